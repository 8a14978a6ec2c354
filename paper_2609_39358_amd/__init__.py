"""MI355X-native hot path of Taliesin (byte-exact KV save / verify / restore).

The compute lives in libtaliesin.so (include/taliesin.h): host C++ for the key
chain and the index, hand-written HIP (gfx950) kernels for save and load.
`paper_2609_39358_amd.taliesin` is the ctypes binding."""
