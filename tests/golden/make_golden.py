"""Writes tests/golden/micro_record.txt using only the oracle.

A fixed 1-layer micro layout (P=16, H=1, D=32, bf16 -> 1 KiB slabs), fixed
identity and fixed inputs; the file is a regression anchor for the record
format, not an independent pin. Run: python tests/golden/make_golden.py"""
import os
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, os.path.dirname(os.path.dirname(HERE)))

import numpy as np  # noqa: E402

from oracle import taliesin_ref as ref  # noqa: E402


def build():
    lay = ref.Layout(1, 1, 32, 1, 16)
    ns = ref.namespace_digest(b"golden-tenant", b"golden-model", lay)
    toks = np.arange(1000, 1016, dtype="<u4")
    key = ref.block_keys(ns, toks.tobytes(), lay.block_bytes)[0]
    slabs = [bytes((7 * i + 13 * s) & 0xFF for i in range(lay.slab_bytes)) for s in range(2)]
    return ns, key, ref.make_record(lay, ns, key, 3, toks, slabs)


if __name__ == "__main__":
    ns, key, rec = build()
    with open(os.path.join(HERE, "micro_record.txt"), "w") as f:
        f.write("# written by tests/golden/make_golden.py (oracle only)\n")
        f.write("ns %s\nkey %s\n" % (ns.hex(), key.hex()))
        for i in range(0, len(rec), 64):
            f.write(rec[i:i + 64].hex() + "\n")
