"""Builds libtaliesin.so in-tree: host runtime (C++17, g++) + HIP kernels
(hipcc, gfx950 only). Run: python -m paper_2609_39358_amd.build"""
import os
import shutil
import subprocess
import sys

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
INCLUDE = os.path.join(ROOT, "include")
OUT = os.path.join(PKG, "libtaliesin.so")
SABOTAGE_OUT = os.path.join(PKG, "libtaliesin_sabotage.so")  # test-only build with switchable checks
BUILD_DIR = os.path.join(PKG, "_build")

HIP_FLAGS = [
    "-O3", "-fPIC", "-std=c++17", "--offload-arch=gfx950",
    # no packed FP32 instructions anywhere (the kernels do no FP32 math)
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    "-Wall", "-Wno-unused-function",
]
CXX_FLAGS = ["-O2", "-fPIC", "-std=c++17", "-Wall", "-Wextra", "-Wno-unused-parameter"]


def _run(cmd, verbose):
    if verbose:
        print(" ".join(cmd), flush=True)
    r = subprocess.run(cmd, stdout=subprocess.PIPE, stderr=subprocess.STDOUT, text=True)
    if r.returncode != 0:
        sys.stderr.write(r.stdout)
        raise RuntimeError("build step failed: " + " ".join(cmd[:3]))
    return r.stdout


def build(verbose: bool = False, extra_hip_flags=(), out: str = OUT, build_dir: str = BUILD_DIR) -> str:
    """Compile and link libtaliesin.so; extra_hip_flags (e.g. -DTL_BATCH_ROWS=16)
    and out/build_dir allow building a variant next to the default library."""
    hipcc = os.environ.get("HIPCC") or shutil.which("hipcc") or "/opt/rocm/bin/hipcc"
    cxx = os.environ.get("CXX") or shutil.which("g++") or "g++"
    os.makedirs(build_dir, exist_ok=True)
    inc = ["-I", INCLUDE, "-I", CSRC]
    objs = []
    for src in ("ctx.cpp", "sha256.cpp", "file_io.cpp"):
        o = os.path.join(build_dir, src + ".o")
        _run([cxx, *CXX_FLAGS, *inc, "-c", os.path.join(CSRC, src), "-o", o], verbose)
        objs.append(o)
    for src in ("kernels.hip", "chain.hip"):
        o = os.path.join(build_dir, src + ".o")
        _run([hipcc, *HIP_FLAGS, *extra_hip_flags, *inc, "-c", os.path.join(CSRC, src), "-o", o], verbose)
        objs.append(o)
    tmp = out + ".tmp"
    _run([hipcc, "-shared", "-fPIC", "--offload-arch=gfx950", "-o", tmp, *objs], verbose)
    os.replace(tmp, out)
    return out


C_ABI_TEST = os.path.join(PKG, "c_abi_roundtrip")  # test program that uses the C ABI alone


def build_c_abi_test(verbose: bool = False) -> str:
    """A C program (tests/native/c_abi_roundtrip.c) linked against the
    release library and the HIP runtime only: the GPU tests run it to check
    the boundary without the Python binding."""
    cc = os.environ.get("CC") or shutil.which("gcc") or "gcc"
    rocm = os.environ.get("ROCM_PATH", "/opt/rocm")
    tmp = C_ABI_TEST + ".tmp"
    _run([cc, "-O1", "-std=c11", "-Wall", "-D__HIP_PLATFORM_AMD__", "-I", INCLUDE, "-I", os.path.join(rocm, "include"),
          os.path.join(ROOT, "tests", "native", "c_abi_roundtrip.c"), "-o", tmp, "-L", PKG, "-ltaliesin",
          "-L", os.path.join(rocm, "lib"), "-lamdhip64", "-Wl,-rpath,$ORIGIN", "-Wl,-rpath," + os.path.join(rocm, "lib")],
         verbose)
    os.replace(tmp, C_ABI_TEST)
    return C_ABI_TEST


def build_all(verbose: bool = False):
    """The release library, the sabotage build used by the sabotage tests and
    the C-ABI test program."""
    out = build(verbose)
    build(verbose, extra_hip_flags=("-DTL_SABOTAGE",), out=SABOTAGE_OUT,
          build_dir=os.path.join(BUILD_DIR, "sabotage"))
    build_c_abi_test(verbose)
    return out


if __name__ == "__main__":
    print(build_all(verbose=True))
