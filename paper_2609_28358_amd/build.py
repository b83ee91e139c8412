"""Build libmxconv.so (the gfx950 HIP kernels and the C ABI) in-tree.

    python -m paper_2609_28358_amd.build

Every source is compiled with hipcc for gfx950 and linked into
paper_2609_28358_amd/libmxconv.so.  Packed-fp32 instruction selection is
disabled for all device code.
"""
import os
import subprocess
import sys
from concurrent.futures import ThreadPoolExecutor

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
CSRC = os.path.join(HERE, "csrc")
BUILD = os.path.join(ROOT, "_build")
LIB = os.path.join(HERE, "libmxconv.so")
SOURCES = ["quantize.hip", "nvfp.hip", "im2col.hip", "conv_gemm.hip", "conv_lean.hip", "conv_lean_bwd.hip",
           "conv_lean_e4m3_fwd.hip", "conv_lean_e4m3_dg.hip", "conv_lean_e2m1_fwd.hip", "conv_lean_e2m1_dg.hip",
           "conv_lean_nv.hip", "conv_lean_nv68.hip", "conv_lean_fp6.hip", "wgrad_lean.hip", "naive.hip", "netops.hip", "mxconv_abi.cpp"]
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
FLAGS = ["--offload-arch=gfx950", "-O3", "-std=c++17", "-fPIC",
         "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
         "-I" + os.path.join(ROOT, "include")]


def _compile(src):
    out = os.path.join(BUILD, os.path.splitext(src)[0] + ".o")
    cmd = [HIPCC] + FLAGS + ["-x", "hip", "-c", os.path.join(CSRC, src), "-o", out]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"hipcc failed for {src}:\n{r.stderr}")
    return out


def build(verbose=False):
    os.makedirs(BUILD, exist_ok=True)
    srcs = [s for s in SOURCES if os.path.exists(os.path.join(CSRC, s))]
    with ThreadPoolExecutor(max_workers=min(os.cpu_count() or 8, 16, len(srcs))) as ex:
        objs = list(ex.map(_compile, srcs))
    tmp = LIB + ".tmp"
    cmd = [HIPCC, "--offload-arch=gfx950", "-shared", "-fPIC", "-o", tmp] + objs
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"link failed:\n{r.stderr}")
    # a kernel instantiation the host pass dropped shows up as an undefined
    # symbol only when the library is loaded: load it at build time, so such
    # a library is never installed
    import ctypes
    try:
        ctypes.CDLL(tmp)
    except OSError as e:
        raise RuntimeError(f"built library does not load: {e}")
    os.replace(tmp, LIB)
    if verbose:
        print("built", LIB)
    return LIB


if __name__ == "__main__":
    build(verbose=True)
    sys.exit(0)
