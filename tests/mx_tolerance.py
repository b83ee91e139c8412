"""Error measure for GEMM outputs checked against the oracle.

Eq. (7) sums exact products of the dequantized block elements; the bound is
the one stated for the path, relative to the sum of absolute products:

    max_i |gpu_i - ref_i| / S_i <= 1e-5,     S_i = sum_k |a_k b_k|

with ref and S computed by the oracle in fp64.  On the GPU every format's
products are exact (FP4 and FP6 pairs on the block-scaled MFMA, FP8 decoded
to bf16 with its E8M0 scale and multiplied on the bf16 matrix cores, NVFP4
decoded to fp16), so only the order of the fp32 additions differs from the
oracle's.  An output with no non-zero product must be exactly zero.

Test infrastructure only.
"""
import numpy as np


def gemm_err(got, ref, sabs, tol=1e-5):
    """Largest |gpu - oracle| / (tol * S) over the outputs (<= 1 passes)."""
    got = np.asarray(got).astype(np.float64)
    zero = sabs == 0
    assert np.all(got[zero] == 0), "outputs with no non-zero products must be exactly 0"
    nz = ~zero
    return float(np.max(np.abs(got[nz] - ref[nz]) / (tol * sabs[nz]))) if nz.any() else 0.0


def rel_err(got, ref, sabs):
    """max |gpu - oracle| / S itself (reported beside the pass/fail ratio)."""
    got = np.asarray(got).astype(np.float64)
    nz = sabs != 0
    return float(np.max(np.abs(got[nz] - ref[nz]) / sabs[nz])) if nz.any() else 0.0
