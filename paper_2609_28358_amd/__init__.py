"""Quantize-once MX convolution (MicroQonv) for MI355X (gfx950).

The product is the C-ABI library libmxconv.so (include/mxconv.h), built from
the hand-written HIP kernels in csrc/.  ``mxconv`` is a thin ctypes binding
with the same entry-point names; PyTorch only supplies device memory and
streams.  There is no CPU fallback: a missing library is an error.
"""
