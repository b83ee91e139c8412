"""The C ABI on the host (no GPU): the library loads, exports every entry
point include/mxconv.h declares, sizes match the stated layouts, and every
argument error is reported before anything is launched.  Calls here either
fail validation or are pure size queries; none reaches a kernel."""
import ctypes
import os
import re

import pytest

import oracle
from paper_2609_28358_amd import mxconv as mx
from paper_2609_28358_amd import synth

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _declared():
    src = open(os.path.join(ROOT, "include", "mxconv.h")).read()
    return sorted(set(re.findall(r"\b(mxconv_\w+)\s*\(", src)))


def test_library_exports_every_declared_symbol():
    L = mx.lib()
    names = _declared()
    assert len(names) >= 12
    for n in names:
        assert hasattr(L, n), n


def test_sizes_match_layout_and_oracle():
    for role in (mx.ACT, mx.WEIGHT):
        for fmt in (mx.E4M3, mx.E2M1, mx.E2M3, mx.E3M2):
            for shape in [(32, 64, 56, 56), (2, 32, 8, 8), (16, 3, 640, 640), (64, 100, 3, 5),
                          (256, 64, 3, 3), (20, 33, 1, 1), (4, 40, 3, 3)]:
                n, c, h, w = shape
                if role == mx.ACT and not (n % 32 == 0 or 32 % n == 0):
                    continue
                slack = 16 if fmt in (mx.E2M3, mx.E3M2) else 0     # FP6 read slack
                if role == mx.ACT and fmt in (mx.E2M3, mx.E3M2) and n < 4:
                    assert mx.codes_bytes(role, fmt, *shape) == 0 and oracle.codes_bytes(role, fmt, *shape) < 0
                    continue
                assert mx.codes_bytes(role, fmt, *shape) == oracle.codes_bytes(role, fmt, *shape) + slack
                assert mx.scales_bytes(role, fmt, *shape) == oracle.scales_bytes(role, fmt, *shape)
    # [N/Bn][H][W][Cp][Bn] codes, [N/Bn][H][W][Cp/32] scales
    assert mx.codes_bytes(mx.ACT, mx.E4M3, 32, 64, 56, 56) == 32 * 64 * 56 * 56
    assert mx.codes_bytes(mx.ACT, mx.E2M1, 16, 3, 640, 640) == 16 * 32 * 640 * 640 // 2
    assert mx.scales_bytes(mx.ACT, mx.E4M3, 16, 3, 640, 640) == 640 * 640
    assert mx.codes_bytes(mx.WEIGHT, mx.E4M3, 20, 33, 3, 3) == 32 * 64 * 9
    assert mx.codes_bytes(mx.ACT, mx.E3M2, 32, 64, 56, 56) == 32 * 64 * 56 * 56 * 3 // 4 + 16


def test_conv_sizes():
    for cv in (synth.conv_dict(32, 64, 64, 56, 56, 3, 1, 1), synth.conv_dict(32, 128, 256, 28, 28, 3, 2, 1),
               dict(n=8, cin=33, cout=20, h=9, w=7, kh=3, kw=2, sh=2, sw=1, ph=1, pw=0)):
        assert mx.out_size(cv) == synth.out_hw(cv) == oracle.conv_out(cv)
        c = mx.conv_struct(cv)
        for fmt in (0, 1, 2, 3):
            slack = 16 if fmt >= 2 else 0
            assert mx.lib().mxconv_im2col_codes_bytes(ctypes.byref(c), fmt) == oracle.load().o_im2col_codes_bytes(
                oracle._ptr(oracle._conv_params(cv)), fmt) + slack
            if fmt < 2 or cv["n"] % 32 == 0:
                assert mx.wgrad_workspace_bytes(cv, fmt if fmt != 3 else mx.pair(1, 3)) > 0


P = ctypes.c_void_p
GOOD = P(0x10000)        # 16-byte aligned, never dereferenced: validation fails first
ODD = P(0x10001)


def test_quantize_errors():
    L = mx.lib()
    q = L.mxconv_quantize
    assert q(None, 0, 0, 0, 0, 32, 32, 4, 4, GOOD, GOOD, None) == -1
    assert q(GOOD, 0, 0, 0, 0, 32, 32, 4, 4, None, GOOD, None) == -1
    assert q(GOOD, 2, 0, 0, 0, 32, 32, 4, 4, GOOD, GOOD, None) == -2     # dtype
    assert q(GOOD, 0, 3, 0, 0, 32, 32, 4, 4, GOOD, GOOD, None) == -2     # layout
    assert q(GOOD, 0, 0, 2, 0, 32, 32, 4, 4, GOOD, GOOD, None) == -2     # role
    assert q(GOOD, 0, 0, 0, 4, 32, 32, 4, 4, GOOD, GOOD, None) == -2     # fmt
    assert q(GOOD, 0, 0, 0, mx.pair(1, 3), 32, 32, 4, 4, GOOD, GOOD, None) == -2   # no pairs here
    assert q(GOOD, 0, 0, 0, 2, 2, 32, 4, 4, GOOD, GOOD, None) == -3      # FP6 with two samples
    assert q(GOOD, 0, 0, 0, 3, 4, 32, 4, 4, GOOD, ODD, None) == -4       # FP6 with four: accepted
    assert q(GOOD, 0, 2, 1, 0, 32, 32, 4, 4, GOOD, GOOD, None) == -2     # CBF weights
    assert q(GOOD, 0, 0, 0, 0, 0, 32, 4, 4, GOOD, GOOD, None) == -2      # empty
    assert q(GOOD, 0, 0, 0, 0, 32, -1, 4, 4, GOOD, GOOD, None) == -2
    assert q(GOOD, 0, 0, 0, 0, 48, 32, 4, 4, GOOD, GOOD, None) == -3     # batch rule
    assert q(GOOD, 0, 0, 0, 0, 3, 32, 4, 4, GOOD, GOOD, None) == -3
    assert q(GOOD, 0, 0, 0, 1, 1, 32, 4, 4, GOOD, GOOD, None) == -3      # E2M1 with one sample
    assert q(ODD, 0, 0, 0, 0, 32, 32, 4, 4, GOOD, GOOD, None) == -4
    assert q(GOOD, 0, 0, 0, 0, 32, 32, 4, 4, GOOD, ODD, None) == -4
    # MXC_KEEP_PAD: a flag on layout; the layout under it is still checked
    hdr = open(os.path.join(ROOT, "include", "mxconv.h")).read()
    assert int(re.search(r"#define MXC_KEEP_PAD (0x[0-9a-fA-F]+)", hdr).group(1), 16) == mx.KEEP_PAD
    assert q(GOOD, 0, mx.KEEP_PAD | 0, 0, 0, 32, 3, 4, 4, GOOD, ODD, None) == -4   # accepted up to alignment
    assert q(GOOD, 0, mx.KEEP_PAD | 3, 0, 0, 32, 3, 4, 4, GOOD, GOOD, None) == -2
    assert q(GOOD, 0, 0x200, 0, 0, 32, 3, 4, 4, GOOD, GOOD, None) == -2



def test_gemm_and_im2col_errors():
    L = mx.lib()
    cv = mx.conv_struct(synth.conv_dict(32, 64, 64, 8, 8, 3, 1, 1))
    r = ctypes.byref(cv)
    for fn in (L.mxconv_fwd, L.mxconv_dgrad):
        assert fn(None, 0, GOOD, GOOD, GOOD, GOOD, GOOD, 0, None) == -1
        assert fn(r, 0, GOOD, None, GOOD, GOOD, GOOD, 0, None) == -1
        assert fn(r, 5, GOOD, GOOD, GOOD, GOOD, GOOD, 0, None) == -2
        assert fn(r, 0, GOOD, GOOD, GOOD, GOOD, GOOD, 1, None) == -2     # NHWC output not offered
        assert fn(r, 0, ODD, GOOD, GOOD, GOOD, GOOD, 0, None) == -4
        assert fn(r, 0, GOOD, GOOD, GOOD, GOOD, ODD, 2, None) == -4
    assert L.mxconv_im2col_cbf(r, 0, GOOD, None, GOOD, GOOD, None) == -1
    assert L.mxconv_im2col_cbf(r, 0, GOOD, GOOD, ODD, GOOD, None) == -4
    # a layer large enough to split the weight-gradient contraction: it needs a
    # workspace, so these calls must fail validation (never reach a kernel)
    big = synth.conv_dict(32, 64, 64, 56, 56, 3, 1, 1)
    rb = ctypes.byref(mx.conv_struct(big))
    need = mx.wgrad_workspace_bytes(big, 0)
    assert need > 0
    assert L.mxconv_wgrad(rb, 0, GOOD, GOOD, GOOD, GOOD, GOOD, None, 0, None) == -6
    assert L.mxconv_wgrad(rb, 0, GOOD, GOOD, GOOD, GOOD, GOOD, GOOD, need - 1, None) == -6
    assert L.mxconv_wgrad(rb, 0, GOOD, GOOD, GOOD, GOOD, GOOD, ODD, need, None) == -4
    bad = [dict(n=32, cin=64, cout=64, h=8, w=8, kh=3, kw=3, sh=0, sw=1, ph=1, pw=1),
           dict(n=32, cin=64, cout=64, h=8, w=8, kh=3, kw=3, sh=1, sw=1, ph=-1, pw=1)]
    for b in bad:
        assert L.mxconv_fwd(ctypes.byref(mx.conv_struct(b)), 0, GOOD, GOOD, GOOD, GOOD, GOOD, 0, None) == -2
    small = mx.conv_struct(dict(n=32, cin=64, cout=64, h=2, w=8, kh=5, kw=3, sh=1, sw=1, ph=1, pw=1))
    assert L.mxconv_fwd(ctypes.byref(small), 0, GOOD, GOOD, GOOD, GOOD, GOOD, 0, None) == -3
    odd_batch = mx.conv_struct(synth.conv_dict(24, 64, 64, 8, 8, 3, 1, 1))
    assert L.mxconv_dgrad(ctypes.byref(odd_batch), 0, GOOD, GOOD, GOOD, GOOD, GOOD, 0, None) == -3


def test_strerror_covers_codes():
    for rc in range(0, -7, -1):
        assert mx.strerror(rc) and mx.strerror(rc) != "unknown error"
    assert mx.strerror(-99) == "unknown error"


def test_naive_sizes():
    L = mx.lib()
    # line matrices: lines x (length rounded up to 64), one scale per 32
    assert L.mxconv_naive_codes_bytes(100, 576, mx.E4M3) == 100 * 576
    assert L.mxconv_naive_codes_bytes(100, 27, mx.E4M3) == 100 * 64
    assert L.mxconv_naive_codes_bytes(100, 65, mx.E2M1) == 100 * 128 // 2
    assert L.mxconv_naive_scales_bytes(100, 65) == 100 * 4
    assert L.mxconv_naive_codes_bytes(0, 5, mx.E4M3) == 0
    assert L.mxconv_naive_codes_bytes(5, 5, 2) == 0
    assert L.mxconv_naive_scales_bytes(5, -1) == 0


def test_naive_errors():
    L = mx.lib()
    c = ctypes.byref(mx.conv_struct(synth.conv_dict(32, 64, 64, 8, 8, 3, 1, 1)))
    bad = ctypes.byref(mx.conv_struct(synth.conv_dict(48, 64, 64, 8, 8, 3, 1, 1)))   # batch rule
    assert L.mxconv_naive_im2col_f32(None, GOOD, GOOD, None) == -1
    assert L.mxconv_naive_im2col_f32(c, GOOD, None, None) == -1
    assert L.mxconv_naive_im2col_f32(bad, GOOD, GOOD, None) == -3
    assert L.mxconv_naive_im2col_f32(c, ODD, GOOD, None) == -4
    q = L.mxconv_naive_quantize_1d
    assert q(None, 4, 4, 0, 0, GOOD, GOOD, None) == -1
    assert q(GOOD, 0, 4, 0, 0, GOOD, GOOD, None) == -2
    assert q(GOOD, 4, 4, 2, 0, GOOD, GOOD, None) == -2
    assert q(GOOD, 4, 4, 0, 5, GOOD, GOOD, None) == -2
    assert q(GOOD, 4, 4, 1, 0, GOOD, ODD, None) == -4
    for fn, extra in ((L.mxconv_naive_fwd, ()), (L.mxconv_naive_dgrad, (GOOD,)), (L.mxconv_naive_wgrad, ())):
        args = [GOOD] * 4 + list(extra) + [GOOD]
        assert fn(None, 0, *args, None) == -1
        assert fn(c, 0, None, *args[1:], None) == -1
        assert fn(c, 3, *args, None) == -2
        assert fn(bad, 0, *args, None) == -3
        assert fn(c, 0, *args[:-1], ODD, None) == -4


def test_fused_errors():
    """mxconv_fwd_quant / mxconv_dgrad_quant: every call below fails validation."""
    L = mx.lib()
    c = ctypes.byref(mx.conv_struct(synth.conv_dict(32, 64, 64, 8, 8, 3, 1, 1)))
    c16 = ctypes.byref(mx.conv_struct(synth.conv_dict(16, 64, 64, 8, 8, 3, 1, 1)))       # batch block 16
    c5 = ctypes.byref(mx.conv_struct(synth.conv_dict(32, 64, 64, 8, 8, 5, 1, 2)))        # kernel width 5
    c21 = ctypes.byref(mx.conv_struct(dict(n=32, cin=64, cout=64, h=8, w=8, kh=3, kw=3, sh=2, sw=1, ph=1, pw=1)))
    f = L.mxconv_fwd_quant          # (cv, fmt, wc, ws, xc, xs, fn, out_fmt, yc, ys, y_act, stream)
    assert f(None, 0, GOOD, GOOD, GOOD, GOOD, 0, 0, GOOD, GOOD, None, None) == -1
    assert f(c, 0, GOOD, GOOD, GOOD, GOOD, 0, 0, None, GOOD, None, None) == -1
    assert f(c, 0, GOOD, GOOD, GOOD, None, 0, 0, GOOD, GOOD, None, None) == -1
    assert f(c, 0, GOOD, GOOD, GOOD, GOOD, 3, 0, GOOD, GOOD, None, None) == -2      # activation
    assert f(c, 0, GOOD, GOOD, GOOD, GOOD, -1, 0, GOOD, GOOD, None, None) == -2
    assert f(c, 0, GOOD, GOOD, GOOD, GOOD, 0, 4, GOOD, GOOD, None, None) == -2      # output format
    assert f(c, mx.pair(1, 3), GOOD, GOOD, GOOD, GOOD, 0, 3, ODD, GOOD, None, None) == -4   # MicroQonv+ accepted
    assert f(c, mx.pair(3, 3), GOOD, GOOD, GOOD, GOOD, 0, 3, GOOD, GOOD, None, None) == -2
    assert f(c, 7, GOOD, GOOD, GOOD, GOOD, 0, 0, GOOD, GOOD, None, None) == -2      # operand format
    assert f(c16, 0, GOOD, GOOD, GOOD, GOOD, 0, 0, GOOD, GOOD, None, None) == -3
    assert f(c5, 0, GOOD, GOOD, GOOD, GOOD, 0, 0, GOOD, GOOD, None, None) == -3
    assert f(c, 0, GOOD, GOOD, GOOD, GOOD, 0, 0, ODD, GOOD, None, None) == -4
    assert f(c, 0, GOOD, GOOD, GOOD, GOOD, 2, 1, GOOD, GOOD, ODD, None) == -4
    d = L.mxconv_dgrad_quant        # (cv, fmt, wc, ws, gc, gs, fn, z, out_fmt, gxc, gxs, gx_act, stream)
    assert d(None, 0, GOOD, GOOD, GOOD, GOOD, 0, None, 0, GOOD, GOOD, None, None) == -1
    assert d(c, 0, GOOD, GOOD, GOOD, GOOD, 1, None, 0, GOOD, GOOD, None, None) == -1   # ReLU needs z
    assert d(c, 0, GOOD, GOOD, GOOD, GOOD, 2, None, 0, GOOD, GOOD, None, None) == -1   # SiLU needs z
    assert d(c, 0, GOOD, GOOD, GOOD, GOOD, 0, None, 0, None, GOOD, None, None) == -1
    assert d(c, 0, GOOD, GOOD, GOOD, GOOD, 4, GOOD, 0, GOOD, GOOD, None, None) == -2
    assert d(c, 0, GOOD, GOOD, GOOD, GOOD, 1, GOOD, 5, GOOD, GOOD, None, None) == -2
    assert d(c, 2, GOOD, GOOD, GOOD, GOOD, 1, GOOD, 2, GOOD, GOOD, ODD, None) == -4
    assert d(c21, 0, GOOD, GOOD, GOOD, GOOD, 0, None, 0, GOOD, GOOD, None, None) == -3  # stride 2x1
    assert d(c16, 0, GOOD, GOOD, GOOD, GOOD, 1, GOOD, 0, GOOD, GOOD, None, None) == -3
    assert d(c, 0, GOOD, GOOD, GOOD, GOOD, 1, ODD, 0, GOOD, GOOD, None, None) == -4
    assert d(c, 0, GOOD, GOOD, GOOD, GOOD, 0, None, 0, GOOD, GOOD, ODD, None) == -4


def test_fp6_format_pairs():
    """The GEMM entry points take one format or MXC_PAIR(first, second); only
    the pairs the kernels are built for pass validation (misaligned outputs
    then stop the accepted ones before any launch)."""
    L = mx.lib()
    r = ctypes.byref(mx.conv_struct(synth.conv_dict(32, 64, 64, 8, 8, 3, 1, 1)))
    accepted = [0, 1, 2, mx.pair(1, 3), 0x10 | (2 << 2) | 2]
    refused = [3, mx.pair(3, 3), mx.pair(0, 1), mx.pair(1, 2), mx.pair(3, 1), 0x20, 0x10 | 15, 4, -1]
    for fn in (L.mxconv_fwd, L.mxconv_dgrad):
        for f in accepted:
            assert fn(r, f, GOOD, GOOD, GOOD, GOOD, ODD, 0, None) == -4, f
        for f in refused:
            assert fn(r, f, GOOD, GOOD, GOOD, GOOD, GOOD, 0, None) == -2, f
    for f in accepted:     # a workspace large enough for any split count, so alignment is what fails
        assert L.mxconv_wgrad(r, f, GOOD, GOOD, GOOD, GOOD, ODD, GOOD, 1 << 40, None) == -4, f
    for f in refused:
        assert L.mxconv_wgrad(r, f, GOOD, GOOD, GOOD, GOOD, GOOD, None, 0, None) == -2, f
    # im2col and the size queries take a single format
    assert L.mxconv_im2col_cbf(r, mx.pair(1, 3), GOOD, GOOD, GOOD, GOOD, None) == -2
    assert L.mxconv_im2col_codes_bytes(r, mx.pair(1, 3)) == 0
    # FP6 runs only on the batch-block-32 kernels: other layers are refused
    # (after validation, with nothing launched)
    for cvd in (synth.conv_dict(32, 64, 64, 8, 8, 5, 1, 2), synth.conv_dict(16, 64, 64, 8, 8, 3, 1, 1)):
        rr = ctypes.byref(mx.conv_struct(cvd))
        for f in (2, mx.pair(1, 3)):
            assert L.mxconv_fwd(rr, f, GOOD, GOOD, GOOD, GOOD, GOOD, 0, None) == -3
            assert L.mxconv_dgrad(rr, f, GOOD, GOOD, GOOD, GOOD, GOOD, 0, None) == -3
    r16 = ctypes.byref(mx.conv_struct(synth.conv_dict(16, 64, 64, 8, 8, 3, 1, 1)))
    assert L.mxconv_wgrad(r16, 2, GOOD, GOOD, GOOD, GOOD, GOOD, None, 0, None) == -3
    # the naive comparator stays MXFP8 / MXFP4
    assert L.mxconv_naive_fwd(r, 2, GOOD, GOOD, GOOD, GOOD, GOOD, None) == -2


def test_quantize_sr_errors():
    L = mx.lib()
    q = L.mxconv_quantize_sr      # (src, dtype, layout, role, fmt, n, c, h, w, seed, codes, scales, stream)
    assert q(None, 0, 0, 0, 0, 32, 32, 4, 4, 1, GOOD, GOOD, None) == -1
    assert q(GOOD, 0, 0, 0, 0, 32, 32, 4, 4, 1, GOOD, None, None) == -1
    assert q(GOOD, 2, 0, 0, 0, 32, 32, 4, 4, 1, GOOD, GOOD, None) == -2
    assert q(GOOD, 0, 2, 1, 0, 32, 32, 4, 4, 1, GOOD, GOOD, None) == -2
    assert q(GOOD, 0, 0, 0, 4, 32, 32, 4, 4, 1, GOOD, GOOD, None) == -2
    assert q(GOOD, 0, 0, 0, 0, 48, 32, 4, 4, 1, GOOD, GOOD, None) == -3
    assert q(GOOD, 0, 0, 0, 3, 2, 32, 4, 4, 1, GOOD, GOOD, None) == -3
    assert q(GOOD, 0, 0, 0, 3, 32, 32, 4, 4, 2 ** 64 - 1, ODD, GOOD, None) == -4


def test_nvfp_errors():
    L = mx.lib()
    q = L.mxconv_nvfp_quantize   # (src, dtype, layout, role, fmt, n, c, h, w, codes, scales, t, ws, ws_bytes, stream)
    wsb = L.mxconv_nvfp_workspace_bytes()
    assert wsb >= 1024 * 4
    assert L.mxconv_nvfp_scales_bytes(0, 1, 64, 40, 3, 3) == oracle.load().o_nvfp_scales_bytes(0, 1, 64, 40, 3, 3)
    assert L.mxconv_nvfp_scales_bytes(0, 1, 4, 32, 1, 1) == 0                       # Bn = 4: no 8x8 blocks
    assert q(None, 0, 2, 0, 1, 32, 32, 4, 4, GOOD, GOOD, GOOD, GOOD, wsb, None) == -1
    assert q(GOOD, 0, 2, 0, 1, 32, 32, 4, 4, GOOD, GOOD, None, GOOD, wsb, None) == -1
    assert q(GOOD, 0, 2, 0, 9, 32, 32, 4, 4, GOOD, GOOD, GOOD, GOOD, wsb, None) == -2
    assert q(GOOD, 0, 1, 0, 1, 32, 32, 4, 4, GOOD, GOOD, GOOD, GOOD, wsb, None) == -3   # NHWC: not on the GPU
    assert q(GOOD, 0, 2, 0, 1, 16, 32, 4, 4, GOOD, GOOD, GOOD, GOOD, wsb, None) == -3   # batch block 16
    assert q(GOOD, 0, 2, 0, 1, 32, 32, 4, 4, GOOD, GOOD, GOOD, None, 0, None) == -6
    assert q(GOOD, 0, 2, 0, 1, 32, 32, 4, 4, GOOD, GOOD, GOOD, GOOD, wsb - 1, None) == -6
    assert q(GOOD, 0, 2, 0, 1, 32, 32, 4, 4, GOOD, GOOD, ODD, GOOD, wsb, None) == -4


def test_quantize_multi_errors():
    L = mx.lib()
    J = mx.MxcQJob

    def job(src=0x10000, dtype=0, layout=2, role=0, fmt=0, n=32, c=32, h=4, w=4, codes=0x10000, scales=0x10000):
        return J(src, dtype, layout, role, fmt, n, c, h, w, codes, scales)

    def call(*jobs):
        arr = (J * max(1, len(jobs)))(*jobs)
        return L.mxconv_quantize_multi(len(jobs), arr, None)

    assert L.mxconv_quantize_multi(mx.QMULTI_MAX + 1, None, None) == -2
    assert L.mxconv_quantize_multi(-1, None, None) == -2
    assert L.mxconv_quantize_multi(2, None, None) == -1
    assert L.mxconv_quantize_multi(0, None, None) == 0                  # nothing to do
    # every job is validated before anything is launched
    assert call(job(), job(src=0)) == -1
    assert call(job(), job(fmt=7)) == -2
    assert call(job(), job(layout=2, role=1)) == -2                     # CBF weights
    assert call(job(), job(n=48)) == -3
    assert call(job(), job(codes=0x10001)) == -4
    # the optional im2col output: NULL outputs, a layer that does not match its
    # tensor, weights, a bad layer, misaligned outputs
    cv = mx.conv_struct(synth.conv_dict(32, 32, 16, 4, 4, 3, 1, 1))

    def colj(conv=cv, cc=0x10000, cs=0x10000, **kw):
        j = job(**kw)
        j.conv = ctypes.pointer(conv)
        j.col_codes, j.col_scales = cc, cs
        return j

    assert call(job(), colj(cc=0)) == -1
    assert call(job(), colj(cs=0)) == -1
    assert call(job(), colj(c=64)) == -3                               # conv.cin != c
    assert call(job(), colj(h=5)) == -3
    assert call(job(), colj(layout=0, role=1)) == -3                   # weights have no im2col
    bad = mx.conv_struct(synth.conv_dict(32, 32, 16, 4, 4, 3, 1, 1))
    bad.sh = 0
    assert call(job(), colj(conv=bad)) == -2
    big = mx.conv_struct(synth.conv_dict(32, 32, 16, 4, 4, 7, 1, 0))  # kernel larger than the padded input
    assert call(job(), colj(conv=big)) == -3
    assert call(job(), colj(cc=0x10008)) == -4
    assert call(job(), colj(cs=0x10001)) == -4


def test_nvfp_gemm_errors():
    L = mx.lib()
    r = ctypes.byref(mx.conv_struct(synth.conv_dict(32, 64, 64, 8, 8, 3, 1, 1)))
    r5 = ctypes.byref(mx.conv_struct(synth.conv_dict(32, 64, 64, 8, 8, 5, 1, 2)))
    for fn in (L.mxconv_nvfp_fwd, L.mxconv_nvfp_dgrad):   # (cv, fmt, wc, ws, wt, xc, xs, xt, out, layout, stream)
        assert fn(None, 1, GOOD, GOOD, GOOD, GOOD, GOOD, GOOD, GOOD, 0, None) == -1
        assert fn(r, 1, GOOD, GOOD, None, GOOD, GOOD, GOOD, GOOD, 0, None) == -1
        assert fn(r, 3, GOOD, GOOD, GOOD, GOOD, GOOD, GOOD, GOOD, 0, None) == -2      # E3M2 x E3M2
        assert fn(r, 0x14, GOOD, GOOD, GOOD, GOOD, GOOD, GOOD, GOOD, 0, None) == -2   # FP4 x FP8
        assert fn(r, 1, GOOD, GOOD, GOOD, GOOD, GOOD, GOOD, GOOD, 1, None) == -2      # NHWC output
        assert fn(r, 1, GOOD, GOOD, GOOD, GOOD, GOOD, ODD, GOOD, 0, None) == -4
        assert fn(r5, 1, GOOD, GOOD, GOOD, GOOD, GOOD, GOOD, GOOD, 0, None) == -3     # kernel width 5
    w = L.mxconv_nvfp_wgrad      # (cv, fmt, gc, gs, gt, xc, xs, xt, gw, ws, ws_bytes, stream)
    assert w(r, 1, GOOD, GOOD, GOOD, GOOD, GOOD, None, GOOD, GOOD, 1 << 30, None) == -1
    assert w(r, 3, GOOD, GOOD, GOOD, GOOD, GOOD, GOOD, GOOD, GOOD, 1 << 30, None) == -2   # E3M2 x E3M2
    assert w(r, 0x12, GOOD, GOOD, GOOD, GOOD, GOOD, GOOD, GOOD, GOOD, 1 << 30, None) == -2  # FP8 x E2M3
    big = ctypes.byref(mx.conv_struct(synth.conv_dict(32, 64, 64, 56, 56, 3, 1, 1)))
    assert w(big, 1, GOOD, GOOD, GOOD, GOOD, GOOD, GOOD, GOOD, None, 0, None) == -6
    r16 = ctypes.byref(mx.conv_struct(synth.conv_dict(16, 64, 64, 8, 8, 3, 1, 1)))
    assert w(r16, 1, GOOD, GOOD, GOOD, GOOD, GOOD, GOOD, GOOD, GOOD, 1 << 30, None) == -3


def test_wgrad_reduce_multi_errors():
    L = mx.lib()
    cv = mx.conv_struct(synth.conv_dict(32, 64, 64, 56, 56, 3, 1, 1))        # needs a split-K workspace
    need = L.mxconv_wgrad_workspace_bytes(ctypes.byref(cv), 0)
    assert need > 0

    def job(conv=cv, fmt=0, ws=0x10000, wsb=None, gw=0x10000):
        return mx.MxcWJob(ctypes.pointer(conv) if conv is not None else None, fmt, ws, need if wsb is None else wsb, gw)

    def call(*jobs):
        arr = (mx.MxcWJob * max(1, len(jobs)))(*jobs)
        return L.mxconv_wgrad_reduce_multi(len(jobs), arr, None)

    assert L.mxconv_wgrad_reduce_multi(mx.WREDUCE_MAX + 1, None, None) == -2
    assert L.mxconv_wgrad_reduce_multi(-1, None, None) == -2
    assert L.mxconv_wgrad_reduce_multi(1, None, None) == -1
    assert L.mxconv_wgrad_reduce_multi(0, None, None) == 0
    assert call(job(), job(conv=None)) == -1
    assert call(job(), job(gw=0)) == -1
    assert call(job(), job(fmt=9)) == -2
    assert call(job(), job(ws=0)) == -6
    assert call(job(), job(wsb=need - 1)) == -6
    assert call(job(), job(gw=0x10004)) == -4
    assert call(job(), job(ws=0x10008)) == -4
    r = ctypes.byref(cv)
    assert L.mxconv_wgrad_deferred(r, 0, GOOD, GOOD, GOOD, GOOD, GOOD, None, 0, None) == -6
    assert L.mxconv_wgrad_deferred(None, 0, GOOD, GOOD, GOOD, GOOD, GOOD, GOOD, need, None) == -1


def test_size_limits():
    """Geometries past the 32-bit block and pixel indices the kernels use are
    refused on the host; the largest admitted sizes are still computed."""
    L = mx.lib()
    # activation blocks (n / Bn) * h * w * (Cp / 32) must stay below 2^31
    assert mx.codes_bytes(mx.ACT, mx.E4M3, 32, 32, 46340, 46340) == 46340 * 46340 * 1024
    assert mx.codes_bytes(mx.ACT, mx.E4M3, 32, 32, 46341, 46341) == 0
    assert mx.scales_bytes(mx.ACT, mx.E4M3, 32, 32, 46341, 46341) == 0
    assert L.mxconv_quantize(GOOD, 0, 2, 0, 0, 32, 32, 46341, 46341, GOOD, GOOD, None) == -3
    # the explicit im2col indexes taps with 16 bits, alone or asked for by a quantize job
    big = mx.conv_struct(synth.conv_dict(32, 32, 32, 300, 300, 257, 1, 128))      # 66049 taps
    assert L.mxconv_im2col_cbf(ctypes.byref(big), 0, GOOD, GOOD, GOOD, GOOD, None) == -3
    j = mx.MxcQJob(0x10000, 0, 2, 0, 0, 32, 32, 300, 300, 0x10000, 0x10000)
    j.conv = ctypes.pointer(big)
    j.col_codes, j.col_scales = 0x10000, 0x10000
    assert L.mxconv_quantize_multi(1, (mx.MxcQJob * 1)(j), None) == -3
    ok = mx.conv_struct(synth.conv_dict(32, 32, 32, 300, 300, 255, 1, 127))       # 65025 taps
    assert L.mxconv_im2col_codes_bytes(ctypes.byref(ok), 0) > 0


def test_backward_errors():
    L = mx.lib()
    cv = mx.conv_struct(synth.conv_dict(32, 64, 64, 56, 56, 3, 1, 1))        # needs a split-K workspace
    r = ctypes.byref(cv)
    need = L.mxconv_wgrad_workspace_bytes(r, 0)
    assert need > 0

    def call(conv=r, fmt=0, gx=GOOD, layout=mx.CBF, gw=GOOD, ws=GOOD, wsb=need, deferred=0, x=GOOD):
        return L.mxconv_backward(conv, fmt, GOOD, GOOD, GOOD, GOOD, x, GOOD, gx, layout, gw, ws, wsb, deferred, None)

    assert call(conv=None) == -1
    assert call(gx=None) == -1
    assert call(gw=None) == -1
    assert call(x=None) == -1
    assert call(layout=7) == -2
    assert call(deferred=2) == -2
    assert call(fmt=9) == -2
    # a mixed pair would make G_Y one format for the input gradient and the
    # other for the weight gradient: refused, while a pair of equal halves
    # passes the format check (and reaches the workspace check here)
    assert call(fmt=mx.pair(mx.E2M1, mx.E3M2)) == -2
    assert call(fmt=mx.pair(mx.E2M1, mx.E2M1), ws=None) == -6
    assert call(ws=None) == -6
    assert call(wsb=need - 1) == -6
    assert call(gw=0x10004) == -4
    assert call(ws=0x10008) == -4
    assert call(x=0x10002) == -4
