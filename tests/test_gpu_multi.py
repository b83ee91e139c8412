"""mxconv_quantize_multi: several quantizations in one call give exactly the
codes and scales of the single calls (and of the oracle), whatever mix of
source kinds, formats and source types the jobs have; a job outside the
one-launch kinds (an NCHW activation) is quantized by its own launch."""
import numpy as np
import pytest
import torch

import oracle
from paper_2609_28358_amd import synth

pytestmark = pytest.mark.gpu

DEV = "cuda:0"


@pytest.fixture(scope="module")
def mx():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2609_28358_amd import mxconv
    mxconv.lib()
    return mxconv


def _jobs(mx):
    x = synth.silu_normal((32, 70, 9, 7), 3)
    x2 = synth.silu_normal((64, 32, 5, 5), 4)
    w = synth.kaiming(64, 70, 3, 3, seed=5)
    w2 = synth.kaiming(20, 48, 1, 1, seed=6)
    xn = synth.normal((16, 40, 4, 6), 1.0, 7)
    return [
        (synth.nchw_to_cbf(x, 32).to(DEV), mx.ACT, 0, mx.CBF, tuple(x.shape), x),
        (w.to(DEV), mx.WEIGHT, 0, mx.NCHW, tuple(w.shape), w),
        (synth.nchw_to_cbf(x2, 32).to(DEV).to(torch.bfloat16), mx.ACT, 3, mx.CBF, tuple(x2.shape),
         x2.to(torch.bfloat16).float()),
        (w2.to(DEV), mx.WEIGHT, 1, mx.NCHW, tuple(w2.shape), w2),
        (xn.to(DEV), mx.ACT, 2, mx.NCHW, tuple(xn.shape), xn),            # its own launch
        (w2.to(DEV).to(torch.bfloat16), mx.WEIGHT, 2, mx.NCHW, tuple(w2.shape), w2.to(torch.bfloat16).float()),
    ]


def test_multi_matches_single_calls_and_oracle(mx):
    jobs = _jobs(mx)
    outs = mx.quantize_multi([(s, r, f, l, sh, None) for s, r, f, l, sh, _ in jobs])
    singles = [mx.quantize(s, r, f, layout=l, shape=sh) for s, r, f, l, sh, _ in jobs]
    torch.cuda.synchronize()
    for (s, r, f, l, sh, ref), o, one in zip(jobs, outs, singles):
        assert torch.equal(o.codes, one.codes) and torch.equal(o.scales, one.scales)
        rc, rs = oracle.quantize(ref.numpy(), oracle.NCHW, r, f, *sh)
        assert np.array_equal(o.scales.cpu().numpy(), rs)
        assert np.array_equal(o.codes.cpu().numpy()[:len(rc)], rc)


def test_multi_layer_operands_full_size(mx):
    """X and W of each benchmark layer, one call per layer, both formats."""
    for li, (name, cv) in enumerate(synth.SWEEP_LAYERS):
        x, w, _ = synth.layer_inputs(cv, 1000 + li, kind="sweep")
        xd, wd = synth.nchw_to_cbf(x, 32).to(DEV), w.to(DEV)
        for fmt in (0, 1):
            qx, qw = mx.quantize_multi([(xd, mx.ACT, fmt, mx.CBF, tuple(x.shape), None),
                                        (wd, mx.WEIGHT, fmt, mx.NCHW, tuple(w.shape), None)])
            sx = mx.quantize(xd, mx.ACT, fmt, layout=mx.CBF, shape=tuple(x.shape))
            sw = mx.quantize(wd, mx.WEIGHT, fmt)
            torch.cuda.synchronize()
            assert torch.equal(qx.codes, sx.codes) and torch.equal(qx.scales, sx.scales)
            assert torch.equal(qw.codes, sw.codes) and torch.equal(qw.scales, sw.scales)


# ------------------------------------------------------------------ with the im2col output
def _col_buffers(mx, cv, fmt):
    import ctypes
    c = mx.conv_struct(cv)
    nb = mx.lib().mxconv_im2col_codes_bytes(ctypes.byref(c), fmt)
    ns = mx.lib().mxconv_im2col_scales_bytes(ctypes.byref(c), fmt)
    # garbage first: every byte must be written by the call
    return (torch.full((nb,), 0xAB, dtype=torch.uint8, device=DEV),
            torch.full((ns,), 0xCD, dtype=torch.uint8, device=DEV))


def _explicit_im2col(mx, cv, fmt, q):
    import ctypes
    cc, cs = _col_buffers(mx, cv, fmt)
    c = mx.conv_struct(cv)
    rc = mx.lib().mxconv_im2col_cbf(ctypes.byref(c), fmt, mx._ptr(q.codes), mx._ptr(q.scales), mx._ptr(cc),
                                    mx._ptr(cs), mx._stream(None))
    assert rc == 0
    return cc, cs


COL_CASES = [
    # (conv, fmt, source kind): fused in the quantizer ...
    (synth.conv_dict(32, 64, 64, 12, 10, 3, 1, 1), 0, "cbf"),
    (synth.conv_dict(32, 64, 64, 12, 10, 3, 1, 1), 1, "cbf"),
    (synth.conv_dict(64, 70, 32, 9, 7, 3, 2, 1), 0, "cbf"),          # stride 2, ragged channels, 2 groups
    (synth.conv_dict(32, 40, 16, 11, 9, 5, 2, 2), 1, "cbf_bf16"),    # 5x5 stride 2, bf16 source
    (synth.conv_dict(32, 96, 48, 7, 8, 1, 1, 0), 0, "cbf"),          # 1x1
    (dict(n=32, cin=33, cout=20, h=9, w=7, kh=3, kw=2, sh=2, sw=1, ph=1, pw=0), 1, "cbf"),
    (synth.conv_dict(32, 32, 32, 6, 6, 2, 2, 0), 0, "cbf"),          # even kernel, no padding
    # ... or an im2col launch of its own after the quantization
    (synth.conv_dict(32, 64, 32, 8, 8, 3, 1, 1), 2, "cbf"),          # FP6 activation
    (synth.conv_dict(32, 32, 32, 6, 6, 1, 1, 1), 0, "cbf"),          # output larger than the input
    (synth.conv_dict(16, 40, 32, 7, 5, 3, 1, 1), 0, "nchw"),         # batch block 16, NCHW source
]


@pytest.mark.parametrize("case", COL_CASES, ids=lambda c: f"k{c[0]['kh']}{c[0]['kw']}s{c[0]['sh']}{c[0]['sw']}"
                         f"p{c[0]['ph']}{c[0]['pw']}_c{c[0]['cin']}_f{c[1]}_{c[2]}")
def test_multi_im2col_output(mx, case):
    """The im2col a job asks for equals the explicit im2col of its codes and
    the oracle's im2col of the oracle's codes, bit for bit, with the codes
    unchanged; the layer's weights ride in the same call."""
    cv, fmt, kind = case
    x, w, _ = synth.layer_inputs(cv, 77, kind="sweep")
    xs = tuple(x.shape)
    if kind == "nchw":
        src, layout, ref = x.to(DEV), mx.NCHW, x
    else:
        src = synth.nchw_to_cbf(x, synth.batch_block(cv["n"])).to(DEV)
        ref = x
        if kind == "cbf_bf16":
            src, ref = src.to(torch.bfloat16), x.to(torch.bfloat16).float()
        layout = mx.CBF
    cc, cs = _col_buffers(mx, cv, fmt)
    for rep in range(2):                                        # a second call over the same buffers
        qx, qw = mx.quantize_multi([(src, mx.ACT, fmt, layout, xs, None, (cv, cc, cs)),
                                    (w.to(DEV), mx.WEIGHT, fmt, mx.NCHW, tuple(w.shape), None)])
        torch.cuda.synchronize()
        ec, es = _explicit_im2col(mx, cv, fmt, mx.quantize(src, mx.ACT, fmt, layout=layout, shape=xs))
        torch.cuda.synchronize()
        assert torch.equal(cs, es), f"scales differ at {torch.nonzero(cs != es)[:8].flatten().tolist()}"
        assert torch.equal(cc, ec), f"codes differ at {torch.nonzero(cc != ec)[:8].flatten().tolist()}"
    oc, os_ = oracle.quantize(ref.numpy(), oracle.NCHW, oracle.ACT, fmt, *xs)
    assert np.array_equal(qx.codes.cpu().numpy()[:len(oc)], oc) and np.array_equal(qx.scales.cpu().numpy(), os_)
    rcc, rcs = oracle.im2col_cbf(cv, fmt, oc, os_)
    assert np.array_equal(cs.cpu().numpy(), rcs)
    assert np.array_equal(cc.cpu().numpy()[:len(rcc)], rcc)


def test_multi_im2col_benchmark_layers(mx):
    """The benchmark layers' X (with its im2col) and W in one call, both formats."""
    for li, (name, cv) in enumerate(synth.SWEEP_LAYERS):
        x, w, _ = synth.layer_inputs(cv, 1000 + li, kind="sweep")
        xd, wd = synth.nchw_to_cbf(x, 32).to(DEV), w.to(DEV)
        for fmt in (0, 1):
            cc, cs = _col_buffers(mx, cv, fmt)
            qx, qw = mx.quantize_multi([(xd, mx.ACT, fmt, mx.CBF, tuple(x.shape), None, (cv, cc, cs)),
                                        (wd, mx.WEIGHT, fmt, mx.NCHW, tuple(w.shape), None)])
            sx = mx.quantize(xd, mx.ACT, fmt, layout=mx.CBF, shape=tuple(x.shape))
            ec, es = _explicit_im2col(mx, cv, fmt, sx)
            torch.cuda.synchronize()
            assert torch.equal(qx.codes, sx.codes) and torch.equal(qx.scales, sx.scales), name
            assert torch.equal(cc, ec) and torch.equal(cs, es), f"{name} fmt {fmt}"
