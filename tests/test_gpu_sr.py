"""GPU parity of stochastic rounding (mxconv_quantize_sr) against the oracle.

Codes and scales bit-exact for every format, source layout and kernel path
(the one-wave-per-block kernel for CBF activations with batch block 32 and
OIHW weights, the slab kernel otherwise), including elements whose scaled
value lies below the fp32 range and blocks that saturate or hold a NaN.
The random bits are keyed by the code position, so the same seed gives the
same codes from any source layout.
"""
import numpy as np
import pytest
import torch

import oracle
from paper_2609_28358_amd import synth

pytestmark = pytest.mark.gpu

DEV = "cuda:0"
FMTS = [0, 1, 2, 3]
IDS = ["e4m3", "e2m1", "e2m3", "e3m2"]


@pytest.fixture(scope="module")
def mx():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2609_28358_amd import mxconv
    mxconv.lib()
    return mxconv


def _check(mx, t, role, fmt, seed, layout, shape, src=None):
    g = mx.quantize_sr((src if src is not None else t).to(DEV), role, fmt, seed, layout=layout, shape=shape)
    torch.cuda.synchronize()
    rc, rs = oracle.quantize_sr(t.float().numpy(), oracle.NCHW, role, fmt, *shape, seed)
    gc, gs = g.codes.cpu().numpy(), g.scales.cpu().numpy()
    assert np.array_equal(gs, rs), f"scales differ at {np.flatnonzero(gs != rs)[:8]}"
    gc = gc[:len(rc)]
    assert np.array_equal(gc, rc), f"codes differ at {np.flatnonzero(gc != rc)[:8]}"
    return g


@pytest.mark.parametrize("fmt", FMTS, ids=IDS)
@pytest.mark.parametrize("shape", [(32, 64, 7, 9), (4, 40, 5, 6), (16, 3, 5, 6), (64, 40, 3, 3), (8, 100, 4, 5)],
                         ids=lambda s: "x".join(map(str, s)))
def test_sr_nchw(mx, fmt, shape):
    t = synth.normal(shape, 1.0, 31 + shape[0]) * torch.exp(synth.normal(shape, 2.0, 6))
    _check(mx, t, mx.ACT, fmt, 1234 + shape[1], mx.NCHW, shape)


@pytest.mark.parametrize("fmt", FMTS, ids=IDS)
@pytest.mark.parametrize("layout", ["nhwc", "cbf32", "cbf8", "bf16"])
def test_sr_layouts(mx, fmt, layout):
    """Every layout gives the oracle's codes; CBF with Bn = 32 runs the
    one-wave-per-block kernel."""
    n = 8 if layout == "cbf8" else 32
    shape = (n, 70, 5, 7)
    t = synth.silu_normal(shape, 3)
    seed = 2 ** 40 + 77
    if layout == "nhwc":
        _check(mx, t, mx.ACT, fmt, seed, mx.NHWC, shape, t.permute(0, 2, 3, 1).contiguous())
    elif layout.startswith("cbf"):
        _check(mx, t, mx.ACT, fmt, seed, mx.CBF, shape, synth.nchw_to_cbf(t, synth.batch_block(n)))
    else:
        tb = t.to(torch.bfloat16)
        _check(mx, tb.float(), mx.ACT, fmt, seed, mx.NCHW, shape, tb)


@pytest.mark.parametrize("fmt", FMTS, ids=IDS)
def test_sr_weights(mx, fmt):
    for shape in [(64, 64, 3, 3), (20, 48, 3, 3), (33, 70, 5, 2)]:
        _check(mx, synth.kaiming(*shape, seed=shape[0]), mx.WEIGHT, fmt, 99, mx.NCHW, shape)


@pytest.mark.parametrize("fmt", FMTS, ids=IDS)
@pytest.mark.parametrize("cbf", [False, True], ids=["slab", "block"])
def test_sr_edge_values(mx, fmt, cbf):
    shape = (32, 64, 2, 4)
    t = synth.normal(shape, 1.0, 9)
    t[:, :32, 0, 0] = 0.0
    t[:, 32:, 0, 0] = -0.0
    t[3, 5, 0, 1] = float("inf")
    t[4, 40, 0, 1] = float("nan")
    t[:, :32, 0, 2] = 2.0 ** -140                          # fp32 subnormals
    t[7, 3, 0, 2] = -(2.0 ** -149)
    t[:, 32:, 0, 2] = 3.0e38
    t[5, 33, 0, 2] = 1e-30                                 # scaled far below the fp32 range
    t[6, 34, 0, 2] = -3e-39
    t[:, :32, 0, 3] = 448.0 * 1.0625                       # saturation
    t[0, 0, 0, 3] = 1.75 * 2 ** 8
    t[:, 32:, 1, 1] = 2.0 ** -10
    src = synth.nchw_to_cbf(t, 32) if cbf else None
    _check(mx, t, mx.ACT, fmt, 5, mx.CBF if cbf else mx.NCHW, shape, src)


@pytest.mark.parametrize("fmt", [0, 1], ids=["e4m3", "e2m1"])
def test_sr_full_size_gradient(mx, fmt):
    """G_Y of the 1x1 64->256 56x56 layer at batch 32 (25.7M elements), CBF,
    every code against the oracle; the same seed twice gives the same codes,
    another seed different ones."""
    name, cv = synth.SWEEP_LAYERS[1]
    _, _, gy = synth.layer_inputs(cv, 1001, kind="sweep")
    src = synth.nchw_to_cbf(gy, 32).to(DEV)
    g = _check(mx, gy, mx.ACT, fmt, 2026, mx.CBF, tuple(gy.shape), src)
    g2 = mx.quantize_sr(src, mx.ACT, fmt, 2026, layout=mx.CBF, shape=tuple(gy.shape))
    g3 = mx.quantize_sr(src, mx.ACT, fmt, 2027, layout=mx.CBF, shape=tuple(gy.shape))
    torch.cuda.synchronize()
    assert torch.equal(g.codes, g2.codes) and torch.equal(g.scales, g3.scales)
    assert not torch.equal(g.codes, g3.codes)
