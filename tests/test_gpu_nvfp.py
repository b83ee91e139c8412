"""GPU parity of the paper-literal NVFP quantizer (Eqs. (4)-(6)) against the
oracle: per-tensor scale T bit-equal, E4M3 block scales and element codes
bit-exact, for every element format, fp32 and bf16 sources, CBF activations
and OIHW weights, and the degenerate tensors (all zero, a NaN, values whose
block scale underflows E4M3)."""
import math

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


def _check(mx, t, role, fmt, layout, src):
    shape = tuple(t.shape)
    g = mx.nvfp_quantize(src.to(DEV), role, fmt, layout=layout, shape=shape)
    torch.cuda.synchronize()
    rc, rs, rt = oracle.nvfp_quantize(t.float().numpy(), oracle.NCHW, role, fmt, *shape)
    gt = float(g.tscale[0].cpu())
    assert (math.isnan(gt) and math.isnan(rt)) or gt == rt, (gt, rt)
    gs, gc = g.scales.cpu().numpy(), g.codes.cpu().numpy()[:len(rc)]
    assert np.array_equal(gs, rs), f"block scales differ at {np.flatnonzero(gs != rs)[:8]}"
    assert np.array_equal(gc, rc), f"codes differ at {np.flatnonzero(gc != rc)[:8]}"
    return g


@pytest.mark.parametrize("fmt", FMTS, ids=IDS)
@pytest.mark.parametrize("shape", [(32, 64, 7, 9), (64, 40, 3, 5), (32, 3, 6, 6), (32, 100, 4, 5)],
                         ids=lambda s: "x".join(map(str, s)))
@pytest.mark.parametrize("bf16", [False, True], ids=["f32", "bf16"])
def test_nvfp_activations(mx, fmt, shape, bf16):
    t = synth.normal(shape, 1.0, 41 + shape[1]) * torch.exp(synth.normal(shape, 1.5, 8))
    if bf16:
        t = t.to(torch.bfloat16).float()
    src = synth.nchw_to_cbf(t, 32)
    _check(mx, t, mx.ACT, fmt, mx.CBF, src.to(torch.bfloat16) if bf16 else src)


@pytest.mark.parametrize("fmt", FMTS, ids=IDS)
def test_nvfp_weights(mx, fmt):
    for shape in [(64, 64, 3, 3), (20, 48, 3, 3), (256, 64, 1, 1), (33, 70, 5, 2)]:
        t = synth.kaiming(*shape, seed=shape[0])
        _check(mx, t, mx.WEIGHT, fmt, mx.NCHW, t)


@pytest.mark.parametrize("fmt", FMTS, ids=IDS)
def test_nvfp_degenerate_tensors(mx, fmt):
    shape = (32, 64, 2, 3)
    z = torch.zeros(shape)
    _check(mx, z, mx.ACT, fmt, mx.CBF, synth.nchw_to_cbf(z, 32))          # T = 0
    t = synth.normal(shape, 1.0, 5)
    t[:, 8:16, 1, 1] *= 1e-30                                             # block scale underflows E4M3
    t[:, 16:24, 0, 2] = -0.0
    _check(mx, t, mx.ACT, fmt, mx.CBF, synth.nchw_to_cbf(t, 32))
    t[3, 40, 1, 0] = float("nan")                                         # T NaN, scales 0x7F, codes 0
    _check(mx, t, mx.ACT, fmt, mx.CBF, synth.nchw_to_cbf(t, 32))


@pytest.mark.parametrize("fmt", [0, 1], ids=["e4m3", "e2m1"])
def test_nvfp_full_size_activation(mx, fmt):
    """X of the 1x1 64->256 56x56 layer at batch 32 and its G_Y (25.7M elements)."""
    name, cv = synth.SWEEP_LAYERS[1]
    x, _, gy = synth.layer_inputs(cv, 1001, kind="sweep")
    for t in (x, gy):
        _check(mx, t, mx.ACT, fmt, mx.CBF, synth.nchw_to_cbf(t, 32))
