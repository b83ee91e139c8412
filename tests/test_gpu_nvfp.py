"""GPU parity of the paper-literal NVFP quantizer (Eqs. (4)-(6)) against the
oracle: per-tensor scale T bit-equal, E4M3 block scales and element codes
bit-exact, for every element format, fp32 and bf16 sources, CBF activations
and OIHW weights, and the degenerate tensors (all zero, a NaN, values whose
block scale underflows E4M3)."""
import math

import numpy as np
import pytest
import torch

import mx_tolerance as mxt
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


# ------------------------------------------------------------------ GEMMs on NVFP operands
TOL = 1e-5

NV_CONVS = [
    synth.conv_dict(32, 64, 64, 12, 10, 3, 1, 1),
    synth.conv_dict(32, 64, 96, 9, 9, 1, 1, 0),
    synth.conv_dict(32, 64, 48, 11, 9, 3, 2, 1),               # stride 2 (input gradient in phases)
    synth.conv_dict(64, 32, 128, 6, 5, 3, 1, 1),               # two batch groups
    synth.conv_dict(32, 128, 64, 8, 8, 1, 2, 0),               # 1x1 stride 2: a phase with no taps
    synth.conv_dict(32, 96, 200, 7, 9, 3, 2, 1),               # ragged channels
    synth.conv_dict(32, 40, 72, 13, 11, 3, 1, 1),
]


def _nv_ids(c):
    return f"n{c['n']}_{c['cin']}to{c['cout']}_{c['h']}x{c['w']}_k{c['kh']}{c['kw']}_s{c['sh']}{c['sw']}"


# element formats of (W, X, G_Y): NVFP4 (the paper's format), NVFP8 (its
# "-8" methods), NVFP6 E2M3 (the "-6" methods, Sec. VI-B) and MicroQonv+
# (NVFP6 E3M2 activations with NVFP4 weights and gradients, Sec. IV-D)
NV_METHODS = {"nvfp4": (1, 1, 1), "nvfp8": (0, 0, 0), "nvfp6": (2, 2, 2), "microqonv_plus": (1, 3, 1)}


def _nv_layer(mx, cv, seed, kind="unit", fmts=(1, 1, 1)):
    x, w, gy = synth.layer_inputs(cv, seed, kind=kind)
    q, d = {}, {}
    for (k, t, role), fmt in zip((("w", w, mx.WEIGHT), ("x", x, mx.ACT), ("gy", gy, mx.ACT)), fmts):
        src = synth.nchw_to_cbf(t, 32) if role == mx.ACT else t
        q[k] = _check(mx, t, role, fmt, mx.CBF if role == mx.ACT else mx.NCHW, src)   # bit-exact quantize first
        rc, rs, rt = oracle.nvfp_quantize(t.numpy(), oracle.NCHW, role, fmt, *t.shape)
        d[k] = oracle.nvfp_dequant(rc, rs, rt, role, fmt, *t.shape)
    return q, d


def _nv_err(got, ref, sabs):
    return mxt.gemm_err(got, ref, sabs, tol=TOL)


# every layer in CBF for every method; the NCHW output epilogue does not
# depend on the element format: every layer for NVFP4, the first for the rest
NV_CASES = ([(cv, "cbf", m) for m in NV_METHODS for cv in NV_CONVS] +
            [(cv, "nchw", "nvfp4") for cv in NV_CONVS] + [(NV_CONVS[0], "nchw", m) for m in NV_METHODS if m != "nvfp4"])


@pytest.mark.parametrize("cv,layout,method", NV_CASES, ids=lambda v: _nv_ids(v) if isinstance(v, dict) else v)
def test_nvfp_gemms(mx, cv, layout, method):
    """Forward, input gradient and weight gradient of the fake-quantized NVFP
    tensors against the oracle's direct convolutions of Eqs. (1)-(3) (fp64),
    within 1e-5 of the sum of absolute products, for every element-format
    combination the GEMMs take."""
    lay = mx.NCHW if layout == "nchw" else mx.CBF
    q, d = _nv_layer(mx, cv, 31, fmts=NV_METHODS[method])
    ho, wo = synth.out_hw(cv)
    y = mx.nvfp_fwd(cv, q["w"], q["x"], layout=lay)
    gw = mx.nvfp_wgrad(cv, q["gy"], q["x"])
    dg_ok = (cv["sh"], cv["sw"]) in ((1, 1), (2, 2))
    gx = mx.nvfp_dgrad(cv, q["w"], q["gy"], layout=lay) if dg_ok else None
    torch.cuda.synchronize()
    if lay == mx.CBF:
        y = synth.cbf_to_nchw(y.cpu(), cv["n"], cv["cout"], ho, wo, 32)
        if gx is not None:
            gx = synth.cbf_to_nchw(gx.cpu(), cv["n"], cv["cin"], cv["h"], cv["w"], 32)
    e = [_nv_err(y.cpu().numpy(), oracle.direct_fwd(cv, d["w"], d["x"]),
                 oracle.direct_fwd(cv, np.abs(d["w"]), np.abs(d["x"]))),
         _nv_err(gw.cpu().numpy(), oracle.direct_wgrad(cv, d["gy"], d["x"]),
                 oracle.direct_wgrad(cv, np.abs(d["gy"]), np.abs(d["x"])))]
    if gx is not None:
        e.append(_nv_err(gx.cpu().numpy(), oracle.direct_dgrad(cv, d["w"], d["gy"]),
                         oracle.direct_dgrad(cv, np.abs(d["w"]), np.abs(d["gy"]))))
    assert max(e) <= 1.0, e


@pytest.mark.parametrize("method", list(NV_METHODS))
def test_nvfp_gemms_full_size_layer(mx, method):
    """The 3x3 s1 64->64 56x56 layer at batch 32: 2048 sampled outputs of
    each GEMM against dot products of the dequantized operands."""
    name, cv = synth.SWEEP_LAYERS[0]
    q, d = _nv_layer(mx, cv, 3000, kind="sweep", fmts=NV_METHODS[method])
    ho, wo = synth.out_hw(cv)
    y = synth.cbf_to_nchw(mx.nvfp_fwd(cv, q["w"], q["x"], layout=mx.CBF).cpu(), cv["n"], cv["cout"], ho, wo, 32).numpy()
    gx = synth.cbf_to_nchw(mx.nvfp_dgrad(cv, q["w"], q["gy"], layout=mx.CBF).cpu(), cv["n"], cv["cin"], cv["h"],
                           cv["w"], 32).numpy()
    gw = mx.nvfp_wgrad(cv, q["gy"], q["x"]).cpu().numpy()
    rng = np.random.default_rng(9)
    xp = np.pad(d["x"], ((0, 0), (0, 0), (1, 1), (1, 1)))
    gp = np.pad(d["gy"], ((0, 0), (0, 0), (1, 1), (1, 1)))
    wf = d["w"][:, :, ::-1, ::-1]
    errs = []
    for _ in range(2048):
        n, co, oy, ox = (int(rng.integers(s)) for s in (cv["n"], cv["cout"], ho, wo))
        t = d["w"][co] * xp[n, :, oy:oy + 3, ox:ox + 3]
        errs.append(abs(y[n, co, oy, ox] - t.sum()) / (TOL * np.abs(t).sum() + 1e-300))
        n, ci, iy, ix = (int(rng.integers(s)) for s in (cv["n"], cv["cin"], cv["h"], cv["w"]))
        t = wf[:, ci] * gp[n, :, iy:iy + 3, ix:ix + 3]
        errs.append(abs(gx[n, ci, iy, ix] - t.sum()) / (TOL * np.abs(t).sum() + 1e-300))
    for _ in range(256):
        co, ci, a, b = (int(rng.integers(s)) for s in (cv["cout"], cv["cin"], 3, 3))
        t = d["gy"][:, co] * xp[:, ci, a:a + ho, b:b + wo]
        errs.append(abs(gw[co, ci, a, b] - t.sum()) / (TOL * np.abs(t).sum() + 1e-300))
    assert max(errs) <= 1.0, max(errs)


def test_nvfp_gemm_refusals(mx):
    """Other element formats and layers outside the batch-block-32 kernels are refused."""
    cv = synth.conv_dict(32, 32, 32, 9, 9, 5, 1, 2)                 # kernel width 5
    q, _ = _nv_layer(mx, cv, 5)
    with pytest.raises(mx.MxconvError, match="code -3"):
        mx.nvfp_fwd(cv, q["w"], q["x"])
    x8 = mx.nvfp_quantize(synth.nchw_to_cbf(synth.normal((32, 32, 9, 9), 1.0, 3), 32).to(DEV), mx.ACT, 0,
                          layout=mx.CBF, shape=(32, 32, 9, 9))
    with pytest.raises(mx.MxconvError, match="code -2"):
        mx.nvfp_fwd(cv, q["w"], x8)                                   # FP4 weights with FP8 activations
    cv3 = synth.conv_dict(32, 32, 32, 9, 9, 3, 1, 1)
    shp = (32, 32, 9, 9)
    x6 = mx.nvfp_quantize(synth.nchw_to_cbf(synth.normal(shp, 1.0, 4), 32).to(DEV), mx.ACT, 3, layout=mx.CBF, shape=shp)
    w6 = mx.nvfp_quantize(synth.kaiming(32, 32, 3, 3, seed=6).to(DEV), mx.WEIGHT, 3, shape=(32, 32, 3, 3))
    with pytest.raises(mx.MxconvError, match="code -2"):
        mx.nvfp_fwd(cv3, w6, x6)                                      # E3M2 x E3M2
