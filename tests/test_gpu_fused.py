"""GPU parity of the fused quantizing epilogues (mxconv_fwd_quant,
mxconv_dgrad_quant) against the oracle.

Each call also returns, through `act_out`, the fp32 values its epilogue
quantized.  Three checks per case:
  * codes and scales equal the oracle quantizer applied to those fp32 values
    (both sides take the rounding decision on the same numbers: bit-exact);
  * with no activation, those values equal the plain mxconv_fwd /
    mxconv_dgrad output bit for bit (same kernel arithmetic);
  * the values agree with the oracle's fp64 result passed through the
    activation (forward) or multiplied by its derivative at z (input
    gradient), within the GEMM bound of test_gpu_parity (1e-5 * S) times
    the activation's Lipschitz constant (1 for ReLU, 1.1 for SiLU), plus
    1e-6 relative: the epilogue evaluates the activation in fp32 with the
    hardware exp2 and reciprocal (about 1 ulp each), and an fp32 result
    cannot be nearer than half an ulp to the fp64 reference anyway.
"""
import numpy as np
import pytest
import torch

import oracle
from paper_2609_28358_amd import synth

pytestmark = pytest.mark.gpu

TOL = 1e-5
DEV = "cuda:0"
LIP = {0: 1.0, 1: 1.0, 2: 1.1}


@pytest.fixture(scope="module")
def mx():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2609_28358_amd import mxconv
    mxconv.lib()
    return mxconv


def _layer(mx, cv, fmt, seed, kind="unit"):
    x, w, gy = synth.layer_inputs(cv, seed, kind=kind)
    q = {k: mx.quantize(t.to(DEV), role, fmt) for k, t, role in
         (("x", x, mx.ACT), ("w", w, mx.WEIGHT), ("gy", gy, mx.ACT))}
    o = {k: oracle.quantize(t.numpy(), oracle.NCHW, role, fmt, *t.shape) for k, t, role in
         (("x", x, oracle.ACT), ("w", w, oracle.WEIGHT), ("gy", gy, oracle.ACT))}
    return q, o


def _bound(cv, fmt, o, which, ref_shape, sabs):
    return TOL * sabs


def _codes_match(mx, act_cbf, shape, ofmt, q):
    """The epilogue's codes equal the oracle quantizer on the values it quantized."""
    n, c, h, w = shape
    a = synth.cbf_to_nchw(act_cbf.cpu(), n, c, h, w, 32).numpy().astype(np.float32)
    rc, rs = oracle.quantize(a, oracle.NCHW, oracle.ACT, ofmt, n, c, h, w)
    gc, gs = q.codes.cpu().numpy(), q.scales.cpu().numpy()
    assert np.array_equal(gs, rs), f"scales differ at {np.flatnonzero(gs != rs)[:8]}"
    assert np.array_equal(gc, rc), f"codes differ at {np.flatnonzero(gc != rc)[:8]}"
    return a


FUSED_CONVS = [
    synth.conv_dict(32, 64, 64, 12, 10, 3, 1, 1),
    synth.conv_dict(32, 64, 96, 9, 9, 1, 1, 0),
    synth.conv_dict(32, 64, 48, 11, 9, 3, 2, 1),               # stride 2 (input gradient in phases)
    synth.conv_dict(64, 32, 128, 6, 5, 3, 1, 1),               # two batch groups
    synth.conv_dict(32, 128, 64, 8, 8, 1, 2, 0),               # 1x1 stride 2: a phase with no taps
    synth.conv_dict(32, 96, 200, 7, 9, 3, 2, 1),               # ragged channels: padded rows in a block
    synth.conv_dict(32, 40, 72, 13, 11, 3, 1, 1),              # ragged on both sides
    synth.conv_dict(32, 16, 16, 48, 64, 3, 1, 1),              # narrow tiles (FP4: 32 rows x 16 pixels)
    synth.conv_dict(64, 16, 32, 64, 64, 3, 2, 1),              # narrow input gradient in phases
]


def _ids(c):
    return f"n{c['n']}_{c['cin']}to{c['cout']}_{c['h']}x{c['w']}_k{c['kh']}{c['kw']}_s{c['sh']}{c['sw']}"


@pytest.mark.parametrize("fn", [0, 1, 2], ids=["none", "relu", "silu"])
@pytest.mark.parametrize("fmt,ofmt", [(0, 0), (1, 1), (0, 1)], ids=["e4m3", "e2m1", "e4m3to2m1"])
@pytest.mark.parametrize("cv", FUSED_CONVS, ids=_ids)
def test_fwd_quant(mx, cv, fmt, ofmt, fn):
    q, o = _layer(mx, cv, fmt, 21)
    ho, wo = synth.out_hw(cv)
    shape = (cv["n"], cv["cout"], ho, wo)
    plain = mx.fwd(cv, q["w"], q["x"], layout=mx.CBF)
    act = torch.full_like(plain, float("nan"))
    yq = mx.fwd_quant(cv, q["w"], q["x"], fn=fn, out_fmt=ofmt, act_out=act)
    torch.cuda.synchronize()
    if fn == mx.FN_NONE:
        assert torch.equal(act, plain)
    a = _codes_match(mx, act, shape, ofmt, yq)
    ry, sy = oracle.fwd(cv, fmt, o["w"], o["x"])
    ref = oracle.act_fn(ry, fn)
    tol = LIP[fn] * _bound(cv, fmt, o, "fwd", ry.shape, sy) + 1e-6 * np.abs(ref)
    err = np.abs(a.astype(np.float64) - ref)
    assert np.all(err <= tol), float(np.max(err / np.maximum(tol, 1e-300)))


@pytest.mark.parametrize("fn", [0, 1, 2], ids=["none", "relu", "silu"])
@pytest.mark.parametrize("fmt,ofmt", [(0, 0), (1, 1), (1, 0)], ids=["e4m3", "e2m1", "e2m1to4m3"])
@pytest.mark.parametrize("cv", FUSED_CONVS, ids=_ids)
def test_dgrad_quant(mx, cv, fmt, ofmt, fn):
    q, o = _layer(mx, cv, fmt, 23)
    shape = (cv["n"], cv["cin"], cv["h"], cv["w"])
    z = synth.normal(shape, 1.5, 77)
    zc = synth.nchw_to_cbf(z, 32).to(DEV)
    plain = mx.dgrad(cv, q["w"], q["gy"], layout=mx.CBF)
    act = torch.full_like(plain, float("nan"))
    gq = mx.dgrad_quant(cv, q["w"], q["gy"], fn=fn, z=zc if fn else None, out_fmt=ofmt, act_out=act)
    torch.cuda.synchronize()
    if fn == mx.FN_NONE:
        assert torch.equal(act, plain)
    a = _codes_match(mx, act, shape, ofmt, gq)
    rgx, sgx = oracle.dgrad(cv, fmt, o["w"], o["gy"])
    d = oracle.act_grad(z.numpy(), fn)
    ref = rgx * d
    tol = LIP[fn] * _bound(cv, fmt, o, "dgrad", rgx.shape, sgx) + 1e-6 * np.abs(rgx) + 1e-30
    err = np.abs(a.astype(np.float64) - ref)
    assert np.all(err <= tol), float(np.max(err / tol))


@pytest.mark.parametrize("fmt", [0, 1], ids=["e4m3", "e2m1"])
def test_fused_full_size_layer(mx, fmt):
    """The 3x3 s1 64->64 56x56 layer at batch 32 with SiLU: every code checked
    against the oracle quantizer, values on 2048 sampled outputs against the
    oracle's fp64 dot products."""
    name, cv = synth.SWEEP_LAYERS[0]
    x, w, gy = synth.layer_inputs(cv, 1000, kind="sweep")
    qx = mx.quantize(synth.nchw_to_cbf(x, 32).to(DEV), mx.ACT, fmt, layout=mx.CBF, shape=tuple(x.shape))
    qw = mx.quantize(w.to(DEV), mx.WEIGHT, fmt)
    ho, wo = synth.out_hw(cv)
    shape = (cv["n"], cv["cout"], ho, wo)
    act = torch.empty((cv["n"] // 32, ho, wo, cv["cout"], 32), dtype=torch.float32, device=DEV)
    yq = mx.fwd_quant(cv, qw, qx, fn=mx.FN_SILU, act_out=act)
    torch.cuda.synchronize()
    a = _codes_match(mx, act, shape, fmt, yq)
    ox = oracle.quantize(x.numpy(), oracle.NCHW, oracle.ACT, fmt, *x.shape)
    ow = oracle.quantize(w.numpy(), oracle.NCHW, oracle.WEIGHT, fmt, *w.shape)
    rng = np.random.default_rng(3)
    idx = np.stack([rng.integers(0, d, 2048) for d in shape], 1)
    r, s = oracle.fwd_at(cv, fmt, ow, ox, idx)
    tol = TOL * s
    ref = oracle.act_fn(r, oracle.FN_SILU)
    got = a[tuple(idx.T)].astype(np.float64)
    assert np.all(np.abs(got - ref) <= 1.1 * tol + 1e-6 * np.abs(ref))


@pytest.mark.parametrize("fmt", [0, 1], ids=["e4m3", "e2m1"])
@pytest.mark.parametrize("cv", FUSED_CONVS[:4], ids=_ids)
def test_fwd_quant_pre_activation_out(mx, cv, fmt):
    """With MXC_FN_PRE_OUT the fp32 output is W * X before the activation (bit
    for bit the plain forward), while the codes are those of SiLU(W * X)
    (equal to the call without the flag)."""
    q, _ = _layer(mx, cv, fmt, 23)
    plain = mx.fwd(cv, q["w"], q["x"], layout=mx.CBF)
    pre = torch.full_like(plain, float("nan"))
    y1 = mx.fwd_quant(cv, q["w"], q["x"], fn=mx.FN_SILU | mx.FN_PRE_OUT, act_out=pre)
    y2 = mx.fwd_quant(cv, q["w"], q["x"], fn=mx.FN_SILU)
    torch.cuda.synchronize()
    assert torch.equal(pre, plain)
    assert torch.equal(y1.codes, y2.codes) and torch.equal(y1.scales, y2.scales)


def test_fused_unsupported_shapes_refused(mx):
    """Layers outside the fused kernels return MXC_ERR_SHAPE, nothing launched."""
    for cv, which in [(synth.conv_dict(16, 32, 32, 8, 8, 3, 1, 1), "both"),        # batch block 16
                      (synth.conv_dict(32, 32, 32, 9, 9, 5, 1, 2), "both"),        # kernel width 5
                      (dict(n=32, cin=48, cout=96, h=10, w=9, kh=7, kw=3, sh=2, sw=1, ph=3, pw=1), "dgrad")]:
        q, _ = _layer(mx, cv, 0, 5)
        if which == "both":
            with pytest.raises(mx.MxconvError, match="code -3"):
                mx.fwd_quant(cv, q["w"], q["x"])
        with pytest.raises(mx.MxconvError, match="code -3"):
            mx.dgrad_quant(cv, q["w"], q["gy"])
