"""GPU parity of the FP6 formats (OCP E2M3 / E3M2) against the oracle.

The two FP6 methods: MicroQonv+ (Sec. IV-D; activations X in E3M2, weights
and gradients in E2M1: fwd and wgrad multiply E2M1 by E3M2, dgrad is plain
E2M1) and the "-6" methods (Sec. VI-B; E2M3 for every operand).

Codes and scales bit-exact (the GPU buffers end with 16 bytes of FP6 read
slack, which are not compared).  GEMM outputs within 1e-5 * S, S = the
oracle's sum of |products|: every product of these format pairs is exact in
the matrix cores' alignment (the smallest product quantum lies above the
truncation quantum), so only fp32 accumulation rounds.  Outputs whose
products are all zero must be exactly zero.
"""
import numpy as np
import pytest
import torch

import mx_tolerance as mxt
import oracle
from paper_2609_28358_amd import synth

pytestmark = pytest.mark.gpu

TOL = 1e-5
DEV = "cuda:0"
E2M1, E2M3, E3M2 = 1, 2, 3
FP6 = [E2M3, E3M2]
# (W, X, G_Y) formats of the two methods
METHODS = {"plus": (E2M1, E3M2, E2M1), "six": (E2M3, E2M3, E2M3)}


@pytest.fixture(scope="module")
def mx():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2609_28358_amd import mxconv
    mxconv.lib()
    return mxconv


def _same_codes(g, ref, what=""):
    gc, gs = g.codes.cpu().numpy(), g.scales.cpu().numpy()
    rc, rs = ref
    assert np.array_equal(gs, rs), f"{what} scales differ at {np.flatnonzero(gs != rs)[:8]}"
    assert len(gc) == len(rc) + (16 if g.fmt in FP6 else 0)
    gc = gc[:len(rc)]
    assert np.array_equal(gc, rc), f"{what} codes differ at {np.flatnonzero(gc != rc)[:8]}"


def _qcheck(mx, t, role, fmt, layout, shape, src=None):
    g = mx.quantize((src if src is not None else t).to(DEV), role, fmt, layout=layout, shape=shape)
    torch.cuda.synchronize()
    _same_codes(g, oracle.quantize(t.float().numpy(), oracle.NCHW, role, fmt, *shape))
    return g


# ------------------------------------------------------------------ quantize
Q_SHAPES = [(32, 64, 7, 9), (4, 32, 8, 8), (16, 3, 5, 6), (64, 40, 3, 3), (8, 100, 4, 5),
            (32, 32, 1, 300), (4, 96, 2, 17)]


@pytest.mark.parametrize("fmt", FP6, ids=["e2m3", "e3m2"])
@pytest.mark.parametrize("shape", Q_SHAPES, ids=lambda s: "x".join(map(str, s)))
def test_quantize_nchw(mx, fmt, shape):
    t = synth.normal(shape, 1.0, 11 + shape[0]) * torch.exp(synth.normal(shape, 2.0, 5))
    _qcheck(mx, t, mx.ACT, fmt, mx.NCHW, shape)


@pytest.mark.parametrize("fmt", FP6, ids=["e2m3", "e3m2"])
@pytest.mark.parametrize("layout", ["nhwc", "cbf", "bf16"])
def test_quantize_layouts_and_bf16(mx, fmt, layout):
    """CBF with batch block 32 runs the one-wave-per-block kernel; the others
    (and CBF with a smaller block) the slab kernel."""
    for shape in [(32, 64, 5, 7), (16, 40, 3, 4), (64, 35, 2, 3), (8, 70, 3, 3)]:
        t = synth.silu_normal(shape, 3)
        if layout == "nhwc":
            _qcheck(mx, t, mx.ACT, fmt, mx.NHWC, shape, t.permute(0, 2, 3, 1).contiguous())
        elif layout == "cbf":
            _qcheck(mx, t, mx.ACT, fmt, mx.CBF, shape, synth.nchw_to_cbf(t, synth.batch_block(shape[0])))
        else:
            tb = t.to(torch.bfloat16)
            _qcheck(mx, tb.float(), mx.ACT, fmt, mx.NCHW, shape, tb)


@pytest.mark.parametrize("fmt", FP6, ids=["e2m3", "e3m2"])
def test_quantize_cbf_medium(mx, fmt):
    for shape in [(32, 70, 41, 37), (64, 64, 40, 29)]:
        t = synth.silu_normal(shape, 7)
        _qcheck(mx, t, mx.ACT, fmt, mx.CBF, shape, synth.nchw_to_cbf(t, 32))


@pytest.mark.parametrize("fmt", FP6, ids=["e2m3", "e3m2"])
def test_quantize_weights(mx, fmt):
    for shape in [(64, 64, 3, 3), (20, 48, 3, 3), (256, 64, 1, 1), (16, 3, 3, 3), (33, 70, 5, 2)]:
        t = synth.kaiming(*shape, seed=shape[0])
        _qcheck(mx, t, mx.WEIGHT, fmt, mx.NCHW, shape)


@pytest.mark.parametrize("fmt", FP6, ids=["e2m3", "e3m2"])
@pytest.mark.parametrize("cbf", [False, True], ids=["nchw", "cbf"])
def test_quantize_edge_values(mx, fmt, cbf):
    shape = (32, 64, 2, 4)
    t = synth.normal(shape, 1.0, 9)
    t[:, :32, 0, 0] = 0.0                                 # all-zero block
    t[:, 32:, 0, 0] = -0.0                                # negative zeros
    t[3, 5, 0, 1] = float("inf")                          # non-finite blocks
    t[4, 40, 0, 1] = float("nan")
    t[:, :32, 0, 2] = 2.0 ** -140                         # fp32 subnormals
    t[7, 3, 0, 2] = -(2.0 ** -149)
    t[:, 32:, 0, 2] = 3.0e38                              # near the fp32 maximum
    t[:, :32, 0, 3] = 7.5 * 1.03                          # saturation and ties
    t[0, 0, 0, 3] = 28.0 * 1.07
    t[:, :32, 1, 0] = torch.tensor([1.0625, 1.1875, 0.0625, 0.1875, 3.875, 3.625, 26.0, 0.21875]).repeat(4)[:32]
    t[:, 32:, 1, 1] = 2.0 ** -10
    src = synth.nchw_to_cbf(t, 32) if cbf else None
    _qcheck(mx, t, mx.ACT, fmt, mx.CBF if cbf else mx.NCHW, shape, src)


def test_quantize_golden_fp6_blocks(mx):
    """The hand-worked FP6 blocks of tests/golden through the GPU kernel."""
    from test_oracle_pins import _golden_blocks, _code_at
    rows = [r for r in _golden_blocks() if r[1] in FP6]
    assert len(rows) >= 4
    for name, fmt, vals, scale, codes in rows:
        x = torch.zeros((32, 32, 1, 1))
        for i, v in enumerate(vals):
            x[i, 0, 0, 0] = v
        g = mx.quantize(x.to(DEV), mx.ACT, fmt)
        torch.cuda.synchronize()
        c, s = g.codes.cpu().numpy(), g.scales.cpu().numpy()
        assert s.tolist() == [scale], name
        assert [_code_at(c, fmt, i) for i in range(len(vals))] == codes, name


# ------------------------------------------------------------------ im2col
@pytest.mark.parametrize("fmt", FP6, ids=["e2m3", "e3m2"])
@pytest.mark.parametrize("cv", [synth.conv_dict(4, 32, 32, 8, 8, 3, 1, 1), synth.conv_dict(32, 64, 64, 9, 7, 3, 2, 1),
                                dict(n=16, cin=40, cout=8, h=6, w=5, kh=3, kw=2, sh=1, sw=2, ph=1, pw=0)],
                         ids=["n4", "n32s2", "n16k32"])
def test_im2col(mx, fmt, cv):
    x = synth.silu_normal((cv["n"], cv["cin"], cv["h"], cv["w"]), 4)
    qx = mx.quantize(x.to(DEV), mx.ACT, fmt)
    cc, cs = mx.im2col_cbf(cv, qx)
    torch.cuda.synchronize()
    ox = oracle.quantize(x.numpy(), oracle.NCHW, oracle.ACT, fmt, *x.shape)
    rc, rs = oracle.im2col_cbf(cv, fmt, *ox)
    assert np.array_equal(cs.cpu().numpy(), rs)
    assert np.array_equal(cc.cpu().numpy()[:len(rc)], rc)


# ------------------------------------------------------------------ GEMMs
def _layer(mx, cv, fmts, seed, kind="unit"):
    fw, fx, fg = fmts
    x, w, gy = synth.layer_inputs(cv, seed, kind=kind)
    q, o = {}, {}
    for k, t, role, f in (("x", x, mx.ACT, fx), ("w", w, mx.WEIGHT, fw), ("gy", gy, mx.ACT, fg)):
        q[k] = mx.quantize(t.to(DEV), role, f)
        o[k] = oracle.quantize(t.numpy(), oracle.NCHW, role, f, *t.shape)
    torch.cuda.synchronize()
    for k in q:   # the GEMMs below see identical operands on both sides
        _same_codes(q[k], o[k], k)
    return q, o


def _err(got, ref, sabs):
    return mxt.gemm_err(got, ref, sabs, tol=TOL)


FP6_CONVS = [
    synth.conv_dict(32, 64, 64, 12, 10, 3, 1, 1),
    synth.conv_dict(32, 64, 96, 9, 9, 1, 1, 0),
    synth.conv_dict(32, 64, 48, 11, 9, 3, 2, 1),               # stride 2 (input gradient in phases)
    synth.conv_dict(64, 32, 128, 6, 5, 3, 1, 1),               # two batch groups
    synth.conv_dict(32, 128, 64, 8, 8, 1, 2, 0),               # 1x1 stride 2: a phase with no taps
    synth.conv_dict(32, 96, 200, 7, 9, 3, 2, 1),               # ragged channels at stride 2
    synth.conv_dict(32, 40, 72, 13, 11, 3, 1, 1),              # ragged on both sides
    synth.conv_dict(32, 32, 256, 5, 6, 3, 1, 1),               # 256 output channels: 4 row groups per tile
    synth.conv_dict(32, 256, 64, 6, 7, 1, 1, 0),               # 256 input channels
    dict(n=32, cin=48, cout=96, h=10, w=9, kh=7, kw=3, sh=2, sw=1, ph=3, pw=1),   # fwd only at 2x1
]


def _ids(c):
    return f"n{c['n']}_{c['cin']}to{c['cout']}_{c['h']}x{c['w']}_k{c['kh']}{c['kw']}_s{c['sh']}{c['sw']}"


def _dgrad_ok(cv):
    return (cv["sh"], cv["sw"]) in ((1, 1), (2, 2))


@pytest.mark.parametrize("method", list(METHODS))
@pytest.mark.parametrize("cv", FP6_CONVS, ids=_ids)
@pytest.mark.parametrize("layout", ["nchw", "cbf"])
def test_gemms(mx, method, cv, layout):
    fmts = METHODS[method]
    lay = mx.NCHW if layout == "nchw" else mx.CBF
    q, o = _layer(mx, cv, fmts, 7)
    fw, fx, fg = fmts
    ho, wo = synth.out_hw(cv)
    y = mx.fwd(cv, q["w"], q["x"], layout=lay)
    gw = mx.wgrad(cv, q["gy"], q["x"])
    gx = mx.dgrad(cv, q["w"], q["gy"], layout=lay) if _dgrad_ok(cv) else None
    torch.cuda.synchronize()
    if lay == mx.CBF:
        y = synth.cbf_to_nchw(y.cpu(), cv["n"], cv["cout"], ho, wo, 32)
        if gx is not None:
            gx = synth.cbf_to_nchw(gx.cpu(), cv["n"], cv["cin"], cv["h"], cv["w"], 32)
    ry, sy = oracle.fwd(cv, (fw, fx), o["w"], o["x"])
    rgw, sgw = oracle.wgrad(cv, (fg, fx), o["gy"], o["x"])
    e = [_err(y.cpu().numpy(), ry, sy), _err(gw.cpu().numpy(), rgw, sgw)]
    if gx is not None:
        rgx, sgx = oracle.dgrad(cv, (fw, fg), o["w"], o["gy"])
        e.append(_err(gx.cpu().numpy(), rgx, sgx))
    assert max(e) <= 1.0, f"fwd/wgrad/dgrad error / allowed = {e}"


@pytest.mark.parametrize("method", list(METHODS))
@pytest.mark.parametrize("li", range(len(synth.SWEEP_LAYERS)), ids=[n for n, _ in synth.SWEEP_LAYERS])
def test_sweep_layer_full_size(mx, method, li):
    """The benchmark's layers at full size with CBF activations in and out:
    codes bit-exact everywhere, GEMM outputs on 2048 seeded samples each
    against the oracle's single-output dot products."""
    fw, fx, fg = METHODS[method]
    name, cv = synth.SWEEP_LAYERS[li]
    x, w, gy = synth.layer_inputs(cv, 2000 + li, kind="sweep")
    ho, wo = synth.out_hw(cv)
    qx = mx.quantize(synth.nchw_to_cbf(x, 32).to(DEV), mx.ACT, fx, layout=mx.CBF, shape=tuple(x.shape))
    qw = mx.quantize(w.to(DEV), mx.WEIGHT, fw)
    qg = mx.quantize(synth.nchw_to_cbf(gy, 32).to(DEV), mx.ACT, fg, layout=mx.CBF, shape=tuple(gy.shape))
    y = mx.fwd(cv, qw, qx, layout=mx.CBF)
    gx = mx.dgrad(cv, qw, qg, layout=mx.CBF)
    gw = mx.wgrad(cv, qg, qx)
    torch.cuda.synchronize()
    o = {}
    for k, t, role, q, f in (("x", x, oracle.ACT, qx, fx), ("w", w, oracle.WEIGHT, qw, fw),
                             ("gy", gy, oracle.ACT, qg, fg)):
        o[k] = oracle.quantize(t.numpy(), oracle.NCHW, role, f, *t.shape)
        _same_codes(q, o[k], k)
    rng = np.random.default_rng(li)
    y = synth.cbf_to_nchw(y.cpu(), cv["n"], cv["cout"], ho, wo, 32).numpy()
    gx = synth.cbf_to_nchw(gx.cpu(), cv["n"], cv["cin"], cv["h"], cv["w"], 32).numpy()
    gw = gw.cpu().numpy()
    S = 2048
    idx = np.stack([rng.integers(0, d, S) for d in (cv["n"], cv["cout"], ho, wo)], 1)
    r, s = oracle.fwd_at(cv, (fw, fx), o["w"], o["x"], idx)
    ey = _err(y[tuple(idx.T)], r, s)
    idx = np.stack([rng.integers(0, d, S) for d in (cv["n"], cv["cin"], cv["h"], cv["w"])], 1)
    r, s = oracle.dgrad_at(cv, (fw, fg), o["w"], o["gy"], idx)
    egx = _err(gx[tuple(idx.T)], r, s)
    idx = np.stack([rng.integers(0, d, S // 8) for d in (cv["cout"], cv["cin"], cv["kh"], cv["kw"])], 1)
    r, s = oracle.wgrad_at(cv, (fg, fx), o["gy"], o["x"], idx)
    egw = _err(gw[tuple(idx.T)], r, s)
    assert max(ey, egx, egw) <= 1.0, (ey, egx, egw)


# ------------------------------------------------------------------ fused epilogues
@pytest.mark.parametrize("fn", [0, 2], ids=["none", "silu"])
@pytest.mark.parametrize("method", list(METHODS))
@pytest.mark.parametrize("cv", FP6_CONVS[:7], ids=_ids)
def test_fused_fp6_outputs(mx, cv, method, fn):
    """Forward writes the next layer's X in the method's activation format
    (E3M2 / E2M3); the input gradient writes the previous layer's G_Y (E2M1 /
    E2M3).  Codes equal the oracle quantizer on the fp32 values the epilogue
    quantized; those equal the plain GEMM (no activation) and the oracle's
    result through the activation within the GEMM bound."""
    fw, fx, fg = METHODS[method]
    q, o = _layer(mx, cv, METHODS[method], 21)
    ho, wo = synth.out_hw(cv)
    plain = mx.fwd(cv, q["w"], q["x"], layout=mx.CBF)
    act = torch.full_like(plain, float("nan"))
    yq = mx.fwd_quant(cv, q["w"], q["x"], fn=fn, out_fmt=fx, act_out=act)
    torch.cuda.synchronize()
    if fn == 0:
        assert torch.equal(act, plain)
    shape = (cv["n"], cv["cout"], ho, wo)
    a = synth.cbf_to_nchw(act.cpu(), *shape, 32).numpy().astype(np.float32)
    _same_codes(yq, oracle.quantize(a, oracle.NCHW, oracle.ACT, fx, *shape), "y")
    ry, sy = oracle.fwd(cv, (fw, fx), o["w"], o["x"])
    ref = oracle.act_fn(ry, fn)
    err = np.abs(a.astype(np.float64) - ref)
    assert np.all(err <= 1.1 * TOL * sy + 1e-6 * np.abs(ref)), float(np.max(err / (1.1 * TOL * sy + 1e-30)))
    if not _dgrad_ok(cv):
        return
    xshape = (cv["n"], cv["cin"], cv["h"], cv["w"])
    z = synth.normal(xshape, 1.5, 77)
    zc = synth.nchw_to_cbf(z, 32).to(DEV)
    plain = mx.dgrad(cv, q["w"], q["gy"], layout=mx.CBF)
    act = torch.full_like(plain, float("nan"))
    gq = mx.dgrad_quant(cv, q["w"], q["gy"], fn=fn, z=zc if fn else None, out_fmt=fg, act_out=act)
    torch.cuda.synchronize()
    if fn == 0:
        assert torch.equal(act, plain)
    a = synth.cbf_to_nchw(act.cpu(), *xshape, 32).numpy().astype(np.float32)
    _same_codes(gq, oracle.quantize(a, oracle.NCHW, oracle.ACT, fg, *xshape), "gx")
    rgx, sgx = oracle.dgrad(cv, (fw, fg), o["w"], o["gy"])
    ref = rgx * oracle.act_grad(z.numpy(), fn)
    err = np.abs(a.astype(np.float64) - ref)
    assert np.all(err <= 1.1 * TOL * sgx + 1e-6 * np.abs(rgx) + 1e-30)


def test_fp6_unsupported_layers_refused(mx):
    """FP6 runs on the batch-block-32 kernels only; other layers are refused."""
    for cv in (synth.conv_dict(16, 32, 32, 8, 8, 3, 1, 1), synth.conv_dict(32, 32, 32, 9, 9, 5, 1, 2)):
        q, _ = _layer(mx, cv, METHODS["six"], 5)
        with pytest.raises(mx.MxconvError, match="code -3"):
            mx.fwd(cv, q["w"], q["x"])
        with pytest.raises(mx.MxconvError, match="code -3"):
            mx.dgrad(cv, q["w"], q["gy"])
