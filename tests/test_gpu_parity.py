"""GPU parity: the HIP path (through the C ABI) against the CPU oracle.

Codes and scales must match bit for bit.  GEMM outputs are compared with
the oracle's fp64 results element by element: |gpu - oracle| <= 1e-5 * S,
S = sum_k |a_k b_k| (the oracle's sum of absolute products, the error scale
of an fp32 accumulation), for every format.  An output whose products are all zero must be exactly zero.  Inputs come from
the seeded generators in paper_2609_28358_amd.synth.
"""
import numpy as np
import pytest
import torch

import mx_tolerance as mxt
import oracle
from paper_2609_28358_amd import synth

pytestmark = pytest.mark.gpu

TOL = 1e-5


@pytest.fixture(scope="module")
def mx():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2609_28358_amd import mxconv
    mxconv.lib()
    return mxconv


DEV = "cuda:0"


def _qcheck(mx, t, role, fmt, layout, shape, src_for_gpu=None):
    """Quantize on both sides; GPU gets `src_for_gpu` (same values, maybe a
    different layout or bf16), the oracle gets the fp32 NCHW tensor `t`."""
    g = mx.quantize((src_for_gpu if src_for_gpu is not None else t).to(DEV), role, fmt, layout=layout,
                    shape=shape)
    torch.cuda.synchronize()
    ref = oracle.quantize(t.float().numpy(), oracle.NCHW, role, fmt, *shape)
    gc, gs = g.codes.cpu().numpy(), g.scales.cpu().numpy()
    assert np.array_equal(gs, ref[1]), f"scales differ at {np.flatnonzero(gs != ref[1])[:8]}"
    assert np.array_equal(gc, ref[0]), f"codes differ at {np.flatnonzero(gc != ref[0])[:8]}"
    return g


Q_SHAPES = [(32, 64, 7, 9), (2, 32, 8, 8), (16, 3, 5, 6), (64, 40, 3, 3), (1, 100, 4, 5),
            (8, 33, 1, 1), (4, 96, 2, 17), (32, 32, 1, 300)]


# E2M1 codes pack two samples per byte, so a batch of one is no E2M1 case
@pytest.mark.parametrize("shape,fmt", [(s, f) for s in Q_SHAPES for f in (0, 1) if not (f == 1 and s[0] == 1)],
                         ids=lambda v: ("e4m3", "e2m1")[v] if isinstance(v, int) else "x".join(map(str, v)))
def test_quantize_nchw_f32(mx, fmt, shape):
    t = synth.normal(shape, 1.0, 11 + shape[0]) * torch.exp(synth.normal(shape, 2.0, 5))
    _qcheck(mx, t, mx.ACT, fmt, mx.NCHW, shape)


NARROW_SHAPES = [(32, 3, 17, 19), (64, 3, 40, 40), (32, 1, 8, 8), (96, 4, 5, 13), (64, 2, 1, 130), (32, 3, 64, 64)]


@pytest.mark.parametrize("fmt", [0, 1], ids=["e4m3", "e2m1"])
@pytest.mark.parametrize("bf16", [False, True], ids=["f32", "bf16"])
@pytest.mark.parametrize("shape", NARROW_SHAPES, ids=lambda s: "x".join(map(str, s)))
def test_quantize_narrow_nchw(mx, fmt, bf16, shape):
    """An input image: NCHW with at most 4 channels and batch block 32 (its
    own kernel; pixel counts that are and are not multiples of the load width,
    partial pixel tiles, U(0, 1) and wide-range values)."""
    t = synth.uniform(shape, 17 + shape[1]) if shape[2] > 16 else (
        synth.normal(shape, 1.0, 3) * torch.exp(synth.normal(shape, 3.0, 4)))
    if bf16:
        tb = t.to(torch.bfloat16)
        _qcheck(mx, tb.float(), mx.ACT, fmt, mx.NCHW, shape, tb)
    else:
        _qcheck(mx, t, mx.ACT, fmt, mx.NCHW, shape)


@pytest.mark.parametrize("fmt", [0, 1], ids=["e4m3", "e2m1"])
@pytest.mark.parametrize("layout", ["nhwc", "cbf", "bf16"])
def test_quantize_layouts_and_bf16(mx, fmt, layout):
    for shape in [(32, 64, 5, 7), (16, 40, 3, 4), (64, 35, 2, 3)]:
        t = synth.silu_normal(shape, 3)
        if layout == "nhwc":
            _qcheck(mx, t, mx.ACT, fmt, mx.NHWC, shape, t.permute(0, 2, 3, 1).contiguous())
        elif layout == "cbf":
            _qcheck(mx, t, mx.ACT, fmt, mx.CBF, shape, synth.nchw_to_cbf(t, synth.batch_block(shape[0])))
        else:
            tb = t.to(torch.bfloat16)
            _qcheck(mx, tb.float(), mx.ACT, fmt, mx.NCHW, shape, tb)


@pytest.mark.parametrize("fmt", [0, 1], ids=["e4m3", "e2m1"])
@pytest.mark.parametrize("bf16", [False, True], ids=["f32", "bf16"])
def test_quantize_cbf_medium(mx, fmt, bf16):
    """CBF activations of a few thousand blocks, with ragged channels and two
    batch groups, fp32 and bf16 sources."""
    for shape in [(32, 70, 41, 37), (64, 64, 40, 29), (32, 100, 61, 47)]:
        t = synth.silu_normal(shape, 7)
        if bf16:
            t = t.to(torch.bfloat16).float()
        src = synth.nchw_to_cbf(t, 32)
        _qcheck(mx, t, mx.ACT, fmt, mx.CBF, shape, src.to(torch.bfloat16) if bf16 else src)


@pytest.mark.parametrize("fmt", [0, 1], ids=["e4m3", "e2m1"])
def test_quantize_weights(mx, fmt):
    for shape in [(64, 64, 3, 3), (20, 48, 3, 3), (256, 64, 1, 1), (16, 3, 3, 3), (33, 70, 5, 2)]:
        t = synth.kaiming(*shape, seed=shape[0])
        _qcheck(mx, t, mx.WEIGHT, fmt, mx.NCHW, shape)


@pytest.mark.parametrize("fmt", [0, 1], ids=["e4m3", "e2m1"])
def test_quantize_edge_values(mx, fmt):
    shape = (32, 64, 2, 4)
    t = synth.normal(shape, 1.0, 9)
    t[:, :32, 0, 0] = 0.0                                 # all-zero block
    t[:, 32:, 0, 0] = -0.0                                # negative zeros
    t[3, 5, 0, 1] = float("inf")                          # non-finite blocks
    t[4, 40, 0, 1] = float("nan")
    t[:, :32, 0, 2] = 2.0 ** -140                         # fp32 subnormals
    t[7, 3, 0, 2] = -(2.0 ** -149)
    t[:, 32:, 0, 2] = 3.0e38                              # near the fp32 maximum
    t[:, :32, 0, 3] = 448.0 * 1.0625                      # saturation and ties
    t[0, 0, 0, 3] = 1.75 * 2 ** 8
    t[:, :32, 1, 0] = torch.tensor([1.0625, 1.1875, 0.75, 1.25, 2.5, 5.0, 1.75, 3.5]).repeat(4)[:32]
    t[:, 32:, 1, 1] = 2.0 ** -10
    _qcheck(mx, t, mx.ACT, fmt, mx.NCHW, shape)


def test_quantize_golden_blocks(mx):
    """The hand-worked blocks of tests/golden through the GPU kernel."""
    from test_oracle_pins import _golden_blocks, _code_at
    for name, fmt, vals, scale, codes in _golden_blocks():
        x = torch.zeros((32, 32, 1, 1))
        for i, v in enumerate(vals):
            x[i, 0, 0, 0] = v
        g = mx.quantize(x.to(DEV), mx.ACT, fmt)
        torch.cuda.synchronize()
        c, s = g.codes.cpu().numpy(), g.scales.cpu().numpy()
        assert s.tolist() == [scale], name
        assert [_code_at(c, fmt, i) for i in range(len(vals))] == codes, name


# ------------------------------------------------------------------ im2col
IM_CONVS = [synth.conv_dict(2, 32, 32, 8, 8, 3, 1, 1), synth.conv_dict(32, 64, 64, 9, 7, 3, 2, 1),
            dict(n=16, cin=40, cout=8, h=6, w=5, kh=3, kw=2, sh=1, sw=2, ph=1, pw=0),
            synth.conv_dict(64, 32, 32, 4, 4, 1, 1, 0)]


@pytest.mark.parametrize("fmt", [0, 1], ids=["e4m3", "e2m1"])
@pytest.mark.parametrize("ci", range(len(IM_CONVS)))
def test_im2col(mx, fmt, ci):
    cv = IM_CONVS[ci]
    x = synth.silu_normal((cv["n"], cv["cin"], cv["h"], cv["w"]), 4)
    qx = mx.quantize(x.to(DEV), mx.ACT, fmt)
    cc, cs = mx.im2col_cbf(cv, qx)
    torch.cuda.synchronize()
    ox = oracle.quantize(x.numpy(), oracle.NCHW, oracle.ACT, fmt, *x.shape)
    rc, rs = oracle.im2col_cbf(cv, fmt, *ox)
    assert np.array_equal(cs.cpu().numpy(), rs) and np.array_equal(cc.cpu().numpy(), rc)


# ------------------------------------------------------------------ GEMMs
_err = mxt.gemm_err


def _all_idx(*dims):
    return np.stack(np.meshgrid(*[np.arange(d) for d in dims], indexing="ij"), -1).reshape(-1, len(dims))


def _layer(mx, cv, fmt, seed, kind="sweep"):
    x, w, gy = synth.layer_inputs(cv, seed, kind=kind)
    q = {k: mx.quantize(t.to(DEV), role, fmt) for k, t, role in
         (("x", x, mx.ACT), ("w", w, mx.WEIGHT), ("gy", gy, mx.ACT))}
    o = {k: oracle.quantize(t.numpy(), oracle.NCHW, role, fmt, *t.shape) for k, t, role in
         (("x", x, oracle.ACT), ("w", w, oracle.WEIGHT), ("gy", gy, oracle.ACT))}
    torch.cuda.synchronize()
    for k in q:   # the GEMMs below see identical operands on both sides
        assert np.array_equal(q[k].codes.cpu().numpy(), o[k][0])
        assert np.array_equal(q[k].scales.cpu().numpy(), o[k][1])
    return q, o


GEMM_CONVS = [
    synth.conv_dict(2, 32, 32, 8, 8, 3, 1, 1),                # the small single-layer case
    synth.conv_dict(32, 64, 64, 12, 10, 3, 1, 1),
    synth.conv_dict(32, 64, 96, 9, 9, 1, 1, 0),
    synth.conv_dict(32, 64, 48, 11, 9, 3, 2, 1),
    synth.conv_dict(16, 3, 16, 13, 12, 3, 2, 1),              # 3-channel input, Bn = 16
    dict(n=8, cin=33, cout=20, h=9, w=7, kh=3, kw=2, sh=2, sw=1, ph=1, pw=0),
    synth.conv_dict(64, 32, 128, 6, 5, 3, 1, 1),              # two batch groups
    synth.conv_dict(4, 40, 70, 10, 11, 5, 2, 2),
    synth.conv_dict(1, 64, 32, 7, 7, 3, 1, 1),                # one sample (E4M3 only)
    synth.conv_dict(32, 128, 64, 8, 8, 1, 2, 0),              # 1x1 stride 2: a phase with no taps
    synth.conv_dict(32, 32, 40, 13, 11, 5, 2, 2),             # 5x5 stride 2, odd sizes
    dict(n=32, cin=48, cout=96, h=10, w=9, kh=7, kw=3, sh=2, sw=1, ph=3, pw=1),
    synth.conv_dict(8, 64, 32, 6, 19, 3, 1, 1),               # Bn = 8: a tile spans 16 pixels
    synth.conv_dict(32, 16, 24, 9, 11, 7, 1, 3),              # 7x7: stages too big for the stream path
    synth.conv_dict(32, 32, 256, 5, 6, 3, 1, 1),              # 256 output channels: 4 row groups per tile
    synth.conv_dict(32, 256, 64, 6, 7, 1, 1, 0),              # 1x1 with 256 input channels (dgrad rows)
    synth.conv_dict(32, 96, 200, 7, 9, 3, 2, 1),              # ragged channels at stride 2
    synth.conv_dict(32, 16, 16, 20, 18, 3, 1, 1),             # one channel block on each side (32 x 32 wgrad tiles)
    synth.conv_dict(64, 3, 16, 24, 22, 3, 2, 1),              # an image layer: 3 channels, stride 2, one block each
    synth.conv_dict(32, 32, 16, 9, 9, 1, 1, 0),
    # FP4 layers with a single 32-row block of outputs run on narrow tiles (32 rows x 16 pixels)
    synth.conv_dict(32, 16, 16, 48, 64, 3, 1, 1),             # fwd and dgrad narrow, stride 1
    synth.conv_dict(64, 3, 16, 128, 96, 3, 2, 1),             # an image layer: fwd narrow at stride 2, dgrad in phases
    synth.conv_dict(32, 32, 16, 40, 80, 1, 1, 0),             # 1x1 narrow
    synth.conv_dict(32, 32, 48, 50, 45, 3, 1, 1),             # dgrad narrow, fwd not (48 outputs)
]


def _ids(c):
    return f"n{c['n']}_{c['cin']}to{c['cout']}_{c['h']}x{c['w']}_k{c['kh']}{c['kw']}_s{c['sh']}{c['sw']}"


@pytest.mark.parametrize("cv,fmt", [(c, f) for c in GEMM_CONVS for f in (0, 1) if not (f == 1 and c["n"] == 1)],
                         ids=lambda v: ("e4m3", "e2m1")[v] if isinstance(v, int) else _ids(v))
@pytest.mark.parametrize("layout", ["nchw", "cbf"])
def test_gemms(mx, fmt, cv, layout):
    lay = mx.NCHW if layout == "nchw" else mx.CBF
    q, o = _layer(mx, cv, fmt, 7, kind="unit")
    bn = synth.batch_block(cv["n"])
    ho, wo = synth.out_hw(cv)
    y = mx.fwd(cv, q["w"], q["x"], layout=lay)
    gx = mx.dgrad(cv, q["w"], q["gy"], layout=lay)
    gw = mx.wgrad(cv, q["gy"], q["x"])
    torch.cuda.synchronize()
    if lay == mx.CBF:
        y = synth.cbf_to_nchw(y.cpu(), cv["n"], cv["cout"], ho, wo, bn)
        gx = synth.cbf_to_nchw(gx.cpu(), cv["n"], cv["cin"], cv["h"], cv["w"], bn)
    ry, sy = oracle.fwd(cv, fmt, o["w"], o["x"])
    rgx, sgx = oracle.dgrad(cv, fmt, o["w"], o["gy"])
    rgw, sgw = oracle.wgrad(cv, fmt, o["gy"], o["x"])
    e = (_err(y.cpu().numpy(), ry, sy), _err(gx.cpu().numpy(), rgx, sgx), _err(gw.cpu().numpy(), rgw, sgw))
    assert max(e) <= 1.0, f"fwd/dgrad/wgrad error / allowed = {e}"


def test_nonfinite_block_propagates(mx):
    cv = synth.conv_dict(32, 32, 32, 4, 4, 3, 1, 1)
    x, w, gy = synth.layer_inputs(cv, 3, kind="unit")
    x[0, 0, 1, 1] = float("inf")
    qx = mx.quantize(x.to(DEV), mx.ACT, mx.E4M3)
    qw = mx.quantize(w.to(DEV), mx.WEIGHT, mx.E4M3)
    y = mx.fwd(cv, qw, qx).cpu()
    # the non-finite block feeds output pixels (0..2, 0..2) of all samples only
    assert torch.isnan(y[:, :, 0:3, 0:3]).all()
    assert torch.isfinite(y[:, :, 3:, :]).all() and torch.isfinite(y[:, :, :, 3:]).all()


# ------------------------------------------------------------------ full-size layers
@pytest.mark.parametrize("fmt", [0, 1], ids=["e4m3", "e2m1"])
@pytest.mark.parametrize("li", range(len(synth.SWEEP_LAYERS)), ids=[n for n, _ in synth.SWEEP_LAYERS])
def test_sweep_layer_full_size(mx, fmt, li):
    """The benchmark's layers at full size, in the launch configuration the
    benchmark times (CBF activations in and out): codes bit-exact everywhere,
    GEMM outputs checked on 2048 seeded samples each by direct dot products."""
    name, cv = synth.SWEEP_LAYERS[li]
    x, w, gy = synth.layer_inputs(cv, 1000 + li, kind="sweep")
    bn = 32
    ho, wo = synth.out_hw(cv)
    qx = mx.quantize(synth.nchw_to_cbf(x, bn).to(DEV), mx.ACT, fmt, layout=mx.CBF, shape=tuple(x.shape))
    qw = mx.quantize(w.to(DEV), mx.WEIGHT, fmt)
    qg = mx.quantize(synth.nchw_to_cbf(gy, bn).to(DEV), mx.ACT, fmt, layout=mx.CBF, shape=tuple(gy.shape))
    y = mx.fwd(cv, qw, qx, layout=mx.CBF)
    gx = mx.dgrad(cv, qw, qg, layout=mx.CBF)
    gw = mx.wgrad(cv, qg, qx)
    torch.cuda.synchronize()
    o = {}
    for k, t, role, q in (("x", x, oracle.ACT, qx), ("w", w, oracle.WEIGHT, qw), ("gy", gy, oracle.ACT, qg)):
        o[k] = oracle.quantize(t.numpy(), oracle.NCHW, role, fmt, *t.shape)
        assert np.array_equal(q.scales.cpu().numpy(), o[k][1]), f"{k} scales"
        assert np.array_equal(q.codes.cpu().numpy(), o[k][0]), f"{k} codes"
    rng = np.random.default_rng(li)
    y = synth.cbf_to_nchw(y.cpu(), cv["n"], cv["cout"], ho, wo, bn).numpy()
    gx = synth.cbf_to_nchw(gx.cpu(), cv["n"], cv["cin"], cv["h"], cv["w"], bn).numpy()
    gw = gw.cpu().numpy()
    S = 2048
    idx = np.stack([rng.integers(0, d, S) for d in (cv["n"], cv["cout"], ho, wo)], 1)
    r, s = oracle.fwd_at(cv, fmt, o["w"], o["x"], idx)
    ey = _err(y[tuple(idx.T)], r, s)
    idx = np.stack([rng.integers(0, d, S) for d in (cv["n"], cv["cin"], cv["h"], cv["w"])], 1)
    r, s = oracle.dgrad_at(cv, fmt, o["w"], o["gy"], idx)
    egx = _err(gx[tuple(idx.T)], r, s)
    idx = np.stack([rng.integers(0, d, S // 8) for d in (cv["cout"], cv["cin"], cv["kh"], cv["kw"])], 1)
    r, s = oracle.wgrad_at(cv, fmt, o["gy"], o["x"], idx)
    egw = _err(gw[tuple(idx.T)], r, s)
    assert max(ey, egx, egw) <= 1.0, (ey, egx, egw)
