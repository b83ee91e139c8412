"""bf16 full-precision tensors between layers: the MXC_CBF_BF16 output layout
and the MXC_FN_BF16 mode of the fused epilogues and of the gradient sum.

The rule under test: the fp32 GEMM result is rounded to bf16 (round to
nearest, ties to even -- oracle.round_bf16, pinned in test_oracle_net) and
that rounded value is what is stored, activated, multiplied and quantized.
  * a bf16 output equals oracle.round_bf16 of the same call's fp32 output,
    bit for bit (same kernel arithmetic), on lean and general-kernel shapes;
  * the bf16 values agree with the oracle's fp64 GEMMs within the GEMM bound
    1e-5 * S plus the rounding, 2^-8 of the magnitude;
  * the fused epilogues' codes equal the oracle quantizer applied to the
    fp32 values they quantized (returned through act_out), bit for bit;
  * the fused input gradient equals the unfused route (bf16 input gradient,
    then mxconv_quantize_sum in bf16 mode) bit for bit;
  * mxconv_quantize_sum on bf16 terms and z: values against the oracle's
    fp64 gradient sum, codes bit for bit on the values it quantized.
"""
import numpy as np
import pytest
import torch

import oracle
from paper_2609_28358_amd import synth

pytestmark = pytest.mark.gpu
DEV = "cuda:0"
TOL = 1e-5
RND = 2.0 ** -8      # bf16 rounding: at most half of a 2^-7 step, relative


@pytest.fixture(scope="module")
def mx():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2609_28358_amd import mxconv
    mxconv.lib()
    return mxconv


def _layer(mx, cv, fmt, seed):
    x, w, gy = synth.layer_inputs(cv, seed, kind="unit")
    q = {k: mx.quantize(t.to(DEV), role, fmt) for k, t, role in
         (("x", x, mx.ACT), ("w", w, mx.WEIGHT), ("gy", gy, mx.ACT))}
    o = {k: oracle.quantize(t.numpy(), oracle.NCHW, role, fmt, *t.shape) for k, t, role in
         (("x", x, oracle.ACT), ("w", w, oracle.WEIGHT), ("gy", gy, oracle.ACT))}
    return q, o


def _bits(t):
    """bf16 tensor -> its 16-bit patterns (numpy uint16)."""
    return t.cpu().contiguous().view(torch.int16).numpy().view(np.uint16)


def _oracle_bits(f32):
    """oracle.round_bf16 of an fp32 tensor -> 16-bit patterns."""
    r = oracle.round_bf16(f32.cpu().numpy())
    return (r.view(np.uint32) >> 16).astype(np.uint16)


def _cbf(t, n, c, h, w):
    return synth.cbf_to_nchw(t.cpu().float(), n, c, h, w, 32).numpy().astype(np.float64)


def _codes_match(act_cbf, shape, ofmt, q):
    n, c, h, w = shape
    a = synth.cbf_to_nchw(act_cbf.cpu(), n, c, h, w, 32).numpy().astype(np.float32)
    rc, rs = oracle.quantize(a, oracle.NCHW, oracle.ACT, ofmt, n, c, h, w)
    assert np.array_equal(q.scales.cpu().numpy(), rs)
    assert np.array_equal(q.codes.cpu().numpy(), rc)
    return a


def _ids(c):
    return f"n{c['n']}_{c['cin']}to{c['cout']}_{c['h']}x{c['w']}_k{c['kh']}{c['kw']}_s{c['sh']}{c['sw']}"


# lean shapes (batch block 32; narrow FP4 tiles, stride-2 phases, ragged
# channels) and general-kernel shapes (batch block 16, kernel width 5)
OUT_CONVS = [
    synth.conv_dict(32, 64, 64, 12, 10, 3, 1, 1),
    synth.conv_dict(32, 96, 200, 7, 9, 3, 2, 1),
    synth.conv_dict(64, 16, 16, 40, 48, 3, 1, 1),
    synth.conv_dict(64, 3, 16, 64, 48, 3, 2, 1),
    synth.conv_dict(16, 32, 48, 9, 8, 3, 1, 1),
    synth.conv_dict(32, 32, 32, 11, 10, 5, 1, 2),
]


@pytest.mark.parametrize("fmt", [0, 1], ids=["e4m3", "e2m1"])
@pytest.mark.parametrize("cv", OUT_CONVS, ids=_ids)
def test_bf16_outputs(mx, cv, fmt):
    """fwd, dgrad and backward into MXC_CBF_BF16."""
    q, o = _layer(mx, cv, fmt, 31)
    n, bn = cv["n"], mx.batch_block(cv["n"])
    ho, wo = synth.out_hw(cv)
    y32 = mx.fwd(cv, q["w"], q["x"], layout=mx.CBF)
    y16 = mx.fwd(cv, q["w"], q["x"], layout=mx.CBF_BF16)
    g32 = mx.dgrad(cv, q["w"], q["gy"], layout=mx.CBF)
    g16 = mx.dgrad(cv, q["w"], q["gy"], layout=mx.CBF_BF16)
    gb, gwb = mx.backward(cv, q["w"], q["gy"], q["x"], layout=mx.CBF_BF16)
    gw = mx.wgrad(cv, q["gy"], q["x"])
    torch.cuda.synchronize()
    assert y16.dtype == torch.bfloat16 and y16.shape == (n // bn, ho, wo, cv["cout"], bn)
    assert np.array_equal(_bits(y16), _oracle_bits(y32))
    assert np.array_equal(_bits(g16), _oracle_bits(g32))
    assert np.array_equal(_bits(gb), _bits(g16))
    assert torch.equal(gwb, gw)
    if bn != 32:
        return
    ry, sy = oracle.fwd(cv, fmt, o["w"], o["x"])
    rg, sg = oracle.dgrad(cv, fmt, o["w"], o["gy"])
    for got, ref, s, shp in ((y16, ry, sy, (n, cv["cout"], ho, wo)), (g16, rg, sg, (n, cv["cin"], cv["h"], cv["w"]))):
        a = _cbf(got, *shp)
        tol = TOL * s + RND * (np.abs(ref) + TOL * s)
        assert np.all(np.abs(a - ref) <= tol), float(np.max(np.abs(a - ref) / np.maximum(tol, 1e-300)))


FUSED_CONVS = [
    synth.conv_dict(32, 64, 64, 12, 10, 3, 1, 1),
    synth.conv_dict(32, 64, 48, 11, 9, 3, 2, 1),
    synth.conv_dict(32, 40, 72, 13, 11, 3, 1, 1),
    synth.conv_dict(32, 16, 16, 48, 64, 3, 1, 1),
    synth.conv_dict(64, 16, 32, 64, 64, 3, 2, 1),
]


@pytest.mark.parametrize("fmt", [0, 1], ids=["e4m3", "e2m1"])
@pytest.mark.parametrize("cv", FUSED_CONVS, ids=_ids)
def test_fwd_quant_bf16(mx, cv, fmt):
    q, o = _layer(mx, cv, fmt, 33)
    n = cv["n"]
    ho, wo = synth.out_hw(cv)
    shape = (n, cv["cout"], ho, wo)
    plain = mx.fwd(cv, q["w"], q["x"], layout=mx.CBF)
    act = torch.full_like(plain, float("nan"))
    pre = torch.full(plain.shape, float("nan"), dtype=torch.bfloat16, device=DEV)
    lin = torch.full_like(plain, float("nan"))
    y1 = mx.fwd_quant(cv, q["w"], q["x"], fn=mx.FN_SILU | mx.FN_BF16, act_out=act)
    y2 = mx.fwd_quant(cv, q["w"], q["x"], fn=mx.FN_SILU | mx.FN_BF16 | mx.FN_PRE_OUT, act_out=pre)
    y0 = mx.fwd_quant(cv, q["w"], q["x"], fn=mx.FN_NONE | mx.FN_BF16, act_out=lin)
    torch.cuda.synchronize()
    # the stored pre-activation is the rounded plain forward; the same codes
    # with and without it
    assert np.array_equal(_bits(pre), _oracle_bits(plain))
    assert torch.equal(y1.codes, y2.codes) and torch.equal(y1.scales, y2.scales)
    # with no activation the quantized values are the rounded GEMM result
    assert np.array_equal(lin.cpu().numpy().view(np.uint32), oracle.round_bf16(plain.cpu().numpy()).view(np.uint32))
    _codes_match(lin, shape, fmt, y0)
    # SiLU of the rounded value, quantized
    a = _codes_match(act, shape, fmt, y1)
    zb = _cbf(pre, *shape)
    ref = oracle.act_fn(zb, oracle.FN_SILU)
    assert np.all(np.abs(a - ref) <= 1e-6 * np.abs(ref) + 1e-30)
    ry, sy = oracle.fwd(cv, fmt, o["w"], o["x"])
    tol = TOL * sy + RND * (np.abs(ry) + TOL * sy)
    assert np.all(np.abs(zb - ry) <= tol)


@pytest.mark.parametrize("fn", [1, 2], ids=["relu", "silu"])
@pytest.mark.parametrize("fmt", [0, 1], ids=["e4m3", "e2m1"])
@pytest.mark.parametrize("cv", FUSED_CONVS, ids=_ids)
def test_dgrad_quant_bf16(mx, cv, fmt, fn):
    q, o = _layer(mx, cv, fmt, 35)
    n = cv["n"]
    shape = (n, cv["cin"], cv["h"], cv["w"])
    z = synth.normal(shape, 1.5, 79)
    zc = synth.nchw_to_cbf(z, 32).to(torch.bfloat16).to(DEV)
    plain16 = mx.dgrad(cv, q["w"], q["gy"], layout=mx.CBF_BF16)
    act = torch.full(plain16.shape, float("nan"), device=DEV)
    g1 = mx.dgrad_quant(cv, q["w"], q["gy"], fn=fn | mx.FN_BF16, z=zc, act_out=act)
    # the unfused route: bf16 input gradient, then the gradient sum in bf16 mode
    g2 = mx.quantize_sum([(plain16, cv["cin"], 0, 0)], shape, fmt, fn=fn | mx.FN_BF16, z=zc)
    torch.cuda.synchronize()
    assert torch.equal(g1.codes, g2.codes) and torch.equal(g1.scales, g2.scales)
    a = _codes_match(act, shape, fmt, g1)
    zb = _cbf(zc, *shape)
    d = oracle.act_grad(zb, fn)
    gb = _cbf(plain16, *shape)
    # SiLU' in fp32 with the hardware exp2 and reciprocal: a few ulp of its
    # largest term, about 1 + |z| (it crosses zero near z = -1.28); ReLU' is
    # exact
    assert np.all(np.abs(a - gb * d) <= 1e-6 * np.abs(gb) * (1.0 + np.abs(zb)) + 1e-30)
    rg, sg = oracle.dgrad(cv, fmt, o["w"], o["gy"])
    tol = TOL * sg + RND * (np.abs(rg) + TOL * sg)
    assert np.all(np.abs(gb - rg) <= tol)


SUM_CASES = [
    (32, 48, 4, 6, [(96, 16, 0), (48, 0, 0)], 2),
    (64, 16, 5, 4, [(48, 32, 1), (16, 0, 0), (32, 16, 0)], 2),
    (32, 64, 3, 3, [(64, 0, 0), (128, 64, 1), (64, 0, 0), (192, 0, 0)], 0),
    (32, 48, 4, 6, [(96, 16, 0), (48, 0, 1)], 1),                # ReLU
]


@pytest.mark.parametrize("fmt", [0, 1], ids=["e4m3", "e2m1"])
@pytest.mark.parametrize("case", SUM_CASES, ids=lambda c: f"n{c[0]}c{c[1]}_{len(c[4])}terms_fn{c[5]}")
def test_quantize_sum_bf16(mx, fmt, case):
    n, c, h, w, tdesc, fn = case
    terms_gpu, terms_o, terms_abs = [], [], []
    for k, (c_src, c_off, down) in enumerate(tdesc):
        hs, ws = (2 * h, 2 * w) if down else (h, w)
        g = synth.nchw_to_cbf(synth.normal((n, c_src, hs, ws), 1e-3 * (k + 1), 170 + k), 32).to(torch.bfloat16)
        terms_gpu.append((g.to(DEV), c_src, c_off, down))
        flat = g.float().numpy().reshape(-1)
        terms_o.append((flat, c_src, c_off, down))
        terms_abs.append((np.abs(flat), c_src, c_off, down))
    zc = synth.nchw_to_cbf(synth.normal((n, c, h, w), 2.0, 190), 32).to(torch.bfloat16)
    vals = torch.full((n // 32, h, w, c, 32), float("nan"), device=DEV)
    g = mx.quantize_sum(terms_gpu, (n, c, h, w), fmt, fn=fn | mx.FN_BF16, z=zc.to(DEV) if fn else None, vals=vals)
    torch.cuda.synchronize()
    v = synth.cbf_to_nchw(vals.cpu(), n, c, h, w, 32).numpy()
    zf = zc.float().numpy().reshape(-1)
    ref = oracle.gradient_sum(terms_o, fn, zf, n, c, h, w)
    sabs = oracle.gradient_sum(terms_abs, oracle.FN_NONE, None, n, c, h, w)
    gscale = np.abs(oracle.act_grad(oracle._cbf_nchw(zf, n, c, h, w), fn))
    tol = 1e-6 * sabs * np.maximum(1.0, gscale) + 1e-6 * np.abs(ref)
    assert np.all(np.abs(v - ref) <= tol)
    rc, rs = oracle.quantize(v.astype(np.float32), oracle.NCHW, oracle.ACT, fmt, n, c, h, w)
    assert np.array_equal(g.scales.cpu().numpy(), rs)
    assert np.array_equal(g.codes.cpu().numpy(), rc)


def test_bf16_arguments_checked(mx):
    """The element type of every full-precision tensor must match the mode;
    the NVFP entry points and the quantizers refuse MXC_CBF_BF16."""
    cv = synth.conv_dict(32, 32, 32, 4, 4, 3, 1, 1)
    q, _ = _layer(mx, cv, 1, 37)
    f32 = torch.zeros((1, 4, 4, 32, 32), device=DEV)
    with pytest.raises(mx.MxconvError):
        mx.fwd_quant(cv, q["w"], q["x"], fn=mx.FN_SILU | mx.FN_BF16 | mx.FN_PRE_OUT, act_out=f32)
    with pytest.raises(mx.MxconvError):
        mx.dgrad_quant(cv, q["w"], q["gy"], fn=mx.FN_SILU | mx.FN_BF16, z=f32)
    with pytest.raises(mx.MxconvError):
        mx.quantize_sum([(f32, 32, 0, 0)], (32, 32, 4, 4), 1, fn=mx.FN_BF16)
    with pytest.raises(mx.MxconvError):
        mx.fwd(cv, q["w"], q["x"], layout=mx.CBF_BF16, out=f32)
    L = mx.lib()
    src = torch.zeros(32 * 32 * 16, device=DEV)
    qt = mx.MxTensor.empty(mx.ACT, 1, (32, 32, 4, 4), DEV)
    rc = L.mxconv_quantize(mx._ptr(src), mx.F32, mx.CBF_BF16, mx.ACT, 1, 32, 32, 4, 4, mx._ptr(qt.codes),
                           mx._ptr(qt.scales), None)
    assert rc == -2
