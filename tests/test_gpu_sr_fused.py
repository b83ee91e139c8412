"""GPU parity of stochastic rounding where the fused path writes gradients:
mxconv_dgrad_quant_sr (the input-gradient epilogue) and mxconv_quantize_sum_sr
(the gradient-sum quantizer), Sec. III-A / Eq. (6).

Each call also hands back the fp32 values it quantized.  Checks per case:
  * those values equal the round-to-nearest call's bit for bit (rounding
    touches only the codes), and that call is held to the oracle's fp64
    result by test_gpu_fused / test_gpu_netops;
  * codes and scales equal the oracle's stochastic quantizer applied to those
    values in the CBF layout with the same seed (the random bits are keyed by
    the code position, so both sides draw the same bits): bit-exact;
  * the same seed reproduces the codes; another seed changes some of them.
"""
import numpy as np
import pytest
import torch

import oracle
from paper_2609_28358_amd import synth

pytestmark = pytest.mark.gpu

DEV = "cuda:0"
SEED = 0x0123456789ABCDEF


@pytest.fixture(scope="module")
def mx():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2609_28358_amd import mxconv
    mxconv.lib()
    return mxconv


def _oracle_sr(vals_cbf, shape, fmt, seed):
    n, c, h, w = shape
    a = synth.cbf_to_nchw(vals_cbf.cpu(), n, c, h, w, 32).numpy().astype(np.float32)
    return oracle.quantize_sr(a, oracle.NCHW, oracle.ACT, fmt, n, c, h, w, seed)


def _match(g, ref):
    rc, rs = ref
    gc, gs = g.codes.cpu().numpy(), g.scales.cpu().numpy()
    assert np.array_equal(gs, rs), f"scales differ at {np.flatnonzero(gs != rs)[:8]}"
    gc = gc[:len(rc)]                       # FP6 buffers end with read-only slack
    assert np.array_equal(gc, rc), f"codes differ at {np.flatnonzero(gc != rc)[:8]}"


CONVS = [
    synth.conv_dict(32, 64, 64, 12, 10, 3, 1, 1),
    synth.conv_dict(32, 64, 48, 11, 9, 3, 2, 1),               # stride 2: input gradient in phases
    synth.conv_dict(64, 32, 128, 6, 5, 3, 1, 1),               # two batch groups
    synth.conv_dict(32, 96, 200, 7, 9, 3, 2, 1),               # ragged channels: padded rows in a block
    synth.conv_dict(32, 128, 64, 8, 8, 1, 1, 0),               # 1x1
    synth.conv_dict(32, 16, 16, 48, 64, 3, 1, 1),              # narrow tiles
]


def _ids(c):
    return f"n{c['n']}_{c['cin']}to{c['cout']}_{c['h']}x{c['w']}_k{c['kh']}{c['kw']}_s{c['sh']}{c['sw']}"


@pytest.mark.parametrize("fn", [0, 2], ids=["none", "silu"])
@pytest.mark.parametrize("fmt,ofmt", [(0, 0), (1, 1), (1, 0), (0, 2), (1, 3)],
                         ids=["e4m3", "e2m1", "e2m1to4m3", "e4m3to2m3", "e2m1to3m2"])
@pytest.mark.parametrize("cv", CONVS, ids=_ids)
def test_dgrad_quant_sr(mx, cv, fmt, ofmt, fn):
    x, w, gy = synth.layer_inputs(cv, 31, kind="unit")
    qw = mx.quantize(w.to(DEV), mx.WEIGHT, fmt)
    qg = mx.quantize(gy.to(DEV), mx.ACT, fmt)
    shape = (cv["n"], cv["cin"], cv["h"], cv["w"])
    zc = synth.nchw_to_cbf(synth.normal(shape, 1.5, 78), 32).to(DEV) if fn else None
    act_rn = torch.full((cv["n"] // 32, cv["h"], cv["w"], cv["cin"], 32), float("nan"), device=DEV)
    act_sr = torch.full_like(act_rn, float("nan"))
    mx.dgrad_quant(cv, qw, qg, fn=fn, z=zc, out_fmt=ofmt, act_out=act_rn)
    g1 = mx.dgrad_quant(cv, qw, qg, fn=fn, z=zc, out_fmt=ofmt, act_out=act_sr, sr_seed=SEED)
    g2 = mx.dgrad_quant(cv, qw, qg, fn=fn, z=zc, out_fmt=ofmt, sr_seed=SEED)
    g3 = mx.dgrad_quant(cv, qw, qg, fn=fn, z=zc, out_fmt=ofmt, sr_seed=SEED + 1)
    torch.cuda.synchronize()
    assert torch.equal(act_sr, act_rn), "stochastic rounding changed the values quantized"
    _match(g1, _oracle_sr(act_sr, shape, ofmt, SEED))
    assert torch.equal(g1.codes, g2.codes) and torch.equal(g1.scales, g2.scales)
    assert not torch.equal(g1.codes, g3.codes), "another seed gave the same codes"


def test_dgrad_quant_sr_bf16(mx):
    """MXC_FN_BF16: z bf16, the product rounded to bf16 first; codes keyed the same way."""
    cv = synth.conv_dict(32, 64, 96, 10, 12, 3, 1, 1)
    x, w, gy = synth.layer_inputs(cv, 33, kind="unit")
    qw = mx.quantize(w.to(DEV), mx.WEIGHT, mx.E2M1)
    qg = mx.quantize(gy.to(DEV), mx.ACT, mx.E2M1)
    shape = (cv["n"], cv["cin"], cv["h"], cv["w"])
    zc = synth.nchw_to_cbf(synth.normal(shape, 1.5, 79), 32).to(DEV).to(torch.bfloat16)
    act_rn = torch.full((1, cv["h"], cv["w"], cv["cin"], 32), float("nan"), device=DEV)
    act_sr = torch.full_like(act_rn, float("nan"))
    fn = mx.FN_SILU | mx.FN_BF16
    mx.dgrad_quant(cv, qw, qg, fn=fn, z=zc, out_fmt=mx.E2M1, act_out=act_rn)
    g = mx.dgrad_quant(cv, qw, qg, fn=fn, z=zc, out_fmt=mx.E2M1, act_out=act_sr, sr_seed=7)
    torch.cuda.synchronize()
    assert torch.equal(act_sr, act_rn)
    _match(g, _oracle_sr(act_sr, shape, mx.E2M1, 7))


SUM_CASES = [
    # n, c, h, w, terms: (c_src, c_off, down), fn
    (32, 32, 6, 5, [(32, 0, 0)], 0),
    (64, 16, 5, 4, [(48, 32, 1), (16, 0, 0), (32, 16, 0)], 2),   # a 16-channel part: padded block
    (32, 64, 3, 3, [(64, 0, 0), (128, 64, 1), (64, 0, 0), (192, 0, 0)], 2),
    (32, 40, 7, 9, [(40, 0, 0), (80, 40, 0)], 0),
]


@pytest.mark.parametrize("bf16", [False, True], ids=["f32", "bf16"])
@pytest.mark.parametrize("fmt", [0, 1], ids=["e4m3", "e2m1"])
@pytest.mark.parametrize("case", SUM_CASES, ids=lambda c: f"n{c[0]}c{c[1]}_{c[2]}x{c[3]}_{len(c[4])}terms_fn{c[5]}")
def test_quantize_sum_sr(mx, fmt, case, bf16):
    n, c, h, w, tdesc, fn = case
    dt = torch.bfloat16 if bf16 else torch.float32
    terms = []
    for k, (c_src, c_off, down) in enumerate(tdesc):
        hs, ws = (2 * h, 2 * w) if down else (h, w)
        g = synth.normal((n, c_src, hs, ws), 1e-3 * (k + 1), 170 + k)
        terms.append((synth.nchw_to_cbf(g, 32).to(DEV).to(dt), c_src, c_off, down))
    zc = synth.nchw_to_cbf(synth.normal((n, c, h, w), 2.0, 190), 32).to(DEV).to(dt) if fn else None
    fnb = fn | (mx.FN_BF16 if bf16 else 0)
    v_rn = torch.full((n // 32, h, w, c, 32), float("nan"), device=DEV)
    v_sr = torch.full_like(v_rn, float("nan"))
    mx.quantize_sum(terms, (n, c, h, w), fmt, fn=fnb, z=zc, vals=v_rn)
    g1 = mx.quantize_sum(terms, (n, c, h, w), fmt, fn=fnb, z=zc, vals=v_sr, sr_seed=SEED)
    g2 = mx.quantize_sum(terms, (n, c, h, w), fmt, fn=fnb, z=zc, sr_seed=SEED)
    g3 = mx.quantize_sum(terms, (n, c, h, w), fmt, fn=fnb, z=zc, sr_seed=SEED ^ (1 << 40))
    torch.cuda.synchronize()
    assert torch.equal(v_sr, v_rn), "stochastic rounding changed the values quantized"
    _match(g1, _oracle_sr(v_sr, (n, c, h, w), fmt, SEED))
    assert torch.equal(g1.codes, g2.codes) and torch.equal(g1.scales, g2.scales)
    assert not torch.equal(g1.codes, g3.codes), "another seed gave the same codes"


def test_sr_full_size_fused_gradient(mx):
    """The sweep's 3x3 64->64 56x56 layer at batch 32, MXFP4: the fused SR input gradient in full."""
    cv = synth.conv_dict(32, 64, 64, 56, 56, 3, 1, 1)
    x, w, gy = synth.layer_inputs(cv, 1001, kind="sweep")
    qw = mx.quantize(w.to(DEV), mx.WEIGHT, mx.E2M1)
    qg = mx.quantize(gy.to(DEV), mx.ACT, mx.E2M1)
    shape = (cv["n"], cv["cin"], cv["h"], cv["w"])
    zc = synth.nchw_to_cbf(synth.normal(shape, 1.0, 80), 32).to(DEV)
    act = torch.empty((1, 56, 56, 64, 32), device=DEV)
    g = mx.dgrad_quant(cv, qw, qg, fn=mx.FN_SILU, z=zc, out_fmt=mx.E2M1, act_out=act, sr_seed=SEED)
    torch.cuda.synchronize()
    _match(g, _oracle_sr(act, shape, mx.E2M1, SEED))
