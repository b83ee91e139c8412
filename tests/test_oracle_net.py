"""Pins of the oracle's network-step functions (no GPU).

concat_cbf (channel concatenation / 2x nearest upsampling on MX blocks):
  * dequantizing its result equals torch.cat of the dequantized parts (each
    zero-padded to whole 32-channel blocks), with F.interpolate(nearest) for
    an upsampled part -- library routines on the same tensors;
  * quantize-once commutation: quantizing the concatenated / upsampled fp32
    tensor gives exactly the blocks concat_cbf copies (Sec. IV-C: no tensor is
    quantized twice because of a concatenation or an upsampling).
gradient_sum (the gradient of a tensor read by several consumers):
  * equals torch autograd through torch.cat, F.interpolate and SiLU in fp64
    on the same tensors.
"""
import numpy as np
import pytest
import torch
import torch.nn.functional as F

import oracle
from paper_2609_28358_amd import synth


def _q(x, fmt):
    n, c, h, w = x.shape
    return oracle.quantize(x.numpy(), oracle.NCHW, oracle.ACT, fmt, n, c, h, w)


def _deq(q, fmt, shape):
    return torch.from_numpy(oracle.dequant(q[0], q[1], oracle.ACT, fmt, *shape))


def _pad32(t):
    c = t.shape[1]
    cp = -(-c // 32) * 32
    return F.pad(t, (0, 0, 0, 0, 0, cp - c))


@pytest.mark.parametrize("fmt", [oracle.E4M3, oracle.E2M1], ids=["e4m3", "e2m1"])
@pytest.mark.parametrize("n", [32, 64, 8])
def test_concat_equals_cat_of_dequantized_parts(fmt, n):
    h, w = 6, 4
    a = synth.silu_normal((n, 40, h, w), 1)           # 40 channels: 2 blocks, the second one padded
    b = synth.silu_normal((n, 16, h // 2, w // 2), 2)  # upsampled part, 16 channels
    c = synth.normal((n, 32, h, w), 0.3, 3)
    qa, qb, qc = _q(a, fmt), _q(b, fmt), _q(c, fmt)
    cc, cs = oracle.concat_cbf([(qa[0], qa[1], 40, 0), (qb[0], qb[1], 16, 1), (qc[0], qc[1], 32, 0)], fmt, n, h, w)
    got = _deq((cc, cs), fmt, (n, 128, h, w))
    ref = torch.cat([_pad32(_deq(qa, fmt, a.shape)),
                     F.interpolate(_pad32(_deq(qb, fmt, b.shape)), scale_factor=2, mode="nearest"),
                     _deq(qc, fmt, c.shape)], 1)
    assert torch.equal(got, ref)


@pytest.mark.parametrize("fmt", [oracle.E4M3, oracle.E2M1], ids=["e4m3", "e2m1"])
def test_concat_commutes_with_quantize(fmt):
    n, h, w = 64, 4, 6
    a = synth.silu_normal((n, 64, h, w), 4)
    b = synth.silu_normal((n, 32, h // 2, w // 2), 5)
    qa, qb = _q(a, fmt), _q(b, fmt)
    cc, cs = oracle.concat_cbf([(qb[0], qb[1], 32, 1), (qa[0], qa[1], 64, 0)], fmt, n, h, w)
    whole = torch.cat([F.interpolate(b, scale_factor=2, mode="nearest"), a], 1).contiguous()
    rc, rs = _q(whole, fmt)
    assert np.array_equal(cc, rc) and np.array_equal(cs, rs)


def _cbf(t):
    return synth.nchw_to_cbf(t.float(), 32).numpy().reshape(-1)


@pytest.mark.parametrize("fn", [oracle.FN_NONE, oracle.FN_SILU], ids=["none", "silu"])
def test_gradient_sum_equals_autograd(fn):
    n, c, h, w = 32, 24, 4, 6
    z = synth.normal((n, c, h, w), 1.5, 7).double().requires_grad_(True)
    a = F.silu(z) if fn == oracle.FN_SILU else z * 1.0
    # consumer 1: concatenated after another tensor, at 2x resolution
    other = synth.normal((n, 8, 2 * h, 2 * w), 1.0, 8).double()
    cat = torch.cat([other, F.interpolate(a, scale_factor=2, mode="nearest")], 1)
    g_cat = synth.normal(tuple(cat.shape), 1e-3, 9).double()
    # consumer 2: read directly, e.g. by a convolution whose input gradient is g_dir
    g_dir = synth.normal((n, c, h, w), 1e-3, 10).double()
    # consumer 3: concatenated first, at the same resolution, with another part after it
    cat2 = torch.cat([a, other[:, :, ::2, ::2]], 1)
    g_cat2 = synth.normal(tuple(cat2.shape), 1e-3, 11).double()
    loss = (cat * g_cat).sum() + (a * g_dir).sum() + (cat2 * g_cat2).sum()
    (ref,) = torch.autograd.grad(loss, z)
    terms = [(_cbf(g_cat), cat.shape[1], 8, 1), (_cbf(g_dir), c, 0, 0), (_cbf(g_cat2), cat2.shape[1], 0, 0)]
    got = oracle.gradient_sum(terms, fn, _cbf(z.detach()), n, c, h, w)
    # every input was drawn in fp32, so both sides see the same numbers; only
    # the fp64 summation order differs
    assert np.max(np.abs(got - ref.numpy())) <= 1e-12 * float(np.max(np.abs(ref.numpy())))


# ---------------------------------------------------------------- bf16 rounding
def test_round_bf16_hand_worked():
    """bf16 keeps 7 fraction bits: near 1 its step is 2^-7.  Ties go to the
    neighbour with an even last bit; past the largest finite bf16 is inf."""
    f = np.float32
    cases = [
        (1.0, 1.0),
        (1.0 + 2.0 ** -8, 1.0),                            # half a step above 1: tie, 1 is even
        (1.0 + 3 * 2.0 ** -8, 1.0 + 2.0 ** -6),            # tie between 1 + 2^-7 (odd) and 1 + 2^-6 (even)
        (1.0 + 2.0 ** -8 + 2.0 ** -20, 1.0 + 2.0 ** -7),   # just above the tie
        (1.0 + 2.0 ** -8 - 2.0 ** -20, 1.0),               # just below it
        (-(1.0 + 3 * 2.0 ** -8), -(1.0 + 2.0 ** -6)),      # the sign is kept
        (3.0e-39, float(np.uint32(0x00210000).view(np.float32))),   # subnormal: the same bit rule
        (float(np.uint32(0x7F7FFFFF).view(np.float32)), np.inf),    # largest fp32 rounds past bf16's max
        (float(np.uint32(0x7F7F7FFF).view(np.float32)), float(np.uint32(0x7F7F0000).view(np.float32))),
        (np.inf, np.inf), (-0.0, -0.0),
    ]
    for x, want in cases:
        got = oracle.round_bf16(np.array([x], f))[0]
        assert got == f(want) and np.signbit(got) == np.signbit(f(want)), (x, got, want)
    assert np.isnan(oracle.round_bf16(np.array([np.nan], f))[0])


def test_round_bf16_matches_torch_cast():
    """Against torch's fp32 -> bfloat16 cast (round to nearest even) on values
    spanning the exponent range, with many exact ties."""
    rng = np.random.default_rng(5)
    x = (rng.standard_normal(200000) * np.exp2(rng.integers(-130, 120, 200000))).astype(np.float32)
    ties = (x.view(np.uint32) & np.uint32(0xFFFF0000)) | np.uint32(0x8000)
    x = np.concatenate([x, ties.view(np.float32)])
    x = x[np.isfinite(x)]
    want = torch.from_numpy(x).to(torch.bfloat16).to(torch.float32).numpy()
    got = oracle.round_bf16(x)
    assert np.array_equal(got.view(np.uint32), want.view(np.uint32))
