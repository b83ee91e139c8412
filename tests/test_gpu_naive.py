"""GPU parity of the naive comparator (quantize after an fp32 im2col, 1-D
blocks along each GEMM's contraction) against the oracle's comparator.

Codes and scales bit for bit; im2col bit for bit (a copy); GEMM outputs
within 1e-5 * S, with S = sum_k |a_k b_k| from the oracle's operands."""
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


def _unpack(codes, fmt, count):
    c = np.asarray(codes, dtype=np.uint8)
    if fmt == 0:
        return c[:count]
    return np.stack([c & 0xF, c >> 4], -1).reshape(-1)[:count]


def _line_to_matrix(lm, rows, cols, direction):
    """GPU line matrix -> (codes [rows][cols], scales in the oracle's layout,
    padding codes, padding scales)."""
    lines, length = (rows, cols) if direction == 0 else (cols, rows)
    lp = (length + 63) // 64 * 64
    codes = _unpack(lm.codes.cpu().numpy(), lm.fmt, lines * lp).reshape(lines, lp)
    scales = lm.scales.cpu().numpy().reshape(lines, lp // 32)
    nbl = (length + 31) // 32
    body, pad_c = codes[:, :length], codes[:, length:]
    sb, pad_s = scales[:, :nbl], scales[:, nbl:]
    if direction == 1:
        body, sb = body.T, sb.T
    return body, np.ascontiguousarray(sb).reshape(-1), pad_c, pad_s


def _matrix(shape, seed):
    rng = np.random.default_rng(seed)
    return (rng.standard_normal(shape) * 2.0 ** rng.uniform(-8, 8, size=shape)).astype(np.float32)


@pytest.mark.parametrize("fmt", [0, 1], ids=["e4m3", "e2m1"])
@pytest.mark.parametrize("direction", [0, 1])
@pytest.mark.parametrize("shape", [(70, 45), (128, 576), (100, 27), (33, 200), (1, 1), (257, 64)],
                         ids=lambda s: f"{s[0]}x{s[1]}")
def test_quantize_1d_bit_exact(mx, fmt, direction, shape):
    m = _matrix(shape, 3 + shape[0])
    if shape[0] > 2:
        m[1, 0] = np.nan                         # a non-finite block
    lm = mx.naive_quantize_1d(torch.from_numpy(m).to(DEV), direction, fmt)
    torch.cuda.synchronize()
    rc, rs = oracle.quantize_1d(m, direction, fmt)
    codes, scales, pad_c, pad_s = _line_to_matrix(lm, *shape, direction)
    assert np.array_equal(scales, rs), "scales differ"
    assert np.array_equal(codes, _unpack(rc, fmt, m.size).reshape(shape)), "codes differ"
    assert not pad_c.any() and not pad_s.any(), "padding not zero"


NAIVE_CONVS = [
    synth.conv_dict(2, 32, 32, 8, 8, 3, 1, 1),
    dict(n=8, cin=33, cout=20, h=9, w=7, kh=3, kw=2, sh=2, sw=1, ph=1, pw=0),
    synth.conv_dict(32, 64, 96, 6, 6, 1, 1, 0),
    synth.conv_dict(4, 40, 70, 7, 6, 3, 2, 1),
    synth.conv_dict(32, 64, 64, 14, 14, 3, 1, 1),       # wgrad splits K (atomic adds)
]


def _nhwc(t):
    return t.permute(0, 2, 3, 1).contiguous()


def _check(got, ref, sabs, what):
    tol = 1e-5 * sabs
    err = np.abs(got.astype(np.float64) - ref)
    zero = sabs == 0
    assert not np.any(got[zero]), f"{what}: nonzero output where every product is zero"
    worst = np.max(err / np.maximum(tol, 1e-300))
    assert worst <= 1.0, f"{what}: error is {worst:.3f} of the allowed bound"


@pytest.mark.parametrize("fmt", [0, 1], ids=["e4m3", "e2m1"])
@pytest.mark.parametrize("cv", NAIVE_CONVS, ids=lambda c: f"n{c['n']}c{c['cin']}o{c['cout']}k{c['kh']}{c['kw']}s{c['sh']}h{c['h']}")
def test_naive_path_matches_oracle(mx, fmt, cv):
    x, w, gy = synth.layer_inputs(cv, 77, kind="unit")
    ho, wo = synth.out_hw(cv)
    P, K, cout = cv["n"] * ho * wo, cv["kh"] * cv["kw"] * cv["cin"], cv["cout"]
    xn, gyn = _nhwc(x), _nhwc(gy)
    wm = w.permute(0, 2, 3, 1).reshape(cout, K).contiguous()
    gym = gyn.reshape(P, cout)

    col = mx.naive_im2col_f32(cv, xn.to(DEV))
    wd, gyd = wm.to(DEV), gym.to(DEV)
    y = mx.naive_fwd(cv, mx.naive_quantize_1d(col, 0, fmt), mx.naive_quantize_1d(wd, 0, fmt))
    gx = mx.naive_dgrad(cv, mx.naive_quantize_1d(gyd, 0, fmt), mx.naive_quantize_1d(wd, 1, fmt))
    gw = mx.naive_wgrad(cv, mx.naive_quantize_1d(gyd, 1, fmt), mx.naive_quantize_1d(col, 1, fmt))
    torch.cuda.synchronize()

    ocol = oracle.naive_im2col(cv, xn.numpy())
    assert np.array_equal(col.cpu().numpy(), ocol), "im2col differs"

    y_ref, sy = oracle.naive_fwd(cv, fmt, xn.numpy(), wm.numpy())
    gx_ref, sgx = oracle.naive_dgrad(cv, fmt, gyn.numpy(), wm.numpy())
    gw_ref, sgw = oracle.naive_wgrad(cv, fmt, gyn.numpy(), xn.numpy())
    _check(y.cpu().numpy(), y_ref, sy, "fwd")
    _check(gx.cpu().numpy(), gx_ref, sgx, "dgrad")
    _check(gw.cpu().numpy(), gw_ref, sgw, "wgrad")
