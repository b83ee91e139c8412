"""Pins for the CPU oracle (no GPU).

Each test checks the oracle against something other than itself: the
hand-worked blocks in tests/golden/, brute-force enumeration of the element
formats, torch's float8 cast, torch's fp64 convolutions, F.unfold, the
brute-force direct convolutions of Eqs. (1)-(3), and invariants of the
quantizer.  A plausible slip in the oracle (a dropped term, a wrong sign or
index, a transposed operand, the wrong rounding) fails at least one.
"""
import math
import os

import numpy as np
import pytest
import torch
import torch.nn.functional as F

import oracle
from paper_2609_28358_amd import synth

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")
FMTS = {"E4M3": oracle.E4M3, "E2M1": oracle.E2M1, "E2M3": oracle.E2M3, "E3M2": oracle.E3M2}
ALL_FMTS = [oracle.E4M3, oracle.E2M1, oracle.E2M3, oracle.E3M2]
# OCP MX element formats: emax, largest finite magnitude, code width
EMAX = {oracle.E4M3: 8, oracle.E2M1: 2, oracle.E2M3: 2, oracle.E3M2: 4}
MAXV = {oracle.E4M3: 448.0, oracle.E2M1: 6.0, oracle.E2M3: 7.5, oracle.E3M2: 28.0}
BITS = {oracle.E4M3: 8, oracle.E2M1: 4, oracle.E2M3: 6, oracle.E3M2: 6}


def _parse_num(t):
    t = t.strip()
    if "0x" in t and "p" in t:
        return float.fromhex(t)
    if t.startswith("0x") or t.startswith("0X"):
        return int(t, 16)
    return float(t)


def _golden_blocks():
    rows = []
    with open(os.path.join(GOLDEN, "mx_blocks.txt")) as f:
        for line in f:
            if not line.strip() or line.startswith("#"):
                continue
            name, fmt, vals, scale, codes = [p.strip() for p in line.split("|")]
            rows.append((name, FMTS[fmt], [_parse_num(v) for v in vals.split()],
                         int(scale), [int(_parse_num(c)) for c in codes.split()]))
    return rows


def _code_at(codes, fmt, pos):
    """Stated code packing (a spec, not the method): FP8 one byte per code,
    FP4 two per byte (even position low), FP6 a little-endian bit string
    with the code at position p in bits 6p .. 6p+5."""
    if fmt == oracle.E4M3:
        return int(codes[pos])
    if BITS[fmt] == 6:
        bit = 6 * pos
        word = int(codes[bit // 8]) | (int(codes[bit // 8 + 1]) << 8 if bit // 8 + 1 < len(codes) else 0)
        return (word >> (bit % 8)) & 0x3F
    b = int(codes[pos // 2])
    return (b >> 4) if pos % 2 else (b & 0xF)


@pytest.mark.parametrize("row", _golden_blocks(), ids=lambda r: r[0])
def test_hand_worked_blocks(row):
    name, fmt, vals, scale, codes = row
    x = np.zeros((32, 32, 1, 1), dtype=np.float32)     # N=32, C=32: one tile
    for i, v in enumerate(vals):
        x[i, 0, 0, 0] = v                               # sample i, channel 0
    c, s = oracle.quantize(x, oracle.NCHW, oracle.ACT, fmt, 32, 32, 1, 1)
    assert s.tolist() == [scale]
    # code position of (channel 0, sample i) is i (samples fastest)
    got = [_code_at(c, fmt, i) for i in range(len(vals))]
    assert got == codes
    # every untouched element is +0
    rest = [_code_at(c, fmt, i) for i in range(len(vals), 32 * 32)]
    assert all(r == 0 for r in rest)


# ---------------------------------------------------------------- elements
def _grid(fmt):
    """(code, value) of every finite non-negative code."""
    if fmt == oracle.E4M3:
        u = torch.arange(0, 0x7F, dtype=torch.uint8)       # 0x7F is NaN
        v = u.view(torch.float8_e4m3fn).double()
        return list(zip(u.tolist(), v.tolist()))
    if fmt == oracle.E2M1:
        mags = [0.0, 0.5, 1.0, 1.5, 2.0, 3.0, 4.0, 6.0]     # E2M1 by definition
    elif fmt == oracle.E2M3:                                 # OCP MX FP6 E2M3, codes 0..31
        mags = [0.0, 0.125, 0.25, 0.375, 0.5, 0.625, 0.75, 0.875,
                1.0, 1.125, 1.25, 1.375, 1.5, 1.625, 1.75, 1.875,
                2.0, 2.25, 2.5, 2.75, 3.0, 3.25, 3.5, 3.75,
                4.0, 4.5, 5.0, 5.5, 6.0, 6.5, 7.0, 7.5]
    else:                                                    # OCP MX FP6 E3M2, codes 0..31
        mags = [0.0, 0.0625, 0.125, 0.1875, 0.25, 0.3125, 0.375, 0.4375,
                0.5, 0.625, 0.75, 0.875, 1.0, 1.25, 1.5, 1.75,
                2.0, 2.5, 3.0, 3.5, 4.0, 5.0, 6.0, 7.0,
                8.0, 10.0, 12.0, 14.0, 16.0, 20.0, 24.0, 28.0]
    return list(enumerate(mags))


def _brute_encode(v, fmt):
    grid = _grid(fmt)
    sign = 1 if math.copysign(1.0, v) < 0 else 0
    a = min(abs(v), MAXV[fmt])
    best = min(abs(a - g) for _, g in grid)
    cands = [c for c, g in grid if abs(a - g) == best]
    if len(cands) > 1:
        cands = [c for c in cands if c % 2 == 0]            # tie -> even code
    assert len(cands) == 1
    return cands[0] | (sign << (BITS[fmt] - 1))


def test_fp6_grids_match_published_limits():
    """The FP6 value lists against the OCP MX figures: largest normal, smallest
    normal, largest and smallest subnormal, 32 distinct magnitudes each."""
    limits = {oracle.E2M3: (7.5, 1.0, 0.875, 0.125), oracle.E3M2: (28.0, 0.25, 0.1875, 0.0625)}
    for fmt, (mx, mn, sub_hi, sub_lo) in limits.items():
        g = [v for _, v in _grid(fmt)]
        assert len(set(g)) == 32 and g == sorted(g)
        assert g[-1] == mx == MAXV[fmt] and g[1] == sub_lo
        normals = [v for v in g if v >= mn]
        assert normals[0] == mn and max(v for v in g if v < mn) == sub_hi
        # top binade of the format is [2^emax, 2^(emax+1))
        assert 2.0 ** EMAX[fmt] <= mx < 2.0 ** (EMAX[fmt] + 1)


@pytest.mark.parametrize("fmt", ALL_FMTS)
def test_encode_matches_brute_force(fmt):
    grid = [g for _, g in _grid(fmt)]
    pts = set()
    for a, b in zip(grid[:-1], grid[1:]):                  # values, midpoints, neighbours
        m = (a + b) / 2
        for t in (a, b, m, np.nextafter(m, -1), np.nextafter(m, 2)):
            pts.add(float(t))
    top = MAXV[fmt]
    for t in (top, top * 1.03, top * 1.07, top * 1.2, 2 ** (EMAX[fmt] + 1) * 0.999):
        pts.add(t)
    rng = np.random.default_rng(7)
    pts.update((rng.random(3000) * 2 ** (EMAX[fmt] + 1)).tolist())
    pts.update((rng.random(2000) * grid[2] * 2).tolist())   # subnormal range
    for v in sorted(pts):
        for s in (v, -v):
            assert oracle.encode(s, fmt) == _brute_encode(s, fmt), (s, fmt)


def _brute_encode_vec(v, fmt):
    """_brute_encode over an array: nearest grid value of min(|v|, max),
    ties to the even code, sign bit from the sign of v."""
    grid = _grid(fmt)
    codes = np.array([c for c, _ in grid], dtype=np.int64)
    vals = np.array([g for _, g in grid], dtype=np.float64)
    order = np.argsort(vals)
    codes, vals = codes[order], vals[order]
    a = np.minimum(np.abs(v.astype(np.float64)), MAXV[fmt])
    hi = np.clip(np.searchsorted(vals, a, side="left"), 1, len(vals) - 1)
    lo = hi - 1
    dlo, dhi = a - vals[lo], vals[hi] - a
    pick_hi = (dhi < dlo) | ((dhi == dlo) & (codes[hi] % 2 == 0))
    c = np.where(pick_hi, codes[hi], codes[lo])
    return c | (np.signbit(v).astype(np.int64) << (BITS[fmt] - 1))


def _unpack_codes(codes, fmt, count):
    """All codes of a packed array, in stored order (packing as in _code_at)."""
    b = codes.astype(np.int64)
    if fmt == oracle.E4M3:
        return b[:count]
    if BITS[fmt] == 4:
        return np.stack([b & 0xF, b >> 4], 1).reshape(-1)[:count]
    b = b[:count // 4 * 3].reshape(-1, 3)
    c = np.stack([b[:, 0] & 63, (b[:, 0] >> 6) | ((b[:, 1] & 15) << 2),
                  (b[:, 1] >> 4) | ((b[:, 2] & 3) << 4), b[:, 2] >> 2], 1)
    return c.reshape(-1)[:count]


@pytest.mark.parametrize("fmt", ALL_FMTS)
def test_encode_brute_force_ten_million(fmt):
    """10^7 random values through the tensor quantizer with every block scale
    forced to 2^0 (an anchor 1.5 * 2^emax per block, all else below 2^(emax+1)),
    so each code is encode(x) itself, against the nearest-value search."""
    blocks = 9766                                        # 32 x 32 elements each: >= 10^7 values
    rng = np.random.default_rng(100 + fmt)
    top = 2.0 ** (EMAX[fmt] + 1)
    n = blocks * 1024
    lin = (rng.random(n) * 2 - 1) * top                  # the whole range, saturation included
    sub = np.exp2(rng.uniform(EMAX[fmt] - 14, EMAX[fmt] + 1, n)) * np.where(rng.random(n) < 0.5, -1, 1)
    v = np.where(rng.random(n) < 0.5, lin, sub).astype(np.float32)
    v = np.where(np.abs(v) >= top, np.float32(0.0), v)  # keep every |x| < 2^(emax+1)
    grid = sorted(g for _, g in _grid(fmt))
    special = []                                         # grid values, midpoints (ties) and their neighbours
    for lo_, hi_ in zip(grid[:-1], grid[1:]):
        m = np.float32((lo_ + hi_) / 2)
        special += [lo_, m, np.nextafter(m, np.float32(-1)), np.nextafter(m, np.float32(top))]
    special += [MAXV[fmt], np.nextafter(np.float32(top), np.float32(0))]
    special = np.array(special, dtype=np.float32)
    special = np.concatenate([special, -special])
    v[1:1 + special.size] = special                      # inside the first block, clear of its anchor
    v = v.reshape(blocks, 32, 32)                        # CBF: [pixel][channel][sample]
    v[:, 0, 0] = 1.5 * 2.0 ** EMAX[fmt]
    codes, scales = oracle.quantize(v.reshape(-1), oracle.CBF, oracle.ACT, fmt, 32, 32, 1, blocks)
    assert np.all(scales == 127)
    got = _unpack_codes(codes, fmt, n)
    want = _brute_encode_vec(v.reshape(-1), fmt)
    bad = np.flatnonzero(got != want)
    assert bad.size == 0, (bad[:5], v.reshape(-1)[bad[:5]], got[bad[:5]], want[bad[:5]])


def test_encode_e4m3_matches_torch_cast():
    rng = np.random.default_rng(11)
    mag = 2.0 ** rng.uniform(-14, 9.2, size=20000)
    v = (mag * np.where(rng.random(20000) < 0.5, -1, 1)).astype(np.float32)
    ref = torch.clamp(torch.from_numpy(v), -448, 448).to(torch.float8_e4m3fn).view(torch.uint8)
    got = [oracle.encode(float(t), oracle.E4M3) for t in v]
    assert got == ref.tolist()


@pytest.mark.parametrize("fmt", ALL_FMTS)
def test_decode_matches_format_grid(fmt):
    for code, val in _grid(fmt):
        assert oracle.decode(code, fmt) == val
        neg = code | (1 << (BITS[fmt] - 1))
        assert oracle.decode(neg, fmt) == -val


# ---------------------------------------------------------------- quantizer
def _rand_tensor(shape, seed, spread=6.0):
    rng = np.random.default_rng(seed)
    mag = 2.0 ** rng.uniform(-spread, spread, size=shape)
    return (rng.standard_normal(shape) * mag).astype(np.float32)


@pytest.mark.parametrize("fmt", ALL_FMTS)
def test_scale_puts_block_max_in_top_binade(fmt):
    n, c, h, w = 32, 64, 3, 2
    x = _rand_tensor((n, c, h, w), 3)
    codes, scales = oracle.quantize(x, oracle.NCHW, oracle.ACT, fmt, n, c, h, w)
    for hh in range(h):
        for ww in range(w):
            for cb in range(2):
                blk = x[:, cb * 32:(cb + 1) * 32, hh, ww].astype(np.float64)
                amax = np.abs(blk).max()
                s = int(scales[(hh * w + ww) * 2 + cb]) - 127
                scaled = amax / 2.0 ** s
                assert 2.0 ** EMAX[fmt] <= scaled < 2.0 ** (EMAX[fmt] + 1)


@pytest.mark.parametrize("fmt", ALL_FMTS)
def test_dequant_error_bound(fmt):
    """|x - deq(q(x))| <= half a quantum of x's binade, except clipping in
    the block's top binade (amax above the format maximum saturates)."""
    n, c, h, w = 32, 32, 2, 2
    x = _rand_tensor((n, c, h, w), 5).astype(np.float64)
    codes, scales = oracle.quantize(x.astype(np.float32), oracle.NCHW, oracle.ACT, fmt, n, c, h, w)
    d = oracle.dequant(codes, scales, oracle.ACT, fmt, n, c, h, w)
    mbits = {oracle.E4M3: 3, oracle.E2M1: 1, oracle.E2M3: 3, oracle.E3M2: 2}[fmt]
    minexp = {oracle.E4M3: -6, oracle.E2M1: 0, oracle.E2M3: 0, oracle.E3M2: -2}[fmt]
    for hh in range(h):
        for ww in range(w):
            s = int(scales[hh * w + ww]) - 127
            for i in range(n):
                for cc in range(c):
                    v = x[i, cc, hh, ww] / 2.0 ** s
                    if abs(v) >= MAXV[fmt]:
                        assert abs(d[i, cc, hh, ww] / 2.0 ** s) == MAXV[fmt]
                        continue
                    e = max(math.floor(math.log2(abs(v))) if v != 0 else minexp, minexp)
                    half_q = 2.0 ** (e - mbits) / 2
                    assert abs(v - d[i, cc, hh, ww] / 2.0 ** s) <= half_q


@pytest.mark.parametrize("fmt", ALL_FMTS)
def test_quantizer_invariants(fmt):
    n, c, h, w = 32, 40, 2, 3                      # ragged channels: padded to 64
    x = _rand_tensor((n, c, h, w), 9)
    codes, scales = oracle.quantize(x, oracle.NCHW, oracle.ACT, fmt, n, c, h, w)
    # sign symmetry: codes(-x) = codes(x) with every real element's sign flipped
    cn, sn = oracle.quantize(-x, oracle.NCHW, oracle.ACT, fmt, n, c, h, w)
    assert np.array_equal(sn, scales)
    d = oracle.dequant(codes, scales, oracle.ACT, fmt, n, c, h, w)
    dn = oracle.dequant(cn, sn, oracle.ACT, fmt, n, c, h, w)
    assert np.array_equal(np.signbit(dn), ~np.signbit(d))
    assert np.array_equal(np.abs(dn), np.abs(d))
    # power-of-two equivariance: scale shifts by k, codes unchanged
    for k in (-5, 3):
        ck, sk = oracle.quantize(x * np.float32(2.0 ** k), oracle.NCHW, oracle.ACT, fmt, n, c, h, w)
        assert np.array_equal(ck, codes)
        assert np.array_equal(sk.astype(int), scales.astype(int) + k)
    # idempotence: re-quantizing the dequantized tensor is the identity
    c2, s2 = oracle.quantize(d.astype(np.float32), oracle.NCHW, oracle.ACT, fmt, n, c, h, w)
    assert np.array_equal(c2, codes) and np.array_equal(s2, scales)


def _fp6_ok(fmt, n):
    """FP6 activation codes fill whole bytes per channel row only with a batch
    block of at least 4, so smaller batches are not a valid FP6 case."""
    fs = fmt if isinstance(fmt, tuple) else (fmt,)
    return n >= 4 or all(BITS[f] != 6 for f in fs)


def _pos(n, c, h, w, bn, H, W, Cp):
    """Stated code layout [N/Bn][H][W][Cp][Bn] (a spec, not the method)."""
    return ((((n // bn) * H + h) * W + w) * Cp + c) * bn + n % bn


@pytest.mark.parametrize("fmt,N", [(f, N) for N in [2, 4, 16, 64] for f in ALL_FMTS if _fp6_ok(f, N)])
def test_layout_single_element(fmt, N):
    C, H, W = 40, 3, 5
    Cp, bn = 64, min(32, N)
    rng = np.random.default_rng(N)
    for _ in range(6):
        n, c, h, w = (int(rng.integers(N)), int(rng.integers(C)), int(rng.integers(H)),
                      int(rng.integers(W)))
        x = np.zeros((N, C, H, W), dtype=np.float32)
        x[n, c, h, w] = -1.0
        codes, scales = oracle.quantize(x, oracle.NCHW, oracle.ACT, fmt, N, C, H, W)
        pos = _pos(n, c, h, w, bn, H, W, Cp)
        # -1.0 alone: scale 2^-emax, element -2^emax = -256 (0xF8), -4 (E2M1
        # 0xE, E2M3 0x38) or -16 (E3M2 0x3C)
        top = {oracle.E4M3: 0xF8, oracle.E2M1: 0xE, oracle.E2M3: 0x38, oracle.E3M2: 0x3C}[fmt]
        nz = [i for i in range(len(codes) * 8 // BITS[fmt]) if _code_at(codes, fmt, i)]
        assert nz == [pos] and _code_at(codes, fmt, pos) == top
        spos = (((n // bn) * H + h) * W + w) * (Cp // 32) + c // 32
        assert [i for i, s in enumerate(scales) if s] == [spos]
        assert scales[spos] == 127 - EMAX[fmt]


@pytest.mark.parametrize("fmt", ALL_FMTS)
def test_source_layouts_agree(fmt):
    N, C, H, W = 64, 40, 3, 4
    x = torch.from_numpy(_rand_tensor((N, C, H, W), 21))
    ref = oracle.quantize(x.numpy(), oracle.NCHW, oracle.ACT, fmt, N, C, H, W)
    nhwc = x.permute(0, 2, 3, 1).contiguous().numpy()
    cbf = synth.nchw_to_cbf(x, 32).numpy()
    for lay, arr in ((oracle.NHWC, nhwc), (oracle.CBF, cbf)):
        got = oracle.quantize(arr, lay, oracle.ACT, fmt, N, C, H, W)
        assert np.array_equal(got[0], ref[0]) and np.array_equal(got[1], ref[1])


def test_weight_role_pads_both_channel_dims():
    """Weight tiles are 32 Cin x 32 Cout at one tap; both dims pad to 32."""
    co, ci = 48, 20
    w = _rand_tensor((co, ci, 3, 3), 4)
    codes, scales = oracle.quantize(w, oracle.NCHW, oracle.WEIGHT, oracle.E4M3, co, ci, 3, 3)
    assert len(codes) == 64 * 3 * 3 * 32 and len(scales) == 2 * 9
    d = oracle.dequant(codes, scales, oracle.WEIGHT, oracle.E4M3, co, ci, 3, 3)
    for cob in range(2):
        for a in range(3):
            for b in range(3):
                blk = w[cob * 32:(cob + 1) * 32, :, a, b].astype(np.float64)
                e = math.floor(math.log2(np.abs(blk).max()))
                assert scales[(cob * 3 + a) * 3 + b] == e - 8 + 127
                err = np.abs(d[cob * 32:(cob + 1) * 32, :, a, b] - blk)
                # half a top-binade quantum, or the clip of [1.75, 2) * 2^e to 448 * 2^s
                clip = np.abs(blk).max() - 1.75 * 2.0 ** e
                assert err.max() <= max(2.0 ** (e - 4), clip)


def test_bad_batch_rejected():
    for n in (3, 48, 20):
        assert oracle.codes_bytes(oracle.ACT, oracle.E4M3, n, 32, 1, 1) < 0
    assert oracle.codes_bytes(oracle.ACT, oracle.E2M1, 1, 32, 1, 1) < 0
    assert oracle.codes_bytes(oracle.ACT, oracle.E4M3, 1, 32, 1, 1) == 32
    for fmt in (oracle.E2M3, oracle.E3M2):
        assert oracle.codes_bytes(oracle.ACT, fmt, 2, 32, 1, 1) < 0
        assert oracle.codes_bytes(oracle.ACT, fmt, 4, 32, 1, 1) == 4 * 32 * 6 // 8
        assert oracle.codes_bytes(oracle.ACT, fmt, 64, 40, 2, 3) == 64 * 64 * 6 * 6 // 8


def test_fp6_bit_string_packing_hand_worked():
    """Four E2M3 samples of one channel holding codes 1, 2, 3, 4 (values
    0.125 .. 0.5 under scale 2^0, set by a 7.5 elsewhere in the block).
    Bit string: 000001 | 000010 | 000011 | 000100, least significant first:
    byte 0 = 01 + (10 << 6) = 0x81, byte 1 = 0000 + (0011 << 4) = 0x30,
    byte 2 = 00 + (000100 << 2) = 0x10."""
    x = np.zeros((4, 32, 1, 1), dtype=np.float32)
    x[:, 0, 0, 0] = [0.125, 0.25, 0.375, 0.5]
    x[0, 5, 0, 0] = 7.5
    codes, scales = oracle.quantize(x, oracle.NCHW, oracle.ACT, oracle.E2M3, 4, 32, 1, 1)
    assert scales.tolist() == [127] and len(codes) == 96
    assert codes[:3].tolist() == [0x81, 0x30, 0x10]
    # channel 5 row starts at byte 15; sample 0 holds 7.5 = 0x1F
    assert codes[15] == 0x1F and codes[16:18].tolist() == [0, 0]
    assert int(np.count_nonzero(codes)) == 4


# ---------------------------------------------------------------- im2col
CONVS = [
    synth.conv_dict(2, 32, 32, 8, 8, 3, 1, 1),
    synth.conv_dict(4, 40, 24, 7, 6, 3, 2, 1),
    synth.conv_dict(32, 32, 64, 5, 5, 1, 1, 0),
    dict(n=8, cin=33, cout=20, h=9, w=7, kh=3, kw=2, sh=2, sw=1, ph=1, pw=0),
    synth.conv_dict(64, 64, 32, 4, 4, 3, 1, 1),
    synth.conv_dict(2, 16, 8, 9, 9, 5, 2, 2),
]


def _conv_fmts(convs, fmts):
    return [(cv, f) for cv in convs for f in fmts if _fp6_ok(f, cv["n"])]


def _cv_fmt_id(v):
    if isinstance(v, dict):
        return f"n{v['n']}c{v['cin']}k{v['kh']}{v['kw']}s{v['sh']}"
    names = {k: n for n, k in FMTS.items()}
    return "-".join(names[t] for t in v) if isinstance(v, tuple) else names[v]


def _unfold_as_tensor(x, cv):
    """fp32 im2col via F.unfold, viewed as (N, C, Ho*Wo*Kh*Kw, 1) with pixel
    index ((ho*Wo+wo)*Kh+kh)*Kw+kw."""
    ho, wo = synth.out_hw(cv)
    u = F.unfold(x, (cv["kh"], cv["kw"]), padding=(cv["ph"], cv["pw"]), stride=(cv["sh"], cv["sw"]))
    n, c = x.shape[:2]
    u = u.reshape(n, c, cv["kh"] * cv["kw"], ho * wo).permute(0, 1, 3, 2)
    return u.reshape(n, c, ho * wo * cv["kh"] * cv["kw"], 1).contiguous()


@pytest.mark.parametrize("cv,fmt", _conv_fmts(CONVS, ALL_FMTS), ids=_cv_fmt_id)
def test_im2col_commutes_with_quantize(fmt, cv):
    """quantize(im2col(X)) == im2col_cbf(quantize(X)), bit for bit (Sec. IV-B:
    quantizing X_{Cin,N} keeps its blocks whole through the CBF im2col)."""
    x = torch.from_numpy(_rand_tensor((cv["n"], cv["cin"], cv["h"], cv["w"]), 31))
    q = oracle.quantize(x.numpy(), oracle.NCHW, oracle.ACT, fmt, cv["n"], cv["cin"], cv["h"], cv["w"])
    col = oracle.im2col_cbf(cv, fmt, *q)
    xu = _unfold_as_tensor(x, cv)
    ref = oracle.quantize(xu.numpy(), oracle.NCHW, oracle.ACT, fmt, cv["n"], cv["cin"], xu.shape[2], 1)
    assert np.array_equal(col[0], ref[0]) and np.array_equal(col[1], ref[1])


def test_im2col_index_map_brute_force():
    cv = CONVS[1]
    fmt = oracle.E4M3
    x = _rand_tensor((cv["n"], cv["cin"], cv["h"], cv["w"]), 2)
    xc, xs = oracle.quantize(x, oracle.NCHW, oracle.ACT, fmt, cv["n"], cv["cin"], cv["h"], cv["w"])
    cc, cs = oracle.im2col_cbf(cv, fmt, xc, xs)
    ho, wo = synth.out_hw(cv)
    bn, Cp = cv["n"], 64
    xt = xc.reshape(1, cv["h"], cv["w"], Cp, bn)
    ct = cc.reshape(1, ho, wo, cv["kh"], cv["kw"], Cp, bn)
    xst = xs.reshape(1, cv["h"], cv["w"], 2)
    cst = cs.reshape(1, ho, wo, cv["kh"], cv["kw"], 2)
    for oh in range(ho):
        for ow in range(wo):
            for a in range(cv["kh"]):
                for b in range(cv["kw"]):
                    ih, iw = oh * cv["sh"] + a - cv["ph"], ow * cv["sw"] + b - cv["pw"]
                    if 0 <= ih < cv["h"] and 0 <= iw < cv["w"]:
                        assert np.array_equal(ct[0, oh, ow, a, b], xt[0, ih, iw])
                        assert np.array_equal(cst[0, oh, ow, a, b], xst[0, ih, iw])
                    else:
                        assert not ct[0, oh, ow, a, b].any() and not cst[0, oh, ow, a, b].any()


# ---------------------------------------------------------------- GEMMs
def _quantized_layer(cv, fmt, seed):
    """fmt: one format for W, X and G_Y, or a (W, X, G_Y) triple."""
    fw, fx, fg = fmt if isinstance(fmt, tuple) else (fmt, fmt, fmt)
    x, w, gy = synth.layer_inputs(cv, seed, kind="unit")
    ho, wo = synth.out_hw(cv)
    qx = oracle.quantize(x.numpy(), oracle.NCHW, oracle.ACT, fx, cv["n"], cv["cin"], cv["h"], cv["w"])
    qw = oracle.quantize(w.numpy(), oracle.NCHW, oracle.WEIGHT, fw, cv["cout"], cv["cin"], cv["kh"], cv["kw"])
    qg = oracle.quantize(gy.numpy(), oracle.NCHW, oracle.ACT, fg, cv["n"], cv["cout"], ho, wo)
    xd = oracle.dequant(*qx, oracle.ACT, fx, cv["n"], cv["cin"], cv["h"], cv["w"])
    wd = oracle.dequant(*qw, oracle.WEIGHT, fw, cv["cout"], cv["cin"], cv["kh"], cv["kw"])
    gd = oracle.dequant(*qg, oracle.ACT, fg, cv["n"], cv["cout"], ho, wo)
    return qx, qw, qg, xd, wd, gd


# (W, X, G_Y) element formats: the single-format methods, MicroQonv+ (FP6
# E3M2 activations, FP4 weights and gradients) and an all-E2M3 "-6" layer
LAYER_FMTS = [oracle.E4M3, oracle.E2M1, (oracle.E2M1, oracle.E3M2, oracle.E2M1),
              (oracle.E2M3, oracle.E2M3, oracle.E2M3)]


def _pairs(fmt):
    """Per-call format pairs (fwd: W, X; dgrad: W, G_Y; wgrad: G_Y, X)."""
    fw, fx, fg = fmt if isinstance(fmt, tuple) else (fmt, fmt, fmt)
    return (fw, fx), (fw, fg), (fg, fx)


def _fmt_id(f):
    names = {v: k for k, v in FMTS.items()}
    return "-".join(names[t] for t in f) if isinstance(f, tuple) else names[f]


def _close(a, b, s):
    scale = np.maximum(s, 1e-300)
    return np.max(np.abs(a - b) / scale) <= 1e-12


@pytest.mark.parametrize("cv,fmt", _conv_fmts(CONVS, LAYER_FMTS), ids=_cv_fmt_id)
def test_gemms_match_torch_fp64(fmt, cv):
    qx, qw, qg, xd, wd, gd = _quantized_layer(cv, fmt, 5)
    pf, pd_, pw = _pairs(fmt)
    st, pd = (cv["sh"], cv["sw"]), (cv["ph"], cv["pw"])
    X, Wt, G = map(torch.from_numpy, (xd, wd, gd))
    y, sy = oracle.fwd(cv, pf, qw, qx)
    gx, sgx = oracle.dgrad(cv, pd_, qw, qg)
    gw, sgw = oracle.wgrad(cv, pw, qg, qx)
    y_ref = F.conv2d(X, Wt, stride=st, padding=pd).numpy()
    gx_ref = torch.nn.grad.conv2d_input(X.shape, Wt, G, stride=st, padding=pd).numpy()
    gw_ref = torch.nn.grad.conv2d_weight(X, Wt.shape, G, stride=st, padding=pd).numpy()
    assert _close(y, y_ref, sy) and _close(gx, gx_ref, sgx) and _close(gw, gw_ref, sgw)
    # the absolute-product sums bound the results and are torch's |.| convs
    sy_ref = F.conv2d(X.abs(), Wt.abs(), stride=st, padding=pd).numpy()
    assert np.allclose(sy, sy_ref, rtol=1e-12, atol=0)
    assert np.all(np.abs(y) <= sy * (1 + 1e-12))
    sgw_ref = torch.nn.grad.conv2d_weight(X.abs(), Wt.shape, G.abs(), stride=st, padding=pd).numpy()
    assert np.allclose(sgw, sgw_ref, rtol=1e-12, atol=0)


@pytest.mark.parametrize("cv,fmt", _conv_fmts(CONVS[:4], [oracle.E4M3, (oracle.E2M1, oracle.E3M2, oracle.E2M1)]),
                         ids=_cv_fmt_id)
def test_gemms_match_direct_definitions(cv, fmt):
    qx, qw, qg, xd, wd, gd = _quantized_layer(cv, fmt, 6)
    pf, pd_, pw = _pairs(fmt)
    y, sy = oracle.fwd(cv, pf, qw, qx)
    gx, sgx = oracle.dgrad(cv, pd_, qw, qg)
    gw, sgw = oracle.wgrad(cv, pw, qg, qx)
    assert _close(y, oracle.direct_fwd(cv, wd, xd), sy)
    assert _close(gx, oracle.direct_dgrad(cv, wd, gd), sgx)
    assert _close(gw, oracle.direct_wgrad(cv, gd, xd), sgw)


@pytest.mark.parametrize("cv,fmt", _conv_fmts(CONVS[:4], [oracle.E2M1, (oracle.E2M3, oracle.E3M2, oracle.E2M1)]),
                         ids=_cv_fmt_id)
def test_single_output_routines_match_full(cv, fmt):
    qx, qw, qg, xd, wd, gd = _quantized_layer(cv, fmt, 8)
    pf, pd_, pw = _pairs(fmt)
    ho, wo = synth.out_hw(cv)
    rng = np.random.default_rng(0)
    y, sy = oracle.fwd(cv, pf, qw, qx)
    idx = np.stack([rng.integers(0, d, 50) for d in (cv["n"], cv["cout"], ho, wo)], 1)
    v, s = oracle.fwd_at(cv, pf, qw, qx, idx)
    assert _close(v, y[tuple(idx.T)], s) and np.allclose(s, sy[tuple(idx.T)], rtol=1e-12)
    gx, sgx = oracle.dgrad(cv, pd_, qw, qg)
    idx = np.stack([rng.integers(0, d, 50) for d in (cv["n"], cv["cin"], cv["h"], cv["w"])], 1)
    v, s = oracle.dgrad_at(cv, pd_, qw, qg, idx)
    assert _close(v, gx[tuple(idx.T)], s) and np.allclose(s, sgx[tuple(idx.T)], rtol=1e-12)
    gw, sgw = oracle.wgrad(cv, pw, qg, qx)
    idx = np.stack([rng.integers(0, d, 50) for d in (cv["cout"], cv["cin"], cv["kh"], cv["kw"])], 1)
    v, s = oracle.wgrad_at(cv, pw, qg, qx, idx)
    assert _close(v, gw[tuple(idx.T)], s) and np.allclose(s, sgw[tuple(idx.T)], rtol=1e-12)


def test_pointwise_conv_is_a_matmul():
    cv = synth.conv_dict(32, 64, 48, 3, 3, 1, 1, 0)
    fmt = oracle.E4M3
    qx, qw, qg, xd, wd, gd = _quantized_layer(cv, fmt, 10)
    y, sy = oracle.fwd(cv, fmt, qw, qx)
    ref = np.einsum("oc,nchw->nohw", wd[:, :, 0, 0], xd)
    assert _close(y, ref, sy)


@pytest.mark.parametrize("fmt", [oracle.E4M3, (oracle.E2M1, oracle.E3M2, oracle.E2M1),
                                 (oracle.E2M3, oracle.E2M3, oracle.E2M3)], ids=_fmt_id)
def test_lossless_inputs_reproduce_plain_convolution(fmt):
    """Inputs already on the MX grid pass through quantization unchanged, so
    the MX convolution equals torch's fp64 convolution of the raw inputs."""
    cv = synth.conv_dict(32, 32, 32, 6, 6, 3, 1, 1)
    fw, fx, _ = fmt if isinstance(fmt, tuple) else (fmt, fmt, fmt)
    qx, qw, qg, xd, wd, gd = _quantized_layer(cv, fmt, 12)
    # xd, wd are exactly representable; quantize them again from fp32
    qx2 = oracle.quantize(xd.astype(np.float32), oracle.NCHW, oracle.ACT, fx, 32, 32, 6, 6)
    qw2 = oracle.quantize(wd.astype(np.float32), oracle.NCHW, oracle.WEIGHT, fw, 32, 32, 3, 3)
    y, sy = oracle.fwd(cv, (fw, fx), qw2, qx2)
    ref = F.conv2d(torch.from_numpy(xd), torch.from_numpy(wd), padding=1).numpy()
    assert _close(y, ref, sy)


# ---------------------------------------------------------------- Table I
def _table1():
    out = {}
    with open(os.path.join(GOLDEN, "table1.txt")) as f:
        for line in f:
            if line.startswith("#") or not line.strip():
                continue
            p = [t.strip() for t in line.split("|")]
            out[p[0]] = [float(t) for t in p[1:]]
    return out


def test_table1_quantization_counts():
    """Per-element quantization counts of Table I at Kh=Kw=3, s=1, p=1:
    quantize-once sees each of X, W, G_Y once; the naive line-block path
    quantizes the im2col'd activations and W, G_Y once per GEMM direction."""
    t1 = _table1()
    cv = synth.conv_dict(32, 32, 32, 8, 8, 3, 1, 1)
    fmt = oracle.E2M1
    x, w, gy = synth.layer_inputs(cv, 1, kind="unit")
    nX, nW, nG = x.numel(), w.numel(), gy.numel()
    # quantize once (MicroQonv)
    counts = []
    for t, role, shape in ((x, oracle.ACT, x.shape), (w, oracle.WEIGHT, w.shape), (gy, oracle.ACT, gy.shape)):
        oracle.counter_reset()
        oracle.quantize(t.numpy(), oracle.NCHW, role, fmt, *shape)
        counts.append(oracle.counter_get())
    assert [counts[0] / nX, counts[1] / nW, counts[2] / nG] == t1["MicroQonv"][:3]
    # naive: im2col'd X quantized along K (fwd) and along (pixel, n) (wgrad);
    # W_f along K and along Cout; G_Yf along (pixel, n) and along Cout
    xu = _unfold_as_tensor(x, cv)                                   # N, C, P*9, 1
    ho, wo = synth.out_hw(cv)
    xcol = xu.reshape(cv["n"], cv["cin"], ho * wo, 9).permute(3, 1, 2, 0).reshape(9 * cv["cin"], -1)
    wf = w.permute(0, 2, 3, 1).reshape(cv["cout"], -1)
    gf = gy.permute(1, 2, 3, 0).reshape(cv["cout"], -1)
    naive = []
    for m in (xcol, wf, gf):
        oracle.counter_reset()
        oracle.quantize_1d(m.numpy(), 0, fmt)
        oracle.quantize_1d(m.numpy(), 1, fmt)
        naive.append(oracle.counter_get())
    assert [naive[0] / nX, naive[1] / nW, naive[2] / nG] == t1["Dacapo"][:3]


def test_quantize_1d_blocks_follow_direction():
    m = _rand_tensor((70, 45), 3)
    r_idx, c_idx = np.meshgrid(np.arange(70), np.arange(45), indexing="ij")
    for d in (0, 1):
        codes, scales = oracle.quantize_1d(m, d, oracle.E4M3)
        if d == 0:      # blocks of 32 along each row: scales [70][2]
            blk = r_idx * 2 + c_idx // 32
        else:           # blocks of 32 down each column: scales [3][45]
            blk = (r_idx // 32) * 45 + c_idx
        s = scales[blk].astype(np.float64) - 127
        for b in np.unique(blk):
            sel = blk == b
            amax = np.abs(m[sel].astype(np.float64)).max()
            sb = s[sel][0]
            assert 2.0 ** 8 <= amax / 2.0 ** sb < 2.0 ** 9
        ref = torch.clamp(torch.from_numpy(m.astype(np.float64) / 2.0 ** s), -448, 448)
        ref = ref.to(torch.float8_e4m3fn).view(torch.uint8).numpy()
        assert np.array_equal(codes.reshape(70, 45), ref)


# ---------------------------------------------------------------- naive comparator
def _nhwc(t):
    return np.ascontiguousarray(t.permute(0, 2, 3, 1).numpy())


def _ohwi(w):
    return np.ascontiguousarray(w.permute(0, 2, 3, 1).reshape(w.shape[0], -1).numpy())


def _int_tensor(shape, seed, lo=-4, hi=4):
    """Small integers: exact under every 1-D block scale of E4M3 and E2M1."""
    g = torch.Generator().manual_seed(seed)
    return torch.randint(lo, hi + 1, shape, generator=g).to(torch.float64)


@pytest.mark.parametrize("cv", CONVS, ids=lambda c: f"n{c['n']}c{c['cin']}k{c['kh']}{c['kw']}s{c['sh']}")
def test_naive_im2col_matches_unfold(cv):
    """The comparator's fp32 im2col is F.unfold with K reordered to (kh, kw, ci)."""
    n, cin, kh, kw = cv["n"], cv["cin"], cv["kh"], cv["kw"]
    x = torch.from_numpy(_rand_tensor((n, cin, cv["h"], cv["w"]), 41))
    ho, wo = synth.out_hw(cv)
    col = oracle.naive_im2col(cv, _nhwc(x))
    u = F.unfold(x, (kh, kw), padding=(cv["ph"], cv["pw"]), stride=(cv["sh"], cv["sw"]))
    ref = u.reshape(n, cin, kh, kw, ho * wo).permute(0, 4, 2, 3, 1).reshape(n * ho * wo, kh * kw * cin)
    assert np.array_equal(col, ref.numpy())


@pytest.mark.parametrize("cv", CONVS, ids=lambda c: f"n{c['n']}c{c['cin']}k{c['kh']}{c['kw']}s{c['sh']}")
def test_naive_col2im_matches_fold(cv):
    """col2im is F.fold (the adjoint of unfold) with the same K order."""
    n, cin, kh, kw = cv["n"], cv["cin"], cv["kh"], cv["kw"]
    ho, wo = synth.out_hw(cv)
    g = np.random.default_rng(5).standard_normal((n * ho * wo, kh * kw * cin))
    gx = oracle.naive_col2im(cv, g)
    u = torch.from_numpy(g).reshape(n, ho * wo, kh, kw, cin).permute(0, 4, 2, 3, 1).reshape(n, cin * kh * kw, -1)
    ref = F.fold(u, (cv["h"], cv["w"]), (kh, kw), padding=(cv["ph"], cv["pw"]), stride=(cv["sh"], cv["sw"]))
    assert np.allclose(gx, ref.permute(0, 2, 3, 1).numpy(), rtol=0, atol=1e-12)


@pytest.mark.parametrize("fmt", [oracle.E4M3, oracle.E2M1])
def test_dequant_1d_inverts_quantize_1d(fmt):
    """Values on the grid come back unchanged through quantize_1d/dequant_1d
    in both directions (each block carries its own power-of-two factor, so a
    scale read from the wrong block shows), and quantize_1d is idempotent."""
    rows, cols = 70, 45
    r, c = np.meshgrid(np.arange(rows), np.arange(cols), indexing="ij")
    base = _int_tensor((rows, cols), 8).numpy()
    for d in (0, 1):
        blk = (r + c // 32) if d == 0 else (r // 32 + c)
        m = (base * np.exp2(blk % 7 - 3)).astype(np.float32)
        codes, scales = oracle.quantize_1d(m, d, fmt)
        assert np.array_equal(oracle.dequant_1d(codes, scales, rows, cols, d, fmt), m)
        x = _rand_tensor((rows, cols), 9 + d)
        codes, scales = oracle.quantize_1d(x, d, fmt)
        dq = oracle.dequant_1d(codes, scales, rows, cols, d, fmt).astype(np.float32)
        c2, s2 = oracle.quantize_1d(dq, d, fmt)
        assert np.array_equal(codes, c2) and np.array_equal(scales, s2)


def _torch_layer(cv, x, w, gy):
    st, pd = (cv["sh"], cv["sw"]), (cv["ph"], cv["pw"])
    y = F.conv2d(x, w, stride=st, padding=pd)
    gx = torch.nn.grad.conv2d_input(x.shape, w, gy, stride=st, padding=pd)
    gw = torch.nn.grad.conv2d_weight(x, w.shape, gy, stride=st, padding=pd)
    return y, gx, gw


@pytest.mark.parametrize("fmt", [oracle.E4M3, oracle.E2M1])
@pytest.mark.parametrize("cv", CONVS[:4], ids=lambda c: f"n{c['n']}c{c['cin']}k{c['kh']}{c['kw']}s{c['sh']}")
def test_naive_gemms_on_lossless_inputs_match_torch(fmt, cv):
    """On small-integer inputs every 1-D quantization is the identity, so the
    comparator's fwd / dgrad / wgrad equal torch's fp64 convolutions."""
    ho, wo = synth.out_hw(cv)
    x = _int_tensor((cv["n"], cv["cin"], cv["h"], cv["w"]), 21)
    w = _int_tensor((cv["cout"], cv["cin"], cv["kh"], cv["kw"]), 22)
    gy = _int_tensor((cv["n"], cv["cout"], ho, wo), 23)
    y_ref, gx_ref, gw_ref = _torch_layer(cv, x, w, gy)
    y, _ = oracle.naive_fwd(cv, fmt, _nhwc(x), _ohwi(w))
    assert np.array_equal(y, _nhwc(y_ref).reshape(-1, cv["cout"]))
    gx, _ = oracle.naive_dgrad(cv, fmt, _nhwc(gy), _ohwi(w))
    assert np.array_equal(gx, _nhwc(gx_ref))
    gw, _ = oracle.naive_wgrad(cv, fmt, _nhwc(gy), _nhwc(x))
    assert np.array_equal(gw, _ohwi(gw_ref))


@pytest.mark.parametrize("fmt", [oracle.E4M3, oracle.E2M1])
def test_naive_gemms_block_along_their_contraction(fmt):
    """One huge element flushes the small ones of its own 1-D block to zero;
    which ones that are shows the direction each GEMM blocks its operand in:
    W along K for fwd and along Cout for dgrad, G_Y along P for wgrad."""
    cv = synth.conv_dict(2, 64, 64, 6, 6, 3, 1, 1)
    ho, wo = synth.out_hw(cv)
    x = _int_tensor((2, 64, 6, 6), 31, 1, 4)
    w = _int_tensor((64, 64, 3, 3), 32, 1, 4)
    gy = _int_tensor((2, 64, ho, wo), 33, 1, 4)
    co0, ci0, a0, b0 = 37, 45, 1, 2
    big = 2.0 ** 20
    wb = w.clone()
    wb[co0, ci0, a0, b0] = big
    k0 = (a0 * 3 + b0) * 64 + ci0
    # fwd: W blocked along K -> same row co0, K block of k0
    wf = wb.permute(0, 2, 3, 1).reshape(64, -1).clone()
    kb = k0 // 32 * 32
    keep = wf[co0, k0].item()
    wf[co0, kb:kb + 32] = 0.0
    wf[co0, k0] = keep
    w_fwd = wf.reshape(64, 3, 3, 64).permute(0, 3, 1, 2)
    y, _ = oracle.naive_fwd(cv, fmt, _nhwc(x), _ohwi(wb))
    y_ref = F.conv2d(x, w_fwd, padding=1)
    assert np.array_equal(y, _nhwc(y_ref).reshape(-1, 64))
    # dgrad: W blocked along Cout -> same column k0, Cout block of co0
    wd = wb.permute(0, 2, 3, 1).reshape(64, -1).clone()
    cb = co0 // 32 * 32
    wd[cb:cb + 32, k0] = 0.0
    wd[co0, k0] = big
    w_dg = wd.reshape(64, 3, 3, 64).permute(0, 3, 1, 2)
    gx, _ = oracle.naive_dgrad(cv, fmt, _nhwc(gy), _ohwi(wb))
    gx_ref = torch.nn.grad.conv2d_input(x.shape, w_dg, gy, padding=1)
    assert np.array_equal(gx, _nhwc(gx_ref))
    # wgrad: G_Y blocked along P = (n, ho, wo) -> same channel, P block of p0
    n0, oh0, ow0, cg = 1, 2, 3, 17
    gyb = gy.clone()
    gyb[n0, cg, oh0, ow0] = big
    gf = gyb.permute(0, 2, 3, 1).reshape(-1, 64).clone()
    p0 = (n0 * ho + oh0) * wo + ow0
    pb = p0 // 32 * 32
    gf[pb:pb + 32, cg] = 0.0
    gf[p0, cg] = big
    gy_wg = gf.reshape(2, ho, wo, 64).permute(0, 3, 1, 2)
    gw, _ = oracle.naive_wgrad(cv, fmt, _nhwc(gyb), _nhwc(x))
    gw_ref = torch.nn.grad.conv2d_weight(x, w.shape, gy_wg, padding=1)
    assert np.array_equal(gw, _ohwi(gw_ref))


def test_naive_step_quantizes_each_tensor_twice():
    """A comparator step (fwd, dgrad, wgrad) quantizes 2|X'| + 2|W| + 2|G_Y|
    elements; at 3x3 s1 p1 that is Table I's baseline count."""
    t1 = _table1()
    cv = synth.conv_dict(32, 32, 32, 8, 8, 3, 1, 1)
    x, w, gy = synth.layer_inputs(cv, 1, kind="unit")
    xn, wn, gn = _nhwc(x), _ohwi(w), _nhwc(gy)
    oracle.counter_reset()
    oracle.naive_fwd(cv, oracle.E4M3, xn, wn)
    oracle.naive_dgrad(cv, oracle.E4M3, gn, wn)
    oracle.naive_wgrad(cv, oracle.E4M3, gn, xn)
    total = oracle.counter_get()
    dac = t1["Dacapo"]
    assert total == dac[0] * x.numel() + dac[1] * w.numel() + dac[2] * gy.numel()


# ------------------------------------------------------------ fused-epilogue activations
def test_act_fn_special_values():
    y = np.array([-3.0, -0.0, 0.0, 0.5, 2.0, 40.0, -40.0])
    assert np.array_equal(oracle.act_fn(y, oracle.FN_NONE), y)
    r = oracle.act_fn(y, oracle.FN_RELU)
    assert np.array_equal(r, [0, 0, 0, 0.5, 2.0, 40.0, 0]) and not np.signbit(r[1])
    s = oracle.act_fn(y, oracle.FN_SILU)
    assert s[2] == 0 and abs(s[3] - 0.5 / (1 + np.exp(-0.5))) < 1e-15
    assert abs(s[5] - 40.0) < 1e-15 and abs(s[6]) < 1e-15          # y and 0 far out on either side
    assert abs(oracle.act_fn(np.array([-1e4]), oracle.FN_SILU)[0]) == 0.0   # exp overflow gives -0


def test_act_grad_is_the_derivative():
    # central differences of act_fn, away from ReLU's kink
    rng = np.random.default_rng(5)
    z = rng.normal(0, 3, 2000)
    z = z[np.abs(z) > 1e-3]
    h = 1e-6
    for fn in (oracle.FN_NONE, oracle.FN_RELU, oracle.FN_SILU):
        fd = (oracle.act_fn(z + h, fn) - oracle.act_fn(z - h, fn)) / (2 * h)
        assert np.max(np.abs(fd - oracle.act_grad(z, fn))) < 1e-7, fn
    g = oracle.act_grad(np.array([0.0, 50.0, -50.0]), oracle.FN_SILU)
    assert g[0] == 0.5 and abs(g[1] - 1) < 1e-15 and abs(g[2]) < 1e-15
    # SiLU' stays in [-0.1, 1.1]: the Lipschitz constant the fused tests use
    zz = np.linspace(-20, 20, 200001)
    gg = oracle.act_grad(zz, oracle.FN_SILU)
    assert gg.max() < 1.1 and gg.min() > -0.1


# ---------------------------------------------------------------- stochastic rounding
def test_philox_known_answers():
    """The counter-based generator against its published known-answer vectors."""
    rows = 0
    with open(os.path.join(GOLDEN, "philox4x32_10_kat.txt")) as f:
        for line in f:
            if not line.strip() or line.startswith("#"):
                continue
            ctr, key, out = [[int(v, 16) for v in part.split()] for part in line.split("|")]
            assert oracle.philox4x32_10(ctr, key).tolist() == out
            rows += 1
    assert rows == 3


def test_sr_bits_follow_the_stated_counter_mapping():
    """Position p takes half (p mod 2) of word (p mod 8) / 2 of the generator
    at counter (p / 8 low, p / 8 high, 0, 0), key = the seed's two halves."""
    for seed in (0, 12345, 2 ** 63 + 977):
        key = [seed & 0xFFFFFFFF, seed >> 32]
        for base in (0, 8 * 1000, 8 * (2 ** 33 + 5)):
            q = base // 8
            w = oracle.philox4x32_10([q & 0xFFFFFFFF, q >> 32, 0, 0], key)
            halves = [(int(w[j // 2]) >> (16 * (j % 2))) & 0xFFFF for j in range(8)]
            assert [oracle.sr_bits(seed, base + j) for j in range(8)] == halves


@pytest.mark.parametrize("fmt", ALL_FMTS)
def test_sr_picks_a_neighbour(fmt):
    """Every stochastic result is one of the two grid values around |x| (by
    enumeration of the grid), the sign is kept, grid values stay exact for
    any random bits, and magnitudes at or above the maximum saturate."""
    grid = [g for _, g in _grid(fmt)]
    rng = np.random.default_rng(fmt + 40)
    top = MAXV[fmt]
    for v in np.concatenate([rng.random(400) * top, rng.random(200) * grid[2] * 2]):
        lo = max(g for g in grid if g <= v)
        hi = min([g for g in grid if g > v] or [top])
        for r in rng.integers(0, 65536, 6):
            for s in (v, -v):
                d = oracle.decode(oracle.encode_sr(s, fmt, int(r)), fmt)
                assert abs(d) in (lo, hi) and (d == 0 or math.copysign(1, d) == math.copysign(1, s))
    for g in grid:
        for r in (0, 1, 12345, 65535):
            assert oracle.decode(oracle.encode_sr(g, fmt, r), fmt) == g
            assert oracle.decode(oracle.encode_sr(-g, fmt, r), fmt) == -g
    for v in (top * 1.01, top * 3, 1e30):
        assert oracle.decode(oracle.encode_sr(v, fmt, 0), fmt) == top


@pytest.mark.parametrize("fmt", ALL_FMTS)
def test_sr_is_exactly_unbiased(fmt):
    """Over all 2^16 values of the random bits, x rounds up exactly
    ceil(frac * 2^16) times; when frac is a multiple of 2^-16 the mean of the
    rounded values is x itself."""
    grid = [g for _, g in _grid(fmt)]
    m = len(grid) // 2
    cases = [(grid[3], grid[4], 12345 / 65536), (grid[1], grid[2], 0.5), (grid[-3], grid[-2], 1 / 65536),
             (grid[-2], grid[-1], 0.7), (grid[m], grid[m + 1], 0.25 + 3 / 65536)]
    for lo, hi, frac in cases:
        x = lo + frac * (hi - lo)
        ups = sum(oracle.decode(oracle.encode_sr(x, fmt, r), fmt) == hi for r in range(65536))
        assert ups == math.ceil(frac * 65536)
        if (frac * 65536).is_integer():
            assert lo + ups / 65536 * (hi - lo) == x


@pytest.mark.parametrize("fmt", [oracle.E4M3, oracle.E2M1, oracle.E3M2])
def test_quantize_sr_tensor(fmt):
    """The tensor quantizer with stochastic rounding: scales are the
    round-to-nearest ones; every element is a neighbour of its exact scaled
    value; the same seed reproduces the codes and another seed changes them;
    and the mean over 256 seeds of the dequantized tensor approaches x within
    four standard errors of the rounding noise (which is at most half a
    quantum per element)."""
    n, c, h, w = 32, 40, 2, 3
    x = _rand_tensor((n, c, h, w), 13)
    rc, rs = oracle.quantize(x, oracle.NCHW, oracle.ACT, fmt, n, c, h, w)
    c1, s1 = oracle.quantize_sr(x, oracle.NCHW, oracle.ACT, fmt, n, c, h, w, 7)
    c1b, _ = oracle.quantize_sr(x, oracle.NCHW, oracle.ACT, fmt, n, c, h, w, 7)
    c2, s2 = oracle.quantize_sr(x, oracle.NCHW, oracle.ACT, fmt, n, c, h, w, 8)
    assert np.array_equal(s1, rs) and np.array_equal(s2, rs)
    assert np.array_equal(c1, c1b) and not np.array_equal(c1, c2)
    xd = x.astype(np.float64)
    acc = np.zeros_like(xd)
    seeds = 256
    for seed in range(seeds):
        cs, ss = oracle.quantize_sr(x, oracle.NCHW, oracle.ACT, fmt, n, c, h, w, 1000 + seed)
        acc += oracle.dequant(cs, ss, oracle.ACT, fmt, n, c, h, w)
    mean = acc / seeds
    # block scales, and the grid spacing q around each scaled element (from
    # the enumerated grid): the rounding noise has standard deviation <= q / 2
    sc = np.zeros_like(xd)
    for hh in range(h):
        for ww in range(w):
            for cb in range(2):
                sc[:, cb * 32:(cb + 1) * 32, hh, ww] = 2.0 ** (int(rs[(hh * w + ww) * 2 + cb]) - 127)
    grid = np.array([g for _, g in _grid(fmt)])
    a = np.abs(xd) / sc
    ok = a < MAXV[fmt]                      # saturated elements are not unbiased
    k = np.clip(np.searchsorted(grid, a, side="right"), 1, len(grid) - 1)
    q = (grid[k] - grid[k - 1]) * sc
    bound = 4 * (q / 2) / np.sqrt(seeds)
    assert np.all(np.abs(mean - xd)[ok] <= bound[ok])


# ---------------------------------------------------------------- NVFP (Eqs. (4)-(6))
def test_nvfp_hand_worked_blocks():
    x = np.zeros((8, 16, 1, 1), dtype=np.float32)
    x[0:3, 0, 0, 0] = [2688.0, 224.0, -1344.0]
    x[0:5, 8, 0, 0] = [1.1, 0.5, 0.46875, -0.1, 0.05]
    codes, scales, t = oracle.nvfp_quantize(x, oracle.NCHW, oracle.ACT, oracle.E2M1, 8, 16, 1, 1)
    rows = []
    with open(os.path.join(GOLDEN, "nvfp_blocks.txt")) as f:
        for line in f:
            if line.strip() and not line.startswith("#"):
                rows.append([p.strip() for p in line.split("|")])
    assert len(rows) == 2
    for tv, blk, bcode, ecodes in rows:
        assert t == float(tv)
        b = int(blk)
        # scales [Np/Bn][H][W][Cp/8][Bn/8]: Cp = 32 -> 4 channel blocks, Bn = 8 -> 1 sample block
        assert scales[b] == int(bcode, 16)
        want = [int(_parse_num(v)) for v in ecodes.split()]
        # code position of (channel 8 b, sample j) is (8 b) * 8 + j
        assert [_code_at(codes, oracle.E2M1, 8 * b * 8 + j) for j in range(len(want))] == want
    assert scales[2:].tolist() == [0, 0]                  # padded channels 16-31


def test_nvfp_element_step_is_a_correctly_rounded_quotient():
    """Eq. (6)'s element step divides x by the fp32 product B T.  Elements
    placed exactly on a rounding tie of the E2M1 grid (x = m B with m a
    midpoint of two grid values, so x / (B T) = m exactly when T = 1) must
    take the tie's even code; a route through the reciprocal, x * fl(1 / BT),
    lands a little above or below m and picks the other neighbour for some of
    them.  The test first checks, in numpy float32 arithmetic, that the
    reciprocal route does move at least a few of these elements, so it pins
    the quotient."""
    mids = [0.25, 0.75, 1.25, 1.75, 2.5, 3.5, 5.0]
    even = {0.25: 0, 0.75: 2, 1.25: 2, 1.75: 4, 2.5: 4, 3.5: 6, 5.0: 6}     # RNE: the even code of the two
    bs = [m / 8.0 * 2.0 ** e for m in range(9, 16) for e in (-3, 0, 4)]     # E4M3 block scales, 1.xxx * 2^e
    nblk = len(bs) + 1
    x = np.zeros((8, 8 * nblk, 1, 1), dtype=np.float32)
    x[0, 0, 0, 0] = 2688.0                        # block 0: amax = 448 * 6, so T = 1
    for k, b in enumerate(bs):
        ch = 8 * (k + 1)
        x[0, ch, 0, 0] = 6.0 * b                  # block max: B = CastE4M3(6 b / (1 * 6)) = b exactly
        for i, m in enumerate(mids):
            x[1 + i, ch, 0, 0] = m * b            # exact in fp32 (b has 4 significant bits)
    codes, scales, t = oracle.nvfp_quantize(x, oracle.NCHW, oracle.ACT, oracle.E2M1, 8, 8 * nblk, 1, 1)
    assert t == 1.0
    moved = 0
    for k, b in enumerate(bs):
        blk = k + 1
        assert float(oracle.decode(int(scales[blk]), oracle.E4M3)) == b
        for i, m in enumerate(mids):
            pos = 8 * blk * 8 + 1 + i             # code position of (channel 8 blk, sample 1 + i)
            assert _code_at(codes, oracle.E2M1, pos) == even[m], (b, m)
            recip = np.float32(np.float32(m * b) * (np.float32(1.0) / np.float32(b)))
            moved += oracle.encode(float(recip), oracle.E2M1) != even[m]
    assert moved >= 5, moved                      # the reciprocal route would fail this test


@pytest.mark.parametrize("fmt", ALL_FMTS)
def test_nvfp_block_scale_cast_matches_torch(fmt):
    """Eq. (5)'s CastE4M3 of every block against torch's float8 E4M3 cast of
    the same fp32 ratio (after clamping to the E4M3 maximum)."""
    n, c, h, w = 32, 64, 3, 2
    x = _rand_tensor((n, c, h, w), 17, spread=4.0)
    codes, scales, t = oracle.nvfp_quantize(x, oracle.NCHW, oracle.ACT, fmt, n, c, h, w)
    tm = np.float32(t) * np.float32(MAXV[fmt])
    ratios = []
    for hh in range(h):
        for ww in range(w):
            for cb8 in range(c // 8):
                for sb8 in range(n // 32 * 4):
                    blk = x[sb8 * 8:(sb8 + 1) * 8, cb8 * 8:(cb8 + 1) * 8, hh, ww]
                    ratios.append(np.float32(np.abs(blk).max()) / tm)
    ref = torch.clamp(torch.tensor(np.array(ratios, dtype=np.float32)), max=448.0).to(torch.float8_e4m3fn)
    # oracle order: [H][W][Cp/8][Bn/8] for one batch group
    assert scales.tolist() == ref.view(torch.uint8).tolist()


@pytest.mark.parametrize("fmt", ALL_FMTS)
def test_nvfp_invariants(fmt):
    """Power-of-two equivariance (codes and block scales unchanged, T scaled
    exactly), source layouts agree, and every dequantized element lies
    within one element-grid step (times B T) of x."""
    n, c, h, w = 32, 40, 2, 3
    x = _rand_tensor((n, c, h, w), 19)
    codes, scales, t = oracle.nvfp_quantize(x, oracle.NCHW, oracle.ACT, fmt, n, c, h, w)
    for k in (-7, 5):
        c2, s2, t2 = oracle.nvfp_quantize(x * np.float32(2.0 ** k), oracle.NCHW, oracle.ACT, fmt, n, c, h, w)
        assert np.array_equal(c2, codes) and np.array_equal(s2, scales) and t2 == t * 2.0 ** k
    xt = torch.from_numpy(x)
    for lay, arr in ((oracle.NHWC, xt.permute(0, 2, 3, 1).contiguous().numpy()),
                     (oracle.CBF, synth.nchw_to_cbf(xt, 32).numpy())):
        c3, s3, t3 = oracle.nvfp_quantize(arr, lay, oracle.ACT, fmt, n, c, h, w)
        assert np.array_equal(c3, codes) and np.array_equal(s3, scales) and t3 == t
    d = oracle.nvfp_dequant(codes, scales, t, oracle.ACT, fmt, n, c, h, w)
    grid = np.array([g for _, g in _grid(fmt)])
    bt = np.zeros_like(d)
    for hh in range(h):
        for ww in range(w):
            for cb8 in range(c // 8 + 1):
                for sb8 in range(4):
                    sc = float(oracle.decode(int(scales[((hh * w + ww) * 8 + cb8) * 4 + sb8]), oracle.E4M3))
                    bt[sb8 * 8:(sb8 + 1) * 8, cb8 * 8:(cb8 + 1) * 8, hh, ww] = sc * t
    a = np.abs(x.astype(np.float64)) / bt
    k = np.clip(np.searchsorted(grid, a, side="right"), 1, len(grid) - 1)
    step = (grid[k] - grid[k - 1]) * bt
    clip = np.maximum(np.abs(x) - MAXV[fmt] * bt, 0)          # E4M3 rounding of B can clip the block max
    assert np.all(np.abs(d - x) <= step * (1 + 1e-6) + clip)


def test_nvfp_special_tensors():
    z = np.zeros((32, 32, 1, 2), dtype=np.float32)
    c, s, t = oracle.nvfp_quantize(z, oracle.NCHW, oracle.ACT, oracle.E2M1, 32, 32, 1, 2)
    assert t == 0.0 and not c.any() and not s.any()
    z[3, 4, 0, 1] = float("nan")
    c, s, t = oracle.nvfp_quantize(z + 1, oracle.NCHW, oracle.ACT, oracle.E2M1, 32, 32, 1, 2)
    assert math.isnan(t) and not c.any() and set(s.tolist()) == {0x7F}
    assert oracle.load().o_nvfp_scales_bytes(oracle.ACT, oracle.E2M1, 4, 32, 1, 1) < 0   # Bn = 4: no 8x8 blocks
    assert oracle.load().o_nvfp_scales_bytes(oracle.ACT, oracle.E2M1, 64, 40, 3, 3) == 2 * 9 * 8 * 4


@pytest.mark.parametrize("fmt", [oracle.E2M1, oracle.E2M3, oracle.E3M2])
def test_nvfp_reduces_error_against_e8m0_blocks(fmt):
    """Sec. III-A: the two-level NVFP scaling has lower quantization error
    than power-of-two block scales.  Mean squared error of NVFP (8x8 blocks,
    E4M3 scales) against the E8M0 32x32-block quantizer, on N(0,1)
    activations and on heavy-tailed gradients."""
    n, c, h, w = 32, 64, 8, 8
    for x in (np.random.default_rng(3).standard_normal((n, c, h, w)).astype(np.float32),
              _rand_tensor((n, c, h, w), 23, spread=3.0)):
        cn, sn, t = oracle.nvfp_quantize(x, oracle.NCHW, oracle.ACT, fmt, n, c, h, w)
        mse_nv = np.mean((oracle.nvfp_dequant(cn, sn, t, oracle.ACT, fmt, n, c, h, w) - x) ** 2)
        cm, sm = oracle.quantize(x, oracle.NCHW, oracle.ACT, fmt, n, c, h, w)
        mse_mx = np.mean((oracle.dequant(cm, sm, oracle.ACT, fmt, n, c, h, w) - x) ** 2)
        assert mse_nv < mse_mx
