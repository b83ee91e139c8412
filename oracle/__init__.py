"""CPU oracle for quantize-once MX convolution (MicroQonv).

TEST INFRASTRUCTURE ONLY.  Only the test suite, ``__graft_entry__.smoke()``
and the CPU-baseline leg of ``bench.py`` may import this package.  The GPU
library never links, loads or calls it, and it shares no code with it.

This module is a thin ctypes layer over ``mxoracle.c`` (plain fp64 loops, see
that file's header for the definitions and the passages of the paper each one
follows).  ``build()`` compiles it with gcc; ``load()`` builds on first use.

Parity: every function here is pinned by the ``-m "not gpu"`` tests in
``tests/test_oracle_pins.py`` (hand-worked blocks, brute-force element
rounding, torch's float8 cast, torch's fp64 convolutions, the brute-force
direct convolutions, invariants) and ``tests/test_oracle_net.py`` (the
network-step functions against torch.cat, F.interpolate and autograd; the
bf16 rounding against hand-worked ties and torch's bfloat16 cast).
Nothing here is "parity unpinned".
"""
import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "mxoracle.c")
_LIB = os.path.join(_HERE, "libmxoracle.so")

E4M3, E2M1, E2M3, E3M2 = 0, 1, 2, 3
BITS = {E4M3: 8, E2M1: 4, E2M3: 6, E3M2: 6}
NCHW, NHWC, CBF = 0, 1, 2
ACT, WEIGHT = 0, 1

_lib = None


def build():
    """Compile the oracle (plain C, -O2, OpenMP over the outermost loops)."""
    cmd = ["gcc", "-O2", "-fopenmp", "-fPIC", "-shared", "-std=c11",
           "-o", _LIB + ".tmp", _SRC, "-lm"]
    subprocess.check_call(cmd)
    os.replace(_LIB + ".tmp", _LIB)


def load():
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(_LIB) or os.path.getmtime(_LIB) < os.path.getmtime(_SRC):
        build()
    lib = ctypes.CDLL(_LIB)
    P = ctypes.c_void_p
    i32, i64, dbl = ctypes.c_int, ctypes.c_int64, ctypes.c_double
    sig = {
        "o_encode": (i32, [dbl, i32]),
        "o_decode": (dbl, [i32, i32]),
        "o_scale_value": (dbl, [i32]),
        "o_scale_code": (i32, [dbl, i32]),
        "o_codes_bytes": (i64, [i32, i32, i32, i32, i32, i32]),
        "o_scales_bytes": (i64, [i32, i32, i32, i32, i32, i32]),
        "o_quantize": (i32, [P, i32, i32, i32, i32, i32, i32, i32, P, P]),
        "o_quantize_sr": (i32, [P, i32, i32, i32, i32, i32, i32, i32, ctypes.c_uint64, P, P]),
        "o_philox4x32_10": (None, [P, P, P]),
        "o_sr_bits": (ctypes.c_uint, [ctypes.c_uint64, i64]),
        "o_encode_sr": (i32, [dbl, i32, ctypes.c_uint]),
        "o_nvfp_scales_bytes": (i64, [i32, i32, i32, i32, i32, i32]),
        "o_nvfp_quantize": (i32, [P, i32, i32, i32, i32, i32, i32, i32, P, P, P]),
        "o_nvfp_dequant": (i32, [P, P, ctypes.c_float, i32, i32, i32, i32, i32, i32, P]),
        "o_dequant": (i32, [P, P, i32, i32, i32, i32, i32, i32, P]),
        "o_conv_out": (i32, [P, P, P]),
        "o_im2col_cbf": (i32, [P, i32, P, P, P, P]),
        "o_im2col_codes_bytes": (i64, [P, i32]),
        "o_im2col_scales_bytes": (i64, [P, i32]),
        "o_fwd": (i32, [P, i32, i32, P, P, P, P, P, P]),
        "o_wgrad": (i32, [P, i32, i32, P, P, P, P, P, P]),
        "o_dgrad": (i32, [P, i32, i32, P, P, P, P, P, P]),
        "o_direct_fwd": (i32, [P, P, P, P]),
        "o_direct_dgrad": (i32, [P, P, P, P]),
        "o_direct_wgrad": (i32, [P, P, P, P]),
        "o_fwd_at": (i32, [P, i32, i32, P, P, P, P, P, i64, P, P]),
        "o_dgrad_at": (i32, [P, i32, i32, P, P, P, P, P, i64, P, P]),
        "o_wgrad_at": (i32, [P, i32, i32, P, P, P, P, P, i64, P, P]),
        "o_quantize_1d": (i32, [P, i64, i64, i32, i32, P, P]),
        "o_dequant_1d": (i32, [P, P, i64, i64, i32, i32, P]),
        "o_naive_im2col": (i32, [P, P, P]),
        "o_naive_col2im": (i32, [P, P, P]),
        "o_counter_get": (i64, []),
        "o_counter_reset": (None, []),
        "o_set_threads": (None, [i32]),
        "o_get_threads": (i32, []),
    }
    for name, (res, args) in sig.items():
        fn = getattr(lib, name)
        fn.restype = res
        fn.argtypes = args
    _lib = lib
    return lib


def _ptr(a):
    return a.ctypes.data_as(ctypes.c_void_p)


def _check(rc, what):
    if rc != 0:
        raise ValueError(f"oracle {what} failed with code {rc}")


def _conv_params(conv):
    """conv: dict with n, cin, cout, h, w, kh, kw, sh, sw, ph, pw."""
    keys = ("n", "cin", "cout", "h", "w", "kh", "kw", "sh", "sw", "ph", "pw")
    return np.array([int(conv[k]) for k in keys], dtype=np.int32)


def set_threads(t):
    load().o_set_threads(int(t))


def get_threads():
    return load().o_get_threads()


def encode(v, fmt):
    return load().o_encode(float(v), fmt)


def decode(code, fmt):
    return load().o_decode(int(code), fmt)


def scale_code(amax, fmt):
    return load().o_scale_code(float(amax), fmt)


def codes_bytes(role, fmt, n, c, h, w):
    return load().o_codes_bytes(role, fmt, n, c, h, w)


def scales_bytes(role, fmt, n, c, h, w):
    return load().o_scales_bytes(role, fmt, n, c, h, w)


def quantize(src, layout, role, fmt, n, c, h, w):
    """src: float32 array holding the logical (n, c, h, w) tensor in `layout`.
    Returns (codes uint8, scales uint8) in the MX-CBF layout."""
    lib = load()
    src = np.ascontiguousarray(src, dtype=np.float32)
    nb = lib.o_codes_bytes(role, fmt, n, c, h, w)
    ns = lib.o_scales_bytes(role, fmt, n, c, h, w)
    if nb < 0:
        raise ValueError("bad geometry")
    codes = np.zeros(nb, dtype=np.uint8)
    scales = np.zeros(ns, dtype=np.uint8)
    _check(lib.o_quantize(_ptr(src), layout, role, fmt, n, c, h, w, _ptr(codes), _ptr(scales)),
           "quantize")
    return codes, scales


def quantize_sr(src, layout, role, fmt, n, c, h, w, seed):
    """quantize() with stochastic rounding of the elements under `seed`."""
    lib = load()
    src = np.ascontiguousarray(src, dtype=np.float32)
    nb = lib.o_codes_bytes(role, fmt, n, c, h, w)
    ns = lib.o_scales_bytes(role, fmt, n, c, h, w)
    if nb < 0:
        raise ValueError("bad geometry")
    codes = np.zeros(nb, dtype=np.uint8)
    scales = np.zeros(ns, dtype=np.uint8)
    _check(lib.o_quantize_sr(_ptr(src), layout, role, fmt, n, c, h, w, int(seed) & (2 ** 64 - 1),
                             _ptr(codes), _ptr(scales)), "quantize_sr")
    return codes, scales


def nvfp_quantize(src, layout, role, fmt, n, c, h, w):
    """Eqs. (4)-(6) literally: returns (codes, E4M3 block scales, T)."""
    lib = load()
    src = np.ascontiguousarray(src, dtype=np.float32)
    nb = lib.o_codes_bytes(role, fmt, n, c, h, w)
    ns = lib.o_nvfp_scales_bytes(role, fmt, n, c, h, w)
    if nb < 0 or ns < 0:
        raise ValueError("bad geometry")
    codes = np.zeros(nb, dtype=np.uint8)
    scales = np.zeros(ns, dtype=np.uint8)
    t = np.zeros(1, dtype=np.float32)
    _check(lib.o_nvfp_quantize(_ptr(src), layout, role, fmt, n, c, h, w, _ptr(codes), _ptr(scales), _ptr(t)),
           "nvfp_quantize")
    return codes, scales, float(t[0])


def nvfp_dequant(codes, scales, tscale, role, fmt, n, c, h, w):
    out = np.zeros((n, c, h, w), dtype=np.float64)
    _check(load().o_nvfp_dequant(_ptr(np.ascontiguousarray(codes)), _ptr(np.ascontiguousarray(scales)),
                                 float(tscale), role, fmt, n, c, h, w, _ptr(out)), "nvfp_dequant")
    return out


def philox4x32_10(ctr, key):
    """Philox4x32-10 of a 4-word counter under a 2-word key."""
    c = np.ascontiguousarray(ctr, dtype=np.uint32)
    k = np.ascontiguousarray(key, dtype=np.uint32)
    out = np.zeros(4, dtype=np.uint32)
    load().o_philox4x32_10(_ptr(c), _ptr(k), _ptr(out))
    return out


def sr_bits(seed, pos):
    return load().o_sr_bits(int(seed) & (2 ** 64 - 1), int(pos))


def encode_sr(v, fmt, r):
    return load().o_encode_sr(float(v), fmt, int(r))


def dequant(codes, scales, role, fmt, n, c, h, w):
    lib = load()
    out = np.zeros((n, c, h, w), dtype=np.float64)
    codes = np.ascontiguousarray(codes, dtype=np.uint8)
    scales = np.ascontiguousarray(scales, dtype=np.uint8)
    _check(lib.o_dequant(_ptr(codes), _ptr(scales), role, fmt, n, c, h, w, _ptr(out)), "dequant")
    return out


def conv_out(conv):
    p = _conv_params(conv)
    ho = ctypes.c_int()
    wo = ctypes.c_int()
    _check(load().o_conv_out(_ptr(p), ctypes.byref(ho), ctypes.byref(wo)), "conv_out")
    return ho.value, wo.value


def im2col_cbf(conv, fmt, xcodes, xscales):
    lib = load()
    p = _conv_params(conv)
    cb = lib.o_im2col_codes_bytes(_ptr(p), fmt)
    sb = lib.o_im2col_scales_bytes(_ptr(p), fmt)
    cc = np.zeros(cb, dtype=np.uint8)
    cs = np.zeros(sb, dtype=np.uint8)
    _check(lib.o_im2col_cbf(_ptr(p), fmt, _ptr(np.ascontiguousarray(xcodes)),
                            _ptr(np.ascontiguousarray(xscales)), _ptr(cc), _ptr(cs)), "im2col")
    return cc, cs


def _fmts(fmt):
    """One element format for both operands, or a pair (first operand's,
    second operand's), in the argument order of the call."""
    if isinstance(fmt, (tuple, list)):
        return int(fmt[0]), int(fmt[1])
    return int(fmt), int(fmt)


def _gemm(name, conv, fmt, a, b, shape):
    lib = load()
    p = _conv_params(conv)
    out = np.zeros(shape, dtype=np.float64)
    sabs = np.zeros(shape, dtype=np.float64)
    (ac, as_), (bc, bs) = a, b
    _check(getattr(lib, name)(_ptr(p), *_fmts(fmt), _ptr(np.ascontiguousarray(ac)),
                              _ptr(np.ascontiguousarray(as_)), _ptr(np.ascontiguousarray(bc)),
                              _ptr(np.ascontiguousarray(bs)), _ptr(out), _ptr(sabs)), name)
    return out, sabs


def fwd(conv, fmt, w, x):
    """w, x: (codes, scales) pairs; fmt: one format, or (W's, X's).
    Returns (Y NCHW fp64, sum|products|)."""
    ho, wo = conv_out(conv)
    return _gemm("o_fwd", conv, fmt, w, x, (conv["n"], conv["cout"], ho, wo))


def dgrad(conv, fmt, w, gy):
    """fmt: one format, or (W's, G_Y's)."""
    return _gemm("o_dgrad", conv, fmt, w, gy, (conv["n"], conv["cin"], conv["h"], conv["w"]))


def wgrad(conv, fmt, gy, x):
    """fmt: one format, or (G_Y's, X's)."""
    return _gemm("o_wgrad", conv, fmt, gy, x, (conv["cout"], conv["cin"], conv["kh"], conv["kw"]))


def _at(name, conv, fmt, a, b, idx):
    lib = load()
    p = _conv_params(conv)
    idx = np.ascontiguousarray(idx, dtype=np.int32).reshape(-1, 4)
    out = np.zeros(len(idx), dtype=np.float64)
    sabs = np.zeros(len(idx), dtype=np.float64)
    (ac, as_), (bc, bs) = a, b
    _check(getattr(lib, name)(_ptr(p), *_fmts(fmt), _ptr(np.ascontiguousarray(ac)),
                              _ptr(np.ascontiguousarray(as_)), _ptr(np.ascontiguousarray(bc)),
                              _ptr(np.ascontiguousarray(bs)), _ptr(idx), len(idx), _ptr(out),
                              _ptr(sabs)), name)
    return out, sabs


def fwd_at(conv, fmt, w, x, idx):
    """idx rows (n, co, ho, wo)."""
    return _at("o_fwd_at", conv, fmt, w, x, idx)


def dgrad_at(conv, fmt, w, gy, idx):
    """idx rows (n, ci, h, w)."""
    return _at("o_dgrad_at", conv, fmt, w, gy, idx)


def wgrad_at(conv, fmt, gy, x, idx):
    """idx rows (co, ci, kh, kw)."""
    return _at("o_wgrad_at", conv, fmt, gy, x, idx)


def direct_fwd(conv, w, x):
    ho, wo = conv_out(conv)
    y = np.zeros((conv["n"], conv["cout"], ho, wo), dtype=np.float64)
    _check(load().o_direct_fwd(_ptr(_conv_params(conv)), _ptr(np.ascontiguousarray(w, np.float64)),
                               _ptr(np.ascontiguousarray(x, np.float64)), _ptr(y)), "direct_fwd")
    return y


def direct_dgrad(conv, w, gy):
    gx = np.zeros((conv["n"], conv["cin"], conv["h"], conv["w"]), dtype=np.float64)
    _check(load().o_direct_dgrad(_ptr(_conv_params(conv)), _ptr(np.ascontiguousarray(w, np.float64)),
                                 _ptr(np.ascontiguousarray(gy, np.float64)), _ptr(gx)), "direct_dgrad")
    return gx


def direct_wgrad(conv, gy, x):
    gw = np.zeros((conv["cout"], conv["cin"], conv["kh"], conv["kw"]), dtype=np.float64)
    _check(load().o_direct_wgrad(_ptr(_conv_params(conv)), _ptr(np.ascontiguousarray(gy, np.float64)),
                                 _ptr(np.ascontiguousarray(x, np.float64)), _ptr(gw)), "direct_wgrad")
    return gw


def quantize_1d(m, direction, fmt):
    """Naive comparator's quantizer on a 2-D fp32 matrix: 1-D blocks of 32
    along rows (direction 0) or columns (direction 1)."""
    lib = load()
    m = np.ascontiguousarray(m, dtype=np.float32)
    rows, cols = m.shape
    bits = BITS[fmt]
    codes = np.zeros((rows * cols * bits + 7) // 8, dtype=np.uint8)
    if direction == 0:
        scales = np.zeros(rows * ((cols + 31) // 32), dtype=np.uint8)
    else:
        scales = np.zeros(((rows + 31) // 32) * cols, dtype=np.uint8)
    _check(lib.o_quantize_1d(_ptr(m), rows, cols, direction, fmt, _ptr(codes), _ptr(scales)),
           "quantize_1d")
    return codes, scales


def dequant_1d(codes, scales, rows, cols, direction, fmt):
    """Fake quantization of a quantize_1d result: fp64 [rows][cols]."""
    out = np.zeros((rows, cols), dtype=np.float64)
    _check(load().o_dequant_1d(_ptr(np.ascontiguousarray(codes)), _ptr(np.ascontiguousarray(scales)),
                               rows, cols, direction, fmt, _ptr(out)), "dequant_1d")
    return out


def naive_im2col(conv, x_nhwc):
    """fp32 im2col of an NHWC tensor: [P][K], P = (n, ho, wo), K = (kh, kw, ci)."""
    p = _conv_params(conv)
    ho, wo = conv_out(conv)
    x = np.ascontiguousarray(x_nhwc, dtype=np.float32)
    col = np.zeros((conv["n"] * ho * wo, conv["kh"] * conv["kw"] * conv["cin"]), dtype=np.float32)
    _check(load().o_naive_im2col(_ptr(p), _ptr(x), _ptr(col)), "naive_im2col")
    return col


def naive_col2im(conv, gcol):
    """Scatter-add of a [P][K] fp64 matrix back to an NHWC tensor."""
    p = _conv_params(conv)
    g = np.ascontiguousarray(gcol, dtype=np.float64)
    gx = np.zeros((conv["n"], conv["h"], conv["w"], conv["cin"]), dtype=np.float64)
    _check(load().o_naive_col2im(_ptr(p), _ptr(g), _ptr(gx)), "naive_col2im")
    return gx


def _fake_1d(m, direction, fmt):
    m = np.ascontiguousarray(m, dtype=np.float32)
    codes, scales = quantize_1d(m, direction, fmt)
    return dequant_1d(codes, scales, m.shape[0], m.shape[1], direction, fmt)


# The naive comparator's three GEMMs (Sec. III-C / Table I baseline), in the
# channels-last GEMM form: X, G_Y and G_X are NHWC, W and G_W are OHWI
# ([Cout][K]).  Each operand is quantized with 1-D blocks along its GEMM's
# contraction dimension, so every tensor is quantized twice per step.  Each
# returns (result, sum of absolute products) in fp64.
def naive_fwd(conv, fmt, x_nhwc, w_ohwi):
    """Y [P][Cout] = X'[P][K] W[Cout][K]^T, X' and W blocked along K."""
    a = _fake_1d(naive_im2col(conv, x_nhwc), 0, fmt)
    b = _fake_1d(np.asarray(w_ohwi, dtype=np.float32).reshape(conv["cout"], -1), 0, fmt)
    return a @ b.T, np.abs(a) @ np.abs(b).T


def naive_dgrad(conv, fmt, gy_nhwc, w_ohwi):
    """G_X' [P][K] = G_Y[P][Cout] W[Cout][K], both blocked along Cout; then col2im."""
    cout = conv["cout"]
    a = _fake_1d(np.asarray(gy_nhwc, dtype=np.float32).reshape(-1, cout), 0, fmt)
    b = _fake_1d(np.asarray(w_ohwi, dtype=np.float32).reshape(cout, -1), 1, fmt)
    return naive_col2im(conv, a @ b), naive_col2im(conv, np.abs(a) @ np.abs(b))


def naive_wgrad(conv, fmt, gy_nhwc, x_nhwc):
    """G_W [Cout][K] = G_Y[P][Cout]^T X'[P][K], both blocked along P."""
    a = _fake_1d(np.asarray(gy_nhwc, dtype=np.float32).reshape(-1, conv["cout"]), 1, fmt)
    b = _fake_1d(naive_im2col(conv, x_nhwc), 1, fmt)
    return a.T @ b, np.abs(a).T @ np.abs(b)


def counter_get():
    return load().o_counter_get()


def counter_reset():
    load().o_counter_reset()


# ---------------------------------------------------------------- fused epilogues
FN_NONE, FN_RELU, FN_SILU = 0, 1, 2


def act_fn(y, fn):
    """The activation between two convolutions, in fp64: identity, ReLU
    (y if y > 0 else 0; the ResNets of Sec. VI) or SiLU y / (1 + exp(-y))
    (the YOLO networks of Sec. VI).  The fused forward epilogue quantizes
    act_fn(Y) as the next layer's X, once (Sec. IV-B, Sec. IV-C)."""
    y = np.asarray(y, dtype=np.float64)
    if fn == FN_NONE:
        return y.copy()
    if fn == FN_RELU:
        return np.where(y > 0, y, 0.0)
    with np.errstate(over="ignore"):
        return y / (1.0 + np.exp(-y))


def act_grad(z, fn):
    """Derivative of act_fn at the pre-activation z, in fp64: 1, [z > 0], or
    for SiLU s (1 + z (1 - s)) with s = 1 / (1 + exp(-z)).  The fused
    input-gradient epilogue quantizes G_X * act_grad(z) as the previous
    layer's G_Y."""
    z = np.asarray(z, dtype=np.float64)
    if fn == FN_NONE:
        return np.ones_like(z)
    if fn == FN_RELU:
        return (z > 0).astype(np.float64)
    with np.errstate(over="ignore"):
        s = 1.0 / (1.0 + np.exp(-z))
    return s * (1.0 + z * (1.0 - s))


# ---------------------------------------------------------------- bf16 master tensors
def round_bf16(x):
    """fp32 -> bf16 (8 significand bits: the fp32 sign, exponent and top 7
    fraction bits), round to nearest with ties to even, returned as fp32.
    Written as the rule: of the two bf16 neighbours -- the fp32 pattern with
    its low 16 bits cleared, and the next bf16 away from zero -- take the one
    the dropped 16 bits are nearer to; on an exact half, the one whose last
    kept bit is 0.  The step past the largest finite bf16 is infinity.  A NaN
    stays a NaN.  Full-precision tensors between layers are held in bf16
    when a network keeps bf16 master tensors."""
    a = np.ascontiguousarray(np.asarray(x, dtype=np.float32))
    u = a.view(np.uint32).astype(np.int64)
    lo = u & 0xFFFF0000
    dropped = u & 0xFFFF
    odd = (lo >> 16) & 1
    up = (dropped > 0x8000) | ((dropped == 0x8000) & (odd == 1))
    r = np.where(up, lo + 0x10000, lo)
    nan = np.isnan(a)
    out = (r & 0xFFFFFFFF).astype(np.uint32).view(np.float32).copy()
    out[nan] = np.float32("nan")
    return out


# ---------------------------------------------------------------- network steps
def _bn(n):
    return 32 if n >= 32 else n


def concat_cbf(parts, fmt, n, h, w):
    """Channel concatenation of MX-CBF activations on whole blocks, each part
    optionally upsampled 2x by nearest neighbour, written out as loops over
    (group, pixel, part, block).  parts: tuples (codes, scales, c, up) of MX
    tensors (n, c, h_k, w_k) with (h_k, w_k) = (h/2, w/2) when up else (h, w).
    A block is 32 channels x Bn samples at one pixel (Sec. IV-A, IV-B), so
    the result copies codes and scales and requantizes nothing.  Returns the
    codes and scales of (n, 32 * sum ceil(c_k / 32), h, w)."""
    bn = _bn(n)
    ng = -(-n // bn)
    bb = 32 * bn * BITS[fmt] // 8
    ncbs = [-(-c // 32) for _, _, c, _ in parts]
    tot = sum(ncbs)
    out_c = np.zeros((ng, h, w, tot, bb), np.uint8)
    out_s = np.zeros((ng, h, w, tot), np.uint8)
    srcs = []
    for (codes, scales, c, up), ncb in zip(parts, ncbs):
        hk, wk = (h // 2, w // 2) if up else (h, w)
        cd = np.asarray(codes, np.uint8)[:ng * hk * wk * ncb * bb].reshape(ng, hk, wk, ncb, bb)
        sc = np.asarray(scales, np.uint8)[:ng * hk * wk * ncb].reshape(ng, hk, wk, ncb)
        srcs.append((cd, sc, ncb, up))
    for g in range(ng):
        for y in range(h):
            for x in range(w):
                off = 0
                for cd, sc, ncb, up in srcs:
                    sy, sx = (y // 2, x // 2) if up else (y, x)
                    for b in range(ncb):
                        out_c[g, y, x, off + b] = cd[g, sy, sx, b]
                        out_s[g, y, x, off + b] = sc[g, sy, sx, b]
                    off += ncb
    return out_c.reshape(-1), out_s.reshape(-1)


def _cbf_nchw(a, n, c, h, w):
    """fp32 CBF [n/32][h][w][c][32] -> fp64 (n, c, h, w)."""
    a = np.asarray(a, np.float32).reshape(n // 32, h, w, c, 32).astype(np.float64)
    return a.transpose(0, 4, 3, 1, 2).reshape(n, c, h, w)


def gradient_sum(terms, fn, z, n, c, h, w):
    """The gradient of a tensor a = fn(z) read by several consumers, in fp64:
    fn'(z) times the sum of the consumers' contributions, each the channel
    slice [c_off, c_off + c) of an fp32 CBF tensor (n, c_src, hs, ws) --
    what a concatenation's gradient hands back to one part -- and, when down,
    summed over the 2x2 source pixels that a nearest-neighbour 2x upsampling
    copied this pixel to.  terms: tuples (src, c_src, c_off, down); z: fp32
    CBF (n, c, h, w) or None for FN_NONE.  Returns fp64 (n, c, h, w)."""
    acc = np.zeros((n, c, h, w))
    for src, c_src, c_off, down in terms:
        hs, ws = (2 * h, 2 * w) if down else (h, w)
        t = _cbf_nchw(src, n, c_src, hs, ws)[:, c_off:c_off + c]
        if down:
            s = np.zeros((n, c, h, w))
            for i in range(2):
                for j in range(2):
                    s += t[:, :, i::2, j::2]
            t = s
        acc += t
    if fn != FN_NONE:
        acc *= act_grad(_cbf_nchw(z, n, c, h, w), fn)
    return acc
