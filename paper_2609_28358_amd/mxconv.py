"""ctypes binding of libmxconv.so (include/mxconv.h).

Argument marshalling only: output tensors are allocated with torch on the
caller's device, pointers and the current HIP stream are passed through, and
every step runs in the library's HIP kernels.  A missing library raises; there
is no fallback path.
"""
import ctypes
import os

import torch

E4M3, E2M1, E2M3, E3M2 = 0, 1, 2, 3
F32, BF16 = 0, 1
NCHW, NHWC, CBF, CBF_BF16 = 0, 1, 2, 3
ACT, WEIGHT = 0, 1
FN_NONE, FN_RELU, FN_SILU = 0, 1, 2
FN_PRE_OUT = 0x100      # or-ed into fwd_quant's fn: act_out receives the pre-activation
FN_BF16 = 0x200         # or-ed into fwd_quant / dgrad_quant / quantize_sum's fn: bf16 full-precision tensors
KEEP_PAD = 0x100        # or-ed into quantize's layout: padding channels' codes already +0, not written

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libmxconv.so")
_lib = None


class MxconvError(RuntimeError):
    pass


QMULTI_MAX = 24
FP6_SLACK = 16          # bytes of read slack at the end of an FP6 code buffer


class MxcConv(ctypes.Structure):
    _fields_ = [(k, ctypes.c_int32) for k in
                ("n", "cin", "cout", "h", "w", "kh", "kw", "sh", "sw", "ph", "pw")]


class MxcWJob(ctypes.Structure):
    _fields_ = [("conv", ctypes.POINTER(MxcConv)), ("fmt", ctypes.c_int32), ("workspace", ctypes.c_void_p),
                ("ws_bytes", ctypes.c_size_t), ("gw", ctypes.c_void_p)]


WREDUCE_MAX = 32
CONCAT_MAX = 4
TERMS_MAX = 4


class MxcPart(ctypes.Structure):
    _fields_ = [("codes", ctypes.c_void_p), ("scales", ctypes.c_void_p), ("ncb", ctypes.c_int32),
                ("up", ctypes.c_int32)]


class MxcTerm(ctypes.Structure):
    _fields_ = [("src", ctypes.c_void_p), ("c_src", ctypes.c_int32), ("c_off", ctypes.c_int32),
                ("down", ctypes.c_int32)]


class MxcQJob(ctypes.Structure):
    _fields_ = [("src", ctypes.c_void_p)] + [(k, ctypes.c_int32) for k in
                                           ("dtype", "layout", "role", "fmt", "n", "c", "h", "w")] + \
               [("codes", ctypes.c_void_p), ("scales", ctypes.c_void_p),
                ("conv", ctypes.POINTER(MxcConv)), ("col_codes", ctypes.c_void_p), ("col_scales", ctypes.c_void_p)]


def lib():
    """Load the in-tree library (built by paper_2609_28358_amd.build)."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise MxconvError(f"{LIB_PATH} is missing: build it with "
                          "`python -m paper_2609_28358_amd.build` (no CPU fallback exists)")
    L = ctypes.CDLL(LIB_PATH)
    P, i32, i64, sz = ctypes.c_void_p, ctypes.c_int, ctypes.c_int64, ctypes.c_size_t
    CP = ctypes.POINTER(MxcConv)
    sigs = {
        "mxconv_codes_bytes": (sz, [i32] * 6),
        "mxconv_scales_bytes": (sz, [i32] * 6),
        "mxconv_out_size": (i32, [CP, ctypes.POINTER(i32), ctypes.POINTER(i32)]),
        "mxconv_im2col_codes_bytes": (sz, [CP, i32]),
        "mxconv_im2col_scales_bytes": (sz, [CP, i32]),
        "mxconv_wgrad_workspace_bytes": (sz, [CP, i32]),
        "mxconv_quantize": (i32, [P, i32, i32, i32, i32, i32, i32, i32, i32, P, P, P]),
        "mxconv_quantize_multi": (i32, [i32, ctypes.POINTER(MxcQJob), P]),
        "mxconv_quantize_sr": (i32, [P, i32, i32, i32, i32, i32, i32, i32, i32, ctypes.c_uint64, P, P, P]),
        "mxconv_nvfp_scales_bytes": (sz, [i32] * 6),
        "mxconv_nvfp_workspace_bytes": (sz, []),
        "mxconv_nvfp_quantize": (i32, [P, i32, i32, i32, i32, i32, i32, i32, i32, P, P, P, P, sz, P]),
        "mxconv_nvfp_fwd": (i32, [CP, i32, P, P, P, P, P, P, P, i32, P]),
        "mxconv_nvfp_dgrad": (i32, [CP, i32, P, P, P, P, P, P, P, i32, P]),
        "mxconv_nvfp_wgrad": (i32, [CP, i32, P, P, P, P, P, P, P, P, sz, P]),
        "mxconv_im2col_cbf": (i32, [CP, i32, P, P, P, P, P]),
        "mxconv_fwd": (i32, [CP, i32, P, P, P, P, P, i32, P]),
        "mxconv_dgrad": (i32, [CP, i32, P, P, P, P, P, i32, P]),
        "mxconv_wgrad": (i32, [CP, i32, P, P, P, P, P, P, sz, P]),
        "mxconv_wgrad_deferred": (i32, [CP, i32, P, P, P, P, P, P, sz, P]),
        "mxconv_backward": (i32, [CP, i32, P, P, P, P, P, P, P, i32, P, P, sz, i32, P]),
        "mxconv_wgrad_reduce_multi": (i32, [i32, ctypes.POINTER(MxcWJob), P]),
        "mxconv_fwd_quant": (i32, [CP, i32, P, P, P, P, i32, i32, P, P, P, P]),
        "mxconv_dgrad_quant": (i32, [CP, i32, P, P, P, P, i32, P, i32, P, P, P, P]),
        "mxconv_dgrad_quant_sr": (i32, [CP, i32, P, P, P, P, i32, P, i32, P, P, P, ctypes.c_uint64, P]),
        "mxconv_naive_codes_bytes": (sz, [i64, i64, i32]),
        "mxconv_naive_scales_bytes": (sz, [i64, i64]),
        "mxconv_naive_im2col_f32": (i32, [CP, P, P, P]),
        "mxconv_naive_quantize_1d": (i32, [P, i64, i64, i32, i32, P, P, P]),
        "mxconv_naive_fwd": (i32, [CP, i32, P, P, P, P, P, P]),
        "mxconv_naive_dgrad": (i32, [CP, i32, P, P, P, P, P, P, P]),
        "mxconv_naive_wgrad": (i32, [CP, i32, P, P, P, P, P, P]),
        "mxconv_wgrad_noalloc": (i32, [CP, i32, P, P, P, P, P, P]),
        "mxconv_concat_cbf": (i32, [i32, i32, i32, i32, i32, ctypes.POINTER(MxcPart), P, P, P]),
        "mxconv_quantize_sum": (i32, [i32, i32, i32, i32, i32, i32, ctypes.POINTER(MxcTerm), i32, P, P, P, P, P]),
        "mxconv_quantize_sum_sr": (i32, [i32, i32, i32, i32, i32, i32, ctypes.POINTER(MxcTerm), i32, P, P, P, P,
                                         ctypes.c_uint64, P]),
        "mxconv_strerror": (ctypes.c_char_p, [i32]),
    }
    for name, (res, args) in sigs.items():
        fn = getattr(L, name)
        fn.restype = res
        fn.argtypes = args
    _lib = L
    return L


def pair(first, second):
    """The `fmt` argument of a GEMM entry point whose two MX operands have
    these formats (first, second in the call's argument order)."""
    return first if first == second else 0x10 | (first << 2) | second


def strerror(rc):
    return lib().mxconv_strerror(rc).decode()


def _check(rc, what):
    if rc != 0:
        raise MxconvError(f"{what}: {strerror(rc)} (code {rc})")


def _ptr(t):
    return ctypes.c_void_p(t.data_ptr()) if t is not None else None


def _stream(stream):
    if stream is None:
        stream = torch.cuda.current_stream()
    return ctypes.c_void_p(stream.cuda_stream)


def conv_struct(cv):
    return MxcConv(*[int(cv[k]) for k in ("n", "cin", "cout", "h", "w", "kh", "kw", "sh", "sw", "ph", "pw")])


def codes_bytes(role, fmt, n, c, h, w):
    return lib().mxconv_codes_bytes(role, fmt, n, c, h, w)


def scales_bytes(role, fmt, n, c, h, w):
    return lib().mxconv_scales_bytes(role, fmt, n, c, h, w)


def out_size(cv):
    ho, wo = ctypes.c_int(), ctypes.c_int()
    _check(lib().mxconv_out_size(ctypes.byref(conv_struct(cv)), ctypes.byref(ho), ctypes.byref(wo)),
           "out_size")
    return ho.value, wo.value


def wgrad_workspace_bytes(cv, fmt):
    return lib().mxconv_wgrad_workspace_bytes(ctypes.byref(conv_struct(cv)), fmt)


class MxTensor:
    """Codes and E8M0 scales of one quantized tensor (device uint8 tensors)."""

    def __init__(self, codes, scales, role, fmt, shape):
        self.codes, self.scales, self.role, self.fmt, self.shape = codes, scales, role, fmt, tuple(shape)

    @staticmethod
    def empty(role, fmt, shape, device):
        n, c, h, w = shape
        nb = codes_bytes(role, fmt, n, c, h, w)
        ns = scales_bytes(role, fmt, n, c, h, w)
        if nb == 0:
            raise MxconvError(f"invalid MX tensor geometry {shape} role {role} fmt {fmt}")
        codes = torch.empty(nb, dtype=torch.uint8, device=device)
        if fmt in (E2M3, E3M2):
            codes[-FP6_SLACK:].zero_()     # read slack, never written by the library: keep it defined
        return MxTensor(codes, torch.empty(ns, dtype=torch.uint8, device=device), role, fmt, shape)


def _quant_args(src, layout, shape):
    if shape is None:
        if layout == NHWC:
            n, h, w, c = src.shape
            shape = (n, c, h, w)
        elif layout == NCHW:
            shape = tuple(src.shape)
        else:
            raise ValueError("shape is required for the CBF layout")
    dtype = {torch.float32: F32, torch.bfloat16: BF16}.get(src.dtype)
    if dtype is None:
        raise MxconvError(f"unsupported dtype {src.dtype}")
    if not src.is_contiguous():
        raise MxconvError("src must be contiguous")
    return dtype, tuple(int(v) for v in shape)


def quantize(src, role, fmt, layout=NCHW, shape=None, out=None, stream=None, keep_pad=False):
    """Quantize `src` (fp32 or bf16 device tensor) once.  `shape` is the
    logical (n, c, h, w); it defaults to src.shape for NCHW.  keep_pad: the
    codes of `out`'s padding channels already hold +0 codes (MXC_KEEP_PAD)."""
    dtype, shape = _quant_args(src, layout, shape)
    if out is None:
        if keep_pad:
            raise MxconvError("keep_pad needs an output whose padding codes are +0")
        out = MxTensor.empty(role, fmt, shape, src.device)
    _check(lib().mxconv_quantize(_ptr(src), dtype, layout | (KEEP_PAD if keep_pad else 0), role, fmt, *shape,
                                 _ptr(out.codes), _ptr(out.scales), _stream(stream)), "mxconv_quantize")
    return out


def quantize_multi(items, stream=None):
    """Several quantize() calls in one library call (one launch for the CBF
    batch-block-32 activations and OIHW weights among them).  items: tuples
    (src, role, fmt, layout, shape, out[, col]); col = (cv, col_codes,
    col_scales) also writes the activation's CBF im2col for layer cv into the
    two uint8 device tensors (sizes: mxconv_im2col_{codes,scales}_bytes).
    Returns the MX tensors."""
    if len(items) > QMULTI_MAX:
        raise MxconvError(f"at most {QMULTI_MAX} tensors per call")
    jobs = (MxcQJob * max(1, len(items)))()
    convs = []                       # kept alive for the call
    outs = []
    for k, item in enumerate(items):
        src, role, fmt, layout, shape, out = item[:6]
        col = item[6] if len(item) > 6 else None
        dtype, shape = _quant_args(src, layout, shape)
        if out is None:
            out = MxTensor.empty(role, fmt, shape, src.device)
        jobs[k] = MxcQJob(src.data_ptr(), dtype, layout, role, fmt, *shape, out.codes.data_ptr(),
                          out.scales.data_ptr())
        if col is not None:
            cv, cc, cs = col
            convs.append(conv_struct(cv))
            jobs[k].conv = ctypes.pointer(convs[-1])
            jobs[k].col_codes = cc.data_ptr()
            jobs[k].col_scales = cs.data_ptr()
        outs.append(out)
    _check(lib().mxconv_quantize_multi(len(items), jobs, _stream(stream)), "mxconv_quantize_multi")
    return outs


def quantize_sr(src, role, fmt, seed, layout=NCHW, shape=None, out=None, stream=None):
    """quantize() with stochastic rounding of the elements under `seed`."""
    dtype, shape = _quant_args(src, layout, shape)
    if out is None:
        out = MxTensor.empty(role, fmt, shape, src.device)
    _check(lib().mxconv_quantize_sr(_ptr(src), dtype, layout, role, fmt, *shape, int(seed) & (2 ** 64 - 1),
                                    _ptr(out.codes), _ptr(out.scales), _stream(stream)), "mxconv_quantize_sr")
    return out


class NvfpTensor:
    """A tensor in the two-level NVFP format: codes (MX-CBF layout), E4M3
    block scales, and the per-tensor scale (a one-element float tensor)."""

    def __init__(self, codes, scales, tscale, role, fmt, shape):
        self.codes, self.scales, self.tscale = codes, scales, tscale
        self.role, self.fmt, self.shape = role, fmt, tuple(shape)


def nvfp_quantize(src, role, fmt, layout=NCHW, shape=None, workspace=None, stream=None):
    """Eqs. (4)-(6) on the GPU: CBF activations (batch block 32) or OIHW weights."""
    dtype, shape = _quant_args(src, layout, shape)
    L = lib()
    nb = L.mxconv_codes_bytes(role, fmt, *shape)
    ns = L.mxconv_nvfp_scales_bytes(role, fmt, *shape)
    if nb == 0 or ns == 0:
        raise MxconvError(f"invalid NVFP tensor geometry {shape} role {role} fmt {fmt}")
    out = NvfpTensor(torch.empty(nb, dtype=torch.uint8, device=src.device),
                     torch.empty(ns, dtype=torch.uint8, device=src.device),
                     torch.empty(4, dtype=torch.float32, device=src.device), role, fmt, shape)
    wsb = L.mxconv_nvfp_workspace_bytes()
    if workspace is None:
        workspace = torch.empty(wsb, dtype=torch.uint8, device=src.device)
    _check(L.mxconv_nvfp_quantize(_ptr(src), dtype, layout, role, fmt, *shape, _ptr(out.codes), _ptr(out.scales),
                                  _ptr(out.tscale), _ptr(workspace), workspace.numel() * workspace.element_size(),
                                  _stream(stream)), "mxconv_nvfp_quantize")
    return out


def nvfp_fwd(cv, w, x, layout=NCHW, out=None, stream=None):
    """Y = W * X on NVFP operands (NvfpTensor): NVFP4, NVFP6 E2M3, NVFP8, or
    NVFP4 weights with NVFP6 E3M2 activations."""
    y = _out((cv["n"], cv["cout"], *out_size(cv)), layout, batch_block(cv["n"]), x.codes.device, out)
    _check(lib().mxconv_nvfp_fwd(ctypes.byref(conv_struct(cv)), pair(w.fmt, x.fmt), _ptr(w.codes), _ptr(w.scales), _ptr(w.tscale),
                                 _ptr(x.codes), _ptr(x.scales), _ptr(x.tscale), _ptr(y), layout, _stream(stream)),
           "mxconv_nvfp_fwd")
    return y


def nvfp_dgrad(cv, w, gy, layout=NCHW, out=None, stream=None):
    gx = _out((cv["n"], cv["cin"], cv["h"], cv["w"]), layout, batch_block(cv["n"]), gy.codes.device, out)
    _check(lib().mxconv_nvfp_dgrad(ctypes.byref(conv_struct(cv)), pair(w.fmt, gy.fmt), _ptr(w.codes), _ptr(w.scales),
                                   _ptr(w.tscale), _ptr(gy.codes), _ptr(gy.scales), _ptr(gy.tscale), _ptr(gx), layout,
                                   _stream(stream)), "mxconv_nvfp_dgrad")
    return gx


def nvfp_wgrad(cv, gy, x, out=None, workspace=None, stream=None):
    gw = out if out is not None else torch.empty((cv["cout"], cv["cin"], cv["kh"], cv["kw"]),
                                                 dtype=torch.float32, device=x.codes.device)
    fmt = pair(gy.fmt, x.fmt)
    need = wgrad_workspace_bytes(cv, fmt)
    if workspace is None and need:
        workspace = torch.empty(need, dtype=torch.uint8, device=x.codes.device)
    wsz = workspace.numel() * workspace.element_size() if workspace is not None else 0
    _check(lib().mxconv_nvfp_wgrad(ctypes.byref(conv_struct(cv)), fmt, _ptr(gy.codes), _ptr(gy.scales),
                                   _ptr(gy.tscale), _ptr(x.codes), _ptr(x.scales), _ptr(x.tscale), _ptr(gw),
                                   _ptr(workspace), wsz, _stream(stream)), "mxconv_nvfp_wgrad")
    return gw


def im2col_cbf(cv, x, stream=None):
    c = conv_struct(cv)
    nb = lib().mxconv_im2col_codes_bytes(ctypes.byref(c), x.fmt)
    ns = lib().mxconv_im2col_scales_bytes(ctypes.byref(c), x.fmt)
    codes = torch.empty(nb, dtype=torch.uint8, device=x.codes.device)
    scales = torch.empty(ns, dtype=torch.uint8, device=x.codes.device)
    _check(lib().mxconv_im2col_cbf(ctypes.byref(c), x.fmt, _ptr(x.codes), _ptr(x.scales), _ptr(codes),
                                   _ptr(scales), _stream(stream)), "mxconv_im2col_cbf")
    return codes, scales


def _want(t, dtype, what):
    """A device tensor argument must have the element type the call reads or
    writes through its pointer."""
    if t is not None and t.dtype != dtype:
        raise MxconvError(f"{what} must be {dtype}, got {t.dtype}")


def _out(shape, layout, bn, device, out):
    n, c, h, w = shape
    dtype = torch.bfloat16 if layout == CBF_BF16 else torch.float32
    if out is not None:
        _want(out, dtype, "the output")
        return out
    if layout in (CBF, CBF_BF16):
        return torch.empty((n // bn, h, w, c, bn), dtype=dtype, device=device)
    return torch.empty((n, c, h, w), dtype=dtype, device=device)


def batch_block(n):
    return 32 if n >= 32 else n


def fwd(cv, w, x, layout=NCHW, out=None, stream=None):
    ho, wo = out_size(cv)
    y = _out((cv["n"], cv["cout"], ho, wo), layout, batch_block(cv["n"]), x.codes.device, out)
    _check(lib().mxconv_fwd(ctypes.byref(conv_struct(cv)), pair(w.fmt, x.fmt), _ptr(w.codes), _ptr(w.scales),
                            _ptr(x.codes), _ptr(x.scales), _ptr(y), layout, _stream(stream)), "mxconv_fwd")
    return y


def dgrad(cv, w, gy, layout=NCHW, out=None, stream=None):
    gx = _out((cv["n"], cv["cin"], cv["h"], cv["w"]), layout, batch_block(cv["n"]), gy.codes.device, out)
    _check(lib().mxconv_dgrad(ctypes.byref(conv_struct(cv)), pair(w.fmt, gy.fmt), _ptr(w.codes), _ptr(w.scales),
                              _ptr(gy.codes), _ptr(gy.scales), _ptr(gx), layout, _stream(stream)),
           "mxconv_dgrad")
    return gx


def wgrad(cv, gy, x, out=None, workspace=None, stream=None, deferred=False):
    """G_W = G_Y * X^T.  deferred: leave the split-K partial sums in the
    workspace for wgrad_reduce_multi (the workspace must then be passed)."""
    gw = out if out is not None else torch.empty((cv["cout"], cv["cin"], cv["kh"], cv["kw"]),
                                                 dtype=torch.float32, device=x.codes.device)
    need = wgrad_workspace_bytes(cv, pair(gy.fmt, x.fmt))
    if workspace is None and need:
        if deferred:
            raise MxconvError("a deferred weight gradient needs the caller's workspace")
        workspace = torch.empty(need, dtype=torch.uint8, device=x.codes.device)
    wsz = workspace.numel() * workspace.element_size() if workspace is not None else 0
    fn, name = (lib().mxconv_wgrad_deferred, "mxconv_wgrad_deferred") if deferred else (lib().mxconv_wgrad,
                                                                                          "mxconv_wgrad")
    _check(fn(ctypes.byref(conv_struct(cv)), pair(gy.fmt, x.fmt), _ptr(gy.codes), _ptr(gy.scales),
              _ptr(x.codes), _ptr(x.scales), _ptr(gw), _ptr(workspace), wsz, _stream(stream)), name)
    return gw


def backward(cv, w, gy, x, layout=NCHW, gx_out=None, gw_out=None, workspace=None, stream=None, deferred=False):
    """Input and weight gradients of one layer from one call: (G_X, G_W), bit
    for bit what dgrad() and wgrad() give (one launch where the layer allows)."""
    f = pair(w.fmt, gy.fmt)
    if pair(gy.fmt, x.fmt) != f:
        raise MxconvError("backward needs the same format pair for (W, G_Y) and (G_Y, X)")
    dev = gy.codes.device
    gx = _out((cv["n"], cv["cin"], cv["h"], cv["w"]), layout, batch_block(cv["n"]), dev, gx_out)
    gw = gw_out if gw_out is not None else torch.empty((cv["cout"], cv["cin"], cv["kh"], cv["kw"]),
                                                       dtype=torch.float32, device=dev)
    need = wgrad_workspace_bytes(cv, f)
    if workspace is None and need:
        if deferred:
            raise MxconvError("a deferred weight gradient needs the caller's workspace")
        workspace = torch.empty(need, dtype=torch.uint8, device=dev)
    wsz = workspace.numel() * workspace.element_size() if workspace is not None else 0
    _check(lib().mxconv_backward(ctypes.byref(conv_struct(cv)), f, _ptr(w.codes), _ptr(w.scales), _ptr(gy.codes),
                                 _ptr(gy.scales), _ptr(x.codes), _ptr(x.scales), _ptr(gx), layout, _ptr(gw),
                                 _ptr(workspace), wsz, 1 if deferred else 0, _stream(stream)), "mxconv_backward")
    return gx, gw


def wgrad_reduce_multi(items, stream=None):
    """Finish deferred weight gradients in one launch.  items: tuples
    (cv, fmt, workspace, gw) of the deferred calls (fmt as passed to them:
    pair(gy.fmt, x.fmt))."""
    if len(items) > WREDUCE_MAX:
        raise MxconvError(f"at most {WREDUCE_MAX} layers per call")
    jobs = (MxcWJob * max(1, len(items)))()
    convs = []
    for k, (cv, fmt, ws, gw) in enumerate(items):
        convs.append(conv_struct(cv))
        jobs[k] = MxcWJob(ctypes.pointer(convs[-1]), fmt, ws.data_ptr() if ws is not None else None,
                          ws.numel() * ws.element_size() if ws is not None else 0, gw.data_ptr())
    _check(lib().mxconv_wgrad_reduce_multi(len(items), jobs, _stream(stream)), "mxconv_wgrad_reduce_multi")


def fwd_quant(cv, w, x, fn=FN_NONE, out_fmt=None, out=None, act_out=None, stream=None):
    """Forward with the quantizing epilogue: MX codes of fn(W * X) for
    (n, cout, Ho, Wo); `act_out` (CBF fp32, optional) receives the values
    that were quantized (with FN_PRE_OUT: W * X; with FN_BF16 | FN_PRE_OUT
    it is bf16 and receives W * X rounded to bf16).  Returns the MxTensor."""
    _want(act_out, torch.bfloat16 if (fn & FN_BF16) and (fn & FN_PRE_OUT) else torch.float32, "act_out")
    ho, wo = out_size(cv)
    out_fmt = x.fmt if out_fmt is None else out_fmt
    shape = (cv["n"], cv["cout"], ho, wo)
    y = out if out is not None else MxTensor.empty(ACT, out_fmt, shape, x.codes.device)
    _check(lib().mxconv_fwd_quant(ctypes.byref(conv_struct(cv)), pair(w.fmt, x.fmt), _ptr(w.codes), _ptr(w.scales),
                                  _ptr(x.codes), _ptr(x.scales), fn, out_fmt, _ptr(y.codes), _ptr(y.scales),
                                  _ptr(act_out), _stream(stream)), "mxconv_fwd_quant")
    return y


def dgrad_quant(cv, w, gy, fn=FN_NONE, z=None, out_fmt=None, out=None, act_out=None, stream=None, sr_seed=None):
    """Input gradient with the quantizing epilogue: MX codes of
    (W^T * G_Y) . fn'(z) for (n, cin, h, w); z is the CBF pre-activation of
    this layer's input (not needed for FN_NONE), fp32, or bf16 with FN_BF16.
    act_out (optional) is fp32.  sr_seed: round the codes stochastically
    (mxconv_dgrad_quant_sr) with this 64-bit seed."""
    _want(z, torch.bfloat16 if fn & FN_BF16 else torch.float32, "z")
    _want(act_out, torch.float32, "act_out")
    out_fmt = gy.fmt if out_fmt is None else out_fmt
    shape = (cv["n"], cv["cin"], cv["h"], cv["w"])
    g = out if out is not None else MxTensor.empty(ACT, out_fmt, shape, gy.codes.device)
    args = (ctypes.byref(conv_struct(cv)), pair(w.fmt, gy.fmt), _ptr(w.codes), _ptr(w.scales), _ptr(gy.codes),
            _ptr(gy.scales), fn, _ptr(z), out_fmt, _ptr(g.codes), _ptr(g.scales), _ptr(act_out))
    if sr_seed is None:
        _check(lib().mxconv_dgrad_quant(*args, _stream(stream)), "mxconv_dgrad_quant")
    else:
        _check(lib().mxconv_dgrad_quant_sr(*args, sr_seed, _stream(stream)), "mxconv_dgrad_quant_sr")
    return g


# ---------------------------------------------------------------- network steps
def concat_cbf(parts, out=None, stream=None):
    """Concatenate MX-CBF activations along channels, whole blocks, in order.
    parts: MxTensors, or (MxTensor, up) with up = 1 for a 2x nearest-neighbour
    upsampling of that part.  Returns the MxTensor of (n, 32 * sum ncb, h, w)."""
    if not 1 <= len(parts) <= CONCAT_MAX:
        raise MxconvError(f"1 to {CONCAT_MAX} parts")
    arr = (MxcPart * len(parts))()
    nb, hw, fmt = 0, None, None
    for k, p in enumerate(parts):
        t, up = (p, 0) if isinstance(p, MxTensor) else p
        n, c, h, w = t.shape
        ncb = (c + 31) // 32
        arr[k] = MxcPart(t.codes.data_ptr(), t.scales.data_ptr(), ncb, up)
        nb += ncb
        hw = (h * 2, w * 2) if up else (h, w)
        fmt, dev = t.fmt, t.codes.device
    shape = (n, 32 * nb, hw[0], hw[1])
    y = out if out is not None else MxTensor.empty(ACT, fmt, shape, dev)
    _check(lib().mxconv_concat_cbf(fmt, shape[0], shape[2], shape[3], len(parts), arr, _ptr(y.codes), _ptr(y.scales),
                                   _stream(stream)), "mxconv_concat_cbf")
    return y


def quantize_sum(terms, shape, fmt, fn=FN_NONE, z=None, out=None, vals=None, stream=None, sr_seed=None):
    """MX codes of fn'(z) . (sum of terms) for the (n, c, h, w) tensor `shape`.
    terms: tuples (src, c_src, c_off, down) with src a CBF device tensor
    [n/32][hs][ws][c_src][32]; terms and z are fp32, or bf16 with FN_BF16;
    vals (optional) is fp32.  sr_seed: round the codes stochastically
    (mxconv_quantize_sum_sr) with this 64-bit seed."""
    if not 1 <= len(terms) <= TERMS_MAX:
        raise MxconvError(f"1 to {TERMS_MAX} terms")
    dt = torch.bfloat16 if fn & FN_BF16 else torch.float32
    _want(z, dt, "z")
    _want(vals, torch.float32, "vals")
    arr = (MxcTerm * len(terms))()
    for k, (src, c_src, c_off, down) in enumerate(terms):
        _want(src, dt, f"term {k}")
        arr[k] = MxcTerm(src.data_ptr(), c_src, c_off, down)
    n, c, h, w = shape
    g = out if out is not None else MxTensor.empty(ACT, fmt, shape, terms[0][0].device)
    args = (fmt, n, c, h, w, len(terms), arr, fn, _ptr(z), _ptr(g.codes), _ptr(g.scales), _ptr(vals))
    if sr_seed is None:
        _check(lib().mxconv_quantize_sum(*args, _stream(stream)), "mxconv_quantize_sum")
    else:
        _check(lib().mxconv_quantize_sum_sr(*args, sr_seed, _stream(stream)), "mxconv_quantize_sum_sr")
    return g


# ---------------------------------------------------------------- naive comparator
# Channels-last GEMM form: P = n*Ho*Wo positions (n, ho, wo), K = kh*kw*cin
# (kh, kw, ci); X, G_Y, G_X NHWC fp32; W, G_W OHWI fp32 ([cout][K]).
class LineMatrix:
    """A 1-D-blocked matrix: codes [lines][Lp] and scales [lines][Lp/32]."""

    def __init__(self, codes, scales, fmt, lines, length):
        self.codes, self.scales, self.fmt, self.lines, self.length = codes, scales, fmt, lines, length


def naive_im2col_f32(cv, x, out=None, stream=None):
    ho, wo = out_size(cv)
    col = out if out is not None else torch.empty((cv["n"] * ho * wo, cv["kh"] * cv["kw"] * cv["cin"]),
                                                  dtype=torch.float32, device=x.device)
    _check(lib().mxconv_naive_im2col_f32(ctypes.byref(conv_struct(cv)), _ptr(x), _ptr(col), _stream(stream)),
           "mxconv_naive_im2col_f32")
    return col


def naive_quantize_1d(m, direction, fmt, out=None, stream=None):
    """Quantize a contiguous fp32 [rows][cols] device matrix with 1-D blocks
    of 32 along its rows (direction 0) or columns (direction 1)."""
    rows, cols = m.shape
    lines, length = (rows, cols) if direction == 0 else (cols, rows)
    if out is None:
        nb = lib().mxconv_naive_codes_bytes(lines, length, fmt)
        ns = lib().mxconv_naive_scales_bytes(lines, length)
        if nb == 0:
            raise MxconvError(f"invalid line matrix {lines} x {length}")
        out = LineMatrix(torch.empty(nb, dtype=torch.uint8, device=m.device),
                         torch.empty(ns, dtype=torch.uint8, device=m.device), fmt, lines, length)
    if m.dtype != torch.float32 or not m.is_contiguous():
        raise MxconvError("naive_quantize_1d needs a contiguous fp32 matrix")
    _check(lib().mxconv_naive_quantize_1d(_ptr(m), rows, cols, direction, fmt, _ptr(out.codes),
                                          _ptr(out.scales), _stream(stream)), "mxconv_naive_quantize_1d")
    return out


def naive_fwd(cv, col_q, w_q, out=None, stream=None):
    ho, wo = out_size(cv)
    y = out if out is not None else torch.empty((cv["n"] * ho * wo, cv["cout"]), dtype=torch.float32,
                                                device=col_q.codes.device)
    _check(lib().mxconv_naive_fwd(ctypes.byref(conv_struct(cv)), col_q.fmt, _ptr(col_q.codes),
                                  _ptr(col_q.scales), _ptr(w_q.codes), _ptr(w_q.scales), _ptr(y),
                                  _stream(stream)), "mxconv_naive_fwd")
    return y


def naive_dgrad(cv, gy_q, wt_q, gcol=None, out=None, stream=None):
    ho, wo = out_size(cv)
    dev = gy_q.codes.device
    if gcol is None:
        gcol = torch.empty((cv["n"] * ho * wo, cv["kh"] * cv["kw"] * cv["cin"]), dtype=torch.float32,
                           device=dev)
    gx = out if out is not None else torch.empty((cv["n"], cv["h"], cv["w"], cv["cin"]),
                                                 dtype=torch.float32, device=dev)
    _check(lib().mxconv_naive_dgrad(ctypes.byref(conv_struct(cv)), gy_q.fmt, _ptr(gy_q.codes),
                                    _ptr(gy_q.scales), _ptr(wt_q.codes), _ptr(wt_q.scales), _ptr(gcol),
                                    _ptr(gx), _stream(stream)), "mxconv_naive_dgrad")
    return gx


def naive_wgrad(cv, gyt_q, xt_q, out=None, stream=None):
    gw = out if out is not None else torch.empty((cv["cout"], cv["kh"] * cv["kw"] * cv["cin"]),
                                                 dtype=torch.float32, device=gyt_q.codes.device)
    _check(lib().mxconv_naive_wgrad(ctypes.byref(conv_struct(cv)), gyt_q.fmt, _ptr(gyt_q.codes),
                                    _ptr(gyt_q.scales), _ptr(xt_q.codes), _ptr(xt_q.scales), _ptr(gw),
                                    _stream(stream)), "mxconv_naive_wgrad")
    return gw
