// mxconv_abi.cpp -- the C ABI of include/mxconv.h: host-side validation,
// size helpers and dispatch to the gfx950 kernels.  Every argument check runs
// on the host before anything is enqueued.
#include <mutex>

#include "mx_internal.h"

namespace mxc {

static bool fmt_ok(int fmt) { return fmt >= MXC_E4M3 && fmt <= MXC_E3M2; }

int geom_init(Geom* g, int role, int fmt, int n, int c, int h, int w) {
    if (!fmt_ok(fmt)) return MXC_ERR_ARG;
    if (role != MXC_ACT && role != MXC_WEIGHT) return MXC_ERR_ARG;
    if (n <= 0 || c <= 0 || h <= 0 || w <= 0) return MXC_ERR_ARG;
    g->n = n; g->c = c; g->h = h; g->w = w;
    g->fmt = fmt;
    g->bits = fmt_bits(fmt);
    g->cp = (c + 31) / 32 * 32;
    g->ncb = g->cp / 32;
    if (role == MXC_WEIGHT) {
        g->bn = 32;
        g->np = (n + 31) / 32 * 32;
    } else {
        if (n >= 32) {
            if (n % 32) return MXC_ERR_SHAPE;
            g->bn = 32;
        } else {
            if (32 % n) return MXC_ERR_SHAPE;
            g->bn = n;
        }
        g->np = n;
        if (fmt == MXC_E2M1 && g->bn < 2) return MXC_ERR_SHAPE;
        if (g->bits == 6 && g->bn < 4) return MXC_ERR_SHAPE;   // whole bytes per channel row
    }
    g->ng = g->np / g->bn;
    // sizes addressed with 32-bit pixel / block indices inside kernels
    if ((long long)g->ng * h * w * g->ncb > 0x7FFFFFFFLL) return MXC_ERR_SHAPE;
    return MXC_OK;
}

// The format pairs the GEMM kernels are built for.
static bool pair_ok(int fa, int fb) {
    if (fa == fb) return fa == MXC_E4M3 || fa == MXC_E2M1 || fa == MXC_E2M3;
    return fa == MXC_E2M1 && fb == MXC_E3M2;
}

int conv_init(Conv* cv, const mxc_conv* p, int fmt, int op) {
    int f1 = fmt, f2 = fmt;
    if (op != CONV_ONE) {
        if ((fmt & ~0x1F) != 0) return MXC_ERR_ARG;
        if (fmt & 0x10) { f1 = (fmt >> 2) & 3; f2 = fmt & 3; }
        if (!fmt_ok(f1) || !fmt_ok(f2) || !pair_ok(f1, f2)) return MXC_ERR_ARG;
    } else if (!fmt_ok(fmt)) {
        return MXC_ERR_ARG;
    }
    if (p->n <= 0 || p->cin <= 0 || p->cout <= 0 || p->h <= 0 || p->w <= 0 || p->kh <= 0 ||
        p->kw <= 0 || p->sh <= 0 || p->sw <= 0 || p->ph < 0 || p->pw < 0)
        return MXC_ERR_ARG;
    cv->n = p->n; cv->cin = p->cin; cv->cout = p->cout; cv->h = p->h; cv->w = p->w;
    cv->kh = p->kh; cv->kw = p->kw; cv->sh = p->sh; cv->sw = p->sw; cv->ph = p->ph; cv->pw = p->pw;
    if (p->h + 2 * p->ph < p->kh || p->w + 2 * p->pw < p->kw) return MXC_ERR_SHAPE;
    cv->ho = (p->h + 2 * p->ph - p->kh) / p->sh + 1;
    cv->wo = (p->w + 2 * p->pw - p->kw) / p->sw + 1;
    // formats of X, G_Y and W (an operand the call does not read takes the
    // format of one it does, for its geometry only)
    int fx = f1, fg = f1, fw = f1;
    if (op == CONV_FWD) { fw = f1; fx = f2; fg = f2; }
    else if (op == CONV_DGRAD) { fw = f1; fg = f2; fx = f2; }
    else if (op == CONV_WGRAD) { fg = f1; fx = f2; fw = f1; }
    cv->fa = f1; cv->fb = f2;
    cv->fmt = f1 == f2 ? f1 : -1;
    cv->bits = f1 == f2 ? fmt_bits(f1) : 0;
    int rc;
    if ((rc = geom_init(&cv->x, MXC_ACT, fx, p->n, p->cin, p->h, p->w))) return rc;
    if ((rc = geom_init(&cv->gy, MXC_ACT, fg, p->n, p->cout, cv->ho, cv->wo))) return rc;
    if ((rc = geom_init(&cv->wt, MXC_WEIGHT, fw, p->cout, p->cin, p->kh, p->kw))) return rc;
    return MXC_OK;
}

}  // namespace mxc

using namespace mxc;

static bool aligned16(const void* p) { return ((uintptr_t)p & 15u) == 0; }
// output layouts of the GEMM entry points: fp32 NCHW / CBF, bf16 CBF
static bool out_layout_ok(int l) { return l == MXC_NCHW || l == MXC_CBF || l == MXC_CBF_BF16; }

extern "C" {

size_t mxconv_codes_bytes(int role, int fmt, int n, int c, int h, int w) {
    Geom g;
    return geom_init(&g, role, fmt, n, c, h, w) ? 0 : geom_codes_bytes(g);
}

size_t mxconv_scales_bytes(int role, int fmt, int n, int c, int h, int w) {
    Geom g;
    return geom_init(&g, role, fmt, n, c, h, w) ? 0 : geom_scales_bytes(g);
}

int mxconv_out_size(const mxc_conv* p, int* ho, int* wo) {
    if (!p || !ho || !wo) return MXC_ERR_NULL;
    Conv cv;
    int rc = conv_init(&cv, p, MXC_E4M3);
    if (rc) return rc;
    *ho = cv.ho; *wo = cv.wo;
    return MXC_OK;
}

size_t mxconv_im2col_codes_bytes(const mxc_conv* p, int fmt) {
    Conv cv;
    if (!p || conv_init(&cv, p, fmt)) return 0;
    return (size_t)cv.x.ng * cv.ho * cv.wo * cv.kh * cv.kw * cv.x.cp * cv.x.bn * cv.x.bits / 8 +
           (cv.x.bits == 6 ? FP6_SLACK : 0);
}

size_t mxconv_im2col_scales_bytes(const mxc_conv* p, int fmt) {
    Conv cv;
    if (!p || conv_init(&cv, p, fmt)) return 0;
    return (size_t)cv.x.ng * cv.ho * cv.wo * cv.kh * cv.kw * cv.x.ncb;
}

size_t mxconv_wgrad_workspace_bytes(const mxc_conv* p, int fmt) {
    Conv cv;
    if (!p || conv_init(&cv, p, fmt, CONV_WGRAD)) return 0;
    return wgrad_workspace(cv);
}

int mxconv_quantize(const void* src, int dtype, int layout, int role, int fmt, int n, int c,
                    int h, int w, void* codes, uint8_t* scales, void* stream) {
    if (!src || !codes || !scales) return MXC_ERR_NULL;
    const bool keep_pad = (layout & MXC_KEEP_PAD) != 0;
    layout &= ~MXC_KEEP_PAD;
    if (dtype != MXC_F32 && dtype != MXC_BF16) return MXC_ERR_ARG;
    if (layout != MXC_NCHW && layout != MXC_NHWC && layout != MXC_CBF) return MXC_ERR_ARG;
    if (layout == MXC_CBF && role != MXC_ACT) return MXC_ERR_ARG;
    Geom g;
    int rc = geom_init(&g, role, fmt, n, c, h, w);
    if (rc) return rc;
    if (!aligned16(src) || !aligned16(codes) || !aligned16(scales)) return MXC_ERR_ALIGN;
    return launch_quantize(src, dtype, layout, role, g, fmt, codes, scales, (hipStream_t)stream, nullptr, keep_pad);
}

int mxconv_quantize_multi(int count, const mxc_qjob* jobs, void* stream) {
    if (count < 0 || count > MXC_QMULTI_MAX) return MXC_ERR_ARG;
    if (count > 0 && !jobs) return MXC_ERR_NULL;
    QuantJob q[MXC_QMULTI_MAX];
    for (int i = 0; i < count; i++) {
        const mxc_qjob& j = jobs[i];
        if (!j.src || !j.codes || !j.scales) return MXC_ERR_NULL;
        if (j.dtype != MXC_F32 && j.dtype != MXC_BF16) return MXC_ERR_ARG;
        if (j.layout != MXC_NCHW && j.layout != MXC_NHWC && j.layout != MXC_CBF) return MXC_ERR_ARG;
        if (j.layout == MXC_CBF && j.role != MXC_ACT) return MXC_ERR_ARG;
        const int rc = geom_init(&q[i].g, j.role, j.fmt, j.n, j.c, j.h, j.w);
        if (rc) return rc;
        if (!aligned16(j.src) || !aligned16(j.codes) || !aligned16(j.scales)) return MXC_ERR_ALIGN;
        q[i].src = j.src; q[i].dtype = j.dtype; q[i].layout = j.layout; q[i].role = j.role; q[i].fmt = j.fmt;
        q[i].codes = j.codes; q[i].scales = j.scales;
        q[i].col = j.conv != nullptr;
        q[i].col_codes = j.col_codes; q[i].col_scales = j.col_scales;
        if (q[i].col) {
            if (!j.col_codes || !j.col_scales) return MXC_ERR_NULL;
            const mxc_conv& p = *j.conv;
            if (j.role != MXC_ACT || p.n != j.n || p.cin != j.c || p.h != j.h || p.w != j.w) return MXC_ERR_SHAPE;
            int rc2 = conv_init(&q[i].cv, j.conv, j.fmt);
            if (!rc2) rc2 = im2col_check(q[i].cv);
            if (rc2) return rc2;
            if (!aligned16(j.col_codes) || !aligned16(j.col_scales)) return MXC_ERR_ALIGN;
        }
    }
    return launch_quantize_multi(count, q, (hipStream_t)stream);
}

int mxconv_quantize_sr(const void* src, int dtype, int layout, int role, int fmt, int n, int c,
                       int h, int w, uint64_t seed, void* codes, uint8_t* scales, void* stream) {
    if (!src || !codes || !scales) return MXC_ERR_NULL;
    if (dtype != MXC_F32 && dtype != MXC_BF16) return MXC_ERR_ARG;
    if (layout != MXC_NCHW && layout != MXC_NHWC && layout != MXC_CBF) return MXC_ERR_ARG;
    if (layout == MXC_CBF && role != MXC_ACT) return MXC_ERR_ARG;
    Geom g;
    int rc = geom_init(&g, role, fmt, n, c, h, w);
    if (rc) return rc;
    if (!aligned16(src) || !aligned16(codes) || !aligned16(scales)) return MXC_ERR_ALIGN;
    return launch_quantize(src, dtype, layout, role, g, fmt, codes, scales, (hipStream_t)stream, &seed);
}

size_t mxconv_nvfp_scales_bytes(int role, int fmt, int n, int c, int h, int w) {
    Geom g;
    if (geom_init(&g, role, fmt, n, c, h, w) || g.bn % 8) return 0;
    return (size_t)g.ng * g.h * g.w * (g.cp / 8) * (g.bn / 8);
}

size_t mxconv_nvfp_workspace_bytes(void) { return (size_t)NVFP_PARTS * sizeof(uint32_t); }

int mxconv_nvfp_quantize(const void* src, int dtype, int layout, int role, int fmt, int n, int c, int h, int w,
                         void* codes, uint8_t* scales, float* tscale, void* workspace, size_t ws_bytes,
                         void* stream) {
    if (!src || !codes || !scales || !tscale) return MXC_ERR_NULL;
    if (dtype != MXC_F32 && dtype != MXC_BF16) return MXC_ERR_ARG;
    if (layout != MXC_NCHW && layout != MXC_NHWC && layout != MXC_CBF) return MXC_ERR_ARG;
    if (layout == MXC_CBF && role != MXC_ACT) return MXC_ERR_ARG;
    Geom g;
    int rc = geom_init(&g, role, fmt, n, c, h, w);
    if (rc) return rc;
    // the GPU kernels read CBF activations with batch block 32 and OIHW weights
    if (!((layout == MXC_CBF && role == MXC_ACT && g.bn == 32) || (layout == MXC_NCHW && role == MXC_WEIGHT)))
        return MXC_ERR_SHAPE;
    if (!workspace || ws_bytes < mxconv_nvfp_workspace_bytes()) return MXC_ERR_WORKSPACE;
    if (!aligned16(src) || !aligned16(codes) || !aligned16(scales) || !aligned16(tscale) || !aligned16(workspace))
        return MXC_ERR_ALIGN;
    return launch_nvfp_quantize(src, dtype, layout, role, g, fmt, codes, scales, tscale, workspace,
                                (hipStream_t)stream);
}

int mxconv_nvfp_fwd(const mxc_conv* p, int fmt, const void* wc, const uint8_t* ws, const float* wt,
                    const void* xc, const uint8_t* xs, const float* xt, float* y, int y_layout, void* stream) {
    if (!p || !wc || !ws || !wt || !xc || !xs || !xt || !y) return MXC_ERR_NULL;
    if (y_layout != MXC_NCHW && y_layout != MXC_CBF) return MXC_ERR_ARG;
    Conv cv;
    int rc = conv_init(&cv, p, fmt, CONV_FWD);
    if (rc) return rc;
    if (!nv_pair_ok(cv.fa, cv.fb)) return MXC_ERR_ARG;
    if (!aligned16(wc) || !aligned16(ws) || !aligned16(wt) || !aligned16(xc) || !aligned16(xs) ||
        !aligned16(xt) || !aligned16(y))
        return MXC_ERR_ALIGN;
    rc = launch_conv_lean(cv, false, wc, ws, xc, xs, y, y_layout, (hipStream_t)stream, nullptr, wt, xt);
    return rc == 1 ? MXC_ERR_SHAPE : rc;
}

int mxconv_nvfp_dgrad(const mxc_conv* p, int fmt, const void* wc, const uint8_t* ws, const float* wt,
                      const void* gc, const uint8_t* gs, const float* gt, float* gx, int gx_layout, void* stream) {
    if (!p || !wc || !ws || !wt || !gc || !gs || !gt || !gx) return MXC_ERR_NULL;
    if (gx_layout != MXC_NCHW && gx_layout != MXC_CBF) return MXC_ERR_ARG;
    Conv cv;
    int rc = conv_init(&cv, p, fmt, CONV_DGRAD);
    if (rc) return rc;
    if (!nv_pair_ok(cv.fa, cv.fb)) return MXC_ERR_ARG;
    if (!aligned16(wc) || !aligned16(ws) || !aligned16(wt) || !aligned16(gc) || !aligned16(gs) ||
        !aligned16(gt) || !aligned16(gx))
        return MXC_ERR_ALIGN;
    rc = launch_conv_lean(cv, true, wc, ws, gc, gs, gx, gx_layout, (hipStream_t)stream, nullptr, wt, gt);
    return rc == 1 ? MXC_ERR_SHAPE : rc;
}

int mxconv_nvfp_wgrad(const mxc_conv* p, int fmt, const void* gc, const uint8_t* gs, const float* gt,
                      const void* xc, const uint8_t* xs, const float* xt, float* gw, void* workspace,
                      size_t ws_bytes, void* stream) {
    if (!p || !gc || !gs || !gt || !xc || !xs || !xt || !gw) return MXC_ERR_NULL;
    Conv cv;
    int rc = conv_init(&cv, p, fmt, CONV_WGRAD);
    if (rc) return rc;
    if (!nv_pair_ok(cv.fa, cv.fb)) return MXC_ERR_ARG;
    if (wgrad_lean_splits(cv) == 0) return MXC_ERR_SHAPE;
    const size_t need = wgrad_workspace(cv);
    if (need && (!workspace || ws_bytes < need)) return MXC_ERR_WORKSPACE;
    if (!aligned16(gc) || !aligned16(gs) || !aligned16(gt) || !aligned16(xc) || !aligned16(xs) ||
        !aligned16(xt) || !aligned16(gw) || (need && !aligned16(workspace)))
        return MXC_ERR_ALIGN;
    return launch_wgrad(cv, gc, gs, xc, xs, gw, workspace, (hipStream_t)stream, gt, xt);
}

int mxconv_im2col_cbf(const mxc_conv* p, int fmt, const void* xc, const uint8_t* xs, void* cc,
                      uint8_t* cs, void* stream) {
    if (!p || !xc || !xs || !cc || !cs) return MXC_ERR_NULL;
    Conv cv;
    int rc = conv_init(&cv, p, fmt);
    if (rc) return rc;
    if (!aligned16(xc) || !aligned16(xs) || !aligned16(cc) || !aligned16(cs)) return MXC_ERR_ALIGN;
    return launch_im2col(cv, xc, xs, cc, cs, (hipStream_t)stream);
}

int mxconv_fwd(const mxc_conv* p, int fmt, const void* wc, const uint8_t* ws, const void* xc,
               const uint8_t* xs, void* y, int y_layout, void* stream) {
    if (!p || !wc || !ws || !xc || !xs || !y) return MXC_ERR_NULL;
    if (!out_layout_ok(y_layout)) return MXC_ERR_ARG;
    Conv cv;
    int rc = conv_init(&cv, p, fmt, CONV_FWD);
    if (rc) return rc;
    if (!aligned16(wc) || !aligned16(ws) || !aligned16(xc) || !aligned16(xs) || !aligned16(y))
        return MXC_ERR_ALIGN;
    return launch_fwd(cv, wc, ws, xc, xs, (float*)y, y_layout, (hipStream_t)stream);
}

int mxconv_dgrad(const mxc_conv* p, int fmt, const void* wc, const uint8_t* ws, const void* gc,
                 const uint8_t* gs, void* gx, int gx_layout, void* stream) {
    if (!p || !wc || !ws || !gc || !gs || !gx) return MXC_ERR_NULL;
    if (!out_layout_ok(gx_layout)) return MXC_ERR_ARG;
    Conv cv;
    int rc = conv_init(&cv, p, fmt, CONV_DGRAD);
    if (rc) return rc;
    if (!aligned16(wc) || !aligned16(ws) || !aligned16(gc) || !aligned16(gs) || !aligned16(gx))
        return MXC_ERR_ALIGN;
    return launch_dgrad(cv, wc, ws, gc, gs, (float*)gx, gx_layout, (hipStream_t)stream);
}

static int wgrad_call(const mxc_conv* p, int fmt, const void* gc, const uint8_t* gs, const void* xc,
                      const uint8_t* xs, float* gw, void* workspace, size_t ws_bytes, void* stream, bool defer) {
    if (!p || !gc || !gs || !xc || !xs || !gw) return MXC_ERR_NULL;
    Conv cv;
    int rc = conv_init(&cv, p, fmt, CONV_WGRAD);
    if (rc) return rc;
    const size_t need = wgrad_workspace(cv);
    if (need && (!workspace || ws_bytes < need)) return MXC_ERR_WORKSPACE;
    if (!aligned16(gc) || !aligned16(gs) || !aligned16(xc) || !aligned16(xs) || !aligned16(gw) ||
        (need && !aligned16(workspace)))
        return MXC_ERR_ALIGN;
    return launch_wgrad(cv, gc, gs, xc, xs, gw, workspace, (hipStream_t)stream, nullptr, nullptr, defer);
}

int mxconv_wgrad(const mxc_conv* p, int fmt, const void* gc, const uint8_t* gs, const void* xc,
                 const uint8_t* xs, float* gw, void* workspace, size_t ws_bytes, void* stream) {
    return wgrad_call(p, fmt, gc, gs, xc, xs, gw, workspace, ws_bytes, stream, false);
}

int mxconv_wgrad_deferred(const mxc_conv* p, int fmt, const void* gc, const uint8_t* gs, const void* xc,
                          const uint8_t* xs, float* gw, void* workspace, size_t ws_bytes, void* stream) {
    return wgrad_call(p, fmt, gc, gs, xc, xs, gw, workspace, ws_bytes, stream, true);
}

int mxconv_backward(const mxc_conv* p, int fmt, const void* wc, const uint8_t* ws, const void* gc,
                    const uint8_t* gs, const void* xc, const uint8_t* xs, void* gx, int gx_layout, float* gw,
                    void* workspace, size_t ws_bytes, int deferred, void* stream) {
    if (!p || !wc || !ws || !gc || !gs || !xc || !xs || !gx || !gw) return MXC_ERR_NULL;
    if (!out_layout_ok(gx_layout)) return MXC_ERR_ARG;
    if (deferred != 0 && deferred != 1) return MXC_ERR_ARG;
    // one fmt names (W, G_Y) for the input gradient and (G_Y, X) for the
    // weight gradient, so G_Y would take both halves of a mixed pair
    if ((fmt & 0x10) && ((fmt >> 2) & 3) != (fmt & 3)) return MXC_ERR_ARG;
    Conv dcv, wcv;
    int rc = conv_init(&dcv, p, fmt, CONV_DGRAD);
    if (rc) return rc;
    rc = conv_init(&wcv, p, fmt, CONV_WGRAD);
    if (rc) return rc;
    const size_t need = wgrad_workspace(wcv);
    if (need && (!workspace || ws_bytes < need)) return MXC_ERR_WORKSPACE;
    if (!aligned16(wc) || !aligned16(ws) || !aligned16(gc) || !aligned16(gs) || !aligned16(xc) ||
        !aligned16(xs) || !aligned16(gx) || !aligned16(gw) || (need && !aligned16(workspace)))
        return MXC_ERR_ALIGN;
    return launch_backward(dcv, wc, ws, gc, gs, (float*)gx, gx_layout, wcv, xc, xs, gw, workspace, (hipStream_t)stream,
                           deferred == 1);
}

int mxconv_wgrad_reduce_multi(int count, const mxc_wjob* jobs, void* stream) {
    if (count < 0 || count > MXC_WREDUCE_MAX) return MXC_ERR_ARG;
    if (count > 0 && !jobs) return MXC_ERR_NULL;
    WReduceJob q[MXC_WREDUCE_MAX];
    for (int i = 0; i < count; i++) {
        const mxc_wjob& j = jobs[i];
        if (!j.conv || !j.gw) return MXC_ERR_NULL;
        const int rc = conv_init(&q[i].cv, j.conv, j.fmt, CONV_WGRAD);
        if (rc) return rc;
        const size_t need = wgrad_workspace(q[i].cv);
        if (need && (!j.workspace || j.ws_bytes < need)) return MXC_ERR_WORKSPACE;
        if (!aligned16(j.gw) || (need && !aligned16(j.workspace))) return MXC_ERR_ALIGN;
        q[i].ws = j.workspace;
        q[i].gw = j.gw;
    }
    return launch_wgrad_reduce_multi(count, q, (hipStream_t)stream);
}

namespace {
// the fused kernels' shapes: batch block 32 (so the output tensor is also in
// blocks of 32 samples), kernel width 1 or 3, the strides the lean kernels run
bool fused_shape(const Conv& cv, bool dg) {
    if (cv.x.bn != 32 || (cv.kw != 1 && cv.kw != 3)) return false;
    return dg ? ((cv.sh == 1 && cv.sw == 1) || (cv.sh == 2 && cv.sw == 2)) : (cv.sw == 1 || cv.sw == 2);
}
}  // namespace

int mxconv_fwd_quant(const mxc_conv* p, int fmt, const void* wc, const uint8_t* ws, const void* xc,
                     const uint8_t* xs, int fn, int out_fmt, void* yc, uint8_t* ysc, void* y_act,
                     void* stream) {
    if (!p || !wc || !ws || !xc || !xs || !yc || !ysc) return MXC_ERR_NULL;
    const bool pre = (fn & MXC_FN_PRE_OUT) != 0, bf16 = (fn & MXC_FN_BF16) != 0;
    fn &= ~(MXC_FN_PRE_OUT | MXC_FN_BF16);
    if (fn < MXC_FN_NONE || fn > MXC_FN_SILU || !fmt_ok(out_fmt)) return MXC_ERR_ARG;
    Conv cv;
    int rc = conv_init(&cv, p, fmt, CONV_FWD);
    if (rc) return rc;
    if (!fused_shape(cv, false)) return MXC_ERR_SHAPE;
    if (!aligned16(wc) || !aligned16(ws) || !aligned16(xc) || !aligned16(xs) || !aligned16(yc) ||
        !aligned16(ysc) || (y_act && !aligned16(y_act)))
        return MXC_ERR_ALIGN;
    FusedEpi q{yc, ysc, out_fmt, fn, nullptr, pre, bf16};
    rc = launch_conv_lean(cv, false, wc, ws, xc, xs, (float*)y_act, MXC_CBF, (hipStream_t)stream, &q);
    return rc == 1 ? MXC_ERR_SHAPE : rc;
}

namespace {
int dgrad_quant_impl(const mxc_conv* p, int fmt, const void* wc, const uint8_t* ws, const void* gc, const uint8_t* gs,
                int fn, const void* z, int out_fmt, void* gxc, uint8_t* gxs, float* gx_act, void* stream, bool sr,
                uint64_t seed) {
    if (!p || !wc || !ws || !gc || !gs || !gxc || !gxs) return MXC_ERR_NULL;
    const bool bf16 = (fn & MXC_FN_BF16) != 0;
    fn &= ~MXC_FN_BF16;
    if (fn < MXC_FN_NONE || fn > MXC_FN_SILU || !fmt_ok(out_fmt)) return MXC_ERR_ARG;
    if (fn != MXC_FN_NONE && !z) return MXC_ERR_NULL;
    Conv cv;
    int rc = conv_init(&cv, p, fmt, CONV_DGRAD);
    if (rc) return rc;
    if (!fused_shape(cv, true)) return MXC_ERR_SHAPE;
    if (!aligned16(wc) || !aligned16(ws) || !aligned16(gc) || !aligned16(gs) || !aligned16(gxc) ||
        !aligned16(gxs) || (gx_act && !aligned16(gx_act)) || (fn != MXC_FN_NONE && !aligned16(z)))
        return MXC_ERR_ALIGN;
    FusedEpi q{gxc, gxs, out_fmt, fn, z, false, bf16};
    q.sr = sr;
    q.seed = seed;
    rc = launch_conv_lean(cv, true, wc, ws, gc, gs, gx_act, MXC_CBF, (hipStream_t)stream, &q);
    return rc == 1 ? MXC_ERR_SHAPE : rc;
}
}  // namespace

int mxconv_dgrad_quant(const mxc_conv* p, int fmt, const void* wc, const uint8_t* ws, const void* gc,
                       const uint8_t* gs, int fn, const void* z, int out_fmt, void* gxc, uint8_t* gxs,
                       float* gx_act, void* stream) {
    return dgrad_quant_impl(p, fmt, wc, ws, gc, gs, fn, z, out_fmt, gxc, gxs, gx_act, stream, false, 0);
}

int mxconv_dgrad_quant_sr(const mxc_conv* p, int fmt, const void* wc, const uint8_t* ws, const void* gc,
                          const uint8_t* gs, int fn, const void* z, int out_fmt, void* gxc, uint8_t* gxs,
                          float* gx_act, uint64_t seed, void* stream) {
    return dgrad_quant_impl(p, fmt, wc, ws, gc, gs, fn, z, out_fmt, gxc, gxs, gx_act, stream, true, seed);
}

// The weight gradient's split-K partial sums for callers that cannot
// allocate: one library-owned array per GPU.  Its name is a host-side
// stand-in; the device address on each GPU is looked up once, with that
// device current, and only that address is handed to kernels.
namespace {
__device__ __attribute__((aligned(256))) uint8_t scratch[MXC_NOALLOC_WS_MAX];
constexpr int SCRATCH_DEVICES = 64;
std::mutex g_scratch_mu;
void* g_scratch_ptr[SCRATCH_DEVICES];

int scratch_for_current_device(void** out) {
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= SCRATCH_DEVICES) return MXC_ERR_HIP;
    std::lock_guard<std::mutex> lock(g_scratch_mu);
    if (!g_scratch_ptr[dev]) {
        void* p = nullptr;
        if (hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)) != hipSuccess || !p) return MXC_ERR_HIP;
        g_scratch_ptr[dev] = p;
    }
    *out = g_scratch_ptr[dev];
    return MXC_OK;
}
}  // namespace

int mxconv_wgrad_noalloc(const mxc_conv* p, int fmt, const void* gc, const uint8_t* gs, const void* xc,
                         const uint8_t* xs, float* gw, void* stream) {
    if (!p || !gc || !gs || !xc || !xs || !gw) return MXC_ERR_NULL;
    Conv cv;
    int rc = conv_init(&cv, p, fmt, CONV_WGRAD);
    if (rc) return rc;
    const size_t need = wgrad_workspace(cv);
    if (need > MXC_NOALLOC_WS_MAX) return MXC_ERR_WORKSPACE;
    if (!aligned16(gc) || !aligned16(gs) || !aligned16(xc) || !aligned16(xs) || !aligned16(gw))
        return MXC_ERR_ALIGN;
    void* ws = nullptr;
    if (need) {
        rc = scratch_for_current_device(&ws);
        if (rc) return rc;
    }
    return launch_wgrad(cv, gc, gs, xc, xs, gw, ws, (hipStream_t)stream, nullptr, nullptr, false);
}

int mxconv_concat_cbf(int fmt, int n, int h, int w, int nparts, const mxc_part* parts, void* codes,
                      uint8_t* scales, void* stream) {
    if (!parts || !codes || !scales) return MXC_ERR_NULL;
    if (nparts < 1 || nparts > MXC_CONCAT_MAX || !fmt_ok(fmt)) return MXC_ERR_ARG;
    int total = 0;
    for (int k = 0; k < nparts; k++) {
        const mxc_part& q = parts[k];
        if (!q.codes || !q.scales) return MXC_ERR_NULL;
        if (q.ncb <= 0 || (q.up != 0 && q.up != 1)) return MXC_ERR_ARG;
        if (q.up && ((h & 1) || (w & 1))) return MXC_ERR_SHAPE;
        if (!aligned16(q.codes) || !aligned16(q.scales)) return MXC_ERR_ALIGN;
        if (total > 0x3FFFFFF - q.ncb) return MXC_ERR_SHAPE;
        total += q.ncb;
    }
    Geom g;
    const int rc = geom_init(&g, MXC_ACT, fmt, n, 32 * total, h, w);
    if (rc) return rc;
    if (!aligned16(codes) || !aligned16(scales)) return MXC_ERR_ALIGN;
    return launch_concat(g, parts, nparts, codes, scales, (hipStream_t)stream);
}

namespace {
int quantize_sum_impl(int fmt, int n, int c, int h, int w, int nterms, const mxc_term* terms, int fn, const void* z,
                 void* codes, uint8_t* scales, float* vals, void* stream, bool sr, uint64_t seed) {
    if (!terms || !codes || !scales) return MXC_ERR_NULL;
    if (nterms < 1 || nterms > MXC_TERMS_MAX) return MXC_ERR_ARG;
    const bool bf16 = (fn & MXC_FN_BF16) != 0;
    fn &= ~MXC_FN_BF16;
    if (fmt != MXC_E4M3 && fmt != MXC_E2M1) return MXC_ERR_ARG;
    if (fn < MXC_FN_NONE || fn > MXC_FN_SILU) return MXC_ERR_ARG;
    if (fn != MXC_FN_NONE && !z) return MXC_ERR_NULL;
    Geom g;
    int rc = geom_init(&g, MXC_ACT, fmt, n, c, h, w);
    if (rc) return rc;
    if (g.bn != 32) return MXC_ERR_SHAPE;
    for (int t = 0; t < nterms; t++) {
        const mxc_term& q = terms[t];
        if (!q.src) return MXC_ERR_NULL;
        if (q.c_src <= 0 || q.c_off < 0 || (q.down != 0 && q.down != 1)) return MXC_ERR_ARG;
        if ((long long)q.c_off + c > q.c_src) return MXC_ERR_SHAPE;
        if (q.down && ((long long)2 * h * 2 * w > 0x7FFFFFFFLL)) return MXC_ERR_SHAPE;
        if (!aligned16(q.src)) return MXC_ERR_ALIGN;
    }
    if (!aligned16(codes) || !aligned16(scales) || (vals && !aligned16(vals)) ||
        (fn != MXC_FN_NONE && !aligned16(z)))
        return MXC_ERR_ALIGN;
    return launch_quantize_sum(g, fmt, terms, nterms, fn, bf16, z, codes, scales, vals, (hipStream_t)stream, sr,
                               seed);
}
}  // namespace

int mxconv_quantize_sum(int fmt, int n, int c, int h, int w, int nterms, const mxc_term* terms, int fn,
                        const void* z, void* codes, uint8_t* scales, float* vals, void* stream) {
    return quantize_sum_impl(fmt, n, c, h, w, nterms, terms, fn, z, codes, scales, vals, stream, false, 0);
}

int mxconv_quantize_sum_sr(int fmt, int n, int c, int h, int w, int nterms, const mxc_term* terms, int fn,
                           const void* z, void* codes, uint8_t* scales, float* vals, uint64_t seed, void* stream) {
    return quantize_sum_impl(fmt, n, c, h, w, nterms, terms, fn, z, codes, scales, vals, stream, true, seed);
}

size_t mxconv_naive_codes_bytes(int64_t lines, int64_t len, int fmt) {
    if (lines <= 0 || len <= 0 || (fmt != MXC_E4M3 && fmt != MXC_E2M1)) return 0;
    const long long lp = naive_line_len(len);
    return (size_t)lines * lp * (fmt == MXC_E4M3 ? 8 : 4) / 8;
}

size_t mxconv_naive_scales_bytes(int64_t lines, int64_t len) {
    if (lines <= 0 || len <= 0) return 0;
    return (size_t)lines * (naive_line_len(len) / 32);
}

int mxconv_naive_im2col_f32(const mxc_conv* p, const float* x, float* col, void* stream) {
    if (!p || !x || !col) return MXC_ERR_NULL;
    Conv cv;
    int rc = conv_init(&cv, p, MXC_E4M3);
    if (rc) return rc;
    if (!aligned16(x) || !aligned16(col)) return MXC_ERR_ALIGN;
    return launch_naive_im2col(cv, x, col, (hipStream_t)stream);
}

int mxconv_naive_quantize_1d(const float* src, int64_t rows, int64_t cols, int dir, int fmt,
                             void* codes, uint8_t* scales, void* stream) {
    if (!src || !codes || !scales) return MXC_ERR_NULL;
    if (rows <= 0 || cols <= 0 || (dir != 0 && dir != 1) || (fmt != MXC_E4M3 && fmt != MXC_E2M1))
        return MXC_ERR_ARG;
    if (!aligned16(src) || !aligned16(codes) || !aligned16(scales)) return MXC_ERR_ALIGN;
    return launch_naive_q1d(src, rows, cols, dir, fmt, codes, scales, (hipStream_t)stream);
}

int mxconv_naive_fwd(const mxc_conv* p, int fmt, const void* cc, const uint8_t* cs, const void* wc,
                     const uint8_t* ws, float* y, void* stream) {
    if (!p || !cc || !cs || !wc || !ws || !y) return MXC_ERR_NULL;
    if (fmt != MXC_E4M3 && fmt != MXC_E2M1) return MXC_ERR_ARG;   // the comparator runs MXFP8 / MXFP4
    Conv cv;
    int rc = conv_init(&cv, p, fmt);
    if (rc) return rc;
    if (!aligned16(cc) || !aligned16(cs) || !aligned16(wc) || !aligned16(ws) || !aligned16(y))
        return MXC_ERR_ALIGN;
    return launch_naive_fwd(cv, cc, cs, wc, ws, y, (hipStream_t)stream);
}

int mxconv_naive_dgrad(const mxc_conv* p, int fmt, const void* gc, const uint8_t* gs,
                       const void* wtc, const uint8_t* wts, float* gcol, float* gx, void* stream) {
    if (!p || !gc || !gs || !wtc || !wts || !gcol || !gx) return MXC_ERR_NULL;
    if (fmt != MXC_E4M3 && fmt != MXC_E2M1) return MXC_ERR_ARG;   // the comparator runs MXFP8 / MXFP4
    Conv cv;
    int rc = conv_init(&cv, p, fmt);
    if (rc) return rc;
    if (!aligned16(gc) || !aligned16(gs) || !aligned16(wtc) || !aligned16(wts) || !aligned16(gcol) ||
        !aligned16(gx))
        return MXC_ERR_ALIGN;
    return launch_naive_dgrad(cv, gc, gs, wtc, wts, gcol, gx, (hipStream_t)stream);
}

int mxconv_naive_wgrad(const mxc_conv* p, int fmt, const void* gtc, const uint8_t* gts,
                       const void* xtc, const uint8_t* xts, float* gw, void* stream) {
    if (!p || !gtc || !gts || !xtc || !xts || !gw) return MXC_ERR_NULL;
    if (fmt != MXC_E4M3 && fmt != MXC_E2M1) return MXC_ERR_ARG;   // the comparator runs MXFP8 / MXFP4
    Conv cv;
    int rc = conv_init(&cv, p, fmt);
    if (rc) return rc;
    if (!aligned16(gtc) || !aligned16(gts) || !aligned16(xtc) || !aligned16(xts) || !aligned16(gw))
        return MXC_ERR_ALIGN;
    return launch_naive_wgrad(cv, gtc, gts, xtc, xts, gw, (hipStream_t)stream);
}

const char* mxconv_strerror(int code) {
    switch (code) {
        case MXC_OK: return "ok";
        case MXC_ERR_NULL: return "a required pointer is NULL";
        case MXC_ERR_ARG: return "bad enum value or non-positive size";
        case MXC_ERR_SHAPE: return "unsupported shape (batch must divide 32 or be a multiple of 32; "
                                   "E2M1 needs at least 2 samples per block, FP6 at least 4; output must be non-empty; "
                                   "FP6 GEMMs need batch block 32 and the lean kernels' shapes)";
        case MXC_ERR_ALIGN: return "device pointer not 16-byte aligned";
        case MXC_ERR_HIP: return "HIP launch error";
        case MXC_ERR_WORKSPACE: return "workspace missing or too small";
        default: return "unknown error";
    }
}

}  // extern "C"
