// conv_lean_bwd.hip -- a layer's input gradient and batch-block-32 weight
// gradient in one launch (conv_lean_bwd_kernel, conv_lean_kern.h).
#include "conv_lean_kern.h"

namespace mxc {

namespace {

template <int F, int KW, int PW, bool DG2, int NB, int NRB = 2, bool KR = false>
int bwd_launch(const LeanArgs& a, const WLArgs& q, int nl, int grid, size_t lds, hipStream_t s) {
    static std::atomic<uint64_t> devs{0};
    if (raise_lds(conv_lean_bwd_kernel<F, KW, PW, DG2, NB, NRB, KR>, devs, lds)) return MXC_ERR_HIP;
    hipLaunchKernelGGL((conv_lean_bwd_kernel<F, KW, PW, DG2, NB, NRB, KR>), dim3(grid), dim3(LT), lds, s, a, q, nl);
    return hipGetLastError() == hipSuccess ? MXC_OK : MXC_ERR_HIP;
}

template <int F, int NB>
int bwd_launch_nb(const LeanArgs& a, const WLArgs& q, int nl, int grid, size_t lds, bool dg2, int kw, int pw, bool kr,
                  hipStream_t s) {
    if constexpr (F == MXC_E2M1) {
        if (pw == NARROW_PW) {
            if (kw == 3 && kr)
                return dg2 ? bwd_launch<F, 3, NARROW_PW, true, NB, 1, true>(a, q, nl, grid, lds, s)
                           : bwd_launch<F, 3, NARROW_PW, false, NB, 1, true>(a, q, nl, grid, lds, s);
            if (dg2) return kw == 3 ? bwd_launch<F, 3, NARROW_PW, true, NB, 1>(a, q, nl, grid, lds, s)
                                    : bwd_launch<F, 1, NARROW_PW, true, NB, 1>(a, q, nl, grid, lds, s);
            return kw == 3 ? bwd_launch<F, 3, NARROW_PW, false, NB, 1>(a, q, nl, grid, lds, s)
                           : bwd_launch<F, 1, NARROW_PW, false, NB, 1>(a, q, nl, grid, lds, s);
        }
    }
    if (dg2) {
        if (kw == 3) return pw == 1 ? bwd_launch<F, 3, 1, true, NB>(a, q, nl, grid, lds, s) : bwd_launch<F, 3, 2, true, NB>(a, q, nl, grid, lds, s);
        return pw == 1 ? bwd_launch<F, 1, 1, true, NB>(a, q, nl, grid, lds, s) : bwd_launch<F, 1, 2, true, NB>(a, q, nl, grid, lds, s);
    }
    if (kw == 3) return pw == 1 ? bwd_launch<F, 3, 1, false, NB>(a, q, nl, grid, lds, s) : bwd_launch<F, 3, 2, false, NB>(a, q, nl, grid, lds, s);
    return pw == 1 ? bwd_launch<F, 1, 1, false, NB>(a, q, nl, grid, lds, s) : bwd_launch<F, 1, 2, false, NB>(a, q, nl, grid, lds, s);
}

template <int F>
int bwd_launch_f(const LeanArgs& a, const WLArgs& q, int nl, int grid, size_t lds, bool dg2, int kw, int pw, bool kr,
                 bool nb1, hipStream_t s) {
    return nb1 ? bwd_launch_nb<F, 1>(a, q, nl, grid, lds, dg2, kw, pw, kr, s)
               : bwd_launch_nb<F, 2>(a, q, nl, grid, lds, dg2, kw, pw, kr, s);
}

}  // namespace

// Input gradient (dcv) and weight gradient (wcv, `splits` ways into wdst) of
// one layer in one launch; returns 1 when the layer or its formats are
// outside the grouped kernel (the caller then launches the two separately).
int launch_lean_bwd(const Conv& dcv, const void* wc, const uint8_t* ws, const void* gc, const uint8_t* gs,
                    float* gx, int layout, const Conv& wcv, const void* xc, const uint8_t* xs, float* wdst,
                    int splits, hipStream_t s) {
    const int f = dcv.fa;
    if ((f != MXC_E4M3 && f != MXC_E2M1) || dcv.fb != f || wcv.fa != f || wcv.fb != f) return 1;
    LeanPlan P;
    const int prc = lean_plan(dcv, true, wc, ws, gc, gs, gx, layout, nullptr, nullptr, nullptr, P);
    if (prc) return prc;
    if (P.rb == 1 && P.pw != NARROW_PW) return 1;        // a narrow shape this kernel is not built for
    WLArgs q;
    const long wg = wgrad_lean_fill(wcv, gc, gs, xc, xs, wdst, splits, nullptr, nullptr, q);
    if (wg < 0) return MXC_ERR_SHAPE;
    LeanArgs& a = P.a;
    const long nl = ((long)(P.dg2 ? a.pofs[4] : a.ntiles) + 7) / 8 * 8;
    if (nl + wg > 0x7FFFFFFFL) return MXC_ERR_SHAPE;
    // ring depth for the combined grid, every workgroup holding at least the
    // LDS the weight-gradient tile sums its four waves through (64 KB, or
    // 16 KB on 32 x 32 tiles)
    const bool nb1 = wgrad_single_block(wcv);
    const long red = nb1 ? 16384 : 65536;
    const long per_cu = (nl + wg + 255) / 256;
    int nbuf = 2;
    for (int b = 4; b > 2; b--) {
        const long need = (long)b * a.stage_bytes > red ? (long)b * a.stage_bytes : red;
        if (per_cu * need <= LDS_MAX) { nbuf = b; break; }
    }
    a.nbuf = nbuf;
    const int used = nbuf < P.nstage ? nbuf : P.nstage;
    size_t lds = lean_lds(a, used);
    if (lds < (size_t)red) lds = (size_t)red;
    const int grid = (int)(nl + wg);
    return f == MXC_E4M3 ? bwd_launch_f<MXC_E4M3>(a, q, (int)nl, grid, lds, P.dg2, dcv.kw, P.pw, P.krow, nb1, s)
                         : bwd_launch_f<MXC_E2M1>(a, q, (int)nl, grid, lds, P.dg2, dcv.kw, P.pw, P.krow, nb1, s);
}
}  // namespace mxc
