// conv_lean.hip -- launch planning for the lean forward / input-gradient
// kernels (conv_lean_kern.h): the tile shape, stage layout and ring depth of
// a layer, then the launch through the translation unit of its formats.
#include "conv_lean_kern.h"

namespace mxc {

// The tile shape, stage layout and ring depth of one launch; returns 0, 1
// when the layer is outside this kernel's shapes, or an MXC_* code.
int lean_plan(const Conv& cv, bool dg, const void* wc, const uint8_t* ws, const void* sc, const uint8_t* ss,
              float* out, int layout, const FusedEpi* q, const float* nv_tw, const float* nv_tx, LeanPlan& P) {
    const bool nv = nv_tw != nullptr;
    if (nv && (q || !nv_pair_ok(cv.fa, cv.fb))) return MXC_ERR_ARG;
    if (cv.x.bn != 32) return 1;
    if (cv.kw != 1 && cv.kw != 3) return 1;
    // input gradient: stride 1, or 2 in both directions (phases); forward:
    // column stride 1 or 2, any row stride
    const bool dg2 = dg && cv.sh == 2 && cv.sw == 2;
    if (dg ? !(dg2 || (cv.sh == 1 && cv.sw == 1)) : (cv.sw != 1 && cv.sw != 2)) return 1;
    LeanArgs& a = P.a;
    a.wc = (const uint8_t*)wc; a.ws = ws; a.sc = (const uint8_t*)sc; a.ss = ss;
    a.out = out; a.layout = layout;
    a.M = dg ? cv.cin : cv.cout;
    a.qcodes = q ? (uint8_t*)q->codes : nullptr;
    a.qscales = q ? q->scales : nullptr;
    a.qfmt = q ? q->fmt : 0;
    a.q_ncb = (a.M + 31) / 32;
    a.fn = q ? q->fn : MXC_FN_NONE;
    a.pre_out = q && q->pre ? 1 : 0;
    a.bf16 = q && q->bf16 ? 1 : 0;
    a.zpre = q ? q->z : nullptr;
    a.sr = q && q->sr ? 1 : 0;
    a.sk0 = q ? (uint32_t)q->seed : 0u;
    a.sk1 = q ? (uint32_t)(q->seed >> 32) : 0u;
    a.tw = nv_tw; a.tx = nv_tx;
    const Geom& src = dg ? cv.gy : cv.x;
    a.hsrc = src.h; a.wsrc = src.w;
    a.hout = dg ? cv.h : cv.ho;
    a.wout = dg ? cv.w : cv.wo;
    a.kh = cv.kh; a.sh = cv.sh; a.ph = cv.ph; a.pw = cv.pw;
    a.kwf = cv.kw;
    a.kcb = src.ncb;
    a.w_rowblocks = dg ? cv.wt.ncb : cv.wt.np / 32;
    a.w_cp = cv.wt.cp; a.w_ncb = cv.wt.ncb; a.w_nco = cv.wt.np / 32;
    a.x_ncb = src.ncb;
    a.xrows = src.ncb == 1 ? src.c : 32;
    if (dg && a.w_nco != src.ncb) return 1;
    // rows per tile: 64 rows x 8 pixels at column stride 1; the forward at
    // column stride 2, whose halo is twice as wide, takes 64 rows x 4 pixels
    // (measured faster in the network step than 128 x 4 or 64 x 8: the
    // five downsampling layers 142 -> 131 µs together)
    const int wgm = 1;
    int pw = !dg && cv.sw == 2 ? 1 : 2;
    // a single 32-row block of FP4 rows: narrow tiles (32 rows x 16 pixels)
    const bool narrow = a.M <= 32 && cv.fa == MXC_E2M1 && cv.fb == MXC_E2M1 && !nv;
    int rb = 2;
    // tiles of a tile shape; for the stride-2 input gradient, per phase
    // (ry, rx), whose pixel grids are the output rows / columns of that parity
    auto count = [&](int wgm_, int pw_, int rb_, bool fill) -> long long {
        const int px_ = pw_ * 4 / wgm_;
        const int rows = 32 * rb_ * wgm_;
        const long long mt = (a.M + rows - 1) / rows;
        if (!dg2) return mt * ((a.wout + px_ - 1) / px_) * a.hout * src.ng;
        long long t = 0;
        for (int ph = 0; ph < 4; ph++) {
            const int gh = (a.hout - (ph >> 1) + 1) / 2, gw = (a.wout - (ph & 1) + 1) / 2;
            t += mt * ((gw + px_ - 1) / px_) * gh * src.ng;
            if (fill) a.pofs[ph + 1] = t <= 0x7FFFFFF0LL ? (int)t : 0;
        }
        return t;
    };
    // Narrow tiles of 8 pixels instead of 16 (half the stage ring, more
    // workgroups on a CU's LDS) where that measured faster in the network
    // step: the forward at column stride 2 and the fused input gradient,
    // except at stride 2 with kernel-row pairing (a single K block), which
    // keeps 16 (210 vs 246 µs on the second layer); the grouped backward
    // (no fused epilogue) keeps 16 as well.
    const bool kr_cand = a.kcb == 1 && cv.kw == 3 && (dg2 ? (cv.kh + 1) / 2 : cv.kh) >= 2;
    const bool half = dg ? (q != nullptr && !(dg2 && kr_cand)) : cv.sw == 2;
    // a layer whose tiles would leave a quarter of the CUs idle takes one
    // pixel per wave instead: twice the workgroups, more waves streaming
    // operands and storing results at once (measured: faster below ~200
    // tiles, slower from ~400)
    if (narrow && count(1, NARROW_PW, 1, false) >= 192) { pw = half ? NARROW_PW2 : NARROW_PW; rb = 1; }
    else if (count(wgm, pw, 2, false) < 192 || nv) pw = 1;
    const int px = pw * 4 / wgm;
    a.mtiles = (a.M + 32 * rb * wgm - 1) / (32 * rb * wgm);
    for (int i = 0; i < 5; i++) a.pofs[i] = 0;
    const long long nt = count(wgm, pw, rb, true);
    if (nt <= 0 || nt > 0x7FFFFFF0LL) return 1;
    a.ntiles = (int)nt;
    // stage layout: DMA slices of the weight blocks, then the halo blocks,
    // rounded to whole 4 KB groups, then the scale entries; at stride 2 the
    // widest phase has (kw + 1) / 2 taps per row
    // (weights: format fa; source: fb; FP4 blocks take half a 1 KB slice)
    const int bpiw = cv.fa == MXC_E2M1 ? 2 : 1, bpix = cv.fb == MXC_E2M1 ? 2 : 1;
    const int kwt = dg2 ? (cv.kw + 1) / 2 : cv.kw;
    const int hp = dg ? px + kwt - 1 : (px - 1) * cv.sw + cv.kw;
    const int na = kwt * 2 * rb * wgm, nb = 2 * hp;
    const int nq = (na / bpiw + nb / bpix + 3) / 4;
    a.stage_bytes = nq * 4096 + (nv ? 4096 : SCALE_REGION);
    // a single K block and two or more kernel rows: stages pair kernel rows
    // (the narrow FP4 kernels; NVFP keeps its own stage layout)
    const int krows = dg2 ? (cv.kh + 1) / 2 : cv.kh;
    const bool krow = a.kcb == 1 && krows >= 2 && rb == 1 && cv.kw == 3 && !nv;
    const int nstage = krow ? (krows + 1) / 2 : krows * ((a.kcb + 1) / 2);
    if (2 * a.stage_bytes > LDS_MAX || nstage < 1) return 1;
    // ring depth: the workgroups that share a CU at this grid size split its
    // LDS; each takes as many stage buffers (2..4) as fit in its share
    const int per_cu = (int)((nt + 255) / 256);
    // the fused input gradient with a bf16 z prefetches its z tiles
    const bool zpf = dg && q && q->bf16 && q->fn != MXC_FN_NONE && !nv;
    const int zsl = a.M <= 16 ? 1 : 2;
    const long zb = zpf ? (long)lean_z_lds(pw, rb, zsl) : 0;
    int nbuf = 2;
    for (int b = 4; b > 2; b--)
        if ((long)per_cu * (b * a.stage_bytes + zb) <= LDS_MAX) { nbuf = b; break; }
    a.nbuf = nbuf;
    const int used = nbuf < nstage ? nbuf : nstage;
    a.zoff = 0; a.zpw = pw; a.zrb = rb; a.zsl = zsl;
    if (zpf) {
        // only where two workgroups still fit a CU's LDS: the kernels hold
        // two per CU by their registers, and halving that costs more than
        // the prefetch saves (measured)
        const size_t ring = lean_ring_lds(a, used);
        if (ring + lean_z_lds(pw, rb, zsl) <= (size_t)LDS_MAX / 2) a.zoff = (int)ring;
    }
    P.wgm = wgm; P.pw = pw; P.rb = rb; P.nstage = nstage; P.used = used; P.dg2 = dg2; P.krow = krow;
    return 0;
}

// Returns 1 when the layer is outside this kernel's shapes (the caller then
// uses the general kernels), else an MXC_* code.
int launch_conv_lean(const Conv& cv, bool dg, const void* wc, const uint8_t* ws, const void* sc,
                     const uint8_t* ss, float* out, int layout, hipStream_t s, const FusedEpi* q,
                     const float* nv_tw, const float* nv_tx) {
    LeanPlan P;
    const int prc = lean_plan(cv, dg, wc, ws, sc, ss, out, layout, q, nv_tw, nv_tx, P);
    if (prc) return prc;
    const LeanArgs& a = P.a;
    const LeanShape h{cv.kw, cv.sw, P.wgm, P.pw, P.rb, P.krow, P.used};
    if (nv_tw) return cv.fa == MXC_E2M1 ? lean_nv(cv.fa, cv.fb, a, dg, h, s) : lean_nv68(cv.fa, cv.fb, a, dg, h, s);
    if (cv.fa == MXC_E4M3 && cv.fb == MXC_E4M3) return dg ? lean_dg_e4m3(a, h, s) : lean_fwd_e4m3(a, h, s);
    if (cv.fa == MXC_E2M1 && cv.fb == MXC_E2M1) return dg ? lean_dg_e2m1(a, h, s) : lean_fwd_e2m1(a, h, s);
    return lean_fp6(cv.fa, cv.fb, a, dg, h, s);
}

}  // namespace mxc
