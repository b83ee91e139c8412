// wgrad_tile.h -- the weight-gradient tile of the batch-block-32 kernel
// (a5), shared by its own kernel and by the grouped backward launch.
// Included inside namespace mxc by .hip files only.
#pragma once

namespace {


constexpr int WT = 256;


struct WLArgs {
    const uint8_t* gc;
    const uint8_t* gs;
    const uint8_t* xc;
    const uint8_t* xs;
    float* dst;
    int direct;                    // 1: dst is G_W (OIHW); 0: partial tiles
    int cout, cin, kh, kw, sh, sw, ph, pw, ho, wo, h, w;
    int gy_ncb, x_ncb, gy_cp, x_cp, ntot;
    int npix, npairs;              // output pixels (all batch groups), pixel pairs (rows x ppr)
    int ppr;                       // pixel pairs per output row: ceil(wo / 2)
    int cot, cit, ntiles;          // 64-row / 64-column tile counts, tiles
    int ppw;                       // pixel pairs per wave
    int nsplit;
    // NVFP4 operands: gs / xs hold E4M3 scales per 8x8 block ([pixel][Cp/8][4]:
    // a row's four sample groups in four consecutive bytes); tg, tx the
    // per-tensor scales
    const float* tg;
    const float* tx;
};

// One operand's fragment for a K step: K block 0 from pixel row p0, K block
// 1 from p1 (rows already offset to this lane's row), zeroed where v0 / v1
// say the block or row does not exist.  FP8: 16 bytes of each (the lane's
// half of the row); FP4 and FP6: the whole row of the lane's own K block
// (ph, vh = p0, v0 or p1, v1 by lane half).  Invalid rows still load from a
// valid address (the caller points them at an existing row) and are zeroed
// afterwards.  The loads name the global address space explicitly: where
// the compiler cannot prove it (a per-lane choice between two pointers) it
// emits flat loads, which also count against the LDS / scalar-load counter,
// so every later wait on that counter drained the whole batch (measured:
// the weight gradient of the image layer ran at a quarter of its speed).
typedef const __attribute__((address_space(1))) v4i g_v4i;
typedef const __attribute__((address_space(1))) v2i g_v2i;
template <int F>
__device__ __forceinline__ v8i row_frag(const uint8_t* p0, const uint8_t* p1, const uint8_t* ph, bool v0, bool v1,
                                        bool vh) {
    v8i o;
    if constexpr (F == MXC_E4M3) {
        const v4i u = *(g_v4i*)p0, v = *(g_v4i*)p1;
#pragma unroll
        for (int e = 0; e < 4; e++) { o[e] = v0 ? u[e] : 0; o[4 + e] = v1 ? v[e] : 0; }
    } else if constexpr (fmt_bits(F) == 6) {
        const v2i a = *(g_v2i*)ph, b = *(g_v2i*)(ph + 8), c = *(g_v2i*)(ph + 16);
        o[0] = a[0]; o[1] = a[1]; o[2] = b[0]; o[3] = b[1]; o[4] = c[0]; o[5] = c[1];
        o[6] = o[7] = 0;
#pragma unroll
        for (int e = 0; e < 6; e++) o[e] = vh ? o[e] : 0;
    } else {
        const v4i u = *(g_v4i*)ph;
#pragma unroll
        for (int e = 0; e < 4; e++) { o[e] = vh ? u[e] : 0; o[4 + e] = 0; }
    }
    return o;
}

// NV: NVFP operands, decoded per fragment (fp16 for FP4 / FP6, bf16 for FP8)
// and multiplied on fp16 / bf16 MFMAs (the 8-sample groups of a row each
// have their own E4M3 scale).
// NB: 32-row blocks per tile side -- 2 (a 64 x 64 tile), or 1 for a layer
// whose G_Y and X both have a single channel block (a 32 x 32 tile: half the
// loads and a quarter of the products per pixel pair, so twice the pairs per
// batch).
// KT: taps of one kernel row per wave (3 for a 3-wide kernel on 32 x 32
// tiles, else 1): each G_Y fragment of a pixel pair is loaded once and
// multiplied with the X fragments of all KT taps, instead of once per tap.
template <int FA, int FB, bool NV = false, int NB = 2, int KT = 1>
__device__ __forceinline__ void wgrad_tile(const WLArgs& p, int bid, int nblk, float (*red)[32 * NB * 32 * NB]) {
    static_assert(!NV || (FA == FB && FA != MXC_E3M2) || (FA == MXC_E2M1 && FB == MXC_E3M2),
                  "NVFP pairs: one format (FP4, E2M3, FP8), or FP4 gradients with E3M2 activations");
    static_assert(NB == 1 || NB == 2, "one or two blocks per tile side");
    static_assert(KT == 1 || (NB == 1 && !NV), "several taps per wave on 32 x 32 MX tiles only");
    constexpr int RS = 32 * NB;                   // tile side; red[wave] holds RS x RS floats
    constexpr int RBA = 32 * fmt_bits(FA) / 8;    // bytes of one block row (32 samples): G_Y
    constexpr int RBB = 32 * fmt_bits(FB) / 8;    // X
    constexpr int TBA = 32 * RBA, TBB = 32 * RBB; // bytes of one block

    const int tid = threadIdx.x, lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    // XCD-aware order: workgroups are dealt round-robin to the 8 XCDs; give
    // each XCD a contiguous range of (split, tile), so the tiles (taps, channel
    // blocks) that read the same pixels share that XCD's L2
    const int per_xcd = (nblk + 7) / 8;
    const int lin = (bid % 8) * per_xcd + bid / 8;
    if (lin >= p.ntiles * p.nsplit) return;
    const int tile = lin % p.ntiles, split = lin / p.ntiles;
    const int tap = tile / (p.cot * p.cit);
    const int rc = tile % (p.cot * p.cit);
    const int cop = rc / p.cit, cip = rc % p.cit;
    const int kwg = p.kw / KT;                    // tap groups per kernel row
    const int th = tap / kwg, tw = (tap % kwg) * KT;   // kernel row, first tap of the group
    const int r = lane & 31, hf = lane >> 5;

    // lane offsets inside one pixel's codes, and block validity
    uint32_t a_off[2], b_off[2];
    bool a_ok[2], b_ok[2];      // the block exists
    bool a_row[2], b_row[2];    // ... and this lane's channel row is real (padding rows hold +0 codes)
#pragma unroll
    for (int i = 0; i < 2; i++) {
        const int cob = 2 * cop + i, cib = 2 * cip + i;
        a_ok[i] = cob < p.gy_ncb;
        b_ok[i] = cib < p.x_ncb;
        a_row[i] = a_ok[i] && cob * 32 + r < p.cout;
        b_row[i] = b_ok[i] && cib * 32 + r < p.cin;
        // a lane without a real row reads row 0 of its block (or of block 0):
        // a line the real rows fetch anyway
        a_off[i] = (uint32_t)(a_ok[i] ? cob : 0) * TBA + (a_row[i] ? r * RBA : 0) + (FA == MXC_E4M3 ? 16 * hf : 0);
        b_off[i] = (uint32_t)(b_ok[i] ? cib : 0) * TBB + (b_row[i] ? r * RBB : 0) + (FB == MXC_E4M3 ? 16 * hf : 0);
    }
    const uint32_t gy_pix = (uint32_t)p.gy_ncb * TBA, x_pix = (uint32_t)p.x_ncb * TBB;

    v16f acc[KT][NB][NB];
#pragma unroll
    for (int t = 0; t < KT; t++)
#pragma unroll
        for (int i = 0; i < NB; i++)
#pragma unroll
            for (int j = 0; j < NB; j++)
#pragma unroll
                for (int e = 0; e < 16; e++) acc[t][i][j][e] = 0.0f;

    const int wid = split * 4 + wave;
    const int q0 = wid * p.ppw;
    const int q1 = min(p.npairs, q0 + p.ppw);

    // operands of one pair (pixels 2 j and 2 j + 1 of an output row)
    struct Ops {
        v8i a[2], b[KT][2];
        int sa[2], sb[KT][2];
        uint32_t na[2], nb[2];     // NV: the four E4M3 scales of the lane's row
    };

    // Pairs run along output rows: pair pj of row crow = (group, oy) holds
    // pixels 2 pj and 2 pj + 1 (a row of odd width ends with a half pair).
    // The wave walks its range with this cursor and per-row bases, so the
    // per-pair work is a few scalar adds and compares; the lane of half hf
    // takes pixel 2 pj + hf for FP4 / FP6 (its K block), both for FP8.
    int crow = q0 / p.ppr, pj = q0 % p.ppr;
    // per-row state: pixel indices and byte offsets of the row's first G_Y
    // pixel and of the tap's X row, scale offsets, and whether that X row exists
    size_t pa_row = 0, px_row = 0, ga_row = 0, xb_row = 0, gs_row = 0, xs_row = 0;
    bool rv = false;
    auto set_row = [&]() {
        const int g = crow / p.ho, oy = crow - g * p.ho;
        const int iy = oy * p.sh + th - p.ph;
        rv = iy >= 0 && iy < p.h;
        pa_row = (size_t)crow * p.wo;
        px_row = rv ? ((size_t)g * p.h + iy) * p.w : 0;
        ga_row = pa_row * gy_pix;
        gs_row = pa_row * p.gy_ncb;
        xb_row = px_row * x_pix;
        xs_row = px_row * p.x_ncb;
    };
    set_row();

    // pixel 2 pj + k of the cursor's row: validity of G_Y (inside the row and
    // the wave's range) and of X (also inside the input), and their pixel
    // offsets within the row bases
    auto load = [&](bool live, Ops& o) {
        int oxk[2];
        bool va[2];
        int ixk[KT][2];
        bool vb[KT][2];
#pragma unroll
        for (int k = 0; k < 2; k++) {
            const int ox = 2 * pj + k;
            va[k] = live && ox < p.wo;
            oxk[k] = va[k] ? ox : 0;
#pragma unroll
            for (int t = 0; t < KT; t++) {
                const int ix = ox * p.sw + tw + t - p.pw;
                vb[t][k] = va[k] && rv && ix >= 0 && ix < p.w;
                ixk[t][k] = vb[t][k] ? ix : 0;
            }
        }
        // the lane's own pixel (FP4 / FP6, and the scales of every format)
        const int oxh = hf ? oxk[1] : oxk[0];
        const bool vah = hf ? va[1] : va[0];
        const uint8_t* const gr = p.gc + ga_row;
        const uint8_t* const xr = p.xc + xb_row;
#pragma unroll
        for (int i = 0; i < NB; i++) {
            const uint8_t* a0 = gr + (uint32_t)oxk[0] * gy_pix + a_off[i];
            const uint8_t* a1 = gr + (uint32_t)oxk[1] * gy_pix + a_off[i];
            const uint8_t* ah = gr + (uint32_t)oxh * gy_pix + a_off[i];
            o.a[i] = row_frag<FA>(a0, a1, ah, va[0] && a_row[i], va[1] && a_row[i], vah && a_row[i]);
            // scale of (row, K block hf): the pixel of this lane's half
            const int cob = 2 * cop + i, cib = 2 * cip + i;
            const bool sav = vah && a_ok[i];
            const uint8_t sa = p.gs[gs_row + (uint32_t)oxh * p.gy_ncb + (a_ok[i] ? cob : 0)];
            o.sa[i] = sav ? sa : 0;
            int ixh = 0;
            bool vbh = false;
#pragma unroll
            for (int t = 0; t < KT; t++) {
                ixh = hf ? ixk[t][1] : ixk[t][0];
                vbh = hf ? vb[t][1] : vb[t][0];
                const uint8_t* b0 = xr + (uint32_t)ixk[t][0] * x_pix + b_off[i];
                const uint8_t* b1 = xr + (uint32_t)ixk[t][1] * x_pix + b_off[i];
                const uint8_t* bh = xr + (uint32_t)ixh * x_pix + b_off[i];
                o.b[t][i] = row_frag<FB>(b0, b1, bh, vb[t][0] && b_row[i], vb[t][1] && b_row[i], vbh && b_row[i]);
                const uint8_t sb = p.xs[xs_row + (uint32_t)ixh * p.x_ncb + (b_ok[i] ? cib : 0)];
                o.sb[t][i] = vbh && b_ok[i] ? sb : 0;
            }
            if constexpr (NV) {
                // E4M3 scales of the lane's row: the four sample groups of a
                // pixel in one word (KT == 1 here)
                const bool sbv = vbh && b_ok[i];
                const uint32_t* ga = (const uint32_t*)p.gs;
                const uint32_t* xa = (const uint32_t*)p.xs;
                const uint32_t ca = (uint32_t)(a_ok[i] ? cob : 0) * 4 + (r >> 3);
                const uint32_t cb = (uint32_t)(b_ok[i] ? cib : 0) * 4 + (r >> 3);
                if constexpr (FA == MXC_E4M3) {
                    // the lane holds samples 16 hf .. 16 hf + 15 of both
                    // pixels: sample groups 2 hf, 2 hf + 1 of each
                    uint32_t wa[2], wb[2];
#pragma unroll
                    for (int k = 0; k < 2; k++) {
                        const uint32_t u = ga[(pa_row + oxk[k]) * (p.gy_cp / 8) + ca];
                        const uint32_t v = xa[(px_row + ixk[0][k]) * (p.x_cp / 8) + cb];
                        wa[k] = va[k] && a_ok[i] ? (u >> (16 * hf)) & 0xFFFFu : 0u;
                        wb[k] = vb[0][k] && b_ok[i] ? (v >> (16 * hf)) & 0xFFFFu : 0u;
                    }
                    o.na[i] = wa[0] | wa[1] << 16;
                    o.nb[i] = wb[0] | wb[1] << 16;
                } else {   // all 32 samples of the lane's own pixel
                    const uint32_t va4 = ga[(pa_row + oxh) * (p.gy_cp / 8) + ca];
                    const uint32_t vb4 = xa[(px_row + ixh) * (p.x_cp / 8) + cb];
                    o.na[i] = sav ? va4 : 0u;
                    o.nb[i] = sbv ? vb4 : 0u;
                }
            }
        }
    };

    // batches of PB pairs: all loads of a batch are in flight together (the
    // loop is bound by memory latency, not by the MFMAs); pairs past the
    // wave's range get zero operands and add nothing
    constexpr int PB = NV ? 2 : NB == 1 ? (KT > 1 ? 4 : 8) : 4;
    for (int q = q0; q < q1; q += PB) {
        Ops o[PB];
#pragma unroll
        for (int b = 0; b < PB; b++) {
            load(q + b < q1, o[b]);
            if (++pj == p.ppr) {                      // next output row
                pj = 0;
                ++crow;
                if (q + b + 1 < q1) set_row();
            }
        }
#pragma unroll
        for (int b = 0; b < PB; b++) {
            if constexpr (NV) {
                uint32_t ad[NB][16], bd[NB][16];
#pragma unroll
                for (int i = 0; i < NB; i++) {
                    nv_decode32<FA>(o[b].a[i], o[b].na[i], ad[i]);
                    nv_decode32<FB>(o[b].b[0][i], o[b].nb[i], bd[i]);
                }
#pragma unroll
                for (int i = 0; i < NB; i++)
#pragma unroll
                    for (int j = 0; j < NB; j++)
                        acc[0][i][j] = FA == MXC_E4M3 ? mfma_x8(ad[i], bd[j], acc[0][i][j])
                                                      : mfma_nv(ad[i], bd[j], acc[0][i][j]);
            } else if constexpr (FA == MXC_E4M3) {   // MXFP8: each fragment decoded to bf16 once
                uint32_t ad[NB][16];
#pragma unroll
                for (int i = 0; i < NB; i++) e4m3_decode32_lane(o[b].a[i], o[b].sa[i], ad[i]);
#pragma unroll
                for (int t = 0; t < KT; t++) {
                    uint32_t bd[NB][16];
#pragma unroll
                    for (int j = 0; j < NB; j++) e4m3_decode32_lane(o[b].b[t][j], o[b].sb[t][j], bd[j]);
#pragma unroll
                    for (int i = 0; i < NB; i++)
#pragma unroll
                        for (int j = 0; j < NB; j++) acc[t][i][j] = mfma_x8(ad[i], bd[j], acc[t][i][j]);
                }
            } else {
#pragma unroll
                for (int t = 0; t < KT; t++)
#pragma unroll
                    for (int i = 0; i < NB; i++)
#pragma unroll
                        for (int j = 0; j < NB; j++)
                            acc[t][i][j] = mfma_mx<FA, FB>(o[b].a[i], o[b].b[t][j], acc[t][i][j], o[b].sa[i],
                                                           o[b].sb[t][j]);
            }
        }
    }
    if constexpr (NV) {   // the per-tensor scales T_GY T_X
        const float tt = *p.tg * *p.tx;
#pragma unroll
        for (int i = 0; i < NB; i++)
#pragma unroll
            for (int j = 0; j < NB; j++)
#pragma unroll
                for (int e = 0; e < 16; e++) acc[0][i][j][e] *= tt;
    }

    // ---- per tap: sum the four waves' tiles, then write
#pragma unroll
    for (int t = 0; t < KT; t++) {
        if (t > 0) __syncthreads();                   // the previous tap's sums are read
#pragma unroll
        for (int i = 0; i < NB; i++)
#pragma unroll
            for (int j = 0; j < NB; j++)
#pragma unroll
                for (int e = 0; e < 16; e++) {
                    const int row = 32 * i + 8 * (e >> 2) + 4 * hf + (e & 3);
                    red[wave][row * RS + 32 * j + r] = acc[t][i][j][e];
                }
        __syncthreads();
        const int ttap = th * p.kw + tw + t;
#pragma unroll 4
        for (int k = 0; k < RS * RS / WT; k++) {
            const int idx = tid + WT * k;
            const int row = idx / RS, col = idx % RS;
            const float v = (red[0][idx] + red[1][idx]) + (red[2][idx] + red[3][idx]);
            const int co = cop * 64 + row, ci = cip * 64 + col;
            if (p.direct) {
                if (co < p.cout && ci < p.cin)
                    p.dst[(((size_t)co * p.cin + ci) * p.kh + th) * p.kw + tw + t] = v;
            } else if (co < p.gy_cp && ci < p.x_cp) {
                p.dst[((size_t)split * p.gy_cp + co) * p.ntot + (size_t)ttap * p.x_cp + ci] = v;
            }
        }
    }
}

// The tile arguments for one layer split `splits` ways over its pixel pairs
// (dst: G_W when splits == 1, else the partial tiles); returns the workgroup
// count (a multiple of 8), or -1 past the 32-bit grid.
inline long wgrad_lean_fill(const Conv& cv, const void* gc, const uint8_t* gs, const void* xc, const uint8_t* xs,
                            float* dst, int splits, const float* nv_tg, const float* nv_tx, WLArgs& a) {
    a.gc = (const uint8_t*)gc; a.gs = gs; a.xc = (const uint8_t*)xc; a.xs = xs;
    a.dst = dst;
    a.tg = nv_tg; a.tx = nv_tx;
    a.direct = splits == 1;
    a.cout = cv.cout; a.cin = cv.cin; a.kh = cv.kh; a.kw = cv.kw; a.sh = cv.sh; a.sw = cv.sw;
    a.ph = cv.ph; a.pw = cv.pw; a.ho = cv.ho; a.wo = cv.wo; a.h = cv.h; a.w = cv.w;
    a.gy_ncb = cv.gy.ncb; a.x_ncb = cv.x.ncb; a.gy_cp = cv.gy.cp; a.x_cp = cv.x.cp;
    a.ntot = cv.kh * cv.kw * cv.x.cp;
    a.npix = cv.x.ng * cv.ho * cv.wo;
    a.ppr = (cv.wo + 1) / 2;
    a.npairs = cv.x.ng * cv.ho * a.ppr;
    a.cot = (cv.gy.ncb + 1) / 2; a.cit = (cv.x.ncb + 1) / 2;
    a.ntiles = cv.kh * (cv.kw / wgrad_taps(cv, nv_tg != nullptr)) * a.cot * a.cit;
    const int waves = splits * 4;
    a.ppw = (a.npairs + waves - 1) / waves;
    a.nsplit = splits;
    const long grid = ((long)a.ntiles * splits + 7) / 8 * 8;
    return grid > 0x7FFFFFFFL ? -1 : grid;
}

}  // namespace
