// conv_gemm.hip -- a3/a4/a5: the three convolution GEMMs on MX operands
// (Sec. II-C and Sec. IV-B: Y_f = W_f X', G_X' = W_f^T G_Yf folded back by
// col2im, G_Wf = G_Yf X'^T), on gfx950 block-scaled MFMA
// (v_mfma_scale_f32_32x32x64_f8f6f4): every 32-element K block of an
// operand row carries its own E8M0 scale, which is exactly Eq. (7).
//
// All three kernels share one scheme.  A workgroup (4 waves) owns a BM x BN
// output tile; a K step is two MX blocks (K = 64).  Per step the operands'
// blocks are copied into LDS in their stored layout -- a block is a
// contiguous [32 rows][Bn samples] slab of codes -- double-buffered so the
// next step's global loads overlap this step's MFMAs.  Whether an operand is
// read along its rows or across them, the transposition happens in the LDS
// read (ds_read_b64_tr_b8 / _b4), so no data is ever rearranged:
//   fwd   A = W   (rows co, K ci): weight block [ci][co], read transposed
//         B = X'  (cols (pixel, n), K ci): X block [ci][n], read transposed;
//             the im2col is implicit, each tap's block is fetched from the
//             source pixel ho*sh+kh-ph, wo*sw+kw-pw (zero outside).
//   dgrad A = W^T (rows ci, K co): weight block [ci][co], read along rows
//         B = G_Y (cols (pixel, n), K co), read transposed; the output is
//             split into sh x sw stride phases so every tap a workgroup
//             visits reaches all its pixels (the col2im becomes a gather).
//   wgrad A = G_Y (rows co, K n) and B = X at the tap-shifted pixel
//             (cols (tap, ci), K n), both read along rows; one K block is
//             one pixel's batch block (padded with zeros when Bn < 32);
//             split over K, partials reduced in fp32 by a second kernel.
#include "mx_internal.h"

namespace mxc {
namespace {

constexpr int BM = 64;    // output rows per workgroup (2 MFMA row blocks)
constexpr int BN = 128;   // output columns per workgroup (4 MFMA column blocks)
constexpr int NT = 256;   // 4 waves: wave w owns rows 32*(w&1), columns 64*(w>>1)
constexpr int SP = 4;     // streamed wgrad: pixel blocks per stage

template <int UNIT> struct Vec;
template <> struct Vec<16> { typedef uint4 T; };
template <> struct Vec<8> { typedef uint2 T; };
template <> struct Vec<4> { typedef uint32_t T; };
template <> struct Vec<2> { typedef unsigned short T; };
template <> struct Vec<1> { typedef uint8_t T; };

template <int UNIT>
__device__ __forceinline__ typename Vec<UNIT>::T vzero() {
    typename Vec<UNIT>::T z;
    __builtin_memset(&z, 0, sizeof(z));
    return z;
}

// MFMA fragment from a K-major LDS tile ([block][k][col] bytes, row stride
// `stride`): lane (col c, half h) receives the elements the block-scaled MFMA
// expects (see mfma_mx), gathered by transposing reads.
template <int FMT>
__device__ __forceinline__ v8i frag_tr(const uint8_t* base, int stride, int colbase) {
    const int l = threadIdx.x & 63;
    const int i = l & 15, gi = l >> 4, cg = gi & 1, h = gi >> 1;
    v8i r;
    if (FMT == MXC_E4M3) {
#pragma unroll
        for (int blk = 0; blk < 2; blk++)
#pragma unroll
            for (int hf = 0; hf < 2; hf++) {
                const int row = blk * 32 + 16 * h + 8 * hf + (i >> 1);
                const int col = colbase + 16 * cg + 8 * (i & 1);
                const v2i v = lds_tr8(base + row * stride + col);
                r[4 * blk + 2 * hf] = v[0];
                r[4 * blk + 2 * hf + 1] = v[1];
            }
    } else {
#pragma unroll
        for (int hf = 0; hf < 2; hf++) {
            const int row = h * 32 + 16 * hf + i;
            const v2i v = lds_tr4(base + row * stride + ((colbase + 16 * cg) >> 1));
            r[2 * hf] = v[0];
            r[2 * hf + 1] = v[1];
        }
        r[4] = r[5] = r[6] = r[7] = 0;
    }
    return r;
}

// MFMA fragment from a row-major LDS tile ([row][block][32 elements], row
// stride `stride`).
template <int FMT>
__device__ __forceinline__ v8i frag_rows(const uint8_t* base, int stride, int rowbase) {
    const int l = threadIdx.x & 63;
    const int r = l & 31, h = l >> 5;
    const uint8_t* p = base + (rowbase + r) * stride;
    v8i out;
    if (FMT == MXC_E4M3) {
        const v4i a = *(const v4i*)(p + 16 * h);
        const v4i b = *(const v4i*)(p + 32 + 16 * h);
        out[0] = a[0]; out[1] = a[1]; out[2] = a[2]; out[3] = a[3];
        out[4] = b[0]; out[5] = b[1]; out[6] = b[2]; out[7] = b[3];
    } else {
        const v4i a = *(const v4i*)(p + 16 * h);
        out[0] = a[0]; out[1] = a[1]; out[2] = a[2]; out[3] = a[3];
        out[4] = out[5] = out[6] = out[7] = 0;
    }
    return out;
}

// ============================================================ fwd / dgrad
struct ConvArgs {
    Conv cv;
    const uint8_t* wc;  // weight codes / scales
    const uint8_t* ws;
    const uint8_t* bc;  // activation operand: X (fwd) or G_Y (dgrad)
    const uint8_t* bs;
    float* out;
    int layout;
    int M;              // real output channels (cout for fwd, cin for dgrad)
    int mtiles, ctiles;
    int hs, wsrc, cps, ncbs;  // activation operand: spatial size, padded channels, blocks
    int kcb;                  // channel blocks along K
    int hout, wout;           // output spatial size
};

template <int FMT, bool DG, int UNIT>
__global__ __launch_bounds__(NT) void conv_kernel(ConvArgs p) {
    constexpr int EB = FMT == MXC_E4M3 ? 8 : 4;     // element bits
    constexpr int ROWB = 32 * EB / 8;               // bytes of one 32-element block row
    constexpr int BSTR = BN * EB / 8 + 16;          // B: K-major row stride
    constexpr int B_BYTES = 64 * BSTR;
    constexpr int ASTR = DG ? 2 * ROWB + 16 : BM * EB / 8 + 16;
    constexpr int A_BYTES = DG ? BM * ASTR : 64 * ASTR;
    constexpr int NU_B = BN * EB / (32 * UNIT);     // B copy units per thread per step
    constexpr int AUNITS = 128 * ROWB / 16;          // A copy units (16 B) per step
    __shared__ __attribute__((aligned(16))) uint8_t lds_a[2][A_BYTES];
    __shared__ __attribute__((aligned(16))) uint8_t lds_b[2][B_BYTES];
    __shared__ int sc_a[2][2][2];                    // [buf][block][row block]
    __shared__ uint8_t sc_b[2][2][BN];               // [buf][block][pixel slot]
    __shared__ int slot_g[BN], slot_y[BN], slot_x[BN];

    const Conv& cv = p.cv;
    const int tid = threadIdx.x;
    const int bn = cv.x.bn;
    const int nps = BN / bn;                         // pixel slots per tile
    const int rb = bn * EB / 8;                      // bytes of one row of an activation block
    const int parts = rb / UNIT;

    // ---- which tile: XCD-aware (tiles sharing columns land on one XCD)
    const int ntile = p.mtiles * p.ctiles;
    const int per_xcd = (gridDim.x + 7) / 8;
    const int lin = (blockIdx.x % 8) * per_xcd + blockIdx.x / 8;
    if (lin >= ntile) return;
    const int mt = lin % p.mtiles, ct = lin / p.mtiles;

    // ---- phase (dgrad) and the taps that reach it
    int ry = 0, rx = 0, kh0 = 0, kw0 = 0, nvh = cv.kh, nvw = cv.kw, gh = cv.ho, gw = cv.wo;
    if (DG) {
        const int ph_id = blockIdx.y;
        ry = ph_id / cv.sw; rx = ph_id % cv.sw;
        kh0 = (ry + cv.ph) % cv.sh; kw0 = (rx + cv.pw) % cv.sw;
        nvh = kh0 < cv.kh ? (cv.kh - kh0 + cv.sh - 1) / cv.sh : 0;
        nvw = kw0 < cv.kw ? (cv.kw - kw0 + cv.sw - 1) / cv.sw : 0;
        gh = ry < cv.h ? (cv.h - ry + cv.sh - 1) / cv.sh : 0;
        gw = rx < cv.w ? (cv.w - rx + cv.sw - 1) / cv.sw : 0;
    }
    const int pph = gh * gw;                          // output pixels in this phase
    const int ng = cv.x.ng;
    if ((long)ct * BN >= (long)ng * pph * bn) return;
    const int nkb = nvh * nvw * p.kcb;                // K blocks
    const int nsteps = (nkb + 1) / 2;

    // ---- pixel slots of this column tile
    for (int s = tid; s < nps; s += NT) {
        const long q = (long)ct * nps + s;            // (group, pixel) index
        const int g = (int)(q / (pph > 0 ? pph : 1)), pp = pph > 0 ? (int)(q % pph) : 0;
        slot_g[s] = (pph > 0 && g < ng) ? g : -1;
        slot_y[s] = pph > 0 ? pp / gw : 0;
        slot_x[s] = pph > 0 ? pp % gw : 0;
    }
    __syncthreads();

    // tap index -> (kh, kw) and the source-pixel offset of the tap
    const int tsh = DG ? cv.sh : 1, tsw = DG ? cv.sw : 1;
    auto tap_of = [&](int ti, int& kh, int& kw) {
        kh = kh0 + (ti / nvw) * tsh;
        kw = kw0 + (ti % nvw) * tsw;
    };

    typename Vec<UNIT>::T rb_regs[NU_B];
    uint4 ra;
    uint8_t rsb = 0;
    int rsa = 0;

    auto load_step = [&](int s) {
        // B: units ordered (block, slot, k, part) so lanes walk contiguous bytes
#pragma unroll
        for (int i = 0; i < NU_B; i++) {
            const int u = tid + NT * i;
            const int part = u % parts;
            const int r1 = u / parts;
            const int k = r1 & 31;
            const int r2 = r1 >> 5;
            const int ps = r2 % nps;
            const int blk = r2 / nps;
            const int b = 2 * s + blk;
            // every load is issued (out-of-range ones read offset 0 and are
            // zeroed), so all of a step's loads are in flight together
            const int g = slot_g[ps];
            const int bb = min(b, nkb - 1);
            const int ti = bb / p.kcb, kc = bb % p.kcb;
            int kh, kw;
            tap_of(ti, kh, kw);
            int sy, sx;
            if (DG) {
                sy = slot_y[ps] + (ry + cv.ph - kh) / cv.sh;
                sx = slot_x[ps] + (rx + cv.pw - kw) / cv.sw;
            } else {
                sy = slot_y[ps] * cv.sh + kh - cv.ph;
                sx = slot_x[ps] * cv.sw + kw - cv.pw;
            }
            const bool ok = b < nkb && g >= 0 && sy >= 0 && sy < p.hs && sx >= 0 && sx < p.wsrc;
            const size_t off = ((((size_t)max(g, 0) * p.hs + sy) * p.wsrc + sx) * p.cps + 32 * kc) *
                                   (size_t)bn * EB / 8 + (size_t)k * rb + part * UNIT;
            const typename Vec<UNIT>::T v = *(const typename Vec<UNIT>::T*)(p.bc + (ok ? off : 0));
            rb_regs[i] = ok ? v : vzero<UNIT>();
        }
        // B scales: one per (block, slot)
        if (tid < 2 * nps) {
            const int blk = tid / nps, ps = tid % nps, b = 2 * s + blk;
            const int g = slot_g[ps];
            uint8_t sc = 0;
            if (b < nkb && g >= 0) {
                const int ti = b / p.kcb, kc = b % p.kcb;
                int kh, kw;
                tap_of(ti, kh, kw);
                int sy, sx;
                if (DG) {
                    sy = slot_y[ps] + (ry + cv.ph - kh) / cv.sh;
                    sx = slot_x[ps] + (rx + cv.pw - kw) / cv.sw;
                } else {
                    sy = slot_y[ps] * cv.sh + kh - cv.ph;
                    sx = slot_x[ps] * cv.sw + kw - cv.pw;
                }
                if (sy >= 0 && sy < p.hs && sx >= 0 && sx < p.wsrc)
                    sc = p.bs[(((size_t)g * p.hs + sy) * p.wsrc + sx) * p.ncbs + kc];
            }
            rsb = sc;
        }
        // A: weight blocks; units ordered (block, row block, k, part)
        ra = make_uint4(0, 0, 0, 0);
        if (tid < AUNITS) {
            const int u = tid;
            const int part = u % (ROWB / 16);
            const int r1 = u / (ROWB / 16);
            const int k = r1 & 31;
            const int mb = (r1 >> 5) & 1;
            const int blk = r1 >> 6;
            const int b = 2 * s + blk;
            const int bb = min(b, nkb - 1);
            const int ti = bb / p.kcb, kc = bb % p.kcb;
            int kh, kw;
            tap_of(ti, kh, kw);
            const int rowblk = 2 * mt + mb;           // block of output rows
            const int cob = DG ? kc : rowblk, cib = DG ? rowblk : kc;
            const bool ok = b < nkb && cob < cv.wt.np / 32 && cib < cv.wt.ncb;
            const size_t off = ((((size_t)cob * cv.kh + kh) * cv.kw + kw) * cv.wt.cp + 32 * cib) *
                                   (size_t)32 * EB / 8 + (size_t)k * ROWB + part * 16;
            const uint4 v = *(const uint4*)(p.wc + (ok ? off : 0));
            ra = ok ? v : make_uint4(0, 0, 0, 0);
        }
        if (tid < 4) {
            const int blk = tid >> 1, mb = tid & 1, b = 2 * s + blk;
            int sc = 0;
            if (b < nkb) {
                const int ti = b / p.kcb, kc = b % p.kcb;
                int kh, kw;
                tap_of(ti, kh, kw);
                const int rowblk = 2 * mt + mb;
                const int cob = DG ? kc : rowblk, cib = DG ? rowblk : kc;
                if (cob < cv.wt.np / 32 && cib < cv.wt.ncb)
                    sc = p.ws[(((size_t)cob * cv.kh + kh) * cv.kw + kw) * cv.wt.ncb + cib];
            }
            rsa = sc;
        }
    };

    auto store_step = [&](int buf) {
#pragma unroll
        for (int i = 0; i < NU_B; i++) {
            const int u = tid + NT * i;
            const int part = u % parts;
            const int r1 = u / parts;
            const int k = r1 & 31;
            const int r2 = r1 >> 5;
            const int ps = r2 % nps;
            const int blk = r2 / nps;
            *(typename Vec<UNIT>::T*)&lds_b[buf][(blk * 32 + k) * BSTR + ps * rb + part * UNIT] = rb_regs[i];
        }
        if (tid < 2 * nps) sc_b[buf][tid / nps][tid % nps] = rsb;
        if (tid < AUNITS) {
            const int u = tid;
            const int part = u % (ROWB / 16);
            const int r1 = u / (ROWB / 16);
            const int k = r1 & 31;
            const int mb = (r1 >> 5) & 1;
            const int blk = r1 >> 6;
            const int off = DG ? (mb * 32 + k) * ASTR + blk * ROWB + part * 16
                               : (blk * 32 + k) * ASTR + mb * ROWB + part * 16;
            *(uint4*)&lds_a[buf][off] = ra;
        }
        if (tid < 4) sc_a[buf][tid >> 1][tid & 1] = rsa;
    };

    const int wave = tid >> 6, lane = tid & 63;
    const int wm = wave & 1, wn = wave >> 1;
    v16f acc[2];
    for (int c = 0; c < 2; c++)
        for (int e = 0; e < 16; e++) acc[c][e] = 0.0f;

    if (nsteps > 0) {
        load_step(0);
        store_step(0);
    }
    __syncthreads();
    for (int s = 0; s < nsteps; s++) {
        const int buf = s & 1;
        if (s + 1 < nsteps) load_step(s + 1);
        const v8i af = DG ? frag_rows<FMT>(lds_a[buf], ASTR, 32 * wm)
                          : frag_tr<FMT>(lds_a[buf], ASTR, 32 * wm);
        const int h = lane >> 5;
        const int sa = sc_a[buf][h][wm];
        AFrag<FMT> ad;
        ad.set(af, sa);
#pragma unroll
        for (int c = 0; c < 2; c++) {
            const int colbase = 64 * wn + 32 * c;
            const v8i bf = frag_tr<FMT>(lds_b[buf], BSTR, colbase);
            const int sb = sc_b[buf][h][(colbase + (lane & 31)) / bn];
            acc[c] = mfma_mx_a<FMT>(ad, bf, acc[c], sb);
        }
        if (s + 1 < nsteps) store_step(buf ^ 1);
        __syncthreads();
    }

    // ---- epilogue: D(row, col) of lane l, value e: col = l%32,
    //      row = 8*(e/4) + 4*(l/32) + e%4
#pragma unroll
    for (int c = 0; c < 2; c++) {
        const int col = 64 * wn + 32 * c + (lane & 31);
        const int ps = col / bn, j = col % bn;
        const int g = slot_g[ps];
        if (g < 0) continue;
        const int oy = DG ? ry + cv.sh * slot_y[ps] : slot_y[ps];
        const int ox = DG ? rx + cv.sw * slot_x[ps] : slot_x[ps];
        const int n = g * bn + j;
#pragma unroll
        for (int e = 0; e < 16; e++) {
            const int m = BM * mt + 32 * wm + 8 * (e >> 2) + 4 * (lane >> 5) + (e & 3);
            if (m >= p.M) continue;
            size_t o;
            if (p.layout != MXC_NCHW)
                o = ((((size_t)g * p.hout + oy) * p.wout + ox) * p.M + m) * bn + j;
            else
                o = (((size_t)n * p.M + m) * p.hout + oy) * p.wout + ox;
            if (p.layout == MXC_CBF_BF16) ((uint16_t*)p.out)[o] = (uint16_t)bf16_bits(acc[c][e]);
            else                          p.out[o] = acc[c][e];
        }
    }
}

template <bool DG, int FMT>
int launch_conv_u(const ConvArgs& a, dim3 grid, hipStream_t s) {
    const int rb = a.cv.x.bn * (FMT == MXC_E4M3 ? 8 : 4) / 8;
    const int unit = rb >= 16 ? 16 : rb;
    switch (unit) {
        case 16: hipLaunchKernelGGL((conv_kernel<FMT, DG, 16>), grid, dim3(NT), 0, s, a); break;
        case 8:  hipLaunchKernelGGL((conv_kernel<FMT, DG, 8>), grid, dim3(NT), 0, s, a); break;
        case 4:  hipLaunchKernelGGL((conv_kernel<FMT, DG, 4>), grid, dim3(NT), 0, s, a); break;
        case 2:  hipLaunchKernelGGL((conv_kernel<FMT, DG, 2>), grid, dim3(NT), 0, s, a); break;
        default: hipLaunchKernelGGL((conv_kernel<FMT, DG, 1>), grid, dim3(NT), 0, s, a); break;
    }
    return hipGetLastError() == hipSuccess ? MXC_OK : MXC_ERR_HIP;
}

int launch_conv(const Conv& cv, bool dg, const void* wc, const uint8_t* ws, const void* bc,
                const uint8_t* bs, float* out, int layout, hipStream_t s) {
    ConvArgs a;
    a.cv = cv;
    a.wc = (const uint8_t*)wc; a.ws = ws; a.bc = (const uint8_t*)bc; a.bs = bs;
    a.out = out; a.layout = layout;
    const Geom& src = dg ? cv.gy : cv.x;
    a.hs = src.h; a.wsrc = src.w; a.cps = src.cp; a.ncbs = src.ncb;
    a.kcb = dg ? cv.wt.np / 32 : cv.wt.ncb;
    a.M = dg ? cv.cin : cv.cout;
    a.hout = dg ? cv.h : cv.ho;
    a.wout = dg ? cv.w : cv.wo;
    a.mtiles = (a.M + BM - 1) / BM;
    // largest phase grid sets the number of column tiles
    long maxp = 0;
    const int nph = dg ? cv.sh * cv.sw : 1;
    for (int ph = 0; ph < nph; ph++) {
        const int ry = dg ? ph / cv.sw : 0, rx = dg ? ph % cv.sw : 0;
        const long gh = dg ? (ry < cv.h ? (cv.h - ry + cv.sh - 1) / cv.sh : 0) : cv.ho;
        const long gw = dg ? (rx < cv.w ? (cv.w - rx + cv.sw - 1) / cv.sw : 0) : cv.wo;
        if (gh * gw > maxp) maxp = gh * gw;
    }
    const long ctiles = ((long)cv.x.ng * maxp * cv.x.bn + BN - 1) / BN;
    const long ntile = ctiles * a.mtiles;
    if (ntile > 0x7FFFFFF0L) return MXC_ERR_SHAPE;
    a.ctiles = (int)ctiles;
    const unsigned gx = (unsigned)((ntile + 7) / 8 * 8);
    const dim3 grid(gx, nph);
    if (cv.fmt == MXC_E4M3)
        return dg ? launch_conv_u<true, MXC_E4M3>(a, grid, s) : launch_conv_u<false, MXC_E4M3>(a, grid, s);
    return dg ? launch_conv_u<true, MXC_E2M1>(a, grid, s) : launch_conv_u<false, MXC_E2M1>(a, grid, s);
}

// ============================================================ wgrad
struct WgradArgs {
    Conv cv;
    const uint8_t* gc;  // G_Y codes / scales
    const uint8_t* gs;
    const uint8_t* xc;  // X codes / scales
    const uint8_t* xs;
    float* part;        // [splits][Cout_p][ntot] partial sums
    int ntot;           // columns: Kh*Kw*Cin_p, column = tap*Cin_p + ci
    int mtiles, ctiles, splits, kbps;   // K blocks per split (even)
};

template <int FMT, int UNIT>
__global__ __launch_bounds__(NT) void wgrad_kernel(WgradArgs p) {
    constexpr int EB = FMT == MXC_E4M3 ? 8 : 4;
    constexpr int ROWB = 32 * EB / 8;
    constexpr int STR = 2 * ROWB + 16;
    __shared__ __attribute__((aligned(16))) uint8_t lds_a[2][BM * STR];
    __shared__ __attribute__((aligned(16))) uint8_t lds_b[2][BN * STR];
    __shared__ int sc_a[2][2][2];
    __shared__ int sc_b[2][2][4];

    const Conv& cv = p.cv;
    const int tid = threadIdx.x;
    const int bn = cv.x.bn;
    const int rb = bn * EB / 8;                  // real bytes of a block row
    const int parts = rb / UNIT;
    const int npix = cv.ho * cv.wo;
    const int nkb = cv.x.ng * npix;              // K blocks: (group, output pixel)

    const int ntile = p.mtiles * p.ctiles * p.splits;
    const int per_xcd = (gridDim.x + 7) / 8;
    const int lin = (blockIdx.x % 8) * per_xcd + blockIdx.x / 8;
    if (lin >= ntile) return;
    const int mt = lin % p.mtiles;
    const int r0 = lin / p.mtiles;
    const int ct = r0 % p.ctiles, sp = r0 / p.ctiles;
    const int kb0 = sp * p.kbps;
    const int kb1 = min(nkb, kb0 + p.kbps);
    const int nsteps = kb1 > kb0 ? (kb1 - kb0 + 1) / 2 : 0;

    // rows shorter than a block are zero-padded once; loads never touch the pad
    if (rb < ROWB) {
        for (int i = tid; i < 2 * BM * STR / 4; i += NT) ((uint32_t*)lds_a)[i] = 0;
        for (int i = tid; i < 2 * BN * STR / 4; i += NT) ((uint32_t*)lds_b)[i] = 0;
        __syncthreads();
    }

    // column block cbk (0..3) of this tile -> (tap, ci block)
    const int cinb = cv.x.ncb;
    // a block row is either split into 16-byte units (at most 2: 32 FP8 codes)
    // or moved as one smaller unit, so A has <= 2*BM*2 = NT units, B <= 2*NT
    constexpr int NUA = 1;
    constexpr int NUB = 2;
    typename Vec<UNIT>::T ra[NUA], rbv[NUB];
    int rs = 0;

    // A units: (block, row, part); B units: (block, column, part); only the
    // real bytes of each row are loaded.
    auto load_step = [&](int s) {
#pragma unroll
        for (int i = 0; i < NUA; i++) {
            const int u = tid + NT * i;
            const int part = u % parts, r1 = u / parts;
            const int row = r1 % BM, blk = r1 / BM;
            const int b = kb0 + 2 * s + blk;
            const int co = BM * mt + row;
            const bool ok = u < 2 * BM * parts && b < kb1 && co < cv.gy.cp;
            const int bb = min(b, nkb - 1);
            const int g = bb / npix, pix = bb % npix;
            const size_t off = (((size_t)g * npix + pix) * cv.gy.cp + co) * (size_t)rb + part * UNIT;
            const typename Vec<UNIT>::T v = *(const typename Vec<UNIT>::T*)(p.gc + (ok ? off : 0));
            ra[i] = ok ? v : vzero<UNIT>();
        }
#pragma unroll
        for (int i = 0; i < NUB; i++) {
            const int u = tid + NT * i;
            const int part = u % parts, r1 = u / parts;
            const int col = r1 % BN, blk = r1 / BN;
            const int b = kb0 + 2 * s + blk;
            const int gcol = BN * ct + col;
            const int tap = gcol / cv.x.cp, ci = gcol % cv.x.cp;
            const int bb = min(b, nkb - 1);
            const int g = bb / npix, pix = bb % npix;
            const int oh = pix / cv.wo, ow = pix % cv.wo;
            const int ih = oh * cv.sh + tap / cv.kw - cv.ph, iw = ow * cv.sw + tap % cv.kw - cv.pw;
            const bool ok = u < 2 * BN * parts && b < kb1 && tap < cv.kh * cv.kw && ih >= 0 && ih < cv.h &&
                            iw >= 0 && iw < cv.w;
            const size_t off = ((((size_t)g * cv.h + ih) * cv.w + iw) * cv.x.cp + ci) * (size_t)rb + part * UNIT;
            const typename Vec<UNIT>::T v = *(const typename Vec<UNIT>::T*)(p.xc + (ok ? off : 0));
            rbv[i] = ok ? v : vzero<UNIT>();
        }
        // scales: 4 for A (block x row block), 8 for B (block x column block)
        rs = 0;
        if (tid < 4) {
            const int blk = tid >> 1, mb = tid & 1, b = kb0 + 2 * s + blk;
            const int cob = 2 * mt + mb;
            if (b < kb1 && cob < cv.gy.ncb) rs = p.gs[(size_t)b * cv.gy.ncb + cob];
        } else if (tid < 12) {
            const int t = tid - 4, blk = t >> 2, cbk = t & 3, b = kb0 + 2 * s + blk;
            const int gcb = 4 * ct + cbk;                 // global column block
            const int tap = gcb / cinb, cib = gcb % cinb;
            if (b < kb1 && tap < cv.kh * cv.kw) {
                const int g = b / npix, pix = b % npix;
                const int oh = pix / cv.wo, ow = pix % cv.wo;
                const int ih = oh * cv.sh + tap / cv.kw - cv.ph, iw = ow * cv.sw + tap % cv.kw - cv.pw;
                if (ih >= 0 && ih < cv.h && iw >= 0 && iw < cv.w)
                    rs = p.xs[(((size_t)g * cv.h + ih) * cv.w + iw) * cinb + cib];
            }
        }
    };

    auto store_step = [&](int buf) {
#pragma unroll
        for (int i = 0; i < NUA; i++) {
            const int u = tid + NT * i;
            if (u < 2 * BM * parts) {
                const int part = u % parts, r1 = u / parts;
                const int row = r1 % BM, blk = r1 / BM;
                *(typename Vec<UNIT>::T*)&lds_a[buf][row * STR + blk * ROWB + part * UNIT] = ra[i];
            }
        }
#pragma unroll
        for (int i = 0; i < NUB; i++) {
            const int u = tid + NT * i;
            if (u < 2 * BN * parts) {
                const int part = u % parts, r1 = u / parts;
                const int col = r1 % BN, blk = r1 / BN;
                *(typename Vec<UNIT>::T*)&lds_b[buf][col * STR + blk * ROWB + part * UNIT] = rbv[i];
            }
        }
        if (tid < 4) sc_a[buf][tid >> 1][tid & 1] = rs;
        else if (tid < 12) sc_b[buf][(tid - 4) >> 2][(tid - 4) & 3] = rs;
    };

    const int wave = tid >> 6, lane = tid & 63;
    const int wm = wave & 1, wn = wave >> 1;
    v16f acc[2];
    for (int c = 0; c < 2; c++)
        for (int e = 0; e < 16; e++) acc[c][e] = 0.0f;

    if (nsteps > 0) {
        load_step(0);
        store_step(0);
    }
    __syncthreads();
    for (int s = 0; s < nsteps; s++) {
        const int buf = s & 1;
        if (s + 1 < nsteps) load_step(s + 1);
        const int h = lane >> 5;
        const v8i af = frag_rows<FMT>(lds_a[buf], STR, 32 * wm);
        const int sa = sc_a[buf][h][wm];
        AFrag<FMT> ad;
        ad.set(af, sa);
#pragma unroll
        for (int c = 0; c < 2; c++) {
            const v8i bf = frag_rows<FMT>(lds_b[buf], STR, 64 * wn + 32 * c);
            const int sb = sc_b[buf][h][2 * wn + c];
            acc[c] = mfma_mx_a<FMT>(ad, bf, acc[c], sb);
        }
        if (s + 1 < nsteps) store_step(buf ^ 1);
        __syncthreads();
    }

    // partial tile -> workspace [split][Cout_p][ntot]
#pragma unroll
    for (int c = 0; c < 2; c++) {
        const int col = BN * ct + 64 * wn + 32 * c + (lane & 31);
        if (col >= p.ntot) continue;
#pragma unroll
        for (int e = 0; e < 16; e++) {
            const int m = BM * mt + 32 * wm + 8 * (e >> 2) + 4 * (lane >> 5) + (e & 3);
            if (m >= cv.gy.cp) continue;
            p.part[((size_t)sp * cv.gy.cp + m) * p.ntot + col] = acc[c][e];
        }
    }
}

// G_W[co][ci][kh][kw] = sum over splits of the partial (co, tap*Cin_p + ci).
// Below 64 splits a thread takes a column and keeps four sums, sum q adding
// splits q, q + 4, q + 8, ... in increasing order, and returns (sum0 + sum1)
// + (sum2 + sum3).  From 64 splits on (the first layers: few columns, many
// splits, where a thread per column left most of the GPU idle behind long
// load chains) sixteen threads share a column: thread q adds splits q, q +
// 16, ... in increasing order and the column's result is the pairwise tree
// ((s0 + s1) + (s2 + s3)) + ... of the sixteen.  Either way a fixed order:
// the result does not depend on timing, and the same bits whether one layer
// or several are reduced by the launch.  A workgroup takes 256 / nr
// consecutive columns (nr = 1 or 16); neighbouring threads read
// neighbouring columns of one split.
struct RedGeom {
    int cout, cin, kh, kw, gy_cp, x_cp, ntot, splits, nr;
};

inline int reduce_nr(int splits) { return splits >= 64 ? 16 : 1; }

__device__ __forceinline__ void reduce_store(float* __restrict__ gw, const RedGeom& r, long i, float sum) {
    const int co = (int)(i / r.ntot), col = (int)(i % r.ntot);
    const int tap = col / r.x_cp, ci = col % r.x_cp;
    if (ci < r.cin)
        gw[(((size_t)co * r.cin + ci) * r.kh + tap / r.kw) * r.kw + tap % r.kw] = sum;
}

__device__ __forceinline__ void reduce_cols(const float* __restrict__ part, float* __restrict__ gw,
                                            const RedGeom& r, long wg) {
    const size_t stride = (size_t)r.gy_cp * r.ntot;
    if (r.nr == 1) {
        const long i = wg * 256 + threadIdx.x;
        if (i >= (long)r.cout * r.ntot) return;
        const float* q = part + (size_t)(i / r.ntot) * r.ntot + (i % r.ntot);
        float a[4] = {0.0f, 0.0f, 0.0f, 0.0f};
        int k = 0;
        for (; k + 8 <= r.splits; k += 8) {                 // eight loads in flight
            float v[8];
#pragma unroll
            for (int j = 0; j < 8; j++) v[j] = __ldg(q + (size_t)(k + j) * stride);
#pragma unroll
            for (int j = 0; j < 8; j++) a[j & 3] += v[j];
        }
        for (; k < r.splits; k++) a[k & 3] += __ldg(q + (size_t)k * stride);
        reduce_store(gw, r, i, (a[0] + a[1]) + (a[2] + a[3]));
        return;
    }
    __shared__ float red[256];
    constexpr int NR = 16, PER = 256 / NR;
    const int t = threadIdx.x, qi = t / PER, cl = t % PER;
    const long i = wg * PER + cl;
    const bool live = i < (long)r.cout * r.ntot;
    float a = 0.0f;
    if (live) {
        const float* q = part + (size_t)(i / r.ntot) * r.ntot + (i % r.ntot);
        int k = qi;
        for (; k + 7 * NR < r.splits; k += 8 * NR) {        // eight loads in flight
            float v[8];
#pragma unroll
            for (int j = 0; j < 8; j++) v[j] = __ldg(q + (size_t)(k + j * NR) * stride);
#pragma unroll
            for (int j = 0; j < 8; j++) a += v[j];
        }
        for (; k < r.splits; k += NR) a += __ldg(q + (size_t)k * stride);
    }
    red[t] = a;
    __syncthreads();
    if (qi != 0 || !live) return;
    float s[NR];
#pragma unroll
    for (int j = 0; j < NR; j++) s[j] = red[j * PER + cl];
#pragma unroll
    for (int w = 1; w < NR; w *= 2)                         // pairwise tree
#pragma unroll
        for (int j = 0; j + w < NR; j += 2 * w) s[j] = s[j] + s[j + w];
    reduce_store(gw, r, i, s[0]);
}

// workgroups of one reduction
long reduce_wgs(const Conv& cv, int splits) {
    const long per = 256 / reduce_nr(splits);
    return ((long)cv.cout * cv.kh * cv.kw * cv.x.cp + per - 1) / per;
}

RedGeom red_geom(const Conv& cv, int splits) {
    RedGeom r;
    r.cout = cv.cout; r.cin = cv.cin; r.kh = cv.kh; r.kw = cv.kw;
    r.gy_cp = cv.gy.cp; r.x_cp = cv.x.cp; r.ntot = cv.kh * cv.kw * cv.x.cp; r.splits = splits;
    r.nr = reduce_nr(splits);
    return r;
}

__global__ __launch_bounds__(256) void wgrad_reduce(const float* __restrict__ part, float* __restrict__ gw,
                                                    RedGeom r) {
    reduce_cols(part, gw, r, blockIdx.x);
}

// Several layers' reductions in one launch: the workgroups of job i take
// [wg0_i, wg0_i + reduce_wgs(job i)); the job is picked with scalar
// selects, as in the batched quantizer.
struct RJob {
    const float* part;
    float* gw;
    RedGeom r;
    int wg0;
};
struct RMulti {
    RJob j[MXC_WREDUCE_MAX];
    int count, nwg;
};

__global__ __launch_bounds__(256) void wgrad_reduce_multi(RMulti m) {
    const int wg = (int)blockIdx.x;
    if (wg >= m.nwg) return;                                      // the whole workgroup
    RJob q = m.j[0];
#pragma unroll
    for (int t = 1; t < MXC_WREDUCE_MAX; t++)
        if (t < m.count && wg >= m.j[t].wg0) q = m.j[t];
    reduce_cols(q.part, q.gw, q.r, wg - q.wg0);
}

int launch_reduce(const Conv& cv, const float* part, float* gw, int splits, hipStream_t s) {
    hipLaunchKernelGGL(wgrad_reduce, dim3((unsigned)reduce_wgs(cv, splits)), dim3(256), 0, s, part, gw,
                       red_geom(cv, splits));
    return hipGetLastError() == hipSuccess ? MXC_OK : MXC_ERR_HIP;
}

struct WgradPlan {
    int mtiles, ctiles, splits, kbps, ntot;
};

bool wstream_ok(const Conv& cv);

WgradPlan wgrad_plan(const Conv& cv) {
    WgradPlan pl;
    pl.ntot = cv.kh * cv.kw * cv.x.cp;
    pl.mtiles = (cv.gy.cp + BM - 1) / BM;
    pl.ctiles = (pl.ntot + BN - 1) / BN;
    const long nkb = (long)cv.x.ng * cv.ho * cv.wo;
    const long tiles = (long)pl.mtiles * pl.ctiles;
    // enough workgroups for the 256 CUs, but long enough K ranges that the
    // partial sums stay small next to the operands
    const bool streamed = wstream_ok(cv);
    const long target = streamed ? 512 : 1024;
    const long min_kb = streamed ? 32 : 16;
    const long gran = streamed ? SP : 2;
    long splits = (target + tiles - 1) / tiles;
    const long max_splits = (nkb + min_kb - 1) / min_kb;
    if (splits > max_splits) splits = max_splits;
    if (splits < 1) splits = 1;
    long kbps = (nkb + splits - 1) / splits;
    kbps = (kbps + gran - 1) / gran * gran;
    splits = (nkb + kbps - 1) / kbps;
    pl.splits = (int)splits;
    pl.kbps = (int)kbps;
    return pl;
}

template <int FMT>
int launch_wgrad_f(const WgradArgs& a, dim3 grid, hipStream_t s) {
    const int rb = a.cv.x.bn * (FMT == MXC_E4M3 ? 8 : 4) / 8;
    const int unit = rb >= 16 ? 16 : rb;
    switch (unit) {
        case 16: hipLaunchKernelGGL((wgrad_kernel<FMT, 16>), grid, dim3(NT), 0, s, a); break;
        case 8:  hipLaunchKernelGGL((wgrad_kernel<FMT, 8>), grid, dim3(NT), 0, s, a); break;
        case 4:  hipLaunchKernelGGL((wgrad_kernel<FMT, 4>), grid, dim3(NT), 0, s, a); break;
        case 2:  hipLaunchKernelGGL((wgrad_kernel<FMT, 2>), grid, dim3(NT), 0, s, a); break;
        default: hipLaunchKernelGGL((wgrad_kernel<FMT, 1>), grid, dim3(NT), 0, s, a); break;
    }
    return hipGetLastError() == hipSuccess ? MXC_OK : MXC_ERR_HIP;
}


// ============================================================ streamed kernels
// Used when a block row is at least 8 bytes (FP8 Bn >= 8, FP4 Bn >= 16).  LDS
// holds whole blocks ("tile-major": a block is 32 rows x Bn codes, exactly as
// stored), streamed in by global_load_lds_dwordx4: every lane moves 16 bytes
// from its own global address to LDS base + 16*lane, so one wave instruction
// fills 1 KB and nothing passes through registers.  Taps in the padding read a
// zero block.  Two stages are double-buffered: the next stage's loads are in
// flight while the current stage's MFMAs run.

__device__ __attribute__((aligned(16))) uint8_t g_zero_block[1024];

typedef __attribute__((address_space(3))) void lds_void;

// 16 bytes per lane from gsrc into lds_base + 16 * lane.
__device__ __forceinline__ void lds_dma16(const void* gsrc, uint8_t* lds_base) {
    __builtin_amdgcn_global_load_lds(gsrc, (lds_void*)lds_base, 16, 0, 0);
}

__device__ __forceinline__ void wait_dma() {
    __builtin_amdgcn_s_waitcnt(0x0F70);   // vmcnt(0): this wave's LDS DMA has landed
}

struct StreamArgs {
    Conv cv;
    const uint8_t* wc;
    const uint8_t* ws;
    const uint8_t* bc;
    const uint8_t* bs;
    float* out;
    int layout;
    int M;                     // real output channels
    int mtiles;
    int P;                     // output pixels per tile (BN / Bn), along one output row
    int kcb;                   // channel blocks along K
    int hs, wsrc, cps, ncbs;   // activation operand geometry
    int hout, wout;            // output spatial size
    int ctiles_max;            // column tiles of the largest phase
    int a_bytes, b_bytes, stage_bytes;   // per-stage LDS regions (A, B, + scales)
};

// fwd / dgrad: one stage = one kernel row (its taps) x two channel blocks.
// B holds the halo of source pixels the row's taps read for the tile's P
// output pixels: [block][halo column] blocks; A holds the weight blocks
// [tap][block][row block].
//
// Address arithmetic is kept off the critical path: Bn is a template
// parameter (pixel / sample splits are shifts), every lane builds the
// stage-invariant part of its DMA source offsets once, and a stage only adds
// one delta per operand.  Offsets are 32-bit (tensors below 4 GB).
constexpr int NDMA = 8;        // DMA instructions per wave per stage (<= 32 KB stages)

template <int FMT, bool DG, int BNS>
__global__ __launch_bounds__(NT) void conv_stream_kernel(StreamArgs p) {
    constexpr int EB = FMT == MXC_E4M3 ? 8 : 4;
    constexpr int TA = 32 * 32 * EB / 8;              // bytes of a weight block
    constexpr int RB = BNS * EB / 8;                  // bytes of an activation block row
    constexpr int TB = 32 * RB;                       // bytes of an activation block
    constexpr int P = BN / BNS;                       // output pixels per tile
    constexpr int LOGB = BNS == 32 ? 5 : BNS == 16 ? 4 : 3;
    extern __shared__ __attribute__((aligned(16))) uint8_t smem[];
    const Conv& cv = p.cv;
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;

    // ---- tile: XCD-aware linear order over (column tile, row tile)
    const int ntile = p.mtiles * p.ctiles_max;
    const int per_xcd = (gridDim.x + 7) / 8;
    const int lin = (blockIdx.x % 8) * per_xcd + blockIdx.x / 8;
    if (lin >= ntile) return;
    const int mt = lin % p.mtiles, ct = lin / p.mtiles;

    // ---- phase and the taps that reach it (fwd: one phase, all taps)
    int ry = 0, rx = 0, kh0 = 0, kw0 = 0, nvh = cv.kh, nvw = cv.kw, gh = cv.ho, gw = cv.wo;
    if (DG) {
        ry = blockIdx.y / cv.sw; rx = blockIdx.y % cv.sw;
        kh0 = (ry + cv.ph) % cv.sh; kw0 = (rx + cv.pw) % cv.sw;
        nvh = kh0 < cv.kh ? (cv.kh - kh0 + cv.sh - 1) / cv.sh : 0;
        nvw = kw0 < cv.kw ? (cv.kw - kw0 + cv.sw - 1) / cv.sw : 0;
        gh = ry < cv.h ? (cv.h - ry + cv.sh - 1) / cv.sh : 0;
        gw = rx < cv.w ? (cv.w - rx + cv.sw - 1) / cv.sw : 0;
    }
    const int nseg = (gw + P - 1) / P;
    const int tiles = cv.x.ng * gh * nseg;
    if (ct >= tiles) return;
    const int seg = ct % nseg;
    const int r0 = ct / nseg;
    const int oyr = r0 % gh, g = r0 / gh;
    const int b0 = seg * P;

    const int CS = DG ? 1 : cv.sw;
    const int ntw = nvw;
    const int HC = (P - 1) * CS + ntw;
    const int cbase = DG ? b0 + (rx + cv.pw - (kw0 + cv.sw * (ntw - 1))) / cv.sw : b0 * cv.sw - cv.pw;
    const int nkk = (p.kcb + 1) / 2;
    const int nstage = ntw > 0 ? nkk * nvh : 0;
    const int a_pieces = ntw * 4 * TA / 16;
    const int b_pieces = 2 * HC * TB / 16;
    const int a_ins = (a_pieces + 63) / 64, b_ins = (b_pieces + 63) / 64;

    // strides (bytes) of the stored tensors
    const uint32_t w_kc = DG ? (uint32_t)cv.kh * cv.kw * cv.wt.cp * 32 * EB / 8 : (uint32_t)TA;   // per K block
    const uint32_t w_kh = (uint32_t)cv.kw * cv.wt.cp * 32 * EB / 8;
    const uint32_t x_row = (uint32_t)p.wsrc * p.cps * RB;
    const uint32_t x_kc = 32u * RB;

    // ---- per-lane DMA descriptors (stage-invariant)
    uint32_t d_off[NDMA];     // invariant source offset
    uint32_t d_zero[NDMA];    // offset inside the zero block
    int d_info[NDMA];         // bit0: B piece, bit1: block 1, bit2: invariant-valid, bit3: lane active
#pragma unroll
    for (int k = 0; k < NDMA; k++) {
        const int ins = wave + 4 * k;
        d_off[k] = 0; d_zero[k] = 0; d_info[k] = 0;
        if (ins >= a_ins + b_ins) continue;
        const bool isA = ins < a_ins;
        const int pc = (isA ? ins : ins - a_ins) * 64 + lane;
        if (isA) {
            const int t = pc / (4 * TA / 16), rem = pc % (4 * TA / 16);
            const int blk = rem / (2 * TA / 16), mb = (rem / (TA / 16)) & 1;
            const int within = (pc % (TA / 16)) * 16;
            const int rowblk = 2 * mt + mb;
            const int kw = DG ? kw0 + cv.sw * t : t;
            const bool ok = DG ? rowblk < cv.wt.ncb : rowblk < cv.wt.np / 32;
            const int cob = DG ? 0 : rowblk, cib = DG ? rowblk : 0;
            d_off[k] = ((((uint32_t)cob * cv.kh) * cv.kw + kw) * cv.wt.cp + 32 * cib) * (uint32_t)(32 * EB / 8) +
                       (uint32_t)blk * w_kc + within;
            d_zero[k] = within;
            d_info[k] = (blk << 1) | (ok ? 4 : 0) | (pc < a_pieces ? 8 : 0);
        } else {
            const int tile = pc / (TB / 16), within = (pc % (TB / 16)) * 16;
            const int blk = tile / HC, hc = tile % HC;
            const int sx = cbase + hc;
            const bool ok = sx >= 0 && sx < p.wsrc;
            d_off[k] = ((uint32_t)g * p.hs * p.wsrc + (ok ? sx : 0)) * (uint32_t)p.cps * RB +
                       (uint32_t)blk * x_kc + within;
            d_zero[k] = within;
            d_info[k] = 1 | (blk << 1) | (ok ? 4 : 0) | (pc < b_pieces ? 8 : 0);
        }
    }
    // scale descriptors: threads [0, ntw*4) A scales, [ntw*4, ntw*4 + 2*HC) B scales
    const int na = ntw * 4;
    uint32_t s_off = 0;
    int s_info = 0;
    if (tid < na) {
        const int t = tid >> 2, blk = (tid >> 1) & 1, mb = tid & 1;
        const int rowblk = 2 * mt + mb, kw = DG ? kw0 + cv.sw * t : t;
        const bool ok = DG ? rowblk < cv.wt.ncb : rowblk < cv.wt.np / 32;
        const int cob = DG ? 0 : rowblk, cib = DG ? rowblk : 0;
        s_off = (((uint32_t)cob * cv.kh) * cv.kw + kw) * cv.wt.ncb + cib +
                (uint32_t)blk * (DG ? (uint32_t)cv.kh * cv.kw * cv.wt.ncb : 1u);
        s_info = (blk << 1) | (ok ? 4 : 0) | 8;
    } else if (tid < na + 2 * HC) {
        const int q = tid - na, blk = q / HC, hc = q % HC;
        const int sx = cbase + hc;
        const bool ok = sx >= 0 && sx < p.wsrc;
        s_off = ((uint32_t)g * p.hs * p.wsrc + (ok ? sx : 0)) * p.ncbs + blk;
        s_info = 1 | (blk << 1) | (ok ? 4 : 0) | 8;
    }

    int sreg = 0;
    auto issue = [&](int st, int buf) {
        uint8_t* base = smem + buf * p.stage_bytes;
        const int kk = st / nvh, ri = st % nvh;
        const int kh = DG ? kh0 + cv.sh * ri : ri;
        const int sy = DG ? oyr + (ry + cv.ph - kh) / cv.sh : oyr * cv.sh + kh - cv.ph;
        const bool row_ok = sy >= 0 && sy < p.hs;
        const bool blk1_ok = 2 * kk + 1 < p.kcb;
        const uint32_t add_a = (uint32_t)kh * w_kh + (uint32_t)(2 * kk) * w_kc;
        const uint32_t add_b = (uint32_t)(row_ok ? sy : 0) * x_row + (uint32_t)(2 * kk) * x_kc;
#pragma unroll
        for (int k = 0; k < NDMA; k++) {
            const int ins = wave + 4 * k;
            if (ins >= a_ins + b_ins) break;
            const int info = d_info[k];
            const bool isB = info & 1;
            const bool ok = (info & 4) && ((info & 2) == 0 || blk1_ok) && (!isB || row_ok);
            const uint8_t* src = ok ? (isB ? p.bc + d_off[k] + add_b : p.wc + d_off[k] + add_a)
                                    : g_zero_block + d_zero[k];
            uint8_t* dst = isB ? base + p.a_bytes + (ins - a_ins) * 1024 : base + ins * 1024;
            if (info & 8) lds_dma16(src, dst);
        }
        sreg = 0;
        if (s_info & 8) {
            const bool isB = s_info & 1;
            const bool ok = (s_info & 4) && ((s_info & 2) == 0 || blk1_ok) && (!isB || row_ok);
            const uint32_t o = isB ? s_off + (uint32_t)(row_ok ? sy : 0) * p.wsrc * p.ncbs + 2 * kk
                                   : s_off + (uint32_t)kh * cv.kw * cv.wt.ncb +
                                         (uint32_t)(2 * kk) * (DG ? (uint32_t)cv.kh * cv.kw * cv.wt.ncb : 1u);
            sreg = ok ? (isB ? p.bs[o] : p.ws[o]) : 0;
        }
    };
    auto store_scales = [&](int buf) {
        if (s_info & 8) smem[buf * p.stage_bytes + p.a_bytes + p.b_bytes + tid] = (uint8_t)sreg;
    };

    const int wm = wave & 1, wn = wave >> 1;
    const int h = lane >> 5;
    // per-lane fragment addresses (bytes from the stage base)
    const int i16 = lane & 15, gi = lane >> 4, cg = gi & 1, hh = gi >> 1;
    int a_lane;                       // A: offset inside a weight block
    if (DG) a_lane = FMT == MXC_E4M3 ? (lane & 31) * 32 + 16 * h : (lane & 31) * 16;
    else    a_lane = FMT == MXC_E4M3 ? (16 * hh + (i16 >> 1)) * 32 + 16 * cg + 8 * (i16 & 1)
                                     : i16 * 16 + 8 * cg;
    int b_lane[2], b_hc[2], s_hc[2];
#pragma unroll
    for (int c = 0; c < 2; c++) {
        const int colbase = 64 * wn + 32 * c;
        const int col = FMT == MXC_E4M3 ? colbase + 16 * cg + 8 * (i16 & 1) : colbase + 16 * cg;
        const int pix = col >> LOGB, jb = (col & (BNS - 1)) * EB / 8;
        b_hc[c] = pix * CS;
        b_lane[c] = FMT == MXC_E4M3 ? (16 * hh + (i16 >> 1)) * RB + jb : i16 * RB + jb;
        s_hc[c] = ((colbase + (lane & 31)) >> LOGB) * CS;
    }

    v16f acc[2];
    for (int c = 0; c < 2; c++)
        for (int e = 0; e < 16; e++) acc[c][e] = 0.0f;

    if (nstage > 0) {
        issue(0, 0);
        wait_dma();
        store_scales(0);
    }
    __syncthreads();
    for (int st = 0; st < nstage; st++) {
        const int buf = st & 1;
        if (st + 1 < nstage) issue(st + 1, buf ^ 1);
        const uint8_t* A = smem + buf * p.stage_bytes;
        const uint8_t* B = A + p.a_bytes;
        const uint8_t* SC = B + p.b_bytes;
        for (int t = 0; t < ntw; t++) {
            const int co = DG ? ntw - 1 - t : t;         // halo column offset of this tap
            const uint8_t* a0 = A + ((t * 2 + 0) * 2 + wm) * TA + a_lane;
            const uint8_t* a1 = a0 + 2 * TA;
            v8i af;
            if (DG) {
                if (FMT == MXC_E4M3) {
                    const v4i x0 = *(const v4i*)a0;
                    const v4i x1 = *(const v4i*)a1;
                    af[0] = x0[0]; af[1] = x0[1]; af[2] = x0[2]; af[3] = x0[3];
                    af[4] = x1[0]; af[5] = x1[1]; af[6] = x1[2]; af[7] = x1[3];
                } else {
                    const v4i x0 = *(const v4i*)(h ? a1 : a0);
                    af[0] = x0[0]; af[1] = x0[1]; af[2] = x0[2]; af[3] = x0[3];
                    af[4] = af[5] = af[6] = af[7] = 0;
                }
            } else {
                if (FMT == MXC_E4M3) {
#pragma unroll
                    for (int blk = 0; blk < 2; blk++)
#pragma unroll
                        for (int hf = 0; hf < 2; hf++) {
                            const v2i v = lds_tr8((blk ? a1 : a0) + hf * 8 * 32);
                            af[4 * blk + 2 * hf] = v[0];
                            af[4 * blk + 2 * hf + 1] = v[1];
                        }
                } else {
                    const uint8_t* ab = hh ? a1 : a0;
#pragma unroll
                    for (int hf = 0; hf < 2; hf++) {
                        const v2i v = lds_tr4(ab + hf * 16 * 16);
                        af[2 * hf] = v[0];
                        af[2 * hf + 1] = v[1];
                    }
                    af[4] = af[5] = af[6] = af[7] = 0;
                }
            }
            const int sa = SC[(t * 2 + h) * 2 + wm];
            AFrag<FMT> ad;
            ad.set(af, sa);
#pragma unroll
            for (int c = 0; c < 2; c++) {
                v8i bf;
                const int hc = b_hc[c] + co;
                if (FMT == MXC_E4M3) {
                    const uint8_t* tb = B + hc * TB + b_lane[c];
#pragma unroll
                    for (int blk = 0; blk < 2; blk++)
#pragma unroll
                        for (int hf = 0; hf < 2; hf++) {
                            const v2i v = lds_tr8(tb + blk * HC * TB + hf * 8 * RB);
                            bf[4 * blk + 2 * hf] = v[0];
                            bf[4 * blk + 2 * hf + 1] = v[1];
                        }
                } else {
                    const uint8_t* tb = B + (hh * HC + hc) * TB + b_lane[c];
#pragma unroll
                    for (int hf = 0; hf < 2; hf++) {
                        const v2i v = lds_tr4(tb + hf * 16 * RB);
                        bf[2 * hf] = v[0];
                        bf[2 * hf + 1] = v[1];
                    }
                    bf[4] = bf[5] = bf[6] = bf[7] = 0;
                }
                const int sb = SC[ntw * 4 + h * HC + s_hc[c] + co];
                acc[c] = mfma_mx_a<FMT>(ad, bf, acc[c], sb);
            }
        }
        if (st + 1 < nstage) {
            wait_dma();
            store_scales(buf ^ 1);
        }
        __syncthreads();
    }

    // ---- epilogue: lane's column is fixed; rows step by 1 / 8
    const int oy = DG ? ry + cv.sh * oyr : oyr;
#pragma unroll
    for (int c = 0; c < 2; c++) {
        const int col = 64 * wn + 32 * c + (lane & 31);
        const int pix = col >> LOGB, j = col & (BNS - 1);
        const int ox_g = b0 + pix;
        if (ox_g >= gw) continue;
        const int ox = DG ? rx + cv.sw * ox_g : ox_g;
        const int m0 = BM * mt + 32 * wm + 4 * h;
        size_t o0, mstride;
        if (p.layout != MXC_NCHW) {
            o0 = ((((size_t)g * p.hout + oy) * p.wout + ox) * p.M + m0) * BNS + j;
            mstride = BNS;
        } else {
            o0 = (((size_t)(g * BNS + j) * p.M + m0) * p.hout + oy) * p.wout + ox;
            mstride = (size_t)p.hout * p.wout;
        }
#pragma unroll
        for (int e = 0; e < 16; e++) {
            const int dm = 8 * (e >> 2) + (e & 3);
            if (m0 + dm >= p.M) continue;
            if (p.layout == MXC_CBF_BF16) ((uint16_t*)p.out)[o0 + dm * mstride] = (uint16_t)bf16_bits(acc[c][e]);
            else                          p.out[o0 + dm * mstride] = acc[c][e];
        }
    }
}

// transposing reads need 8 consecutive FP8 samples / 16 consecutive FP4 samples
// of one block row, i.e. rows of at least 8 bytes
bool stream_ok(const Conv& cv) { return cv.x.bn * cv.bits >= 64; }

int launch_conv_stream(const Conv& cv, bool dg, const void* wc, const uint8_t* ws, const void* bc,
                       const uint8_t* bs, float* out, int layout, hipStream_t s) {
    StreamArgs a;
    a.cv = cv;
    a.wc = (const uint8_t*)wc; a.ws = ws; a.bc = (const uint8_t*)bc; a.bs = bs;
    a.out = out; a.layout = layout;
    const Geom& src = dg ? cv.gy : cv.x;
    a.hs = src.h; a.wsrc = src.w; a.cps = src.cp; a.ncbs = src.ncb;
    a.kcb = dg ? cv.wt.np / 32 : cv.wt.ncb;
    a.M = dg ? cv.cin : cv.cout;
    a.hout = dg ? cv.h : cv.ho;
    a.wout = dg ? cv.w : cv.wo;
    a.mtiles = (a.M + BM - 1) / BM;
    a.P = BN / cv.x.bn;
    const int EB = cv.bits;
    const int TA = 32 * 32 * EB / 8, TB = 32 * cv.x.bn * EB / 8;
    // LDS: the largest stage over the phases
    long maxtiles = 0;
    int max_ntw = 0, max_hc = 0;
    const int nph = dg ? cv.sh * cv.sw : 1;
    for (int ph = 0; ph < nph; ph++) {
        const int ry = dg ? ph / cv.sw : 0, rx = dg ? ph % cv.sw : 0;
        const int kw0 = dg ? (rx + cv.pw) % cv.sw : 0;
        const int nvw = dg ? (kw0 < cv.kw ? (cv.kw - kw0 + cv.sw - 1) / cv.sw : 0) : cv.kw;
        const long gh = dg ? (ry < cv.h ? (cv.h - ry + cv.sh - 1) / cv.sh : 0) : cv.ho;
        const long gw = dg ? (rx < cv.w ? (cv.w - rx + cv.sw - 1) / cv.sw : 0) : cv.wo;
        const long tiles = (long)cv.x.ng * gh * ((gw + a.P - 1) / a.P);
        if (tiles > maxtiles) maxtiles = tiles;
        const int hcv = (a.P - 1) * (dg ? 1 : cv.sw) + nvw;
        if (nvw > max_ntw) max_ntw = nvw;
        if (hcv > max_hc) max_hc = hcv;
    }
    a.a_bytes = max_ntw * 4 * TA;
    a.b_bytes = 2 * max_hc * TB;
    // each wave issues at most NDMA 1 KB DMA instructions per stage
    if ((a.a_bytes + 1023) / 1024 + (a.b_bytes + 1023) / 1024 > 4 * NDMA)
        return launch_conv(cv, dg, wc, ws, bc, bs, out, layout, s);
    a.stage_bytes = (a.a_bytes + a.b_bytes + max_ntw * 4 + 2 * max_hc + 15) / 16 * 16;
    const size_t lds = 2 * (size_t)a.stage_bytes;
    if (lds > 64 * 1024) return launch_conv(cv, dg, wc, ws, bc, bs, out, layout, s);
    const long ntile = maxtiles * a.mtiles;
    if (ntile > 0x7FFFFFF0L) return MXC_ERR_SHAPE;
    a.ctiles_max = (int)maxtiles;
    const dim3 grid((unsigned)((ntile + 7) / 8 * 8), nph);
#define MXC_LAUNCH_CS(F, D, B) hipLaunchKernelGGL((conv_stream_kernel<F, D, B>), grid, dim3(NT), lds, s, a)
    const int bn = cv.x.bn;
    if (cv.fmt == MXC_E4M3) {
        if (bn == 32)      { if (dg) MXC_LAUNCH_CS(MXC_E4M3, true, 32); else MXC_LAUNCH_CS(MXC_E4M3, false, 32); }
        else if (bn == 16) { if (dg) MXC_LAUNCH_CS(MXC_E4M3, true, 16); else MXC_LAUNCH_CS(MXC_E4M3, false, 16); }
        else               { if (dg) MXC_LAUNCH_CS(MXC_E4M3, true, 8);  else MXC_LAUNCH_CS(MXC_E4M3, false, 8); }
    } else {
        if (bn == 32)      { if (dg) MXC_LAUNCH_CS(MXC_E2M1, true, 32); else MXC_LAUNCH_CS(MXC_E2M1, false, 32); }
        else               { if (dg) MXC_LAUNCH_CS(MXC_E2M1, true, 16); else MXC_LAUNCH_CS(MXC_E2M1, false, 16); }
    }
#undef MXC_LAUNCH_CS
    return hipGetLastError() == hipSuccess ? MXC_OK : MXC_ERR_HIP;
}


// wgrad: output tile BM x BN as in wgrad_kernel; one stage = SP pixel blocks
// (SP/2 MFMA K steps).  LDS blocks are full 32 x 32-element MFMA blocks; a
// batch block shorter than 32 samples is padded with zero pieces.
struct WStreamArgs {
    Conv cv;
    const uint8_t* gc;
    const uint8_t* gs;
    const uint8_t* xc;
    const uint8_t* xs;
    float* part;
    int ntot, mtiles, ctiles, splits, kbps;   // kbps: K blocks per split, a multiple of SP
};

template <int FMT>
__global__ __launch_bounds__(NT) void wgrad_stream_kernel(WStreamArgs p) {
    constexpr int EB = FMT == MXC_E4M3 ? 8 : 4;
    constexpr int ROWB = 32 * EB / 8;                  // bytes of a 32-element row
    constexpr int TT = 32 * ROWB;                      // bytes of an LDS block
    constexpr int A_BYTES = SP * 2 * TT, B_BYTES = SP * 4 * TT;
    constexpr int STAGE = A_BYTES + B_BYTES + 32;      // + scales (SP*2 + SP*4 bytes)
    __shared__ __attribute__((aligned(16))) uint8_t smem[2 * STAGE];
    const Conv& cv = p.cv;
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int bn = cv.x.bn;
    const int rb = bn * EB / 8;                        // real bytes of a row (>= 16)
    const int npix = cv.ho * cv.wo;
    const int nkb = cv.x.ng * npix;
    const int cinb = cv.x.ncb, taps = cv.kh * cv.kw;

    const int ntile = p.mtiles * p.ctiles * p.splits;
    const int per_xcd = (gridDim.x + 7) / 8;
    const int lin = (blockIdx.x % 8) * per_xcd + blockIdx.x / 8;
    if (lin >= ntile) return;
    const int mt = lin % p.mtiles;
    const int r0 = lin / p.mtiles;
    const int ct = r0 % p.ctiles, sp = r0 / p.ctiles;
    const int kb0 = sp * p.kbps;
    const int kb1 = min(nkb, kb0 + p.kbps);
    const int nstage = kb1 > kb0 ? (kb1 - kb0 + SP - 1) / SP : 0;

    // ---- per-lane DMA descriptors.  An LDS block is 1 KB (FP8) or 512 B (FP4),
    // so one 1 KB instruction carries blocks of a single pixel slot pi; the
    // stage only supplies that slot's K block (group, output pixel).
    constexpr int PT = TT / 16;
    constexpr int NINS = (A_BYTES + B_BYTES) / 1024;    // instructions per stage
    constexpr int NK = NINS / 4;                        // per wave
    static_assert(NINS % 4 == 0, "stage must split evenly over 4 waves");
    const uint32_t gy_pix = (uint32_t)cv.gy.cp * rb;    // bytes of one G_Y pixel (all blocks)
    const uint32_t x_pix = (uint32_t)cv.x.cp * rb;
    uint32_t d_off[NK];
    int d_pi[NK], d_kh[NK], d_kw[NK], d_ok[NK], d_b[NK];
#pragma unroll
    for (int k = 0; k < NK; k++) {
        const int ins = wave + 4 * k;
        const int pc = ins * 64 + lane;
        const int tile = pc / PT, within = (pc % PT) * 16;
        const int row = within / ROWB, byte = within % ROWB;
        d_b[k] = tile >= SP * 2;
        if (!d_b[k]) {
            const int pi = tile >> 1, mb = tile & 1, cob = 2 * mt + mb;
            d_pi[k] = pi; d_kh[k] = 0; d_kw[k] = 0;
            d_ok[k] = byte < rb && cob < cv.gy.ncb;
            d_off[k] = (uint32_t)(32 * cob + row) * rb + byte;
        } else {
            const int t2 = tile - SP * 2, pi = t2 >> 2, cbk = t2 & 3;
            const int gcb = 4 * ct + cbk, tap = gcb / cinb, cib = gcb % cinb;
            d_pi[k] = pi; d_kh[k] = tap / cv.kw; d_kw[k] = tap % cv.kw;
            d_ok[k] = byte < rb && tap < taps;
            d_off[k] = (uint32_t)(32 * cib + row) * rb + byte;
        }
    }
    // scale descriptors: threads [0, 2*SP) G_Y scales, [2*SP, 6*SP) X scales
    int s_pi = 0, s_kh = 0, s_kw = 0, s_ok = 0, s_idx = 0;
    if (tid < SP * 2) {
        const int mb = tid & 1, cob = 2 * mt + mb;
        s_pi = tid >> 1; s_ok = cob < cv.gy.ncb; s_idx = cob;
    } else if (tid < SP * 6) {
        const int t2 = tid - SP * 2, cbk = t2 & 3;
        const int gcb = 4 * ct + cbk, tap = gcb / cinb;
        s_pi = t2 >> 2; s_ok = tap < taps; s_kh = tap / cv.kw; s_kw = tap % cv.kw; s_idx = gcb % cinb;
    }

    int sreg = 0;
    auto issue = [&](int st, int buf) {
        uint8_t* base = smem + buf * STAGE;
        const int bst = kb0 + st * SP;
        // positions (group, oh, ow) of the stage's SP K blocks (wave-uniform)
        int pg[SP], poh[SP], pw[SP];
        {
            const int g0 = bst / npix, px = bst % npix;
            int gg = g0, oh = px / cv.wo, ow = px % cv.wo;
#pragma unroll
            for (int i = 0; i < SP; i++) {
                pg[i] = gg; poh[i] = oh; pw[i] = ow;
                ow++;
                const bool wrap = ow == cv.wo;
                ow = wrap ? 0 : ow;
                oh += wrap ? 1 : 0;
                const bool wrap2 = oh == cv.ho;
                oh = wrap2 ? 0 : oh;
                gg += wrap2 ? 1 : 0;
            }
        }
#pragma unroll
        for (int k = 0; k < NK; k++) {
            const int ins = wave + 4 * k;
            const int pi = d_pi[k];
            const int b = bst + pi;
            const int gg = pi == 0 ? pg[0] : pi == 1 ? pg[1] : pi == 2 ? pg[2] : pg[3];
            const int oh = pi == 0 ? poh[0] : pi == 1 ? poh[1] : pi == 2 ? poh[2] : poh[3];
            const int ow = pi == 0 ? pw[0] : pi == 1 ? pw[1] : pi == 2 ? pw[2] : pw[3];
            bool ok = d_ok[k] && b < kb1;
            uint32_t off;
            const uint8_t* src;
            if (!d_b[k]) {
                off = (uint32_t)b * gy_pix + d_off[k];
                src = p.gc;
            } else {
                const int ih = oh * cv.sh + d_kh[k] - cv.ph, iw = ow * cv.sw + d_kw[k] - cv.pw;
                ok = ok && ih >= 0 && ih < cv.h && iw >= 0 && iw < cv.w;
                off = (((uint32_t)gg * cv.h + ih) * cv.w + iw) * x_pix + d_off[k];
                src = p.xc;
            }
            // a piece invalid in this stage reads the zero block at its offset
            // inside the block (< 1 KB), never at its tensor offset
            lds_dma16(ok ? src + off : g_zero_block + (lane & (PT - 1)) * 16, base + ins * 1024);
        }
        sreg = 0;
        if (tid < SP * 6) {
            const int pi = s_pi, b = bst + pi;
            const int gg = pi == 0 ? pg[0] : pi == 1 ? pg[1] : pi == 2 ? pg[2] : pg[3];
            const int oh = pi == 0 ? poh[0] : pi == 1 ? poh[1] : pi == 2 ? poh[2] : poh[3];
            const int ow = pi == 0 ? pw[0] : pi == 1 ? pw[1] : pi == 2 ? pw[2] : pw[3];
            if (tid < SP * 2) {
                if (s_ok && b < kb1) sreg = p.gs[(size_t)b * cv.gy.ncb + s_idx];
            } else {
                const int ih = oh * cv.sh + s_kh - cv.ph, iw = ow * cv.sw + s_kw - cv.pw;
                if (s_ok && b < kb1 && ih >= 0 && ih < cv.h && iw >= 0 && iw < cv.w)
                    sreg = p.xs[(((size_t)gg * cv.h + ih) * cv.w + iw) * cinb + s_idx];
            }
        }
    };
    auto store_scales = [&](int buf) {
        if (tid < SP * 6) smem[buf * STAGE + A_BYTES + B_BYTES + tid] = (uint8_t)sreg;
    };

    const int wm = wave & 1, wn = wave >> 1, h = lane >> 5, r = lane & 31;
    v16f acc[2];
    for (int c = 0; c < 2; c++)
        for (int e = 0; e < 16; e++) acc[c][e] = 0.0f;

    if (nstage > 0) {
        issue(0, 0);
        wait_dma();
        store_scales(0);
    }
    __syncthreads();
    for (int st = 0; st < nstage; st++) {
        const int buf = st & 1;
        if (st + 1 < nstage) issue(st + 1, buf ^ 1);
        const uint8_t* A = smem + buf * STAGE;
        const uint8_t* B = A + A_BYTES;
        const uint8_t* SC = B + B_BYTES;
#pragma unroll
        for (int ks = 0; ks < SP / 2; ks++) {
            v8i af;
            if (FMT == MXC_E4M3) {
                const v4i x0 = *(const v4i*)(A + ((2 * ks) * 2 + wm) * TT + r * ROWB + 16 * h);
                const v4i x1 = *(const v4i*)(A + ((2 * ks + 1) * 2 + wm) * TT + r * ROWB + 16 * h);
                af[0] = x0[0]; af[1] = x0[1]; af[2] = x0[2]; af[3] = x0[3];
                af[4] = x1[0]; af[5] = x1[1]; af[6] = x1[2]; af[7] = x1[3];
            } else {
                const v4i x0 = *(const v4i*)(A + ((2 * ks + h) * 2 + wm) * TT + r * ROWB);
                af[0] = x0[0]; af[1] = x0[1]; af[2] = x0[2]; af[3] = x0[3];
                af[4] = af[5] = af[6] = af[7] = 0;
            }
            const int sa = SC[(2 * ks + h) * 2 + wm];
            AFrag<FMT> ad;
            ad.set(af, sa);
#pragma unroll
            for (int c = 0; c < 2; c++) {
                const int cbk = 2 * wn + c;
                v8i bf;
                if (FMT == MXC_E4M3) {
                    const v4i y0 = *(const v4i*)(B + ((2 * ks) * 4 + cbk) * TT + r * ROWB + 16 * h);
                    const v4i y1 = *(const v4i*)(B + ((2 * ks + 1) * 4 + cbk) * TT + r * ROWB + 16 * h);
                    bf[0] = y0[0]; bf[1] = y0[1]; bf[2] = y0[2]; bf[3] = y0[3];
                    bf[4] = y1[0]; bf[5] = y1[1]; bf[6] = y1[2]; bf[7] = y1[3];
                } else {
                    const v4i y0 = *(const v4i*)(B + ((2 * ks + h) * 4 + cbk) * TT + r * ROWB);
                    bf[0] = y0[0]; bf[1] = y0[1]; bf[2] = y0[2]; bf[3] = y0[3];
                    bf[4] = bf[5] = bf[6] = bf[7] = 0;
                }
                const int sb = SC[SP * 2 + (2 * ks + h) * 4 + cbk];
                acc[c] = mfma_mx_a<FMT>(ad, bf, acc[c], sb);
            }
        }
        if (st + 1 < nstage) {
            wait_dma();
            store_scales(buf ^ 1);
        }
        __syncthreads();
    }

#pragma unroll
    for (int c = 0; c < 2; c++) {
        const int col = BN * ct + 64 * wn + 32 * c + (lane & 31);
        if (col >= p.ntot) continue;
#pragma unroll
        for (int e = 0; e < 16; e++) {
            const int m = BM * mt + 32 * wm + 8 * (e >> 2) + 4 * (lane >> 5) + (e & 3);
            if (m >= cv.gy.cp) continue;
            p.part[((size_t)sp * cv.gy.cp + m) * p.ntot + col] = acc[c][e];
        }
    }
}

bool wstream_ok(const Conv& cv) { return cv.x.bn * cv.bits >= 128; }   // rows of >= 16 bytes

// the general kernels above run one format for both operands, FP8 or FP4;
// FP6 and mixed pairs run only on the batch-block-32 kernels
bool general_fmt(const Conv& cv) { return cv.fmt == MXC_E4M3 || cv.fmt == MXC_E2M1; }

}  // namespace

int launch_fwd(const Conv& cv, const void* wc, const uint8_t* ws, const void* xc, const uint8_t* xs,
               float* y, int layout, hipStream_t s) {
    const int rc = launch_conv_lean(cv, false, wc, ws, xc, xs, y, layout, s);
    if (rc != 1) return rc;
    if (!general_fmt(cv)) return MXC_ERR_SHAPE;
    if (stream_ok(cv)) return launch_conv_stream(cv, false, wc, ws, xc, xs, y, layout, s);
    return launch_conv(cv, false, wc, ws, xc, xs, y, layout, s);
}

int launch_dgrad(const Conv& cv, const void* wc, const uint8_t* ws, const void* gc, const uint8_t* gs,
                 float* gx, int layout, hipStream_t s) {
    const int rc = launch_conv_lean(cv, true, wc, ws, gc, gs, gx, layout, s);
    if (rc != 1) return rc;
    if (!general_fmt(cv)) return MXC_ERR_SHAPE;
    if (stream_ok(cv)) return launch_conv_stream(cv, true, wc, ws, gc, gs, gx, layout, s);
    return launch_conv(cv, true, wc, ws, gc, gs, gx, layout, s);
}

size_t wgrad_workspace(const Conv& cv) {
    const int ls = wgrad_lean_splits(cv);
    if (ls > 0) return ls > 1 ? (size_t)ls * cv.gy.cp * cv.kh * cv.kw * cv.x.cp * sizeof(float) : 0;
    if (!general_fmt(cv)) return 0;
    const WgradPlan pl = wgrad_plan(cv);
    return (size_t)pl.splits * cv.gy.cp * pl.ntot * sizeof(float);
}

int launch_wgrad(const Conv& cv, const void* gc, const uint8_t* gs, const void* xc, const uint8_t* xs,
                 float* gw, void* ws, hipStream_t s, const float* nv_tg, const float* nv_tx, bool defer) {
    const int ls = wgrad_lean_splits(cv);
    if (nv_tg && ls == 0) return MXC_ERR_SHAPE;
    if (ls > 0) {
        const int rc = launch_wgrad_lean(cv, gc, gs, xc, xs, ls > 1 ? (float*)ws : gw, ls, s, nv_tg, nv_tx);
        if (rc || ls == 1 || defer) return rc;
        return launch_reduce(cv, (const float*)ws, gw, ls, s);
    }
    if (!general_fmt(cv)) return MXC_ERR_SHAPE;
    const WgradPlan pl = wgrad_plan(cv);
    WgradArgs a;
    a.cv = cv;
    a.gc = (const uint8_t*)gc; a.gs = gs; a.xc = (const uint8_t*)xc; a.xs = xs;
    a.part = (float*)ws;
    a.ntot = pl.ntot; a.mtiles = pl.mtiles; a.ctiles = pl.ctiles; a.splits = pl.splits; a.kbps = pl.kbps;
    const long ntile = (long)pl.mtiles * pl.ctiles * pl.splits;
    if (ntile > 0x7FFFFFF0L) return MXC_ERR_SHAPE;
    const dim3 grid((unsigned)((ntile + 7) / 8 * 8));
    int rc;
    if (wstream_ok(cv)) {
        WStreamArgs w;
        w.cv = cv;
        w.gc = a.gc; w.gs = gs; w.xc = a.xc; w.xs = xs; w.part = a.part;
        w.ntot = pl.ntot; w.mtiles = pl.mtiles; w.ctiles = pl.ctiles; w.splits = pl.splits; w.kbps = pl.kbps;
        if (cv.fmt == MXC_E4M3) hipLaunchKernelGGL((wgrad_stream_kernel<MXC_E4M3>), grid, dim3(NT), 0, s, w);
        else                    hipLaunchKernelGGL((wgrad_stream_kernel<MXC_E2M1>), grid, dim3(NT), 0, s, w);
        rc = hipGetLastError() == hipSuccess ? MXC_OK : MXC_ERR_HIP;
    } else {
        rc = cv.fmt == MXC_E4M3 ? launch_wgrad_f<MXC_E4M3>(a, grid, s) : launch_wgrad_f<MXC_E2M1>(a, grid, s);
    }
    if (rc || defer) return rc;
    return launch_reduce(cv, (const float*)ws, gw, pl.splits, s);
}

int launch_backward(const Conv& dcv, const void* wc, const uint8_t* ws, const void* gc, const uint8_t* gs,
                    float* gx, int layout, const Conv& wcv, const void* xc, const uint8_t* xs, float* gw,
                    void* wsp, hipStream_t s, bool defer) {
    const int ls = wgrad_lean_splits(wcv);
    if (ls > 0) {
        const int rc = launch_lean_bwd(dcv, wc, ws, gc, gs, gx, layout, wcv, xc, xs, ls > 1 ? (float*)wsp : gw, ls, s);
        if (rc != 1) {
            if (rc || ls == 1 || defer) return rc;
            return launch_reduce(wcv, (const float*)wsp, gw, ls, s);
        }
    }
    const int rc = launch_dgrad(dcv, wc, ws, gc, gs, gx, layout, s);
    if (rc) return rc;
    return launch_wgrad(wcv, gc, gs, xc, xs, gw, wsp, s, nullptr, nullptr, defer);
}

int wgrad_pending_splits(const Conv& cv) {
    const int ls = wgrad_lean_splits(cv);
    if (ls > 0) return ls > 1 ? ls : 0;
    return general_fmt(cv) ? wgrad_plan(cv).splits : 0;
}

int launch_wgrad_reduce_multi(int count, const WReduceJob* jobs, hipStream_t s) {
    RMulti m;
    int nq = 0;
    long nwg = 0;
    for (int i = 0; i < count; i++) {
        const int splits = wgrad_pending_splits(jobs[i].cv);
        if (splits == 0) continue;                        // G_W was written by the weight-gradient kernel
        const long wgs = reduce_wgs(jobs[i].cv, splits);
        if (nwg + wgs > 0x7FFFFFFFL) return MXC_ERR_SHAPE;
        RJob& d = m.j[nq++];
        d.part = (const float*)jobs[i].ws; d.gw = jobs[i].gw; d.r = red_geom(jobs[i].cv, splits); d.wg0 = (int)nwg;
        nwg += wgs;
    }
    if (nq == 0) return MXC_OK;
    m.count = nq;
    m.nwg = (int)nwg;
    for (int i = nq; i < MXC_WREDUCE_MAX; i++) m.j[i] = m.j[nq - 1];
    hipLaunchKernelGGL(wgrad_reduce_multi, dim3((unsigned)nwg), dim3(256), 0, s, m);
    return hipGetLastError() == hipSuccess ? MXC_OK : MXC_ERR_HIP;
}

}  // namespace mxc
