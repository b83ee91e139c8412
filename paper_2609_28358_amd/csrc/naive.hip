// naive.hip -- a6: the comparator the method is measured against (Sec. III-C,
// the baseline column of Table I).  It performs the full-precision im2col
// first and then quantizes every GEMM operand with 1-D blocks of 32 along
// that GEMM's contraction dimension, so each tensor is quantized twice per
// training step (once per GEMM it enters).  The matrices are in
// channels-last GEMM form: P = N*Ho*Wo output positions ordered (n, ho, wo),
// K = Kh*Kw*Cin ordered (kh, kw, ci); X, G_Y, G_X are NHWC and W, G_W are
// OHWI, i.e. [Cout][K].
//
//   naive_im2col_kernel  X (NHWC fp32) -> X' [P][K] fp32
//   naive_q1d_kernel     fp32 [rows][cols] -> MX "line matrix": codes
//                        [lines][Lp] with the blocked dimension contiguous
//                        (dir 0: blocks along cols, lines = rows; dir 1:
//                        blocks along rows, written transposed, lines =
//                        cols), Lp = blocked length rounded up to 64, zero
//                        padded; scales [lines][Lp/32]
//   naive_gemm_kernel    C[M][N] fp32 = A[M][Kp] B[N][Kp]^T on the scaled
//                        MFMA, both operands line matrices (K contiguous)
//   naive_col2im_kernel  G_X' [P][K] fp32 -> G_X (NHWC), a gather over taps
//
// Same element encoding as the quantize-once path (shared device helpers);
// only the block shape and the data flow differ.
#include "mx_internal.h"

namespace mxc {
namespace {

constexpr int NT = 256;

struct NaiveGeom {
    int n, cin, h, w, kh, kw, sh, sw, ph, pw, ho, wo;
    long long P, K;
};

NaiveGeom naive_geom(const Conv& cv) {
    NaiveGeom g;
    g.n = cv.n; g.cin = cv.cin; g.h = cv.h; g.w = cv.w; g.kh = cv.kh; g.kw = cv.kw;
    g.sh = cv.sh; g.sw = cv.sw; g.ph = cv.ph; g.pw = cv.pw; g.ho = cv.ho; g.wo = cv.wo;
    g.P = (long long)cv.n * cv.ho * cv.wo;
    g.K = (long long)cv.kh * cv.kw * cv.cin;
    return g;
}

int grid_for(long long work) {
    long long b = (work + NT - 1) / NT;
    return (int)(b < 65536 ? (b < 1 ? 1 : b) : 65536);
}

// ---------------------------------------------------------------- im2col
// VEC consecutive k share one tap when cin % VEC == 0.
template <int VEC>
__global__ __launch_bounds__(NT) void naive_im2col_kernel(const float* __restrict__ x,
                                                          float* __restrict__ col, NaiveGeom g) {
    const long long kq = g.K / VEC;
    const long long total = g.P * kq;
    for (long long i = (long long)blockIdx.x * NT + threadIdx.x; i < total;
         i += (long long)gridDim.x * NT) {
        const long long p = i / kq;
        const int k = (int)(i - p * kq) * VEC;
        const int ci = k % g.cin, t = k / g.cin;
        const int b = t % g.kw, a = t / g.kw;
        const int ow = (int)(p % g.wo);
        const long long q = p / g.wo;
        const int oh = (int)(q % g.ho), n = (int)(q / g.ho);
        const int ih = oh * g.sh + a - g.ph, iw = ow * g.sw + b - g.pw;
        const bool in = ih >= 0 && ih < g.h && iw >= 0 && iw < g.w;
        const size_t src = (((size_t)n * g.h + (in ? ih : 0)) * g.w + (in ? iw : 0)) * g.cin + ci;
        if (VEC == 4) {
            float4 v = in ? *(const float4*)(x + src) : make_float4(0.f, 0.f, 0.f, 0.f);
            *(float4*)(col + (size_t)i * 4) = v;
        } else {
            col[i] = in ? x[src] : 0.0f;
        }
    }
}

// ---------------------------------------------------------------- col2im
// G_X[n][ih][iw][ci] = sum over taps (a, b) whose output pixel exists of
// G_X'[(n, oh, ow)][(a, b, ci)].
template <int VEC>
__global__ __launch_bounds__(NT) void naive_col2im_kernel(const float* __restrict__ gcol,
                                                          float* __restrict__ gx, NaiveGeom g) {
    const int cq = g.cin / VEC;
    const long long total = (long long)g.n * g.h * g.w * cq;
    for (long long i = (long long)blockIdx.x * NT + threadIdx.x; i < total;
         i += (long long)gridDim.x * NT) {
        const int ci = (int)(i % cq) * VEC;
        long long r = i / cq;
        const int iw = (int)(r % g.w);
        r /= g.w;
        const int ih = (int)(r % g.h), n = (int)(r / g.h);
        float4 acc = make_float4(0.f, 0.f, 0.f, 0.f);
        for (int a = 0; a < g.kh; a++) {
            const int th = ih + g.ph - a;
            if (th < 0 || th % g.sh) continue;
            const int oh = th / g.sh;
            if (oh >= g.ho) continue;
            for (int b = 0; b < g.kw; b++) {
                const int tw = iw + g.pw - b;
                if (tw < 0 || tw % g.sw) continue;
                const int ow = tw / g.sw;
                if (ow >= g.wo) continue;
                const size_t o = (((size_t)n * g.ho + oh) * g.wo + ow) * g.K + (a * g.kw + b) * g.cin + ci;
                if (VEC == 4) {
                    const float4 v = *(const float4*)(gcol + o);
                    acc.x += v.x; acc.y += v.y; acc.z += v.z; acc.w += v.w;
                } else {
                    acc.x += gcol[o];
                }
            }
        }
        if (VEC == 4) *(float4*)(gx + (size_t)i * 4) = acc;
        else gx[i] = acc.x;
    }
}

// ---------------------------------------------------------------- 1-D quantize
// One thread per block of 32.  dir 0: block b of row `line` holds
// src[line][32b .. 32b+31]; threads walk b fastest.  dir 1: block b of
// column `line` holds src[32b .. 32b+31][line]; threads walk the columns
// fastest so each of the 32 loads is coalesced across the wave.
template <int FMT, int DIR, int VEC>
__global__ __launch_bounds__(NT) void naive_q1d_kernel(const float* __restrict__ src, long long rows,
                                                       long long cols, long long lp,
                                                       uint8_t* __restrict__ codes,
                                                       uint8_t* __restrict__ scales) {
    const long long lines = DIR == 0 ? rows : cols;
    const long long len = DIR == 0 ? cols : rows;
    const long long nb = lp / 32;
    const long long total = lines * nb;
    for (long long t = (long long)blockIdx.x * NT + threadIdx.x; t < total;
         t += (long long)gridDim.x * NT) {
        long long line, b;
        if (DIR == 0) { line = t / nb; b = t - line * nb; }
        else          { b = t / lines; line = t - b * lines; }
        const long long e0 = 32 * b;
        float4 x[8];
        if (DIR == 0 && VEC == 4) {
            const float* s = src + line * cols + e0;
#pragma unroll
            for (int q = 0; q < 8; q++)
                x[q] = e0 + 4 * q < len ? *(const float4*)(s + 4 * q) : make_float4(0.f, 0.f, 0.f, 0.f);
        } else {
            float v[32];
#pragma unroll
            for (int q = 0; q < 32; q++) {
                const long long e = e0 + q;
                const size_t at = DIR == 0 ? (size_t)(line * cols + e) : (size_t)(e * cols + line);
                v[q] = e < len ? src[at] : 0.0f;
            }
#pragma unroll
            for (int q = 0; q < 8; q++) x[q] = make_float4(v[4 * q], v[4 * q + 1], v[4 * q + 2], v[4 * q + 3]);
        }
        uint32_t m = 0;
#pragma unroll
        for (int q = 0; q < 8; q++) {
            m = max(m, __float_as_uint(x[q].x) & 0x7FFFFFFFu);
            m = max(m, __float_as_uint(x[q].y) & 0x7FFFFFFFu);
            m = max(m, __float_as_uint(x[q].z) & 0x7FFFFFFFu);
            m = max(m, __float_as_uint(x[q].w) & 0x7FFFFFFFu);
        }
        constexpr int EMAX = FMT == MXC_E4M3 ? 8 : 2;
        const uint32_t sc = scale_code_from_bits<EMAX>(m);
        scales[line * nb + b] = (uint8_t)sc;
        const float inv = inv_scale(sc);
        const bool bad = sc == 0xFFu;
        if (FMT == MXC_E4M3) {
            uint32_t w[8];
#pragma unroll
            for (int q = 0; q < 8; q++) w[q] = bad ? 0u : pack4_e4m3(x[q], inv);
            uint4* d = (uint4*)(codes + line * lp + e0);
            d[0] = make_uint4(w[0], w[1], w[2], w[3]);
            d[1] = make_uint4(w[4], w[5], w[6], w[7]);
        } else {
            uint32_t w[4];
#pragma unroll
            for (int q = 0; q < 4; q++) w[q] = bad ? 0u : pack8_e2m1(x[2 * q], x[2 * q + 1], inv);
            *(uint4*)(codes + (line * lp + e0) / 2) = make_uint4(w[0], w[1], w[2], w[3]);
        }
    }
}

// ---------------------------------------------------------------- GEMM
// C[M][N] = A[M][Kp] B[N][Kp]^T, both operands line matrices (codes K
// contiguous, one scale per 32 K).  Four waves in a WM x WN arrangement, each
// owning 64 x 64 outputs (2 x 2 MFMAs of 32 x 32 x 64 per K step).  Operands
// are read straight from memory into the MFMA fragments (no LDS): lane l
// holds row l % 32 and K half l / 32 of each fragment.  Rows past M / N read
// the last row and are never stored.  blockIdx.y splits K; with more than one
// split the results are added atomically into C, which the launcher zeroes.
template <int FMT, int WM, int WN>
__global__ __launch_bounds__(NT) void naive_gemm_kernel(const uint8_t* __restrict__ a,
                                                        const uint8_t* __restrict__ as,
                                                        const uint8_t* __restrict__ b,
                                                        const uint8_t* __restrict__ bs, int m, int n,
                                                        int ksteps, int steps_per_split, int tiles_m,
                                                        float* __restrict__ c) {
    constexpr int RB = FMT == MXC_E4M3 ? 64 : 32;        // code bytes per row per K step
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int h = lane >> 5, r = lane & 31;
    const int tm = blockIdx.x % tiles_m, tn = blockIdx.x / tiles_m;
    const int mbase = (tm * WM + wave % WM) * 64, nbase = (tn * WN + wave / WM) * 64;
    const int k0 = blockIdx.y * steps_per_split;
    const int k1 = min(ksteps, k0 + steps_per_split);
    const size_t rowb = (size_t)ksteps * RB, rows_s = (size_t)ksteps * 2;

    const uint8_t* ap[2];
    const uint8_t* bp[2];
    const uint8_t* asp[2];
    const uint8_t* bsp[2];
#pragma unroll
    for (int i = 0; i < 2; i++) {
        const int ra = min(mbase + 32 * i + r, m - 1), rb = min(nbase + 32 * i + r, n - 1);
        ap[i] = a + ra * rowb + 16 * h;
        bp[i] = b + rb * rowb + 16 * h;
        asp[i] = as + ra * rows_s + h;
        bsp[i] = bs + rb * rows_s + h;
    }
    auto frag = [&](const uint8_t* p, int k) {
        v8i f;
        const v4i lo = *(const v4i*)(p + (size_t)k * RB);
        f[0] = lo[0]; f[1] = lo[1]; f[2] = lo[2]; f[3] = lo[3];
        if (FMT == MXC_E4M3) {
            const v4i hi = *(const v4i*)(p + (size_t)k * RB + 32);
            f[4] = hi[0]; f[5] = hi[1]; f[6] = hi[2]; f[7] = hi[3];
        } else {
            f[4] = f[5] = f[6] = f[7] = 0;
        }
        return f;
    };

    v16f acc[2][2];
#pragma unroll
    for (int i = 0; i < 2; i++)
#pragma unroll
        for (int j = 0; j < 2; j++)
#pragma unroll
            for (int e = 0; e < 16; e++) acc[i][j][e] = 0.0f;

    if (k0 < k1) {
        v8i fa[2], fb[2];
        int sa[2], sb[2];
#pragma unroll
        for (int i = 0; i < 2; i++) {
            fa[i] = frag(ap[i], k0); fb[i] = frag(bp[i], k0);
            sa[i] = asp[i][2 * k0]; sb[i] = bsp[i][2 * k0];
        }
        for (int k = k0; k < k1; k++) {
            // next step's operands are loaded before this step's MFMAs issue
            const int kn = k + 1 < k1 ? k + 1 : k;
            v8i na[2], nb[2];
            int nsa[2], nsb[2];
#pragma unroll
            for (int i = 0; i < 2; i++) {
                na[i] = frag(ap[i], kn); nb[i] = frag(bp[i], kn);
                nsa[i] = asp[i][2 * kn]; nsb[i] = bsp[i][2 * kn];
            }
            if constexpr (FMT == MXC_E4M3) {   // each fragment decoded to bf16 once (exact products)
                uint32_t ad[2][16], bd[2][16];
#pragma unroll
                for (int i = 0; i < 2; i++) {
                    e4m3_decode32_lane(fa[i], sa[i], ad[i]);
                    e4m3_decode32_lane(fb[i], sb[i], bd[i]);
                }
#pragma unroll
                for (int i = 0; i < 2; i++)
#pragma unroll
                    for (int j = 0; j < 2; j++) acc[i][j] = mfma_x8(ad[i], bd[j], acc[i][j]);
            } else {
#pragma unroll
                for (int i = 0; i < 2; i++)
#pragma unroll
                    for (int j = 0; j < 2; j++) acc[i][j] = mfma_mx<FMT>(fa[i], fb[j], acc[i][j], sa[i], sb[j]);
            }
#pragma unroll
            for (int i = 0; i < 2; i++) { fa[i] = na[i]; fb[i] = nb[i]; sa[i] = nsa[i]; sb[i] = nsb[i]; }
        }
    }

    const bool split = gridDim.y > 1;
#pragma unroll
    for (int j = 0; j < 2; j++) {
        const int col = nbase + 32 * j + r;
        if (col >= n) continue;
#pragma unroll
        for (int i = 0; i < 2; i++)
#pragma unroll
            for (int e = 0; e < 16; e++) {
                const int row = mbase + 32 * i + 8 * (e >> 2) + 4 * h + (e & 3);
                if (row >= m) continue;
                float* o = c + (size_t)row * n + col;
                if (split) unsafeAtomicAdd(o, acc[i][j][e]);
                else *o = acc[i][j][e];
            }
    }
}

__global__ __launch_bounds__(NT) void naive_zero_kernel(float* __restrict__ p, long long count) {
    for (long long i = (long long)blockIdx.x * NT + threadIdx.x; i < count; i += (long long)gridDim.x * NT)
        p[i] = 0.0f;
}

template <int FMT, int WM, int WN>
void gemm_t(const uint8_t* a, const uint8_t* as, const uint8_t* b, const uint8_t* bs, int m, int n,
            int ksteps, float* c, hipStream_t s) {
    const int tiles_m = (m + 64 * WM - 1) / (64 * WM), tiles_n = (n + 64 * WN - 1) / (64 * WN);
    const int tiles = tiles_m * tiles_n;
    // split K only when the tile grid alone cannot fill the chip
    int splits = 1;
    if (tiles < 512) {
        splits = min(1024 / tiles, max(1, ksteps / 8));
        if (splits < 1) splits = 1;
    }
    const int per = (ksteps + splits - 1) / splits;
    splits = (ksteps + per - 1) / per;
    if (splits > 1)
        hipLaunchKernelGGL(naive_zero_kernel, dim3(grid_for((long long)m * n)), dim3(NT), 0, s, c,
                           (long long)m * n);
    hipLaunchKernelGGL((naive_gemm_kernel<FMT, WM, WN>), dim3(tiles, splits), dim3(NT), 0, s, a, as, b,
                       bs, m, n, ksteps, per, tiles_m, c);
}

template <int FMT>
void gemm_fmt(const uint8_t* a, const uint8_t* as, const uint8_t* b, const uint8_t* bs, int m, int n,
              int ksteps, float* c, hipStream_t s) {
    if (n <= 64)      gemm_t<FMT, 4, 1>(a, as, b, bs, m, n, ksteps, c, s);
    else if (m <= 64) gemm_t<FMT, 1, 4>(a, as, b, bs, m, n, ksteps, c, s);
    else              gemm_t<FMT, 2, 2>(a, as, b, bs, m, n, ksteps, c, s);
}

int gemm(int fmt, const void* a, const uint8_t* as, const void* b, const uint8_t* bs, long long m,
         long long n, long long klen, float* c, hipStream_t s) {
    const long long lp = naive_line_len(klen);
    if (m > 0x7FFFFFFFLL || n > 0x7FFFFFFFLL || lp / 64 > 0x7FFFFFFFLL) return MXC_ERR_SHAPE;
    const int ksteps = (int)(lp / 64);
    if (fmt == MXC_E4M3) gemm_fmt<MXC_E4M3>((const uint8_t*)a, as, (const uint8_t*)b, bs, (int)m, (int)n, ksteps, c, s);
    else                 gemm_fmt<MXC_E2M1>((const uint8_t*)a, as, (const uint8_t*)b, bs, (int)m, (int)n, ksteps, c, s);
    return hipGetLastError() == hipSuccess ? MXC_OK : MXC_ERR_HIP;
}

}  // namespace

int launch_naive_im2col(const Conv& cv, const float* x, float* col, hipStream_t s) {
    const NaiveGeom g = naive_geom(cv);
    if (cv.cin % 4 == 0)
        hipLaunchKernelGGL(naive_im2col_kernel<4>, dim3(grid_for(g.P * g.K / 4)), dim3(NT), 0, s, x, col, g);
    else
        hipLaunchKernelGGL(naive_im2col_kernel<1>, dim3(grid_for(g.P * g.K)), dim3(NT), 0, s, x, col, g);
    return hipGetLastError() == hipSuccess ? MXC_OK : MXC_ERR_HIP;
}

int launch_naive_q1d(const float* src, long long rows, long long cols, int dir, int fmt, void* codes,
                     uint8_t* scales, hipStream_t s) {
    const long long len = dir == 0 ? cols : rows, lines = dir == 0 ? rows : cols;
    const long long lp = naive_line_len(len);
    const int grid = grid_for(lines * (lp / 32));
    uint8_t* cd = (uint8_t*)codes;
    const bool v4 = cols % 4 == 0;
#define Q1D(F, D, V) hipLaunchKernelGGL((naive_q1d_kernel<F, D, V>), dim3(grid), dim3(NT), 0, s, src, rows, \
                                        cols, lp, cd, scales)
    if (fmt == MXC_E4M3) {
        if (dir == 1) Q1D(MXC_E4M3, 1, 1);
        else if (v4)  Q1D(MXC_E4M3, 0, 4);
        else          Q1D(MXC_E4M3, 0, 1);
    } else {
        if (dir == 1) Q1D(MXC_E2M1, 1, 1);
        else if (v4)  Q1D(MXC_E2M1, 0, 4);
        else          Q1D(MXC_E2M1, 0, 1);
    }
#undef Q1D
    return hipGetLastError() == hipSuccess ? MXC_OK : MXC_ERR_HIP;
}

int launch_naive_fwd(const Conv& cv, const void* cc, const uint8_t* cs, const void* wc,
                     const uint8_t* ws, float* y, hipStream_t s) {
    const NaiveGeom g = naive_geom(cv);
    return gemm(cv.fmt, cc, cs, wc, ws, g.P, cv.cout, g.K, y, s);
}

int launch_naive_dgrad(const Conv& cv, const void* gc, const uint8_t* gs, const void* wtc,
                       const uint8_t* wts, float* gcol, float* gx, hipStream_t s) {
    const NaiveGeom g = naive_geom(cv);
    int rc = gemm(cv.fmt, gc, gs, wtc, wts, g.P, g.K, cv.cout, gcol, s);
    if (rc) return rc;
    const long long nx = (long long)cv.n * cv.h * cv.w * cv.cin;
    if (cv.cin % 4 == 0)
        hipLaunchKernelGGL(naive_col2im_kernel<4>, dim3(grid_for(nx / 4)), dim3(NT), 0, s, gcol, gx, g);
    else
        hipLaunchKernelGGL(naive_col2im_kernel<1>, dim3(grid_for(nx)), dim3(NT), 0, s, gcol, gx, g);
    return hipGetLastError() == hipSuccess ? MXC_OK : MXC_ERR_HIP;
}

int launch_naive_wgrad(const Conv& cv, const void* gtc, const uint8_t* gts, const void* xtc,
                       const uint8_t* xts, float* gw, hipStream_t s) {
    const NaiveGeom g = naive_geom(cv);
    return gemm(cv.fmt, gtc, gts, xtc, xts, cv.cout, g.K, g.P, gw, s);
}

}  // namespace mxc
