// quantize.hip -- a1: quantize a float tensor once into MX-CBF codes and
// E8M0 scales (Sec. III-A Eqs. (4)-(6), OCP-MX form, with the square blocks of
// Sec. IV-B: 32 channels x Bn samples at one pixel).
//
// One workgroup (256 threads) handles slabs of 256 "units"; a unit is 32
// consecutive elements of one block in code order ([c][j], j fastest), so a
// slab is TT = 256/Bn consecutive pixels of one (batch group, channel block).
//   1. load: every thread reads 32 elements, lanes walking the source's
//      contiguous dimension (pixels for NCHW, channels for NHWC, samples for
//      CBF), and stores them into an LDS slab in code order (16-byte chunks
//      XOR-swizzled per unit to spread banks);
//   2. each thread takes one unit: max |x| over its 32 elements, then over the
//      Bn lanes that share the block (xor shuffles);
//   3. scale code from the exponent bits; elements scaled by 2^-s (exact) and
//      encoded with the hardware converts, codes stored as 16-byte vectors.
// Traffic: 4 (or 2) bytes read and 1, 3/4 or 1/2 byte written per element
// (FP8, FP6, FP4), plus one scale byte per block; HBM-bound.
//
// CBF sources with Bn = 32 and OIHW weights skip the slab: their blocks need
// no transposition, so one wave quantizes one block straight from its
// registers (quantize_block_kernel).
#include "mx_internal.h"

namespace mxc {
namespace {

constexpr int QT = 256;            // threads per workgroup

__device__ __forceinline__ int swz(int u) { return ((u >> 5) ^ (u >> 1)) & 7; }

// Four consecutive source elements as floats (bf16 widened exactly).
template <int DTYPE, int VEC>
__device__ __forceinline__ float4 load4(const void* src, size_t i) {
    if (VEC == 4) {
        if (DTYPE == MXC_F32) return __ldg((const float4*)((const float*)src + i));
        const uint2 b = __ldg((const uint2*)((const unsigned short*)src + i));
        return make_float4(__uint_as_float(b.x << 16), __uint_as_float(b.x & 0xFFFF0000u),
                           __uint_as_float(b.y << 16), __uint_as_float(b.y & 0xFFFF0000u));
    }
    float v;
    if (DTYPE == MXC_F32) v = __ldg((const float*)src + i);
    else v = __uint_as_float((uint32_t)__ldg((const unsigned short*)src + i) << 16);
    return make_float4(v, 0.0f, 0.0f, 0.0f);
}

// VEC = 4: every thread moves 8 runs of 4 consecutive elements along the
// source's contiguous dimension (16-byte loads); VEC = 1: 32 single elements.
// All loads of a slab are issued before any is consumed (addresses of
// out-of-range elements are clamped to the tensor's first element and the
// value replaced by zero), so each thread has its whole slab share in flight.
__device__ __forceinline__ float comp(const float4& v, int t) {
    return t == 0 ? v.x : t == 1 ? v.y : t == 2 ? v.z : v.w;
}

// Stochastic codes of N consecutive elements x[0 .. N/4) whose first code
// position is 8 q0; GEN selects the encoder that also handles fp32 subnormals.
template <int FMT, int N, bool GEN>
__device__ __forceinline__ void sr_codes(uint32_t* cd, const float4* x, uint64_t q0, int s, float inv, bool bad,
                                         uint32_t k0, uint32_t k1) {
#pragma unroll
    for (int g8 = 0; g8 < N / 8; g8++) {
        const uint4 w = sr_words(q0 + g8, k0, k1);
#pragma unroll
        for (int j = 0; j < 8; j++) {
            const int k = 8 * g8 + j;
            const float xv = comp(x[k >> 2], k & 3);
            const uint32_t r = sr_half(w, j);
            const uint32_t c = GEN ? encode_sr<FMT>(xv, s, inv, r) : encode_sr_normal<FMT>(xv, s, inv, r);
            cd[k] = bad ? 0u : c;
        }
    }
}

// Codes of 32 consecutive elements (x[0..7]) at code position e0 (a multiple
// of 8) by stochastic rounding, written at their place in the code array.
template <int FMT>
__device__ __forceinline__ void store_sr32(uint8_t* __restrict__ codes, size_t e0, const float4* x, int s,
                                           float inv, bool bad, uint32_t k0, uint32_t k1) {
    uint32_t cd[32];
    bool gen = false;
#pragma unroll
    for (int k = 0; k < 32; k++) gen |= sr_needs_general(comp(x[k >> 2], k & 3));
    // wave-uniform choice: only a wave holding an fp32 subnormal takes the general path
    if (__builtin_amdgcn_ballot_w64(gen) != 0)
        sr_codes<FMT, 32, true>(cd, x, (uint64_t)(e0 >> 3), s, inv, bad, k0, k1);
    else
        sr_codes<FMT, 32, false>(cd, x, (uint64_t)(e0 >> 3), s, inv, bad, k0, k1);
    if constexpr (FMT == MXC_E4M3) {
        uint32_t w[8];
#pragma unroll
        for (int q = 0; q < 8; q++) w[q] = cd[4 * q] | cd[4 * q + 1] << 8 | cd[4 * q + 2] << 16 | cd[4 * q + 3] << 24;
        uint4* dst = (uint4*)(codes + e0);
        dst[0] = make_uint4(w[0], w[1], w[2], w[3]);
        dst[1] = make_uint4(w[4], w[5], w[6], w[7]);
    } else if constexpr (fmt_bits(FMT) == 6) {
        uint32_t w[6] = {0u, 0u, 0u, 0u, 0u, 0u};
#pragma unroll
        for (int k = 0; k < 32; k++) {
            const int bit = 6 * k;
            w[bit >> 5] |= cd[k] << (bit & 31);
            if ((bit & 31) > 26) w[(bit >> 5) + 1] |= cd[k] >> (32 - (bit & 31));
        }
        uint2* dst = (uint2*)(codes + e0 / 4 * 3);
        dst[0] = make_uint2(w[0], w[1]);
        dst[1] = make_uint2(w[2], w[3]);
        dst[2] = make_uint2(w[4], w[5]);
    } else {
        uint32_t w[4];
#pragma unroll
        for (int q = 0; q < 4; q++) {
            uint32_t v = 0u;
#pragma unroll
            for (int t = 0; t < 8; t++) v |= cd[8 * q + t] << (4 * t);
            w[q] = v;
        }
        *(uint4*)(codes + e0 / 2) = make_uint4(w[0], w[1], w[2], w[3]);
    }
}

template <int LAYOUT, int DTYPE, int FMT, int VEC, bool SR>
__global__ __launch_bounds__(QT) void quantize_kernel(const void* __restrict__ src, Geom g,
                                                      uint8_t* __restrict__ codes,
                                                      uint8_t* __restrict__ scales,
                                                      int nslabs, int pixblocks, int slabs_per_wg,
                                                      uint32_t k0, uint32_t k1) {
    __shared__ __attribute__((aligned(16))) float slab[QT * 32];
    const int tid = threadIdx.x;
    const int bn = g.bn, tt = QT / bn;
    const int hw = g.h * g.w;
    constexpr int NL = 32 / VEC;              // loads per thread per slab

    // XCD-aware order: workgroups are dealt round-robin to the 8 XCDs, so give
    // each XCD a contiguous range of slabs (neighbouring pixel blocks share
    // cache lines in NCHW).
    const int nwg = gridDim.x;
    const int per_xcd = (nwg + 7) / 8;
    const int wg = (blockIdx.x % 8) * per_xcd + blockIdx.x / 8;

    for (int it = 0; it < slabs_per_wg; it++) {
        const int slab_id = wg * slabs_per_wg + it;
        if (slab_id >= nslabs) return;
        const int pb = slab_id % pixblocks;
        const int rest = slab_id / pixblocks;
        const int cb = rest % g.ncb;
        const int ng = rest / g.ncb;
        const int p0 = pb * tt;

        // ---- 1. load (all loads first), then store into the slab in code order
        float4 v[NL];
        int ci0[NL];
#pragma unroll
        for (int r = 0; r < NL; r++) {
            const int e = (tid + QT * r) * VEC;
            int pl, cl, j;
            if (LAYOUT == MXC_NCHW) {
                pl = e % tt; const int r1 = e / tt; cl = r1 & 31; j = r1 >> 5;
            } else if (LAYOUT == MXC_NHWC) {
                cl = e & 31; const int r1 = e >> 5; pl = r1 % tt; j = r1 / tt;
            } else {
                j = e % bn; const int r1 = e / bn; cl = r1 & 31; pl = r1 >> 5;
            }
            const int pix = p0 + pl, c = cb * 32 + cl, n = ng * bn + j;
            const bool ok = pix < hw && c < g.c && n < g.n;
            size_t gi;
            if (LAYOUT == MXC_NCHW)      gi = ((size_t)n * g.c + c) * hw + pix;
            else if (LAYOUT == MXC_NHWC) gi = ((size_t)n * hw + pix) * g.c + c;
            else                         gi = (((size_t)ng * hw + pix) * g.c + c) * bn + j;
            v[r] = load4<DTYPE, VEC>(src, ok ? gi : 0);
            if (!ok) v[r] = make_float4(0.0f, 0.0f, 0.0f, 0.0f);
            ci0[r] = (pl * 32 + cl) * bn + j;          // canonical index of the first element
        }
#pragma unroll
        for (int r = 0; r < NL; r++) {
            if (LAYOUT == MXC_CBF && VEC == 4) {
                // four consecutive samples: one 16-byte chunk of the slab
                const int u = ci0[r] >> 5, k = ci0[r] & 31;
                *(float4*)&slab[u * 32 + (((k >> 2) ^ swz(u)) << 2)] = v[r];
                continue;
            }
            const float x4[4] = {v[r].x, v[r].y, v[r].z, v[r].w};
#pragma unroll
            for (int q = 0; q < VEC; q++) {
                // the q-th element steps along the contiguous dimension
                int ci;
                if (LAYOUT == MXC_NCHW)      ci = ci0[r] + q * 32 * bn;
                else if (LAYOUT == MXC_NHWC) ci = ci0[r] + q * bn;
                else                         ci = ci0[r] + q;
                const int u = ci >> 5, k = ci & 31;
                slab[u * 32 + ((((k >> 2) ^ swz(u))) << 2) + (k & 3)] = x4[q];
            }
        }
        __syncthreads();

        // ---- 2. one unit per thread; block max over the bn lanes of a block
        const int u = tid;
        float4 x[8];
        uint32_t m = 0;
#pragma unroll
        for (int q = 0; q < 8; q++) {
            x[q] = *(const float4*)&slab[u * 32 + ((q ^ swz(u)) << 2)];
            m = max(m, __float_as_uint(x[q].x) & 0x7FFFFFFFu);
            m = max(m, __float_as_uint(x[q].y) & 0x7FFFFFFFu);
            m = max(m, __float_as_uint(x[q].z) & 0x7FFFFFFFu);
            m = max(m, __float_as_uint(x[q].w) & 0x7FFFFFFFu);
        }
        for (int off = 1; off < bn; off <<= 1) m = max(m, (uint32_t)__shfl_xor((int)m, off));
        __syncthreads();   // the slab is reused by the next iteration

        const int pl = u / bn, part = u % bn;      // pixel in slab, unit within the block
        const int pix = p0 + pl;
        if (pix >= hw) continue;
        const uint32_t sc = scale_code_from_bits<fmt_emax(FMT)>(m);
        const size_t blk = ((size_t)ng * hw + pix) * g.ncb + cb;
        if (part == 0) scales[blk] = (uint8_t)sc;
        const float inv = inv_scale(sc);
        const bool bad = sc == 0xFFu;
        const size_t e0 = (((size_t)ng * hw + pix) * g.cp + cb * 32) * bn + part * 32;

        // ---- 3. encode and store
        if constexpr (SR) {
            store_sr32<FMT>(codes, e0, x, (int)sc - 127, inv, bad, k0, k1);
        } else if (FMT == MXC_E4M3) {
            uint32_t w[8];
#pragma unroll
            for (int q = 0; q < 8; q++) w[q] = bad ? 0u : pack4_e4m3(x[q], inv);
            uint4* dst = (uint4*)(codes + e0);
            dst[0] = make_uint4(w[0], w[1], w[2], w[3]);
            dst[1] = make_uint4(w[4], w[5], w[6], w[7]);
        } else if constexpr (fmt_bits(FMT) == 6) {
            // 32 codes = 24 bytes at byte 3/4 e0 (a multiple of 24)
            const v6i w = pack32_fp6<FMT>(x, inv);
            uint2* dst = (uint2*)(codes + e0 / 4 * 3);
            dst[0] = bad ? make_uint2(0, 0) : make_uint2(w[0], w[1]);
            dst[1] = bad ? make_uint2(0, 0) : make_uint2(w[2], w[3]);
            dst[2] = bad ? make_uint2(0, 0) : make_uint2(w[4], w[5]);
        } else {
            uint32_t w[4];
#pragma unroll
            for (int q = 0; q < 4; q++) w[q] = bad ? 0u : pack8_e2m1(x[2 * q], x[2 * q + 1], inv);
            *(uint4*)(codes + e0 / 2) = make_uint4(w[0], w[1], w[2], w[3]);
        }
    }
}

// One wave per 32 x 32 block, for the two sources whose blocks need no
// transposition: a CBF activation with Bn = 32 (a block is 1024 contiguous
// source elements in code order) and OIHW weights (a block is a gather of
// 32 Cout x 32 Cin at one tap).  Block index b = scale index; its codes are
// the 1024 elements at b * 1024.  Lane l holds the four element runs
// [256 q + 4 l, 256 q + 4 l + 4), q = 0..3, so every load and store
// instruction of the wave covers one contiguous range.
// SRC 0: CBF activation, SRC 1: NCHW-ordered weights (n = Cout).
// FP6 (768-byte blocks): lane l holds the 16 consecutive elements [16 l,
// 16 l + 16) -- half a channel row -- and writes their 12 bytes of codes, so
// the wave's store is one contiguous 768-byte run.
// The same layout serves stochastic rounding in every format (positions
// 16 l .. 16 l + 15 take their random bits from two generator calls).
template <int SRC, int DTYPE, int FMT, bool SR>
__device__ __forceinline__ void quantize_block16(const void* __restrict__ src, const Geom& g,
                                                 uint8_t* __restrict__ codes, uint8_t* __restrict__ scales,
                                                 int blk, int lane, uint32_t k0, uint32_t k1) {
    const int cb = blk % g.ncb, rest = blk / g.ncb;
    const int c = cb * 32 + (lane >> 1);                     // channel (input channel) of the half row
    const int j0 = 16 * (lane & 1);                          // first sample (output channel)
    float4 x[4];
    if (SRC == 0) {
        const bool ok = c < g.c;
        const size_t i0 = ((size_t)rest * g.c + (ok ? c : 0)) * 32 + j0;
#pragma unroll
        for (int q = 0; q < 4; q++) {
            if (DTYPE == MXC_F32) {
                x[q] = load_nt((const float*)src + i0 + 4 * q);
            } else {
                const uint2 b = load_nt((const unsigned short*)src + i0 + 4 * q);
                x[q] = make_float4(__uint_as_float(b.x << 16), __uint_as_float(b.x & 0xFFFF0000u),
                                   __uint_as_float(b.y << 16), __uint_as_float(b.y & 0xFFFF0000u));
            }
            if (!ok) x[q] = make_float4(0.f, 0.f, 0.f, 0.f);
        }
    } else {
        const int hw = g.h * g.w;
        const int cob = rest / hw, tap = rest % hw;
        float v[16];
#pragma unroll
        for (int k = 0; k < 16; k++) {
            const int n = cob * 32 + j0 + k;
            const bool ok = c < g.c && n < g.n;
            const size_t i = ok ? ((size_t)n * g.c + c) * hw + tap : 0;
            v[k] = DTYPE == MXC_F32 ? __ldg((const float*)src + i)
                                    : __uint_as_float((uint32_t)__ldg((const unsigned short*)src + i) << 16);
            if (!ok) v[k] = 0.0f;
        }
#pragma unroll
        for (int q = 0; q < 4; q++) x[q] = make_float4(v[4 * q], v[4 * q + 1], v[4 * q + 2], v[4 * q + 3]);
    }
    uint32_t m = 0;
#pragma unroll
    for (int q = 0; q < 4; q++) {
        m = max(m, __float_as_uint(x[q].x) & 0x7FFFFFFFu);
        m = max(m, __float_as_uint(x[q].y) & 0x7FFFFFFFu);
        m = max(m, __float_as_uint(x[q].z) & 0x7FFFFFFFu);
        m = max(m, __float_as_uint(x[q].w) & 0x7FFFFFFFu);
    }
    m = wave_max_u32(m);
    const uint32_t sc = scale_code_from_bits<fmt_emax(FMT)>(m);
    if (lane == 0) scales[blk] = (uint8_t)sc;
    const bool bad = sc == 0xFFu;
    const float inv = inv_scale(sc);
    if constexpr (!SR) {
        const v6i w = pack16_fp6<FMT>(x, inv);
        v3i out;
        out[0] = bad ? 0 : w[0]; out[1] = bad ? 0 : w[1]; out[2] = bad ? 0 : w[2];
        *(v3i*)(codes + (size_t)blk * 768 + 12 * lane) = out;
    } else {
        uint32_t cd[16];
        const uint64_t q0 = (uint64_t)blk * 128 + 2 * lane;       // (1024 blk + 16 lane) / 8
        bool gen = false;
#pragma unroll
        for (int k = 0; k < 16; k++) gen |= sr_needs_general(comp(x[k >> 2], k & 3));
        const int s = (int)sc - 127;
        if (__builtin_amdgcn_ballot_w64(gen) != 0)   // wave-uniform
            sr_codes<FMT, 16, true>(cd, x, q0, s, inv, bad, k0, k1);
        else
            sr_codes<FMT, 16, false>(cd, x, q0, s, inv, bad, k0, k1);
        if constexpr (FMT == MXC_E4M3) {
            uint32_t w[4];
#pragma unroll
            for (int q = 0; q < 4; q++) w[q] = cd[4 * q] | cd[4 * q + 1] << 8 | cd[4 * q + 2] << 16 | cd[4 * q + 3] << 24;
            *(uint4*)(codes + (size_t)blk * 1024 + 16 * lane) = make_uint4(w[0], w[1], w[2], w[3]);
        } else if constexpr (fmt_bits(FMT) == 6) {
            uint32_t w[3] = {0u, 0u, 0u};
#pragma unroll
            for (int k = 0; k < 16; k++) {
                const int bit = 6 * k;
                w[bit >> 5] |= cd[k] << (bit & 31);
                if ((bit & 31) > 26) w[(bit >> 5) + 1] |= cd[k] >> (32 - (bit & 31));
            }
            v3i out;
            out[0] = (int)w[0]; out[1] = (int)w[1]; out[2] = (int)w[2];
            *(v3i*)(codes + (size_t)blk * 768 + 12 * lane) = out;
        } else {
            uint32_t w[2] = {0u, 0u};
#pragma unroll
            for (int k = 0; k < 16; k++) w[k >> 3] |= cd[k] << (4 * (k & 7));
            *(uint2*)(codes + (size_t)blk * 512 + 8 * lane) = make_uint2(w[0], w[1]);
        }
    }
}

// Optional im2col output of a CBF activation quantized one block per wave
// (Sec. IV-A: the quantized blocks are what the channel-batch-first im2col
// moves).  The wave of block (group gi, pixel (y, x), channel block cb) copies
// its codes and scale to every im2col position (output pixel, tap) whose
// source pixel is (y, x), and writes the zero blocks of the padding taps of
// output pixel (y, x) itself; with Ho <= h and Wo <= w every output pixel has
// such a wave, so every im2col block is written exactly once.  All indices are
// wave-uniform.  Layout as mxconv_im2col_cbf: [Np/32][Ho][Wo][Kh][Kw][Cp][32].
struct ColOut {
    uint8_t* codes;                // nullptr: no im2col output
    uint8_t* scales;
    int ho, wo, kh, kw, sh, sw, ph, pw;
};

// One im2col block: the wave's 16 (FP8) or 8 (FP4) contiguous code bytes per
// lane, or zeros, and the scale byte.
template <int FMT>
__device__ __forceinline__ void col_put(const ColOut& col, size_t bi, int lane, uint4 v, uint32_t sc, bool zero) {
    if constexpr (FMT == MXC_E4M3)
        store_nt(col.codes + bi * 1024 + 16 * lane, zero ? make_uint4(0u, 0u, 0u, 0u) : v);
    else
        store_nt(col.codes + bi * 512 + 8 * lane, zero ? make_uint2(0u, 0u) : make_uint2(v.x, v.y));
    if (lane == 0) col.scales[bi] = zero ? (uint8_t)0 : (uint8_t)sc;
}

template <int FMT>
__device__ __forceinline__ void col_scatter(const ColOut& col, const Geom& g, int blk, int lane,
                                            const uint32_t* wq, uint32_t sc) {
    // the quantizer leaves lane l with the codes of rows 8 q + l / 8 (q = 0..3);
    // one pass through 1 KB of LDS gives each lane 16 (FP8) or 8 (FP4)
    // consecutive bytes of the stored block, so each copy is one wide store.
    // LDS operations of a wave complete in order: waiting for the writes
    // (and keeping the compiler from moving the read above them) suffices.
    __shared__ __attribute__((aligned(16))) uint32_t stage[QT / 64][256];
    uint32_t* st = stage[threadIdx.x >> 6];
    if constexpr (FMT == MXC_E4M3) {
#pragma unroll
        for (int q = 0; q < 4; q++) st[lane + 64 * q] = wq[q];
    } else {
#pragma unroll
        for (int q = 0; q < 4; q++) ((unsigned short*)st)[lane + 64 * q] = (unsigned short)wq[q];
    }
    __asm__ volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
    uint4 v;
    if constexpr (FMT == MXC_E4M3) {
        v = ((const uint4*)st)[lane];
    } else {
        const uint2 h = ((const uint2*)st)[lane];
        v = make_uint4(h.x, h.y, 0u, 0u);
    }
    const int cb = blk % g.ncb;
    int r = blk / g.ncb;
    const int x = r % g.w;
    r /= g.w;
    const int y = r % g.h, gi = r / g.h;
    const int taps = col.kh * col.kw;
    auto block = [&](int oh, int ow, int tap) {
        return ((((size_t)gi * col.ho + oh) * col.wo + ow) * taps + tap) * g.ncb + cb;
    };
    for (int a = 0; a < col.kh; a++) {                   // output rows whose tap row a reads y
        const int t = y + col.ph - a;
        if (t < 0) break;
        if (t % col.sh) continue;
        const int oh = t / col.sh;
        if (oh >= col.ho) continue;
        for (int b = 0; b < col.kw; b++) {
            const int u = x + col.pw - b;
            if (u < 0) break;
            if (u % col.sw) continue;
            const int ow = u / col.sw;
            if (ow < col.wo) col_put<FMT>(col, block(oh, ow, a * col.kw + b), lane, v, sc, false);
        }
    }
    if (y < col.ho && x < col.wo) {                      // padding taps of output pixel (y, x)
        for (int a = 0; a < col.kh; a++) {
            const int iy = y * col.sh + a - col.ph;
            const bool rowout = iy < 0 || iy >= g.h;
            for (int b = 0; b < col.kw; b++) {
                const int ix = x * col.sw + b - col.pw;
                if (rowout || ix < 0 || ix >= g.w) col_put<FMT>(col, block(y, x, a * col.kw + b), lane, v, sc, true);
            }
        }
    }
}

template <int SRC, int DTYPE, int FMT, bool SR>
__device__ __forceinline__ void quantize_block_body(const void* __restrict__ src, const Geom& g,
                                                    uint8_t* __restrict__ codes, uint8_t* __restrict__ scales,
                                                    int blk, int lane, uint32_t k0, uint32_t k1,
                                                    const ColOut* col = nullptr) {
    if constexpr (SR || fmt_bits(FMT) == 6) {
        quantize_block16<SRC, DTYPE, FMT, SR>(src, g, codes, scales, blk, lane, k0, k1);
        return;
    }
    const int cb = blk % g.ncb, rest = blk / g.ncb;          // rest = (group, pixel) or (Cout block, tap)
    const int j = 4 * (lane & 7);                            // first sample (output channel) of the run
    float4 x[4];
    if (SRC == 0) {
#pragma unroll
        for (int q = 0; q < 4; q++) {
            const int c = cb * 32 + 8 * q + (lane >> 3);
            const bool ok = c < g.c;
            const size_t i = ((size_t)rest * g.c + (ok ? c : 0)) * 32 + j;
            if (DTYPE == MXC_F32) {
                x[q] = load_nt((const float*)src + i);
            } else {
                const uint2 b = load_nt((const unsigned short*)src + i);
                x[q] = make_float4(__uint_as_float(b.x << 16), __uint_as_float(b.x & 0xFFFF0000u),
                                   __uint_as_float(b.y << 16), __uint_as_float(b.y & 0xFFFF0000u));
            }
            if (!ok) x[q] = make_float4(0.f, 0.f, 0.f, 0.f);
        }
    } else {
        const int hw = g.h * g.w;
        const int cob = rest / hw, tap = rest % hw;
        float v[16];
#pragma unroll
        for (int k = 0; k < 16; k++) {
            const int c = cb * 32 + 8 * (k >> 2) + (lane >> 3);
            const int n = cob * 32 + j + (k & 3);
            const bool ok = c < g.c && n < g.n;
            const size_t i = ok ? ((size_t)n * g.c + c) * hw + tap : 0;
            v[k] = DTYPE == MXC_F32 ? __ldg((const float*)src + i)
                                    : __uint_as_float((uint32_t)__ldg((const unsigned short*)src + i) << 16);
            if (!ok) v[k] = 0.0f;
        }
#pragma unroll
        for (int q = 0; q < 4; q++) x[q] = make_float4(v[4 * q], v[4 * q + 1], v[4 * q + 2], v[4 * q + 3]);
    }
    uint32_t m = 0;
#pragma unroll
    for (int q = 0; q < 4; q++) {
        m = max(m, __float_as_uint(x[q].x) & 0x7FFFFFFFu);
        m = max(m, __float_as_uint(x[q].y) & 0x7FFFFFFFu);
        m = max(m, __float_as_uint(x[q].z) & 0x7FFFFFFFu);
        m = max(m, __float_as_uint(x[q].w) & 0x7FFFFFFFu);
    }
    m = wave_max_u32(m);
    const uint32_t sc = scale_code_from_bits<fmt_emax(FMT)>(m);
    if (lane == 0) scales[blk] = (uint8_t)sc;
    const float inv = inv_scale(sc);
    const bool bad = sc == 0xFFu;
    uint32_t wq[4];                                          // the lane's codes of rows 8 q + lane / 8
    if (FMT == MXC_E4M3) {
        uint32_t* d = (uint32_t*)(codes + (size_t)blk * 1024) + lane;
#pragma unroll
        for (int q = 0; q < 4; q++) {
            wq[q] = bad ? 0u : pack4_e4m3(x[q], inv);
            d[64 * q] = wq[q];
        }
    } else {
        unsigned short* d = (unsigned short*)(codes + (size_t)blk * 512) + lane;
#pragma unroll
        for (int q = 0; q < 4; q++) {
            wq[q] = bad ? 0u : pack4_e2m1(x[q], inv);
            d[64 * q] = (unsigned short)wq[q];
        }
    }
    if (SRC == 0 && col && col->codes) col_scatter<FMT>(*col, g, blk, lane, wq, sc);
}

// NCHW activations with at most NARROW_C channels (a network's input image)
// and a batch block of 32.  Their single channel block per pixel holds only
// C real rows, and in NCHW those rows are C x 32 planes apart, so a block is
// never one contiguous run.  A workgroup takes one 32-sample group and
// NARROW_P consecutive pixels: it reads the C x 32 source rows of those
// pixels as contiguous 16-byte pieces, transposes them through LDS
// ([pixel][channel][sample], rows padded by one float against bank
// conflicts), and each wave then quantizes a quarter of the pixels, four
// blocks at a time (16 lanes per block, below).  Channels C .. 31 are zero
// codes, written with 16-byte stores; with keep_pad they are not written
// (the buffer already holds them), and a block's stores shrink to its C
// real rows.
constexpr int NARROW_C = 4;
constexpr int NARROW_P = 64;

template <int DTYPE, int FMT, bool VECLOAD>
__global__ __launch_bounds__(QT) void quantize_narrow_kernel(const void* __restrict__ src, Geom g,
                                                             uint8_t* __restrict__ codes,
                                                             uint8_t* __restrict__ scales, int tiles,
                                                             int keep_pad) {
    constexpr int PS = NARROW_C * 32 + 1;                     // floats per pixel row
    __shared__ float t[NARROW_P * PS];
    const int tid = threadIdx.x;
    const int hw = g.h * g.w;
    const int grp = blockIdx.x / tiles, p0 = (blockIdx.x - grp * tiles) * NARROW_P;
    constexpr int VEC = DTYPE == MXC_F32 ? 4 : 8;            // elements per 16-byte load
    constexpr int LPR = NARROW_P / VEC;                       // lanes per source row
    constexpr int RPP = QT / LPR;                             // rows per pass
    const int rows = 32 * g.c;
    const int k = tid % LPR;
    // every pass's 16-byte load is issued before the first is used (the
    // passes are independent), then the values go to LDS
    constexpr int MAXP = 32 * NARROW_C / RPP;                 // passes for NARROW_C channels
    uint4 raw[MAXP];
#pragma unroll
    for (int q = 0; q < MAXP; q++) {
        const int r = tid / LPR + q * RPP;
        const int n = r / g.c, c = r - n * g.c;
        const int sample = grp * 32 + n;
        const int px = p0 + k * VEC;
        const size_t base = ((size_t)sample * g.c + c) * hw;
        raw[q] = make_uint4(0u, 0u, 0u, 0u);
        if (r >= rows) continue;
        if (VECLOAD && sample < g.n && px + VEC <= hw) {
            const v4i b = __builtin_nontemporal_load((const v4i*)((const uint8_t*)src + (base + px) * (DTYPE == MXC_F32 ? 4 : 2)));
            raw[q] = make_uint4((uint32_t)b[0], (uint32_t)b[1], (uint32_t)b[2], (uint32_t)b[3]);
        } else {
            float v[VEC];
#pragma unroll
            for (int e = 0; e < VEC; e++) {
                const bool ok = sample < g.n && px + e < hw;
                const size_t i = ok ? base + px + e : 0;
                const float x = DTYPE == MXC_F32 ? __ldg((const float*)src + i)
                                                 : __uint_as_float((uint32_t)__ldg((const unsigned short*)src + i) << 16);
                v[e] = ok ? x : 0.0f;
            }
            if constexpr (DTYPE == MXC_F32)
                raw[q] = make_uint4(__float_as_uint(v[0]), __float_as_uint(v[1]), __float_as_uint(v[2]), __float_as_uint(v[3]));
            else   // back to bf16 pairs (exact: the values are bf16)
                raw[q] = make_uint4(__float_as_uint(v[0]) >> 16 | (__float_as_uint(v[1]) & 0xFFFF0000u),
                                    __float_as_uint(v[2]) >> 16 | (__float_as_uint(v[3]) & 0xFFFF0000u),
                                    __float_as_uint(v[4]) >> 16 | (__float_as_uint(v[5]) & 0xFFFF0000u),
                                    __float_as_uint(v[6]) >> 16 | (__float_as_uint(v[7]) & 0xFFFF0000u));
        }
    }
#pragma unroll
    for (int q = 0; q < MAXP; q++) {
        const int r = tid / LPR + q * RPP;
        if (r >= rows) continue;
        const int n = r / g.c, c = r - n * g.c;
        const uint32_t w4[4] = {raw[q].x, raw[q].y, raw[q].z, raw[q].w};
        float v[VEC];
        if constexpr (DTYPE == MXC_F32) {
#pragma unroll
            for (int e = 0; e < 4; e++) v[e] = __uint_as_float(w4[e]);
        } else {
#pragma unroll
            for (int e = 0; e < 4; e++) {
                v[2 * e] = __uint_as_float(w4[e] << 16);
                v[2 * e + 1] = __uint_as_float(w4[e] & 0xFFFF0000u);
            }
        }
#pragma unroll
        for (int e = 0; e < VEC; e++) t[(k * VEC + e) * PS + c * 32 + n] = v[e];
    }
    __syncthreads();
    // Four pixels per pass of a wave: 16 lanes per pixel, lane (l % 16) holds
    // row (l / 4) % 4 and samples 8 (l % 4) .. +7 of its pixel's block (rows
    // 4 .. 31 are padding: NARROW_C <= 4), so the block maximum is a
    // reduction inside one 16-lane DPP row and the scale a per-lane value.
    const int lane = tid & 63, wave = tid >> 6;
    const int ps = lane >> 4, row = (lane >> 2) & 3, jj = 8 * (lane & 3);
    constexpr int RB = FMT == MXC_E4M3 ? 32 : 16;              // bytes of one code row
    constexpr int PPW = NARROW_P / (QT / 64);                 // pixels per wave
    for (int i = 0; i < PPW; i += 4) {
        const int pl = wave * PPW + i + ps, pix = p0 + pl;
        const bool live = pix < hw;
        float x[8];
#pragma unroll
        for (int e = 0; e < 8; e++) x[e] = 0.0f;
        if (row < g.c) {                                      // pixels past hw hold zeros in t
            const float* tp = t + pl * PS + row * 32 + jj;
#pragma unroll
            for (int e = 0; e < 8; e++) x[e] = tp[e];
        }
        uint32_t m = 0;
#pragma unroll
        for (int e = 0; e < 8; e++) m = max(m, __float_as_uint(x[e]) & 0x7FFFFFFFu);
        m = max(m, (uint32_t)__builtin_amdgcn_mov_dpp((int)m, 0xB1, 0xF, 0xF, false));   // quad_perm 1,0,3,2
        m = max(m, (uint32_t)__builtin_amdgcn_mov_dpp((int)m, 0x4E, 0xF, 0xF, false));   // quad_perm 2,3,0,1
        m = max(m, (uint32_t)__builtin_amdgcn_mov_dpp((int)m, 0x141, 0xF, 0xF, false));  // row_half_mirror
        m = max(m, (uint32_t)__builtin_amdgcn_mov_dpp((int)m, 0x140, 0xF, 0xF, false));  // row_mirror
        const uint32_t sc = scale_code_from_bits<fmt_emax(FMT)>(m);
        const size_t blk = (size_t)grp * hw + pix;             // one channel block per pixel
        if (!live) continue;
        if ((lane & 15) == 0) scales[blk] = (uint8_t)sc;
        const float inv = inv_scale(sc);
        const bool bad = sc == 0xFFu;
        const float4 lo = make_float4(x[0], x[1], x[2], x[3]), hi = make_float4(x[4], x[5], x[6], x[7]);
        uint8_t* const b = codes + blk * (32 * RB);
        if (!keep_pad || row < g.c) {
            if (FMT == MXC_E4M3)
                *(uint2*)(b + row * RB + jj) = bad ? make_uint2(0u, 0u) : make_uint2(pack4_e4m3(lo, inv), pack4_e4m3(hi, inv));
            else
                *(uint32_t*)(b + row * RB + jj / 2) =
                    bad ? 0u : (uint32_t)pack4_e2m1(lo, inv) | (uint32_t)pack4_e2m1(hi, inv) << 16;
        }
        if (!keep_pad) {                                      // rows 4 .. 31: +0 codes, 16 bytes a store
            constexpr int NZ = 28 * RB / 16;
            for (int q = lane & 15; q < NZ; q += 16) *(uint4*)(b + 4 * RB + 16 * q) = make_uint4(0u, 0u, 0u, 0u);
        }
    }
}

template <int DTYPE, int FMT>
int launch_qn(const void* src, const Geom& g, void* codes, uint8_t* scales, hipStream_t s, bool keep_pad) {
    const int hw = g.h * g.w;
    const int tiles = (hw + NARROW_P - 1) / NARROW_P;
    const long grid = (long)g.ng * tiles;
    if (grid > 0x7FFFFFFFL) return MXC_ERR_SHAPE;
    constexpr int VEC = DTYPE == MXC_F32 ? 4 : 8;
    if (hw % VEC == 0)
        hipLaunchKernelGGL((quantize_narrow_kernel<DTYPE, FMT, true>), dim3((unsigned)grid), dim3(QT), 0, s, src, g,
                           (uint8_t*)codes, scales, tiles, keep_pad ? 1 : 0);
    else
        hipLaunchKernelGGL((quantize_narrow_kernel<DTYPE, FMT, false>), dim3((unsigned)grid), dim3(QT), 0, s, src, g,
                           (uint8_t*)codes, scales, tiles, keep_pad ? 1 : 0);
    return hipGetLastError() == hipSuccess ? MXC_OK : MXC_ERR_HIP;
}

template <int SRC, int DTYPE, int FMT, bool SR>
__global__ __launch_bounds__(QT) void quantize_block_kernel(const void* __restrict__ src, Geom g,
                                                            uint8_t* __restrict__ codes,
                                                            uint8_t* __restrict__ scales, int nblocks,
                                                            uint32_t k0, uint32_t k1) {
    const int blk = blockIdx.x * (QT / 64) + (threadIdx.x >> 6);
    if (blk >= nblocks) return;
    quantize_block_body<SRC, DTYPE, FMT, SR>(src, g, codes, scales, blk, threadIdx.x & 63, k0, k1);
}

// Several tensors of the one-wave-per-block kind (CBF activations with
// Bn = 32, OIHW weights) in one launch: the waves of job i take blocks
// [blk0_i, blk0_i + nblocks_i).  Each tensor keeps its own source kind,
// source type and element format; the wave picks the job and the kernel
// body by a uniform branch.
struct QJob {
    const void* src;
    uint8_t* codes;
    uint8_t* scales;
    Geom g;
    int kind, dtype, fmt;          // kind 0: CBF activation, 1: OIHW weights
    int blk0, nblocks;
    ColOut col;                    // kind 0, FP8 / FP4: optional im2col output
};
constexpr int QMULTI_MAX = MXC_QMULTI_MAX;     // 24 x 136 bytes of kernel arguments
struct QMulti {
    QJob j[QMULTI_MAX];
    int count, nblocks;
};

template <int SRC>
__device__ __forceinline__ void qmulti_dispatch(const QJob& q, int blk, int lane) {
#define QM_CASE(D, F) quantize_block_body<SRC, D, F, false>(q.src, q.g, q.codes, q.scales, blk, lane, 0u, 0u, &q.col)
    if (q.dtype == MXC_F32) {
        switch (q.fmt) {
            case MXC_E4M3: QM_CASE(MXC_F32, MXC_E4M3); break;
            case MXC_E2M3: QM_CASE(MXC_F32, MXC_E2M3); break;
            case MXC_E3M2: QM_CASE(MXC_F32, MXC_E3M2); break;
            default:       QM_CASE(MXC_F32, MXC_E2M1); break;
        }
    } else {
        switch (q.fmt) {
            case MXC_E4M3: QM_CASE(MXC_BF16, MXC_E4M3); break;
            case MXC_E2M3: QM_CASE(MXC_BF16, MXC_E2M3); break;
            case MXC_E3M2: QM_CASE(MXC_BF16, MXC_E3M2); break;
            default:       QM_CASE(MXC_BF16, MXC_E2M1); break;
        }
    }
#undef QM_CASE
}

__global__ __launch_bounds__(QT) void quantize_multi_kernel(QMulti m) {
    // the wave's block index is uniform: keep it (and the job choice) scalar
    const int blk = __builtin_amdgcn_readfirstlane(blockIdx.x * (QT / 64) + (threadIdx.x >> 6));
    if (blk >= m.nblocks) return;
    // the job: its index from the start blocks, then one copy of it
    int jt = 0;
#pragma unroll
    for (int t = 1; t < QMULTI_MAX; t++)
        if (t < m.count && blk >= m.j[t].blk0) jt = t;
    const QJob q = m.j[jt];
    if (q.kind == 0) qmulti_dispatch<0>(q, blk - q.blk0, threadIdx.x & 63);
    else             qmulti_dispatch<1>(q, blk - q.blk0, threadIdx.x & 63);
}

template <int SRC, int DTYPE, int FMT, bool SR>
int launch_qb(const void* src, const Geom& g, void* codes, uint8_t* scales, hipStream_t s, uint32_t k0,
              uint32_t k1) {
    const long long nb = (long long)g.ng * g.h * g.w * g.ncb;
    if (nb > 0x7FFFFFFFLL - 4) return MXC_ERR_SHAPE;
    const int grid = (int)((nb + 3) / 4);
    hipLaunchKernelGGL((quantize_block_kernel<SRC, DTYPE, FMT, SR>), dim3(grid), dim3(QT), 0, s, src, g,
                       (uint8_t*)codes, scales, (int)nb, k0, k1);
    return hipGetLastError() == hipSuccess ? MXC_OK : MXC_ERR_HIP;
}

template <int LAYOUT, int DTYPE, int FMT, bool SR>
int launch_q(const void* src, const Geom& g, void* codes, uint8_t* scales, hipStream_t s, uint32_t k0,
             uint32_t k1) {
    const int tt = QT / g.bn;
    const int hw = g.h * g.w;
    const int pixblocks = (hw + tt - 1) / tt;
    const long nslabs = (long)g.ng * g.ncb * pixblocks;
    // 16-byte loads need runs of 4 along the contiguous dimension that never
    // straddle a row: pixels (NCHW), channels (NHWC) or samples (CBF)
    bool vec4;
    if (LAYOUT == MXC_NCHW)      vec4 = hw % 4 == 0 && tt % 4 == 0;
    else if (LAYOUT == MXC_NHWC) vec4 = g.c % 4 == 0;
    else                         vec4 = g.bn % 4 == 0;
    // NCHW: neighbouring pixel blocks share cache lines, keep a few together
    const int spw = LAYOUT == MXC_NCHW ? 2 : 1;
    if (nslabs > 0x7FFFFFFFL / spw) return MXC_ERR_SHAPE;
    const int nwg = (int)((nslabs + spw - 1) / spw);
    const int grid = (nwg + 7) / 8 * 8;     // whole rounds over the 8 XCDs
    if (vec4)
        hipLaunchKernelGGL((quantize_kernel<LAYOUT, DTYPE, FMT, 4, SR>), dim3(grid), dim3(QT), 0, s, src, g,
                           (uint8_t*)codes, scales, (int)nslabs, pixblocks, spw, k0, k1);
    else
        hipLaunchKernelGGL((quantize_kernel<LAYOUT, DTYPE, FMT, 1, SR>), dim3(grid), dim3(QT), 0, s, src, g,
                           (uint8_t*)codes, scales, (int)nslabs, pixblocks, spw, k0, k1);
    return hipGetLastError() == hipSuccess ? MXC_OK : MXC_ERR_HIP;
}

// format and rounding dispatch: F(LAUNCHER, FMT, SR) expands to one launch
#define MXC_FMT_SR_SWITCH(CALL)                                          \
    switch (fmt) {                                                       \
        case MXC_E4M3: return sr ? CALL(MXC_E4M3, true) : CALL(MXC_E4M3, false); \
        case MXC_E2M3: return sr ? CALL(MXC_E2M3, true) : CALL(MXC_E2M3, false); \
        case MXC_E3M2: return sr ? CALL(MXC_E3M2, true) : CALL(MXC_E3M2, false); \
        default:       return sr ? CALL(MXC_E2M1, true) : CALL(MXC_E2M1, false); \
    }

template <int LAYOUT, int DTYPE>
int launch_q_fmt(const void* src, const Geom& g, int fmt, bool sr, void* codes, uint8_t* scales,
                 hipStream_t s, uint32_t k0, uint32_t k1) {
#define Q_CALL(F, R) launch_q<LAYOUT, DTYPE, F, R>(src, g, codes, scales, s, k0, k1)
    MXC_FMT_SR_SWITCH(Q_CALL)
#undef Q_CALL
}

template <int SRC, int DTYPE>
int launch_qb_fmt(const void* src, const Geom& g, int fmt, bool sr, void* codes, uint8_t* scales, hipStream_t s,
                  uint32_t k0, uint32_t k1) {
#define QB_CALL(F, R) launch_qb<SRC, DTYPE, F, R>(src, g, codes, scales, s, k0, k1)
    MXC_FMT_SR_SWITCH(QB_CALL)
#undef QB_CALL
}

template <int LAYOUT>
int launch_q_dt(const void* src, int dtype, const Geom& g, int fmt, bool sr, void* codes,
                uint8_t* scales, hipStream_t s, uint32_t k0, uint32_t k1) {
    return dtype == MXC_F32 ? launch_q_fmt<LAYOUT, MXC_F32>(src, g, fmt, sr, codes, scales, s, k0, k1)
                            : launch_q_fmt<LAYOUT, MXC_BF16>(src, g, fmt, sr, codes, scales, s, k0, k1);
}

}  // namespace

int launch_quantize_multi(int count, const QuantJob* jobs, hipStream_t s) {
    QMulti m;
    int nq = 0;
    long long nb = 0;
    int deferred[QMULTI_MAX];      // jobs whose im2col runs as its own launch afterwards
    int nd = 0;
    for (int i = 0; i < count; i++) {
        const QuantJob& q = jobs[i];
        const bool block = (q.layout == MXC_CBF && q.role == MXC_ACT && q.g.bn == 32) ||
                           (q.layout == MXC_NCHW && q.role == MXC_WEIGHT);
        const long long qb = (long long)q.g.ng * q.g.h * q.g.w * q.g.ncb;
        if (!block || nq == QMULTI_MAX || nb + qb > 0x7FFFFFFFLL - 4) {
            // a tensor of another kind: its own launch
            const int rc = launch_quantize(q.src, q.dtype, q.layout, q.role, q.g, q.fmt, q.codes, q.scales, s);
            if (rc) return rc;
            if (q.col) deferred[nd++] = i;
            continue;
        }
        QJob& d = m.j[nq++];
        d.src = q.src; d.codes = (uint8_t*)q.codes; d.scales = q.scales; d.g = q.g;
        d.kind = q.role == MXC_WEIGHT ? 1 : 0; d.dtype = q.dtype; d.fmt = q.fmt;
        d.blk0 = (int)nb; d.nblocks = (int)qb;
        d.col.codes = nullptr; d.col.scales = nullptr;
        if (q.col) {
            // fused: FP8 / FP4 activation blocks, and an output no larger than the input
            if ((q.fmt == MXC_E4M3 || q.fmt == MXC_E2M1) && q.cv.ho <= q.g.h && q.cv.wo <= q.g.w) {
                d.col.codes = (uint8_t*)q.col_codes; d.col.scales = q.col_scales;
                d.col.ho = q.cv.ho; d.col.wo = q.cv.wo; d.col.kh = q.cv.kh; d.col.kw = q.cv.kw;
                d.col.sh = q.cv.sh; d.col.sw = q.cv.sw; d.col.ph = q.cv.ph; d.col.pw = q.cv.pw;
            } else {
                deferred[nd++] = i;
            }
        }
        nb += qb;
    }
    if (nq > 0) {
        m.count = nq;
        m.nblocks = (int)nb;
        for (int i = nq; i < QMULTI_MAX; i++) m.j[i] = m.j[nq - 1];
        hipLaunchKernelGGL(quantize_multi_kernel, dim3((unsigned)((nb + 3) / 4)), dim3(QT), 0, s, m);
        if (hipGetLastError() != hipSuccess) return MXC_ERR_HIP;
    }
    for (int k = 0; k < nd; k++) {
        const QuantJob& q = jobs[deferred[k]];
        const int rc = launch_im2col(q.cv, q.codes, q.scales, q.col_codes, q.col_scales, s);
        if (rc) return rc;
    }
    return MXC_OK;
}

int launch_quantize(const void* src, int dtype, int layout, int role, const Geom& g, int fmt, void* codes,
                    uint8_t* scales, hipStream_t s, const uint64_t* seed, bool keep_pad) {
    const bool sr = seed != nullptr;
    const uint32_t k0 = sr ? (uint32_t)*seed : 0u, k1 = sr ? (uint32_t)(*seed >> 32) : 0u;
    // blocks that are contiguous (CBF, Bn = 32) or a small gather (weights): one wave per block
    const int blocksrc = (layout == MXC_CBF && g.bn == 32) ? 0 : (role == MXC_WEIGHT && layout == MXC_NCHW) ? 1 : -1;
    if (blocksrc == 0)
        return dtype == MXC_F32 ? launch_qb_fmt<0, MXC_F32>(src, g, fmt, sr, codes, scales, s, k0, k1)
                                : launch_qb_fmt<0, MXC_BF16>(src, g, fmt, sr, codes, scales, s, k0, k1);
    if (blocksrc == 1)
        return dtype == MXC_F32 ? launch_qb_fmt<1, MXC_F32>(src, g, fmt, sr, codes, scales, s, k0, k1)
                                : launch_qb_fmt<1, MXC_BF16>(src, g, fmt, sr, codes, scales, s, k0, k1);
    // a few-channel NCHW activation (an input image), round to nearest
    if (layout == MXC_NCHW && role == MXC_ACT && g.bn == 32 && g.c <= NARROW_C && !sr &&
        (fmt == MXC_E4M3 || fmt == MXC_E2M1)) {
        if (dtype == MXC_F32)
            return fmt == MXC_E4M3 ? launch_qn<MXC_F32, MXC_E4M3>(src, g, codes, scales, s, keep_pad)
                                   : launch_qn<MXC_F32, MXC_E2M1>(src, g, codes, scales, s, keep_pad);
        return fmt == MXC_E4M3 ? launch_qn<MXC_BF16, MXC_E4M3>(src, g, codes, scales, s, keep_pad)
                               : launch_qn<MXC_BF16, MXC_E2M1>(src, g, codes, scales, s, keep_pad);
    }
    switch (layout) {
        case MXC_NCHW: return launch_q_dt<MXC_NCHW>(src, dtype, g, fmt, sr, codes, scales, s, k0, k1);
        case MXC_NHWC: return launch_q_dt<MXC_NHWC>(src, dtype, g, fmt, sr, codes, scales, s, k0, k1);
        default:       return launch_q_dt<MXC_CBF>(src, dtype, g, fmt, sr, codes, scales, s, k0, k1);
    }
}

}  // namespace mxc
