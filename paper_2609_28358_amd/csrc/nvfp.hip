// nvfp.hip -- the paper's own two-level format, Eqs. (4)-(6): a per-tensor
// fp32 scale T = amax / (448 * emax_val) (Eq. (4)), an FP8 E4M3 scale per
// 8x8 block B = CastE4M3(bmax / (T * emax_val)) (Eq. (5); 8 channels x 8
// samples, Sec. IV-B with B = 64) and elements Round(x / (B * T)) (Eq. (6))
// in any of the four element formats.  Every step gives the IEEE fp32
// result rounded to nearest even (divisions included), in this order, so
// that each rounding decision is the reference's.
//
// Two launches, no atomics and no memset: nvfp_amax_kernel writes one
// partial maximum of |x| per workgroup into the workspace; the quantize
// kernel re-reduces those partials in every workgroup (at most NVFP_PARTS
// words, an L2 hit), forms T, and quantizes the 8x8 blocks.
// Sources: channel-batch-first fp32 / bf16 activations with a batch block of
// 32, or OIHW weights (blocks of 8 Cin x 8 Cout at one tap).
#include "mx_internal.h"

namespace mxc {
namespace {

constexpr int NT = 256;

template <int DTYPE>
__device__ __forceinline__ float ld1(const void* src, size_t i) {
    if (DTYPE == MXC_F32) return __ldg((const float*)src + i);
    return __uint_as_float((uint32_t)__ldg((const unsigned short*)src + i) << 16);
}

// |x| as fp32 bit patterns of the 16 bytes at u (four fp32 or eight bf16)
template <int DTYPE>
__device__ __forceinline__ uint32_t absmax16(uint4 u) {
    if (DTYPE == MXC_F32)
        return max(max(u.x & 0x7FFFFFFFu, u.y & 0x7FFFFFFFu), max(u.z & 0x7FFFFFFFu, u.w & 0x7FFFFFFFu));
    const uint32_t hi = max(max(u.x & 0x7FFF0000u, u.y & 0x7FFF0000u), max(u.z & 0x7FFF0000u, u.w & 0x7FFF0000u));
    const uint32_t lo = max(max(u.x << 16, u.y << 16), max(u.z << 16, u.w << 16)) & 0x7FFF0000u;
    return max(hi, lo);
}

// The source is 16-byte aligned: whole 16-byte chunks are read as such and
// the last count % (16 / size) elements one by one.
template <int DTYPE>
__global__ __launch_bounds__(NT) void nvfp_amax_kernel(const void* __restrict__ src, size_t count,
                                                       uint32_t* __restrict__ parts) {
    __shared__ uint32_t red[NT / 64];
    uint32_t m = 0;
    const size_t stride = (size_t)gridDim.x * NT;
    constexpr int EPV = DTYPE == MXC_F32 ? 4 : 8;
    const size_t nvec = count / EPV, first = nvec * EPV;
    for (size_t i = (size_t)blockIdx.x * NT + threadIdx.x; i < nvec; i += stride)
        m = max(m, absmax16<DTYPE>(__ldg((const uint4*)src + i)));
    for (size_t i = first + (size_t)blockIdx.x * NT + threadIdx.x; i < count; i += stride)
        m = max(m, __float_as_uint(ld1<DTYPE>(src, i)) & 0x7FFFFFFFu);   // NaN patterns sort above inf
    m = wave_max_u32(m);
    if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = m;
    __syncthreads();
    if (threadIdx.x == 0) parts[blockIdx.x] = max(max(red[0], red[1]), max(red[2], red[3]));
}

// eight consecutive codes of a block row, stored at their place in the code array
template <int FMT>
__device__ __forceinline__ void store8(uint8_t* __restrict__ codes, size_t pos, const float* q) {
    if constexpr (FMT == MXC_E4M3) {
        const uint32_t a = pack4_e4m3(make_float4(q[0], q[1], q[2], q[3]), 1.0f);
        const uint32_t b = pack4_e4m3(make_float4(q[4], q[5], q[6], q[7]), 1.0f);
        *(uint2*)(codes + pos) = make_uint2(a, b);
    } else if constexpr (FMT == MXC_E2M1) {
        *(uint32_t*)(codes + pos / 2) =
            pack8_e2m1(make_float4(q[0], q[1], q[2], q[3]), make_float4(q[4], q[5], q[6], q[7]), 1.0f);
    } else {
        v16f ev, od;
#pragma unroll
        for (int i = 0; i < 16; i++) { ev[i] = 0.0f; od[i] = 0.0f; }
#pragma unroll
        for (int i = 0; i < 4; i++) { ev[i] = q[2 * i]; od[i] = q[2 * i + 1]; }
        const v6i w = cvt32_fp6<FMT>(ev, od);                    // 8 codes = the first 48 bits
        uint8_t* d = codes + pos / 4 * 3;                        // pos is a multiple of 8: 6-byte aligned
        *(uint16_t*)d = (uint16_t)w[0];
        *(uint16_t*)(d + 2) = (uint16_t)((uint32_t)w[0] >> 16);
        *(uint16_t*)(d + 4) = (uint16_t)w[1];
    }
}

template <int FMT>
constexpr float emax_val() {
    return FMT == MXC_E4M3 ? 448.0f : FMT == MXC_E2M1 ? 6.0f : FMT == MXC_E2M3 ? 7.5f : 28.0f;
}

// Eq. (4) in every workgroup from the partial maxima: T = amax / (448 emax_val),
// NaN when any element is not finite.
template <int FMT>
__device__ __forceinline__ float tensor_scale(const uint32_t* __restrict__ parts, int nparts) {
    __shared__ uint32_t red[NT / 64];
    uint32_t m = 0;
    for (int i = threadIdx.x; i < nparts; i += NT) m = max(m, parts[i]);
    m = wave_max_u32(m);
    if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = m;
    __syncthreads();
    const uint32_t amax_bits = max(max(red[0], red[1]), max(red[2], red[3]));
    return amax_bits >= 0x7F800000u ? __uint_as_float(0x7FC00000u)
                                    : __uint_as_float(amax_bits) / (448.0f * emax_val<FMT>());
}

// Eq. (5) for a block with maximum |x| bit pattern bm: the E4M3 scale code,
// and B * T in fp32 (0 when T or B is 0; the code is 0x7F for a NaN T).
template <int FMT>
__device__ __forceinline__ uint32_t block_scale(float T, uint32_t bm, float& bt) {
    bt = 0.0f;
    if (T != T) return 0x7Fu;
    if (T == 0.0f) return 0u;
    const float tm = T * emax_val<FMT>();
    const float ratio = __uint_as_float(bm) / tm;
    const uint32_t bcode = pack4_e4m3(make_float4(ratio, 0.f, 0.f, 0.f), 1.0f) & 0xFFu;
    const uint32_t e = (bcode >> 3) & 0xFu, mt = bcode & 7u;     // E4M3 value of the code (exact)
    const float B = e ? __uint_as_float(((e + 120u) << 23) | (mt << 20)) : (float)mt * 0.001953125f;
    bt = B * T;
    return bcode;
}

// Eq. (6): x / (B T) correctly rounded to fp32, as x times an fp64
// reciprocal: the fp64 product is within 2^-52 (relative) of the exact
// quotient, while a quotient of two fp32 numbers is never an fp32 rounding
// midpoint and lies at least about 2^-48 (relative) away from one, so
// rounding the product to fp32 gives the correctly rounded quotient.
// (Quotients below the fp32 normal range round to a zero code either way.)
// B T = 0 gives +0 for every element.
__device__ __forceinline__ void scale_row(const float* v, float bt, float* q) {
    const double rcp = 1.0 / (double)bt;
#pragma unroll
    for (int j = 0; j < 8; j++) q[j] = bt != 0.0f ? (float)((double)v[j] * rcp) : 0.0f;
}

// CBF activations (Bn = 32).  A unit is 16 channel rows x 32 samples of
// one pixel (two 8-row block groups, eight 8x8 blocks); lane l holds row
// l / 4 and samples 8 (l % 4) .. +7 of it, so loads and code stores are
// contiguous across the wave.  Each wave takes UPW consecutive units and
// issues all their loads before the per-tensor scale is reduced, so the
// source stream overlaps that prologue.  The block maximum is reduced over
// the eight lanes of a block (same l % 4 and l / 32): DPP rotations by 4 and
// 8 within a 16-lane row, then a swap of the two rows of a 32-lane half.
constexpr int UPW = 4;

template <int DTYPE, int FMT>
__global__ __launch_bounds__(NT) void nvfp_act_kernel(const void* __restrict__ src, Geom g,
                                                      uint8_t* __restrict__ codes, uint8_t* __restrict__ scales,
                                                      float* __restrict__ tscale, const uint32_t* __restrict__ parts,
                                                      int nparts, int units) {
    const int lane = threadIdx.x & 63, sb8 = lane & 3;
    const int u0 = (blockIdx.x * (NT / 64) + (threadIdx.x >> 6)) * UPW;    // wave-uniform
    const unsigned kpg = (unsigned)g.cp / 16;                              // units per pixel group
    constexpr int EW = DTYPE == MXC_F32 ? 2 : 1;                           // 16-byte words per block row
    uint4 raw[UPW][EW];
#pragma unroll
    for (int t = 0; t < UPW; t++) {
        const unsigned u = (unsigned)min(u0 + t, units - 1);
        const unsigned pg = u / kpg, k = u - pg * kpg;
        const int c = 16 * (int)k + (lane >> 2);
        const size_t at = ((size_t)pg * g.c + (c < g.c ? c : 0)) * 32 + 8 * sb8;
        const uint4* p = DTYPE == MXC_F32 ? (const uint4*)((const float*)src + at)
                                          : (const uint4*)((const unsigned short*)src + at);
#pragma unroll
        for (int e = 0; e < EW; e++) raw[t][e] = __ldg(p + e);
    }
    const float T = tensor_scale<FMT>(parts, nparts);
    if (blockIdx.x == 0 && threadIdx.x == 0) *tscale = T;
#pragma unroll
    for (int t = 0; t < UPW; t++) {
        if (u0 + t >= units) break;                                        // wave-uniform
        const unsigned u = (unsigned)(u0 + t);
        const unsigned pg = u / kpg, k = u - pg * kpg;
        const int c = 16 * (int)k + (lane >> 2);
        float v[8];
        if (DTYPE == MXC_F32) {
            const uint32_t w[8] = {raw[t][0].x, raw[t][0].y, raw[t][0].z, raw[t][0].w,
                                   raw[t][EW - 1].x, raw[t][EW - 1].y, raw[t][EW - 1].z, raw[t][EW - 1].w};
#pragma unroll
            for (int j = 0; j < 8; j++) v[j] = __uint_as_float(w[j]);
        } else {
            const uint32_t w[4] = {raw[t][0].x, raw[t][0].y, raw[t][0].z, raw[t][0].w};
#pragma unroll
            for (int j = 0; j < 4; j++) {
                v[2 * j] = __uint_as_float(w[j] << 16);
                v[2 * j + 1] = __uint_as_float(w[j] & 0xFFFF0000u);
            }
        }
        uint32_t bm = 0;
#pragma unroll
        for (int j = 0; j < 8; j++) {
            if (c >= g.c) v[j] = 0.0f;
            bm = max(bm, __float_as_uint(v[j]) & 0x7FFFFFFFu);
        }
        bm = max(bm, (uint32_t)__builtin_amdgcn_mov_dpp((int)bm, 0x124, 0xF, 0xF, false));   // row_ror:4
        bm = max(bm, (uint32_t)__builtin_amdgcn_mov_dpp((int)bm, 0x128, 0xF, 0xF, false));   // row_ror:8
        bm = max(bm, (uint32_t)__shfl_xor((int)bm, 16));
        float bt;
        const uint32_t bcode = block_scale<FMT>(T, bm, bt);
        if (((lane >> 2) & 7) == 0)
            scales[((size_t)pg * (g.cp / 8) + 2 * k + (lane >> 5)) * 4 + sb8] = (uint8_t)bcode;
        float q[8];
        scale_row(v, bt, q);
        store8<FMT>(codes, ((size_t)pg * g.cp + c) * 32 + 8 * sb8, q);
    }
}

// OIHW weights: one thread per 8x8 block (8 Cin x 8 Cout at one tap).
template <int DTYPE, int FMT>
__global__ __launch_bounds__(NT) void nvfp_weight_kernel(const void* __restrict__ src, Geom g,
                                                         uint8_t* __restrict__ codes, uint8_t* __restrict__ scales,
                                                         float* __restrict__ tscale, const uint32_t* __restrict__ parts,
                                                         int nparts, long long nblocks) {
    const float T = tensor_scale<FMT>(parts, nparts);
    if (blockIdx.x == 0 && threadIdx.x == 0) *tscale = T;
    const long long b = (long long)blockIdx.x * NT + threadIdx.x;
    if (b >= nblocks) return;
    // block b = ((32-Cout block, tap) * (Cp / 8) + cb8) * 4 + sb8
    const int sb8 = (int)(b & 3);
    const long long r = b >> 2;
    const int cb8 = (int)(r % (g.cp / 8));
    const long long pg = r / (g.cp / 8);
    const int hw = g.h * g.w;
    const long long cob = pg / hw;
    const int tap = (int)(pg % hw);
    float v[8][8];
    uint32_t bm = 0;
#pragma unroll
    for (int i = 0; i < 8; i++) {
        const int c = cb8 * 8 + i;
#pragma unroll
        for (int j = 0; j < 8; j++) {
            const long long n = cob * 32 + sb8 * 8 + j;
            const bool ok = c < g.c && n < g.n;
            v[i][j] = ok ? ld1<DTYPE>(src, ((size_t)n * g.c + c) * hw + tap) : 0.0f;
            bm = max(bm, __float_as_uint(v[i][j]) & 0x7FFFFFFFu);
        }
    }
    float bt;
    scales[b] = (uint8_t)block_scale<FMT>(T, bm, bt);
#pragma unroll
    for (int i = 0; i < 8; i++) {
        float q[8];
        scale_row(v[i], bt, q);
        store8<FMT>(codes, ((size_t)pg * g.cp + cb8 * 8 + i) * 32 + 8 * sb8, q);
    }
}

template <int SRC, int DTYPE, int FMT>
int launch_nq(const void* src, const Geom& g, void* codes, uint8_t* scales, float* tscale, uint32_t* parts,
              hipStream_t s) {
    const size_t count = (size_t)g.n * g.c * g.h * g.w;
    const int nparts = (int)min((size_t)NVFP_PARTS, (count + NT * 32 - 1) / (NT * 32));
    hipLaunchKernelGGL((nvfp_amax_kernel<DTYPE>), dim3(nparts), dim3(NT), 0, s, src, count, parts);
    if (SRC == 0) {
        const long long units = (long long)g.ng * g.h * g.w * (g.cp / 16);
        if (units > 0x7FFFFFFFLL - (long long)NT / 64 * UPW) return MXC_ERR_SHAPE;
        const long long per_wg = NT / 64 * UPW;
        hipLaunchKernelGGL((nvfp_act_kernel<DTYPE, FMT>), dim3((unsigned)((units + per_wg - 1) / per_wg)), dim3(NT), 0,
                           s, src, g, (uint8_t*)codes, scales, tscale, parts, nparts, (int)units);
    } else {
        const long long nblocks = (long long)g.ng * g.h * g.w * (g.cp / 8) * 4;
        const long long grid = (nblocks + NT - 1) / NT;
        if (grid > 0x7FFFFFFFLL) return MXC_ERR_SHAPE;
        hipLaunchKernelGGL((nvfp_weight_kernel<DTYPE, FMT>), dim3((unsigned)grid), dim3(NT), 0, s, src, g,
                           (uint8_t*)codes, scales, tscale, parts, nparts, nblocks);
    }
    return hipGetLastError() == hipSuccess ? MXC_OK : MXC_ERR_HIP;
}

template <int SRC, int DTYPE>
int launch_nq_fmt(const void* src, const Geom& g, int fmt, void* codes, uint8_t* scales, float* tscale,
                  uint32_t* parts, hipStream_t s) {
    switch (fmt) {
        case MXC_E4M3: return launch_nq<SRC, DTYPE, MXC_E4M3>(src, g, codes, scales, tscale, parts, s);
        case MXC_E2M3: return launch_nq<SRC, DTYPE, MXC_E2M3>(src, g, codes, scales, tscale, parts, s);
        case MXC_E3M2: return launch_nq<SRC, DTYPE, MXC_E3M2>(src, g, codes, scales, tscale, parts, s);
        default:       return launch_nq<SRC, DTYPE, MXC_E2M1>(src, g, codes, scales, tscale, parts, s);
    }
}

}  // namespace

int launch_nvfp_quantize(const void* src, int dtype, int layout, int role, const Geom& g, int fmt, void* codes,
                         uint8_t* scales, float* tscale, void* ws, hipStream_t s) {
    uint32_t* parts = (uint32_t*)ws;
    if (layout == MXC_CBF && role == MXC_ACT && g.bn == 32)
        return dtype == MXC_F32 ? launch_nq_fmt<0, MXC_F32>(src, g, fmt, codes, scales, tscale, parts, s)
                                : launch_nq_fmt<0, MXC_BF16>(src, g, fmt, codes, scales, tscale, parts, s);
    if (layout == MXC_NCHW && role == MXC_WEIGHT)
        return dtype == MXC_F32 ? launch_nq_fmt<1, MXC_F32>(src, g, fmt, codes, scales, tscale, parts, s)
                                : launch_nq_fmt<1, MXC_BF16>(src, g, fmt, codes, scales, tscale, parts, s);
    return MXC_ERR_SHAPE;
}

}  // namespace mxc
