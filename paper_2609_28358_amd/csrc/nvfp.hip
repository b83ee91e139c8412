// nvfp.hip -- the paper's own two-level format, Eqs. (4)-(6): a per-tensor
// fp32 scale T = amax / (448 * emax_val) (Eq. (4)), an FP8 E4M3 scale per
// 8x8 block B = CastE4M3(bmax / (T * emax_val)) (Eq. (5); 8 channels x 8
// samples, Sec. IV-B with B = 64) and elements Round(x / (B * T)) (Eq. (6))
// in any of the four element formats.  Every step is one IEEE fp32
// operation rounded to nearest even (divisions included), in this order, so
// that each rounding decision is the reference's.
//
// Two launches, no atomics and no memset: nvfp_amax_kernel writes one
// partial maximum of |x| per workgroup into the workspace; nvfp_quant_kernel
// re-reduces those partials in every workgroup (at most NVFP_PARTS words, an
// L2 hit), forms T, and quantizes one 8x8 block per thread.
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

template <int DTYPE>
__global__ __launch_bounds__(NT) void nvfp_amax_kernel(const void* __restrict__ src, size_t count,
                                                       uint32_t* __restrict__ parts) {
    __shared__ uint32_t red[NT / 64];
    uint32_t m = 0;
    const size_t stride = (size_t)gridDim.x * NT;
    for (size_t i = (size_t)blockIdx.x * NT + threadIdx.x; i < count; i += stride)
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

// SRC 0: CBF activation (Bn = 32); SRC 1: OIHW weights.  One thread per 8x8 block.
template <int SRC, int DTYPE, int FMT>
__global__ __launch_bounds__(NT) void nvfp_quant_kernel(const void* __restrict__ src, Geom g,
                                                        uint8_t* __restrict__ codes, uint8_t* __restrict__ scales,
                                                        float* __restrict__ tscale, const uint32_t* __restrict__ parts,
                                                        int nparts, long long nblocks) {
    __shared__ uint32_t red[NT / 64];
    uint32_t m = 0;
    for (int i = threadIdx.x; i < nparts; i += NT) m = max(m, parts[i]);
    m = wave_max_u32(m);
    if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = m;
    __syncthreads();
    const uint32_t amax_bits = max(max(red[0], red[1]), max(red[2], red[3]));
    const bool nonfinite = amax_bits >= 0x7F800000u;
    constexpr float EMAXV = FMT == MXC_E4M3 ? 448.0f : FMT == MXC_E2M1 ? 6.0f : FMT == MXC_E2M3 ? 7.5f : 28.0f;
    const float T = nonfinite ? __uint_as_float(0x7FC00000u) : __uint_as_float(amax_bits) / (448.0f * EMAXV);
    if (blockIdx.x == 0 && threadIdx.x == 0) *tscale = T;
    const long long b = (long long)blockIdx.x * NT + threadIdx.x;
    if (b >= nblocks) return;
    // block b = ((pixel group) * (Cp / 8) + cb8) * 4 + sb8; the pixel group is
    // (batch group, h, w) for activations, (32-Cout block, tap) for weights
    const int sb8 = (int)(b & 3);
    const long long r = b >> 2;
    const int cb8 = (int)(r % (g.cp / 8));
    const long long pg = r / (g.cp / 8);
    const int hw = g.h * g.w;
    float v[8][8];
    uint32_t bm = 0;
#pragma unroll
    for (int i = 0; i < 8; i++) {
        const int c = cb8 * 8 + i;
        if (SRC == 0) {
            const bool ok = c < g.c;
            const size_t base = ((size_t)pg * g.c + (ok ? c : 0)) * 32 + 8 * sb8;
            float4 a, bb;
            if (DTYPE == MXC_F32) {
                a = __ldg((const float4*)((const float*)src + base));
                bb = __ldg((const float4*)((const float*)src + base + 4));
            } else {
                const uint4 u = __ldg((const uint4*)((const unsigned short*)src + base));
                a = make_float4(__uint_as_float(u.x << 16), __uint_as_float(u.x & 0xFFFF0000u),
                                __uint_as_float(u.y << 16), __uint_as_float(u.y & 0xFFFF0000u));
                bb = make_float4(__uint_as_float(u.z << 16), __uint_as_float(u.z & 0xFFFF0000u),
                                 __uint_as_float(u.w << 16), __uint_as_float(u.w & 0xFFFF0000u));
            }
            v[i][0] = ok ? a.x : 0.f; v[i][1] = ok ? a.y : 0.f; v[i][2] = ok ? a.z : 0.f; v[i][3] = ok ? a.w : 0.f;
            v[i][4] = ok ? bb.x : 0.f; v[i][5] = ok ? bb.y : 0.f; v[i][6] = ok ? bb.z : 0.f; v[i][7] = ok ? bb.w : 0.f;
        } else {
            const long long cob = pg / hw;
            const int tap = (int)(pg % hw);
#pragma unroll
            for (int j = 0; j < 8; j++) {
                const long long n = cob * 32 + sb8 * 8 + j;
                const bool ok = c < g.c && n < g.n;
                v[i][j] = ok ? ld1<DTYPE>(src, ((size_t)n * g.c + c) * hw + tap) : 0.0f;
            }
        }
#pragma unroll
        for (int j = 0; j < 8; j++) bm = max(bm, __float_as_uint(v[i][j]) & 0x7FFFFFFFu);
    }
    // Eq. (5): B = CastE4M3(bmax / (T * emax_val)); Eq. (6): x / (B * T)
    uint32_t bcode = 0;
    float bt = 0.0f;
    if (nonfinite) {
        bcode = 0x7Fu;
    } else if (T != 0.0f) {
        const float tm = T * EMAXV;
        const float ratio = __uint_as_float(bm) / tm;
        bcode = pack4_e4m3(make_float4(ratio, 0.f, 0.f, 0.f), 1.0f) & 0xFFu;
        const uint32_t e = (bcode >> 3) & 0xFu, mt = bcode & 7u;     // E4M3 value of the code (exact)
        const float B = e ? __uint_as_float(((e + 120u) << 23) | (mt << 20)) : (float)mt * 0.001953125f;
        bt = B * T;
    }
    scales[b] = (uint8_t)bcode;
#pragma unroll
    for (int i = 0; i < 8; i++) {
        float q[8];
#pragma unroll
        for (int j = 0; j < 8; j++) q[j] = bt != 0.0f ? v[i][j] / bt : 0.0f;
        const size_t pos = ((size_t)pg * g.cp + cb8 * 8 + i) * 32 + 8 * sb8;   // code position of (row, first sample)
        store8<FMT>(codes, pos, q);
    }
}

template <int SRC, int DTYPE, int FMT>
int launch_nq(const void* src, const Geom& g, void* codes, uint8_t* scales, float* tscale, uint32_t* parts,
              hipStream_t s) {
    const size_t count = (size_t)g.n * g.c * g.h * g.w;
    const int nparts = (int)min((size_t)NVFP_PARTS, (count + NT * 16 - 1) / (NT * 16));
    hipLaunchKernelGGL((nvfp_amax_kernel<DTYPE>), dim3(nparts), dim3(NT), 0, s, src, count, parts);
    const long long nblocks = (long long)g.ng * g.h * g.w * (g.cp / 8) * 4;
    const long long grid = (nblocks + NT - 1) / NT;
    if (grid > 0x7FFFFFFFLL) return MXC_ERR_SHAPE;
    hipLaunchKernelGGL((nvfp_quant_kernel<SRC, DTYPE, FMT>), dim3((unsigned)grid), dim3(NT), 0, s, src, g,
                       (uint8_t*)codes, scales, tscale, parts, nparts, nblocks);
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
