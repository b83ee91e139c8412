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
//   3. scale code from the exponent bits, elements encoded with integer
//      round-to-nearest-even, codes stored as 16-byte vectors.
// Traffic: 4 (or 2) bytes read and 1 (or 1/2) byte written per element, plus
// one scale byte per block; HBM-bound.
#include "mx_internal.h"

namespace mxc {
namespace {

constexpr int QT = 256;            // threads per workgroup
constexpr int SLABS_PER_WG = 4;    // consecutive slabs per workgroup

__device__ __forceinline__ int swz(int u) { return ((u >> 5) ^ (u >> 1)) & 7; }

template <int DTYPE>
__device__ __forceinline__ float load_elem(const void* src, size_t i) {
    if (DTYPE == MXC_F32) return __ldg((const float*)src + i);
    uint32_t b = (uint32_t)__ldg((const unsigned short*)src + i);
    return __uint_as_float(b << 16);
}

template <int LAYOUT, int DTYPE, int FMT>
__global__ __launch_bounds__(QT) void quantize_kernel(const void* __restrict__ src, Geom g,
                                                      uint8_t* __restrict__ codes,
                                                      uint8_t* __restrict__ scales,
                                                      int nslabs, int pixblocks) {
    __shared__ __attribute__((aligned(16))) float slab[QT * 32];
    const int tid = threadIdx.x;
    const int bn = g.bn, tt = QT / bn;
    const int hw = g.h * g.w;

    // XCD-aware order: workgroups are dealt round-robin to the 8 XCDs, so give
    // each XCD a contiguous range of slabs (neighbouring pixel blocks share
    // cache lines in NCHW).
    const int nwg = gridDim.x;
    const int per_xcd = (nwg + 7) / 8;
    const int wg = (blockIdx.x % 8) * per_xcd + blockIdx.x / 8;
    if (wg >= nwg) return;

    for (int it = 0; it < SLABS_PER_WG; it++) {
        const int slab_id = wg * SLABS_PER_WG + it;
        if (slab_id >= nslabs) return;
        const int pb = slab_id % pixblocks;
        const int rest = slab_id / pixblocks;
        const int cb = rest % g.ncb;
        const int ng = rest / g.ncb;
        const int p0 = pb * tt;

        // ---- 1. load into the slab (code order, swizzled chunks)
#pragma unroll 8
        for (int r = 0; r < 32; r++) {
            const int e = tid + QT * r;
            int pl, cl, j;
            if (LAYOUT == MXC_NCHW) {
                pl = e % tt; const int r1 = e / tt; cl = r1 & 31; j = r1 >> 5;
            } else if (LAYOUT == MXC_NHWC) {
                cl = e & 31; const int r1 = e >> 5; pl = r1 % tt; j = r1 / tt;
            } else {
                j = e % bn; const int r1 = e / bn; cl = r1 & 31; pl = r1 >> 5;
            }
            const int pix = p0 + pl, c = cb * 32 + cl, n = ng * bn + j;
            float v = 0.0f;
            if (pix < hw && c < g.c && n < g.n) {
                size_t gi;
                if (LAYOUT == MXC_NCHW)      gi = ((size_t)n * g.c + c) * hw + pix;
                else if (LAYOUT == MXC_NHWC) gi = ((size_t)n * hw + pix) * g.c + c;
                else                         gi = (((size_t)ng * hw + pix) * g.c + c) * bn + j;
                v = load_elem<DTYPE>(src, gi);
            }
            const int ci = (pl * 32 + cl) * bn + j;      // canonical index in the slab
            const int u = ci >> 5, k = ci & 31;
            slab[u * 32 + ((((k >> 2) ^ swz(u))) << 2) + (k & 3)] = v;
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
        constexpr int EMAX = FMT == MXC_E4M3 ? 8 : 2;
        const uint32_t sc = scale_code_from_bits<EMAX>(m);
        const size_t blk = ((size_t)ng * hw + pix) * g.ncb + cb;
        if (part == 0) scales[blk] = (uint8_t)sc;
        const float inv = inv_scale(sc);
        const bool bad = sc == 0xFFu;
        const size_t e0 = (((size_t)ng * hw + pix) * g.cp + cb * 32) * bn + part * 32;

        // ---- 3. encode and store
        if (FMT == MXC_E4M3) {
            uint32_t w[8];
#pragma unroll
            for (int q = 0; q < 8; q++) {
                uint32_t c0 = enc_e4m3(x[q].x * inv), c1 = enc_e4m3(x[q].y * inv);
                uint32_t c2 = enc_e4m3(x[q].z * inv), c3 = enc_e4m3(x[q].w * inv);
                w[q] = bad ? 0u : (c0 | (c1 << 8) | (c2 << 16) | (c3 << 24));
            }
            uint4* dst = (uint4*)(codes + e0);
            dst[0] = make_uint4(w[0], w[1], w[2], w[3]);
            dst[1] = make_uint4(w[4], w[5], w[6], w[7]);
        } else {
            uint32_t w[4];
#pragma unroll
            for (int q = 0; q < 4; q++) {
                const float4 a = x[2 * q], b = x[2 * q + 1];
                uint32_t t = enc_e2m1(a.x * inv) | (enc_e2m1(a.y * inv) << 4) |
                             (enc_e2m1(a.z * inv) << 8) | (enc_e2m1(a.w * inv) << 12) |
                             (enc_e2m1(b.x * inv) << 16) | (enc_e2m1(b.y * inv) << 20) |
                             (enc_e2m1(b.z * inv) << 24) | (enc_e2m1(b.w * inv) << 28);
                w[q] = bad ? 0u : t;
            }
            *(uint4*)(codes + e0 / 2) = make_uint4(w[0], w[1], w[2], w[3]);
        }
    }
}

template <int LAYOUT, int DTYPE, int FMT>
int launch_q(const void* src, const Geom& g, void* codes, uint8_t* scales, hipStream_t s) {
    const int tt = QT / g.bn;
    const int pixblocks = (g.h * g.w + tt - 1) / tt;
    const long nslabs = (long)g.ng * g.ncb * pixblocks;
    if (nslabs > 0x7FFFFFFFL / SLABS_PER_WG) return MXC_ERR_SHAPE;
    const int nwg = (int)((nslabs + SLABS_PER_WG - 1) / SLABS_PER_WG);
    const int grid = (nwg + 7) / 8 * 8;     // whole rounds over the 8 XCDs
    hipLaunchKernelGGL((quantize_kernel<LAYOUT, DTYPE, FMT>), dim3(grid), dim3(QT), 0, s, src, g,
                       (uint8_t*)codes, scales, (int)nslabs, pixblocks);
    return hipGetLastError() == hipSuccess ? MXC_OK : MXC_ERR_HIP;
}

template <int LAYOUT, int DTYPE>
int launch_q_fmt(const void* src, const Geom& g, int fmt, void* codes, uint8_t* scales,
                 hipStream_t s) {
    return fmt == MXC_E4M3 ? launch_q<LAYOUT, DTYPE, MXC_E4M3>(src, g, codes, scales, s)
                           : launch_q<LAYOUT, DTYPE, MXC_E2M1>(src, g, codes, scales, s);
}

template <int LAYOUT>
int launch_q_dt(const void* src, int dtype, const Geom& g, int fmt, void* codes,
                uint8_t* scales, hipStream_t s) {
    return dtype == MXC_F32 ? launch_q_fmt<LAYOUT, MXC_F32>(src, g, fmt, codes, scales, s)
                            : launch_q_fmt<LAYOUT, MXC_BF16>(src, g, fmt, codes, scales, s);
}

}  // namespace

int launch_quantize(const void* src, int dtype, int layout, const Geom& g, int fmt, void* codes,
                    uint8_t* scales, hipStream_t s) {
    switch (layout) {
        case MXC_NCHW: return launch_q_dt<MXC_NCHW>(src, dtype, g, fmt, codes, scales, s);
        case MXC_NHWC: return launch_q_dt<MXC_NHWC>(src, dtype, g, fmt, codes, scales, s);
        default:       return launch_q_dt<MXC_CBF>(src, dtype, g, fmt, codes, scales, s);
    }
}

}  // namespace mxc
