// netops.hip -- the two operations a whole network's training step needs
// between its convolutions, written so that every tensor is still quantized
// exactly once (Sec. IV-C).
//
// Concatenation and 2x upsampling on MX codes.  A quantization block is 32
// channels x Bn samples at one pixel (Sec. IV-B's square block in the
// channel-batch-first layout of Sec. IV-A), so concatenating activations
// along channels (whole blocks) or repeating each pixel 2x2 (nearest-
// neighbour upsampling) only moves whole blocks: codes and scales are copied,
// never requantized.  One thread per 16-byte destination chunk, as in a
// streaming copy; threads with chunk index below the block count of a pixel
// also copy that pixel's scale bytes.
//
// The gradient of a tensor a = fn(z) that several consumers read.  Its
// gradient is the sum of what each consumer's input gradient hands back --
// fp32 slices of wider tensors (the consumer was a concatenation) or the
// 2x2 pixel sums of a tensor twice as large (the consumer was an upsampling)
// -- times fn'(z), and it is quantized once, as the G_Y operand of the layer
// that produced a.  One wave per 32-channel x 32-sample block, the lane
// layout of the one-block-per-wave quantizer: lane l holds channels
// 8 q + l / 8 (q = 0..3) and samples 4 (l % 8) .. +3, so every load of a
// term is a 16-byte vector and the wave's codes are one contiguous run.
#include "mx_internal.h"

namespace mxc {
namespace {

struct ConcatArgs {
    const uint8_t* codes[MXC_CONCAT_MAX];
    const uint8_t* scales[MXC_CONCAT_MAX];
    int ncb[MXC_CONCAT_MAX];          // channel blocks of each part
    int off[MXC_CONCAT_MAX + 1];      // first destination block of each part, off[nparts] = total
    int up[MXC_CONCAT_MAX];
    int nparts;
    int h, w;                         // destination pixel grid
    int bb16;                         // 16-byte chunks per block
};

__global__ __launch_bounds__(256) void concat_kernel(ConcatArgs a, uint8_t* __restrict__ dst,
                                                     uint8_t* __restrict__ sdst, long long nchunks) {
    const long long i = (long long)blockIdx.x * 256 + threadIdx.x;
    if (i >= nchunks) return;
    const int run16 = a.off[a.nparts] * a.bb16;           // chunks of one destination pixel
    const long long pix = i / run16;
    const int within = (int)(i - pix * run16);
    const int blk = within / a.bb16, in = within - blk * a.bb16;
    int k = 0;
#pragma unroll
    for (int t = 1; t < MXC_CONCAT_MAX; t++)
        if (t < a.nparts && blk >= a.off[t]) k = t;
    const int x = (int)(pix % a.w);
    const long long gy = pix / a.w;                        // (group, row)
    const int y = (int)(gy % a.h);
    const long long g = gy / a.h;
    long long spix;
    if (a.up[k]) spix = (g * (a.h >> 1) + (y >> 1)) * (a.w >> 1) + (x >> 1);
    else spix = pix;
    const int sb = blk - a.off[k];
    const uint4* src = (const uint4*)(a.codes[k] + ((size_t)spix * a.ncb[k] + sb) * 16 * a.bb16) + in;
    store_nt(dst + ((size_t)pix * run16 + within) * 16, __ldg(src));
    if (within < a.off[a.nparts]) {                        // this pixel's scale byte of block `within`
        int kk = 0;
#pragma unroll
        for (int t = 1; t < MXC_CONCAT_MAX; t++)
            if (t < a.nparts && within >= a.off[t]) kk = t;
        const long long sp = a.up[kk] ? (g * (a.h >> 1) + (y >> 1)) * (a.w >> 1) + (x >> 1) : pix;
        sdst[(size_t)pix * a.off[a.nparts] + within] = a.scales[kk][(size_t)sp * a.ncb[kk] + within - a.off[kk]];
    }
}

struct SumArgs {
    const void* src[MXC_TERMS_MAX];   // fp32, or bf16 (BF)
    int c_src[MXC_TERMS_MAX];
    int c_off[MXC_TERMS_MAX];
    int down[MXC_TERMS_MAX];
    int nterms;
    int c, h, w, ncb;                 // destination (n, c, h, w), channel blocks
    int fn;
    const void* z;                    // CBF [n/32][h][w][c][32] (fn != NONE), fp32 or bf16 (BF)
    float* vals;                      // optional: the values quantized
    int sr;                           // codes by stochastic rounding, generator key (k0, k1)
    uint32_t k0, k1;
};

// Four consecutive elements at index i of an fp32 or (BF) bf16 tensor.
template <bool BF>
__device__ __forceinline__ float4 load4(const void* s, size_t i) {
    if constexpr (BF) return bf16_unpack4(load_nt((const unsigned short*)s + i));
    else              return load_nt((const float*)s + i);
}

// Term t at destination pixel (g, y, x), channel ch, samples j .. j+3.
template <bool BF>
__device__ __forceinline__ float4 term4(const SumArgs& a, int t, long long g, int y, int x, int ch, int j) {
    const void* s = a.src[t];
    const int cs = a.c_src[t];
    const int col = a.c_off[t] + ch;
    if (!a.down[t]) {
        const size_t i = ((((size_t)g * a.h + y) * a.w + x) * cs + col) * 32 + j;
        return load4<BF>(s, i);
    }
    const int hs = 2 * a.h, ws = 2 * a.w;
    const size_t r0 = ((size_t)g * hs + 2 * y) * ws + 2 * x, r1 = r0 + ws;
    const float4 p = load4<BF>(s, (r0 * cs + col) * 32 + j);
    const float4 q = load4<BF>(s, ((r0 + 1) * cs + col) * 32 + j);
    const float4 u = load4<BF>(s, (r1 * cs + col) * 32 + j);
    const float4 v = load4<BF>(s, ((r1 + 1) * cs + col) * 32 + j);
    return make_float4((p.x + q.x) + (u.x + v.x), (p.y + q.y) + (u.y + v.y), (p.z + q.z) + (u.z + v.z),
                       (p.w + q.w) + (u.w + v.w));
}

template <int FMT, bool BF>
__global__ __launch_bounds__(256) void quantize_sum_kernel(SumArgs a, uint8_t* __restrict__ codes,
                                                           uint8_t* __restrict__ scales, long long nblocks) {
    const long long blk = (long long)blockIdx.x * 4 + (threadIdx.x >> 6);
    if (blk >= nblocks) return;
    const int lane = threadIdx.x & 63;
    const int cb = (int)(blk % a.ncb);
    const long long pix = blk / a.ncb;                     // (group, y, x)
    const int x = (int)(pix % a.w);
    const long long gy = pix / a.w;
    const int y = (int)(gy % a.h);
    const long long g = gy / a.h;
    const int j = 4 * (lane & 7);
    float4 v[4];
#pragma unroll
    for (int q = 0; q < 4; q++) {
        const int ch = cb * 32 + 8 * q + (lane >> 3);
        float4 s = make_float4(0.f, 0.f, 0.f, 0.f);
        if (ch < a.c) {
            s = term4<BF>(a, 0, g, y, x, ch, j);
            for (int t = 1; t < a.nterms; t++) {
                const float4 u = term4<BF>(a, t, g, y, x, ch, j);
                s.x += u.x; s.y += u.y; s.z += u.z; s.w += u.w;
            }
            if (a.fn != MXC_FN_NONE) {
                const float4 zz = load4<BF>(a.z, ((size_t)pix * a.c + ch) * 32 + j);
                with_fn(a.fn, [&](auto t) {
                    constexpr int F = decltype(t)::fn;
                    s.x *= fn_grad_c<F>(zz.x);
                    s.y *= fn_grad_c<F>(zz.y);
                    s.z *= fn_grad_c<F>(zz.z);
                    s.w *= fn_grad_c<F>(zz.w);
                });
            }
            if (a.vals) store_nt(a.vals + ((size_t)pix * a.c + ch) * 32 + j, s);
        }
        v[q] = s;
    }
    uint32_t m = 0;
#pragma unroll
    for (int q = 0; q < 4; q++) {
        m = max(m, __float_as_uint(v[q].x) & 0x7FFFFFFFu);
        m = max(m, __float_as_uint(v[q].y) & 0x7FFFFFFFu);
        m = max(m, __float_as_uint(v[q].z) & 0x7FFFFFFFu);
        m = max(m, __float_as_uint(v[q].w) & 0x7FFFFFFFu);
    }
    m = wave_max_u32(m);
    const uint32_t sc = scale_code_from_bits<fmt_emax(FMT)>(m);
    if (lane == 0) scales[blk] = (uint8_t)sc;
    const float inv = inv_scale(sc);
    const bool bad = sc == 0xFFu;
    uint32_t run[4];   // the codes of v[q]: channel row 8 q + lane / 8, samples j .. j + 3
    if (a.sr) {        // stochastic rounding, keyed by code position blk 1024 + 32 row + sample
        const int s = (int)sc - 127;
#pragma unroll
        for (int q = 0; q < 4; q++) {
            uint32_t cd[4];
            sr_codes4<FMT>(v[q], (uint64_t)blk * 1024 + (8 * q + (lane >> 3)) * 32 + j, s, inv, a.k0, a.k1, cd);
            run[q] = FMT == MXC_E4M3 ? cd[0] | cd[1] << 8 | cd[2] << 16 | cd[3] << 24
                                     : cd[0] | cd[1] << 4 | cd[2] << 8 | cd[3] << 12;
        }
    } else {
#pragma unroll
        for (int q = 0; q < 4; q++)
            run[q] = FMT == MXC_E4M3 ? pack4_e4m3(v[q], inv) : (uint32_t)pack4_e2m1(v[q], inv);
    }
    if constexpr (FMT == MXC_E4M3) {
        uint32_t* d = (uint32_t*)(codes + (size_t)blk * 1024) + lane;
#pragma unroll
        for (int q = 0; q < 4; q++) d[64 * q] = bad ? 0u : run[q];
    } else {
        unsigned short* d = (unsigned short*)(codes + (size_t)blk * 512) + lane;
#pragma unroll
        for (int q = 0; q < 4; q++) d[64 * q] = bad ? (unsigned short)0 : (unsigned short)run[q];
    }
}

// bf16 terms and z: the same sums with 16-byte loads.  Lane l takes channels
// 16 hh + l / 4 (hh = 0, 1) of the block and samples 8 (l % 4) .. + 7 (eight
// bf16 = 16 bytes per load, half the load instructions of the layout above),
// and writes their codes as one 4-byte (FP4) or 8-byte (FP8) piece: each
// store instruction of the wave covers 16 whole channel rows.
__device__ __forceinline__ void bf16x8(uint4 u, float* f) {
    const float4 a = bf16_unpack4(make_uint2(u.x, u.y)), b = bf16_unpack4(make_uint2(u.z, u.w));
    f[0] = a.x; f[1] = a.y; f[2] = a.z; f[3] = a.w; f[4] = b.x; f[5] = b.y; f[6] = b.z; f[7] = b.w;
}
__device__ __forceinline__ uint4 load16_nt(const uint16_t* p) {   // 16 bytes, bits only
    const float4 f = load_nt((const float*)p);
    return make_uint4(__float_as_uint(f.x), __float_as_uint(f.y), __float_as_uint(f.z), __float_as_uint(f.w));
}

template <int FMT>
__global__ __launch_bounds__(256) void quantize_sum_bf_kernel(SumArgs a, uint8_t* __restrict__ codes,
                                                              uint8_t* __restrict__ scales, long long nblocks) {
    const long long blk = (long long)blockIdx.x * 4 + (threadIdx.x >> 6);
    if (blk >= nblocks) return;
    const int lane = threadIdx.x & 63;
    const int cb = (int)(blk % a.ncb);
    const long long pix = blk / a.ncb;                     // (group, y, x)
    const int x = (int)(pix % a.w);
    const long long gy = pix / a.w;
    const int y = (int)(gy % a.h);
    const long long g = gy / a.h;
    const int j = 8 * (lane & 3);
    const int hs = 2 * a.h, ws = 2 * a.w;
    const size_t r0 = ((size_t)g * hs + 2 * y) * ws + 2 * x, r1 = r0 + ws;   // a 2x2 source patch (down)
    float v[2][8];
#pragma unroll
    for (int hh = 0; hh < 2; hh++) {
        const int ch = cb * 32 + 16 * hh + (lane >> 2);
#pragma unroll
        for (int e = 0; e < 8; e++) v[hh][e] = 0.0f;
        if (ch >= a.c) continue;
        for (int t = 0; t < a.nterms; t++) {
            const uint16_t* src = (const uint16_t*)a.src[t];
            const int cs = a.c_src[t], col = a.c_off[t] + ch;
            float u[8];
            if (!a.down[t]) {
                bf16x8(load16_nt(src + ((size_t)pix * cs + col) * 32 + j), u);
            } else {
                float p0[8], p1[8], p2[8], p3[8];
                bf16x8(load16_nt(src + (r0 * cs + col) * 32 + j), p0);
                bf16x8(load16_nt(src + ((r0 + 1) * cs + col) * 32 + j), p1);
                bf16x8(load16_nt(src + (r1 * cs + col) * 32 + j), p2);
                bf16x8(load16_nt(src + ((r1 + 1) * cs + col) * 32 + j), p3);
#pragma unroll
                for (int e = 0; e < 8; e++) u[e] = (p0[e] + p1[e]) + (p2[e] + p3[e]);
            }
            if (t == 0) {
#pragma unroll
                for (int e = 0; e < 8; e++) v[hh][e] = u[e];
            } else {
#pragma unroll
                for (int e = 0; e < 8; e++) v[hh][e] += u[e];
            }
        }
        if (a.fn != MXC_FN_NONE) {
            float z[8];
            bf16x8(load16_nt((const uint16_t*)a.z + ((size_t)pix * a.c + ch) * 32 + j), z);
            with_fn(a.fn, [&](auto t) {
#pragma unroll
                for (int e = 0; e < 8; e++) v[hh][e] *= fn_grad_c<decltype(t)::fn>(z[e]);
            });
        }
        if (a.vals) {
            float* o = a.vals + ((size_t)pix * a.c + ch) * 32 + j;
            store_nt(o, make_float4(v[hh][0], v[hh][1], v[hh][2], v[hh][3]));
            store_nt(o + 4, make_float4(v[hh][4], v[hh][5], v[hh][6], v[hh][7]));
        }
    }
    uint32_t m = 0;
#pragma unroll
    for (int hh = 0; hh < 2; hh++)
#pragma unroll
        for (int e = 0; e < 8; e++) m = max(m, __float_as_uint(v[hh][e]) & 0x7FFFFFFFu);
    m = wave_max_u32(m);
    const uint32_t sc = scale_code_from_bits<fmt_emax(FMT)>(m);
    if (lane == 0) scales[blk] = (uint8_t)sc;
    const float inv = inv_scale(sc);
    const bool bad = sc == 0xFFu;
#pragma unroll
    for (int hh = 0; hh < 2; hh++) {
        const float4 lo = make_float4(v[hh][0], v[hh][1], v[hh][2], v[hh][3]);
        const float4 hi = make_float4(v[hh][4], v[hh][5], v[hh][6], v[hh][7]);
        const int row = 16 * hh + (lane >> 2);
        uint32_t clo, chi;   // the codes of lo and hi (samples j .. j + 3, j + 4 .. j + 7)
        if (a.sr) {          // stochastic rounding: positions blk 1024 + 32 row + j .., one generator call
            const int s = (int)sc - 127;
            const uint4 w = sr_words(((uint64_t)blk * 1024 + row * 32 + j) >> 3, a.k0, a.k1);
            const uint32_t r[8] = {w.x & 0xFFFFu, w.x >> 16, w.y & 0xFFFFu, w.y >> 16,
                                   w.z & 0xFFFFu, w.z >> 16, w.w & 0xFFFFu, w.w >> 16};
            uint32_t cd[8];
#pragma unroll
            for (int e = 0; e < 8; e++) cd[e] = encode_sr<FMT>(v[hh][e], s, inv, r[e]);
            constexpr int NB = FMT == MXC_E4M3 ? 8 : 4;
            clo = cd[0] | cd[1] << NB | cd[2] << (2 * NB) | cd[3] << (3 * NB);
            chi = cd[4] | cd[5] << NB | cd[6] << (2 * NB) | cd[7] << (3 * NB);
        } else if constexpr (FMT == MXC_E4M3) {
            clo = pack4_e4m3(lo, inv);
            chi = pack4_e4m3(hi, inv);
        } else {
            clo = pack4_e2m1(lo, inv);
            chi = pack4_e2m1(hi, inv);
        }
        if constexpr (FMT == MXC_E4M3) {
            const uint2 c = bad ? make_uint2(0u, 0u) : make_uint2(clo, chi);
            *(uint2*)(codes + (size_t)blk * 1024 + row * 32 + j) = c;
        } else {
            const uint32_t c = bad ? 0u : (clo | chi << 16);
            *(uint32_t*)(codes + (size_t)blk * 512 + row * 16 + j / 2) = c;
        }
    }
}

}  // namespace

int launch_concat(const Geom& dst, const mxc_part* parts, int nparts, void* codes, uint8_t* scales,
                  hipStream_t s) {
    ConcatArgs a{};
    int off = 0;
    for (int k = 0; k < nparts; k++) {
        a.codes[k] = (const uint8_t*)parts[k].codes;
        a.scales[k] = parts[k].scales;
        a.ncb[k] = parts[k].ncb;
        a.up[k] = parts[k].up;
        a.off[k] = off;
        off += parts[k].ncb;
    }
    a.off[nparts] = off;
    a.nparts = nparts;
    a.h = dst.h;
    a.w = dst.w;
    a.bb16 = 32 * dst.bn * dst.bits / 8 / 16;
    const long long nchunks = (long long)dst.ng * dst.h * dst.w * off * a.bb16;
    if (nchunks <= 0) return MXC_OK;
    const long long grid = (nchunks + 255) / 256;
    if (grid > 0x7FFFFFFFLL) return MXC_ERR_SHAPE;
    hipLaunchKernelGGL(concat_kernel, dim3((unsigned)grid), dim3(256), 0, s, a, (uint8_t*)codes, scales, nchunks);
    return hipGetLastError() == hipSuccess ? MXC_OK : MXC_ERR_HIP;
}

int launch_quantize_sum(const Geom& dst, int fmt, const mxc_term* terms, int nterms, int fn, bool bf16,
                        const void* z, void* codes, uint8_t* scales, float* vals, hipStream_t s, bool sr,
                        uint64_t seed) {
    SumArgs a{};
    a.sr = sr ? 1 : 0;
    a.k0 = (uint32_t)seed;
    a.k1 = (uint32_t)(seed >> 32);
    for (int t = 0; t < nterms; t++) {
        a.src[t] = terms[t].src;
        a.c_src[t] = terms[t].c_src;
        a.c_off[t] = terms[t].c_off;
        a.down[t] = terms[t].down;
    }
    a.nterms = nterms;
    a.c = dst.c; a.h = dst.h; a.w = dst.w; a.ncb = dst.ncb;
    a.fn = fn;
    a.z = z;
    a.vals = vals;
    const long long nblocks = (long long)dst.ng * dst.h * dst.w * dst.ncb;
    if (nblocks <= 0) return MXC_OK;
    const long long grid = (nblocks + 3) / 4;
    if (grid > 0x7FFFFFFFLL) return MXC_ERR_SHAPE;
    const dim3 gd((unsigned)grid);
    uint8_t* const cd = (uint8_t*)codes;
    if (fmt == MXC_E4M3) {
        if (bf16) hipLaunchKernelGGL((quantize_sum_bf_kernel<MXC_E4M3>), gd, dim3(256), 0, s, a, cd, scales, nblocks);
        else      hipLaunchKernelGGL((quantize_sum_kernel<MXC_E4M3, false>), gd, dim3(256), 0, s, a, cd, scales, nblocks);
    } else {
        if (bf16) hipLaunchKernelGGL((quantize_sum_bf_kernel<MXC_E2M1>), gd, dim3(256), 0, s, a, cd, scales, nblocks);
        else      hipLaunchKernelGGL((quantize_sum_kernel<MXC_E2M1, false>), gd, dim3(256), 0, s, a, cd, scales, nblocks);
    }
    return hipGetLastError() == hipSuccess ? MXC_OK : MXC_ERR_HIP;
}

}  // namespace mxc
