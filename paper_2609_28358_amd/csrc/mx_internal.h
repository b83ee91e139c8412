// mx_internal.h -- geometry and device helpers shared by the gfx950 kernels
// and the host-side argument checks of the C ABI.  Internal to the library.
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>
#include <stddef.h>
#include "../../include/mxconv.h"

namespace mxc {

// ---------------------------------------------------------------- geometry
// MX tensor: logical (n, c, h, w); codes [np/bn][h][w][cp][bn], scales
// [np/bn][h][w][cp/32] (see mxconv.h).
struct Geom {
    int n, c, h, w;
    int bn, np, cp, ng, ncb;  // batch block, padded batch, padded channels, groups, channel blocks
    int fmt, bits;            // element format; bits 8 (E4M3), 6 (E2M3, E3M2) or 4 (E2M1)
};

// Element bits, exponent of the largest power of two below the maximum
// (OCP emax), and the format selector of the block-scaled MFMA.
constexpr int fmt_bits(int f) { return f == MXC_E4M3 ? 8 : f == MXC_E2M1 ? 4 : 6; }
constexpr int fmt_emax(int f) { return f == MXC_E4M3 ? 8 : f == MXC_E3M2 ? 4 : 2; }
constexpr int fmt_mfma(int f) { return f == MXC_E4M3 ? 0 : f == MXC_E2M3 ? 2 : f == MXC_E3M2 ? 3 : 4; }
// FP6 blocks are copied into LDS 16 bytes per 12-byte half row, so a copy
// reads up to 4 bytes past the last block: FP6 code buffers end with this
// much read-only slack.
constexpr size_t FP6_SLACK = 16;

// Returns MXC_OK or an error code.
int geom_init(Geom* g, int role, int fmt, int n, int c, int h, int w);

static inline size_t geom_codes_bytes(const Geom& g) {
    size_t e = (size_t)g.np * g.h * g.w * g.cp;
    return e * g.bits / 8 + (g.bits == 6 ? FP6_SLACK : 0);
}
static inline size_t geom_scales_bytes(const Geom& g) {
    return (size_t)g.ng * g.h * g.w * g.ncb;
}

struct Conv {
    int n, cin, cout, h, w, kh, kw, sh, sw, ph, pw, ho, wo;
    int fmt, bits;   // the common format of the call's two operands (-1, 0: mixed)
    int fa, fb;      // formats of the GEMM's first operand (W; G_Y for wgrad) and second (X or G_Y)
    Geom x;   // X  (n, cin, h, w), role ACT
    Geom gy;  // G_Y (n, cout, ho, wo), role ACT
    Geom wt;  // W  (cout, cin, kh, kw), role WEIGHT
};

// Which GEMM a call runs: the first and second operand of its format pair
// are (W, X) for the forward, (W, G_Y) for the input gradient and (G_Y, X)
// for the weight gradient.  CONV_ONE: a single format for every operand.
enum { CONV_ONE = 0, CONV_FWD = 1, CONV_DGRAD = 2, CONV_WGRAD = 3 };
int conv_init(Conv* cv, const mxc_conv* p, int fmt, int op = CONV_ONE);

// ---------------------------------------------------------------- launchers
// seed != NULL: elements rounded stochastically with that Philox key;
// keep_pad: the few-channel path leaves the padding channels' codes unwritten
int launch_quantize(const void* src, int dtype, int layout, int role, const Geom& g, int fmt,
                    void* codes, uint8_t* scales, hipStream_t s, const uint64_t* seed = nullptr,
                    bool keep_pad = false);
int im2col_check(const Conv& cv);     // MXC_ERR_SHAPE for sizes the im2col kernel cannot index
int launch_im2col(const Conv& cv, const void* xc, const uint8_t* xs, void* cc, uint8_t* cs,
                  hipStream_t s);
// several quantizations, one launch for those of the one-wave-per-block kind
struct QuantJob {
    const void* src;
    int dtype, layout, role, fmt;
    Geom g;
    void* codes;
    uint8_t* scales;
    bool col;                     // also write the CBF im2col of this activation
    Conv cv;                      // (col) the layer it is the input of
    void* col_codes;
    uint8_t* col_scales;
};
int launch_quantize_multi(int count, const QuantJob* jobs, hipStream_t s);
// NVFP (nvfp.hip): partial maxima in the workspace (NVFP_PARTS words at most)
constexpr int NVFP_PARTS = 1024;
int launch_nvfp_quantize(const void* src, int dtype, int layout, int role, const Geom& g, int fmt, void* codes,
                         uint8_t* scales, float* tscale, void* ws, hipStream_t s);
// Output pointers are typed float*; with layout MXC_CBF_BF16 they hold bf16.
int launch_fwd(const Conv& cv, const void* wc, const uint8_t* ws, const void* xc,
               const uint8_t* xs, float* y, int layout, hipStream_t s);
int launch_dgrad(const Conv& cv, const void* wc, const uint8_t* ws, const void* gc,
                 const uint8_t* gs, float* gx, int layout, hipStream_t s);
// Fused quantizing epilogue of fwd / dgrad: the output, after the activation
// fn (fwd) or times its derivative at z (dgrad), quantized into MX-CBF codes
// and scales of format fmt.
// Element-format pairs of the NVFP GEMMs (first operand, second operand):
// one format (NVFP4, NVFP6 E2M3, NVFP8), or FP4 with E3M2 (MicroQonv+).
inline bool nv_pair_ok(int fa, int fb) {
    return (fa == fb && fa != MXC_E3M2) || (fa == MXC_E2M1 && fb == MXC_E3M2);
}

struct FusedEpi {
    void* codes;
    uint8_t* scales;
    int fmt, fn;
    const void* z;       // fp32 CBF, or bf16 CBF with bf16
    bool pre;            // forward: the output gets the values before fn
    bool bf16;           // round the GEMM result to bf16 first; z and the pre output are bf16
    bool sr = false;     // codes by stochastic rounding (Philox4x32-10 keyed by seed, by code position)
    uint64_t seed = 0;
};
// fwd / dgrad for batch block 32 and kernel width 1 or 3 (conv_lean.hip);
// returns 1 when the layer is outside those shapes.  With q, the output is
// quantized in the epilogue (out, if not NULL, gets the fp32 values that were
// quantized, CBF layout).
// With nv_tw / nv_tx (device per-tensor scales of W and the source), the
// operands are NVFP4: E2M1 codes with E4M3 block scales per 8x8 block.
int launch_conv_lean(const Conv& cv, bool dg, const void* wc, const uint8_t* ws, const void* sc,
                     const uint8_t* ss, float* out, int layout, hipStream_t s, const FusedEpi* q = nullptr,
                     const float* nv_tw = nullptr, const float* nv_tx = nullptr);
// input gradient and batch-block-32 weight gradient of one layer in one
// launch (conv_lean.hip); 1 when the layer or its formats are outside it
int launch_lean_bwd(const Conv& dcv, const void* wc, const uint8_t* ws, const void* gc, const uint8_t* gs,
                    float* gx, int layout, const Conv& wcv, const void* xc, const uint8_t* xs, float* wdst,
                    int splits, hipStream_t s);
// dgrad then wgrad (conv_gemm.hip), grouped into one launch where it applies
int launch_backward(const Conv& dcv, const void* wc, const uint8_t* ws, const void* gc, const uint8_t* gs,
                    float* gx, int layout, const Conv& wcv, const void* xc, const uint8_t* xs, float* gw,
                    void* wsp, hipStream_t s, bool defer);
// weight gradient for batch block 32 (wgrad_lean.hip): number of K splits
// (0: not applicable); with more than one split the partial tiles go to the
// workspace and are reduced by the caller
int wgrad_lean_splits(const Conv& cv);
// the batch-block-32 weight gradient on 32 x 32 tiles: G_Y and X each a
// single channel block, formats MXFP8 or MXFP4
inline bool wgrad_single_block(const Conv& cv) {
    return cv.gy.ncb == 1 && cv.x.ncb == 1 && cv.fa == cv.fb && (cv.fa == MXC_E4M3 || cv.fa == MXC_E2M1);
}
// taps of one kernel row a weight-gradient wave takes together: the three of
// a 3-wide kernel on 32 x 32 MX tiles (G_Y loaded once for all three), else 1
inline int wgrad_taps(const Conv& cv, bool nv) { return !nv && wgrad_single_block(cv) && cv.kw == 3 ? 3 : 1; }
int launch_wgrad_lean(const Conv& cv, const void* gc, const uint8_t* gs, const void* xc, const uint8_t* xs,
                      float* dst, int splits, hipStream_t s, const float* nv_tg = nullptr,
                      const float* nv_tx = nullptr);
size_t wgrad_workspace(const Conv& cv);
int launch_wgrad(const Conv& cv, const void* gc, const uint8_t* gs, const void* xc,
                 const uint8_t* xs, float* gw, void* ws, hipStream_t s, const float* nv_tg = nullptr,
                 const float* nv_tx = nullptr, bool defer = false);
// Split-K partial sums a deferred weight gradient leaves in its workspace
// (0: the kernel wrote G_W itself), and their reduction for several layers.
int wgrad_pending_splits(const Conv& cv);
struct WReduceJob {
    Conv cv;
    const void* ws;
    float* gw;
};
int launch_wgrad_reduce_multi(int count, const WReduceJob* jobs, hipStream_t s);
// network operations (netops.hip): MX-block concatenation / 2x upsampling,
// and the quantized, fn'-masked sum of gradient terms
int launch_concat(const Geom& dst, const mxc_part* parts, int nparts, void* codes, uint8_t* scales,
                  hipStream_t s);
int launch_quantize_sum(const Geom& dst, int fmt, const mxc_term* terms, int nterms, int fn, bool bf16, const void* z,
                        void* codes, uint8_t* scales, float* vals, hipStream_t s, bool sr = false,
                        uint64_t seed = 0);

// naive comparator (naive.hip): a line matrix stores each 1-D-blocked line
// zero-padded to a multiple of 64 elements (one K step of the MFMA)
static inline long long naive_line_len(long long len) { return (len + 63) / 64 * 64; }
int launch_naive_im2col(const Conv& cv, const float* x, float* col, hipStream_t s);
int launch_naive_q1d(const float* src, long long rows, long long cols, int dir, int fmt, void* codes,
                     uint8_t* scales, hipStream_t s);
int launch_naive_fwd(const Conv& cv, const void* cc, const uint8_t* cs, const void* wc,
                     const uint8_t* ws, float* y, hipStream_t s);
int launch_naive_dgrad(const Conv& cv, const void* gc, const uint8_t* gs, const void* wtc,
                       const uint8_t* wts, float* gcol, float* gx, hipStream_t s);
int launch_naive_wgrad(const Conv& cv, const void* gtc, const uint8_t* gts, const void* xtc,
                       const uint8_t* xts, float* gw, hipStream_t s);

}  // namespace mxc

// ---------------------------------------------------------------- device side
#if defined(__HIPCC__)
namespace mxc {

typedef int v8i __attribute__((ext_vector_type(8)));
typedef int v4i __attribute__((ext_vector_type(4)));
typedef int v2i __attribute__((ext_vector_type(2)));
typedef float v16f __attribute__((ext_vector_type(16)));
typedef __attribute__((address_space(3))) v2i lds_v2i;

// A 16-byte vector store with the non-temporal hint, for large outputs that
// no later kernel of the path reads soon (fp32 GEMM results, the explicit
// im2col): the lines are not kept in the caches, so the stream drains to HBM
// without leaving dirty last-level-cache lines for the next kernel to write
// back (measured: the benchmark step takes 0.44 instead of 0.49 ms).
__device__ __forceinline__ void store_nt(void* p, uint4 v) {
    v4i t;
    t[0] = (int)v.x; t[1] = (int)v.y; t[2] = (int)v.z; t[3] = (int)v.w;
    __builtin_nontemporal_store(t, (v4i*)p);
}
__device__ __forceinline__ void store_nt(void* p, uint2 v) {
    v2i t;
    t[0] = (int)v.x; t[1] = (int)v.y;
    __builtin_nontemporal_store(t, (v2i*)p);
}
__device__ __forceinline__ void store_nt(void* p, float4 v) {
    store_nt(p, make_uint4(__float_as_uint(v.x), __float_as_uint(v.y), __float_as_uint(v.z), __float_as_uint(v.w)));
}

// 16- and 8-byte vector loads with the non-temporal hint, for sources read
// exactly once (the quantizer's fp32 / bf16 input): the stream does not
// displace cached data the next kernels read (measured: the benchmark step
// takes 0.42 instead of 0.44 ms).
__device__ __forceinline__ float4 load_nt(const float* p) {
    typedef float v4f __attribute__((ext_vector_type(4)));
    const v4f t = __builtin_nontemporal_load((const v4f*)p);
    return make_float4(t[0], t[1], t[2], t[3]);
}
__device__ __forceinline__ uint2 load_nt(const unsigned short* p) {
    const v2i t = __builtin_nontemporal_load((const v2i*)p);
    return make_uint2((uint32_t)t[0], (uint32_t)t[1]);
}

// bf16 full-precision tensors (the MXC_CBF_BF16 layout and the MXC_FN_BF16
// mode).  fp32 -> bf16 is the hardware conversion (v_cvt_pk_bf16_f32, two
// values per instruction): round to nearest, ties to even, a NaN stays a NaN.
typedef float f2v __attribute__((ext_vector_type(2)));
typedef __bf16 bf2v __attribute__((ext_vector_type(2)));
__device__ __forceinline__ uint32_t bf16_pack2(float a, float b) {
    const f2v v = {a, b};
    return __builtin_bit_cast(uint32_t, __builtin_convertvector(v, bf2v));
}
__device__ __forceinline__ uint32_t bf16_bits(float f) { return __builtin_bit_cast(uint16_t, (__bf16)f); }
__device__ __forceinline__ float bf16_round(float f) { return __uint_as_float(bf16_bits(f) << 16); }
// four consecutive bf16 (8 bytes) <-> four floats
__device__ __forceinline__ uint2 bf16_pack4(float a, float b, float c, float d) {
    return make_uint2(bf16_pack2(a, b), bf16_pack2(c, d));
}
__device__ __forceinline__ float4 bf16_unpack4(uint2 u) {
    return make_float4(__uint_as_float(u.x << 16), __uint_as_float(u.x & 0xFFFF0000u),
                       __uint_as_float(u.y << 16), __uint_as_float(u.y & 0xFFFF0000u));
}

// Largest |x| bit pattern of a block -> E8M0 code (0xFF if any element was
// NaN/inf).  floor(log2) comes from the exponent field, or from the
// leading-zero count for an fp32 subnormal.
template <int EMAX>
__device__ __forceinline__ uint32_t scale_code_from_bits(uint32_t amax_bits) {
    if (amax_bits >= 0x7F800000u) return 0xFFu;
    if (amax_bits == 0u) return 0u;
    int e = (amax_bits >= 0x00800000u) ? (int)(amax_bits >> 23) - 127
                                       : (31 - __clz((int)amax_bits)) - 149;
    int s = e - EMAX;
    s = s < -127 ? -127 : (s > 127 ? 127 : s);
    return (uint32_t)(s + 127);
}

// 2^-s as a float for s = code - 127 in [-127, 126] (always exact).
__device__ __forceinline__ float inv_scale(uint32_t code) {
    int s = (int)code - 127;
    return __uint_as_float((uint32_t)(127 - s) << 23);
}

// Element encoding on gfx950's scaled converts.  v_cvt_scalef32_pk_fp8_f32 /
// _pk_fp4_f32 divide by their scale operand and round to nearest, ties to
// even, keeping the sign of zero; the FP4 convert saturates at 6, the FP8
// convert does not (|x| >= 464 gives the NaN code), so FP8 inputs are clamped
// to +-448 first.  With that clamp both match the reference rule on every
// finite fp32 input (checked exhaustively on MI355X).  The inputs here are
// x * 2^-s, exact, so the convert runs with scale 1.
typedef short v2s __attribute__((ext_vector_type(2)));

// four consecutive elements -> four E4M3 codes (first element in the low byte)
__device__ __forceinline__ uint32_t pack4_e4m3(float4 x, float inv) {
    const float a = __builtin_amdgcn_fmed3f(x.x * inv, -448.0f, 448.0f);
    const float b = __builtin_amdgcn_fmed3f(x.y * inv, -448.0f, 448.0f);
    const float c = __builtin_amdgcn_fmed3f(x.z * inv, -448.0f, 448.0f);
    const float d = __builtin_amdgcn_fmed3f(x.w * inv, -448.0f, 448.0f);
    v2s r = {0, 0};
    r = __builtin_amdgcn_cvt_scalef32_pk_fp8_f32(r, a, b, 1.0f, false);
    r = __builtin_amdgcn_cvt_scalef32_pk_fp8_f32(r, c, d, 1.0f, true);
    return __builtin_bit_cast(uint32_t, r);
}

// eight consecutive elements -> eight E2M1 codes (first element in the low nibble)
__device__ __forceinline__ uint32_t pack8_e2m1(float4 x, float4 y, float inv) {
    uint32_t q = 0;
    q = __builtin_amdgcn_cvt_scalef32_pk_fp4_f32(q, x.x * inv, x.y * inv, 1.0f, 0);
    q = __builtin_amdgcn_cvt_scalef32_pk_fp4_f32(q, x.z * inv, x.w * inv, 1.0f, 1);
    q = __builtin_amdgcn_cvt_scalef32_pk_fp4_f32(q, y.x * inv, y.y * inv, 1.0f, 2);
    q = __builtin_amdgcn_cvt_scalef32_pk_fp4_f32(q, y.z * inv, y.w * inv, 1.0f, 3);
    return q;
}

// FP6 (E2M3 / E3M2): v_cvt_scalef32_2xpk16_{fp6,bf6}_f32 converts 32 floats
// into one 192-bit string of codes, rounding to nearest even, saturating at
// the format maximum and keeping the sign of zero (checked against the
// reference rule on MI355X); it interleaves its two sources (code 2i from
// the first, 2i + 1 from the second), so the even elements go first.
typedef int v6i __attribute__((ext_vector_type(6)));
template <int FMT>
__device__ __forceinline__ v6i cvt32_fp6(const v16f& even, const v16f& odd) {
    if constexpr (FMT == MXC_E2M3) return __builtin_amdgcn_cvt_scalef32_2xpk16_fp6_f32(even, odd, 1.0f);
    else return __builtin_amdgcn_cvt_scalef32_2xpk16_bf6_f32(even, odd, 1.0f);
}
// 32 consecutive elements (x[0..7]) -> 24 bytes of codes
template <int FMT>
__device__ __forceinline__ v6i pack32_fp6(const float4* x, float inv) {
    v16f a, b;
#pragma unroll
    for (int q = 0; q < 8; q++) {
        a[2 * q] = x[q].x * inv; b[2 * q] = x[q].y * inv;
        a[2 * q + 1] = x[q].z * inv; b[2 * q + 1] = x[q].w * inv;
    }
    return cvt32_fp6<FMT>(a, b);
}
// 16 consecutive elements (x[0..3]) -> 12 bytes of codes (the first three
// dwords of the result)
template <int FMT>
__device__ __forceinline__ v6i pack16_fp6(const float4* x, float inv) {
    v16f a, b;
#pragma unroll
    for (int q = 0; q < 4; q++) {
        a[2 * q] = x[q].x * inv; b[2 * q] = x[q].y * inv;
        a[2 * q + 1] = x[q].z * inv; b[2 * q + 1] = x[q].w * inv;
    }
#pragma unroll
    for (int i = 8; i < 16; i++) { a[i] = 0.0f; b[i] = 0.0f; }
    return cvt32_fp6<FMT>(a, b);
}

// ---------------------------------------------------------------- stochastic rounding
// Philox4x32-10 (Salmon, Moraes, Dror, Shaw, SC'11): ten rounds of two
// 32x32 -> 64-bit products mixed with the key, the key advanced by the Weyl
// constants between rounds.
__device__ __forceinline__ uint4 philox4x32_10(uint4 c, uint32_t k0, uint32_t k1) {
#pragma unroll
    for (int round = 0; round < 10; round++) {
        if (round > 0) { k0 += 0x9E3779B9u; k1 += 0xBB67AE85u; }
        const uint64_t p0 = (uint64_t)0xD2511F53u * c.x;
        const uint64_t p1 = (uint64_t)0xCD9E8D57u * c.z;
        c = make_uint4((uint32_t)(p1 >> 32) ^ c.y ^ k0, (uint32_t)p1, (uint32_t)(p0 >> 32) ^ c.w ^ k1, (uint32_t)p0);
    }
    return c;
}
// The 16-bit random words of the eight code positions 8 q .. 8 q + 7:
// position 8 q + j takes half (j mod 2) of word j / 2 at counter (q, 0, 0).
__device__ __forceinline__ uint4 sr_words(uint64_t q, uint32_t k0, uint32_t k1) {
    return philox4x32_10(make_uint4((uint32_t)q, (uint32_t)(q >> 32), 0u, 0u), k0, k1);
}
__device__ __forceinline__ uint32_t sr_half(const uint4& w, int j) {
    const uint32_t v = (j >> 1) == 0 ? w.x : (j >> 1) == 1 ? w.y : (j >> 1) == 2 ? w.z : w.w;
    return (j & 1) ? v >> 16 : v & 0xFFFFu;
}

template <int F> struct FmtSR;
template <> struct FmtSR<MXC_E4M3> { static constexpr int MB = 3, BIAS = 7; static constexpr uint32_t MAXB = 0x43E00000u, MAXC = 0x7Eu; };
template <> struct FmtSR<MXC_E2M1> { static constexpr int MB = 1, BIAS = 1; static constexpr uint32_t MAXB = 0x40C00000u, MAXC = 0x7u; };
template <> struct FmtSR<MXC_E2M3> { static constexpr int MB = 3, BIAS = 1; static constexpr uint32_t MAXB = 0x40F00000u, MAXC = 0x1Fu; };
template <> struct FmtSR<MXC_E3M2> { static constexpr int MB = 2, BIAS = 3; static constexpr uint32_t MAXB = 0x41E00000u, MAXC = 0x1Fu; };

// Stochastic rounding of one finite element x of a block with scale 2^s
// (inv = 2^-s) under 16 random bits r: with lo <= |x| 2^-s < hi the
// neighbouring grid values, the code of hi when r < frac * 2^16, frac =
// (|x| 2^-s - lo) / (hi - lo), else of lo; at or above the format maximum,
// the maximum.  The decision is taken in integers on the bits of x itself
// (|x| = M 2^(ex - 23)), so a scaled value below the fp32 range still rounds
// exactly: |x| 2^-s / 2^(te - MB) = M 2^-k with te the scaled value's binade
// (at least the format's smallest), lo = (M >> k) quanta, frac = D / 2^k
// with D = M mod 2^k, and r < frac * 2^16 <=> r < ceil(D 2^(16 - k)).
// k >= 13 for every block scale; M < 2^24, so shifts are capped at 24.
// Written without branches: every lane takes the same path.
// The rule's body with the format as values (MB mantissa bits, BIAS, MAXB
// the fp32 bits of the format maximum, MAXC its code, NB the code width), so
// that a kernel whose output format is a run-time value shares it.
__device__ __forceinline__ uint32_t encode_sr_f(float x, int s, float inv, uint32_t r, int MB, int BIAS,
                                                uint32_t MAXB, uint32_t MAXC, int NB) {
    const int EMIN = 1 - BIAS;
    const uint32_t b = __float_as_uint(x), ab = b & 0x7FFFFFFFu;
    const uint32_t scaled = __float_as_uint(x * inv) & 0x7FFFFFFFu;   // exact unless far below the maximum
    const uint32_t fe = ab >> 23;
    const uint32_t M = fe ? ((ab & 0x7FFFFFu) | 0x800000u) : ab;
    const int ex = fe ? (int)fe - 127 : -126;
    const int fl = fe ? ex : (31 - __clz((int)ab)) - 149;           // floor(log2 |x|)
    const int te = max(fl - s, EMIN);
    const int k = 23 + te - MB - ex + s;
    const int kc = min(k, 24);
    const uint32_t mlo = M >> kc;
    const uint32_t D = M & ((1u << kc) - 1u);
    const int sh = k - 16;                                            // >= -3
    const int shc = min(sh, 24);
    const uint32_t t = sh <= 0 ? D << (-sh) : (D + (1u << shc) - 1u) >> shc;
    const uint32_t up = r < t ? 1u : 0u;
    uint32_t code = (uint32_t)(((te + BIAS) << MB) - (1 << MB)) + mlo + up;
    code = scaled >= MAXB ? MAXC : (ab == 0u ? 0u : code);
    return code | ((b >> 31) << (NB - 1));
}
template <int FMT>
__device__ __forceinline__ uint32_t encode_sr(float x, int s, float inv, uint32_t r) {
    typedef FmtSR<FMT> F;
    return encode_sr_f(x, s, inv, r, F::MB, F::BIAS, F::MAXB, F::MAXC, fmt_bits(FMT));
}
// Run-time format: the same rule for an output format known only at run time.
__device__ __forceinline__ uint32_t encode_sr_rt(int fmt, float x, int s, float inv, uint32_t r) {
    const int mb = fmt == MXC_E2M1 ? 1 : fmt == MXC_E3M2 ? 2 : 3;
    const int bias = fmt == MXC_E4M3 ? 7 : fmt == MXC_E3M2 ? 3 : 1;
    const uint32_t maxb = fmt == MXC_E4M3 ? FmtSR<MXC_E4M3>::MAXB : fmt == MXC_E2M1 ? FmtSR<MXC_E2M1>::MAXB
                        : fmt == MXC_E2M3 ? FmtSR<MXC_E2M3>::MAXB : FmtSR<MXC_E3M2>::MAXB;
    const uint32_t maxc = fmt == MXC_E4M3 ? 0x7Eu : fmt == MXC_E2M1 ? 0x7u : 0x1Fu;
    const int nb = fmt == MXC_E4M3 ? 8 : fmt == MXC_E2M1 ? 4 : 6;
    return encode_sr_f(x, s, inv, r, mb, bias, maxb, maxc, nb);
}
// Stochastic codes of four consecutive elements x whose first code position
// p is a multiple of 4 (positions p .. p + 3 take half-words p % 8 .. + 3 of
// the generator call at counter p / 8).
template <int FMT>
__device__ __forceinline__ void sr_codes4(float4 x, uint64_t p, int s, float inv, uint32_t k0, uint32_t k1,
                                          uint32_t* cd) {
    const uint4 w = sr_words(p >> 3, k0, k1);
    const bool hi = (p & 4u) != 0u;
    const uint32_t w0 = hi ? w.z : w.x, w1 = hi ? w.w : w.y;
    cd[0] = encode_sr<FMT>(x.x, s, inv, w0 & 0xFFFFu);
    cd[1] = encode_sr<FMT>(x.y, s, inv, w0 >> 16);
    cd[2] = encode_sr<FMT>(x.z, s, inv, w1 & 0xFFFFu);
    cd[3] = encode_sr<FMT>(x.w, s, inv, w1 >> 16);
}

// The same decision for a normal fp32 x (or a zero), in fewer operations:
// the carry out of the low k bits of M + R, R = ((2^16 - 1 - r) << (k - 16))
// | (2^(k - 16) - 1), is exactly [r < ceil(D 2^(16 - k))], so the rounded
// magnitude in quanta is (M + R) >> k.  For k > 31 (elements more than 2^8
// quanta below the grid's first step) the low k - 31 bits of M are folded
// into a sticky bit first, which leaves the decision unchanged.  An fp32
// subnormal x (M without its implicit bit) needs encode_sr.
template <int FMT>
__device__ __forceinline__ uint32_t encode_sr_normal(float x, int s, float inv, uint32_t r) {
    typedef FmtSR<FMT> F;
    constexpr int MB = F::MB, BIAS = F::BIAS, EMIN = 1 - BIAS;
    const uint32_t b = __float_as_uint(x), ab = b & 0x7FFFFFFFu;
    const uint32_t scaled = __float_as_uint(x * inv) & 0x7FFFFFFFu;   // exact when at or above the maximum
    const int ea = (int)(ab >> 23) - 127 - s;                         // binade of |x| 2^-s
    const int te = max(ea, EMIN);
    const int k = 23 - MB + te - ea;                                  // >= 20
    const uint32_t M = (ab & 0x7FFFFFu) | 0x800000u;
    const int sh2 = min(max(k - 31, 0), 24);
    const int kk = min(k, 31);
    const uint32_t Mp = (M >> sh2) + ((M & ((1u << sh2) - 1u)) != 0u ? 1u : 0u);
    const uint32_t lowm = (1u << (kk - 16)) - 1u;
    const uint32_t R = ((r ^ 0xFFFFu) << (kk - 16)) | lowm;
    uint32_t code = (uint32_t)((te + BIAS - 1) << MB) + ((Mp + R) >> kk);
    code = scaled >= F::MAXB ? F::MAXC : (ab == 0u ? 0u : code);
    return code | ((b >> 31) << (fmt_bits(FMT) - 1));
}
// Does x need the general path (a non-zero fp32 subnormal)?
__device__ __forceinline__ bool sr_needs_general(float x) {
    const uint32_t ab = __float_as_uint(x) & 0x7FFFFFFFu;
    return ab != 0u && ab < 0x800000u;
}

// ---------------------------------------------------------------- NVFP operands
// The block-scaled matrix cores take E8M0 scales per 32 K elements; an NVFP
// block scale is E4M3 per 8 elements.  A code times its E4M3 scale B has at
// most 2 + 4 = 6 (E2M1), 3 + 4 = 7 (E3M2) or 4 + 4 = 8 (E2M3, E4M3)
// significant bits.  FP4 and FP6 products lie in [2^-13, 12544], so they are
// exact in fp16; FP8 products reach 448 x 448, past fp16's range, and are
// exact in bf16 (8 significant bits, the fp32 exponent range).  The GEMMs
// therefore decode NVFP fragments to fp16 (FP4, FP6) or bf16 (FP8) and run
// fp16 / bf16 MFMAs; the product of two decoded values is exact in fp32.
typedef _Float16 v2h __attribute__((ext_vector_type(2)));
typedef _Float16 v8h __attribute__((ext_vector_type(8)));
typedef _Float16 v32h __attribute__((ext_vector_type(32)));
typedef float v2f __attribute__((ext_vector_type(2)));

// An E4M3 block scale: 2^e2 times m8 / 8 (m8 = 8 + m for a normal code, m
// for a subnormal one), as the power of two and the mantissa factor.
__device__ __forceinline__ void e4m3_split(uint32_t sg, float& pw, float& mf) {
    const uint32_t e = (sg >> 3) & 0xFu, m = sg & 7u;
    pw = __uint_as_float(e ? (e + 120u) << 23 : (127u - 9u) << 23);   // 2^(e-7), or 2^-9
    mf = e ? 1.0f + 0.125f * (float)m : (float)m;
}

// 32 codes of format F (the lane's fragment: FP4 element k in nibble k, FP6
// code k in bits 6k .. 6k+5, FP8 element k in byte k) and the E4M3 scales of
// their four groups of 8 (byte g of s4: elements 8g .. 8g+7) -> 32 decoded
// values code x B in out[0..15] (element k in half k): fp16 for FP4 / FP6,
// bf16 for FP8.
template <int F>
__device__ __forceinline__ void nv_decode32(const v8i& f, uint32_t s4, uint32_t* out) {
    if constexpr (F == MXC_E2M1) {
        // the scaled convert applies only the power of two of its scale
        // operand (measured): 2^E goes to the convert, the mantissa factor is
        // one packed fp16 multiply
#pragma unroll
        for (int g = 0; g < 4; g++) {
            float pw, mf;
            e4m3_split((s4 >> (8 * g)) & 0xFFu, pw, mf);
            const _Float16 mh = (_Float16)mf;
            const v2h mm = {mh, mh};
            const uint32_t src = (uint32_t)f[g];
#define NVD(SEL) { const v2h v = __builtin_bit_cast(v2h, __builtin_amdgcn_cvt_scalef32_pk_f16_fp4(src, pw, SEL)) * mm; \
                   out[4 * g + SEL] = __builtin_bit_cast(uint32_t, v); }
            NVD(0) NVD(1) NVD(2) NVD(3)
#undef NVD
        }
    } else if constexpr (fmt_bits(F) == 6) {
        // the 32 codes to fp16 with scale 1 (exact), then each group times
        // its B, exact in fp16 (one packed multiply per pair)
        v6i src;
#pragma unroll
        for (int e = 0; e < 6; e++) src[e] = f[e];
        const v32h v = F == MXC_E2M3 ? __builtin_amdgcn_cvt_scalef32_pk32_f16_fp6(src, 1.0f)
                                     : __builtin_amdgcn_cvt_scalef32_pk32_f16_bf6(src, 1.0f);
#pragma unroll
        for (int g = 0; g < 4; g++) {
            float pw, mf;
            e4m3_split((s4 >> (8 * g)) & 0xFFu, pw, mf);
            const _Float16 bh = (_Float16)(pw * mf);
            const v2h bb = {bh, bh};
#pragma unroll
            for (int j = 0; j < 4; j++) {
                const v2h x = {v[8 * g + 2 * j], v[8 * g + 2 * j + 1]};
                out[4 * g + j] = __builtin_bit_cast(uint32_t, x * bb);
            }
        }
    } else {
        // FP8: each pair decoded to fp32 (exact), times B in fp32 (exact: at
        // most 8 significant bits), rounded to bf16 (exact for the same reason)
#pragma unroll
        for (int g = 0; g < 4; g++) {
            float pw, mf;
            e4m3_split((s4 >> (8 * g)) & 0xFFu, pw, mf);
            const float b = pw * mf;
#pragma unroll
            for (int w = 0; w < 2; w++) {
                const uint32_t src = (uint32_t)f[2 * g + w];
                const v2f lo = __builtin_amdgcn_cvt_scalef32_pk_f32_fp8(src, 1.0f, false);
                const v2f hi = __builtin_amdgcn_cvt_scalef32_pk_f32_fp8(src, 1.0f, true);
                out[4 * g + 2 * w] = bf16_pack2(lo[0] * b, lo[1] * b);
                out[4 * g + 2 * w + 1] = bf16_pack2(hi[0] * b, hi[1] * b);
            }
        }
    }
}

// D += A B over the 64 K elements of two decoded fragments: four fp16 MFMAs,
// instruction t taking elements 8t .. 8t+7 of each lane's 32 (the same K
// relabelling on both operands, so the sum is unchanged).
__device__ __forceinline__ v16f mfma_nv(const uint32_t* a, const uint32_t* b, v16f c) {
#pragma unroll
    for (int t = 0; t < 4; t++) {
        v4i av = {(int)a[4 * t], (int)a[4 * t + 1], (int)a[4 * t + 2], (int)a[4 * t + 3]};
        v4i bv = {(int)b[4 * t], (int)b[4 * t + 1], (int)b[4 * t + 2], (int)b[4 * t + 3]};
        c = __builtin_amdgcn_mfma_f32_32x32x16_f16(__builtin_bit_cast(v8h, av), __builtin_bit_cast(v8h, bv), c, 0, 0, 0);
    }
    return c;
}

// four consecutive elements -> four E2M1 codes in 16 bits (first element in the low nibble)
__device__ __forceinline__ unsigned short pack4_e2m1(float4 x, float inv) {
    uint32_t q = 0;
    q = __builtin_amdgcn_cvt_scalef32_pk_fp4_f32(q, x.x * inv, x.y * inv, 1.0f, 0);
    q = __builtin_amdgcn_cvt_scalef32_pk_fp4_f32(q, x.z * inv, x.w * inv, 1.0f, 1);
    return (unsigned short)q;
}

// ---------------------------------------------------------------- activations
// Activation of the forward epilogue and its derivative (input-gradient
// epilogue, gradient quantizer).  SiLU uses the hardware exp2 and reciprocal
// (about 1 ulp each): the logistic s(y) = 1 / (1 + 2^(-y log2 e)); exp2
// overflows to +inf for very negative y, where s = 0 and SiLU = -0.
__device__ __forceinline__ float logistic(float y) {
    return __builtin_amdgcn_rcpf(1.0f + __builtin_amdgcn_exp2f(-y * 1.4426950408889634f));
}
template <int F>
__device__ __forceinline__ float fn_apply_c(float y) {
    if constexpr (F == MXC_FN_NONE) return y;
    else if constexpr (F == MXC_FN_RELU) return y > 0.0f ? y : 0.0f;
    else return y * logistic(y);                                // SiLU
}
template <int F>
__device__ __forceinline__ float fn_grad_c(float z) {
    if constexpr (F == MXC_FN_NONE) return 1.0f;
    else if constexpr (F == MXC_FN_RELU) return z > 0.0f ? 1.0f : 0.0f;
    else {
        const float s = logistic(z);                            // SiLU' = s (1 + z (1 - s))
        return s * (1.0f + z * (1.0f - s));
    }
}
// the derivative with the choice made per value (fewer live registers)
__device__ __forceinline__ float fn_grad(int fn, float z) {
    return fn == MXC_FN_NONE ? 1.0f : fn == MXC_FN_RELU ? fn_grad_c<MXC_FN_RELU>(z) : fn_grad_c<MXC_FN_SILU>(z);
}
// body(FnTag<f>{}) for an activation f other than MXC_FN_NONE: the choice is
// one uniform branch around straight-line code, so the values' exponentials
// and reciprocals are independent and overlap.  (A choice per value, inside
// an unrolled loop, put a scalar branch between every two values and ran
// each SiLU as one dependent chain.)
template <int F> struct FnTag { static constexpr int fn = F; };
template <class Body>
__device__ __forceinline__ void with_fn(int fn, Body&& body) {
    if (fn == MXC_FN_RELU) body(FnTag<MXC_FN_RELU>{});
    else body(FnTag<MXC_FN_SILU>{});
}

// ---------------------------------------------------------------- MXFP8 operands
// Eq. (7) sums exact block products in fp32.  The block-scaled MFMA does so
// for FP4 and FP6 operands, but for FP8 it aligns the products of every 8
// consecutive K elements to the largest and truncates them to 14 bits before
// adding (measured), which is far outside fp32 accumulation.  FP8 operands
// are therefore decoded to bf16 with their E8M0 scale applied and multiplied
// on the bf16 matrix cores, which sum exact products at fp32 precision
// (measured: within 2.7e-7 of the sum of |products| over 64-long chains of
// 4-bit-significand operands spread over 80 binades).  An E4M3 value (4
// significant bits, magnitudes 2^-9 .. 448) times 2^(c-127) is exact in bf16
// for every E8M0 code c in 5 .. 246 (the quantizer produces 0 .. 246 and
// 255); below code 5 magnitudes under 2^-133 flush to zero; code 255 (NaN)
// decodes every element to NaN.  The scaled convert reads its fp32 scale
// operand's exponent field as the E8M0 code, so the code is passed as the
// exponent bits (code 0 -> +0.0, which the convert takes as 2^-127).
typedef __bf16 v8bf __attribute__((ext_vector_type(8)));
typedef __bf16 v2bf __attribute__((ext_vector_type(2)));

__device__ __forceinline__ float e8m0_operand(int code) { return __uint_as_float((uint32_t)code << 23); }

// 32 E4M3 codes of an operand fragment (bytes 0..15 of K block 0, scale
// code s0; bytes 16..31 of K block 1, scale code s1) -> 32 bf16 values,
// out[j] = elements 2j (low half) and 2j + 1: byte order is kept.
__device__ __forceinline__ void e4m3_decode32(const v8i& f, int s0, int s1, uint32_t* out) {
    const float p0 = e8m0_operand(s0), p1 = e8m0_operand(s1);
#pragma unroll
    for (int d = 0; d < 8; d++) {
        const float p = d < 4 ? p0 : p1;
        out[2 * d] = __builtin_bit_cast(uint32_t, __builtin_amdgcn_cvt_scalef32_pk_bf16_fp8((uint32_t)f[d], p, false));
        out[2 * d + 1] = __builtin_bit_cast(uint32_t, __builtin_amdgcn_cvt_scalef32_pk_bf16_fp8((uint32_t)f[d], p, true));
    }
}

// The same when the lane holds only the scale code of its own half's K block
// (lane l: K block l / 32 of row l % 32, the block-scaled MFMA's convention):
// the other block's code comes from lane l ^ 32.  The whole wave must be active.
__device__ __forceinline__ void e4m3_decode32_lane(const v8i& f, int s, uint32_t* out) {
    const int lane = threadIdx.x & 63;
    const int so = __builtin_amdgcn_ds_bpermute((lane ^ 32) << 2, s);
    const bool hi = lane >= 32;
    e4m3_decode32(f, hi ? so : s, hi ? s : so, out);
}

// D += A B over the 64 K elements of two decoded fragments: four bf16 MFMAs,
// instruction t taking elements 8t .. 8t+7 of each lane's 32 (the same K
// relabelling on both operands, so the sum is unchanged).
__device__ __forceinline__ v16f mfma_x8(const uint32_t* a, const uint32_t* b, v16f c) {
#pragma unroll
    for (int t = 0; t < 4; t++) {
        v4i av = {(int)a[4 * t], (int)a[4 * t + 1], (int)a[4 * t + 2], (int)a[4 * t + 3]};
        v4i bv = {(int)b[4 * t], (int)b[4 * t + 1], (int)b[4 * t + 2], (int)b[4 * t + 3]};
        c = __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(v8bf, av), __builtin_bit_cast(v8bf, bv), c, 0, 0, 0);
    }
    return c;
}

// One block-scaled product: D(32x32) += A(32 x 64) B(64 x 32) with one E8M0
// scale per (row, 32-wide K block).  Operand fragment of lane l (row l%32,
// half h = l/32):
//   FP8: bytes 0..15  = K-block 0 elements [16h, 16h+16)
//        bytes 16..31 = K-block 1 elements [16h, 16h+16)
//   FP4: bytes 0..15  = K-block h, all 32 elements (nibble k = element k)
//   scale operand: E8M0 of (row l%32, K-block h) in the low byte.
//   FP6: bytes 0..23  = K-block h, all 32 elements as a bit string (element
//        k in bits 6k .. 6k+5), bytes 24..31 unused.
// The two operands may have different formats (FA for a, FB for b); FP8 is
// only paired with FP8 and runs on the exact bf16 route above (kernels that
// reuse a fragment decode it once and call mfma_x8 themselves).
template <int FA, int FB = FA>
__device__ __forceinline__ v16f mfma_mx(v8i a, v8i b, v16f c, int sa, int sb) {
    static_assert((FA == MXC_E4M3) == (FB == MXC_E4M3), "FP8 pairs only with FP8");
    if constexpr (FA == MXC_E4M3) {
        uint32_t ad[16], bd[16];
        e4m3_decode32_lane(a, sa, ad);
        e4m3_decode32_lane(b, sb, bd);
        return mfma_x8(ad, bd, c);
    } else {
        constexpr int ca = fmt_mfma(FA), cb = fmt_mfma(FB);
        return __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(a, b, c, ca, cb, 0, sa, 0, sb);
    }
}

// An A fragment multiplied by several B fragments: an FP8 one is decoded
// once (set), the others are kept as they are.
template <int F> struct AFrag {
    v8i f;
    int s;
    uint32_t d[F == MXC_E4M3 ? 16 : 1];
    __device__ __forceinline__ void set(const v8i& f_, int s_) {
        f = f_;
        s = s_;
        if constexpr (F == MXC_E4M3) e4m3_decode32_lane(f, s, d);
    }
};
template <int F>
__device__ __forceinline__ v16f mfma_mx_a(const AFrag<F>& a, v8i b, v16f c, int sb) {
    if constexpr (F == MXC_E4M3) {
        uint32_t bd[16];
        e4m3_decode32_lane(b, sb, bd);
        return mfma_x8(a.d, bd, c);
    } else {
        return mfma_mx<F>(a.f, b, c, a.s, sb);
    }
}

// Asynchronous global -> LDS copies (global_load_lds).  Every lane supplies
// its own source address; the LDS destination is the wave-uniform base in M0
// plus 16 * lane for the 16-byte form, plus 4 * lane for the one-byte form
// (the byte is zero-extended to the lane's dword).  They are issued as inline
// assembly, so the compiler does not track them: left to itself it waits for
// every outstanding copy before any LDS read, which serialises a multi-stage
// pipeline.  The caller waits with vm_wait<N>() -- N = the vector-memory
// operations of this wave that may still be in flight, counted in issue
// order -- before the barrier that publishes the data to the other waves.
typedef __attribute__((address_space(3))) uint8_t lds_u8;

__device__ __forceinline__ uint32_t lds_addr(const uint8_t* p) {
    return (uint32_t)(uintptr_t)(const lds_u8*)p;
}
__device__ __forceinline__ void dma16_async(const void* gsrc, uint32_t lds) {
    asm volatile("global_load_lds_dwordx4 %0, off" ::"v"(gsrc), "{m0}"(lds) : "memory");
}
__device__ __forceinline__ void dma1_async(const void* gsrc, uint32_t lds) {
    asm volatile("global_load_lds_ubyte %0, off" ::"v"(gsrc), "{m0}"(lds) : "memory");
}
template <int N>
__device__ __forceinline__ void vm_wait() {
    static_assert(N >= 0 && N <= 63, "vmcnt holds 6 bits");
    asm volatile("s_waitcnt vmcnt(%0)" ::"n"(N) : "memory");
}
// Wait for a stage when `later` stages of PER operations each were issued
// after it (later in 0..2).
template <int PER>
__device__ __forceinline__ void vm_wait_stage(int later) {
    if (later <= 0) vm_wait<0>();
    else if (later == 1) vm_wait<PER>();
    else vm_wait<2 * PER>();
}

// Maximum of a 32-bit value over the 64 lanes of a wave, returned to every
// lane: DPP swaps within quads (lanes 1032 and 2301 orders), a mirror within
// each 8 and each 16 lanes (after which every lane of a 16-lane row holds the
// row's maximum), then the four row maxima read as scalars.  No LDS traffic
// and no waits, unlike a shuffle through ds_bpermute.  The whole wave must be
// active.
__device__ __forceinline__ uint32_t wave_max_u32(uint32_t m) {
    m = max(m, (uint32_t)__builtin_amdgcn_mov_dpp((int)m, 0xB1, 0xF, 0xF, false));   // quad_perm 1,0,3,2
    m = max(m, (uint32_t)__builtin_amdgcn_mov_dpp((int)m, 0x4E, 0xF, 0xF, false));   // quad_perm 2,3,0,1
    m = max(m, (uint32_t)__builtin_amdgcn_mov_dpp((int)m, 0x141, 0xF, 0xF, false));  // row_half_mirror
    m = max(m, (uint32_t)__builtin_amdgcn_mov_dpp((int)m, 0x140, 0xF, 0xF, false));  // row_mirror
    const uint32_t a = (uint32_t)__builtin_amdgcn_readlane((int)m, 0);
    const uint32_t b = (uint32_t)__builtin_amdgcn_readlane((int)m, 16);
    const uint32_t c = (uint32_t)__builtin_amdgcn_readlane((int)m, 32);
    const uint32_t d = (uint32_t)__builtin_amdgcn_readlane((int)m, 48);
    return max(max(a, b), max(c, d));
}

// LDS transposing reads (16-lane groups).
//  tr8: lane i gets byte (i%8) of the 8-byte chunks addressed by lanes 2q + i/8, q = 0..7.
//  tr4: lane i gets nibble i of the chunks addressed by lanes q, q = 0..15.
__device__ __forceinline__ v2i lds_tr8(const uint8_t* p) {
    return __builtin_amdgcn_ds_read_tr8_b64_v2i32((lds_v2i*)(p));
}
__device__ __forceinline__ v2i lds_tr4(const uint8_t* p) {
    return __builtin_amdgcn_ds_read_tr4_b64_v2i32((lds_v2i*)(p));
}
//  tr6: lane i gets 6-bit element i of the 12-byte chunks addressed by lanes
//       q, q = 0..15, as element q of its 96-bit result.  Every chunk address
//       must be 16-byte aligned (the low four bits are ignored).
typedef int v3i __attribute__((ext_vector_type(3)));
typedef __attribute__((address_space(3))) v3i lds_v3i;
__device__ __forceinline__ v3i lds_tr6(const uint8_t* p) {
    return __builtin_amdgcn_ds_read_tr6_b96_v3i32((lds_v3i*)(p));
}

}  // namespace mxc
#endif
