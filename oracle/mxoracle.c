/*
 * mxoracle.c -- CPU oracle for quantize-once MX convolution (MicroQonv).
 *
 * TEST INFRASTRUCTURE ONLY.  Nothing in the product path may link, load or
 * call this file: only the test suite, the smoke check and the CPU-baseline
 * leg of the benchmark do.  It shares no code, header, table or constant
 * with the GPU library; the only thing the two sides have in common is the
 * seeded input generator, which holds none of the method's arithmetic.
 *
 * Everything here is a plain, slow, obviously-correct definition written
 * in fp64 loops (OpenMP only splits the outermost loop of the big ones):
 *
 *   o_encode / o_decode   one element to/from FP8 E4M3, FP4 E2M1, FP6 E2M3
 *                         or FP6 E3M2 (OCP MX element formats; the paper's
 *                         number formats are introduced in Sec. II-D and
 *                         Sec. III-A; its FP6 variants: E3M2 activations
 *                         for MicroQonv+ in Sec. IV-D, E2M3 for the "-6"
 *                         methods in Sec. VI-B).
 *   o_quantize            microscaling quantizer, Sec. III-A Eqs. (4)-(6) in
 *                         its OCP-MX form: one E8M0 power-of-two scale per
 *                         square block (Sec. IV-B), elements rounded to
 *                         nearest-even with saturation.
 *   o_dequant             fake quantization: element value times the block
 *                         scale (Sec. III-A, below Eq. (6)).
 *   o_nvfp_quantize /     the paper's own two-level format, Eqs. (4)-(6)
 *   o_nvfp_dequant          literally: a per-tensor scale T, an FP8 E4M3
 *                         scale per 8x8 square block (Sec. IV-B: B = 64),
 *                         elements of any of the four element formats.
 *   o_quantize_sr         the same quantizer with stochastic rounding of the
 *                         elements, the option Eq. (6) offers and Sec. III-A
 *                         applies to gradients; random bits from
 *                         o_philox4x32_10 (Salmon et al., SC'11).
 *   o_im2col_cbf          channel-batch-first im2col applied to MX codes
 *                         (Sec. IV-A; Fig. 3).
 *   o_fwd / o_wgrad /     the three GEMMs of Sec. IV-B,
 *   o_dgrad                 Y_f = W_f X',  G_Wf = G_Yf X'^T,  G_X' = W_f^T G_Yf,
 *                         on dequantized operands, with the reordering back to
 *                         NCHW/OIHW (a col2im scatter-add for G_X').  Each
 *                         operand carries its own element format (MicroQonv+
 *                         pairs FP4 weights and gradients with FP6 activations).
 *   o_direct_*            brute-force definitions of Eqs. (1)-(3).
 *   o_*_at                single outputs of Eqs. (1)-(3), for sampled checks
 *                         at sizes where the full GEMMs are too slow.
 *   o_quantize_1d         the naive comparator's quantizer: 1-D blocks of 32
 *                         along one matrix direction (Sec. III-C, Dacapo).
 *   o_dequant_1d          its fake quantization.
 *   o_naive_im2col /      the naive comparator's fp32 im2col (channels-last
 *   o_naive_col2im          GEMM form) and the col2im scatter-add back.
 *
 * Readings of the paper that this file fixes (the paper uses NVFP with 8x8
 * blocks; the build uses OCP MX):
 *   - scale code = clamp(floor(log2 amax) - emax, -127, 127) + 127 where
 *     emax is 8 for E4M3, 2 for E2M1 and E2M3, 4 for E3M2; amax == 0 gives
 *     code 0; a block holding a NaN or infinity gets code 0xFF and all-zero
 *     element codes.
 *   - elements: x * 2^-s rounded to nearest, ties to even, magnitudes above
 *     the format maximum saturate (448, 6, 7.5 or 28); the sign of zero is
 *     kept.
 *   - block = 32 channels x Bn batch samples at one pixel, Bn = min(32, N);
 *     for weights 32 input channels x 32 output channels at one tap.
 *   - code layout [N/Bn][H][W][Cp][Bn] (Bn fastest), scales
 *     [N/Bn][H][W][Cp/32]; FP4 packs two consecutive codes per byte, the
 *     even one in the low nibble.  Cp = C rounded up to 32; padding is +0.
 *   - stochastic rounding (o_encode_sr): with lo <= |x| < hi the two
 *     neighbouring grid values and frac = (|x| - lo) / (hi - lo), the element
 *     becomes hi when r < frac * 2^16 for its 16 random bits r, else lo;
 *     grid values stay exact, magnitudes at or above the format maximum
 *     saturate, the scale rule is unchanged.  The bits of the code at linear
 *     position p: Philox4x32-10 with key (seed mod 2^32, seed / 2^32) and
 *     counter (p / 8 mod 2^32, p / 2^35, 0, 0) gives four words w0..w3;
 *     j = p mod 8 selects bits 16 (j mod 2) .. 16 (j mod 2) + 15 of w[j / 2].
 *   - NVFP (Eqs. (4)-(6)), every step one fp32 operation rounded to nearest
 *     even (the paper fixes no precision; its simulation runs in fp32):
 *     T = fl(amax / fl(448 * emax_val)) over the whole tensor (emax_val =
 *     the element format's largest value); per 8-channel x 8-sample block
 *     (weights: 8 Cin x 8 Cout) B = CastE4M3(fl(bmax / fl(T * emax_val)))
 *     with E4M3 rounding to nearest even, saturating at 448; element code =
 *     encode(fl(x / fl(B * T))) (round to nearest even, saturating).  T = 0
 *     or B = 0 gives zero codes.  A non-finite element anywhere makes T NaN,
 *     every block scale the E4M3 NaN code 0x7F and every element code 0.
 *     Codes use the MX-CBF code layout with Bn a multiple of 8 (n a multiple
 *     of 32, or 8 or 16); block scales are E4M3 bytes in the layout
 *     [Np/Bn][H][W][Cp/8][Bn/8].
 *   - FP6 codes are packed as one little-endian bit string: the code at
 *     linear position p occupies bits 6p .. 6p+5 (bit 0 = least significant
 *     bit of byte 0), so 32 samples of one channel take 24 bytes.  The same
 *     rule with 4 bits is the FP4 nibble order above.  FP6 activations need
 *     Bn >= 4 so that every channel row starts on a byte.
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>
#include <fenv.h>
#ifdef _OPENMP
#include <omp.h>
#endif

enum { O_E4M3 = 0, O_E2M1 = 1, O_E2M3 = 2, O_E3M2 = 3 };
enum { O_NCHW = 0, O_NHWC = 1, O_CBF = 2 };
enum { O_ACT = 0, O_WEIGHT = 1 };

/* ------------------------------------------------------------------ */
/* element formats                                                     */
/* ------------------------------------------------------------------ */
typedef struct {
    int bits, mbits, bias, emax;
    double maxval;      /* largest finite magnitude */
    double min_normal;  /* 2^(1-bias) */
    double quantum;     /* subnormal spacing 2^(1-bias-mbits) */
} o_fmt;

static int fmt_get(int fmt, o_fmt *f)
{
    if (fmt == O_E4M3) {
        f->bits = 8; f->mbits = 3; f->bias = 7; f->emax = 8;
        f->maxval = 448.0; f->min_normal = ldexp(1.0, -6); f->quantum = ldexp(1.0, -9);
        return 0;
    }
    if (fmt == O_E2M1) {
        f->bits = 4; f->mbits = 1; f->bias = 1; f->emax = 2;
        f->maxval = 6.0; f->min_normal = 1.0; f->quantum = 0.5;
        return 0;
    }
    if (fmt == O_E2M3) {                /* max 2^2 * 1.875, no inf / NaN */
        f->bits = 6; f->mbits = 3; f->bias = 1; f->emax = 2;
        f->maxval = 7.5; f->min_normal = 1.0; f->quantum = 0.125;
        return 0;
    }
    if (fmt == O_E3M2) {                /* max 2^4 * 1.75, no inf / NaN */
        f->bits = 6; f->mbits = 2; f->bias = 3; f->emax = 4;
        f->maxval = 28.0; f->min_normal = 0.25; f->quantum = 0.0625;
        return 0;
    }
    return -2;
}

/* Round v (already divided by the block scale) to the element format:
 * nearest value, ties to the even code, saturating, sign of zero kept.
 * The route is frexp + nearbyint in the default rounding mode, which is
 * round-half-to-even. */
int o_encode(double v, int fmt)
{
    o_fmt f;
    if (fmt_get(fmt, &f)) return -1;
    int sign = signbit(v) ? 1 : 0;
    double a = fabs(v);
    if (a > f.maxval) a = f.maxval;
    int code;
    if (a < f.min_normal) {
        code = (int)nearbyint(a / f.quantum);          /* 0 .. 2^mbits */
    } else {
        int e2;
        double m = frexp(a, &e2);                       /* a = m 2^e2, m in [0.5,1) */
        int ue = e2 - 1;                                /* a = (1+frac) 2^ue */
        double frac = m * 2.0 - 1.0;
        int q = (int)nearbyint(frac * (double)(1 << f.mbits));
        code = ((ue + f.bias) << f.mbits) + q;          /* q == 2^mbits carries */
    }
    return code | (sign << (f.bits - 1));
}

double o_decode(int code, int fmt)
{
    o_fmt f;
    if (fmt_get(fmt, &f)) return NAN;
    int sign = (code >> (f.bits - 1)) & 1;
    int mag = code & ((1 << (f.bits - 1)) - 1);
    if (fmt == O_E4M3 && mag == 0x7F) return NAN;
    int ef = mag >> f.mbits, mf = mag & ((1 << f.mbits) - 1);
    double v;
    if (ef == 0) v = mf * f.quantum;
    else v = ldexp(1.0 + (double)mf / (double)(1 << f.mbits), ef - f.bias);
    return sign ? -v : v;
}

/* E8M0 scale code -> 2^(code-127); 0xFF is NaN. */
double o_scale_value(int scode)
{
    if (scode == 0xFF) return NAN;
    return ldexp(1.0, scode - 127);
}

/* Scale code of a block with largest magnitude amax (finite). */
int o_scale_code(double amax, int fmt)
{
    o_fmt f;
    if (fmt_get(fmt, &f)) return -1;
    if (amax == 0.0) return 0;
    int e2;
    frexp(amax, &e2);
    int e = e2 - 1;                                  /* floor(log2 amax) */
    int s = e - f.emax;
    if (s < -127) s = -127;
    if (s > 127) s = 127;
    return s + 127;
}

/* Philox4x32-10 (Salmon, Moraes, Dror, Shaw, "Parallel random numbers: as
 * easy as 1, 2, 3", SC'11): ten rounds of two 32x32->64-bit products mixed
 * with the key, the key advanced by the Weyl constants between rounds. */
void o_philox4x32_10(const uint32_t ctr[4], const uint32_t key[2], uint32_t out[4])
{
    uint32_t c0 = ctr[0], c1 = ctr[1], c2 = ctr[2], c3 = ctr[3];
    uint32_t k0 = key[0], k1 = key[1];
    for (int round = 0; round < 10; round++) {
        if (round > 0) { k0 += 0x9E3779B9u; k1 += 0xBB67AE85u; }
        uint64_t p0 = (uint64_t)0xD2511F53u * c0;
        uint64_t p1 = (uint64_t)0xCD9E8D57u * c2;
        uint32_t n0 = (uint32_t)(p1 >> 32) ^ c1 ^ k0;
        uint32_t n1 = (uint32_t)p1;
        uint32_t n2 = (uint32_t)(p0 >> 32) ^ c3 ^ k1;
        uint32_t n3 = (uint32_t)p0;
        c0 = n0; c1 = n1; c2 = n2; c3 = n3;
    }
    out[0] = c0; out[1] = c1; out[2] = c2; out[3] = c3;
}

/* The 16 random bits of code position pos (see the header). */
unsigned o_sr_bits(uint64_t seed, int64_t pos)
{
    uint64_t q = (uint64_t)pos >> 3;
    uint32_t ctr[4] = {(uint32_t)q, (uint32_t)(q >> 32), 0u, 0u};
    uint32_t key[2] = {(uint32_t)seed, (uint32_t)(seed >> 32)};
    uint32_t w[4];
    o_philox4x32_10(ctr, key, w);
    int j = (int)(pos & 7);
    return (w[j >> 1] >> (16 * (j & 1))) & 0xFFFFu;
}

/* Stochastic rounding of v (already divided by the block scale) to the
 * element format, with the 16 random bits r. */
int o_encode_sr(double v, int fmt, unsigned r)
{
    o_fmt f;
    if (fmt_get(fmt, &f)) return -1;
    int neg = signbit(v) ? 1 : 0;
    double a = fabs(v);
    double pick;
    if (a >= f.maxval) {
        pick = f.maxval;
    } else {
        double q;                                       /* grid spacing at a */
        if (a < f.min_normal) {
            q = f.quantum;
        } else {
            int e2;
            frexp(a, &e2);                              /* a in [2^(e2-1), 2^e2) */
            q = ldexp(1.0, e2 - 1 - f.mbits);
        }
        double lo = floor(a / q) * q;                   /* exact: q is a power of two */
        double frac = (a - lo) / q;                     /* in [0, 1), exact */
        pick = ((double)r < frac * 65536.0) ? lo + q : lo;
    }
    return o_encode(neg ? -pick : pick, fmt);           /* pick is on the grid */
}

/* ------------------------------------------------------------------ */
/* tensor geometry of an MX tensor                                     */
/* ------------------------------------------------------------------ */
typedef struct { int n, c, h, w, bn, np, cp, bits; } o_geom;

static int geom_init(o_geom *g, int role, int fmt, int n, int c, int h, int w)
{
    o_fmt f;
    if (fmt_get(fmt, &f)) return -2;
    if (n <= 0 || c <= 0 || h <= 0 || w <= 0) return -2;
    g->n = n; g->c = c; g->h = h; g->w = w; g->bits = f.bits;
    g->cp = (c + 31) / 32 * 32;
    if (role == O_WEIGHT) {
        g->bn = 32;
        g->np = (n + 31) / 32 * 32;
    } else if (role == O_ACT) {
        if (n >= 32) {
            if (n % 32) return -3;
            g->bn = 32;
        } else {
            if (32 % n) return -3;
            g->bn = n;
        }
        g->np = n;
        if (fmt == O_E2M1 && g->bn == 1) return -3;
        if (f.bits == 6 && g->bn < 4) return -3;
    } else {
        return -2;
    }
    return 0;
}

int64_t o_codes_bytes(int role, int fmt, int n, int c, int h, int w)
{
    o_geom g;
    if (geom_init(&g, role, fmt, n, c, h, w)) return -1;
    int64_t elems = (int64_t)g.np * g.h * g.w * g.cp;
    return elems * g.bits / 8;
}

int64_t o_scales_bytes(int role, int fmt, int n, int c, int h, int w)
{
    o_geom g;
    if (geom_init(&g, role, fmt, n, c, h, w)) return -1;
    return (int64_t)(g.np / g.bn) * g.h * g.w * (g.cp / 32);
}

/* linear position of element (nb, hh, ww, cc, j) in the code array */
static int64_t code_pos(const o_geom *g, int nb, int hh, int ww, int cc, int j)
{
    return ((((int64_t)nb * g->h + hh) * g->w + ww) * g->cp + cc) * g->bn + j;
}

static int64_t scale_pos(const o_geom *g, int nb, int hh, int ww, int cb)
{
    return (((int64_t)nb * g->h + hh) * g->w + ww) * (g->cp / 32) + cb;
}

static void put_code(uint8_t *codes, int bits, int64_t pos, int code)
{
    if (bits == 8) { codes[pos] = (uint8_t)code; return; }
    if (bits == 6) {                    /* bit string, bit 6*pos + t = bit t of the code */
        for (int t = 0; t < 6; t++) {
            int64_t bit = 6 * pos + t;
            uint8_t m = (uint8_t)(1u << (bit & 7));
            if ((code >> t) & 1) codes[bit >> 3] |= m;
            else codes[bit >> 3] &= (uint8_t)~m;
        }
        return;
    }
    uint8_t *b = &codes[pos >> 1];
    if (pos & 1) *b = (uint8_t)((*b & 0x0F) | (code << 4));
    else         *b = (uint8_t)((*b & 0xF0) | (code & 0x0F));
}

static int get_code(const uint8_t *codes, int bits, int64_t pos)
{
    if (bits == 8) return codes[pos];
    if (bits == 6) {
        int code = 0;
        for (int t = 0; t < 6; t++) {
            int64_t bit = 6 * pos + t;
            code |= ((codes[bit >> 3] >> (bit & 7)) & 1) << t;
        }
        return code;
    }
    uint8_t b = codes[pos >> 1];
    return (pos & 1) ? (b >> 4) : (b & 0x0F);
}

/* value of logical element (n, c, h, w) of a float source in a layout */
static double src_at(const float *src, int layout, const o_geom *g, int n, int c, int h, int w)
{
    int64_t i;
    if (layout == O_NCHW)      i = (((int64_t)n * g->c + c) * g->h + h) * g->w + w;
    else if (layout == O_NHWC) i = (((int64_t)n * g->h + h) * g->w + w) * g->c + c;
    else {                                  /* [N/Bn][H][W][C][Bn], real C */
        int nb = n / g->bn, j = n % g->bn;
        i = ((((int64_t)nb * g->h + h) * g->w + w) * g->c + c) * g->bn + j;
    }
    return (double)src[i];
}

static int64_t o_quantized_count = 0;
int64_t o_counter_get(void) { return o_quantized_count; }
void o_counter_reset(void) { o_quantized_count = 0; }

void o_set_threads(int t)
{
#ifdef _OPENMP
    if (t > 0) omp_set_num_threads(t);
#else
    (void)t;
#endif
}

int o_get_threads(void)
{
#ifdef _OPENMP
    return omp_get_max_threads();
#else
    return 1;
#endif
}

/* Quantize a float tensor into MX-CBF codes and E8M0 scales.
 * src: logical (n, c, h, w) tensor in `layout` (weights: OIHW, i.e. NCHW
 * with n = Cout, c = Cin).  codes/scales sized by o_codes_bytes/o_scales_bytes.
 * Returns 0, or a negative error. */
static int quantize_impl(const float *src, int layout, int role, int fmt,
                         int n, int c, int h, int w, int sr, uint64_t seed,
                         uint8_t *codes, uint8_t *scales);

int o_quantize(const float *src, int layout, int role, int fmt,
               int n, int c, int h, int w, uint8_t *codes, uint8_t *scales)
{
    return quantize_impl(src, layout, role, fmt, n, c, h, w, 0, 0, codes, scales);
}

/* As o_quantize, with every element rounded stochastically (Eq. (6)'s
 * stochastic option) under `seed`. */
int o_quantize_sr(const float *src, int layout, int role, int fmt,
                  int n, int c, int h, int w, uint64_t seed, uint8_t *codes, uint8_t *scales)
{
    return quantize_impl(src, layout, role, fmt, n, c, h, w, 1, seed, codes, scales);
}

static int quantize_impl(const float *src, int layout, int role, int fmt,
                         int n, int c, int h, int w, int sr, uint64_t seed,
                         uint8_t *codes, uint8_t *scales)
{
    o_geom g;
    o_fmt f;
    int rc = geom_init(&g, role, fmt, n, c, h, w);
    if (rc) return rc;
    fmt_get(fmt, &f);
    if (layout < O_NCHW || layout > O_CBF) return -2;
    if (layout == O_CBF && role != O_ACT) return -2;
    int ngroups = g.np / g.bn, ncb = g.cp / 32;
    int64_t ntiles = (int64_t)ngroups * g.h * g.w * ncb;
    fesetround(FE_TONEAREST);
    #pragma omp parallel for schedule(static)
    for (int64_t t = 0; t < ntiles; t++) {
        int cb = (int)(t % ncb);
        int64_t r = t / ncb;
        int ww = (int)(r % g.w); r /= g.w;
        int hh = (int)(r % g.h);
        int nb = (int)(r / g.h);
        double vals[32][32];
        double amax = 0.0;
        int nonfinite = 0;
        for (int ci = 0; ci < 32; ci++) {
            for (int j = 0; j < g.bn; j++) {
                int nn = nb * g.bn + j, cc = cb * 32 + ci;
                double x = (nn < g.n && cc < g.c) ? src_at(src, layout, &g, nn, cc, hh, ww) : 0.0;
                vals[ci][j] = x;
                if (!isfinite(x)) nonfinite = 1;
                else if (fabs(x) > amax) amax = fabs(x);
            }
        }
        int scode = nonfinite ? 0xFF : o_scale_code(amax, fmt);
        scales[scale_pos(&g, nb, hh, ww, cb)] = (uint8_t)scode;
        int s = scode - 127;
        for (int ci = 0; ci < 32; ci++) {
            for (int j = 0; j < g.bn; j++) {
                int64_t pos = code_pos(&g, nb, hh, ww, cb * 32 + ci, j);
                int code = nonfinite ? 0
                         : sr ? o_encode_sr(ldexp(vals[ci][j], -s), fmt, o_sr_bits(seed, pos))
                              : o_encode(ldexp(vals[ci][j], -s), fmt);
                put_code(codes, g.bits, pos, code);
            }
        }
    }
    o_quantized_count += (int64_t)g.n * g.c * g.h * g.w;
    return 0;
}

/* Dequantize to a real-sized fp64 tensor (n, c, h, w) in NCHW order. */
int o_dequant(const uint8_t *codes, const uint8_t *scales, int role, int fmt,
              int n, int c, int h, int w, double *out)
{
    o_geom g;
    int rc = geom_init(&g, role, fmt, n, c, h, w);
    if (rc) return rc;
    #pragma omp parallel for schedule(static)
    for (int nn = 0; nn < n; nn++)
        for (int cc = 0; cc < c; cc++)
            for (int hh = 0; hh < h; hh++)
                for (int ww = 0; ww < w; ww++) {
                    int nb = nn / g.bn, j = nn % g.bn;
                    int code = get_code(codes, g.bits, code_pos(&g, nb, hh, ww, cc, j));
                    int sc = scales[scale_pos(&g, nb, hh, ww, cc / 32)];
                    out[(((int64_t)nn * c + cc) * h + hh) * w + ww] =
                        o_decode(code, fmt) * o_scale_value(sc);
                }
    return 0;
}

/* ------------------------------------------------------------------ */
/* NVFP, Eqs. (4)-(6) literally                                         */
/* ------------------------------------------------------------------ */
static int nvfp_geom(o_geom *g, int role, int fmt, int n, int c, int h, int w)
{
    int rc = geom_init(g, role, fmt, n, c, h, w);
    if (rc) return rc;
    if (g->bn % 8) return -3;                           /* 8x8 blocks */
    return 0;
}

int64_t o_nvfp_scales_bytes(int role, int fmt, int n, int c, int h, int w)
{
    o_geom g;
    if (nvfp_geom(&g, role, fmt, n, c, h, w)) return -1;
    return (int64_t)(g.np / g.bn) * g.h * g.w * (g.cp / 8) * (g.bn / 8);
}

static int64_t nvfp_scale_pos(const o_geom *g, int nb, int hh, int ww, int cb8, int sb8)
{
    return ((((int64_t)nb * g->h + hh) * g->w + ww) * (g->cp / 8) + cb8) * (g->bn / 8) + sb8;
}

/* Quantize into NVFP: codes (o_codes_bytes), E4M3 block scales
 * (o_nvfp_scales_bytes) and the per-tensor scale *tscale. */
int o_nvfp_quantize(const float *src, int layout, int role, int fmt, int n, int c, int h, int w,
                    uint8_t *codes, uint8_t *scales, float *tscale)
{
    o_geom g;
    o_fmt f;
    int rc = nvfp_geom(&g, role, fmt, n, c, h, w);
    if (rc) return rc;
    fmt_get(fmt, &f);
    if (layout < O_NCHW || layout > O_CBF) return -2;
    if (layout == O_CBF && role != O_ACT) return -2;
    const float emaxv = (float)f.maxval;
    /* Eq. (4): the per-tensor scale */
    float amax = 0.0f;
    int nonfinite = 0;
    for (int nn = 0; nn < n; nn++)
        for (int cc = 0; cc < c; cc++)
            for (int hh = 0; hh < h; hh++)
                for (int ww = 0; ww < w; ww++) {
                    float x = (float)src_at(src, layout, &g, nn, cc, hh, ww);
                    if (!isfinite(x)) nonfinite = 1;
                    else if (fabsf(x) > amax) amax = fabsf(x);
                }
    volatile float denom_t = 448.0f * emaxv;
    float T = nonfinite ? NAN : amax / denom_t;
    *tscale = T;
    volatile float tm = T * emaxv;                     /* T x max B_ef, rounded to fp32 */
    int ngroups = g.np / g.bn;
    for (int nb = 0; nb < ngroups; nb++)
      for (int hh = 0; hh < g.h; hh++)
        for (int ww = 0; ww < g.w; ww++)
          for (int cb8 = 0; cb8 < g.cp / 8; cb8++)
            for (int sb8 = 0; sb8 < g.bn / 8; sb8++) {
                float v[8][8];
                float bmax = 0.0f;
                for (int i = 0; i < 8; i++)
                    for (int j = 0; j < 8; j++) {
                        int nn = nb * g.bn + sb8 * 8 + j, cc = cb8 * 8 + i;
                        v[i][j] = (nn < g.n && cc < g.c) ? (float)src_at(src, layout, &g, nn, cc, hh, ww) : 0.0f;
                        if (fabsf(v[i][j]) > bmax) bmax = fabsf(v[i][j]);
                    }
                int bcode;
                float B = 0.0f;
                if (nonfinite) {
                    bcode = 0x7F;
                } else if (T == 0.0f) {
                    bcode = 0;
                } else {
                    volatile float ratio = bmax / tm;     /* Eq. (5), before the cast */
                    bcode = o_encode((double)ratio, O_E4M3);
                    B = (float)o_decode(bcode, O_E4M3);
                }
                scales[nvfp_scale_pos(&g, nb, hh, ww, cb8, sb8)] = (uint8_t)bcode;
                volatile float bt = B * T;                /* B_scale x T_scale, rounded to fp32 */
                for (int i = 0; i < 8; i++)
                    for (int j = 0; j < 8; j++) {
                        int code = 0;
                        if (!nonfinite && bt != 0.0f) {
                            volatile float q = v[i][j] / bt;   /* Eq. (6), before the rounding */
                            code = o_encode((double)q, fmt);
                        }
                        put_code(codes, g.bits, code_pos(&g, nb, hh, ww, cb8 * 8 + i, sb8 * 8 + j), code);
                    }
            }
    o_quantized_count += (int64_t)g.n * g.c * g.h * g.w;
    return 0;
}

/* Fake quantization: code value x B x T, exact in fp64, real-sized NCHW. */
int o_nvfp_dequant(const uint8_t *codes, const uint8_t *scales, float tscale, int role, int fmt,
                   int n, int c, int h, int w, double *out)
{
    o_geom g;
    int rc = nvfp_geom(&g, role, fmt, n, c, h, w);
    if (rc) return rc;
    for (int nn = 0; nn < n; nn++)
        for (int cc = 0; cc < c; cc++)
            for (int hh = 0; hh < h; hh++)
                for (int ww = 0; ww < w; ww++) {
                    int nb = nn / g.bn, j = nn % g.bn;
                    int code = get_code(codes, g.bits, code_pos(&g, nb, hh, ww, cc, j));
                    int b = scales[nvfp_scale_pos(&g, nb, hh, ww, cc / 8, j / 8)];
                    out[(((int64_t)nn * c + cc) * h + hh) * w + ww] =
                        o_decode(code, fmt) * o_decode(b, O_E4M3) * (double)tscale;
                }
    return 0;
}

/* ------------------------------------------------------------------ */
/* convolution geometry                                                */
/* ------------------------------------------------------------------ */
typedef struct { int n, cin, cout, h, w, kh, kw, sh, sw, ph, pw, ho, wo; } o_conv;

static int conv_init(o_conv *cv, const int *p)
{
    cv->n = p[0]; cv->cin = p[1]; cv->cout = p[2]; cv->h = p[3]; cv->w = p[4];
    cv->kh = p[5]; cv->kw = p[6]; cv->sh = p[7]; cv->sw = p[8]; cv->ph = p[9]; cv->pw = p[10];
    if (cv->n <= 0 || cv->cin <= 0 || cv->cout <= 0 || cv->h <= 0 || cv->w <= 0 ||
        cv->kh <= 0 || cv->kw <= 0 || cv->sh <= 0 || cv->sw <= 0 || cv->ph < 0 || cv->pw < 0)
        return -2;
    /* cross-correlation with zero padding, dilation 1 */
    cv->ho = (cv->h + 2 * cv->ph - cv->kh) / cv->sh + 1;
    cv->wo = (cv->w + 2 * cv->pw - cv->kw) / cv->sw + 1;
    if (cv->h + 2 * cv->ph < cv->kh || cv->w + 2 * cv->pw < cv->kw) return -3;
    return 0;
}

int o_conv_out(const int *p, int *ho, int *wo)
{
    o_conv cv;
    int rc = conv_init(&cv, p);
    if (rc) return rc;
    *ho = cv.ho; *wo = cv.wo;
    return 0;
}

/* Channel-batch-first im2col on MX codes (Sec. IV-A):
 *   X'[nb][ho][wo][kh][kw][c][j] = X[nb][ho*sh+kh-ph][wo*sw+kw-pw][c][j],
 * copying codes and the block's scale; taps that fall in the zero padding
 * become all-zero blocks with scale code 0 (the quantization of a +0 block). */
int o_im2col_cbf(const int *p, int fmt, const uint8_t *xcodes, const uint8_t *xscales,
                 uint8_t *ccodes, uint8_t *cscales)
{
    o_conv cv;
    o_geom gx, gc;
    int rc = conv_init(&cv, p);
    if (rc) return rc;
    if ((rc = geom_init(&gx, O_ACT, fmt, cv.n, cv.cin, cv.h, cv.w))) return rc;
    /* the im2col tensor viewed as an activation tensor with
     * H = Ho*Wo*Kh*Kw pixels and W = 1 */
    if ((rc = geom_init(&gc, O_ACT, fmt, cv.n, cv.cin, cv.ho * cv.wo * cv.kh * cv.kw, 1))) return rc;
    int ngroups = cv.n / gx.bn;
    for (int nb = 0; nb < ngroups; nb++)
      for (int oh = 0; oh < cv.ho; oh++)
        for (int ow = 0; ow < cv.wo; ow++)
          for (int a = 0; a < cv.kh; a++)
            for (int b = 0; b < cv.kw; b++) {
              int ih = oh * cv.sh + a - cv.ph, iw = ow * cv.sw + b - cv.pw;
              int inside = ih >= 0 && ih < cv.h && iw >= 0 && iw < cv.w;
              int pix = ((oh * cv.wo + ow) * cv.kh + a) * cv.kw + b;
              for (int cb = 0; cb < gx.cp / 32; cb++)
                cscales[scale_pos(&gc, nb, pix, 0, cb)] =
                    inside ? xscales[scale_pos(&gx, nb, ih, iw, cb)] : 0;
              for (int cc = 0; cc < gx.cp; cc++)
                for (int j = 0; j < gx.bn; j++)
                  put_code(ccodes, gc.bits, code_pos(&gc, nb, pix, 0, cc, j),
                           inside ? get_code(xcodes, gx.bits, code_pos(&gx, nb, ih, iw, cc, j)) : 0);
            }
    return 0;
}

int64_t o_im2col_codes_bytes(const int *p, int fmt)
{
    o_conv cv;
    if (conv_init(&cv, p)) return -1;
    return o_codes_bytes(O_ACT, fmt, cv.n, cv.cin, cv.ho * cv.wo * cv.kh * cv.kw, 1);
}

int64_t o_im2col_scales_bytes(const int *p, int fmt)
{
    o_conv cv;
    if (conv_init(&cv, p)) return -1;
    return o_scales_bytes(O_ACT, fmt, cv.n, cv.cin, cv.ho * cv.wo * cv.kh * cv.kw, 1);
}

/* ------------------------------------------------------------------ */
/* the three GEMMs of Sec. IV-B on dequantized operands                */
/* ------------------------------------------------------------------ */
/* Dequantized X' as a (Kh Kw Cin) x (Ho Wo N) matrix: row (kh, kw, ci) with
 * ci fastest, column (ho, wo, n) with n fastest (the paper's X'_{Cin,N}). */
static double *build_xcol(const o_conv *cv, int fmt, const uint8_t *xcodes, const uint8_t *xscales)
{
    int pp[11] = {cv->n, cv->cin, cv->cout, cv->h, cv->w, cv->kh, cv->kw, cv->sh, cv->sw, cv->ph, cv->pw};
    int64_t cb = o_im2col_codes_bytes(pp, fmt), sb = o_im2col_scales_bytes(pp, fmt);
    uint8_t *cc = (uint8_t *)calloc((size_t)cb, 1), *cs = (uint8_t *)calloc((size_t)sb, 1);
    int hcol = cv->ho * cv->wo * cv->kh * cv->kw;
    double *xd = (double *)malloc(sizeof(double) * (size_t)cv->n * cv->cin * hcol);
    int64_t K = (int64_t)cv->kh * cv->kw * cv->cin, NC = (int64_t)cv->ho * cv->wo * cv->n;
    double *xcol = (double *)malloc(sizeof(double) * (size_t)(K * NC));
    o_im2col_cbf(pp, fmt, xcodes, xscales, cc, cs);
    o_dequant(cc, cs, O_ACT, fmt, cv->n, cv->cin, hcol, 1, xd);     /* [n][ci][pix] */
    #pragma omp parallel for schedule(static)
    for (int64_t pix = 0; pix < (int64_t)cv->ho * cv->wo; pix++)
        for (int a = 0; a < cv->kh; a++)
            for (int b = 0; b < cv->kw; b++)
                for (int ci = 0; ci < cv->cin; ci++)
                    for (int nn = 0; nn < cv->n; nn++) {
                        int64_t row = ((int64_t)a * cv->kw + b) * cv->cin + ci;
                        int64_t col = pix * cv->n + nn;
                        int64_t p4 = (pix * cv->kh + a) * cv->kw + b;
                        xcol[row * NC + col] = xd[((int64_t)nn * cv->cin + ci) * hcol + p4];
                    }
    free(cc); free(cs); free(xd);
    return xcol;
}

/* W_f as Cout x (Kh Kw Cin), row-major. */
static double *build_wf(const o_conv *cv, int fmt, const uint8_t *wcodes, const uint8_t *wscales)
{
    double *wd = (double *)malloc(sizeof(double) * (size_t)cv->cout * cv->cin * cv->kh * cv->kw);
    o_dequant(wcodes, wscales, O_WEIGHT, fmt, cv->cout, cv->cin, cv->kh, cv->kw, wd);
    int64_t K = (int64_t)cv->kh * cv->kw * cv->cin;
    double *wf = (double *)malloc(sizeof(double) * (size_t)(cv->cout * K));
    for (int co = 0; co < cv->cout; co++)
        for (int ci = 0; ci < cv->cin; ci++)
            for (int a = 0; a < cv->kh; a++)
                for (int b = 0; b < cv->kw; b++)
                    wf[co * K + ((int64_t)a * cv->kw + b) * cv->cin + ci] =
                        wd[(((int64_t)co * cv->cin + ci) * cv->kh + a) * cv->kw + b];
    free(wd);
    return wf;
}

/* G_Yf as Cout x (Ho Wo N), row-major, column (ho, wo, n) with n fastest. */
static double *build_gyf(const o_conv *cv, int fmt, const uint8_t *gcodes, const uint8_t *gscales)
{
    int64_t NC = (int64_t)cv->ho * cv->wo * cv->n;
    double *gd = (double *)malloc(sizeof(double) * (size_t)(NC * cv->cout));
    o_dequant(gcodes, gscales, O_ACT, fmt, cv->n, cv->cout, cv->ho, cv->wo, gd);
    double *gf = (double *)malloc(sizeof(double) * (size_t)(NC * cv->cout));
    for (int nn = 0; nn < cv->n; nn++)
        for (int co = 0; co < cv->cout; co++)
            for (int oh = 0; oh < cv->ho; oh++)
                for (int ow = 0; ow < cv->wo; ow++)
                    gf[co * NC + ((int64_t)oh * cv->wo + ow) * cv->n + nn] =
                        gd[(((int64_t)nn * cv->cout + co) * cv->ho + oh) * cv->wo + ow];
    free(gd);
    return gf;
}

/* Forward: Y_f = W_f X', reordered to Y[n][co][ho][wo]; W in element format
 * wfmt, X in xfmt.  sabs (optional) receives sum_k |W_f[co][k] X'[k][col]|,
 * the scale of the rounding error. */
int o_fwd(const int *p, int wfmt, int xfmt, const uint8_t *wcodes, const uint8_t *wscales,
          const uint8_t *xcodes, const uint8_t *xscales, double *y, double *sabs)
{
    o_conv cv;
    o_geom g;
    int rc = conv_init(&cv, p);
    if (rc) return rc;
    if ((rc = geom_init(&g, O_ACT, xfmt, cv.n, cv.cin, cv.h, cv.w))) return rc;
    if ((rc = geom_init(&g, O_WEIGHT, wfmt, cv.cout, cv.cin, cv.kh, cv.kw))) return rc;
    double *xcol = build_xcol(&cv, xfmt, xcodes, xscales);
    double *wf = build_wf(&cv, wfmt, wcodes, wscales);
    int64_t K = (int64_t)cv.kh * cv.kw * cv.cin, NC = (int64_t)cv.ho * cv.wo * cv.n;
    #pragma omp parallel for schedule(dynamic)
    for (int co = 0; co < cv.cout; co++) {
        double *acc = (double *)calloc((size_t)NC, sizeof(double));
        double *aab = (double *)calloc((size_t)NC, sizeof(double));
        for (int64_t k = 0; k < K; k++) {
            double a = wf[co * K + k];
            const double *xr = &xcol[k * NC];
            for (int64_t col = 0; col < NC; col++) {
                acc[col] += a * xr[col];
                aab[col] += fabs(a * xr[col]);
            }
        }
        for (int64_t col = 0; col < NC; col++) {
            int nn = (int)(col % cv.n);
            int64_t pix = col / cv.n;
            int64_t o = ((int64_t)nn * cv.cout + co) * cv.ho * cv.wo + pix;
            y[o] = acc[col];
            if (sabs) sabs[o] = aab[col];
        }
        free(acc); free(aab);
    }
    free(xcol); free(wf);
    return 0;
}

/* Weight gradient: G_Wf = G_Yf X'^T, reordered to G_W[co][ci][kh][kw]; G_Y in
 * element format gfmt, X in xfmt. */
int o_wgrad(const int *p, int gfmt, int xfmt, const uint8_t *gcodes, const uint8_t *gscales,
            const uint8_t *xcodes, const uint8_t *xscales, double *gw, double *sabs)
{
    o_conv cv;
    o_geom g;
    int rc = conv_init(&cv, p);
    if (rc) return rc;
    if ((rc = geom_init(&g, O_ACT, xfmt, cv.n, cv.cin, cv.h, cv.w))) return rc;
    if ((rc = geom_init(&g, O_ACT, gfmt, cv.n, cv.cout, cv.ho, cv.wo))) return rc;
    double *xcol = build_xcol(&cv, xfmt, xcodes, xscales);
    double *gf = build_gyf(&cv, gfmt, gcodes, gscales);
    int64_t K = (int64_t)cv.kh * cv.kw * cv.cin, NC = (int64_t)cv.ho * cv.wo * cv.n;
    #pragma omp parallel for schedule(dynamic) collapse(2)
    for (int co = 0; co < cv.cout; co++)
        for (int64_t k = 0; k < K; k++) {
            double acc = 0.0, aab = 0.0;
            const double *gr = &gf[co * NC], *xr = &xcol[k * NC];
            for (int64_t col = 0; col < NC; col++) {
                acc += gr[col] * xr[col];
                aab += fabs(gr[col] * xr[col]);
            }
            int ci = (int)(k % cv.cin);
            int64_t tap = k / cv.cin;
            int a = (int)(tap / cv.kw), b = (int)(tap % cv.kw);
            int64_t o = (((int64_t)co * cv.cin + ci) * cv.kh + a) * cv.kw + b;
            gw[o] = acc;
            if (sabs) sabs[o] = aab;
        }
    free(xcol); free(gf);
    return 0;
}

/* Input gradient: G_X' = W_f^T G_Yf, then the col2im scatter-add that turns
 * the (Kh Kw Cin) x (Ho Wo N) matrix back into G_X[n][ci][h][w]; W in element
 * format wfmt, G_Y in gfmt. */
int o_dgrad(const int *p, int wfmt, int gfmt, const uint8_t *wcodes, const uint8_t *wscales,
            const uint8_t *gcodes, const uint8_t *gscales, double *gx, double *sabs)
{
    o_conv cv;
    o_geom g;
    int rc = conv_init(&cv, p);
    if (rc) return rc;
    if ((rc = geom_init(&g, O_ACT, gfmt, cv.n, cv.cout, cv.ho, cv.wo))) return rc;
    if ((rc = geom_init(&g, O_WEIGHT, wfmt, cv.cout, cv.cin, cv.kh, cv.kw))) return rc;
    double *wf = build_wf(&cv, wfmt, wcodes, wscales);
    double *gf = build_gyf(&cv, gfmt, gcodes, gscales);
    int64_t K = (int64_t)cv.kh * cv.kw * cv.cin, NC = (int64_t)cv.ho * cv.wo * cv.n;
    double *gcol = (double *)malloc(sizeof(double) * (size_t)(K * NC));
    double *scol = (double *)malloc(sizeof(double) * (size_t)(K * NC));
    #pragma omp parallel for schedule(dynamic)
    for (int64_t k = 0; k < K; k++) {
        double *acc = &gcol[k * NC], *aab = &scol[k * NC];
        for (int64_t col = 0; col < NC; col++) { acc[col] = 0.0; aab[col] = 0.0; }
        for (int co = 0; co < cv.cout; co++) {
            double a = wf[co * K + k];
            const double *gr = &gf[co * NC];
            for (int64_t col = 0; col < NC; col++) {
                acc[col] += a * gr[col];
                aab[col] += fabs(a * gr[col]);
            }
        }
    }
    int64_t nx = (int64_t)cv.n * cv.cin * cv.h * cv.w;
    for (int64_t i = 0; i < nx; i++) { gx[i] = 0.0; if (sabs) sabs[i] = 0.0; }
    /* col2im: parallel over (n, ci) rows, which own disjoint outputs */
    #pragma omp parallel for schedule(static) collapse(2)
    for (int nn = 0; nn < cv.n; nn++)
        for (int ci = 0; ci < cv.cin; ci++)
            for (int oh = 0; oh < cv.ho; oh++)
                for (int ow = 0; ow < cv.wo; ow++)
                    for (int a = 0; a < cv.kh; a++)
                        for (int b = 0; b < cv.kw; b++) {
                            int ih = oh * cv.sh + a - cv.ph, iw = ow * cv.sw + b - cv.pw;
                            if (ih < 0 || ih >= cv.h || iw < 0 || iw >= cv.w) continue;
                            int64_t k = ((int64_t)a * cv.kw + b) * cv.cin + ci;
                            int64_t col = ((int64_t)oh * cv.wo + ow) * cv.n + nn;
                            int64_t o = (((int64_t)nn * cv.cin + ci) * cv.h + ih) * cv.w + iw;
                            gx[o] += gcol[k * NC + col];
                            if (sabs) sabs[o] += scol[k * NC + col];
                        }
    free(wf); free(gf); free(gcol); free(scol);
    return 0;
}

/* ------------------------------------------------------------------ */
/* brute-force definitions, Eqs. (1)-(3), on fp64 NCHW tensors          */
/* ------------------------------------------------------------------ */
int o_direct_fwd(const int *p, const double *w, const double *x, double *y)
{
    o_conv cv;
    int rc = conv_init(&cv, p);
    if (rc) return rc;
    #pragma omp parallel for schedule(static) collapse(2)
    for (int nn = 0; nn < cv.n; nn++)
        for (int co = 0; co < cv.cout; co++)
            for (int oh = 0; oh < cv.ho; oh++)
                for (int ow = 0; ow < cv.wo; ow++) {
                    double s = 0.0;
                    for (int ci = 0; ci < cv.cin; ci++)
                        for (int a = 0; a < cv.kh; a++)
                            for (int b = 0; b < cv.kw; b++) {
                                int ih = oh * cv.sh + a - cv.ph, iw = ow * cv.sw + b - cv.pw;
                                if (ih < 0 || ih >= cv.h || iw < 0 || iw >= cv.w) continue;
                                s += w[(((int64_t)co * cv.cin + ci) * cv.kh + a) * cv.kw + b] *
                                     x[(((int64_t)nn * cv.cin + ci) * cv.h + ih) * cv.w + iw];
                            }
                    y[(((int64_t)nn * cv.cout + co) * cv.ho + oh) * cv.wo + ow] = s;
                }
    return 0;
}

/* G_X[n][ci][h][w] = sum over (co, kh, kw, ho, wo) with ho*sh+kh-ph == h and
 * wo*sw+kw-pw == w of W[co][ci][kh][kw] G_Y[n][co][ho][wo] (Eq. (2): the
 * convolution of G_Y with the channel-swapped kernel). */
int o_direct_dgrad(const int *p, const double *w, const double *gy, double *gx)
{
    o_conv cv;
    int rc = conv_init(&cv, p);
    if (rc) return rc;
    #pragma omp parallel for schedule(static) collapse(2)
    for (int nn = 0; nn < cv.n; nn++)
        for (int ci = 0; ci < cv.cin; ci++)
            for (int ih = 0; ih < cv.h; ih++)
                for (int iw = 0; iw < cv.w; iw++) {
                    double s = 0.0;
                    for (int co = 0; co < cv.cout; co++)
                        for (int a = 0; a < cv.kh; a++)
                            for (int b = 0; b < cv.kw; b++) {
                                int th = ih + cv.ph - a, tw = iw + cv.pw - b;
                                if (th < 0 || tw < 0 || th % cv.sh || tw % cv.sw) continue;
                                int oh = th / cv.sh, ow = tw / cv.sw;
                                if (oh >= cv.ho || ow >= cv.wo) continue;
                                s += w[(((int64_t)co * cv.cin + ci) * cv.kh + a) * cv.kw + b] *
                                     gy[(((int64_t)nn * cv.cout + co) * cv.ho + oh) * cv.wo + ow];
                            }
                    gx[(((int64_t)nn * cv.cin + ci) * cv.h + ih) * cv.w + iw] = s;
                }
    return 0;
}

int o_direct_wgrad(const int *p, const double *gy, const double *x, double *gw)
{
    o_conv cv;
    int rc = conv_init(&cv, p);
    if (rc) return rc;
    #pragma omp parallel for schedule(static) collapse(2)
    for (int co = 0; co < cv.cout; co++)
        for (int ci = 0; ci < cv.cin; ci++)
            for (int a = 0; a < cv.kh; a++)
                for (int b = 0; b < cv.kw; b++) {
                    double s = 0.0;
                    for (int nn = 0; nn < cv.n; nn++)
                        for (int oh = 0; oh < cv.ho; oh++)
                            for (int ow = 0; ow < cv.wo; ow++) {
                                int ih = oh * cv.sh + a - cv.ph, iw = ow * cv.sw + b - cv.pw;
                                if (ih < 0 || ih >= cv.h || iw < 0 || iw >= cv.w) continue;
                                s += gy[(((int64_t)nn * cv.cout + co) * cv.ho + oh) * cv.wo + ow] *
                                     x[(((int64_t)nn * cv.cin + ci) * cv.h + ih) * cv.w + iw];
                            }
                    gw[(((int64_t)co * cv.cin + ci) * cv.kh + a) * cv.kw + b] = s;
                }
    return 0;
}

/* ------------------------------------------------------------------ */
/* single outputs, straight from the MX codes (sampled checks)         */
/* ------------------------------------------------------------------ */
static double mx_elem(const uint8_t *codes, const uint8_t *scales, const o_geom *g, int fmt,
                      int nn, int cc, int hh, int ww)
{
    int nb = nn / g->bn, j = nn % g->bn;
    int code = get_code(codes, g->bits, code_pos(g, nb, hh, ww, cc, j));
    return o_decode(code, fmt) * o_scale_value(scales[scale_pos(g, nb, hh, ww, cc / 32)]);
}

/* idx: cnt x 4 ints (n, co, ho, wo); out/sabs: cnt doubles */
int o_fwd_at(const int *p, int wfmt, int xfmt, const uint8_t *wcodes, const uint8_t *wscales,
             const uint8_t *xcodes, const uint8_t *xscales, const int *idx, int64_t cnt,
             double *out, double *sabs)
{
    o_conv cv;
    o_geom gw, gx;
    int rc = conv_init(&cv, p);
    if (rc) return rc;
    if ((rc = geom_init(&gw, O_WEIGHT, wfmt, cv.cout, cv.cin, cv.kh, cv.kw))) return rc;
    if ((rc = geom_init(&gx, O_ACT, xfmt, cv.n, cv.cin, cv.h, cv.w))) return rc;
    #pragma omp parallel for schedule(dynamic)
    for (int64_t i = 0; i < cnt; i++) {
        int nn = idx[4 * i], co = idx[4 * i + 1], oh = idx[4 * i + 2], ow = idx[4 * i + 3];
        double s = 0.0, sa = 0.0;
        for (int ci = 0; ci < cv.cin; ci++)
            for (int a = 0; a < cv.kh; a++)
                for (int b = 0; b < cv.kw; b++) {
                    int ih = oh * cv.sh + a - cv.ph, iw = ow * cv.sw + b - cv.pw;
                    if (ih < 0 || ih >= cv.h || iw < 0 || iw >= cv.w) continue;
                    double t = mx_elem(wcodes, wscales, &gw, wfmt, co, ci, a, b) *
                               mx_elem(xcodes, xscales, &gx, xfmt, nn, ci, ih, iw);
                    s += t; sa += fabs(t);
                }
        out[i] = s; sabs[i] = sa;
    }
    return 0;
}

/* idx: cnt x 4 ints (n, ci, h, w) */
int o_dgrad_at(const int *p, int wfmt, int gfmt, const uint8_t *wcodes, const uint8_t *wscales,
               const uint8_t *gcodes, const uint8_t *gscales, const int *idx, int64_t cnt,
               double *out, double *sabs)
{
    o_conv cv;
    o_geom gw, gg;
    int rc = conv_init(&cv, p);
    if (rc) return rc;
    if ((rc = geom_init(&gw, O_WEIGHT, wfmt, cv.cout, cv.cin, cv.kh, cv.kw))) return rc;
    if ((rc = geom_init(&gg, O_ACT, gfmt, cv.n, cv.cout, cv.ho, cv.wo))) return rc;
    #pragma omp parallel for schedule(dynamic)
    for (int64_t i = 0; i < cnt; i++) {
        int nn = idx[4 * i], ci = idx[4 * i + 1], ih = idx[4 * i + 2], iw = idx[4 * i + 3];
        double s = 0.0, sa = 0.0;
        for (int co = 0; co < cv.cout; co++)
            for (int a = 0; a < cv.kh; a++)
                for (int b = 0; b < cv.kw; b++) {
                    int th = ih + cv.ph - a, tw = iw + cv.pw - b;
                    if (th < 0 || tw < 0 || th % cv.sh || tw % cv.sw) continue;
                    int oh = th / cv.sh, ow = tw / cv.sw;
                    if (oh >= cv.ho || ow >= cv.wo) continue;
                    double t = mx_elem(wcodes, wscales, &gw, wfmt, co, ci, a, b) *
                               mx_elem(gcodes, gscales, &gg, gfmt, nn, co, oh, ow);
                    s += t; sa += fabs(t);
                }
        out[i] = s; sabs[i] = sa;
    }
    return 0;
}

/* idx: cnt x 4 ints (co, ci, kh, kw) */
int o_wgrad_at(const int *p, int gfmt, int xfmt, const uint8_t *gcodes, const uint8_t *gscales,
               const uint8_t *xcodes, const uint8_t *xscales, const int *idx, int64_t cnt,
               double *out, double *sabs)
{
    o_conv cv;
    o_geom gx, gg;
    int rc = conv_init(&cv, p);
    if (rc) return rc;
    if ((rc = geom_init(&gx, O_ACT, xfmt, cv.n, cv.cin, cv.h, cv.w))) return rc;
    if ((rc = geom_init(&gg, O_ACT, gfmt, cv.n, cv.cout, cv.ho, cv.wo))) return rc;
    #pragma omp parallel for schedule(dynamic)
    for (int64_t i = 0; i < cnt; i++) {
        int co = idx[4 * i], ci = idx[4 * i + 1], a = idx[4 * i + 2], b = idx[4 * i + 3];
        double s = 0.0, sa = 0.0;
        for (int nn = 0; nn < cv.n; nn++)
            for (int oh = 0; oh < cv.ho; oh++)
                for (int ow = 0; ow < cv.wo; ow++) {
                    int ih = oh * cv.sh + a - cv.ph, iw = ow * cv.sw + b - cv.pw;
                    if (ih < 0 || ih >= cv.h || iw < 0 || iw >= cv.w) continue;
                    double t = mx_elem(gcodes, gscales, &gg, gfmt, nn, co, oh, ow) *
                               mx_elem(xcodes, xscales, &gx, xfmt, nn, ci, ih, iw);
                    s += t; sa += fabs(t);
                }
        out[i] = s; sabs[i] = sa;
    }
    return 0;
}

/* ------------------------------------------------------------------ */
/* naive comparator's quantizer (Sec. III-C: quantize in line blocks)   */
/* ------------------------------------------------------------------ */
/* m: rows x cols fp32 matrix, row-major.  dir 0: blocks of 32 consecutive
 * elements along a row (the last block of a row is short if cols % 32);
 * dir 1: blocks of 32 consecutive elements down a column.  codes: one
 * code per element at the element's own position (FP4: two per byte,
 * even position low); scales: dir 0 -> [rows][ceil(cols/32)],
 * dir 1 -> [ceil(rows/32)][cols]. */
int o_quantize_1d(const float *m, int64_t rows, int64_t cols, int dir, int fmt,
                  uint8_t *codes, uint8_t *scales)
{
    o_fmt f;
    if (fmt_get(fmt, &f)) return -2;
    if (rows <= 0 || cols <= 0 || (dir != 0 && dir != 1)) return -2;
    int64_t nbr = dir == 0 ? rows : (rows + 31) / 32;
    int64_t nbc = dir == 0 ? (cols + 31) / 32 : cols;
    /* codes are produced one per element and packed afterwards: two FP4
     * codes of different blocks can share a byte */
    uint8_t *one = (uint8_t *)malloc((size_t)(rows * cols));
    if (!one) return -1;
    fesetround(FE_TONEAREST);
    #pragma omp parallel for schedule(static)
    for (int64_t bi = 0; bi < nbr * nbc; bi++) {
        int64_t br = bi / nbc, bc = bi % nbc;
        int64_t pos[32];
        int cnt = 0;
        for (int t = 0; t < 32; t++) {
            int64_t r = dir == 0 ? br : br * 32 + t;
            int64_t c = dir == 0 ? bc * 32 + t : bc;
            if (r < rows && c < cols) pos[cnt++] = r * cols + c;
        }
        double amax = 0.0;
        int nonfinite = 0;
        for (int t = 0; t < cnt; t++) {
            double x = m[pos[t]];
            if (!isfinite(x)) nonfinite = 1;
            else if (fabs(x) > amax) amax = fabs(x);
        }
        int scode = nonfinite ? 0xFF : o_scale_code(amax, fmt);
        scales[bi] = (uint8_t)scode;
        for (int t = 0; t < cnt; t++) {
            int code = nonfinite ? 0 : o_encode(ldexp((double)m[pos[t]], -(scode - 127)), fmt);
            one[pos[t]] = (uint8_t)code;
        }
    }
    for (int64_t i = 0; i < rows * cols; i++) put_code(codes, f.bits, i, one[i]);
    free(one);
    o_quantized_count += rows * cols;
    return 0;
}

/* ------------------------------------------------------------------ */
/* naive comparator (Sec. III-C; the baseline column of Table I): the  */
/* full-precision im2col comes first and every GEMM operand is then    */
/* quantized with 1-D blocks of 32 along its contraction dimension     */
/* ------------------------------------------------------------------ */

/* Fake quantization of a matrix quantized by o_quantize_1d (same layouts:
 * codes in the matrix's own row-major order, scales [rows][ceil(cols/32)]
 * for dir 0 and [ceil(rows/32)][cols] for dir 1). */
int o_dequant_1d(const uint8_t *codes, const uint8_t *scales, int64_t rows, int64_t cols,
                 int dir, int fmt, double *out)
{
    o_fmt f;
    if (fmt_get(fmt, &f)) return -2;
    if (rows <= 0 || cols <= 0 || (dir != 0 && dir != 1)) return -2;
    int64_t nbc = (cols + 31) / 32;
    for (int64_t r = 0; r < rows; r++)
        for (int64_t c = 0; c < cols; c++) {
            int64_t bi = dir == 0 ? r * nbc + c / 32 : (r / 32) * cols + c;
            int64_t pos = r * cols + c;
            out[pos] = o_decode(get_code(codes, f.bits, pos), fmt) * o_scale_value(scales[bi]);
        }
    return 0;
}

/* fp32 im2col in channels-last GEMM form: col[p][k] with p = (n, ho, wo)
 * and k = (kh, kw, ci), x in NHWC.  col[p][k] = x[n][ho*sh+kh-ph][wo*sw+kw-pw][ci],
 * zero where the tap falls into the padding. */
int o_naive_im2col(const int *p, const float *x, float *col)
{
    o_conv cv;
    int rc = conv_init(&cv, p);
    if (rc) return rc;
    int64_t K = (int64_t)cv.kh * cv.kw * cv.cin;
    for (int nn = 0; nn < cv.n; nn++)
        for (int oh = 0; oh < cv.ho; oh++)
            for (int ow = 0; ow < cv.wo; ow++) {
                int64_t row = ((int64_t)nn * cv.ho + oh) * cv.wo + ow;
                for (int a = 0; a < cv.kh; a++)
                    for (int b = 0; b < cv.kw; b++)
                        for (int ci = 0; ci < cv.cin; ci++) {
                            int ih = oh * cv.sh + a - cv.ph, iw = ow * cv.sw + b - cv.pw;
                            int inside = ih >= 0 && ih < cv.h && iw >= 0 && iw < cv.w;
                            int64_t k = ((int64_t)a * cv.kw + b) * cv.cin + ci;
                            col[row * K + k] = inside ? x[(((int64_t)nn * cv.h + ih) * cv.w + iw) * cv.cin + ci]
                                                      : 0.0f;
                        }
            }
    return 0;
}

/* col2im: G_X[n][h][w][ci] (NHWC) = sum of gcol[p][k] over every (p, k) that
 * o_naive_im2col reads from (n, h, w, ci) -- the scatter-add that turns
 * G_X' back into G_X (Sec. IV-B). */
int o_naive_col2im(const int *p, const double *gcol, double *gx)
{
    o_conv cv;
    int rc = conv_init(&cv, p);
    if (rc) return rc;
    int64_t K = (int64_t)cv.kh * cv.kw * cv.cin;
    int64_t nx = (int64_t)cv.n * cv.h * cv.w * cv.cin;
    for (int64_t i = 0; i < nx; i++) gx[i] = 0.0;
    for (int nn = 0; nn < cv.n; nn++)
        for (int oh = 0; oh < cv.ho; oh++)
            for (int ow = 0; ow < cv.wo; ow++) {
                int64_t row = ((int64_t)nn * cv.ho + oh) * cv.wo + ow;
                for (int a = 0; a < cv.kh; a++)
                    for (int b = 0; b < cv.kw; b++) {
                        int ih = oh * cv.sh + a - cv.ph, iw = ow * cv.sw + b - cv.pw;
                        if (ih < 0 || ih >= cv.h || iw < 0 || iw >= cv.w) continue;
                        for (int ci = 0; ci < cv.cin; ci++) {
                            int64_t k = ((int64_t)a * cv.kw + b) * cv.cin + ci;
                            gx[(((int64_t)nn * cv.h + ih) * cv.w + iw) * cv.cin + ci] += gcol[row * K + k];
                        }
                    }
            }
    return 0;
}
