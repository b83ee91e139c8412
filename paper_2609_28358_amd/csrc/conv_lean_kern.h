// conv_lean_kern.h -- the lean forward / input-gradient kernels (a3 / a4 for
// the common layer shapes) and their launch templates, shared by the
// translation units that instantiate them: one per element format and
// direction (conv_lean_*.hip), so that they compile in parallel;
// conv_lean.hip plans a launch (tile shape, stage layout, ring depth) and
// calls the one that serves its formats.
//
// Forward (Sec. II-C, Y_f = W_f X') and input gradient (G_X' = W_f^T G_Yf folded back by col2im,
// computed as a gather) on MX-CBF operands with a batch block of 32, kernel
// width 1 or 3; forward with column stride 1 or 2 (any row stride), input
// gradient with stride 1 or 2 x 2.
//
// Stride-2 input gradient: the output pixels split into four phases (row
// parity ry, column parity rx).  A phase only meets the taps whose offset has
// its parity, kh = kh0 + 2 i and kw = kw0 + 2 j, and its pixel (ry + 2 yi,
// rx + 2 xi) reads G_Y at row yi + (ry + ph - kh) / 2 and column
// xi + (rx + pw - kw) / 2: on the phase's own pixel grid that is a stride-1
// gather with ceil((K - k0) / 2) taps per dimension, which is the stride-1
// kernel with a smaller kernel.  One launch covers the four phases.
//
// One workgroup (4 waves) computes a tile of BM = 64*WGM output channels x
// PX = 4*PW/WGM output pixels of one output row x 32 samples; each wave owns
// 64 channels x PW pixels (2 x PW MFMAs of 32 x 32 x 64 per tap and K step).
// The K loop runs over stages (kernel row, pair of 32-channel blocks).  A
// stage holds, in LDS, the weight blocks of its kernel row ([tap][block]
// [row block]) and the source pixels its taps reach in that row (the halo:
// [block][pixel]), both as whole stored blocks.  They are streamed with
// global_load_lds (16 bytes per lane straight into LDS): each wave
// instruction moves one 1 KB slice; every lane's source offset is fixed for
// the tile and a stage adds one uniform delta; padding taps and missing
// blocks read a zero block through a select, not a branch.  The E8M0
// scales of a stage stream the same way, one byte per lane.  Stages rotate
// through a ring of 2 to 4 LDS buffers: while one stage computes, the next
// ones stream in (the host picks the ring depth from the LDS left per
// workgroup at the layer's occupancy).
// The fragments of each source pixel are read from LDS once per stage and
// reused by every tap that reaches it.  The MFMAs compute the transposed
// tile (samples x channels) so that each lane ends up holding four
// consecutive samples of one channel: one 16-byte store in the CBF layout.
#pragma once

#include <atomic>

#include "mx_internal.h"

namespace mxc {
#include "wgrad_tile.h"

struct LeanArgs {
    const uint8_t* wc;        // weight codes / scales
    const uint8_t* ws;
    const uint8_t* sc;        // source activation codes / scales (X or G_Y)
    const uint8_t* ss;
    float* out;
    int layout;
    int M;                    // real output channels
    int mtiles;               // row tiles
    int hout, wout;           // output spatial size
    int hsrc, wsrc;           // source spatial size
    int kh, sh, ph, pw;       // kernel rows, row stride, padding
    int kcb;                  // 32-channel blocks of the source (K blocks per tap)
    int w_rowblocks;          // valid 32-row blocks of the weight operand
    int w_cp;                 // weight Cin_p
    int w_ncb;                // weight scale blocks per tap (Cin_p / 32)
    int w_nco;                // weight Cout_p / 32
    int x_ncb;                // source scale blocks per pixel
    int ntiles;
    int stage_bytes;          // bytes between stage buffers
    int nbuf;                 // ring depth, 2..4
    int kwf;                  // full kernel width
    int pofs[5];              // stride-2 input gradient: first tile of each phase (ry, rx) = 00, 01, 10, 11
    // fused quantizing epilogue (qcodes != NULL): the output tile, after the
    // activation (forward) or the activation's derivative at zpre (input
    // gradient), is quantized into the MX-CBF tensor (qcodes, qscales) of
    // format qfmt with q_ncb 32-channel blocks per pixel; `out`, if not NULL,
    // receives the fp32 values that were quantized (CBF layout)
    uint8_t* qcodes;
    uint8_t* qscales;
    int qfmt, q_ncb, fn;
    int pre_out;              // forward: `out` receives the values before the activation
    int bf16;                 // the GEMM result is rounded to bf16 first; zpre and the pre_out output are bf16
    int xrows;                // real channel rows of the source's blocks (its channels if it has one block, else 32)
    int zoff;                 // > 0: the fused input gradient's bf16 z tiles are prefetched to LDS at this offset
    int zpw, zrb;             // (host) the tile shape the z region is sized for
    int zsl;                  // 1 KB slots of 16 rows per z tile: 1 if the layer has at most 16 rows, else 2
    const void* zpre;
    int sr;                   // fused epilogue: codes by stochastic rounding, generator key (sk0, sk1)
    uint32_t sk0, sk1;
    // NVFP4 operands (the NV kernels): per-tensor scales of W and the source;
    // the scale arrays ws / ss then hold E4M3 scales per 8x8 block, the 16 of
    // one 32-row block in 16 consecutive bytes
    const float* tw;
    const float* tx;
};

// Taps and output pixel grid of one phase; the stride-1 kernels use the
// trivial phase (every tap, every pixel).
struct Phase {
    int ry, rx;               // output row / column parity
    int kh0, nvh;             // first kernel row, kernel rows
    int kw0;                  // first kernel column
    int gh, gw;               // output rows / columns of the phase
    int c0;                   // G_Y column of phase column 0 for kernel column kw0
    int r0;                   // G_Y row of phase row 0 for kernel row kh0
};

// The tile shape of one launch, as the host planned it.
struct LeanShape {
    int kw, sw;               // kernel width, column stride
    int wgm, pw, rb;          // row groups, pixels per wave, 32-row blocks per wave
    bool kr;                  // stages pair kernel rows
    int nb;                   // stage buffers in use
};

namespace {


constexpr int LT = 256;

__device__ __attribute__((aligned(16))) uint8_t g_zero_lean[1024];

// LDS of one stage: NQ 4 KB groups of DMA slices (weight blocks, then halo
// blocks), then 1 KB of scale entries (entry e at byte 4 e: one dword per
// lane of the one-byte copies).
constexpr int SCALE_REGION = 1024;
constexpr int LDS_MAX = 160 * 1024;       // LDS of one CU



// One tile.  DG with S = 2 is a phase of the stride-2 input gradient and KW
// its taps per row (the halo is then a stride-1 one on the phase grid).
// Each wave owns 64 channels x PW pixels (PW = 2, or 1 for layers with few
// tiles: twice the workgroups, so more waves stream and store at once).
//
// Element formats: FW of the weights, FX of the source activation.  A stored
// block is 32 rows x 32 codes: 1024 bytes (FP8), 768 (FP6) or 512 (FP4).  In
// LDS an FP8 or FP4 block keeps its stored layout; an FP6 block takes 1 KB,
// each 12-byte half row (16 codes) at the start of its own 16-byte slot --
// the alignment the 6-bit transposing read needs.  One wave copy
// instruction moves 1 KB of LDS: two FP4 blocks, or one FP8 block, or one
// FP6 block with lane j reading the 16 bytes at 12 j (the last 4 of them
// belong to the next half row and are never read back).
// bf16 tiles of one output block (32 channels x 32 samples at one pixel: 2 KB
// contiguous in the CBF layout, 64 bytes per channel row) pass through 2 KB of
// LDS per wave, so that global memory sees whole 1 KB runs of 16 bytes per
// lane rather than the accumulator layout's 8-byte pieces of 32 rows (twice
// the rows touched per instruction, and four times the instructions per
// block).  The 16-byte chunk c of row r sits at r * 64 + ((c ^ ((r / 2) % 4))
// * 16): rows two apart land on different chunks.
__device__ __forceinline__ int bf16_lds(int row, int chunk) { return row * 64 + ((chunk ^ ((row >> 1) & 3)) << 4); }

// v *= fn'(z) for the lane's 16 values, z from a bf16 tile in LDS (zero where
// zr is false), at most four values in flight
template <int F>
__device__ __forceinline__ void grad_lds4(float* v, const uint8_t* zt, bool zr, int r, int h) {
#pragma unroll
    for (int e4 = 0; e4 < 4; e4++) {
        const float4 z = zr ? bf16_unpack4(*(const uint2*)(zt + bf16_lds(r, e4) + 8 * h)) : make_float4(0.f, 0.f, 0.f, 0.f);
        v[4 * e4] *= fn_grad_c<F>(z.x);
        v[4 * e4 + 1] *= fn_grad_c<F>(z.y);
        v[4 * e4 + 2] *= fn_grad_c<F>(z.z);
        v[4 * e4 + 3] *= fn_grad_c<F>(z.w);
        __builtin_amdgcn_sched_barrier(0);
    }
}

// Lane (r, h) = (lane % 32, lane / 32) holds samples 8 e4 + 4 h .. + 3 of row r
// in v[4 e4 .. 4 e4 + 3] (the MFMA accumulator layout).  Rows >= rows are
// not written.
__device__ __forceinline__ void store_bf16_tile(uint8_t* lds, const float* v, uint16_t* dst, int rows, int lane) {
    const int r = lane & 31, h = lane >> 5;
#pragma unroll
    for (int e4 = 0; e4 < 4; e4++)
        *(uint2*)(lds + bf16_lds(r, e4) + 8 * h) = bf16_pack4(v[4 * e4], v[4 * e4 + 1], v[4 * e4 + 2], v[4 * e4 + 3]);
#pragma unroll
    for (int i = 0; i < 2; i++) {
        const int k = lane + 64 * i, row = k >> 2, c = k & 3;
        const uint4 d = *(const uint4*)(lds + bf16_lds(row, c));
        if (row < rows) store_nt(dst + row * 32 + c * 8, d);
    }
}

// The inverse: z[4 e4 .. 4 e4 + 3] of lane (r, h) = samples 8 e4 + 4 h .. + 3
// of row r of the bf16 tile at src, as floats; rows >= rows read as 0.
__device__ __forceinline__ void load_bf16_tile(uint8_t* lds, const uint16_t* src, int rows, int lane, float* z) {
#pragma unroll
    for (int i = 0; i < 2; i++) {
        const int k = lane + 64 * i, row = k >> 2, c = k & 3;
        uint4 d = make_uint4(0u, 0u, 0u, 0u);
        if (row < rows) {   // 16 bytes moved as four fp32 lanes: bits only, no arithmetic
            const float4 f = load_nt((const float*)(src + row * 32 + c * 8));
            d = make_uint4(__float_as_uint(f.x), __float_as_uint(f.y), __float_as_uint(f.z), __float_as_uint(f.w));
        }
        *(uint4*)(lds + bf16_lds(row, c)) = d;
    }
    const int r = lane & 31, h = lane >> 5;
#pragma unroll
    for (int e4 = 0; e4 < 4; e4++) {
        const float4 f = bf16_unpack4(*(const uint2*)(lds + bf16_lds(r, e4) + 8 * h));
        z[4 * e4] = f.x; z[4 * e4 + 1] = f.y; z[4 * e4 + 2] = f.z; z[4 * e4 + 3] = f.w;
    }
}

template <int F> struct LdsBlock {
    static constexpr int TBG = 32 * 32 * fmt_bits(F) / 8;        // stored block bytes
    static constexpr int TBL = F == MXC_E2M1 ? 512 : 1024;       // LDS block bytes
    static constexpr int BPI = 1024 / TBL;                       // blocks per copy instruction
    static constexpr int STEP = fmt_bits(F) == 6 ? 12 : 16;      // source bytes between lanes
};

// NV: NVFP4 operands (both E2M1 codes with E4M3 8x8 block scales and a
// per-tensor scale, Eqs. (4)-(6)): a stage also carries the 16 block scales of
// each 32-row block it holds (4 KB of scale entries instead of 1 KB), the
// fragments are decoded to fp16 and multiplied on fp16 MFMAs, and the result
// is multiplied by the two per-tensor scales.
// Q: the kernel may run the fused quantizing epilogue (p.qcodes); the
// grouped backward kernel never does and compiles it out.
template <int FW, int FX, bool DG, int KW, int S, int WGM, int PW, bool NV = false, int NRB = 2, bool KR = false,
          bool Q = true>
__device__ __forceinline__ void lean_tile(const LeanArgs& p, int lin, const Phase& f) {
    static_assert(!NV || (FW == FX && FW != MXC_E3M2) || (FW == MXC_E2M1 && FX == MXC_E3M2),
                  "NVFP pairs: one format (FP4, E2M3, FP8), or FP4 weights with E3M2 activations");
    // X8: MXFP8 operands, decoded once per fragment to bf16 (exact products,
    // fp32 accumulation); NV or X8: the products run on decoded fragments
    // (NVFP8 on bf16 MFMAs, NVFP4 / NVFP6 on fp16 MFMAs)
    constexpr bool X8 = FX == MXC_E4M3 && !NV;
    constexpr bool NV8 = NV && FX == MXC_E4M3;
    constexpr bool DEC = NV || X8;
    typedef LdsBlock<FW> BW;
    typedef LdsBlock<FX> BX;
    constexpr int TBW = BW::TBG, TBX = BX::TBG;     // stored block bytes (weights, activations)
    constexpr int RBW_G = 32 * fmt_bits(FW) / 8;    // stored bytes of one 32-code row of a weight block
    constexpr int RB = 32 * fmt_bits(FX) / 8;       // stored bytes of one channel row of an activation block
    static_assert(NRB == 1 || NRB == 2, "one or two 32-row blocks per wave");
    constexpr int RBW = NRB * WGM;                   // 32-row blocks per tile
    constexpr int PX = PW * 4 / WGM;                // output pixels per tile
    constexpr int CS = DG ? 1 : S;                  // halo columns per output pixel step
    constexpr int DS = DG ? S : 1;                  // tap step of a phase (stride-2 input gradient)
    constexpr int HP = (PX - 1) * CS + KW;          // halo pixels
    constexpr int NA = KW * 2 * RBW;                // weight blocks per stage
    constexpr int NB = 2 * HP;                      // activation blocks per stage
    constexpr int NSW = NA / BW::BPI;               // weight slices (1 KB) per stage
    constexpr int NSX = NB / BX::BPI;               // activation slices per stage
    constexpr int NQ = (NSW + NSX + 3) / 4;         // DMA instructions per thread per stage
    constexpr int ND = (PW - 1) * CS + KW;          // distinct halo pixels of a wave
    constexpr int NSA = KW * 2 * RBW;               // weight scales per stage
    constexpr int NSB = 2 * HP;                     // activation scales per stage
    static_assert(NA % BW::BPI == 0 && NB % BX::BPI == 0, "whole slices");
    static_assert(NSA + NSB <= LT, "scale staging needs one thread per scale");
    static_assert(2 * (NQ + 1) <= 63, "two stages in flight must fit the vmcnt counter");
    static_assert(S == 1 || S == 2, "stride 1 or 2");
    constexpr int A_BYTES = NSW * 1024;
    extern __shared__ __attribute__((aligned(16))) uint8_t smem[];

    const int tid = threadIdx.x, lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);

    // ---- tile: (row tile, pixel segment, output row of the phase, group)
    const int nseg = (f.gw + PX - 1) / PX;
    const int mt = lin % p.mtiles;
    int r = lin / p.mtiles;
    const int seg = r % nseg;
    r /= nseg;
    const int yi = r % f.gh, g = r / f.gh;
    const int x0 = seg * PX;                                       // first pixel on the phase grid
    const int cbase = DG ? x0 + f.c0 - (KW - 1) : x0 * S - p.pw;   // first halo column

    // ---- strides (bytes)
    const uint32_t w_tap = (uint32_t)p.w_cp * RBW_G;               // one tap of one 32-Cout block
    const uint32_t w_cob = (uint32_t)p.kh * p.kwf * w_tap;         // one 32-Cout block
    const uint32_t x_pix = (uint32_t)p.kcb * TBX;                  // one source pixel
    const uint32_t x_row = (uint32_t)p.wsrc * x_pix;

    // ---- per-lane DMA pieces: instruction q of this wave moves LDS slice
    // (4q + wave) of the stage; its block(s) and this lane's 16 bytes
    const uint32_t in_w = (uint32_t)(BW::BPI == 2 ? (lane & 31) : lane) * BW::STEP;   // lane offset in a block
    const uint32_t in_x = (uint32_t)(BX::BPI == 2 ? (lane & 31) : lane) * BX::STEP;
    uint32_t off[NQ];
    uint32_t flg[NQ];        // bit0 tile-valid, bit1 K block 1, bit2 activation block
#pragma unroll
    for (int q = 0; q < NQ; q++) {
        const int slice = 4 * q + wave;
        flg[q] = 0;
        off[q] = 0;
        if (slice < NSW) {
            // [tap t][K half kb][row block rb]
            const int blk = slice * BW::BPI + (BW::BPI == 2 ? (lane >> 5) : 0);
            const int rb = blk % RBW, kb = (blk / RBW) & 1, t = blk / (2 * RBW);
            const int rowblk = mt * RBW + rb;
            // K half kb: 32-channel block 2 kk + kb, or with KR kernel row 2 st + kb
            const uint32_t kbo = KR ? 0u : (uint32_t)kb;
            if (DG) {   // rows = input channels (block rowblk of Cin_p), K = output channels
                off[q] = kbo * w_cob + (uint32_t)(f.kw0 + DS * t) * w_tap + (uint32_t)rowblk * TBW;
            } else {    // rows = output channels (32-Cout block rowblk), K = input channels
                off[q] = (uint32_t)rowblk * w_cob + (uint32_t)t * w_tap + kbo * TBW;
            }
            if (KR) off[q] += (uint32_t)(kb * DS) * p.kwf * w_tap;
            off[q] += in_w;
            flg[q] = (rowblk < p.w_rowblocks ? 1u : 0u) | (uint32_t)kb << 1;
        } else if (slice < NSW + NSX) {
            // [K half kb][halo pixel hc]
            const int b = (slice - NSW) * BX::BPI + (BX::BPI == 2 ? (lane >> 5) : 0);
            const int kb = b / HP, hc = b % HP;
            const int col = cbase + hc;
            const bool ok = col >= 0 && col < p.wsrc;
            // channel rows past a single block's real channels hold +0 codes:
            // read the zero block there instead (FP8 / FP4 rows of 32 / 16 bytes)
            const bool row_real = fmt_bits(FX) == 6 || (int)(in_x / RB) < p.xrows;
            off[q] = (uint32_t)(ok ? col : 0) * x_pix + (KR ? 0u : (uint32_t)kb) * TBX + in_x;
            // KR: the next kernel row reads the source row below (forward) or
            // above (input gradient); offsets wrap modulo 2^32 and are added
            // to the row base before the pointer
            if (KR && kb) off[q] += DG ? 0u - x_row : x_row;
            flg[q] = (ok && row_real ? 1u : 0u) | (uint32_t)kb << 1 | 4u;
        }
    }
    // scale entries: thread e copies entry e; [0, NSA) weight scales
    // [t][kb][rb], [NSA, NSA+NSB) halo scales [kb][hc], the rest zero
    uint32_t s_off = 0, s_flg = 0;
    if (tid < NSA) {
        const int rb = tid % RBW, kb = (tid / RBW) & 1, t = tid / (2 * RBW);
        const int rowblk = mt * RBW + rb;
        const uint32_t kbo = KR ? 0u : (uint32_t)kb;
        if (DG) s_off = (kbo * p.kh * p.kwf + f.kw0 + DS * t) * p.w_ncb + rowblk;
        else    s_off = ((uint32_t)rowblk * p.kh * p.kwf + t) * p.w_ncb + kbo;
        if (KR) s_off += (uint32_t)(kb * DS) * p.kwf * p.w_ncb;
        s_flg = (rowblk < p.w_rowblocks ? 1u : 0u) | (uint32_t)kb << 1 | 8u;
    } else if (tid < NSA + NSB) {
        const int q = tid - NSA, kb = q / HP, hc = q % HP;
        const int col = cbase + hc;
        const bool ok = col >= 0 && col < p.wsrc;
        s_off = (uint32_t)(ok ? col : 0) * p.x_ncb + (KR ? 0u : (uint32_t)kb);
        if (KR && kb) s_off += DG ? 0u - (uint32_t)p.wsrc * p.x_ncb : (uint32_t)p.wsrc * p.x_ncb;
        s_flg = (ok ? 1u : 0u) | (uint32_t)kb << 1 | 4u | 8u;
    }
    // Which per-stage condition a lane's copy needs, as bits to test against
    // the stage's mask: a copy is issued from memory when the test passes,
    // else from the zero block.  Bitwise tests keep the copies free of the
    // branches that short-circuit conditions compile to.
    //   KR (mask: 1 row 0 in range, 2 row 1 in range, 4 always, 8 row 1
    //   exists): activation copies need 1 or 2, weight copies 4 or 8; any
    //   bit passes.
    //   otherwise (mask: 1 always, 2 second K block exists, 4 row in range):
    //   every needed bit must pass.
    // A lane whose copy is never valid needs bit 16, which no mask has.
    auto need_of = [&](uint32_t fl) -> uint32_t {
        if (!(fl & 1u)) return 16u;
        const bool isb = fl & 4u, k1 = fl & 2u;
        if (KR) return isb ? (k1 ? 2u : 1u) : (k1 ? 8u : 4u);
        return 1u | (k1 ? 2u : 0u) | (isb ? 4u : 0u);
    };
    uint32_t need[NQ];
#pragma unroll
    for (int q = 0; q < NQ; q++) need[q] = need_of(flg[q]);
    const uint32_t s_need = (s_flg & 8u) ? need_of(s_flg) : 16u;

    // stages: (kernel row, pair of 32-channel K blocks), or with krow (a
    // single K block) pairs of kernel rows, the K halves of a stage holding
    // the two rows, so no stage carries a zero block
    const int nkk = (p.kcb + 1) / 2;
    const int nstage = KR ? (f.nvh + 1) / 2 : f.nvh * nkk;
    const uint8_t* const zero = g_zero_lean;
    // both scale tensors in scalar registers: a per-lane choice between the
    // two argument fields would otherwise be made by a vector load from the
    // argument block, whose wait would also drain every copy in flight
    const uint8_t* wsp = p.ws;
    const uint8_t* ssp = p.ss;
    asm("" : "+s"(wsp), "+s"(ssp));

    // stage st = (kernel row kh, K pair kk): issue its copies into buffer
    // buf.  Every wave issues exactly NQ + 1 copies per stage.
    auto issue_rows = [&](int st, int buf) {   // KR: K half kb = kernel row 2 st + kb
        const int ki0 = 2 * st;
        const bool has1 = ki0 + 1 < f.nvh;
        const int kh0 = f.kh0 + DS * ki0;
        const int sy0 = DG ? yi + f.r0 - ki0 : yi * p.sh + kh0 - p.ph;
        const int sy1 = DG ? sy0 - 1 : sy0 + 1;
        const bool ok0 = sy0 >= 0 && sy0 < p.hsrc;
        const bool ok1 = has1 && sy1 >= 0 && sy1 < p.hsrc;
        const uint8_t* abase = p.wc + (uint32_t)kh0 * p.kwf * w_tap;
        const uint32_t row = (uint32_t)g * p.hsrc + (uint32_t)sy0;   // may wrap: only used where valid
        const uint32_t xrow = row * x_row;
        const uint8_t* lds = smem + buf * p.stage_bytes;
        const uint32_t okm = (ok0 ? 1u : 0u) | (ok1 ? 2u : 0u) | 4u | (has1 ? 8u : 0u);
#pragma unroll
        for (int q = 0; q < NQ; q++) {
            const bool isb = flg[q] & 4u;
            const bool ok = (okm & need[q]) != 0u;
            const uint8_t* src = isb ? p.sc + (xrow + off[q]) : abase + off[q];
            dma16_async(ok ? src : zero + (isb ? in_x : in_w), lds_addr(lds + (4 * q + wave) * 1024));
        }
        const bool isb = s_flg & 4u;
        const bool ok = (okm & s_need) != 0u;
        const uint32_t o = isb ? s_off + row * p.wsrc * p.x_ncb : s_off + (uint32_t)kh0 * p.kwf * p.w_ncb;
        if constexpr (NV)
            dma16_async(ok ? (isb ? ssp : wsp) + 16 * o : zero, lds_addr(lds + NQ * 4096 + wave * 1024));
        else
            dma1_async(ok ? (isb ? ssp : wsp) + o : zero, lds_addr(lds + NQ * 4096 + wave * 256));
    };
    // stages are issued in order 0, 1, 2, ...: (kk, ki) = (st % nkk, st / nkk)
    // is kept as a counter pair instead of two scalar divisions per stage
    int iss_kk = 0, iss_ki = 0;
    auto issue = [&](int st, int buf) {
        if constexpr (KR) { issue_rows(st, buf); return; }
        const int kk = iss_kk, ki = iss_ki;
        if (++iss_kk == nkk) { iss_kk = 0; ++iss_ki; }
        const int kh = f.kh0 + DS * ki;
        const int sy = DG ? yi + f.r0 - ki : yi * p.sh + kh - p.ph;
        const bool row_ok = sy >= 0 && sy < p.hsrc;
        const bool kb1_ok = 2 * kk + 1 < p.kcb;
        const uint8_t* abase = p.wc + (DG ? (uint32_t)(2 * kk) * w_cob : (uint32_t)(2 * kk) * TBW) +
                               (uint32_t)kh * p.kwf * w_tap;
        const uint8_t* bbase = p.sc + ((uint32_t)g * p.hsrc + (row_ok ? sy : 0)) * x_row + (uint32_t)(2 * kk) * TBX;
        const uint8_t* lds = smem + buf * p.stage_bytes;
        const uint32_t okm = 1u | (kb1_ok ? 2u : 0u) | (row_ok ? 4u : 0u);
#pragma unroll
        for (int q = 0; q < NQ; q++) {
            const bool isb = flg[q] & 4u;
            const bool ok = (okm & need[q]) == need[q];
            const uint8_t* src = (isb ? bbase : abase) + off[q];
            dma16_async(ok ? src : zero + (isb ? in_x : in_w), lds_addr(lds + (4 * q + wave) * 1024));
        }
        const bool isb = s_flg & 4u;
        const bool ok = (okm & s_need) == s_need;
        const uint32_t o = isb ? s_off + ((uint32_t)g * p.hsrc + (row_ok ? sy : 0)) * p.wsrc * p.x_ncb + 2 * kk
                               : s_off + (uint32_t)kh * p.kwf * p.w_ncb +
                                     (DG ? (uint32_t)(2 * kk) * p.kh * p.kwf * p.w_ncb : (uint32_t)(2 * kk));
        if constexpr (NV)   // the 16 block scales of the 32-row block: 16 bytes per entry
            dma16_async(ok ? (isb ? ssp : wsp) + 16 * o : zero, lds_addr(lds + NQ * 4096 + wave * 1024));
        else
            dma1_async(ok ? (isb ? ssp : wsp) + o : zero, lds_addr(lds + NQ * 4096 + wave * 256));
    };

    // ---- wave geometry and per-lane fragment offsets
    const int wm = wave % WGM, wn = wave / WGM;       // 64-row group, pixel pair
    const int h = lane >> 5, i16 = lane & 15, gi = lane >> 4, cg = gi & 1, hh = gi >> 1;
    // FP6 in LDS: half row (row k, half c) in the 16-byte slot 2 k + c
    int a_lane;
    if (DG) a_lane = FW == MXC_E4M3 ? (lane & 31) * 32 + 16 * h : fmt_bits(FW) == 6 ? (lane & 31) * 32 : (lane & 31) * 16;
    else    a_lane = FW == MXC_E4M3 ? (16 * hh + (i16 >> 1)) * 32 + 16 * cg + 8 * (i16 & 1)
                   : fmt_bits(FW) == 6 ? 32 * i16 + 16 * cg : i16 * 16 + 8 * cg;
    const int b_lane = FX == MXC_E4M3 ? (16 * hh + (i16 >> 1)) * RB + 16 * cg + 8 * (i16 & 1)
                     : fmt_bits(FX) == 6 ? 32 * i16 + 16 * cg : i16 * RB + 8 * cg;
    const int hbase = PW * wn * CS;                   // first halo pixel of the wave

    v16f acc[NRB][PW];
#pragma unroll
    for (int i = 0; i < NRB; i++)
#pragma unroll
        for (int j = 0; j < PW; j++)
#pragma unroll
            for (int e = 0; e < 16; e++) acc[i][j][e] = 0.0f;

    // ring of nbuf buffers: stages st + 1 .. st + nbuf - 2 are in flight
    // while stage st computes; the barrier after the wait both publishes
    // stage st and frees the buffer of stage st - 1 for the next copy
    const int nbuf = p.nbuf;
    for (int j = 0; j < nbuf - 1 && j < nstage; j++) issue(j, j);
    // the fused input gradient's z tiles (bf16, 2 KB per output block) are
    // copied to LDS now, behind the first stages, so the epilogue finds them
    // there instead of waiting on a load per block; each wave copies the
    // tiles of its own blocks, so no barrier is needed, and the stage waits
    // below let the NZ younger copies stay in flight
    constexpr int NZB = PW * NRB;                   // output blocks of a wave
    constexpr int NZ = DG && !NV ? 2 * NZB : 0;     // at most this many z copies (1 KB each): zsl per block
    static_assert(2 * (NQ + 1) + NZ <= 63, "two stages and the z copies must fit the vmcnt counter");
    const bool zpf = DG && !NV && p.zoff > 0;
    const int npro = min(nbuf - 1, nstage);         // stages issued before the z copies
    const int zsl = p.zsl;
    uint8_t* const zl = smem + p.zoff + wave * (NZB * 1024 * zsl);
    if (zpf) {
        const int yz = f.ry + DS * yi;
#pragma unroll
        for (int cn = 0; cn < PW; cn++) {
#pragma unroll
            for (int rb = 0; rb < NRB; rb++) {
                const int xi = x0 + PW * wn + cn;
                const int cb = mt * RBW + NRB * wm + rb;
                const bool live = xi < f.gw && cb < p.q_ncb;
                const size_t pix = ((size_t)g * p.hout + yz) * p.wout + (f.rx + DS * (live ? xi : 0));
                const int rows = min(32, p.M - cb * 32);
                const uint16_t* zb = (const uint16_t*)p.zpre + (pix * p.M + (size_t)(live ? cb : 0) * 32) * 32;
                for (int i = 0; i < zsl; i++) {
                    // LDS slot lane of rows 16 i .. 16 i + 15 holds row 16 i + lane / 4,
                    // stored chunk lane % 4 = chunk c ^ ((row / 2) % 4) (the layout of bf16_lds)
                    const int row = 16 * i + (lane >> 2), c = (lane & 3) ^ ((row >> 1) & 3);
                    const bool ok = live && row < rows;
                    dma16_async(ok ? (const void*)(zb + row * 32 + c * 8) : (const void*)(zero + lane * 16),
                                lds_addr(zl + (cn * NRB + rb) * 1024 * zsl + i * 1024));
                }
            }
        }
    }
    int buf = 0;
    for (int st = 0; st < nstage; st++) {
        const int later = min(nbuf - 2, nstage - 1 - st);
        if (NZ > 0 && zpf && st < npro) {           // the zsl * NZB z copies are younger than this stage
            if (zsl == 2) {
                if (later <= 0) vm_wait<NZ>();
                else if (later == 1) vm_wait<NQ + 1 + NZ>();
                else vm_wait<2 * (NQ + 1) + NZ>();
            } else {
                if (later <= 0) vm_wait<NZ / 2>();
                else if (later == 1) vm_wait<NQ + 1 + NZ / 2>();
                else vm_wait<2 * (NQ + 1) + NZ / 2>();
            }
        } else {
            vm_wait_stage<NQ + 1>(later);
        }
        __syncthreads();
        if (st + nbuf - 1 < nstage) issue(st + nbuf - 1, buf == 0 ? nbuf - 1 : buf - 1);
        const uint8_t* A = smem + buf * p.stage_bytes;
        const uint8_t* B = A + A_BYTES;
        const uint8_t* SC = A + NQ * 4096;
        buf = buf + 1 == nbuf ? 0 : buf + 1;

        // fragments of the wave's ND halo pixels (both K halves)
        v8i bf[ND];
        int sb[ND];
        uint32_t bfd[DEC ? ND : 1][16];         // NV: decoded to fp16; X8: to bf16
#pragma unroll
        for (int d = 0; d < ND; d++) {
            const int hc = hbase + d;
            if (FX == MXC_E4M3) {
                const uint8_t* tb = B + hc * BX::TBL + b_lane;
#pragma unroll
                for (int kb = 0; kb < 2; kb++)
#pragma unroll
                    for (int hf = 0; hf < 2; hf++) {
                        const v2i v = lds_tr8(tb + kb * HP * BX::TBL + hf * 8 * RB);
                        bf[d][4 * kb + 2 * hf] = v[0];
                        bf[d][4 * kb + 2 * hf + 1] = v[1];
                    }
            } else if (fmt_bits(FX) == 6) {
                // channels 0..15, then 16..31, of this lane's sample
                const uint8_t* tb = B + (hh * HP + hc) * BX::TBL + b_lane;
                const v3i lo = lds_tr6(tb), hi = lds_tr6(tb + 512);
                bf[d][0] = lo[0]; bf[d][1] = lo[1]; bf[d][2] = lo[2];
                bf[d][3] = hi[0]; bf[d][4] = hi[1]; bf[d][5] = hi[2];
                bf[d][6] = bf[d][7] = 0;
            } else {
                const uint8_t* tb = B + (hh * HP + hc) * BX::TBL + b_lane;
#pragma unroll
                for (int hf = 0; hf < 2; hf++) {
                    const v2i v = lds_tr4(tb + hf * 16 * RB);
                    bf[d][2 * hf] = v[0];
                    bf[d][2 * hf + 1] = v[1];
                }
                bf[d][4] = bf[d][5] = bf[d][6] = bf[d][7] = 0;
            }
            sb[d] = SC[4 * (NSA + h * HP + hc)];
            if constexpr (X8)   // both K blocks' scales (h = 0, 1) of the pixel
                e4m3_decode32(bf[d], SC[4 * (NSA + hc)], SC[4 * (NSA + HP + hc)], bfd[d]);
            if constexpr (NV) {
                // scale of (channel group o, this lane's sample group): byte
                // 4 o + (lane % 32) / 8 of a K block's entry, word o
                const int sh = 8 * ((lane & 31) >> 3);
                uint32_t s4;
                if constexpr (FX == MXC_E4M3) {
                    // the lane holds channels 16 h .. 16 h + 15 of both K blocks:
                    // groups 2 h, 2 h + 1 of each
                    const uint4 u0 = *(const uint4*)(SC + 16 * (NSA + hc));
                    const uint4 u1 = *(const uint4*)(SC + 16 * (NSA + HP + hc));
                    const uint32_t w0 = h ? u0.z : u0.x, w1 = h ? u0.w : u0.y;
                    const uint32_t w2 = h ? u1.z : u1.x, w3 = h ? u1.w : u1.y;
                    s4 = ((w0 >> sh) & 0xFFu) | ((w1 >> sh) & 0xFFu) << 8 | ((w2 >> sh) & 0xFFu) << 16 |
                         ((w3 >> sh) & 0xFFu) << 24;
                } else {   // all 32 channels of K block h
                    const uint4 u = *(const uint4*)(SC + 16 * (NSA + h * HP + hc));
                    s4 = ((u.x >> sh) & 0xFFu) | ((u.y >> sh) & 0xFFu) << 8 | ((u.z >> sh) & 0xFFu) << 16 |
                         ((u.w >> sh) & 0xFFu) << 24;
                }
                nv_decode32<FX>(bf[d], s4, bfd[d]);
            }
        }
#pragma unroll
        for (int t = 0; t < KW; t++) {
            v8i af[NRB];
            int sa[NRB];
#pragma unroll
            for (int rb = 0; rb < NRB; rb++) {
                const int rbi = NRB * wm + rb;
                const uint8_t* a0 = A + ((t * 2 + 0) * RBW + rbi) * BW::TBL + a_lane;
                const uint8_t* a1 = a0 + RBW * BW::TBL;
                if (DG) {
                    if (FW == MXC_E4M3) {
                        const v4i u0 = *(const v4i*)a0;
                        const v4i u1 = *(const v4i*)a1;
                        af[rb][0] = u0[0]; af[rb][1] = u0[1]; af[rb][2] = u0[2]; af[rb][3] = u0[3];
                        af[rb][4] = u1[0]; af[rb][5] = u1[1]; af[rb][6] = u1[2]; af[rb][7] = u1[3];
                    } else if (fmt_bits(FW) == 6) {
                        // the lane's row: 12 bytes from each of its two slots
                        const uint8_t* ar = h ? a1 : a0;
                        const v3i u0 = *(const v3i*)ar;
                        const v3i u1 = *(const v3i*)(ar + 16);
                        af[rb][0] = u0[0]; af[rb][1] = u0[1]; af[rb][2] = u0[2];
                        af[rb][3] = u1[0]; af[rb][4] = u1[1]; af[rb][5] = u1[2];
                        af[rb][6] = af[rb][7] = 0;
                    } else {
                        const v4i u0 = *(const v4i*)(h ? a1 : a0);
                        af[rb][0] = u0[0]; af[rb][1] = u0[1]; af[rb][2] = u0[2]; af[rb][3] = u0[3];
                        af[rb][4] = af[rb][5] = af[rb][6] = af[rb][7] = 0;
                    }
                } else {
                    if (FW == MXC_E4M3) {
#pragma unroll
                        for (int kb = 0; kb < 2; kb++)
#pragma unroll
                            for (int hf = 0; hf < 2; hf++) {
                                const v2i v = lds_tr8((kb ? a1 : a0) + hf * 8 * 32);
                                af[rb][4 * kb + 2 * hf] = v[0];
                                af[rb][4 * kb + 2 * hf + 1] = v[1];
                            }
                    } else if (fmt_bits(FW) == 6) {
                        const uint8_t* ab = hh ? a1 : a0;
                        const v3i lo = lds_tr6(ab), hi = lds_tr6(ab + 512);
                        af[rb][0] = lo[0]; af[rb][1] = lo[1]; af[rb][2] = lo[2];
                        af[rb][3] = hi[0]; af[rb][4] = hi[1]; af[rb][5] = hi[2];
                        af[rb][6] = af[rb][7] = 0;
                    } else {
                        const uint8_t* ab = hh ? a1 : a0;
#pragma unroll
                        for (int hf = 0; hf < 2; hf++) {
                            const v2i v = lds_tr4(ab + hf * 16 * 16);
                            af[rb][2 * hf] = v[0];
                            af[rb][2 * hf + 1] = v[1];
                        }
                        af[rb][4] = af[rb][5] = af[rb][6] = af[rb][7] = 0;
                    }
                }
                sa[rb] = SC[4 * ((t * 2 + h) * RBW + rbi)];
            }
            uint32_t afd[DEC ? NRB : 1][16];
            if constexpr (X8) {
#pragma unroll
                for (int rb = 0; rb < NRB; rb++) {
                    const int rbi = NRB * wm + rb;
                    e4m3_decode32(af[rb], SC[4 * ((t * 2 + 0) * RBW + rbi)], SC[4 * ((t * 2 + 1) * RBW + rbi)], afd[rb]);
                }
            }
            if constexpr (NV) {
                // an entry holds byte 4 (Cin group) + (Cout group)
#pragma unroll
                for (int rb = 0; rb < NRB; rb++) {
                    const int rbi = NRB * wm + rb;
                    const int q8 = (lane & 31) >> 3, sh = 8 * q8;
                    uint32_t s4;
                    if constexpr (FW == MXC_E4M3) {
                        // K elements 16 h .. 16 h + 15 of both K blocks: groups 2 h, 2 h + 1
                        const uint4 u0 = *(const uint4*)(SC + 16 * ((t * 2 + 0) * RBW + rbi));
                        const uint4 u1 = *(const uint4*)(SC + 16 * ((t * 2 + 1) * RBW + rbi));
                        if (DG) {   // rows = input channels (word q8), K = output channels (its bytes)
                            const uint32_t a = q8 == 0 ? u0.x : q8 == 1 ? u0.y : q8 == 2 ? u0.z : u0.w;
                            const uint32_t b = q8 == 0 ? u1.x : q8 == 1 ? u1.y : q8 == 2 ? u1.z : u1.w;
                            s4 = ((a >> (16 * h)) & 0xFFFFu) | ((b >> (16 * h)) & 0xFFFFu) << 16;
                        } else {    // rows = output channels (byte q8), K = input channels (the words)
                            const uint32_t w0 = h ? u0.z : u0.x, w1 = h ? u0.w : u0.y;
                            const uint32_t w2 = h ? u1.z : u1.x, w3 = h ? u1.w : u1.y;
                            s4 = ((w0 >> sh) & 0xFFu) | ((w1 >> sh) & 0xFFu) << 8 | ((w2 >> sh) & 0xFFu) << 16 |
                                 ((w3 >> sh) & 0xFFu) << 24;
                        }
                    } else {
                        const uint4 u = *(const uint4*)(SC + 16 * ((t * 2 + h) * RBW + rbi));
                        if (DG) {   // rows = input channels: the lane's channel group row, K groups o
                            s4 = q8 == 0 ? u.x : q8 == 1 ? u.y : q8 == 2 ? u.z : u.w;
                        } else {    // columns = output channels: byte 4 o + (lane % 32) / 8
                            s4 = ((u.x >> sh) & 0xFFu) | ((u.y >> sh) & 0xFFu) << 8 | ((u.z >> sh) & 0xFFu) << 16 |
                                 ((u.w >> sh) & 0xFFu) << 24;
                        }
                    }
                    nv_decode32<FW>(af[rb], s4, afd[rb]);
                }
            }
#pragma unroll
            for (int cn = 0; cn < PW; cn++) {
                const int d = DG ? cn + (KW - 1 - t) : cn * CS + t;
#pragma unroll
                for (int rb = 0; rb < NRB; rb++) {  // transposed product: rows = samples, columns = channels
                    if constexpr (NV8) acc[rb][cn] = mfma_x8(bfd[d], afd[rb], acc[rb][cn]);
                    else if constexpr (NV) acc[rb][cn] = mfma_nv(bfd[d], afd[rb], acc[rb][cn]);
                    else if constexpr (X8) acc[rb][cn] = mfma_x8(bfd[d], afd[rb], acc[rb][cn]);
                    else acc[rb][cn] = mfma_mx<FX, FW>(bf[d], af[rb], acc[rb][cn], sb[d], sa[rb]);
                }
            }
        }
    }

    // ---- epilogue.  The tile was computed transposed: in acc[rb][cn] lane l
    // holds output channel 32 rb + l % 32 of the wave's 64, and samples
    // 8 (e / 4) + 4 (l / 32) + e % 4 -- four consecutive samples per group of
    // 4 registers.  In the CBF output the 32 channels of one (rb, cn) are one
    // contiguous 4 KB run, so each wave passes them through 4 KB of LDS
    // (16-byte chunks XOR-swizzled by row against bank conflicts) and writes
    // them back as four fully contiguous 1 KB stores.
    if constexpr (NV) {   // Eq. (6)'s fake-quantized operands carry T_W T_X
        const float tt = *p.tw * *p.tx;
#pragma unroll
        for (int rb = 0; rb < NRB; rb++)
#pragma unroll
            for (int cn = 0; cn < PW; cn++)
#pragma unroll
                for (int e = 0; e < 16; e++) acc[rb][cn][e] *= tt;
    }
    const int m = mt * 32 * RBW + 32 * NRB * wm + (lane & 31);
    if ((p.layout == MXC_CBF || p.layout == MXC_CBF_BF16) && !(Q && p.qcodes))
        __syncthreads();                                 // every wave is done with the stage buffers
    uint8_t* const ep = smem + wave * 4096;
    const int er = lane >> 3, ec = lane & 7;            // read-back: row er + 8 i, chunk ec
    const int y = f.ry + DS * yi;
    if (zpf) vm_wait<0>();                               // the z copies (a phase with no taps ran no stage)
    if (Q && p.qcodes) {
        // ---- fused quantizing epilogue: acc[rb][cn] is one whole MX block of
        // the output (32 channels x 32 samples at one pixel); lane l holds
        // channel l % 32 and samples 8 (e / 4) + 4 (l / 32) + e % 4.  The
        // codes are assembled in 1 KB of LDS per wave in stored order and
        // written as one contiguous run (16 or 8 bytes per lane).
        __syncthreads();                                 // every wave is done with the stage buffers
        uint8_t* const ep = smem + wave * 1024;
        const int r = lane & 31;
        // the fp32 output of one block (32 channels x 32 samples, 4 KB
        // contiguous in CBF): through 4 KB of LDS per wave (16-byte chunks
        // XOR-swizzled by row) and out as four whole 1 KB non-temporal runs
        uint8_t* const ep4 = smem + 4096 + wave * 4096;
        auto store_block = [&](const float* val, size_t pix, int cb) {
#pragma unroll
            for (int e4 = 0; e4 < 4; e4++)
                *(float4*)(ep4 + r * 128 + (((2 * e4 + h) ^ (r & 7)) << 4)) =
                    make_float4(val[4 * e4], val[4 * e4 + 1], val[4 * e4 + 2], val[4 * e4 + 3]);
            float* o = p.out + (pix * p.M + (size_t)cb * 32) * 32;
#pragma unroll
            for (int i = 0; i < 4; i++) {
                const int row = er + 8 * i;
                const float4 w = *(const float4*)(ep4 + row * 128 + ((ec ^ (row & 7)) << 4));
                if (cb * 32 + row < p.M) store_nt(o + row * 32 + 4 * ec, w);
            }
        };
#pragma unroll
        for (int cn = 0; cn < PW; cn++) {
            const int xi = x0 + PW * wn + cn;
            if (xi >= f.gw) continue;
            const size_t pix = ((size_t)g * p.hout + y) * p.wout + (f.rx + DS * xi);
#pragma unroll
            for (int rb = 0; rb < NRB; rb++) {
                const int cb = mt * RBW + NRB * wm + rb;
                if (cb >= p.q_ncb) continue;
                const int c = cb * 32 + r;
                const bool real = c < p.M;
                float v[16];
#pragma unroll
                for (int e = 0; e < 16; e++) v[e] = acc[rb][cn][e];
                // with bf16, the value a bf16 tensor holds is the value used
                // from here on
                auto to_bf16 = [](float* w, int n) {
#pragma unroll
                    for (int e = 0; e < n; e += 2) {
                        const uint32_t u = bf16_pack2(w[e], w[e + 1]);
                        w[e] = __uint_as_float(u << 16);
                        w[e + 1] = __uint_as_float(u & 0xFFFF0000u);
                    }
                };
                const int rows = min(32, p.M - cb * 32);
                const bool q8 = p.qfmt == MXC_E4M3, q6 = p.qfmt == MXC_E2M3 || p.qfmt == MXC_E3M2;
                if (!DG && rows <= 16 && !q6) {
                    // ---- a forward block with at most 16 real rows (a
                    // 16-channel layer): lanes 16..31 of each half hold padding rows.
                    // Lane (r + 16, h) takes samples 16 + 4 h .. (e4 = 2, 3)
                    // of row r from lane (r, h), which keeps e4 = 0, 1, so
                    // each lane activates and quantizes 8 values instead of
                    // 16 (the values, codes and stored bytes are unchanged).
                    const int row = r & 15, k0 = (r >> 4) * 2;
                    // (v_permlane16_swap(a, b) swaps the odd 16-lane rows of
                    // a with the even rows of b: its first result keeps a in
                    // lanes 0..15 and 32..47 and takes b's lanes 0..15 and
                    // 32..47 into lanes 16..31 and 48..63 -- with a = v[i]
                    // and b = v[8 + i], exactly u[i], in registers)
                    float u[8];
#pragma unroll
                    for (int i = 0; i < 8; i++)
                        u[i] = __uint_as_float(__builtin_amdgcn_permlane16_swap(
                            __float_as_uint(v[i]), __float_as_uint(v[8 + i]), false, false)[0]);
                    if (p.bf16) to_bf16(u, 8);
                    // the values of one block through LDS to global memory:
                    // bf16 (2 KB, 64-byte rows) or fp32 (4 KB, 128-byte rows)
                    auto stage_out = [&](const float* w, bool as_bf16, void* dst) {
                        if (as_bf16) {
#pragma unroll
                            for (int k = 0; k < 2; k++)
                                *(uint2*)(ep4 + bf16_lds(row, k0 + k) + 8 * h) =
                                    bf16_pack4(w[4 * k], w[4 * k + 1], w[4 * k + 2], w[4 * k + 3]);
                            const int rr = lane >> 2, ch = lane & 3;      // rows 0..15: one chunk per lane
                            const uint4 d = *(const uint4*)(ep4 + bf16_lds(rr, ch));
                            if (rr < rows) store_nt((uint16_t*)dst + rr * 32 + ch * 8, d);
                        } else {
#pragma unroll
                            for (int k = 0; k < 2; k++)
                                *(float4*)(ep4 + row * 128 + (((2 * (k0 + k) + h) ^ (row & 7)) << 4)) =
                                    make_float4(w[4 * k], w[4 * k + 1], w[4 * k + 2], w[4 * k + 3]);
#pragma unroll
                            for (int i = 0; i < 2; i++) {
                                const int rr = er + 8 * i;
                                const float4 d = *(const float4*)(ep4 + rr * 128 + ((ec ^ (rr & 7)) << 4));
                                if (rr < rows) store_nt((float*)dst + rr * 32 + 4 * ec, d);
                            }
                        }
                    };
                    const size_t ob = (pix * p.M + (size_t)cb * 32) * 32;   // the block in a CBF tensor
                    if (p.out && p.pre_out)
                        stage_out(u, p.bf16, p.bf16 ? (void*)((uint16_t*)p.out + ob) : (void*)(p.out + ob));
                    if (p.fn != MXC_FN_NONE)
                        with_fn(p.fn, [&](auto t) {
#pragma unroll
                            for (int i = 0; i < 8; i++) u[i] = fn_apply_c<decltype(t)::fn>(u[i]);
                        });
                    if (p.out && !p.pre_out) stage_out(u, false, p.out + ob);
                    uint32_t mm = 0;
#pragma unroll
                    for (int i = 0; i < 8; i++) mm = max(mm, __float_as_uint(u[i]) & 0x7FFFFFFFu);
                    mm = wave_max_u32(mm);
                    const uint32_t sc = q8 ? scale_code_from_bits<8>(mm) : scale_code_from_bits<2>(mm);
                    const float inv = inv_scale(sc);
                    const bool bad = sc == 0xFFu;
                    if (lane == 0) p.qscales[pix * p.q_ncb + cb] = (uint8_t)sc;
                    if (q8) {   // 32-byte rows; rows 16..31 are +0 codes
#pragma unroll
                        for (int k = 0; k < 2; k++)
                            *(uint32_t*)(ep + row * 32 + 8 * (k0 + k) + 4 * h) =
                                bad ? 0u : pack4_e4m3(make_float4(u[4 * k], u[4 * k + 1], u[4 * k + 2], u[4 * k + 3]), inv);
                        *(uint2*)(ep + 512 + 8 * lane) = make_uint2(0u, 0u);
                        const uint4 chunk = *(const uint4*)(ep + lane * 16);
                        *(uint4*)(p.qcodes + (pix * p.q_ncb + cb) * 1024 + lane * 16) = chunk;
                    } else {    // 16-byte rows
#pragma unroll
                        for (int k = 0; k < 2; k++)
                            *(unsigned short*)(ep + row * 16 + 4 * (k0 + k) + 2 * h) =
                                bad ? (unsigned short)0
                                    : pack4_e2m1(make_float4(u[4 * k], u[4 * k + 1], u[4 * k + 2], u[4 * k + 3]), inv);
                        *(uint32_t*)(ep + 256 + 4 * lane) = 0u;
                        const uint2 chunk = *(const uint2*)(ep + lane * 8);
                        *(uint2*)(p.qcodes + (pix * p.q_ncb + cb) * 512 + lane * 8) = chunk;
                    }
                    continue;
                }
                if (p.bf16) to_bf16(v, 16);
                if (p.out && p.pre_out) {   // the pre-activation, for the backward pass
                    if (p.bf16) store_bf16_tile(ep4, v, (uint16_t*)p.out + (pix * p.M + (size_t)cb * 32) * 32, rows, lane);
                    else        store_block(v, pix, cb);
                }
                // The activation (forward) or its derivative at z (input
                // gradient).  The forward takes one uniform branch on fn
                // around the 16 values, so that their exponentials and
                // reciprocals overlap.  The input gradient, with z from its
                // LDS tile, does the same four values at a time (scheduling
                // barriers): all sixteen at once took its kernels past the
                // registers of three waves per SIMD (measured on the second
                // layer of the network step: 234 -> 275 µs); its other z
                // sources choose fn per value.
                if constexpr (DG) {
                    if (p.fn != MXC_FN_NONE) {
                        if (zpf) {
                            const uint8_t* zt = zl + (cn * NRB + rb) * 1024 * zsl;
                            const bool zr = r < 16 * zsl;    // rows past the copied slots: padding, z = 0
                            if (p.fn == MXC_FN_RELU) grad_lds4<MXC_FN_RELU>(v, zt, zr, r, h);
                            else                     grad_lds4<MXC_FN_SILU>(v, zt, zr, r, h);
                        } else if (p.bf16) {
                            float zz[16];
                            load_bf16_tile(ep4, (const uint16_t*)p.zpre + (pix * p.M + (size_t)cb * 32) * 32, rows, lane, zz);
#pragma unroll
                            for (int e = 0; e < 16; e++) {
                                v[e] *= fn_grad(p.fn, zz[e]);
                                if ((e & 3) == 3) __builtin_amdgcn_sched_barrier(0);
                            }
                        } else {
                            const size_t zo = (pix * p.M + (real ? c : 0)) * 32 + 4 * h;
#pragma unroll
                            for (int e4 = 0; e4 < 4; e4++) {
                                float4 z = make_float4(0.f, 0.f, 0.f, 0.f);
                                if (real) z = *(const float4*)((const float*)p.zpre + zo + 8 * e4);
                                v[4 * e4] *= fn_grad(p.fn, z.x);
                                v[4 * e4 + 1] *= fn_grad(p.fn, z.y);
                                v[4 * e4 + 2] *= fn_grad(p.fn, z.z);
                                v[4 * e4 + 3] *= fn_grad(p.fn, z.w);
                                __builtin_amdgcn_sched_barrier(0);
                            }
                        }
                    }
                } else if (p.fn != MXC_FN_NONE) {
                    with_fn(p.fn, [&](auto t) {
#pragma unroll
                        for (int e = 0; e < 16; e++) v[e] = fn_apply_c<decltype(t)::fn>(v[e]);
                    });
                }
                if (p.out && !p.pre_out) store_block(v, pix, cb);
                uint32_t m = 0;
#pragma unroll
                for (int e = 0; e < 16; e++) m = max(m, __float_as_uint(v[e]) & 0x7FFFFFFFu);
                m = wave_max_u32(m);
                const uint32_t sc = q8 ? scale_code_from_bits<8>(m)
                                  : p.qfmt == MXC_E3M2 ? scale_code_from_bits<4>(m) : scale_code_from_bits<2>(m);
                const float inv = inv_scale(sc);
                const bool bad = sc == 0xFFu;
                if (lane == 0) p.qscales[pix * p.q_ncb + cb] = (uint8_t)sc;
                // the lane's 16 codes: run e4 (samples 8 e4 + 4 h .. + 3) in
                // bits [nb * 4 e4, nb * 4 (e4 + 1)) of run[e4]
                uint32_t run[4];
                if (DG && p.sr) {
                    // stochastic rounding (gradients): the code of (channel r,
                    // sample n) sits at position (pix q_ncb + cb) 1024 + 32 r + n
                    // of the code tensor, which keys its random half-word
                    const int s = (int)sc - 127;
                    const uint64_t q0 = (((uint64_t)pix * p.q_ncb + cb) * 1024 + 32 * r) >> 3;
                    const int nb = q8 ? 8 : q6 ? 6 : 4;
#pragma unroll
                    for (int e4 = 0; e4 < 4; e4++) {
                        const uint4 w = sr_words(q0 + e4, p.sk0, p.sk1);
                        const uint32_t w0 = h ? w.z : w.x, w1 = h ? w.w : w.y;
                        const uint32_t rr[4] = {w0 & 0xFFFFu, w0 >> 16, w1 & 0xFFFFu, w1 >> 16};
                        uint32_t u = 0u;
#pragma unroll
                        for (int t = 0; t < 4; t++)
                            u |= encode_sr_rt(p.qfmt, v[4 * e4 + t], s, inv, rr[t]) << (nb * t);
                        run[e4] = bad ? 0u : u;
                    }
                } else if (q6) {
                    float4 xv[4];
#pragma unroll
                    for (int e4 = 0; e4 < 4; e4++) xv[e4] = make_float4(v[4 * e4], v[4 * e4 + 1], v[4 * e4 + 2], v[4 * e4 + 3]);
                    const v6i w = p.qfmt == MXC_E2M3 ? pack16_fp6<MXC_E2M3>(xv, inv) : pack16_fp6<MXC_E3M2>(xv, inv);
                    const uint32_t w0 = bad ? 0u : (uint32_t)w[0], w1 = bad ? 0u : (uint32_t)w[1],
                                   w2 = bad ? 0u : (uint32_t)w[2];
                    run[0] = w0 & 0xFFFFFFu;
                    run[1] = (w0 >> 24) | ((w1 & 0xFFFFu) << 8);
                    run[2] = (w1 >> 16) | ((w2 & 0xFFu) << 16);
                    run[3] = w2 >> 8;
                } else if (q8) {
#pragma unroll
                    for (int e4 = 0; e4 < 4; e4++)
                        run[e4] = bad ? 0u : pack4_e4m3(make_float4(v[4 * e4], v[4 * e4 + 1], v[4 * e4 + 2], v[4 * e4 + 3]), inv);
                } else {
#pragma unroll
                    for (int e4 = 0; e4 < 4; e4++)
                        run[e4] = bad ? 0u
                                      : pack4_e2m1(make_float4(v[4 * e4], v[4 * e4 + 1], v[4 * e4 + 2], v[4 * e4 + 3]), inv);
                }
                if (q6) {
                    // 24 bits per run, stored at byte 6 e4 + 3 h of the channel's 24-byte row
#pragma unroll
                    for (int e4 = 0; e4 < 4; e4++) {
                        uint8_t* d = ep + r * 24 + 6 * e4 + 3 * h;
                        d[0] = (uint8_t)run[e4];
                        d[1] = (uint8_t)(run[e4] >> 8);
                        d[2] = (uint8_t)(run[e4] >> 16);
                    }
                    if (lane < 48) {
                        const uint4 chunk = *(const uint4*)(ep + lane * 16);
                        *(uint4*)(p.qcodes + (pix * p.q_ncb + cb) * 768 + lane * 16) = chunk;
                    }
                } else if (q8) {
#pragma unroll
                    for (int e4 = 0; e4 < 4; e4++) *(uint32_t*)(ep + r * 32 + 8 * e4 + 4 * h) = run[e4];
                    const uint4 chunk = *(const uint4*)(ep + lane * 16);
                    *(uint4*)(p.qcodes + (pix * p.q_ncb + cb) * 1024 + lane * 16) = chunk;
                } else {
#pragma unroll
                    for (int e4 = 0; e4 < 4; e4++) *(unsigned short*)(ep + r * 16 + 4 * e4 + 2 * h) = (unsigned short)run[e4];
                    const uint2 chunk = *(const uint2*)(ep + lane * 8);
                    *(uint2*)(p.qcodes + (pix * p.q_ncb + cb) * 512 + lane * 8) = chunk;
                }
            }
        }
        return;
    }
#pragma unroll
    for (int cn = 0; cn < PW; cn++) {
        const int xi = x0 + PW * wn + cn;
        if (xi >= f.gw) continue;
        const int x = f.rx + DS * xi;
        if (p.layout == MXC_CBF_BF16) {
            uint16_t* px = (uint16_t*)p.out + (((size_t)g * p.hout + y) * p.wout + x) * p.M * 32;
#pragma unroll
            for (int rb = 0; rb < NRB; rb++) {
                const int m0 = mt * 32 * RBW + 32 * NRB * wm + 32 * rb;
                if (m0 >= p.M) continue;
                float v[16];
#pragma unroll
                for (int e = 0; e < 16; e++) v[e] = acc[rb][cn][e];
                store_bf16_tile(ep, v, px + (size_t)m0 * 32, min(32, p.M - m0), lane);
            }
        } else if (p.layout == MXC_CBF) {
            float* px = p.out + (((size_t)g * p.hout + y) * p.wout + x) * p.M * 32;
#pragma unroll
            for (int rb = 0; rb < NRB; rb++) {
                const int m0 = mt * 32 * RBW + 32 * NRB * wm + 32 * rb;
                if (m0 >= p.M) continue;
                const int r = lane & 31;
#pragma unroll
                for (int e4 = 0; e4 < 4; e4++)
                    *(float4*)(ep + r * 128 + (((2 * e4 + h) ^ (r & 7)) << 4)) =
                        make_float4(acc[rb][cn][4 * e4], acc[rb][cn][4 * e4 + 1],
                                    acc[rb][cn][4 * e4 + 2], acc[rb][cn][4 * e4 + 3]);
                float* o = px + (size_t)m0 * 32;
#pragma unroll
                for (int i = 0; i < 4; i++) {
                    const int row = er + 8 * i;
                    const float4 v = *(const float4*)(ep + row * 128 + ((ec ^ (row & 7)) << 4));
                    if (m0 + row < p.M) store_nt(o + row * 32 + 4 * ec, v);
                }
            }
        } else {
            const size_t hw = (size_t)p.hout * p.wout;
            float* px = p.out + (size_t)y * p.wout + x;
#pragma unroll
            for (int rb = 0; rb < NRB; rb++) {
                const int mm = m + 32 * rb;
                if (mm >= p.M) continue;
#pragma unroll
                for (int e = 0; e < 16; e++) {
                    const int n = 8 * (e >> 2) + 4 * h + (e & 3);
                    px[((size_t)(g * 32 + n) * p.M + mm) * hw] = acc[rb][cn][e];
                }
            }
        }
    }
}

// Workgroup `bid` of `nblk` (a multiple of 8).
template <int FW, int FX, bool DG, int KW, int S, int WGM, int PW, bool NV = false, int NRB = 2, bool KR = false,
          bool Q = true>
__device__ __forceinline__ void lean_body(const LeanArgs& p, int bid, int nblk) {
    // XCD-aware order: consecutive tiles (same output row) on one XCD
    const int per_xcd = (nblk + 7) / 8;
    const int lin = (bid % 8) * per_xcd + bid / 8;
    if (lin >= p.ntiles) return;
    Phase f;
    f.ry = 0; f.rx = 0; f.kh0 = 0; f.nvh = p.kh; f.kw0 = 0;
    f.gh = p.hout; f.gw = p.wout; f.c0 = p.pw; f.r0 = p.ph;
    lean_tile<FW, FX, DG, KW, S, WGM, PW, NV, NRB, KR, Q>(p, lin, f);
}

// Every lean kernel asks for at least two waves per SIMD.  Left to itself
// the compiler gives these kernels about 290 registers per lane (64 of them
// accumulation registers): one wave per SIMD, one workgroup per CU, and the
// latency of each stage and epilogue exposed.  Held to 256 they fit in 120
// to 170 with no spills, so two or three workgroups share a CU (measured on
// the network step: the forward kernels about 18% faster, the narrow
// stride-2 input gradient 21%).
template <int FW, int FX, bool DG, int KW, int S, int WGM, int PW, bool NV = false, int NRB = 2, bool KR = false>
__global__ __launch_bounds__(LT) __attribute__((amdgpu_waves_per_eu(2))) void conv_lean_kernel(LeanArgs p) {
    lean_body<FW, FX, DG, KW, S, WGM, PW, NV, NRB, KR>(p, blockIdx.x, gridDim.x);
}

// Stride-2 input gradient for kernel width KWF (1 or 3): the four phases in
// one launch, tiles of phase (ry, rx) at [pofs[2 ry + rx], pofs[2 ry + rx + 1]).
template <int FW, int FX, int KWF, int WGM, int PW, bool NV = false, int NRB = 2, bool KR = false, bool Q = true>
__device__ __forceinline__ void lean_dg2_body(const LeanArgs& p, int bid, int nblk) {
    const int per_xcd = (nblk + 7) / 8;
    int lin = (bid % 8) * per_xcd + bid / 8;
    if (lin >= p.pofs[4]) return;
    int ph = 0;
    while (ph < 3 && lin >= p.pofs[ph + 1]) ph++;
    lin -= p.pofs[ph];
    Phase f;
    f.ry = ph >> 1; f.rx = ph & 1;
    f.kh0 = (f.ry + p.ph) & 1;
    f.kw0 = (f.rx + p.pw) & 1;
    f.nvh = f.kh0 < p.kh ? (p.kh - f.kh0 + 1) / 2 : 0;
    const int nvw = f.kw0 < KWF ? (KWF - f.kw0 + 1) / 2 : 0;
    if (nvw == 0) f.nvh = 0;                       // no tap reaches the phase: its pixels are zero
    f.gh = (p.hout - f.ry + 1) / 2; f.gw = (p.wout - f.rx + 1) / 2;
    f.c0 = (f.rx + p.pw - f.kw0) / 2; f.r0 = (f.ry + p.ph - f.kh0) / 2;
    if (KWF == 3 && nvw == 2) lean_tile<FW, FX, true, 2, 2, WGM, PW, NV, NRB, KR, Q>(p, lin, f);
    else                      lean_tile<FW, FX, true, 1, 2, WGM, PW, NV, NRB, KR, Q>(p, lin, f);
}

template <int FW, int FX, int KWF, int WGM, int PW, bool NV = false, int NRB = 2, bool KR = false>
__global__ __launch_bounds__(LT) __attribute__((amdgpu_waves_per_eu(2))) void conv_lean_dg2_kernel(LeanArgs p) {
    lean_dg2_body<FW, FX, KWF, WGM, PW, NV, NRB, KR>(p, blockIdx.x, gridDim.x);
}

// The input gradient of a layer (stride 1 with KW taps per row, or, with
// DG2, the four stride-2 phases of kernel width KW) and its weight gradient
// in one launch: the last nl workgroups take input-gradient tiles, the ones
// before them weight-gradient tiles (dispatched first: measured faster than
// the other order).  Both only read the quantized G_Y (with W, resp. X), so
// neither waits for the other, and the tail of one fills the CUs the other
// leaves idle.  Both counts are multiples of 8, so each part keeps its own
// kernel's XCD mapping.  Format F for every operand.
template <int F, int KW, int PW, bool DG2, int NB, int NRB = 2, bool KR = false>
__global__ __launch_bounds__(LT) __attribute__((amdgpu_waves_per_eu(2))) void conv_lean_bwd_kernel(LeanArgs p, WLArgs q, int nl) {
    extern __shared__ __attribute__((aligned(16))) uint8_t smem[];
    const int b = blockIdx.x;
    const int nw = (int)gridDim.x - nl;
    if (b >= nw) {
        if constexpr (DG2) lean_dg2_body<F, F, KW, 1, PW, false, NRB, KR, false>(p, b - nw, nl);
        else               lean_body<F, F, true, KW, 1, 1, PW, false, NRB, KR, false>(p, b - nw, nl);
    } else {
        wgrad_tile<F, F, false, NB, (NB == 1 && KW == 3) ? 3 : 1>(q, b, nw, (float (*)[32 * NB * 32 * NB])smem);
    }
}

// LDS bytes of one launch: the stage ring, and at least the 4 x 4 KB the
// epilogue stages through.
inline size_t lean_ring_lds(const LeanArgs& a, int nbufs_used) {
    const size_t lds = (size_t)nbufs_used * a.stage_bytes;
    const size_t epi = a.qcodes ? 5 * 4096 : 4 * 4096;     // the fused epilogue: codes + fp32 staging
    return lds < epi ? epi : lds;
}
// bytes of the prefetched z tiles: 4 waves x (pixels x row blocks per wave)
// x 1 KB per 16 rows of the layer's rows (at most 32)
inline size_t lean_z_lds(int pw, int rb, int zsl) { return (size_t)4 * pw * rb * zsl * 1024; }
inline size_t lean_lds(const LeanArgs& a, int nbufs_used) {
    return a.zoff > 0 ? (size_t)a.zoff + lean_z_lds(a.zpw, a.zrb, a.zsl) : lean_ring_lds(a, nbufs_used);
}

// Dynamic LDS above 64 KB needs the kernel's attribute raised, once per
// device: `devs` holds one bit per device that has it (devices past the 64th
// raise it on every launch).  Concurrent first calls may both raise it, which
// is harmless.
template <typename K>
int raise_lds(K kernel, std::atomic<uint64_t>& devs, size_t lds) {
    if (lds > 65536) {
        int dev = 0;
        if (hipGetDevice(&dev) != hipSuccess) return MXC_ERR_HIP;
        const uint64_t bit = dev < 64 ? (uint64_t)1 << dev : 0;
        if (!bit || !(devs.load(std::memory_order_acquire) & bit)) {
            if (hipFuncSetAttribute((const void*)kernel, hipFuncAttributeMaxDynamicSharedMemorySize, LDS_MAX) !=
                hipSuccess)
                return MXC_ERR_HIP;
            devs.fetch_or(bit, std::memory_order_release);
        }
    }
    return MXC_OK;
}

template <typename K>
int lean_launch(K kernel, std::atomic<uint64_t>& devs, const LeanArgs& a, int ntiles, size_t lds, hipStream_t s) {
    if (raise_lds(kernel, devs, lds)) return MXC_ERR_HIP;
    const int grid = (ntiles + 7) / 8 * 8;
    hipLaunchKernelGGL(kernel, dim3(grid), dim3(LT), lds, s, a);
    return hipGetLastError() == hipSuccess ? MXC_OK : MXC_ERR_HIP;
}

template <int FW, int FX, bool DG, int KW, int S, int WGM, int PW, bool NV = false, int NRB = 2, bool KR = false>
int launch_lean_t(const LeanArgs& a, int nbufs_used, hipStream_t s) {
    static std::atomic<uint64_t> devs{0};
    return lean_launch(conv_lean_kernel<FW, FX, DG, KW, S, WGM, PW, NV, NRB, KR>, devs, a, a.ntiles, lean_lds(a, nbufs_used), s);
}

template <int FW, int FX, int KWF, int PW, bool NV = false, int NRB = 2, bool KR = false>
int launch_lean_dg2(const LeanArgs& a, int nbufs_used, hipStream_t s) {
    static std::atomic<uint64_t> devs{0};
    return lean_launch(conv_lean_dg2_kernel<FW, FX, KWF, 1, PW, NV, NRB, KR>, devs, a, a.pofs[4], lean_lds(a, nbufs_used), s);
}

// Narrow tiles: output channels (forward) or input channels (input gradient)
// in a single 32-row block, FP4 operands: each wave owns 32 rows x 4 pixels
// (the same products per wave as 64 rows x 2 pixels, none of them on padding
// rows), a tile 32 rows x 16 pixels.
constexpr int NARROW_PW = 4;
// ... or 32 rows x 2 pixels (a tile 32 x 8: half the stage, so more
// workgroups share a CU's LDS)
constexpr int NARROW_PW2 = 2;
template <int FW, int FX>
constexpr bool narrow_ok() { return FW == MXC_E2M1 && FX == MXC_E2M1; }

// (WGM, PW, NRB) in use: (1, 1, 2), (1, 2, 2) and narrow (1, NARROW_PW, 1),
// (1, NARROW_PW2, 1); the NV kernels run (1, 1, 2)
template <int FW, int FX, bool DG, int KW, int S, bool NV = false>
int launch_lean_w(const LeanArgs& a, const LeanShape& h, hipStream_t s) {
    const int wgm = h.wgm, pw = h.pw, nb = h.nb;
    if constexpr (NV) return launch_lean_t<FW, FX, DG, KW, S, 1, 1, true>(a, nb, s);
    if constexpr (narrow_ok<FW, FX>())
        if (h.rb == 1) {
            if (pw == NARROW_PW) {
                if constexpr (KW == 3)
                    if (h.kr) return launch_lean_t<FW, FX, DG, KW, S, 1, NARROW_PW, false, 1, true>(a, nb, s);
                return launch_lean_t<FW, FX, DG, KW, S, 1, NARROW_PW, false, 1>(a, nb, s);
            }
            if (pw == NARROW_PW2) {
                if constexpr (KW == 3)
                    if (h.kr) return launch_lean_t<FW, FX, DG, KW, S, 1, NARROW_PW2, false, 1, true>(a, nb, s);
                return launch_lean_t<FW, FX, DG, KW, S, 1, NARROW_PW2, false, 1>(a, nb, s);
            }
            return MXC_ERR_ARG;
        }
    if (wgm != 1) return MXC_ERR_ARG;
    return pw == 1 ? launch_lean_t<FW, FX, DG, KW, S, 1, 1>(a, nb, s) : launch_lean_t<FW, FX, DG, KW, S, 1, 2>(a, nb, s);
}

template <int FW, int FX, bool DG, bool NV = false>
int launch_lean_f(const LeanArgs& a, const LeanShape& h, hipStream_t s) {
    const int kw = h.kw, sw = h.sw, pw = h.pw, nb = h.nb;
    if constexpr (DG) {
        if (sw == 2) {
            if constexpr (NV) return kw == 3 ? launch_lean_dg2<FW, FX, 3, 1, true>(a, nb, s) : launch_lean_dg2<FW, FX, 1, 1, true>(a, nb, s);
            if constexpr (narrow_ok<FW, FX>())
                if (h.rb == 1) {
                    if (pw == NARROW_PW)
                        return kw == 3 ? (h.kr ? launch_lean_dg2<FW, FX, 3, NARROW_PW, false, 1, true>(a, nb, s)
                                               : launch_lean_dg2<FW, FX, 3, NARROW_PW, false, 1>(a, nb, s))
                                       : launch_lean_dg2<FW, FX, 1, NARROW_PW, false, 1>(a, nb, s);
                    if (pw == NARROW_PW2)
                        return kw == 3 ? (h.kr ? launch_lean_dg2<FW, FX, 3, NARROW_PW2, false, 1, true>(a, nb, s)
                                               : launch_lean_dg2<FW, FX, 3, NARROW_PW2, false, 1>(a, nb, s))
                                       : launch_lean_dg2<FW, FX, 1, NARROW_PW2, false, 1>(a, nb, s);
                    return MXC_ERR_ARG;
                }
            if (kw == 3) return pw == 1 ? launch_lean_dg2<FW, FX, 3, 1>(a, nb, s) : launch_lean_dg2<FW, FX, 3, 2>(a, nb, s);
            return pw == 1 ? launch_lean_dg2<FW, FX, 1, 1>(a, nb, s) : launch_lean_dg2<FW, FX, 1, 2>(a, nb, s);
        }
        return kw == 3 ? launch_lean_w<FW, FX, DG, 3, 1, NV>(a, h, s) : launch_lean_w<FW, FX, DG, 1, 1, NV>(a, h, s);
    } else {
        if (kw == 3) return sw == 2 ? launch_lean_w<FW, FX, DG, 3, 2, NV>(a, h, s) : launch_lean_w<FW, FX, DG, 3, 1, NV>(a, h, s);
        return sw == 2 ? launch_lean_w<FW, FX, DG, 1, 2, NV>(a, h, s) : launch_lean_w<FW, FX, DG, 1, 1, NV>(a, h, s);
    }
}

}  // namespace

// The launch plan of one layer (conv_lean.hip).
struct LeanPlan {
    LeanArgs a;
    int wgm, pw, rb, nstage, used;
    bool dg2;
    bool krow;    // stages pair kernel rows (a single K block, kernel width 3)
};

// The tile shape, stage layout and ring depth of one launch; returns 0, 1
// when the layer is outside these kernels' shapes, or an MXC_* code.
int lean_plan(const Conv& cv, bool dg, const void* wc, const uint8_t* ws, const void* sc, const uint8_t* ss,
              float* out, int layout, const FusedEpi* q, const float* nv_tw, const float* nv_tx, LeanPlan& P);

// Per-format launches (one translation unit each):
int lean_fwd_e4m3(const LeanArgs& a, const LeanShape& h, hipStream_t s);
int lean_dg_e4m3(const LeanArgs& a, const LeanShape& h, hipStream_t s);
int lean_fwd_e2m1(const LeanArgs& a, const LeanShape& h, hipStream_t s);
int lean_dg_e2m1(const LeanArgs& a, const LeanShape& h, hipStream_t s);
int lean_nv(int fw, int fx, const LeanArgs& a, bool dg, const LeanShape& h, hipStream_t s);
int lean_nv68(int fw, int fx, const LeanArgs& a, bool dg, const LeanShape& h, hipStream_t s);
int lean_fp6(int fw, int fx, const LeanArgs& a, bool dg, const LeanShape& h, hipStream_t s);

}  // namespace mxc
