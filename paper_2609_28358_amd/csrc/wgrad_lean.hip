// wgrad_lean.hip -- a5 for batch block 32: G_Wf = G_Yf X'^T (Sec. II-C,
// Sec. IV-B), contracted over (output pixel, sample).
//
// With Bn = 32 the contraction runs along the samples of a block row, which
// the CBF layout stores contiguously: a G_Y block is [32 Cout][32 samples]
// and the X block of a tap's input pixel is [32 Cin][32 samples].  So both
// MFMA operands are read straight from memory into registers (16 bytes per
// lane; an FP6 row is 24 bytes), with no LDS staging and no transposition:
// G_Y and X may have different element formats.  One 32 x 32 x 64 MFMA
// contracts the 32 samples of two consecutive output pixels (K block 0 =
// pixel P0, K block 1 = pixel P1), each K block with its own E8M0 scales.
// Taps that fall into the padding read a zero block.
//
// Work split: a tile is 64 Cout x 64 Cin at one tap; each wave of a
// workgroup accumulates the tile over its own range of pixel pairs, the four
// waves are summed through LDS, and the workgroup writes one partial tile
// ([split][Cout_p][tap * Cin_p + ci], reduced by wgrad_reduce) or, with a
// single split, the final OIHW values.  Pixel pairs are processed in
// batches whose loads are all issued before the first MFMA.
#include "mx_internal.h"

namespace mxc {
#include "wgrad_tile.h"

namespace {

template <int FA, int FB, bool NV = false, int NB = 2, int KT = 1>
__global__ __launch_bounds__(WT) void wgrad_lean_kernel(WLArgs p) {
    __shared__ float red[4][32 * NB * 32 * NB];
    wgrad_tile<FA, FB, NV, NB, KT>(p, blockIdx.x, gridDim.x, red);
}

}  // namespace

// Splits of the lean weight-gradient kernel for this layer, or 0 when it does
// not apply (batch block below 32).
int wgrad_lean_splits(const Conv& cv) {
    if (cv.x.bn != 32) return 0;
    const long npix = (long)cv.x.ng * cv.ho * cv.wo;
    const long npairs = (npix + 1) / 2;
    const long ntiles = (long)cv.kh * (cv.kw / wgrad_taps(cv, false)) * ((cv.gy.ncb + 1) / 2) * ((cv.x.ncb + 1) / 2);
    if (npix > 0x3FFFFFFFL || ntiles > 0x7FFFFFL) return 0;
    // about two workgroups per CU, each wave with at least 4 pixel pairs; a
    // layer on 32 x 32 tiles (one channel block on each side) keeps a quarter
    // of the LDS per workgroup, so about five fit on a CU, each wave with at
    // least 8 pairs
    const bool nb1 = wgrad_single_block(cv);
    long splits = (nb1 ? 1280 : 512) / ntiles;
    const long cap = npairs / (4 * (nb1 ? 8 : 4));
    if (splits > cap) splits = cap;
    if (splits < 1) splits = 1;
    return (int)splits;
}

int launch_wgrad_lean(const Conv& cv, const void* gc, const uint8_t* gs, const void* xc, const uint8_t* xs,
                      float* dst, int splits, hipStream_t s, const float* nv_tg, const float* nv_tx) {
    WLArgs a;
    const long grid = wgrad_lean_fill(cv, gc, gs, xc, xs, dst, splits, nv_tg, nv_tx, a);
    if (grid < 0) return MXC_ERR_SHAPE;
    const dim3 gd((unsigned)grid);
    if (nv_tg) {
        if (cv.fa == MXC_E2M1 && cv.fb == MXC_E2M1)
            hipLaunchKernelGGL((wgrad_lean_kernel<MXC_E2M1, MXC_E2M1, true>), gd, dim3(WT), 0, s, a);
        else if (cv.fa == MXC_E2M1 && cv.fb == MXC_E3M2)
            hipLaunchKernelGGL((wgrad_lean_kernel<MXC_E2M1, MXC_E3M2, true>), gd, dim3(WT), 0, s, a);
        else if (cv.fa == MXC_E2M3 && cv.fb == MXC_E2M3)
            hipLaunchKernelGGL((wgrad_lean_kernel<MXC_E2M3, MXC_E2M3, true>), gd, dim3(WT), 0, s, a);
        else if (cv.fa == MXC_E4M3 && cv.fb == MXC_E4M3)
            hipLaunchKernelGGL((wgrad_lean_kernel<MXC_E4M3, MXC_E4M3, true>), gd, dim3(WT), 0, s, a);
        else
            return MXC_ERR_ARG;
        return hipGetLastError() == hipSuccess ? MXC_OK : MXC_ERR_HIP;
    }
    const bool nb1 = wgrad_single_block(cv);
    const bool kt3 = wgrad_taps(cv, false) == 3;
    if (cv.fa == MXC_E4M3 && cv.fb == MXC_E4M3) {
        if (kt3)      hipLaunchKernelGGL((wgrad_lean_kernel<MXC_E4M3, MXC_E4M3, false, 1, 3>), gd, dim3(WT), 0, s, a);
        else if (nb1) hipLaunchKernelGGL((wgrad_lean_kernel<MXC_E4M3, MXC_E4M3, false, 1>), gd, dim3(WT), 0, s, a);
        else          hipLaunchKernelGGL((wgrad_lean_kernel<MXC_E4M3, MXC_E4M3>), gd, dim3(WT), 0, s, a);
    } else if (cv.fa == MXC_E2M1 && cv.fb == MXC_E2M1) {
        if (kt3)      hipLaunchKernelGGL((wgrad_lean_kernel<MXC_E2M1, MXC_E2M1, false, 1, 3>), gd, dim3(WT), 0, s, a);
        else if (nb1) hipLaunchKernelGGL((wgrad_lean_kernel<MXC_E2M1, MXC_E2M1, false, 1>), gd, dim3(WT), 0, s, a);
        else          hipLaunchKernelGGL((wgrad_lean_kernel<MXC_E2M1, MXC_E2M1>), gd, dim3(WT), 0, s, a);
    }
    else if (cv.fa == MXC_E2M3 && cv.fb == MXC_E2M3) hipLaunchKernelGGL((wgrad_lean_kernel<MXC_E2M3, MXC_E2M3>), gd, dim3(WT), 0, s, a);
    else if (cv.fa == MXC_E2M1 && cv.fb == MXC_E3M2) hipLaunchKernelGGL((wgrad_lean_kernel<MXC_E2M1, MXC_E3M2>), gd, dim3(WT), 0, s, a);
    else return MXC_ERR_ARG;
    return hipGetLastError() == hipSuccess ? MXC_OK : MXC_ERR_HIP;
}

}  // namespace mxc
