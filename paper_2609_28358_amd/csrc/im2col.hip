// im2col.hip -- a2: explicit channel-batch-first im2col on MX codes
// (Sec. IV-A: X'_{Cin,N} = im2col of the channel-batch-first X_{Cin,N}).
//
// X'[g][ho][wo][kh][kw][Cp][Bn] = X[g][ho*sh+kh-ph][wo*sw+kw-pw][Cp][Bn]:
// for one (group, output pixel, tap) the destination run and the source
// pixel's run are both Cp*Bn codes long and contiguous, so the kernel is a
// 16-byte-vector copy (one chunk per thread, non-temporal stores); blocks stay whole, so nothing is requantized, and
// padding taps become zero codes with scale code 0.  Pure HBM stream:
// |X'| codes written, the source re-read from L2/MALL across taps.
#include "mx_internal.h"

namespace mxc {
namespace {

// One thread per 16-byte destination chunk, as in a plain streaming copy.
// Grid: x = chunks of one output row (output column, chunk within the run),
// y = (source group, output row), z = tap (kh, kw); all index arithmetic
// except a shift and a mask is per workgroup and scalar.  The run length in
// chunks is a power of two for the usual channel counts (POW2: shift and
// mask), else one division.  Threads with chunk index below the block count
// also copy the scale bytes.
template <int POW2>
__global__ __launch_bounds__(256) void im2col_kernel(const uint4* __restrict__ src,
                                                     const uint8_t* __restrict__ ssrc,
                                                     uint4* __restrict__ dst,
                                                     uint8_t* __restrict__ sdst, Conv cv,
                                                     int run16, int log2run) {
    const int i = blockIdx.x * 256 + threadIdx.x;
    const int ow = POW2 ? i >> log2run : i / run16;
    if (ow >= cv.wo) return;
    const int within = POW2 ? i & (run16 - 1) : i - ow * run16;
    const int g = blockIdx.y / cv.ho, oh = blockIdx.y % cv.ho;
    const int tap = blockIdx.z, a = tap / cv.kw, b = tap % cv.kw;
    const int ih = oh * cv.sh + a - cv.ph, iw = ow * cv.sw + b - cv.pw;
    const bool inside = ih >= 0 && ih < cv.h && iw >= 0 && iw < cv.w;
    const size_t srun = ((size_t)g * cv.h + (inside ? ih : 0)) * cv.w + (inside ? iw : 0);
    const size_t run = ((size_t)blockIdx.y * cv.wo + ow) * (cv.kh * cv.kw) + tap;
    store_nt(dst + run * run16 + within, inside ? __ldg(src + srun * run16 + within) : make_uint4(0, 0, 0, 0));
    const int ncb = cv.x.ncb;
    if (within < ncb) sdst[run * ncb + within] = inside ? ssrc[srun * ncb + within] : 0;
}

}  // namespace

int im2col_check(const Conv& cv) {
    const long run16 = (long)cv.x.cp * cv.x.bn * cv.x.bits / 8 / 16;   // run bytes: a multiple of 16 (FP6: Bn >= 4)
    const long row = (long)cv.wo * run16;            // chunks of one output row, one tap
    const long rows = (long)cv.x.ng * cv.ho;
    if (row > 0x7FFFFFFFL - 256 || rows > 0x7FFFFFFFL || cv.kh * cv.kw > 65535 || cv.x.ncb > run16)
        return MXC_ERR_SHAPE;
    return MXC_OK;
}

int launch_im2col(const Conv& cv, const void* xc, const uint8_t* xs, void* cc, uint8_t* cs,
                  hipStream_t s) {
    const int rc = im2col_check(cv);
    if (rc) return rc;
    const int run16 = (int)((long)cv.x.cp * cv.x.bn * cv.x.bits / 8 / 16);
    const long row = (long)cv.wo * run16;
    const long rows = (long)cv.x.ng * cv.ho;
    int log2run = -1;
    for (int k = 0; k < 31; k++)
        if ((1 << k) == run16) log2run = k;
    const dim3 grid((unsigned)((row + 255) / 256), (unsigned)rows, (unsigned)(cv.kh * cv.kw));
    if (log2run >= 0)
        hipLaunchKernelGGL(im2col_kernel<1>, grid, dim3(256), 0, s, (const uint4*)xc, xs, (uint4*)cc, cs, cv,
                           run16, log2run);
    else
        hipLaunchKernelGGL(im2col_kernel<0>, grid, dim3(256), 0, s, (const uint4*)xc, xs, (uint4*)cc, cs, cv,
                           run16, 0);
    return hipGetLastError() == hipSuccess ? MXC_OK : MXC_ERR_HIP;
}

}  // namespace mxc
