// im2col.hip -- a2: explicit channel-batch-first im2col on MX codes
// (Sec. IV-A: X'_{Cin,N} = im2col of the channel-batch-first X_{Cin,N}).
//
// X'[g][ho][wo][kh][kw][Cp][Bn] = X[g][ho*sh+kh-ph][wo*sw+kw-pw][Cp][Bn]:
// for one (group, output pixel, tap) the destination run and the source
// pixel's run are both Cp*Bn codes long and contiguous, so the kernel is a
// 16-byte-vector copy; blocks stay whole, so nothing is requantized, and
// padding taps become zero codes with scale code 0.  Pure HBM stream:
// |X'| codes written, the source re-read from L2/MALL across taps.
#include "mx_internal.h"

namespace mxc {
namespace {

__global__ __launch_bounds__(256) void im2col_kernel(const uint4* __restrict__ src,
                                                     const uint8_t* __restrict__ ssrc,
                                                     uint4* __restrict__ dst,
                                                     uint8_t* __restrict__ sdst, Conv cv,
                                                     long total16, int run16) {
    const long o = (long)blockIdx.x * blockDim.x + threadIdx.x;
    if (o >= total16) return;
    const long r = o / run16;            // (g, ho, wo, kh, kw) run index
    const int within = (int)(o % run16);
    long t = r;
    const int b = (int)(t % cv.kw); t /= cv.kw;
    const int a = (int)(t % cv.kh); t /= cv.kh;
    const int ow = (int)(t % cv.wo); t /= cv.wo;
    const int oh = (int)(t % cv.ho);
    const long g = t / cv.ho;
    const int ih = oh * cv.sh + a - cv.ph, iw = ow * cv.sw + b - cv.pw;
    const bool inside = ih >= 0 && ih < cv.h && iw >= 0 && iw < cv.w;
    const long srun = (g * cv.h + ih) * cv.w + iw;
    dst[o] = inside ? __ldg(&src[srun * run16 + within]) : make_uint4(0, 0, 0, 0);
    if (within == 0) {
        const int ncb = cv.x.ncb;
        for (int c = 0; c < ncb; c++) sdst[r * ncb + c] = inside ? ssrc[srun * ncb + c] : 0;
    }
}

}  // namespace

int launch_im2col(const Conv& cv, const void* xc, const uint8_t* xs, void* cc, uint8_t* cs,
                  hipStream_t s) {
    const long run_bytes = (long)cv.x.cp * cv.x.bn * cv.bits / 8;   // multiple of 32
    const int run16 = (int)(run_bytes / 16);
    const long runs = (long)cv.x.ng * cv.ho * cv.wo * cv.kh * cv.kw;
    const long total16 = runs * run16;
    const long grid = (total16 + 255) / 256;
    if (grid > 0x7FFFFFFFL) return MXC_ERR_SHAPE;
    hipLaunchKernelGGL(im2col_kernel, dim3((unsigned)grid), dim3(256), 0, s, (const uint4*)xc, xs,
                       (uint4*)cc, cs, cv, total16, run16);
    return hipGetLastError() == hipSuccess ? MXC_OK : MXC_ERR_HIP;
}

}  // namespace mxc
