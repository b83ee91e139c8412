// conv_lean_e2m1_fwd.hip -- the lean forward kernels on MXFP4 operands (one translation unit per format and direction,
// so that the kernel instantiations compile in parallel).
#include "conv_lean_kern.h"

namespace mxc {

int lean_fwd_e2m1(const LeanArgs& a, const LeanShape& h, hipStream_t s) {
    return launch_lean_f<MXC_E2M1, MXC_E2M1, false>(a, h, s);
}

}  // namespace mxc
