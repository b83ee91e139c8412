// conv_lean_fp6.hip -- the lean forward and input-gradient kernels with FP6 operands (all E2M3, and
// E2M1 weights / gradients with E3M2 activations) (one translation unit per format and direction,
// so that the kernel instantiations compile in parallel).
#include "conv_lean_kern.h"

namespace mxc {

int lean_fp6(int fw, int fx, const LeanArgs& a, bool dg, const LeanShape& h, hipStream_t s) {
    if (fw == MXC_E2M3 && fx == MXC_E2M3)
        return dg ? launch_lean_f<MXC_E2M3, MXC_E2M3, true>(a, h, s) : launch_lean_f<MXC_E2M3, MXC_E2M3, false>(a, h, s);
    if (fw == MXC_E2M1 && fx == MXC_E3M2)
        return dg ? launch_lean_f<MXC_E2M1, MXC_E3M2, true>(a, h, s) : launch_lean_f<MXC_E2M1, MXC_E3M2, false>(a, h, s);
    return MXC_ERR_ARG;
}

}  // namespace mxc
