// conv_lean_nv.hip -- the lean forward and input-gradient kernels on NVFP
// operands with FP4 weights: NVFP4, and FP4 weights / gradients with NVFP6
// E3M2 activations (one translation unit per format group, so that the
// kernel instantiations compile in parallel).
#include "conv_lean_kern.h"

namespace mxc {

int lean_nv(int fw, int fx, const LeanArgs& a, bool dg, const LeanShape& h, hipStream_t s) {
    if (fw == MXC_E2M1 && fx == MXC_E2M1)
        return dg ? launch_lean_f<MXC_E2M1, MXC_E2M1, true, true>(a, h, s)
                  : launch_lean_f<MXC_E2M1, MXC_E2M1, false, true>(a, h, s);
    if (fw == MXC_E2M1 && fx == MXC_E3M2)
        return dg ? launch_lean_f<MXC_E2M1, MXC_E3M2, true, true>(a, h, s)
                  : launch_lean_f<MXC_E2M1, MXC_E3M2, false, true>(a, h, s);
    return MXC_ERR_ARG;
}

}  // namespace mxc
