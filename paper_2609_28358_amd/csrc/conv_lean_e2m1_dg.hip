// conv_lean_e2m1_dg.hip -- the lean input-gradient kernels on MXFP4 operands (one translation unit per format and direction,
// so that the kernel instantiations compile in parallel).
#include "conv_lean_kern.h"

namespace mxc {

int lean_dg_e2m1(const LeanArgs& a, const LeanShape& h, hipStream_t s) {
    return launch_lean_f<MXC_E2M1, MXC_E2M1, true>(a, h, s);
}

}  // namespace mxc
