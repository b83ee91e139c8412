// conv_lean_e4m3_dg.hip -- the lean input-gradient kernels on MXFP8 operands (one translation unit per format and direction,
// so that the kernel instantiations compile in parallel).
#include "conv_lean_kern.h"

namespace mxc {

int lean_dg_e4m3(const LeanArgs& a, const LeanShape& h, hipStream_t s) {
    return launch_lean_f<MXC_E4M3, MXC_E4M3, true>(a, h, s);
}

}  // namespace mxc
