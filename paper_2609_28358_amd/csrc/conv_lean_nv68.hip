// conv_lean_nv68.hip -- the lean forward and input-gradient kernels on NVFP6
// E2M3 and NVFP8 E4M3 operands (one translation unit per format group, so
// that the kernel instantiations compile in parallel).
#include "conv_lean_kern.h"

namespace mxc {

int lean_nv68(int fw, int fx, const LeanArgs& a, bool dg, const LeanShape& h, hipStream_t s) {
    if (fw == MXC_E2M3 && fx == MXC_E2M3)
        return dg ? launch_lean_f<MXC_E2M3, MXC_E2M3, true, true>(a, h, s)
                  : launch_lean_f<MXC_E2M3, MXC_E2M3, false, true>(a, h, s);
    if (fw == MXC_E4M3 && fx == MXC_E4M3)
        return dg ? launch_lean_f<MXC_E4M3, MXC_E4M3, true, true>(a, h, s)
                  : launch_lean_f<MXC_E4M3, MXC_E4M3, false, true>(a, h, s);
    return MXC_ERR_ARG;
}

}  // namespace mxc
