// W4A4 GEMM instantiations: the 3 x 3 convolution as an implicit GEMM, in the
// per-group and in the static (LDM) setting.
#include "w4a4_gemm_kernel.h"

namespace quartz {

hipError_t launch_gemm_conv(const GemmLaunch& a, hipStream_t stream)
{
    return launch_mode<false, false, true>(a, stream);
}

hipError_t launch_gemm_conv_static(const GemmLaunch& a, hipStream_t stream)
{
    return launch_mode<false, true, true>(a, stream);
}

}  // namespace quartz
