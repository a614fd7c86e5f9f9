// W4A4 GEMM instantiations: the asymmetric mode (zero points and weight
// group sums).
#include "w4a4_gemm_kernel.h"

namespace quartz {

hipError_t launch_gemm_asym(const GemmLaunch& a, hipStream_t stream)
{
    return launch_mode<false, false, true>(a, stream);
}

}  // namespace quartz
