// W4A4 GEMM instantiations: the LDM setting (static activation scale,
// per-channel weight scales).
#include "w4a4_gemm_kernel.h"

namespace quartz {

hipError_t launch_gemm_static(const GemmLaunch& a, hipStream_t stream)
{
    return launch_mode<false, false, true, false>(a, stream);
}

}  // namespace quartz
