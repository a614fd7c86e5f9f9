// W4A4 GEMM instantiations: the output quantized for the next layer.
#include "w4a4_gemm_kernel.h"

namespace quartz {

hipError_t launch_gemm_quant(const GemmLaunch& a, hipStream_t stream)
{
    return launch_mode<false, true, false, false>(a, stream);
}

}  // namespace quartz
