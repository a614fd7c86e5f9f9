// The linear layer's kernel (w4a4_linear_kernel.h) in the asymmetric mode
// (zero points and weight group sums), its own translation unit so the
// instantiations compile in parallel with the others.
#include "w4a4_linear_kernel.h"

namespace quartz {

hipError_t launch_linear_asym(const GemmLaunch& a, hipStream_t stream)
{
    return launch_linear_mode<false, false, true>(a, stream);
}

}  // namespace quartz
