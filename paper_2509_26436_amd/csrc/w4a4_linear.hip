// The linear layer's kernel (w4a4_linear_kernel.h): per-group bf16 or
// quantized output and the LDM setting, plus its schedule and residency.
#include "w4a4_linear_kernel.h"

namespace quartz {
GemmSchedule linear_schedule(int64_t M, int64_t N, int64_t K, int blocks, bool split)
{
    return gemm_schedule_tiles(M, N, K, blocks, split, LBM, LBN);
}

int linear_resident_blocks()
{
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0)
        return 0;
    constexpr int kMaxDevices = 64;
    static std::atomic<int> cache[kMaxDevices];
    if (dev < kMaxDevices) {
        const int c = cache[dev].load(std::memory_order_relaxed);
        if (c > 0)
            return c;
    }
    int cus = 0, per_cu = 0;
    if (hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess ||
        hipOccupancyMaxActiveBlocksPerMultiprocessor(
            &per_cu, reinterpret_cast<const void*>(&w4a4_linear_kernel<16, false, true, false, true, false>),
            kLinThreads, 0) != hipSuccess)
        return 0;
    const int n = cus * std::max(per_cu, 1);
    if (dev < kMaxDevices)
        cache[dev].store(n, std::memory_order_relaxed);
    return n;
}

hipError_t launch_linear(const GemmLaunch& a, hipStream_t stream)
{
    return a.qout.codes ? launch_linear_mode<false, true>(a, stream)
                        : launch_linear_mode<false, false>(a, stream);
}

hipError_t launch_linear_static(const GemmLaunch& a, hipStream_t stream)
{
    return launch_linear_mode<true, false>(a, stream);
}

}  // namespace quartz
