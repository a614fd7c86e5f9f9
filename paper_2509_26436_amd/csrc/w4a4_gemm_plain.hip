// W4A4 GEMM template instantiations: the exact integer accumulator, plus the
// occupancy query the template's persistent grid is sized by.
#include "w4a4_gemm_kernel.h"

namespace quartz {

hipError_t launch_gemm_i32(const GemmLaunch& a, hipStream_t stream)
{
    return launch_mode<true, false>(a, stream);
}

int device_compute_units()
{
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0)
        return 256;
    constexpr int kMaxDevices = 64;
    static std::atomic<int> cache[kMaxDevices];
    if (dev < kMaxDevices) {
        const int c = cache[dev].load(std::memory_order_relaxed);
        if (c > 0)
            return c;
    }
    int cus = 0;
    if (hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess ||
        cus <= 0)
        return 256;
    if (dev < kMaxDevices)
        cache[dev].store(cus, std::memory_order_relaxed);
    return cus;
}

int gemm_resident_blocks()
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
            &per_cu, reinterpret_cast<const void*>(&w4a4_gemm_kernel<16, false, false, true, false, true>),
            kThreadsPerBlock, 0) != hipSuccess)
        return 0;
    const int n = cus * std::max(per_cu, 1);
    if (dev < kMaxDevices)
        cache[dev].store(n, std::memory_order_relaxed);
    return n;
}

}  // namespace quartz
