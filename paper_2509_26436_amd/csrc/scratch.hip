// Device scratch of quartz_w4a4_linear_noalloc: a file-scope array that takes
// the place of the caller's stream-K workspace, for callers that cannot
// allocate (graph capture, serving loops).  Each device the library runs on
// holds its own copy of the array until the process ends.
//
// Size: the workspace of quartz_w4a4_linear_ws is the split tiles' counters
// (fewer than two rounds of tiles x 8 math waves x 4 bytes: under 16 KiB for
// 256 workgroups) followed by two 128 KiB partial-sum slots per splitting
// workgroup (64 MiB for 256).  The array holds that worst case for a
// persistent grid of up to 256 workgroups, one per compute unit of an MI355X.
#include <mutex>

#include "quartz_internal.h"

namespace quartz {
namespace {

constexpr size_t kScratchCounterBytes = size_t(64) << 10;
constexpr size_t kScratchBytes = (size_t(64) << 20) + kScratchCounterBytes;

__device__ __align__(256) uint8_t scratch[kScratchBytes];

// Clears the counter part with a kernel (not a memset node, so that a
// captured graph replays it correctly): counters must read zero when a GEMM
// starts, whatever the last call on this device left behind.
__global__ __launch_bounds__(256) void clear_words_kernel(uint32_t* __restrict__ p, uint32_t words)
{
    const uint32_t i = blockIdx.x * 256u + threadIdx.x;
    if (i < words)
        p[i] = 0u;
}

constexpr int kMaxDevices = 64;

}  // namespace

size_t noalloc_scratch_bytes()
{
    return kScratchBytes;
}

hipError_t noalloc_scratch(void** out)
{
    *out = nullptr;
    int dev = 0;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess)
        return e;
    if (dev < 0 || dev >= kMaxDevices)
        return hipErrorInvalidDevice;
    // resolved once per device, with that device current: each device holds
    // its own copy of the array at its own address
    static std::mutex mu;
    static void* ptr[kMaxDevices] = {};
    std::lock_guard<std::mutex> lock(mu);
    if (!ptr[dev]) {
        void* p = nullptr;
        e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
        if (e != hipSuccess)
            return e;
        if (!p)
            return hipErrorInvalidSymbol;
        ptr[dev] = p;
    }
    *out = ptr[dev];
    return hipSuccess;
}

hipError_t clear_noalloc_counters(void* ptr, size_t counter_bytes, hipStream_t stream)
{
    if (counter_bytes > kScratchCounterBytes)
        return hipErrorInvalidValue;
    const uint32_t words = (uint32_t)((counter_bytes + 3) / 4);
    if (words == 0)
        return hipSuccess;
    clear_words_kernel<<<dim3((words + 255) / 256), dim3(256), 0, stream>>>(
        static_cast<uint32_t*>(ptr), words);
    return hipGetLastError();
}

}  // namespace quartz
