// libdart internal: validation of device-side preconditions (target ids in
// range, strictly increasing offsets with the right ends, 0/1 masks), run
// before the real kernels when DART_CHECK=1 so that malformed device data is
// reported as DART_ERR_INVALID_ARG instead of being read out of range. The
// calls synchronise the stream, so this is a debugging mode.
#include "internal.h"

#include <stdlib.h>

#include <mutex>

namespace {

// Violation flags of the last validation on this device: bit 0 ids, bit 1
// offsets, bit 2 mask. Every thread that finds a violation stores the same
// nonzero word, so concurrent stores need no atomics.
__device__ unsigned int g_flags[3];

constexpr int kCheckThreads = 256;
constexpr int64_t kCheckMaxBlocks = 1024;

__global__ void __launch_bounds__(kCheckThreads)
check_ids_kernel(const int32_t* __restrict__ v, int64_t n, int64_t bound, unsigned int* flag) {
    for (int64_t i = blockIdx.x * (int64_t)kCheckThreads + threadIdx.x; i < n;
         i += (int64_t)gridDim.x * kCheckThreads) {
        const int64_t x = v[i];
        if (x < 0 || x >= bound) *flag = 1u;
    }
}

__global__ void __launch_bounds__(kCheckThreads)
check_offsets_kernel(const int32_t* __restrict__ v, int64_t n, int64_t bound, unsigned int* flag) {
    for (int64_t i = blockIdx.x * (int64_t)kCheckThreads + threadIdx.x; i <= n;
         i += (int64_t)gridDim.x * kCheckThreads) {
        const int64_t x = v[i];
        const bool bad = (i == 0 && x != 0) || (i == n && x != bound) || (i < n && x >= v[i + 1]);
        if (bad) *flag = 1u;
    }
}

__global__ void __launch_bounds__(kCheckThreads)
check_mask_kernel(const uint8_t* __restrict__ v, int64_t n, unsigned int* flag) {
    for (int64_t i = blockIdx.x * (int64_t)kCheckThreads + threadIdx.x; i < n;
         i += (int64_t)gridDim.x * kCheckThreads)
        if (v[i] > 1) *flag = 1u;
}

unsigned blocks_for(int64_t n) {
    const int64_t b = (n + kCheckThreads) / kCheckThreads;
    return (unsigned)(b < kCheckMaxBlocks ? b : kCheckMaxBlocks);
}

}  // namespace

namespace dart_check {

bool enabled() {
    const char* e = getenv("DART_CHECK");
    return e && e[0] == '1' && e[1] == '\0';
}

dart_status_t run(hipStream_t stream, std::initializer_list<Item> items) {
    if (!enabled()) return DART_OK;
    // the validation waits for its result: not possible under graph capture
    if (const dart_status_t st = may_synchronize(stream); st != DART_OK) return st;
    // one validation at a time in the process: the flags are shared by every
    // call on a device
    static std::mutex mu;
    std::lock_guard<std::mutex> lock(mu);
    // the flags of the stream's device
    const int dev = stream_device(stream);
    if (dev < 0) return DART_ERR_HIP;
    DeviceGuard on_dev(dev);
    if (!on_dev.ok) return DART_ERR_HIP;
    unsigned int* flags = nullptr;
    if (hipGetSymbolAddress(reinterpret_cast<void**>(&flags), HIP_SYMBOL(g_flags)) != hipSuccess)
        return DART_ERR_HIP;
    unsigned int host[3] = {0u, 0u, 0u};
    if (hipMemcpyAsync(flags, host, sizeof host, hipMemcpyHostToDevice, stream) != hipSuccess)
        return DART_ERR_HIP;
    for (const Item& it : items) {
        if (!it.ptr) continue;
        switch (it.kind) {
            case Item::Ids:
                if (it.n > 0)
                    hipLaunchKernelGGL(check_ids_kernel, dim3(blocks_for(it.n)), dim3(kCheckThreads),
                                       0, stream, static_cast<const int32_t*>(it.ptr), it.n, it.bound,
                                       flags + 0);
                break;
            case Item::Offsets:
                hipLaunchKernelGGL(check_offsets_kernel, dim3(blocks_for(it.n + 1)),
                                   dim3(kCheckThreads), 0, stream,
                                   static_cast<const int32_t*>(it.ptr), it.n, it.bound, flags + 1);
                break;
            case Item::Mask:
                if (it.n > 0)
                    hipLaunchKernelGGL(check_mask_kernel, dim3(blocks_for(it.n)), dim3(kCheckThreads),
                                       0, stream, static_cast<const uint8_t*>(it.ptr), it.n, flags + 2);
                break;
        }
        if (hipGetLastError() != hipSuccess) return DART_ERR_HIP;
    }
    if (hipMemcpyAsync(host, flags, sizeof host, hipMemcpyDeviceToHost, stream) != hipSuccess ||
        hipStreamSynchronize(stream) != hipSuccess)
        return DART_ERR_HIP;
    return (host[0] | host[1] | host[2]) ? DART_ERR_INVALID_ARG : DART_OK;
}

}  // namespace dart_check
