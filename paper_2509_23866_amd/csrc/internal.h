// libdart internal helpers shared by its sources; not part of the C ABI.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include <initializer_list>

#include "dart.h"

#pragma GCC visibility push(hidden)

// Makes dev the current device for the caller's scope and restores the
// previous one after.
struct DeviceGuard {
    int prev = -1;
    bool ok = false;
    explicit DeviceGuard(int dev) {
        if (hipGetDevice(&prev) != hipSuccess) return;
        ok = prev == dev || hipSetDevice(dev) == hipSuccess;
    }
    ~DeviceGuard() {
        if (ok) (void)hipSetDevice(prev);
    }
    DeviceGuard(const DeviceGuard&) = delete;
    DeviceGuard& operator=(const DeviceGuard&) = delete;
};

// The device a stream belongs to (the current device for the null stream);
// -1 on a HIP error.
inline int stream_device(hipStream_t stream) {
    int dev = -1;
    if ((stream ? hipStreamGetDevice(stream, &dev) : hipGetDevice(&dev)) != hipSuccess) return -1;
    return dev;
}

// Whether a 1-D launch of blocks workgroups of threads work-items each fits
// the dispatch (at most 2^32 - 1 work-items in the grid).
inline bool grid_fits(int64_t blocks, int64_t threads) {
    return blocks >= 0 && threads > 0 && blocks <= 0xFFFFFFFFll / threads;
}

// DART_OK when work on the stream may wait for the host (the stream is not
// being captured into a graph), DART_ERR_UNSUPPORTED when it is being captured,
// DART_ERR_HIP when HIP cannot tell.
inline dart_status_t may_synchronize(hipStream_t stream) {
    hipStreamCaptureStatus cs = hipStreamCaptureStatusNone;
    if (hipStreamIsCapturing(stream, &cs) != hipSuccess) return DART_ERR_HIP;
    return cs == hipStreamCaptureStatusNone ? DART_OK : DART_ERR_UNSUPPORTED;
}

// The optional validation of device-side preconditions (DART_CHECK=1 in the
// environment).
namespace dart_check {

// One device array to validate.
//   Ids:     n int32 values, each in [0, bound)
//   Offsets: n + 1 int32 values, 0 = v[0] < v[1] < ... < v[n] = bound
//   Mask:    n uint8 values, each 0 or 1
struct Item {
    enum Kind { Ids, Offsets, Mask } kind;
    const void* ptr;
    int64_t n;
    int64_t bound;
};

// True when DART_CHECK=1 is set (read on every call, so it can be switched at
// run time).
__attribute__((visibility("hidden"))) bool enabled();

// With checks enabled: runs the validation kernels for every item on stream,
// waits for them and returns DART_ERR_INVALID_ARG if any precondition fails
// (DART_ERR_HIP on a HIP error). With checks disabled: DART_OK, nothing runs.
__attribute__((visibility("hidden"))) dart_status_t run(hipStream_t stream,
                                                        std::initializer_list<Item> items);

}  // namespace dart_check

#pragma GCC visibility pop
