// Device (HIP) twin of the counter-based logits generator in synth/gen.py.
// Same element definition as synth_host.c; every double operation is an
// explicitly rounded intrinsic, so nothing is contracted into an FMA.
// This file holds no arithmetic of the policy-update method.
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace {

__device__ __forceinline__ uint64_t splitmix64(uint64_t x) {
    x += 0x9E3779B97F4A7C15ull;
    x = (x ^ (x >> 30)) * 0xBF58476D1CE4E5B9ull;
    x = (x ^ (x >> 27)) * 0x94D049BB133111EBull;
    return x ^ (x >> 31);
}

__device__ __forceinline__ uint16_t f32_to_bf16_rne(float f) {
    uint32_t u = __float_as_uint(f);
    if ((u & 0x7F800000u) == 0x7F800000u && (u & 0x007FFFFFu)) return (uint16_t)((u >> 16) | 0x40u);
    u += 0x7FFFu + ((u >> 16) & 1u);
    return (uint16_t)(u >> 16);
}

constexpr int kThreads = 256;
constexpr int kColsPerBlock = 4096;

__global__ void __launch_bounds__(kThreads)
synth_logits_kernel(void* __restrict__ out, int dtype, int64_t V, int64_t ld, int64_t chunks,
                    uint64_t key0, double sigma, const int32_t* __restrict__ kind,
                    const int32_t* __restrict__ src_row, const int32_t* __restrict__ spike_col,
                    const double* __restrict__ spike_val, const double* __restrict__ Q) {
    const int64_t t = (int64_t)blockIdx.x / chunks;
    const int64_t c0 = ((int64_t)blockIdx.x % chunks) * kColsPerBlock;
    const uint64_t rowkey = key0 ^ ((uint64_t)(uint32_t)src_row[t] << 28);
    const bool gauss = kind[t] == 0;
    const int64_t sc = spike_col[t];
    const double sv = spike_val[t];
    for (int64_t j = threadIdx.x; j < kColsPerBlock; j += kThreads) {
        const int64_t v = c0 + j;
        if (v >= V) break;
        double base = 0.0;
        if (gauss) base = __dmul_rn(sigma, Q[splitmix64(rowkey ^ (uint64_t)v) >> 48]);
        const double value = __dadd_rn(base, v == sc ? sv : 0.0);
        const float f = __double2float_rn(value);
        if (dtype == 0)
            static_cast<float*>(out)[t * ld + v] = f;
        else
            static_cast<uint16_t*>(out)[t * ld + v] = f32_to_bf16_rne(f);
    }
}

}  // namespace

// Fills out[T, ld] (device memory) with rows 0..T-1. All pointers are device
// pointers. Returns 0 on success, 1 on a bad argument, 2 on a launch error.
extern "C" int synth_logits_device(void* out, int dtype, int64_t T, int64_t V, int64_t ld,
                                   uint64_t key0, double sigma, const int32_t* kind,
                                   const int32_t* src_row, const int32_t* spike_col,
                                   const double* spike_val, const double* Q, hipStream_t stream) {
    if (!out || !kind || !src_row || !spike_col || !spike_val || !Q) return 1;
    if (T < 1 || V < 1 || ld < V || (dtype != 0 && dtype != 1)) return 1;
    const int64_t chunks = (V + kColsPerBlock - 1) / kColsPerBlock;
    const int64_t blocks = T * chunks;
    if (blocks > 0x7FFFFFFFll) return 1;
    hipLaunchKernelGGL(synth_logits_kernel, dim3((unsigned)blocks), dim3(kThreads), 0, stream, out,
                       dtype, V, ld, chunks, key0, sigma, kind, src_row, spike_col, spike_val, Q);
    return hipGetLastError() == hipSuccess ? 0 : 2;
}
