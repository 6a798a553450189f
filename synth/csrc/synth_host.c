/* Host (C + OpenMP) twin of the counter-based logits generator in synth/gen.py.
 *
 * Element (t, v) of the logits, for row t = rows[i]:
 *   h     = splitmix64(key0 ^ (0 << 56 | src_row[t] << 28 | v))
 *   base  = kind[t] == 0 ? sigma * Q[h >> 48] : 0.0          (IEEE double multiply)
 *   value = base + (v == spike_col[t] ? spike_val[t] : 0.0)  (IEEE double add)
 * rounded to float32, then (bf16 workloads) to bfloat16, both round-to-nearest-even.
 * Build with -ffp-contract=off so the multiply and add are never fused.
 * This file holds no arithmetic of the policy-update method. */
#include <stdint.h>
#include <string.h>

static inline uint64_t splitmix64(uint64_t x) {
    x += 0x9E3779B97F4A7C15ull;
    x = (x ^ (x >> 30)) * 0xBF58476D1CE4E5B9ull;
    x = (x ^ (x >> 27)) * 0x94D049BB133111EBull;
    return x ^ (x >> 31);
}

static inline uint16_t f32_to_bf16_rne(float f) {
    uint32_t u;
    memcpy(&u, &f, 4);
    if ((u & 0x7F800000u) == 0x7F800000u && (u & 0x007FFFFFu)) return (uint16_t)((u >> 16) | 0x40u);
    u += 0x7FFFu + ((u >> 16) & 1u);
    return (uint16_t)(u >> 16);
}

/* out: [nrows, ld] row-major; row i of out holds global row rows[i]. dtype 0 = f32, 1 = bf16. */
void synth_logits_host(void* out, int dtype, int64_t nrows, const int64_t* rows, int64_t V,
                       int64_t ld, uint64_t key0, double sigma, const int32_t* kind,
                       const int32_t* src_row, const int32_t* spike_col, const double* spike_val,
                       const double* Q, int nthreads) {
    if (nthreads < 1) nthreads = 1;
#pragma omp parallel for schedule(dynamic, 1) num_threads(nthreads)
    for (int64_t i = 0; i < nrows; ++i) {
        const int64_t t = rows[i];
        const uint64_t rowkey = key0 ^ ((uint64_t)(uint32_t)src_row[t] << 28);
        const int gauss = kind[t] == 0;
        const int64_t sc = spike_col[t];
        const double sv = spike_val[t];
        for (int64_t v = 0; v < V; ++v) {
            double base = 0.0;
            if (gauss) {
                const uint64_t h = splitmix64(rowkey ^ (uint64_t)v);
                base = sigma * Q[h >> 48];
            }
            const double value = base + (v == sc ? sv : 0.0);
            const float f = (float)value;
            if (dtype == 0)
                ((float*)out)[i * ld + v] = f;
            else
                ((uint16_t*)out)[i * ld + v] = f32_to_bf16_rne(f);
        }
    }
}
