// libdart: DART's policy-update hot path as hand-written HIP for gfx950 (CDNA4).
//
// Paper: DART, arXiv 2509.23866 — token entropy and step entropy (Sec. 4.3),
// high-entropy step selection (Sec. 4.3, indicator of Eq. 2), truncated
// importance sampling (Sec. 4.4), clipped surrogate (Eq. 1, Eq. 2).
//
// Kernels of the path, all launched on the caller's stream:
//   tok_stats_kernel    one workgroup per logits row; one streaming pass with an
//                       online (max, normaliser, entropy) triple in fp32 per lane,
//                       merged across lanes and waves; target logit gathered.
//   step_mean_kernel    one wave per step: mean entropy, fp64 sums in a fixed order.
//   step_select_kernel  one workgroup per group of steps: direct rank of the
//                       step keys (small groups) or radix select of the k-th
//                       largest 32-bit key with LDS histograms; index-ordered ties.
//   tis_coef_kernel     many workgroups: per-token ratio, TIS weight, clip gate and
//                       loss coefficient; partial sums of the loss in fp64
//                       (tis_coef_step_kernel: one workgroup, step-level ratios).
//   tis_loss_finalize_kernel  adds the partial sums in a fixed order.
//   select_coef_kernel  one workgroup: step_select_kernel's and tis_coef_kernel's
//                       device code back to back (up to 4096 tokens), the
//                       offsets and mask handed over in LDS.
//   tis_grad_kernel     one workgroup per 4 KB chunk of a row; second streaming
//                       pass writing coef * (onehot - softmax) in the logits dtype.
// The two streaming kernels are HBM-bound (no matrix contraction anywhere):
// 16-byte non-temporal loads and stores, several loads in flight per lane,
// base-2 exponentials.
#include <hip/hip_runtime.h>
#include <hip/hip_bf16.h>
#include <math.h>
#include <stdint.h>

#include <mutex>
#include <type_traits>

#include "internal.h"
#include "dart.h"

namespace {

constexpr float kLog2e = 1.44269504088896340736f;
constexpr float kLn2 = 0.69314718055994530942f;

typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));

// ------------------------------------------------------------------------
// element access
// ------------------------------------------------------------------------

template <dart_dtype_t D>
struct Elt;
template <>
struct Elt<DART_BF16> {
    using T = uint16_t;
    static constexpr int kPerVec = 8;  // elements per 16-byte vector
};
template <>
struct Elt<DART_F32> {
    using T = float;
    static constexpr int kPerVec = 4;
};

template <dart_dtype_t D>
__device__ __forceinline__ void unpack(const u32x4 v, float* z);

template <>
__device__ __forceinline__ void unpack<DART_BF16>(const u32x4 v, float* z) {
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        z[2 * i] = __uint_as_float(v[i] << 16);
        z[2 * i + 1] = __uint_as_float(v[i] & 0xFFFF0000u);
    }
}

template <>
__device__ __forceinline__ void unpack<DART_F32>(const u32x4 v, float* z) {
#pragma unroll
    for (int i = 0; i < 4; ++i) z[i] = __uint_as_float(v[i]);
}

template <dart_dtype_t D>
__device__ __forceinline__ float load_one(const void* row, int64_t col) {
    if constexpr (D == DART_BF16)
        return __uint_as_float((uint32_t)static_cast<const uint16_t*>(row)[col] << 16);
    else
        return static_cast<const float*>(row)[col];
}

template <dart_dtype_t D>
__device__ __forceinline__ void store_one(void* row, int64_t col, float x) {
    if constexpr (D == DART_BF16) {
        __hip_bfloat16 b = __float2bfloat16(x);  // round to nearest even
        static_cast<__hip_bfloat16*>(row)[col] = b;
    } else {
        static_cast<float*>(row)[col] = x;
    }
}

template <dart_dtype_t D>
__device__ __forceinline__ u32x4 pack(const float* d);

template <>
__device__ __forceinline__ u32x4 pack<DART_BF16>(const float* d) {
    u32x4 v;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        __hip_bfloat162 p = __float22bfloat162_rn(make_float2(d[2 * i], d[2 * i + 1]));
        v[i] = *reinterpret_cast<const uint32_t*>(&p);
    }
    return v;
}

template <>
__device__ __forceinline__ u32x4 pack<DART_F32>(const float* d) {
    u32x4 v;
#pragma unroll
    for (int i = 0; i < 4; ++i) v[i] = __float_as_uint(d[i]);
    return v;
}

// ------------------------------------------------------------------------
// online (max, normaliser, entropy) triple
// ------------------------------------------------------------------------
// For the elements seen so far, with m their maximum and x_v = (z_v - m) log2(e):
//   s = sum_v 2^{x_v},   w = sum_v 2^{x_v} x_v.
// Then lse = m + ln2 log2(s) and H = ln2 (log2(s) - w / s). Two triples merge
// by rescaling to the larger maximum: s' = 2^{d} s, w' = 2^{d} (w + d s),
// d = (m - m_new) log2(e). An empty triple has s == 0 and m == -inf.
struct Triple {
    float m, s, w;
};

__device__ __forceinline__ Triple triple_empty() { return Triple{-INFINITY, 0.f, 0.f}; }

// Adds N elements exactly: the running maximum is updated once per call, then
// every element costs one FMA, one clamp, one exp2, one add and one FMA. The
// clamp keeps 2^x * x finite for -inf logits (2^-256 is 0 in fp32, so no finite
// value moves).
// The logits enter scaled by k = inv_temp * log2(e) (inv_temp > 0); m is kept
// in units of inv_temp * z.
template <int N>
__device__ __forceinline__ void triple_add_exact(Triple& a, const float* z, float inv_temp,
                                                 float k) {
    float cm = z[0];
#pragma unroll
    for (int i = 1; i < N; ++i) cm = fmaxf(cm, z[i]);
    cm *= inv_temp;
    if (cm > a.m) {
        if (a.s > 0.f) {
            const float d = (a.m - cm) * kLog2e;
            const float sc = __builtin_amdgcn_exp2f(d);
            a.w = sc * fmaf(d, a.s, a.w);
            a.s *= sc;
        }
        a.m = cm;
    }
    if (a.m == -INFINITY) return;
    const float mb = a.m * kLog2e;
    float s = 0.f, w = 0.f;
#pragma unroll
    for (int i = 0; i < N; ++i) {
        const float x = fmaxf(fmaf(z[i], k, -mb), -256.f);
        const float e = __builtin_amdgcn_exp2f(x);
        s += e;
        w = fmaf(e, x, w);
    }
    a.s += s;
    a.w += w;
}

// Adds N elements against a lazy reference: the triple's m need not be the
// maximum, only some value that keeps every 2^x term small. A lane takes its
// first finite element as the reference and keeps it while a chunk's terms sum
// below 2^30 (x <= ~30, so fp32 keeps H and lse to a few 1e-6) and are not NaN;
// otherwise (a much larger logit, or a -inf logit making 0 * -inf) the chunk is
// redone exactly, which also moves the reference to the chunk maximum. Per
// element this costs one FMA, one exp2, one add and one FMA: the per-element
// maximum and clamp leave the hot loop.
template <int N>
__device__ __forceinline__ void triple_add(Triple& a, const float* z, float inv_temp, float k) {
    if (a.m == -INFINITY) a.m = z[0] * inv_temp;
    if (a.m != -INFINITY) {
        const float mb = a.m * kLog2e;
        float s = 0.f, w = 0.f;
#pragma unroll
        for (int i = 0; i < N; ++i) {
            const float x = fmaf(z[i], k, -mb);
            const float e = __builtin_amdgcn_exp2f(x);
            s += e;
            w = fmaf(e, x, w);
        }
        if (s < 0x1p30f && w == w) {
            a.s += s;
            a.w += w;
            return;
        }
    }
    triple_add_exact<N>(a, z, inv_temp, k);
}

__device__ __forceinline__ Triple triple_merge(const Triple a, const Triple b) {
    if (b.s == 0.f) return a;
    if (a.s == 0.f) return b;
    const float m = fmaxf(a.m, b.m);
    const float da = (a.m - m) * kLog2e;
    const float db = (b.m - m) * kLog2e;
    const float ca = __builtin_amdgcn_exp2f(da);
    const float cb = __builtin_amdgcn_exp2f(db);
    Triple r;
    r.m = m;
    r.s = ca * a.s + cb * b.s;
    r.w = ca * fmaf(da, a.s, a.w) + cb * fmaf(db, b.s, b.w);
    return r;
}

__device__ __forceinline__ Triple triple_wave_reduce(Triple a) {
#pragma unroll
    for (int off = 32; off >= 1; off >>= 1) {
        Triple b;
        b.m = __shfl_xor(a.m, off);
        b.s = __shfl_xor(a.s, off);
        b.w = __shfl_xor(a.w, off);
        a = triple_merge(a, b);
    }
    return a;
}

// The statistics pass uses THREADS threads per row and UNROLL 16-byte vectors
// per lane per iteration: vector j of the aligned body is read by lane
// j % THREADS in iteration j / (THREADS * UNROLL), so every wave reads 1 KiB
// contiguous per load. With PIPE the iteration loop is unrolled twice over two
// register sets, so the loads of the next iteration are issued before the
// current one is consumed (2 * UNROLL vectors in flight per lane). NTL / NTS
// select non-temporal loads / stores. The entry points instantiate the
// configurations chosen by measurement on MI355X (V = 152064 bf16 rows): the
// read-only statistics pass peaks with 12 waves per row (768 threads); the
// read+write gradient pass with one-shot workgroups of 128 threads x 2
// vectors over 4 KB chunks of a row (best of 32..1024 threads x 1..8 vectors,
// ~15% faster than one 1024-thread workgroup per row and faster than a plain
// elementwise copy). Non-temporal loads and stores win in both; register
// double-buffering does not.
constexpr int kStatsThreads = 768;
constexpr int kStatsUnroll = 4;
constexpr int64_t kStatsMaxRows = int64_t(1) << 22;  // rows per launch of the statistics
static_assert(kStatsMaxRows * kStatsThreads <= 0xFFFFFFFFll, "statistics grid");
constexpr int kGradThreads = 128;
constexpr int kGradUnroll = 2;
constexpr int64_t kGradMaxBlocks = 1ll << 24;
constexpr bool kPipe = false;
constexpr bool kNtLoad = true;
constexpr bool kNtStore = true;

template <bool NT>
__device__ __forceinline__ u32x4 vload(const u32x4* p) {
    if constexpr (NT)
        return __builtin_nontemporal_load(p);
    else
        return *p;
}

template <bool NT>
__device__ __forceinline__ void vstore(const u32x4 v, u32x4* p) {
    if constexpr (NT)
        __builtin_nontemporal_store(v, p);
    else
        *p = v;
}

struct RowLayout {
    int64_t head;      // scalar elements before the first 16-byte boundary
    int64_t nvec;      // aligned 16-byte vectors
    int64_t body_end;  // first element after the vectors
    bool vector_ok;
};

template <dart_dtype_t D>
__device__ __forceinline__ RowLayout row_layout(const void* row, int64_t V) {
    using E = typename Elt<D>::T;
    constexpr int EPV = Elt<D>::kPerVec;
    RowLayout L;
    const uintptr_t addr = reinterpret_cast<uintptr_t>(row);
    L.vector_ok = (addr % sizeof(E)) == 0;
    int64_t head = (int64_t)(((16 - (addr & 15)) & 15) / sizeof(E));
    if (!L.vector_ok) head = V;
    if (head > V) head = V;
    L.head = head;
    L.nvec = (V - head) / EPV;
    L.body_end = head + L.nvec * EPV;
    return L;
}

// Runs body(v, it) over the full iterations of the aligned body, with the
// loads of iteration it+1 in flight while iteration it is consumed when PIPE.
template <int THREADS, int UNROLL, bool PIPE, bool NTL, class Body>
__device__ __forceinline__ void stream_iterations(const u32x4* vrow, int64_t nfull, int tid,
                                                  Body&& body) {
    constexpr int PER_IT = THREADS * UNROLL;
    auto load = [&](u32x4* v, int64_t it) {
#pragma unroll
        for (int u = 0; u < UNROLL; ++u) v[u] = vload<NTL>(vrow + it * PER_IT + u * THREADS + tid);
    };
    if constexpr (!PIPE) {
        for (int64_t it = 0; it < nfull; ++it) {
            u32x4 v[UNROLL];
            load(v, it);
            body(v, it);
        }
    } else {
        u32x4 a[UNROLL], b[UNROLL];
        if (nfull > 0) load(a, 0);
        int64_t it = 0;
        for (; it + 1 < nfull; it += 2) {
            load(b, it + 1);
            body(a, it);
            if (it + 2 < nfull) load(a, it + 2);
            body(b, it + 1);
        }
        if (it < nfull) body(a, it);
    }
}

// ------------------------------------------------------------------------
// K1: token statistics
// ------------------------------------------------------------------------

template <dart_dtype_t D, int THREADS, int UNROLL, bool PIPE, bool NTL>
__global__ void __launch_bounds__(THREADS)
tok_stats_kernel(const void* __restrict__ logits, int64_t V, int64_t ld,
                 const int32_t* __restrict__ target, float inv_temp, float* __restrict__ logp,
                 float* __restrict__ entropy, float* __restrict__ lse) {
    using E = typename Elt<D>::T;
    constexpr int EPV = Elt<D>::kPerVec;
    constexpr int PER_IT = THREADS * UNROLL;
    __shared__ Triple partial[THREADS / 64];

    const int64_t t = blockIdx.x;
    const int tid = threadIdx.x;
    const E* row = static_cast<const E*>(logits) + t * ld;
    // an out-of-range target id (a broken precondition) yields NaN, never a stray read
    const int64_t y_in = target[t];
    const bool y_ok = y_in >= 0 && y_in < V;
    const int64_t y = y_ok ? y_in : -1;
    const RowLayout L = row_layout<D>(row, V);
    const u32x4* vrow = reinterpret_cast<const u32x4*>(row + L.head);

    // The target element is left out of the lane sums and added once at the
    // end, so that 1 - p_target (and logp near 0) keep full relative accuracy.
    const int64_t vy = (y >= L.head && y < L.body_end) ? (y - L.head) / EPV : -1;
    const int64_t it_y = vy >= 0 ? vy / PER_IT : -1;
    const int64_t nfull = L.nvec / PER_IT;

    const float k = inv_temp * kLog2e;
    Triple acc = triple_empty();
    stream_iterations<THREADS, UNROLL, PIPE, NTL>(vrow, nfull, tid, [&](const u32x4* v, int64_t it) {
        float z[UNROLL * EPV];
#pragma unroll
        for (int u = 0; u < UNROLL; ++u) unpack<D>(v[u], z + u * EPV);
        if (it == it_y) {
#pragma unroll
            for (int u = 0; u < UNROLL; ++u)
#pragma unroll
                for (int e = 0; e < EPV; ++e) {
                    const int64_t col = L.head + (it * PER_IT + u * THREADS + tid) * EPV + e;
                    if (col == y) z[u * EPV + e] = -INFINITY;
                }
        }
        triple_add<UNROLL * EPV>(acc, z, inv_temp, k);
    });
    for (int64_t j = nfull * PER_IT + tid; j < L.nvec; j += THREADS) {
        float z[EPV];
        unpack<D>(vload<NTL>(vrow + j), z);
        if (j == vy) {
#pragma unroll
            for (int e = 0; e < EPV; ++e)
                if (L.head + j * EPV + e == y) z[e] = -INFINITY;
        }
        triple_add<EPV>(acc, z, inv_temp, k);
    }
    const int64_t nscalar = L.head + (V - L.body_end);
    for (int64_t q = tid; q < nscalar; q += THREADS) {
        const int64_t col = q < L.head ? q : L.body_end + (q - L.head);
        float z1[1] = {col == y ? -INFINITY : load_one<D>(row, col)};
        triple_add<1>(acc, z1, inv_temp, k);
    }

    acc = triple_wave_reduce(acc);
    const int wave = tid >> 6;
    if ((tid & 63) == 0) partial[wave] = acc;
    __syncthreads();
    if (tid != 0) return;
    Triple x = partial[0];
#pragma unroll
    for (int i = 1; i < THREADS / 64; ++i) x = triple_merge(x, partial[i]);

    // add the target element
    const float zy = y_ok ? load_one<D>(row, y) * inv_temp : __builtin_nanf("");
    const float M = fmaxf(x.m, zy);
    float sx = 0.f, wx = 0.f;
    if (x.s > 0.f) {
        const float dx = (x.m - M) * kLog2e;
        const float cx = __builtin_amdgcn_exp2f(dx);
        sx = cx * x.s;
        wx = cx * fmaf(dx, x.s, x.w);
    }
    const float xy = (zy - M) * kLog2e;
    const float ey = zy == -INFINITY ? 0.f : __builtin_amdgcn_exp2f(xy);
    const float s = sx + ey;
    const float w = ey > 0.f ? fmaf(ey, xy, wx) : wx;
    const float log2s = log2f(s);
    const float ln_s = log2s * kLn2;
    lse[t] = M + ln_s;
    entropy[t] = fmaxf(kLn2 * (log2s - w / s), 0.f);
    // p_y = ey / (sx + ey): -log1p(sx / ey) is exact to a few ulps when p_y -> 1
    logp[t] = sx < ey ? -log1pf(sx / ey) : (zy - M) - ln_s;
}

// ------------------------------------------------------------------------
// K2: step entropy + top-k step selection
// ------------------------------------------------------------------------

constexpr int kSelThreads = 1024;
constexpr int kSelWaves = kSelThreads / 64;
constexpr int kSelLdsKeys = 8192;  // groups up to this many steps keep their keys in LDS
constexpr int kSelLdsTokens = 16384;  // one group of up to this many tokens: means fused in
constexpr int kSelRankMax = 256;   // groups up to this many steps are ranked directly

// Wave sums in a fixed order on the DPP network (no LDS round trips): pairs
// (quad_perm 1,0,3,2), quads (quad_perm 2,3,0,1), half-rows (row_half_mirror),
// rows of 16 (row_mirror), then rows 0+1 and 2+3 (row_bcast15 into rows 1, 3)
// and all four (row_bcast31 into rows 2, 3); lane 63 holds the total, which
// every lane receives. The whole wave must be active. A 64-bit value moves as
// two 32-bit halves under the same control.
template <int CTRL, int ROW_MASK = 0xf>
__device__ __forceinline__ uint64_t dpp_u64(uint64_t x) {
    const int lo = __builtin_amdgcn_update_dpp(0, (int)(uint32_t)x, CTRL, ROW_MASK, 0xf, false);
    const int hi =
        __builtin_amdgcn_update_dpp(0, (int)(uint32_t)(x >> 32), CTRL, ROW_MASK, 0xf, false);
    return ((uint64_t)(uint32_t)hi << 32) | (uint32_t)lo;
}

__device__ __forceinline__ uint64_t lane63_u64(uint64_t x) {
    const uint32_t lo = (uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)x, 63);
    const uint32_t hi = (uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)(x >> 32), 63);
    return ((uint64_t)hi << 32) | lo;
}

template <class Add>
__device__ __forceinline__ uint64_t wave_reduce_u64(uint64_t x, Add add) {
    x = add(x, dpp_u64<0xB1>(x));
    x = add(x, dpp_u64<0x4E>(x));
    x = add(x, dpp_u64<0x141>(x));
    x = add(x, dpp_u64<0x140>(x));
    x = add(x, dpp_u64<0x142, 0xa>(x));
    x = add(x, dpp_u64<0x143, 0xc>(x));
    return lane63_u64(x);
}

__device__ __forceinline__ double wave_sum(double x) {
    const uint64_t r = wave_reduce_u64(__double_as_longlong(x), [](uint64_t a, uint64_t b) {
        return (uint64_t)__double_as_longlong(__longlong_as_double(a) + __longlong_as_double(b));
    });
    return __longlong_as_double(r);
}

__device__ __forceinline__ int64_t wave_sum_i64(int64_t x) {
    return (int64_t)wave_reduce_u64((uint64_t)x, [](uint64_t a, uint64_t b) { return a + b; });
}

// Workgroup barrier for data exchanged through LDS only: waits for the wave's
// LDS accesses (lgkmcnt) but not for its global stores, which the fence of
// __syncthreads would wait for (~1 us each time in the one-workgroup kernels);
// the empty asm statements keep the compiler from moving memory accesses
// across it.
__device__ __forceinline__ void lds_barrier() {
    __builtin_amdgcn_s_waitcnt(0xF | (0x7 << 4) | (0x3 << 14));  // lgkmcnt(0)
    asm volatile("" ::: "memory");
    __builtin_amdgcn_s_barrier();
    asm volatile("" ::: "memory");
}

// Token range of step s, clamped to [0, T] so that malformed offsets (a broken
// precondition) give meaningless numbers but never an out-of-bounds access.
__device__ __forceinline__ void step_bounds(const int32_t* off, int64_t s, int64_t T, int64_t& b,
                                            int64_t& e) {
    b = min(max((int64_t)off[s], (int64_t)0), T);
    e = min(max((int64_t)off[s + 1], b), T);
}

// Order-preserving map of a float to uint32 (larger float -> larger key); -0 == +0.
__device__ __forceinline__ uint32_t float_key(float f) {
    uint32_t u = __float_as_uint(f == 0.f ? 0.f : f);
    return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}

// Step means: one wave per step, lanes stride the step's tokens, fixed
// butterfly order (identical steps give identical means wherever they sit).
// Grid: ceil(S / waves per workgroup), so every step runs in parallel.
__global__ void __launch_bounds__(kSelThreads)
step_mean_kernel(const float* __restrict__ H, int64_t T, const int32_t* __restrict__ off,
                 int64_t S, float* __restrict__ step_H) {
    const int lane = threadIdx.x & 63;
    const int64_t s = (int64_t)blockIdx.x * kSelWaves + (threadIdx.x >> 6);
    if (s >= S) return;
    int64_t b, e;
    step_bounds(off, s, T, b, e);
    double sum = 0.0;
    for (int64_t i = b + lane; i < e; i += 64) sum += (double)H[i];
    sum = wave_sum(sum);
    if (lane == 0) step_H[s] = (float)(sum / (double)(e - b));
}

// k = clamp(ceil(rho * n - 1e-6), 0, n), with the two double operations
// rounded separately (no contraction) so that it equals the host's count.
__device__ __forceinline__ int64_t kept_steps_dev(int64_t n, double rho) {
    double k = ceil(__dsub_rn(__dmul_rn(rho, (double)n), 1e-6));
    k = fmin(fmax(k, 0.0), (double)n);
    return (int64_t)k;
}

// One workgroup per group of steps: group g is steps [grp[g], grp[g+1]) (or all
// S steps when grp is null, with k given); it keeps the ceil(rho S_g) steps of
// highest mean entropy (step_H, from step_mean_kernel) among its own, equal
// means lower step index first: by direct rank in small groups, else by a
// radix select of the k-th key and a scan over the keys equal to it.
// FUSED (one group, T <= kSelLdsTokens, S <= kSelLdsKeys): the workgroup first
// computes the step means itself, from the token entropies and offsets staged
// in LDS, in the order of step_mean_kernel (so with bit-identical results),
// and writes them to step_H.
// LDS of the selection; with the means fused in, also the token entropies
// and the clamped offsets (off_l[s] = first token of step s, off_l[S] = end)
struct SelLds {
    uint32_t keys[kSelLdsKeys];
    uint32_t hist[256];
    uint32_t sel_bin;
    int64_t sel_remaining;
    int64_t wave_count[kSelWaves];
};

template <bool FUSED>
__device__ __forceinline__ void select_steps(const float* __restrict__ H, int64_t T,
                                             const int32_t* __restrict__ off, int64_t S,
                                             const int32_t* __restrict__ grp, double rho,
                                             int64_t k_all, float* __restrict__ step_H,
                                             uint8_t* __restrict__ mask,
                                             int32_t* __restrict__ n_kept, SelLds& sl,
                                             float* H_l, int32_t* off_l,
                                             uint8_t* mask_l = nullptr) {
    uint32_t* keys = sl.keys;
    uint32_t* hist = sl.hist;
    uint32_t& sel_bin = sl.sel_bin;
    int64_t& sel_remaining = sl.sel_remaining;
    int64_t* wave_count = sl.wave_count;

    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = tid >> 6;
    if constexpr (FUSED) {
#pragma unroll 4
        for (int64_t i = tid; i < T; i += kSelThreads) H_l[i] = H[i];
        for (int64_t s = tid; s < S; s += kSelThreads) {
            int64_t b, e;
            step_bounds(off, s, T, b, e);
            off_l[s] = (int32_t)b;
            if (s == S - 1) off_l[S] = (int32_t)e;
        }
        __syncthreads();
        for (int64_t s = wave; s < S; s += kSelWaves) {
            const int64_t b = off_l[s], e = max((int64_t)off_l[s + 1], b);
            double sum = 0.0;
            for (int64_t i = b + lane; i < e; i += 64) sum += (double)H_l[i];
            sum = wave_sum(sum);
            const float m = (float)(sum / (double)(e - b));
            if (lane == 0) {
                step_H[s] = m;
                keys[s] = float_key(m);
            }
        }
        lds_barrier();  // the keys; the step means in global memory are not read here
    }
    int64_t gs = 0, ge = S, k = k_all;
    if (grp) {
        gs = min(max((int64_t)grp[blockIdx.x], (int64_t)0), S);
        ge = min(max((int64_t)grp[blockIdx.x + 1], gs), S);
        k = kept_steps_dev(ge - gs, rho);
    }
    const int64_t Sg = ge - gs;

    if (k <= 0 || k >= Sg) {
        for (int64_t s = gs + tid; s < ge; s += kSelThreads) {
            mask[s] = k > 0 ? 1 : 0;
            if (mask_l) mask_l[s] = k > 0 ? 1 : 0;
        }
        if (tid == 0 && n_kept) n_kept[blockIdx.x] = (int32_t)(k > 0 ? Sg : 0);
        return;
    }

    // the group's keys, read once (LDS when they fit)
    const bool staged = Sg <= kSelLdsKeys;
    if (staged && !FUSED) {
        for (int64_t i = tid; i < Sg; i += kSelThreads) keys[i] = float_key(step_H[gs + i]);
        __syncthreads();
    }
    auto key_at = [&](int64_t i) -> uint32_t {
        return staged ? keys[i] : float_key(step_H[gs + i]);
    };

    if (Sg <= kSelRankMax) {
        // small group: the rank of each step among the group (higher key
        // first, equal keys lower index first) decides directly
        for (int64_t i = tid; i < Sg; i += kSelThreads) {
            const uint32_t ki = keys[i];
            int64_t rank = 0;
            for (int64_t j = 0; j < Sg; ++j) {
                const uint32_t kj = keys[j];
                rank += (kj > ki || (kj == ki && j < i)) ? 1 : 0;
            }
            mask[gs + i] = rank < k ? 1 : 0;
            if (mask_l) mask_l[gs + i] = rank < k ? 1 : 0;
        }
        if (tid == 0 && n_kept) n_kept[blockIdx.x] = (int32_t)k;
        return;
    }

    // radix select of the k-th largest key, 8 bits per pass from the top
    uint32_t prefix = 0, pmask = 0;
    int64_t remaining = k;
    for (int shift = 24; shift >= 0; shift -= 8) {
        for (int i = tid; i < 256; i += kSelThreads) hist[i] = 0;
        __syncthreads();
        for (int64_t i = tid; i < Sg; i += kSelThreads) {
            const uint32_t key = key_at(i);
            if ((key & pmask) == prefix) atomicAdd(&hist[(key >> shift) & 255u], 1u);
        }
        __syncthreads();
        if (wave == 0) {
            // lane l holds bins 255-4l .. 252-4l (descending key order)
            const int b0 = 255 - 4 * lane;
            const uint32_t c0 = hist[b0], c1 = hist[b0 - 1], c2 = hist[b0 - 2], c3 = hist[b0 - 3];
            const int64_t local = (int64_t)c0 + c1 + c2 + c3;
            int64_t incl = local;
#pragma unroll
            for (int d = 1; d < 64; d <<= 1) {
                const int64_t o = __shfl_up(incl, d);
                if (lane >= d) incl += o;
            }
            const int64_t excl = incl - local;
            if (excl < remaining && remaining <= incl) {
                int64_t r = remaining - excl;
                int bin = b0;
                if (r > c0) {
                    r -= c0;
                    bin = b0 - 1;
                    if (r > c1) {
                        r -= c1;
                        bin = b0 - 2;
                        if (r > c2) {
                            r -= c2;
                            bin = b0 - 3;
                        }
                    }
                }
                sel_bin = (uint32_t)bin;
                sel_remaining = r;
            }
        }
        __syncthreads();
        prefix |= sel_bin << shift;
        pmask |= 255u << shift;
        remaining = sel_remaining;
        __syncthreads();
    }

    // keep keys above the k-th; of the keys equal to it keep the first
    // `remaining` in step order (block scan over tiles of kSelThreads steps)
    int64_t carry = 0;
    for (int64_t base = 0; base < Sg; base += kSelThreads) {
        const int64_t i = base + tid;
        const uint32_t key = i < Sg ? key_at(i) : 0u;
        const bool eq = i < Sg && key == prefix;
        const uint64_t ballot = __ballot(eq);
        const int before = __popcll(ballot & ((1ull << lane) - 1ull));
        if (lane == 0) wave_count[wave] = __popcll(ballot);
        __syncthreads();
        int64_t wave_before = 0, total = 0;
        for (int w = 0; w < kSelWaves; ++w) {
            if (w < wave) wave_before += wave_count[w];
            total += wave_count[w];
        }
        if (i < Sg) {
            const int64_t rank = carry + wave_before + before;
            const uint8_t m = (key > prefix || (eq && rank < remaining)) ? 1 : 0;
            mask[gs + i] = m;
            if (mask_l) mask_l[gs + i] = m;
        }
        carry += total;
        __syncthreads();
    }
    if (tid == 0 && n_kept) n_kept[blockIdx.x] = (int32_t)k;
}

template <bool FUSED>
__global__ void __launch_bounds__(kSelThreads)
step_select_kernel(const float* __restrict__ H, int64_t T, const int32_t* __restrict__ off,
                   int64_t S, const int32_t* __restrict__ grp, double rho, int64_t k_all,
                   float* __restrict__ step_H, uint8_t* __restrict__ mask,
                   int32_t* __restrict__ n_kept) {
    __shared__ SelLds sl;
    if constexpr (FUSED) {
        __shared__ float H_l[kSelLdsTokens];
        __shared__ int32_t off_l[kSelLdsKeys + 1];
        select_steps<true>(H, T, off, S, grp, rho, k_all, step_H, mask, n_kept, sl, H_l, off_l);
    } else {
        select_steps<false>(H, T, off, S, grp, rho, k_all, step_H, mask, n_kept, sl, nullptr,
                            nullptr);
    }
}

// ------------------------------------------------------------------------
// step-wise GRPO advantage (Sec. 3.3)
// ------------------------------------------------------------------------

constexpr int kAdvThreads = 256;

// One workgroup per group. Over the group's steps (each step counts its
// trajectory's reward once): mean and population standard deviation, summed
// per trajectory with weight = its step count, in fp64, in a fixed order; then
// every token of trajectory i gets (R_i - mean) / sd (0 when sd == 0).
__global__ void __launch_bounds__(kAdvThreads)
grpo_advantage_kernel(const float* __restrict__ reward, const int32_t* __restrict__ traj_off,
                      int64_t n_traj, const int32_t* __restrict__ grp_off,
                      const int32_t* __restrict__ off, int64_t S, int64_t T,
                      float* __restrict__ adv, float* __restrict__ group_mean,
                      float* __restrict__ group_std) {
    __shared__ double red[2][kAdvThreads / 64];
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int64_t i0 = min(max((int64_t)grp_off[blockIdx.x], (int64_t)0), n_traj);
    const int64_t i1 = min(max((int64_t)grp_off[blockIdx.x + 1], i0), n_traj);
    auto steps_of = [&](int64_t i, int64_t& a, int64_t& b) {
        a = min(max((int64_t)traj_off[i], (int64_t)0), S);
        b = min(max((int64_t)traj_off[i + 1], a), S);
    };
    auto block_sum2 = [&](double& x, double& y) {
        x = wave_sum(x);
        y = wave_sum(y);
        if (lane == 0) {
            red[0][wave] = x;
            red[1][wave] = y;
        }
        __syncthreads();
        x = 0.0;
        y = 0.0;
        for (int i = 0; i < kAdvThreads / 64; ++i) {
            x += red[0][i];
            y += red[1][i];
        }
        __syncthreads();
    };
    double cnt = 0.0, sum = 0.0;
    for (int64_t i = i0 + tid; i < i1; i += kAdvThreads) {
        int64_t a, b;
        steps_of(i, a, b);
        cnt += (double)(b - a);
        sum += (double)(b - a) * (double)reward[i];
    }
    block_sum2(cnt, sum);
    const double mean = cnt > 0.0 ? sum / cnt : 0.0;
    double sq = 0.0, unused = 0.0;
    for (int64_t i = i0 + tid; i < i1; i += kAdvThreads) {
        int64_t a, b;
        steps_of(i, a, b);
        const double d = (double)reward[i] - mean;
        sq += (double)(b - a) * d * d;
    }
    block_sum2(sq, unused);
    const double sd = cnt > 0.0 ? sqrt(sq / cnt) : 0.0;
    if (tid == 0) {
        if (group_mean) group_mean[blockIdx.x] = (float)mean;
        if (group_std) group_std[blockIdx.x] = (float)sd;
    }
    for (int64_t i = i0; i < i1; ++i) {
        int64_t a, b;
        steps_of(i, a, b);
        const float A = sd > 0.0 ? (float)(((double)reward[i] - mean) / sd) : 0.f;
        const int64_t t0 = min(max((int64_t)off[a], (int64_t)0), T);
        const int64_t t1 = min(max((int64_t)off[b], t0), T);
        for (int64_t t = t0 + tid; t < t1; t += kAdvThreads) adv[t] = A;
    }
}

// ------------------------------------------------------------------------
// K3: per-token TIS / clip coefficient and the loss
// ------------------------------------------------------------------------

struct LossConfig {
    float eps_low, eps_high, C, log_C;
    int kl, agg, ratio;
    float beta;
};

// Per token t of step s (M = 1 if the step is kept, else 0):
//   loss term  l_t = -M om_t (w o - beta kl_t),  o = min(r A, clip(r) A)
//   coefficient g_t = dL/dlogp_t = -M (Om w [u <= c] r A dlog - om_t beta dkl_t)
// with om_t the aggregation weight (1/N, 1/T or 1/(K |s|)). Token ratios use
// r = exp(logp - lp_old) and w = min(exp(lp_old - lp_roll), C) per token
// (Om = om_t, dlog = 1); step ratios use the sum (product) or mean (geometric
// mean) of the token log-ratios of the step and its mean advantage, shared by
// all its tokens (Om = om |s|, dlog = 1 or 1/|s|).
//
// Token ratios run on many workgroups (one CU cannot keep enough loads in
// flight to read T tokens quickly); each writes the partial sums of its
// tokens to a small workspace, and tis_loss_finalize_kernel adds them in
// workgroup order. Step ratios run on one workgroup, one wave per step.
// Every sum is in fp64 and in a fixed order: per lane in token order, then a
// fixed butterfly, then waves, then workgroups.

// partial sums per workgroup, in this order
enum { kPartLoss = 0, kPartW, kPartClip, kPartCap, kPartKl, kParts };

constexpr int kCoefThreads = 256;  // workgroup of the many-workgroup launch
constexpr int kCoefWaves = kCoefThreads / 64;
constexpr int kCoefOneThreads = 1024;  // workgroup of the one-workgroup launch
constexpr int kCoefBatch = 4;  // tokens per lane whose loads are in flight together
constexpr int kCoefChunk = kCoefThreads * kCoefBatch;  // tokens per workgroup iteration
constexpr int kCoefMaxBlocks = 1024;
// up to this many tokens the one-workgroup launch is used even with a
// workspace: one launch instead of two (the finalize kernel). Measured on
// MI355X: at T = 512 one workgroup saves ~2.5 us a step; at T = 4096 the
// many-workgroup launch saves ~5 us.
constexpr int64_t kCoefOneBlockMaxT = 2048;
// up to this many tokens the selection and the loss run in one workgroup in
// dart_select_tis_loss_fwd. Measured on MI355X (back to back, S = T / 64):
// 11.0 vs 14.8 us for the two calls at T = 2048, 14.2 vs 16.6 at 4096, 21.0 vs
// 17.7 at 6144, 44 vs 29 at 16384 (the one workgroup's arithmetic grows with T).
constexpr int64_t kSelCoefMaxT = 4096;
constexpr int kCoefLdsSteps = 8192;  // offsets and mask of up to this many steps go to LDS
constexpr int kStepCoefThreads = 1024;
constexpr int kStepCoefWaves = kStepCoefThreads / 64;

// workgroups of the many-workgroup launch for T tokens
__host__ __device__ constexpr int64_t coef_blocks(int64_t T) {
    return (T + kCoefChunk - 1) / kCoefChunk < kCoefMaxBlocks ? (T + kCoefChunk - 1) / kCoefChunk
                                                                : kCoefMaxBlocks;
}

// workspace: kParts doubles per workgroup, then N and K
__host__ __device__ constexpr int64_t coef_workspace_doubles(int64_t nblocks) {
    return nblocks * kParts + 2;
}

// KL estimators of D_KL(pi_theta || pi_ref) from the sampled token, with
// delta = log pi_ref - log pi_theta: k1 = -delta, k2 = delta^2 / 2,
// k3 = exp(delta) - delta - 1 (GRPO's), and their derivatives w.r.t.
// log pi_theta. In double: k3 cancels to O(delta^2) for small delta.
__device__ __forceinline__ void kl_terms(int kl, double delta, double& value, double& dlogp) {
    value = 0.0;
    dlogp = 0.0;
    if (kl == DART_KL_K1) {
        value = -delta;
        dlogp = 1.0;
    } else if (kl == DART_KL_K2) {
        value = 0.5 * delta * delta;
        dlogp = -delta;
    } else if (kl == DART_KL_K3) {
        const double e = exp(delta);
        value = e - delta - 1.0;
        dlogp = 1.0 - e;
    }
}

// Kept tokens N and kept steps K over all S steps, block-wide; with
// off_l/mask_l non-null the (clamped) offsets and the mask are also staged.
template <int THREADS>
__device__ __forceinline__ void count_kept(const int32_t* __restrict__ off,
                                           const uint8_t* __restrict__ mask, int64_t S, int64_t T,
                                           int32_t* off_l, uint8_t* mask_l,
                                           int64_t (*red)[THREADS / 64], int64_t& N, int64_t& K) {
    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = tid >> 6;
    int64_t n_local = 0, k_local = 0;
#pragma unroll 4
    for (int64_t s = tid; s < S; s += THREADS) {
        int64_t b, e;
        step_bounds(off, s, T, b, e);
        const uint8_t m = mask[s];
        if (off_l) {
            off_l[s] = (int32_t)b;
            mask_l[s] = m;
            if (s == S - 1) off_l[S] = (int32_t)e;
        }
        if (m) {
            n_local += e - b;
            k_local += 1;
        }
    }
    n_local = wave_sum_i64(n_local);
    k_local = wave_sum_i64(k_local);
    if (lane == 0) {
        red[0][wave] = n_local;
        red[1][wave] = k_local;
    }
    __syncthreads();
    N = 0;
    K = 0;
    for (int i = 0; i < THREADS / 64; ++i) {
        N += red[0][i];
        K += red[1][i];
    }
}

// N and K from offsets and mask already in LDS (as count_kept stages them).
template <int THREADS>
__device__ __forceinline__ void count_kept_lds(const int32_t* off_l, const uint8_t* mask_l,
                                               int64_t S, int64_t (*red)[THREADS / 64],
                                               int64_t& N, int64_t& K) {
    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = tid >> 6;
    int64_t n_local = 0, k_local = 0;
    // step s ends at max(off_l[s + 1], off_l[s]): the clamped end of step_bounds
    for (int64_t s = tid; s < S; s += THREADS)
        if (mask_l[s]) {
            n_local += (int64_t)max(off_l[s + 1], off_l[s]) - off_l[s];
            k_local += 1;
        }
    n_local = wave_sum_i64(n_local);
    k_local = wave_sum_i64(k_local);
    if (lane == 0) {
        red[0][wave] = n_local;
        red[1][wave] = k_local;
    }
    lds_barrier();
    N = 0;
    K = 0;
    for (int i = 0; i < THREADS / 64; ++i) {
        N += red[0][i];
        K += red[1][i];
    }
}

// Sums the kParts per-lane values over the block in a fixed order (butterfly
// within each wave, then a butterfly over the wave totals in wave 0); the
// result is valid in thread 0.
template <int THREADS>
__device__ __forceinline__ void block_sum_parts(double (&acc)[kParts],
                                                double (*red)[THREADS / 64]) {
    constexpr int WAVES = THREADS / 64;
    static_assert(WAVES <= 64, "one wave adds the wave totals");
    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = tid >> 6;
#pragma unroll
    for (int i = 0; i < kParts; ++i) acc[i] = wave_sum(acc[i]);
    if (lane == 0)
#pragma unroll
        for (int i = 0; i < kParts; ++i) red[i][wave] = acc[i];
    lds_barrier();
    if (wave == 0)
#pragma unroll
        for (int i = 0; i < kParts; ++i) acc[i] = wave_sum(lane < WAVES ? red[i][lane] : 0.0);
}

// Loss and stats = {clip fraction, mean TIS weight, capped fraction, N, mean
// KL, K} (the first nstats of them) from the summed parts.
__device__ __forceinline__ void write_loss(const double (&acc)[kParts], double N, double K,
                                           double* loss, float* stats, int nstats) {
    const double inv_n = N > 0 ? 1.0 / N : 0.0;
    loss[0] = acc[kPartLoss];
    if (stats) {
        const float out[6] = {(float)(acc[kPartClip] * inv_n), (float)(acc[kPartW] * inv_n),
                              (float)(acc[kPartCap] * inv_n), (float)N,
                              (float)(acc[kPartKl] * inv_n), (float)K};
        for (int j = 0; j < nstats; ++j) stats[j] = out[j];
    }
}

// Token ratios. Workgroup b takes chunks b, b + grid, ... of THREADS *
// kCoefBatch tokens; lane tokens are THREADS apart within a chunk (coalesced).
// The step of each token is found by binary search over the offsets. With
// part != null each workgroup writes its partial sums there (workgroup 0 also
// N and K); with part == null the grid is one workgroup, which writes the loss
// and stats itself.
template <int THREADS>
struct CoefRed {
    int64_t i[2][THREADS / 64];
    double d[kParts][THREADS / 64];
};

// The lane's tokens of one chunk of THREADS * kCoefBatch tokens (zeros past T).
struct CoefTokens {
    float A[kCoefBatch], lp[kCoefBatch], lpo[kCoefBatch], lpr[kCoefBatch], lpf[kCoefBatch];
};

template <int THREADS>
__device__ __forceinline__ void load_coef_tokens(CoefTokens& x, int64_t c, int64_t T,
                                                 const float* __restrict__ logp,
                                                 const float* __restrict__ lp_old,
                                                 const float* __restrict__ lp_roll,
                                                 const float* __restrict__ lp_ref,
                                                 const float* __restrict__ adv, bool with_kl) {
    constexpr int CHUNK = THREADS * kCoefBatch;
#pragma unroll
    for (int j = 0; j < kCoefBatch; ++j) {
        const int64_t t = c * CHUNK + threadIdx.x + (int64_t)j * THREADS;
        x.A[j] = x.lp[j] = x.lpo[j] = x.lpr[j] = x.lpf[j] = 0.f;
        if (t < T) {
            x.A[j] = adv[t];
            x.lp[j] = logp[t];
            x.lpo[j] = lp_old[t];
            x.lpr[j] = lp_roll[t];
            if (with_kl) x.lpf[j] = lp_ref[t];
        }
    }
}

// PRE: the caller has put the clamped offsets (off_l[s] = first token of step
// s, off_l[S] = T) and the mask in LDS (S <= kCoefLdsSteps) and loaded this
// workgroup's first chunk into x; else both happen here.
template <bool GENERAL, int THREADS, bool PRE = false>
__device__ __forceinline__ void coef_tokens(
    int64_t T, const float* __restrict__ logp, const float* __restrict__ lp_old,
    const float* __restrict__ lp_roll, const float* __restrict__ lp_ref,
    const float* __restrict__ adv, const int32_t* __restrict__ off, int64_t S,
    const uint8_t* __restrict__ mask, const LossConfig& cfg, float* __restrict__ coef,
    double* __restrict__ part, double* __restrict__ loss, float* __restrict__ stats, int nstats,
    int32_t* off_l, uint8_t* mask_l, CoefRed<THREADS>& red, CoefTokens& x) {
    constexpr int CHUNK = THREADS * kCoefBatch;
    auto& red_i = red.i;
    auto& red_d = red.d;

    const int tid = threadIdx.x;
    const bool with_kl = GENERAL && cfg.kl != DART_KL_NONE;
    const int64_t nchunks = (T + CHUNK - 1) / CHUNK;
    // the lane's tokens of a chunk: loaded before they are needed (the first
    // chunk's loads are in flight while the kept counts are taken)
    float(&A)[kCoefBatch] = x.A;
    float(&lp)[kCoefBatch] = x.lp;
    float(&lpo)[kCoefBatch] = x.lpo;
    float(&lpr)[kCoefBatch] = x.lpr;
    float(&lpf)[kCoefBatch] = x.lpf;
    auto load_chunk = [&](int64_t c) {
        load_coef_tokens<THREADS>(x, c, T, logp, lp_old, lp_roll, lp_ref, adv, with_kl);
    };
    if (!PRE && (int64_t)blockIdx.x < nchunks) load_chunk(blockIdx.x);

    const bool staged = PRE || S <= kCoefLdsSteps;
    int64_t N, K;
    if constexpr (PRE)
        count_kept_lds<THREADS>(off_l, mask_l, S, red_i, N, K);
    else
        count_kept<THREADS>(off, mask, S, T, staged ? off_l : nullptr, staged ? mask_l : nullptr,
                            red_i, N, K);
    if (part && blockIdx.x == 0 && tid == 0) {
        part[(int64_t)gridDim.x * kParts] = (double)N;
        part[(int64_t)gridDim.x * kParts + 1] = (double)K;
    }

    const double inv_n = N > 0 ? 1.0 / (double)N : 0.0;
    const float lo = 1.f - cfg.eps_low, hi = 1.f + cfg.eps_high;
    const double beta = (double)cfg.beta;
    auto weight = [&](int64_t len) -> double {
        if (GENERAL && cfg.agg == DART_AGG_TOKEN_MEAN_ALL) return 1.0 / (double)T;
        if (GENERAL && cfg.agg == DART_AGG_STEP_MEAN) return 1.0 / ((double)K * (double)len);
        return inv_n;
    };
    // largest power of two below S (binary search over step indices [0, S-1])
    int64_t top = 0;
    if (S > 1) {
        top = 1;
        while (top * 2 <= S - 1) top *= 2;
    }

    double acc[kParts] = {0.0, 0.0, 0.0, 0.0, 0.0};
    // the token loop, compiled twice: offsets and mask in LDS or in global
    // memory (a run-time choice per access would serialise the probes)
    auto token_loop = [&](auto staged_tag) {
        constexpr bool STAGED = decltype(staged_tag)::value;
        auto off_at = [&](int64_t i) -> int64_t {
            if constexpr (STAGED)
                return (int64_t)off_l[i];
            else
                return min(max((int64_t)off[i], (int64_t)0), T);
        };
        for (int64_t c = blockIdx.x; c < nchunks; c += gridDim.x) {
            if (c != (int64_t)blockIdx.x) load_chunk(c);
            const int64_t base = c * CHUNK + tid;
            // step of each token: the last s with off[s] <= t, the lane's tokens
            // searched together (every probe of a round issued before any is used)
            int64_t st[kCoefBatch];
#pragma unroll
            for (int j = 0; j < kCoefBatch; ++j) st[j] = 0;
            for (int64_t stride = top; stride > 0; stride >>= 1) {
                int64_t probe[kCoefBatch];
#pragma unroll
                for (int j = 0; j < kCoefBatch; ++j) probe[j] = off_at(min(st[j] + stride, S - 1));
#pragma unroll
                for (int j = 0; j < kCoefBatch; ++j) {
                    const int64_t t = base + (int64_t)j * THREADS;
                    st[j] = (st[j] + stride < S && probe[j] <= t) ? st[j] + stride : st[j];
                }
            }
#pragma unroll
            for (int j = 0; j < kCoefBatch; ++j) {
                const int64_t t = base + (int64_t)j * THREADS;
                if (t >= T) break;
                const bool kept = N > 0 && (STAGED ? mask_l[st[j]] : mask[st[j]]) != 0;
                if (!kept) {
                    coef[t] = 0.f;
                    continue;
                }
                const double om = weight(off_at(st[j] + 1) - off_at(st[j]));
                const float r = expf(lp[j] - lpo[j]);
                const float d = lpo[j] - lpr[j];
                const bool capped = d >= cfg.log_C;
                const float wf = capped ? cfg.C : fminf(expf(d), cfg.C);
                const float rc = fminf(fmaxf(r, lo), hi);
                const float u = r * A[j];
                const float cl = rc * A[j];
                const bool gate = u <= cl;
                const double w = (double)wf;
                const double obj = w * (double)fminf(u, cl);
                const double dobj = gate ? w * (double)A[j] * (double)r : 0.0;
                double klv = 0.0, kld = 0.0;
                if (with_kl) kl_terms(cfg.kl, (double)lpf[j] - (double)lp[j], klv, kld);
                acc[kPartLoss] -= om * (obj - beta * klv);
                coef[t] = (float)(-(om * dobj - om * beta * kld));
                acc[kPartW] += w;
                acc[kPartClip] += gate ? 0.0 : 1.0;
                acc[kPartCap] += capped ? 1.0 : 0.0;
                acc[kPartKl] += klv;
            }
        }
    };
    if (staged)
        token_loop(std::true_type{});
    else
        token_loop(std::false_type{});
    block_sum_parts<THREADS>(acc, red_d);
    if (tid != 0) return;
    if (part)
#pragma unroll
        for (int i = 0; i < kParts; ++i) part[(int64_t)blockIdx.x * kParts + i] = acc[i];
    else
        write_loss(acc, (double)N, (double)K, loss, stats, nstats);
}

template <bool GENERAL, int THREADS>
__global__ void __launch_bounds__(THREADS)
tis_coef_kernel(int64_t T, const float* __restrict__ logp, const float* __restrict__ lp_old,
                const float* __restrict__ lp_roll, const float* __restrict__ lp_ref,
                const float* __restrict__ adv, const int32_t* __restrict__ off, int64_t S,
                const uint8_t* __restrict__ mask, LossConfig cfg, float* __restrict__ coef,
                double* __restrict__ part, double* __restrict__ loss, float* __restrict__ stats,
                int nstats) {
    __shared__ int32_t off_l[kCoefLdsSteps + 1];
    __shared__ uint8_t mask_l[kCoefLdsSteps];
    __shared__ CoefRed<THREADS> red;
    CoefTokens x;
    coef_tokens<GENERAL, THREADS>(T, logp, lp_old, lp_roll, lp_ref, adv, off, S, mask, cfg, coef,
                                  part, loss, stats, nstats, off_l, mask_l, red, x);
}

// Step selection and token coefficients of one group in one workgroup (T <=
// kSelCoefMaxT <= kSelLdsTokens, S <= kSelLdsKeys, token ratios, token mean
// over kept tokens): select_steps with the means fused in, then coef_tokens of the
// one-workgroup launch, the two sharing the staged offsets. Its outputs are
// those of step_select_kernel<true> followed by tis_coef_kernel<false,
// kCoefOneThreads>, bit for bit.
__global__ void __launch_bounds__(kSelThreads)
select_coef_kernel(const float* __restrict__ H, int64_t T, const int32_t* __restrict__ off,
                   int64_t S, double rho, int64_t k, float* __restrict__ step_H,
                   uint8_t* __restrict__ mask, int32_t* __restrict__ n_kept,
                   const float* __restrict__ logp, const float* __restrict__ lp_old,
                   const float* __restrict__ lp_roll, const float* __restrict__ adv,
                   LossConfig cfg, float* __restrict__ coef, double* __restrict__ loss,
                   float* __restrict__ stats, int nstats) {
    static_assert(kSelThreads == kCoefOneThreads, "one workgroup size for both parts");
    static_assert(kSelCoefMaxT <= kSelLdsTokens, "the entropies fit the selection's LDS");
    static_assert(kSelLdsKeys <= kCoefLdsSteps, "the staged offsets serve both parts");
    __shared__ SelLds sl;
    __shared__ float H_l[kSelLdsTokens];
    __shared__ int32_t off_l[kSelLdsKeys + 1];
    __shared__ uint8_t mask_l[kCoefLdsSteps];
    __shared__ CoefRed<kCoefOneThreads> red;
    // the first chunk of tokens is in flight during the selection
    CoefTokens x;
    load_coef_tokens<kCoefOneThreads>(x, 0, T, logp, lp_old, lp_roll, nullptr, adv, false);
    select_steps<true>(H, T, off, S, nullptr, rho, k, step_H, mask, n_kept, sl, H_l, off_l,
                       mask_l);
    lds_barrier();  // the staged offsets and the mask in LDS
    coef_tokens<false, kCoefOneThreads, true>(T, logp, lp_old, lp_roll, nullptr, adv, off, S,
                                              mask, cfg, coef, nullptr, loss, stats, nstats,
                                              off_l, mask_l, red, x);
}

// Step ratios: one workgroup, one wave per step, the step's sums first.
__global__ void __launch_bounds__(kStepCoefThreads)
tis_coef_step_kernel(int64_t T, const float* __restrict__ logp, const float* __restrict__ lp_old,
                     const float* __restrict__ lp_roll, const float* __restrict__ lp_ref,
                     const float* __restrict__ adv, const int32_t* __restrict__ off, int64_t S,
                     const uint8_t* __restrict__ mask, LossConfig cfg, float* __restrict__ coef,
                     double* __restrict__ loss, float* __restrict__ stats, int nstats) {
    __shared__ int64_t red_i[2][kStepCoefWaves];
    __shared__ double red_d[kParts][kStepCoefWaves];

    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = tid >> 6;
    int64_t N, K;
    count_kept<kStepCoefThreads>(off, mask, S, T, nullptr, nullptr, red_i, N, K);

    const double inv_n = N > 0 ? 1.0 / (double)N : 0.0;
    const float lo = 1.f - cfg.eps_low, hi = 1.f + cfg.eps_high;
    const bool with_kl = cfg.kl != DART_KL_NONE;
    const double beta = (double)cfg.beta;
    double acc[kParts] = {0.0, 0.0, 0.0, 0.0, 0.0};
    for (int64_t s = wave; s < S; s += kStepCoefWaves) {
        int64_t b, e;
        step_bounds(off, s, T, b, e);
        const int64_t len = e - b;
        const bool kept = mask[s] != 0 && N > 0;
        if (!kept) {
            for (int64_t t = b + lane; t < e; t += 64) coef[t] = 0.f;
            continue;
        }
        double om = inv_n;
        if (cfg.agg == DART_AGG_TOKEN_MEAN_ALL) om = 1.0 / (double)T;
        if (cfg.agg == DART_AGG_STEP_MEAN) om = 1.0 / ((double)K * (double)len);
        double slr = 0.0, slw = 0.0, sa = 0.0, dlog = 1.0;
        for (int64_t t = b + lane; t < e; t += 64) {
            slr += (double)logp[t] - (double)lp_old[t];
            slw += (double)lp_old[t] - (double)lp_roll[t];
            sa += (double)adv[t];
        }
        slr = wave_sum(slr);
        slw = wave_sum(slw);
        sa = wave_sum(sa);
        if (cfg.ratio == DART_RATIO_STEP_GEOMEAN) {
            slr /= (double)len;
            slw /= (double)len;
            dlog = 1.0 / (double)len;
        }
        const double r_s = exp(slr);
        const bool capped = slw >= (double)cfg.log_C;
        const double w = capped ? (double)cfg.C : fmin(exp(slw), (double)cfg.C);
        const double A_s = sa / (double)len;
        const double om_obj = om * (double)len;
        const double rc = fmin(fmax(r_s, (double)lo), (double)hi);
        const double u = r_s * A_s;
        const double cl = rc * A_s;
        const bool gate = u <= cl;
        const double obj = w * fmin(u, cl);
        const double dobj = gate ? w * r_s * A_s * dlog : 0.0;
        for (int64_t t = b + lane; t < e; t += 64) {
            double klv = 0.0, kld = 0.0;
            if (with_kl) kl_terms(cfg.kl, (double)lp_ref[t] - (double)logp[t], klv, kld);
            acc[kPartLoss] -= om * (obj - beta * klv);
            coef[t] = (float)(-(om_obj * dobj - om * beta * kld));
            acc[kPartW] += w;
            acc[kPartClip] += gate ? 0.0 : 1.0;
            acc[kPartCap] += capped ? 1.0 : 0.0;
            acc[kPartKl] += klv;
        }
    }
    block_sum_parts<kStepCoefThreads>(acc, red_d);
    if (tid == 0) write_loss(acc, (double)N, (double)K, loss, stats, nstats);
}

// Adds the nblocks partial sums in workgroup order and writes the loss and
// stats.
__global__ void __launch_bounds__(kCoefThreads)
tis_loss_finalize_kernel(const double* __restrict__ part, int64_t nblocks,
                         double* __restrict__ loss, float* __restrict__ stats, int nstats) {
    __shared__ double red_d[kParts][kCoefWaves];
    double acc[kParts] = {0.0, 0.0, 0.0, 0.0, 0.0};
    for (int64_t b = threadIdx.x; b < nblocks; b += kCoefThreads)
#pragma unroll
        for (int i = 0; i < kParts; ++i) acc[i] += part[b * kParts + i];
    block_sum_parts<kCoefThreads>(acc, red_d);
    if (threadIdx.x == 0)
        write_loss(acc, part[nblocks * kParts], part[nblocks * kParts + 1], loss, stats, nstats);
}

// ------------------------------------------------------------------------
// K4: dlogits = coef * (onehot(target) - softmax(z))
// ------------------------------------------------------------------------

// dlogits[t, v] = it * g_t * (onehot(y_t)[v] - exp(it * z_tv - lse_t)), it the
// inverse temperature, written in the logits dtype (bf16 rounded to nearest
// even). The body of each row is cut into chunks of THREADS * UNROLL 16-byte
// vectors, and workgroup b takes chunk b % nchunk of row b / nchunk in one
// shot (every load of the lane in flight before its first store); chunk 0 also
// takes the row's unaligned head and tail elements. Small one-shot workgroups
// walking along the rows keep HBM busier than long per-row loops. The target
// element uses 1 - p_y = -expm1(logp_y), accurate when p_y -> 1. dlogits may
// be the logits buffer itself (in place): each element is read, then written,
// by the same lane. With DART_GRAD_SKIP_ZERO_ROWS a row whose coefficient is
// zero is written without reading the logits.
template <dart_dtype_t D, int THREADS, int UNROLL, bool NTL, bool NTS>
__global__ void __launch_bounds__(THREADS)
tis_grad_kernel(const void* logits, int64_t V, int64_t ld,
                      const int32_t* __restrict__ target, const float* __restrict__ lse,
                      const float* __restrict__ logp, const float* __restrict__ coef,
                      float inv_temp, uint32_t flags, void* dlogits, int64_t ld_out, int64_t T,
                      int64_t nchunk) {
    using E = typename Elt<D>::T;
    constexpr int EPV = Elt<D>::kPerVec;
    constexpr int PER = THREADS * UNROLL;
    const int tid = threadIdx.x;
    const int64_t nblocks = T * nchunk;
    for (int64_t b = blockIdx.x; b < nblocks; b += gridDim.x) {
        const int64_t t = b / nchunk;
        const int64_t c = b - t * nchunk;
        const E* row = static_cast<const E*>(logits) + t * ld;
        E* orow = static_cast<E*>(dlogits) + t * ld_out;
        const int64_t y_in = target[t];
        const int64_t y = (y_in >= 0 && y_in < V) ? y_in : -1;
        const float g = coef[t] * inv_temp;
        const float neg_g = -g;
        const float k = inv_temp * kLog2e;
        const float lb = lse[t] * kLog2e;
        const float dy = g * -expm1f(logp[t]);
        RowLayout L = row_layout<D>(row, V);
        const RowLayout Lo = row_layout<D>(orow, V);
        if (L.head != Lo.head || !Lo.vector_ok) L = RowLayout{V, 0, V, false};
        const bool zero_row = (flags & DART_GRAD_SKIP_ZERO_ROWS) && g == 0.f;

        const u32x4* vrow = reinterpret_cast<const u32x4*>(row + L.head);
        u32x4* vout = reinterpret_cast<u32x4*>(orow + L.head);
        const int64_t base = c * PER + tid;
        if (zero_row) {
            const u32x4 zero = {0u, 0u, 0u, 0u};
#pragma unroll
            for (int u = 0; u < UNROLL; ++u) {
                const int64_t j = base + (int64_t)u * THREADS;
                if (j < L.nvec) vstore<NTS>(zero, vout + j);
            }
        } else {
            u32x4 v[UNROLL];
#pragma unroll
            for (int u = 0; u < UNROLL; ++u) {
                const int64_t j = base + (int64_t)u * THREADS;
                if (j < L.nvec) v[u] = vload<NTL>(vrow + j);
            }
#pragma unroll
            for (int u = 0; u < UNROLL; ++u) {
                const int64_t j = base + (int64_t)u * THREADS;
                if (j >= L.nvec) continue;
                float z[EPV];
                unpack<D>(v[u], z);
#pragma unroll
                for (int e = 0; e < EPV; ++e) {
                    z[e] = neg_g * __builtin_amdgcn_exp2f(fmaf(z[e], k, -lb));
                    if (L.head + j * EPV + e == y) z[e] = dy;
                }
                vstore<NTS>(pack<D>(z), vout + j);
            }
        }
        if (c == 0) {
            const int64_t nscalar = L.head + (V - L.body_end);
            for (int64_t q = tid; q < nscalar; q += THREADS) {
                const int64_t col = q < L.head ? q : L.body_end + (q - L.head);
                float d = 0.f;
                if (!zero_row) {
                    const float x = load_one<D>(row, col);
                    d = col == y ? dy : neg_g * __builtin_amdgcn_exp2f(fmaf(x, k, -lb));
                }
                store_one<D>(orow, col, d);
            }
        }
    }
}

// ------------------------------------------------------------------------
// host helpers
// ------------------------------------------------------------------------

bool bad_dtype(dart_dtype_t d) { return d != DART_F32 && d != DART_BF16; }

size_t elem_size(dart_dtype_t d) { return d == DART_F32 ? 4 : 2; }

// dlogits may alias logits exactly (same base, same row stride); any other
// overlap of the two [T, ld] row ranges is rejected.
bool bad_overlap(const void* logits, int64_t ld, const void* dlogits, int64_t ld_out, int64_t T,
                 int64_t V, size_t es) {
    const uintptr_t a0 = reinterpret_cast<uintptr_t>(logits);
    const uintptr_t a1 = a0 + (uintptr_t)(((T - 1) * ld + V) * (int64_t)es);
    const uintptr_t b0 = reinterpret_cast<uintptr_t>(dlogits);
    const uintptr_t b1 = b0 + (uintptr_t)(((T - 1) * ld_out + V) * (int64_t)es);
    const bool alias = a0 == b0 && ld == ld_out;
    return !alias && a0 < b1 && b0 < a1;
}

dart_status_t launch_status() {
    return hipGetLastError() == hipSuccess ? DART_OK : DART_ERR_HIP;
}

// K3 and the loss reduction for one configuration: step ratios on one
// workgroup; token ratios on up to kCoefMaxBlocks workgroups plus the
// finalize kernel when a workspace is given and T > kCoefOneBlockMaxT, else
// on one workgroup.
dart_status_t launch_tis_coef(bool general, int64_t T, const float* logp, const float* lp_old,
                              const float* lp_roll, const float* lp_ref, const float* adv,
                              const int32_t* off, int64_t S, const uint8_t* mask,
                              const LossConfig& cfg, float* coef, double* loss, float* stats,
                              int nstats, void* workspace, hipStream_t stream) {
    if (general && cfg.ratio != DART_RATIO_TOKEN) {
        hipLaunchKernelGGL(tis_coef_step_kernel, dim3(1), dim3(kStepCoefThreads), 0, stream, T,
                           logp, lp_old, lp_roll, lp_ref, adv, off, S, mask, cfg, coef, loss,
                           stats, nstats);
        return launch_status();
    }
    if (!workspace || T <= kCoefOneBlockMaxT) {
        if (general)
            hipLaunchKernelGGL((tis_coef_kernel<true, kCoefOneThreads>), dim3(1),
                               dim3(kCoefOneThreads), 0, stream, T, logp, lp_old, lp_roll, lp_ref,
                               adv, off, S, mask, cfg, coef, nullptr, loss, stats, nstats);
        else
            hipLaunchKernelGGL((tis_coef_kernel<false, kCoefOneThreads>), dim3(1),
                               dim3(kCoefOneThreads), 0, stream, T, logp, lp_old, lp_roll, lp_ref,
                               adv, off, S, mask, cfg, coef, nullptr, loss, stats, nstats);
        return launch_status();
    }
    const int64_t nblocks = coef_blocks(T);
    double* part = static_cast<double*>(workspace);
    if (general)
        hipLaunchKernelGGL((tis_coef_kernel<true, kCoefThreads>), dim3((unsigned)nblocks),
                           dim3(kCoefThreads), 0, stream, T, logp, lp_old, lp_roll, lp_ref, adv,
                           off, S, mask, cfg, coef, part, nullptr, nullptr, 0);
    else
        hipLaunchKernelGGL((tis_coef_kernel<false, kCoefThreads>), dim3((unsigned)nblocks),
                           dim3(kCoefThreads), 0, stream, T, logp, lp_old, lp_roll, lp_ref, adv,
                           off, S, mask, cfg, coef, part, nullptr, nullptr, 0);
    hipLaunchKernelGGL(tis_loss_finalize_kernel, dim3(1), dim3(kCoefThreads), 0, stream, part,
                       nblocks, loss, stats, nstats);
    return launch_status();
}

// A workspace is either absent or large enough and 8-byte aligned.
bool bad_workspace(const void* workspace, size_t bytes, int64_t T) {
    if (!workspace) return false;
    return bytes < (size_t)coef_workspace_doubles(coef_blocks(T)) * sizeof(double) ||
           reinterpret_cast<uintptr_t>(workspace) % sizeof(double) != 0;
}

// Host-side argument rules of dart_tis_loss_fwd_bwd (both halves), workspace
// aside: true when the call must return DART_ERR_INVALID_ARG.
bool bad_fwd_bwd_args(const void* logits, dart_dtype_t dtype, int64_t T, int64_t V, int64_t ld,
                      const int32_t* target, const float* logp, const float* lse,
                      const float* logp_old, const float* logp_rollout, const float* adv,
                      const int32_t* step_offsets, int64_t S, const uint8_t* step_mask,
                      float eps_low, float eps_high, float C, const void* dlogits, int64_t ld_out,
                      const double* loss, const float* tok_coef) {
    if (!logits || !target || !lse || !dlogits) return true;
    if (bad_dtype(dtype) || V < 1 || ld < V || ld_out < V) return true;
    const size_t es = elem_size(dtype);
    if (reinterpret_cast<uintptr_t>(logits) % es || reinterpret_cast<uintptr_t>(dlogits) % es)
        return true;
    if (!logp || !logp_old || !logp_rollout || !adv || !step_offsets || !step_mask || !loss ||
        !tok_coef)
        return true;
    if (T < 1 || S < 1 || S > T || T > 0x7FFFFFFFll) return true;
    if (!(eps_low >= 0.f) || !(eps_high >= 0.f) || !(C > 0.f)) return true;
    return bad_overlap(logits, ld, dlogits, ld_out, T, V, es);
}

// The loss of dart_tis_loss_fwd: token ratios, token mean over kept tokens,
// no KL term.
LossConfig plain_loss_config(float eps_low, float eps_high, float C) {
    LossConfig cfg;
    cfg.eps_low = eps_low;
    cfg.eps_high = eps_high;
    cfg.C = C;
    cfg.log_C = isinf(C) ? INFINITY : (float)log((double)C);
    cfg.kl = DART_KL_NONE;
    cfg.beta = 0.f;
    cfg.agg = DART_AGG_TOKEN_MEAN;
    cfg.ratio = DART_RATIO_TOKEN;
    return cfg;
}

}  // namespace

// Scratch of dart_tis_loss_fwd_bwd_noalloc: the loss kernels' per-workgroup
// partial sums and the kept counts, sized for the largest many-workgroup
// launch (kCoefMaxBlocks workgroups, 40,976 bytes), so every T fits. Each
// device holds its own copy for the life of the process. Host code never
// passes the array's name to a kernel (on the host it is only a stand-in for
// the symbol): the device address comes from hipGetSymbolAddress, once per
// device, with that device current.
constexpr int64_t kNoAllocScratchDoubles = coef_workspace_doubles(kCoefMaxBlocks);
constexpr size_t kNoAllocScratchBytes = (size_t)kNoAllocScratchDoubles * sizeof(double);
static __device__ __align__(256) double scratch[kNoAllocScratchDoubles];

constexpr int kMaxScratchDevices = 64;
static std::mutex g_scratch_mu;
static void* g_scratch_ptr[kMaxScratchDevices] = {};

// The device address of dev's scratch array (null on a HIP error or a device
// index beyond kMaxScratchDevices).
static void* device_scratch(int dev) {
    if (dev < 0 || dev >= kMaxScratchDevices) return nullptr;
    std::lock_guard<std::mutex> lock(g_scratch_mu);
    if (!g_scratch_ptr[dev]) {
        DeviceGuard on_dev(dev);
        if (!on_dev.ok) return nullptr;
        void* ptr = nullptr;
        if (hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch)) != hipSuccess || !ptr) return nullptr;
        g_scratch_ptr[dev] = ptr;
    }
    return g_scratch_ptr[dev];
}

extern "C" {

const char* dart_status_string(dart_status_t status) {
    switch (status) {
        case DART_OK: return "DART_OK";
        case DART_ERR_INVALID_ARG: return "DART_ERR_INVALID_ARG";
        case DART_ERR_UNSUPPORTED: return "DART_ERR_UNSUPPORTED";
        case DART_ERR_HIP: return "DART_ERR_HIP";
    }
    return "DART_ERR_UNKNOWN";
}

int64_t dart_kept_steps(int64_t S, double rho) {
    if (S < 0 || !(rho >= 0.0 && rho <= 1.0)) return -1;
    double k = ceil(rho * (double)S - 1e-6);
    if (k < 0.0) k = 0.0;
    if (k > (double)S) k = (double)S;
    return (int64_t)k;
}

size_t dart_tis_loss_workspace_bytes(int64_t T) {
    if (T < 1 || T > 0x7FFFFFFFll) return 0;
    return (size_t)coef_workspace_doubles(coef_blocks(T)) * sizeof(double);
}

dart_status_t dart_tok_stats_ex(const void* logits, dart_dtype_t dtype, int64_t T, int64_t V,
                                int64_t ld, const int32_t* target, float inv_temp, float* logp,
                                float* entropy, float* lse, hipStream_t stream) {
    if (!logits || !target || !logp || !entropy || !lse) return DART_ERR_INVALID_ARG;
    if (bad_dtype(dtype) || T < 1 || V < 1 || ld < V || T > 0x7FFFFFFFll)
        return DART_ERR_INVALID_ARG;
    if (!(inv_temp > 0.f) || isinf(inv_temp)) return DART_ERR_INVALID_ARG;
    if (reinterpret_cast<uintptr_t>(logits) % elem_size(dtype)) return DART_ERR_INVALID_ARG;
    if (const dart_status_t ck = dart_check::run(
            stream, {{dart_check::Item::Ids, target, T, V}}); ck != DART_OK)
        return ck;
    // one workgroup per row, at most kStatsMaxRows rows per launch (a dispatch
    // holds at most 2^32 - 1 work-items)
    const size_t esz = elem_size(dtype);
    for (int64_t r0 = 0; r0 < T; r0 += kStatsMaxRows) {
        const int64_t rows = T - r0 < kStatsMaxRows ? T - r0 : kStatsMaxRows;
        const void* lr = static_cast<const char*>(logits) + (size_t)r0 * (size_t)ld * esz;
        const dim3 grid((unsigned)rows), block(kStatsThreads);
        if (dtype == DART_BF16)
            hipLaunchKernelGGL(
                (tok_stats_kernel<DART_BF16, kStatsThreads, kStatsUnroll, kPipe, kNtLoad>), grid,
                block, 0, stream, lr, V, ld, target + r0, inv_temp, logp + r0, entropy + r0,
                lse + r0);
        else
            hipLaunchKernelGGL(
                (tok_stats_kernel<DART_F32, kStatsThreads, kStatsUnroll, kPipe, kNtLoad>), grid,
                block, 0, stream, lr, V, ld, target + r0, inv_temp, logp + r0, entropy + r0,
                lse + r0);
    }
    return launch_status();
}

dart_status_t dart_tok_stats(const void* logits, dart_dtype_t dtype, int64_t T, int64_t V,
                             int64_t ld, const int32_t* target, float* logp, float* entropy,
                             float* lse, hipStream_t stream) {
    return dart_tok_stats_ex(logits, dtype, T, V, ld, target, 1.f, logp, entropy, lse, stream);
}

dart_status_t dart_step_select(const float* entropy, int64_t T, const int32_t* step_offsets,
                               int64_t S, double rho, float* step_entropy, uint8_t* step_mask,
                               int32_t* n_kept_steps, hipStream_t stream) {
    if (!entropy || !step_offsets || !step_entropy || !step_mask) return DART_ERR_INVALID_ARG;
    if (T < 1 || S < 1 || S > T || T > 0x7FFFFFFFll) return DART_ERR_INVALID_ARG;
    const int64_t k = dart_kept_steps(S, rho);
    if (k < 0) return DART_ERR_INVALID_ARG;
    if (const dart_status_t ck = dart_check::run(
            stream, {{dart_check::Item::Offsets, step_offsets, S, T}}); ck != DART_OK)
        return ck;
    if (!grid_fits((S + kSelWaves - 1) / kSelWaves, kSelThreads)) return DART_ERR_UNSUPPORTED;
    if (T <= kSelLdsTokens && S <= kSelLdsKeys) {
        hipLaunchKernelGGL(step_select_kernel<true>, dim3(1), dim3(kSelThreads), 0, stream,
                           entropy, T, step_offsets, S, nullptr, rho, k, step_entropy, step_mask,
                           n_kept_steps);
        return launch_status();
    }
    hipLaunchKernelGGL(step_mean_kernel, dim3((unsigned)((S + kSelWaves - 1) / kSelWaves)),
                       dim3(kSelThreads), 0, stream, entropy, T, step_offsets, S, step_entropy);
    hipLaunchKernelGGL(step_select_kernel<false>, dim3(1), dim3(kSelThreads), 0, stream, entropy,
                       T, step_offsets, S, nullptr, rho, k, step_entropy, step_mask, n_kept_steps);
    return launch_status();
}

dart_status_t dart_step_select_groups(const float* entropy, int64_t T,
                                     const int32_t* step_offsets, int64_t S,
                                     const int32_t* group_step_offsets, int64_t G, double rho,
                                     float* step_entropy, uint8_t* step_mask,
                                     int32_t* n_kept_steps, hipStream_t stream) {
    if (!entropy || !step_offsets || !group_step_offsets || !step_entropy || !step_mask)
        return DART_ERR_INVALID_ARG;
    if (T < 1 || S < 1 || S > T || T > 0x7FFFFFFFll || G < 1 || G > S || G > 0x7FFFFFFFll)
        return DART_ERR_INVALID_ARG;
    if (dart_kept_steps(S, rho) < 0) return DART_ERR_INVALID_ARG;
    if (!grid_fits((S + kSelWaves - 1) / kSelWaves, kSelThreads) || !grid_fits(G, kSelThreads))
        return DART_ERR_UNSUPPORTED;
    if (const dart_status_t ck = dart_check::run(
            stream, {{dart_check::Item::Offsets, step_offsets, S, T},
                     {dart_check::Item::Offsets, group_step_offsets, G, S}}); ck != DART_OK)
        return ck;
    hipLaunchKernelGGL(step_mean_kernel, dim3((unsigned)((S + kSelWaves - 1) / kSelWaves)),
                       dim3(kSelThreads), 0, stream, entropy, T, step_offsets, S, step_entropy);
    hipLaunchKernelGGL(step_select_kernel<false>, dim3((unsigned)G), dim3(kSelThreads), 0, stream,
                       entropy, T, step_offsets, S, group_step_offsets, rho, (int64_t)0,
                       step_entropy, step_mask, n_kept_steps);
    return launch_status();
}

dart_status_t dart_grpo_advantage(const float* reward, int64_t n_traj,
                                  const int32_t* traj_step_offsets,
                                  const int32_t* group_traj_offsets, int64_t G,
                                  const int32_t* step_offsets, int64_t S, int64_t T, float* adv,
                                  float* group_mean, float* group_std, hipStream_t stream) {
    if (!reward || !traj_step_offsets || !group_traj_offsets || !step_offsets || !adv)
        return DART_ERR_INVALID_ARG;
    if (n_traj < 1 || G < 1 || G > n_traj || S < 1 || S > T || T > 0x7FFFFFFFll ||
        G > 0x7FFFFFFFll)
        return DART_ERR_INVALID_ARG;
    if (!grid_fits(G, kAdvThreads)) return DART_ERR_UNSUPPORTED;
    if (const dart_status_t ck = dart_check::run(
            stream, {{dart_check::Item::Offsets, traj_step_offsets, n_traj, S},
                     {dart_check::Item::Offsets, group_traj_offsets, G, n_traj},
                     {dart_check::Item::Offsets, step_offsets, S, T}}); ck != DART_OK)
        return ck;
    hipLaunchKernelGGL(grpo_advantage_kernel, dim3((unsigned)G), dim3(kAdvThreads), 0, stream,
                       reward, traj_step_offsets, n_traj, group_traj_offsets, step_offsets, S, T,
                       adv, group_mean, group_std);
    return launch_status();
}

dart_status_t dart_tis_loss_fwd_ex(int64_t T, const float* logp, const float* logp_old,
                                   const float* logp_rollout, const float* logp_ref,
                                   const float* adv, const int32_t* step_offsets, int64_t S,
                                   const uint8_t* step_mask, const dart_loss_config_t* config,
                                   double* loss, float* tok_coef, float* stats, void* workspace,
                                   size_t workspace_bytes, hipStream_t stream) {
    if (!config) return DART_ERR_INVALID_ARG;
    const dart_loss_config_t& c = *config;
    if (c.kl < DART_KL_NONE || c.kl > DART_KL_K3 || c.aggregation < DART_AGG_TOKEN_MEAN ||
        c.aggregation > DART_AGG_STEP_MEAN || c.ratio < DART_RATIO_TOKEN ||
        c.ratio > DART_RATIO_STEP_PRODUCT)
        return DART_ERR_INVALID_ARG;
    if (c.kl != DART_KL_NONE && (!logp_ref || !(c.beta >= 0.f) || isinf(c.beta)))
        return DART_ERR_INVALID_ARG;
    if (!logp || !logp_old || !logp_rollout || !adv || !step_offsets || !step_mask || !loss ||
        !tok_coef)
        return DART_ERR_INVALID_ARG;
    if (T < 1 || S < 1 || S > T || T > 0x7FFFFFFFll) return DART_ERR_INVALID_ARG;
    if (!(c.eps_low >= 0.f) || !(c.eps_high >= 0.f) || !(c.C > 0.f)) return DART_ERR_INVALID_ARG;
    if (bad_workspace(workspace, workspace_bytes, T)) return DART_ERR_INVALID_ARG;
    if (const dart_status_t ck = dart_check::run(
            stream, {{dart_check::Item::Offsets, step_offsets, S, T},
                     {dart_check::Item::Mask, step_mask, S, 0}}); ck != DART_OK)
        return ck;
    LossConfig cfg;
    cfg.eps_low = c.eps_low;
    cfg.eps_high = c.eps_high;
    cfg.C = c.C;
    cfg.log_C = isinf(c.C) ? INFINITY : (float)log((double)c.C);
    cfg.kl = c.kl;
    cfg.beta = c.kl == DART_KL_NONE ? 0.f : c.beta;
    cfg.agg = c.aggregation;
    cfg.ratio = c.ratio;
    return launch_tis_coef(true, T, logp, logp_old, logp_rollout,
                           c.kl == DART_KL_NONE ? nullptr : logp_ref, adv, step_offsets, S,
                           step_mask, cfg, tok_coef, loss, stats, 6, workspace, stream);
}

dart_status_t dart_tis_loss_fwd(int64_t T, const float* logp, const float* logp_old,
                                const float* logp_rollout, const float* adv,
                                const int32_t* step_offsets, int64_t S, const uint8_t* step_mask,
                                float eps_low, float eps_high, float C, double* loss,
                                float* tok_coef, float* stats, void* workspace,
                                size_t workspace_bytes, hipStream_t stream) {
    if (!logp || !logp_old || !logp_rollout || !adv || !step_offsets || !step_mask || !loss ||
        !tok_coef)
        return DART_ERR_INVALID_ARG;
    if (T < 1 || S < 1 || S > T || T > 0x7FFFFFFFll) return DART_ERR_INVALID_ARG;
    if (!(eps_low >= 0.f) || !(eps_high >= 0.f) || !(C > 0.f)) return DART_ERR_INVALID_ARG;
    if (bad_workspace(workspace, workspace_bytes, T)) return DART_ERR_INVALID_ARG;
    if (const dart_status_t ck = dart_check::run(
            stream, {{dart_check::Item::Offsets, step_offsets, S, T},
                     {dart_check::Item::Mask, step_mask, S, 0}}); ck != DART_OK)
        return ck;
    return launch_tis_coef(false, T, logp, logp_old, logp_rollout, nullptr, adv, step_offsets, S,
                           step_mask, plain_loss_config(eps_low, eps_high, C), tok_coef, loss,
                           stats, 4, workspace, stream);
}

dart_status_t dart_select_tis_loss_fwd(int64_t T, const float* entropy, const float* logp,
                                       const float* logp_old, const float* logp_rollout,
                                       const float* adv, const int32_t* step_offsets, int64_t S,
                                       double rho, float eps_low, float eps_high, float C,
                                       float* step_entropy, uint8_t* step_mask,
                                       int32_t* n_kept_steps, double* loss, float* tok_coef,
                                       float* stats, void* workspace, size_t workspace_bytes,
                                       hipStream_t stream) {
    // the argument rules of dart_step_select and dart_tis_loss_fwd, all checked
    // before anything is enqueued
    if (!entropy || !step_offsets || !step_entropy || !step_mask || !logp || !logp_old ||
        !logp_rollout || !adv || !loss || !tok_coef)
        return DART_ERR_INVALID_ARG;
    if (T < 1 || S < 1 || S > T || T > 0x7FFFFFFFll) return DART_ERR_INVALID_ARG;
    const int64_t k = dart_kept_steps(S, rho);
    if (k < 0) return DART_ERR_INVALID_ARG;
    if (!(eps_low >= 0.f) || !(eps_high >= 0.f) || !(C > 0.f)) return DART_ERR_INVALID_ARG;
    if (bad_workspace(workspace, workspace_bytes, T)) return DART_ERR_INVALID_ARG;
    if (T > kSelCoefMaxT || S > kSelLdsKeys) {
        // beyond what one workgroup does faster: the two calls in turn
        const dart_status_t st = dart_step_select(entropy, T, step_offsets, S, rho, step_entropy,
                                                  step_mask, n_kept_steps, stream);
        if (st != DART_OK) return st;
        return dart_tis_loss_fwd(T, logp, logp_old, logp_rollout, adv, step_offsets, S, step_mask,
                                 eps_low, eps_high, C, loss, tok_coef, stats, workspace,
                                 workspace_bytes, stream);
    }
    if (const dart_status_t ck = dart_check::run(
            stream, {{dart_check::Item::Offsets, step_offsets, S, T}}); ck != DART_OK)
        return ck;
    hipLaunchKernelGGL(select_coef_kernel, dim3(1), dim3(kSelThreads), 0, stream, entropy, T,
                       step_offsets, S, rho, k, step_entropy, step_mask, n_kept_steps, logp,
                       logp_old, logp_rollout, adv, plain_loss_config(eps_low, eps_high, C),
                       tok_coef, loss, stats, 4);
    return launch_status();
}

dart_status_t dart_tis_grad_ex(const void* logits, dart_dtype_t dtype, int64_t T, int64_t V,
                               int64_t ld, const int32_t* target, const float* logp,
                               const float* lse, const float* tok_coef, float inv_temp,
                               uint32_t flags, void* dlogits, int64_t ld_out, hipStream_t stream) {
    if (!logits || !target || !logp || !lse || !tok_coef || !dlogits) return DART_ERR_INVALID_ARG;
    if (bad_dtype(dtype) || T < 1 || V < 1 || ld < V || ld_out < V || T > 0x7FFFFFFFll)
        return DART_ERR_INVALID_ARG;
    if (!(inv_temp > 0.f) || isinf(inv_temp) || (flags & ~DART_GRAD_SKIP_ZERO_ROWS))
        return DART_ERR_INVALID_ARG;
    const size_t es = elem_size(dtype);
    if (reinterpret_cast<uintptr_t>(logits) % es || reinterpret_cast<uintptr_t>(dlogits) % es)
        return DART_ERR_INVALID_ARG;
    if (bad_overlap(logits, ld, dlogits, ld_out, T, V, es)) return DART_ERR_INVALID_ARG;
    if (const dart_status_t ck = dart_check::run(
            stream, {{dart_check::Item::Ids, target, T, V}}); ck != DART_OK)
        return ck;
    // chunks of kGradThreads * kGradUnroll vectors per row; a grid of at most
    // kGradMaxBlocks workgroups strides over the T * nchunk chunks
    const int64_t per = (int64_t)kGradThreads * kGradUnroll;
    const int64_t nvec = V / (int64_t)(16 / es);
    const int64_t nchunk = nvec > 0 ? (nvec + per - 1) / per : 1;
    const int64_t nblocks = T * nchunk < kGradMaxBlocks ? T * nchunk : kGradMaxBlocks;
    const dim3 grid((unsigned)nblocks), block(kGradThreads);
    if (dtype == DART_BF16)
        hipLaunchKernelGGL((tis_grad_kernel<DART_BF16, kGradThreads, kGradUnroll, kNtLoad, kNtStore>),
                           grid, block, 0, stream, logits, V, ld, target, lse, logp, tok_coef,
                           inv_temp, flags, dlogits, ld_out, T, nchunk);
    else
        hipLaunchKernelGGL((tis_grad_kernel<DART_F32, kGradThreads, kGradUnroll, kNtLoad, kNtStore>),
                           grid, block, 0, stream, logits, V, ld, target, lse, logp, tok_coef,
                           inv_temp, flags, dlogits, ld_out, T, nchunk);
    return launch_status();
}

dart_status_t dart_tis_grad(const void* logits, dart_dtype_t dtype, int64_t T, int64_t V,
                            int64_t ld, const int32_t* target, const float* logp,
                            const float* lse, const float* tok_coef, void* dlogits,
                            int64_t ld_out, hipStream_t stream) {
    return dart_tis_grad_ex(logits, dtype, T, V, ld, target, logp, lse, tok_coef, 1.f, 0u,
                            dlogits, ld_out, stream);
}

dart_status_t dart_tis_loss_fwd_bwd(const void* logits, dart_dtype_t dtype, int64_t T, int64_t V,
                                    int64_t ld, const int32_t* target, const float* logp,
                                    const float* lse, const float* logp_old,
                                    const float* logp_rollout, const float* adv,
                                    const int32_t* step_offsets, int64_t S,
                                    const uint8_t* step_mask, float eps_low, float eps_high,
                                    float C, void* dlogits, int64_t ld_out, double* loss,
                                    float* tok_coef, float* stats, void* workspace,
                                    size_t workspace_bytes, hipStream_t stream) {
    // validate both halves before enqueuing either
    if (!logits || !target || !lse || !dlogits) return DART_ERR_INVALID_ARG;
    if (bad_dtype(dtype) || V < 1 || ld < V || ld_out < V) return DART_ERR_INVALID_ARG;
    const size_t es = elem_size(dtype);
    if (reinterpret_cast<uintptr_t>(logits) % es || reinterpret_cast<uintptr_t>(dlogits) % es)
        return DART_ERR_INVALID_ARG;
    if (T >= 1 && bad_overlap(logits, ld, dlogits, ld_out, T, V, es)) return DART_ERR_INVALID_ARG;
    // with checks on, all device data is validated before either half enqueues
    if (T >= 1 && S >= 1 && S <= T) {
        const dart_status_t ck = dart_check::run(
            stream, {{dart_check::Item::Ids, target, T, V},
                     {dart_check::Item::Offsets, step_offsets, S, T},
                     {dart_check::Item::Mask, step_mask, S, 0}});
        if (ck != DART_OK) return ck;
    }
    dart_status_t st = dart_tis_loss_fwd(T, logp, logp_old, logp_rollout, adv, step_offsets, S,
                                         step_mask, eps_low, eps_high, C, loss, tok_coef, stats,
                                         workspace, workspace_bytes, stream);
    if (st != DART_OK) return st;
    return dart_tis_grad(logits, dtype, T, V, ld, target, logp, lse, tok_coef, dlogits, ld_out,
                         stream);
}


dart_status_t dart_tis_loss_fwd_bwd_noalloc(const void* logits, dart_dtype_t dtype, int64_t T,
                                            int64_t V, int64_t ld, const int32_t* target,
                                            const float* logp, const float* lse,
                                            const float* logp_old, const float* logp_rollout,
                                            const float* adv, const int32_t* step_offsets,
                                            int64_t S, const uint8_t* step_mask, float eps_low,
                                            float eps_high, float C, void* dlogits, int64_t ld_out,
                                            double* loss, float* tok_coef, float* stats,
                                            hipStream_t stream) {
    // host-side rules first: a bad argument is reported before any HIP call
    if (bad_fwd_bwd_args(logits, dtype, T, V, ld, target, logp, lse, logp_old, logp_rollout, adv,
                         step_offsets, S, step_mask, eps_low, eps_high, C, dlogits, ld_out, loss,
                         tok_coef))
        return DART_ERR_INVALID_ARG;
    // the workspace this T needs must fit the scratch array (always true for
    // T <= INT32_MAX: the many-workgroup launch is capped at kCoefMaxBlocks)
    if (dart_tis_loss_workspace_bytes(T) > kNoAllocScratchBytes) return DART_ERR_UNSUPPORTED;
    const int dev = stream_device(stream);
    if (dev < 0) return DART_ERR_HIP;
    void* ws = device_scratch(dev);
    if (!ws) return DART_ERR_HIP;
    // every argument rule of dart_tis_loss_fwd_bwd applies unchanged
    return dart_tis_loss_fwd_bwd(logits, dtype, T, V, ld, target, logp, lse, logp_old,
                                 logp_rollout, adv, step_offsets, S, step_mask, eps_low, eps_high,
                                 C, dlogits, ld_out, loss, tok_coef, stats, ws,
                                 kNoAllocScratchBytes, stream);
}

}  // extern "C"
