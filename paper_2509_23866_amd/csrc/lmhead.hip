// libdart, LM-head part: the token statistics of the policy-update hot path
// computed straight from the LM head's inputs, so that the [T, V] logits are
// never written to memory.
//
// Paper: DART, arXiv 2509.23866. The statistics are those of Sec. 4.3 (token
// entropy, the target's log-prob of Eq. 1) for logits z = h W^T, where h [T, d]
// are the final hidden states of the T action tokens and W [V, d] the LM-head
// weight of the policy (the 7B VLM of Sec. 5.1: d = 3584, V = 152064).
//
//   lmhead_stats_kernel  one 256 x 256 tile of z per workgroup on MFMA
//                        (v_mfma_f32_32x32x16_bf16, fp32 accumulation), K = d in
//                        slices of 64 loaded straight into an LDS ring; the tile
//                        is reduced in the epilogue to one (max, normaliser,
//                        entropy) triple per row over its 256 columns (the
//                        target column kept apart) and written to a workspace.
//   lmhead_merge_kernel  one wave per row: merges the row's V / 256 triples in
//                        a fixed order, adds the target logit, writes logp, H
//                        and lse exactly as tok_stats_kernel defines them.
#include <hip/hip_runtime.h>
#include <math.h>
#include <rocblas/rocblas.h>
#include <stdint.h>

#include <mutex>

#include "dart.h"

namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));

// Waits until at most N loads of this wave are outstanding (vmcnt), leaving
// the LDS and export counters alone.
template <int N>
__device__ __forceinline__ void wait_vmcnt() {
    static_assert(N >= 0 && N < 64, "vmcnt");
    __builtin_amdgcn_s_waitcnt((N & 0xF) | ((N >> 4) << 14) | (0x7 << 4) | (0xF << 8));
}

// Workgroup barrier of the LDS ring: the caller has waited for its own loads
// into LDS (vmcnt); lgkmcnt(0) retires its LDS reads; the empty asm
// statements keep the compiler from moving memory accesses across it. Unlike
// __syncthreads it carries no fence, which would wait for every load in flight.
__device__ __forceinline__ void lds_ring_barrier() {
    __builtin_amdgcn_s_waitcnt(0xF | (0x3 << 14) | (0x7 << 4));  // lgkmcnt(0)
    asm volatile("" ::: "memory");
    __builtin_amdgcn_s_barrier();
    asm volatile("" ::: "memory");
}

// Tile configuration: BM tokens x BN vocabulary entries per workgroup, K in
// slices of 64 through an NS-buffer LDS ring filled by direct global->LDS
// loads (no staging registers), WM x WN waves each owning a (BM/WM) x (BN/WN)
// block of 32 x 32 MFMA tiles.
template <int BM_, int BN_, int WM_, int WN_, int NS_>
struct Cfg {
    static constexpr int BM = BM_, BN = BN_, BK = 64, WM = WM_, WN = WN_, NS = NS_;
    static constexpr int THREADS = 64 * WM * WN, WAVES = WM * WN;
    static constexpr int TM = BM / WM / 32, TN = BN / WN / 32;  // MFMA tiles per wave
    static constexpr int IA = BM / 8 / WAVES, IB = BN / 8 / WAVES;  // load instructions per slice
    static constexpr int CROW = BN + 1;  // LDS row of the fp32 result tile
    // the epilogue stages EPI rows of the fp32 tile at a time through LDS
    static constexpr int EPI = (BM * CROW * 4 <= 159 * 1024) ? BM : BM / 2;
    static_assert(BM % (32 * WM) == 0 && BN % (32 * WN) == 0, "tile shape");
    static_assert(IA * 8 * WAVES == BM && IB * 8 * WAVES == BN, "rows per wave");
    static_assert(THREADS % EPI == 0 || EPI % THREADS == 0, "epilogue rows");
    struct alignas(16) Smem {
        union {
            struct {
                // slice buffers: 64 bf16 (8 chunks of 16 B) per row, chunk c of
                // row r stored in slot c ^ (r % 8)
                uint16_t a[NS][BM][64];
                uint16_t b[NS][BN][64];
            } in;
            float c[EPI][CROW];
        };
    };
};
// Measured on MI355X at T = 4096, d = 3584, V = 152064 among 128/256-square
// tiles, 4 or 8 waves, 2-4 ring buffers and register-staged loads: 256 x 256
// with 8 waves as 4 x 2 (64 x 128 per wave) and 2 buffers is the fastest.
using LmCfg = Cfg<256, 256, 4, 2, 2>;
constexpr int kMergeWaves = 4;

struct Triple {
    float m, s, w;  // reference, sum of e^{z-m}, sum of e^{z-m} (z-m), natural units
};

// float -> bf16 bits, round to nearest even (NaN kept a quiet NaN)
__device__ __forceinline__ uint16_t bf16_bits(float f) {
    uint32_t u = __float_as_uint(f);
    if ((u & 0x7F800000u) == 0x7F800000u && (u & 0x007FFFFFu)) return (uint16_t)((u >> 16) | 0x40u);
    u += 0x7FFFu + ((u >> 16) & 1u);
    return (uint16_t)(u >> 16);
}

__device__ __forceinline__ uint32_t pack_bf16x2(float lo, float hi) {
    return (uint32_t)bf16_bits(lo) | ((uint32_t)bf16_bits(hi) << 16);
}

// Exact merge of two partial triples; an empty triple has s == 0.
__device__ __forceinline__ Triple merge(const Triple& a, const Triple& b) {
    if (b.s == 0.f) return a;
    if (a.s == 0.f) return b;
    const float m = fmaxf(a.m, b.m);
    const float ca = expf(a.m - m), cb = expf(b.m - m);
    Triple r;
    r.m = m;
    r.s = ca * a.s + cb * b.s;
    r.w = ca * fmaf(a.m - m, a.s, a.w) + cb * fmaf(b.m - m, b.s, b.w);
    return r;
}

// acc = this wave's block of the tile A[m0:m0+BM, :] B[n0:n0+BN, :]^T (A [M, K]
// and B [N, K] row-major bf16, rows 16-byte aligned, K % 8 == 0). Rows past M
// or N read clamped copies of the last row (their results are not used); K
// past the end is zeroed in LDS. Layout of acc[i][j]: value v of lane l is row
// i*32 + (v/4)*8 + (l/32)*4 + v%4, column j*32 + l%32 of the wave's block,
// which starts at row (wave / WN) * BM/WM, column (wave % WN) * BN/WN. Ends
// on a barrier with no loads in flight, so the caller may reuse the LDS.
template <class C>
__device__ __forceinline__ void gemm_tile(const uint16_t* __restrict__ A, int64_t M, int64_t lda,
                                          const uint16_t* __restrict__ B, int64_t N, int64_t ldb,
                                          int64_t K, int64_t m0, int64_t n0,
                                          typename C::Smem& sm,
                                          f32x16 (&acc)[C::TM][C::TN]) {
#if defined(__HIP_DEVICE_COMPILE__)  // the gfx950 builtins below have no host form
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int wr = (wave / C::WN) * (C::BM / C::WM), wc = (wave % C::WN) * (C::BN / C::WN);
#pragma unroll
    for (int i = 0; i < C::TM; ++i)
#pragma unroll
        for (int j = 0; j < C::TN; ++j)
#pragma unroll
            for (int v = 0; v < 16; ++v) acc[i][j][v] = 0.f;

    // one load instruction fills 8 rows x 8 slots (1 KB): lane l writes slot
    // l % 8 of row r0 + l / 8, i.e. chunk (l % 8) ^ (row % 8) of that row
    const int lrow = lane >> 3, lslot = lane & 7;
    auto issue = [&](int64_t kt, int buf) {
#pragma unroll
        for (int q = 0; q < C::IA; ++q) {
            const int r0 = (q * C::WAVES + wave) * 8, r = r0 + lrow;
            const int c = lslot ^ (r & 7);
            const int64_t row = min(m0 + r, M - 1), k = min(kt * 64 + c * 8, K - 8);
            __builtin_amdgcn_global_load_lds(A + row * lda + k, &sm.in.a[buf][r0][0], 16, 0, 0);
        }
#pragma unroll
        for (int q = 0; q < C::IB; ++q) {
            const int r0 = (q * C::WAVES + wave) * 8, r = r0 + lrow;
            const int c = lslot ^ (r & 7);
            const int64_t row = min(n0 + r, N - 1), k = min(kt * 64 + c * 8, K - 8);
            __builtin_amdgcn_global_load_lds(B + row * ldb + k, &sm.in.b[buf][r0][0], 16, 0, 0);
        }
    };
    auto operand = [&](const uint16_t (*tile)[64], int r, int c) {
        return __builtin_bit_cast(
            bf16x8, *reinterpret_cast<const u32x4*>(&tile[r][(c ^ (r & 7)) * 8]));
    };

    const int64_t nk = (K + 63) / 64;
    constexpr int PER = C::IA + C::IB;  // loads per wave and slice
#pragma unroll
    for (int s = 0; s < C::NS - 1; ++s)
        if (s < nk) issue(s, s);
    for (int64_t kt = 0; kt < nk; ++kt) {
        // slice kt has landed (up to NS-2 newer slices stay in flight)
        if (kt + C::NS - 2 < nk)
            wait_vmcnt<(C::NS - 2) * PER>();
        else
            wait_vmcnt<0>();
        lds_ring_barrier();
        const int buf = (int)(kt % C::NS);
        if ((K & 63) && kt == nk - 1) {
            // a partial last slice: zero the chunks past K (they hold clamped copies)
            const u32x4 z = {0u, 0u, 0u, 0u};
            for (int e = tid; e < (C::BM + C::BN) * 8; e += C::THREADS) {
                const int r = e >> 3, c = e & 7;
                if (kt * 64 + c * 8 < K) continue;
                if (r < C::BM)
                    *reinterpret_cast<u32x4*>(&sm.in.a[buf][r][(c ^ (r & 7)) * 8]) = z;
                else
                    *reinterpret_cast<u32x4*>(
                        &sm.in.b[buf][r - C::BM][(c ^ ((r - C::BM) & 7)) * 8]) = z;
            }
            lds_ring_barrier();
        }
        // the buffer refilled here was last read in iteration kt-1, before the barrier
        if (kt + C::NS - 1 < nk) issue(kt + C::NS - 1, (int)((kt + C::NS - 1) % C::NS));

        // the operands of k-step ks+1 are read while the MFMAs of k-step ks issue
        bf16x8 af[2][C::TM], bfr[2][C::TN];
        auto read_step = [&](int ks, int set) {
            const int c = ks * 2 + (lane >> 5);
#pragma unroll
            for (int i = 0; i < C::TM; ++i) af[set][i] = operand(sm.in.a[buf], wr + i * 32 + (lane & 31), c);
#pragma unroll
            for (int j = 0; j < C::TN; ++j) bfr[set][j] = operand(sm.in.b[buf], wc + j * 32 + (lane & 31), c);
        };
        read_step(0, 0);
#pragma unroll
        for (int ks = 0; ks < 4; ++ks) {
            const int cs = ks & 1;
            if (ks < 3) read_step(ks + 1, cs ^ 1);
#pragma unroll
            for (int i = 0; i < C::TM; ++i)
#pragma unroll
                for (int j = 0; j < C::TN; ++j)
                    acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(af[cs][i], bfr[cs][j],
                                                                        acc[i][j], 0, 0, 0);
            if (ks < 3) {
                // interleave: one LDS read, then a share of the MFMAs
#pragma unroll
                for (int g = 0; g < C::TM + C::TN; ++g) {
                    __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
                    __builtin_amdgcn_sched_group_barrier(0x008, (C::TM * C::TN) / (C::TM + C::TN), 0);
                }
            }
        }
    }
    __syncthreads();
#endif
}

// Logical tile of workgroup b: the hardware places workgroup b on XCD b % 8,
// so each XCD gets a contiguous run of logical tiles; tiles run token-tile
// fastest, so the token tiles sharing one slice of W run together on one XCD
// and read it from that XCD's L2.
__device__ __forceinline__ void tile_of_block(int64_t nmt, int64_t nvt, int64_t& mt, int64_t& vt) {
    const int64_t nb = nmt * nvt, q = nb / 8, rr = nb % 8;
    const int64_t b = blockIdx.x, x = b % 8, sl = b / 8;
    const int64_t lg = x * q + min(x, rr) + sl;
    mt = lg % nmt;
    vt = lg / nmt;
}

// part[t * nvt + vt] receives the triple of row t over the tile's columns
// other than target[t]; the workgroup holding target[t] writes z_y[t].
template <class C>
__global__ void __launch_bounds__(C::THREADS)
lmhead_stats_kernel(const uint16_t* __restrict__ h, int64_t T, int64_t ldh,
                    const uint16_t* __restrict__ w, int64_t V, int64_t ldw, int64_t d,
                    const int32_t* __restrict__ target, int64_t nmt, int64_t nvt,
                    float4* __restrict__ part, float* __restrict__ z_y) {
    __shared__ typename C::Smem sm;
    int64_t mt, vt;
    tile_of_block(nmt, nvt, mt, vt);
    const int64_t m0 = mt * C::BM, n0 = vt * C::BN;
    f32x16 acc[C::TM][C::TN];
    gemm_tile<C>(h, T, ldh, w, V, ldw, d, m0, n0, sm, acc);

    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int wr = (wave / C::WN) * (C::BM / C::WM), wc = (wave % C::WN) * (C::BN / C::WN);
    for (int e0 = 0; e0 < C::BM; e0 += C::EPI) {
        if (e0) __syncthreads();
        // rows [e0, e0 + EPI) of the tile to LDS
#pragma unroll
        for (int i = 0; i < C::TM; ++i)
#pragma unroll
            for (int j = 0; j < C::TN; ++j)
#pragma unroll
                for (int v = 0; v < 16; ++v) {
                    const int row = wr + i * 32 + (v >> 2) * 8 + (lane >> 5) * 4 + (v & 3) - e0;
                    if (row >= 0 && row < C::EPI) sm.c[row][wc + j * 32 + (lane & 31)] = acc[i][j][v];
                }
        __syncthreads();
        // P threads per row, BN / P columns each: maximum, then the sums; the
        // P partial triples merged in lane order
        constexpr int P = C::THREADS >= C::EPI ? C::THREADS / C::EPI : 1;
        constexpr int NC = C::BN / P;
        for (int r = tid / P; r < C::EPI; r += C::THREADS / P) {
            const int part_id = tid % P;
            const int64_t t = m0 + e0 + r;
            const int64_t y = t < T ? (int64_t)target[t] : -1;
            const int c0 = part_id * NC;
            int ncol = (int)min((int64_t)NC, V - (n0 + c0));
            if (ncol < 0) ncol = 0;
            const int yc = (int)(y - n0 - c0);  // the target's column here, if 0 <= yc < ncol
            float mx = -INFINITY;
            for (int c = 0; c < ncol; ++c)
                if (c != yc) mx = fmaxf(mx, sm.c[r][c0 + c]);
            Triple mine = {mx, 0.f, 0.f};
            if (mx > -INFINITY) {
                for (int c = 0; c < ncol; ++c) {
                    if (c == yc) continue;
                    const float x = sm.c[r][c0 + c] - mx;
                    const float e = expf(x);
                    mine.s += e;
                    mine.w = fmaf(e, x, mine.w);
                }
            }
#pragma unroll
            for (int off = 1; off < P; off <<= 1) {
                Triple o;
                o.m = __shfl_xor(mine.m, off);
                o.s = __shfl_xor(mine.s, off);
                o.w = __shfl_xor(mine.w, off);
                mine = (part_id & off) ? merge(o, mine) : merge(mine, o);
            }
            if (t < T && part_id == 0) part[t * nvt + vt] = make_float4(mine.m, mine.s, mine.w, 0.f);
            if (t < T && yc >= 0 && yc < ncol) z_y[t] = sm.c[r][c0 + yc];
        }
    }
}

// dlogits = g_t (onehot(y_t) - exp(z - lse_t)) for rows [0, M) of the chunk
// (h and out already offset to the chunk's first row), written in bf16
// (nearest even) to out [M, ld_out]: the gradient pass of the logits path
// with the logits formed on the fly. The target element is
// g_t * -expm1(logp_t), accurate when p_y -> 1. The fp32 tile is staged
// through LDS so that each row leaves as 16-byte vectors.
template <class C>
__global__ void __launch_bounds__(C::THREADS)
lmhead_dlogits_kernel(const uint16_t* __restrict__ h, int64_t M, int64_t ldh,
                      const uint16_t* __restrict__ w, int64_t V, int64_t ldw, int64_t d,
                      const int32_t* __restrict__ target, const float* __restrict__ lse,
                      const float* __restrict__ logp, const float* __restrict__ coef,
                      uint16_t* __restrict__ out, int64_t ld_out, int64_t nmt, int64_t nvt) {
    __shared__ typename C::Smem sm;
    int64_t mt, vt;
    tile_of_block(nmt, nvt, mt, vt);
    const int64_t m0 = mt * C::BM, n0 = vt * C::BN;
    f32x16 acc[C::TM][C::TN];
    gemm_tile<C>(h, M, ldh, w, V, ldw, d, m0, n0, sm, acc);

    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int wr = (wave / C::WN) * (C::BM / C::WM), wc = (wave % C::WN) * (C::BN / C::WN);
    constexpr int CHUNKS = C::BN / 8;  // 16-byte output chunks per tile row
    for (int e0 = 0; e0 < C::BM; e0 += C::EPI) {
        if (e0) __syncthreads();
#pragma unroll
        for (int i = 0; i < C::TM; ++i)
#pragma unroll
            for (int j = 0; j < C::TN; ++j)
#pragma unroll
                for (int v = 0; v < 16; ++v) {
                    const int row = wr + i * 32 + (v >> 2) * 8 + (lane >> 5) * 4 + (v & 3) - e0;
                    if (row >= 0 && row < C::EPI) sm.c[row][wc + j * 32 + (lane & 31)] = acc[i][j][v];
                }
        __syncthreads();
        for (int e = tid; e < C::EPI * CHUNKS; e += C::THREADS) {
            const int r = e / CHUNKS, ch = e % CHUNKS;
            const int64_t t = m0 + e0 + r;
            const int64_t col0 = n0 + ch * 8;
            if (t >= M || col0 >= V) continue;
            const float g = coef[t], lb = lse[t];
            const int64_t y = target[t];
            const float dy = g * -expm1f(logp[t]);
            float dz[8];
#pragma unroll
            for (int q = 0; q < 8; ++q) {
                const int64_t col = col0 + q;
                const float x = sm.c[r][ch * 8 + q];
                dz[q] = col == y ? dy : -g * expf(x - lb);
            }
            uint16_t* dst = out + t * ld_out + col0;
            if (col0 + 8 <= V) {
                u32x4 pk;
                pk.x = pack_bf16x2(dz[0], dz[1]);
                pk.y = pack_bf16x2(dz[2], dz[3]);
                pk.z = pack_bf16x2(dz[4], dz[5]);
                pk.w = pack_bf16x2(dz[6], dz[7]);
                __builtin_nontemporal_store(pk, reinterpret_cast<u32x4*>(dst));
            } else {
                for (int q = 0; q < 8 && col0 + q < V; ++q) dst[q] = bf16_bits(dz[q]);
            }
        }
    }
}

// One wave per row: the row's nvt triples merged lane-strided in index order,
// then across lanes by a butterfly; the target logit is added last, as in
// tok_stats_kernel: lse = M + log S, H = log S - W / S, and logp from
// -log1p(s_rest / e_y) when the target dominates.
__global__ void __launch_bounds__(kMergeWaves * 64)
lmhead_merge_kernel(const float4* __restrict__ part, const float* __restrict__ z_y, int64_t T,
                    int64_t nvt, int64_t V, const int32_t* __restrict__ target,
                    float* __restrict__ logp, float* __restrict__ entropy,
                    float* __restrict__ lse) {
    const int lane = threadIdx.x & 63;
    const int64_t t = (int64_t)blockIdx.x * kMergeWaves + (threadIdx.x >> 6);
    if (t >= T) return;
    Triple acc = {-INFINITY, 0.f, 0.f};
    for (int64_t j = lane; j < nvt; j += 64) {
        const float4 p = part[t * nvt + j];
        acc = merge(acc, Triple{p.x, p.y, p.z});
    }
#pragma unroll
    for (int off = 32; off >= 1; off >>= 1) {
        Triple o;
        o.m = __shfl_xor(acc.m, off);
        o.s = __shfl_xor(acc.s, off);
        o.w = __shfl_xor(acc.w, off);
        acc = merge(acc, o);
    }
    if (lane != 0) return;
    const int64_t y = target[t];
    const float zy = (y >= 0 && y < V) ? z_y[t] : __builtin_nanf("");
    const float M = acc.s > 0.f ? fmaxf(acc.m, zy) : zy;
    float sx = 0.f, wx = 0.f;
    if (acc.s > 0.f) {
        const float dx = acc.m - M;
        const float cx = expf(dx);
        sx = cx * acc.s;
        wx = cx * fmaf(dx, acc.s, acc.w);
    }
    const float xy = zy - M;
    const float ey = expf(xy);
    const float S = sx + ey;
    const float W = fmaf(ey, xy, wx);
    const float ln_s = logf(S);
    lse[t] = M + ln_s;
    entropy[t] = fmaxf(ln_s - W / S, 0.f);
    logp[t] = sx < ey ? -log1pf(sx / ey) : xy - ln_s;
}

int64_t vocab_tiles(int64_t V) { return (V + LmCfg::BN - 1) / LmCfg::BN; }

// Host-side argument rules shared by the LM-head entry points.
bool bad_lmhead_args(const void* hidden, int64_t T, int64_t d, int64_t ld_h, const void* weight,
                     int64_t V, int64_t ld_w) {
    if (!hidden || !weight) return true;
    if (T < 1 || V < 1 || d < 8 || T > 0x7FFFFFFFll || V > 0x7FFFFFFFll || d > 0x7FFFFFFFll)
        return true;
    if (d % 8 || ld_h < d || ld_w < d || ld_h % 8 || ld_w % 8) return true;
    return reinterpret_cast<uintptr_t>(hidden) % 16 || reinterpret_cast<uintptr_t>(weight) % 16;
}

dart_status_t launch_dlogits(const uint16_t* hidden, int64_t rows, int64_t d, int64_t ld_h,
                             const uint16_t* weight, int64_t V, int64_t ld_w,
                             const int32_t* target, const float* lse, const float* logp,
                             const float* coef, uint16_t* out, int64_t ld_out,
                             hipStream_t stream) {
    const int64_t nmt = (rows + LmCfg::BM - 1) / LmCfg::BM, nvt = vocab_tiles(V);
    if (nmt * nvt > 0x7FFFFFFFll) return DART_ERR_UNSUPPORTED;
    hipLaunchKernelGGL(lmhead_dlogits_kernel<LmCfg>, dim3((unsigned)(nmt * nvt)),
                       dim3(LmCfg::THREADS), 0, stream, hidden, rows, ld_h, weight, V, ld_w, d,
                       target, lse, logp, coef, out, ld_out, nmt, nvt);
    return hipGetLastError() == hipSuccess ? DART_OK : DART_ERR_HIP;
}

// One rocBLAS handle per device, created on first use and kept until the
// process ends; calls that use it are serialised by the mutex (the handle's
// stream is set per call).
constexpr int kMaxDevices = 64;
std::mutex g_blas_mu;
rocblas_handle g_blas[kMaxDevices] = {};

// A handle belongs to the device current when it is created.
rocblas_handle blas_handle(int dev) {
    if (dev < 0 || dev >= kMaxDevices) return nullptr;
    if (g_blas[dev]) return g_blas[dev];
    int cur = 0;
    if (hipGetDevice(&cur) != hipSuccess) return nullptr;
    if (cur != dev && hipSetDevice(dev) != hipSuccess) return nullptr;
    if (rocblas_create_handle(&g_blas[dev]) != rocblas_status_success) g_blas[dev] = nullptr;
    if (cur != dev) (void)hipSetDevice(cur);
    return g_blas[dev];
}

}  // namespace

extern "C" {

size_t dart_lmhead_stats_workspace_bytes(int64_t T, int64_t V) {
    if (T < 1 || V < 1 || T > 0x7FFFFFFFll || V > 0x7FFFFFFFll) return 0;
    return (size_t)T * (size_t)vocab_tiles(V) * sizeof(float4) + (size_t)T * sizeof(float);
}

dart_status_t dart_lmhead_tok_stats(const void* hidden, int64_t T, int64_t d, int64_t ld_h,
                                    const void* weight, int64_t V, int64_t ld_w,
                                    const int32_t* target, float* logp, float* entropy,
                                    float* lse, void* workspace, size_t workspace_bytes,
                                    hipStream_t stream) {
    if (bad_lmhead_args(hidden, T, d, ld_h, weight, V, ld_w)) return DART_ERR_INVALID_ARG;
    if (!target || !logp || !entropy || !lse || !workspace ||
        reinterpret_cast<uintptr_t>(workspace) % 16)
        return DART_ERR_INVALID_ARG;
    if (workspace_bytes < dart_lmhead_stats_workspace_bytes(T, V)) return DART_ERR_INVALID_ARG;
    const int64_t nmt = (T + LmCfg::BM - 1) / LmCfg::BM, nvt = vocab_tiles(V);
    if (nmt * nvt > 0x7FFFFFFFll) return DART_ERR_UNSUPPORTED;
    float4* part = static_cast<float4*>(workspace);
    float* z_y = reinterpret_cast<float*>(part + T * nvt);
    hipLaunchKernelGGL(lmhead_stats_kernel<LmCfg>, dim3((unsigned)(nmt * nvt)), dim3(LmCfg::THREADS),
                       0, stream,
                       static_cast<const uint16_t*>(hidden), T, ld_h,
                       static_cast<const uint16_t*>(weight), V, ld_w, d, target, nmt, nvt, part,
                       z_y);
    hipLaunchKernelGGL(lmhead_merge_kernel, dim3((unsigned)((T + kMergeWaves - 1) / kMergeWaves)),
                       dim3(kMergeWaves * 64), 0, stream, part, z_y, T, nvt, V, target, logp,
                       entropy, lse);
    return hipGetLastError() == hipSuccess ? DART_OK : DART_ERR_HIP;
}

dart_status_t dart_lmhead_dlogits(const void* hidden, int64_t T, int64_t d, int64_t ld_h,
                                  const void* weight, int64_t V, int64_t ld_w,
                                  const int32_t* target, const float* lse, const float* logp,
                                  const float* tok_coef, void* dlogits, int64_t ld_out,
                                  hipStream_t stream) {
    if (bad_lmhead_args(hidden, T, d, ld_h, weight, V, ld_w)) return DART_ERR_INVALID_ARG;
    if (!target || !lse || !logp || !tok_coef || !dlogits || ld_out < V || ld_out % 8 ||
        reinterpret_cast<uintptr_t>(dlogits) % 16)
        return DART_ERR_INVALID_ARG;
    return launch_dlogits(static_cast<const uint16_t*>(hidden), T, d, ld_h,
                          static_cast<const uint16_t*>(weight), V, ld_w, target, lse, logp,
                          tok_coef, static_cast<uint16_t*>(dlogits), ld_out, stream);
}

size_t dart_lmhead_backward_workspace_bytes(int64_t chunk_rows, int64_t V) {
    if (chunk_rows < 1 || V < 1 || chunk_rows > 0x7FFFFFFFll || V > 0x7FFFFFFFll) return 0;
    return (size_t)chunk_rows * (size_t)((V + 7) / 8 * 8) * 2;
}

dart_status_t dart_lmhead_backward(const void* hidden, int64_t T, int64_t d, int64_t ld_h,
                                   const void* weight, int64_t V, int64_t ld_w,
                                   const int32_t* target, const float* lse, const float* logp,
                                   const float* tok_coef, float* dhidden, int64_t ld_dh,
                                   float* dweight, int64_t ld_dw, int64_t chunk_rows,
                                   void* workspace, size_t workspace_bytes, hipStream_t stream) {
    if (bad_lmhead_args(hidden, T, d, ld_h, weight, V, ld_w)) return DART_ERR_INVALID_ARG;
    if (!target || !lse || !logp || !tok_coef || !dhidden || !dweight || !workspace)
        return DART_ERR_INVALID_ARG;
    if (ld_dh < d || ld_dw < d || chunk_rows < 1 ||
        reinterpret_cast<uintptr_t>(workspace) % 16)
        return DART_ERR_INVALID_ARG;
    // the BLAS library takes 32-bit sizes and leading dimensions
    const int64_t kI32 = 0x7FFFFFFFll;
    if (ld_h > kI32 || ld_w > kI32 || ld_dh > kI32 || ld_dw > kI32) return DART_ERR_UNSUPPORTED;
    if (chunk_rows > T) chunk_rows = T;
    if (workspace_bytes < dart_lmhead_backward_workspace_bytes(chunk_rows, V))
        return DART_ERR_INVALID_ARG;
    int dev = 0;
    if ((stream ? hipStreamGetDevice(stream, &dev) : hipGetDevice(&dev)) != hipSuccess)
        return DART_ERR_HIP;
    std::lock_guard<std::mutex> lock(g_blas_mu);
    rocblas_handle blas = blas_handle(dev);
    if (!blas || rocblas_set_stream(blas, stream) != rocblas_status_success) return DART_ERR_HIP;
    const int64_t ld_dz = (V + 7) / 8 * 8;
    uint16_t* dz = static_cast<uint16_t*>(workspace);
    const uint16_t* h = static_cast<const uint16_t*>(hidden);
    const uint16_t* w = static_cast<const uint16_t*>(weight);
    const float one = 1.f, zero = 0.f;
    for (int64_t r0 = 0; r0 < T; r0 += chunk_rows) {
        const int64_t rows = T - r0 < chunk_rows ? T - r0 : chunk_rows;
        dart_status_t st = launch_dlogits(h + r0 * ld_h, rows, d, ld_h, w, V, ld_w, target + r0,
                                          lse + r0, logp + r0, tok_coef + r0, dz, ld_dz, stream);
        if (st != DART_OK) return st;
        // rocBLAS is column-major: a row-major [R, C] matrix with row stride ld
        // is its column-major [C, R] transpose with leading dimension ld.
        // dh[rows, d] = dz[rows, V] W[V, d]   <=>   dh^T = W^T dz^T
        if (rocblas_gemm_ex(blas, rocblas_operation_none, rocblas_operation_none, (rocblas_int)d,
                            (rocblas_int)rows, (rocblas_int)V, &one, w, rocblas_datatype_bf16_r,
                            (rocblas_int)ld_w, dz, rocblas_datatype_bf16_r, (rocblas_int)ld_dz,
                            &zero, dhidden + r0 * ld_dh, rocblas_datatype_f32_r,
                            (rocblas_int)ld_dh, dhidden + r0 * ld_dh, rocblas_datatype_f32_r,
                            (rocblas_int)ld_dh, rocblas_datatype_f32_r, rocblas_gemm_algo_standard,
                            0, 0) != rocblas_status_success)
            return DART_ERR_HIP;
        // dW[V, d] (+)= dz^T[V, rows] h[rows, d]   <=>   dW^T = h^T dz
        if (rocblas_gemm_ex(blas, rocblas_operation_none, rocblas_operation_transpose,
                            (rocblas_int)d, (rocblas_int)V, (rocblas_int)rows, &one, h + r0 * ld_h,
                            rocblas_datatype_bf16_r, (rocblas_int)ld_h, dz,
                            rocblas_datatype_bf16_r, (rocblas_int)ld_dz, r0 == 0 ? &zero : &one,
                            dweight, rocblas_datatype_f32_r, (rocblas_int)ld_dw, dweight,
                            rocblas_datatype_f32_r, (rocblas_int)ld_dw, rocblas_datatype_f32_r,
                            rocblas_gemm_algo_standard, 0, 0) != rocblas_status_success)
            return DART_ERR_HIP;
    }
    return hipGetLastError() == hipSuccess ? DART_OK : DART_ERR_HIP;
}

}  // extern "C"
