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
#include <stdint.h>

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
    if (!hidden || !weight || !target || !logp || !entropy || !lse || !workspace)
        return DART_ERR_INVALID_ARG;
    if (T < 1 || V < 1 || d < 8 || T > 0x7FFFFFFFll || V > 0x7FFFFFFFll || d > 0x7FFFFFFFll)
        return DART_ERR_INVALID_ARG;
    if (d % 8 || ld_h < d || ld_w < d || ld_h % 8 || ld_w % 8) return DART_ERR_INVALID_ARG;
    if (reinterpret_cast<uintptr_t>(hidden) % 16 || reinterpret_cast<uintptr_t>(weight) % 16 ||
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

}  // extern "C"
