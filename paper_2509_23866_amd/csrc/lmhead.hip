// libdart, LM-head part: the token statistics and the gradient of the
// policy-update hot path computed straight from the LM head's inputs, so that
// the [T, V] logits are never written to memory.
//
// Paper: DART, arXiv 2509.23866. The statistics are those of Sec. 4.3 (token
// entropy, the target's log-prob of Eq. 1) for logits z = h W^T, where h [T, d]
// are the final hidden states of the T action tokens and W [V, d] the LM-head
// weight of the policy (the 7B VLM of Sec. 5.1); the gradient is the chain
// rule of Eq. 2's loss through them. Both kernels scale the fp32 tile by an
// inverse sampling temperature before the epilogue (1 in the paper, App. A.4;
// multiplying by 1 changes no bit).
//
//   lmhead_stats_kernel   one 256 x 256 tile of z per workgroup on MFMA
//                         (v_mfma_f32_32x32x16_bf16, fp32 accumulation), K = d
//                         in slices of 64 loaded straight into two LDS buffers;
//                         the tile is reduced in the epilogue to one (max,
//                         normaliser, entropy) triple per row over its 256
//                         columns (the target column kept apart), written to a
//                         workspace.
//   lmhead_merge_kernel   one wave per row: merges the row's V / 256 triples in
//                         a fixed order, adds the target logit, writes logp, H
//                         and lse exactly as tok_stats_kernel defines them.
//   lmhead_dlogits_kernel the same tile, its epilogue writing
//                         dz = g (onehot - softmax) in bf16.
// The backward forms dz block by block (rows x vocabulary entries, the blocked
// entry point optionally over the rows with a non-zero coefficient only) and
// adds dh = dz W and dW = dz^T h per block with the ROCm BLAS library.
#include <hip/hip_runtime.h>
#include <math.h>
#include <rocblas/rocblas.h>
#include <stdint.h>

#include <mutex>
#include <type_traits>
#include <vector>

#include "internal.h"
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
[[maybe_unused]] __device__ __forceinline__ void lds_ring_barrier() {
    __builtin_amdgcn_s_waitcnt(0xF | (0x3 << 14) | (0x7 << 4));  // lgkmcnt(0)
    asm volatile("" ::: "memory");
    __builtin_amdgcn_s_barrier();
    asm volatile("" ::: "memory");
}

// Tile configuration: BM tokens x BN vocabulary entries per workgroup, K in
// slices of 64 through an NS-buffer LDS ring filled by direct global->LDS
// loads (no staging registers), WM x WN waves each owning a (BM/WM) x (BN/WN)
// block of 32 x 32 MFMA tiles.
// A K slice of BK bf16 per tile row is BK/8 chunks of 16 B. Chunk c of row r
// sits in LDS slot c ^ swz(r). gfx950's LDS serves 16-byte-per-lane reads 16
// lanes at a time across 64 four-byte banks (16 bank quads); a row of CH
// chunks covers CH quads, so 16 / CH consecutive rows tile the banks once and
// the swizzle shifts each such run of rows: the 16 rows that one read cycle
// takes (same chunk c) land in 16 distinct quads. With the plain c ^ (r % 8)
// of a 32-bank LDS, the bank-conflict counter showed half of all LDS cycles
// in two-way conflicts.
template <int CH>
__device__ __forceinline__ int swz(int r) { return (r / (16 / CH)) % CH; }

template <int BM_, int BN_, int WM_, int WN_, int NS_, int BK_ = 64>
struct Cfg {
    static constexpr int BM = BM_, BN = BN_, BK = BK_, WM = WM_, WN = WN_, NS = NS_;
    static_assert(NS == 2, "the K loop alternates two LDS buffers");
    static constexpr int CH = BK / 8;          // 16-byte chunks per row and slice
    static constexpr int LROWS = 64 / CH;      // rows one load instruction fills
    static constexpr int KSTEPS = BK / 16;     // MFMA k-steps per slice
    static constexpr int THREADS = 64 * WM * WN, WAVES = WM * WN;
    static constexpr int TM = BM / WM / 32, TN = BN / WN / 32;  // MFMA tiles per wave
    // a wave's TM row blocks of 32 sit RS = WM * 32 rows apart, so that each
    // epilogue pass over EPI = RS rows takes one block from every wave
    static constexpr int RS = BM / TM;
    static constexpr int IA = BM / LROWS / WAVES, IB = BN / LROWS / WAVES;  // loads per slice
    // LDS row of the fp32 result tile: BN + 16 floats, so that consecutive
    // rows start one bank quad apart: the 16 lanes of one 16-byte read cycle
    // (4 rows x 4 adjacent 16-byte pieces) fall in 16 distinct quads
    static constexpr int CROW = BN + 16;
    // the epilogue stages EPI rows of the fp32 tile at a time through LDS:
    // one 32-row block of every wave
    static constexpr int EPI = RS;
    static_assert(BK == 32 || BK == 64, "slice depth");
    static_assert(BM % (32 * WM) == 0 && BN % (32 * WN) == 0, "tile shape");
    static_assert(IA * LROWS * WAVES == BM && IB * LROWS * WAVES == BN, "rows per wave");
    static_assert(THREADS % EPI == 0 || EPI % THREADS == 0, "epilogue rows");
    struct alignas(16) Smem {
        union {
            struct {
                // slice buffers: BK bf16 per row, chunk c of row r in slot c ^ swz(r)
                uint16_t a[NS][BM][BK];
                uint16_t b[NS][BN][BK];
            } in;
            struct {
                float c[EPI][CROW];
                float4 rowp[EPI];  // per-row constants of the gradient epilogue
            };
        };
    };
};
// Measured on MI355X at T = 4096, d = 3584, V = 152064 among 128/256-square
// tiles, 4 or 8 waves, 2-4 buffers, 32- or 64-wide slices and register-staged
// loads: 256 x 256 with 8 waves as 4 x 2 (64 x 128 per wave) and two 64-wide
// buffers is the fastest.
using LmCfg = Cfg<256, 256, 4, 2, 2>;
static_assert(sizeof(LmCfg::Smem) <= 160 * 1024, "LDS per workgroup");
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

// acc = this wave's part of the tile A[m0:m0+BM, :] B[n0:n0+BN, :]^T (A [M, K]
// and B [N, K] row-major bf16, rows 16-byte aligned, K % 8 == 0). Rows past M
// or N read clamped copies of the last row (their results are not used); K
// past the end is zeroed in LDS. Layout of acc[i][j]: value v of lane l is
// tile row (wave / WN) * 32 + i * RS + (v/4)*8 + (l/32)*4 + v%4, column
// (wave % WN) * BN/WN + j*32 + l%32. Ends on a barrier with no loads in
// flight, so the caller may reuse the LDS.
template <class C>
__device__ __forceinline__ void gemm_tile(const uint16_t* __restrict__ A, int64_t M, int64_t lda,
                                          const uint16_t* __restrict__ B, int64_t N, int64_t ldb,
                                          int64_t K, int64_t m0, int64_t n0,
                                          typename C::Smem& sm,
                                          f32x16 (&acc)[C::TM][C::TN]) {
#if defined(__HIP_DEVICE_COMPILE__)  // the gfx950 builtins below have no host form
    const int tid = threadIdx.x, lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);  // uniform: addresses in SGPRs
    const int wr = (wave / C::WN) * 32, wc = (wave % C::WN) * (C::BN / C::WN);
#pragma unroll
    for (int i = 0; i < C::TM; ++i)
#pragma unroll
        for (int j = 0; j < C::TN; ++j)
#pragma unroll
            for (int v = 0; v < 16; ++v) acc[i][j][v] = 0.f;

    // One load instruction fills LROWS rows x CH slots (1 KB): lane l writes
    // slot l % CH of row r0 + l / CH, i.e. chunk (l % CH) ^ swz(row) of that
    // row. Each lane's source offsets within the tile are fixed for the whole
    // K loop (rows past M or N clamped to the last row), so a full slice's
    // load is a uniform base plus a per-lane 32-bit offset.
    constexpr int CH = C::CH, BK = C::BK;
    const int lrow = lane / CH, lslot = lane % CH;
    const char* a_tile = reinterpret_cast<const char*>(A + m0 * lda);
    const char* b_tile = reinterpret_cast<const char*>(B + n0 * ldb);
    uint32_t aoff[C::IA], boff[C::IB];
#pragma unroll
    for (int q = 0; q < C::IA; ++q) {
        const int r = (q * C::WAVES + wave) * C::LROWS + lrow;
        aoff[q] = (uint32_t)(((min(m0 + r, M - 1) - m0) * lda + (lslot ^ swz<CH>(r)) * 8) * 2);
    }
#pragma unroll
    for (int q = 0; q < C::IB; ++q) {
        const int r = (q * C::WAVES + wave) * C::LROWS + lrow;
        boff[q] = (uint32_t)(((min(n0 + r, N - 1) - n0) * ldb + (lslot ^ swz<CH>(r)) * 8) * 2);
    }
    auto lds_a = [&](int buf, int q) { return &sm.in.a[buf][(q * C::WAVES + wave) * C::LROWS][0]; };
    auto lds_b = [&](int buf, int q) { return &sm.in.b[buf][(q * C::WAVES + wave) * C::LROWS][0]; };
    const int64_t nk = (K + BK - 1) / BK;
    // slice kt into buffer buf; a slice that ends past K clamps each chunk's
    // column to K - 8 (those chunks are zeroed after landing)
    auto issue = [&](int64_t kt, int buf) {
        if ((kt + 1) * BK <= K) {
            const int64_t kb = kt * BK * 2;
#pragma unroll
            for (int q = 0; q < C::IA; ++q)
                __builtin_amdgcn_global_load_lds(a_tile + kb + aoff[q], lds_a(buf, q), 16, 0, 0);
#pragma unroll
            for (int q = 0; q < C::IB; ++q)
                __builtin_amdgcn_global_load_lds(b_tile + kb + boff[q], lds_b(buf, q), 16, 0, 0);
        } else {
#pragma unroll
            for (int q = 0; q < C::IA; ++q) {
                const int r = (q * C::WAVES + wave) * C::LROWS + lrow;
                const int64_t k = min(kt * BK + (lslot ^ swz<CH>(r)) * 8, K - 8);
                __builtin_amdgcn_global_load_lds(A + min(m0 + r, M - 1) * lda + k, lds_a(buf, q), 16, 0, 0);
            }
#pragma unroll
            for (int q = 0; q < C::IB; ++q) {
                const int r = (q * C::WAVES + wave) * C::LROWS + lrow;
                const int64_t k = min(kt * BK + (lslot ^ swz<CH>(r)) * 8, K - 8);
                __builtin_amdgcn_global_load_lds(B + min(n0 + r, N - 1) * ldb + k, lds_b(buf, q), 16, 0, 0);
            }
        }
    };
    // a partial last slice: zero the chunks past K (they hold clamped copies)
    auto zero_tail = [&](int64_t kt, int buf) {
        const u32x4 z = {0u, 0u, 0u, 0u};
        for (int e = tid; e < (C::BM + C::BN) * CH; e += C::THREADS) {
            const int r = e / CH, c = e % CH;
            if (kt * BK + c * 8 < K) continue;
            if (r < C::BM)
                *reinterpret_cast<u32x4*>(&sm.in.a[buf][r][(c ^ swz<CH>(r)) * 8]) = z;
            else
                *reinterpret_cast<u32x4*>(
                    &sm.in.b[buf][r - C::BM][(c ^ swz<CH>(r - C::BM)) * 8]) = z;
        }
    };

    // MFMA operands: lane l reads row (l % 32) of each 32-row block, chunk
    // 2 ks + l / 32. The rows' swizzle depends only on l % 32 (blocks start at
    // multiples of 32), so one byte offset per k-step serves every block, the
    // block and the buffer entering as immediate offsets.
    uint32_t rda[C::KSTEPS], rdb[C::KSTEPS];
#pragma unroll
    for (int ks = 0; ks < C::KSTEPS; ++ks) {
        const int c = ks * 2 + (lane >> 5), ra = wr + (lane & 31), rb = wc + (lane & 31);
        rda[ks] = (uint32_t)(ra * BK + (c ^ swz<CH>(ra)) * 8) * 2;
        rdb[ks] = (uint32_t)(rb * BK + (c ^ swz<CH>(rb)) * 8) * 2;
    }
    bf16x8 af[2][C::TM], bfr[2][C::TN];
    auto read_step = [&](auto bufc, int ks, int set) {
        constexpr int buf = decltype(bufc)::value;
        const char* ba = reinterpret_cast<const char*>(&sm.in.a[buf][0][0]);
        const char* bb = reinterpret_cast<const char*>(&sm.in.b[buf][0][0]);
#pragma unroll
        for (int i = 0; i < C::TM; ++i)
            af[set][i] = __builtin_bit_cast(
                bf16x8, *reinterpret_cast<const u32x4*>(ba + rda[ks] + i * C::RS * BK * 2));
#pragma unroll
        for (int j = 0; j < C::TN; ++j)
            bfr[set][j] = __builtin_bit_cast(
                bf16x8, *reinterpret_cast<const u32x4*>(bb + rdb[ks] + j * 32 * BK * 2));
    };
    auto mfmas = [&](int set) {
#pragma unroll
        for (int i = 0; i < C::TM; ++i)
#pragma unroll
            for (int j = 0; j < C::TN; ++j)
                acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(af[set][i], bfr[set][j],
                                                                    acc[i][j], 0, 0, 0);
    };

    // two LDS buffers: slice kt+1 loads while slice kt is multiplied
    auto slice = [&](auto bufc, int64_t kt) {
        constexpr int buf = decltype(bufc)::value;
        // slice kt has landed for this wave; the barrier makes it so for all,
        // and every wave has finished reading the other buffer (slice kt-1)
        wait_vmcnt<0>();
        lds_ring_barrier();
        if ((K % BK) && kt == nk - 1) {
            zero_tail(kt, buf);
            lds_ring_barrier();
        }
        if (kt + 1 < nk) issue(kt + 1, buf ^ 1);
        // the operands of k-step ks+1 are read while the MFMAs of k-step ks issue
        read_step(bufc, 0, 0);
#pragma unroll
        for (int ks = 0; ks < C::KSTEPS; ++ks) {
            const int cs = ks & 1;
            if (ks < C::KSTEPS - 1) read_step(bufc, ks + 1, cs ^ 1);
            mfmas(cs);
            if (ks < C::KSTEPS - 1) {
                // interleave: one LDS read, then a share of the MFMAs
#pragma unroll
                for (int g = 0; g < C::TM + C::TN; ++g) {
                    __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
                    __builtin_amdgcn_sched_group_barrier(0x008, (C::TM * C::TN) / (C::TM + C::TN), 0);
                }
            }
        }
    };
    issue(0, 0);
    for (int64_t kt = 0; kt < nk; kt += 2) {
        slice(std::integral_constant<int, 0>{}, kt);
        if (kt + 1 < nk) slice(std::integral_constant<int, 1>{}, kt + 1);
    }
    __syncthreads();
#else
    (void)A, (void)M, (void)lda, (void)B, (void)N, (void)ldb, (void)K, (void)m0, (void)n0;
    (void)sm, (void)acc;
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
                    const int32_t* __restrict__ target, float scale, int64_t nmt, int64_t nvt,
                    float4* __restrict__ part, float* __restrict__ z_y) {
    __shared__ typename C::Smem sm;
    int64_t mt, vt;
    tile_of_block(nmt, nvt, mt, vt);
    const int64_t m0 = mt * C::BM, n0 = vt * C::BN;
    f32x16 acc[C::TM][C::TN];
    gemm_tile<C>(h, T, ldh, w, V, ldw, d, m0, n0, sm, acc);

    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int wr = (wave / C::WN) * 32, wc = (wave % C::WN) * (C::BN / C::WN);
#pragma unroll
    for (int e0 = 0; e0 < C::BM; e0 += C::EPI) {
        if (e0) __syncthreads();
        // rows [e0, e0 + EPI) of the tile to LDS
#pragma unroll
        for (int i = 0; i < C::TM; ++i)
#pragma unroll
            for (int j = 0; j < C::TN; ++j)
#pragma unroll
                for (int v = 0; v < 16; ++v) {
                    const int row = wr + i * C::RS + (v >> 2) * 8 + (lane >> 5) * 4 + (v & 3) - e0;
                    if (row >= 0 && row < C::EPI)
                        sm.c[row][wc + j * 32 + (lane & 31)] = acc[i][j][v] * scale;
                }
        __syncthreads();
        // P threads per row; thread p takes the 16-byte pieces p, p + P, ...
        // of the row (columns 16 c + 4 p + u) into registers: maximum over the
        // row's columns other than the target, then the sums in base-2 units
        // against it; the P partial triples merged in lane order
        constexpr int P = C::THREADS / C::EPI, NX = C::BN / P;
        static_assert(C::THREADS == C::EPI * P && P == 4, "four threads per epilogue row");
        const int r = tid / P, p = tid % P;
        const int64_t t = m0 + e0 + r;
        const int64_t yrel = (t < T ? (int64_t)target[t] : -1) - n0;
        // columns below vlim exist; the target sits at column y32 (-1: not here)
        const int vlim = (int)min(V - n0, (int64_t)C::BN);
        const int y32 = yrel >= 0 && yrel < vlim ? (int)yrel : -1;
        // the thread's 64 columns in two halves of 32 registers, each folded
        // into a triple (maximum, then the sums in base-2 units against it)
        // and merged; columns past V and the target's column drop out as -inf
        constexpr int NH = NX / 2;
        Triple mine = {-INFINITY, 0.f, 0.f};
#pragma unroll
        for (int hh = 0; hh < 2; ++hh) {
            float x[NH];
            float mx = -INFINITY;
#pragma unroll
            for (int c4 = 0; c4 < NH / 4; ++c4) {
                const int cc = hh * (NH / 4) + c4;
                const float4 q = *reinterpret_cast<const float4*>(&sm.c[r][16 * cc + 4 * p]);
                const float qv[4] = {q.x, q.y, q.z, q.w};
#pragma unroll
                for (int u = 0; u < 4; ++u) {
                    const int col = 16 * cc + 4 * p + u;
                    x[4 * c4 + u] = col < vlim && col != y32 ? qv[u] : -INFINITY;
                    mx = fmaxf(mx, x[4 * c4 + u]);
                }
            }
            Triple part_h = {mx, 0.f, 0.f};
            if (mx > -INFINITY) {
                // e = 2^xl with xl = (x - mx) log2(e) floored at -200, where 2^xl
                // is already 0 in fp32, so that dropped columns add 0
                constexpr float kLog2e = 1.4426950408889634f;
                const float ml = mx * kLog2e;
                float s2 = 0.f, w2 = 0.f;
#pragma unroll
                for (int i = 0; i < NH; ++i) {
                    const float xl = fmaxf(fmaf(x[i], kLog2e, -ml), -200.f);
                    const float e = __builtin_amdgcn_exp2f(xl);
                    s2 += e;
                    w2 = fmaf(e, xl, w2);
                }
                part_h.s = s2;
                part_h.w = w2 * 0.6931471805599453f;
            }
            mine = merge(mine, part_h);
        }
#pragma unroll
        for (int off = 1; off < P; off <<= 1) {
            Triple o;
            o.m = __shfl_xor(mine.m, off);
            o.s = __shfl_xor(mine.s, off);
            o.w = __shfl_xor(mine.w, off);
            mine = (p & off) ? merge(o, mine) : merge(mine, o);
        }
        if (t < T && p == 0) part[t * nvt + vt] = make_float4(mine.m, mine.s, mine.w, 0.f);
        if (t < T && y32 >= 0 && ((y32 >> 2) & (P - 1)) == p) z_y[t] = sm.c[r][y32];
    }
}

// dlogits = s g_t (onehot(y_t) - exp(s z - lse_t)) (s = scale, the inverse
// temperature; lse_t that of s z) for rows [0, M) of the block
// (h and out already offset to the block's first row) and the V vocabulary
// entries vbase .. vbase + V - 1 (w already offset to entry vbase), written in
// bf16 (nearest even) to out [M, ld_out]: the gradient pass of the logits
// path with the logits formed on the fly. The target element is
// s g_t * -expm1(logp_t), accurate when p_y -> 1. The fp32 tile is staged
// through LDS so that each row leaves as 16-byte vectors.
template <class C>
__global__ void __launch_bounds__(C::THREADS)
lmhead_dlogits_kernel(const uint16_t* __restrict__ h, int64_t M, int64_t ldh,
                      const uint16_t* __restrict__ w, int64_t V, int64_t ldw, int64_t d,
                      const int32_t* __restrict__ target, const float* __restrict__ lse,
                      const float* __restrict__ logp, const float* __restrict__ coef,
                      float scale, uint16_t* __restrict__ out, int64_t ld_out, int64_t vbase,
                      int64_t nmt, int64_t nvt) {
    __shared__ typename C::Smem sm;
    int64_t mt, vt;
    tile_of_block(nmt, nvt, mt, vt);
    const int64_t m0 = mt * C::BM, n0 = vt * C::BN;
    f32x16 acc[C::TM][C::TN];
    gemm_tile<C>(h, M, ldh, w, V, ldw, d, m0, n0, sm, acc);

    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int wr = (wave / C::WN) * 32, wc = (wave % C::WN) * (C::BN / C::WN);
    constexpr int CHUNKS = C::BN / 8;  // 16-byte output chunks per tile row
#pragma unroll
    for (int e0 = 0; e0 < C::BM; e0 += C::EPI) {
        if (e0) __syncthreads();
#pragma unroll
        for (int i = 0; i < C::TM; ++i)
#pragma unroll
            for (int j = 0; j < C::TN; ++j)
#pragma unroll
                for (int v = 0; v < 16; ++v) {
                    const int row = wr + i * C::RS + (v >> 2) * 8 + (lane >> 5) * 4 + (v & 3) - e0;
                    if (row >= 0 && row < C::EPI)
                        sm.c[row][wc + j * 32 + (lane & 31)] = acc[i][j][v] * scale;
                }
        // per-row constants: -g, -lse log2(e), the target's gradient
        // g (-expm1(logp)) (accurate when p_y -> 1), the target's column here;
        // g carries the inverse temperature (the chain rule through scale z)
        if (tid < C::EPI) {
            const int64_t t = m0 + e0 + tid;
            float4 rp = make_float4(0.f, 0.f, 0.f, __int_as_float(-1));
            if (t < M) {
                const float g = coef[t] * scale;
                const int64_t yrel = (int64_t)target[t] - vbase - n0;
                rp = make_float4(-g, -lse[t] * 1.4426950408889634f, g * -expm1f(logp[t]),
                                 __int_as_float(yrel >= 0 && yrel < C::BN ? (int)yrel : -1));
            }
            sm.rowp[tid] = rp;
        }
        __syncthreads();
        for (int e = tid; e < C::EPI * CHUNKS; e += C::THREADS) {
            const int r = e / CHUNKS, ch = e % CHUNKS;
            const int64_t t = m0 + e0 + r;
            const int64_t col0 = n0 + ch * 8;
            if (t >= M || col0 >= V) continue;
            const float4 rp = sm.rowp[r];
            const int yc = __float_as_int(rp.w) - ch * 8;  // the target's index in this chunk
            // the chunk's two 16-byte halves, read in an order that alternates
            // every 8 chunks so that the 16 lanes of one LDS read cycle hit 16
            // distinct bank quads
            const int sw = (ch >> 3) & 1;
            const float4 a = *reinterpret_cast<const float4*>(&sm.c[r][ch * 8 + 4 * sw]);
            const float4 b = *reinterpret_cast<const float4*>(&sm.c[r][ch * 8 + 4 - 4 * sw]);
            const float4 lo = sw ? b : a, hi = sw ? a : b;
            const float xs[8] = {lo.x, lo.y, lo.z, lo.w, hi.x, hi.y, hi.z, hi.w};
            float dz[8];
#pragma unroll
            for (int q = 0; q < 8; ++q) {
                const float e2 = __builtin_amdgcn_exp2f(fmaf(xs[q], 1.4426950408889634f, rp.y));
                dz[q] = q == yc ? rp.z : rp.x * e2;
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

// Rows whose coefficient is not 0, in increasing order: map[0 .. n) and
// count[0] = n. One workgroup walks the rows 1024 at a time; the position of
// each kept row is its wave's ballot prefix plus the earlier waves' counts.
constexpr int kCompactThreads = 1024;
__global__ void __launch_bounds__(kCompactThreads)
compact_rows_kernel(const float* __restrict__ coef, int64_t T, int32_t* __restrict__ map,
                    int32_t* __restrict__ count) {
    __shared__ int wave_n[kCompactThreads / 64];
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    int64_t base = 0;
    for (int64_t t0 = 0; t0 < T; t0 += kCompactThreads) {
        const int64_t t = t0 + tid;
        const bool keep = t < T && coef[t] != 0.f;
        const uint64_t ballot = __ballot(keep);
        const int before = __popcll(ballot & ((uint64_t(1) << lane) - 1));
        if (lane == 0) wave_n[wave] = __popcll(ballot);
        __syncthreads();
        int off = 0, total = 0;
        for (int w = 0; w < kCompactThreads / 64; ++w) {
            off += w < wave ? wave_n[w] : 0;
            total += wave_n[w];
        }
        if (keep) map[base + off + before] = (int32_t)t;
        base += total;
        __syncthreads();
    }
    if (tid == 0) count[0] = (int32_t)base;
}

// Row i < count of the compact problem: hidden row map[i] and its per-row
// values, one workgroup per row (grid-stride over the rows).
__global__ void __launch_bounds__(64)
gather_rows_kernel(const int32_t* __restrict__ map, const int32_t* __restrict__ count,
                   const uint16_t* __restrict__ h, int64_t ld_h, int64_t d,
                   const int32_t* __restrict__ target, const float* __restrict__ lse,
                   const float* __restrict__ logp, const float* __restrict__ coef,
                   uint16_t* __restrict__ h_c, int32_t* __restrict__ target_c,
                   float* __restrict__ lse_c, float* __restrict__ logp_c, float* __restrict__ coef_c) {
    const int64_t n = count[0];
    for (int64_t i = blockIdx.x; i < n; i += gridDim.x) {
        const int64_t t = map[i];
        const u32x4* src = reinterpret_cast<const u32x4*>(h + t * ld_h);
        u32x4* dst = reinterpret_cast<u32x4*>(h_c + i * d);
        for (int64_t j = threadIdx.x; j < d / 8; j += 64) dst[j] = src[j];
        if (threadIdx.x == 0) {
            target_c[i] = target[t];
            lse_c[i] = lse[t];
            logp_c[i] = logp[t];
            coef_c[i] = coef[t];
        }
    }
}

// An element of a gradient output: fp32, or bf16 bits rounded to nearest even.
__device__ __forceinline__ void put(float* p, float v) { *p = v; }
__device__ __forceinline__ void put(uint16_t* p, float v) { *p = bf16_bits(v); }

// Rows [0, rows) of a row-major matrix set to 0 (columns [0, cols)).
template <class O>
__global__ void __launch_bounds__(256)
zero_rows_kernel(O* __restrict__ m, int64_t rows, int64_t cols, int64_t ld) {
    for (int64_t r = blockIdx.x; r < rows; r += gridDim.x)
        for (int64_t c = threadIdx.x; c < cols; c += 256) put(m + r * ld + c, 0.f);
}

// dh[map[i]] = dh_c[i] for i < count (grid-stride over the rows).
template <class O>
__global__ void __launch_bounds__(256)
scatter_rows_kernel(const int32_t* __restrict__ map, const int32_t* __restrict__ count,
                    const float* __restrict__ dh_c, int64_t d, O* __restrict__ dh, int64_t ld_dh) {
    const int64_t n = count[0];
    for (int64_t i = blockIdx.x; i < n; i += gridDim.x) {
        const int64_t t = map[i];
        for (int64_t c = threadIdx.x; c < d; c += 256) put(dh + t * ld_dh + c, dh_c[i * d + c]);
    }
}

// dst[r, c] = bf16(src[r, c]) for rows [0, rows), columns [0, cols).
__global__ void __launch_bounds__(256)
to_bf16_kernel(const float* __restrict__ src, int64_t ld_src, int64_t rows, int64_t cols,
               uint16_t* __restrict__ dst, int64_t ld_dst) {
    for (int64_t r = blockIdx.x; r < rows; r += gridDim.x)
        for (int64_t c = threadIdx.x; c < cols; c += 256)
            dst[r * ld_dst + c] = bf16_bits(src[r * ld_src + c]);
}

// Workgroups of the row kernels above: one per row up to this many.
constexpr int64_t kRowBlocks = 65536;

// The MFMA tile addresses its rows by 32-bit byte offsets from the tile's first
// row: (BM - 1) rows of ld elements must stay below 2^31 bytes.
constexpr int64_t kMaxLd = int64_t(1) << 22;

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
                             const float* coef, float scale, uint16_t* out, int64_t ld_out,
                             int64_t vbase, hipStream_t stream) {
    const int64_t nmt = (rows + LmCfg::BM - 1) / LmCfg::BM, nvt = vocab_tiles(V);
    if (!grid_fits(nmt * nvt, LmCfg::THREADS) || ld_h > kMaxLd || ld_w > kMaxLd)
        return DART_ERR_UNSUPPORTED;
    hipLaunchKernelGGL(lmhead_dlogits_kernel<LmCfg>, dim3((unsigned)(nmt * nvt)),
                       dim3(LmCfg::THREADS), 0, stream, hidden, rows, ld_h, weight, V, ld_w, d,
                       target, lse, logp, coef, scale, out, ld_out, vbase, nmt, nvt);
    return hipGetLastError() == hipSuccess ? DART_OK : DART_ERR_HIP;
}

// One rocBLAS handle per device and stream, created on the first call on that
// stream and kept until the process ends. A handle owns a device workspace that
// some of the library's kernels use, so two streams never share one: their
// GEMMs may run at the same time. Calls are serialised by the mutex (the
// lookup, and the enqueueing on one handle).
std::mutex g_blas_mu;
struct BlasEntry {
    int dev;
    hipStream_t stream;
    rocblas_handle handle;
};
std::vector<BlasEntry> g_blas;

// The handle of (dev, stream), bound to that stream; dev must be current (a
// handle belongs to the device current when it is created). The caller holds
// g_blas_mu.
rocblas_handle blas_handle(int dev, hipStream_t stream) {
    for (const BlasEntry& e : g_blas)
        if (e.dev == dev && e.stream == stream)
            // the stream may be a new one at the address of a destroyed one
            return rocblas_set_stream(e.handle, stream) == rocblas_status_success ? e.handle
                                                                                 : nullptr;
    rocblas_handle h = nullptr;
    if (rocblas_create_handle(&h) != rocblas_status_success) return nullptr;
    if (rocblas_set_stream(h, stream) != rocblas_status_success) {
        (void)rocblas_destroy_handle(h);
        return nullptr;
    }
    g_blas.push_back({dev, stream, h});
    return h;
}

}  // namespace

extern "C" {

size_t dart_lmhead_stats_workspace_bytes(int64_t T, int64_t V) {
    if (T < 1 || V < 1 || T > 0x7FFFFFFFll || V > 0x7FFFFFFFll) return 0;
    return (size_t)T * (size_t)vocab_tiles(V) * sizeof(float4) + (size_t)T * sizeof(float);
}

dart_status_t dart_lmhead_tok_stats_ex(const void* hidden, int64_t T, int64_t d, int64_t ld_h,
                                       const void* weight, int64_t V, int64_t ld_w,
                                       const int32_t* target, float inv_temp, float* logp,
                                       float* entropy, float* lse, void* workspace,
                                       size_t workspace_bytes, hipStream_t stream) {
    if (bad_lmhead_args(hidden, T, d, ld_h, weight, V, ld_w)) return DART_ERR_INVALID_ARG;
    if (!(inv_temp > 0.f) || isinf(inv_temp)) return DART_ERR_INVALID_ARG;
    if (!target || !logp || !entropy || !lse || !workspace ||
        reinterpret_cast<uintptr_t>(workspace) % 16)
        return DART_ERR_INVALID_ARG;
    if (const dart_status_t ck = dart_check::run(
            stream, {{dart_check::Item::Ids, target, T, V}}); ck != DART_OK)
        return ck;

    if (workspace_bytes < dart_lmhead_stats_workspace_bytes(T, V)) return DART_ERR_INVALID_ARG;
    const int64_t nmt = (T + LmCfg::BM - 1) / LmCfg::BM, nvt = vocab_tiles(V);
    if (!grid_fits(nmt * nvt, LmCfg::THREADS) ||
        !grid_fits((T + kMergeWaves - 1) / kMergeWaves, kMergeWaves * 64) || ld_h > kMaxLd ||
        ld_w > kMaxLd)
        return DART_ERR_UNSUPPORTED;
    float4* part = static_cast<float4*>(workspace);
    float* z_y = reinterpret_cast<float*>(part + T * nvt);
    hipLaunchKernelGGL(lmhead_stats_kernel<LmCfg>, dim3((unsigned)(nmt * nvt)), dim3(LmCfg::THREADS),
                       0, stream,
                       static_cast<const uint16_t*>(hidden), T, ld_h,
                       static_cast<const uint16_t*>(weight), V, ld_w, d, target, inv_temp, nmt,
                       nvt, part, z_y);
    hipLaunchKernelGGL(lmhead_merge_kernel, dim3((unsigned)((T + kMergeWaves - 1) / kMergeWaves)),
                       dim3(kMergeWaves * 64), 0, stream, part, z_y, T, nvt, V, target, logp,
                       entropy, lse);
    return hipGetLastError() == hipSuccess ? DART_OK : DART_ERR_HIP;
}

dart_status_t dart_lmhead_tok_stats(const void* hidden, int64_t T, int64_t d, int64_t ld_h,
                                    const void* weight, int64_t V, int64_t ld_w,
                                    const int32_t* target, float* logp, float* entropy,
                                    float* lse, void* workspace, size_t workspace_bytes,
                                    hipStream_t stream) {
    return dart_lmhead_tok_stats_ex(hidden, T, d, ld_h, weight, V, ld_w, target, 1.f, logp,
                                    entropy, lse, workspace, workspace_bytes, stream);
}

dart_status_t dart_lmhead_dlogits_ex(const void* hidden, int64_t T, int64_t d, int64_t ld_h,
                                     const void* weight, int64_t V, int64_t ld_w,
                                     const int32_t* target, const float* lse, const float* logp,
                                     const float* tok_coef, float inv_temp, void* dlogits,
                                     int64_t ld_out, hipStream_t stream) {
    if (bad_lmhead_args(hidden, T, d, ld_h, weight, V, ld_w)) return DART_ERR_INVALID_ARG;
    if (!(inv_temp > 0.f) || isinf(inv_temp)) return DART_ERR_INVALID_ARG;
    if (!target || !lse || !logp || !tok_coef || !dlogits || ld_out < V || ld_out % 8 ||
        reinterpret_cast<uintptr_t>(dlogits) % 16)
        return DART_ERR_INVALID_ARG;
    if (const dart_status_t ck = dart_check::run(
            stream, {{dart_check::Item::Ids, target, T, V}}); ck != DART_OK)
        return ck;

    return launch_dlogits(static_cast<const uint16_t*>(hidden), T, d, ld_h,
                          static_cast<const uint16_t*>(weight), V, ld_w, target, lse, logp,
                          tok_coef, inv_temp, static_cast<uint16_t*>(dlogits), ld_out, 0, stream);
}

dart_status_t dart_lmhead_dlogits(const void* hidden, int64_t T, int64_t d, int64_t ld_h,
                                  const void* weight, int64_t V, int64_t ld_w,
                                  const int32_t* target, const float* lse, const float* logp,
                                  const float* tok_coef, void* dlogits, int64_t ld_out,
                                  hipStream_t stream) {
    return dart_lmhead_dlogits_ex(hidden, T, d, ld_h, weight, V, ld_w, target, lse, logp, tok_coef,
                                  1.f, dlogits, ld_out, stream);
}

size_t dart_lmhead_backward_workspace_bytes(int64_t chunk_rows, int64_t V) {
    if (chunk_rows < 1 || V < 1 || chunk_rows > 0x7FFFFFFFll || V > 0x7FFFFFFFll) return 0;
    return (size_t)chunk_rows * (size_t)((V + 7) / 8 * 8) * 2;
}

}  // extern "C"

namespace {

constexpr uint32_t kBackwardFlags = DART_LMHEAD_SKIP_ZERO_ROWS | DART_LMHEAD_BF16_GRADS;

int64_t ceil8(int64_t x) { return (x + 7) / 8 * 8; }
size_t align256(size_t x) { return (x + 255) / 256 * 256; }

// How a backward call runs and where its parts sit in the workspace (byte
// offsets, each part 256-byte aligned; total is the end of the last part).
struct BackwardPlan {
    bool bf16, skip;
    int64_t rows, cols;  // block of rows x vocabulary entries, at most T x V
    bool acc_w;          // dW summed over row blocks into bf16: through fp32
    bool acc_h;          // dh summed over vocabulary blocks into bf16: through fp32
    size_t dz, accw, acch, h_c, dh_c, target_c, lse_c, logp_c, coef_c, map, count, total;
};

// total = 0 when the sizes do not fit the address arithmetic.
BackwardPlan plan_backward(int64_t T, int64_t d, int64_t V, int64_t chunk_rows,
                           int64_t chunk_cols, uint32_t flags) {
    BackwardPlan P = {};
    P.bf16 = flags & DART_LMHEAD_BF16_GRADS;
    P.skip = flags & DART_LMHEAD_SKIP_ZERO_ROWS;
    P.rows = chunk_rows < T ? chunk_rows : T;
    P.cols = chunk_cols < V ? chunk_cols : V;
    // with rows skipped, dh is summed in the compact fp32 rows
    P.acc_w = P.bf16 && P.rows < T;
    P.acc_h = P.bf16 && P.cols < V && !P.skip;
    const double big = double(int64_t(1) << 60);
    if ((double)P.rows * (double)ceil8(P.cols) * 2 > big || (double)V * (double)d * 4 > big ||
        (double)T * (double)d * 6 > big)
        return P;
    size_t end = 0;
    auto take = [&](size_t bytes) {
        const size_t at = align256(end);
        end = at + bytes;
        return at;
    };
    P.dz = take((size_t)P.rows * (size_t)ceil8(P.cols) * 2);
    if (P.acc_w) P.accw = take((size_t)V * (size_t)d * 4);
    if (P.acc_h) P.acch = take((size_t)T * (size_t)d * 4);
    if (P.skip) {
        P.h_c = take((size_t)T * (size_t)d * 2);
        P.dh_c = take((size_t)T * (size_t)d * 4);
        P.target_c = take((size_t)T * 4);
        P.lse_c = take((size_t)T * 4);
        P.logp_c = take((size_t)T * 4);
        P.coef_c = take((size_t)T * 4);
        P.map = take((size_t)T * 4);
        P.count = take(4);
    }
    P.total = end;
    return P;
}

// A gradient output: row-major, fp32 or bf16.
struct Grad {
    void* p;
    int64_t ld;
    bool bf16;
    void* row(int64_t r) const {
        return static_cast<char*>(p) + r * ld * (bf16 ? 2 : 4);
    }
};

// rocBLAS is column-major: a row-major [R, C] matrix with row stride ld is
// its column-major [C, R] transpose with leading dimension ld. Both products
// take bf16 inputs and accumulate in fp32; accumulate adds to the output.
// dh[rows, d] (+)= dz[rows, K] W[K, d]   <=>   dh^T = W^T dz^T
bool gemm_dh(rocblas_handle blas, const uint16_t* dz, int64_t ld_dz, int64_t rows, int64_t K,
             const uint16_t* w, int64_t ld_w, int64_t d, bool accumulate, const Grad& out) {
    const float one = 1.f, zero = 0.f;
    const rocblas_datatype ot = out.bf16 ? rocblas_datatype_bf16_r : rocblas_datatype_f32_r;
    return rocblas_gemm_ex(blas, rocblas_operation_none, rocblas_operation_none, (rocblas_int)d,
                           (rocblas_int)rows, (rocblas_int)K, &one, w, rocblas_datatype_bf16_r,
                           (rocblas_int)ld_w, dz, rocblas_datatype_bf16_r, (rocblas_int)ld_dz,
                           accumulate ? &one : &zero, out.p, ot, (rocblas_int)out.ld, out.p, ot,
                           (rocblas_int)out.ld, rocblas_datatype_f32_r, rocblas_gemm_algo_standard,
                           0, 0) == rocblas_status_success;
}

// dW[cols, d] (+)= dz[K, cols]^T h[K, d]   <=>   dW^T = h^T dz
bool gemm_dw(rocblas_handle blas, const uint16_t* h, int64_t ld_h, int64_t K, const uint16_t* dz,
             int64_t ld_dz, int64_t cols, int64_t d, bool accumulate, const Grad& out) {
    const float one = 1.f, zero = 0.f;
    const rocblas_datatype ot = out.bf16 ? rocblas_datatype_bf16_r : rocblas_datatype_f32_r;
    return rocblas_gemm_ex(blas, rocblas_operation_none, rocblas_operation_transpose,
                           (rocblas_int)d, (rocblas_int)cols, (rocblas_int)K, &one, h,
                           rocblas_datatype_bf16_r, (rocblas_int)ld_h, dz, rocblas_datatype_bf16_r,
                           (rocblas_int)ld_dz, accumulate ? &one : &zero, out.p, ot,
                           (rocblas_int)out.ld, out.p, ot, (rocblas_int)out.ld,
                           rocblas_datatype_f32_r, rocblas_gemm_algo_standard, 0,
                           0) == rocblas_status_success;
}

void launch_to_bf16(const float* src, int64_t rows, int64_t cols, const Grad& dst,
                    hipStream_t stream) {
    const unsigned blocks = (unsigned)(rows < kRowBlocks ? rows : kRowBlocks);
    hipLaunchKernelGGL(to_bf16_kernel, dim3(blocks), dim3(256), 0, stream, src, cols, rows, cols,
                       static_cast<uint16_t*>(dst.p), dst.ld);
}

// The gradient pass over rows [0, T) of h in blocks of rows x vocabulary
// entries: per block, its dlogits into dz (bf16), then the block's share of
// dh (summed over the vocabulary blocks of its rows) and of dW (summed over
// the row blocks of its entries). A sum goes into its fp32 output directly,
// or, for a bf16 output that more than one block adds to, into acc_h ([T, d])
// or acc_w ([V, d]) and is rounded to bf16 once at the end; an output that
// one block writes is that GEMM's fp32 result rounded once.
dart_status_t backward_core(rocblas_handle blas, const uint16_t* h, int64_t T, int64_t d,
                            int64_t ld_h, const uint16_t* w, int64_t V, int64_t ld_w,
                            const int32_t* target, const float* lse, const float* logp,
                            const float* coef, float scale, const Grad& dh, const Grad& dw,
                            int64_t R,
                            int64_t C, uint16_t* dz, float* acc_h, float* acc_w,
                            hipStream_t stream) {
    if (R > T) R = T;
    if (C > V) C = V;
    const int64_t ld_dz = ceil8(C);
    const bool via_h = dh.bf16 && C < V, via_w = dw.bf16 && R < T;
    const Grad sum_h = via_h ? Grad{acc_h, d, false} : dh;
    const Grad sum_w = via_w ? Grad{acc_w, d, false} : dw;
    for (int64_t r0 = 0; r0 < T; r0 += R) {
        const int64_t rows = T - r0 < R ? T - r0 : R;
        const uint16_t* hr = h + r0 * ld_h;
        for (int64_t c0 = 0; c0 < V; c0 += C) {
            const int64_t cols = V - c0 < C ? V - c0 : C;
            const uint16_t* wc = w + c0 * ld_w;
            const dart_status_t st =
                launch_dlogits(hr, rows, d, ld_h, wc, cols, ld_w, target + r0, lse + r0,
                               logp + r0, coef + r0, scale, dz, ld_dz, c0, stream);
            if (st != DART_OK) return st;
            if (!gemm_dh(blas, dz, ld_dz, rows, cols, wc, ld_w, d, c0 > 0,
                         Grad{sum_h.row(r0), sum_h.ld, sum_h.bf16}) ||
                !gemm_dw(blas, hr, ld_h, rows, dz, ld_dz, cols, d, r0 > 0,
                         Grad{sum_w.row(c0), sum_w.ld, sum_w.bf16}))
                return DART_ERR_HIP;
        }
    }
    if (via_h) launch_to_bf16(acc_h, T, d, dh, stream);
    if (via_w) launch_to_bf16(acc_w, V, d, dw, stream);
    return hipGetLastError() == hipSuccess ? DART_OK : DART_ERR_HIP;
}

template <class O>
void launch_zero_rows(void* m, int64_t rows, int64_t cols, int64_t ld, hipStream_t stream) {
    const unsigned blocks = (unsigned)(rows < kRowBlocks ? rows : kRowBlocks);
    hipLaunchKernelGGL(zero_rows_kernel<O>, dim3(blocks), dim3(256), 0, stream,
                       static_cast<O*>(m), rows, cols, ld);
}

}  // namespace

extern "C" {

size_t dart_lmhead_backward_ex_workspace_bytes(int64_t T, int64_t d, int64_t V,
                                               int64_t chunk_rows, int64_t chunk_cols,
                                               uint32_t flags) {
    if (T < 1 || d < 1 || V < 1 || chunk_rows < 1 || chunk_cols < 1 || T > 0x7FFFFFFFll ||
        d > 0x7FFFFFFFll || V > 0x7FFFFFFFll || (flags & ~kBackwardFlags))
        return 0;
    return plan_backward(T, d, V, chunk_rows, chunk_cols, flags).total;
}

dart_status_t dart_lmhead_backward_ex(const void* hidden, int64_t T, int64_t d, int64_t ld_h,
                                      const void* weight, int64_t V, int64_t ld_w,
                                      const int32_t* target, const float* lse, const float* logp,
                                      const float* tok_coef, float inv_temp, void* dhidden,
                                      int64_t ld_dh, void* dweight, int64_t ld_dw,
                                      int64_t chunk_rows, int64_t chunk_cols, uint32_t flags,
                                      void* workspace, size_t workspace_bytes,
                                      hipStream_t stream) {
    if (bad_lmhead_args(hidden, T, d, ld_h, weight, V, ld_w)) return DART_ERR_INVALID_ARG;
    if (!(inv_temp > 0.f) || isinf(inv_temp)) return DART_ERR_INVALID_ARG;
    if (!target || !lse || !logp || !tok_coef || !dhidden || !dweight || !workspace)
        return DART_ERR_INVALID_ARG;
    if (ld_dh < d || ld_dw < d || chunk_rows < 1 || chunk_cols < 1 ||
        (flags & ~kBackwardFlags) || reinterpret_cast<uintptr_t>(workspace) % 16)
        return DART_ERR_INVALID_ARG;
    // the BLAS library takes 32-bit sizes and leading dimensions
    const int64_t kI32 = 0x7FFFFFFFll;
    if (ld_h > kI32 || ld_w > kI32 || ld_dh > kI32 || ld_dw > kI32) return DART_ERR_UNSUPPORTED;
    const BackwardPlan P = plan_backward(T, d, V, chunk_rows, chunk_cols, flags);
    if (P.total == 0) return DART_ERR_UNSUPPORTED;
    if (workspace_bytes < P.total) return DART_ERR_INVALID_ARG;
    // skipping rows waits for the kept-row count: not possible under graph capture
    if (P.skip)
        if (const dart_status_t st = may_synchronize(stream); st != DART_OK) return st;
    if (const dart_status_t ck = dart_check::run(
            stream, {{dart_check::Item::Ids, target, T, V}}); ck != DART_OK)
        return ck;

    const int dev = stream_device(stream);
    if (dev < 0) return DART_ERR_HIP;
    // the stream's device is current while the BLAS library works
    DeviceGuard on_dev(dev);
    if (!on_dev.ok) return DART_ERR_HIP;
    std::lock_guard<std::mutex> lock(g_blas_mu);
    rocblas_handle blas = blas_handle(dev, stream);
    if (!blas) return DART_ERR_HIP;
    const uint16_t* h = static_cast<const uint16_t*>(hidden);
    const uint16_t* w = static_cast<const uint16_t*>(weight);
    char* ws = static_cast<char*>(workspace);
    uint16_t* dz = reinterpret_cast<uint16_t*>(ws + P.dz);
    float* acc_w = P.acc_w ? reinterpret_cast<float*>(ws + P.accw) : nullptr;
    float* acc_h = P.acc_h ? reinterpret_cast<float*>(ws + P.acch) : nullptr;
    const Grad dh{dhidden, ld_dh, P.bf16}, dw{dweight, ld_dw, P.bf16};
    if (!P.skip)
        return backward_core(blas, h, T, d, ld_h, w, V, ld_w, target, lse, logp, tok_coef,
                             inv_temp, dh, dw, P.rows, P.cols, dz, acc_h, acc_w, stream);

    // rows with a zero coefficient have dz = 0: they add nothing to dW and
    // their rows of dh are 0, so the GEMMs run over the other rows only
    int32_t* map = reinterpret_cast<int32_t*>(ws + P.map);
    int32_t* count = reinterpret_cast<int32_t*>(ws + P.count);
    uint16_t* h_c = reinterpret_cast<uint16_t*>(ws + P.h_c);
    float* dh_c = reinterpret_cast<float*>(ws + P.dh_c);
    int32_t* target_c = reinterpret_cast<int32_t*>(ws + P.target_c);
    float* lse_c = reinterpret_cast<float*>(ws + P.lse_c);
    float* logp_c = reinterpret_cast<float*>(ws + P.logp_c);
    float* coef_c = reinterpret_cast<float*>(ws + P.coef_c);
    hipLaunchKernelGGL(compact_rows_kernel, dim3(1), dim3(kCompactThreads), 0, stream, tok_coef,
                       T, map, count);
    const unsigned row_blocks = (unsigned)(T < kRowBlocks ? T : kRowBlocks);
    hipLaunchKernelGGL(gather_rows_kernel, dim3(row_blocks), dim3(64), 0, stream, map, count, h,
                       ld_h, d, target, lse, logp, tok_coef, h_c, target_c, lse_c, logp_c, coef_c);
    if (P.bf16)
        launch_zero_rows<uint16_t>(dhidden, T, d, ld_dh, stream);
    else
        launch_zero_rows<float>(dhidden, T, d, ld_dh, stream);
    if (hipGetLastError() != hipSuccess) return DART_ERR_HIP;
    // the GEMM sizes are host values: wait for the count
    int32_t n = 0;
    if (hipMemcpyAsync(&n, count, sizeof n, hipMemcpyDeviceToHost, stream) != hipSuccess ||
        hipStreamSynchronize(stream) != hipSuccess)
        return DART_ERR_HIP;
    if (n == 0) {
        if (P.bf16)
            launch_zero_rows<uint16_t>(dweight, V, d, ld_dw, stream);
        else
            launch_zero_rows<float>(dweight, V, d, ld_dw, stream);
        return hipGetLastError() == hipSuccess ? DART_OK : DART_ERR_HIP;
    }
    const dart_status_t st =
        backward_core(blas, h_c, n, d, d, w, V, ld_w, target_c, lse_c, logp_c, coef_c, inv_temp,
                      Grad{dh_c, d, false}, dw, P.rows, P.cols, dz, nullptr, acc_w, stream);
    if (st != DART_OK) return st;
    const unsigned nb = (unsigned)(n < kRowBlocks ? n : kRowBlocks);
    if (P.bf16)
        hipLaunchKernelGGL(scatter_rows_kernel<uint16_t>, dim3(nb), dim3(256), 0, stream, map,
                           count, dh_c, d, static_cast<uint16_t*>(dhidden), ld_dh);
    else
        hipLaunchKernelGGL(scatter_rows_kernel<float>, dim3(nb), dim3(256), 0, stream, map, count,
                           dh_c, d, static_cast<float*>(dhidden), ld_dh);
    return hipGetLastError() == hipSuccess ? DART_OK : DART_ERR_HIP;
}

dart_status_t dart_lmhead_backward(const void* hidden, int64_t T, int64_t d, int64_t ld_h,
                                   const void* weight, int64_t V, int64_t ld_w,
                                   const int32_t* target, const float* lse, const float* logp,
                                   const float* tok_coef, float* dhidden, int64_t ld_dh,
                                   float* dweight, int64_t ld_dw, int64_t chunk_rows,
                                   void* workspace, size_t workspace_bytes, hipStream_t stream) {
    return dart_lmhead_backward_ex(hidden, T, d, ld_h, weight, V, ld_w, target, lse, logp,
                                   tok_coef, 1.f, dhidden, ld_dh, dweight, ld_dw, chunk_rows, V,
                                   0u, workspace, workspace_bytes, stream);
}

}  // extern "C"
