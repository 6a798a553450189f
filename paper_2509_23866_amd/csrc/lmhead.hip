// libdart, LM-head part: the token statistics and the gradient of the
// policy-update hot path computed straight from the LM head's inputs, so that
// the [T, V] logits are never written to memory.
//
// Paper: DART, arXiv 2509.23866. The statistics are those of Sec. 4.3 (token
// entropy, the target's log-prob of Eq. 1) for logits z = h W^T, where h [T, d]
// are the final hidden states of the T action tokens and W [V, d] the LM-head
// weight of the policy (the 7B VLM of Sec. 5.1); the gradient is the chain
// rule of Eq. 2's loss through them. Both kernels apply an inverse sampling
// temperature s (1 in the paper, App. A.4) in their epilogues: the fp32 tile
// stays unscaled, and s enters the factor of the base-2 exponent (s log2 e)
// and the row maximum (s > 0), so that s = 1 changes no bit.
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
// adds dh = dz W and dW = dz^T h per block in one launch of
// lmhead_bwd_gemms_kernel (the same MFMA tile, its operands stored with K as
// their row index read through LDS transpose loads).
#include <hip/hip_runtime.h>
#include <math.h>
#include <stdint.h>

#include <type_traits>
#include <vector>

#include "internal.h"
#include "dart.h"

namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));

// Waits until at most N loads of this wave are outstanding (vmcnt), leaving
// the LDS and export counters alone.
template <int N>
__device__ __forceinline__ void wait_vmcnt() {
    static_assert(N >= 0 && N < 64, "vmcnt");
    __builtin_amdgcn_s_waitcnt((N & 0xF) | ((N >> 4) << 14) | (0x7 << 4) | (0xF << 8));
}

// A buffer resource over [base, base + bytes) (bytes capped at 2^32 - 1): raw
// loads past its end return zero. Dword 3 selects 32-bit data, untyped.
__device__ __forceinline__ __amdgpu_buffer_rsrc_t tile_rsrc(const void* base, int64_t bytes) {
    const uint32_t n = bytes > 0xFFFFFFFFll ? 0xFFFFFFFFu : (uint32_t)bytes;
    return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), (short)0, (int)n, 0x00020000);
}

__device__ __forceinline__ __attribute__((address_space(3))) void* lds_ptr(void* p) {
    return (__attribute__((address_space(3))) void*)p;
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

// float -> bf16 bits, round to nearest even, a NaN kept quiet with its
// payload: the __bf16 conversion, which is gfx950's v_cvt_pk_bf16_f32 (two
// values per instruction; the same bits as the integer rounding
// u + 0x7FFF + ((u >> 16) & 1) for every one of the 2^32 fp32 inputs, checked
// on the GPU)
typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
__device__ __forceinline__ uint16_t bf16_bits(float f) {
    return __builtin_bit_cast(uint16_t, (__bf16)f);
}

__device__ __forceinline__ uint32_t pack_bf16x2(float lo, float hi) {
    const bf16x2_t v = {(__bf16)lo, (__bf16)hi};
    return __builtin_bit_cast(uint32_t, v);
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
// or N read as zero (their results are not used); K past the end is zeroed in
// LDS. Layout of acc[i][j]: value v of lane l is
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
    // row. The loads are buffer loads into LDS: each operand's tile rows are a
    // buffer resource whose range ends at the matrix's last element, so rows
    // past M or N read as zero (their results are not used). A lane's byte
    // offset within its instruction's rows is the same for every instruction
    // and slice (the swizzle repeats every 16 rows, and the rows of one
    // instruction of every wave together are a multiple of that), so one VGPR
    // serves all of an operand's loads; the instruction's rows and the slice
    // enter as a scalar offset.
    constexpr int CH = C::CH, BK = C::BK;
    const int lrow = lane / CH, lslot = lane % CH;
    static_assert((C::WAVES * C::LROWS) % (16 / CH * CH) == 0, "swizzle period");
    const int r_lane = wave * C::LROWS + lrow;  // row of the lane in instruction 0
    const uint32_t voff_a = (uint32_t)((r_lane * lda + (lslot ^ swz<CH>(r_lane)) * 8) * 2);
    const uint32_t voff_b = (uint32_t)((r_lane * ldb + (lslot ^ swz<CH>(r_lane)) * 8) * 2);
    const uint32_t qstride_a = (uint32_t)(C::WAVES * C::LROWS * lda * 2);
    const uint32_t qstride_b = (uint32_t)(C::WAVES * C::LROWS * ldb * 2);
    const __amdgpu_buffer_rsrc_t rsrc_a = tile_rsrc(A + m0 * lda, (M - m0) * lda * 2);
    const __amdgpu_buffer_rsrc_t rsrc_b = tile_rsrc(B + n0 * ldb, (N - n0) * ldb * 2);
    // rows of instruction q of wave `wave + hh * HW`
    auto lds_a = [&](int buf, int q, int hh) {
        return &sm.in.a[buf][(q * C::WAVES + wave + hh * (C::WAVES / 2)) * C::LROWS][0];
    };
    auto lds_b = [&](int buf, int q, int hh) {
        return &sm.in.b[buf][(q * C::WAVES + wave + hh * (C::WAVES / 2)) * C::LROWS][0];
    };
    const int64_t nk = (K + BK - 1) / BK;
    // slice kt into buffer buf; a slice that ends past K reads chunks past K
    // (in the row padding, the next row or, at the end, as zero) that are
    // zeroed after landing
    // The first half of the waves (one per SIMD) issue every load of a
    // slice: their own rows and those of the wave HW above, with the same lane
    // offsets (the rows between them are a whole number of swizzle periods).
    // Issuing a slice's 64 loads holds each issuing wave for ~700 cycles; the
    // other wave of its SIMD multiplies meanwhile.
    constexpr int HW = C::WAVES / 2;
    static_assert((HW * C::LROWS) % 16 == 0, "swizzle period");
    const uint32_t hstride_a = (uint32_t)(HW * C::LROWS * lda * 2);
    const uint32_t hstride_b = (uint32_t)(HW * C::LROWS * ldb * 2);
    auto issue = [&](int64_t kt, int buf) {
        if (wave >= HW) return;
        const uint32_t kb = (uint32_t)(kt * BK * 2);
#pragma unroll
        for (int q = 0; q < C::IA; ++q)
#pragma unroll
            for (int hh = 0; hh < 2; ++hh)
                __builtin_amdgcn_raw_ptr_buffer_load_lds(rsrc_a, lds_ptr(lds_a(buf, q, hh)), 16,
                                                        voff_a, kb + q * qstride_a + hh * hstride_a,
                                                        0, 0);
#pragma unroll
        for (int q = 0; q < C::IB; ++q)
#pragma unroll
            for (int hh = 0; hh < 2; ++hh)
                __builtin_amdgcn_raw_ptr_buffer_load_lds(rsrc_b, lds_ptr(lds_b(buf, q, hh)), 16,
                                                        voff_b, kb + q * qstride_b + hh * hstride_b,
                                                        0, 0);
    };
    // a partial last slice: zero the chunks past K
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
    // The B offsets include the B buffers' start (64 KB into the LDS) and are
    // kept opaque to the compiler, so that the buffer and the 32-column block
    // enter as the read's 16-bit immediate (below 64 KB); folded into the
    // immediate, they did not fit, and every B read cost an address add.
    uint32_t rda[C::KSTEPS], rdb[C::KSTEPS];
    const char* const lds0 = reinterpret_cast<const char*>(&sm);
    const uint32_t b_at = (uint32_t)(reinterpret_cast<const char*>(&sm.in.b[0][0][0]) - lds0);
#pragma unroll
    for (int ks = 0; ks < C::KSTEPS; ++ks) {
        const int c = ks * 2 + (lane >> 5), ra = wr + (lane & 31), rb = wc + (lane & 31);
        rda[ks] = (uint32_t)(ra * BK + (c ^ swz<CH>(ra)) * 8) * 2;
        rdb[ks] = b_at + (uint32_t)(rb * BK + (c ^ swz<CH>(rb)) * 8) * 2;
        asm volatile("" : "+v"(rdb[ks]));
    }
    static_assert((C::NS - 1) * C::BN * BK * 2 + (C::TN - 1) * 32 * BK * 2 < 65536,
                  "B read immediates");
    bf16x8 af[2][C::TM], bfr[2][C::TN];
    auto read_step = [&](auto bufc, int ks, int set) {
        constexpr int buf = decltype(bufc)::value;
        const char* ba = reinterpret_cast<const char*>(&sm.in.a[buf][0][0]);
#pragma unroll
        for (int i = 0; i < C::TM; ++i)
            af[set][i] = __builtin_bit_cast(
                bf16x8, *reinterpret_cast<const u32x4*>(ba + rda[ks] + i * C::RS * BK * 2));
#pragma unroll
        for (int j = 0; j < C::TN; ++j)
            bfr[set][j] = __builtin_bit_cast(
                bf16x8, *reinterpret_cast<const u32x4*>(lds0 + rdb[ks] + buf * C::BN * BK * 2 +
                                                        j * 32 * BK * 2));
    };
    // the MFMAs of row blocks [i0, i1) of one k-step
    auto mfmas = [&](int set, int i0 = 0, int i1 = C::TM) {
#pragma unroll
        for (int i = 0; i < C::TM; ++i)
#pragma unroll
            for (int j = 0; j < C::TN; ++j)
                if (i >= i0 && i < i1)
                    acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(af[set][i], bfr[set][j],
                                                                        acc[i][j], 0, 0, 0);
    };
    // Every wave holds back the last k-step's MFMAs of its last row block
    // and issues them after the next slice's barrier (and its loads), while
    // the first operand reads of that slice are in flight.
    constexpr int LASTSET = (C::KSTEPS - 1) & 1;

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
        __builtin_amdgcn_s_setprio(1);
        if (kt > 0) mfmas(LASTSET, C::TM - 1, C::TM);
#pragma unroll
        for (int ks = 0; ks < C::KSTEPS; ++ks) {
            const int cs = ks & 1;
            if (ks < C::KSTEPS - 1) read_step(bufc, ks + 1, cs ^ 1);
            mfmas(cs, 0, ks == C::KSTEPS - 1 ? C::TM - 1 : C::TM);
            if (ks < C::KSTEPS - 1) {
                // interleave: one LDS read, then a share of the MFMAs
#pragma unroll
                for (int g = 0; g < C::TM + C::TN; ++g) {
                    __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
                    __builtin_amdgcn_sched_group_barrier(0x008, (C::TM * C::TN) / (C::TM + C::TN), 0);
                }
            }
        }
        __builtin_amdgcn_s_setprio(0);
    };
    // the loop body has no condition on the accumulators: an odd last slice
    // runs after it (a conditional second slice in the body made the compiler
    // copy every accumulator at the join)
    issue(0, 0);
    int64_t kt = 0;
    for (; kt + 1 < nk; kt += 2) {
        slice(std::integral_constant<int, 0>{}, kt);
        slice(std::integral_constant<int, 1>{}, kt + 1);
    }
    if (kt < nk) slice(std::integral_constant<int, 0>{}, kt);
    mfmas(LASTSET, C::TM - 1, C::TM);
    __syncthreads();
#else
    (void)A, (void)M, (void)lda, (void)B, (void)N, (void)ldb, (void)K, (void)m0, (void)n0;
    (void)sm, (void)acc;
#endif
}

// Logical tile of workgroup b: the hardware places workgroup b on XCD b % 8,
// so each XCD gets a contiguous run of logical tiles. Logical tiles come in
// groups of G token tiles x every vocabulary tile, token tile fastest within
// a group, so the ~32 tiles an XCD runs at once share G tiles of h and a few
// slices of W in its L2. (Token tile fastest over all of them made each XCD
// read a different h tile per workgroup: at T = 152569 that re-read the 1.09
// GB of h from HBM once per vocabulary slice, 15% slower than groups of 4.)
__device__ __forceinline__ void tile_of_block(int64_t nmt, int64_t nvt, int64_t& mt, int64_t& vt) {
    const int64_t nb = nmt * nvt, q = nb / 8, rr = nb % 8;
    const int64_t b = blockIdx.x, x = b % 8, sl = b / 8;
    const int64_t lg = x * q + min(x, rr) + sl;
    constexpr int64_t G = 4;  // token tiles per group
    const int64_t g = lg / (G * nvt), first = g * G;
    const int64_t gm = nmt - first < G ? nmt - first : G;
    const int64_t in = lg - first * nvt;
    mt = first + in % gm;
    vt = in / gm;
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
    static_assert(C::EPI == C::RS, "one row block of every wave per pass");
#pragma unroll
    for (int ip = 0; ip < C::TM; ++ip) {
        const int e0 = ip * C::EPI;
        // LDS-only barriers: the workgroup exchanges nothing but LDS here, and a
        // __syncthreads fence would also wait for the previous pass's stores
        if (ip) lds_ring_barrier();
        // rows [e0, e0 + EPI) of the tile to LDS: row block ip of every wave
#pragma unroll
        for (int j = 0; j < C::TN; ++j)
#pragma unroll
            for (int v = 0; v < 16; ++v)
                sm.c[wr + (v >> 2) * 8 + (lane >> 5) * 4 + (v & 3)][wc + j * 32 + (lane & 31)] =
                    acc[ip][j][v];
        lds_ring_barrier();
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
        // only the tile's last columns past V and a row's target column drop
        // out: the selects run only in threads that hold such a column
        const bool masked = vlim < C::BN || (y32 >= 0 && ((y32 >> 2) & (P - 1)) == p);
        // the tile stays unscaled in LDS: the inverse temperature enters the
        // base-2 exponent's factor (1 at scale 1: the same bits)
        const float c2 = scale * 1.4426950408889634f;
        Triple mine = {-INFINITY, 0.f, 0.f};
#pragma unroll
        for (int hh = 0; hh < 2; ++hh) {
            // the half's eight 16-byte reads, issued together; the empty asm
            // keeps the compiler from turning the selects below into
            // per-element predicated reads
            static_assert(NH / 4 == 8, "eight vectors per half row");
            f32x4 q[8];
#pragma unroll
            for (int c4 = 0; c4 < 8; ++c4)
                q[c4] = *reinterpret_cast<const f32x4*>(&sm.c[r][16 * (hh * 8 + c4) + 4 * p]);
            asm volatile("" : "+v"(q[0]), "+v"(q[1]), "+v"(q[2]), "+v"(q[3]), "+v"(q[4]),
                         "+v"(q[5]), "+v"(q[6]), "+v"(q[7]));
            float x[NH];
#pragma unroll
            for (int c4 = 0; c4 < 8; ++c4)
#pragma unroll
                for (int u = 0; u < 4; ++u) x[4 * c4 + u] = q[c4][u];
            if (masked) {
#pragma unroll
                for (int c4 = 0; c4 < 8; ++c4)
#pragma unroll
                    for (int u = 0; u < 4; ++u) {
                        const int col = 16 * (hh * 8 + c4) + 4 * p + u;
                        x[4 * c4 + u] = col < vlim && col != y32 ? x[4 * c4 + u] : -INFINITY;
                    }
            }
            float mx = -INFINITY;
#pragma unroll
            for (int i = 0; i < NH; ++i) mx = fmaxf(mx, x[i]);
            // scale > 0: the maximum of the scaled row is the scaled maximum
            Triple part_h = {mx * scale, 0.f, 0.f};
            if (mx > -INFINITY) {
                // e = 2^xl with xl = (x - mx) scale log2(e); where a column was
                // dropped (-inf) xl is floored at -200, where 2^xl is already 0
                // in fp32, so that it adds 0 (other columns are finite)
                const float ml = mx * c2;
                float s2 = 0.f, w2 = 0.f;
                if (masked) {
#pragma unroll
                    for (int i = 0; i < NH; ++i) {
                        const float xl = fmaxf(fmaf(x[i], c2, -ml), -200.f);
                        const float e = __builtin_amdgcn_exp2f(xl);
                        s2 += e;
                        w2 = fmaf(e, xl, w2);
                    }
                } else {
#pragma unroll
                    for (int i = 0; i < NH; ++i) {
                        const float xl = fmaf(x[i], c2, -ml);
                        const float e = __builtin_amdgcn_exp2f(xl);
                        s2 += e;
                        w2 = fmaf(e, xl, w2);
                    }
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
        if (t < T && y32 >= 0 && ((y32 >> 2) & (P - 1)) == p) z_y[t] = sm.c[r][y32] * scale;
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
                      int64_t nmt, int64_t nvt, const int32_t* __restrict__ dyn_rows,
                      int64_t dyn_base) {
    __shared__ typename C::Smem sm;
    // with dyn_rows, the block holds only rows below *dyn_rows - dyn_base (the
    // grid covers the most it can hold): the tiles are laid over the live rows'
    // tiles, so that they spread over every XCD, and the workgroups past them
    // (the last ones dispatched) have nothing to do
    if (dyn_rows) {
        const int64_t live = (int64_t)*dyn_rows - dyn_base;
        M = live < M ? (live > 0 ? live : 0) : M;
        nmt = (M + C::BM - 1) / C::BM;
        if ((int64_t)blockIdx.x >= nmt * nvt) return;
    }
    int64_t mt, vt;
    tile_of_block(nmt, nvt, mt, vt);
    const int64_t m0 = mt * C::BM, n0 = vt * C::BN;
    f32x16 acc[C::TM][C::TN];
    gemm_tile<C>(h, M, ldh, w, V, ldw, d, m0, n0, sm, acc);

    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int wr = (wave / C::WN) * 32, wc = (wave % C::WN) * (C::BN / C::WN);
    constexpr int CHUNKS = C::BN / 8;  // 16-byte output chunks per tile row
    static_assert(C::EPI == C::RS, "one row block of every wave per pass");
    // the tile stays unscaled in LDS: the inverse temperature enters the
    // base-2 exponent's factor (1 at scale 1: the same bits)
    const float c2 = scale * 1.4426950408889634f;
#pragma unroll
    for (int ip = 0; ip < C::TM; ++ip) {
        const int e0 = ip * C::EPI;
        // LDS-only barriers: a __syncthreads fence here would also wait for
        // the previous pass's gradient stores
        if (ip) lds_ring_barrier();
#pragma unroll
        for (int j = 0; j < C::TN; ++j)
#pragma unroll
            for (int v = 0; v < 16; ++v)
                sm.c[wr + (v >> 2) * 8 + (lane >> 5) * 4 + (v & 3)][wc + j * 32 + (lane & 31)] =
                    acc[ip][j][v];
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
        lds_ring_barrier();
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
            uint16_t* dst = out + t * ld_out + col0;
            if ((unsigned)yc >= 8u && col0 + 8 <= V) {
                // no target here (all but one chunk of a row): every element
                // takes the same formula, each half is rounded in the order
                // it was read, and only the four packed words follow the swap
                const float xa[4] = {a.x, a.y, a.z, a.w}, xb[4] = {b.x, b.y, b.z, b.w};
                float da[4], db[4];
#pragma unroll
                for (int q = 0; q < 4; ++q) {
                    da[q] = rp.x * __builtin_amdgcn_exp2f(fmaf(xa[q], c2, rp.y));
                    db[q] = rp.x * __builtin_amdgcn_exp2f(fmaf(xb[q], c2, rp.y));
                }
                const uint32_t a01 = pack_bf16x2(da[0], da[1]), a23 = pack_bf16x2(da[2], da[3]);
                const uint32_t b01 = pack_bf16x2(db[0], db[1]), b23 = pack_bf16x2(db[2], db[3]);
                u32x4 pk;
                pk.x = sw ? b01 : a01;
                pk.y = sw ? b23 : a23;
                pk.z = sw ? a01 : b01;
                pk.w = sw ? a23 : b23;
                __builtin_nontemporal_store(pk, reinterpret_cast<u32x4*>(dst));
                continue;
            }
            const float4 lo = sw ? b : a, hi = sw ? a : b;
            const float xs[8] = {lo.x, lo.y, lo.z, lo.w, hi.x, hi.y, hi.z, hi.w};
            float dz[8];
#pragma unroll
            for (int q = 0; q < 8; ++q) {
                const float e2 = __builtin_amdgcn_exp2f(fmaf(xs[q], c2, rp.y));
                dz[q] = q == yc ? rp.z : rp.x * e2;
            }
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

// ---------------------------------------------------------------------------
// Backward GEMMs on the matrix cores: C[M, N] (+)= A B with B stored [K][N]
// (N contiguous), for dh = dz W (A = the dz block read along its rows, K
// contiguous; B = the block's rows of W) and dW = dz^T h (A = the dz block
// read down its columns, M contiguous; B = the block's rows of h). The tile,
// waves, K slices and LDS ring are those of the forward tile; what differs is
// how an operand stored with K as its row index reaches the MFMA.
//
// Such an operand's slice sits in LDS as BK rows of 256 elements (its k rows
// as they are stored), chunk c (8 elements, 16 bytes) of row k in slot
// c ^ (4 (k mod 4)). The MFMA wants, in lane l, 8 consecutive k of one column;
// ds_read_b64_tr_b16 transposes 4 x 16 blocks within each 16 lanes: lane l
// receives element l % 4 of the 8 bytes that lane 16 (l / 16) + 4 j + (l % 16) / 4
// loaded, for j = 0..3 (whatever addresses the lanes gave). So lane L of a
// group points at row k0 + L / 4, columns 4 (L % 4) .. + 3 of its group's 16
// columns, and receives column L at rows k0 .. k0 + 3; two such reads give the
// 8 k of one MFMA operand. In one read, the 32 lanes of a half-wave take 4
// rows x 32 columns; the swizzle puts the 4 rows' chunks in 16 distinct bank
// quads (gfx950: 64 banks of 4 bytes), so the reads do not conflict.
// ---------------------------------------------------------------------------

typedef short s16x4 __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) s16x4* lds_s16x4_ptr;

// Elements of one transposed operand row in LDS (the tile width).
constexpr int kTw = 256;
static_assert(LmCfg::BM == kTw && LmCfg::BN == kTw, "transposed rows are one tile wide");

// Slot of chunk c of row k of a transposed operand tile.
__device__ __forceinline__ int tr_slot(int c, int k) { return c ^ (4 * (k & 3)); }

// acc = this wave's part of C[m0:m0+BM, n0:n0+BN] = A B over k in [0, K).
// A_KMAJ: A(m, k) = A[m lda + k], else A(m, k) = A[k lda + m]. B(k, n) =
// B[k ldb + n]. Rows and columns past M, N read zero or whatever lies there
// in the matrices (their results are not stored); k past K is zero in LDS
// (also inside a chunk that straddles K), so the stored row padding up to a
// multiple of 8 may hold anything. lda >= ceil8(K) (A_KMAJ) or ceil8(M),
// ldb >= ceil8(N); rows 16-byte aligned. Layout of acc as in gemm_tile. Ends
// on a barrier with no loads in flight.
template <class C, bool A_KMAJ>
__device__ __forceinline__ void gemm_tile_bwd(const uint16_t* __restrict__ A, int64_t lda,
                                              const uint16_t* __restrict__ B, int64_t ldb,
                                              int64_t M, int64_t N, int64_t K, int64_t m0,
                                              int64_t n0, typename C::Smem& sm,
                                              f32x16 (&acc)[C::TM][C::TN]) {
#if defined(__HIP_DEVICE_COMPILE__)
    static_assert(C::BK == 64 && C::BM == kTw && C::BN == kTw, "backward tile");
    const int tid = threadIdx.x, lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int wr = (wave / C::WN) * 32, wc = (wave % C::WN) * (C::BN / C::WN);
#pragma unroll
    for (int i = 0; i < C::TM; ++i)
#pragma unroll
        for (int j = 0; j < C::TN; ++j)
#pragma unroll
            for (int v = 0; v < 16; ++v) acc[i][j][v] = 0.f;

    constexpr int CH = C::CH, BK = C::BK;
    // transposed operands: one load instruction fills 2 rows of 32 chunks
    constexpr int TQ = BK / 2 / C::WAVES;  // load instructions per wave and slice
    static_assert(TQ * 2 * C::WAVES == BK, "transposed rows per wave");
    const int trow = lane >> 5, tslot = lane & 31;
    const int64_t nk = (K + BK - 1) / BK;

    // Buffer loads into LDS, as in gemm_tile: one per-lane offset VGPR per
    // operand, the instruction's rows and the slice as scalar offsets (or,
    // for a transposed operand, the slice in the resource base). A transposed
    // operand's resource ends at the last element of row K - 1 that exists
    // (columns < ceil8(len)), so k rows past K read as zero; chunks past len
    // within a row read the row padding or the next row (their results are
    // not stored).
    const int lrow = lane / CH, lslot = lane % CH;
    static_assert((C::WAVES * C::LROWS) % (16 / CH * CH) == 0, "swizzle period");
    static_assert(C::WAVES % 2 == 0, "transposed swizzle period");
    const int tr_k = wave * 2 + trow;  // transposed row of the lane in instruction 0
    const int tr_c = 8 * tr_slot(tslot, tr_k);
    uint32_t voff_a, qstride_a;
    if constexpr (A_KMAJ) {
        const int r_lane = wave * C::LROWS + lrow;
        voff_a = (uint32_t)((r_lane * lda + (lslot ^ swz<CH>(r_lane)) * 8) * 2);
        qstride_a = (uint32_t)(C::WAVES * C::LROWS * lda * 2);
    } else {
        voff_a = (uint32_t)((tr_k * lda + tr_c) * 2);
        qstride_a = (uint32_t)(C::WAVES * 2 * lda * 2);
    }
    const uint32_t voff_b = (uint32_t)((tr_k * ldb + tr_c) * 2);
    const uint32_t qstride_b = (uint32_t)(C::WAVES * 2 * ldb * 2);
    const __amdgpu_buffer_rsrc_t rsrc_ak = tile_rsrc(A + m0 * lda, (M - m0) * lda * 2);
    // resource of a transposed operand's slice kt: rows kt*BK .. K-1 from column t0
    auto tr_rsrc = [&](const uint16_t* X, int64_t ld, int64_t t0, int64_t len, int64_t kt) {
        const int64_t first = kt * BK * ld + t0;
        const int64_t end = (K - 1) * ld + (len + 7) / 8 * 8;
        return tile_rsrc(X + first, (end - first) * 2);
    };

    // instruction q of wave `wave + hh * HW`
    constexpr int HW = C::WAVES / 2;
    auto lds_a = [&](int buf, int q, int hh) {
        constexpr int per = A_KMAJ ? C::LROWS * BK : 2 * kTw;  // elements per instruction
        return &sm.in.a[buf][0][0] + (q * C::WAVES + wave + hh * HW) * per;
    };
    auto lds_b = [&](int buf, int q, int hh) {
        return &sm.in.b[buf][0][0] + (q * C::WAVES + wave + hh * HW) * 2 * kTw;
    };

    // As in gemm_tile, the first half of the waves issue every load, their
    // own rows and those of the wave HW above (HW * LROWS K-major rows or
    // 2 HW transposed rows further: whole swizzle periods, so the same lane
    // offsets)
    static_assert((HW * C::LROWS) % 16 == 0 && (2 * HW) % 4 == 0, "swizzle periods");
    const uint32_t hstride_ak = (uint32_t)(HW * C::LROWS * lda * 2);
    const uint32_t hstride_at = (uint32_t)(2 * HW * lda * 2);
    const uint32_t hstride_b = (uint32_t)(2 * HW * ldb * 2);
    auto issue = [&](int64_t kt, int buf) {
        if (wave >= HW) return;
        if constexpr (A_KMAJ) {
            const uint32_t kb = (uint32_t)(kt * BK * 2);
#pragma unroll
            for (int q = 0; q < C::IA; ++q)
#pragma unroll
                for (int hh = 0; hh < 2; ++hh)
                    __builtin_amdgcn_raw_ptr_buffer_load_lds(
                        rsrc_ak, lds_ptr(lds_a(buf, q, hh)), 16, voff_a,
                        kb + q * qstride_a + hh * hstride_ak, 0, 0);
        } else {
            const __amdgpu_buffer_rsrc_t ra = tr_rsrc(A, lda, m0, M, kt);
#pragma unroll
            for (int q = 0; q < TQ; ++q)
#pragma unroll
                for (int hh = 0; hh < 2; ++hh)
                    __builtin_amdgcn_raw_ptr_buffer_load_lds(ra, lds_ptr(lds_a(buf, q, hh)), 16,
                                                            voff_a, q * qstride_a + hh * hstride_at,
                                                            0, 0);
        }
        const __amdgpu_buffer_rsrc_t rb = tr_rsrc(B, ldb, n0, N, kt);
#pragma unroll
        for (int q = 0; q < TQ; ++q)
#pragma unroll
            for (int hh = 0; hh < 2; ++hh)
                __builtin_amdgcn_raw_ptr_buffer_load_lds(rb, lds_ptr(lds_b(buf, q, hh)), 16, voff_b,
                                                        q * qstride_b + hh * hstride_b, 0, 0);
    };
    // the partial last slice of a K-major A: k >= K set to 0, also inside the
    // chunk that straddles K (transposed operands read zero rows there)
    auto zero_tail = [&](int64_t kt, int buf) {
        const int kv = (int)(K - kt * BK);  // valid k in this slice, 1 .. BK-1
        uint16_t* a = &sm.in.a[buf][0][0];
        for (int e = tid; e < BK * kTw; e += C::THREADS) {
            // [BM][BK] rows with swizzled chunks: element e is row e / BK,
            // slot (e % BK) / 8, holding chunk slot ^ swz(row)
            const int r = e / BK, sl = (e % BK) / 8;
            const int kk = ((sl ^ swz<CH>(r)) * 8) + (e % 8);
            if (kk >= kv) a[e] = 0;
        }
    };

    // MFMA operand offsets. A (K-major): as gemm_tile. Transposed: lane l
    // points at row ks*16 + 8 (l / 32) + 4 h + (l / 4) % 4 and columns
    // mb + 16 ((l / 16) % 2) + 4 (l % 4) of its 32-column block mb (a multiple
    // of 32, so the chunk is (mb / 8) | ((l / 16) % 2) * 2 | (l % 4) / 2).
    const int kq = (lane >> 2) & 3;
    const int tr_lane_row = 8 * (lane >> 5) + kq;
    const int tr_delta = 2 * ((lane >> 4) & 1) + ((lane & 3) >> 1);
    auto tr_off = [&](int mb) -> uint32_t {
        const int slot = ((mb / 8) ^ (4 * kq)) | tr_delta;
        return (uint32_t)(tr_lane_row * kTw * 2 + slot * 16 + 8 * (lane & 1));
    };
    uint32_t rda[A_KMAJ ? C::KSTEPS : C::TM], rdb[C::TN];
    if constexpr (A_KMAJ) {
#pragma unroll
        for (int ks = 0; ks < C::KSTEPS; ++ks) {
            const int c = ks * 2 + (lane >> 5), ra = wr + (lane & 31);
            rda[ks] = (uint32_t)(ra * BK + (c ^ swz<CH>(ra)) * 8) * 2;
        }
    } else {
#pragma unroll
        for (int i = 0; i < C::TM; ++i) rda[i] = tr_off(wr + i * C::RS);
    }
    // B's offsets carry its buffers' start (64 KB into the LDS), opaque to the
    // compiler, so that the buffer, the k-step and the half enter as the
    // read's 16-bit immediate (as in gemm_tile)
    const char* const lds0 = reinterpret_cast<const char*>(&sm);
    const uint32_t b_at = (uint32_t)(reinterpret_cast<const char*>(&sm.in.b[0][0][0]) - lds0);
#pragma unroll
    for (int j = 0; j < C::TN; ++j) {
        rdb[j] = b_at + tr_off(wc + j * 32);
        asm volatile("" : "+v"(rdb[j]));
    }
    static_assert((C::NS - 1) * C::BN * BK * 2 + (C::KSTEPS - 1) * 16 * kTw * 2 + 4 * kTw * 2 <
                      65536,
                  "B read immediates");

    auto tr_pair = [&](const char* base, uint32_t off, int ks) -> bf16x8 {
        const int k0 = ks * 16 * kTw * 2;
        const s16x4 lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
            (lds_s16x4_ptr)(base + off + k0));
        const s16x4 hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
            (lds_s16x4_ptr)(base + off + k0 + 4 * kTw * 2));
        typedef short s16x8 __attribute__((ext_vector_type(8)));
        const s16x8 v = {lo[0], lo[1], lo[2], lo[3], hi[0], hi[1], hi[2], hi[3]};
        return __builtin_bit_cast(bf16x8, v);
    };
    bf16x8 af[2][C::TM], bfr[2][C::TN];
    auto read_step = [&](auto bufc, int ks, int set) {
        constexpr int buf = decltype(bufc)::value;
        const char* ba = reinterpret_cast<const char*>(&sm.in.a[buf][0][0]);
        const char* bb = lds0 + buf * C::BN * BK * 2;
#pragma unroll
        for (int i = 0; i < C::TM; ++i) {
            if constexpr (A_KMAJ)
                af[set][i] = __builtin_bit_cast(
                    bf16x8, *reinterpret_cast<const u32x4*>(ba + rda[ks] + i * C::RS * BK * 2));
            else
                af[set][i] = tr_pair(ba, rda[i], ks);
        }
#pragma unroll
        for (int j = 0; j < C::TN; ++j) bfr[set][j] = tr_pair(bb, rdb[j], ks);
    };
    auto mfmas = [&](int set) {
#pragma unroll
        for (int i = 0; i < C::TM; ++i)
#pragma unroll
            for (int j = 0; j < C::TN; ++j)
                acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(af[set][i], bfr[set][j],
                                                                    acc[i][j], 0, 0, 0);
    };
    auto slice = [&](auto bufc, int64_t kt) {
        constexpr int buf = decltype(bufc)::value;
        wait_vmcnt<0>();
        lds_ring_barrier();
        if (A_KMAJ && (K % BK) && kt == nk - 1) {
            zero_tail(kt, buf);
            lds_ring_barrier();
        }
        if (kt + 1 < nk) issue(kt + 1, buf ^ 1);
        read_step(bufc, 0, 0);
        __builtin_amdgcn_s_setprio(1);
        constexpr int NREAD = (A_KMAJ ? C::TM : 2 * C::TM) + 2 * C::TN;
#pragma unroll
        for (int ks = 0; ks < C::KSTEPS; ++ks) {
            const int cs = ks & 1;
            if (ks < C::KSTEPS - 1) read_step(bufc, ks + 1, cs ^ 1);
            mfmas(cs);
            if (ks < C::KSTEPS - 1) {
#pragma unroll
                for (int g = 0; g < C::TM * C::TN; ++g) {
                    __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
                    __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
                }
                __builtin_amdgcn_sched_group_barrier(0x100, NREAD - C::TM * C::TN, 0);
            }
        }
        __builtin_amdgcn_s_setprio(0);
    };
    if (nk > 0) issue(0, 0);
    int64_t kt = 0;
    for (; kt + 1 < nk; kt += 2) {
        slice(std::integral_constant<int, 0>{}, kt);
        slice(std::integral_constant<int, 1>{}, kt + 1);
    }
    if (kt < nk) slice(std::integral_constant<int, 0>{}, kt);
    __syncthreads();
#else
    (void)A, (void)lda, (void)B, (void)ldb, (void)M, (void)N, (void)K, (void)m0, (void)n0;
    (void)sm, (void)acc;
#endif
}

// One GEMM of the backward: C[M, N] (+)= A B with gemm_tile_bwd's operands,
// written to out [M, ldc] (fp32, or bf16 bits rounded to nearest even); vec:
// out 16-byte aligned and ldc a multiple of 16 bytes' worth of elements.
struct BwdGemm {
    const uint16_t* A;
    int64_t lda;
    const uint16_t* B;
    int64_t ldb;
    int64_t M, N, K;
    void* out;
    int64_t ldc;
    int vec;
    int64_t nmt, nnt;  // tiles
    // optional device row count: M (dyn_m) or K (dyn_k) is at most
    // *dyn - dyn_base (the grid covers the host values, the most there can be)
    const int32_t* dyn;
    int64_t dyn_base;
    bool dyn_m, dyn_k;
};

// Output modes of a backward GEMM: fp32 written, fp32 added to, bf16 written.
enum BwdOut { kOutF32 = 0, kOutF32Acc = 1, kOutBf16 = 2 };

// Logical tile of the workgroup with index b among the nb workgroups of one
// GEMM whose first workgroup sits on XCD 0 (workgroup i of a launch runs on
// XCD i % 8): each XCD takes a contiguous run of logical tiles, column tile
// fastest, so the tiles that share a row block of A run together on one XCD
// and read it from that XCD's L2.
__device__ __forceinline__ void tile_of_block_nfast(int64_t b, int64_t nmt, int64_t nnt,
                                                    int64_t& mt, int64_t& nt) {
    const int64_t nb = nmt * nnt, q = nb / 8, rr = nb % 8;
    const int64_t x = b % 8, sl = b / 8;
    const int64_t lg = x * q + min(x, rr) + sl;
    nt = lg % nnt;
    mt = lg / nnt;
}

// Tile b of GEMM g: the MFMA tile, then the fp32 result through LDS, 128 rows
// at a time, so that each row leaves as 16-byte vectors (vec), else one
// element at a time.
template <class C, bool A_KMAJ, int OUT>
__device__ __forceinline__ void bwd_gemm_tile(const BwdGemm& g, int64_t b, typename C::Smem& sm) {
    using OutT = typename std::conditional<OUT == kOutBf16, uint16_t, float>::type;
    constexpr bool ACC = OUT == kOutF32Acc;
    int64_t M = g.M, K = g.K, nmt = g.nmt;
    const int64_t N = g.N;
    if (g.dyn) {
        const int64_t live = (int64_t)*g.dyn - g.dyn_base;
        const int64_t lim = live > 0 ? live : 0;
        if (g.dyn_k && lim < K) K = lim;
        // no rows of this block to add: nothing to do
        if (K == 0 && ACC) return;
        if (g.dyn_m && lim < M) {
            // the tiles laid over the live rows' tiles (spread over every XCD)
            M = lim;
            nmt = (M + C::BM - 1) / C::BM;
            if (b >= nmt * g.nnt) return;
        }
    }
    int64_t mt, nt;
    tile_of_block_nfast(b, nmt, g.nnt, mt, nt);
    const int64_t m0 = mt * C::BM, n0 = nt * C::BN;
    f32x16 acc[C::TM][C::TN];
    gemm_tile_bwd<C, A_KMAJ>(g.A, g.lda, g.B, g.ldb, M, N, K, m0, n0, sm, acc);

    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int wr = (wave / C::WN) * 32, wc = (wave % C::WN) * (C::BN / C::WN);
    constexpr bool F32 = OUT != kOutBf16;
    constexpr int EPV = F32 ? 4 : 8;  // elements per 16-byte vector
    constexpr int VPR = C::BN / EPV;  // vectors per tile row
    OutT* out = static_cast<OutT*>(g.out);
    static_assert(C::EPI == C::RS, "one row block of every wave per pass");
#pragma unroll
    for (int ip = 0; ip < C::TM; ++ip) {
        const int e0 = ip * C::EPI;
        // LDS-only barriers: a __syncthreads fence here would also wait for
        // the previous pass's stores
        if (ip) lds_ring_barrier();
#pragma unroll
        for (int j = 0; j < C::TN; ++j)
#pragma unroll
            for (int v = 0; v < 16; ++v)
                sm.c[wr + (v >> 2) * 8 + (lane >> 5) * 4 + (v & 3)][wc + j * 32 + (lane & 31)] =
                    acc[ip][j][v];
        lds_ring_barrier();
        for (int e = tid; e < C::EPI * VPR; e += C::THREADS) {
            const int r = e / VPR, cv = e % VPR;
            const int64_t m = m0 + e0 + r, n = n0 + (int64_t)cv * EPV;
            if (m >= M || n >= N) continue;
            const float* src = &sm.c[r][cv * EPV];
            OutT* dst = out + m * g.ldc + n;
            if (g.vec && n + EPV <= N) {
                if constexpr (F32) {
                    float4 x = *reinterpret_cast<const float4*>(src);
                    if constexpr (ACC) {
                        const float4 o = *reinterpret_cast<const float4*>(dst);
                        x.x += o.x, x.y += o.y, x.z += o.z, x.w += o.w;
                    }
                    *reinterpret_cast<float4*>(dst) = x;
                } else {
                    const float4 lo = *reinterpret_cast<const float4*>(src);
                    const float4 hi = *reinterpret_cast<const float4*>(src + 4);
                    u32x4 pk;
                    pk.x = pack_bf16x2(lo.x, lo.y);
                    pk.y = pack_bf16x2(lo.z, lo.w);
                    pk.z = pack_bf16x2(hi.x, hi.y);
                    pk.w = pack_bf16x2(hi.z, hi.w);
                    *reinterpret_cast<u32x4*>(dst) = pk;
                }
            } else {
                for (int q = 0; q < EPV && n + q < N; ++q) {
                    if constexpr (F32)
                        dst[q] = ACC ? dst[q] + src[q] : src[q];
                    else
                        dst[q] = bf16_bits(src[q]);
                }
            }
        }
    }
}

// The two GEMMs of one backward block in one launch: dh = dz W (dz read
// along its rows) on the first n_dh workgroups (a multiple of 8; those past
// dh's tiles return at once), dW = dz^T h (dz read down its columns) on the
// rest. dh has few tiles with a long sum (a block's rows x d) and dW many
// with a short one, so dW's tiles fill the compute units that dh leaves
// free, and both start from the dz block just written.
template <class C, int DH_OUT, int DW_OUT>
__global__ void __launch_bounds__(C::THREADS)
lmhead_bwd_gemms_kernel(BwdGemm dh, BwdGemm dw, int64_t n_dh) {
    __shared__ typename C::Smem sm;
    const int64_t b = blockIdx.x;
    if (b < n_dh) {
        if (b < dh.nmt * dh.nnt) bwd_gemm_tile<C, true, DH_OUT>(dh, b, sm);
    } else {
        bwd_gemm_tile<C, false, DW_OUT>(dw, b - n_dh, sm);
    }
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
                             int64_t vbase, hipStream_t stream, const int32_t* dyn_rows = nullptr,
                             int64_t dyn_base = 0) {
    const int64_t nmt = (rows + LmCfg::BM - 1) / LmCfg::BM, nvt = vocab_tiles(V);
    if (!grid_fits(nmt * nvt, LmCfg::THREADS) || ld_h > kMaxLd || ld_w > kMaxLd)
        return DART_ERR_UNSUPPORTED;
    hipLaunchKernelGGL(lmhead_dlogits_kernel<LmCfg>, dim3((unsigned)(nmt * nvt)),
                       dim3(LmCfg::THREADS), 0, stream, hidden, rows, ld_h, weight, V, ld_w, d,
                       target, lse, logp, coef, scale, out, ld_out, vbase, nmt, nvt, dyn_rows,
                       dyn_base);
    return hipGetLastError() == hipSuccess ? DART_OK : DART_ERR_HIP;
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

// The GEMM description of one backward output (out.p at the block's first
// row); mode: kOutF32, kOutF32Acc or kOutBf16.
BwdGemm make_bwd_gemm(const uint16_t* A, int64_t lda, const uint16_t* B, int64_t ldb, int64_t M,
                      int64_t N, int64_t K, const Grad& out) {
    BwdGemm g;
    g.A = A, g.lda = lda, g.B = B, g.ldb = ldb, g.M = M, g.N = N, g.K = K;
    g.out = out.p, g.ldc = out.ld;
    const size_t esz = out.bf16 ? 2 : 4;
    g.vec = reinterpret_cast<uintptr_t>(out.p) % 16 == 0 && (out.ld * esz) % 16 == 0;
    g.nmt = (M + LmCfg::BM - 1) / LmCfg::BM;
    g.nnt = (N + LmCfg::BN - 1) / LmCfg::BN;
    g.dyn = nullptr, g.dyn_base = 0, g.dyn_m = g.dyn_k = false;
    return g;
}

int out_mode(const Grad& out, bool accumulate) {
    return out.bf16 ? kOutBf16 : accumulate ? kOutF32Acc : kOutF32;
}

template <int DH, int DW>
void launch_bwd_gemms_t(const BwdGemm& dh, const BwdGemm& dw, int64_t n_dh, int64_t blocks,
                        hipStream_t stream) {
    hipLaunchKernelGGL((lmhead_bwd_gemms_kernel<LmCfg, DH, DW>), dim3((unsigned)blocks),
                       dim3(LmCfg::THREADS), 0, stream, dh, dw, n_dh);
}

template <int DH>
void launch_bwd_gemms_dw(int dw_mode, const BwdGemm& dh, const BwdGemm& dw, int64_t n_dh,
                         int64_t blocks, hipStream_t stream) {
    if (dw_mode == kOutF32) launch_bwd_gemms_t<DH, kOutF32>(dh, dw, n_dh, blocks, stream);
    else if (dw_mode == kOutF32Acc) launch_bwd_gemms_t<DH, kOutF32Acc>(dh, dw, n_dh, blocks, stream);
    else launch_bwd_gemms_t<DH, kOutBf16>(dh, dw, n_dh, blocks, stream);
}

// One block's dh[rows, d] (+)= dz[rows, cols] W[cols, d] and
// dW[cols, d] (+)= dz[rows, cols]^T h[rows, d], in one launch. A bf16 output
// is never added to (sums over blocks go through fp32). With dyn_rows, the
// block's rows are at most *dyn_rows - dyn_base (read on the device).
dart_status_t launch_bwd_gemms(const uint16_t* dz, int64_t ld_dz, int64_t rows, int64_t cols,
                               const uint16_t* w, int64_t ld_w, const uint16_t* h, int64_t ld_h,
                               int64_t d, const Grad& dh_out, bool dh_acc, const Grad& dw_out,
                               bool dw_acc, hipStream_t stream, const int32_t* dyn_rows,
                               int64_t dyn_base) {
    if ((dh_out.bf16 && dh_acc) || (dw_out.bf16 && dw_acc)) return DART_ERR_INVALID_ARG;
    if (ld_dz > kMaxLd || ld_w > kMaxLd || ld_h > kMaxLd || dh_out.ld > kMaxLd ||
        dw_out.ld > kMaxLd)
        return DART_ERR_UNSUPPORTED;
    BwdGemm dh = make_bwd_gemm(dz, ld_dz, w, ld_w, rows, d, cols, dh_out);
    BwdGemm dw = make_bwd_gemm(dz, ld_dz, h, ld_h, cols, d, rows, dw_out);
    // the block's rows are dh's M and dW's K
    dh.dyn = dw.dyn = dyn_rows;
    dh.dyn_base = dw.dyn_base = dyn_base;
    dh.dyn_m = dw.dyn_k = dyn_rows != nullptr;
    const int64_t n_dh = (dh.nmt * dh.nnt + 7) / 8 * 8;
    const int64_t blocks = n_dh + dw.nmt * dw.nnt;
    if (!grid_fits(blocks, LmCfg::THREADS)) return DART_ERR_UNSUPPORTED;
    const int dhm = out_mode(dh_out, dh_acc), dwm = out_mode(dw_out, dw_acc);
    if (dhm == kOutF32) launch_bwd_gemms_dw<kOutF32>(dwm, dh, dw, n_dh, blocks, stream);
    else if (dhm == kOutF32Acc) launch_bwd_gemms_dw<kOutF32Acc>(dwm, dh, dw, n_dh, blocks, stream);
    else launch_bwd_gemms_dw<kOutBf16>(dwm, dh, dw, n_dh, blocks, stream);
    return hipGetLastError() == hipSuccess ? DART_OK : DART_ERR_HIP;
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
// one block writes is that GEMM's fp32 result rounded once. With dyn_rows, T
// is the most rows there can be and only the first *dyn_rows are formed (the
// count is read on the device: blocks past it have nothing to do, and the
// first row block writes dW even when it holds no rows).
dart_status_t backward_core(const uint16_t* h, int64_t T, int64_t d,
                            int64_t ld_h, const uint16_t* w, int64_t V, int64_t ld_w,
                            const int32_t* target, const float* lse, const float* logp,
                            const float* coef, float scale, const Grad& dh, const Grad& dw,
                            int64_t R,
                            int64_t C, uint16_t* dz, float* acc_h, float* acc_w,
                            hipStream_t stream, const int32_t* dyn_rows = nullptr) {
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
                               logp + r0, coef + r0, scale, dz, ld_dz, c0, stream, dyn_rows, r0);
            if (st != DART_OK) return st;
            const dart_status_t sg = launch_bwd_gemms(
                dz, ld_dz, rows, cols, wc, ld_w, hr, ld_h, d,
                Grad{sum_h.row(r0), sum_h.ld, sum_h.bf16}, c0 > 0,
                Grad{sum_w.row(c0), sum_w.ld, sum_w.bf16}, r0 > 0, stream, dyn_rows, r0);
            if (sg != DART_OK) return sg;
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
    // the MFMA tiles address rows by 32-bit offsets from a tile's first row
    if (ld_h > kMaxLd || ld_w > kMaxLd || ld_dh > kMaxLd || ld_dw > kMaxLd)
        return DART_ERR_UNSUPPORTED;
    const BackwardPlan P = plan_backward(T, d, V, chunk_rows, chunk_cols, flags);
    if (P.total == 0) return DART_ERR_UNSUPPORTED;
    if (workspace_bytes < P.total) return DART_ERR_INVALID_ARG;
    if (const dart_status_t ck = dart_check::run(
            stream, {{dart_check::Item::Ids, target, T, V}}); ck != DART_OK)
        return ck;

    const uint16_t* h = static_cast<const uint16_t*>(hidden);
    const uint16_t* w = static_cast<const uint16_t*>(weight);
    char* ws = static_cast<char*>(workspace);
    uint16_t* dz = reinterpret_cast<uint16_t*>(ws + P.dz);
    float* acc_w = P.acc_w ? reinterpret_cast<float*>(ws + P.accw) : nullptr;
    float* acc_h = P.acc_h ? reinterpret_cast<float*>(ws + P.acch) : nullptr;
    const Grad dh{dhidden, ld_dh, P.bf16}, dw{dweight, ld_dw, P.bf16};
    if (!P.skip)
        return backward_core(h, T, d, ld_h, w, V, ld_w, target, lse, logp, tok_coef,
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
    // the kernels read the kept-row count on the device: T rows at most
    const dart_status_t st =
        backward_core(h_c, T, d, d, w, V, ld_w, target_c, lse_c, logp_c, coef_c, inv_temp,
                      Grad{dh_c, d, false}, dw, P.rows, P.cols, dz, nullptr, acc_w, stream, count);
    if (st != DART_OK) return st;
    const unsigned nb = (unsigned)(T < kRowBlocks ? T : kRowBlocks);
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
