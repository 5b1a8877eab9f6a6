// Grouped fp32 MFMA GEMM for gfx950 with fused epilogues.
//
// One launch covers every tile of a list of independent products (all
// factors' products of one dependency level of the step). Each product
// carries its own epilogue (flags and coefficient set, decided at run time
// per problem), so products with different epilogues share a launch. A
// workgroup of 256 threads computes one 128 x 128 tile of C = A * B; its
// four waves each own a 64 x 64 sub-tile held as 4 x 4 blocks of
// v_mfma_f32_16x16x4_f32 accumulators (this form reads and writes half as
// many accumulator registers per flop as the 32 x 32 one). K is consumed in
// slabs of 32 staged through double-buffered LDS (one barrier per slab): while
// the waves run the MFMAs of slab k, slab k+1 streams into the other buffer.
// K-contiguous operands go straight from global memory to LDS
// (global_load_lds_dwordx4, no register staging); an MN-contiguous operand
// (the NN kernel's B) is held in registers and written to LDS after the MFMAs.
//
// Within a slab, lane l of a wave contributes k = 16*kg + 4*q + s to the MFMA
// of step s (s = 0..3) of 16-wide k group kg, with q = quarter(l / 16): the
// four lane groups take disjoint quarters of each group, so a K-contiguous
// operand is read from LDS as one 16-byte load per lane per 16 k values. The
// same k map is used for A and B, so every product A[i][k] * B[k][j] is
// formed exactly once.
#pragma once

#include <hip/hip_runtime.h>

#include "jorge_types.hpp"

namespace jorge {

typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef float f32x16 __attribute__((ext_vector_type(16)));

// Accumulator layout. A wave's 64 x 64 quadrant (wy, wx) of its tile is a
// 4 x 4 grid of 16 x 16 blocks; block b = 4 i + j (rows 16 i, columns 16 j of
// the quadrant) is one v_mfma_f32_16x16x4_f32 accumulator, in which lane l
// holds column l % 16, rows 4 (l / 16) .. 4 (l / 16) + 3. Each lane thus
// holds, for each of its 16 blocks, four consecutive rows of one column.
// Row and column of the first of those four values, relative to the tile:
__device__ __forceinline__ int acc_row(int b, int lane, int wy) { return wy * 64 + (b >> 2) * 16 + (lane >> 4) * 4; }
__device__ __forceinline__ int acc_col(int b, int lane, int wx) { return wx * 64 + (b & 3) * 16 + (lane & 15); }

// The k quarter that lane group g (lanes 16 g .. 16 g + 15) reads: groups 1
// and 2 swapped. A 16-byte LDS read is served in passes that pair lanes
// 0-7 with 32-39 (8-15 with 40-47, ...); with the swap, the two halves of a
// pass read chunks an odd distance apart, which the XOR layout below puts in
// opposite halves of the banks (with the identity map they collide 2-way).
__device__ __forceinline__ int quarter(int g) { return ((g & 1) << 1) | (g >> 1); }

constexpr int kTile = 128;                    // tile rows = tile columns
constexpr int kSlab = 32;                     // K per LDS stage
constexpr int kGemmThreads = 256;
// A K-contiguous operand slab (128 rows x 32 k) sits in LDS as 16 blocks of
// 8 rows of 128 bytes, the 1 KB one wave-wide 16-byte load to LDS writes:
// lane L loads row L / 8 of the block, so eight consecutive lanes read one
// contiguous 128-byte row of global memory. The lane loads logical chunk
// (L % 8) ^ (L / 8) (k = 4c .. 4c+3 is chunk c), so chunk c of block row r
// sits at physical chunk c ^ r: eight lanes reading one chunk of 8 rows hit
// 8 distinct 16-byte bank groups, and the 128-byte pad between blocks moves
// the next 8 rows to the other half of a 64-bank LDS.
constexpr int kLdsBlock = 8 * 32 + 32;        // floats per 8-row block, with its pad
// Row stride of an M/N-contiguous operand in LDS: 132 floats puts the rows
// that the four lane groups read in one step (4 apart) on distinct quarters
// of the banks.
constexpr int kLdsMN = kTile + 4;
constexpr int kLdsOperand = 16 * kLdsBlock;   // floats per operand per stage (>= kSlab * kLdsMN)
static_assert(kLdsOperand >= kSlab * kLdsMN, "LDS operand buffer too small");
static_assert(kLdsOperand / 2 >= 2 * 64 * 16, "a small-mode stage (two 64 x 16 slabs) must fit in half an operand buffer");

// Pointers into global memory (address space 1): loads through them compile
// to global_load rather than flat_load, which would also count against the
// LDS wait counter and make every LDS wait drain the in-flight prefetch.
typedef __attribute__((address_space(1))) const f32x4 global_f32x4;
typedef __attribute__((address_space(1))) const float global_f32;

__device__ __forceinline__ f32x4 gload4(const float* p) {
    return *(global_f32x4*)p;
}

typedef __attribute__((address_space(1))) void global_void;
typedef __attribute__((address_space(3))) void lds_void;

// Byte offsets, from the operand's base at k = 0, of the four 16-byte chunks
// this lane loads for each 128 x 32 K-contiguous operand slab of a tile. Wave
// w fills LDS blocks 4w .. 4w+3 with one 16-byte load per lane each. Rows
// past the extent `lim` are clamped to the last valid one: they only feed
// outputs that the epilogue discards. The offsets do not change along K, so
// they are computed once per tile.
struct SlabLanes {
    unsigned o[4];
};

__device__ __forceinline__ void slab_lanes(int ld, int mn0, int lim, SlabLanes& L) {
    const int lane = threadIdx.x & 63;
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const int chunk = (lane & 7) ^ (lane >> 3);
#pragma unroll
    for (int j = 0; j < 4; ++j) {
        const int row = min(mn0 + (wave * 4 + j) * 8 + (lane >> 3), lim - 1);
        L.o[j] = (unsigned)row * (unsigned)ld * 4u + (unsigned)chunk * 16u;
    }
}

typedef __attribute__((address_space(1))) const char gcchar;

// Global -> LDS directly: the slab at k0 of an operand whose lane offsets
// are L. The uniform part of the address (base + k0) stays in scalar
// registers, so each load is one instruction with no address arithmetic.
// The loads complete asynchronously (vmcnt).
__device__ __forceinline__ void load_slab_lds(const float* __restrict__ base, const SlabLanes& L, int k0, float* s) {
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const gcchar* g = (const gcchar*)(base + k0);
#pragma unroll
    for (int j = 0; j < 4; ++j)
        __builtin_amdgcn_global_load_lds((global_void*)(g + L.o[j]), (lds_void*)(s + (wave * 4 + j) * kLdsBlock), 16,
                                         0, 0);
}

// Global -> registers: one 32 x 128 MN-contiguous operand slab, four 16-byte
// loads per thread (columns past `lim` clamped as above).
__device__ __forceinline__ void load_slab_mn(const float* __restrict__ base, int ld, int mn0, int lim,
                                             int k0, f32x4 (&r)[4]) {
    const int tid = threadIdx.x;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        const int u = tid + i * kGemmThreads;
        const int col = min(mn0 + (u & 31) * 4, lim - 4);
        r[i] = gload4(base + (size_t)(k0 + (u >> 5)) * ld + col);
    }
}

// Registers -> LDS for the MN-contiguous operand.
__device__ __forceinline__ void store_slab_mn(float* s, const f32x4 (&r)[4]) {
    const int tid = threadIdx.x;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        const int u = tid + i * kGemmThreads;
        *reinterpret_cast<f32x4*>(s + (u >> 5) * kLdsMN + (u & 31) * 4) = r[i];
    }
}

// LDS -> MFMA operand registers: values for k = k .. k+3 (k a multiple of 4)
// at row/column mn.
template <bool KMAJ>
__device__ __forceinline__ void fragment(const float* s, int mn, int k, float (&f)[4]) {
    if constexpr (KMAJ) {
        const int r = mn & 7;
        const f32x4 v =
            *reinterpret_cast<const f32x4*>(s + (mn >> 3) * kLdsBlock + r * 32 + (((k >> 2) ^ r) << 2));
        f[0] = v[0]; f[1] = v[1]; f[2] = v[2]; f[3] = v[3];
    } else {
#pragma unroll
        for (int q = 0; q < 4; ++q) f[q] = s[(k + q) * kLdsMN + mn];
    }
}

// Which of a wave's 16 blocks it multiplies: every block; on a diagonal
// tile of a symmetric result, only blocks on or above the diagonal (i <= j)
// of a diagonal quadrant; or none, for the quadrant below the diagonal. The
// epilogue of a symmetric result never reads the blocks left out.
enum BlockSet : int { BS_ALL = 0, BS_UPPER = 1, BS_NONE = 2 };

// Fragments of one 16-wide k group of a slab for the calling wave: A rows
// wy*64 + 16 i + (lane % 16) and B columns wx*64 + 16 i + (lane % 16), at k
// = kg*16 + 4 quarter(lane / 16) .. + 3.
template <bool AK, bool BK>
__device__ __forceinline__ void group_fragments(const float* sa, const float* sb, int wy, int wx, int lane, int kg,
                                                float (&a)[4][4], float (&b)[4][4]) {
    const int r = lane & 15, q = quarter(lane >> 4);
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        fragment<AK>(sa, wy * 64 + i * 16 + r, kg * 16 + q * 4, a[i]);
        fragment<BK>(sb, wx * 64 + i * 16 + r, kg * 16 + q * 4, b[i]);
    }
}

// The 64 MFMAs of one 16-wide k group (the blocks of block set BS).
template <int BS>
__device__ __forceinline__ void group_mma(const float (&a)[4][4], const float (&b)[4][4], f32x4 (&acc)[16]) {
#pragma unroll
    for (int st = 0; st < 4; ++st)
#pragma unroll
        for (int i = 0; i < 4; ++i)
#pragma unroll
            for (int j = 0; j < 4; ++j)
                if (BS == BS_ALL || i <= j)
                    acc[i * 4 + j] = __builtin_amdgcn_mfma_f32_16x16x4f32(a[i][st], b[j][st], acc[i * 4 + j], 0, 0, 0);
}

// The MFMAs of one LDS slab (sa, sb) of two 16-wide k groups, whose first
// group's fragments the caller has already read into (fa, fb). The second
// group's fragments are read while the first group's MFMAs run. Between the
// two groups, `sync` makes the next slab (nsa, nsb) visible to every wave
// (and ends every wave's reads of this slab); the next slab's first-group
// fragments are then read into (fa, fb) while the second group's MFMAs run,
// so neither the barrier nor that LDS latency leaves the matrix pipe idle.
// `issue` starts the loads of a later slab into the stage that is free; the
// compiler's own schedule spreads those loads and the LDS reads among the
// MFMAs (it measured 2-4% faster than a fixed interleave).
template <bool AK, bool BK, int BS, class Issue, class Sync>
__device__ __forceinline__ void mma_slab(const float* sa, const float* sb, const float* nsa, const float* nsb, int wy,
                                         int wx, int lane, float (&fa)[4][4], float (&fb)[4][4], f32x4 (&acc)[16],
                                         Issue&& issue, Sync&& sync) {
    static_assert(kSlab == 32, "a slab is two 16-wide k groups");
    if constexpr (BS == BS_NONE) {
        issue();
        sync();
        return;
    }
    float a[4][4], b[4][4];
    group_fragments<AK, BK>(sa, sb, wy, wx, lane, 1, a, b);
    // These reads too go first: the barrier in `sync` waits for them.
    __builtin_amdgcn_sched_barrier(0);
    issue();
    group_mma<BS>(fa, fb, acc);
    sync();
    group_fragments<AK, BK>(nsa, nsb, wy, wx, lane, 0, fa, fb);
    // Keep those reads ahead of the MFMAs (the scheduler would sink them).
    __builtin_amdgcn_sched_barrier(0);
    group_mma<BS>(a, b, acc);
}

// Sum of one double per lane over a 64-lane wave, in a fixed order.
__device__ __forceinline__ double wave_sum(double v) {
#pragma unroll
    for (int off = 32; off > 0; off >>= 1) v += __shfl_xor(v, off);
    return v;
}

// Sum of one double per thread over the workgroup, in a fixed order.
__device__ __forceinline__ double block_sum_256(double v, double* red) {
#pragma unroll
    for (int off = 32; off > 0; off >>= 1) v += __shfl_xor(v, off);
    if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = v;
    __syncthreads();
    return (red[0] + red[1]) + (red[2] + red[3]);
}

// Operand base pointer, leading dimension and local k of one slab: the
// second K segment (k >= K1) reads A2 / B2.
struct SlabSrc {
    const float* a;
    const float* b;
    int lda, ldb, k;
};

__device__ __forceinline__ SlabSrc slab_src(const GemmProblem& p, int k0) {
    if (k0 < p.K1) return {p.A, p.B, p.lda, p.ldb, k0};
    return {p.A2, p.B2, p.lda2, p.ldb2, k0 - p.K1};
}

// One LDS stage of the GEMM: the A and B operand slabs. The two stages of
// the double buffer are separate __shared__ objects, so the compiler can see
// that loads into one stage never alias reads of the other and does not wait
// for the in-flight prefetch before reading the current stage.
struct GemmStageLds {
    float a[kLdsOperand];
    float b[kLdsOperand];
};

// Lane offsets of a tile's operand slabs for both K segments.
struct TileLanes {
    SlabLanes a, b, a2, b2;
};

// Starts the copy of slab k0 (absolute K) of tile (row0, col0) into stage st.
// K-contiguous operands load to LDS directly; the MN-contiguous B is held in rb
// until store_b (after the MFMAs of the other stage).
template <bool BK>
__device__ __forceinline__ void issue_slab(const GemmProblem& p, const TileLanes& tl, int col0, int k0,
                                           GemmStageLds& st, f32x4 (&rb)[4]) {
    // Segment selection by selects, not branches, so the loads stay in the
    // scheduling region of the MFMAs they are interleaved with.
    const bool two = k0 >= p.K1;
    const int k = two ? k0 - p.K1 : k0;
    SlabLanes la, lb;
#pragma unroll
    for (int j = 0; j < 4; ++j) {
        la.o[j] = two ? tl.a2.o[j] : tl.a.o[j];
        if constexpr (BK) lb.o[j] = two ? tl.b2.o[j] : tl.b.o[j];
    }
    load_slab_lds(two ? p.A2 : p.A, la, k, st.a);
    if constexpr (BK) load_slab_lds(two ? p.B2 : p.B, lb, k, st.b);
    else load_slab_mn(two ? p.B2 : p.B, two ? p.ldb2 : p.ldb, col0, p.N, k, rb);
}

template <bool BK>
__device__ __forceinline__ void finish_slab(GemmStageLds& st, const f32x4 (&rb)[4]) {
    if constexpr (!BK) store_slab_mn(st.b, rb);
    // This wave's loads to LDS have landed and its reads of the other stage
    // are complete; the barrier makes every wave's loads visible and lets the
    // other stage be refilled.
    asm volatile("s_waitcnt vmcnt(0) lgkmcnt(0)" ::: "memory");
    __syncthreads();
}

// The slab loop of gemm_mainloop for the calling wave's block set BS (one
// copy per set, so the loop itself has no branches on it). Slab 0 is in s0
// and its first-group fragments in (fa, fb).
template <bool AK, bool BK, int BS>
__device__ __forceinline__ void slab_loop(const GemmProblem& p, const TileLanes& tl, int col0, int k0, int nk,
                                          GemmStageLds& s0, GemmStageLds& s1, f32x4 (&rb)[4], int wy, int wx,
                                          int lane, float (&fa)[4][4], float (&fb)[4][4], f32x4 (&acc)[16]) {
    // Raised issue priority while this wave runs its MFMAs (lowered around
    // each barrier): the two waves sharing a SIMD then alternate between
    // MFMA and memory phases.
    auto sync_to = [&](GemmStageLds& st) {
        __builtin_amdgcn_s_setprio(0);
        finish_slab<BK>(st, rb);
        __builtin_amdgcn_s_setprio(1);
    };
    // Pairs of slabs: slab kt is in s0, kt+1 goes to s1 and kt+2 back to s0.
    // The loop has no other exit, so the accumulators stay in place.
    int kt = 0;
    __builtin_amdgcn_s_setprio(1);
    for (; kt + 2 <= nk; kt += 2) {
        mma_slab<AK, BK, BS>(s0.a, s0.b, s1.a, s1.b, wy, wx, lane, fa, fb, acc,
                             [&] { issue_slab<BK>(p, tl, col0, k0 + (kt + 1) * kSlab, s1, rb); },
                             [&] { sync_to(s1); });
        // Past the last slab the load repeats slab nk - 1 into the idle stage
        // (never multiplied), which keeps the loop free of branches.
        const int kn = min(kt + 2, nk - 1);
        mma_slab<AK, BK, BS>(s1.a, s1.b, s0.a, s0.b, wy, wx, lane, fa, fb, acc,
                             [&] { issue_slab<BK>(p, tl, col0, k0 + kn * kSlab, s0, rb); },
                             [&] { sync_to(s0); });
    }
    if (kt < nk)  // odd slab count: the last slab is in s0; nothing follows it
        mma_slab<AK, BK, BS>(s0.a, s0.b, s1.a, s1.b, wy, wx, lane, fa, fb, acc, [] {}, [] {});
    __builtin_amdgcn_s_setprio(0);
}

// The product of one 128 x 128 tile (tm, tn) of problem p over K range
// [k0, k1), accumulated by the whole workgroup into acc. Every thread of the
// workgroup must call it. Waves return without waiting for each other, so
// LDS may be written after it only behind a barrier (the grouped kernel
// writes none). The slab loop is unrolled by two so each half reads one stage
// and fills the other.
template <bool AK, bool BK>
__device__ __forceinline__ void gemm_mainloop(const GemmProblem& p, int tm, int tn, int k0, int k1,
                                              GemmStageLds& s0, GemmStageLds& s1, f32x4 (&acc)[16]) {
    static_assert(AK, "the A operand is always K-contiguous");
    const int row0 = tm * kTile, col0 = tn * kTile;
    const int lane = threadIdx.x & 63, wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const int wy = wave >> 1, wx = wave & 1;

#pragma unroll
    for (int b = 0; b < 16; ++b)
#pragma unroll
        for (int e = 0; e < 4; ++e) acc[b][e] = 0.0f;

    TileLanes tl;
    slab_lanes(p.lda, row0, p.M, tl.a);
    slab_lanes(p.lda2, row0, p.M, tl.a2);
    if constexpr (BK) {
        slab_lanes(p.ldb, col0, p.N, tl.b);
        slab_lanes(p.ldb2, col0, p.N, tl.b2);
    }
    f32x4 rb[4];
    const int nk = (k1 - k0) / kSlab;
    issue_slab<BK>(p, tl, col0, k0, s0, rb);
    finish_slab<BK>(s0, rb);
    float fa[4][4], fb[4][4];
    group_fragments<AK, BK>(s0.a, s0.b, wy, wx, lane, 0, fa, fb);
    // A quadrant that lies wholly past the product's padded extent (a product
    // 32 or 64 rows or columns wide, or an edge tile) multiplies nothing: its
    // outputs are discarded. On a diagonal tile of a symmetric result the
    // quadrant below the diagonal is not needed and the diagonal quadrants
    // only on and above it.
    if (row0 + wy * 64 >= p.M || col0 + wx * 64 >= p.N) {
        slab_loop<AK, BK, BS_NONE>(p, tl, col0, k0, nk, s0, s1, rb, wy, wx, lane, fa, fb, acc);
    } else if (p.upper && tm == tn) {
        if (wy > wx) slab_loop<AK, BK, BS_NONE>(p, tl, col0, k0, nk, s0, s1, rb, wy, wx, lane, fa, fb, acc);
        else if (wy == wx) slab_loop<AK, BK, BS_UPPER>(p, tl, col0, k0, nk, s0, s1, rb, wy, wx, lane, fa, fb, acc);
        else slab_loop<AK, BK, BS_ALL>(p, tl, col0, k0, nk, s0, s1, rb, wy, wx, lane, fa, fb, acc);
    } else {
        slab_loop<AK, BK, BS_ALL>(p, tl, col0, k0, nk, s0, s1, rb, wy, wx, lane, fa, fb, acc);
    }
    // No closing barrier: every load into LDS has landed (the last slab's
    // wait), and nothing after the main loop writes LDS, so each wave goes on
    // to its epilogue as soon as its own MFMAs are issued.
}

// Partial products of split tiles: thread t (= 64 wave + lane) keeps its 64
// accumulators as 16 float4 (one per block), float4 b of a partial at
// b * 1024 + 4 t (coalesced across threads).
__device__ __forceinline__ void store_partial(float* __restrict__ blk, const f32x4 (&acc)[16]) {
#pragma unroll
    for (int b = 0; b < 16; ++b) *reinterpret_cast<f32x4*>(blk + b * 1024 + 4 * threadIdx.x) = acc[b];
}

// The 64 values of one partial product that thread t of the computing workgroup kept.
__device__ __forceinline__ void load_partial(const float* __restrict__ blk, int t, f32x4 (&v)[16]) {
#pragma unroll
    for (int b = 0; b < 16; ++b) v[b] = *(global_f32x4*)(blk + b * 1024 + 4 * t);
}

__device__ __forceinline__ void add_partial(const f32x4 (&v)[16], f32x4 (&acc)[16]) {
#pragma unroll
    for (int b = 0; b < 16; ++b) {
        acc[b][0] += v[b][0]; acc[b][1] += v[b][1];
        acc[b][2] += v[b][2]; acc[b][3] += v[b][3];
    }
}

typedef __attribute__((address_space(1))) float gfloat;
typedef __attribute__((address_space(1))) f32x4 gfloat4;
typedef __attribute__((address_space(1))) char gchar;

// Global accesses at a 32-bit byte offset from a uniform base: they compile to
// the base-in-SGPR, offset-in-VGPR form with no 64-bit address arithmetic.
// Every matrix here spans at most 32768^2 floats, so byte offsets fit in 32 bits.
__device__ __forceinline__ float ld_at(const float* base, unsigned byte_off) {
    return *(const gfloat*)((const gchar*)base + byte_off);
}
__device__ __forceinline__ void st_at(float* base, unsigned byte_off, float v) {
    *(gfloat*)((gchar*)base + byte_off) = v;
}
__device__ __forceinline__ void st4_at(float* base, unsigned byte_off, f32x4 v) {
    *(gfloat4*)((gchar*)base + byte_off) = v;
}

// The epilogue body for one combination of flags F and symmetry UP, known
// at compile time. value = ci [row == col < valid_m] + cx X + cc acc.
// Offsets are 32-bit (every matrix has fewer than 2^32 elements) from
// uniform base pointers; per-element masks are only evaluated on edge tiles
// and on diagonal tiles of symmetric results.
template <int F, bool UP, bool MASKED>
__device__ __forceinline__ double epilogue_body(const GemmProblem& p, int tm, int tn, const f32x4 (&acc)[16],
                                                float ci, float cx, float cc, int lane, int wave) {
    constexpr bool kReadX = (F & EF_READX) != 0;
    constexpr bool kRead = (F & (EF_READX | EF_DOT)) != 0;
    const int row0 = tm * kTile, col0 = tn * kTile;
    const int wy = wave >> 1, wx = wave & 1;
    const bool diag = MASKED && UP && tm == tn;
    const bool ident = kReadX && ci != 0.f && tm == tn;
    constexpr double w_off = UP ? 2.0 : 1.0;   // off-diagonal tiles of a symmetric result
    float* C = p.C;
    float* C2 = p.C2;
    const float* X = p.X;
    // Row strides in bytes.
    const unsigned sc = 4u * p.ldc, sc2 = 4u * p.ldc2, sx = 4u * p.ldx;

    // Every X value the thread will use is loaded before anything is stored,
    // so one memory round trip serves the whole tile (X may be C itself, and
    // the compiler keeps loads after earlier stores it cannot tell apart).
    // Masked tiles clamp positions outside M x N to the last row and column
    // and drop those values; every position the thread uses is also one it
    // writes, and no other thread writes it.
    f32x4 xv[16];
    if constexpr (kRead) {
#pragma unroll
        for (int b = 0; b < 16; ++b) {
            const int col = col0 + acc_col(b, lane, wx);
            const int colc = MASKED ? min(col, p.N - 1) : col;
            // rowb .. rowb+3 are all inside M when rowb is (M is a multiple of 4).
            const int rowb = row0 + acc_row(b, lane, wy);
            const int rowc = MASKED ? min(rowb, p.M - 4) : rowb;
            const unsigned ox = (unsigned)rowc * sx + 4u * (unsigned)colc;
#pragma unroll
            for (int e = 0; e < 4; ++e) xv[b][e] = ld_at(X, ox + e * sx);
        }
    }

    double part = 0.0;
#pragma unroll
    for (int b = 0; b < 16; ++b) {
        const int col = col0 + acc_col(b, lane, wx);
        const int rowb = row0 + acc_row(b, lane, wy);
        // rowb .. rowb+3 are all inside M when rowb is (M is a multiple of 4).
        if (MASKED && (rowb >= p.M || col >= p.N)) continue;
        // X at positions this thread writes (read and written by the same thread).
        f32x4 x;
        f32x4 out;
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            const float v = acc[b][e];
            float o = cc * v;
            if constexpr (kRead) x[e] = xv[b][e];
            if constexpr (kReadX) {
                const float id = (ident && rowb + e == col && col < p.valid_m) ? ci : 0.0f;
                o = (id + cx * x[e]) + o;
            }
            out[e] = o;
        }
        if (!diag) {
#pragma unroll
            for (int e = 0; e < 4; ++e) {
                if constexpr ((F & EF_NORM) != 0) part += w_off * (double)out[e] * (double)out[e];
                if constexpr ((F & EF_DOT) != 0) part += w_off * (double)acc[b][e] * (double)x[e];
            }
            if constexpr ((F & EF_STORE) != 0) {
                const unsigned oc = (unsigned)rowb * sc + 4u * (unsigned)col;
#pragma unroll
                for (int e = 0; e < 4; ++e) st_at(C, oc + e * sc, out[e]);
                if constexpr (UP) st4_at(C, (unsigned)col * sc + 4u * (unsigned)rowb, out);
            }
            if constexpr ((F & EF_STORE_T) != 0) st4_at(C2, (unsigned)col * sc2 + 4u * (unsigned)rowb, out);
        } else {
            // Diagonal tile of a symmetric result: element (row, col) with
            // row <= col is written at both positions.
#pragma unroll
            for (int e = 0; e < 4; ++e) {
                const int row = rowb + e;
                if (row > col) continue;
                const double w = row != col ? 2.0 : 1.0;
                if constexpr ((F & EF_NORM) != 0) part += w * (double)out[e] * (double)out[e];
                if constexpr ((F & EF_DOT) != 0) part += w * (double)acc[b][e] * (double)x[e];
                if constexpr ((F & EF_STORE) != 0) {
                    st_at(C, (unsigned)row * sc + 4u * (unsigned)col, out[e]);
                    if (row != col) st_at(C, (unsigned)col * sc + 4u * (unsigned)row, out[e]);
                }
            }
        }
    }
    return part;
}

// The epilogue for a flag combination without a compiled body (not used by
// the launch tables the library builds; kept so every combination works).
__device__ __forceinline__ double epilogue_generic(const GemmProblem& p, int tm, int tn, const f32x4 (&acc)[16],
                                                float ci, float cx, float cc, int lane, int wave) {
    double part = 0.0;
    const int F = p.flags;
    const bool up = p.upper != 0;
    const int row0 = tm * kTile, col0 = tn * kTile;
    const int wy = wave >> 1, wx = wave & 1;
    float* C = p.C;
    float* C2 = p.C2;
    const float* X = p.X;
    const unsigned sc = 4u * p.ldc, sc2 = 4u * p.ldc2, sx = 4u * p.ldx;
#pragma unroll
    for (int b = 0; b < 16; ++b) {
        const int col = col0 + acc_col(b, lane, wx);
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            const int row = row0 + acc_row(b, lane, wy) + e;
            if (row >= p.M || col >= p.N || (up && row > col)) continue;
            const float v = acc[b][e];
            const float xe = (F & (EF_READX | EF_DOT)) ? ld_at(X, (unsigned)row * sx + 4u * (unsigned)col) : 0.f;
            float o = cc * v;
            if (F & EF_READX) o = (((row == col && row < p.valid_m) ? ci : 0.0f) + cx * xe) + o;
            const double w = (up && row != col) ? 2.0 : 1.0;
            if (F & EF_NORM) part += w * (double)o * (double)o;
            if (F & EF_DOT) part += w * (double)v * (double)xe;
            if (F & EF_STORE) {
                st_at(C, (unsigned)row * sc + 4u * (unsigned)col, o);
                if (up && row != col) st_at(C, (unsigned)col * sc + 4u * (unsigned)row, o);
            }
            if (F & EF_STORE_T) st_at(C2, (unsigned)col * sc2 + 4u * (unsigned)row, o);
        }
    }
    return part;
}

// m = beta1 m + (1 - beta1) acc on the dense valid_m x valid_n momentum.
template <bool MASKED>
__device__ __forceinline__ double epilogue_momentum(const GemmProblem& p, int tm, int tn,
                                                    const f32x4 (&acc)[16], float beta1, int lane, int wave) {
    const int row0 = tm * kTile, col0 = tn * kTile;
    const int wy = wave >> 1, wx = wave & 1;
    float* mom = p.mom;
    const unsigned sm = 4u * p.ldmom;
    // All of this thread's momentum values are loaded before any is stored
    // (one memory round trip per tile); masked tiles clamp positions outside
    // the dense valid_m x valid_n momentum to its last row and column and
    // drop those values.
    f32x4 mv[16];
#pragma unroll
    for (int b = 0; b < 16; ++b) {
        const int col = col0 + acc_col(b, lane, wx);
        const int colc = MASKED ? min(col, p.valid_n - 1) : col;
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            const int row = row0 + acc_row(b, lane, wy) + e;
            const int rowc = MASKED ? min(row, p.valid_m - 1) : row;
            mv[b][e] = ld_at(mom, (unsigned)rowc * sm + 4u * (unsigned)colc);
        }
    }
    double part = 0.0;
#pragma unroll
    for (int b = 0; b < 16; ++b) {
        const int col = col0 + acc_col(b, lane, wx);
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            const int row = row0 + acc_row(b, lane, wy) + e;
            if (MASKED && !(row < p.valid_m && col < p.valid_n)) continue;
            const unsigned o = (unsigned)row * sm + 4u * (unsigned)col;
            const float mn = beta1 * mv[b][e] + (1.0f - beta1) * acc[b][e];
            st_at(mom, o, mn);
            part += (double)mn * (double)mn;
        }
    }
    return part;
}

// The epilogue of quadrant `wave` of tile (tm, tn) of problem p for the
// product in acc (this lane's accumulators); beta1 is the momentum of
// EF_MOMENTUM. One uniform switch picks the compiled body for the problem's
// flags. The wave's partial sum (norm, dot product) goes to sub-slot `wave`
// of the tile's slot.
//
// Symmetric results (p.upper): only tiles with tm <= tn are computed. An
// element (row, col) with row <= col is written at (row, col) and at
// (col, row), elements below the diagonal of a diagonal tile are skipped,
// so the stored matrix is bitwise symmetric whatever the product's rounding.
// The epilogue reads X only at the positions it is about to write, by the
// same thread, so X may alias C (an in-place update).
__device__ __forceinline__ void gemm_epilogue(const GemmProblem& p, int tm, int tn, int slot, float beta1,
                                              const f32x4 (&acc)[16], int lane, int wave) {
    const int flags = p.flags;
    double part = 0.0;
    if (flags & EF_MOMENTUM) {
        // Interior tiles of the dense valid_m x valid_n momentum need no masks.
        if ((tm + 1) * kTile <= p.valid_m && (tn + 1) * kTile <= p.valid_n)
            part = epilogue_momentum<false>(p, tm, tn, acc, beta1, lane, wave);
        else
            part = epilogue_momentum<true>(p, tm, tn, acc, beta1, lane, wave);
    } else {
        float ci = 0.f, cx = 0.f, cc = 1.f;
        if (p.coef != CO_ONE) {
            const FactorScalars* sc = p.sc;
            switch (p.coef) {
                case CO_POLY: ci = 1.f; cx = -sc->a; cc = sc->b; break;
                case CO_SCALE: cc = sc->sf; break;
                case CO_WMIX: cx = sc->a; cc = -sc->b; break;
                case CO_SYR2K: cx = sc->sf; cc = -0.5f * sc->sf; break;
                case CO_LITUPD: cx = sc->sf; cc = -sc->sf; break;
                case CO_VSER: cx = sc->b; cc = -sc->e; break;
                case CO_POLY3: ci = 1.f; cx = -sc->a; break;
                case CO_WMIX3: cx = sc->a; cc = -1.f; break;
                default: break;
            }
        }
        const int key = flags | (p.upper ? 256 : 0);
        const bool masked = (tm + 1) * kTile > p.M || (tn + 1) * kTile > p.N || (p.upper && tm == tn);
        switch (key) {
            case EF_STORE: part = masked ? epilogue_body<EF_STORE, false, true>(p, tm, tn, acc, ci, cx, cc, lane, wave)
                            : epilogue_body<EF_STORE, false, false>(p, tm, tn, acc, ci, cx, cc, lane, wave); break;
            case EF_STORE | 256: part = masked ? epilogue_body<EF_STORE, true, true>(p, tm, tn, acc, ci, cx, cc, lane, wave)
                            : epilogue_body<EF_STORE, true, false>(p, tm, tn, acc, ci, cx, cc, lane, wave); break;
            case EF_STORE_T: part = masked ? epilogue_body<EF_STORE_T, false, true>(p, tm, tn, acc, ci, cx, cc, lane, wave)
                            : epilogue_body<EF_STORE_T, false, false>(p, tm, tn, acc, ci, cx, cc, lane, wave); break;
            case EF_DOT | 256: part = masked ? epilogue_body<EF_DOT, true, true>(p, tm, tn, acc, ci, cx, cc, lane, wave)
                            : epilogue_body<EF_DOT, true, false>(p, tm, tn, acc, ci, cx, cc, lane, wave); break;
            case EF_STORE | EF_STORE_T | EF_NORM:
                part = masked ? epilogue_body<EF_STORE | EF_STORE_T | EF_NORM, false, true>(p, tm, tn, acc, ci, cx, cc, lane, wave)
                            : epilogue_body<EF_STORE | EF_STORE_T | EF_NORM, false, false>(p, tm, tn, acc, ci, cx, cc, lane, wave);
                break;
            case EF_STORE_T | EF_READX:
                part = masked ? epilogue_body<EF_STORE_T | EF_READX, false, true>(p, tm, tn, acc, ci, cx, cc, lane, wave)
                            : epilogue_body<EF_STORE_T | EF_READX, false, false>(p, tm, tn, acc, ci, cx, cc, lane, wave);
                break;
            case EF_STORE | EF_READX:
                part = masked ? epilogue_body<EF_STORE | EF_READX, false, true>(p, tm, tn, acc, ci, cx, cc, lane, wave)
                            : epilogue_body<EF_STORE | EF_READX, false, false>(p, tm, tn, acc, ci, cx, cc, lane, wave);
                break;
            case EF_STORE | EF_STORE_T:
                part = masked ? epilogue_body<EF_STORE | EF_STORE_T, false, true>(p, tm, tn, acc, ci, cx, cc, lane, wave)
                              : epilogue_body<EF_STORE | EF_STORE_T, false, false>(p, tm, tn, acc, ci, cx, cc, lane, wave);
                break;
            case EF_STORE | EF_STORE_T | EF_READX:
                part = masked ? epilogue_body<EF_STORE | EF_STORE_T | EF_READX, false, true>(p, tm, tn, acc, ci, cx, cc, lane, wave)
                              : epilogue_body<EF_STORE | EF_STORE_T | EF_READX, false, false>(p, tm, tn, acc, ci, cx,
                                                                                              cc, lane, wave);
                break;
            case EF_STORE | EF_READX | 256:
                part = masked ? epilogue_body<EF_STORE | EF_READX, true, true>(p, tm, tn, acc, ci, cx, cc, lane, wave)
                            : epilogue_body<EF_STORE | EF_READX, true, false>(p, tm, tn, acc, ci, cx, cc, lane, wave);
                break;
            default:  // any other combination: every flag tested at run time
                part = epilogue_generic(p, tm, tn, acc, ci, cx, cc, lane, wave);
                break;
        }
    }
    if (flags & (EF_NORM | EF_DOT | EF_MOMENTUM)) {
        const double total = wave_sum(part);
        if (lane == 0) p.partials[(size_t)slot * kWaveSlots + wave] = total;
    }
}

// Small-mode operand slab: 64 rows x 16 k in LDS as 4 groups of 16 rows of
// 64 bytes, each group the 1 KB that one wave-wide 16-byte load to LDS
// writes. Lane L of a load fills row L / 4 of its group; it reads logical
// chunk (L % 4) ^ ((row / 4) % 4) of that row (chunk c holds k = 4c .. 4c+3),
// so chunk c of row r sits at physical chunk c ^ ((r / 4) % 4): sixteen lanes
// reading one chunk of sixteen consecutive rows hit sixteen distinct 16-byte
// bank groups.
constexpr int kSmallSlab = 16;                    // K per slab of a small-mode block
constexpr int kSmallOperand = 64 * kSmallSlab;    // floats per operand slab

// One wave loads a 64 x 16 K-contiguous slab (rows past lim clamped).
__device__ __forceinline__ void small_load(const float* __restrict__ base, int ld, int mn0, int lim, int k0,
                                           float* s) {
    const int lane = threadIdx.x & 63;
#pragma unroll
    for (int j = 0; j < 4; ++j) {
        const int r = j * 16 + (lane >> 2);
        const int row = min(mn0 + r, lim - 1);
        const int chunk = (lane & 3) ^ ((r >> 2) & 3);
        const float* g = base + (size_t)row * ld + k0 + chunk * 4;
        __builtin_amdgcn_global_load_lds((global_void*)g, (lds_void*)(s + j * 256), 16, 0, 0);
    }
}

// Values for k = k .. k+3 (k a multiple of 4 below 16) at row mn of a small-mode slab.
__device__ __forceinline__ void small_fragment(const float* s, int mn, int k, float (&f)[4]) {
    const f32x4 v = *reinterpret_cast<const f32x4*>(s + mn * kSmallSlab + (((k >> 2) ^ ((mn >> 2) & 3)) << 2));
    f[0] = v[0]; f[1] = v[1]; f[2] = v[2]; f[3] = v[3];
}

// The MFMAs of one small-mode slab: lane l contributes k = 4 (l / 16) + s
// to step s, for A and B alike (as in mma_slab). UPPER: a block on the
// diagonal of a symmetric result, whose 16 x 16 blocks below the diagonal are
// left out. BI x BJ: the 16 x 16 blocks of the 64 x 64 block that lie inside
// the product (a product 32 rows or columns wide fills half of it; the
// others are left out rather than computed from padding and discarded).
template <bool UPPER, int BI, int BJ>
__device__ __forceinline__ void small_mma(const float* sa, const float* sb, int lane, f32x4 (&acc)[16]) {
    const int r = lane & 15, g = lane >> 4;
    float a[BI][4], b[BJ][4];
#pragma unroll
    for (int i = 0; i < BI; ++i) small_fragment(sa, i * 16 + r, g * 4, a[i]);
#pragma unroll
    for (int j = 0; j < BJ; ++j) small_fragment(sb, j * 16 + r, g * 4, b[j]);
#pragma unroll
    for (int st = 0; st < 4; ++st)
#pragma unroll
        for (int i = 0; i < BI; ++i)
#pragma unroll
            for (int j = 0; j < BJ; ++j)
                if (!UPPER || i <= j)
                    acc[i * 4 + j] = __builtin_amdgcn_mfma_f32_16x16x4f32(a[i][st], b[j][st], acc[i * 4 + j], 0, 0, 0);
}

// Starts the loads of slab k0 of a small-mode block into stage s (A then B).
__device__ __forceinline__ void small_issue(const GemmProblem& p, int row0, int col0, int k0, float* s) {
    const SlabSrc src = slab_src(p, k0);
    small_load(src.a, src.lda, row0, p.M, src.k, s);
    small_load(src.b, src.ldb, col0, p.N, src.k, s + kSmallOperand);
}

// The K loop of a small-mode block computed by the calling wave alone in its
// own LDS stages s0, s1 (2 x 64 x 16 floats each), with no workgroup barrier:
// slab k + 1 loads while slab k is multiplied. One copy per block shape, so
// the loop has no branches on it.
template <bool UPPER, int BI, int BJ>
__device__ __forceinline__ void small_loop(const GemmProblem& p, int row0, int col0, int nk, float* s0, float* s1,
                                           int lane, f32x4 (&acc)[16]) {
    small_issue(p, row0, col0, 0, s0);
    for (int kt = 0; kt < nk; ++kt) {
        float* cur = (kt & 1) ? s1 : s0;
        float* nxt = (kt & 1) ? s0 : s1;
        // The other stage's slab was read by the previous step's MFMAs; refill it.
        asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
        if (kt + 1 < nk) {
            small_issue(p, row0, col0, (kt + 1) * kSmallSlab, nxt);
            asm volatile("s_waitcnt vmcnt(8)" ::: "memory");  // all but the 8 loads just issued: slab kt
        } else {
            asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
        }
        small_mma<UPPER, BI, BJ>(cur, cur + kSmallOperand, lane, acc);
    }
}

// One small-mode block: its K loop, then the epilogue of the block's
// quadrant, and the zeroing of the partial sums of its tile's quadrants that
// no block computes. The block's shape (on the diagonal of a symmetric
// result or not; 2 or 4 of its 16-row and 16-column strips inside the
// product) is uniform over the wave and picks the loop once.
__device__ __forceinline__ void small_unit(const GemmProblem& p, const SmallUnit& su, float* s0, float* s1,
                                           float beta1, int lane) {
    f32x4 acc[16];
#pragma unroll
    for (int b = 0; b < 16; ++b)
#pragma unroll
        for (int e = 0; e < 4; ++e) acc[b][e] = 0.0f;
    const int row0 = su.bm * kSmallDim, col0 = su.bn * kSmallDim;
    const int nk = p.K / kSmallSlab;
    const bool diag = p.upper && su.bm == su.bn;   // uniform: the block is read with scalar loads
    // Strips inside the product: M and N are multiples of 32.
    const int bi = min(4, (p.M - row0) / 16), bj = min(4, (p.N - col0) / 16);
    if (diag) {
        if (bi == 4 && bj == 4) small_loop<true, 4, 4>(p, row0, col0, nk, s0, s1, lane, acc);
        else if (bi == 4) small_loop<true, 4, 2>(p, row0, col0, nk, s0, s1, lane, acc);
        else if (bj == 4) small_loop<true, 2, 4>(p, row0, col0, nk, s0, s1, lane, acc);
        else small_loop<true, 2, 2>(p, row0, col0, nk, s0, s1, lane, acc);
    } else {
        if (bi == 4 && bj == 4) small_loop<false, 4, 4>(p, row0, col0, nk, s0, s1, lane, acc);
        else if (bi == 4) small_loop<false, 4, 2>(p, row0, col0, nk, s0, s1, lane, acc);
        else if (bj == 4) small_loop<false, 2, 4>(p, row0, col0, nk, s0, s1, lane, acc);
        else small_loop<false, 2, 2>(p, row0, col0, nk, s0, s1, lane, acc);
    }
    const int quadrant = ((su.bm & 1) << 1) | (su.bn & 1);
    gemm_epilogue(p, su.bm >> 1, su.bn >> 1, su.slot, beta1, acc, lane, quadrant);
    if (su.zero_mask && lane == 0) {
#pragma unroll
        for (int q = 0; q < kWaveSlots; ++q)
            if ((su.zero_mask >> q) & 1) p.partials[(size_t)su.slot * kWaveSlots + q] = 0.0;
    }
}

// Grouped launch: one workgroup per work unit of the list. The list is in
// dispatch order: consecutive workgroups go round-robin to the 8 XCDs, and
// the host arranged it so each XCD's share is balanced and reuses operand
// panels in its own L2. Units of split tiles leave their partial product in
// ws for gemm_fixup. A small-mode unit is a group of up to four 64 x 64
// blocks (small), one per wave, each in its own quarter of the LDS.
template <bool AK, bool BK>
__global__ __launch_bounds__(kGemmThreads, 2) void gemm_grouped(const GemmProblem* __restrict__ probs,
                                                                const TileDesc* __restrict__ tiles,
                                                                const SmallUnit* __restrict__ small,
                                                                float beta1, float* __restrict__ ws) {
    __shared__ __attribute__((aligned(16))) GemmStageLds s0;
    __shared__ __attribute__((aligned(16))) GemmStageLds s1;
    const TileDesc td = tiles[blockIdx.x];
    if (td.part == kSmallGroup) {
        if constexpr (BK) {
            const int w = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);  // uniform: its block is read with scalar loads
            if (w < td.tn) {
                const SmallUnit su = small[td.tm + w];
                // Wave w's two stages: half w % 2 of the A and B buffers of s0 or s1.
                GemmStageLds& st = (w >> 1) ? s1 : s0;
                const int half = (w & 1) * (kLdsOperand / 2);
                small_unit(probs[su.prob], su, st.a + half, st.b + half, beta1, threadIdx.x & 63);
            }
        }
        return;
    }
    const GemmProblem p = probs[td.prob];
    f32x4 acc[16];
    gemm_mainloop<AK, BK>(p, td.tm, td.tn, td.k0, td.k1, s0, s1, acc);
    if (td.part >= 0)
        store_partial(ws + (size_t)td.part * kSplitBlock, acc);
    else
        gemm_epilogue(p, td.tm, td.tn, td.slot, beta1, acc, threadIdx.x & 63, threadIdx.x >> 6);
}

// Split tiles of a grouped launch: sums the partial products in K order
// (a fixed order, so results are deterministic) and runs the epilogue. One
// single-wave workgroup per 64 x 64 quadrant of each split tile (workgroup b:
// tile b / 4, quadrant b % 4), so a tile's pieces are read by four
// workgroups in parallel; each takes the accumulators that wave b % 4 of the
// computing workgroups kept.
constexpr int kFixupThreads = 64;
__global__ __launch_bounds__(kFixupThreads) void gemm_fixup(const GemmProblem* __restrict__ probs,
                                                            const FixupDesc* __restrict__ fix, float beta1,
                                                            const float* __restrict__ ws) {
    const FixupDesc fd = fix[blockIdx.x / kWaveSlots];
    const int wave = blockIdx.x % kWaveSlots, lane = threadIdx.x;
    const int t = wave * 64 + lane;  // thread of the computing workgroup
    const GemmProblem p = probs[fd.prob];
    f32x4 acc[16];
#pragma unroll
    for (int b = 0; b < 16; ++b)
#pragma unroll
        for (int e = 0; e < 4; ++e) acc[b][e] = 0.0f;
    // Partials are added in K order; the loads of the next one are in flight
    // while the current one is added (nsplit >= 2).
    const float* blk = ws + (size_t)fd.part0 * kSplitBlock;
    f32x4 v0[16], v1[16];
    load_partial(blk, t, v0);
    int s = 0;
    for (; s + 2 <= fd.nsplit; s += 2) {
        load_partial(blk + (size_t)(s + 1) * kSplitBlock, t, v1);
        add_partial(v0, acc);
        if (s + 2 < fd.nsplit) load_partial(blk + (size_t)(s + 2) * kSplitBlock, t, v0);
        add_partial(v1, acc);
    }
    if (s < fd.nsplit) add_partial(v0, acc);
    gemm_epilogue(p, fd.tm, fd.tn, fd.slot, beta1, acc, lane, wave);
}

}  // namespace jorge
