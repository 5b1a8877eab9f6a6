// Bandwidth-bound and scalar kernels of the Jorge step for gfx950.
#pragma once

#include <hip/hip_runtime.h>

#include "jorge_gemm.hpp"
#include "jorge_types.hpp"

namespace jorge {

constexpr int kEwThreads = 256;

// Fixed-order sum of n doubles by one wave (every lane gets the total).
__device__ __forceinline__ double wave_sum_array(const double* __restrict__ x, int n) {
    double v = 0.0;
    for (int i = threadIdx.x & 63; i < n; i += 64) v += x[i];
    return wave_sum(v);
}

// Zeroes n 16-byte words (a fill kernel rather than a memset, so that the
// clearing is an ordinary kernel node if the caller captures it).
__global__ __launch_bounds__(kEwThreads) void zero_kernel(f32x4* __restrict__ p, size_t n) {
    const f32x4 z = {0.0f, 0.0f, 0.0f, 0.0f};
    for (size_t i = (size_t)blockIdx.x * kEwThreads + threadIdx.x; i < n; i += (size_t)gridDim.x * kEwThreads) p[i] = z;
}

// A_hat = eps^(-1/4) I on the valid diagonal of every factor (the arena is zeroed before).
__global__ void init_factors_kernel(const FactorDev* __restrict__ f, float l0) {
    const FactorDev F = f[blockIdx.x];
    for (int i = threadIdx.x; i < F.d; i += blockDim.x) F.A[(size_t)i * F.dp + i] = l0;
}

// Gradient stage-in over 64 x 64 blocks: copies G (dense m x n, caller's
// buffer) into the padded operand Gp and its transpose Gpt, updates
// m_SGD = beta1 m_SGD + G (Algorithm 3) and writes the block's sum of m_SGD^2.
// Each thread moves groups of four consecutive elements: 16-byte accesses
// where the layer's rows allow them (n a multiple of 4, G 16-byte aligned),
// element by element otherwise. Rows are read and the transpose is written
// in 256-byte runs per 16 threads; the transpose goes through LDS.
__global__ __launch_bounds__(kEwThreads) void stagein_kernel(const LayerDev* __restrict__ layers,
                                                             const StageTile* __restrict__ tiles,
                                                             int layer_base, PtrBatch grads,
                                                             float beta1) {
    __shared__ float blk[64][65];
    __shared__ double red[4];
    const StageTile st = tiles[blockIdx.x];
    const LayerDev& L = layers[st.layer];
    const float* __restrict__ G = grads.p[st.layer - layer_base];
    const int m = L.m, n = L.n;
    const bool vec = (n & 3) == 0 && (reinterpret_cast<uintptr_t>(G) & 15) == 0;
    double part = 0.0;
    // Row r, columns c .. c+3 of the block, for q = 16 r + c / 4.
    if (vec) {
        // Every load of the thread is issued before its first store, so
        // eight 16-byte loads are in flight at once (no store overwrites what
        // a later load of the thread reads, which the compiler cannot prove
        // by itself). The loads are unconditional: a position outside the
        // layer reads the nearest one inside it (n >= 4) and its values are
        // dropped.
        constexpr int kIt = 64 * 16 / kEwThreads;
        float* __restrict__ msgd = L.msgd;
        float* __restrict__ Gp = L.Gp;
        const size_t np = (size_t)L.np;
        f32x4 g[kIt], ms[kIt];
#pragma unroll
        for (int i = 0; i < kIt; ++i) {
            const int q = threadIdx.x + i * kEwThreads;
            const int gr = min(st.r0 + (q >> 4), m - 1), gc = min(st.c0 + (q & 15) * 4, n - 4);
            const size_t gi = (size_t)gr * n + gc;
            g[i] = gload4(G + gi);
            ms[i] = gload4(msgd + gi);
        }
#pragma unroll
        for (int i = 0; i < kIt; ++i) {
            const int q = threadIdx.x + i * kEwThreads, r = q >> 4, c = (q & 15) * 4;
            const int gr = st.r0 + r, gc = st.c0 + c;
#pragma unroll
            for (int j = 0; j < 4; ++j) blk[r][c + j] = g[i][j];
            if (gr >= m || gc >= n) continue;  // gc + 3 < n: n and gc are multiples of 4
            const size_t gi = (size_t)gr * n + gc;
            f32x4 v;
#pragma unroll
            for (int j = 0; j < 4; ++j) v[j] = beta1 * ms[i][j] + g[i][j];
            *(gfloat4*)(Gp + (size_t)gr * np + gc) = g[i];
            *(gfloat4*)(msgd + gi) = v;
#pragma unroll
            for (int j = 0; j < 4; ++j) part += (double)v[j] * (double)v[j];
        }
    } else {
        for (int q = threadIdx.x; q < 64 * 16; q += kEwThreads) {
            const int r = q >> 4, c = (q & 15) * 4, gr = st.r0 + r, gc = st.c0 + c;
            if (gr >= m || gc >= n) continue;
            const size_t gi = (size_t)gr * n + gc;
            f32x4 g;
#pragma unroll
            for (int j = 0; j < 4; ++j) {
                g[j] = 0.0f;
                if (gc + j < n) {
                    g[j] = G[gi + j];
                    L.Gp[(size_t)gr * L.np + gc + j] = g[j];
                    const float w = beta1 * L.msgd[gi + j] + g[j];
                    L.msgd[gi + j] = w;
                    part += (double)w * (double)w;
                }
            }
#pragma unroll
            for (int j = 0; j < 4; ++j) blk[r][c + j] = g[j];
        }
    }
    __syncthreads();
    // Column c, rows r .. r+3 of the block: Gpt[c][r..r+3] (mp is a multiple of 32).
    for (int q = threadIdx.x; q < 64 * 16; q += kEwThreads) {
        const int c = q >> 4, r = (q & 15) * 4, gr = st.r0 + r, gc = st.c0 + c;
        if (gc >= n || gr >= m) continue;
        float* dst = L.Gpt + (size_t)gc * L.mp + gr;
        if (gr + 3 < m) {
            f32x4 t;
#pragma unroll
            for (int j = 0; j < 4; ++j) t[j] = blk[r + j][c];
            *reinterpret_cast<f32x4*>(dst) = t;
        } else {
            for (int j = 0; gr + j < m; ++j) dst[j] = blk[r + j][c];
        }
    }
    const double total = block_sum_256(part, red);
    if (threadIdx.x == 0) L.part_sgd[st.slot] = total;
}

// (beta, c, s) of one factor update from nu = ||X||_F (Algorithm 2; Appendix
// A.1, Eq. 8-9). The dynamic branch forms c = 1/nu and s = (1 + 1/nu)^(1/4)
// directly, never 1 - beta.
__device__ __forceinline__ FactorScalars factor_scalars(double nu, double beta2, int mode) {
    bool dyn = false;
    if (mode == 1) dyn = nu > 0.0;                           // DYNAMIC
    else if (mode == 2) dyn = nu > beta2 / (1.0 - beta2);    // CLAMPED: nu/(nu+1) > beta2
    FactorScalars out;
    if (dyn) {
        out.beta = nu / (nu + 1.0);
        out.c = 1.0 / nu;
        out.s = pow(1.0 + 1.0 / nu, 0.25);
    } else {
        out.beta = beta2;
        out.c = (1.0 - beta2) / beta2;
        out.s = pow(beta2, -0.25);
    }
    out.nu = nu;
    out.a = (float)(0.25 * out.c);
    out.b = (float)(0.15625 * out.c * out.c);
    out.sf = (float)out.s;
    out.e = (float)(0.1171875 * out.c * out.c * out.c);
    return out;
}

// nu = ||X||_F from the per-tile partial sums, then the factor's scalars.
// One wave per factor of the list (the factors of the grouped levels). The factored form's partials are terms of an inner
// product of two positive semidefinite matrices whose exact sum is ||X||_F^2;
// a sum that rounding left below zero is read as zero.
__global__ void factor_finalize_kernel(const FactorDev* __restrict__ f, const int* __restrict__ list,
                                       double beta2, int mode) {
    const FactorDev F = f[list[blockIdx.x]];
    const double nu = sqrt(fmax(0.0, wave_sum_array(F.partials, F.nparts * kWaveSlots)));
    if (threadIdx.x == 0) *F.sc = factor_scalars(nu, beta2, mode);
}

// A_hat <- (Z + Z^T)/2 (or Z when not symmetrizing) for the pair of 64 x 64
// tiles (ti, tj), (tj, ti) of a factor in the explicit form; a diagonal tile
// (ti = tj) is its own partner and is read once. fp32 addition commutes, so
// the result is bitwise symmetric. za, zb: 64 x 65 floats of LDS each. All
// threads of the workgroup call it; it ends with a barrier so the LDS can be
// reused. Global memory is addressed as such (not through generic pointers).
__device__ __forceinline__ void symmetrize_pair(const FactorDev& F, int ti, int tj, int symmetrize,
                                                float (*za)[65], float (*zb)[65]) {
    const int dp = F.dp, i0 = ti * 64, j0 = tj * 64;
    const int tid = threadIdx.x;
    const bool diag = ti == tj;
    float (*const pb)[65] = diag ? za : zb;  // the partner tile's LDS copy
    // 64 rows x 16 float4 per tile, 4 per thread; every load before the first LDS store.
    f32x4 va[4], vb[4];
#pragma unroll
    for (int q = 0; q < 4; ++q) {
        const int u = tid + q * kEwThreads, r = u >> 4, c = (u & 15) * 4;
        if (i0 + r < dp && j0 + c < dp) va[q] = gload4(F.Z + (size_t)(i0 + r) * dp + j0 + c);
        if (!diag && j0 + r < dp && i0 + c < dp) vb[q] = gload4(F.Z + (size_t)(j0 + r) * dp + i0 + c);
    }
#pragma unroll
    for (int q = 0; q < 4; ++q) {
        const int u = tid + q * kEwThreads, r = u >> 4, c = (u & 15) * 4;
        if (i0 + r < dp && j0 + c < dp) {
            za[r][c] = va[q][0]; za[r][c + 1] = va[q][1]; za[r][c + 2] = va[q][2]; za[r][c + 3] = va[q][3];
        }
        if (!diag && j0 + r < dp && i0 + c < dp) {
            zb[r][c] = vb[q][0]; zb[r][c + 1] = vb[q][1]; zb[r][c + 2] = vb[q][2]; zb[r][c + 3] = vb[q][3];
        }
    }
    __syncthreads();
#pragma unroll
    for (int q = 0; q < 4; ++q) {
        const int u = tid + q * kEwThreads, r = u >> 4, c = (u & 15) * 4;
        if (i0 + r < dp && j0 + c < dp) {
            f32x4 v;
#pragma unroll
            for (int e = 0; e < 4; ++e)
                v[e] = symmetrize ? 0.5f * (za[r][c + e] + pb[c + e][r]) : za[r][c + e];
            *(gfloat4*)(F.A + (size_t)(i0 + r) * dp + j0 + c) = v;
        }
        if (!diag && j0 + r < dp && i0 + c < dp) {
            f32x4 v;
#pragma unroll
            for (int e = 0; e < 4; ++e)
                v[e] = symmetrize ? 0.5f * (zb[r][c + e] + za[c + e][r]) : zb[r][c + e];
            *(gfloat4*)(F.A + (size_t)(j0 + r) * dp + i0 + c) = v;
        }
    }
    __syncthreads();
}

__global__ __launch_bounds__(kEwThreads) void symmetrize_kernel(const FactorDev* __restrict__ f,
                                                                const SymTile* __restrict__ tiles,
                                                                int symmetrize) {
    __shared__ float za[64][65];
    __shared__ float zb[64][65];
    const SymTile st = tiles[blockIdx.x];
    symmetrize_pair(f[st.factor], st.ti, st.tj, symmetrize, za, zb);
}

// ---------------------------------------------------------------- LDS chain
// The whole update of a small factor (padded size dp <= 64) by one
// workgroup, in the explicit order of Algorithm 2 with every matrix resident
// in LDS: M = H H^T (H streamed from global memory in 32-column slabs),
// A^2, A^4, X = A^4 M with ||X||_F, (beta, c, s) (Appendix A.1, Eq. 8-9),
// P = I - (c/4) X + (5c^2/32) X X (Eq. 6), Z = s A P and A <- (Z + Z^T)/2
// (or Z). With series order 3, P = I - a X + X V with V = b X - e X X keeps
// the cubic term of Eq. 5. One launch replaces the grouped levels for these
// factors.
// Each of the four waves owns one 32 x 32 block of a 64 x 64 product
// (v_mfma_f32_32x32x2_f32); blocks outside dp are skipped.
constexpr int kChainMax = 64;
constexpr int kChainLd = kChainMax + 1;          // LDS row stride: column reads hit 32 distinct banks
constexpr int kChainMat = kChainMax * kChainLd;  // floats per LDS matrix
constexpr int kChainSlabLd = kSlab + 1;

struct ChainLds {
    float A[kChainMat];
    float M[kChainMat];
    float T1[kChainMat];
    float T2[kChainMat];
    float H[kChainMax * kChainSlabLd];
    double red[4];
    float coef[4];  // a, b, s, e
};

// acc += A (rows wy*32.., lda) x B (cols wx*32.., ldb) over k in [0, K): both
// operands in LDS; BT reads B transposed (B[k][col] = Bm[col][k]).
// K is a multiple of 32; each group of 16 k has all its LDS reads issued
// before its 8 MFMAs.
template <bool BT>
__device__ __forceinline__ void chain_mma(const float* a, int lda, const float* b, int ldb, int K, int wy, int wx,
                                          f32x16& acc) {
    const int lane = threadIdx.x & 63, r = lane & 31, h = lane >> 5;
    for (int t0 = 0; t0 < K; t0 += 16) {
        float av[8], bv[8];
#pragma unroll
        for (int u = 0; u < 8; ++u) {
            const int t = t0 + 2 * u + h;
            av[u] = a[(wy * 32 + r) * lda + t];
            bv[u] = BT ? b[(wx * 32 + r) * ldb + t] : b[t * ldb + wx * 32 + r];
        }
#pragma unroll
        for (int u = 0; u < 8; ++u) acc = __builtin_amdgcn_mfma_f32_32x32x2f32(av[u], bv[u], acc, 0, 0, 0);
    }
}

// C (LDS) = the wave's accumulator block; f(row, col, value) gives the stored value.
template <typename Fn>
__device__ __forceinline__ void chain_store(float* c, int wy, int wx, const f32x16& acc, Fn f) {
    const int lane = threadIdx.x & 63, h = lane >> 5;
    const int col = wx * 32 + (lane & 31);
#pragma unroll
    for (int e = 0; e < 16; ++e) {
        const int row = wy * 32 + 8 * (e >> 2) + 4 * h + (e & 3);
        c[row * kChainLd + col] = f(row, col, acc[e]);
    }
}

__global__ __launch_bounds__(kGemmThreads) void lds_chain_kernel(const FactorDev* __restrict__ f,
                                                                 const int* __restrict__ list, double beta2,
                                                                 int mode, int symmetrize, int order) {
    __shared__ __attribute__((aligned(16))) ChainLds sm;
    const FactorDev F = f[list[blockIdx.x]];
    const int dp = F.dp, tid = threadIdx.x;
    const int wave = tid >> 6, wy = wave >> 1, wx = wave & 1;
    const bool active = wy * 32 < dp && wx * 32 < dp;  // this wave's block lies inside dp x dp
    auto zero = [](f32x16& a) {
#pragma unroll
        for (int e = 0; e < 16; ++e) a[e] = 0.0f;
    };

    for (int e = tid; e < dp * dp; e += kGemmThreads) sm.A[(e / dp) * kChainLd + e % dp] = F.A[e];

    // M = H H^T, H streamed in slabs of 32 columns: each thread holds its
    // (up to) 8 floats of the next slab in registers while the current one is
    // multiplied. Thread t covers rows t/8 and 32 + t/8, columns 4 (t%8) .. +3.
    f32x16 acc;
    zero(acc);
    const int hr = tid >> 3, hc = (tid & 7) * 4;
    f32x4 hv[2];
    auto load_h = [&](int k0) {
#pragma unroll
        for (int q = 0; q < 2; ++q) {
            const int r = hr + 32 * q;
            if (r < dp) hv[q] = *(const f32x4*)(F.H + (size_t)r * F.kp + k0 + hc);
        }
    };
    load_h(0);
    for (int k0 = 0; k0 < F.kp; k0 += kSlab) {
        __syncthreads();  // the previous slab's products are done with sm.H
#pragma unroll
        for (int q = 0; q < 2; ++q) {
            const int r = hr + 32 * q;
            if (r < dp) {
#pragma unroll
                for (int e = 0; e < 4; ++e) sm.H[r * kChainSlabLd + hc + e] = hv[q][e];
            }
        }
        __syncthreads();
        if (k0 + kSlab < F.kp) load_h(k0 + kSlab);
        if (active) chain_mma<true>(sm.H, kChainSlabLd, sm.H, kChainSlabLd, kSlab, wy, wx, acc);
    }
    if (active) chain_store(sm.M, wy, wx, acc, [](int, int, float v) { return v; });
    __syncthreads();
    // A^2 -> T1, A^4 -> T2
    zero(acc);
    if (active) {
        chain_mma<false>(sm.A, kChainLd, sm.A, kChainLd, dp, wy, wx, acc);
        chain_store(sm.T1, wy, wx, acc, [](int, int, float v) { return v; });
    }
    __syncthreads();
    zero(acc);
    if (active) {
        chain_mma<false>(sm.T1, kChainLd, sm.T1, kChainLd, dp, wy, wx, acc);
        chain_store(sm.T2, wy, wx, acc, [](int, int, float v) { return v; });
    }
    __syncthreads();
    // X = A^4 M -> T1, with ||X||_F^2
    zero(acc);
    double part = 0.0;
    if (active) {
        chain_mma<false>(sm.T2, kChainLd, sm.M, kChainLd, dp, wy, wx, acc);
        chain_store(sm.T1, wy, wx, acc, [&](int, int, float v) {
            part += (double)v * (double)v;
            return v;
        });
    }
    const double nu2 = block_sum_256(part, sm.red);
    if (tid == 0) {
        const FactorScalars fs = factor_scalars(sqrt(nu2), beta2, mode);
        *F.sc = fs;
        sm.coef[0] = fs.a;
        sm.coef[1] = fs.b;
        sm.coef[2] = fs.sf;
        sm.coef[3] = fs.e;
    }
    __syncthreads();
    const float a = sm.coef[0], b = sm.coef[1], sf = sm.coef[2], ce = sm.coef[3];
    const int d = F.d;
    // P (the matrix the product with A reads) and Z, in buffers free at that point.
    float* P = sm.T2;
    float* Z = sm.M;
    if (order == 3) {
        // V = b X - e X X -> T2, then P = I - a X + X V -> M
        zero(acc);
        if (active) {
            chain_mma<false>(sm.T1, kChainLd, sm.T1, kChainLd, dp, wy, wx, acc);
            chain_store(sm.T2, wy, wx, acc,
                        [&](int row, int col, float v) { return b * sm.T1[row * kChainLd + col] - ce * v; });
        }
        __syncthreads();
        zero(acc);
        if (active) {
            chain_mma<false>(sm.T1, kChainLd, sm.T2, kChainLd, dp, wy, wx, acc);
            chain_store(sm.M, wy, wx, acc, [&](int row, int col, float v) {
                const float id = (row == col && row < d) ? 1.0f : 0.0f;
                return (id - a * sm.T1[row * kChainLd + col]) + v;
            });
        }
        P = sm.M;
        Z = sm.T1;
    } else {
        // P = I - a X + b X X -> T2
        zero(acc);
        if (active) {
            chain_mma<false>(sm.T1, kChainLd, sm.T1, kChainLd, dp, wy, wx, acc);
            chain_store(sm.T2, wy, wx, acc, [&](int row, int col, float v) {
                const float id = (row == col && row < d) ? 1.0f : 0.0f;
                return (id - a * sm.T1[row * kChainLd + col]) + b * v;
            });
        }
    }
    __syncthreads();
    // Z = s A P
    zero(acc);
    if (active) {
        chain_mma<false>(sm.A, kChainLd, P, kChainLd, dp, wy, wx, acc);
        chain_store(Z, wy, wx, acc, [&](int, int, float v) { return sf * v; });
    }
    __syncthreads();
    // A <- (Z + Z^T)/2 or Z; fp32 addition commutes, so the result is bitwise symmetric.
    for (int e = tid; e < dp * dp; e += kGemmThreads) {
        const int r = e / dp, c = e % dp;
        const float z = Z[r * kChainLd + c];
        F.A[e] = symmetrize ? 0.5f * (z + Z[c * kChainLd + r]) : z;
    }
}

// ---------------------------------------------------------------- LDS chain, sizes 96 and 128
// The same whole-factor update (explicit order of Algorithm 2, symmetric
// factors) for padded sizes 64 < dp <= 128, by one workgroup of eight waves
// (two per SIMD, so one wave's MFMAs run while the other waits at a barrier
// or for memory). Two dp x dp matrices stay in LDS and A is read from global
// memory when a product needs it: M = H H^T (H streamed in 32-column slabs,
// the next slab held in registers while the current one is multiplied), A^2,
// A^4, X = A^4 M with ||X||_F, (beta, c, s) (Appendix A.1, Eq. 8-9),
// P = I - (c/4) X + (5c^2/32) X X (Eq. 6; with series order 3,
// P = I - a X + X V, V = b X - e X X), Z = s A P and A <- (Z + Z^T)/2.
// Every product is C = A B with both operands held as rows that are
// contiguous in k: A's rows, and B's columns, i.e. the rows of B^T. The
// symmetric operands (A, A^2, A^4, M) are their own transposes; X is stored
// beside X^T, and P and V only transposed.
// Wave w owns the 64 x 32 piece at rows 64 (w / 4), columns 32 (w % 4) of
// the product, as 4 x 2 blocks of v_mfma_f32_16x16x4_f32; lane l reads 16
// bytes of its row for k = k0 + 4 (l / 16) .. + 3 and feeds them to the four
// steps of a 16-deep k group (A and B alike, so every A[i][k] B[k][j] is
// formed once). Blocks outside dp are skipped.
constexpr int kChain2Max = 128;
constexpr int kC2Threads = 512;          // eight waves
constexpr int kC2Waves = kC2Threads / 64;
constexpr int kC2PieceCols = 32;         // a wave's piece: 64 rows x 32 columns
constexpr int kC2Ld = kChain2Max + 4;    // LDS row stride: 16-byte reads of 16 rows fall in distinct bank quads
constexpr int kC2Mat = kChain2Max * kC2Ld;
constexpr int kC2HLd = kSlab + 4;        // H slab row stride

struct Chain2Lds {
    float m0[kC2Mat];
    float m1[kC2Mat];
    float h[kChain2Max * kC2HLd];
    double red[kC2Waves];
    float coef[4];  // a, b, s, e
};

// Fragments of one 16-deep k group: lane l's 16 bytes of rows 16 i + l % 16
// of its piece (A) and of its columns (B), at k = k0 + 4 (l / 16) .. + 3.
template <int NBI, int NBJ>
__device__ __forceinline__ void c2_frags(const float* pa, int lda, const float* pb, int ldb, int k0, f32x4 (&fa)[NBI],
                                         f32x4 (&fb)[NBJ]) {
#pragma unroll
    for (int i = 0; i < NBI; ++i) fa[i] = *reinterpret_cast<const f32x4*>(pa + 16 * i * lda + k0);
#pragma unroll
    for (int j = 0; j < NBJ; ++j) fb[j] = *reinterpret_cast<const f32x4*>(pb + 16 * j * ldb + k0);
}

template <int NBI, int NBJ>
__device__ __forceinline__ void c2_group(const f32x4 (&fa)[NBI], const f32x4 (&fb)[NBJ], f32x4 (&acc)[8]) {
#pragma unroll
    for (int st = 0; st < 4; ++st)
#pragma unroll
        for (int i = 0; i < NBI; ++i)
#pragma unroll
            for (int j = 0; j < NBJ; ++j)
                acc[i * 2 + j] = __builtin_amdgcn_mfma_f32_16x16x4f32(fa[i][st], fb[j][st], acc[i * 2 + j], 0, 0, 0);
}

// acc += a (rows, stride lda) x b^T (rows, stride ldb) over k in [0, K) (K a
// multiple of 32) for the NBI x NBJ blocks of the calling wave's piece that
// lie inside the product. The next group's fragments are read while the
// current group's MFMAs run.
template <int NBI, int NBJ>
__device__ __forceinline__ void c2_mma_t(const float* a, int lda, const float* b, int ldb, int K, int wy, int wx,
                                         f32x4 (&acc)[8]) {
    const int lane = threadIdx.x & 63, r = lane & 15, q = lane >> 4;
    const float* pa = a + (wy * 64 + r) * lda + 4 * q;
    const float* pb = b + (wx * kC2PieceCols + r) * ldb + 4 * q;
    f32x4 fa0[NBI], fb0[NBJ], fa1[NBI], fb1[NBJ];
    c2_frags<NBI, NBJ>(pa, lda, pb, ldb, 0, fa0, fb0);
    for (int k0 = 0; k0 < K; k0 += 32) {
        c2_frags<NBI, NBJ>(pa, lda, pb, ldb, k0 + 16, fa1, fb1);
        __builtin_amdgcn_sched_barrier(0);
        c2_group<NBI, NBJ>(fa0, fb0, acc);
        // past the last group the read repeats group 0 (never multiplied): no branch in the loop
        c2_frags<NBI, NBJ>(pa, lda, pb, ldb, k0 + 32 < K ? k0 + 32 : 0, fa0, fb0);
        __builtin_amdgcn_sched_barrier(0);
        c2_group<NBI, NBJ>(fa1, fb1, acc);
    }
}

// The wave's part of a product: nbi (2 or 4) x 2 of its 4 x 2 blocks lie
// inside it (uniform per wave); a wave with none returns.
__device__ __forceinline__ void c2_mma(const float* a, int lda, const float* b, int ldb, int K, int wy, int wx,
                                       int nbi, f32x4 (&acc)[8]) {
    if (nbi == 4) c2_mma_t<4, 2>(a, lda, b, ldb, K, wy, wx, acc);
    else if (nbi == 2) c2_mma_t<2, 2>(a, lda, b, ldb, K, wy, wx, acc);
}

__device__ __forceinline__ void c2_zero(f32x4 (&acc)[8]) {
#pragma unroll
    for (int b = 0; b < 8; ++b) acc[b] = f32x4{0.0f, 0.0f, 0.0f, 0.0f};
}

// The wave's blocks to LDS: m[row][col] = f(row, col, value), row-major
// (stride kC2Ld); with T, m[col][row] instead (four consecutive rows of a
// column are one 16-byte store).
template <bool T, typename Fn>
__device__ __forceinline__ void c2_store(float* m, int wy, int wx, int nbi, const f32x4 (&acc)[8], Fn f) {
    const int lane = threadIdx.x & 63;
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 2; ++j) {
            if (i >= nbi) continue;
            const int row = wy * 64 + 16 * i + 4 * (lane >> 4), col = wx * kC2PieceCols + 16 * j + (lane & 15);
            f32x4 v;
#pragma unroll
            for (int e = 0; e < 4; ++e) v[e] = f(row + e, col, acc[i * 2 + j][e]);
            if constexpr (T) {
                *reinterpret_cast<f32x4*>(m + col * kC2Ld + row) = v;
            } else {
#pragma unroll
                for (int e = 0; e < 4; ++e) m[(row + e) * kC2Ld + col] = v[e];
            }
        }
}

// A (dp x dp, global, row stride dp) into LDS rows of stride kC2Ld.
__device__ __forceinline__ void c2_load_a(float* m, const float* __restrict__ A, int dp) {
    const int nv = dp * dp / 4;
    for (int v = threadIdx.x; v < nv; v += kC2Threads) {
        const int e = 4 * v, r = e / dp, c = e - r * dp;
        *reinterpret_cast<f32x4*>(m + r * kC2Ld + c) = gload4(A + e);
    }
}

// Sum of one double per thread over the workgroup's eight waves, in a fixed order.
__device__ __forceinline__ double c2_block_sum(double v, double* red) {
    v = wave_sum(v);
    if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = v;
    __syncthreads();
    return ((red[0] + red[1]) + (red[2] + red[3])) + ((red[4] + red[5]) + (red[6] + red[7]));
}

__global__ __launch_bounds__(kC2Threads) void lds_chain128_kernel(const FactorDev* __restrict__ f,
                                                                  const int* __restrict__ list, double beta2,
                                                                  int mode, int order) {
    static_assert(kC2Waves == 8, "the block sum and the piece layout assume eight waves");
    __shared__ __attribute__((aligned(16))) Chain2Lds sm;
    const FactorDev F = f[list[blockIdx.x]];
    const int dp = F.dp, d = F.d, tid = threadIdx.x;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6), wy = wave >> 2, wx = wave & 3;
    // 16-row blocks of this wave's piece inside dp (dp is 96 or 128: 2 or 4);
    // its two 16-column blocks are inside dp or outside it together.
    const int nbi = min(4, (dp - wy * 64) / 16);
    const bool active = nbi > 0 && wx * kC2PieceCols < dp;
    f32x4 acc[8];

    // M = H H^T, H (dp x kp, row stride kp) in 32-column slabs; thread t
    // moves two 16-byte pieces of each slab: row (t + 512 p) / 8, columns
    // 4 ((t + 512 p) % 8) .. + 3.
    c2_zero(acc);
    f32x4 hv[2];
    auto load_h = [&](int k0) {
#pragma unroll
        for (int p = 0; p < 2; ++p) {
            const int u = tid + kC2Threads * p, r = u >> 3;
            if (r < dp) hv[p] = gload4(F.H + (size_t)r * F.kp + k0 + 4 * (u & 7));
        }
    };
    load_h(0);
    for (int k0 = 0; k0 < F.kp; k0 += kSlab) {
        __syncthreads();  // every wave is done with the previous slab
#pragma unroll
        for (int p = 0; p < 2; ++p) {
            const int u = tid + kC2Threads * p, r = u >> 3;
            if (r < dp) *reinterpret_cast<f32x4*>(sm.h + r * kC2HLd + 4 * (u & 7)) = hv[p];
        }
        __syncthreads();
        if (k0 + kSlab < F.kp) load_h(k0 + kSlab);
        if (active) c2_mma(sm.h, kC2HLd, sm.h, kC2HLd, kSlab, wy, wx, nbi, acc);
    }
    if (active) c2_store<false>(sm.m0, wy, wx, nbi, acc, [](int, int, float v) { return v; });
    c2_load_a(sm.m1, F.A, dp);
    __syncthreads();
    // A^2 and A^4, each over the last in m1
    for (int pw = 0; pw < 2; ++pw) {
        c2_zero(acc);
        if (active) c2_mma(sm.m1, kC2Ld, sm.m1, kC2Ld, dp, wy, wx, nbi, acc);
        __syncthreads();
        if (active) c2_store<false>(sm.m1, wy, wx, nbi, acc, [](int, int, float v) { return v; });
        __syncthreads();
    }
    // X = A^4 M (M symmetric: its rows are its columns) with ||X||_F^2; X to
    // m0, X^T to m1.
    c2_zero(acc);
    double part = 0.0;
    if (active) {
        c2_mma(sm.m1, kC2Ld, sm.m0, kC2Ld, dp, wy, wx, nbi, acc);
#pragma unroll
        for (int b = 0; b < 8; ++b)
#pragma unroll
            for (int e = 0; e < 4; ++e) part += (double)acc[b][e] * (double)acc[b][e];
    }
    const double nu2 = c2_block_sum(part, sm.red);  // (its barrier also ends the reads of m0 and m1)
    if (active) {
        c2_store<false>(sm.m0, wy, wx, nbi, acc, [](int, int, float v) { return v; });
        c2_store<true>(sm.m1, wy, wx, nbi, acc, [](int, int, float v) { return v; });
    }
    if (tid == 0) {
        const FactorScalars fs = factor_scalars(sqrt(nu2), beta2, mode);
        *F.sc = fs;
        sm.coef[0] = fs.a;
        sm.coef[1] = fs.b;
        sm.coef[2] = fs.sf;
        sm.coef[3] = fs.e;
    }
    __syncthreads();
    const float a = sm.coef[0], b = sm.coef[1], sf = sm.coef[2], ce = sm.coef[3];
    const float* X = sm.m0;
    // X X (B = X, whose rows-in-k are the rows of X^T in m1)
    c2_zero(acc);
    if (active) c2_mma(sm.m0, kC2Ld, sm.m1, kC2Ld, dp, wy, wx, nbi, acc);
    __syncthreads();
    if (order == 3) {
        // V = b X - e X X, stored transposed over X^T; then X V
        if (active)
            c2_store<true>(sm.m1, wy, wx, nbi, acc,
                           [&](int row, int col, float v) { return b * X[row * kC2Ld + col] - ce * v; });
        __syncthreads();
        c2_zero(acc);
        if (active) c2_mma(sm.m0, kC2Ld, sm.m1, kC2Ld, dp, wy, wx, nbi, acc);
        __syncthreads();
        // P = I - a X + X V, stored transposed
        if (active)
            c2_store<true>(sm.m1, wy, wx, nbi, acc, [&](int row, int col, float v) {
                const float id = (row == col && row < d) ? 1.0f : 0.0f;
                return (id - a * X[row * kC2Ld + col]) + v;
            });
    } else {
        // P = I - a X + b X X, stored transposed
        if (active)
            c2_store<true>(sm.m1, wy, wx, nbi, acc, [&](int row, int col, float v) {
                const float id = (row == col && row < d) ? 1.0f : 0.0f;
                return (id - a * X[row * kC2Ld + col]) + b * v;
            });
    }
    __syncthreads();  // every read of X is done: A can replace it
    c2_load_a(sm.m0, F.A, dp);
    __syncthreads();
    // Z = s A P (B = P: its rows-in-k are the rows of P^T in m1)
    c2_zero(acc);
    if (active) c2_mma(sm.m0, kC2Ld, sm.m1, kC2Ld, dp, wy, wx, nbi, acc);
    __syncthreads();
    if (active) c2_store<false>(sm.m0, wy, wx, nbi, acc, [&](int, int, float v) { return sf * v; });
    __syncthreads();
    // A <- (Z + Z^T)/2: fp32 addition commutes, so the result is bitwise symmetric.
    const int nv = dp * dp / 4;
    for (int v = tid; v < nv; v += kC2Threads) {
        const int e = 4 * v, r = e / dp, c = e - r * dp;
        f32x4 o;
#pragma unroll
        for (int q = 0; q < 4; ++q) o[q] = 0.5f * (sm.m0[r * kC2Ld + c + q] + sm.m0[(c + q) * kC2Ld + r]);
        *(gfloat4*)(F.A + e) = o;
    }
}

// Per-layer norms of m and m_SGD from their partial sums, and the grafted
// step g (Algorithm 3) with the decoupled decay rate lr * wd (Section 4). One
// wave per layer.
__global__ void layer_finalize_kernel(const LayerDev* __restrict__ layers, double lr, double wd,
                                      int graft) {
    const LayerDev L = layers[blockIdx.x];
    const double nm = sqrt(wave_sum_array(L.part_m, L.n_part_m * kWaveSlots));
    const double ns = sqrt(wave_sum_array(L.part_sgd, L.n_part_sgd));
    if (threadIdx.x != 0) return;
    // A NaN or infinity anywhere in this step's G reaches m_SGD = beta1 m_SGD + G,
    // and with it this norm: the layer's flag records it for the host.
    if (!isfinite(ns)) *L.nonfinite = 1;
    double g = lr;
    if (graft) g = nm > 0.0 ? lr * ns / nm : 0.0;
    LayerScalars out;
    out.norm_m = nm;
    out.norm_sgd = ns;
    out.g = g;
    out.gf = (float)g;
    out.lw = (float)(lr * wd);
    *L.ls = out;
}

// theta <- theta (1 - lr wd) - g m over a flat chunk of one layer, evaluated as
// theta - (lr wd theta + g m): the small correction is formed first, so the
// stored parameter is rounded once (1 - lr wd in fp32 would itself be off by up
// to 2^-25, a systematic error of that size on every parameter).
__global__ __launch_bounds__(kEwThreads) void weight_kernel(const LayerDev* __restrict__ layers,
                                                            const FlatChunk* __restrict__ chunks,
                                                            int layer_base, MutPtrBatch params) {
    const FlatChunk ck = chunks[blockIdx.x];
    const LayerDev& L = layers[ck.layer];
    float* __restrict__ th = params.p[ck.layer - layer_base];
    const float g = L.ls->gf, lw = L.ls->lw;
    const float* __restrict__ m = L.mom;
    if ((ck.count & 3) == 0 && (reinterpret_cast<uintptr_t>(th) & 15) == 0) {
        const int n4 = ck.count >> 2;
        // Global (not generic) accesses, four per array per thread in flight:
        // each group of four iterations issues its loads before its stores,
        // then the remainder goes one by one.
        gfloat4* t4 = (gfloat4*)(th + ck.start);
        const global_f32x4* m4 = (const global_f32x4*)(m + ck.start);
        int e = threadIdx.x;
        for (; e + 3 * kEwThreads < n4; e += 4 * kEwThreads) {
            f32x4 t[4], mv[4];
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                t[i] = t4[e + i * kEwThreads];
                mv[i] = m4[e + i * kEwThreads];
            }
#pragma unroll
            for (int i = 0; i < 4; ++i) {
#pragma unroll
                for (int q = 0; q < 4; ++q) t[i][q] = t[i][q] - (lw * t[i][q] + g * mv[i][q]);
                t4[e + i * kEwThreads] = t[i];
            }
        }
        for (; e < n4; e += kEwThreads) {
            f32x4 t = t4[e];
            const f32x4 mv = m4[e];
#pragma unroll
            for (int q = 0; q < 4; ++q) t[q] = t[q] - (lw * t[q] + g * mv[q]);
            t4[e] = t;
        }
    } else {
        for (int e = threadIdx.x; e < ck.count; e += kEwThreads) {
            const int i = ck.start + e;
            th[i] = th[i] - (lw * th[i] + g * m[i]);
        }
    }
}

}  // namespace jorge
