// Plain structs shared by the host runtime and the gfx950 kernels.
#pragma once

#include <stdint.h>

namespace jorge {

// What the epilogue of a grouped GEMM does with one tile of the product
// (bit flags, combined per problem).
enum EpiFlags : int {
    EF_STORE = 1,      // write the value to C (row-major)
    EF_STORE_T = 2,    // write the value transposed to C2 (C2[col][row])
    EF_NORM = 4,       // add the tile's sum of value^2 to the partial-sum slot
    EF_DOT = 8,        // add the tile's sum of acc * X[row][col] (weighted for symmetric halves)
    EF_MOMENTUM = 16,  // m = beta1 m + (1 - beta1) acc on the dense momentum, plus sum of m^2
    EF_READX = 32,     // the value reads X[row][col] (coefficient cx below)
};

// Coefficient sets: value = ci [row == col < valid_m] + cx X[row][col] + cc acc,
// with (a, b, e, s) = (c/4, 5c^2/32, 15c^3/128, beta^(-1/4)) of the factor
// being updated (e: the cubic term of Eq. 5, kept only with series order 3).
enum Coef : int {
    CO_ONE = 0,     // (0, 0, 1)          plain product
    CO_POLY = 1,    // (1, -a, b)         P = I - (c/4) X + (5c^2/32) X X      (Eq. 6)
    CO_SCALE = 2,   // (0, 0, s)          Z = s A P
    CO_WMIX = 3,    // (0, a, -b)         W = A^5 H (a I - b S)
    CO_SYR2K = 4,   // (0, s, -s/2)       A <- s A - (s/2) (W H^T + H W^T)
    CO_LITUPD = 5,  // (0, s, -s)         A <- s A - s W H^T
    CO_VSER = 6,    // (0, b, -e)         V = b X - e X X        (series order 3)
    CO_POLY3 = 7,   // (1, -a, 1)         P = I - a X + X V  = I - a X + b X^2 - e X^3
    CO_WMIX3 = 8,   // (0, a, -1)         W = a A^5 H - A^5 H V(S) = A^5 H (a I - b S + e S^2)
};

// Scalars of one factor update, written on the device by the finalize kernel.
struct FactorScalars {
    double nu;    // ||X||_F
    double beta;  // beta used for this update
    double c;     // (1 - beta) / beta
    double s;     // beta^(-1/4)
    float a;      // c / 4            (fp32 copy for the epilogue)
    float b;      // 5 c^2 / 32
    float sf;     // s
    float e;      // 15 c^3 / 128
};

// Scalars of one layer's weight update, written by the layer finalize kernel.
struct LayerScalars {
    double norm_m;    // ||m_t||_F
    double norm_sgd;  // ||m_SGD,t||_F
    double g;         // step applied to m_t
    float gf;         // g as fp32
    float lw;         // lr * weight_decay as fp32 (theta <- theta - (lw theta + g m))
};

// One product of a grouped launch. With both operands K-major (the "NT"
// kernel) the product is C = A B^T: A is M x K row-major, B is N x K
// row-major. With B MN-major (the "NN" kernel) B is K x N row-major.
// K may consist of two segments: slabs with k >= K1 read A2 and B2 (at
// k - K1) instead of A and B, which forms sums such as W H^T + H W^T in one
// accumulation. M, N, K, K1 are padded extents (K and K1 multiples of 32,
// leading dimensions multiples of 4).
struct GemmProblem {
    const float* A;
    const float* B;
    const float* A2;
    const float* B2;
    float* C;
    float* C2;                 // EF_STORE_T destination
    const float* X;            // EF_READX / EF_DOT operand
    const FactorScalars* sc;   // coefficients (any Coef but CO_ONE)
    float* mom;                // EF_MOMENTUM: dense valid_m x valid_n momentum
    double* partials;          // EF_NORM, EF_DOT, EF_MOMENTUM: kWaveSlots doubles per tile slot
    int M, N, K, K1;
    int lda, ldb, lda2, ldb2;
    int ldc, ldc2, ldx, ldmom;
    int valid_m, valid_n;      // unpadded extent (identity / momentum masks)
    int flags;                 // EpiFlags
    int coef;                  // Coef
    int upper;                 // 1: symmetric result, only tiles tm <= tn are computed
                               //    and each is written with its mirror image
    int pad0;
};

// One work unit of a grouped launch: tile (tm, tn) of a problem over the K
// range [k0, k1). A unit of a split tile (part >= 0) writes its partial
// product to block `part` of the launch's split workspace instead of running
// the epilogue; a fixup unit then sums the parts and runs it.
struct TileDesc {
    int prob;  // index into the launch's problem table
    int tm;    // tile row
    int tn;    // tile column
    int slot;  // partial-sum slot within the problem
    int k0;    // K range (multiples of 32)
    int k1;
    int part;  // split workspace block, -1 for a whole tile, kSmallGroup for small-mode blocks
    int pad0;
};

// Small mode: a product with at most 64 rows or columns and a short K is
// computed in 64 x 64 blocks, one wave per block, up to four blocks per
// workgroup. Block (bm, bn) is quadrant ((bm & 1), (bn & 1)) of 128 x 128 tile
// (bm / 2, bn / 2), with that tile's partial-sum slot; zero_mask lists the
// quadrants of the tile that no block computes (outside the product, or below
// the diagonal of a symmetric result), whose partial sums this block sets to 0.
struct SmallUnit {
    int prob;
    int bm;
    int bn;
    int slot;
    int zero_mask;
    int pad0, pad1, pad2;
};
constexpr int kSmallDim = 64;     // rows or columns at most
constexpr int kSmallMaxK = 256;   // K at most
// TileDesc.part of a small-mode workgroup: tm = its first SmallUnit, tn = their
// number (1 to 4), [k0, k1) = [0, the longest K among them).
constexpr int kSmallGroup = -2;

// A split tile of a grouped launch: its nsplit partial products sit in
// workspace blocks part0 .. part0 + nsplit - 1, in K order.
struct FixupDesc {
    int prob;
    int tm;
    int tn;
    int slot;
    int part0;
    int nsplit;
    int pad0, pad1;
};

// Floats per split-workspace block: one 128 x 128 tile.
constexpr int kSplitBlock = 128 * 128;
// Partial sums of a GEMM tile's epilogue (norms, dot products): one double
// per 64 x 64 quadrant, each written by the wave that owns it; consumers sum
// all kWaveSlots * (tile slots) of them in index order.
constexpr int kWaveSlots = 4;

// Device view of a factor (L_hat or R_hat of one layer).
struct FactorDev {
    float* A;              // state, dp x dp, ld = dp, zero outside the d x d block
    FactorScalars* sc;
    double* partials;      // partial sums of ||X||_F^2: kWaveSlots per tile slot
    float* Z;              // explicit form: the unsymmetrized product s A P (dp x dp)
    const float* H;        // the statistic's factor, row-major d x k (ld kp, zero padded)
    int d, dp;
    int k, kp;
    int nparts;
    int explicit_form;     // 1: explicit powers; 0: factored through the statistic's factor
};

// Device view of a layer.
struct LayerDev {
    float* Gp;             // padded copy of G, mp x np, ld = np, zero padding
    float* Gpt;            // its transpose, np x mp, ld = mp
    float* T;              // L_hat G, mp x np
    float* mom;            // m_t, dense m x n
    float* msgd;           // m_SGD, dense m x n
    double* part_m;        // sums of m_ij^2: kWaveSlots per tile slot
    double* part_sgd;      // per-block sums of m_SGD,ij^2
    LayerScalars* ls;
    int* nonfinite;        // set to 1 by a step whose ||m_SGD|| is not finite; cleared by the host
    int m, n, mp, np;
    int n_part_m, n_part_sgd;
};

// A 64 x 64 block of one layer's gradient for the stage-in kernel.
struct StageTile {
    int layer;
    int r0;
    int c0;
    int slot;
};

// A contiguous range of one layer's m*n elements for the weight update.
struct FlatChunk {
    int layer;
    int start;
    int count;
    int pad0;
};

// A pair of 64 x 64 tiles (ti, tj), ti <= tj, of one factor to symmetrize.
struct SymTile {
    int factor;
    int ti;
    int tj;
    int pad0;
};

// User pointers passed by value as kernel arguments, one batch of layers per launch
// (2 KB of pointers, within the 4 KB a kernel's arguments may take).
constexpr int kPtrBatch = 256;
struct PtrBatch {
    const float* p[kPtrBatch];
};
struct MutPtrBatch {
    float* p[kPtrBatch];
};

}  // namespace jorge
