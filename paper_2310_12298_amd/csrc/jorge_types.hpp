// Plain structs shared by the host runtime and the gfx950 kernels.
#pragma once

#include <stdint.h>

namespace jorge {

// Epilogues of the grouped GEMM (what is done with C = A * B of one tile).
enum Epilogue : int {
    EPI_STORE = 0,     // C
    EPI_SYM = 1,       // C and its mirror C^T (upper tiles of a symmetric product only)
    EPI_NORM = 2,      // C, plus the tile's sum of C_ij^2 (for ||X||_F)
    EPI_POLY = 3,      // I - a X + b C with C = X X  (truncated series of Eq. 6)
    EPI_SCALE = 4,     // s C                          (s A_hat P)
    EPI_MOMENTUM = 5,  // m = beta1 m + (1-beta1) C, plus the tile's sum of m_ij^2
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
    float pad;
};

// Scalars of one layer's weight update, written by the layer finalize kernel.
struct LayerScalars {
    double norm_m;    // ||m_t||_F
    double norm_sgd;  // ||m_SGD,t||_F
    double g;         // step applied to m_t
    float gf;         // g as fp32
    float decay;      // 1 - lr * weight_decay as fp32
};

// One product C = A * B of a grouped launch. Operand layouts are fixed per
// kernel instantiation: a "K-major" operand has K contiguous (A row-major,
// or B stored as B^T row-major), an "MN-major" one has M (N) contiguous.
// M, N, K are the padded extents (K a multiple of 32, ld's multiples of 4).
struct GemmProblem {
    const float* A;
    const float* B;
    float* C;
    const float* X;            // EPI_POLY: the X of the polynomial
    const FactorScalars* sc;   // EPI_POLY, EPI_SCALE
    float* mom;                // EPI_MOMENTUM: dense valid_m x valid_n momentum
    double* partials;          // EPI_NORM, EPI_MOMENTUM: one double per tile slot
    int M, N, K;
    int lda, ldb, ldc, ldx, ldmom;
    int valid_m, valid_n;      // unpadded extent (identity / momentum masks)
    int pad0;
};

struct TileDesc {
    int prob;  // index into the launch's problem table
    int tm;    // tile row
    int tn;    // tile column
    int slot;  // partial-sum slot within the problem
};

// Device view of a factor (L_hat or R_hat of one layer).
struct FactorDev {
    float* A;              // state, dp x dp, ld = dp, zero outside the d x d block
    float* W0;             // workspace: statistic M, later Z
    float* W1;             // workspace: A^2, later X
    float* W2;             // workspace: A^4, later P
    FactorScalars* sc;
    double* partials;      // per-tile sums of X_ij^2
    const float* gop;      // Gram operand with K contiguous: Gp (L side) or Gpt (R side)
    int gk;                // its K (np or mp), also its row stride
    int d, dp;
    int nparts;
};

// Device view of a layer.
struct LayerDev {
    float* Gp;             // padded copy of G, mp x np, ld = np, zero padding
    float* Gpt;            // its transpose, np x mp, ld = mp
    float* T;              // L_hat G, mp x np
    float* mom;            // m_t, dense m x n
    float* msgd;           // m_SGD, dense m x n
    double* part_m;        // per-tile sums of m_ij^2
    double* part_sgd;      // per-block sums of m_SGD,ij^2
    LayerScalars* ls;
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

// User pointers passed by value as kernel arguments, one batch of layers per launch.
constexpr int kPtrBatch = 128;
struct PtrBatch {
    const float* p[kPtrBatch];
};
struct MutPtrBatch {
    float* p[kPtrBatch];
};

}  // namespace jorge
