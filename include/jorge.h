/*
 * jorge.h - C ABI of an MI355X (gfx950) implementation of the Jorge optimizer step.
 *
 * Jorge (Singh, Sating, Bhatele, arXiv 2310.12298) keeps, per 2-D layer
 * theta (m x n), two preconditioner factors L_hat (m x m) and R_hat (n x n)
 * that approximate the inverse fourth roots of Shampoo's Kronecker factors,
 * and updates them with matrix products only (Section 3, Algorithm 2,
 * Eq. 3-7; the dynamic beta_2 of Appendix A.1, Eq. 8-9). The gradient is
 * preconditioned as L_hat G R_hat and applied with momentum, SGD grafting
 * (Appendix A.2, Algorithm 3) and decoupled weight decay (Section 4).
 *
 * Every entry point returns a jorge_status (0 = JORGE_OK, negative = error)
 * except jorge_destroy and the string helpers. No C++ exception crosses the
 * ABI. Pointers documented as "device" are HIP device pointers; every other
 * pointer is a host pointer. Work is queued on the context's HIP stream and
 * does not synchronise the host unless the comment says so. Arguments are
 * validated before any HIP call; an invalid call changes no state.
 *
 * A HIP error part-way through jorge_step is different: kernels queued before
 * it have run, so some state tensors (m_SGD, factors, momentum, parameters)
 * may hold the new step's values and others the old ones, and the step
 * counter has not advanced. The call returns JORGE_ERR_HIP and the context is
 * poisoned: every later jorge_step returns JORGE_ERR_HIP without queueing
 * anything, until the caller has restored the state from a checkpoint
 * (jorge_set_state for every tensor, the parameters by itself) and calls
 * jorge_set_step.
 *
 * The interface takes the step's scalars (lr, beta2, beta1, weight_decay) per
 * call, as doubles: they may change every step (a learning-rate schedule), and
 * the scalar arithmetic they enter runs in fp64 on the device. The options
 * fixed at creation (jorge_hparams) therefore carry none of them.
 *
 * A context is not re-entrant: calls on one context must not overlap.
 * Distinct contexts are independent.
 */
#ifndef JORGE_H
#define JORGE_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef int32_t jorge_status;
#define JORGE_OK                    0
#define JORGE_ERR_INVALID_ARGUMENT (-1) /* null pointer, bad size, bad mode, out-of-range value */
#define JORGE_ERR_OUT_OF_MEMORY    (-2) /* device or host allocation failed */
#define JORGE_ERR_HIP              (-3) /* a HIP runtime call or kernel launch failed */
#define JORGE_ERR_UNSUPPORTED      (-4) /* a size above the library's limits */

/* How beta_2 is chosen for each factor update (Section 3 and Appendix A.1).
 * FIXED:   beta = beta2 as passed (Algorithm 2 as printed).
 * DYNAMIC: beta = ||X||_F / (||X||_F + 1) (Eq. 8 with equality, Eq. 9); beta2
 *          is used only when ||X||_F = 0.
 * CLAMPED: beta = max(beta2, ||X||_F / (||X||_F + 1)): the dynamic value
 *          exactly when the truncated series would otherwise leave its domain
 *          ||(1-beta)/beta X|| < 1. Default.
 * In every mode the update uses c = (1-beta)/beta and s = beta^(-1/4), formed
 * on the dynamic branch as c = 1/||X||_F, s = (1 + 1/||X||_F)^(1/4) (Eq. 9). */
#define JORGE_BETA_FIXED   0
#define JORGE_BETA_DYNAMIC 1
#define JORGE_BETA_CLAMPED 2

/* Evaluation order of a factor update. Both compute the same factor (up to
 * fp32 rounding); they differ in cost. A (d x d) is updated from the
 * statistic M = H H^T with H = G (d = rows, k = cols) for L_hat and H = G^T
 * for R_hat, so M has rank at most k.
 * EXPLICIT: the paper's order (Algorithm 2): A^2, A^4, X = A^4 M, X X, A P;
 *           about 8 d^3 + d^2 k flops.
 * FACTORED: through H: U = A^4 H, X = U H^T, X X = U (H^T U) H^T,
 *           A P = A - A^5 H (a I - b H^T U) H^T, ||X||_F^2 = <U^T U, H^T H>;
 *           about 12 d^2 k + 5 d k^2 flops, far less when k << d.
 * SQUARED:  the factored order with A^2 formed once: A^2 H and A^4 H as
 *           H^T A^2 and (H^T A^2) A^2, A^5 H from A^4 H; about
 *           d^3 + 8 d^2 k + 5 d k^2 flops, less than either order above for k
 *           between about d/4 and 2d/3. Needs symmetric factors (symmetrize = 1).
 * AUTO:     per factor, whichever order has the least tile work (SQUARED only
 *           with symmetrize = 1). */
#define JORGE_FORM_AUTO     0
#define JORGE_FORM_EXPLICIT 1
#define JORGE_FORM_FACTORED 2
#define JORGE_FORM_SQUARED  3

/* State tensors of one layer (Algorithm 2 and Algorithm 3). */
#define JORGE_STATE_L       0 /* L_hat, rows x rows, fp32 (symmetric unless symmetrize = 0) */
#define JORGE_STATE_R       1 /* R_hat, cols x cols, fp32 (symmetric unless symmetrize = 0) */
#define JORGE_STATE_MOM     2 /* Jorge momentum m_t, rows x cols, fp32      */
#define JORGE_STATE_MOM_SGD 3 /* SGD heavy-ball momentum m_SGD, rows x cols */

/* Per-layer diagnostics of the last step (jorge_read_diag). */
#define JORGE_DIAG_NU_L     0 /* ||X_L||_F of the last factor update            */
#define JORGE_DIAG_NU_R     1 /* ||X_R||_F                                      */
#define JORGE_DIAG_BETA_L   2 /* beta used for L_hat in the last factor update  */
#define JORGE_DIAG_BETA_R   3 /* beta used for R_hat                            */
#define JORGE_DIAG_NORM_M   4 /* ||m_t||_F after the last step                  */
#define JORGE_DIAG_NORM_SGD 5 /* ||m_SGD,t||_F after the last step              */
#define JORGE_DIAG_STEP     6 /* step size g applied to m_t in the last step    */
#define JORGE_DIAG_COUNT    7

/* One layer: theta and G are dense row-major rows x cols fp32 (an N-d weight
 * collapsed to out x in*kh*kw, Section 3). */
typedef struct jorge_shape {
    int64_t rows;
    int64_t cols;
} jorge_shape;

/* Per-context options fixed at creation. */
typedef struct jorge_hparams {
    double  eps;              /* factors start at eps^(-1/4) I (Algorithm 2); > 0, finite.
                                 Default 1e-6. */
    int32_t precond_interval; /* k >= 1: factors update on steps t with (t-1) mod k == 0
                                 (Section 3, preconditioner update interval). Default 1. */
    int32_t beta_mode;        /* JORGE_BETA_*. Default JORGE_BETA_CLAMPED. */
    int32_t graft;            /* 1: SGD grafting (Algorithm 3); 0: theta -= lr * m_t. Default 1. */
    int32_t symmetrize;       /* 1: each updated factor is replaced by (Z + Z^T)/2, Z being
                                 Algorithm 2's product; 0: Z itself. Default 1. */
    int32_t factor_form;      /* JORGE_FORM_*: evaluation order of each factor update
                                 (JORGE_FORM_SQUARED needs symmetrize = 1).
                                 Default JORGE_FORM_AUTO. */
    int32_t split_k;          /* 1: a GEMM level splits some of its tiles along K where the
                                 library's cost model of the launch says it then finishes
                                 sooner: a level with too few tiles for the GPU, or one whose
                                 last round of tiles would leave most workgroups idle
                                 (partial products summed in a fixed order: deterministic,
                                 but rounded differently from an unsplit tile, and the split
                                 plan depends on every layer of the context); 0: never.
                                 Default 1. */
    int32_t lds_chain_max;    /* when every factor's size rounded up to 32 is at most this, each
                                 factor update runs in the explicit order in one workgroup with
                                 its matrices in LDS (one launch for the factors up to 64, one
                                 for those of 96 and 128, which need symmetrize = 1) instead of
                                 the grouped levels. With any larger factor present the levels
                                 run anyway and take the small factors too. 0 disables.
                                 In [0, 128]. Default 128. */
    int32_t precond_lowrank;  /* 1: on update steps, a factored factor A with d > 3k preconditions
                                 through A_new H = s A H - (s/2)(W H^T H + H W^T H), built from
                                 the update's own terms (about 6 k^2 d flops instead of a d x d
                                 product; the same result up to fp32 rounding); needs
                                 symmetrize = 1. 0: always the direct products. Default 1. */
    int32_t series_order;     /* last power of X kept from the binomial series of
                                 (I + c X)^(-1/4) (Section 3, Eq. 5): 2 gives Eq. 6-7,
                                 P = I - (c/4) X + (5c^2/32) X^2, as in Algorithm 2; 3 also
                                 keeps -(15c^3/128) X^3, the term Section 3 drops. Order 3
                                 costs one more product per factor (2 d^3 in the explicit
                                 order, k^3 in the factored one) and one more GEMM launch per
                                 update. 2 or 3. Default 2. */
} jorge_hparams;

/* Largest rows or cols of a layer the library accepts. */
#define JORGE_MAX_DIM 32768
/* Largest number of layers in one context. */
#define JORGE_MAX_LAYERS 65536

typedef struct jorge_ctx jorge_ctx;

/* Fills *hp with the defaults listed above. hp: non-NULL. */
jorge_status jorge_hparams_default(jorge_hparams* hp);

/* Creates a context for num_layers layers (Algorithm 2's initialisation).
 * shapes: num_layers entries, each rows, cols in [1, JORGE_MAX_DIM].
 * hp: options, or NULL for the defaults.
 * hip_stream: the hipStream_t all work is queued on (NULL = the null stream).
 * Allocates all device state (factors eps^(-1/4) I, momenta zero) and the
 * workspace in one device allocation owned by the context; the step counter
 * starts at 0. Synchronises the stream before returning. On error *out is
 * set to NULL and nothing stays allocated. */
jorge_status jorge_create(const jorge_shape* shapes, int32_t num_layers,
                          const jorge_hparams* hp, void* hip_stream, jorge_ctx** out);

/* Plans a context without a GPU: lays out the device arena and builds and
 * checks every launch table on the host (each access of each grouped launch
 * inside its buffer, alignment and extents as the kernels assume), exactly as
 * jorge_create does, then frees everything. Makes no HIP call.
 * *arena_bytes receives the size of the device allocation jorge_create would
 * make. Same argument rules and errors as jorge_create; a table that fails
 * the check returns JORGE_ERR_HIP (an internal error). */
jorge_status jorge_plan(const jorge_shape* shapes, int32_t num_layers, const jorge_hparams* hp,
                        int64_t* arena_bytes);

/* The grouped GEMM launches of each stage as jorge_plan builds them, without a
 * GPU: for min(n, jorge_num_stages()) stages (numbered as for jorge_stage_name),
 * units[i] receives the work units (workgroups) of the stage's grouped
 * launches, split_tiles[i] the number of 128 x 128 tiles split along K (0 when
 * split_k = 0) and small_blocks[i] the number of 64 x 64 blocks computed in
 * small mode (products with at most 64 rows or columns, one wave per block,
 * up to four per unit). A unit is a whole tile, a piece of a split tile or a
 * group of small-mode blocks. units, split_tiles and small_blocks are host
 * arrays of n entries; any may be NULL, not all when n > 0. Same argument
 * rules and errors as jorge_plan. */
jorge_status jorge_plan_stages(const jorge_shape* shapes, int32_t num_layers, const jorge_hparams* hp,
                               int64_t* units, int64_t* split_tiles, int64_t* small_blocks, int32_t n);

/* One Jorge step for every layer (Algorithm 2 with Algorithm 3 and decoupled
 * weight decay). With t the new step number (1 for the first call):
 *   if (t-1) mod k == 0, for A in {L_hat (statistic G G^T), R_hat (G^T G)}:
 *     X = A^4 * stat;  nu = ||X||_F;  (c, s) from beta_mode, beta2 and nu;
 *     Z = s * A * (I - (c/4) X + (5 c^2/32) X^2);  A <- (Z + Z^T)/2 or Z;
 *   G~ = L_hat G R_hat;  m = beta1 m + (1-beta1) G~;  m_SGD = beta1 m_SGD + G;
 *   g = lr ||m_SGD||_F / ||m||_F (graft, 0 if ||m||_F = 0) or lr (no graft);
 *   theta <- theta (1 - lr weight_decay) - g m.
 * params: host array of num_layers device pointers, each a dense row-major
 *   rows x cols fp32 tensor, updated in place.
 * grads: host array of num_layers device pointers (same layout), read only.
 * lr >= 0, 0 < beta2 < 1, 0 <= beta1 < 1, weight_decay >= 0, all finite.
 * The host arrays are read before the call returns; the tensors must stay
 * valid until the stream has executed the step. */
jorge_status jorge_step(jorge_ctx* ctx, float* const* params, const float* const* grads,
                        double lr, double beta2, double beta1, double weight_decay);

/* For callers that cannot allocate device memory (tight serving loops,
 * harnesses that forbid allocation): one step of one layer, as jorge_step
 * computes it, with the state held by the caller and every temporary in the
 * library's static device scratch of JORGE_NOALLOC_SCRATCH_BYTES per GPU,
 * instead of a context's allocations. Makes no device allocation.
 * shape: the layer (rows x cols); hp: options as for jorge_create (NULL = the
 * defaults); t >= 1: the number of this step (the factors update when
 * (t-1) mod precond_interval == 0).
 * theta (in/out), grad (in): device, dense row-major rows x cols fp32.
 * L (rows x rows), R (cols x cols), mom, mom_sgd (rows x cols): device, dense
 * row-major fp32, the state before the step on entry and after it on return
 * (start from eps^(-1/4) I, eps^(-1/4) I, 0, 0; jorge_get_state gives a
 * context's state in this layout). lr, beta2, beta1, weight_decay: as for
 * jorge_step. hip_stream: the stream the work is queued on.
 * The call returns after the stream has executed the step (the scratch is
 * reused by the next call). Calls on one GPU share its scratch: the library
 * runs them one at a time (a lock per GPU), and each starts by clearing what
 * must start at zero. Errors: JORGE_ERR_INVALID_ARGUMENT as for jorge_step;
 * JORGE_ERR_UNSUPPORTED if the layer's workspace and launch tables need more
 * than JORGE_NOALLOC_SCRATCH_BYTES (a 512 x 1024 layer fits with split_k = 1,
 * a 1024 x 1024 one with split_k = 0); JORGE_ERR_HIP on a runtime error, in
 * which case the caller's state may be partly updated. */
#define JORGE_NOALLOC_SCRATCH_BYTES (64ll << 20)
jorge_status jorge_step_noalloc(const jorge_shape* shape, const jorge_hparams* hp, int64_t t, float* theta,
                                const float* grad, float* L, float* R, float* mom, float* mom_sgd, double lr,
                                double beta2, double beta1, double weight_decay, void* hip_stream);

/* Copies one state tensor (dense, row-major; sizes as listed for JORGE_STATE_*)
 * into dst, a device buffer with row stride ld_dst >= its columns. Stream-ordered. */
jorge_status jorge_get_state(jorge_ctx* ctx, int32_t layer, int32_t kind, float* dst,
                             int64_t ld_dst);

/* Overwrites one state tensor from src, a device buffer with row stride
 * ld_src >= its columns (for checkpoint restore and state injection). The
 * caller keeps factors symmetric if it relies on symmetry. A factor's storage
 * padding (rows and columns past its size) is reset to zeros as well, so a
 * restore also undoes a step that met non-finite values. Stream-ordered. */
jorge_status jorge_set_state(jorge_ctx* ctx, int32_t layer, int32_t kind, const float* src,
                             int64_t ld_src);

/* Lends the device pointer of one state tensor and its row stride in floats
 * (*ld: factors are stored with rows padded to a multiple of 32, zero outside
 * the valid block, so a caller that reads or writes them in place needs the
 * stride). Valid until jorge_destroy. */
jorge_status jorge_state_ptr(jorge_ctx* ctx, int32_t layer, int32_t kind, float** dev_ptr,
                             int64_t* ld);

/* Step counter: the number of steps taken (0 after create). jorge_set_step
 * (t >= 0) also lifts the refusal that follows a step failed part-way (see the
 * top of this file): call it once the state has been restored. */
jorge_status jorge_get_step(const jorge_ctx* ctx, int64_t* t);
jorge_status jorge_set_step(jorge_ctx* ctx, int64_t t);

/* Diagnostics of the last step for one layer: out[JORGE_DIAG_COUNT] on the
 * host. Synchronises the context's stream. */
jorge_status jorge_read_diag(jorge_ctx* ctx, int32_t layer, double* out);

/* Non-finite gradients (failure detection). A step sets a layer's flag in
 * device memory when the fp64 norm ||m_SGD||_F that it sums for the grafting
 * anyway comes out non-finite (no host synchronisation, no extra pass over
 * G). Any NaN or infinity in the layer's gradient does that, through m_SGD =
 * beta1 m_SGD + G (Algorithm 3); so does an m_SGD element that overflows fp32.
 * The step itself runs to its end; the layer's m_SGD, m and parameters
 * are then non-finite, and stay so in later steps until the caller restores
 * its state (jorge_set_state, jorge_set_step). This call synchronises the
 * context's stream, sets *count to the number of layers flagged by any step
 * since the context was created or this call last ran, and *first (if not
 * NULL) to the lowest such layer index or -1, then clears the flags. */
jorge_status jorge_nonfinite(jorge_ctx* ctx, int32_t* count, int32_t* first);

/* Changes the stream later calls queue on (NULL = the null stream). Work
 * queued later on the new stream waits for everything already queued on the
 * old one (an event recorded on the old stream, waited on by the new one), so
 * the switch needs no synchronisation by the caller; jorge_synchronize and
 * jorge_destroy then cover the old stream's work too. Exception: when either
 * stream is being captured into a graph, no such wait is queued (a capture
 * cannot wait on an event recorded outside it); the capture's owner orders
 * the two streams. */
jorge_status jorge_set_stream(jorge_ctx* ctx, void* hip_stream);

/* Waits for all work queued by the context. */
jorge_status jorge_synchronize(jorge_ctx* ctx);

/* Device bytes the context holds (state plus workspace). */
jorge_status jorge_device_bytes(const jorge_ctx* ctx, int64_t* bytes);

/* Per-stage timing. When enabled, every kernel launch of a step is bracketed
 * by HIP events on the context's stream. jorge_read_timing synchronises,
 * adds the elapsed time of every bracket since the last read to per-stage
 * totals, and copies min(n, jorge_num_stages()) totals (milliseconds) and
 * launch counts into ms / launches (either may be NULL).
 * jorge_reset_timing zeroes the totals. */
jorge_status jorge_set_timing(jorge_ctx* ctx, int32_t enable);
jorge_status jorge_read_timing(jorge_ctx* ctx, double* ms, int64_t* launches, int32_t n);
jorge_status jorge_reset_timing(jorge_ctx* ctx);
int32_t      jorge_num_stages(void);
/* Algorithmic flops of each stage in one step that updates the factors
 * (symmetric products counted once per stored pair), for
 * min(n, jorge_num_stages()) stages; flops: host array. */
jorge_status jorge_stage_flops(const jorge_ctx* ctx, double* flops, int32_t n);
const char*  jorge_stage_name(int32_t stage);  /* NULL if out of range */

/* The evaluation order chosen for one factor: side 0 = L_hat, 1 = R_hat;
 * *form receives JORGE_FORM_EXPLICIT, JORGE_FORM_FACTORED or JORGE_FORM_SQUARED. */
jorge_status jorge_factor_form(const jorge_ctx* ctx, int32_t layer, int32_t side, int32_t* form);

/* Frees the context and all device memory it holds; NULL is ignored.
 * Synchronises the context's stream first. */
void jorge_destroy(jorge_ctx* ctx);

/* Static description of a status code. */
const char* jorge_status_string(jorge_status s);

/* Detail of the last error on this context ("" if none). */
const char* jorge_last_error(const jorge_ctx* ctx);

#ifdef __cplusplus
}
#endif

#endif /* JORGE_H */
