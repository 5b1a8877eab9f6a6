// Host runtime and C ABI of the Jorge optimizer step on gfx950.
//
// A context owns one device arena holding, per layer, the factors L_hat and
// R_hat (padded to multiples of 32, zero outside the valid block), the
// workspace of each factor's update, the padded gradient and its transpose,
// the intermediate L_hat G, both momenta and the partial-sum slots; and the
// device tables that describe every grouped launch. Tables are built once at
// creation, so a step is a fixed sequence of launches on one stream with no
// host sync.
//
// Each factor A (d x d) is updated from the statistic M = H H^T, where H is
// G (L side, d = m, k = n) or G^T (R side, d = n, k = m) (Algorithm 2,
// Appendix A.1). Two evaluation orders give the same factor:
//
//   explicit (the paper's order):  A^2, A^4, X = A^4 M, nu = ||X||_F,
//     P = I - (c/4) X + (5c^2/32) X X, Z = s A P, A <- (Z + Z^T)/2.
//   factored, through H (rank of M is at most k):  with U = A^4 H,
//     X = U H^T, X X = U S H^T with S = H^T U (k x k), so
//     P = I - U (aI - bS) H^T and A P = A - W H^T with W = A^5 H (aI - bS);
//     nu^2 = ||U H^T||_F^2 = <U^T U, H^T H>; the symmetrized factor is
//     s A - (s/2)(W H^T + H W^T). It costs about 12 d^2 k + 5 d k^2 flops
//     against 8 d^3 + d^2 k.
//   squared (symmetric factors): the factored order with A^2 formed once, so
//     that A^2 H and A^4 H take one product each: about d^3 + 8 d^2 k + 5 d k^2
//     flops, the cheapest of the three for k between about d/4 and 2d/3.
// Each factor takes the order with the least tile work (hp.factor_form can
// force one).
//
// Update step, as dependency levels (every GEMM of a level is one grouped
// launch; "Yt_j" is (A^j H)^T, k x d):
//   stage-in  Gp <- G, Gpt <- G^T, m_SGD <- beta1 m_SGD + G, partial sums of m_SGD^2
//   gram      explicit: M = H H^T, A^2      factored: Q = H^T H, Yt_1 = H^T A^T
//                                           squared: Q, A^2 (and A H)
//   pow4      explicit: A^4                 factored: Yt_2          squared: Yt_2 = H^T A^2
//   xform     explicit: X, X^T, ||X||^2     factored: Yt_3, S = Yt_2 Yt_2^T
//                                           squared: Yt_4 = Yt_2 A^2, S
//   chain4                                  factored: Yt_4
//                                           squared: A^5 H, <U^T U, Q>
//   chain5                                  factored: A^5 H (stored d x k), <U^T U, Q>
//   ffinal    nu = ||X||_F, beta, c, s per factor
//   poly      explicit: P^T                 factored: W = a A^5 H - b A^5 H S
//             (series order 3: V = b X - e X X   /   V = b S - e S S)
//   poly2     (series order 3 only) explicit: P^T = (I - a X + X V)^T   factored: W = a A^5 H - A^5 H V
//   update    explicit: Z = s A P           factored: A <- s A - (s/2)(W H^T + H W^T)
//   symm      explicit: A <- (Z + Z^T)/2
//   precond   T = L_hat G, then G~ = T R_hat fused with m <- beta1 m + (1-beta1) G~;
//             on update steps a factored factor with d > 3k supplies A_new H from the
//             update's own terms instead (low-rank preconditioning)
//   lfinal    ||m||, ||m_SGD||, grafted step g
//   weight    theta <- theta (1 - lr wd) - g m
// When every factor has padded size up to hp.lds_chain_max (at most 128), the
// levels are replaced by LDS chain kernels, which run each factor's whole
// explicit-order update in one workgroup with its matrices in LDS
// (lds_chain_kernel up to 64, lds_chain128_kernel for 96 and 128; one launch
// each for all their factors).
// Non-update steps run stage-in, precond, lfinal and weight only.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <cstdio>
#include <cstring>
#include <functional>
#include <mutex>
#include <new>
#include <queue>
#include <string>
#include <vector>

#include "../../include/jorge.h"
#include "jorge_gemm.hpp"
#include "jorge_kernels.hpp"
#include "jorge_types.hpp"

using namespace jorge;

namespace {

// Timed stages: one per dependency level of the update (see above).
enum Stage : int {
    ST_STAGEIN = 0, ST_GRAM, ST_POW4, ST_XFORM, ST_CHAIN4, ST_CHAIN5, ST_FFINAL, ST_POLY, ST_UPDATE,
    ST_SYMM, ST_PRECOND_L, ST_PRECOND_R, ST_LFINAL, ST_WEIGHT, ST_FIXUP, ST_LDS_CHAIN, ST_UPRECOND_L,
    ST_UPRECOND_R, ST_POLY2, ST_COUNT
};
const char* const kStageNames[ST_COUNT] = {
    "stage_in", "gram", "pow4", "xform", "chain4", "chain5", "factor_finalize", "poly", "update",
    "symmetrize", "precond_L", "precond_R", "layer_finalize", "weight", "split_fixup", "lds_chain",
    "uprecond_L", "uprecond_R", "poly2"};
// The GEMM levels of an update step, in launch order (poly2 is empty unless
// the series keeps its cubic term).
constexpr int kLevels[] = {ST_GRAM, ST_POW4, ST_XFORM, ST_CHAIN4, ST_CHAIN5, ST_POLY, ST_POLY2, ST_UPDATE};

constexpr size_t kAlign = 256;
constexpr int kFlatChunkElems = 16384;
constexpr int kGroupRows = 8;  // tile rows per group in the tile ordering
constexpr int kXcds = 8;  // workgroup b of a launch runs on XCD b % 8, in increasing b
constexpr int kSlots = 512;   // resident GEMM workgroups: 256 CUs x 2
constexpr int kMinSplitK = 64;  // shortest K piece of a split tile

inline int64_t round_up(int64_t x, int64_t m) { return (x + m - 1) / m * m; }
inline int64_t tiles_of(int64_t x) { return (x + kTile - 1) / kTile; }

struct GemmStage {
    bool kmajor_b = false;          // the NT launch (K-contiguous B): small mode is available
    std::vector<GemmProblem> probs;
    std::vector<TileDesc> tiles;    // work units, in dispatch order once uploaded
    std::vector<SmallUnit> small;   // small-mode blocks (grouped by four into units of tiles)
    std::vector<FixupDesc> fix;     // split tiles
    int nparts = 0;                 // split-workspace blocks the stage uses
    double flops = 0.0;             // algorithmic flops of all its products
    GemmProblem* dprobs = nullptr;
    TileDesc* dtiles = nullptr;
    SmallUnit* dsmall = nullptr;
    FixupDesc* dfix = nullptr;
    int ntiles() const { return (int)tiles.size(); }
};

struct LayerHost {
    int m, n, mp, np;
    size_t off_Gp, off_Gpt, off_T, off_mom, off_msgd, off_part_m, off_part_sgd, off_ls;
    int n_part_m = 0, n_part_sgd = 0;
    int fL, fR;
};

// One factor: A (d x d) with statistic H H^T, H being d x k.
//   explicit workspace: w[0] M (kept until the next step's gram level: a factored factor of the
//   same layer reads it as its H^T H), w[1] A^2, then X, then Z, w[2] A^4 then P^T (with the cubic
//   term, V^T), w[3] X^T (with the cubic term, then P^T) (dp x dp each)
//   factored workspace: w[0], w[1] kp x dp (Yt_j, A^5 H, W), w[2] Q = H^T H, w[3] S (kp x kp),
//   and with series order 3 s2: b S - e S^2 (kp x kp)
struct FactorHost {
    int layer, side, d, dp, k, kp;
    bool expl = true;
    bool squared = false;  // (not explicit) the squared order: A^2 formed, the chain in steps of A^2
    bool chain = false;  // small: the whole update in one workgroup (an LDS chain kernel), explicit order
    // Low-rank preconditioning on update steps (factored, symmetric, d > 3k): the
    // layer's A_new H comes from the chain's A H, W, Q and H^T W (see add_factored).
    bool lrp = false;
    size_t off_y1 = 0, off_wt = 0, off_v2t = 0, off_xa = 0;
    size_t off_A, off_part, off_sc;
    size_t off_w[4];
    size_t off_s2 = 0;
    size_t off_a2 = 0;     // the squared order's A^2 (dp x dp)
    int nparts = 0;
};

struct Launch {  // one timed launch: stage id and its bracketing events
    int stage;
    hipEvent_t start, stop;
};

}  // namespace

struct jorge_ctx {
    jorge_hparams hp{};
    hipStream_t stream = nullptr;
    int64_t t = 0;
    int device = 0;
    std::vector<LayerHost> layers;
    std::vector<FactorHost> factors;
    char* arena = nullptr;
    size_t arena_bytes = 0;
    size_t off_nonfinite = 0;  // int per layer (count rounded up to 4): non-finite ||m_SGD|| seen
    std::vector<std::pair<size_t, size_t>> regions;  // (offset, bytes) of every arena buffer
    // device tables
    LayerDev* dlayers = nullptr;
    FactorDev* dfactors = nullptr;
    StageTile* dstage = nullptr;
    FlatChunk* dflat = nullptr;
    SymTile* dsym = nullptr;
    std::vector<StageTile> stage_tiles;
    std::vector<FlatChunk> flat_chunks;
    std::vector<int> stage_batch_start, flat_batch_start;  // first block of each layer batch
    std::vector<SymTile> sym_tiles;
    // factors of the grouped levels, of the LDS chain (padded size <= 64) and of
    // the LDS chain for padded sizes 96 and 128
    std::vector<int> grouped, chain, chain2;
    int* dgrouped = nullptr;
    int* dchain = nullptr;
    int* dchain2 = nullptr;
    double chain_flops = 0.0;  // algorithmic flops of the chains' factor updates
    float* splitws = nullptr;     // partial products of split tiles (shared by the stages, in turn)
    int64_t splitws_blocks = 0;
    // Per stage: products with both operands K-major, and (literal mode only)
    // powers of non-symmetric factors, which need an MN-major B.
    GemmStage nt[ST_COUNT], nn[ST_COUNT];
    // timing
    bool timing = false;
    std::vector<hipEvent_t> free_events;
    std::vector<Launch> pending;
    double stage_ms[ST_COUNT] = {};
    int64_t stage_launches[ST_COUNT] = {};
    std::string last_error;
    hipEvent_t order_event = nullptr;  // orders a stream switch (jorge_set_stream)
    // jorge_step_noalloc: every device pointer of the context lies in lent
    // memory (free_ctx frees none), and the device tables go to a pool there
    // (upload() copies into it) instead of allocations of their own.
    bool lent = false;
    char* pool = nullptr;
    size_t pool_bytes = 0, pool_used = 0;
    // A step failed after its first launch: part of the state may be updated
    // and part not. Further steps are refused until jorge_set_step.
    bool poisoned = false;
};

// Device scratch of jorge_step_noalloc: the arena, split workspace and launch
// tables of its one-layer step live here instead of in allocations. Each GPU
// the library runs on holds its own copy from module load to process end. In
// host code this name is only a stand-in for the symbol: kernels and copies
// take the per-device address that hipGetSymbolAddress returns.
static __device__ __align__(256) unsigned char scratch[JORGE_NOALLOC_SCRATCH_BYTES];

namespace {

jorge_status fail(jorge_ctx* c, jorge_status s, const std::string& msg) {
    if (c) c->last_error = msg;
    return s;
}

// A failed runtime call is reported once, here: its error is also taken off
// the runtime's last-error state (where a later launch check would find it
// again); errors that stay with the device, such as a fault, remain.
jorge_status hip_fail(jorge_ctx* c, hipError_t e, const char* what) {
    (void)hipGetLastError();
    std::string msg = std::string(what) + ": " + hipGetErrorString(e);
    return fail(c, e == hipErrorOutOfMemory ? JORGE_ERR_OUT_OF_MEMORY : JORGE_ERR_HIP, msg);
}

#define JORGE_HIP(ctx, call)                                    \
    do {                                                        \
        hipError_t e_ = (call);                                 \
        if (e_ != hipSuccess) return hip_fail((ctx), e_, #call); \
    } while (0)

hipEvent_t take_event(jorge_ctx* c) {
    if (!c->free_events.empty()) {
        hipEvent_t e = c->free_events.back();
        c->free_events.pop_back();
        return e;
    }
    hipEvent_t e = nullptr;
    if (hipEventCreate(&e) != hipSuccess) return nullptr;
    return e;
}

// Brackets one launch with events when timing is on.
struct TimedLaunch {
    jorge_ctx* c;
    int stage;
    hipStream_t stream;
    hipEvent_t start = nullptr, stop = nullptr;
    TimedLaunch(jorge_ctx* ctx, int st) : TimedLaunch(ctx, st, ctx->stream) {}
    TimedLaunch(jorge_ctx* ctx, int st, hipStream_t s) : c(ctx), stage(st), stream(s) {
        if (!c->timing) return;
        start = take_event(c);
        stop = take_event(c);
        if (start) (void)hipEventRecord(start, stream);
    }
    void finish() {
        if (!c->timing || !start || !stop) return;
        (void)hipEventRecord(stop, stream);
        c->pending.push_back({stage, start, stop});
    }
};

// A product for add_problem: C = A B^T (NT) or A B (NN) with the given
// padded extents; everything else of the problem is zero until set.
GemmProblem product(const float* A, int lda, const float* B, int ldb, int M, int N, int K) {
    GemmProblem p{};
    p.A = A; p.lda = lda;
    p.B = B; p.ldb = ldb;
    p.M = M; p.N = N; p.K = K; p.K1 = K;
    p.coef = CO_ONE;
    return p;
}

// Adds a product's tiles in grouped order: bands of kGroupRows tile rows,
// walked column by column, so concurrently running workgroups share panels.
// flops: the product's algorithmic flops. Returns the number of partial-sum
// slots (one per tile).
// Whether a product may run in small mode (64 x 64 blocks, one wave each):
// a product of the NT launch with at most 64 rows or columns and a short K.
bool small_eligible(const GemmStage& st, const GemmProblem& p) {
    return st.kmajor_b && p.K <= kSmallMaxK && (p.M <= kSmallDim || p.N <= kSmallDim);
}

int add_problem(GemmStage& st, const GemmProblem& p, double flops) {
    const int idx = (int)st.probs.size();
    st.probs.push_back(p);
    st.flops += flops;
    const int tm_n = (int)tiles_of(p.M), tn_n = (int)tiles_of(p.N);
    int slot = 0;
    for (int g = 0; g < tm_n; g += kGroupRows)
        for (int tn = 0; tn < tn_n; ++tn)
            for (int tm = g; tm < std::min(g + kGroupRows, tm_n); ++tm) {
                if (p.upper && tm > tn) continue;
                st.tiles.push_back({idx, tm, tn, slot++, 0, p.K, -1, 0});
            }
    return slot;
}

// Small mode pays where a launch has enough units to keep every CU busy:
// then the padding of 128 x 128 tiles costs throughput, while a level with
// few units is bound by its longest unit, which a one-wave block lengthens. In a stage with at least kSlots tiles, every eligible
// product's tiles are replaced by its 64 x 64 blocks: those quadrants of its
// tiles that lie inside the product (and on or above the diagonal of a
// symmetric result), each with its tile's partial-sum slot; the tile's first
// block zeroes the partial sums of the others. The blocks are then grouped,
// longest K first, four to a unit of the tile list.
void make_small(GemmStage& st) {
    if (st.tiles.size() < (size_t)kSlots) return;
    std::vector<char> small(st.probs.size(), 0);
    bool any = false;
    for (size_t i = 0; i < st.probs.size(); ++i) any |= (small[i] = small_eligible(st, st.probs[i]));
    if (!any) return;
    std::vector<TileDesc> keep;
    keep.reserve(st.tiles.size());
    for (const TileDesc& t : st.tiles) {
        if (!small[t.prob]) {
            keep.push_back(t);
            continue;
        }
        const GemmProblem& p = st.probs[t.prob];
        const int bm_n = (p.M + kSmallDim - 1) / kSmallDim, bn_n = (p.N + kSmallDim - 1) / kSmallDim;
        int zero = 0, first = -1;
        for (int q = 0; q < kWaveSlots; ++q) {
            const int bm = 2 * t.tm + (q >> 1), bn = 2 * t.tn + (q & 1);
            if (bm >= bm_n || bn >= bn_n || (p.upper && bm > bn)) {
                zero |= 1 << q;
                continue;
            }
            if (first < 0) first = (int)st.small.size();
            st.small.push_back({t.prob, bm, bn, t.slot, 0, 0, 0, 0});
        }
        if (p.flags & (EF_NORM | EF_DOT | EF_MOMENTUM)) st.small[first].zero_mask = zero;
    }
    st.tiles.swap(keep);
    std::stable_sort(st.small.begin(), st.small.end(), [&](const SmallUnit& a, const SmallUnit& b) {
        return st.probs[a.prob].K > st.probs[b.prob].K;
    });
    for (size_t i = 0; i < st.small.size(); i += kWaveSlots) {
        const int n = (int)std::min<size_t>(kWaveSlots, st.small.size() - i);
        int K = 0;
        for (int j = 0; j < n; ++j) K = std::max(K, st.probs[st.small[i + j].prob].K);
        st.tiles.push_back({st.small[i].prob, (int)i, n, -1, 0, K, kSmallGroup, 0});
    }
}

int tile_count(int M, int N) { return (int)(tiles_of(M) * tiles_of(N)); }


// Puts work units in dispatch order. The units are sorted by K, longest
// first, and then by problem and by the start of their K range (the pieces of
// split tiles that cover one K range stay together); each problem's tiles
// stay in bands of kGroupRows tile rows walked column by column. Runs of
// consecutive units of one problem, one column and one K range (they share
// the B panel and neighbouring A panels) are dealt,
// in that order, to the XCD with the least accumulated work (K of the unit),
// so every XCD gets a balanced, largest-first share whose units reuse panels
// in its own L2. The shares are then interleaved so that XCD x's i-th unit
// sits at slot kXcds * i + x; once a share is used up, its slots take the
// next unit of the longest remaining share.
void order_for_xcds(std::vector<TileDesc>& tiles) {
    const size_t n = tiles.size();
    if (n == 0) return;
    // Longest K range first; within one length, by problem (in list order)
    // and then by the start of the K range, so the pieces of split tiles that
    // share a K range stay together (stable: tile order is kept otherwise).
    std::vector<int> first_of;
    {
        int mx = 0;
        for (const TileDesc& t : tiles) mx = std::max(mx, t.prob);
        first_of.assign(mx + 1, INT32_MAX);
        for (size_t i = 0; i < n; ++i) first_of[tiles[i].prob] = std::min(first_of[tiles[i].prob], (int)i);
    }
    std::stable_sort(tiles.begin(), tiles.end(), [&](const TileDesc& a, const TileDesc& b) {
        const int la = a.k1 - a.k0, lb = b.k1 - b.k0;
        if (la != lb) return la > lb;
        if (first_of[a.prob] != first_of[b.prob]) return first_of[a.prob] < first_of[b.prob];
        return a.k0 < b.k0;
    });
    std::vector<std::vector<TileDesc>> share(kXcds);
    std::vector<int64_t> work(kXcds, 0);
    for (size_t i = 0; i < n;) {
        size_t j = i + 1;
        while (j < n && tiles[j].prob == tiles[i].prob && tiles[j].tn == tiles[i].tn &&
               tiles[j].k0 == tiles[i].k0 && tiles[j].tm / kGroupRows == tiles[i].tm / kGroupRows)
            ++j;
        const int x = (int)(std::min_element(work.begin(), work.end()) - work.begin());
        for (size_t k = i; k < j; ++k) share[x].push_back(tiles[k]);
        work[x] += (int64_t)(j - i) * (tiles[i].k1 - tiles[i].k0);
        i = j;
    }
    std::vector<size_t> next(kXcds, 0);
    std::vector<TileDesc> out;
    out.reserve(n);
    for (size_t b = 0; b < n; ++b) {
        int x = (int)(b % kXcds);
        if (next[x] == share[x].size()) {
            size_t best = 0;
            for (int y = 0; y < kXcds; ++y)
                if (share[y].size() - next[y] > best) {
                    best = share[y].size() - next[y];
                    x = y;
                }
        }
        out.push_back(share[x][next[x]++]);
    }
    tiles.swap(out);
}

// Cost model of a grouped launch for the split planner, in units of one k
// step of a 128 x 128 tile on a whole compute unit (0.058 us). Workgroup b
// runs on XCD b mod kXcds, on one of that XCD's CUs. A CU holds two work
// units at a time; two resident units share its throughput, a unit alone on
// a CU runs at kLoneRate of it. A work unit costs its K plus its own
// prologue and epilogue; the fixup launch costs a fixed start plus the
// traffic of all partial products (64 KB each). Fitted on MI355X to the
// per-level times of 512 x 4608 and 64 x 576 layers with the long tiles cut
// into 1 .. 8 equal pieces or into pieces of a fixed length (most levels
// within 5%).
constexpr int kCus = kSlots / 2;
constexpr int kCusPerXcd = kCus / kXcds;
constexpr double kLoneRate = 0.9;
constexpr int64_t kUnitCost = 64;
constexpr int64_t kFixupStart = 200;
constexpr int64_t kFixupPartsPerK = 5;
// A split plan is kept only if the model puts it this much below the unsplit launch
// (the partial products' traffic also slows the other units, which the model leaves out).
constexpr double kSplitGain = 0.97;

// Duration of a list of units (in dispatch order) on ncu CUs: placed one per
// CU, then a second per CU; later, each unit goes to a CU with a free place,
// CUs with no resident unit first. Each CU shares its throughput between its
// resident units.
double launch_span(const std::vector<int64_t>& work, int ncu) {
    struct Cu {
        double rem[2];
        int n = 0;
        double last = 0.0;
        unsigned ver = 0;
    };
    std::vector<Cu> cu(ncu);
    typedef std::pair<double, std::pair<int, unsigned>> Ev;  // (time, (cu, version))
    std::priority_queue<Ev, std::vector<Ev>, std::greater<Ev>> events;
    auto rate = [](int n) { return n == 1 ? kLoneRate : 0.5; };  // of each resident unit
    auto next_done = [&](const Cu& c) {
        const double m = c.n == 1 ? c.rem[0] : std::min(c.rem[0], c.rem[1]);
        return c.last + m / rate(c.n);
    };
    size_t next = 0;
    for (int round = 0; round < 2; ++round)
        for (int i = 0; i < ncu && next < work.size(); ++i) cu[i].rem[cu[i].n++] = (double)work[next++];
    for (int i = 0; i < ncu; ++i)
        if (cu[i].n) events.push({next_done(cu[i]), {i, cu[i].ver}});
    double span = 0.0;
    std::vector<int> freed;
    while (!events.empty()) {
        // Every completion at this time, then the placements.
        const double now = events.top().first;
        freed.clear();
        while (!events.empty() && events.top().first <= now) {
            const Ev e = events.top();
            events.pop();
            Cu& c = cu[e.second.first];
            if (e.second.second != c.ver) continue;
            const double done_work = (e.first - c.last) * rate(c.n);
            for (int j = 0; j < c.n; ++j) c.rem[j] -= done_work;
            c.last = e.first;
            const int done = (c.n == 2 && c.rem[1] < c.rem[0]) ? 1 : 0;
            c.rem[done] = c.rem[c.n - 1];
            --c.n;
            ++c.ver;
            span = std::max(span, e.first);
            freed.push_back(e.second.first);
        }
        std::sort(freed.begin(), freed.end());
        freed.erase(std::unique(freed.begin(), freed.end()), freed.end());
        std::stable_sort(freed.begin(), freed.end(), [&](int a, int b) { return cu[a].n < cu[b].n; });
        for (int pass = 0; pass < 2; ++pass)
            for (int i : freed)
                if (next < work.size() && cu[i].n == pass) cu[i].rem[cu[i].n++] = (double)work[next++];
        for (int i : freed)  // each was brought up to now by its completion
            if (cu[i].n) events.push({next_done(cu[i]), {i, ++cu[i].ver}});
    }
    return span;
}

// The K lengths of a tile of length K cut into pieces of length P (a multiple
// of 32): whole pieces of P, and the rest as a last piece of its own when it
// is at least kMinSplitK long, else added to the last whole piece. A single
// piece means the tile stays whole.
std::vector<int64_t> cut_tile(int64_t K, int64_t P) {
    std::vector<int64_t> out;
    if (P <= 0 || P >= K) return {K};
    for (int64_t k = 0; k + P <= K; k += P) out.push_back(P);
    const int64_t rest = K - P * (int64_t)out.size();
    if (rest >= kMinSplitK) out.push_back(rest);
    else out.back() += rest;
    return out;
}

// Piece length that cuts K into q pieces of about equal length.
int64_t piece_len(int64_t K, int q) { return round_up((K + q - 1) / q, kSlab); }

// The work units of tiles cut into pieces of length plen[i] (0: whole), in
// tile order with each tile's pieces in K order; parts counts the pieces of
// cut tiles.
std::vector<TileDesc> cut_units(const std::vector<TileDesc>& tiles, const std::vector<int64_t>& plen,
                                int64_t* parts) {
    std::vector<TileDesc> units;
    units.reserve(tiles.size());
    *parts = 0;
    for (size_t i = 0; i < tiles.size(); ++i) {
        const TileDesc& t = tiles[i];
        const std::vector<int64_t> pieces = cut_tile(t.k1 - t.k0, plen[i]);
        if (pieces.size() > 1) *parts += (int64_t)pieces.size();
        int k = t.k0;
        for (int64_t len : pieces) {
            TileDesc u = t;
            u.k0 = k;
            u.k1 = k + (int)len;
            k = u.k1;
            units.push_back(u);
        }
    }
    return units;
}

// Modelled duration of a stage whose tiles are cut into pieces of length
// plen[i] (0: whole): the units in dispatch order, each XCD's share on its CUs,
// plus the fixup launch.
double modelled_cost(const std::vector<TileDesc>& tiles, const std::vector<int64_t>& plen) {
    int64_t parts = 0;
    std::vector<TileDesc> units = cut_units(tiles, plen, &parts);
    order_for_xcds(units);
    std::vector<std::vector<int64_t>> per(kXcds);
    for (size_t b = 0; b < units.size(); ++b) per[b % kXcds].push_back(units[b].k1 - units[b].k0 + kUnitCost);
    double cost = 0.0;
    for (const auto& w : per) cost = std::max(cost, launch_span(w, kCusPerXcd));
    if (parts) cost += (double)(kFixupStart + parts / kFixupPartsPerK);
    return cost;
}

// Splits the K range of some tiles of a stage when the cost model above says
// the launch then finishes sooner: a level with too few tiles to keep every CU
// busy, a level held up by a few long tiles, or one whose last round of tiles
// would leave CUs idle. Candidates, tiles taken longest first: no split;
// every long tile (more than half the longest) in q = 2 .. 8 equal pieces;
// every tile longer than P in pieces of P, for P a share of the stage's work
// per CU (1, 1/2, 1/3, 1/4, 1/6, 1/8) or the longest tile over q; and all but
// the last one or two rounds of kSlots tiles kept whole with every later tile
// in 2 .. 6 pieces. Pieces are never shorter than kMinSplitK. Each piece leaves a
// partial product in the split workspace; a fixup unit per split tile sums
// them in K order and runs the epilogue, so results do not depend on the
// schedule.
void split_stage(GemmStage& st) {
    const size_t n = st.tiles.size();
    if (n == 0) return;
    std::vector<size_t> idx(n);
    for (size_t i = 0; i < n; ++i) idx[i] = i;
    std::stable_sort(idx.begin(), idx.end(), [&](size_t a, size_t b) {
        return st.tiles[a].k1 - st.tiles[a].k0 > st.tiles[b].k1 - st.tiles[b].k0;
    });
    std::vector<int64_t> klen(n);
    int64_t W = 0;
    for (size_t i = 0; i < n; ++i) {
        klen[i] = st.tiles[idx[i]].k1 - st.tiles[idx[i]].k0;
        W += klen[i];
    }
    // Candidates give piece lengths in longest-first order; the model takes them in tile order.
    std::vector<int64_t> in_order(n, 0);
    auto cost_of = [&](const std::vector<int64_t>& plen) {
        for (size_t i = 0; i < n; ++i) in_order[idx[i]] = st.tiles[idx[i]].part == kSmallGroup ? 0 : plen[i];
        return modelled_cost(st.tiles, in_order);
    };
    const std::vector<int64_t> none(n, 0);
    std::vector<int64_t> best = none;
    const double base = cost_of(none);
    // No plan finishes before the CUs have shared out all the work (splitting only adds units).
    if (kSplitGain * base <= (double)(W + (int64_t)n * kUnitCost) / kCus) return;
    double best_cost = base;
    auto consider = [&](const std::vector<int64_t>& plen) {
        const double c = cost_of(plen);
        if (c < best_cost) {
            best_cost = c;
            best = plen;
        }
    };
    for (int q = 2; q <= 8; ++q) {  // the long tiles in q equal pieces
        std::vector<int64_t> plen(n, 0);
        for (size_t i = 0; i < n && 2 * klen[i] > klen[0]; ++i)
            if (klen[i] >= (int64_t)q * kMinSplitK) plen[i] = piece_len(klen[i], q);
        consider(plen);
    }
    std::vector<int64_t> lens;
    for (int m : {1, 2, 3, 4, 6, 8}) lens.push_back(round_up((W + (int64_t)m * kCus - 1) / ((int64_t)m * kCus), kSlab));
    for (int q = 2; q <= 8; ++q) lens.push_back(piece_len(klen[0], q));
    for (int64_t P : lens) {  // pieces of a fixed length
        P = std::max<int64_t>(P, kMinSplitK);
        std::vector<int64_t> plen(n, 0);
        for (size_t i = 0; i < n; ++i)
            if (klen[i] > P) plen[i] = P;
        consider(plen);
    }
    const size_t rounds = (n - 1) / kSlots;  // whole rounds before the last one
    for (size_t h = kSlots * (rounds > 2 ? rounds - 1 : 1); h < n; h += kSlots)  // the last rounds cut
        for (int q = 2; q <= 6; ++q) {
            std::vector<int64_t> plen(n, 0);
            for (size_t i = h; i < n; ++i)
                if (klen[i] >= (int64_t)q * kMinSplitK) plen[i] = piece_len(klen[i], q);
            consider(plen);
        }
    if (!(best_cost < kSplitGain * base)) return;
    std::vector<int64_t> plen_of(n, 0);
    for (size_t i = 0; i < n; ++i) plen_of[idx[i]] = st.tiles[idx[i]].part == kSmallGroup ? 0 : best[i];
    // The same units as the model's, with their workspace blocks and fixups.
    int64_t parts = 0;
    std::vector<TileDesc> out = cut_units(st.tiles, plen_of, &parts);
    for (size_t u = 0; u < out.size();) {
        size_t v = u + 1;
        while (v < out.size() && out[v].prob == out[u].prob && out[v].tm == out[u].tm && out[v].tn == out[u].tn &&
               out[v].k0 == out[v - 1].k1)
            ++v;
        if (v - u > 1) {
            st.fix.push_back({out[u].prob, out[u].tm, out[u].tn, out[u].slot, st.nparts, (int)(v - u), 0, 0});
            for (size_t q = u; q < v; ++q) out[q].part = st.nparts++;
        }
        u = v;
    }
    st.tiles.swap(out);
}

template <bool AK, bool BK>
jorge_status launch_gemm(jorge_ctx* c, const GemmStage& st, int stage, float beta1) {
    if (st.ntiles() == 0) return JORGE_OK;
    TimedLaunch tl(c, stage);
    hipLaunchKernelGGL((gemm_grouped<AK, BK>), dim3(st.ntiles()), dim3(kGemmThreads), 0, c->stream,
                       st.dprobs, st.dtiles, st.dsmall, beta1, c->splitws);
    tl.finish();
    JORGE_HIP(c, hipGetLastError());
    if (!st.fix.empty()) {
        TimedLaunch tf(c, ST_FIXUP);
        hipLaunchKernelGGL(gemm_fixup, dim3((unsigned)st.fix.size() * kWaveSlots), dim3(kFixupThreads), 0,
                           c->stream, st.dprobs, st.dfix, beta1, c->splitws);
        tf.finish();
        JORGE_HIP(c, hipGetLastError());
    }
    return JORGE_OK;
}

bool finite_pos(double x) { return std::isfinite(x) && x > 0.0; }

jorge_status validate_hparams(const jorge_hparams* hp) {
    if (!finite_pos(hp->eps)) return JORGE_ERR_INVALID_ARGUMENT;
    if (hp->precond_interval < 1) return JORGE_ERR_INVALID_ARGUMENT;
    if (hp->beta_mode < JORGE_BETA_FIXED || hp->beta_mode > JORGE_BETA_CLAMPED)
        return JORGE_ERR_INVALID_ARGUMENT;
    if ((hp->graft != 0 && hp->graft != 1) || (hp->symmetrize != 0 && hp->symmetrize != 1))
        return JORGE_ERR_INVALID_ARGUMENT;
    if (hp->factor_form < JORGE_FORM_AUTO || hp->factor_form > JORGE_FORM_SQUARED)
        return JORGE_ERR_INVALID_ARGUMENT;
    if (hp->factor_form == JORGE_FORM_SQUARED && hp->symmetrize != 1) return JORGE_ERR_INVALID_ARGUMENT;
    if (hp->split_k != 0 && hp->split_k != 1) return JORGE_ERR_INVALID_ARGUMENT;
    if (hp->lds_chain_max < 0 || hp->lds_chain_max > kChain2Max) return JORGE_ERR_INVALID_ARGUMENT;
    if (hp->precond_lowrank != 0 && hp->precond_lowrank != 1) return JORGE_ERR_INVALID_ARGUMENT;
    if (hp->series_order != 2 && hp->series_order != 3) return JORGE_ERR_INVALID_ARGUMENT;
    return JORGE_OK;
}

// Tile work (128 x 128 tiles times K) of one product, as the grouped launch runs it.
int64_t tile_work(int64_t M, int64_t N, int64_t K, bool upper) {
    const int64_t tm = tiles_of(M), tn = tiles_of(N);
    return (upper ? tm * (tm + 1) / 2 : tm * tn) * K;
}

// The order with the least tile work for a factor of padded size dp with
// statistic rank kp (same product lists as build_tables); ties go to the
// explicit, then the factored order. lrp: the factor would precondition in
// low rank if not explicit (the squared order then also forms A H).
int choose_form(int64_t dp, int64_t kp, bool sym, int order, bool lrp) {
    int64_t e = tile_work(dp, dp, kp, true) + 2 * tile_work(dp, dp, dp, sym) + 3 * tile_work(dp, dp, dp, false);
    int64_t f = tile_work(kp, kp, dp, true) + 5 * tile_work(kp, dp, dp, false) + tile_work(kp, kp, dp, sym) +
                tile_work(kp, kp, dp, true) + tile_work(dp, kp, kp, false) +
                (sym ? tile_work(dp, dp, 2 * kp, true) : tile_work(dp, dp, kp, false));
    // A^2, Q, three chain products, S, nu, W and the SYR2K (and A H)
    int64_t q = tile_work(dp, dp, dp, true) + tile_work(kp, kp, dp, true) + 3 * tile_work(kp, dp, dp, false) +
                2 * tile_work(kp, kp, dp, true) + tile_work(dp, kp, kp, false) + tile_work(dp, dp, 2 * kp, true) +
                (lrp ? tile_work(kp, dp, dp, false) : 0);
    if (order == 3) {  // X V, and S S
        e += tile_work(dp, dp, dp, false);
        f += tile_work(kp, kp, kp, sym);
        q += tile_work(kp, kp, kp, true);
    }
    if (sym && q < std::min(e, f)) return JORGE_FORM_SQUARED;
    return e <= f ? JORGE_FORM_EXPLICIT : JORGE_FORM_FACTORED;
}

// Builds every offset; returns the arena size in bytes.
size_t plan(jorge_ctx* c) {
    size_t off = 0;
    auto take = [&](size_t bytes) {
        const size_t o = off;
        c->regions.push_back({o, bytes});
        off = (size_t)round_up((int64_t)(off + bytes), kAlign);
        return o;
    };
    const bool sym = c->hp.symmetrize != 0;
    // The LDS chains take the factor updates (explicit order, one workgroup per
    // factor) when every factor of the context has padded size up to
    // lds_chain_max, replacing the grouped levels altogether (sizes 96 and 128
    // need symmetric factors). With any larger factor present the levels run
    // anyway, and the small factors' tiles fill slots of theirs that would
    // otherwise idle: taking the small factors out to the chains, on a second
    // stream beside the levels or before them, measured no faster.
    int max_dp = 0;
    for (const auto& L : c->layers) max_dp = std::max(max_dp, std::max(L.mp, L.np));
    const bool all_small = max_dp <= c->hp.lds_chain_max && (max_dp <= kChainMax || sym);
    for (auto& L : c->layers) {
        for (int side = 0; side < 2; ++side) {
            FactorHost F{};
            F.layer = (int)(&L - &c->layers[0]);
            F.side = side;
            F.d = side == 0 ? L.m : L.n;
            F.dp = side == 0 ? L.mp : L.np;
            F.k = side == 0 ? L.n : L.m;
            F.kp = side == 0 ? L.np : L.mp;
            // A_new H (d x k) replaces a d x d product in the preconditioning when
            // 6 k^2 d < 2 d^2 k, i.e. d > 3 k (both orders then cost 2 k^2 d more).
            const bool lrp_ok = sym && c->hp.precond_lowrank && (int64_t)F.d > 3 * (int64_t)F.k;
            const int level_form = c->hp.factor_form != JORGE_FORM_AUTO
                                       ? c->hp.factor_form
                                       : choose_form(F.dp, F.kp, sym, c->hp.series_order, lrp_ok);
            F.chain = all_small;
            const int form = F.chain ? JORGE_FORM_EXPLICIT : level_form;
            F.expl = form == JORGE_FORM_EXPLICIT;
            F.squared = form == JORGE_FORM_SQUARED;
            const size_t dd = (size_t)F.dp * F.dp * sizeof(float);
            F.off_A = take(dd);
            if (F.chain) {
                F.nparts = 1;  // unused: the chain kernel reduces ||X|| itself
                // the explicit order's algorithmic flops (symmetric products counted once)
                const double d = F.d, k = F.k;
                c->chain_flops += d * d * k + (sym ? 2.0 : 4.0) * d * d * d +
                                  (c->hp.series_order == 3 ? 8.0 : 6.0) * d * d * d;
            } else if (F.expl) {
                for (int w = 0; w < 4; ++w) F.off_w[w] = take(dd);
                F.nparts = tile_count(F.dp, F.dp);
            } else {
                const size_t kd = (size_t)F.kp * F.dp * sizeof(float), kk = (size_t)F.kp * F.kp * sizeof(float);
                F.off_w[0] = take(kd);
                F.off_w[1] = take(kd);
                F.off_w[2] = take(kk);
                F.off_w[3] = take(kk);
                if (c->hp.series_order == 3) F.off_s2 = take(kk);
                if (F.squared) F.off_a2 = take(dd);
                F.nparts = tile_count(F.kp, F.kp);
            }
            F.lrp = !F.expl && lrp_ok;
            if (F.lrp) {
                const size_t kd = (size_t)F.kp * F.dp * sizeof(float), kk = (size_t)F.kp * F.kp * sizeof(float);
                F.off_y1 = take(kd);   // A H, d x k
                F.off_wt = take(kd);   // W^T, k x d
                F.off_v2t = take(kk);  // H^T W, k x k
                F.off_xa = take(kd);   // A_new H, d x k
            }
            F.off_part = take((size_t)F.nparts * kWaveSlots * sizeof(double));
            F.off_sc = take(sizeof(FactorScalars));
            (side == 0 ? L.fL : L.fR) = (int)c->factors.size();
            c->factors.push_back(F);
        }
        const size_t padded = (size_t)L.mp * L.np * sizeof(float);
        const size_t dense = (size_t)L.m * L.n * sizeof(float);
        L.off_Gp = take(padded);
        L.off_Gpt = take(padded);
        L.off_T = take(padded);
        L.off_mom = take(dense);
        L.off_msgd = take(dense);
        L.n_part_m = tile_count(L.mp, L.np);
        L.off_part_m = take((size_t)L.n_part_m * kWaveSlots * sizeof(double));
        L.n_part_sgd = ((L.m + 63) / 64) * ((L.n + 63) / 64);
        L.off_part_sgd = take((size_t)L.n_part_sgd * sizeof(double));
        L.off_ls = take(sizeof(LayerScalars));
    }
    c->off_nonfinite = take(round_up((int64_t)c->layers.size(), 4) * sizeof(int));
    return off;
}

template <typename T>
T* at(jorge_ctx* c, size_t off) { return reinterpret_cast<T*>(c->arena + off); }

// The products of one factor's update in the explicit order.
void add_explicit(jorge_ctx* c, const FactorHost& F, const FactorDev& fd, const float* Hr) {
    const bool sym = c->hp.symmetrize != 0;
    const int dp = F.dp, kp = F.kp;
    const double d = F.d, k = F.k;
    float* A = fd.A;
    float* W0 = at<float>(c, F.off_w[0]);
    float* W1 = at<float>(c, F.off_w[1]);
    float* W2 = at<float>(c, F.off_w[2]);
    float* W3 = at<float>(c, F.off_w[3]);
    // M = H H^T
    GemmProblem m = product(Hr, kp, Hr, kp, dp, dp, kp);
    m.C = W0; m.ldc = dp; m.flags = EF_STORE; m.upper = 1;
    add_problem(c->nt[ST_GRAM], m, d * d * k);
    // A^2 and A^4: symmetric products of symmetric factors; general in the literal mode.
    GemmProblem p2 = product(A, dp, A, dp, dp, dp, dp);
    p2.C = W1; p2.ldc = dp; p2.flags = EF_STORE; p2.upper = sym;
    add_problem(sym ? c->nt[ST_GRAM] : c->nn[ST_GRAM], p2, (sym ? 1 : 2) * d * d * d);
    GemmProblem p4 = product(W1, dp, W1, dp, dp, dp, dp);
    p4.C = W2; p4.ldc = dp; p4.flags = EF_STORE; p4.upper = sym;
    add_problem(sym ? c->nt[ST_POW4] : c->nn[ST_POW4], p4, (sym ? 1 : 2) * d * d * d);
    // X = A^4 M (M symmetric, so it is its own K-major B), stored with its transpose.
    GemmProblem x = product(W2, dp, W0, dp, dp, dp, dp);
    x.C = W1; x.ldc = dp; x.C2 = W3; x.ldc2 = dp;
    x.flags = EF_STORE | EF_STORE_T | EF_NORM; x.partials = fd.partials;
    add_problem(c->nt[ST_XFORM], x, 2 * d * d * d);
    float* Pt;  // P^T, the K-major B of A P
    if (c->hp.series_order == 3) {
        // V = b X - e X X, stored transposed over A^4 (the K-major B of X V) ...
        GemmProblem v = product(W1, dp, W3, dp, dp, dp, dp);
        v.C2 = W2; v.ldc2 = dp; v.X = W1; v.ldx = dp; v.sc = fd.sc;
        v.flags = EF_STORE_T | EF_READX; v.coef = CO_VSER;
        add_problem(c->nt[ST_POLY], v, 2 * d * d * d);
        // ... then P = I - a X + X V, stored transposed over X^T.
        GemmProblem p = product(W1, dp, W2, dp, dp, dp, dp);
        p.C2 = W3; p.ldc2 = dp; p.X = W1; p.ldx = dp; p.sc = fd.sc;
        p.flags = EF_STORE_T | EF_READX; p.coef = CO_POLY3; p.valid_m = p.valid_n = F.d;
        add_problem(c->nt[ST_POLY2], p, 2 * d * d * d);
        Pt = W3;
    } else {
        // P = I - a X + b X X, stored transposed over A^4.
        GemmProblem p = product(W1, dp, W3, dp, dp, dp, dp);
        p.C2 = W2; p.ldc2 = dp; p.X = W1; p.ldx = dp; p.sc = fd.sc;
        p.flags = EF_STORE_T | EF_READX; p.coef = CO_POLY; p.valid_m = p.valid_n = F.d;
        add_problem(c->nt[ST_POLY], p, 2 * d * d * d);
        Pt = W2;
    }
    // Z = s A P, over X
    GemmProblem z = product(A, dp, Pt, dp, dp, dp, dp);
    z.C = W1; z.ldc = dp; z.sc = fd.sc; z.flags = EF_STORE; z.coef = CO_SCALE;
    add_problem(c->nt[ST_UPDATE], z, 2 * d * d * d);
    const int fi = (int)(&F - &c->factors[0]);
    for (int ti = 0; ti * 64 < dp; ++ti)
        for (int tj = ti; tj * 64 < dp; ++tj) c->sym_tiles.push_back({fi, ti, tj, 0});
}

// The products of one factor's update in the factored order (through H).
// Hr: H row-major (dp x kp, ld kp); Ht: H^T row-major (kp x dp, ld dp).
// Mo: the other factor's statistic when that factor is in the explicit order
// (H^T H is exactly it: G^T G for L_hat, G G^T for R_hat; kp x kp, ld kp,
// computed in the gram level and kept until the next step's), or null.
int add_factored(jorge_ctx* c, const FactorHost& F, const FactorDev& fd, const float* Hr, const float* Ht,
                 const float* Mo) {
    const bool sym = c->hp.symmetrize != 0;
    const int dp = F.dp, kp = F.kp;
    const double d = F.d, k = F.k;
    float* A = fd.A;
    float* P0 = at<float>(c, F.off_w[0]);
    float* P1 = at<float>(c, F.off_w[1]);
    float* Q = at<float>(c, F.off_w[2]);
    float* S = at<float>(c, F.off_w[3]);
    // Q = H^T H, unless the other factor's statistic already is.
    if (Mo) {
        Q = const_cast<float*>(Mo);
    } else {
        GemmProblem q = product(Ht, dp, Ht, dp, kp, kp, dp);
        q.C = Q; q.ldc = kp; q.flags = EF_STORE; q.upper = 1;
        add_problem(c->nt[ST_GRAM], q, k * k * d);
    }
    // Yt_4 = (A^4 H)^T is built in Yt4; A^5 H goes to Y5 (d x k) and W to Wb.
    float* Yt4;
    float* Y5;
    float* Wb;
    int last;  // level of A^5 H and nu
    if (!F.squared) {
        // Yt_{j+1} = Yt_j A^T, starting from Yt_0 = H^T: P0, P1, P0, P1.
        const float* src = Ht;
        float* dst[4] = {P0, P1, P0, P1};
        const int lvl[4] = {ST_GRAM, ST_POW4, ST_XFORM, ST_CHAIN4};
        for (int j = 0; j < 4; ++j) {
            GemmProblem y = product(src, dp, A, dp, kp, dp, dp);
            y.C = dst[j]; y.ldc = dp; y.flags = EF_STORE;
            if (j == 0 && F.lrp) {  // keep A H (= Yt_1^T) for the preconditioning
                y.C2 = at<float>(c, F.off_y1); y.ldc2 = kp; y.flags |= EF_STORE_T;
            }
            add_problem(c->nt[lvl[j]], y, 2 * k * d * d);
            src = dst[j];
        }
        Yt4 = P1; Y5 = P0; Wb = P1; last = ST_CHAIN5;
    } else {
        // Squared order: A^2 (symmetric), Yt_2 = H^T A^2 into P1, Yt_4 = Yt_2 A^2 into P0.
        float* A2 = at<float>(c, F.off_a2);
        GemmProblem a2 = product(A, dp, A, dp, dp, dp, dp);
        a2.C = A2; a2.ldc = dp; a2.flags = EF_STORE; a2.upper = 1;
        add_problem(c->nt[ST_GRAM], a2, d * d * d);
        if (F.lrp) {  // A H for the preconditioning, stored d x k
            GemmProblem y1 = product(Ht, dp, A, dp, kp, dp, dp);
            y1.C2 = at<float>(c, F.off_y1); y1.ldc2 = kp; y1.flags = EF_STORE_T;
            add_problem(c->nt[ST_GRAM], y1, 2 * k * d * d);
        }
        GemmProblem y2 = product(Ht, dp, A2, dp, kp, dp, dp);
        y2.C = P1; y2.ldc = dp; y2.flags = EF_STORE;
        add_problem(c->nt[ST_POW4], y2, 2 * k * d * d);
        GemmProblem y4 = product(P1, dp, A2, dp, kp, dp, dp);
        y4.C = P0; y4.ldc = dp; y4.flags = EF_STORE;
        add_problem(c->nt[ST_XFORM], y4, 2 * k * d * d);
        Yt4 = P0; Y5 = P1; Wb = P0; last = ST_CHAIN4;
    }
    // S = H^T A^4 H: Yt_2 Yt_2^T for symmetric factors (Yt_2 is in P1 at the xform level).
    if (sym) {
        GemmProblem s = product(P1, dp, P1, dp, kp, kp, dp);
        s.C = S; s.ldc = kp; s.flags = EF_STORE; s.upper = 1;
        add_problem(c->nt[ST_XFORM], s, k * k * d);
    }
    // A^5 H = (Yt_4 A^T)^T, stored d x k; ||X||^2 = <Yt_4 Yt_4^T, Q>.
    GemmProblem y5 = product(Yt4, dp, A, dp, kp, dp, dp);
    y5.C2 = Y5; y5.ldc2 = kp; y5.flags = EF_STORE_T;
    add_problem(c->nt[last], y5, 2 * k * d * d);
    GemmProblem nu = product(Yt4, dp, Yt4, dp, kp, kp, dp);
    nu.X = Q; nu.ldx = kp; nu.flags = EF_DOT; nu.upper = 1; nu.partials = fd.partials;
    const int slots = add_problem(c->nt[last], nu, k * k * d);
    // Literal mode (factored order only): S^T = U^T H = Yt_4 H (general).
    if (!sym) {
        GemmProblem s = product(Yt4, dp, Ht, dp, kp, kp, dp);
        s.C = S; s.ldc = kp; s.flags = EF_STORE;
        add_problem(c->nt[ST_CHAIN5], s, 2 * k * k * d);
    }
    // W = a A^5 H - b A^5 H S (B = S^T row-major), into Wb. With the cubic
    // term, W = a A^5 H - A^5 H V with V = b S - e S S (X^r = U S^(r-1) H^T),
    // one level later: V^T = b S^T - e S^T S^T (S^T symmetric, or the literal
    // mode's S^T as an MN-major B), then W.
    const bool cubic = c->hp.series_order == 3;
    const float* wb = S;
    if (cubic) {
        float* V = at<float>(c, F.off_s2);
        GemmProblem v = product(S, kp, S, kp, kp, kp, kp);
        v.C = V; v.ldc = kp; v.X = S; v.ldx = kp; v.sc = fd.sc;
        v.flags = EF_STORE | EF_READX; v.coef = CO_VSER; v.upper = sym;
        add_problem(sym ? c->nt[ST_POLY] : c->nn[ST_POLY], v, (sym ? 1 : 2) * k * k * k);
        wb = V;
    }
    GemmProblem w = product(Y5, kp, wb, kp, dp, kp, kp);
    w.C = Wb; w.ldc = kp; w.X = Y5; w.ldx = kp; w.sc = fd.sc;
    w.flags = EF_STORE | EF_READX; w.coef = cubic ? CO_WMIX3 : CO_WMIX;
    if (F.lrp) {  // and W^T for H^T W
        w.C2 = at<float>(c, F.off_wt); w.ldc2 = dp; w.flags |= EF_STORE_T;
    }
    add_problem(c->nt[cubic ? ST_POLY2 : ST_POLY], w, 2 * d * k * k);
    if (F.lrp) {
        // H^T W (k x k) in the update level, beside the SYR2K.
        GemmProblem v = product(Ht, dp, at<float>(c, F.off_wt), dp, kp, kp, dp);
        v.C = at<float>(c, F.off_v2t); v.ldc = kp; v.flags = EF_STORE;
        add_problem(c->nt[ST_UPDATE], v, 2 * k * k * d);
        // A_new H = s A H - (s/2)(W H^T H + H W^T H), in the first preconditioning level:
        // K segments [W | H] x [Q | (H^T W)^T]^T (Q is symmetric), coefficients of the SYR2K.
        GemmProblem x = product(Wb, kp, Q, kp, dp, kp, kp);
        x.A2 = Hr; x.lda2 = kp; x.B2 = at<float>(c, F.off_v2t); x.ldb2 = kp; x.K = 2 * kp;
        x.C = at<float>(c, F.off_xa); x.ldc = kp;
        x.X = at<float>(c, F.off_y1); x.ldx = kp; x.sc = fd.sc;
        x.flags = EF_STORE | EF_READX; x.coef = CO_SYR2K;
        add_problem(c->nt[ST_UPRECOND_L], x, 2 * d * k * 2 * k);
    }
    // A <- s A - (s/2)(W H^T + H W^T) (symmetric, in place) or s A - s W H^T.
    GemmProblem u = product(Wb, kp, Hr, kp, dp, dp, kp);
    u.C = A; u.ldc = dp; u.X = A; u.ldx = dp; u.sc = fd.sc; u.flags = EF_STORE | EF_READX;
    if (sym) {
        u.A2 = Hr; u.lda2 = kp; u.B2 = Wb; u.ldb2 = kp;
        u.K = 2 * kp;
        u.coef = CO_SYR2K;
        u.upper = 1;
        add_problem(c->nt[ST_UPDATE], u, d * d * 2 * k);
    } else {
        u.coef = CO_LITUPD;
        add_problem(c->nt[ST_UPDATE], u, 2 * d * d * k);
    }
    return slots;
}

// Fills the host-side launch tables (device pointers already known).
void build_tables(jorge_ctx* c, std::vector<LayerDev>& ld, std::vector<FactorDev>& fd) {
    const int nl = (int)c->layers.size();
    for (auto& F : c->factors) {
        FactorDev d{};
        d.A = at<float>(c, F.off_A);
        d.sc = at<FactorScalars>(c, F.off_sc);
        d.partials = at<double>(c, F.off_part);
        d.Z = (F.expl && !F.chain) ? at<float>(c, F.off_w[1]) : nullptr;
        const auto& L = c->layers[F.layer];
        d.H = at<float>(c, F.side == 0 ? L.off_Gp : L.off_Gpt);
        d.d = F.d;
        d.dp = F.dp;
        d.k = F.k;
        d.kp = F.kp;
        d.nparts = F.nparts;
        d.explicit_form = F.expl ? 1 : 0;
        fd.push_back(d);
    }
    for (int li = 0; li < nl; ++li) {
        auto& L = c->layers[li];
        LayerDev d{};
        d.Gp = at<float>(c, L.off_Gp);
        d.Gpt = at<float>(c, L.off_Gpt);
        d.T = at<float>(c, L.off_T);
        d.mom = at<float>(c, L.off_mom);
        d.msgd = at<float>(c, L.off_msgd);
        d.part_m = at<double>(c, L.off_part_m);
        d.part_sgd = at<double>(c, L.off_part_sgd);
        d.ls = at<LayerScalars>(c, L.off_ls);
        d.nonfinite = at<int>(c, c->off_nonfinite) + li;
        d.m = L.m; d.n = L.n; d.mp = L.mp; d.np = L.np;
        d.n_part_m = L.n_part_m;
        d.n_part_sgd = L.n_part_sgd;
        ld.push_back(d);
    }
    // Per-layer block lists, batched by kPtrBatch layers (user pointers go in kernel arguments).
    for (int li = 0; li < nl; ++li) {
        if (li % kPtrBatch == 0) {
            c->stage_batch_start.push_back((int)c->stage_tiles.size());
            c->flat_batch_start.push_back((int)c->flat_chunks.size());
        }
        const auto& L = c->layers[li];
        int slot = 0;
        for (int r = 0; r < L.m; r += 64)
            for (int q = 0; q < L.n; q += 64) c->stage_tiles.push_back({li, r, q, slot++});
        const int64_t total = (int64_t)L.m * L.n;
        for (int64_t st = 0; st < total; st += kFlatChunkElems)
            c->flat_chunks.push_back({li, (int)st, (int)std::min<int64_t>(kFlatChunkElems, total - st), 0});
    }
    c->stage_batch_start.push_back((int)c->stage_tiles.size());
    c->flat_batch_start.push_back((int)c->flat_chunks.size());

    // Factors in decreasing size, so large tiles come first within a stage.
    std::vector<int> order(c->factors.size());
    for (size_t i = 0; i < order.size(); ++i) order[i] = (int)i;
    std::stable_sort(order.begin(), order.end(),
                     [&](int a, int b) { return c->factors[a].dp > c->factors[b].dp; });
    for (int fi : order) {
        FactorHost& F = c->factors[fi];
        const LayerDev& l = ld[F.layer];
        // H row-major (d x k) and H^T row-major (k x d): G and G^T for L, the reverse for R.
        const float* Hr = F.side == 0 ? l.Gp : l.Gpt;
        const float* Ht = F.side == 0 ? l.Gpt : l.Gp;
        if (F.chain) {
            (F.dp <= kChainMax ? c->chain : c->chain2).push_back(fi);
            continue;
        }
        c->grouped.push_back(fi);
        if (F.expl) {
            add_explicit(c, F, fd[fi], Hr);
        } else {
            const auto& L = c->layers[F.layer];
            const FactorHost& O = c->factors[F.side == 0 ? L.fR : L.fL];
            // (The explicit factor keeps its statistic until the next step's gram level,
            // past the low-rank preconditioning that reads Q.)
            const float* Mo = (O.expl && !O.chain) ? at<float>(c, O.off_w[0]) : nullptr;
            F.nparts = add_factored(c, F, fd[fi], Hr, Ht, Mo);
            fd[fi].nparts = F.nparts;
        }
    }
    // Preconditioning, largest layers first.
    const bool sym = c->hp.symmetrize != 0;
    std::vector<int> lorder(nl);
    for (int i = 0; i < nl; ++i) lorder[i] = i;
    std::stable_sort(lorder.begin(), lorder.end(), [&](int a, int b) {
        return (int64_t)c->layers[a].mp * c->layers[a].np * (c->layers[a].mp + c->layers[a].np) >
               (int64_t)c->layers[b].mp * c->layers[b].np * (c->layers[b].mp + c->layers[b].np);
    });
    for (int li : lorder) {
        const auto& L = c->layers[li];
        const LayerDev& l = ld[li];
        const double m = L.m, n = L.n;
        const FactorHost& FL = c->factors[L.fL];
        const FactorHost& FR = c->factors[L.fR];
        // Non-update steps (and update steps of layers without a low-rank factor):
        // T = L_hat G (B^T = Gpt, both K-major), then G~ = T R_hat fused with the
        // momentum (R_hat is its own K-major B when symmetric).
        GemmProblem a = product(fd[L.fL].A, L.mp, l.Gpt, L.mp, L.mp, L.np, L.mp);
        a.C = l.T; a.ldc = L.np; a.flags = EF_STORE;
        GemmProblem b = product(l.T, L.np, fd[L.fR].A, L.np, L.mp, L.np, L.np);
        b.mom = l.mom; b.ldmom = L.n; b.partials = l.part_m;
        b.valid_m = L.m; b.valid_n = L.n; b.flags = EF_MOMENTUM;
        add_problem(c->nt[ST_PRECOND_L], a, 2 * m * m * n);
        add_problem(sym ? c->nt[ST_PRECOND_R] : c->nn[ST_PRECOND_R], b, 2 * m * n * n);
        if (FR.lrp) {
            // G R_new = (R_new G^T)^T is in the factor's x buffer (n x m); G~ = L_hat (G R_new).
            GemmProblem g = product(fd[L.fL].A, L.mp, at<float>(c, FR.off_xa), L.mp, L.mp, L.np, L.mp);
            g.mom = l.mom; g.ldmom = L.n; g.partials = l.part_m;
            g.valid_m = L.m; g.valid_n = L.n; g.flags = EF_MOMENTUM;
            add_problem(c->nt[ST_UPRECOND_R], g, 2 * m * m * n);
        } else if (FL.lrp) {
            // L_new G is in the factor's x buffer (m x n); G~ = (L_new G) R_hat.
            GemmProblem g = product(at<float>(c, FL.off_xa), L.np, fd[L.fR].A, L.np, L.mp, L.np, L.np);
            g.mom = l.mom; g.ldmom = L.n; g.partials = l.part_m;
            g.valid_m = L.m; g.valid_n = L.n; g.flags = EF_MOMENTUM;
            add_problem(c->nt[ST_UPRECOND_R], g, 2 * m * n * n);
        } else {
            add_problem(c->nt[ST_UPRECOND_L], a, 2 * m * m * n);
            add_problem(sym ? c->nt[ST_UPRECOND_R] : c->nn[ST_UPRECOND_R], b, 2 * m * n * n);
        }
    }
}

// Whether [p, p + bytes) lies inside one arena buffer.
bool in_buffer(const jorge_ctx* c, const void* p, int64_t bytes) {
    const char* q = static_cast<const char*>(p);
    if (bytes <= 0 || q < c->arena || q + bytes > c->arena + c->arena_bytes) return false;
    const size_t off = (size_t)(q - c->arena);
    auto it = std::upper_bound(c->regions.begin(), c->regions.end(), std::make_pair(off, SIZE_MAX));
    if (it == c->regions.begin()) return false;
    --it;
    return off + (size_t)bytes <= it->first + it->second;
}

bool aligned16(const void* p, int ld) { return (reinterpret_cast<uintptr_t>(p) & 15) == 0 && ld % 4 == 0; }

// Checks, on the host, that every access a grouped launch makes stays inside
// the buffer its pointer starts in and meets the kernel's alignment and
// extent assumptions (the tile loads and the vector stores of the epilogue).
// Returns an empty string, or a description of the first violation.
std::string check_stage(const jorge_ctx* c, const GemmStage& st, bool bk, const char* name) {
    auto fl = [](int64_t last) { return (last + 1) * (int64_t)sizeof(float); };
    for (size_t i = 0; i < st.probs.size(); ++i) {
        const GemmProblem& p = st.probs[i];
        const std::string where = std::string(name) + " problem " + std::to_string(i) + ": ";
        if (p.M <= 0 || p.N <= 0 || p.K <= 0 || p.M % 32 || p.N % 32 || p.K % kSlab || p.K1 % kSlab ||
            p.K1 <= 0 || p.K1 > p.K)
            return where + "extents";
        const int k1 = p.K1, k2 = p.K - p.K1;
        if (!aligned16(p.A, p.lda) || !in_buffer(c, p.A, fl((int64_t)(p.M - 1) * p.lda + k1 - 1)))
            return where + "A";
        const int64_t blast = bk ? (int64_t)(p.N - 1) * p.ldb + k1 - 1 : (int64_t)(k1 - 1) * p.ldb + p.N - 1;
        if (!aligned16(p.B, p.ldb) || !in_buffer(c, p.B, fl(blast))) return where + "B";
        if (k2 > 0) {
            if (!aligned16(p.A2, p.lda2) || !in_buffer(c, p.A2, fl((int64_t)(p.M - 1) * p.lda2 + k2 - 1)))
                return where + "A2";
            const int64_t b2 = bk ? (int64_t)(p.N - 1) * p.ldb2 + k2 - 1 : (int64_t)(k2 - 1) * p.ldb2 + p.N - 1;
            if (!aligned16(p.B2, p.ldb2) || !in_buffer(c, p.B2, fl(b2))) return where + "B2";
        }
        if (p.flags & EF_STORE) {
            int64_t last = (int64_t)(p.M - 1) * p.ldc + p.N - 1;
            if (p.upper) last = std::max(last, (int64_t)(p.N - 1) * p.ldc + p.M - 1);
            if ((p.upper && (p.M != p.N || !aligned16(p.C, p.ldc))) || !in_buffer(c, p.C, fl(last)))
                return where + "C";
        }
        if ((p.flags & EF_STORE_T) && (!aligned16(p.C2, p.ldc2) ||
                                       !in_buffer(c, p.C2, fl((int64_t)(p.N - 1) * p.ldc2 + p.M - 1))))
            return where + "C2";
        if ((p.flags & (EF_READX | EF_DOT)) && !in_buffer(c, p.X, fl((int64_t)(p.M - 1) * p.ldx + p.N - 1)))
            return where + "X";
        if ((p.flags & EF_READX) && (p.coef == CO_POLY || p.coef == CO_POLY3) &&
            (p.valid_m > p.M || p.valid_m > p.N))
            return where + "identity extent";
        if ((p.flags & EF_MOMENTUM) &&
            (p.valid_m > p.M || p.valid_n > p.N ||
             !in_buffer(c, p.mom, fl((int64_t)(p.valid_m - 1) * p.ldmom + p.valid_n - 1))))
            return where + "momentum";
        if (p.coef != CO_ONE && !in_buffer(c, p.sc, (int64_t)sizeof(FactorScalars))) return where + "scalars";
    }
    // Every tile of every problem is covered exactly once: whole, or by split
    // units whose K ranges tile [0, K) and whose parts match one fixup.
    std::vector<int> parts_seen(st.nparts, 0);
    std::vector<const TileDesc*> part_unit(st.nparts, nullptr);
    auto check_tile = [&](int prob, int tm, int tn, int slot) -> std::string {
        if (prob < 0 || prob >= (int)st.probs.size()) return std::string(name) + ": tile problem";
        const GemmProblem& p = st.probs[prob];
        if (tm < 0 || tn < 0 || tm >= tiles_of(p.M) || tn >= tiles_of(p.N) || (p.upper && tm > tn))
            return std::string(name) + ": tile index";
        if ((p.flags & (EF_NORM | EF_DOT | EF_MOMENTUM)) &&
            (slot < 0 || !in_buffer(c, p.partials, (int64_t)(slot + 1) * kWaveSlots * (int64_t)sizeof(double))))
            return std::string(name) + ": partial slot";
        return "";
    };
    // The products in small mode: those with blocks.
    std::vector<char> is_small(st.probs.size(), 0);
    for (const SmallUnit& u : st.small)
        if (u.prob >= 0 && u.prob < (int)st.probs.size()) is_small[u.prob] = 1;
    // Small-mode units: groups of 1 to 4 blocks, each block in exactly one group,
    // the group's K range that of its longest block.
    std::vector<int> small_seen(st.small.size(), 0);
    for (const TileDesc& t : st.tiles) {
        if (t.part != kSmallGroup) continue;
        if (!bk || t.tn < 1 || t.tn > kWaveSlots || t.tm < 0 || (size_t)t.tm + t.tn > st.small.size() || t.k0 != 0)
            return std::string(name) + ": small-mode group";
        int K = 0;
        for (int j = 0; j < t.tn; ++j) {
            if (small_seen[t.tm + j]++) return std::string(name) + ": small-mode block in two groups";
            const int pi = st.small[t.tm + j].prob;
            if (pi < 0 || pi >= (int)st.probs.size()) return std::string(name) + ": small-mode problem";
            K = std::max(K, st.probs[pi].K);
        }
        if (t.k1 != K) return std::string(name) + ": small-mode group K";
    }
    // Every block of every small-mode problem is computed once; with partial sums,
    // each tile's quadrants are computed or zeroed, never both.
    std::vector<std::vector<int>> blocks(st.probs.size()), quads(st.probs.size());
    for (size_t i = 0; i < st.small.size(); ++i) {
        if (!small_seen[i]) return std::string(name) + ": small-mode block in no group";
        const SmallUnit& u = st.small[i];
        const GemmProblem& p = st.probs[u.prob];
        const int bm_n = (p.M + kSmallDim - 1) / kSmallDim, bn_n = (p.N + kSmallDim - 1) / kSmallDim;
        const std::string e = check_tile(u.prob, u.bm / 2, u.bn / 2, u.slot);
        if (!e.empty()) return e;
        if (!small_eligible(st, p) || u.bm < 0 || u.bn < 0 || u.bm >= bm_n || u.bn >= bn_n || (p.upper && u.bm > u.bn) ||
            u.zero_mask < 0 || u.zero_mask >= (1 << kWaveSlots))
            return std::string(name) + ": small-mode block";
        auto& b = blocks[u.prob];
        if (b.empty()) b.assign((size_t)bm_n * bn_n, 0);
        if (b[(size_t)u.bm * bn_n + u.bn]++) return std::string(name) + ": small-mode block twice";
        if (p.flags & (EF_NORM | EF_DOT | EF_MOMENTUM)) {
            auto& q = quads[u.prob];
            const int tn_n = (int)tiles_of(p.N);
            if (q.empty()) q.assign((size_t)tiles_of(p.M) * tn_n, 0);
            int& m = q[(size_t)(u.bm / 2) * tn_n + u.bn / 2];
            const int mine = (1 << (((u.bm & 1) << 1) | (u.bn & 1))) | u.zero_mask;
            if (m & mine) return std::string(name) + ": small-mode partial sum written twice";
            m |= mine;
        }
    }
    for (size_t i = 0; i < st.probs.size(); ++i) {
        const GemmProblem& p = st.probs[i];
        if (!is_small[i]) continue;
        const int bm_n = (p.M + kSmallDim - 1) / kSmallDim, bn_n = (p.N + kSmallDim - 1) / kSmallDim;
        for (int bm = 0; bm < bm_n; ++bm)
            for (int bn = 0; bn < bn_n; ++bn)
                if ((!p.upper || bm <= bn) && (blocks[i].empty() || blocks[i][(size_t)bm * bn_n + bn] != 1))
                    return std::string(name) + ": small-mode coverage";
        if (p.flags & (EF_NORM | EF_DOT | EF_MOMENTUM)) {
            const int tm_n = (int)tiles_of(p.M), tn_n = (int)tiles_of(p.N);
            for (int tm = 0; tm < tm_n; ++tm)
                for (int tn = p.upper ? tm : 0; tn < tn_n; ++tn)
                    if (quads[i][(size_t)tm * tn_n + tn] != (1 << kWaveSlots) - 1)
                        return std::string(name) + ": small-mode partial sums";
        }
    }
    int64_t whole = 0, pieces = 0;
    for (const TileDesc& t : st.tiles) {
        if (t.part == kSmallGroup) continue;
        const std::string e = check_tile(t.prob, t.tm, t.tn, t.slot);
        if (!e.empty()) return e;
        const GemmProblem& p = st.probs[t.prob];
        if (t.k0 < 0 || t.k1 > p.K || t.k0 >= t.k1 || t.k0 % kSlab || t.k1 % kSlab)
            return std::string(name) + ": unit K range";
        if (t.part < 0) {
            if (t.k0 != 0 || t.k1 != p.K) return std::string(name) + ": whole tile K range";
            ++whole;
        } else {
            if (t.part >= st.nparts || parts_seen[t.part]++) return std::string(name) + ": split part";
            part_unit[t.part] = &t;
            ++pieces;
        }
    }
    for (const FixupDesc& f : st.fix) {
        const std::string e = check_tile(f.prob, f.tm, f.tn, f.slot);
        if (!e.empty()) return e;
        if (f.nsplit < 2 || f.part0 < 0 || f.part0 + f.nsplit > st.nparts) return std::string(name) + ": fixup";
        int k = 0;
        for (int q = 0; q < f.nsplit; ++q) {  // the parts are this tile's, in K order, covering [0, K)
            const TileDesc* u = part_unit[f.part0 + q];
            if (!u || u->prob != f.prob || u->tm != f.tm || u->tn != f.tn || u->slot != f.slot || u->k0 != k)
                return std::string(name) + ": fixup parts";
            k = u->k1;
        }
        if (k != st.probs[f.prob].K) return std::string(name) + ": fixup K coverage";
        pieces -= f.nsplit;
    }
    int64_t tiles_total = 0;
    for (size_t i = 0; i < st.probs.size(); ++i) {
        const GemmProblem& p = st.probs[i];
        if (is_small[i]) continue;
        const int64_t a = tiles_of(p.M), b = tiles_of(p.N);
        tiles_total += p.upper ? a * (a + 1) / 2 : a * b;
    }
    if (pieces != 0 || whole + (int64_t)st.fix.size() != tiles_total) return std::string(name) + ": coverage";
    return "";
}

std::string check_tables(const jorge_ctx* c, const std::vector<FactorDev>& fd) {
    for (int i = 0; i < ST_COUNT; ++i) {
        std::string e = check_stage(c, c->nt[i], true, kStageNames[i]);
        if (e.empty()) e = check_stage(c, c->nn[i], false, kStageNames[i]);
        if (!e.empty()) return e;
    }
    for (const SymTile& t : c->sym_tiles) {
        const FactorDev& F = fd[t.factor];
        const int64_t dd = (int64_t)F.dp * F.dp * (int64_t)sizeof(float);
        if (!F.Z || t.ti < 0 || t.ti > t.tj || t.tj * 64 >= F.dp || F.dp % 4 || !in_buffer(c, F.Z, dd) ||
            !in_buffer(c, F.A, dd))
            return "symmetrize tile";
    }
    for (const FactorDev& F : fd)
        if (!in_buffer(c, F.partials, (int64_t)F.nparts * kWaveSlots * (int64_t)sizeof(double)) || F.nparts < 1)
            return "factor partials";
    // The LDS chain kernels: A (dp x dp), H (dp x kp), scalars; dp <= 64 for
    // lds_chain_kernel, 64 < dp <= 128 (symmetric factors) for lds_chain128_kernel.
    for (int which = 0; which < 2; ++which)
        for (int fi : which ? c->chain2 : c->chain) {
            const FactorDev& F = fd[fi];
            const bool size_ok = which ? (F.dp > kChainMax && F.dp <= kChain2Max && c->hp.symmetrize)
                                       : F.dp <= kChainMax;
            if (!size_ok || F.dp % 32 || F.kp % kSlab || F.kp < kSlab ||
                !in_buffer(c, F.A, (int64_t)F.dp * F.dp * (int64_t)sizeof(float)) ||
                !in_buffer(c, F.H, (int64_t)F.dp * F.kp * (int64_t)sizeof(float)) ||
                !in_buffer(c, F.sc, (int64_t)sizeof(FactorScalars)))
                return "lds chain factor";
        }
    if (c->grouped.size() + c->chain.size() + c->chain2.size() != fd.size()) return "factor lists";
    return "";
}

// Layer list and arena offsets of a context (no device work).
jorge_status layout_context(jorge_ctx* c, const jorge_shape* shapes, int32_t num_layers) {
    try {
        c->layers.resize(num_layers);
        for (int32_t i = 0; i < num_layers; ++i) {
            LayerHost& L = c->layers[i];
            L.m = (int)shapes[i].rows;
            L.n = (int)shapes[i].cols;
            L.mp = (int)round_up(L.m, 32);
            L.np = (int)round_up(L.n, 32);
        }
        c->arena_bytes = plan(c);
    } catch (const std::bad_alloc&) {
        return JORGE_ERR_OUT_OF_MEMORY;
    }
    return JORGE_OK;
}

// Launch tables for the arena at c->arena, checked on the host.
jorge_status tables_context(jorge_ctx* c, std::vector<LayerDev>& ld, std::vector<FactorDev>& fd) {
    try {
        for (int i = 0; i < ST_COUNT; ++i) c->nt[i].kmajor_b = true;
        build_tables(c, ld, fd);
        for (int i = 0; i < ST_COUNT; ++i)
            for (GemmStage* st : {&c->nt[i], &c->nn[i]}) {
                make_small(*st);
                if (c->hp.split_k) split_stage(*st);
                order_for_xcds(st->tiles);
                c->splitws_blocks = std::max<int64_t>(c->splitws_blocks, st->nparts);
            }
        const std::string e = check_tables(c, fd);
        if (!e.empty()) return fail(c, JORGE_ERR_HIP, "launch table check failed: " + e);
    } catch (const std::bad_alloc&) {
        return JORGE_ERR_OUT_OF_MEMORY;
    }
    return JORGE_OK;
}

jorge_status validate_args(const jorge_shape* shapes, int32_t num_layers, const jorge_hparams* hp,
                           jorge_hparams* h) {
    if (!shapes || num_layers <= 0) return JORGE_ERR_INVALID_ARGUMENT;
    if (num_layers > JORGE_MAX_LAYERS) return JORGE_ERR_UNSUPPORTED;
    jorge_hparams_default(h);
    if (hp) *h = *hp;
    if (validate_hparams(h) != JORGE_OK) return JORGE_ERR_INVALID_ARGUMENT;
    for (int32_t i = 0; i < num_layers; ++i) {
        if (shapes[i].rows <= 0 || shapes[i].cols <= 0) return JORGE_ERR_INVALID_ARGUMENT;
        if (shapes[i].rows > JORGE_MAX_DIM || shapes[i].cols > JORGE_MAX_DIM) return JORGE_ERR_UNSUPPORTED;
    }
    return JORGE_OK;
}

template <typename T>
jorge_status upload(jorge_ctx* c, const std::vector<T>& v, T** dptr) {
    *dptr = nullptr;
    if (v.empty()) return JORGE_OK;
    const size_t bytes = v.size() * sizeof(T);
    if (c->pool) {  // stream-ordered copy into the lent pool; the caller keeps v alive until it is done
        if (c->pool_used + bytes > c->pool_bytes)
            return fail(c, JORGE_ERR_UNSUPPORTED, "launch tables exceed the scratch left for them");
        *dptr = reinterpret_cast<T*>(c->pool + c->pool_used);
        c->pool_used = (size_t)round_up((int64_t)(c->pool_used + bytes), kAlign);
        JORGE_HIP(c, hipMemcpyAsync(*dptr, v.data(), bytes, hipMemcpyHostToDevice, c->stream));
        return JORGE_OK;
    }
    JORGE_HIP(c, hipMalloc(reinterpret_cast<void**>(dptr), bytes));
    JORGE_HIP(c, hipMemcpy(*dptr, v.data(), bytes, hipMemcpyHostToDevice));
    return JORGE_OK;
}

// Bytes the device tables of a built context take, each rounded to kAlign.
template <typename T>
size_t table_bytes(const std::vector<T>& v) { return (size_t)round_up((int64_t)(v.size() * sizeof(T)), kAlign); }

jorge_status upload_stage(jorge_ctx* c, GemmStage& st) {
    jorge_status s = upload(c, st.probs, &st.dprobs);
    if (s != JORGE_OK) return s;
    if ((s = upload(c, st.fix, &st.dfix)) != JORGE_OK) return s;
    if ((s = upload(c, st.small, &st.dsmall)) != JORGE_OK) return s;
    return upload(c, st.tiles, &st.dtiles);
}

// Every device table of a context whose host tables are built.
jorge_status upload_tables(jorge_ctx* c, const std::vector<LayerDev>& ld, const std::vector<FactorDev>& fd) {
    jorge_status st;
    if ((st = upload(c, ld, &c->dlayers)) != JORGE_OK) return st;
    if ((st = upload(c, fd, &c->dfactors)) != JORGE_OK) return st;
    if ((st = upload(c, c->stage_tiles, &c->dstage)) != JORGE_OK) return st;
    if ((st = upload(c, c->flat_chunks, &c->dflat)) != JORGE_OK) return st;
    if ((st = upload(c, c->sym_tiles, &c->dsym)) != JORGE_OK) return st;
    if ((st = upload(c, c->grouped, &c->dgrouped)) != JORGE_OK) return st;
    if ((st = upload(c, c->chain, &c->dchain)) != JORGE_OK) return st;
    if ((st = upload(c, c->chain2, &c->dchain2)) != JORGE_OK) return st;
    for (int i = 0; i < ST_COUNT; ++i)
        for (GemmStage* s : {&c->nt[i], &c->nn[i]})
            if ((st = upload_stage(c, *s)) != JORGE_OK) return st;
    return JORGE_OK;
}

// What upload_tables places in a lent pool.
size_t tables_bytes(const jorge_ctx* c, const std::vector<LayerDev>& ld, const std::vector<FactorDev>& fd) {
    size_t b = table_bytes(ld) + table_bytes(fd) + table_bytes(c->stage_tiles) + table_bytes(c->flat_chunks) +
               table_bytes(c->sym_tiles) + table_bytes(c->grouped) + table_bytes(c->chain) +
               table_bytes(c->chain2);
    for (int i = 0; i < ST_COUNT; ++i)
        for (const GemmStage* s : {&c->nt[i], &c->nn[i]})
            b += table_bytes(s->probs) + table_bytes(s->fix) + table_bytes(s->small) + table_bytes(s->tiles);
    return b;
}

void free_ctx(jorge_ctx* c) {
    if (!c) return;
    if (c->lent) {
        delete c;
        return;
    }
    for (int i = 0; i < ST_COUNT; ++i)
        for (GemmStage* st : {&c->nt[i], &c->nn[i]}) {
            if (st->dprobs) (void)hipFree(st->dprobs);
            if (st->dtiles) (void)hipFree(st->dtiles);
            if (st->dsmall) (void)hipFree(st->dsmall);
            if (st->dfix) (void)hipFree(st->dfix);
        }
    if (c->splitws) (void)hipFree(c->splitws);
    if (c->dlayers) (void)hipFree(c->dlayers);
    if (c->dfactors) (void)hipFree(c->dfactors);
    if (c->dstage) (void)hipFree(c->dstage);
    if (c->dflat) (void)hipFree(c->dflat);
    if (c->dsym) (void)hipFree(c->dsym);
    if (c->dgrouped) (void)hipFree(c->dgrouped);
    if (c->dchain) (void)hipFree(c->dchain);
    if (c->dchain2) (void)hipFree(c->dchain2);
    if (c->arena) (void)hipFree(c->arena);
    for (auto& l : c->pending) {
        (void)hipEventDestroy(l.start);
        (void)hipEventDestroy(l.stop);
    }
    for (auto e : c->free_events) (void)hipEventDestroy(e);
    if (c->order_event) (void)hipEventDestroy(c->order_event);
    delete c;
}

jorge_status launch_stage(jorge_ctx* c, int stage, float beta1) {
    jorge_status s = launch_gemm<true, true>(c, c->nt[stage], stage, beta1);
    if (s != JORGE_OK) return s;
    return launch_gemm<true, false>(c, c->nn[stage], stage, beta1);
}

jorge_status run_update(jorge_ctx* c, double beta2) {
    jorge_status s;
    // The LDS chains: every factor of the context (the levels below are then empty).
    if (!c->chain2.empty()) {
        TimedLaunch tl(c, ST_LDS_CHAIN);
        hipLaunchKernelGGL(lds_chain128_kernel, dim3((unsigned)c->chain2.size()), dim3(kC2Threads), 0, c->stream,
                           c->dfactors, c->dchain2, beta2, (int)c->hp.beta_mode, (int)c->hp.series_order);
        tl.finish();
        JORGE_HIP(c, hipGetLastError());
    }
    if (!c->chain.empty()) {
        TimedLaunch tl(c, ST_LDS_CHAIN);
        hipLaunchKernelGGL(lds_chain_kernel, dim3((unsigned)c->chain.size()), dim3(kGemmThreads), 0, c->stream,
                           c->dfactors, c->dchain, beta2, (int)c->hp.beta_mode, (int)c->hp.symmetrize,
                           (int)c->hp.series_order);
        tl.finish();
        JORGE_HIP(c, hipGetLastError());
    }
    for (int lv : kLevels) {
        if (lv == ST_POLY && !c->grouped.empty()) {  // every grouped factor's nu is complete after chain5
            TimedLaunch tl(c, ST_FFINAL);
            hipLaunchKernelGGL(factor_finalize_kernel, dim3((unsigned)c->grouped.size()), dim3(64), 0,
                               c->stream, c->dfactors, c->dgrouped, beta2, (int)c->hp.beta_mode);
            tl.finish();
            JORGE_HIP(c, hipGetLastError());
        }
        if ((s = launch_stage(c, lv, 0.f)) != JORGE_OK) return s;
    }
    if (!c->sym_tiles.empty()) {
        TimedLaunch tl(c, ST_SYMM);
        hipLaunchKernelGGL(symmetrize_kernel, dim3((unsigned)c->sym_tiles.size()), dim3(kEwThreads), 0,
                           c->stream, c->dfactors, c->dsym, (int)c->hp.symmetrize);
        tl.finish();
        JORGE_HIP(c, hipGetLastError());
    }
    return JORGE_OK;
}

// jorge_step_noalloc: per device, the scratch's device address (set on the
// first call on that device) and the lock that serialises calls.
constexpr int kMaxDevices = 64;
struct NoallocDevice {
    std::mutex mu;
    char* base = nullptr;
};
NoallocDevice g_noalloc[kMaxDevices];

// The launches of step t (everything jorge_step queues after validating).
jorge_status launch_step(jorge_ctx* c, float* const* params, const float* const* grads, int64_t t, double lr,
                         double beta2, double beta1, double weight_decay) {
    const int nl = (int)c->layers.size();
    const bool update = (t - 1) % c->hp.precond_interval == 0;
    const int nbatch = (nl + kPtrBatch - 1) / kPtrBatch;
    for (int b = 0; b < nbatch; ++b) {
        PtrBatch pb{};
        for (int i = b * kPtrBatch; i < std::min(nl, (b + 1) * kPtrBatch); ++i) pb.p[i - b * kPtrBatch] = grads[i];
        const int c0 = c->stage_batch_start[b], c1 = c->stage_batch_start[b + 1];
        TimedLaunch tl(c, ST_STAGEIN);
        hipLaunchKernelGGL(stagein_kernel, dim3(c1 - c0), dim3(kEwThreads), 0, c->stream, c->dlayers,
                           c->dstage + c0, b * kPtrBatch, pb, (float)beta1);
        tl.finish();
        JORGE_HIP(c, hipGetLastError());
    }
    jorge_status s;
    if (update && (s = run_update(c, beta2)) != JORGE_OK) return s;
    // Update steps take the preconditioning tables that reuse the update's low-rank terms.
    if ((s = launch_stage(c, update ? ST_UPRECOND_L : ST_PRECOND_L, 0.f)) != JORGE_OK) return s;
    if ((s = launch_stage(c, update ? ST_UPRECOND_R : ST_PRECOND_R, (float)beta1)) != JORGE_OK) return s;
    {
        TimedLaunch tl(c, ST_LFINAL);
        hipLaunchKernelGGL(layer_finalize_kernel, dim3(nl), dim3(64), 0, c->stream, c->dlayers, lr,
                           weight_decay, (int)c->hp.graft);
        tl.finish();
        JORGE_HIP(c, hipGetLastError());
    }
    for (int b = 0; b < nbatch; ++b) {
        MutPtrBatch pb{};
        for (int i = b * kPtrBatch; i < std::min(nl, (b + 1) * kPtrBatch); ++i) pb.p[i - b * kPtrBatch] = params[i];
        const int c0 = c->flat_batch_start[b], c1 = c->flat_batch_start[b + 1];
        TimedLaunch tl(c, ST_WEIGHT);
        hipLaunchKernelGGL(weight_kernel, dim3(c1 - c0), dim3(kEwThreads), 0, c->stream, c->dlayers,
                           c->dflat + c0, b * kPtrBatch, pb);
        tl.finish();
        JORGE_HIP(c, hipGetLastError());
    }
    return JORGE_OK;
}


bool valid_kind(const jorge_ctx* c, int32_t layer, int32_t kind) {
    return c && layer >= 0 && layer < (int32_t)c->layers.size() && kind >= JORGE_STATE_L &&
           kind <= JORGE_STATE_MOM_SGD;
}

// Device pointer, rows, cols and row stride of one state tensor.
void state_view(jorge_ctx* c, int32_t layer, int32_t kind, float** p, int64_t* rows, int64_t* cols,
                int64_t* ld) {
    const auto& L = c->layers[layer];
    if (kind == JORGE_STATE_L || kind == JORGE_STATE_R) {
        const auto& F = c->factors[kind == JORGE_STATE_L ? L.fL : L.fR];
        *p = at<float>(c, F.off_A);
        *rows = *cols = F.d;
        *ld = F.dp;
    } else {
        *p = at<float>(c, kind == JORGE_STATE_MOM ? L.off_mom : L.off_msgd);
        *rows = L.m;
        *cols = L.n;
        *ld = L.n;
    }
}

}  // namespace

extern "C" {

jorge_status jorge_hparams_default(jorge_hparams* hp) {
    if (!hp) return JORGE_ERR_INVALID_ARGUMENT;
    hp->eps = 1e-6;
    hp->precond_interval = 1;
    hp->beta_mode = JORGE_BETA_CLAMPED;
    hp->graft = 1;
    hp->symmetrize = 1;
    hp->factor_form = JORGE_FORM_AUTO;
    hp->split_k = 1;
    hp->lds_chain_max = kChain2Max;
    hp->precond_lowrank = 1;
    hp->series_order = 2;
    return JORGE_OK;
}

jorge_status jorge_create(const jorge_shape* shapes, int32_t num_layers, const jorge_hparams* hp,
                          void* hip_stream, jorge_ctx** out) {
    if (!out) return JORGE_ERR_INVALID_ARGUMENT;
    *out = nullptr;
    jorge_hparams h;
    jorge_status st = validate_args(shapes, num_layers, hp, &h);
    if (st != JORGE_OK) return st;
    jorge_ctx* c = new (std::nothrow) jorge_ctx();
    if (!c) return JORGE_ERR_OUT_OF_MEMORY;
    c->hp = h;
    c->stream = reinterpret_cast<hipStream_t>(hip_stream);
    auto bail = [&](jorge_status s) {
        free_ctx(c);
        return s;
    };
    if ((st = layout_context(c, shapes, num_layers)) != JORGE_OK) return bail(st);
    if (hipGetDevice(&c->device) != hipSuccess) return bail(JORGE_ERR_HIP);
    // As in hip_fail: the failed allocation's error leaves the last-error state.
    auto alloc_failed = [&](hipError_t err) {
        (void)hipGetLastError();
        return bail(err == hipErrorOutOfMemory ? JORGE_ERR_OUT_OF_MEMORY : JORGE_ERR_HIP);
    };
    hipError_t e = hipMalloc(reinterpret_cast<void**>(&c->arena), c->arena_bytes);
    if (e != hipSuccess) return alloc_failed(e);
    if (hipMemsetAsync(c->arena, 0, c->arena_bytes, c->stream) != hipSuccess) return bail(JORGE_ERR_HIP);
    std::vector<LayerDev> ld;
    std::vector<FactorDev> fd;
    if ((st = tables_context(c, ld, fd)) != JORGE_OK) return bail(st);
    if (c->splitws_blocks > 0) {
        e = hipMalloc(reinterpret_cast<void**>(&c->splitws), (size_t)c->splitws_blocks * kSplitBlock * sizeof(float));
        if (e != hipSuccess) return alloc_failed(e);
    }
    if ((st = upload_tables(c, ld, fd)) != JORGE_OK) return bail(st);
    hipLaunchKernelGGL(init_factors_kernel, dim3((unsigned)c->factors.size()), dim3(256), 0, c->stream,
                       c->dfactors, (float)std::pow(h.eps, -0.25));
    if (hipGetLastError() != hipSuccess) return bail(JORGE_ERR_HIP);
    if (hipStreamSynchronize(c->stream) != hipSuccess) return bail(JORGE_ERR_HIP);
    *out = c;
    return JORGE_OK;
}

// Lays out and builds the tables of a context on the host only (jorge_plan,
// jorge_plan_stages); on success *out owns a context with no device memory.
jorge_status plan_only(const jorge_shape* shapes, int32_t num_layers, const jorge_hparams* hp, jorge_ctx** out) {
    *out = nullptr;
    jorge_hparams h;
    jorge_status st = validate_args(shapes, num_layers, hp, &h);
    if (st != JORGE_OK) return st;
    jorge_ctx* c = new (std::nothrow) jorge_ctx();
    if (!c) return JORGE_ERR_OUT_OF_MEMORY;
    c->hp = h;
    std::vector<LayerDev> ld;
    std::vector<FactorDev> fd;
    if ((st = layout_context(c, shapes, num_layers)) == JORGE_OK) {
        // Tables against a stand-in base address: pointers are only compared, never used.
        c->arena = reinterpret_cast<char*>(uintptr_t(1) << 44);
        st = tables_context(c, ld, fd);
        c->arena = nullptr;
    }
    if (st != JORGE_OK) {
        delete c;
        return st;
    }
    *out = c;
    return JORGE_OK;
}

jorge_status jorge_plan(const jorge_shape* shapes, int32_t num_layers, const jorge_hparams* hp,
                        int64_t* arena_bytes) {
    if (!arena_bytes) return JORGE_ERR_INVALID_ARGUMENT;
    jorge_ctx* c = nullptr;
    const jorge_status st = plan_only(shapes, num_layers, hp, &c);
    if (st != JORGE_OK) return st;
    *arena_bytes = (int64_t)c->arena_bytes + c->splitws_blocks * kSplitBlock * (int64_t)sizeof(float);
    delete c;
    return JORGE_OK;
}

jorge_status jorge_plan_stages(const jorge_shape* shapes, int32_t num_layers, const jorge_hparams* hp,
                               int64_t* units, int64_t* split_tiles, int64_t* small_blocks, int32_t n) {
    if (n < 0 || (n > 0 && !units && !split_tiles && !small_blocks)) return JORGE_ERR_INVALID_ARGUMENT;
    jorge_ctx* c = nullptr;
    const jorge_status st = plan_only(shapes, num_layers, hp, &c);
    if (st != JORGE_OK) return st;
    for (int i = 0; i < std::min<int>(n, ST_COUNT); ++i) {
        if (units) units[i] = (int64_t)c->nt[i].tiles.size() + (int64_t)c->nn[i].tiles.size();
        if (split_tiles) split_tiles[i] = (int64_t)c->nt[i].fix.size() + (int64_t)c->nn[i].fix.size();
        if (small_blocks) small_blocks[i] = (int64_t)c->nt[i].small.size() + (int64_t)c->nn[i].small.size();
    }
    delete c;
    return JORGE_OK;
}

jorge_status jorge_step(jorge_ctx* c, float* const* params, const float* const* grads, double lr,
                        double beta2, double beta1, double weight_decay) {
    if (!c || !params || !grads) return JORGE_ERR_INVALID_ARGUMENT;
    if (!(std::isfinite(lr) && lr >= 0.0) || !(beta2 > 0.0 && beta2 < 1.0) ||
        !(beta1 >= 0.0 && beta1 < 1.0) || !(std::isfinite(weight_decay) && weight_decay >= 0.0))
        return fail(c, JORGE_ERR_INVALID_ARGUMENT, "jorge_step: hyperparameter out of range");
    const int nl = (int)c->layers.size();
    for (int i = 0; i < nl; ++i)
        if (!params[i] || !grads[i]) return fail(c, JORGE_ERR_INVALID_ARGUMENT, "jorge_step: null tensor");
    if (c->poisoned)
        return fail(c, JORGE_ERR_HIP,
                    "jorge_step: an earlier step failed part-way; restore the state (jorge_set_state) and "
                    "the step counter (jorge_set_step) first");
    const int64_t t = c->t + 1;
    const jorge_status s = launch_step(c, params, grads, t, lr, beta2, beta1, weight_decay);
    if (s != JORGE_OK) {
        c->poisoned = true;
        return s;
    }
    c->t = t;
    return JORGE_OK;
}

jorge_status jorge_step_noalloc(const jorge_shape* shape, const jorge_hparams* hp, int64_t t, float* theta,
                                const float* grad, float* L, float* R, float* mom, float* mom_sgd, double lr,
                                double beta2, double beta1, double weight_decay, void* hip_stream) {
    jorge_hparams h;
    jorge_status st = validate_args(shape, 1, hp, &h);
    if (st != JORGE_OK) return st;
    if (t < 1 || !theta || !grad || !L || !R || !mom || !mom_sgd) return JORGE_ERR_INVALID_ARGUMENT;
    if (!(std::isfinite(lr) && lr >= 0.0) || !(beta2 > 0.0 && beta2 < 1.0) || !(beta1 >= 0.0 && beta1 < 1.0) ||
        !(std::isfinite(weight_decay) && weight_decay >= 0.0))
        return JORGE_ERR_INVALID_ARGUMENT;
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) return JORGE_ERR_HIP;
    // One call at a time per device: the scratch is shared.
    std::lock_guard<std::mutex> lock(g_noalloc[dev].mu);
    if (!g_noalloc[dev].base) {
        void* ptr = nullptr;
        if (hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch)) != hipSuccess || !ptr) return JORGE_ERR_HIP;
        g_noalloc[dev].base = static_cast<char*>(ptr);
    }
    char* const base = g_noalloc[dev].base;
    jorge_ctx* c = new (std::nothrow) jorge_ctx();
    if (!c) return JORGE_ERR_OUT_OF_MEMORY;
    struct Owner {  // on every return: waits for queued work (it reads c's host tables), frees c
        jorge_ctx* c;
        bool synced = false;
        ~Owner() {
            if (c->lent && !synced) (void)hipStreamSynchronize(c->stream);
            free_ctx(c);  // host side only: every device pointer of c lies in the scratch
        }
    } owner{c};
    c->hp = h;
    c->stream = reinterpret_cast<hipStream_t>(hip_stream);
    c->device = dev;
    if ((st = layout_context(c, shape, 1)) != JORGE_OK) return st;
    // Everything below lies in the scratch: the arena at its start, then the
    // split workspace, then the launch tables.
    c->lent = true;
    c->arena = base;
    std::vector<LayerDev> ld;
    std::vector<FactorDev> fd;
    if ((st = tables_context(c, ld, fd)) != JORGE_OK) return st;
    const size_t arena = (size_t)round_up((int64_t)c->arena_bytes, kAlign);
    const size_t split = (size_t)round_up(c->splitws_blocks * kSplitBlock * (int64_t)sizeof(float), kAlign);
    const size_t need = arena + split + tables_bytes(c, ld, fd);
    if (need > (size_t)JORGE_NOALLOC_SCRATCH_BYTES) {
        char msg[160];
        std::snprintf(msg, sizeof msg, "jorge_step_noalloc: a %lld x %lld layer needs %zu bytes of scratch, above %lld",
                      (long long)shape->rows, (long long)shape->cols, need, (long long)JORGE_NOALLOC_SCRATCH_BYTES);
        return fail(c, JORGE_ERR_UNSUPPORTED, msg);
    }
    c->splitws = c->splitws_blocks > 0 ? reinterpret_cast<float*>(base + arena) : nullptr;
    c->pool = base + arena + split;
    c->pool_bytes = JORGE_NOALLOC_SCRATCH_BYTES - arena - split;
    // The scratch keeps the last call's contents: the arena's padding and
    // partial sums must start at zero.
    const size_t words = c->arena_bytes / 16;
    hipLaunchKernelGGL(zero_kernel, dim3((unsigned)std::min<size_t>((words + kEwThreads - 1) / kEwThreads, 4096)),
                       dim3(kEwThreads), 0, c->stream, reinterpret_cast<f32x4*>(base), words);
    JORGE_HIP(c, hipGetLastError());
    if ((st = upload_tables(c, ld, fd)) != JORGE_OK) return st;
    // The caller's state in (dense row-major) and, after the step, out.
    const auto& Lh = c->layers[0];
    const int m = Lh.m, n = Lh.n;
    float* const A[2] = {at<float>(c, c->factors[Lh.fL].off_A), at<float>(c, c->factors[Lh.fR].off_A)};
    float* const U[2] = {L, R};
    const int dims[2] = {m, n}, lds[2] = {Lh.mp, Lh.np};
    float* const mm = at<float>(c, Lh.off_mom);
    float* const ms = at<float>(c, Lh.off_msgd);
    const size_t mn = (size_t)m * n * sizeof(float);
    for (int s = 0; s < 2; ++s)
        JORGE_HIP(c, hipMemcpy2DAsync(A[s], lds[s] * sizeof(float), U[s], dims[s] * sizeof(float),
                                      dims[s] * sizeof(float), dims[s], hipMemcpyDeviceToDevice, c->stream));
    JORGE_HIP(c, hipMemcpyAsync(mm, mom, mn, hipMemcpyDeviceToDevice, c->stream));
    JORGE_HIP(c, hipMemcpyAsync(ms, mom_sgd, mn, hipMemcpyDeviceToDevice, c->stream));
    float* const params[1] = {theta};
    const float* const grads[1] = {grad};
    if ((st = launch_step(c, params, grads, t, lr, beta2, beta1, weight_decay)) != JORGE_OK) return st;
    for (int s = 0; s < 2; ++s)
        JORGE_HIP(c, hipMemcpy2DAsync(U[s], dims[s] * sizeof(float), A[s], lds[s] * sizeof(float),
                                      dims[s] * sizeof(float), dims[s], hipMemcpyDeviceToDevice, c->stream));
    JORGE_HIP(c, hipMemcpyAsync(mom, mm, mn, hipMemcpyDeviceToDevice, c->stream));
    JORGE_HIP(c, hipMemcpyAsync(mom_sgd, ms, mn, hipMemcpyDeviceToDevice, c->stream));
    // The host tables the copies above read, and the scratch, are reused once this returns.
    JORGE_HIP(c, hipStreamSynchronize(c->stream));
    owner.synced = true;
    return JORGE_OK;
}

jorge_status jorge_get_state(jorge_ctx* c, int32_t layer, int32_t kind, float* dst, int64_t ld_dst) {
    if (!valid_kind(c, layer, kind) || !dst) return JORGE_ERR_INVALID_ARGUMENT;
    float* p;
    int64_t rows, cols, ld;
    state_view(c, layer, kind, &p, &rows, &cols, &ld);
    if (ld_dst < cols) return fail(c, JORGE_ERR_INVALID_ARGUMENT, "jorge_get_state: ld_dst < cols");
    JORGE_HIP(c, hipMemcpy2DAsync(dst, ld_dst * sizeof(float), p, ld * sizeof(float), cols * sizeof(float),
                                  rows, hipMemcpyDeviceToDevice, c->stream));
    return JORGE_OK;
}

jorge_status jorge_set_state(jorge_ctx* c, int32_t layer, int32_t kind, const float* src, int64_t ld_src) {
    if (!valid_kind(c, layer, kind) || !src) return JORGE_ERR_INVALID_ARGUMENT;
    float* p;
    int64_t rows, cols, ld;
    state_view(c, layer, kind, &p, &rows, &cols, &ld);
    if (ld_src < cols) return fail(c, JORGE_ERR_INVALID_ARGUMENT, "jorge_set_state: ld_src < cols");
    if ((kind == JORGE_STATE_L || kind == JORGE_STATE_R) && ld > cols) {
        // A factor's padding rows and columns must hold zeros, which the step
        // keeps; a step that met a non-finite value filled them with it
        // (0 * NaN), so a restored factor gets them cleared too.
        const size_t words = (size_t)ld * ld / 4;
        hipLaunchKernelGGL(zero_kernel, dim3((unsigned)std::min<size_t>((words + kEwThreads - 1) / kEwThreads, 4096)),
                           dim3(kEwThreads), 0, c->stream, reinterpret_cast<f32x4*>(p), words);
        JORGE_HIP(c, hipGetLastError());
    }
    JORGE_HIP(c, hipMemcpy2DAsync(p, ld * sizeof(float), src, ld_src * sizeof(float), cols * sizeof(float),
                                  rows, hipMemcpyDeviceToDevice, c->stream));
    return JORGE_OK;
}

jorge_status jorge_state_ptr(jorge_ctx* c, int32_t layer, int32_t kind, float** dev_ptr, int64_t* ld) {
    if (!valid_kind(c, layer, kind) || !dev_ptr || !ld) return JORGE_ERR_INVALID_ARGUMENT;
    int64_t rows, cols;
    state_view(c, layer, kind, dev_ptr, &rows, &cols, ld);
    return JORGE_OK;
}

jorge_status jorge_get_step(const jorge_ctx* c, int64_t* t) {
    if (!c || !t) return JORGE_ERR_INVALID_ARGUMENT;
    *t = c->t;
    return JORGE_OK;
}

jorge_status jorge_set_step(jorge_ctx* c, int64_t t) {
    if (!c || t < 0) return JORGE_ERR_INVALID_ARGUMENT;
    c->t = t;
    c->poisoned = false;
    return JORGE_OK;
}

jorge_status jorge_read_diag(jorge_ctx* c, int32_t layer, double* out) {
    if (!c || !out || layer < 0 || layer >= (int32_t)c->layers.size()) return JORGE_ERR_INVALID_ARGUMENT;
    const auto& L = c->layers[layer];
    FactorScalars fl, fr;
    LayerScalars ls;
    JORGE_HIP(c, hipMemcpyAsync(&fl, at<FactorScalars>(c, c->factors[L.fL].off_sc), sizeof(fl),
                                hipMemcpyDeviceToHost, c->stream));
    JORGE_HIP(c, hipMemcpyAsync(&fr, at<FactorScalars>(c, c->factors[L.fR].off_sc), sizeof(fr),
                                hipMemcpyDeviceToHost, c->stream));
    JORGE_HIP(c, hipMemcpyAsync(&ls, at<LayerScalars>(c, L.off_ls), sizeof(ls), hipMemcpyDeviceToHost,
                                c->stream));
    JORGE_HIP(c, hipStreamSynchronize(c->stream));
    out[JORGE_DIAG_NU_L] = fl.nu;
    out[JORGE_DIAG_NU_R] = fr.nu;
    out[JORGE_DIAG_BETA_L] = fl.beta;
    out[JORGE_DIAG_BETA_R] = fr.beta;
    out[JORGE_DIAG_NORM_M] = ls.norm_m;
    out[JORGE_DIAG_NORM_SGD] = ls.norm_sgd;
    out[JORGE_DIAG_STEP] = ls.g;
    return JORGE_OK;
}

jorge_status jorge_nonfinite(jorge_ctx* c, int32_t* count, int32_t* first) {
    if (!c || !count) return JORGE_ERR_INVALID_ARGUMENT;
    const size_t nl = c->layers.size(), words = (nl + 3) / 4;
    std::vector<int> flags;
    try {
        flags.assign(nl, 0);
    } catch (const std::bad_alloc&) {
        return JORGE_ERR_OUT_OF_MEMORY;
    }
    // Read, then clear behind the read on the same stream.
    JORGE_HIP(c, hipMemcpyAsync(flags.data(), at<int>(c, c->off_nonfinite), nl * sizeof(int), hipMemcpyDeviceToHost,
                                c->stream));
    hipLaunchKernelGGL(zero_kernel, dim3((unsigned)((words + kEwThreads - 1) / kEwThreads)), dim3(kEwThreads), 0,
                       c->stream, at<f32x4>(c, c->off_nonfinite), words);
    JORGE_HIP(c, hipGetLastError());
    JORGE_HIP(c, hipStreamSynchronize(c->stream));
    int32_t n = 0, f = -1;
    for (size_t i = 0; i < nl; ++i)
        if (flags[i]) {
            if (f < 0) f = (int32_t)i;
            ++n;
        }
    *count = n;
    if (first) *first = f;
    return JORGE_OK;
}

jorge_status jorge_set_stream(jorge_ctx* c, void* hip_stream) {
    if (!c) return JORGE_ERR_INVALID_ARGUMENT;
    const hipStream_t s = reinterpret_cast<hipStream_t>(hip_stream);
    if (s == c->stream) return JORGE_OK;
    // Work queued later on the new stream waits for all work already queued
    // on the old one. Not when either stream is being captured into a graph:
    // a capture cannot wait on an event recorded outside it, nor the reverse,
    // and the capture's owner orders the streams (torch.cuda.graph
    // synchronises the device before it starts capturing).
    hipStreamCaptureStatus cap_new = hipStreamCaptureStatusNone, cap_old = hipStreamCaptureStatusNone;
    JORGE_HIP(c, hipStreamIsCapturing(s, &cap_new));
    if (cap_new == hipStreamCaptureStatusNone && hipStreamIsCapturing(c->stream, &cap_old) == hipSuccess &&
        cap_old == hipStreamCaptureStatusNone) {
        if (!c->order_event) JORGE_HIP(c, hipEventCreateWithFlags(&c->order_event, hipEventDisableTiming));
        JORGE_HIP(c, hipEventRecord(c->order_event, c->stream));
        JORGE_HIP(c, hipStreamWaitEvent(s, c->order_event, 0));
    }
    c->stream = s;
    return JORGE_OK;
}

jorge_status jorge_synchronize(jorge_ctx* c) {
    if (!c) return JORGE_ERR_INVALID_ARGUMENT;
    JORGE_HIP(c, hipStreamSynchronize(c->stream));
    return JORGE_OK;
}

jorge_status jorge_device_bytes(const jorge_ctx* c, int64_t* bytes) {
    if (!c || !bytes) return JORGE_ERR_INVALID_ARGUMENT;
    *bytes = (int64_t)c->arena_bytes + c->splitws_blocks * kSplitBlock * (int64_t)sizeof(float);
    return JORGE_OK;
}

jorge_status jorge_set_timing(jorge_ctx* c, int32_t enable) {
    if (!c || (enable != 0 && enable != 1)) return JORGE_ERR_INVALID_ARGUMENT;
    c->timing = enable != 0;
    return JORGE_OK;
}

jorge_status jorge_read_timing(jorge_ctx* c, double* ms, int64_t* launches, int32_t n) {
    if (!c || n < 0) return JORGE_ERR_INVALID_ARGUMENT;
    for (auto& l : c->pending) {
        JORGE_HIP(c, hipEventSynchronize(l.stop));
        float t = 0.f;
        JORGE_HIP(c, hipEventElapsedTime(&t, l.start, l.stop));
        c->stage_ms[l.stage] += t;
        c->stage_launches[l.stage] += 1;
        c->free_events.push_back(l.start);
        c->free_events.push_back(l.stop);
    }
    c->pending.clear();
    for (int i = 0; i < std::min<int>(n, ST_COUNT); ++i) {
        if (ms) ms[i] = c->stage_ms[i];
        if (launches) launches[i] = c->stage_launches[i];
    }
    return JORGE_OK;
}

jorge_status jorge_reset_timing(jorge_ctx* c) {
    if (!c) return JORGE_ERR_INVALID_ARGUMENT;
    jorge_status s = jorge_read_timing(c, nullptr, nullptr, 0);
    for (int i = 0; i < ST_COUNT; ++i) {
        c->stage_ms[i] = 0.0;
        c->stage_launches[i] = 0;
    }
    return s;
}

int32_t jorge_num_stages(void) { return ST_COUNT; }

jorge_status jorge_stage_flops(const jorge_ctx* c, double* flops, int32_t n) {
    if (!c || !flops || n < 0) return JORGE_ERR_INVALID_ARGUMENT;
    for (int i = 0; i < std::min<int>(n, ST_COUNT); ++i)
        flops[i] = c->nt[i].flops + c->nn[i].flops + (i == ST_LDS_CHAIN ? c->chain_flops : 0.0);
    return JORGE_OK;
}

jorge_status jorge_factor_form(const jorge_ctx* c, int32_t layer, int32_t side, int32_t* form) {
    if (!c || !form || layer < 0 || layer >= (int32_t)c->layers.size() || (side != 0 && side != 1))
        return JORGE_ERR_INVALID_ARGUMENT;
    const auto& L = c->layers[layer];
    const FactorHost& F = c->factors[side == 0 ? L.fL : L.fR];
    *form = F.expl ? JORGE_FORM_EXPLICIT : F.squared ? JORGE_FORM_SQUARED : JORGE_FORM_FACTORED;
    return JORGE_OK;
}

const char* jorge_stage_name(int32_t stage) {
    return (stage >= 0 && stage < ST_COUNT) ? kStageNames[stage] : nullptr;
}

void jorge_destroy(jorge_ctx* c) {
    if (!c) return;
    (void)hipStreamSynchronize(c->stream);
    free_ctx(c);
}

const char* jorge_status_string(jorge_status s) {
    switch (s) {
        case JORGE_OK: return "ok";
        case JORGE_ERR_INVALID_ARGUMENT: return "invalid argument";
        case JORGE_ERR_OUT_OF_MEMORY: return "out of memory";
        case JORGE_ERR_HIP: return "HIP runtime error";
        case JORGE_ERR_UNSUPPORTED: return "unsupported size";
        default: return "unknown status";
    }
}

const char* jorge_last_error(const jorge_ctx* c) { return c ? c->last_error.c_str() : ""; }

}  // extern "C"
