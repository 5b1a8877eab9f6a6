// Host runtime and C ABI of the Jorge optimizer step on gfx950.
//
// A context owns one device arena holding, per layer, the factors L_hat and
// R_hat (padded to multiples of 32, zero outside the valid block), three
// workspace matrices per factor, the padded gradient, the intermediate
// L_hat G, both momenta and the partial-sum slots; and the device tables that
// describe every grouped launch. Tables are built once at creation, so a
// step is a fixed sequence of launches on one stream with no host sync.
//
// Update step (Algorithm 2, Appendix A.1, Algorithm 3, Section 4):
//   stage-in   Gp <- G, Gpt <- G^T, m_SGD <- beta1 m_SGD + G, partial sums of m_SGD^2
//   gram       M_L = G G^T, M_R = G^T G and A^2 = A A     (one launch, symmetric tiles only)
//   pow4       A^4 = A^2 A^2                              (symmetric tiles only)
//   xform      X = A^4 M, partial sums of X^2
//   ffinal     nu = ||X||_F, beta, c, s per factor
//   poly       P = I - (c/4) X + (5c^2/32) X X
//   update     Z = s A P
//   symm       A <- (Z + Z^T)/2
//   precond    T = L_hat G, then G~ = T R_hat fused with m <- beta1 m + (1-beta1) G~
//   lfinal     ||m||, ||m_SGD||, grafted step g
//   weight     theta <- theta (1 - lr wd) - g m
// Non-update steps run stage-in, precond, lfinal and weight only.
//
// Factors no larger than hp.small_factor_max skip the grouped launches: one
// workgroup per factor runs its whole update (chain_kernel) on a second
// stream, forked after stage-in and joined before preconditioning.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <cstdio>
#include <cstring>
#include <new>
#include <string>
#include <vector>

#include "../../include/jorge.h"
#include "jorge_gemm.hpp"
#include "jorge_kernels.hpp"
#include "jorge_types.hpp"

using namespace jorge;

namespace {

// Timed stages. With symmetric factors the Gram products and A^2 share the
// "gram" launch and "pow2" has none; the literal mode launches pow2 apart.
enum Stage : int {
    ST_STAGEIN = 0, ST_GRAM, ST_POW2, ST_POW4, ST_XFORM, ST_FFINAL, ST_POLY, ST_UPDATE, ST_SYMM,
    ST_CHAIN, ST_PRECOND_L, ST_PRECOND_R, ST_LFINAL, ST_WEIGHT, ST_COUNT
};
const char* const kStageNames[ST_COUNT] = {
    "stage_in", "gram", "pow2", "pow4", "xform", "factor_finalize", "poly", "update", "symmetrize",
    "small_chain", "precond_L", "precond_R", "layer_finalize", "weight"};

constexpr size_t kAlign = 256;
constexpr int kFlatChunkElems = 16384;
constexpr int kGroupRows = 8;  // tile rows per group in the tile ordering

inline int64_t round_up(int64_t x, int64_t m) { return (x + m - 1) / m * m; }

struct GemmStage {
    std::vector<GemmProblem> probs;
    std::vector<TileDesc> tiles;
    GemmProblem* dprobs = nullptr;
    TileDesc* dtiles = nullptr;
    int ntiles() const { return (int)tiles.size(); }
};

struct LayerHost {
    int m, n, mp, np;
    size_t off_Gp, off_Gpt, off_T, off_mom, off_msgd, off_part_m, off_part_sgd, off_ls;
    int n_part_m = 0, n_part_sgd = 0;
    int fL, fR;
};

struct FactorHost {
    int layer, side, d, dp;
    bool small = false;  // updated by chain_kernel rather than the grouped launches
    size_t off_A, off_W0, off_W1, off_W2, off_part, off_sc;
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
    // device tables
    LayerDev* dlayers = nullptr;
    FactorDev* dfactors = nullptr;
    StageTile* dstage = nullptr;
    FlatChunk* dflat = nullptr;
    SymTile* dsym = nullptr;
    int* dbig = nullptr;     // indices of the factors in the grouped launches
    int* dsmall = nullptr;   // indices of the factors updated by chain_kernel, costliest first
    std::vector<int> big, small;
    hipStream_t side = nullptr;                   // stream of chain_kernel
    hipEvent_t ev_fork = nullptr, ev_join = nullptr;
    std::vector<StageTile> stage_tiles;
    std::vector<FlatChunk> flat_chunks;
    std::vector<int> stage_batch_start, flat_batch_start;  // first block of each layer batch
    std::vector<SymTile> sym_tiles;
    GemmStage gram, pow2, pow4, xform, poly, update, pre_l, pre_r;
    // timing
    bool timing = false;
    std::vector<hipEvent_t> free_events;
    std::vector<Launch> pending;
    double stage_ms[ST_COUNT] = {};
    int64_t stage_launches[ST_COUNT] = {};
    std::string last_error;
};

namespace {

jorge_status fail(jorge_ctx* c, jorge_status s, const std::string& msg) {
    if (c) c->last_error = msg;
    return s;
}

jorge_status hip_fail(jorge_ctx* c, hipError_t e, const char* what) {
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

// Adds a product's tiles in grouped order: bands of kGroupRows tile rows,
// walked column by column, so concurrently running workgroups share panels.
void add_problem(GemmStage& st, const GemmProblem& p, bool upper_only) {
    const int idx = (int)st.probs.size();
    st.probs.push_back(p);
    const int tm_n = (p.M + kTile - 1) / kTile, tn_n = (p.N + kTile - 1) / kTile;
    int slot = 0;
    for (int g = 0; g < tm_n; g += kGroupRows)
        for (int tn = 0; tn < tn_n; ++tn)
            for (int tm = g; tm < std::min(g + kGroupRows, tm_n); ++tm) {
                if (upper_only && tm > tn) continue;
                st.tiles.push_back({idx, tm, tn, slot++});
            }
}

int tile_count(int M, int N) { return ((M + kTile - 1) / kTile) * ((N + kTile - 1) / kTile); }

constexpr int kXcds = 8;  // workgroup b of a launch runs on XCD b % 8, in increasing b

// Puts a stage's tiles in dispatch order. The tiles are sorted by K, longest
// first; each problem's tiles stay in bands of kGroupRows tile rows walked
// column by column. Runs of consecutive tiles of one problem and one column (they
// share the B panel and neighbouring A panels) are dealt, in that order, to
// the XCD with the least accumulated work (K of the tile), so every XCD gets
// a balanced, largest-first share whose tiles reuse panels in its own L2.
// The shares are then interleaved so that XCD x's i-th tile sits at slot
// kXcds * i + x; once a share is used up, its slots take the next tile of the
// longest remaining share.
void order_for_xcds(GemmStage& st) {
    const size_t n = st.tiles.size();
    if (n == 0) return;
    // Longest K first (stable: each problem's tiles stay together and in order).
    std::stable_sort(st.tiles.begin(), st.tiles.end(), [&](const TileDesc& a, const TileDesc& b) {
        return st.probs[a.prob].K > st.probs[b.prob].K;
    });
    std::vector<std::vector<TileDesc>> share(kXcds);
    std::vector<int64_t> work(kXcds, 0);
    for (size_t i = 0; i < n;) {
        size_t j = i + 1;
        while (j < n && st.tiles[j].prob == st.tiles[i].prob && st.tiles[j].tn == st.tiles[i].tn &&
               st.tiles[j].tm / kGroupRows == st.tiles[i].tm / kGroupRows)
            ++j;
        const int x = (int)(std::min_element(work.begin(), work.end()) - work.begin());
        for (size_t k = i; k < j; ++k) share[x].push_back(st.tiles[k]);
        work[x] += (int64_t)(j - i) * st.probs[st.tiles[i].prob].K;
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
    st.tiles.swap(out);
}

template <bool AK, bool BK, int EPI>
jorge_status launch_gemm(jorge_ctx* c, const GemmStage& st, int stage, float beta1) {
    if (st.ntiles() == 0) return JORGE_OK;
    TimedLaunch tl(c, stage);
    hipLaunchKernelGGL((gemm_grouped<AK, BK, EPI>), dim3(st.ntiles()), dim3(kGemmThreads), 0, c->stream,
                       st.dprobs, st.dtiles, beta1);
    tl.finish();
    JORGE_HIP(c, hipGetLastError());
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
    if (hp->small_factor_max < 0 || hp->small_factor_max > 4096) return JORGE_ERR_INVALID_ARGUMENT;
    return JORGE_OK;
}

// Builds every offset and launch table; returns the arena size in bytes.
size_t plan(jorge_ctx* c) {
    size_t off = 0;
    auto take = [&](size_t bytes) {
        const size_t o = off;
        off = (size_t)round_up((int64_t)(off + bytes), kAlign);
        return o;
    };
    for (auto& L : c->layers) {
        for (int side = 0; side < 2; ++side) {
            FactorHost F{};
            F.layer = (int)(&L - &c->layers[0]);
            F.side = side;
            F.d = side == 0 ? L.m : L.n;
            F.dp = side == 0 ? L.mp : L.np;
            const size_t mat = (size_t)F.dp * F.dp * sizeof(float);
            F.off_A = take(mat);
            F.off_W0 = take(mat);
            F.off_W1 = take(mat);
            F.off_W2 = take(mat);
            F.nparts = tile_count(F.dp, F.dp);
            F.off_part = take((size_t)F.nparts * sizeof(double));
            F.off_sc = take(sizeof(FactorScalars));
            F.small = F.dp <= c->hp.small_factor_max;
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
        L.off_part_m = take((size_t)L.n_part_m * sizeof(double));
        L.n_part_sgd = ((L.m + 63) / 64) * ((L.n + 63) / 64);
        L.off_part_sgd = take((size_t)L.n_part_sgd * sizeof(double));
        L.off_ls = take(sizeof(LayerScalars));
    }
    return off;
}

template <typename T>
T* at(jorge_ctx* c, size_t off) { return reinterpret_cast<T*>(c->arena + off); }

// Fills the host-side launch tables (device pointers already known).
void build_tables(jorge_ctx* c, std::vector<LayerDev>& ld, std::vector<FactorDev>& fd) {
    const int nl = (int)c->layers.size();
    for (auto& F : c->factors) {
        FactorDev d{};
        d.A = at<float>(c, F.off_A);
        d.W0 = at<float>(c, F.off_W0);
        d.W1 = at<float>(c, F.off_W1);
        d.W2 = at<float>(c, F.off_W2);
        d.sc = at<FactorScalars>(c, F.off_sc);
        d.partials = at<double>(c, F.off_part);
        d.d = F.d;
        d.dp = F.dp;
        d.nparts = F.nparts;
        const auto& L = c->layers[F.layer];
        d.gop = at<float>(c, F.side == 0 ? L.off_Gp : L.off_Gpt);
        d.gk = F.side == 0 ? L.np : L.mp;
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

    // Factors in decreasing size, so large tiles are dispatched first.
    std::vector<int> order(c->factors.size());
    for (size_t i = 0; i < order.size(); ++i) order[i] = (int)i;
    std::stable_sort(order.begin(), order.end(),
                     [&](int a, int b) { return c->factors[a].dp > c->factors[b].dp; });
    for (int fi : order) {
        const auto& F = c->factors[fi];
        if (F.small) continue;
        c->big.push_back(fi);
        const FactorDev& d = fd[fi];
        const auto& L = c->layers[F.layer];
        const LayerDev& l = ld[F.layer];
        GemmProblem g{};
        g.M = g.N = g.K = F.dp;
        g.lda = g.ldb = g.ldc = g.ldx = F.dp;
        g.valid_m = g.valid_n = F.d;
        // Gram statistic into W0: G G^T = Gp Gp^T (K = np) and G^T G = Gpt Gpt^T (K = mp),
        // both with K-contiguous operands.
        GemmProblem s = g;
        s.C = d.W0;
        s.A = s.B = F.side == 0 ? l.Gp : l.Gpt;
        s.K = F.side == 0 ? L.np : L.mp;
        s.lda = s.ldb = s.K;
        add_problem(c->gram, s, true);
        // With symmetric factors A^2 and A^4 are symmetric products (upper tiles, mirrored);
        // the literal mode keeps non-symmetric factors and needs the general product.
        const bool sym = c->hp.symmetrize != 0;
        GemmProblem p2 = g; p2.A = p2.B = d.A; p2.C = d.W1; add_problem(c->pow2, p2, sym);
        GemmProblem p4 = g; p4.A = p4.B = d.W1; p4.C = d.W2; add_problem(c->pow4, p4, sym);
        GemmProblem px = g; px.A = d.W2; px.B = d.W0; px.C = d.W1; px.partials = d.partials;
        add_problem(c->xform, px, false);
        GemmProblem pp = g; pp.A = pp.B = pp.X = d.W1; pp.C = d.W2; pp.sc = d.sc;
        add_problem(c->poly, pp, false);
        GemmProblem pu = g; pu.A = d.A; pu.B = d.W2; pu.C = d.W0; pu.sc = d.sc;
        add_problem(c->update, pu, false);
        for (int ti = 0; ti * 64 < F.dp; ++ti)
            for (int tj = ti; tj * 64 < F.dp; ++tj) c->sym_tiles.push_back({fi, ti, tj, 0});
    }
    // Small factors, costliest first (tile-K products of the Gram and the chain).
    std::vector<std::pair<int64_t, int>> sc;
    for (size_t fi = 0; fi < c->factors.size(); ++fi) {
        const auto& F = c->factors[fi];
        if (!F.small) continue;
        const int64_t nt = (F.dp + kTile - 1) / kTile, sym = nt * (nt + 1) / 2;
        sc.push_back({sym * fd[fi].gk + (2 * sym + 3 * nt * nt) * F.dp, (int)fi});
    }
    std::stable_sort(sc.begin(), sc.end(), [](const auto& a, const auto& b) { return a.first > b.first; });
    for (const auto& e : sc) c->small.push_back(e.second);
    // Preconditioning, largest layers first.
    std::vector<int> lorder(nl);
    for (int i = 0; i < nl; ++i) lorder[i] = i;
    std::stable_sort(lorder.begin(), lorder.end(), [&](int a, int b) {
        return (int64_t)c->layers[a].mp * c->layers[a].np * (c->layers[a].mp + c->layers[a].np) >
               (int64_t)c->layers[b].mp * c->layers[b].np * (c->layers[b].mp + c->layers[b].np);
    });
    for (int li : lorder) {
        const auto& L = c->layers[li];
        const LayerDev& l = ld[li];
        GemmProblem a{};  // T = L_hat G: A = L_hat, B^T = Gpt (both K-major)
        a.A = fd[L.fL].A; a.B = l.Gpt; a.C = l.T;
        a.M = L.mp; a.N = L.np; a.K = L.mp;
        a.lda = L.mp; a.ldb = L.mp; a.ldc = L.np;
        a.valid_m = L.m; a.valid_n = L.n;
        add_problem(c->pre_l, a, false);
        GemmProblem b{};  // G~ = T R_hat: A = T (K-major), B = R_hat (K-major when symmetric)
        b.A = l.T; b.B = fd[L.fR].A;
        b.M = L.mp; b.N = L.np; b.K = L.np;
        b.lda = L.np; b.ldb = L.np;
        b.mom = l.mom; b.ldmom = L.n; b.partials = l.part_m;
        b.valid_m = L.m; b.valid_n = L.n;
        add_problem(c->pre_r, b, false);
    }
}

template <typename T>
jorge_status upload(jorge_ctx* c, const std::vector<T>& v, T** dptr) {
    *dptr = nullptr;
    if (v.empty()) return JORGE_OK;
    JORGE_HIP(c, hipMalloc(reinterpret_cast<void**>(dptr), v.size() * sizeof(T)));
    JORGE_HIP(c, hipMemcpy(*dptr, v.data(), v.size() * sizeof(T), hipMemcpyHostToDevice));
    return JORGE_OK;
}

// Moves every problem and tile of `from` into `into` (same kernel instantiation),
// so independent products share one launch.
void merge_stage(GemmStage& into, GemmStage& from) {
    const int base = (int)into.probs.size();
    into.probs.insert(into.probs.end(), from.probs.begin(), from.probs.end());
    for (TileDesc t : from.tiles) {
        t.prob += base;
        into.tiles.push_back(t);
    }
    from.probs.clear();
    from.tiles.clear();
}

jorge_status upload_stage(jorge_ctx* c, GemmStage& st) {
    order_for_xcds(st);
    jorge_status s = upload(c, st.probs, &st.dprobs);
    if (s != JORGE_OK) return s;
    return upload(c, st.tiles, &st.dtiles);
}

void free_ctx(jorge_ctx* c) {
    if (!c) return;
    for (GemmStage* st : {&c->gram, &c->pow2, &c->pow4, &c->xform, &c->poly, &c->update, &c->pre_l,
                          &c->pre_r}) {
        if (st->dprobs) (void)hipFree(st->dprobs);
        if (st->dtiles) (void)hipFree(st->dtiles);
    }
    if (c->dlayers) (void)hipFree(c->dlayers);
    if (c->dfactors) (void)hipFree(c->dfactors);
    if (c->dstage) (void)hipFree(c->dstage);
    if (c->dflat) (void)hipFree(c->dflat);
    if (c->dsym) (void)hipFree(c->dsym);
    if (c->dbig) (void)hipFree(c->dbig);
    if (c->dsmall) (void)hipFree(c->dsmall);
    if (c->ev_fork) (void)hipEventDestroy(c->ev_fork);
    if (c->ev_join) (void)hipEventDestroy(c->ev_join);
    if (c->side) (void)hipStreamDestroy(c->side);
    if (c->arena) (void)hipFree(c->arena);
    for (auto& l : c->pending) {
        (void)hipEventDestroy(l.start);
        (void)hipEventDestroy(l.stop);
    }
    for (auto e : c->free_events) (void)hipEventDestroy(e);
    delete c;
}

jorge_status run_update(jorge_ctx* c, double beta2) {
    jorge_status s;
    if ((s = launch_gemm<true, true, EPI_SYM>(c, c->gram, ST_GRAM, 0.f)) != JORGE_OK) return s;
    if (c->hp.symmetrize) {  // A^2 ran inside the gram launch
        if ((s = launch_gemm<true, true, EPI_SYM>(c, c->pow4, ST_POW4, 0.f)) != JORGE_OK) return s;
    } else {
        if ((s = launch_gemm<true, false, EPI_STORE>(c, c->pow2, ST_POW2, 0.f)) != JORGE_OK) return s;
        if ((s = launch_gemm<true, false, EPI_STORE>(c, c->pow4, ST_POW4, 0.f)) != JORGE_OK) return s;
    }
    if ((s = launch_gemm<true, true, EPI_NORM>(c, c->xform, ST_XFORM, 0.f)) != JORGE_OK) return s;
    if (!c->big.empty()) {
        TimedLaunch tl(c, ST_FFINAL);
        hipLaunchKernelGGL(factor_finalize_kernel, dim3((unsigned)c->big.size()), dim3(64), 0, c->stream,
                           c->dfactors, c->dbig, beta2, (int)c->hp.beta_mode);
        tl.finish();
        JORGE_HIP(c, hipGetLastError());
    }
    if ((s = launch_gemm<true, false, EPI_POLY>(c, c->poly, ST_POLY, 0.f)) != JORGE_OK) return s;
    if ((s = launch_gemm<true, false, EPI_SCALE>(c, c->update, ST_UPDATE, 0.f)) != JORGE_OK) return s;
    if (!c->sym_tiles.empty()) {
        TimedLaunch tl(c, ST_SYMM);
        hipLaunchKernelGGL(symmetrize_kernel, dim3((unsigned)c->sym_tiles.size()), dim3(kEwThreads), 0,
                           c->stream, c->dfactors, c->dsym, (int)c->hp.symmetrize);
        tl.finish();
        JORGE_HIP(c, hipGetLastError());
    }
    return JORGE_OK;
}

// Small factors: fork the side stream after stage-in, one chain_kernel launch.
jorge_status fork_small(jorge_ctx* c, double beta2) {
    if (c->small.empty()) return JORGE_OK;
    JORGE_HIP(c, hipEventRecord(c->ev_fork, c->stream));
    JORGE_HIP(c, hipStreamWaitEvent(c->side, c->ev_fork, 0));
    TimedLaunch tl(c, ST_CHAIN, c->side);
    if (c->hp.symmetrize)
        hipLaunchKernelGGL(chain_kernel<1>, dim3((unsigned)c->small.size()), dim3(kGemmThreads), 0, c->side,
                           c->dfactors, c->dsmall, beta2, (int)c->hp.beta_mode);
    else
        hipLaunchKernelGGL(chain_kernel<0>, dim3((unsigned)c->small.size()), dim3(kGemmThreads), 0, c->side,
                           c->dfactors, c->dsmall, beta2, (int)c->hp.beta_mode);
    tl.finish();
    JORGE_HIP(c, hipGetLastError());
    JORGE_HIP(c, hipEventRecord(c->ev_join, c->side));
    return JORGE_OK;
}

jorge_status join_small(jorge_ctx* c) {
    if (c->small.empty()) return JORGE_OK;
    JORGE_HIP(c, hipStreamWaitEvent(c->stream, c->ev_join, 0));
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
    hp->small_factor_max = 0;
    return JORGE_OK;
}

jorge_status jorge_create(const jorge_shape* shapes, int32_t num_layers, const jorge_hparams* hp,
                          void* hip_stream, jorge_ctx** out) {
    if (!out) return JORGE_ERR_INVALID_ARGUMENT;
    *out = nullptr;
    if (!shapes || num_layers <= 0) return JORGE_ERR_INVALID_ARGUMENT;
    if (num_layers > JORGE_MAX_LAYERS) return JORGE_ERR_UNSUPPORTED;
    jorge_hparams h;
    jorge_hparams_default(&h);
    if (hp) h = *hp;
    if (validate_hparams(&h) != JORGE_OK) return JORGE_ERR_INVALID_ARGUMENT;
    for (int32_t i = 0; i < num_layers; ++i) {
        if (shapes[i].rows <= 0 || shapes[i].cols <= 0) return JORGE_ERR_INVALID_ARGUMENT;
        if (shapes[i].rows > JORGE_MAX_DIM || shapes[i].cols > JORGE_MAX_DIM) return JORGE_ERR_UNSUPPORTED;
    }
    jorge_ctx* c = new (std::nothrow) jorge_ctx();
    if (!c) return JORGE_ERR_OUT_OF_MEMORY;
    c->hp = h;
    c->stream = reinterpret_cast<hipStream_t>(hip_stream);
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
        free_ctx(c);
        return JORGE_ERR_OUT_OF_MEMORY;
    }
    jorge_status st = JORGE_OK;
    auto bail = [&](jorge_status s) {
        free_ctx(c);
        return s;
    };
    if (hipGetDevice(&c->device) != hipSuccess) return bail(JORGE_ERR_HIP);
    hipError_t e = hipMalloc(reinterpret_cast<void**>(&c->arena), c->arena_bytes);
    if (e != hipSuccess) return bail(e == hipErrorOutOfMemory ? JORGE_ERR_OUT_OF_MEMORY : JORGE_ERR_HIP);
    if (hipMemsetAsync(c->arena, 0, c->arena_bytes, c->stream) != hipSuccess) return bail(JORGE_ERR_HIP);
    std::vector<LayerDev> ld;
    std::vector<FactorDev> fd;
    try {
        build_tables(c, ld, fd);
    } catch (const std::bad_alloc&) {
        return bail(JORGE_ERR_OUT_OF_MEMORY);
    }
    if ((st = upload(c, ld, &c->dlayers)) != JORGE_OK) return bail(st);
    if ((st = upload(c, fd, &c->dfactors)) != JORGE_OK) return bail(st);
    if ((st = upload(c, c->stage_tiles, &c->dstage)) != JORGE_OK) return bail(st);
    if ((st = upload(c, c->flat_chunks, &c->dflat)) != JORGE_OK) return bail(st);
    if ((st = upload(c, c->sym_tiles, &c->dsym)) != JORGE_OK) return bail(st);
    if ((st = upload(c, c->big, &c->dbig)) != JORGE_OK) return bail(st);
    if ((st = upload(c, c->small, &c->dsmall)) != JORGE_OK) return bail(st);
    if (!c->small.empty()) {
        if (hipStreamCreateWithFlags(&c->side, hipStreamNonBlocking) != hipSuccess ||
            hipEventCreateWithFlags(&c->ev_fork, hipEventDisableTiming) != hipSuccess ||
            hipEventCreateWithFlags(&c->ev_join, hipEventDisableTiming) != hipSuccess)
            return bail(JORGE_ERR_HIP);
    }
    if (c->hp.symmetrize) merge_stage(c->gram, c->pow2);
    for (GemmStage* s : {&c->gram, &c->pow2, &c->pow4, &c->xform, &c->poly, &c->update, &c->pre_l,
                         &c->pre_r})
        if ((st = upload_stage(c, *s)) != JORGE_OK) return bail(st);
    hipLaunchKernelGGL(init_factors_kernel, dim3((unsigned)c->factors.size()), dim3(256), 0, c->stream,
                       c->dfactors, (float)std::pow(h.eps, -0.25));
    if (hipGetLastError() != hipSuccess) return bail(JORGE_ERR_HIP);
    if (hipStreamSynchronize(c->stream) != hipSuccess) return bail(JORGE_ERR_HIP);
    *out = c;
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
    const int64_t t = c->t + 1;
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
    if (update) {
        if ((s = fork_small(c, beta2)) != JORGE_OK) return s;
        if ((s = run_update(c, beta2)) != JORGE_OK) return s;
        if ((s = join_small(c)) != JORGE_OK) return s;
    }
    if ((s = launch_gemm<true, true, EPI_STORE>(c, c->pre_l, ST_PRECOND_L, 0.f)) != JORGE_OK) return s;
    s = c->hp.symmetrize ? launch_gemm<true, true, EPI_MOMENTUM>(c, c->pre_r, ST_PRECOND_R, (float)beta1)
                         : launch_gemm<true, false, EPI_MOMENTUM>(c, c->pre_r, ST_PRECOND_R, (float)beta1);
    if (s != JORGE_OK) return s;
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
    c->t = t;
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

jorge_status jorge_set_stream(jorge_ctx* c, void* hip_stream) {
    if (!c) return JORGE_ERR_INVALID_ARGUMENT;
    c->stream = reinterpret_cast<hipStream_t>(hip_stream);
    return JORGE_OK;
}

jorge_status jorge_synchronize(jorge_ctx* c) {
    if (!c) return JORGE_ERR_INVALID_ARGUMENT;
    JORGE_HIP(c, hipStreamSynchronize(c->stream));
    return JORGE_OK;
}

jorge_status jorge_device_bytes(const jorge_ctx* c, int64_t* bytes) {
    if (!c || !bytes) return JORGE_ERR_INVALID_ARGUMENT;
    *bytes = (int64_t)c->arena_bytes;
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
