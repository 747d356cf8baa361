// C ABI of the GMC device library (declared in include/gmc.h): argument
// checks, the context and its device scratch, and the launch order of one
// iteration of Algorithm 1.
#include <algorithm>
#include <cmath>
#include <cstdio>
#include <cstring>
#include <mutex>
#include <new>
#include <string>
#include <vector>

#include "../../include/gmc.h"
#include "gmc_internal.h"

using namespace gmc;

namespace {

// profiled stages: fused pass (vector kernel), fused pass (element-wise
// kernel), selection, emit, aggregate, apply
constexpr int kStages = 6;
constexpr int64_t kMaxPendingEvents = 4096;

thread_local std::string g_init_error = "no error";

// The kept fraction as the caller means it: the fraction p/q with the
// smallest denominator q <= 2^20 whose binary64 quotient is the given ratio
// (0.07 is 7/100, 1/1024 itself).  q = 0 when there is none: then the ratio
// is used at its exact binary value mant * 2^-shift.
struct KeepRatio {
    int64_t p = 0, q = 0;
    uint64_t mant = 0;
    int shift = 0;
};

}  // namespace

struct gmc_ctx {
    // problem
    int64_t d = 0;
    int32_t K = 0;
    int32_t comp = 0;
    double ratio = 0, beta = 0, eta = 0;
    KeepRatio keep;                // ratio as the fraction it stands for
    double lambda = 0;             // GMC+ detach coefficient
    int32_t rule = kRuleGmc;       // update rule
    uint64_t seed = 0;
    float c = 0, s = 0, h = 1, b = 0, q = 0;  // see derive_constants
    int64_t t = 0;
    hipStream_t stream = nullptr;
    hipEvent_t stream_ev = nullptr;  // orders a new stream after the old one (gmc_set_stream)
    int device = 0;
    bool started = false;
    std::string err = "no error";

    // configuration
    std::vector<int64_t> seg_off;  // top-s segments (host)
    int32_t block = 4096;          // RBGS block length
    int force_full = 0;
    int margin = 4;                // speculative threshold rank, quarters of k (k)
    int cap_mult = 64;
    int32_t stratum = 100;         // sampled-threshold top-s: components per sample stratum
    int sparse_w = 0;              // GMC_OPT_SPARSE_MOMENTUM
    bool seeded = false;           // the first step's thresholds were drawn from a sample
    int change_list = 0;           // GMC_OPT_CHANGE_LIST: 0 by size, 1 always, 2 never, 3 whole ranges
    int32_t dl_stride = kDlistStride;  // int2 per range of the change list (kDlistStrideFull with 3)
    // device word: the epoch of the last pass that wrote a non-finite w; the
    // record of a pass counts while it equals nf_epoch (bumped to drop it)
    int32_t* nf = nullptr;
    int32_t nf_epoch = 1;

    // the last server pass's bitmap of changed components (sparse_w)
    uint32_t* wbits = nullptr;
    bool wbits_valid = false;
    const float* wbits_in = nullptr;   // that pass's w_t ...
    const float* wbits_out = nullptr;  // ... and w_{t+1}
    int64_t wbits_t = -1;              // the step the bitmap serves
    int64_t sparse_steps = 0;          // worker passes that used it
    // the bitmap still describes its pass's two buffers (cleared by calls
    // that write w or drop the marks), and the step at which a worker pass
    // last read w through it (-1: the last worker pass did not): together
    // they let the next server pass, writing over that pass's input buffer,
    // skip the components where the buffer already holds w_{t+1}
    bool wbits_pair = false;
    int64_t wbits_used_t = -1;
    int64_t sparse_applies = 0;        // server passes that wrote w only where it changes

    // derived
    std::vector<int32_t> seg_k;
    int64_t k_tot = 0;
    int32_t nb = 0, n_sel = 0;

    // device scratch (one allocation, carved)
    bool prepared = false;
    void* mem = nullptr;
    size_t mem_bytes = 0;
    TopkGeometry geo{};
    TopkScratch scr{};
    int32_t* rowptr = nullptr;
    int2* dlist = nullptr;         // the last top-s server pass's change list (dl_stride per range)
    int32_t n_ranges = 0;
    uint32_t* rbgs_bitmap = nullptr;
    int32_t* rbgs_blocks = nullptr;
    int32_t* rbgs_slot = nullptr;
    int32_t* rbgs_prev = nullptr;    // the previous step's blocks
    int32_t* rbgs_visit = nullptr;   // the sparse server pass's ranges
    uint32_t* rbgs_rbits = nullptr;  // zeroed bitmap of ranges (large d)
    int32_t* rbgs_meta = nullptr;    // [0] ranges in rbgs_visit (-1: all), [1] non-finite flag
    int64_t* stats = nullptr;

    // profiling
    uint32_t profile = 0;  // bit i: time stage i
    double prof_ms[kStages] = {0};
    int64_t prof_n[kStages] = {0};
    std::vector<std::pair<hipEvent_t, hipEvent_t>> pending[kStages];
};

namespace {

gmc_status fail(gmc_ctx* ctx, gmc_status st, const std::string& msg) {
    if (ctx) ctx->err = msg; else g_init_error = msg;
    return st;
}

gmc_status hip_fail(gmc_ctx* ctx, hipError_t e, const char* what) {
    std::string m = std::string(what) + ": " + hipGetErrorString(e);
    return fail(ctx, GMC_EDEVICE, m);
}

#define GMC_HIP(ctx, call)                                  \
    do {                                                    \
        hipError_t e_ = (call);                             \
        if (e_ != hipSuccess) return hip_fail(ctx, e_, #call); \
    } while (0)

#define GMC_TRY(x)                       \
    do {                                 \
        gmc_status st_ = (x);            \
        if (st_ != GMC_OK) return st_;   \
    } while (0)

// Constants of the update rule at the current eta, each formed in binary64
// and rounded once: c multiplies w_t - w_{t-1} in the workers' vector, h the
// gradient, s the server's sum, b the server's momentum term, q the residual
// in GMC+'s detach.
void derive_constants(gmc_ctx* ctx) {
    const double beta = ctx->beta, eta = ctx->eta, K = (double)ctx->K;
    ctx->h = 1.0f;
    ctx->b = 0.0f;
    if (ctx->rule == kRuleServerMomentum) {
        ctx->c = 0.0f;
        ctx->s = (float)(eta / K);
        ctx->b = (float)beta;
    } else if (ctx->rule == kRuleLrInResidual) {
        ctx->c = (float)beta;
        ctx->s = (float)(1.0 / K);
        ctx->h = (float)eta;
    } else {
        ctx->c = (float)(beta / eta);
        ctx->s = (float)(eta / K);
    }
    ctx->q = (float)(ctx->lambda * eta);
}

KeepRatio read_ratio(double ratio) {
    KeepRatio r;
    const int64_t q_max = int64_t(1) << 20;
    for (int64_t q = 1; q <= q_max; ++q) {
        const double scaled = ratio * (double)q;
        const int64_t p = (int64_t)std::floor(scaled + 0.5);
        if (p >= 1 && p <= q && (double)p / (double)q == ratio) {
            r.p = p;
            r.q = q;
            return r;
        }
    }
    int e = 0;
    const double f = std::frexp(ratio, &e);  // ratio = f * 2^e, f in [1/2, 1)
    r.mant = (uint64_t)std::ldexp(f, 53);
    r.shift = 53 - e;
    return r;
}

// top-s keeps ceil(n * ratio) of a segment of n (the paper's s; s = d/1024
// in Section 5.1), in exact integer arithmetic, clamped to [1, n]
int64_t count_for(int64_t n, const KeepRatio& r) {
    int64_t k;
    if (r.q > 0) {
        k = (n * r.p + r.q - 1) / r.q;  // n < 2^31, p <= q <= 2^20
    } else if (r.shift >= 120) {
        k = 1;  // n * mant < 2^84
    } else {
        const unsigned __int128 prod = (unsigned __int128)(uint64_t)n * r.mant;
        const unsigned __int128 ceil_add = ((unsigned __int128)1 << r.shift) - 1;
        k = (int64_t)((prod + ceil_add) >> r.shift);
    }
    return std::max<int64_t>(1, std::min<int64_t>(k, n));
}

// top-s contexts whose parameter vectors outgrow the Infinity Cache keep the
// server pass's change list for the next worker pass
bool use_dlist(const gmc_ctx* ctx) {
    if (ctx->comp == GMC_RBGS || ctx->dlist == nullptr || ctx->change_list == 2) return false;
    return ctx->change_list == 1 || ctx->change_list == 3 || 8 * ctx->d > kDlistMinParamBytes;
}

// Drops the record of the last server pass's changes (bitmap, change list
// and the non-finite flag): the next worker pass reads w densely and the
// next server pass writes w everywhere.
void drop_record(gmc_ctx* ctx) {
    ctx->wbits_valid = false;
    ctx->wbits_pair = false;
    ctx->wbits_used_t = -1;
    ctx->nf_epoch += 1;
}

void release(gmc_ctx* ctx) {
    if (ctx->mem) {
        (void)hipSetDevice(ctx->device);
        (void)hipDeviceSynchronize();
        (void)hipFree(ctx->mem);
    }
    ctx->mem = nullptr;
    ctx->mem_bytes = 0;
    ctx->prepared = false;
}

struct Carver {
    char* base;
    size_t off = 0;
    template <class T>
    T* take(size_t n) {
        off = (off + 255) & ~(size_t)255;
        T* p = reinterpret_cast<T*>(base + off);
        off += n * sizeof(T);
        return p;
    }
};

// Host-side tables of the top-s geometry.
struct TopkTables {
    std::vector<int32_t> seg_start, seg_out;
    std::vector<int32_t> chunk_start, chunk_len, chunk_seg, chunk_cgrp;
    std::vector<int32_t> cgrp_lo, cgrp_hi, cgrp_seg, cgrp_rank, seg_cgrp_lo, seg_cgrps;
    std::vector<int32_t> slice_seg, slice_rank, seg_slices, seg_slice_lo;
    std::vector<int32_t> pair_k, pair_cap;
    std::vector<int64_t> pair_cand;
    std::vector<int2> tile_map;       // per worker: launched tile -> (segment, first tile in the segment)
    std::vector<int32_t> seg_tile_stride;
    std::vector<int2> seed_map;       // first-step sample: (segment, first run) per workgroup
    std::vector<int32_t> seg_seed_groups, seg_seed_runs, seg_seed_rank;
    int64_t cand_total = 0;
};

int64_t pair_capacity(const gmc_ctx* ctx, int64_t n, int64_t k) {
    return std::min<int64_t>(n, (int64_t)ctx->cap_mult * k + 2048);
}

// Candidates the selection launches are sized for: the speculative threshold
// aims at a few k (the margin, then the growth of the residual from one step
// to the next); longer lists, up to the capacity, are walked in strides.
constexpr int64_t kLaunchMult = 8;
int64_t pair_launch(const gmc_ctx* ctx, int64_t n, int64_t k) {
    return std::min<int64_t>(pair_capacity(ctx, n, k), kLaunchMult * k + 2048);
}

TopkTables build_tables(const gmc_ctx* ctx) {
    TopkTables T;
    const int n_seg = (int)ctx->seg_off.size() - 1;
    int64_t out = 0;
    for (int sg = 0; sg <= n_seg; ++sg) T.seg_start.push_back((int32_t)ctx->seg_off[sg]);
    for (int sg = 0; sg < n_seg; ++sg) {
        const int64_t lo = ctx->seg_off[sg], hi = ctx->seg_off[sg + 1], n = hi - lo;
        // chunks of kChunk elements
        const int32_t first_chunk = (int32_t)T.chunk_start.size();
        for (int64_t a = lo; a < hi; a += kChunk) {
            const int32_t len = (int32_t)std::min<int64_t>(kChunk, hi - a);
            T.chunk_start.push_back((int32_t)a);
            T.chunk_len.push_back(len);
            T.chunk_seg.push_back(sg);
        }
        const int32_t last_chunk = (int32_t)T.chunk_start.size();
        // compaction groups
        T.seg_cgrp_lo.push_back((int32_t)T.cgrp_lo.size());
        int32_t rank = 0;
        for (int32_t c = first_chunk; c < last_chunk; c += kCompactChunks) {
            for (int32_t c2 = c; c2 < std::min(c + kCompactChunks, last_chunk); ++c2)
                T.chunk_cgrp.push_back((int32_t)T.cgrp_lo.size());
            T.cgrp_lo.push_back(c);
            T.cgrp_hi.push_back(std::min(c + kCompactChunks, last_chunk));
            T.cgrp_seg.push_back(sg);
            T.cgrp_rank.push_back(rank++);
        }
        T.seg_cgrps.push_back(rank);
        // slices of the selection passes
        const int64_t lc = pair_launch(ctx, n, ctx->seg_k[sg]);
        int64_t w = std::max((n + kSliceElems - 1) / kSliceElems, (lc + kSliceCands - 1) / kSliceCands);
        w = std::max<int64_t>(1, std::min<int64_t>(w, kMaxSlices));
        T.seg_slice_lo.push_back((int32_t)T.slice_seg.size());
        T.seg_slices.push_back((int32_t)w);
        for (int32_t r = 0; r < w; ++r) {
            T.slice_seg.push_back(sg);
            T.slice_rank.push_back(r);
        }
        T.seg_out.push_back((int32_t)out);
        out += ctx->seg_k[sg];
        // copy tiles: a list of c candidates takes at most c/kTile whole
        // tiles plus a partial one per group
        const int64_t nlaunch = (lc + kTile - 1) / kTile + rank;
        T.seg_tile_stride.push_back((int32_t)nlaunch);
        for (int64_t i = 0; i < nlaunch; ++i) T.tile_map.push_back(make_int2(sg, (int)i));
        // first-step sample of a large segment: whole runs of kSeedRun every
        // kSeedStride; the rank aims at kSeedMult k candidates
        const int64_t runs = n >= kSeedMinLen ? n / kSeedStride : 0;
        const int64_t groups = (runs + kSeedRunsPerGroup - 1) / kSeedRunsPerGroup;
        int64_t rank_s = 0;
        if (runs > 0) {
            const int64_t m = runs * kSeedRun;
            const int64_t want = (int64_t)kSeedMult * ctx->seg_k[sg];
            rank_s = std::max<int64_t>(1, std::min<int64_t>(m, (want * m + n - 1) / n));
        }
        T.seg_seed_groups.push_back((int32_t)groups);
        T.seg_seed_runs.push_back((int32_t)runs);
        T.seg_seed_rank.push_back((int32_t)rank_s);
        for (int64_t gi = 0; gi < groups; ++gi) T.seed_map.push_back(make_int2(sg, (int)(gi * kSeedRunsPerGroup)));
    }
    for (int k = 0; k < ctx->K; ++k) {
        for (int sg = 0; sg < n_seg; ++sg) {
            const int64_t n = ctx->seg_off[sg + 1] - ctx->seg_off[sg];
            const int64_t cap = pair_capacity(ctx, n, ctx->seg_k[sg]);
            T.pair_k.push_back(ctx->seg_k[sg]);
            T.pair_cap.push_back((int32_t)cap);
            T.pair_cand.push_back(T.cand_total);
            T.cand_total += cap;
        }
    }
    return T;
}

gmc_status prepare(gmc_ctx* ctx) {
    if (ctx->prepared) return GMC_OK;
    release(ctx);
    GMC_HIP(ctx, hipSetDevice(ctx->device));
    const int32_t K = ctx->K;
    const int64_t d = ctx->d;
    ctx->n_ranges = (int32_t)((d + kAggTopkRange - 1) / kAggTopkRange);

    TopkTables T;
    const bool approx = ctx->comp == GMC_TOPK_APPROX;
    const int64_t samp_n = approx ? (ctx->d + ctx->stratum - 1) / ctx->stratum : 0;
    size_t bytes = 0;
    auto add = [&](size_t n, size_t sz) { bytes = ((bytes + 255) & ~(size_t)255) + n * sz; };
    add(8, sizeof(int64_t));  // stats
    add((size_t)(ctx->d + 31) / 32, 4);  // bitmap of the components the last server pass changed
    if (ctx->comp == GMC_RBGS) {
        add((size_t)(ctx->nb + 31) / 32, 4);
        add((size_t)ctx->n_sel, 4);
        add((size_t)ctx->nb, 4);
        const size_t rr = (size_t)((ctx->d + kAggRange - 1) / kAggRange);
        add((size_t)ctx->n_sel, 4);
        add(rr, 4);
        add((rr + 31) / 32, 4);
        add(2, 4);
    } else {
        T = build_tables(ctx);
        const size_t nc = T.chunk_start.size(), ng = T.cgrp_lo.size(), nsl = T.slice_seg.size();
        const size_t ns = T.seg_out.size(), np = (size_t)K * ns;
        add(ns + 1, 4); add(ns, 4);
        add(nc, 4); add(nc, 4); add(nc, 4); add(nc, 4);
        add(ng, 4); add(ng, 4); add(ng, 4); add(ng, 4); add(ns, 4); add(ns, 4);
        add(nsl, 4); add(nsl, 4); add(ns, 4); add(ns, 4);
        add(np, 4); add(np, 4); add(np, 8);
        add(T.tile_map.size(), sizeof(int2)); add(ns, 4);
        add(T.seed_map.size() + 1, sizeof(int2)); add(ns, 4); add(ns, 4); add(ns, 4);
        add(np, sizeof(PairState));
        add(np * kBins, 4);
        add(np * kBins, 4);
        add((size_t)K * nc, 4); add((size_t)2 * kGrpSub * K * ng, 4);
        add((size_t)K * nc * kChunk, sizeof(int2));
        add((size_t)T.cand_total, 4); add((size_t)T.cand_total, 4);
        for (int q = 0; q < 4; ++q) add((size_t)K * nsl, 4);
        add((size_t)K * nsl * kSlHist, 4);
        add((size_t)K * nsl * kWavesPerGroup, 4);
        add((size_t)K * (ctx->n_ranges + 1), 4);
        add((size_t)ctx->n_ranges * ctx->dl_stride, sizeof(int2));
        add(1, 4);
        if (approx) add((size_t)K * samp_n, 4);
    }
    bytes += 256;
    void* mem = nullptr;
    hipError_t e = hipMalloc(&mem, bytes);
    if (e != hipSuccess) {
        (void)hipGetLastError();
        return fail(ctx, GMC_ENOMEM, "hipMalloc of " + std::to_string(bytes) + " bytes of scratch failed");
    }
    ctx->mem = mem;
    ctx->mem_bytes = bytes;
    GMC_HIP(ctx, hipMemset(mem, 0, bytes));
    Carver cv{reinterpret_cast<char*>(mem)};
    ctx->stats = cv.take<int64_t>(8);
    ctx->wbits = cv.take<uint32_t>((size_t)(ctx->d + 31) / 32);
    ctx->wbits_valid = false;
    ctx->wbits_pair = false;
    ctx->wbits_used_t = -1;
    if (ctx->comp == GMC_RBGS) {
        ctx->rbgs_bitmap = cv.take<uint32_t>((ctx->nb + 31) / 32);
        ctx->rbgs_blocks = cv.take<int32_t>(ctx->n_sel);
        ctx->rbgs_slot = cv.take<int32_t>(ctx->nb);
        const size_t rr = (size_t)((ctx->d + kAggRange - 1) / kAggRange);
        ctx->rbgs_prev = cv.take<int32_t>(ctx->n_sel);
        ctx->rbgs_visit = cv.take<int32_t>(rr);
        ctx->rbgs_rbits = cv.take<uint32_t>((rr + 31) / 32);
        ctx->rbgs_meta = cv.take<int32_t>(2);
    } else {
        const size_t nc = T.chunk_start.size(), ng = T.cgrp_lo.size(), nsl = T.slice_seg.size();
        const size_t ns = T.seg_out.size(), np = (size_t)K * ns;
        auto put = [&](const std::vector<int32_t>& v, const int32_t** dst) -> gmc_status {
            int32_t* d = cv.take<int32_t>(v.size() + (v.empty() ? 1 : 0));
            if (!v.empty()) GMC_HIP(ctx, hipMemcpy(d, v.data(), v.size() * 4, hipMemcpyHostToDevice));
            *dst = d;
            return GMC_OK;
        };
        TopkGeometry& g = ctx->geo;
        g.K = K;
        g.n_seg = (int32_t)ns;
        g.n_chunks = (int32_t)nc;
        g.n_cgroups = (int32_t)ng;
        g.n_slices = (int32_t)nsl;
        g.approx = approx ? 1 : 0;
        g.stratum = ctx->stratum;
        g.samp_n = (int32_t)samp_n;
        g.samp_r = approx ? (int32_t)count_for(samp_n, ctx->keep) : 0;
        GMC_TRY(put(T.seg_start, &g.seg_start));
        GMC_TRY(put(T.seg_out, &g.seg_out));
        GMC_TRY(put(T.chunk_start, &g.chunk_start));
        GMC_TRY(put(T.chunk_len, &g.chunk_len));
        GMC_TRY(put(T.chunk_seg, &g.chunk_seg));
        GMC_TRY(put(T.chunk_cgrp, &g.chunk_cgrp));
        GMC_TRY(put(T.cgrp_lo, &g.cgrp_lo));
        GMC_TRY(put(T.cgrp_hi, &g.cgrp_hi));
        GMC_TRY(put(T.cgrp_seg, &g.cgrp_seg));
        GMC_TRY(put(T.cgrp_rank, &g.cgrp_rank));
        GMC_TRY(put(T.seg_cgrp_lo, &g.seg_cgrp_lo));
        GMC_TRY(put(T.seg_cgrps, &g.seg_cgrps));
        GMC_TRY(put(T.slice_seg, &g.slice_seg));
        GMC_TRY(put(T.slice_rank, &g.slice_rank));
        GMC_TRY(put(T.seg_slices, &g.seg_slices));
        GMC_TRY(put(T.seg_slice_lo, &g.seg_slice_lo));
        GMC_TRY(put(T.pair_k, &g.pair_k));
        GMC_TRY(put(T.pair_cap, &g.pair_cap));
        int64_t* pcd = cv.take<int64_t>(np);
        GMC_HIP(ctx, hipMemcpy(pcd, T.pair_cand.data(), np * 8, hipMemcpyHostToDevice));
        g.pair_cand = pcd;
        int2* tm = cv.take<int2>(T.tile_map.size());
        GMC_HIP(ctx, hipMemcpy(tm, T.tile_map.data(), T.tile_map.size() * sizeof(int2), hipMemcpyHostToDevice));
        g.tile_map = tm;
        g.tiles_per_worker = (int32_t)T.tile_map.size();
        GMC_TRY(put(T.seg_tile_stride, &g.seg_tile_stride));
        int2* sm = cv.take<int2>(T.seed_map.size() + 1);
        if (!T.seed_map.empty())
            GMC_HIP(ctx, hipMemcpy(sm, T.seed_map.data(), T.seed_map.size() * sizeof(int2), hipMemcpyHostToDevice));
        g.seed_map = sm;
        g.n_seed_groups = (int32_t)T.seed_map.size();
        GMC_TRY(put(T.seg_seed_groups, &g.seg_seed_groups));
        GMC_TRY(put(T.seg_seed_runs, &g.seg_seed_runs));
        GMC_TRY(put(T.seg_seed_rank, &g.seg_seed_rank));
        TopkScratch& sc = ctx->scr;
        sc.pair = cv.take<PairState>(np);
        std::vector<PairState> init(np);
        for (auto& ps : init) {
            std::memset(&ps, 0, sizeof ps);
            ps.tau = kNoThreshold;
        }
        GMC_HIP(ctx, hipMemcpy(sc.pair, init.data(), np * sizeof(PairState), hipMemcpyHostToDevice));
        sc.hist = cv.take<uint32_t>(np * kBins);
        sc.hist2 = cv.take<uint32_t>(np * kBins);
        sc.run_cnt = cv.take<uint32_t>((size_t)K * nc);
        sc.grp_acc = cv.take<uint32_t>((size_t)2 * kGrpSub * K * ng);
        sc.slot = cv.take<int2>((size_t)K * nc * kChunk);
        sc.cand_idx = cv.take<int32_t>((size_t)T.cand_total);
        sc.cand_val = cv.take<float>((size_t)T.cand_total);
        sc.sl_above = cv.take<uint32_t>((size_t)K * nsl);
        sc.sl_ties = cv.take<uint32_t>((size_t)K * nsl);
        sc.sl_out = cv.take<uint32_t>((size_t)K * nsl);
        sc.sl_tiebase = cv.take<uint32_t>((size_t)K * nsl);
        sc.sl_hist = cv.take<uint32_t>((size_t)K * nsl * kSlHist);
        sc.sl_run = cv.take<uint32_t>((size_t)K * nsl * kWavesPerGroup);
        sc.stats = ctx->stats;
        ctx->rowptr = cv.take<int32_t>((size_t)K * (ctx->n_ranges + 1));
        ctx->dlist = cv.take<int2>((size_t)ctx->n_ranges * ctx->dl_stride);
        ctx->nf = cv.take<int32_t>(1);
        sc.rowptr = ctx->rowptr;  // the emit kernel writes them for gmc_iteration's server pass
        sc.n_ranges = ctx->n_ranges;
        sc.samp = approx ? cv.take<float>((size_t)K * samp_n) : nullptr;
    }
    if (cv.off > bytes) return fail(ctx, GMC_ENOMEM, "internal: scratch layout overflow");
    ctx->prepared = true;
    return GMC_OK;
}

// -- profiling ---------------------------------------------------------------
// The stage events only time: recorded without the system-scope fence (a
// cache write-back and invalidate that would lengthen the step they time).

gmc_status prof_begin(gmc_ctx* ctx, int stage, hipEvent_t* ev) {
    *ev = nullptr;
    if (!((ctx->profile >> stage) & 1u)) return GMC_OK;
    GMC_HIP(ctx, hipEventCreateWithFlags(ev, hipEventDisableSystemFence));
    GMC_HIP(ctx, hipEventRecord(*ev, ctx->stream));
    return GMC_OK;
}

gmc_status prof_fold(gmc_ctx* ctx, int stage) {
    for (auto& pr : ctx->pending[stage]) {
        GMC_HIP(ctx, hipEventSynchronize(pr.second));
        float ms = 0.f;
        GMC_HIP(ctx, hipEventElapsedTime(&ms, pr.first, pr.second));
        ctx->prof_ms[stage] += ms;
        ctx->prof_n[stage] += 1;
        (void)hipEventDestroy(pr.first);
        (void)hipEventDestroy(pr.second);
    }
    ctx->pending[stage].clear();
    return GMC_OK;
}

gmc_status prof_end(gmc_ctx* ctx, int stage, hipEvent_t start) {
    if (!start) return GMC_OK;
    hipEvent_t stop;
    GMC_HIP(ctx, hipEventCreateWithFlags(&stop, hipEventDisableSystemFence));
    GMC_HIP(ctx, hipEventRecord(stop, ctx->stream));
    ctx->pending[stage].emplace_back(start, stop);
    if ((int64_t)ctx->pending[stage].size() >= kMaxPendingEvents) return prof_fold(ctx, stage);
    return GMC_OK;
}

void prof_clear(gmc_ctx* ctx) {
    for (int s = 0; s < kStages; ++s) {
        for (auto& pr : ctx->pending[s]) {
            (void)hipEventDestroy(pr.first);
            (void)hipEventDestroy(pr.second);
        }
        ctx->pending[s].clear();
        ctx->prof_ms[s] = 0;
        ctx->prof_n[s] = 0;
    }
}

#define GMC_LAUNCH(ctx, call)                                  \
    do {                                                       \
        hipError_t e_ = (call);                                \
        if (e_ != hipSuccess) return hip_fail(ctx, e_, #call); \
    } while (0)


}  // namespace

// ----------------------------------------------------------------------------
// Scratch of gmc_aggregate_static, for callers that cannot allocate: the
// server pass's row pointers, K * (ceil(d / kAggTopkRange) + 1) int32.  One
// copy per GPU, held until the process ends.  Host code never passes the
// array's name to a kernel (on the host it is only a stand-in for the
// symbol): it takes each device's address once with hipGetSymbolAddress and
// passes that.
// ----------------------------------------------------------------------------

static __device__ __align__(256) unsigned char scratch[GMC_STATIC_SCRATCH_BYTES];

namespace {

constexpr int kStaticDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch_ptr[kStaticDevices] = {};

// The current device's address of the static scratch (looked up on the
// device's first call, with that device current).
gmc_status static_scratch(int device, void** out) {
    if (device < 0 || device >= kStaticDevices)
        return fail(nullptr, GMC_EDEVICE, "gmc_aggregate_static: device id beyond the supported 64");
    std::lock_guard<std::mutex> lock(g_scratch_mu);
    if (!g_scratch_ptr[device]) {
        void* p = nullptr;
        hipError_t e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
        if (e != hipSuccess || !p) {
            (void)hipGetLastError();
            return fail(nullptr, GMC_EDEVICE,
                        std::string("gmc_aggregate_static: hipGetSymbolAddress: ") + hipGetErrorString(e));
        }
        g_scratch_ptr[device] = p;
    }
    *out = g_scratch_ptr[device];
    return GMC_OK;
}

}  // namespace

// ============================================================================
// C ABI
// ============================================================================

extern "C" {

gmc_status gmc_init(gmc_ctx** out, int64_t d, int32_t K, int32_t compressor, double ratio, double beta,
                    double eta, uint64_t seed) {
    if (!out) return fail(nullptr, GMC_EINVAL, "gmc_init: out is NULL");
    *out = nullptr;
    if (d < 1 || d > 0x7fffffffLL) return fail(nullptr, GMC_EINVAL, "gmc_init: d must be in [1, 2^31)");
    if (K < 1 || K > GMC_MAX_WORKERS) return fail(nullptr, GMC_EINVAL, "gmc_init: K must be in [1, 64]");
    if (compressor != GMC_TOPK_GLOBAL && compressor != GMC_TOPK_SEGMENTED && compressor != GMC_RBGS &&
        compressor != GMC_TOPK_APPROX)
        return fail(nullptr, GMC_EINVAL, "gmc_init: unknown compressor");
    if (!(ratio > 0.0 && ratio <= 1.0)) return fail(nullptr, GMC_EINVAL, "gmc_init: ratio must be in (0, 1]");
    if (!(beta >= 0.0 && beta < 1.0)) return fail(nullptr, GMC_EINVAL, "gmc_init: beta must be in [0, 1)");
    if (!(eta > 0.0 && std::isfinite(eta))) return fail(nullptr, GMC_EINVAL, "gmc_init: eta must be > 0 and finite");
    gmc_ctx* ctx = new (std::nothrow) gmc_ctx;
    if (!ctx) return fail(nullptr, GMC_ENOMEM, "gmc_init: host allocation failed");
    ctx->d = d;
    ctx->K = K;
    ctx->comp = compressor;
    ctx->ratio = ratio;
    ctx->beta = beta;
    ctx->eta = eta;
    ctx->seed = seed;
    derive_constants(ctx);
    ctx->seg_off = {0, d};
    ctx->keep = read_ratio(ratio);
    ctx->seg_k = {(int32_t)count_for(d, ctx->keep)};
    ctx->k_tot = ctx->seg_k[0];
    if (compressor == GMC_RBGS) {
        ctx->block = (int32_t)std::min<int64_t>(4096, d);
        ctx->nb = (int32_t)((d + ctx->block - 1) / ctx->block);
        ctx->n_sel = (int32_t)count_for(ctx->nb, ctx->keep);
    }
    hipError_t e = hipGetDevice(&ctx->device);
    if (e != hipSuccess) {
        delete ctx;
        return fail(nullptr, GMC_EDEVICE, std::string("gmc_init: hipGetDevice: ") + hipGetErrorString(e));
    }
    gmc_status st = prepare(ctx);
    if (st != GMC_OK) {
        g_init_error = ctx->err;
        release(ctx);
        delete ctx;
        return st;
    }
    *out = ctx;
    return GMC_OK;
}

gmc_status gmc_set_segments(gmc_ctx* ctx, int32_t n_seg, const int64_t* seg_off) {
    if (!ctx) return fail(nullptr, GMC_EINVAL, "gmc_set_segments: ctx is NULL");
    if (ctx->started) return fail(ctx, GMC_ESTATE, "gmc_set_segments: segments are fixed after the first step");
    if (ctx->comp == GMC_RBGS) return fail(ctx, GMC_EINVAL, "gmc_set_segments: not a top-s context");
    if (!seg_off || n_seg < 1 || n_seg > ctx->d) return fail(ctx, GMC_EINVAL, "gmc_set_segments: bad n_seg or NULL table");
    if ((ctx->comp == GMC_TOPK_GLOBAL || ctx->comp == GMC_TOPK_APPROX) && n_seg != 1)
        return fail(ctx, GMC_EINVAL, "gmc_set_segments: this compressor works on one segment");
    if (seg_off[0] != 0 || seg_off[n_seg] != ctx->d)
        return fail(ctx, GMC_EINVAL, "gmc_set_segments: offsets must start at 0 and end at d");
    for (int32_t i = 0; i < n_seg; ++i)
        if (seg_off[i + 1] <= seg_off[i]) return fail(ctx, GMC_EINVAL, "gmc_set_segments: offsets must increase strictly");
    ctx->seg_off.assign(seg_off, seg_off + n_seg + 1);
    ctx->seg_k.clear();
    ctx->k_tot = 0;
    for (int32_t i = 0; i < n_seg; ++i) {
        const int64_t k = count_for(seg_off[i + 1] - seg_off[i], ctx->keep);
        ctx->seg_k.push_back((int32_t)k);
        ctx->k_tot += k;
    }
    ctx->prepared = false;
    return prepare(ctx);
}

gmc_status gmc_set_block(gmc_ctx* ctx, int32_t block) {
    if (!ctx) return fail(nullptr, GMC_EINVAL, "gmc_set_block: ctx is NULL");
    if (ctx->started) return fail(ctx, GMC_ESTATE, "gmc_set_block: the block length is fixed after the first step");
    if (ctx->comp != GMC_RBGS) return fail(ctx, GMC_EINVAL, "gmc_set_block: not an RBGS context");
    if (block < 1 || block > ctx->d) return fail(ctx, GMC_EINVAL, "gmc_set_block: block must be in [1, d]");
    ctx->block = block;
    ctx->nb = (int32_t)((ctx->d + block - 1) / block);
    ctx->n_sel = (int32_t)count_for(ctx->nb, ctx->keep);
    ctx->prepared = false;
    return prepare(ctx);
}

gmc_status gmc_set_stream(gmc_ctx* ctx, void* hip_stream) {
    if (!ctx) return fail(nullptr, GMC_EINVAL, "gmc_set_stream: ctx is NULL");
    hipStream_t next = reinterpret_cast<hipStream_t>(hip_stream);
    if (next == ctx->stream) return GMC_OK;
    if (ctx->started) {
        // work of earlier calls may still be pending on the old stream and
        // shares the context's scratch with what comes next
        GMC_HIP(ctx, hipSetDevice(ctx->device));
        if (!ctx->stream_ev) GMC_HIP(ctx, hipEventCreateWithFlags(&ctx->stream_ev, hipEventDisableTiming));
        GMC_HIP(ctx, hipEventRecord(ctx->stream_ev, ctx->stream));
        GMC_HIP(ctx, hipStreamWaitEvent(next, ctx->stream_ev, 0));
    }
    ctx->stream = next;
    return GMC_OK;
}

int64_t gmc_message_len(const gmc_ctx* ctx) {
    if (!ctx) return -1;
    if (ctx->comp == GMC_TOPK_APPROX) return ctx->d;  // the count varies, up to d
    return ctx->comp == GMC_RBGS ? (int64_t)ctx->n_sel * ctx->block : ctx->k_tot;
}

int64_t gmc_index_len(const gmc_ctx* ctx) {
    if (!ctx) return -1;
    if (ctx->comp == GMC_TOPK_APPROX) return ctx->d;
    return ctx->comp == GMC_RBGS ? (int64_t)ctx->n_sel : ctx->k_tot;
}

int64_t gmc_count(int64_t n, double ratio) {
    if (n < 1 || n > 0x7fffffffLL || !(ratio > 0.0 && ratio <= 1.0)) return -1;
    return count_for(n, read_ratio(ratio));
}

}  // extern "C"

namespace {

gmc_status step_impl(gmc_ctx* ctx, const float* w_t_dev, const float* w_prev_dev, const float* const* grads_dev,
                     float* const* err_dev, float* const* y_dev, int32_t* idx_dev, float* val_dev,
                     int64_t* msg_len_dev, bool defer_zero = false) {
    StepArgs a{};
    a.defer_zero = defer_zero && ctx->comp != GMC_RBGS ? 1 : 0;
    a.w_t = w_t_dev;
    a.w_prev = w_prev_dev;
    a.c = ctx->c;
    a.h = ctx->h;
    a.q = ctx->q;
    a.rule = ctx->rule;
    a.detach = y_dev ? 1 : 0;
    a.d = (int32_t)ctx->d;
    a.seed = ctx->seed;
    a.t = (uint64_t)ctx->t;
    // w_t - w_prev is +0 outside the bitmap when w_t, w_prev are the last
    // server pass's output and input and no step ran since; after a pass in
    // place (output = input) the caller passes w_prev = NULL instead
    const bool rec = ctx->sparse_w && ctx->wbits_valid && ctx->wbits_t == ctx->t && w_t_dev == ctx->wbits_out;
    const bool rec_inplace = rec && ctx->wbits_in == ctx->wbits_out;
    a.wbits = (rec && (rec_inplace ? w_prev_dev == nullptr : w_prev_dev == ctx->wbits_in)) ? ctx->wbits : nullptr;
    // the top-s worker pass takes w_t - w_prev from that pass's change list
    // (written beside the bitmap) when it does not need w_t itself
    a.dlist = (a.wbits && use_dlist(ctx) && !y_dev) ? ctx->dlist : nullptr;
    a.dl_stride = ctx->dl_stride;
    if (!w_prev_dev && !(a.dlist && ctx->dl_stride == kDlistStrideFull && ctx->comp != GMC_RBGS && !y_dev))
        return fail(ctx, GMC_ESTATE,
                    "gmc_step: w_prev may be NULL only right after a server pass that updated w_t in place and "
                    "listed its changes (GMC_OPT_SPARSE_MOMENTUM with GMC_OPT_CHANGE_LIST 3)");
    ctx->wbits_valid = false;
    ctx->wbits_used_t = a.wbits ? ctx->t : -1;
    // workgroup order: w read everywhere (dense momentum term or GMC+'s
    // detached points) in runs of 2 chunks; at the changed components only,
    // runs of 1, or each chunk's workers on one XCD when the components the
    // last server pass changed (at most K times a top-s message) reach 5% of d
    const int64_t per_worker = ctx->comp == GMC_TOPK_APPROX ? count_for(ctx->d, ctx->keep) : ctx->k_tot;
    const bool dense_marks = ctx->comp != GMC_RBGS && (int64_t)ctx->K * per_worker * 20 >= ctx->d;
    a.run = (!a.wbits || y_dev) ? 2 : ((dense_marks && !a.dlist) ? 0 : 1);
    if (a.wbits) ++ctx->sparse_steps;
    for (int k = 0; k < ctx->K; ++k) {
        if (!grads_dev[k] || !err_dev[k] || (y_dev && !y_dev[k]))
            return fail(ctx, GMC_EINVAL, "gmc_step: NULL worker pointer");
        a.wp.g[k] = grads_dev[k];
        a.wp.e[k] = err_dev[k];
        a.wp.y[k] = y_dev ? y_dev[k] : nullptr;
    }
    GMC_TRY(prepare(ctx));
    GMC_HIP(ctx, hipSetDevice(ctx->device));
    ctx->started = true;
    const int64_t row_i = gmc_index_len(ctx), row_v = gmc_message_len(ctx);
    hipEvent_t ev;
    if (ctx->comp == GMC_RBGS) {
        GMC_TRY(prof_begin(ctx, 2, &ev));
        GMC_LAUNCH(ctx, launch_rbgs_sample(ctx->seed, (uint64_t)ctx->t, ctx->nb, ctx->n_sel, (int32_t)ctx->d,
                                           ctx->block, ctx->K, ctx->rbgs_bitmap, ctx->rbgs_blocks, ctx->rbgs_slot,
                                           idx_dev, row_i, msg_len_dev, ctx->rbgs_prev, ctx->rbgs_visit,
                                           ctx->rbgs_rbits, ctx->rbgs_meta, ctx->stream));
        GMC_TRY(prof_end(ctx, 2, ev));
        GMC_TRY(prof_begin(ctx, 0, &ev));
        uint64_t vec_mask = 0;
        const bool shared_ok = ((uintptr_t)w_t_dev & 15u) == 0 && ((uintptr_t)w_prev_dev & 15u) == 0 &&
                               ((uintptr_t)val_dev & 15u) == 0 && (row_v & 3) == 0 && (ctx->block & 3) == 0;
        for (int k = 0; k < ctx->K && shared_ok; ++k)
            if ((((uintptr_t)grads_dev[k] | (uintptr_t)err_dev[k] | (uintptr_t)a.wp.y[k]) & 15u) == 0)
                vec_mask |= 1ull << k;
        GMC_LAUNCH(ctx, launch_rbgs_fused(a, ctx->K, ctx->block, ctx->rbgs_slot, val_dev, row_v, vec_mask,
                                          ctx->stream));
        GMC_TRY(prof_end(ctx, 0, ev));
    } else {
        // worker k takes the vector pass when its rows and w_t, w_prev are 16-byte aligned
        uint64_t vec_mask = 0;
        const bool w_ok = ((uintptr_t)w_t_dev & 15u) == 0 && ((uintptr_t)w_prev_dev & 15u) == 0;
        for (int k = 0; k < ctx->K && w_ok; ++k)
            if ((((uintptr_t)grads_dev[k] | (uintptr_t)err_dev[k] | (uintptr_t)a.wp.y[k]) & 15u) == 0)
                vec_mask |= 1ull << k;
        // the vector kernel takes every chunk of the workers in vec_mask
        // (partial and unaligned ones element-wise); the element-wise kernel
        // every chunk of the others
        const uint64_t all = ctx->K == 64 ? ~0ull : ((1ull << ctx->K) - 1ull);
        // the context's first step: speculative thresholds from a sample of u
        if (!ctx->seeded && !ctx->force_full) GMC_LAUNCH(ctx, launch_topk_seed(a, ctx->geo, ctx->scr, ctx->stream));
        ctx->seeded = true;
        if (vec_mask) {
            GMC_TRY(prof_begin(ctx, 0, &ev));
            GMC_LAUNCH(ctx, launch_topk_fused_vec(a, ctx->geo, ctx->scr, vec_mask, ctx->stream));
            GMC_TRY(prof_end(ctx, 0, ev));
        }
        if (vec_mask != all) {
            GMC_TRY(prof_begin(ctx, 1, &ev));
            GMC_LAUNCH(ctx, launch_topk_fused_gen(a, ctx->geo, ctx->scr, vec_mask, ctx->stream));
            GMC_TRY(prof_end(ctx, 1, ev));
        }
        GMC_TRY(prof_begin(ctx, 2, &ev));
        GMC_LAUNCH(ctx, launch_topk_compact(a, ctx->geo, ctx->scr, ctx->force_full, ctx->margin, ctx->stream));
        for (int pass = 2; pass <= 3; ++pass)
            GMC_LAUNCH(ctx, launch_topk_hist(pass, a, ctx->geo, ctx->scr, ctx->force_full, ctx->margin, msg_len_dev,
                                             ctx->k_tot, ctx->stream));
        if (ctx->comp == GMC_TOPK_APPROX)  // exact top-s counts in the third pass
            GMC_LAUNCH(ctx, launch_topk_count(a, ctx->geo, ctx->scr, msg_len_dev, ctx->k_tot, ctx->stream));
        GMC_TRY(prof_end(ctx, 2, ev));
        GMC_TRY(prof_begin(ctx, 3, &ev));
        GMC_LAUNCH(ctx, launch_topk_emit(a, ctx->geo, ctx->scr, idx_dev, val_dev, row_v, ctx->stream));
        GMC_TRY(prof_end(ctx, 3, ev));
    }
    ctx->t += 1;
    return GMC_OK;
}

}  // namespace

extern "C" {

gmc_status gmc_step(gmc_ctx* ctx, const float* w_t_dev, const float* w_prev_dev, const float* const* grads_dev,
                    float* const* err_dev, int32_t* idx_dev, float* val_dev, int64_t* msg_len_dev) {
    if (!ctx) return fail(nullptr, GMC_EINVAL, "gmc_step: ctx is NULL");
    if (!w_t_dev || !grads_dev || !err_dev || !idx_dev || !val_dev || !msg_len_dev)
        return fail(ctx, GMC_EINVAL, "gmc_step: NULL argument");
    return step_impl(ctx, w_t_dev, w_prev_dev, grads_dev, err_dev, nullptr, idx_dev, val_dev, msg_len_dev);
}

gmc_status gmc_step_detach(gmc_ctx* ctx, const float* w_t_dev, const float* w_prev_dev,
                           const float* const* grads_dev, float* const* err_dev, float* const* w_k_dev,
                           int32_t* idx_dev, float* val_dev, int64_t* msg_len_dev) {
    if (!ctx) return fail(nullptr, GMC_EINVAL, "gmc_step_detach: ctx is NULL");
    if (!w_t_dev || !w_prev_dev || !grads_dev || !err_dev || !w_k_dev || !idx_dev || !val_dev || !msg_len_dev)
        return fail(ctx, GMC_EINVAL, "gmc_step_detach: NULL argument");
    if (ctx->rule == kRuleServerMomentum)
        return fail(ctx, GMC_EINVAL,
                    "gmc_step_detach: with momentum on the server w_{t+1} differs from w_t everywhere; "
                    "use gmc_detach after the apply");
    return step_impl(ctx, w_t_dev, w_prev_dev, grads_dev, err_dev, w_k_dev, idx_dev, val_dev, msg_len_dev);
}

}  // extern "C"

namespace {

// rowptr_ready: the messages are the ones the context's last gmc_step just
// emitted (gmc_iteration), whose emit kernel also wrote the row pointers
gmc_status aggregate_impl(gmc_ctx* ctx, const int32_t* idx_dev, const float* val_dev, const int64_t* msg_len_dev,
                          FinishArgs& f, bool rowptr_ready = false) {
    GMC_TRY(prepare(ctx));
    GMC_HIP(ctx, hipSetDevice(ctx->device));
    f.s = ctx->s;
    f.b = ctx->b;
    f.q = ctx->q;
    // the bitmap for the next worker pass: not with momentum on the server
    // (w_{t+1} differs from w_t everywhere there); in place only for top-s
    // with a change list that holds whole ranges (the next worker pass then
    // has no w_{t-1} and takes w_{t+1} - w_t from it) and without GMC+'s
    // detached points
    const bool inplace = f.w_in && f.w_in == f.w_out;
    const bool mark = ctx->sparse_w && f.w_in && f.w_out && ctx->rule != kRuleServerMomentum &&
                      (!inplace || (ctx->comp != GMC_RBGS && ctx->dl_stride == kDlistStrideFull && !f.detach));
    f.wbits = mark ? ctx->wbits : nullptr;
    f.dlist = (mark && use_dlist(ctx)) ? ctx->dlist : nullptr;
    f.dl_stride = ctx->dl_stride;
    f.nf = ctx->nf;
    f.nf_epoch = ctx->nf_epoch;
    // out of place: w_out is the last pass's input buffer and w_in its
    // output, and the worker pass in between read them through that pass's
    // bitmap: w_out still holds w_{t-1}, which equals w_t off the marks, and
    // w_{t+1} equals w_t off the marks and this pass's sent components.  In
    // place: w_in is the last pass's output, so it holds w_t everywhere.
    const bool chain = mark && ctx->wbits_pair && ctx->wbits_used_t == ctx->t - 1 && ctx->wbits_out == f.w_in;
    f.sparse_apply = (chain && (inplace || ctx->wbits_in == f.w_out)) ? 1 : 0;
    f.inplace = (f.sparse_apply && inplace) ? 1 : 0;
    if (f.sparse_apply) ++ctx->sparse_applies;
    ctx->wbits_used_t = -1;
    ctx->wbits_pair = mark;
    ctx->wbits_valid = mark;
    ctx->wbits_in = f.w_in;
    ctx->wbits_out = f.w_out;
    ctx->wbits_t = ctx->t;
    const int64_t row_i = gmc_index_len(ctx), row_v = gmc_message_len(ctx);
    hipEvent_t ev;
    GMC_TRY(prof_begin(ctx, 4, &ev));
    if (ctx->comp == GMC_RBGS) {
        GMC_LAUNCH(ctx, launch_agg_rbgs(ctx->K, (int32_t)ctx->d, ctx->block, ctx->n_sel, ctx->rbgs_slot, val_dev,
                                        row_v, f, ctx->rbgs_visit, ctx->rbgs_meta,
                                        ctx->stream));
    } else {
        if (!rowptr_ready)
            GMC_LAUNCH(ctx, launch_agg_rowptr(ctx->K, (int32_t)ctx->d, idx_dev, row_i, msg_len_dev, ctx->rowptr,
                                              ctx->n_ranges, ctx->stream));
        GMC_LAUNCH(ctx, launch_agg_topk(ctx->K, (int32_t)ctx->d, idx_dev, row_i, val_dev, row_v, ctx->rowptr,
                                        ctx->n_ranges, f, ctx->stream));
    }
    GMC_TRY(prof_end(ctx, 4, ev));
    return GMC_OK;
}

}  // namespace

extern "C" {

gmc_status gmc_aggregate(gmc_ctx* ctx, const int32_t* idx_dev, const float* val_dev, const int64_t* msg_len_dev,
                         float* update_dev) {
    if (!ctx) return fail(nullptr, GMC_EINVAL, "gmc_aggregate: ctx is NULL");
    if (!idx_dev || !val_dev || !msg_len_dev || !update_dev) return fail(ctx, GMC_EINVAL, "gmc_aggregate: NULL argument");
    if (!ctx->started) return fail(ctx, GMC_ESTATE, "gmc_aggregate: no gmc_step has been taken yet");
    FinishArgs f{};
    f.update = update_dev;
    return aggregate_impl(ctx, idx_dev, val_dev, msg_len_dev, f);
}

gmc_status gmc_aggregate_apply(gmc_ctx* ctx, const int32_t* idx_dev, const float* val_dev,
                               const int64_t* msg_len_dev, const float* w_dev, float* w_out_dev,
                               float* update_dev) {
    if (!ctx) return fail(nullptr, GMC_EINVAL, "gmc_aggregate_apply: ctx is NULL");
    if (!idx_dev || !val_dev || !msg_len_dev || !w_dev || !w_out_dev)
        return fail(ctx, GMC_EINVAL, "gmc_aggregate_apply: NULL argument");
    if (update_dev && (update_dev == w_out_dev || update_dev == w_dev))
        return fail(ctx, GMC_EINVAL, "gmc_aggregate_apply: update may not alias w or w_out");
    if (ctx->rule == kRuleServerMomentum)
        return fail(ctx, GMC_EINVAL, "gmc_aggregate_apply: momentum on the server needs w_{t-1}; use gmc_finish");
    if (!ctx->started) return fail(ctx, GMC_ESTATE, "gmc_aggregate_apply: no gmc_step has been taken yet");
    FinishArgs f{};
    f.w_in = w_dev;
    f.w_out = w_out_dev;
    f.update = update_dev;
    return aggregate_impl(ctx, idx_dev, val_dev, msg_len_dev, f);
}

gmc_status gmc_finish(gmc_ctx* ctx, const int32_t* idx_dev, const float* val_dev, const int64_t* msg_len_dev,
                      const float* w_dev, const float* w_prev_dev, float* w_out_dev, float* update_dev,
                      const float* const* err_dev, float* const* w_k_dev) {
    if (!ctx) return fail(nullptr, GMC_EINVAL, "gmc_finish: ctx is NULL");
    if (!idx_dev || !val_dev || !msg_len_dev || !w_dev || !w_out_dev)
        return fail(ctx, GMC_EINVAL, "gmc_finish: NULL argument");
    if (update_dev && (update_dev == w_out_dev || update_dev == w_dev || update_dev == w_prev_dev))
        return fail(ctx, GMC_EINVAL, "gmc_finish: update may not alias w, w_prev or w_out");
    if (ctx->rule == kRuleServerMomentum && !w_prev_dev)
        return fail(ctx, GMC_EINVAL, "gmc_finish: momentum on the server needs w_prev");
    if (w_prev_dev && w_prev_dev == w_dev) return fail(ctx, GMC_EINVAL, "gmc_finish: w_prev may not alias w");
    if (!ctx->started) return fail(ctx, GMC_ESTATE, "gmc_finish: no gmc_step has been taken yet");
    FinishArgs f{};
    f.w_in = w_dev;
    f.w_prev = ctx->rule == kRuleServerMomentum ? w_prev_dev : nullptr;
    f.w_out = w_out_dev;
    f.update = update_dev;
    if (w_k_dev) {
        if (ctx->rule == kRuleServerMomentum)
            return fail(ctx, GMC_EINVAL, "gmc_finish: detached points with momentum on the server: use gmc_detach");
        if (!err_dev) return fail(ctx, GMC_EINVAL, "gmc_finish: detached points need err");
        f.detach = 1;
        f.rows16 = 1;
        for (int k = 0; k < ctx->K; ++k) {
            if (!err_dev[k] || !w_k_dev[k]) return fail(ctx, GMC_EINVAL, "gmc_finish: NULL worker pointer");
            f.e[k] = err_dev[k];
            f.y[k] = w_k_dev[k];
            if ((((uintptr_t)err_dev[k] | (uintptr_t)w_k_dev[k]) & 15u) != 0) f.rows16 = 0;
        }
    }
    return aggregate_impl(ctx, idx_dev, val_dev, msg_len_dev, f);
}

gmc_status gmc_detach(gmc_ctx* ctx, const float* w_dev, const float* const* err_dev, float* const* w_k_dev) {
    if (!ctx) return fail(nullptr, GMC_EINVAL, "gmc_detach: ctx is NULL");
    if (!w_dev || !err_dev || !w_k_dev) return fail(ctx, GMC_EINVAL, "gmc_detach: NULL argument");
    DetachArgs a{};
    a.w = w_dev;
    a.q = ctx->q;
    a.d = (int32_t)ctx->d;
    for (int k = 0; k < ctx->K; ++k) {
        if (!err_dev[k] || !w_k_dev[k]) return fail(ctx, GMC_EINVAL, "gmc_detach: NULL worker pointer");
        a.e[k] = err_dev[k];
        a.y[k] = w_k_dev[k];
    }
    GMC_HIP(ctx, hipSetDevice(ctx->device));
    GMC_LAUNCH(ctx, launch_detach(a, ctx->K, ctx->stream));
    return GMC_OK;
}

gmc_status gmc_iteration(gmc_ctx* ctx, const float* w_t_dev, float* w_prev_io_dev, const float* const* grads_dev,
                         float* const* err_dev, int32_t* idx_dev, float* val_dev, int64_t* msg_len_dev) {
    if (!ctx) return fail(nullptr, GMC_EINVAL, "gmc_iteration: ctx is NULL");
    if (!w_t_dev || !w_prev_io_dev || !grads_dev || !err_dev || !idx_dev || !val_dev || !msg_len_dev)
        return fail(ctx, GMC_EINVAL, "gmc_iteration: NULL argument");
    if (w_t_dev == w_prev_io_dev) return fail(ctx, GMC_EINVAL, "gmc_iteration: w_prev_io may not alias w_t");
    // the top-s emit leaves the residual's zeros at the sent components to
    // the server pass, which stages every message entry anyway: scattered
    // writes there overlap its chain of dependent loads, while at the emit's
    // end they hold up the launch
    const bool defer = ctx->comp != GMC_RBGS;
    GMC_TRY(step_impl(ctx, w_t_dev, w_prev_io_dev, grads_dev, err_dev, nullptr, idx_dev, val_dev, msg_len_dev,
                      defer));
    FinishArgs f{};
    f.zero_e = defer ? 1 : 0;
    for (int k = 0; defer && k < ctx->K; ++k) f.ez[k] = err_dev[k];
    f.w_in = w_t_dev;
    f.w_out = w_prev_io_dev;
    f.w_prev = ctx->rule == kRuleServerMomentum ? w_prev_io_dev : nullptr;  // read before written, per component
    return aggregate_impl(ctx, idx_dev, val_dev, msg_len_dev, f, true);
}

gmc_status gmc_iteration_inplace(gmc_ctx* ctx, float* w_dev, const float* w_prev_dev, const float* const* grads_dev,
                                 float* const* err_dev, int32_t* idx_dev, float* val_dev, int64_t* msg_len_dev) {
    if (!ctx) return fail(nullptr, GMC_EINVAL, "gmc_iteration_inplace: ctx is NULL");
    if (!w_dev || !grads_dev || !err_dev || !idx_dev || !val_dev || !msg_len_dev)
        return fail(ctx, GMC_EINVAL, "gmc_iteration_inplace: NULL argument");
    if (ctx->comp == GMC_RBGS || ctx->rule == kRuleServerMomentum)
        return fail(ctx, GMC_EINVAL, "gmc_iteration_inplace: top-s under GMC_RULE_GMC or GMC_RULE_LR_IN_RESIDUAL only");
    if (!ctx->sparse_w || ctx->dl_stride != kDlistStrideFull)
        return fail(ctx, GMC_EINVAL,
                    "gmc_iteration_inplace: needs GMC_OPT_SPARSE_MOMENTUM and GMC_OPT_CHANGE_LIST 3, which keep "
                    "w_{t+1} - w_t for the next iteration");
    GMC_TRY(step_impl(ctx, w_dev, w_prev_dev, grads_dev, err_dev, nullptr, idx_dev, val_dev, msg_len_dev, true));
    FinishArgs f{};
    f.zero_e = 1;
    for (int k = 0; k < ctx->K; ++k) f.ez[k] = err_dev[k];
    f.w_in = w_dev;
    f.w_out = w_dev;
    return aggregate_impl(ctx, idx_dev, val_dev, msg_len_dev, f, true);
}

gmc_status gmc_apply(gmc_ctx* ctx, float* w_dev, float* w_prev_out_dev, const float* update_dev) {
    if (!ctx) return fail(nullptr, GMC_EINVAL, "gmc_apply: ctx is NULL");
    if (!w_dev || !update_dev) return fail(ctx, GMC_EINVAL, "gmc_apply: NULL argument");
    if (w_prev_out_dev == w_dev) return fail(ctx, GMC_EINVAL, "gmc_apply: w_prev_out may not alias w");
    if (ctx->rule == kRuleServerMomentum)
        return fail(ctx, GMC_EINVAL, "gmc_apply: momentum on the server needs w_{t-1}; use gmc_finish");
    if (!ctx->started) return fail(ctx, GMC_ESTATE, "gmc_apply: no gmc_step has been taken yet");
    drop_record(ctx);
    GMC_HIP(ctx, hipSetDevice(ctx->device));
    hipEvent_t ev;
    GMC_TRY(prof_begin(ctx, 5, &ev));
    GMC_LAUNCH(ctx, launch_apply((int32_t)ctx->d, w_dev, w_prev_out_dev, update_dev, ctx->stream));
    GMC_TRY(prof_end(ctx, 5, ev));
    return GMC_OK;
}

gmc_status gmc_set_rule(gmc_ctx* ctx, int32_t rule) {
    if (!ctx) return fail(nullptr, GMC_EINVAL, "gmc_set_rule: ctx is NULL");
    if (rule != kRuleGmc && rule != kRuleServerMomentum && rule != kRuleLrInResidual)
        return fail(ctx, GMC_EINVAL, "gmc_set_rule: unknown rule");
    if (ctx->started) return fail(ctx, GMC_ESTATE, "gmc_set_rule: the rule is fixed after the first step");
    ctx->rule = rule;
    derive_constants(ctx);
    return GMC_OK;
}

gmc_status gmc_set_eta(gmc_ctx* ctx, double eta) {
    if (!ctx) return fail(nullptr, GMC_EINVAL, "gmc_set_eta: ctx is NULL");
    if (!(eta > 0.0 && std::isfinite(eta))) return fail(ctx, GMC_EINVAL, "gmc_set_eta: eta must be > 0 and finite");
    ctx->eta = eta;
    derive_constants(ctx);
    return GMC_OK;
}

gmc_status gmc_set_lambda(gmc_ctx* ctx, double lambda) {
    if (!ctx) return fail(nullptr, GMC_EINVAL, "gmc_set_lambda: ctx is NULL");
    if (!(lambda >= 0.0 && lambda <= 1.0)) return fail(ctx, GMC_EINVAL, "gmc_set_lambda: lambda must be in [0, 1]");
    ctx->lambda = lambda;
    derive_constants(ctx);
    return GMC_OK;
}

gmc_status gmc_get_step(const gmc_ctx* ctx, int64_t* t) {
    if (!ctx || !t) return fail(nullptr, GMC_EINVAL, "gmc_get_step: NULL argument");
    *t = ctx->t;
    return GMC_OK;
}

gmc_status gmc_set_step(gmc_ctx* ctx, int64_t t) {
    if (!ctx) return fail(nullptr, GMC_EINVAL, "gmc_set_step: ctx is NULL");
    if (t < 0) return fail(ctx, GMC_EINVAL, "gmc_set_step: t must be >= 0");
    ctx->t = t;
    drop_record(ctx);  // a resume may bring other parameters
    return GMC_OK;
}

gmc_status gmc_set_option(gmc_ctx* ctx, int32_t option, int64_t value) {
    if (!ctx) return fail(nullptr, GMC_EINVAL, "gmc_set_option: ctx is NULL");
    switch (option) {
        case GMC_OPT_FORCE_FULL_SELECT:
            ctx->force_full = value ? 1 : 0;
            return GMC_OK;
        case GMC_OPT_CAND_MARGIN:
            if (value < 4 || value > 4096)
                return fail(ctx, GMC_EINVAL, "gmc_set_option: margin (quarters of k) must be in [4, 4096]");
            ctx->margin = (int)value;
            return GMC_OK;
        case GMC_OPT_CAND_CAP_MULT:
            if (value < 1 || value > 1024) return fail(ctx, GMC_EINVAL, "gmc_set_option: cap multiple must be in [1, 1024]");
            if (ctx->started) return fail(ctx, GMC_ESTATE, "gmc_set_option: capacity is fixed after the first step");
            ctx->cap_mult = (int)value;
            ctx->prepared = false;
            return prepare(ctx);
        case GMC_OPT_SAMPLE_STRATUM:
            if (ctx->comp != GMC_TOPK_APPROX)
                return fail(ctx, GMC_EINVAL, "gmc_set_option: the sample stratum belongs to GMC_TOPK_APPROX");
            if (value < 1 || value > ctx->d) return fail(ctx, GMC_EINVAL, "gmc_set_option: stratum must be in [1, d]");
            if (ctx->started) return fail(ctx, GMC_ESTATE, "gmc_set_option: the stratum is fixed after the first step");
            ctx->stratum = (int32_t)value;
            ctx->prepared = false;
            return prepare(ctx);
        case GMC_OPT_SPARSE_MOMENTUM:
            ctx->sparse_w = value ? 1 : 0;
            drop_record(ctx);
            return GMC_OK;
        case GMC_OPT_CHANGE_LIST: {
            if (value < 0 || value > 3)
                return fail(ctx, GMC_EINVAL, "gmc_set_option: change list must be 0, 1, 2 or 3");
            const int32_t stride = value == 3 ? kDlistStrideFull : kDlistStride;
            if (stride != ctx->dl_stride && ctx->started)
                return fail(ctx, GMC_ESTATE, "gmc_set_option: change list 3 is set or cleared before the first step only");
            ctx->change_list = (int)value;
            drop_record(ctx);  // the list of the last pass may not have been written
            if (stride != ctx->dl_stride) {
                ctx->dl_stride = stride;
                ctx->prepared = false;
                return prepare(ctx);
            }
            return GMC_OK;
        }
        case GMC_OPT_PROFILE:
            if (ctx->profile) GMC_HIP(ctx, hipStreamSynchronize(ctx->stream));
            prof_clear(ctx);
            ctx->profile = (uint32_t)value & ((1u << kStages) - 1u);
            return GMC_OK;
        default:
            return fail(ctx, GMC_EINVAL, "gmc_set_option: unknown option");
    }
}

gmc_status gmc_stats(gmc_ctx* ctx, int64_t* out, int32_t n) {
    if (!ctx || !out || n < 0) return fail(ctx, GMC_EINVAL, "gmc_stats: bad argument");
    GMC_HIP(ctx, hipSetDevice(ctx->device));
    GMC_HIP(ctx, hipStreamSynchronize(ctx->stream));
    int64_t host[8] = {0};
    if (ctx->stats) GMC_HIP(ctx, hipMemcpy(host, ctx->stats, sizeof host, hipMemcpyDeviceToHost));
    host[0] = ctx->t;
    host[5] = ctx->sparse_steps;
    host[6] = ctx->sparse_applies;
    for (int32_t i = 0; i < n && i < 8; ++i) out[i] = host[i];
    return GMC_OK;
}

gmc_status gmc_pair_stats(gmc_ctx* ctx, int32_t* mode, int64_t* cand, int32_t n, int32_t* n_pairs) {
    if (!ctx || !n_pairs || n < 0 || (n > 0 && (!mode || !cand)))
        return fail(ctx, GMC_EINVAL, "gmc_pair_stats: bad argument");
    if (ctx->comp == GMC_RBGS) return fail(ctx, GMC_EINVAL, "gmc_pair_stats: RBGS selects no (worker, segment) pairs");
    if (!ctx->started) return fail(ctx, GMC_ESTATE, "gmc_pair_stats: no step taken yet");
    const int32_t np = ctx->K * ctx->geo.n_seg;
    *n_pairs = np;
    GMC_HIP(ctx, hipSetDevice(ctx->device));
    GMC_HIP(ctx, hipStreamSynchronize(ctx->stream));
    std::vector<PairState> host((size_t)np);
    GMC_HIP(ctx, hipMemcpy(host.data(), ctx->scr.pair, sizeof(PairState) * (size_t)np, hipMemcpyDeviceToHost));
    for (int32_t i = 0; i < n && i < np; ++i) {
        mode[i] = host[(size_t)i].mode == 0 ? 0 : 1;  // collected full data is the full-data path
        cand[i] = (int64_t)host[(size_t)i].cand_used;
    }
    return GMC_OK;
}

gmc_status gmc_profile_read(gmc_ctx* ctx, double* ms, int64_t* launches, int32_t n) {
    if (!ctx || !ms || !launches || n < 0) return fail(ctx, GMC_EINVAL, "gmc_profile_read: bad argument");
    GMC_HIP(ctx, hipSetDevice(ctx->device));
    for (int s = 0; s < kStages; ++s) GMC_TRY(prof_fold(ctx, s));
    for (int32_t i = 0; i < n && i < kStages; ++i) {
        ms[i] = ctx->prof_ms[i];
        launches[i] = ctx->prof_n[i];
    }
    return GMC_OK;
}

const char* gmc_last_error(const gmc_ctx* ctx) {
    return ctx ? ctx->err.c_str() : g_init_error.c_str();
}

void gmc_destroy(gmc_ctx* ctx) {
    if (!ctx) return;
    prof_clear(ctx);
    release(ctx);
    if (ctx->stream_ev) (void)hipEventDestroy(ctx->stream_ev);
    delete ctx;
}

gmc_status gmc_aggregate_static(int64_t d, int32_t K, double eta, const int32_t* idx_dev, int64_t index_len,
                                const float* val_dev, int64_t message_len, const int64_t* msg_len_dev,
                                float* update_dev, void* hip_stream) {
    if (d < 1 || d > 0x7fffffffLL) return fail(nullptr, GMC_EINVAL, "gmc_aggregate_static: d must be in [1, 2^31)");
    if (K < 1 || K > GMC_MAX_WORKERS) return fail(nullptr, GMC_EINVAL, "gmc_aggregate_static: K must be in [1, 64]");
    if (!(eta > 0.0 && std::isfinite(eta)))
        return fail(nullptr, GMC_EINVAL, "gmc_aggregate_static: eta must be > 0 and finite");
    if (index_len < 0 || message_len < index_len || index_len > 0x7fffffffLL)
        return fail(nullptr, GMC_EINVAL, "gmc_aggregate_static: need 0 <= index_len <= message_len, index_len < 2^31");
    if (!idx_dev || !val_dev || !msg_len_dev || !update_dev)
        return fail(nullptr, GMC_EINVAL, "gmc_aggregate_static: NULL argument");
    const int32_t n_ranges = (int32_t)((d + kAggTopkRange - 1) / kAggTopkRange);
    const size_t need = (size_t)K * (size_t)(n_ranges + 1) * sizeof(int32_t);
    if (need > (size_t)GMC_STATIC_SCRATCH_BYTES)
        return fail(nullptr, GMC_EINVAL,
                    "gmc_aggregate_static: K * (ceil(d/4096) + 1) row pointers need " + std::to_string(need) +
                        " bytes, more than the static scratch's " + std::to_string((size_t)GMC_STATIC_SCRATCH_BYTES));
    int device = 0;
    hipError_t e = hipGetDevice(&device);
    if (e != hipSuccess) return hip_fail(nullptr, e, "gmc_aggregate_static: hipGetDevice");
    void* ptr = nullptr;
    GMC_TRY(static_scratch(device, &ptr));
    hipStream_t st = reinterpret_cast<hipStream_t>(hip_stream);
    int32_t* rowptr = reinterpret_cast<int32_t*>(ptr);  // every entry is written before it is read
    FinishArgs f{};
    f.update = update_dev;
    f.s = (float)(eta / (double)K);
    e = launch_agg_rowptr(K, (int32_t)d, idx_dev, index_len, msg_len_dev, rowptr, n_ranges, st);
    if (e != hipSuccess) return hip_fail(nullptr, e, "gmc_aggregate_static: row pointers");
    e = launch_agg_topk(K, (int32_t)d, idx_dev, index_len, val_dev, message_len, rowptr, n_ranges, f, st);
    if (e != hipSuccess) return hip_fail(nullptr, e, "gmc_aggregate_static: sum");
    return GMC_OK;
}

gmc_status gmc_calib_copy(void* hip_stream, float* dst_dev, const float* src_dev, int64_t n) {
    if (!dst_dev || !src_dev || n < 0) return fail(nullptr, GMC_EINVAL, "gmc_calib_copy: bad argument");
    if (n == 0) return GMC_OK;
    hipError_t e = launch_calib_copy(dst_dev, src_dev, n, reinterpret_cast<hipStream_t>(hip_stream));
    if (e != hipSuccess) return hip_fail(nullptr, e, "gmc_calib_copy");
    return GMC_OK;
}

gmc_status gmc_calib_stream(void* hip_stream, float* e_dev, const float* g_dev, int64_t row_pitch, int32_t K,
                            int64_t d) {
    if (!e_dev || !g_dev) return fail(nullptr, GMC_EINVAL, "gmc_calib_stream: NULL argument");
    if (d < 1 || d >= (int64_t(1) << 31) || K < 1 || row_pitch < d)
        return fail(nullptr, GMC_EINVAL, "gmc_calib_stream: need 1 <= d < 2^31, K >= 1, row_pitch >= d");
    const int64_t span = (int64_t)(K - 1) * row_pitch + d;  // elements each buffer covers
    if ((e_dev < g_dev + span) && (g_dev < e_dev + span))
        return fail(nullptr, GMC_EINVAL, "gmc_calib_stream: e and g overlap");
    hipError_t e = launch_calib_stream(e_dev, g_dev, row_pitch, K, (int32_t)d, reinterpret_cast<hipStream_t>(hip_stream));
    if (e != hipSuccess) return hip_fail(nullptr, e, "gmc_calib_stream");
    return GMC_OK;
}

}  // extern "C"
