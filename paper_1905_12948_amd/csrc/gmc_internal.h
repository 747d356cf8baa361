// Internal declarations of the GMC device library: launch geometry, the
// device-side scratch layout and the kernel launchers.  Not part of the ABI.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace gmc {

constexpr int kMaxWorkers = 64;

// Fused worker pass: chunks of kChunk consecutive elements of a segment; the
// vector kernel gives one workgroup (256 threads x 8 floats) to each (chunk,
// worker), the element-wise kernel one wavefront.
constexpr int kWave = 64;
constexpr int kWavesPerGroup = 4;
constexpr int kGroup = kWave * kWavesPerGroup;  // 256 threads
constexpr int kVecIters = 8;
constexpr int kChunk = kWave * 4 * kVecIters;   // 2048 elements

// Selection: the fused pass leaves each (worker, chunk)'s candidates in the
// chunk's own staging slot; compaction groups of kCompactChunks chunks pack
// them, in index order, into the pair's candidate list, in tiles of kTile
// candidates (one workgroup each).  The histogram, count and emit passes
// read the list (or, on the full-data path, the segment's u) as "slices":
// seg_slices even shares, one workgroup each.
constexpr int kCompactChunks = 256;        // chunks per compaction group (one per thread)
// Each group's total is kept as kGrpSub sub-totals, chunk c adding into
// c % kGrpSub: the device-scope adds of a group's chunks then spread over
// that many addresses (with only a few groups, a small workload's adds all
// met on a handful of words and stretched its worker pass).
constexpr int kGrpSub = 16;
constexpr int kTile = kGroup * 8;          // candidates one copy workgroup moves
constexpr int64_t kSliceElems = 1 << 19;   // full-data elements per slice (at most)
constexpr int64_t kSliceCands = 8192;      // usual candidates per slice (more when a list runs long)
constexpr int64_t kHistSliceCands = 4096;  // candidates per second-pass workgroup (one round of loads each)
constexpr int kMaxSlices = 256;
constexpr int kSlHist = 513;               // per slice: suffix sums of a 512-bin histogram + a count above

// Radix select over the 31-bit magnitude key in three digits: 11 + 11 + 9.
constexpr int kBins = 2048;
constexpr int kShift1 = 20, kShift2 = 9;

// Aggregation range per workgroup (RBGS), and for top-s with the number of
// message entries one workgroup stages in LDS.
constexpr int kAggRange = 2048;
constexpr int kAggTopkRange = 4096;
constexpr int kAggTopkStage = 512;
// sparse messages (few entries per range on average) stage fewer, so that
// eight workgroups fit on a CU instead of seven
constexpr int kAggTopkStageSmall = 128;

constexpr uint32_t kNoThreshold = 0xffffffffu;  // no speculative candidates

// The components a top-s server pass changed, per range of kAggTopkRange:
// a block of dl_stride int2 (kDlistStride, or kDlistStrideFull for a list
// that holds every component of a range, which in-place server passes
// need), [0] = {count, 0} (-1: more than the block holds), then {offset in
// the range, bits of fl(w_{t+1} - w_t)} per changed component, in no
// particular order.
constexpr int kDlistStride = 512;
constexpr int kDlistStrideFull = kAggTopkRange + 1;
// The list is kept when the two parameter vectors (8 d bytes) outgrow the
// 256 MB Infinity Cache: below that, the worker pass's reads of w_t and w_prev
// at the marked cache lines are served by that cache (and warm it for the
// server pass), above it every XCD fetches them from HBM.
constexpr int64_t kDlistMinParamBytes = int64_t(256) << 20;

// A full-data pair whose first digit leaves few components at or above its
// bin (at most 1/kCollectDiv of the segment) is "collected": the second pass
// also gathers those components, in index order, into the pair's staging
// rows, and the third pass and the emit read only them.
constexpr int kModeCollected = 3;
constexpr int64_t kCollectDiv = 8;

// First-step threshold from a sample (topk_seed_kernel): runs of kSeedRun
// consecutive components every kSeedStride of each segment of at least
// kSeedMinLen components, kSeedRunsPerGroup runs per workgroup; the threshold
// sits at the sample's key of rank about kSeedMult k |S| / n.
constexpr int kSeedRun = 32;
constexpr int kSeedStride = 512;
constexpr int kSeedRunsPerGroup = 256;
constexpr int64_t kSeedMinLen = 1 << 16;
constexpr int kSeedMult = 4;

// Update rules: GMC (Algorithm 1) and the two other ways of combining
// momentum with error feedback that the appendix compares it with.
constexpr int kRuleGmc = 0;             // u = (e + g) - (beta/eta)(w_t - w_{t-1})
constexpr int kRuleServerMomentum = 1;  // u = e + g; the server adds beta (w_t - w_{t-1})
constexpr int kRuleLrInResidual = 2;    // u = (e + eta g) - beta (w_t - w_{t-1})

struct WorkerPtrs {
    const float* g[kMaxWorkers];
    float* e[kMaxWorkers];
    float* y[kMaxWorkers];  // GMC+ detached points (written when StepArgs::detach)
};

// Per (worker, segment) pair state, kept in device memory across kernels.
struct PairState {
    uint32_t tau;       // candidate threshold key of the next fused pass
    uint32_t unused0;
    int32_t mode;       // 0 = resolve from candidates, 1 = full data, 3 = full data collected
                        // by the second pass (kModeCollected)
    uint32_t prefix;    // radix digits fixed so far
    int32_t need;       // components still to take below the prefix
    uint32_t T;         // threshold key: k-th largest magnitude key
    int32_t r;          // components with key == T to take (lowest index)
    uint32_t done;      // finished workgroups of the current kernel
    uint32_t cand_used; // candidates of this step (cand is reset for the next)
    uint32_t tau_used;  // the candidate threshold this step's fused pass used
    uint32_t unused1, unused2;
    // exact top-s: the first pass puts the next step's threshold at the floor
    // of the 11-bit bin tau_bin holding the key of rank margin*k/4; with
    // tau_fine the second pass narrows it to the floor of the 22-bit bin
    // holding that key, the tau_need-th of bin tau_bin from the top
    uint32_t tau_bin;
    uint32_t tau_need;
    uint32_t tau_fine;
    uint32_t pad;
};

// Static geometry of the top-s selection (built on the host at init).
struct TopkGeometry {
    int32_t K, n_seg, n_chunks, n_cgroups, n_slices;
    // sampled-threshold top-s (one segment): each worker's sample holds one
    // component per stratum of `stratum`; the threshold is its samp_r-th
    // largest key
    int32_t approx, stratum, samp_n, samp_r;
    const int32_t* seg_start;     // [n_seg+1] segment offsets
    const int32_t* seg_out;       // [n_seg] offset of the segment in a message row
    const int32_t* chunk_start;   // [n_chunks]
    const int32_t* chunk_len;     // [n_chunks]
    const int32_t* chunk_seg;     // [n_chunks]
    const int32_t* chunk_cgrp;    // [n_chunks] compaction group of the chunk
    const int32_t* cgrp_lo;       // [n_cgroups] first chunk of the group
    const int32_t* cgrp_hi;       // [n_cgroups] one past its last chunk
    const int32_t* cgrp_seg;      // [n_cgroups] its segment
    const int32_t* cgrp_rank;     // [n_cgroups] its index within the segment
    const int32_t* seg_cgrp_lo;   // [n_seg] first group of the segment
    const int32_t* seg_cgrps;     // [n_seg] groups of the segment
    const int32_t* slice_seg;     // [n_slices] segment of the slice
    const int32_t* slice_rank;    // [n_slices] index of the slice within its segment
    const int32_t* seg_slices;    // [n_seg] slices of the segment
    const int32_t* seg_slice_lo;  // [n_seg] first slice of the segment
    const int32_t* pair_k;        // [K*n_seg]
    const int32_t* pair_cap;      // [K*n_seg]
    const int64_t* pair_cand;     // [K*n_seg] start of the pair's candidate list
    // copy tiles (kTile candidates of one compaction group; a group's tiles
    // follow the groups before it).  Launch: tiles_per_worker workgroups per
    // worker, tile-major (workgroup b is worker b % K's entry tt = b / K);
    // it takes segment tile_map[tt].x's tiles tile_map[tt].y,
    // + seg_tile_stride[seg], ... (the launch is sized for the usual
    // candidate count, the stride covers longer lists)
    int32_t tiles_per_worker;
    const int2* tile_map;             // [tiles_per_worker]
    const int32_t* seg_tile_stride;   // [n_seg] workgroups launched per (worker, segment)
    // first-step sample: workgroup g of a worker takes segment seed_map[g].x's
    // runs seed_map[g].y, +1, ... (kSeedRunsPerGroup of them, fewer at the
    // segment's end); seg_seed_groups[seg] workgroups per (worker, segment),
    // seg_seed_runs[seg] runs, seg_seed_rank[seg] the rank in the sample (0:
    // the segment is not sampled)
    int32_t n_seed_groups;
    const int2* seed_map;             // [n_seed_groups]
    const int32_t* seg_seed_groups;   // [n_seg]
    const int32_t* seg_seed_runs;     // [n_seg]
    const int32_t* seg_seed_rank;     // [n_seg]
};

struct TopkScratch {
    PairState* pair;              // [K*n_seg]
    uint32_t* hist;               // [K*n_seg][kBins]
    uint32_t* hist2;              // [K*n_seg][kBins] second-digit histogram of the threshold's bin
    uint32_t* run_cnt;            // [K*n_chunks] candidates of (worker, chunk)
    // [2][kGrpSub][K*n_cgroups] candidates of (worker, compaction group),
    // added up by the fused pass of the steps of each parity of t, chunk c
    // into sub-total c % kGrpSub (grp_slot); the emit of the step clears its
    // half for the step after next
    uint32_t* grp_acc;
    int2* slot;                   // [K*n_chunks][kChunk] candidates of (worker, chunk) in index
                                  // order: (index, bit pattern of u)
    int32_t* cand_idx;            // [sum cap] candidate lists, ascending index
    float* cand_val;              // [sum cap]
    uint32_t* sl_above;           // [K*n_slices] kept-above-threshold count of each slice
    uint32_t* sl_ties;            // [K*n_slices] at-threshold count
    uint32_t* sl_out;             // [K*n_slices] message offset of the slice's first kept component
    uint32_t* sl_tiebase;         // [K*n_slices] at-threshold components in earlier slices
    uint32_t* sl_hist;            // [K*n_slices][kSlHist] third-pass counts per slice (exact top-s)
    uint32_t* sl_run;             // [K*n_slices][kWavesPerGroup] components each quarter of a
                                  // collected slice gathered (kModeCollected)
    float* samp;                  // [K][samp_n] the sample's values (sampled-threshold top-s)
    int32_t* rowptr;              // [K][n_ranges+1] server-pass row pointers, also written by the emit
    int32_t n_ranges;             // ranges of kAggTopkRange components
    int64_t* stats;               // [8]
};

struct StepArgs {
    const float* w_t;
    const float* w_prev;
    WorkerPtrs wp;
    float c;         // coefficient of w_t - w_{t-1} in u (beta/eta; lr-in-residual: beta)
    float h;         // coefficient of g in u (1; lr-in-residual: eta)
    float q;         // lambda*eta of GMC+'s detach
    int32_t rule;    // kRule*
    int32_t detach;  // 1: also write y_k = w_t - q u_k (completed by the server pass)
    int32_t d;
    uint64_t seed;   // sample draws of the sampled-threshold top-s
    uint64_t t;      // step
    // nullable: the previous server pass's bitmap (FinishArgs::wbits) when
    // w_t and w_prev are that pass's output and input; the vector passes then
    // read w_t, w_prev only at the marked components, since elsewhere
    // w_t - w_prev is exactly +0
    const uint32_t* wbits;
    // workgroup order of the vector worker passes: runs of `run` chunks of
    // one worker (2: w read everywhere; 1: w read at sparse changes), or 0:
    // each chunk's K workers on one XCD (w read at dense changes)
    int32_t run;
    // 1: the emit leaves the residual's zeros at the kept components to the
    // server pass that follows in the same call (FinishArgs::zero_e)
    int32_t defer_zero;
    // nullable (with wbits, top-s): the previous server pass's list of the
    // components it changed and by how much (FinishArgs::dlist); the vector
    // worker pass then takes w_t - w_prev from it and reads neither buffer.
    // With w_prev NULL (the last server pass updated w_t in place, and its
    // list holds every change) every worker path takes it from the list.
    const int2* dlist;
    int32_t dl_stride;  // int2 per range of dlist
};

// The server pass after the sum over workers: update = -(s * sum), the
// apply rule, and the completion of GMC+'s detached points at the components
// some worker sent (where w_{t+1} differs from w_t).
struct FinishArgs {
    const float* w_in;    // w_t; NULL: no apply
    const float* w_prev;  // w_{t-1} for momentum on the server, else NULL
    float* w_out;         // w_{t+1}; NULL: no apply
    float* update;        // nullable
    float s;              // server scale (eta/K; lr-in-residual: 1/K)
    float b;              // server momentum coefficient (beta) when w_prev is set
    float q;              // lambda*eta
    int32_t detach;       // 1: y_k = w_{t+1} - q e_k at the sent components
    int32_t rows16;       // 1: every e[k] and y[k] is 16-byte aligned
    // nullable, [ceil(d/32)]: bit j set where some worker sent j or w_{t+1}[j]
    // is not finite; everywhere else w_{t+1}[j] equals w_t[j] bit for bit
    uint32_t* wbits;
    // 1 (with wbits): wbits holds, on entry, the previous pass's marks, and
    // w_out holds that pass's input w_{t-1}, which equals w_in = w_t off
    // those marks: w_out is written only in the 32-component words where
    // the old marks or this pass's sent components fall
    int32_t sparse_apply;
    // nullable (with wbits): the list of the components this pass changes
    // and fl(w_{t+1} - w_t) there, dl_stride int2 per range
    int2* dlist;
    int32_t dl_stride;
    // 1 (with sparse_apply, w_out == w_in): the previous pass also updated
    // this buffer in place, so it already holds w_t everywhere and only the
    // words of this pass's sent components are written; the previous marks
    // are visited as well once some pass has written a non-finite w (nf)
    int32_t inplace;
    // nf[0] == nf_epoch: some pass since the recorded components were last
    // dropped wrote a non-finite w_{t+1} (the passes with wbits store the
    // epoch there when they do; the host bumps it to drop the record)
    int32_t* nf;
    int32_t nf_epoch;
    const float* e[kMaxWorkers];  // e_{t+1,k}
    float* y[kMaxWorkers];        // w_{t+1,k}
    // 1: e_{t+1,k}[j] = v - v (+0 for a finite v) for each entry (j, v) of
    // worker k's message, the residual u - C(u) at the kept components, which
    // the step before this pass left to it (StepArgs::defer_zero)
    int32_t zero_e;
    float* ez[kMaxWorkers];
};

// Dense detached points: y_k = w - q e_k for every component and worker.
struct DetachArgs {
    const float* w;
    float q;
    int32_t d;
    const float* e[kMaxWorkers];
    float* y[kMaxWorkers];
};

// ----------------------------------------------------------------------------
// launchers (gmc_kernels.hip); each returns the launch status
// ----------------------------------------------------------------------------
// vec_mask: bit k set when worker k's rows (and w_t, w_prev) are 16-byte
// aligned.  The vector kernel takes every chunk of those workers, the
// element-wise kernel every chunk of the others.
// the first step's speculative thresholds from a sample of u (before the
// fused pass; pairs whose segment is not sampled keep no threshold)
hipError_t launch_topk_seed(const StepArgs& a, const TopkGeometry& g, const TopkScratch& s, hipStream_t st);
hipError_t launch_topk_fused_vec(const StepArgs& a, const TopkGeometry& g, const TopkScratch& s,
                                 uint64_t vec_mask, hipStream_t st);
hipError_t launch_topk_fused_gen(const StepArgs& a, const TopkGeometry& g, const TopkScratch& s,
                                 uint64_t vec_mask, hipStream_t st);
// count, then copy and the first histogram pass (the copy itself takes it
// for the pairs of exact top-s that resolve from their candidates)
hipError_t launch_topk_compact(const StepArgs& a, const TopkGeometry& g, const TopkScratch& s, int force_full,
                               int margin, hipStream_t st);
// passes 2 and 3 (pass 1 runs in launch_topk_compact's second kernel); pass 3
// of exact top-s also lays out the message (per-slice offsets and msg_len),
// the sampled-threshold top-s takes launch_topk_count for that
hipError_t launch_topk_hist(int pass, const StepArgs& a, const TopkGeometry& g, const TopkScratch& s,
                            int force_full, int margin, int64_t* msg_len, int64_t msg_total, hipStream_t st);
hipError_t launch_topk_count(const StepArgs& a, const TopkGeometry& g, const TopkScratch& s,
                             int64_t* msg_len, int64_t msg_total, hipStream_t st);
hipError_t launch_topk_emit(const StepArgs& a, const TopkGeometry& g, const TopkScratch& s,
                            int32_t* idx, float* val, int64_t row_len, hipStream_t st);

// also keeps the previous step's blocks (prev, [n_sel]) and lays out the
// sparse server pass's ranges (visit, [ceil(d/kAggRange)]; meta[0] their
// count, -1: all; meta[1] the non-finite flag the server pass raises; rbits
// a zeroed bitmap of ceil(d/kAggRange) bits for large d)
hipError_t launch_rbgs_sample(uint64_t seed, uint64_t t, int32_t nb, int32_t n_sel, int32_t d,
                              int32_t B, int32_t K, uint32_t* bitmap, int32_t* blocks,
                              int32_t* block_slot, int32_t* idx, int64_t idx_row,
                              int64_t* msg_len, int32_t* prev, int32_t* visit, uint32_t* rbits, int32_t* meta,
                              hipStream_t st);
// vec_mask: workers whose rows (g, e, detached points) are 16-byte aligned,
// with w_t, w_prev and the message rows aligned and B a multiple of 4 (else 0)
hipError_t launch_rbgs_fused(const StepArgs& a, int32_t K, int32_t B, const int32_t* block_slot,
                             float* val, int64_t val_row, uint64_t vec_mask, hipStream_t st);

hipError_t launch_agg_rowptr(int32_t K, int32_t d, const int32_t* idx, int64_t idx_row,
                             const int64_t* msg_len, int32_t* rowptr, int32_t n_ranges,
                             hipStream_t st);
// update (nullable) = -(s * sum); with w_out: w_out = w_in + update (plus
// b (w_in - w_prev) with w_prev) as well; see FinishArgs
hipError_t launch_agg_topk(int32_t K, int32_t d, const int32_t* idx, int64_t idx_row,
                           const float* val, int64_t val_row, const int32_t* rowptr,
                           int32_t n_ranges, const FinishArgs& f, hipStream_t st);
// block_slot: the last step's table from launch_rbgs_sample; visit, meta:
// its range list for a sparse apply (meta[1]: the non-finite flag it raises)
hipError_t launch_agg_rbgs(int32_t K, int32_t d, int32_t B, int32_t n_sel, const int32_t* block_slot,
                           const float* val, int64_t val_row, const FinishArgs& f, const int32_t* visit,
                           int32_t* meta, hipStream_t st);
hipError_t launch_detach(const DetachArgs& a, int32_t K, hipStream_t st);

hipError_t launch_apply(int32_t d, float* w, float* w_prev_out, const float* update,
                        hipStream_t st);

// plain copy of n floats (memory-counter calibration)
hipError_t launch_calib_copy(float* dst, const float* src, int64_t n, hipStream_t st);
// e[k][j] += g[k][j] in the fused worker pass's launch shape (stream ceiling)
hipError_t launch_calib_stream(float* e, const float* g, int64_t pitch, int32_t K, int32_t d, hipStream_t st);

}  // namespace gmc
