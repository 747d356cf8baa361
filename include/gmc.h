/*
 * gmc.h -- C ABI of the MI355X (gfx950) library for the data-parallel hot
 * path of Global Momentum Compression (GMC, Algorithm 1), of GMC+ (Algorithm
 * 2: RBGS and the detached points), and of the two other ways of combining
 * momentum with error feedback that the paper's appendix compares GMC with.
 *
 * One call sequence is one iteration t of Algorithm 1 for K workers that
 * live on one GPU as K device-resident vectors:
 *
 *   gmc_step       each worker k forms u_k = e_{t,k} + g_{t,k}
 *                  - (beta/eta)(w_t - w_{t-1}), compresses it (top-s or RBGS)
 *                  into a sparse message C(u_k), and keeps the residual
 *                  e_{t+1,k} = u_k - C(u_k)                 (Algorithm 1, workers)
 *   gmc_aggregate  the server's update w_{t+1} - w_t = -(eta/K) sum_k C(u_k),
 *                  materialised as a dense vector          (Algorithm 1, server)
 *   gmc_apply      w_{t+1} = w_t + (w_{t+1} - w_t)          (Algorithm 1, workers)
 *
 * gmc_aggregate_apply and gmc_finish fuse the last two; gmc_step_detach,
 * gmc_finish and gmc_detach also produce GMC+'s detached points
 * w_{t+1,k} = w_{t+1} - lambda eta e_{t+1,k} (Algorithm 2).
 *
 * Conventions shared by every entry point:
 *   - Arguments named *_dev are device pointers to memory the caller owns
 *     (e.g. PyTorch tensors).  The context owns only its scratch memory.
 *   - All device work is enqueued on the context's stream (gmc_set_stream;
 *     default: the null stream) and is asynchronous: outputs are valid once
 *     that stream has been synchronised.  Host arrays passed in are read
 *     before the call returns.
 *   - Arithmetic is IEEE binary32 with one rounding per operation and no
 *     fused multiply-add contraction; denormals are kept.  c = fl32(beta/eta)
 *     and s = fl32(eta/K) are formed in binary64 and rounded once.
 *     u = fl(fl(e + g) - fl(c * fl(w_t - w_prev))).  The server sums the K
 *     messages in worker order 0..K-1 starting from +0.0f and writes
 *     update = -(s * sum); components no worker sent get -(s * +0) = -0.0f,
 *     so w + update equals w - s * sum bit for bit everywhere.
 *   - Counts: a fraction ratio of n items keeps count(n, ratio) =
 *     min(n, max(1, ceil(n p / q))) of them, in exact integer arithmetic,
 *     with the ratio read as the fraction p/q of smallest denominator
 *     q <= 2^20 whose binary64 quotient equals it (0.07 is 7/100, so 7% of
 *     100 is 7 although 0.07 * 100 is 7.000000000000001 in binary64); a ratio
 *     that no such fraction gives is taken at its exact binary value.
 *     gmc_count evaluates the rule on the host.
 *   - top-s keeps, per segment of n components, k = count(n, ratio)
 *     components (the s of top-s, Section 1), ranked by the
 *     magnitude bits bits(u) & 0x7FFFFFFF (NaN above Inf, -0 equal to +0),
 *     ties broken towards the lower index.  A kept component leaves
 *     u - u behind in the residual (+0.0f for finite u).
 *   - RBGS keeps whole blocks: block b covers [b*B, min((b+1)*B, d)); n_sel =
 *     count(nb, ratio) of the nb = ceil(d/B) blocks are
 *     drawn by Floyd's sampling algorithm from a SplitMix64 stream whose state
 *     starts at seed XOR mix64(t + 1); every worker uses the same blocks
 *     (Section 4: same random seed on all workers), so only values travel.
 *   - Indices are int32: d must be below 2^31.
 *   - Every call returns a gmc_status; on failure gmc_last_error() describes
 *     the cause.  Invalid arguments never reach the device.
 *   - Call order: the server-side calls (gmc_aggregate, gmc_aggregate_apply,
 *     gmc_finish, gmc_apply) return GMC_ESTATE until the context's first
 *     gmc_step (or gmc_step_detach, gmc_iteration) has been enqueued: before
 *     it the context holds no selection (RBGS: no block table) to aggregate.
 *   - A context is not thread safe; calls on one context must not overlap.
 */
#ifndef GMC_H
#define GMC_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef struct gmc_ctx gmc_ctx;

typedef enum {
    GMC_TOPK_GLOBAL = 0,    /* top-s over the whole vector (one segment)          */
    GMC_TOPK_SEGMENTED = 1, /* top-s per segment (per tensor), see gmc_set_segments */
    GMC_RBGS = 2,           /* random blocks shared by all workers                */
    GMC_TOPK_APPROX = 3     /* the experiments' sampled-threshold top-s, whole vector
                               (Section 5.1): see below                            */
} gmc_compressor;

/*
 * GMC_TOPK_APPROX: worker k's sample S at step t holds one component per
 * stratum of L consecutive components (L = 100 by default, the paper's
 * |S| = d/100; GMC_OPT_SAMPLE_STRATUM): stratum i = [iL, min((i+1)L, d))
 * contributes the component at offset ((x >> 32) * len_i) >> 32, x the
 * i-th output (i = 0, 1, ...) of a SplitMix64 stream started at
 * seed XOR mix64(t + 1) XOR mix64((k + 1) << 32).  theta is the key ranked
 * r = count(|S|, ratio) from the top among the sample's
 * magnitude keys (ratio = 1/1024 in the paper), and the message keeps every
 * component whose key is >= theta, in ascending order: about ratio * d of
 * them, a number that varies (msg_len).  Message capacity: d per worker.
 */

typedef enum {
    GMC_OK = 0,
    GMC_EINVAL = -1,  /* an argument is out of range, NULL or misaligned      */
    GMC_ENOMEM = -2,  /* device or host allocation failed                      */
    GMC_EDEVICE = -3, /* a HIP runtime call failed                             */
    GMC_ESTATE = -4   /* call out of order (e.g. configuration after a step)   */
} gmc_status;

#define GMC_MAX_WORKERS 64

/*
 * Create a context for d parameters and K workers (Algorithm 1, "Input":
 * compressor, K, w_0 is the caller's, eta, beta).
 *   d      1 <= d < 2^31
 *   K      1 <= K <= GMC_MAX_WORKERS
 *   compressor  a gmc_compressor value
 *   ratio  (0, 1]: fraction kept per segment (top-s) or of blocks (RBGS)
 *   beta   momentum coefficient, [0, 1)
 *   eta    learning rate, > 0 and finite
 *   seed   RBGS seed (ignored by top-s)
 * The step counter t starts at 0 (w_{-1} = w_0 and e_{0,k} = 0 are the
 * caller's initial buffers).  Allocates the context's scratch on the current
 * HIP device.  *out is set to NULL on failure.
 */
gmc_status gmc_init(gmc_ctx** out, int64_t d, int32_t K, int32_t compressor, double ratio,
                    double beta, double eta, uint64_t seed);

/*
 * GMC_TOPK_SEGMENTED only: set the segments (tensors) top-s works on: the
 * top-s compressor of Section 1 is applied to each segment on its own, with
 * k = count(segment length, ratio) (per-tensor top-s).
 * seg_off is a host array of n_seg+1 strictly increasing offsets, seg_off[0]
 * = 0, seg_off[n_seg] = d.  Before the first step only (GMC_ESTATE after).
 * Default: one segment [0, d).
 */
gmc_status gmc_set_segments(gmc_ctx* ctx, int32_t n_seg, const int64_t* seg_off);

/* GMC_RBGS only: block length B of the random blockwise compressor (RBGS,
 * Sections 4 and 5.2: whole blocks of consecutive components, drawn with a
 * seed the workers share).  1 <= B <= d; a multiple of 4 takes the vector
 * path, any B is accepted.  Before the first step only (GMC_ESTATE after).
 * Default 4096. */
gmc_status gmc_set_block(gmc_ctx* ctx, int32_t block);

/* Stream all later calls enqueue on (a hipStream_t; NULL = null stream).
 * When the stream changes after work has been enqueued, the new stream is
 * made to wait for everything enqueued so far on the old one (an event), so
 * consecutive calls on one context stay ordered across the change. */
gmc_status gmc_set_stream(gmc_ctx* ctx, void* hip_stream);

/* Per-worker message capacity the caller must provide, in elements:
 * top-s: k_tot = sum over segments of k; RBGS: n_sel * B; sampled-threshold
 * top-s: d. */
int64_t gmc_message_len(const gmc_ctx* ctx);

/* Per-worker index capacity: top-s: k_tot (element indices);
 * RBGS: n_sel (block ids); sampled-threshold top-s: d. */
int64_t gmc_index_len(const gmc_ctx* ctx);

/* The count rule on the host, no device work and no context: how many of
 * n items a fraction ratio keeps (the top-s count of a segment of n,
 * Section 1; RBGS blocks out of nb; the sampled threshold's rank in a sample
 * of n).  1 <= n < 2^31, 0 < ratio <= 1; returns -1 for other arguments. */
int64_t gmc_count(int64_t n, double ratio);

/*
 * One worker-side pass of Algorithm 1 for all K workers at step t, then
 * t <- t + 1.
 *   w_t_dev, w_prev_dev   [d] fp32: w_t and w_{t-1}; read only.  w_prev_dev
 *                         may be NULL right after a top-s server pass that
 *                         updated w_t_dev in place and kept its changes
 *                         (GMC_OPT_SPARSE_MOMENTUM with GMC_OPT_CHANGE_LIST
 *                         3): w_t - w_{t-1} is then that pass's exact
 *                         fl(w_{t+1} - w_t), bit for bit what the two
 *                         vectors give; GMC_ESTATE otherwise (no such pass,
 *                         or its record was dropped), and not with
 *                         gmc_step_detach
 *   grads_dev             host array of K device pointers, each [d] fp32:
 *                         g_{t,k}; read only
 *   err_dev               host array of K device pointers, each [d] fp32:
 *                         e_{t,k} in, e_{t+1,k} = u - C(u) out (in place)
 *   idx_dev               [K][gmc_index_len] int32 out: top-s: ascending
 *                         element indices, segment after segment; RBGS:
 *                         ascending block ids, the same row for every worker
 *   val_dev               [K][gmc_message_len] fp32 out: u_k at the kept
 *                         components, in idx order (RBGS: block after block)
 *   msg_len_dev           [K] int64 out: values written per worker (k_tot,
 *                         RBGS: n_sel blocks' worth, sampled-threshold
 *                         top-s: the number kept)
 * Device buffers must not overlap each other, except that w_t_dev and
 * w_prev_dev may be one buffer (w_{-1} = w_0 at t = 0).  Pointers that are not
 * 16-byte aligned are accepted (slower path).  w is never written.
 */
gmc_status gmc_step(gmc_ctx* ctx, const float* w_t_dev, const float* w_prev_dev,
                    const float* const* grads_dev, float* const* err_dev,
                    int32_t* idx_dev, float* val_dev, int64_t* msg_len_dev);

/*
 * The server's update (Algorithm 1, server): update_dev[j] =
 * -(s * sum_k val_k(j)) over the workers whose message holds j, in worker
 * order; -0.0f where no worker sent j.  idx/val/msg_len are K messages in the
 * layout gmc_step writes (top-s rows must be strictly ascending and in
 * [0, d); RBGS rows are the block ids of the last gmc_step).
 *   update_dev  [d] fp32 out, dense
 */
gmc_status gmc_aggregate(gmc_ctx* ctx, const int32_t* idx_dev, const float* val_dev,
                         const int64_t* msg_len_dev, float* update_dev);

/*
 * The server's update and the workers' apply in one pass (Algorithm 1,
 * server and workers): with update = -(s * sum_k C(u_k)) exactly as
 * gmc_aggregate computes it,
 *   w_out_dev[j] = w_dev[j] + update[j]   for every j in [0, d),
 * and update_dev[j] = update[j] when update_dev is not NULL.  w_out_dev may
 * equal w_dev (in place: for top-s under GMC_OPT_SPARSE_MOMENTUM with
 * GMC_OPT_CHANGE_LIST 3 the pass keeps its changes, and the next gmc_step
 * passes w_prev = NULL); otherwise the two must not overlap.  Out of place
 * the caller keeps w_{t+1} in w_out_dev and w_t in w_dev, i.e. swaps the
 * roles of its two parameter buffers for the next gmc_step instead of
 * copying w into w_prev.  update_dev may not alias either.  Not with
 * GMC_RULE_SERVER_MOMENTUM (GMC_EINVAL; use gmc_finish).
 */
gmc_status gmc_aggregate_apply(gmc_ctx* ctx, const int32_t* idx_dev, const float* val_dev,
                               const int64_t* msg_len_dev, const float* w_dev, float* w_out_dev,
                               float* update_dev);

/*
 * Workers' apply (Algorithm 1): w_prev_out_dev[j] = w_dev[j] (when not NULL),
 * then w_dev[j] = w_dev[j] + update_dev[j], for every j in [0, d).  Not with
 * GMC_RULE_SERVER_MOMENTUM (GMC_EINVAL; gmc_finish applies that rule).
 *   w_dev           [d] fp32 in/out
 *   w_prev_out_dev  [d] fp32 out or NULL; may not alias w_dev
 *   update_dev      [d] fp32 in
 */
gmc_status gmc_apply(gmc_ctx* ctx, float* w_dev, float* w_prev_out_dev, const float* update_dev);

/*
 * Update rules (before the first step only; default GMC_RULE_GMC):
 *   GMC_RULE_GMC              Algorithm 1: u = (e + g) - c (w_t - w_{t-1}) with
 *                             c = fl32(beta/eta); update = -(fl32(eta/K) * sum)
 *   GMC_RULE_SERVER_MOMENTUM  appendix, momentum on the server: u = e + g;
 *                             update = -(fl32(eta/K) * sum) and
 *                             w_{t+1} = (w_t + update) + fl32(beta) (w_t - w_{t-1}),
 *                             so the apply needs w_{t-1} (gmc_finish only)
 *   GMC_RULE_LR_IN_RESIDUAL   appendix, learning rate inside the residual:
 *                             u = (e + fl32(eta) g) - fl32(beta) (w_t - w_{t-1});
 *                             update = -(fl32(1/K) * sum)
 * Each operation is one binary32 rounding, left to right as written.
 */
enum { GMC_RULE_GMC = 0, GMC_RULE_SERVER_MOMENTUM = 1, GMC_RULE_LR_IN_RESIDUAL = 2 };
gmc_status gmc_set_rule(gmc_ctx* ctx, int32_t rule);

/* Learning rate of the following iterations (eta > 0, finite), e.g. the
 * cosine schedule of Section 5.1; the rule's constants are re-derived from
 * it (in binary64, rounded once).  Any time between iterations. */
gmc_status gmc_set_eta(gmc_ctx* ctx, double eta);

/* GMC+'s detach coefficient lambda in [0, 1] (Algorithm 2; default 0, which
 * makes the detached points equal to w_{t+1}).  q = fl32(lambda * eta) at the
 * current eta.  Any time between iterations. */
gmc_status gmc_set_lambda(gmc_ctx* ctx, double lambda);

/*
 * gmc_step for GMC+ (Algorithm 2): the same worker pass, and in the same
 * streaming pass w_k_dev[k][j] = w_t[j] - q u_k[j], which is already the
 * detached point w_{t+1,k}[j] = w_{t+1}[j] - q e_{t+1,k}[j] at every component
 * that no worker sends (there e_{t+1,k} = u_k and w_{t+1} = w_t, bit for bit).
 * gmc_finish with the same w_k_dev completes the others.
 *   w_k_dev  host array of K device pointers, each [d] fp32 out
 * Not with GMC_RULE_SERVER_MOMENTUM (w_{t+1} differs from w_t everywhere):
 * GMC_EINVAL; use gmc_detach there.
 */
gmc_status gmc_step_detach(gmc_ctx* ctx, const float* w_t_dev, const float* w_prev_dev,
                           const float* const* grads_dev, float* const* err_dev, float* const* w_k_dev,
                           int32_t* idx_dev, float* val_dev, int64_t* msg_len_dev);

/*
 * The server pass of an iteration under the context's rule (the sum as in
 * gmc_aggregate, then the apply), and optionally the completion of GMC+'s
 * detached points:
 *   w_dev       [d] fp32 in: w_t
 *   w_prev_dev  [d] fp32 in: w_{t-1}; required by GMC_RULE_SERVER_MOMENTUM,
 *               ignored (may be NULL) otherwise; may equal w_out_dev (the
 *               caller's buffer swap), not w_dev
 *   w_out_dev   [d] fp32 out: w_{t+1}; may equal w_dev (in place)
 *   update_dev  [d] fp32 out or NULL: -(s * sum), the sparse part
 *   err_dev, w_k_dev  NULL, or host arrays of K device pointers: e_{t+1,k}
 *               (as gmc_step_detach left them) and the detached points that
 *               gmc_step_detach started; every component some worker sent
 *               gets w_k[j] = w_{t+1}[j] - q e_{t+1,k}[j] (Algorithm 2)
 */
gmc_status gmc_finish(gmc_ctx* ctx, const int32_t* idx_dev, const float* val_dev, const int64_t* msg_len_dev,
                      const float* w_dev, const float* w_prev_dev, float* w_out_dev, float* update_dev,
                      const float* const* err_dev, float* const* w_k_dev);

/*
 * One whole iteration of Algorithm 1 for all K workers: gmc_step(w_t,
 * w_prev_io, ...) and then the server pass, which writes w_{t+1} over
 * w_prev_io (the caller swaps the roles of its two buffers for the next
 * iteration, as after gmc_finish out of place).  Results equal those of
 * gmc_step followed by gmc_finish(w_t, w_prev_io, w_out = w_prev_io) bit for
 * bit; the call pattern GMC_OPT_SPARSE_MOMENTUM serves.
 *   w_t_dev        [d] fp32 in
 *   w_prev_io_dev  [d] fp32: w_{t-1} in, w_{t+1} out; may not alias w_t_dev
 * The remaining arguments are gmc_step's.
 */
gmc_status gmc_iteration(gmc_ctx* ctx, const float* w_t_dev, float* w_prev_io_dev, const float* const* grads_dev,
                         float* const* err_dev, int32_t* idx_dev, float* val_dev, int64_t* msg_len_dev);

/*
 * One whole iteration of Algorithm 1 with the parameters updated in place
 * (one buffer instead of two): gmc_step(w, w_prev, ...) and then the server
 * pass w <- w + update.  The workers' momentum term needs w_t - w_{t-1},
 * which the in-place pass keeps as its change list (every component it
 * changed, with fl(w_{t+1} - w_t)), so the next iteration passes
 * w_prev_dev = NULL.  Top-s (global, segmented or sampled threshold) under
 * GMC_RULE_GMC or GMC_RULE_LR_IN_RESIDUAL, with GMC_OPT_SPARSE_MOMENTUM and
 * GMC_OPT_CHANGE_LIST 3 (GMC_EINVAL otherwise).  Results equal gmc_iteration's
 * bit for bit.  The server pass then writes w only in the 32-component words
 * of the components sent now, where an out-of-place pass also rewrites those
 * the previous pass changed.
 *   w_dev       [d] fp32: w_t in, w_{t+1} out
 *   w_prev_dev  [d] fp32 w_{t-1}, read only; NULL after an in-place
 *               iteration whose record stands (GMC_ESTATE if it was dropped:
 *               gmc_set_step, the options that drop the recorded
 *               components, gmc_apply).  At t = 0 pass w_dev (w_{-1} = w_0).
 * A caller that saves a run to resume it exactly needs w_{t-1} as well: it
 * runs the last iteration before the save as gmc_step(w, NULL, ...) and
 * gmc_aggregate_apply(w, w_next) into a second buffer, saves w (now w_{t-1})
 * and w_next (w_t), and a resumed context (gmc_set_step) starts with
 * gmc_iteration_inplace(w_next, w, ...), then NULL.
 * The remaining arguments are gmc_step's.
 */
gmc_status gmc_iteration_inplace(gmc_ctx* ctx, float* w_dev, const float* w_prev_dev, const float* const* grads_dev,
                                 float* const* err_dev, int32_t* idx_dev, float* val_dev, int64_t* msg_len_dev);

/*
 * GMC+'s detached points as one dense pass (Algorithm 2, detach):
 * w_k_dev[k][j] = w_dev[j] - q err_dev[k][j] for every worker and component,
 * with w_dev = w_{t+1} and err = e_{t+1,k}; any rule.
 */
gmc_status gmc_detach(gmc_ctx* ctx, const float* w_dev, const float* const* err_dev, float* const* w_k_dev);

/* Step counter t (RBGS draws depend on (seed, t)); for checkpoint/resume. */
gmc_status gmc_get_step(const gmc_ctx* ctx, int64_t* t);
gmc_status gmc_set_step(gmc_ctx* ctx, int64_t t);

/*
 * Tuning and test options (value semantics per option):
 *   GMC_OPT_FORCE_FULL_SELECT  1: every top-s selection takes the full-data
 *                              path (no speculative candidates)
 *   GMC_OPT_CAND_MARGIN        rank of the next step's speculative threshold,
 *                              in quarters of k (4..4096; default 4: the
 *                              threshold sits at the floor of the 22-bit key
 *                              bin holding this step's key of rank k, and
 *                              the residual's growth brings about 1.3-2 k
 *                              candidates the next step)
 *   GMC_OPT_CAND_CAP_MULT      candidate capacity as a multiple of k (>= 1);
 *                              reallocates scratch; before the first step
 *   GMC_OPT_PROFILE            bit mask of the stages to time with HIP events
 *                              on the context's stream (0: off); see
 *                              gmc_profile_read for the stage numbers.  The
 *                              events are recorded without a system-scope
 *                              fence: they time, they do not order host reads
 *   GMC_OPT_SAMPLE_STRATUM     GMC_TOPK_APPROX: components per sample stratum
 *                              L in [1, d] (default 100); before the first step
 *   GMC_OPT_SPARSE_MOMENTUM    1: the caller promises not to change either
 *                              parameter buffer between a server pass and the
 *                              next server pass (default 0).  Setting the
 *                              option (to either value) drops the recorded
 *                              components: a caller who wrote w in place or
 *                              swapped in other contents under the same
 *                              pointers sets it again before the next
 *                              gmc_step, which then reads w densely once.
 *                              gmc_set_step and gmc_apply drop them too.  Then a server
 *                              pass out of place (gmc_aggregate_apply,
 *                              gmc_finish, gmc_iteration; not with momentum on
 *                              the server) records which components it
 *                              changed, and when the next gmc_step gets that
 *                              pass's output as w_t and its input as w_prev,
 *                              the worker pass reads w_t and w_prev only there:
 *                              everywhere else w_t - w_prev is exactly +0, as
 *                              in Algorithm 1, where the workers receive the
 *                              server's sparse w_{t+1} - w_t.  The server pass
 *                              that follows, writing over w_prev's buffer,
 *                              writes w_{t+1} only in the 32-component words
 *                              where it differs from w_{t-1} (the recorded
 *                              components and the ones sent now).  Results
 *                              are bit for bit those of the dense path; other
 *                              calls, or other buffers, fall back to it.  A
 *                              server pass in place records its changes only
 *                              with GMC_OPT_CHANGE_LIST 3 (gmc_step with
 *                              w_prev = NULL, gmc_iteration_inplace).
 */
/*
 *   GMC_OPT_CHANGE_LIST        with GMC_OPT_SPARSE_MOMENTUM, top-s: the server
 *                              pass also lists the components it changed and
 *                              fl(w_{t+1} - w_t) there, and the next worker
 *                              pass takes w_t - w_prev from that list instead
 *                              of reading both parameter vectors at the marked
 *                              cache lines.  0 (default): when the two vectors
 *                              (8 d bytes) outgrow the 256 MB Infinity Cache;
 *                              1: always; 2: never; 3: always, with room for
 *                              every component of each 4096-component range
 *                              (8 d bytes of scratch instead of d bytes), so
 *                              that a server pass in place (gmc_aggregate_apply
 *                              or gmc_finish with w_out = w,
 *                              gmc_iteration_inplace) keeps its changes too
 *                              and the next gmc_step may pass w_prev = NULL.
 *                              Results are the same bit for bit.  Setting it
 *                              drops the recorded components, as
 *                              GMC_OPT_SPARSE_MOMENTUM does; setting or
 *                              clearing 3 reallocates scratch and is allowed
 *                              before the first step only (GMC_ESTATE).
 */
enum {
    GMC_OPT_FORCE_FULL_SELECT = 1,
    GMC_OPT_CAND_MARGIN = 2,
    GMC_OPT_CAND_CAP_MULT = 3,
    GMC_OPT_PROFILE = 4,
    GMC_OPT_SAMPLE_STRATUM = 5,
    GMC_OPT_SPARSE_MOMENTUM = 6,
    GMC_OPT_CHANGE_LIST = 7
};
gmc_status gmc_set_option(gmc_ctx* ctx, int32_t option, int64_t value);

/*
 * Diagnostics, synchronising the context's stream first.  Writes up to n of:
 *   [0] steps taken  [1] top-s segment selections resolved from candidates
 *   [2] selections that took the full-data path  [3] candidates collected
 *   [4] selections whose count check failed (must stay 0)
 *   [5] worker passes that read w only at the last server pass's changed
 *       components (GMC_OPT_SPARSE_MOMENTUM)
 *   [6] server passes that wrote w_{t+1} only where their output buffer
 *       did not hold it yet (GMC_OPT_SPARSE_MOMENTUM)
 */
gmc_status gmc_stats(gmc_ctx* ctx, int64_t* out, int32_t n);

/*
 * Per-(worker, segment) selection diagnostics of the last gmc_step (top-s
 * compressors), synchronising the context's stream first.  Pair p = k *
 * n_seg + segment; for p < min(n, K * n_seg): mode[p] = 0 when the pair's
 * top-s was resolved from its speculative candidates, 1 when it took the
 * full-data path (too few or too many candidates), and cand[p] = the
 * candidates the worker pass collected for it.  *n_pairs = K * n_seg.
 * GMC_EINVAL for RBGS, GMC_ESTATE before the first step.
 */
gmc_status gmc_pair_stats(gmc_ctx* ctx, int32_t* mode, int64_t* cand, int32_t n, int32_t* n_pairs);

/*
 * Stage timings of the stages GMC_OPT_PROFILE selects: for each stage i < n,
 * total milliseconds and timed launches since the option was last set.
 * Stages: 0 fused worker pass (vector kernel; RBGS: its fused gather pass),
 * 1 fused worker pass (element-wise kernel), 2 selection (RBGS: block draw),
 * 3 emit, 4 aggregate, 5 apply.  Synchronises the context's stream.
 */
gmc_status gmc_profile_read(gmc_ctx* ctx, double* ms, int64_t* launches, int32_t n);

/*
 * For callers that cannot allocate device memory (code under HIP graph
 * capture, tight serving loops, harnesses that forbid hipMalloc):
 * gmc_aggregate for messages of element indices (the top-s compressors:
 * rows of index_len strictly ascending indices in [0, d), msg_len[k] of them
 * valid, values in rows of message_len) without a context, with the GMC
 * rule's scale s = fl32(eta/K): update_dev[j] = -(s * sum_k val_k(j)) in
 * worker order, -0.0f where no worker sent j, bit for bit what gmc_aggregate
 * of a top-s context with the same d, K and eta writes.  Enqueued on
 * hip_stream (NULL: the null stream); asynchronous.
 *   Allocates nothing: its scratch (the row pointers, 4 K (ceil(d/4096) + 1)
 *   bytes) is a static device array of GMC_STATIC_SCRATCH_BYTES that each GPU
 *   holds from the first call on it until the process ends; larger problems
 *   get GMC_EINVAL.  Every call on a GPU shares that GPU's array (each call
 *   writes every entry it reads), so calls that overlap on one GPU (other
 *   streams, other threads) race: order them.  Argument errors are reported
 *   through gmc_last_error(NULL).
 */
#define GMC_STATIC_SCRATCH_BYTES (8u << 20)
gmc_status gmc_aggregate_static(int64_t d, int32_t K, double eta, const int32_t* idx_dev, int64_t index_len,
                                const float* val_dev, int64_t message_len, const int64_t* msg_len_dev,
                                float* update_dev, void* hip_stream);

/*
 * Measurement support, not part of the method: a plain copy of n floats
 * (dst_dev[i] = src_dev[i]) on hip_stream, the reference kernel of known
 * traffic against which memory counters are scaled.  Buffers must not overlap.
 */
gmc_status gmc_calib_copy(void* hip_stream, float* dst_dev, const float* src_dev, int64_t n);

/*
 * Measurement support, not part of the method: a plain stream with the
 * access pattern of the fused worker pass of gmc_step (two streamed reads
 * and one streamed write per worker-element, one workgroup per (chunk of
 * 2048 components, worker), the K workers of a chunk consecutive):
 * e_dev[k*row_pitch + j] += g_dev[k*row_pitch + j] for k < K, j < d, on
 * hip_stream.  Its rate is the ceiling the memory system gives that pattern.
 *   row_pitch >= d; 1 <= d < 2^31; K >= 1; the two K-row regions must not
 *   overlap.  Rows that are not 16-byte aligned take an element-wise path.
 */
gmc_status gmc_calib_stream(void* hip_stream, float* e_dev, const float* g_dev, int64_t row_pitch, int32_t K,
                            int64_t d);

/* Message for the last non-OK status of this context (or of gmc_init when
 * ctx is NULL); never NULL. */
const char* gmc_last_error(const gmc_ctx* ctx);

/* Free the context and its scratch (synchronises its stream).  NULL is a no-op. */
void gmc_destroy(gmc_ctx* ctx);

#ifdef __cplusplus
}
#endif

#endif /* GMC_H */
