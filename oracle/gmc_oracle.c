/*
 * GMC oracle: a plain, slow, single-threaded CPU statement of what one
 * iteration of Global Momentum Compression computes (Algorithm 1, GMC, of
 * "Global Momentum Compression for Sparse Communication in Distributed
 * Learning", Shi, Zhao, Xie, Gao, Li).
 *
 * TEST INFRASTRUCTURE.  Only the test suite, the smoke check and the bench's
 * CPU-baseline leg may load or call this library.  It shares no code, header,
 * table or helper with the device library; the only thing the two sides have
 * in common is the seeded input generator.
 *
 * Arithmetic: IEEE-754 binary32, one rounding per operation, no contraction
 * into fused multiply-adds (built with -ffp-contract=off, SSE2 scalar float,
 * no fast-math), denormals kept.  The paper states the update in real
 * arithmetic; binary32 is the precision of the device path and the selection
 * of the compressor is an integer decision taken on binary32 values, so both
 * sides must take it on the same bits.
 *
 * Readings of points on which the paper is silent (each one is listed with
 * its reason in the design notes of the repository):
 *   - c = fl32(beta/eta) and s = fl32(eta/K), each formed in double and
 *     rounded once;
 *   - u = fl(fl(e + g) - fl(c * fl(w_t - w_prev))), evaluated left to right as
 *     printed in step "e_{t+1/2,k} = e_{t,k} + grad - (beta/eta)(w_t - w_{t-1})";
 *   - the number kept per segment of n components is
 *     k = min(n, max(1, ceil(n p / q))) in exact integer arithmetic, with the
 *     ratio read as the fraction p/q of smallest denominator (q <= 2^20)
 *     that rounds to it (0.07 is 7/100), else as its exact binary value;
 *   - top-s ranks by the magnitude bits |u| = bits(u) & 0x7FFFFFFF (NaN above
 *     Inf, -0 equal to +0) and breaks ties by the lower index;
 *   - the server sum over workers runs in worker order 0..K-1 from +0.0f and
 *     the scale eta/K is applied once afterwards: delta = -(s * acc);
 *   - RBGS draws its blocks with Floyd's sampling algorithm fed by a SplitMix64
 *     stream whose state is seed XOR mix(t+1); the same blocks on every worker.
 *
 * PARITY UNPINNED: the exact RBGS block ids (orc_rbgs_draw, orc_rbgs_blocks)
 * and the exact positions of the sampled-threshold sample
 * (orc_sample_positions).  The paper prints no draw; these functions follow
 * their stated definitions, and the tests pin the SplitMix64 mix to its
 * published outputs and the samplers to properties (distinct, in range,
 * uniform), not to values the paper fixes.
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

/* ------------------------------------------------------------------------- */
/* Constants and counts                                                       */
/* ------------------------------------------------------------------------- */

/*
 * The ratio read as the fraction the caller means: the smallest denominator
 * q <= 2^20 for which some integer p in [1, q] gives p/q == ratio after
 * rounding to binary64.  0.07 is read as 7/100, 0.001 as 1/1000, 1/1024 as
 * itself.  Returns 0 when no such fraction exists.
 */
static int ratio_as_fraction(double ratio, int64_t* p_out, int64_t* q_out)
{
    for (int64_t q = 1; q <= ((int64_t)1 << 20); ++q) {
        double p = floor(ratio * (double)q + 0.5);
        if (p < 1.0 || p > (double)q) continue;
        if (p / (double)q == ratio) {
            *p_out = (int64_t)p;
            *q_out = q;
            return 1;
        }
    }
    return 0;
}

/*
 * Components kept from a segment of n (top-s keeps s components, Section 1;
 * the experiments set s = d/1024, Section 5.1): ceil(n p / q) in exact
 * integer arithmetic for the ratio read as p/q, clamped to [1, n].  A ratio
 * that no such fraction gives is taken at its exact binary value
 * m 2^-sh (m an integer below 2^53): ceil(n m / 2^sh), also exact.
 */
int64_t orc_count(int64_t n, double ratio)
{
    int64_t p, q, k;
    if (ratio_as_fraction(ratio, &p, &q)) {
        k = (n * p + q - 1) / q;
    } else {
        int e;
        double f = frexp(ratio, &e);                /* ratio = f 2^e, f in [1/2, 1) */
        uint64_t m = (uint64_t)ldexp(f, 53);         /* ratio = m 2^(e - 53) exactly */
        int sh = 53 - e;
        if (sh >= 120) {
            k = 1;                                   /* n m < 2^84: the quotient is in (0, 1) */
        } else {
            unsigned __int128 num = (unsigned __int128)(uint64_t)n * m;
            unsigned __int128 one = 1;
            k = (int64_t)((num + ((one << sh) - 1)) >> sh);
        }
    }
    if (k < 1) k = 1;
    if (k > n) k = n;
    return k;
}

/* beta/eta multiplies the parameter difference in the global momentum term;
 * eta/K scales the server's sum (Algorithm 1, server update). */
void orc_constants(double beta, double eta, int K, float* c, float* s)
{
    *c = (float)(beta / eta);
    *s = (float)(eta / (double)K);
}

/* ------------------------------------------------------------------------- */
/* Worker side: global momentum plus error feedback (Algorithm 1, workers)    */
/* ------------------------------------------------------------------------- */

/*
 * u = e_{t,k} + g_{t,k} - (beta/eta) (w_t - w_{t-1})          (Algorithm 1)
 *
 * -(w_t - w_{t-1})/eta is the paper's global momentum (Section 2.3); beta
 * times it enters every worker's pre-compression vector.
 */
void orc_precompress(int64_t d, float c, const float* w_t, const float* w_prev,
                     const float* g, const float* e, float* u)
{
    for (int64_t j = 0; j < d; ++j) {
        float diff = w_t[j] - w_prev[j];
        float mom = c * diff;
        float acc = e[j] + g[j];
        u[j] = acc - mom;
    }
}

/* Magnitude key: the sign bit cleared. */
static uint32_t key_of(float x)
{
    uint32_t b;
    memcpy(&b, &x, sizeof b);
    return b & 0x7fffffffu;
}

typedef struct {
    uint32_t key;
    int64_t pos;
} keyed;

/* Strict total order: larger magnitude first, then lower position. */
static int cmp_rank(const void* a, const void* b)
{
    const keyed* x = (const keyed*)a;
    const keyed* y = (const keyed*)b;
    if (x->key != y->key) return x->key > y->key ? -1 : 1;
    if (x->pos != y->pos) return x->pos < y->pos ? -1 : 1;
    return 0;
}

static int cmp_i64(const void* a, const void* b)
{
    int64_t x = *(const int64_t*)a, y = *(const int64_t*)b;
    return (x > y) - (x < y);
}

/*
 * top-s: the k positions of u[0..n) with the largest |u|, ties to the lower
 * position, returned in ascending position order.  A full sort under the
 * ranking order, then the first k: slow and plain.  Returns 0, or -1 if the
 * scratch allocation fails.
 */
int orc_topk(int64_t n, const float* u, int64_t k, int64_t* out_pos)
{
    keyed* r = (keyed*)malloc((size_t)(n > 0 ? n : 1) * sizeof(keyed));
    if (!r) return -1;
    for (int64_t j = 0; j < n; ++j) {
        r[j].key = key_of(u[j]);
        r[j].pos = j;
    }
    qsort(r, (size_t)n, sizeof(keyed), cmp_rank);
    for (int64_t i = 0; i < k; ++i) out_pos[i] = r[i].pos;
    free(r);
    qsort(out_pos, (size_t)k, sizeof(int64_t), cmp_i64);
    return 0;
}

/*
 * C(u) for top-s applied to each segment [seg_off[i], seg_off[i+1]) of u, and
 * the residual e_{t+1,k} = u - C(u), written over u in place (a kept
 * component becomes u - u = +0.0f, every other component keeps u).
 * Messages: idx (int32, ascending) and val = u[idx], segment after segment.
 * Returns the message length, or -1 on allocation failure.
 */
int64_t orc_compress_topk(float* u, int64_t n_seg, const int64_t* seg_off, double ratio,
                          int32_t* idx, float* val)
{
    int64_t m = 0;
    for (int64_t s = 0; s < n_seg; ++s) {
        int64_t lo = seg_off[s], n = seg_off[s + 1] - lo;
        int64_t k = orc_count(n, ratio);
        int64_t* pos = (int64_t*)malloc((size_t)k * sizeof(int64_t));
        if (!pos) return -1;
        if (orc_topk(n, u + lo, k, pos) != 0) {
            free(pos);
            return -1;
        }
        for (int64_t i = 0; i < k; ++i) {
            int64_t j = lo + pos[i];
            idx[m] = (int32_t)j;
            val[m] = u[j];
            ++m;
        }
        free(pos);
    }
    for (int64_t i = 0; i < m; ++i) {
        float sent = val[i];
        u[idx[i]] = u[idx[i]] - sent;   /* u - C(u) at a kept component */
    }
    return m;
}

/* ------------------------------------------------------------------------- */
/* RBGS: random blocks with a seed shared by all workers (Sections 4, 5.2)    */
/* ------------------------------------------------------------------------- */

/* SplitMix64 output mixing function (Steele, Lea, Flood, OOPSLA 2014). */
uint64_t orc_splitmix64_mix(uint64_t z)
{
    z = (z ^ (z >> 30)) * 0xbf58476d1ce4e5b9ULL;
    z = (z ^ (z >> 27)) * 0x94d049bb133111ebULL;
    return z ^ (z >> 31);
}

/* Draw i (i = 0, 1, ...) of step t: output i of a SplitMix64 generator whose
 * state starts at seed XOR mix(t + 1) and advances by the golden gamma. */
uint64_t orc_rbgs_draw(uint64_t seed, uint64_t t, uint64_t i)
{
    const uint64_t gamma = 0x9e3779b97f4a7c15ULL;
    uint64_t state = seed ^ orc_splitmix64_mix(t + 1);
    return orc_splitmix64_mix(state + (i + 1) * gamma);
}

static int cmp_i32(const void* a, const void* b)
{
    int32_t x = *(const int32_t*)a, y = *(const int32_t*)b;
    return (x > y) - (x < y);
}

/*
 * n_sel distinct block ids out of nb, sorted ascending: Floyd's sampling
 * algorithm (Bentley and Floyd, "Programming Pearls: A Sample of
 * Brilliance", CACM 1987).  For J = nb-n_sel .. nb-1 draw r uniform on
 * [0, J]; keep r, or J when r was already kept.  The draw maps the top 32
 * random bits onto [0, J] by multiply-shift.
 */
void orc_rbgs_blocks(uint64_t seed, uint64_t t, int32_t nb, int32_t n_sel, int32_t* blocks)
{
    int32_t have = 0;
    for (int64_t J = (int64_t)nb - n_sel; J < nb; ++J) {
        uint64_t x = orc_rbgs_draw(seed, t, (uint64_t)(J - ((int64_t)nb - n_sel)));
        int32_t r = (int32_t)(((x >> 32) * (uint64_t)(J + 1)) >> 32);
        int dup = 0;
        for (int32_t q = 0; q < have; ++q)
            if (blocks[q] == r) dup = 1;
        blocks[have++] = dup ? (int32_t)J : r;
    }
    qsort(blocks, (size_t)n_sel, sizeof(int32_t), cmp_i32);
}

/*
 * C(u) for RBGS: every component of the selected blocks (block b covers
 * [b*B, min((b+1)*B, d))), in ascending block order; the residual u - C(u)
 * is written over u.  Returns the message length.
 */
int64_t orc_compress_rbgs(float* u, int64_t d, int64_t B, const int32_t* blocks, int32_t n_sel,
                          float* val)
{
    int64_t m = 0;
    for (int32_t q = 0; q < n_sel; ++q) {
        int64_t lo = (int64_t)blocks[q] * B, hi = lo + B;
        if (hi > d) hi = d;
        for (int64_t j = lo; j < hi; ++j) {
            float sent = u[j];
            val[m++] = sent;
            u[j] = u[j] - sent;
        }
    }
    return m;
}

/* ------------------------------------------------------------------------- */
/* Server side (Algorithm 1, server) and the workers' apply                   */
/* ------------------------------------------------------------------------- */

/*
 * delta = w_{t+1} - w_t = -(eta/K) sum_k C(u_k):
 * acc = +0.0f; acc += C(u_k) for k = 0..K-1 in order (only the components
 * worker k sent are nonzero in C(u_k)); delta = -(s * acc), dense over d.
 * idx[k], val[k], len[k] are worker k's message.
 */
int orc_aggregate(int64_t d, int K, float s, const int32_t* const* idx,
                  const float* const* val, const int64_t* len, float* delta)
{
    float* acc = (float*)malloc((size_t)(d > 0 ? d : 1) * sizeof(float));
    if (!acc) return -1;
    for (int64_t j = 0; j < d; ++j) acc[j] = 0.0f;
    for (int k = 0; k < K; ++k)
        for (int64_t i = 0; i < len[k]; ++i)
            acc[idx[k][i]] = acc[idx[k][i]] + val[k][i];
    for (int64_t j = 0; j < d; ++j) delta[j] = -(s * acc[j]);
    free(acc);
    return 0;
}

/* w_{t+1} = w_t + (w_{t+1} - w_t)   (Algorithm 1, workers' last step) */
void orc_apply(int64_t d, float* w, const float* delta)
{
    for (int64_t j = 0; j < d; ++j) w[j] = w[j] + delta[j];
}

/* ------------------------------------------------------------------------- */
/* GMC+: the detached point (Algorithm 2)                                     */
/* ------------------------------------------------------------------------- */

/* lambda * eta, the coefficient of the residual in the detach step, formed
 * in double and rounded once. */
float orc_detach_constant(double lambda, double eta)
{
    return (float)(lambda * eta);
}

/*
 * w_{t+1,k} = w_{t+1} - (lambda eta) e_{t+1,k}        (Algorithm 2, detach)
 *
 * GMC+ takes worker k's next stochastic gradient at this point instead of at
 * w_{t+1}; with lambda = 0 the point is w_{t+1} and GMC+ is GMC.  q is
 * orc_detach_constant(lambda, eta).
 */
void orc_detach(int64_t d, float q, const float* w_next, const float* e_next, float* w_k)
{
    for (int64_t j = 0; j < d; ++j) {
        float r = q * e_next[j];
        w_k[j] = w_next[j] - r;
    }
}

/* ------------------------------------------------------------------------- */
/* Other ways of combining momentum and error feedback (appendix)             */
/* ------------------------------------------------------------------------- */

/*
 * Constants of the three update rules, each formed in double and rounded
 * once to binary32:
 *   variant 0, GMC (Algorithm 1):        c = beta/eta (worker), s = eta/K, h = 1;
 *   variant 1, momentum on the server:   c = beta (server), s = eta/K, h = 1;
 *   variant 2, lr inside the residual:   c = beta (worker), s = 1/K, h = eta.
 * A learning-rate schedule changes eta between iterations; the constants are
 * then those of the iteration's eta.
 */
void orc_variant_constants(int variant, double beta, double eta, int K, float* c, float* s, float* h)
{
    float c_gmc, s_gmc;
    orc_constants(beta, eta, K, &c_gmc, &s_gmc);
    const float b = (float)beta;
    if (variant == 1) {
        *c = b;
        *s = s_gmc;
        *h = 1.0f;
    } else if (variant == 2) {
        *c = (float)beta;
        *s = (float)(1.0 / (double)K);
        *h = (float)eta;
    } else {
        *c = c_gmc;
        *s = s_gmc;
        *h = 1.0f;
    }
}

/* Momentum on the server: the worker's vector carries no momentum term,
 * u = e_{t,k} + g_{t,k}. */
void orc_precompress_plain(int64_t d, const float* g, const float* e, float* u)
{
    for (int64_t j = 0; j < d; ++j) u[j] = e[j] + g[j];
}

/* Learning rate inside the residual:
 * u = e_{t,k} + eta g_{t,k} - beta (w_t - w_{t-1}), left to right, with
 * h = eta and b = beta in binary32. */
void orc_precompress_lr(int64_t d, float h, float b, const float* w_t, const float* w_prev,
                        const float* g, const float* e, float* u)
{
    for (int64_t j = 0; j < d; ++j) {
        float dw = w_t[j] - w_prev[j];
        float pull = b * dw;
        float sg = h * g[j];
        float sum = e[j] + sg;
        u[j] = sum - pull;
    }
}

/* Momentum on the server: w_{t+1} = w_t - (eta/K) sum_k C(u_k) + beta (w_t - w_{t-1}),
 * left to right: (w_t + delta) + b (w_t - w_{t-1}) with delta from
 * orc_aggregate and b = beta in binary32. */
void orc_apply_server_momentum(int64_t d, float b, const float* w_t, const float* w_prev,
                               const float* delta, float* w_next)
{
    for (int64_t j = 0; j < d; ++j) {
        float moved = w_t[j] + delta[j];
        float back = w_t[j] - w_prev[j];
        float push = b * back;
        w_next[j] = moved + push;
    }
}

/* ------------------------------------------------------------------------- */
/* The experiments' approximate top-s (Section 5.1)                           */
/* ------------------------------------------------------------------------- */

/* Draw i of worker k's sample at step t: output i of a SplitMix64 generator
 * whose state starts at seed XOR mix(t + 1) XOR mix((k + 1) * 2^32). */
uint64_t orc_sample_draw(uint64_t seed, uint64_t t, uint64_t k, uint64_t i)
{
    const uint64_t gamma = 0x9e3779b97f4a7c15ULL;
    uint64_t state = seed ^ orc_splitmix64_mix(t + 1) ^ orc_splitmix64_mix((k + 1) << 32);
    return orc_splitmix64_mix(state + (i + 1) * gamma);
}

/*
 * The random subset S of Section 5.1, one component per stratum: stratum i
 * covers [i L, min((i + 1) L, n)) and contributes the component at offset
 * ((x_i >> 32) * len_i) >> 32 with x_i = orc_sample_draw(seed, t, k, i).
 * |S| = ceil(n / L) (L = 100: the paper's |S| = d/100).  Writes the
 * positions in ascending order and returns |S|.
 */
int64_t orc_sample_positions(uint64_t seed, uint64_t t, uint64_t k, int64_t n, int64_t L, int64_t* pos)
{
    int64_t m = (n + L - 1) / L;
    for (int64_t i = 0; i < m; ++i) {
        int64_t lo = i * L;
        int64_t len = n - lo < L ? n - lo : L;
        uint64_t x = orc_sample_draw(seed, t, k, (uint64_t)i);
        pos[i] = lo + (int64_t)(((x >> 32) * (uint64_t)len) >> 32);
    }
    return m;
}

static int cmp_key_desc(const void* a, const void* b)
{
    uint32_t x = *(const uint32_t*)a, y = *(const uint32_t*)b;
    return (x < y) - (x > y);
}

/*
 * Approximate top-s (Section 5.1): theta is the magnitude key ranked r-th
 * from the top among the sample's components, r = orc_count(|S|, ratio)
 * (ratio 1/1024 in the paper), and C(u) keeps every component of u whose key
 * is >= theta, in ascending order; the message length varies around n ratio.
 * u becomes the residual u - C(u).  idx and val hold up to n entries.
 * Returns the number kept, or -1 if the scratch allocation fails.
 */
int64_t orc_compress_approx(float* u, int64_t n, uint64_t seed, uint64_t t, uint64_t k, int64_t L,
                            double ratio, int32_t* idx, float* val)
{
    int64_t m = (n + L - 1) / L;
    int64_t* pos = (int64_t*)malloc((size_t)(m > 0 ? m : 1) * sizeof(int64_t));
    uint32_t* keys = (uint32_t*)malloc((size_t)(m > 0 ? m : 1) * sizeof(uint32_t));
    if (!pos || !keys) {
        free(pos);
        free(keys);
        return -1;
    }
    orc_sample_positions(seed, t, k, n, L, pos);
    for (int64_t i = 0; i < m; ++i) keys[i] = key_of(u[pos[i]]);
    qsort(keys, (size_t)m, sizeof(uint32_t), cmp_key_desc);
    int64_t r = orc_count(m, ratio);
    uint32_t theta = keys[r - 1];
    int64_t cnt = 0;
    for (int64_t j = 0; j < n; ++j) {
        if (key_of(u[j]) >= theta) {
            const float kept = u[j];
            idx[cnt] = (int32_t)j;
            val[cnt] = kept;
            u[j] = kept - kept;
            ++cnt;
        }
    }
    free(pos);
    free(keys);
    return cnt;
}
