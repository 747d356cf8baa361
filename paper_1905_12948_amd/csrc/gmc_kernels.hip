// HIP kernels of the GMC hot path for CDNA4 (gfx950, wave64).
//
// One iteration of Algorithm 1 (GMC) for K workers resident on one GPU:
//
//   topk_fused   u_k = (e_k + g_k) - c (w_t - w_prev) for every worker, written
//                over e_k; components whose magnitude key reaches the pair's
//                speculative threshold are kept as candidates
//   topk_compact packs each pair's candidates into a list in index order
//   topk_hist    three radix-select passes (11 + 11 + 9 bits of the key) over
//                the candidates, or over all of u when the candidates cannot
//                prove they hold the top k; the last workgroup of each
//                (worker, segment) picks the digit.  The first pass runs
//                with the compaction copy; the third also counts, per slice,
//                the components above and at the threshold and lays out the
//                message (the sampled-threshold top-s, whose passes run over
//                its sample, counts in topk_count)
//   topk_emit    ordered compaction of the kept components into the message,
//                residual u - u at the kept components, and the server
//                pass's row pointers
//   rbgs_*       shared block draw and the fused pass that gathers whole blocks
//   agg_*        the server sum over workers in worker order, the update and
//                w_{t+1} = w_t + update
//   apply        w_prev <- w (optional), w <- w + update
//
// Arithmetic is binary32 with one rounding per operation; the library is
// built with -ffp-contract=off so no multiply-add is fused.
#include "gmc_internal.h"

namespace gmc {

namespace {

__device__ __forceinline__ uint32_t key_of(float x) { return __float_as_uint(x) & 0x7fffffffu; }

__device__ __forceinline__ uint64_t lanemask_lt() {
    const uint32_t lane = threadIdx.x & (kWave - 1);
    return lane == 0 ? 0ull : (~0ull >> (64 - lane));
}

__device__ __forceinline__ uint32_t popc64(uint64_t x) { return (uint32_t)__popcll(x); }

__device__ __forceinline__ uint64_t ballot(bool p) { return __ballot(p); }

// Exclusive prefix over lanes of a small count v in [0, 7], and the wave total.
__device__ __forceinline__ uint32_t wave_prefix_small(uint32_t v, uint32_t* total) {
    const uint64_t b0 = ballot(v & 1u), b1 = ballot(v & 2u), b2 = ballot(v & 4u);
    const uint64_t lt = lanemask_lt();
    *total = popc64(b0) + 2u * popc64(b1) + 4u * popc64(b2);
    return popc64(b0 & lt) + 2u * popc64(b1 & lt) + 4u * popc64(b2 & lt);
}

__device__ __forceinline__ float4 ld4(const float* p) { return *reinterpret_cast<const float4*>(p); }
__device__ __forceinline__ void st4(float* p, float4 v) { *reinterpret_cast<float4*>(p) = v; }

// Streaming (nontemporal) access for data touched once per step: the K
// workers' g and e rows are gigabytes, far beyond any cache level.
__device__ __forceinline__ float4 ld4_stream(const float* p) {
    float4 v;
    v.x = __builtin_nontemporal_load(p + 0);
    v.y = __builtin_nontemporal_load(p + 1);
    v.z = __builtin_nontemporal_load(p + 2);
    v.w = __builtin_nontemporal_load(p + 3);
    return v;
}
__device__ __forceinline__ void st4_stream(float* p, float4 v) {
    __builtin_nontemporal_store(v.x, p + 0);
    __builtin_nontemporal_store(v.y, p + 1);
    __builtin_nontemporal_store(v.z, p + 2);
    __builtin_nontemporal_store(v.w, p + 3);
}

__device__ __forceinline__ bool aligned16(const void* p) {
    return (reinterpret_cast<uintptr_t>(p) & 15u) == 0;
}

// The sub-total of (worker k, compaction group cg) that chunk adds into, in
// the half of grp_acc of the parity of t.
__device__ __forceinline__ uint32_t* grp_slot(const TopkScratch& s, const TopkGeometry& g, uint64_t t, int k, int cg,
                                              int chunk) {
    const size_t nz = (size_t)g.K * g.n_cgroups;
    return s.grp_acc + ((size_t)(t & 1) * kGrpSub + (size_t)(chunk % kGrpSub)) * nz + (size_t)k * g.n_cgroups + cg;
}

// The candidates of (worker k, compaction group cg) of the step of t: the sum
// of the group's sub-totals.
__device__ __forceinline__ uint32_t grp_total(const TopkScratch& s, const TopkGeometry& g, uint64_t t, int k, int cg) {
    const size_t nz = (size_t)g.K * g.n_cgroups;
    const uint32_t* p = s.grp_acc + (size_t)(t & 1) * kGrpSub * nz + (size_t)k * g.n_cgroups + cg;
    uint32_t v = 0;
#pragma unroll
    for (int i = 0; i < kGrpSub; ++i) v += p[(size_t)i * nz];
    return v;
}

// u = (e + g) - m, two roundings, in this order.
__device__ __forceinline__ float precompress(float e, float g, float m) {
    const float acc = e + g;
    return acc - m;
}

// u under an update rule, from e, g and the two parameter vectors:
//   GMC (Algorithm 1)         (e + g) - c (w_t - w_prev)
//   momentum on the server    e + g
//   lr inside the residual    (e + h g) - c (w_t - w_prev)
template <int kRule>
__device__ __forceinline__ float rule_u(float e, float g, float wt, float wp, float c, float h) {
    if (kRule == kRuleServerMomentum) return e + g;
    const float m = c * (wt - wp);
    if (kRule == kRuleLrInResidual) {
        const float sg = h * g;
        const float acc = e + sg;
        return acc - m;
    }
    return precompress(e, g, m);
}

// rule_u with w_t - w_prev given: diff = fl(w_t - w_prev), bit for bit the
// same result.
template <int kRule>
__device__ __forceinline__ float rule_u_diff(float e, float g, float diff, float c, float h) {
    if (kRule == kRuleServerMomentum) return e + g;
    const float m = c * diff;
    if (kRule == kRuleLrInResidual) {
        const float sg = h * g;
        const float acc = e + sg;
        return acc - m;
    }
    return precompress(e, g, m);
}

__device__ __forceinline__ float rule_u_rt(int rule, float e, float g, float wt, float wp, float c, float h) {
    if (rule == kRuleServerMomentum) return rule_u<kRuleServerMomentum>(e, g, wt, wp, c, h);
    if (rule == kRuleLrInResidual) return rule_u<kRuleLrInResidual>(e, g, wt, wp, c, h);
    return rule_u<kRuleGmc>(e, g, wt, wp, c, h);
}

__device__ __forceinline__ float rule_u_diff_rt(int rule, float e, float g, float diff, float c, float h) {
    if (rule == kRuleServerMomentum) return rule_u_diff<kRuleServerMomentum>(e, g, diff, c, h);
    if (rule == kRuleLrInResidual) return rule_u_diff<kRuleLrInResidual>(e, g, diff, c, h);
    return rule_u_diff<kRuleGmc>(e, g, diff, c, h);
}

// The output mix of SplitMix64 (Steele, Lea and Flood, OOPSLA 2014).
__device__ __forceinline__ uint64_t splitmix64_mix(uint64_t z) {
    z = (z ^ (z >> 30)) * 0xbf58476d1ce4e5b9ull;
    z = (z ^ (z >> 27)) * 0x94d049bb133111ebull;
    return z ^ (z >> 31);
}

// Sampled-threshold top-s (Section 5.1): worker k's sample at step t holds
// one component per stratum of L consecutive components, at offset
// ((x >> 32) * len) >> 32 of stratum i, x the i-th output of a SplitMix64
// stream started at seed ^ mix(t + 1) ^ mix((k + 1) << 32).
__device__ __forceinline__ uint64_t sample_state(uint64_t seed, uint64_t t, int k) {
    return seed ^ splitmix64_mix(t + 1) ^ splitmix64_mix((uint64_t)(k + 1) << 32);
}

__device__ __forceinline__ int32_t sample_pos(uint64_t state, int32_t i, int32_t L, int32_t n) {
    const uint64_t x = splitmix64_mix(state + (uint64_t)(i + 1) * 0x9e3779b97f4a7c15ull);
    const int32_t lo = i * L;
    const int32_t len = n - lo < L ? n - lo : L;
    return lo + (int32_t)(((x >> 32) * (uint64_t)len) >> 32);
}

// Records the sample components among the four at [j, j + 4).
__device__ __forceinline__ void sample_float4(float* samp, uint64_t state, int32_t j, float4 u, int32_t L,
                                              int32_t n) {
    for (int32_t i = j / L; (int64_t)i * L < (int64_t)j + 4 && (int64_t)i * L < n; ++i) {
        const int32_t o = sample_pos(state, i, L, n) - j;
        if (o >= 0 && o < 4) samp[i] = o == 0 ? u.x : o == 1 ? u.y : o == 2 ? u.z : u.w;
    }
}

// Workgroup order of the streaming passes over (chunk, worker) (StepArgs::run,
// chosen on the host): runs of `run` consecutive chunks of one worker, the K
// workers of a run one after the other; or, with run == 0, chunk c on XCD
// c mod 8 with its K workers consecutive there.  Workgroups are dispatched
// round-robin over the 8 XCDs (workgroup b on XCD b mod 8), so with runs of
// 1 every XCD's cache pulls the w_t, w_prev lines a chunk reads, with runs of
// 2 four of them, with run 0 one.  Measured with w read everywhere, on the
// ResNet-50-sized step (K = 16) and the RBGS step (K = 8): runs of 1, 2, 4, 8
// chunks took 893/888/904/926 us and 671/629/628/630 us.  When w is read only
// at the changed components (the sparse momentum term) runs of 1 stream best
// (on a stream of the same shape without w, 804 us against 824 us for runs of
// 2; run 0 slows the ResNet-50-sized pass by 10%), unless the changed
// components are dense: at the ResNet-18-sized workload (8 workers sending
// 1% each) run 0 takes 186 us against 200 us.
constexpr int kXcds = 8;

__device__ __forceinline__ void run_order(int b, int K, int run, int* chunk, int* k) {
    if (run == 0) {
        const int x = b % kXcds, sl = b / kXcds;
        *k = sl % K;
        *chunk = (sl / K) * kXcds + x;
        return;
    }
    const int grp = b / (run * K), r = b % (run * K);
    *k = r / run;
    *chunk = grp * run + r % run;
}

__host__ __device__ inline int64_t run_order_grid(int64_t n_chunks, int K, int run) {
    if (run == 0) return (n_chunks + kXcds - 1) / kXcds * kXcds * K;
    return (n_chunks + run - 1) / run * run * K;
}

// The previous server pass's mark word of the components at j (a.wbits set).
// The top-s vector pass loads it before its stream of e and g: a wait for the
// word then leaves those loads in flight (vmcnt counts in issue order).
__device__ __forceinline__ uint32_t mark_word(const StepArgs& a, int64_t j) {
    return a.wbits ? a.wbits[j >> 5] : 0u;
}

// w_t and w_prev of the four components at j for the worker passes (word:
// mark_word(a, j)).  With the previous server pass's bitmap (a.wbits),
// unmarked components have w_t == w_prev, finite: w_t - w_prev is exactly +0
// there, so the loads are skipped (w_t is still read when the detached points
// need it) and the momentum term comes out +0, bit for bit what the dense
// loads give.
template <bool kDetach>
__device__ __forceinline__ void load_w4(const StepArgs& a, int64_t j, uint32_t word, float4* wt, float4* wv) {
    if (a.wbits) {
        const uint32_t marked = (word >> (j & 31)) & 0xfu;
        if (marked) {
            *wt = ld4(a.w_t + j);
            *wv = ld4(a.w_prev + j);
        } else if (kDetach) {
            *wt = ld4(a.w_t + j);
            *wv = *wt;
        } else {
            *wt = *wv = make_float4(0.f, 0.f, 0.f, 0.f);
        }
        return;
    }
    *wt = ld4(a.w_t + j);
    *wv = ld4(a.w_prev + j);
}

// GMC+'s detached point from w and the residual: w - q e (Algorithm 2).
__device__ __forceinline__ float detached(float w, float e, float q) {
    const float r = q * e;
    return w - r;
}

// Block-wide (256 threads) exclusive scan of one uint32 per thread; returns
// the thread's exclusive prefix and writes the total to *total.
__device__ __forceinline__ uint32_t block_scan_excl(uint32_t v, uint32_t* total, uint32_t* sh /*[kWavesPerGroup]*/) {
    const uint32_t lane = threadIdx.x & (kWave - 1), wave = threadIdx.x >> 6;
    uint32_t x = v;
    // inclusive wave scan (Hillis-Steele via shuffles)
#pragma unroll
    for (int o = 1; o < kWave; o <<= 1) {
        const uint32_t y = __shfl_up(x, o, kWave);
        if (lane >= (uint32_t)o) x += y;
    }
    if (lane == kWave - 1) sh[wave] = x;
    __syncthreads();
    uint32_t before = 0, all = 0;
#pragma unroll
    for (int w = 0; w < kWavesPerGroup; ++w) {
        const uint32_t t = sh[w];
        if (w < (int)wave) before += t;
        all += t;
    }
    __syncthreads();
    *total = all;
    return before + x - v;
}

// Cross-workgroup hand-off without cache flushes.  Everything one workgroup
// hands to another inside a kernel travels through agent-scope atomics
// (read-modify-writes, or loads/stores that bypass the non-coherent caches);
// these two helpers only order them: the producer waits until its atomics
// have completed before it signals, the consumer issues its reads only after
// it has seen the signal.  (An agent-scope fence would write back and
// invalidate the whole L2 in every workgroup.)
__device__ __forceinline__ void order_release() {
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup");
    __builtin_amdgcn_s_waitcnt(0 | (0x7 << 4) | (0xf << 8));  // vmcnt(0)
}

__device__ __forceinline__ void order_acquire() {
    __builtin_amdgcn_s_waitcnt(0 | (0x7 << 4) | (0xf << 8));  // vmcnt(0)
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup");
}

__device__ __forceinline__ uint32_t load_agent(const uint32_t* p) {
    return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

__device__ __forceinline__ void store_agent(uint32_t* p, uint32_t v) {
    __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

}  // namespace

// ============================================================================
// fused worker pass for top-s
// ============================================================================

// ---------------------------------------------------------------------------
// Vector path: one workgroup per (chunk, worker), 8 components per thread.
//
// Consecutive workgroups take the K workers of one chunk, so w_t and w_prev
// of the chunk are fetched from memory once and re-read from cache by the
// other K-1 workgroups.  g and e are streamed with nontemporal accesses.  A
// worker's candidates of the chunk go, in index order, to the chunk's own
// slot in the staging area (kChunk entries, so it can never overflow): the
// streaming pass takes no atomics; the compaction kernel packs the slots.
// ---------------------------------------------------------------------------

__device__ void fused_chunk_wave(const StepArgs& a, const TopkGeometry& g, const TopkScratch& s, int chunk,
                                 int k, const float* dl);

// w_t - w_prev of the components [start, start + len) (len <= kChunk) from
// the last server pass's change list into dl (LDS): fl(w_{t+1} - w_t) of
// every component that pass changed, +0 for the others.  False when a range
// of the chunk overflowed its list (never for a list that holds whole
// ranges).  The whole workgroup calls it; cnt: 2 words of LDS.
__device__ bool scatter_changes(const StepArgs& a, int start, int len, float* dl, int32_t* cnt) {
    const int nt = (int)blockDim.x;
    const int r0 = start / kAggTopkRange, nr = (start + len - 1) / kAggTopkRange - r0 + 1;  // 1 or 2 ranges
    for (int i = threadIdx.x; i < kChunk; i += nt) dl[i] = 0.0f;
    if (threadIdx.x == 0) {
        cnt[0] = a.dlist[(size_t)r0 * a.dl_stride].x;
        cnt[1] = nr > 1 ? a.dlist[(size_t)(r0 + 1) * a.dl_stride].x : 0;
    }
    __syncthreads();
    const int32_t n0 = cnt[0], n1 = cnt[1];
    const bool ok = n0 >= 0 && n1 >= 0;
    for (int h2 = 0; ok && h2 < nr; ++h2) {
        const int32_t c = h2 ? n1 : n0;
        const int2* L = a.dlist + (size_t)(r0 + h2) * a.dl_stride;
        for (int32_t e = 1 + (int32_t)threadIdx.x; e <= c; e += nt) {
            const int2 en = L[e];
            const int j = (r0 + h2) * kAggTopkRange + en.x;
            if (j >= start && j < start + len) dl[j - start] = __int_as_float(en.y);
        }
    }
    __syncthreads();
    return ok;
}

template <int kRule, bool kDetach, bool kApprox>
__global__ __launch_bounds__(kGroup) void topk_fused_vec_kernel(StepArgs a, TopkGeometry g, TopkScratch s,
                                                                uint64_t vec_mask) {
    __shared__ uint32_t wtot[2][kWavesPerGroup];
    __shared__ union {
        int2 stage[kChunk];  // the chunk's candidates, in index order
        float dl[kChunk];    // w_t - w_prev of the chunk's components (from the change list)
    } sm;
    __shared__ int32_t dl_cnt[2];
    int2* const stage = sm.stage;
    int chunk, k;
    run_order(blockIdx.x, g.K, a.run, &chunk, &k);
    if (chunk >= g.n_chunks || !((vec_mask >> k) & 1ull)) return;  // padding, or the element-wise kernel's
    // one segment (global top-s): the chunk's place is arithmetic, no table lookup
    const bool one = g.n_seg == 1;
    const int start = one ? chunk * kChunk : g.chunk_start[chunk];
    const int len = one ? min(kChunk, a.d - start) : g.chunk_len[chunk];
    if ((start & 3) != 0 || len != kChunk) {  // partial or unaligned chunk: element-wise, one wavefront
        // with w_prev NULL (the last server pass updated w in place) w_t -
        // w_prev exists only in that pass's change list, which holds whole
        // ranges
        const float* dl = nullptr;
        if (a.w_prev == nullptr) {
            scatter_changes(a, start, len, sm.dl, dl_cnt);
            dl = sm.dl;
        }
        if (threadIdx.x < kWave) fused_chunk_wave(a, g, s, chunk, k, dl);
        return;
    }
    const int lane = threadIdx.x & (kWave - 1), wave = threadIdx.x >> 6;
    const int seg = one ? 0 : g.chunk_seg[chunk];
    const int p = k * g.n_seg + seg;
    const uint32_t tau = s.pair[p].tau;
    const float c = a.c, h = a.h;
    const int o0 = threadIdx.x * 4;               // components o0..o0+3 and 1024+o0..1024+o0+3
    float* ep = a.wp.e[k] + start + o0;
    const float* gp = a.wp.g[k] + start + o0;
    constexpr bool kNeedW = kRule != kRuleServerMomentum || kDetach;
    // w_t - w_prev from the last server pass's change list (unless a range
    // of the chunk overflowed its list): the chunk's changed components are
    // scattered into LDS, every other one is exactly +0
    bool use_list = !kDetach && kNeedW && a.dlist != nullptr;
    float4 u[2], gv[2], wt[2], wv[2];
    uint32_t mw[2] = {0u, 0u};  // the mark words first, then the stream (see mark_word)
    if (kNeedW && !use_list) {
#pragma unroll
        for (int i = 0; i < 2; ++i) mw[i] = mark_word(a, (int64_t)start + o0 + i * (kGroup * 4));
    }
#pragma unroll
    for (int i = 0; i < 2; ++i) {
        u[i] = ld4_stream(ep + i * (kGroup * 4));
        gv[i] = ld4_stream(gp + i * (kGroup * 4));
    }
#pragma unroll
    for (int i = 0; i < 2; ++i) {
        wt[i] = wv[i] = make_float4(0.f, 0.f, 0.f, 0.f);
        if (kNeedW && !use_list) load_w4<kDetach>(a, (int64_t)start + o0 + i * (kGroup * 4), mw[i], &wt[i], &wv[i]);
    }
    if (use_list) {
        const int r0 = start / kAggTopkRange, nr = (start + len - 1) / kAggTopkRange - r0 + 1;  // 1 or 2 ranges
        int2 head0 = make_int2(0, 0), head1 = make_int2(0, 0);
        if ((int)threadIdx.x < kWave) {
            head0 = a.dlist[(size_t)r0 * a.dl_stride + threadIdx.x];
            if (nr > 1) head1 = a.dlist[(size_t)(r0 + 1) * a.dl_stride + threadIdx.x];
        }
#pragma unroll
        for (int i = 0; i < kChunk / kGroup; ++i) sm.dl[i * kGroup + threadIdx.x] = 0.0f;
        if (threadIdx.x == 0) {
            dl_cnt[0] = head0.x;
            dl_cnt[1] = nr > 1 ? head1.x : 0;
        }
        __syncthreads();
        const int32_t n0 = dl_cnt[0], n1 = dl_cnt[1];
        use_list = n0 >= 0 && n1 >= 0;
        if (use_list) {
            auto put = [&](int2 en, int rr) {
                const int j = rr * kAggTopkRange + en.x;
                if (j >= start && j < start + len) sm.dl[j - start] = __int_as_float(en.y);
            };
#pragma unroll
            for (int h2 = 0; h2 < 2; ++h2) {
                if (h2 >= nr) break;
                const int32_t cnt = h2 ? n1 : n0;
                if (threadIdx.x >= 1 && (int32_t)threadIdx.x <= cnt && (int)threadIdx.x < kWave)
                    put(h2 ? head1 : head0, r0 + h2);
                for (int32_t e2 = kWave + threadIdx.x; e2 <= cnt; e2 += kGroup)
                    put(a.dlist[(size_t)(r0 + h2) * a.dl_stride + e2], r0 + h2);
            }
        }
        __syncthreads();
        if (!use_list) {  // a range's list overflowed (w_prev is then set): the marks and the two parameter vectors
#pragma unroll
            for (int i = 0; i < 2; ++i) {
                const int64_t j = (int64_t)start + o0 + i * (kGroup * 4);
                load_w4<kDetach>(a, j, mark_word(a, j), &wt[i], &wv[i]);
            }
        }
    }
    uint32_t flags = 0;
#pragma unroll
    for (int i = 0; i < 2; ++i) {
        if (use_list) {
            const float4 df = *reinterpret_cast<const float4*>(&sm.dl[o0 + i * (kGroup * 4)]);
            u[i].x = rule_u_diff<kRule>(u[i].x, gv[i].x, df.x, c, h);
            u[i].y = rule_u_diff<kRule>(u[i].y, gv[i].y, df.y, c, h);
            u[i].z = rule_u_diff<kRule>(u[i].z, gv[i].z, df.z, c, h);
            u[i].w = rule_u_diff<kRule>(u[i].w, gv[i].w, df.w, c, h);
        } else {
            u[i].x = rule_u<kRule>(u[i].x, gv[i].x, wt[i].x, wv[i].x, c, h);
            u[i].y = rule_u<kRule>(u[i].y, gv[i].y, wt[i].y, wv[i].y, c, h);
            u[i].z = rule_u<kRule>(u[i].z, gv[i].z, wt[i].z, wv[i].z, c, h);
            u[i].w = rule_u<kRule>(u[i].w, gv[i].w, wt[i].w, wv[i].w, c, h);
        }
        st4_stream(ep + i * (kGroup * 4), u[i]);
        if (kDetach) {
            const float q = a.q;
            st4_stream(a.wp.y[k] + start + o0 + i * (kGroup * 4),
                       make_float4(detached(wt[i].x, u[i].x, q), detached(wt[i].y, u[i].y, q),
                                   detached(wt[i].z, u[i].z, q), detached(wt[i].w, u[i].w, q)));
        }
        flags |= (key_of(u[i].x) >= tau ? 1u : 0u) << (i * 4 + 0);
        flags |= (key_of(u[i].y) >= tau ? 1u : 0u) << (i * 4 + 1);
        flags |= (key_of(u[i].z) >= tau ? 1u : 0u) << (i * 4 + 2);
        flags |= (key_of(u[i].w) >= tau ? 1u : 0u) << (i * 4 + 3);
    }
    if (kApprox) {
        const uint64_t sst = sample_state(a.seed, a.t, k);
        float* sp = s.samp + (size_t)k * g.samp_n;
#pragma unroll
        for (int i = 0; i < 2; ++i) sample_float4(sp, sst, start + o0 + i * (kGroup * 4), u[i], g.stratum, a.d);
    }
    const size_t run_slot = (size_t)k * g.n_chunks + chunk;
    if (__syncthreads_or(flags != 0u) == 0) {
        if (threadIdx.x == 0) s.run_cnt[run_slot] = 0u;
        return;
    }
    // position in index order: (i, thread, q)
    uint32_t pre[2];
#pragma unroll
    for (int i = 0; i < 2; ++i) {
        uint32_t tot;
        pre[i] = wave_prefix_small((uint32_t)__popc((flags >> (i * 4)) & 0xfu), &tot);
        if (lane == 0) wtot[i][wave] = tot;
    }
    __syncthreads();
    uint32_t total = 0, pos[2];
#pragma unroll
    for (int i = 0; i < 2; ++i) {
        uint32_t before = 0;
#pragma unroll
        for (int w = 0; w < kWavesPerGroup; ++w) {
            if (w < wave) before += wtot[i][w];
        }
        pos[i] = total + before + pre[i];
#pragma unroll
        for (int w = 0; w < kWavesPerGroup; ++w) total += wtot[i][w];
    }
    // the chunk's compaction group (a table lookup with several segments),
    // loaded now so that its latency overlaps the staging
    const int cg = one ? chunk / kCompactChunks : g.chunk_cgrp[chunk];
    // gather the candidates in LDS, then write the slot with consecutive
    // threads on consecutive entries (a few whole lines instead of one
    // partial line per candidate)
#pragma unroll
    for (int i = 0; i < 2; ++i) {
        const uint32_t bits = (flags >> (i * 4)) & 0xfu;
        uint32_t q = pos[i];
        const int j = start + o0 + i * (kGroup * 4);
        if (bits & 1u) { stage[q] = make_int2(j + 0, __float_as_int(u[i].x)); ++q; }
        if (bits & 2u) { stage[q] = make_int2(j + 1, __float_as_int(u[i].y)); ++q; }
        if (bits & 4u) { stage[q] = make_int2(j + 2, __float_as_int(u[i].z)); ++q; }
        if (bits & 8u) { stage[q] = make_int2(j + 3, __float_as_int(u[i].w)); }
    }
    __syncthreads();
    int2* sp = s.slot + run_slot * kChunk;
    for (uint32_t q = threadIdx.x; q < total; q += kGroup) sp[q] = stage[q];
    // the count and the device-scope add into the group's total come last:
    // nothing after them waits for their completion (a wait on the add,
    // which travels to the memory-side atomic unit, held up every wave of
    // the workgroup through the staging barriers: 20-30 us per pass)
    if (threadIdx.x == 0) {
        s.run_cnt[run_slot] = total;
        atomicAdd(grp_slot(s, g, a.t, k, cg, chunk), total);
    }
}


// Element-wise pass of one wavefront over one (chunk, worker): the chunks the
// vector path cannot take (a segment's partial last chunk, chunks with an
// unaligned start) and the workers whose rows are not 16-byte aligned.  dl
// (nullable, LDS): w_t - w_prev of the chunk's components (scatter_changes),
// used instead of the two parameter vectors.
__device__ void fused_chunk_wave(const StepArgs& a, const TopkGeometry& g, const TopkScratch& s, int chunk,
                                 int k, const float* dl) {
    const int lane = threadIdx.x & (kWave - 1);
    const int start = g.chunk_start[chunk];
    const int len = g.chunk_len[chunk];
    const int seg = g.chunk_seg[chunk];
    const float c = a.c;
    constexpr int kIt = kChunk / kWave;  // 32
    const int p = k * g.n_seg + seg;
    const uint32_t tau = s.pair[p].tau;
    float* e = a.wp.e[k];
    const float* gr = a.wp.g[k];
    uint32_t flags = 0;
    const uint64_t sst = g.approx ? sample_state(a.seed, a.t, k) : 0ull;
#pragma unroll 4
    for (int i = 0; i < kIt; ++i) {
        const int o = i * kWave + lane;
        if (o < len) {
            const int j = start + o;
            const float u = dl ? rule_u_diff_rt(a.rule, e[j], gr[j], dl[o], c, a.h)
                               : rule_u_rt(a.rule, e[j], gr[j], a.w_t[j], a.w_prev[j], c, a.h);
            e[j] = u;
            if (a.detach) a.wp.y[k][j] = detached(a.w_t[j], u, a.q);
            flags |= (key_of(u) >= tau ? 1u : 0u) << i;
            if (g.approx) {
                const int32_t q = j / g.stratum;
                if (sample_pos(sst, q, g.stratum, a.d) == j) s.samp[(size_t)k * g.samp_n + q] = u;
            }
        }
    }
    // the chunk's slot, in index order (iteration-major, then lane)
    const size_t run_slot = (size_t)k * g.n_chunks + chunk;
    int2* sp = s.slot + run_slot * kChunk;
    const uint64_t lt = lanemask_lt();
    uint32_t base = 0;
    for (int i = 0; i < kIt; ++i) {
        const uint64_t b = ballot((flags >> i) & 1u);
        if ((flags >> i) & 1u) {
            const uint32_t q = base + popc64(b & lt);
            const int j = start + i * kWave + lane;
            sp[q] = make_int2(j, __float_as_int(e[j]));  // re-read of this lane's own store
        }
        base += popc64(b);
    }
    if (lane == 0) {
        s.run_cnt[run_slot] = base;
        if (base)
            atomicAdd(grp_slot(s, g, a.t, k, g.chunk_cgrp[chunk], chunk), base);
    }
}

// The element-wise kernel: one workgroup of one wavefront per (chunk,
// worker) for the workers outside vec_mask (the vector kernel takes every
// chunk of the others, partial ones included).
__global__ __launch_bounds__(kWave) void topk_fused_gen_kernel(StepArgs a, TopkGeometry g, TopkScratch s,
                                                               uint64_t vec_mask) {
    __shared__ float dl[kChunk];
    __shared__ int32_t dl_cnt[2];
    const int64_t wid = blockIdx.x;
    if (wid >= (int64_t)g.n_chunks * g.K) return;
    const int chunk = (int)(wid / g.K), k = (int)(wid % g.K);
    if ((vec_mask >> k) & 1ull) return;  // the vector kernel's
    const float* d = nullptr;
    if (a.w_prev == nullptr) {  // w_t - w_prev from the last in-place server pass's list
        scatter_changes(a, g.chunk_start[chunk], g.chunk_len[chunk], dl, dl_cnt);
        d = dl;
    }
    fused_chunk_wave(a, g, s, chunk, k, d);
}

template <bool kApprox>
static hipError_t launch_fused_vec_rule(const StepArgs& a, const TopkGeometry& g, const TopkScratch& s,
                                       uint64_t vec_mask, hipStream_t st) {
    const int grid = (int)run_order_grid(g.n_chunks, g.K, a.run);
    if (a.rule == kRuleServerMomentum) {
        if (a.detach) return hipErrorInvalidValue;  // the detached points need w_{t+1} = w_t off the sent set
        hipLaunchKernelGGL((topk_fused_vec_kernel<kRuleServerMomentum, false, kApprox>), dim3(grid), dim3(kGroup), 0,
                           st, a, g, s, vec_mask);
    } else if (a.rule == kRuleLrInResidual) {
        if (a.detach)
            hipLaunchKernelGGL((topk_fused_vec_kernel<kRuleLrInResidual, true, kApprox>), dim3(grid), dim3(kGroup),
                               0, st, a, g, s, vec_mask);
        else
            hipLaunchKernelGGL((topk_fused_vec_kernel<kRuleLrInResidual, false, kApprox>), dim3(grid), dim3(kGroup),
                               0, st, a, g, s, vec_mask);
    } else {
        if (a.detach)
            hipLaunchKernelGGL((topk_fused_vec_kernel<kRuleGmc, true, kApprox>), dim3(grid), dim3(kGroup), 0, st, a,
                               g, s, vec_mask);
        else
            hipLaunchKernelGGL((topk_fused_vec_kernel<kRuleGmc, false, kApprox>), dim3(grid), dim3(kGroup), 0, st,
                               a, g, s, vec_mask);
    }
    return hipGetLastError();
}

hipError_t launch_topk_fused_vec(const StepArgs& a, const TopkGeometry& g, const TopkScratch& s,
                                 uint64_t vec_mask, hipStream_t st) {
    return g.approx ? launch_fused_vec_rule<true>(a, g, s, vec_mask, st)
                    : launch_fused_vec_rule<false>(a, g, s, vec_mask, st);
}

hipError_t launch_topk_fused_gen(const StepArgs& a, const TopkGeometry& g, const TopkScratch& s,
                                 uint64_t vec_mask, hipStream_t st) {
    const int64_t grid = (int64_t)g.n_chunks * g.K;
    hipLaunchKernelGGL(topk_fused_gen_kernel, dim3((unsigned)grid), dim3(kWave), 0, st, a, g, s, vec_mask);
    return hipGetLastError();
}

// ============================================================================
// selection
//
// The input of a (worker, segment) pair's selection is either its candidate
// list (mode 0: the fused pass collected every component whose key reaches
// the speculative threshold, and there are at least k and at most the
// capacity of them) or all of the segment's u (mode 1, the full-data path).
// Both are in ascending index order.  The histogram, count and emit passes
// read them as flat slices, one workgroup per slice; the count pass scans
// the slices' counts so that each emit workgroup knows where its kept
// components go.
// ============================================================================

namespace {

constexpr int kSliceLoads = 16;      // independent loads in flight per thread
constexpr int kSliceLoads4 = 8;      // 16-byte loads in flight per thread over contiguous u
constexpr int kEmitLoads = 4;        // staged elements per thread in the emit pass
constexpr int kEmitStage = kGroup * kEmitLoads;  // elements staged in LDS per round
constexpr int kFullRound = kGroup * 16;          // full-data elements per round of the emit

// A workgroup's slice of a pair's selection input.
struct Slice {
    int64_t lo, hi;          // positions in the input array
    const float* val;        // mode 0: candidate values; mode 1: u of the segment (held in e);
                             // mode 2: the sample
    const int32_t* idx;      // mode 0: candidate indices; mode 1: NULL (index = seg_lo + position)
    int32_t seg_lo;
};

__device__ __forceinline__ Slice open_slice(int mode, uint32_t cand, int k, int seg, int p, int w, int W,
                                            const StepArgs& a, const TopkGeometry& g, const TopkScratch& s) {
    Slice v;
    v.seg_lo = g.seg_start[seg];
    const int64_t total = mode == 0   ? (int64_t)cand
                          : mode == 2 ? (int64_t)g.samp_n
                                      : (int64_t)(g.seg_start[seg + 1] - v.seg_lo);
    v.lo = total * w / W;
    v.hi = total * (w + 1) / W;
    if (mode == 0) {
        v.val = s.cand_val + g.pair_cand[p];
        v.idx = s.cand_idx + g.pair_cand[p];
    } else if (mode == 2) {  // the sample (sampled-threshold top-s; values only)
        v.val = s.samp + (size_t)k * g.samp_n;
        v.idx = nullptr;
    } else {
        v.val = a.wp.e[k] + v.seg_lo;
        v.idx = nullptr;
    }
    return v;
}

// Run q of a collected slice (kModeCollected): the components wave q of the
// second pass gathered from its quarter of the full-data slice w of W, in
// index order, at that quarter's positions in the pair's staging rows (the
// pair's slot area: indices in its first n words, values in the next n, n the
// segment's length; the quarter is at most that long, so runs never overlap).
__device__ __forceinline__ Slice collected_run(const TopkGeometry& g, const TopkScratch& s, int k, int seg, int w,
                                               int W, int q) {
    const int64_t n = g.seg_start[seg + 1] - g.seg_start[seg];
    const int64_t lo = n * w / W, len = n * (w + 1) / W - lo;
    int32_t* base = reinterpret_cast<int32_t*>(s.slot + ((size_t)k * g.n_chunks + g.cgrp_lo[g.seg_cgrp_lo[seg]]) * kChunk);
    Slice v;
    v.seg_lo = g.seg_start[seg];
    v.idx = base;
    v.val = reinterpret_cast<const float*>(base + n);
    v.lo = lo + len * q / kWavesPerGroup;
    v.hi = v.lo + s.sl_run[((size_t)k * g.n_slices + g.seg_slice_lo[seg] + w) * kWavesPerGroup + q];
    return v;
}

// f(key, index) for every element of the slice; loads are issued
// kSliceLoads at a time per thread.
template <bool kNeedIdx, class F>
__device__ __forceinline__ void for_slice(const Slice& v, F f) {
    for (int64_t b = v.lo; b < v.hi; b += (int64_t)kGroup * kSliceLoads) {
        float x[kSliceLoads];
        int32_t j[kSliceLoads];
#pragma unroll
        for (int i = 0; i < kSliceLoads; ++i) {
            const int64_t pos = b + (int64_t)i * kGroup + threadIdx.x;
            x[i] = 0.0f;
            j[i] = 0;
            if (pos < v.hi) {
                x[i] = v.val[pos];
                if (kNeedIdx) j[i] = v.idx ? v.idx[pos] : v.seg_lo + (int32_t)pos;
            }
        }
#pragma unroll
        for (int i = 0; i < kSliceLoads; ++i) {
            const int64_t pos = b + (int64_t)i * kGroup + threadIdx.x;
            if (pos < v.hi) f(key_of(x[i]), j[i]);
        }
    }
}

// f(key) for every element of a contiguous slice (no index array: the full
// data, or the sample), with 16-byte loads, kSliceLoads4 of them in flight
// per thread (32 KB per workgroup: the full-data passes are bound by the
// bytes in flight); the head up to the first 16-byte boundary and the tail
// element-wise.  The order of the calls is not the index order.
template <class F>
__device__ __forceinline__ void for_slice_contig(const Slice& v, F f) {
    const float* p = v.val;
    int64_t lo = v.lo;
    const int64_t hi = v.hi;
    const int64_t mis = (int64_t)((reinterpret_cast<uintptr_t>(p + lo) >> 2) & 3u);
    const int64_t head = mis ? (4 - mis < hi - lo ? 4 - mis : hi - lo) : 0;
    if ((int64_t)threadIdx.x < head) f(key_of(p[lo + threadIdx.x]));
    lo += head;
    const int64_t n4 = (hi - lo) / 4;
    const float4* p4 = reinterpret_cast<const float4*>(p + lo);
    for (int64_t b = 0; b < n4; b += (int64_t)kGroup * kSliceLoads4) {
        float4 x[kSliceLoads4];
        // every load unconditional (a position past the end reads the last
        // float4, dropped below), so all kSliceLoads4 are in flight at once
#pragma unroll
        for (int i = 0; i < kSliceLoads4; ++i) {
            const int64_t q = b + i * kGroup + threadIdx.x;
            x[i] = p4[q < n4 ? q : n4 - 1];
        }
#pragma unroll
        for (int i = 0; i < kSliceLoads4; ++i) {
            if (b + i * kGroup + threadIdx.x < n4) {
                f(key_of(x[i].x));
                f(key_of(x[i].y));
                f(key_of(x[i].z));
                f(key_of(x[i].w));
            }
        }
    }
    const int64_t t0 = lo + n4 * 4;
    if (t0 + (int64_t)threadIdx.x < hi) f(key_of(p[t0 + threadIdx.x]));
}

// The bin b (scanning from the top) with above(b) < need <= above(b) + h[b],
// above(b) = sum of the bins above b; h in LDS, nbins a multiple of kGroup.
// Returns -1 if the bins hold fewer than need elements.
__device__ int find_bin(const uint32_t* h, int nbins, uint32_t need, uint32_t* above_out, uint32_t* sh_wsum,
                        int* sh_res) {
    const int per = nbins / kGroup;
    const int t = threadIdx.x;
    const int rt = kGroup - 1 - t;  // thread rt owns the per bins ending (from the top) at rank rt
    uint32_t mine = 0;
    for (int q = 0; q < per; ++q) mine += h[rt * per + q];
    uint32_t total;
    uint32_t above = block_scan_excl(mine, &total, sh_wsum);  // bins above this thread's, in reverse order
    if (t == 0) sh_res[0] = -1;
    __syncthreads();
    for (int q = per - 1; q >= 0; --q) {
        const uint32_t hb = h[rt * per + q];
        if (above < need && need <= above + hb) {
            sh_res[0] = rt * per + q;
            sh_res[1] = (int)above;
        }
        above += hb;
    }
    __syncthreads();
    const int b = sh_res[0];
    *above_out = (uint32_t)sh_res[1];
    __syncthreads();
    return b;
}

// Workgroup -> (worker, segment, slice) of the histogram and count passes.
struct SliceId {
    int k, seg, p, w, W;
};

__device__ __forceinline__ SliceId slice_id(const TopkGeometry& g, int blk) {
    SliceId id;
    id.k = blk / g.n_slices;
    const int r = blk % g.n_slices;
    id.seg = g.slice_seg[r];
    id.w = g.slice_rank[r];
    id.W = g.seg_slices[id.seg];
    id.p = id.k * g.n_seg + id.seg;
    return id;
}

// Signals that this workgroup's contribution (global atomics) is complete;
// true in exactly one workgroup of the pair, the last to finish.
__device__ __forceinline__ bool finish_slice(uint32_t* done, int W, int* sh_flag) {
    order_release();
    __syncthreads();
    if (threadIdx.x == 0) *sh_flag = atomicAdd(done, 1u) == (uint32_t)W - 1u;
    __syncthreads();
    if (!*sh_flag) return false;
    order_acquire();
    return true;
}

// The last workgroup of a pair, once T and r are known: from each slice's
// counts of kept components above T and at T (get(slice, &A, &Ti), the
// segment's slices in index order) the message offset of each slice's first
// kept component and the at-T components in earlier slices (the r ties kept
// go to the lowest indices); then the message length.  carry: 2 words of LDS.
template <class Get>
__device__ void scan_slices(const SliceId& id, int W, int32_t r, Get get, const TopkGeometry& g,
                            const TopkScratch& s, int64_t* msg_len, int64_t msg_total, uint32_t* sh_wsum,
                            uint32_t* carry) {
    const size_t base = (size_t)id.k * g.n_slices + g.seg_slice_lo[id.seg];
    if (threadIdx.x == 0) {
        carry[0] = 0;  // ties before
        carry[1] = 0;  // kept before
    }
    __syncthreads();
    for (int c0 = 0; c0 < W; c0 += kGroup) {
        const int i = c0 + threadIdx.x;
        uint32_t A = 0, Ti = 0;
        if (i < W) get(base + i, &A, &Ti);
        uint32_t tot_t;
        const uint32_t tie_pre = carry[0] + block_scan_excl(Ti, &tot_t, sh_wsum);
        int64_t take = (int64_t)r - (int64_t)tie_pre;
        if (take < 0) take = 0;
        if (take > (int64_t)Ti) take = Ti;
        const uint32_t sel = A + (uint32_t)take;
        uint32_t tot_s;
        const uint32_t sel_pre = carry[1] + block_scan_excl(sel, &tot_s, sh_wsum);
        if (i < W) {
            s.sl_tiebase[base + i] = tie_pre;
            s.sl_out[base + i] = sel_pre;
        }
        __syncthreads();
        if (threadIdx.x == 0) {
            carry[0] += tot_t;
            carry[1] += tot_s;
        }
        __syncthreads();
    }
    if (threadIdx.x == 0) {
        if (g.approx) {
            msg_len[id.k] = (int64_t)carry[1];  // one segment; the count varies
        } else {
            if (carry[1] != (uint32_t)g.pair_k[id.p]) atomicAdd((unsigned long long*)&s.stats[4], 1ull);
            if (id.seg == 0) msg_len[id.k] = msg_total;
        }
    }
}

}  // namespace

// ----------------------------------------------------------------------------
// histogram passes: 11 + 11 + 9 bits of the 31-bit magnitude key
// ----------------------------------------------------------------------------

// The last workgroup of a pair after a histogram pass: reads and clears the
// pair's global histogram, picks the digit and updates the pair's state; pass
// 1 also sets the next step's candidate threshold.  h: [kBins] in LDS.
// The pair's global histogram gh into LDS h (nbins, a multiple of kGroup),
// clearing gh for the next step; all of a thread's loads in flight at once.
template <int nbins>
__device__ __forceinline__ void take_hist(uint32_t* h, uint32_t* gh) {
    constexpr int per = nbins / kGroup;
    uint32_t v[per];
#pragma unroll
    for (int i = 0; i < per; ++i) v[i] = load_agent(&gh[threadIdx.x + i * kGroup]);
#pragma unroll
    for (int i = 0; i < per; ++i) {
        h[threadIdx.x + i * kGroup] = v[i];
        store_agent(&gh[threadIdx.x + i * kGroup], 0u);
    }
    __syncthreads();
}

// take_hist for two histograms at once.
template <int nbins>
__device__ __forceinline__ void take_hist2(uint32_t* h, uint32_t* gh, uint32_t* h2, uint32_t* gh2) {
    constexpr int per = nbins / kGroup;
    uint32_t v[per], v2[per];
#pragma unroll
    for (int i = 0; i < per; ++i) {
        v[i] = load_agent(&gh[threadIdx.x + i * kGroup]);
        v2[i] = load_agent(&gh2[threadIdx.x + i * kGroup]);
    }
#pragma unroll
    for (int i = 0; i < per; ++i) {
        h[threadIdx.x + i * kGroup] = v[i];
        h2[threadIdx.x + i * kGroup] = v2[i];
        store_agent(&gh[threadIdx.x + i * kGroup], 0u);
        store_agent(&gh2[threadIdx.x + i * kGroup], 0u);
    }
    __syncthreads();
}

// ----------------------------------------------------------------------------
// first-step threshold from a sample
//
// A context's first step has no previous selection to place the speculative
// threshold with, so without one every pair would take the full-data path
// (three histogram passes and the emit, each over all of u).  Before that
// step's worker pass this kernel computes u, as the worker pass will, at a
// regular sample of each large segment (runs of kSeedRun consecutive
// components every kSeedStride: a sixteenth of the components, whole cache
// lines), and sets the pair's threshold at the floor of the 11-bit key bin
// holding the sample's key of rank about kSeedMult k |S| / n.  The worker
// pass then collects about that many candidates and the selection resolves
// from them.  The threshold only decides which components are candidates:
// the candidates still have to prove that they hold the top k (at least k of
// them, at most the capacity) or the pair takes the full-data path, so the
// results never depend on it.
// ----------------------------------------------------------------------------

__global__ __launch_bounds__(kGroup) void topk_seed_kernel(StepArgs a, TopkGeometry g, TopkScratch s) {
    static_assert(kSeedRunsPerGroup * kSeedRun == kGroup * 32, "32 sample components per thread");
    static_assert(kGroup % kSeedRun == 0 && kSeedRun <= kSeedStride, "whole runs per wave step");
    __shared__ uint32_t h[kBins];
    __shared__ uint32_t sh_wsum[kWavesPerGroup];
    __shared__ int sh_res[2];
    __shared__ int sh_last;
    const int k = blockIdx.x / g.n_seed_groups;
    const int2 sm = g.seed_map[blockIdx.x % g.n_seed_groups];
    const int seg = sm.x;
    const int p = k * g.n_seg + seg;
    PairState* ps = &s.pair[p];
    const int W = g.seg_seed_groups[seg];
    const int runs = g.seg_seed_runs[seg];
    const int run_hi = min(sm.y + kSeedRunsPerGroup, runs);
    const int64_t seg_lo = g.seg_start[seg];
    for (int b = threadIdx.x; b < kBins; b += kGroup) h[b] = 0u;
    __syncthreads();
    const float* e = a.wp.e[k];
    const float* gr = a.wp.g[k];
    const float c = a.c, hh = a.h;
    constexpr int kRunsPerStep = kGroup / kSeedRun;  // runs one pass of the workgroup covers
    constexpr int kUnroll = 8;
    for (int i0 = 0; i0 < 32; i0 += kUnroll) {
        float ev[kUnroll], gv[kUnroll], wt[kUnroll], wp[kUnroll];
        bool in[kUnroll];
#pragma unroll
        for (int u = 0; u < kUnroll; ++u) {
            const int run = sm.y + (i0 + u) * kRunsPerStep + (int)threadIdx.x / kSeedRun;
            in[u] = run < run_hi;
            const int64_t j = seg_lo + (int64_t)run * kSeedStride + (threadIdx.x % kSeedRun);
            ev[u] = gv[u] = wt[u] = wp[u] = 0.0f;
            if (in[u]) {
                ev[u] = e[j];
                gv[u] = gr[j];
                wt[u] = a.w_t[j];
                wp[u] = a.w_prev[j];
            }
        }
#pragma unroll
        for (int u = 0; u < kUnroll; ++u)
            if (in[u]) atomicAdd(&h[key_of(rule_u_rt(a.rule, ev[u], gv[u], wt[u], wp[u], c, hh)) >> kShift1], 1u);
    }
    __syncthreads();
    uint32_t* gh = s.hist + (size_t)p * kBins;
    const bool solo = W == 1;
    for (int b = threadIdx.x; !solo && b < kBins; b += kGroup)
        if (h[b]) atomicAdd(&gh[b], h[b]);
    if (!finish_slice(&ps->done, W, &sh_last)) return;
    if (!solo) take_hist<kBins>(h, gh);
    uint32_t above = 0;
    const int bin = find_bin(h, kBins, (uint32_t)g.seg_seed_rank[seg], &above, sh_wsum, sh_res);
    if (threadIdx.x == 0) {
        ps->tau = bin < 0 ? 0u : (uint32_t)bin << kShift1;  // fewer sampled than the rank: every component
        store_agent(&ps->done, 0u);
    }
}

hipError_t launch_topk_seed(const StepArgs& a, const TopkGeometry& g, const TopkScratch& s, hipStream_t st) {
    if (g.n_seed_groups == 0) return hipSuccess;
    hipLaunchKernelGGL(topk_seed_kernel, dim3(g.K * g.n_seed_groups), dim3(kGroup), 0, st, a, g, s);
    return hipGetLastError();
}

// margin: the speculative threshold's rank, in quarters of k.  h2/gh2: the
// second pass's histogram of the threshold's bin (PASS 2 only; gh2 holds it
// unless that bin is the one h covers).
template <int PASS>
__device__ void finish_digit(PairState* ps, int p, uint32_t* h, uint32_t* gh, int kp, int mode, uint32_t cand,
                             uint32_t prefix, int margin, int force_full, bool approx, const TopkGeometry& g,
                             const TopkScratch& s, uint32_t* sh_wsum, int* sh_res, uint32_t* h2 = nullptr,
                             uint32_t* gh2 = nullptr, uint32_t* T_out = nullptr, int32_t* r_out = nullptr,
                             bool solo = false) {
    constexpr int nbins = PASS == 3 ? 512 : kBins;
    // second pass: the threshold's bin histogram comes in with T's.  A pair
    // that one workgroup covered (solo) has its whole histogram in LDS
    // already and never wrote the global one.
    // the pair's fields this pick reads, loaded before the histogram is taken
    // (a load after take_hist would also wait for its clearing stores: vmcnt
    // counts in issue order)
    const uint32_t need = PASS == 1 ? (uint32_t)kp : (uint32_t)ps->need;
    const uint32_t tau_prev = PASS == 1 ? ps->tau : 0u;
    const uint32_t tau_fine = PASS == 2 ? ps->tau_fine : 0u;
    const uint32_t tau_bin = PASS == 2 ? ps->tau_bin : 0u;
    const uint32_t tau_need = PASS == 2 ? ps->tau_need : 0u;
    const uint32_t cand_used = PASS == 3 ? ps->cand_used : 0u;
    const uint32_t tau_used = PASS == 3 ? ps->tau_used : 0u;
    const bool fine2 = PASS == 2 && tau_fine != 0u && tau_bin != prefix;
    if (!solo) {
        if (fine2) take_hist2<kBins>(h, gh, h2, gh2);
        else take_hist<nbins>(h, gh);
    }
    uint32_t above = 0;
    const int bin = find_bin(h, nbins, need, &above, sh_wsum, sh_res);
    if (PASS == 3 && T_out) {  // every thread: the threshold and the ties to take
        *T_out = (prefix << 9) | (uint32_t)(bin < 0 ? 0 : bin);
        *r_out = (int32_t)(need - above);
    }

    if (PASS == 1) {
        // speculative threshold of the next step: the floor of the bin that
        // holds the key of rank margin*k/4 this step (the second pass of
        // exact top-s narrows it to 22 bits)
        const uint64_t want64 = ((uint64_t)margin * (uint64_t)kp + 3) / 4;
        uint32_t total, want, ab2 = 0;
        int tb;
        if (want64 == (uint64_t)need && bin >= 0) {
            // rank k itself (the default margin): T's bin, found above, in a
            // histogram of at least k keys
            total = want = need;
            ab2 = above;
            tb = bin;
        } else {
            uint32_t mine = 0;
            for (int b = threadIdx.x; b < nbins; b += kGroup) mine += h[b];
            block_scan_excl(mine, &total, sh_wsum);
            want = (uint32_t)(want64 < total ? want64 : total);
            tb = find_bin(h, nbins, want, &ab2, sh_wsum, sh_res);
        }
        if (threadIdx.x == 0) {
            const bool widen = want64 > total;
            if (widen && tb > 0) --tb;  // too few counted: widen by one bin
            if (tb < 0) tb = 0;
            ps->tau_used = tau_prev;
            ps->tau = (uint32_t)tb << kShift1;
            ps->tau_fine = (!approx && !widen) ? 1u : 0u;
            ps->tau_bin = (uint32_t)tb;
            ps->tau_need = want - ab2;
            ps->mode = mode;
            ps->cand_used = cand;
            if (!approx) {
                atomicAdd((unsigned long long*)&s.stats[mode == 0 ? 1 : 2], 1ull);
                if (mode == 0) atomicAdd((unsigned long long*)&s.stats[3], (unsigned long long)cand);
            }
        }
    }
    if (threadIdx.x == 0) {
        if (bin < 0) atomicAdd((unsigned long long*)&s.stats[4], 1ull);  // cannot happen for valid counts
        const uint32_t b = bin < 0 ? 0u : (uint32_t)bin;
        if (PASS == 1) {
            ps->prefix = b;
            ps->need = (int32_t)(need - above);
            // a full-data pair with few components at or above the digit's
            // bin: the second pass collects them for the third and the emit
            if (mode == 1 && !approx) {
                const int sg = p % g.n_seg;
                const int64_t n = g.seg_start[sg + 1] - g.seg_start[sg];
                if ((int64_t)above + (int64_t)h[b] <= n / kCollectDiv) ps->mode = kModeCollected;
            }
        } else if (PASS == 2) {
            ps->prefix = (prefix << 11) | b;
            ps->need = (int32_t)(need - above);
        } else {
            const uint32_t T = (prefix << 9) | b;
            ps->T = T;
            ps->r = (int32_t)(need - above);
            if (approx) {
                // keep every component at or above the sample's threshold;
                // the candidates hold them all when T reaches the threshold
                // the fused pass collected with and none were dropped
                ps->r = 0x7fffffff;
                const uint32_t cu = cand_used;
                const int m = (!force_full && T >= tau_used && cu <= (uint32_t)g.pair_cap[p]) ? 0 : 1;
                ps->mode = m;
                atomicAdd((unsigned long long*)&s.stats[m == 0 ? 1 : 2], 1ull);
                if (m == 0) atomicAdd((unsigned long long*)&s.stats[3], (unsigned long long)cu);
            }
        }
        if (PASS != 2) store_agent(&ps->done, 0u);
    }
    if (PASS == 2) {
        // the speculative threshold at the floor of the 22-bit bin holding
        // the key of rank margin*k/4: the tau_need-th key of bin tau_bin
        if (tau_fine) {
            const uint32_t tb = tau_bin, tn = tau_need;
            int sb = bin;  // the threshold at T's own rank in T's bin: the bin found above
            if (fine2 || tn != need) {
                uint32_t ab = 0;
                sb = find_bin(fine2 ? h2 : h, kBins, tn, &ab, sh_wsum, sh_res);
            }
            if (threadIdx.x == 0 && sb >= 0) ps->tau = (tb << kShift1) | ((uint32_t)sb << kShift2);
        }
        if (threadIdx.x == 0) store_agent(&ps->done, 0u);
    }
}

// The candidates the fused pass collected for pair (k, seg): the sum of its
// compaction groups' totals (grp_acc of the step's parity).
__device__ uint32_t pair_candidates(const StepArgs& a, const TopkGeometry& g, const TopkScratch& s, int k, int seg,
                                    uint32_t* sh_wsum) {
    const int g0 = g.seg_cgrp_lo[seg], ng = g.seg_cgrps[seg];
    uint32_t mine = 0;
    for (int r = threadIdx.x; r < ng; r += kGroup) mine += grp_total(s, g, a.t, k, g0 + r);
    uint32_t all;
    block_scan_excl(mine, &all, sh_wsum);
    return all;
}

// The third pass of exact top-s also takes the count of the kept components
// per slice: each workgroup stores its slice's count above T's 22-bit bin and
// the suffix sums of its 512-bin histogram of that bin (sl_hist, kSlHist
// words per slice), from which the last workgroup reads, once it has T, each
// slice's counts above and at T and lays out the message.
template <int PASS>
__device__ void hist_pass(const StepArgs& a, const TopkGeometry& g, const TopkScratch& s, int force_full,
                          int margin, int64_t* msg_len, int64_t msg_total, int blk) {
    constexpr int nbins = PASS == 3 ? 512 : kBins;
    __shared__ uint32_t h[kBins];
    __shared__ uint32_t h2[PASS == 2 ? kBins : 1];
    __shared__ uint32_t sh_wsum[kWavesPerGroup];
    __shared__ int sh_res[2];
    __shared__ int sh_last;
    __shared__ uint32_t carry[2];

    const SliceId id = slice_id(g, blk);
    PairState* ps = &s.pair[id.p];
    // sampled-threshold top-s: the passes select over the sample, rank samp_r
    const bool approx = g.approx != 0;
    const int kp = approx ? g.samp_r : g.pair_k[id.p];
    const uint32_t cand = PASS == 1 ? pair_candidates(a, g, s, id.k, id.seg, sh_wsum) : ps->cand_used;
    // the compaction copy takes the first pass of the exact top-s pairs that
    // resolve from their candidates
    if (PASS == 1 && !approx && !force_full && cand >= (uint32_t)kp && cand <= (uint32_t)g.pair_cap[id.p]) return;
    const int mode = approx      ? 2
                     : PASS == 1 ? ((force_full || cand < (uint32_t)kp || cand > (uint32_t)g.pair_cap[id.p]) ? 1 : 0)
                                 : ps->mode;
    const uint32_t prefix = PASS == 1 ? 0u : ps->prefix;
    // a candidate list is histogrammed in slices of about kHistSliceCands,
    // one round of loads per workgroup (each merges its slice's histogram
    // into the pair's with one global atomic per nonzero bin); the other
    // workgroups of the pair leave at once
    // the third pass of exact top-s counts per slice for the emit kernel, so
    // it keeps the emit's slices
    const bool count = PASS == 3 && !approx;
    const int W = (mode == 0 && !count) ? max(1, min(id.W, (int)((cand + kHistSliceCands - 1) / kHistSliceCands)))
                                        : id.W;
    if (id.w >= W) return;
    // second pass: also the second digit of the speculative threshold's bin
    // when it is not T's
    const uint32_t tbin = ps->tau_bin;
    const bool fine2 = PASS == 2 && ps->tau_fine != 0u && tbin != prefix;

    for (int b = threadIdx.x; b < nbins; b += kGroup) {
        h[b] = 0u;
        if (PASS == 2) h2[b] = 0u;
    }
    __syncthreads();
    const bool collected = mode == kModeCollected;
    const Slice v = open_slice(collected ? 1 : mode, cand, id.k, id.seg, id.p, id.w, W, a, g, s);
    uint32_t above = 0;  // third pass: keys above T's 22-bit bin
    auto body = [&](uint32_t key) {
        if (PASS == 1) {
            atomicAdd(&h[key >> kShift1], 1u);
        } else if (PASS == 2) {
            const uint32_t d1 = key >> kShift1;
            if (d1 == prefix) atomicAdd(&h[(key >> kShift2) & (kBins - 1)], 1u);
            else if (fine2 && d1 == tbin) atomicAdd(&h2[(key >> kShift2) & (kBins - 1)], 1u);
        } else {
            const uint32_t d12 = key >> kShift2;
            if (d12 == prefix) atomicAdd(&h[key & 511u], 1u);
            else if (count && d12 > prefix) ++above;
        }
    };
    if (PASS == 2 && collected) {
        // each wave streams its quarter of the slice, histograms it as above
        // and gathers, in index order, the components whose first digit is
        // at or above the prefix (all that the selection can keep) into its
        // run of the staging rows: ballots only, no workgroup barrier
        const int lane = threadIdx.x & (kWave - 1), wave = threadIdx.x >> 6;
        const uint64_t lt = lanemask_lt();
        const Slice run = collected_run(g, s, id.k, id.seg, id.w, W, 0);
        int32_t* ci = const_cast<int32_t*>(run.idx);
        float* cv = const_cast<float*>(run.val);
        const int64_t len = v.hi - v.lo;
        const int64_t ql = v.lo + len * wave / kWavesPerGroup, qh = v.lo + len * (wave + 1) / kWavesPerGroup;
        uint32_t cnt = 0;
        // one component per lane (the quarter's unaligned head and its tail)
        auto one = [&](int64_t pos, bool in) {
            const float x = in ? v.val[pos] : 0.0f;
            const uint32_t key = key_of(x);
            if (in) body(key);
            const bool take = in && (key >> kShift1) >= prefix;
            const uint64_t bal = ballot(take);
            if (take) {
                const int64_t o = ql + cnt + popc64(bal & lt);
                ci[o] = v.seg_lo + (int32_t)pos;
                cv[o] = x;
            }
            cnt += popc64(bal);
        };
        const int64_t mis = (int64_t)((reinterpret_cast<uintptr_t>(v.val + ql) >> 2) & 3u);
        const int64_t head = mis ? (4 - mis < qh - ql ? 4 - mis : qh - ql) : 0;
        one(ql + lane, lane < head);
        const int64_t lo4 = ql + head;
        const int64_t n4 = (qh - lo4) / 4;
        const float4* p4 = reinterpret_cast<const float4*>(v.val + lo4);
        // the body: float4 (i, lane) holds components lo4 + 4 (i * 64 + lane) + c,
        // index order i, lane, c
        for (int64_t b0 = 0; b0 < n4; b0 += (int64_t)kWave * kSliceLoads4) {
            float4 x[kSliceLoads4];
#pragma unroll
            for (int i = 0; i < kSliceLoads4; ++i) {
                const int64_t q = b0 + i * kWave + lane;
                x[i] = q < n4 ? p4[q] : make_float4(0.f, 0.f, 0.f, 0.f);
            }
#pragma unroll
            for (int i = 0; i < kSliceLoads4; ++i) {
                const int64_t q = b0 + i * kWave + lane;
                const bool in = q < n4;
                const float xs[4] = {x[i].x, x[i].y, x[i].z, x[i].w};
                uint32_t take = 0;
#pragma unroll
                for (int c = 0; c < 4; ++c) {
                    const uint32_t key = key_of(xs[c]);
                    if (in) body(key);
                    take |= (in && (key >> kShift1) >= prefix ? 1u : 0u) << c;
                }
                uint32_t tot;
                const uint32_t pre = wave_prefix_small((uint32_t)__popc(take), &tot);
                if (take) {
                    int64_t o = ql + cnt + pre;
                    const int64_t pos = lo4 + 4 * q;
#pragma unroll
                    for (int c = 0; c < 4; ++c) {
                        if ((take >> c) & 1u) {
                            ci[o] = v.seg_lo + (int32_t)(pos + c);
                            cv[o] = xs[c];
                            ++o;
                        }
                    }
                }
                cnt += tot;
            }
        }
        const int64_t t0 = lo4 + 4 * n4;
        one(t0 + lane, t0 + lane < qh);
        if (lane == 0)
            s.sl_run[((size_t)id.k * g.n_slices + g.seg_slice_lo[id.seg] + id.w) * kWavesPerGroup + wave] = cnt;
    } else if (PASS == 3 && collected) {
        for (int q = 0; q < kWavesPerGroup; ++q)
            for_slice<false>(collected_run(g, s, id.k, id.seg, id.w, W, q), [&](uint32_t key, int32_t) { body(key); });
    } else if (v.idx == nullptr) {
        for_slice_contig(v, body);
    } else {
        for_slice<false>(v, [&](uint32_t key, int32_t) { body(key); });
    }
    __syncthreads();
    uint32_t* gh = s.hist + (size_t)id.p * kBins;
    uint32_t* gh2 = s.hist2 + (size_t)id.p * kBins;
    const bool solo = W == 1;  // the pair's whole histogram is this workgroup's
    for (int b = threadIdx.x; !solo && b < nbins; b += kGroup) {
        if (h[b]) atomicAdd(&gh[b], h[b]);
        if (fine2 && h2[b]) atomicAdd(&gh2[b], h2[b]);
    }
    uint32_t* sh = nullptr;
    if (count) {
        // this slice's count above the bin and, for b < 512, S[b] = its keys
        // in the bin with low bits >= b (thread t owns bins 511-2t, 510-2t)
        sh = s.sl_hist + ((size_t)id.k * g.n_slices + g.seg_slice_lo[id.seg] + id.w) * kSlHist;
        uint32_t tot;
        block_scan_excl(above, &tot, sh_wsum);
        if (threadIdx.x == 0) store_agent(&sh[512], tot);
        const int b_hi = 511 - 2 * (int)threadIdx.x;
        const uint32_t hh = h[b_hi], hl = h[b_hi - 1];
        const uint32_t ex = block_scan_excl(hh + hl, &tot, sh_wsum);
        store_agent(&sh[b_hi], ex + hh);
        store_agent(&sh[b_hi - 1], ex + hh + hl);
    }
    if (!finish_slice(&ps->done, W, &sh_last)) return;

    uint32_t T = 0;
    int32_t r = 0;
    finish_digit<PASS>(ps, id.p, h, gh, kp, mode, cand, prefix, margin, force_full, approx, g, s, sh_wsum, sh_res,
                       PASS == 2 ? h2 : nullptr, gh2, &T, &r, solo);
    if (count) {
        // each slice's counts above T and at T: above the bin, plus S[b+1];
        // at T, S[b] - S[b+1] (b = T's low 9 bits)
        const uint32_t b = T & 511u;
        scan_slices(id, W, r, [&](size_t sl, uint32_t* A, uint32_t* Ti) {
            const uint32_t* S = s.sl_hist + sl * kSlHist;
            const uint32_t sb = load_agent(&S[b]), sb1 = b < 511u ? load_agent(&S[b + 1]) : 0u;
            *A = load_agent(&S[512]) + sb1;
            *Ti = sb - sb1;
        }, g, s, msg_len, msg_total, sh_wsum, carry);
    }
}

template <int PASS>
__global__ __launch_bounds__(kGroup) void topk_hist_kernel(StepArgs a, TopkGeometry g, TopkScratch s,
                                                           int force_full, int margin, int64_t* msg_len,
                                                           int64_t msg_total) {
    hist_pass<PASS>(a, g, s, force_full, margin, msg_len, msg_total, blockIdx.x);
}

hipError_t launch_topk_hist(int pass, const StepArgs& a, const TopkGeometry& g, const TopkScratch& s,
                            int force_full, int margin, int64_t* msg_len, int64_t msg_total, hipStream_t st) {
    const int grid = g.K * g.n_slices;
    if (pass != 2 && pass != 3) return hipErrorInvalidValue;  // pass 1 runs with the compaction copy
    if (pass == 2)
        hipLaunchKernelGGL(topk_hist_kernel<2>, dim3(grid), dim3(kGroup), 0, st, a, g, s, force_full, margin, msg_len,
                           msg_total);
    else
        hipLaunchKernelGGL(topk_hist_kernel<3>, dim3(grid), dim3(kGroup), 0, st, a, g, s, force_full, margin, msg_len,
                           msg_total);
    return hipGetLastError();
}

// ----------------------------------------------------------------------------
// compaction of the candidates
// ----------------------------------------------------------------------------

// The pair's candidates go, tile by tile (kTile candidates of one compaction
// group each, the groups in index order), to the pair's list, so the list
// comes out in ascending index order.  The tiles are laid out from the
// groups' totals (grp_acc): group r holds ceil(total_r / kTile) tiles, its
// candidates go to the list at the totals of the groups before it, and within
// the group each chunk's candidates at the counts of the chunks before it.
// Workgroup (worker, tile_map entry (seg, i)) takes the pair's tiles i, i +
// stride, ... (stride = the workgroups launched for the pair, sized for the
// usual count); the grid is tile-major, the K workers' entries consecutive.  For the pairs of exact top-s that resolve from their
// candidates the copy also histograms the first digit, and the last of the
// pair's workgroups picks it (the first histogram pass then skips the pair).
constexpr int kMaxCopyTiles = 256;  // tiles of one workgroup (at most about cap_mult / 8 + 2)

__device__ void compact_copy(const StepArgs& a, const TopkGeometry& g, const TopkScratch& s, int force_full, int margin,
                             int blk) {
    __shared__ uint32_t pre[kCompactChunks];
    __shared__ uint32_t h[kBins];
    __shared__ uint32_t sh_wsum[kWavesPerGroup];
    __shared__ int sh_res[2];
    __shared__ int sh_last;
    __shared__ uint32_t carry[2];
    __shared__ int32_t my_grp[kMaxCopyTiles];     // this workgroup's m-th tile: its group,
    __shared__ uint32_t my_base[kMaxCopyTiles];   // the group's first position in the list,
    __shared__ uint32_t my_tot[kMaxCopyTiles];    // the group's candidates,
    __shared__ uint32_t my_tile[kMaxCopyTiles];   // the tile within the group
    static_assert(kCompactChunks == kGroup, "one chunk per thread");
    // tile-major: the K workers' i-th tiles are consecutive workgroups, so
    // the tiles that hold candidates (the first ones of every pair) are
    // dispatched first and the spare ones after them
    const int k = blk % g.K;
    const int2 tm = g.tile_map[blk / g.K];
    const int seg = tm.x;
    const int p = k * g.n_seg + seg;
    PairState* ps = &s.pair[p];
    const uint32_t i0 = (uint32_t)tm.y;
    const uint32_t stride = (uint32_t)g.seg_tile_stride[seg];
    // the pair's groups: totals, list bases and tiles, in blocks of kGroup
    const int g0 = g.seg_cgrp_lo[seg], ng = g.seg_cgrps[seg];
    if (threadIdx.x == 0) {
        carry[0] = 0u;  // candidates before the block
        carry[1] = 0u;  // tiles before the block
    }
    __syncthreads();
    for (int r0 = 0; r0 < ng; r0 += kGroup) {
        const int r = r0 + (int)threadIdx.x;
        const uint32_t tot = r < ng ? grp_total(s, g, a.t, k, g0 + r) : 0u;
        const uint32_t nt = (tot + kTile - 1) / kTile;
        uint32_t bt, btt;
        const uint32_t base = carry[0] + block_scan_excl(tot, &bt, sh_wsum);
        const uint32_t tp = carry[1] + block_scan_excl(nt, &btt, sh_wsum);
        // this workgroup's tiles i0 + m stride that fall in [tp, tp + nt)
        if (nt) {
            uint32_t tt = i0 >= tp ? i0 : i0 + (tp - i0 + stride - 1) / stride * stride;
            for (; tt < tp + nt; tt += stride) {
                const uint32_t m = (tt - i0) / stride;
                if (m < (uint32_t)kMaxCopyTiles) {
                    my_grp[m] = g0 + r;
                    my_base[m] = base;
                    my_tot[m] = tot;
                    my_tile[m] = tt - tp;
                }
            }
        }
        __syncthreads();
        if (threadIdx.x == 0) {
            carry[0] += bt;
            carry[1] += btt;
        }
        __syncthreads();
    }
    const uint32_t all = carry[0];
    const bool copy = all <= (uint32_t)g.pair_cap[p];
    const uint32_t n_tiles = copy ? carry[1] : 0u;
    if (i0 >= n_tiles) return;
    const uint32_t n_wg = n_tiles < stride ? n_tiles : stride;  // workgroups of the pair with tiles
    const uint32_t n_my = (n_tiles - i0 + stride - 1) / stride;
    const bool fuse = !g.approx && !force_full && all >= (uint32_t)g.pair_k[p];
    if (fuse)
        for (int b = threadIdx.x; b < kBins; b += kGroup) h[b] = 0u;
    int32_t* ci0 = s.cand_idx + g.pair_cand[p];
    float* cv0 = s.cand_val + g.pair_cand[p];
    for (uint32_t m = 0; m < n_my && m < (uint32_t)kMaxCopyTiles; ++m) {
        const int cg = my_grp[m];
        const int clo = g.cgrp_lo[cg], nch = g.cgrp_hi[cg] - clo;
        const uint32_t base = my_base[m];
        const size_t slot0 = (size_t)k * g.n_chunks + clo;
        // each chunk's first position within the group
        const uint32_t cnt = (int)threadIdx.x < nch ? s.run_cnt[slot0 + threadIdx.x] : 0u;
        uint32_t gt;
        const uint32_t cpre = block_scan_excl(cnt, &gt, sh_wsum);
        if ((int)threadIdx.x < nch) pre[threadIdx.x] = cpre;
        __syncthreads();
        // the group's candidates are its chunks' runs (equal to its total,
        // which only decided the layout)
        const uint32_t total = my_tot[m] < gt ? my_tot[m] : gt;
        const uint32_t lo = my_tile[m] * kTile;
        const uint32_t hi = lo + kTile < total ? lo + kTile : total;
        int32_t* ci = ci0 + base;
        float* cv = cv0 + base;
        // the eight loads of a thread go out together: no load sits under a
        // per-element branch (a position past the tile's end reads the
        // tile's first candidate, and its value is dropped)
        int32_t jv[8];
        float xv[8];
        if (lo < hi) {
            uint32_t q[8];
            int a0[8];  // the chunk c with pre[c] <= q < pre[c+1]: the last c with pre[c] <= q
#pragma unroll
            for (int i = 0; i < 8; ++i) {
                const uint32_t q0 = lo + i * kGroup + threadIdx.x;
                q[i] = q0 < hi ? q0 : lo;
                a0[i] = 0;
            }
            // the eight searches step by step: eight LDS reads per step
#pragma unroll
            for (int st = kCompactChunks / 2; st > 0; st >>= 1) {
#pragma unroll
                for (int i = 0; i < 8; ++i) {
                    const int c = a0[i] + st < nch ? a0[i] + st : nch - 1;
                    a0[i] = (a0[i] + st < nch && pre[c] <= q[i]) ? a0[i] + st : a0[i];
                }
            }
#pragma unroll
            for (int i = 0; i < 8; ++i) {
                const int2 c = s.slot[(slot0 + a0[i]) * kChunk + (q[i] - pre[a0[i]])];
                jv[i] = c.x;
                xv[i] = __int_as_float(c.y);
            }
        }
#pragma unroll
        for (int i = 0; i < 8; ++i) {
            const uint32_t q = lo + i * kGroup + threadIdx.x;
            if (q < hi) {
                ci[q] = jv[i];
                cv[q] = xv[i];
                if (fuse) atomicAdd(&h[key_of(xv[i]) >> kShift1], 1u);
            }
        }
        __syncthreads();  // the searches are done with pre before the next tile's scan
    }
    if (!fuse) return;
    __syncthreads();
    uint32_t* gh = s.hist + (size_t)p * kBins;
    const bool solo = n_wg == 1;  // the pair's whole histogram is this workgroup's
    for (int b = threadIdx.x; !solo && b < kBins; b += kGroup)
        if (h[b]) atomicAdd(&gh[b], h[b]);
    if (!finish_slice(&ps->done, (int)n_wg, &sh_last)) return;
    finish_digit<1>(ps, p, h, gh, g.pair_k[p], 0, all, 0u, margin, 0, false, g, s, sh_wsum, sh_res, nullptr,
                    nullptr, nullptr, nullptr, solo);
}

// The copy and the first histogram pass in one launch: the first
// K * tiles_per_worker workgroups copy (with the first pass of the pairs that
// resolve from their candidates), the K * n_slices after them take the first
// pass of the others (full data, or the sample of the sampled-threshold
// top-s); both decide which pairs those are from the groups' totals.
__global__ __launch_bounds__(kGroup) void topk_copy_pass1_kernel(StepArgs a, TopkGeometry g, TopkScratch s,
                                                                 int force_full, int margin) {
    const int n_copy = g.K * g.tiles_per_worker;
    if ((int)blockIdx.x < n_copy)
        compact_copy(a, g, s, force_full, margin, blockIdx.x);
    else
        hist_pass<1>(a, g, s, force_full, margin, nullptr, 0, (int)blockIdx.x - n_copy);
}

hipError_t launch_topk_compact(const StepArgs& a, const TopkGeometry& g, const TopkScratch& s, int force_full,
                               int margin, hipStream_t st) {
    const int64_t grid = (int64_t)g.K * g.tiles_per_worker + (int64_t)g.K * g.n_slices;
    hipLaunchKernelGGL(topk_copy_pass1_kernel, dim3((unsigned)grid), dim3(kGroup), 0, st, a, g, s, force_full, margin);
    return hipGetLastError();
}

// ----------------------------------------------------------------------------
// per-slice counts above / at the threshold, then the scan over the slices
// ----------------------------------------------------------------------------

__global__ __launch_bounds__(kGroup) void topk_count_kernel(StepArgs a, TopkGeometry g, TopkScratch s,
                                                            int64_t* msg_len, int64_t msg_total) {
    __shared__ uint32_t red[2][kWavesPerGroup];
    __shared__ uint32_t sh_wsum[kWavesPerGroup];
    __shared__ int sh_last;
    __shared__ uint32_t carry[2];

    const SliceId id = slice_id(g, blockIdx.x);
    PairState* ps = &s.pair[id.p];
    const int mode = ps->mode;
    const uint32_t T = ps->T;
    const Slice v = open_slice(mode, ps->cand_used, id.k, id.seg, id.p, id.w, id.W, a, g, s);
    uint32_t above = 0, ties = 0;
    auto tally = [&](uint32_t key) {
        above += key > T;
        ties += key == T;
    };
    if (v.idx == nullptr) for_slice_contig(v, tally);
    else for_slice<false>(v, [&](uint32_t key, int32_t) { tally(key); });
    for (int o = kWave / 2; o > 0; o >>= 1) {
        above += __shfl_down(above, o, kWave);
        ties += __shfl_down(ties, o, kWave);
    }
    const int lane = threadIdx.x & (kWave - 1), wave = threadIdx.x >> 6;
    if (lane == 0) {
        red[0][wave] = above;
        red[1][wave] = ties;
    }
    __syncthreads();
    const size_t base = (size_t)id.k * g.n_slices + g.seg_slice_lo[id.seg];
    if (threadIdx.x == 0) {
        uint32_t A = 0, Ti = 0;
        for (int w = 0; w < kWavesPerGroup; ++w) {
            A += red[0][w];
            Ti += red[1][w];
        }
        store_agent(&s.sl_above[base + id.w], A);
        store_agent(&s.sl_ties[base + id.w], Ti);
    }
    if (!finish_slice(&ps->done, id.W, &sh_last)) return;

    // last workgroup of the pair: scan the segment's slices in index order
    scan_slices(id, id.W, ps->r, [&](size_t sl, uint32_t* A, uint32_t* Ti) {
        *A = load_agent(&s.sl_above[sl]);
        *Ti = load_agent(&s.sl_ties[sl]);
    }, g, s, msg_len, msg_total, sh_wsum, carry);
    if (threadIdx.x == 0) store_agent(&ps->done, 0u);
}

hipError_t launch_topk_count(const StepArgs& a, const TopkGeometry& g, const TopkScratch& s,
                             int64_t* msg_len, int64_t msg_total, hipStream_t st) {
    hipLaunchKernelGGL(topk_count_kernel, dim3(g.K * g.n_slices), dim3(kGroup), 0, st, a, g, s, msg_len,
                       msg_total);
    return hipGetLastError();
}

// ----------------------------------------------------------------------------
// ordered emission of the kept components
//
// One workgroup per slice.  The slice's elements are staged in LDS in rounds
// of kEmitStage (coalesced loads, all in flight together); in a round each
// thread owns kEmitLoads consecutive elements, one block-wide scan of its
// (above, tie) counts places them, and the thread writes its kept ones in
// order.  LDS rows are padded by one word per 4 entries, so consecutive
// threads' rows start an odd number of words apart and their strided reads
// hit distinct banks.
// ----------------------------------------------------------------------------

__device__ __forceinline__ int stage_slot(int q) { return q + (q >> 2); }

__global__ __launch_bounds__(kGroup) void topk_emit_kernel(StepArgs a, TopkGeometry g, TopkScratch s,
                                                           int32_t* idx, float* val, int64_t row_len) {
    static_assert(kEmitLoads % 4 == 0 && (kEmitLoads + kEmitLoads / 4) % 2 == 1,
                  "one pad word per 4 entries; each thread's row then starts an odd number of words on");
    constexpr int kStageSlots = kEmitStage + kEmitStage / 4;
    __shared__ union {
        struct {  // candidate path: the staged round
            int32_t idx[kStageSlots];
            float val[kStageSlots];
        } st;
        struct {  // full-data path: the round's (i, wave) counts and its values
            uint32_t cnt[2 * kWave + 1];
            float x[kFullRound];
        } full;
    } lds;
    int32_t* const st_idx = lds.st.idx;
    float* const st_val = lds.st.val;
    __shared__ uint32_t sh_wsum[kWavesPerGroup];

    // this step's group totals have been read (the copy and the first pass):
    // clear them for the step after next, which adds into the same half
    {
        const size_t nz = (size_t)kGrpSub * g.K * g.n_cgroups;
        uint32_t* z = s.grp_acc + (size_t)(a.t & 1) * nz;
        for (size_t i = (size_t)blockIdx.x * kGroup + threadIdx.x; i < nz; i += (size_t)gridDim.x * kGroup) z[i] = 0u;
    }
    const SliceId id = slice_id(g, blockIdx.x);
    const PairState* ps = &s.pair[id.p];
    const int mode = ps->mode;
    const uint32_t T = ps->T;
    const int64_t r = ps->r;
    const size_t sl = (size_t)id.k * g.n_slices + g.seg_slice_lo[id.seg] + id.w;
    const uint32_t out0 = s.sl_out[sl];
    int64_t quota = r - (int64_t)s.sl_tiebase[sl];  // ties this slice may still take, in index order
    if (quota < 0) quota = 0;
    // capacity of the segment's part of the row: k (top-s) or the whole
    // segment (sampled threshold)
    const uint32_t kseg = g.approx ? (uint32_t)(g.seg_start[id.seg + 1] - g.seg_start[id.seg])
                                   : (uint32_t)g.pair_k[id.p];
    int32_t* irow = idx + (size_t)id.k * row_len + g.seg_out[id.seg];
    float* vrow = val + (size_t)id.k * row_len + g.seg_out[id.seg];
    float* e = a.wp.e[id.k];

    // a collected pair's slice spans the full-data slice; its input is the
    // four runs the second pass gathered
    const bool collected = mode == kModeCollected;
    const Slice v = open_slice(collected ? 1 : mode, ps->cand_used, id.k, id.seg, id.p, id.w, id.W, a, g, s);
    // The server pass's row pointers: the slices' index spans [B(w), B(w+1))
    // tile the segment (B(0) its start, B(W) its end, B(w) the index of the
    // slice's first element), so each range start r*R of the segment lies in
    // one span, and there it is the row position of the first kept component
    // at or after it: this slice's first position plus its kept components
    // with a lower index.
    const int64_t seg_lo = g.seg_start[id.seg], seg_hi = g.seg_start[id.seg + 1];
    const int64_t in_total = mode == 0 ? (int64_t)ps->cand_used : seg_hi - seg_lo;
    auto index_at = [&](int64_t pos) -> int64_t {
        return pos < in_total ? (v.idx ? (int64_t)v.idx[pos] : seg_lo + pos) : seg_hi;
    };
    const int64_t span_lo = id.w == 0 ? seg_lo : index_at(v.lo);
    const int64_t span_hi = id.w == id.W - 1 ? seg_hi : index_at(v.hi);
    const int32_t row0 = g.seg_out[id.seg] + (int32_t)out0;  // this slice's first row position
    int32_t* rp = s.rowptr + (size_t)id.k * (s.n_ranges + 1);
    constexpr int64_t R = kAggTopkRange;
    int64_t prev_last = span_lo - 1;  // the index before the round's first element
    uint32_t run_above = 0, run_ties = 0;  // over the earlier rounds
    if (mode == 1) {
        // Full data: the slice is a run of consecutive components of which
        // few are kept, so it is streamed in rounds of kFullRound (coalesced
        // loads, 16 per thread in flight) and only the kept components are
        // placed: element (i, wave, lane) of a round has index order
        // i-major, then wave, then lane, and its rank among the round's kept
        // components comes from ballots and one scan of the 64 (i, wave)
        // counts.  A range start at element j (j a multiple of R) gets the
        // row position of the first kept component at or after it.
        constexpr int kIt = kFullRound / kGroup;  // 16
        static_assert(kIt * kWavesPerGroup == kWave, "one (i, wave) count per lane of the scanning wave");
        const int lane = threadIdx.x & (kWave - 1), wave = threadIdx.x >> 6;
        const uint64_t lt = lanemask_lt();
        uint32_t* cnt = lds.full.cnt;  // [kIt][kWavesPerGroup]: above << 16 | ties
        float* xs = lds.full.x;        // the round's values, element (i, thread) at i * kGroup + thread
        // the next round's loads are issued as soon as the current round's
        // values are counted and parked in LDS, so they are in flight during
        // the current round's scan and placement
        float x[kIt];
        auto load_round = [&](int64_t s0) {
#pragma unroll
            for (int i = 0; i < kIt; ++i) {
                const int64_t q = s0 + i * kGroup + threadIdx.x;
                x[i] = q < v.hi ? v.val[q] : 0.0f;
            }
        };
        if (v.lo < v.hi) load_round(v.lo);
        for (int64_t s0 = v.lo; s0 < v.hi; s0 += kFullRound) {
#pragma unroll
            for (int i = 0; i < kIt; ++i) {
                const bool in = s0 + i * kGroup + threadIdx.x < v.hi;
                const uint32_t key = key_of(x[i]);
                const uint64_t ba = ballot(in && key > T), bt = ballot(in && key == T);
                if (lane == 0) cnt[i * kWavesPerGroup + wave] = (popc64(ba) << 16) | popc64(bt);
                xs[i * kGroup + threadIdx.x] = x[i];
            }
            if (s0 + kFullRound < v.hi) load_round(s0 + kFullRound);
            __syncthreads();
            if (wave == 0) {  // exclusive scan of the 64 counts in index order, and the round's total
                const uint32_t c = cnt[lane];
                uint32_t incl = c;
#pragma unroll
                for (int o = 1; o < kWave; o <<= 1) {
                    const uint32_t y = __shfl_up(incl, o, kWave);
                    if (lane >= o) incl += y;
                }
                cnt[kWave + lane] = incl - c;
                if (lane == kWave - 1) cnt[2 * kWave] = incl;
            }
            __syncthreads();
#pragma unroll
            for (int i = 0; i < kIt; ++i) {
                const int64_t q = s0 + i * kGroup + threadIdx.x;
                const float xi = xs[i * kGroup + threadIdx.x];
                const uint32_t key = key_of(xi);
                const bool in = q < v.hi;
                const uint64_t ba = ballot(in && key > T), bt = ballot(in && key == T);
                const uint32_t pre = cnt[kWave + i * kWavesPerGroup + wave];
                const uint32_t a_before = run_above + (pre >> 16) + popc64(ba & lt);
                const uint32_t t_before = run_ties + (pre & 0xffffu) + popc64(bt & lt);
                const int64_t j = seg_lo + q;
                const int64_t tk = (int64_t)t_before < quota ? (int64_t)t_before : quota;
                if (q < v.hi && (j & (R - 1)) == 0) rp[j / R] = row0 + (int32_t)(a_before + (uint32_t)tk);
                const bool above = (ba >> lane) & 1ull, tie = (bt >> lane) & 1ull;
                if (above || (tie && (int64_t)t_before < quota)) {
                    const uint32_t o = out0 + a_before + (uint32_t)tk;
                    if (o < kseg) {  // always, when the counts are consistent
                        irow[o] = (int32_t)j;
                        vrow[o] = xi;
                        if (!a.defer_zero) e[j] = xi - xi;  // residual u - C(u) at a kept component
                    }
                }
            }
            const uint32_t tot = cnt[2 * kWave];
            run_above += tot >> 16;
            run_ties += tot & 0xffffu;
            __syncthreads();  // the counts and values are read before the next round writes them
        }
        if (v.hi > v.lo) prev_last = seg_lo + v.hi - 1;
    }
    // the candidates (or a collected slice's runs), staged in rounds
    auto emit_list = [&](const Slice& vl) {
    for (int64_t s0 = vl.lo; s0 < vl.hi; s0 += kEmitStage) {
        const int32_t ns = (int32_t)(vl.hi - s0 < kEmitStage ? vl.hi - s0 : kEmitStage);
        // all of a thread's loads go out before the first is stored: a
        // position past the round's end reads the round's first element
        // (dropped), so no load sits under a per-element branch
        float xl[kEmitLoads];
        int32_t jl[kEmitLoads];
        if (vl.idx) {
#pragma unroll
            for (int i = 0; i < kEmitLoads; ++i) {
                const int32_t q = i * kGroup + threadIdx.x;
                const int64_t pos = s0 + (q < ns ? q : 0);
                xl[i] = vl.val[pos];
                jl[i] = vl.idx[pos];
            }
        } else {
#pragma unroll
            for (int i = 0; i < kEmitLoads; ++i) {
                const int32_t q = i * kGroup + threadIdx.x;
                const int64_t pos = s0 + (q < ns ? q : 0);
                xl[i] = vl.val[pos];
                jl[i] = vl.seg_lo + (int32_t)pos;
            }
        }
#pragma unroll
        for (int i = 0; i < kEmitLoads; ++i) {
            const int32_t q = i * kGroup + threadIdx.x;
            if (q < ns) {
                st_val[stage_slot(q)] = xl[i];
                st_idx[stage_slot(q)] = jl[i];
            }
        }
        __syncthreads();
        const int32_t q0 = threadIdx.x * kEmitLoads;
        uint32_t na = 0, nt = 0;
#pragma unroll
        for (int i = 0; i < kEmitLoads; ++i) {
            if (q0 + i < ns) {
                const uint32_t key = key_of(st_val[stage_slot(q0 + i)]);
                na += key > T;
                nt += key == T;
            }
        }
        uint32_t tot;
        const uint32_t pre = block_scan_excl((na << 16) | nt, &tot, sh_wsum);  // counts < 2^16
        uint32_t a_before = run_above + (pre >> 16), t_before = run_ties + (pre & 0xffffu);
        int32_t kbv[kEmitLoads];  // kept components of the slice before each element
#pragma unroll
        for (int i = 0; i < kEmitLoads; ++i) {
            kbv[i] = 0;
            if (q0 + i >= ns) continue;
            const float x = st_val[stage_slot(q0 + i)];
            const uint32_t key = key_of(x);
            kbv[i] = (int32_t)(a_before + (uint32_t)((int64_t)t_before < quota ? (int64_t)t_before : quota));
            bool take = false;
            uint32_t o = 0;
            if (key > T) {
                take = true;
                o = out0 + a_before + (uint32_t)((int64_t)t_before < quota ? (int64_t)t_before : quota);
                ++a_before;
            } else if (key == T) {
                take = (int64_t)t_before < quota;
                o = out0 + a_before + t_before;
                ++t_before;
            }
            if (take && o < kseg) {  // o < kseg always holds when the counts are consistent
                const int32_t j = st_idx[stage_slot(q0 + i)];
                irow[o] = j;
                vrow[o] = x;
                if (!a.defer_zero) e[j] = x - x;  // residual u - C(u) at a kept component
            }
        }
        run_above += tot >> 16;
        run_ties += tot & 0xffffu;
        // row pointers of the range starts in (prev_last, the round's last
        // index]: the row position of the round's first element at or after
        // each, all threads sharing the range starts.  A thread's range
        // starts ascend, so each answer is at or after its previous one, and
        // where the indices leave a gap (clustered candidates: thousands of
        // range starts between two kept components) it is that one: one LDS
        // read, else a binary search over the staged indices after it.
        __syncthreads();  // the round's values are read; the stage now holds the counts
        int32_t* st_kb = reinterpret_cast<int32_t*>(st_val);
#pragma unroll
        for (int i = 0; i < kEmitLoads; ++i)
            if (q0 + i < ns) st_kb[stage_slot(q0 + i)] = kbv[i];
        __syncthreads();
        const int64_t j_end = st_idx[stage_slot(ns - 1)];
        int32_t found = 0;  // the answer for this thread's previous range start
        for (int64_t rr = (prev_last + R) / R + threadIdx.x; rr * R <= j_end; rr += kGroup) {
            const int64_t start = rr * R;
            // the first element whose index is >= start (the last one is)
            if ((int64_t)st_idx[stage_slot(found)] < start) {
                int32_t lo = found + 1, hi = ns - 1;
                while (lo < hi) {
                    const int32_t mid = (lo + hi) >> 1;
                    if ((int64_t)st_idx[stage_slot(mid)] < start) lo = mid + 1; else hi = mid;
                }
                found = lo;
            }
            rp[rr] = row0 + st_kb[stage_slot(found)];
        }
        prev_last = j_end;
        __syncthreads();  // the stage is read before the next round overwrites it
    }
    };
    if (collected) {
        for (int q = 0; q < kWavesPerGroup; ++q) emit_list(collected_run(g, s, id.k, id.seg, id.w, id.W, q));
    } else if (mode != 1) {
        emit_list(v);
    }
    // range starts after the slice's last element, up to the span's end
    const int32_t kept = (int32_t)(run_above + (uint32_t)((int64_t)run_ties < quota ? (int64_t)run_ties : quota));
    for (int64_t rr = (prev_last + R) / R + threadIdx.x; rr * R < span_hi; rr += kGroup) rp[rr] = row0 + kept;
    if (threadIdx.x == 0 && id.seg == g.n_seg - 1 && id.w == id.W - 1) rp[s.n_ranges] = row0 + kept;  // the row's length
}

hipError_t launch_topk_emit(const StepArgs& a, const TopkGeometry& g, const TopkScratch& s,
                            int32_t* idx, float* val, int64_t row_len, hipStream_t st) {
    hipLaunchKernelGGL(topk_emit_kernel, dim3(g.K * g.n_slices), dim3(kGroup), 0, st, a, g, s, idx, val,
                       row_len);
    return hipGetLastError();
}

// ============================================================================
// RBGS: block draw shared by all workers, fused gather pass
// ============================================================================

namespace {

constexpr int kLdsBitmapWords = 8192;  // 262144 blocks

}  // namespace

// One workgroup.  Floyd's algorithm (one lane; the draws are sequential by
// definition) marks n_sel of nb blocks in a bitmap; the workgroup then
// compacts the bitmap into the ascending block list and the block -> slot map.
// It also keeps the previous step's block list (prev) and lays out the ranges
// of kAggRange components a sparse server pass must visit (visit, meta[0]):
// those of this step's blocks and the previous step's, ascending, or every
// range (meta[0] = -1) when the last server pass raised meta[1] (a non-finite
// w outside the sent blocks, which stays marked).
__global__ __launch_bounds__(kGroup) void rbgs_sample_kernel(uint64_t seed, uint64_t t, int32_t nb,
                                                             int32_t n_sel, int32_t d, int32_t B,
                                                             int32_t K, uint32_t* gbitmap,
                                                             int32_t* blocks, int32_t* block_slot,
                                                             int32_t* idx, int64_t idx_row,
                                                             int64_t* msg_len, int32_t* prev, int32_t* visit,
                                                             uint32_t* grbits, int32_t* meta) {
    __shared__ uint32_t lbits[kLdsBitmapWords];
    __shared__ uint32_t wsum[kWavesPerGroup];
    __shared__ uint32_t carry;
    __shared__ int32_t sh_nf;
    for (int i = threadIdx.x; i < n_sel; i += kGroup) prev[i] = blocks[i];
    if (threadIdx.x == 0) sh_nf = meta[1];
    __syncthreads();  // the old list is read before it is rewritten
    const int nwords = (nb + 31) / 32;
    uint32_t* bits = nwords <= kLdsBitmapWords ? lbits : gbitmap;
    for (int w = threadIdx.x; w < nwords; w += kGroup) bits[w] = 0u;
    __threadfence_block();
    __syncthreads();
    if (threadIdx.x == 0) {
        const uint64_t gamma = 0x9e3779b97f4a7c15ull;
        const uint64_t state = seed ^ splitmix64_mix(t + 1);
        const int64_t J0 = (int64_t)nb - n_sel;
        for (int64_t J = J0; J < nb; ++J) {
            const uint64_t x = splitmix64_mix(state + (uint64_t)(J - J0 + 1) * gamma);
            const uint32_t r = (uint32_t)(((x >> 32) * (uint64_t)(J + 1)) >> 32);
            const bool have = (bits[r >> 5] >> (r & 31)) & 1u;
            const uint32_t pick = have ? (uint32_t)J : r;
            bits[pick >> 5] |= 1u << (pick & 31);
        }
        carry = 0;
    }
    __threadfence_block();
    __syncthreads();
    for (int w0 = 0; w0 < nwords; w0 += kGroup) {
        const int w = w0 + threadIdx.x;
        const uint32_t word = w < nwords ? bits[w] : 0u;
        uint32_t tot;
        uint32_t pos = carry + block_scan_excl((uint32_t)__popc(word), &tot, wsum);
        if (w < nwords) {
            for (int bb = 0; bb < 32; ++bb) {
                const int b = w * 32 + bb;
                if (b >= nb) break;
                if ((word >> bb) & 1u) {
                    blocks[pos] = b;
                    block_slot[b] = (int32_t)pos;
                    ++pos;
                } else {
                    block_slot[b] = -1;
                }
            }
        }
        __syncthreads();
        if (threadIdx.x == 0) carry += tot;
        __syncthreads();
    }
    __threadfence_block();
    __syncthreads();
    // message length: all selected blocks are full except possibly block nb-1
    const int32_t last = blocks[n_sel - 1];
    const int64_t last_len = (int64_t)d - (int64_t)last * B < B ? (int64_t)d - (int64_t)last * B : B;
    const int64_t m = (int64_t)(n_sel - 1) * B + last_len;
    for (int i = threadIdx.x; i < K * n_sel; i += kGroup) {
        const int kk = i / n_sel, q = i % n_sel;
        idx[(size_t)kk * idx_row + q] = blocks[q];
    }
    for (int kk = threadIdx.x; kk < K; kk += kGroup) msg_len[kk] = m;
    if (bits == gbitmap)
        for (int w = threadIdx.x; w < nwords; w += kGroup) gbitmap[w] = 0u;

    // the sparse server pass's ranges
    const int32_t n_ranges = (int32_t)(((int64_t)d + kAggRange - 1) / kAggRange);
    if (sh_nf) {
        if (threadIdx.x == 0) {
            meta[0] = -1;
            meta[1] = 0;
        }
        return;
    }
    const int rwords = (n_ranges + 31) / 32;
    const bool in_lds = rwords <= kLdsBitmapWords;
    uint32_t* rb = in_lds ? lbits : grbits;
    __syncthreads();  // every thread is done with the block bitmap
    if (in_lds)
        for (int w = threadIdx.x; w < rwords; w += kGroup) lbits[w] = 0u;
    __syncthreads();
    for (int i = threadIdx.x; i < 2 * n_sel; i += kGroup) {
        const int64_t b = i < n_sel ? blocks[i] : prev[i - n_sel];
        const int64_t lo = b * B, hi = (b + 1) * B < d ? (b + 1) * B : d;
        for (int64_t r = lo / kAggRange; r <= (hi - 1) / kAggRange; ++r) atomicOr(&rb[r >> 5], 1u << (r & 31));
    }
    if (!in_lds) __threadfence();  // the global bitmap's atomics are visible to the loads below
    __syncthreads();
    if (threadIdx.x == 0) carry = 0;
    __syncthreads();
    for (int w0 = 0; w0 < rwords; w0 += kGroup) {
        const int w = w0 + threadIdx.x;
        const uint32_t word = w < rwords ? (in_lds ? rb[w] : load_agent(&rb[w])) : 0u;
        uint32_t tot;
        uint32_t pos = carry + block_scan_excl((uint32_t)__popc(word), &tot, wsum);
        for (int bb = 0; bb < 32; ++bb)
            if ((word >> bb) & 1u) visit[pos++] = w * 32 + bb;
        if (!in_lds && w < rwords) store_agent(&rb[w], 0u);  // clear for the next step
        __syncthreads();
        if (threadIdx.x == 0) carry += tot;
        __syncthreads();
    }
    if (threadIdx.x == 0) meta[0] = (int32_t)carry;
}

hipError_t launch_rbgs_sample(uint64_t seed, uint64_t t, int32_t nb, int32_t n_sel, int32_t d,
                              int32_t B, int32_t K, uint32_t* bitmap, int32_t* blocks,
                              int32_t* block_slot, int32_t* idx, int64_t idx_row,
                              int64_t* msg_len, int32_t* prev, int32_t* visit, uint32_t* rbits, int32_t* meta,
                              hipStream_t st) {
    hipLaunchKernelGGL(rbgs_sample_kernel, dim3(1), dim3(kGroup), 0, st, seed, t, nb, n_sel, d, B, K,
                       bitmap, blocks, block_slot, idx, idx_row, msg_len, prev, visit, rbits, meta);
    return hipGetLastError();
}

// Each thread owns 4 consecutive elements per iteration; a selected block's
// components are copied to the message at slot*B + offset (every selected
// block but the last is full, so this is the concatenation in block order).
__global__ __launch_bounds__(kGroup) void rbgs_fused_kernel(StepArgs a, int32_t K, int32_t B,
                                                            const int32_t* block_slot, float* val,
                                                            int64_t val_row, int64_t j_begin,
                                                            uint64_t vec_mask, int64_t vec_end) {
    const int32_t d = a.d;
    const int64_t j0 = j_begin + ((int64_t)blockIdx.x * kGroup + threadIdx.x) * 4;
    if (j0 >= d) return;
    // workers in vec_mask had [0, vec_end) done by the vector kernel
    const uint64_t skip = j0 < vec_end ? vec_mask : 0ull;
    const float c = a.c, h = a.h, qd = a.q;
    const int rule = a.rule;
    const bool full = j0 + 4 <= d;
    const bool vec = full && (B & 3) == 0 && aligned16(a.w_t) && aligned16(a.w_prev) && aligned16(val) &&
                     (val_row & 3) == 0;
    if (vec) {
        const int32_t j = (int32_t)j0;
        const int32_t b = j / B;
        const int32_t slot = block_slot[b];
        const float4 wt = ld4(a.w_t + j), wp = ld4(a.w_prev + j);
        const int64_t vpos = (int64_t)slot * B + (j - (int64_t)b * B);
        for (int k = 0; k < K; ++k) {
            if ((skip >> k) & 1ull) continue;
            float* e = a.wp.e[k];
            const float* gr = a.wp.g[k];
            float* y = a.wp.y[k];
            if (aligned16(e) && aligned16(gr) && (!a.detach || aligned16(y))) {
                const float4 ev = ld4(e + j), gv = ld4(gr + j);
                float4 u;
                u.x = rule_u_rt(rule, ev.x, gv.x, wt.x, wp.x, c, h);
                u.y = rule_u_rt(rule, ev.y, gv.y, wt.y, wp.y, c, h);
                u.z = rule_u_rt(rule, ev.z, gv.z, wt.z, wp.z, c, h);
                u.w = rule_u_rt(rule, ev.w, gv.w, wt.w, wp.w, c, h);
                if (slot >= 0) {
                    st4(val + (size_t)k * val_row + vpos, u);
                    st4(e + j, make_float4(u.x - u.x, u.y - u.y, u.z - u.z, u.w - u.w));
                } else {
                    st4(e + j, u);
                    // unsent: e_{t+1} = u and w_{t+1} = w_t here, so this is final
                    if (a.detach)
                        st4(y + j, make_float4(detached(wt.x, u.x, qd), detached(wt.y, u.y, qd),
                                               detached(wt.z, u.z, qd), detached(wt.w, u.w, qd)));
                }
            } else {
                const float wtq[4] = {wt.x, wt.y, wt.z, wt.w}, wpq[4] = {wp.x, wp.y, wp.z, wp.w};
                for (int q = 0; q < 4; ++q) {
                    const float u = rule_u_rt(rule, e[j + q], gr[j + q], wtq[q], wpq[q], c, h);
                    if (slot >= 0) {
                        val[(size_t)k * val_row + vpos + q] = u;
                        e[j + q] = u - u;
                    } else {
                        e[j + q] = u;
                        if (a.detach) y[j + q] = detached(wtq[q], u, qd);
                    }
                }
            }
        }
        return;
    }
    for (int q = 0; q < 4; ++q) {
        const int64_t jj = j0 + q;
        if (jj >= d) break;
        const int32_t j = (int32_t)jj;
        const int32_t b = j / B;
        const int32_t slot = block_slot[b];
        const float wtj = a.w_t[j], wpj = a.w_prev[j];
        const int64_t vpos = (int64_t)slot * B + (j - (int64_t)b * B);
        const uint64_t skip_j = j < vec_end ? vec_mask : 0ull;
        for (int k = 0; k < K; ++k) {
            if ((skip_j >> k) & 1ull) continue;
            float* e = a.wp.e[k];
            const float u = rule_u_rt(rule, e[j], a.wp.g[k][j], wtj, wpj, c, h);
            if (slot >= 0) {
                val[(size_t)k * val_row + vpos] = u;
                e[j] = u - u;
            } else {
                e[j] = u;
                if (a.detach) a.wp.y[k][j] = detached(wtj, u, qd);
            }
        }
    }
}

// Vector path of the RBGS worker pass: one workgroup per (chunk of kChunk
// components, worker), 8 components per thread, like the top-s pass: w_t
// and w_prev through the cache, g, e (and the detached points) streamed.  B
// is a multiple of 4, so each float4 lies in one block; a selected block's
// components go to the message, the rest stay in the residual.
template <int kRule, bool kDetach>
__global__ __launch_bounds__(kGroup) void rbgs_vec_kernel(StepArgs a, int32_t K, int32_t B,
                                                          const int32_t* block_slot, float* val, int64_t val_row,
                                                          uint64_t vec_mask) {
    int chunk, k;
    run_order(blockIdx.x, K, a.run, &chunk, &k);
    const int64_t chunk0 = (int64_t)chunk * kChunk;
    if (chunk0 >= a.d || !((vec_mask >> k) & 1ull)) return;  // padding, or the element-wise kernel's
    if (chunk0 + kChunk > a.d) {  // the partial last chunk, element by element
        const float wq = a.q;
        for (int64_t j = chunk0 + threadIdx.x; j < a.d; j += kGroup) {
            const int32_t b = (int32_t)(j / B);
            const int32_t slot = block_slot[b];
            const float wtj = a.w_t[j], wpj = a.w_prev[j];
            const float u = rule_u<kRule>(a.wp.e[k][j], a.wp.g[k][j], wtj, wpj, a.c, a.h);
            if (slot >= 0) {
                val[(size_t)k * val_row + (int64_t)slot * B + (j - (int64_t)b * B)] = u;
                a.wp.e[k][j] = u - u;
            } else {
                a.wp.e[k][j] = u;
                if (kDetach) a.wp.y[k][j] = detached(wtj, u, wq);
            }
        }
        return;
    }
    const int o0 = threadIdx.x * 4;
    const int64_t start = chunk0 + o0;
    float* ep = a.wp.e[k] + start;
    const float* gp = a.wp.g[k] + start;
    constexpr bool kNeedW = kRule != kRuleServerMomentum || kDetach;
    const float c = a.c, h = a.h;
    float4 u[2], gv[2], wt[2], wv[2];
#pragma unroll
    for (int i = 0; i < 2; ++i) {
        u[i] = ld4_stream(ep + i * (kGroup * 4));
        gv[i] = ld4_stream(gp + i * (kGroup * 4));
        if (kNeedW)
            load_w4<kDetach>(a, start + i * (kGroup * 4), mark_word(a, start + i * (kGroup * 4)), &wt[i], &wv[i]);
        else
            wt[i] = wv[i] = make_float4(0.f, 0.f, 0.f, 0.f);
    }
#pragma unroll
    for (int i = 0; i < 2; ++i) {
        const int64_t j = start + i * (kGroup * 4);
        const int32_t b = (int32_t)(j / B);
        const int32_t slot = block_slot[b];
        u[i].x = rule_u<kRule>(u[i].x, gv[i].x, wt[i].x, wv[i].x, c, h);
        u[i].y = rule_u<kRule>(u[i].y, gv[i].y, wt[i].y, wv[i].y, c, h);
        u[i].z = rule_u<kRule>(u[i].z, gv[i].z, wt[i].z, wv[i].z, c, h);
        u[i].w = rule_u<kRule>(u[i].w, gv[i].w, wt[i].w, wv[i].w, c, h);
        if (slot >= 0) {
            st4(val + (size_t)k * val_row + (int64_t)slot * B + (j - (int64_t)b * B), u[i]);
            st4_stream(ep + i * (kGroup * 4),
                       make_float4(u[i].x - u[i].x, u[i].y - u[i].y, u[i].z - u[i].z, u[i].w - u[i].w));
        } else {
            st4_stream(ep + i * (kGroup * 4), u[i]);
            // unsent: e_{t+1} = u and w_{t+1} = w_t here, so this is final
            if (kDetach) {
                const float q = a.q;
                st4_stream(a.wp.y[k] + j, make_float4(detached(wt[i].x, u[i].x, q), detached(wt[i].y, u[i].y, q),
                                                      detached(wt[i].z, u[i].z, q), detached(wt[i].w, u[i].w, q)));
            }
        }
    }
}

hipError_t launch_rbgs_fused(const StepArgs& a, int32_t K, int32_t B, const int32_t* block_slot,
                             float* val, int64_t val_row, uint64_t vec_mask, hipStream_t st) {
    // vector kernel over all chunks (the partial last one element by
    // element) for the workers in vec_mask (B a multiple of 4 and the message
    // rows 16-byte aligned, checked by the caller), element-wise kernel for
    // the rest
    const int64_t n_chunks = vec_mask ? ((int64_t)a.d + kChunk - 1) / kChunk : 0;
    const int64_t vec_end = vec_mask ? (int64_t)a.d : 0;
    if (n_chunks > 0) {
        const dim3 grid((unsigned)run_order_grid(n_chunks, K, a.run));
        if (a.rule == kRuleServerMomentum) {
            if (a.detach) return hipErrorInvalidValue;
            hipLaunchKernelGGL((rbgs_vec_kernel<kRuleServerMomentum, false>), grid, dim3(kGroup), 0, st, a, K, B,
                               block_slot, val, val_row, vec_mask);
        } else if (a.rule == kRuleLrInResidual) {
            if (a.detach)
                hipLaunchKernelGGL((rbgs_vec_kernel<kRuleLrInResidual, true>), grid, dim3(kGroup), 0, st, a, K, B,
                                   block_slot, val, val_row, vec_mask);
            else
                hipLaunchKernelGGL((rbgs_vec_kernel<kRuleLrInResidual, false>), grid, dim3(kGroup), 0, st, a, K, B,
                                   block_slot, val, val_row, vec_mask);
        } else {
            if (a.detach)
                hipLaunchKernelGGL((rbgs_vec_kernel<kRuleGmc, true>), grid, dim3(kGroup), 0, st, a, K, B, block_slot,
                                   val, val_row, vec_mask);
            else
                hipLaunchKernelGGL((rbgs_vec_kernel<kRuleGmc, false>), grid, dim3(kGroup), 0, st, a, K, B,
                                   block_slot, val, val_row, vec_mask);
        }
        const hipError_t e = hipGetLastError();
        if (e != hipSuccess) return e;
    }
    const uint64_t all = K == 64 ? ~0ull : ((1ull << K) - 1ull);
    if (vec_mask == all) return hipSuccess;
    const int64_t j_begin = 0;
    const int64_t threads = ((int64_t)a.d - j_begin + 3) / 4;
    const int grid = (int)((threads + kGroup - 1) / kGroup);
    hipLaunchKernelGGL(rbgs_fused_kernel, dim3(grid), dim3(kGroup), 0, st, a, K, B, block_slot, val, val_row,
                       j_begin, vec_mask, vec_end);
    return hipGetLastError();
}

// ============================================================================
// server: sum over workers in worker order, dense update
// ============================================================================

// w_{t+1} at one component: w_t + update, or with momentum on the server
// (w_t + update) + b (w_t - w_{t-1}).
__device__ __forceinline__ float next_w(float x, float dl, const float* w_prev, int64_t j, float b) {
    const float moved = x + dl;
    if (!w_prev) return moved;
    const float back = x - w_prev[j];
    const float push = b * back;
    return moved + push;
}

__device__ __forceinline__ uint32_t not_finite(float x) {
    return (__float_as_uint(x) & 0x7f800000u) == 0x7f800000u ? 1u : 0u;
}

// Bits of the four components at q of a range for the next worker pass:
// some worker sent the component (hit) or w_{t+1} there is not finite.
__device__ __forceinline__ uint32_t mark4(const unsigned char* hit, int q, float4 wn) {
    return (hit[q] || not_finite(wn.x) ? 1u : 0u) | (hit[q + 1] || not_finite(wn.y) ? 2u : 0u) |
           (hit[q + 2] || not_finite(wn.z) ? 4u : 0u) | (hit[q + 3] || not_finite(wn.w) ? 8u : 0u);
}

// Stores the range's bitmap words (wb in LDS, one bit per component) once
// every thread has marked its components.
__device__ __forceinline__ void flush_marks(const uint32_t* wb, int64_t base, int64_t n, uint32_t* wbits) {
    __syncthreads();
    const int words = (int)((n + 31) / 32);
    if ((int)threadIdx.x < words) wbits[(base >> 5) + threadIdx.x] = wb[threadIdx.x];
}

// Sparse apply (f.sparse_apply): the range's words of the previous pass's
// marks (read before this pass overwrites them), or-ed with the components
// some worker sent now.  Where a word is zero, w_out already holds w_{t+1}:
// w_{t-1} = w_t there (unmarked), and w_{t+1} = w_t + (-0) = w_t (finite,
// nothing sent).
__device__ __forceinline__ void visit_words(uint32_t* wv, const unsigned char* hit, int64_t base, int64_t n,
                                            const uint32_t* wbits) {
    const int words = (int)((n + 31) / 32);
    for (int w = threadIdx.x; w < words; w += kGroup) {
        uint32_t m = wbits[(base >> 5) + w];
        const int lim = n - w * 32 < 32 ? (int)(n - w * 32) : 32;
        for (int b = 0; b < lim; ++b) m |= hit[w * 32 + b] ? (1u << b) : 0u;
        wv[w] = m;
    }
    __syncthreads();
}

// Writes update = -(s * acc) for the n components of a range starting at base
// (when f.update is not NULL) and, with kApply, w_out = next_w(w_in, update),
// only in the words wv marks when wv is not NULL (sparse apply); with f.wbits
// also marks the components for the next worker pass in wb.
template <bool kApply>
__device__ __forceinline__ void write_update(const float* acc, const unsigned char* hit, uint32_t* wb, int64_t base,
                                             int64_t n, const FinishArgs& f, const uint32_t* wv,
                                             int32_t* nf_flag = nullptr) {
    const float s = f.s;
    const bool vec = n == kAggRange && (base & 3) == 0 && (f.update == nullptr || aligned16(f.update)) &&
                     (!kApply || (aligned16(f.w_in) && aligned16(f.w_out) &&
                                  (f.w_prev == nullptr || aligned16(f.w_prev))));
    if (vec) {
        for (int q = threadIdx.x * 4; q < kAggRange; q += kGroup * 4) {
            const int64_t j = base + q;
            const float4 dl = make_float4(-(s * acc[q]), -(s * acc[q + 1]), -(s * acc[q + 2]), -(s * acc[q + 3]));
            if (f.update) st4(f.update + j, dl);
            if (kApply && (!wv || wv[q >> 5])) {
                const float4 x = ld4(f.w_in + j);
                float4 nx = make_float4(x.x + dl.x, x.y + dl.y, x.z + dl.z, x.w + dl.w);
                if (f.w_prev) {  // momentum on the server
                    const float4 p = ld4(f.w_prev + j);
                    const float b = f.b;
                    nx = make_float4(nx.x + b * (x.x - p.x), nx.y + b * (x.y - p.y), nx.z + b * (x.z - p.z),
                                     nx.w + b * (x.w - p.w));
                }
                st4(f.w_out + j, nx);
                if (f.wbits) atomicOr(&wb[q >> 5], mark4(hit, q, nx) << (q & 31));
            }
        }
        return;
    }
    for (int q = threadIdx.x; q < n; q += kGroup) {
        const int64_t j = base + q;
        const float dl = -(s * acc[q]);
        if (f.update) f.update[j] = dl;
        if (kApply && (!wv || wv[q >> 5])) {
            const float wn = next_w(f.w_in[j], dl, f.w_prev, j, f.b);
            f.w_out[j] = wn;
            if (f.wbits && (hit[q] || not_finite(wn))) atomicOr(&wb[q >> 5], 1u << (q & 31));
            if (nf_flag && !hit[q] && not_finite(wn)) atomicOr(nf_flag, 1);
        }
    }
}

// GMC+: the detached points at the components of the range some worker sent
// (hit[q] != 0), where w_{t+1} may differ from w_t: y_k = w_{t+1} - q e_{t+1,k}
// for every worker k, with w_{t+1} read back from w_out after the
// workgroup's writes (w_out may alias w_in or w_prev).  Elsewhere the fused
// worker pass already wrote the final value w_t - q u_k.
__device__ __forceinline__ void finish_detach(const unsigned char* hit, int64_t base, int64_t n, int32_t K,
                                              const FinishArgs& f) {
    __syncthreads();  // this workgroup's w_out writes are visible to all its threads
    for (int q = threadIdx.x; q < n; q += kGroup) {
        if (!hit[q]) continue;
        const int64_t j = base + q;
        const float wn = f.w_out[j];
        for (int k = 0; k < K; ++k) f.y[k][j] = detached(wn, f.e[k][j], f.q);
    }
}

// rowptr[k][r] = first message position of worker k whose index is >= r*R
// with R = kAggTopkRange (a lower bound by binary search over the worker's
// ascending row);
// rowptr[k][n_ranges] = the row's length.  Any row content keeps every entry
// within [0, length].
__global__ __launch_bounds__(kGroup) void agg_rowptr_kernel(int32_t K, int32_t d, const int32_t* idx,
                                                            int64_t idx_row, const int64_t* msg_len,
                                                            int32_t* rowptr, int32_t n_ranges) {
    const int k = blockIdx.y;
    const int32_t r = blockIdx.x * kGroup + threadIdx.x;
    if (r > n_ranges) return;
    int64_t L = msg_len[k];
    if (L < 0) L = 0;
    if (L > idx_row) L = idx_row;
    int32_t* rp = rowptr + (size_t)k * (n_ranges + 1);
    if (r == n_ranges) {
        rp[r] = (int32_t)L;
        return;
    }
    const int64_t target = (int64_t)r * kAggTopkRange;
    const int32_t* row = idx + (size_t)k * idx_row;
    int64_t lo = 0, hi = L;
    while (lo < hi) {
        const int64_t mid = (lo + hi) >> 1;
        if ((int64_t)row[mid] < target) lo = mid + 1; else hi = mid;
    }
    rp[r] = (int32_t)lo;
}

hipError_t launch_agg_rowptr(int32_t K, int32_t d, const int32_t* idx, int64_t idx_row,
                             const int64_t* msg_len, int32_t* rowptr, int32_t n_ranges,
                             hipStream_t st) {
    const int gx = (n_ranges + 1 + kGroup - 1) / kGroup;
    hipLaunchKernelGGL(agg_rowptr_kernel, dim3(gx, K), dim3(kGroup), 0, st, K, d, idx, idx_row, msg_len,
                       rowptr, n_ranges);
    return hipGetLastError();
}

// One workgroup per range of kAggTopkRange components (16 per thread).  The
// workgroup first issues its loads of w_t (fused apply; a sparse apply loads
// only the words that change) and of the previous pass's marks, then fetches the K workers' entries of the range
// into LDS together (one round of loads) and adds them to the range's
// accumulator one worker after the other; a range with more entries than the
// staging holds reads them worker by worker instead.  Sent components are
// kept as a bitmap (hb), so a workgroup needs about 22 KB of LDS (seven fit
// on a CU) with a stage of kStage = 512 entries, 19 KB (eight) with 128 for
// sparse messages: the kernel is bound by its chain of dependent loads, so
// residency counts, and twice the components per chain halves the chains.
template <bool kApply, int kStage>
__global__ __launch_bounds__(kGroup) void agg_topk_kernel(int32_t K, int32_t d, const int32_t* idx,
                                                          int64_t idx_row, const float* val, int64_t val_row,
                                                          const int32_t* rowptr, int32_t n_ranges, FinishArgs f) {
    constexpr int R = kAggTopkRange, NW = R / 32, V = R / (kGroup * 4);
    static_assert(V * kGroup * 4 == R && NW <= kGroup, "whole float4 per thread, one word per thread");
    __shared__ float acc[R];
    __shared__ uint32_t hb[NW];  // components some worker sent
    __shared__ uint32_t wb[NW];  // marks for the next worker pass
    __shared__ uint32_t wv[NW];  // sparse apply: the words to write (old marks | sent)
    __shared__ int32_t st_idx[kStage];
    __shared__ float st_val[kStage];
    __shared__ int32_t src[kMaxWorkers];
    __shared__ int32_t pre[kMaxWorkers + 1];
    __shared__ uint32_t dl_n;    // entries of the change list
    const int r = blockIdx.x;
    const int t = threadIdx.x;
    // the change list of this range: the components this pass marks, with
    // fl(w_{t+1} - w_t), for the next worker pass
    int2* const dlr = (kApply && f.wbits && f.dlist) ? f.dlist + (size_t)r * f.dl_stride : nullptr;
    const uint32_t dl_cap = (uint32_t)f.dl_stride - 1u;
    auto list_change = [&](int q, float wn, float x) {
        const uint32_t pos = atomicAdd(&dl_n, 1u);
        if (pos < dl_cap) dlr[1 + pos] = make_int2(q, __float_as_int(wn - x));
    };
    const int64_t base = (int64_t)r * R;
    const int64_t n = (int64_t)d - base < R ? (int64_t)d - base : R;
    const int words = (int)((n + 31) / 32);
    const float s = f.s;
    const bool vec = n == R && (f.update == nullptr || aligned16(f.update)) &&
                     (!kApply || (aligned16(f.w_in) && aligned16(f.w_out) &&
                                  (f.w_prev == nullptr || aligned16(f.w_prev))));
    const bool sparse = kApply && f.sparse_apply;
    // this thread's components: [base + 1024 i + 4 t, +4), i < V
    float4 wx[V], px[V];
#pragma unroll
    for (int i = 0; i < V; ++i) {
        wx[i] = px[i] = make_float4(0.f, 0.f, 0.f, 0.f);
        if (kApply && vec && !sparse) {
            wx[i] = ld4(f.w_in + base + i * (kGroup * 4) + t * 4);
            if (f.w_prev) px[i] = ld4(f.w_prev + base + i * (kGroup * 4) + t * 4);
        }
    }
    if (t == 0) dl_n = 0u;
    // in place, w already holds w_t everywhere: only this pass's sent
    // components are written, and the previous marks are visited only once
    // a non-finite w has been written (they then keep their marks, and the
    // next worker pass its NaN momentum term)
    const bool old_marks = sparse && (!f.inplace || (f.nf && *f.nf == f.nf_epoch));
    bool nonfinite = false;  // this thread wrote a non-finite w_{t+1}
    if (t < NW) {
        hb[t] = 0u;
        wb[t] = 0u;
        wv[t] = (old_marks && t < words) ? f.wbits[(base >> 5) + t] : 0u;
    }
    if (t < K) {
        const int32_t* rp = rowptr + (size_t)t * (n_ranges + 1);
        const int32_t lo = rp[r], hi = rp[r + 1];
        src[t] = lo;
        pre[t + 1] = hi > lo ? hi - lo : 0;
    }
    // sparse apply: whether the previous pass marked the range anywhere
    const bool marked = __syncthreads_or(sparse && t < NW && wv[t] != 0u) != 0;
    // a sparse apply's range with no old marks and no entries changes
    // nothing: w_out holds w_{t-1}, equal to w_t = w_{t+1} there, and its
    // marks stay clear
    if (sparse && !marked && f.update == nullptr && !__syncthreads_or(t < K && pre[t + 1] > 0)) {
        if (dlr && t == 0) dlr[0] = make_int2(0, 0);
        return;
    }
    for (int q = t; q < R; q += kGroup) acc[q] = 0.0f;
    // sparse apply: w_t is fetched only in the 32-component words the
    // output changes: those of the previous pass's marks now, those of this
    // pass's entries as soon as the entries are staged (their loads then
    // overlap the ordered sum); a dense range's are fetched after the sum
    const bool hb_early = sparse && vec;  // hb is complete before the sum
    uint32_t got = 0u;                    // bit i: wx[i] holds w_t
    if (hb_early) {
#pragma unroll
        for (int i = 0; i < V; ++i) {
            const int q = i * (kGroup * 4) + t * 4;
            if (wv[q >> 5]) {
                wx[i] = ld4(f.w_in + base + q);
                got |= 1u << i;
            }
        }
    }
    if (t == 0) {
        pre[0] = 0;
        for (int k = 0; k < K; ++k) pre[k + 1] += pre[k];
    }
    __syncthreads();
    const int32_t total = pre[K];
    if (total <= kStage) {
        for (int32_t i = t; i < total; i += kGroup) {
            int k = 0;
            while (i >= pre[k + 1]) ++k;
            const int64_t q = (int64_t)src[k] + (i - pre[k]);
            const int32_t j = idx[(size_t)k * idx_row + q];
            const float v = val[(size_t)k * val_row + q];
            st_idx[i] = j;
            st_val[i] = v;
            if (f.zero_e && j - base >= 0 && j - base < n) f.ez[k][j] = v - v;
        }
        __syncthreads();
        if (hb_early) {
            for (int32_t i = t; i < total; i += kGroup) {
                const int64_t j = (int64_t)st_idx[i] - base;
                if (j >= 0 && j < R) atomicOr(&hb[j >> 5], 1u << (j & 31));
            }
            __syncthreads();
#pragma unroll
            for (int i = 0; i < V; ++i) {
                const int q = i * (kGroup * 4) + t * 4;
                if (!((got >> i) & 1u) && hb[q >> 5]) {
                    wx[i] = ld4(f.w_in + base + q);
                    got |= 1u << i;
                }
            }
        }
        for (int k = 0; k < K; ++k) {
            if (pre[k + 1] > pre[k]) {
                for (int32_t i = pre[k] + t; i < pre[k + 1]; i += kGroup) {
                    const int64_t j = (int64_t)st_idx[i] - base;
                    if (j >= 0 && j < R) {
                        acc[j] = acc[j] + st_val[i];
                        if (!hb_early) atomicOr(&hb[j >> 5], 1u << (j & 31));
                    }
                }
                __syncthreads();  // worker k's additions land before worker k+1's
            }
        }
    } else {
        // a dense range (up to K entries per component): worker after
        // worker straight from the messages, kDirect loads in flight per
        // thread (eight with the larger stage, for dense messages: a worker
        // sending 2048 entries of the range then takes one round trip; the
        // sparse-message kernel keeps four and its registers)
        constexpr int kDirect = kStage >= 512 ? 8 : 4;
        for (int k = 0; k < K; ++k) {
            const int32_t cnt = pre[k + 1] - pre[k];
            const int32_t* ip = idx + (size_t)k * idx_row + src[k];
            const float* vp = val + (size_t)k * val_row + src[k];
            for (int32_t i0 = 0; i0 < cnt; i0 += kDirect * kGroup) {
                int32_t jj[kDirect];
                float vv[kDirect];
#pragma unroll
                for (int u = 0; u < kDirect; ++u) {
                    const int32_t i = i0 + u * kGroup + t;
                    jj[u] = -1;
                    vv[u] = 0.0f;
                    if (i < cnt) {
                        jj[u] = ip[i];
                        vv[u] = vp[i];
                    }
                }
#pragma unroll
                for (int u = 0; u < kDirect; ++u) {
                    const int64_t j = (int64_t)jj[u] - base;
                    if (i0 + u * kGroup + t < cnt && j >= 0 && j < R) {
                        acc[j] = acc[j] + vv[u];
                        atomicOr(&hb[j >> 5], 1u << (j & 31));
                        if (f.zero_e && j < n) f.ez[k][jj[u]] = vv[u] - vv[u];
                    }
                }
            }
            __syncthreads();  // worker k's additions land before worker k+1's
        }
    }
    __syncthreads();
    if (sparse) {
        if (t < NW) wv[t] |= hb[t];
        __syncthreads();
    }
    if (vec) {
        uint32_t lm[V];  // the change list: marked components of each float4 and their changes
        float4 ld[V];
#pragma unroll
        for (int i = 0; i < V; ++i) {
            lm[i] = 0u;
            ld[i] = make_float4(0.f, 0.f, 0.f, 0.f);
            const int q = i * (kGroup * 4) + t * 4;
            const float4 dl = make_float4(-(s * acc[q]), -(s * acc[q + 1]), -(s * acc[q + 2]), -(s * acc[q + 3]));
            if (f.update) st4(f.update + base + q, dl);
            if (kApply && (!sparse || wv[q >> 5])) {
                const float4 x = (sparse && !((got >> i) & 1u)) ? ld4(f.w_in + base + q) : wx[i];
                float4 nx = make_float4(x.x + dl.x, x.y + dl.y, x.z + dl.z, x.w + dl.w);
                if (f.w_prev) {  // momentum on the server
                    const float4 pp = px[i];
                    const float b = f.b;
                    nx = make_float4(nx.x + b * (x.x - pp.x), nx.y + b * (x.y - pp.y), nx.z + b * (x.z - pp.z),
                                     nx.w + b * (x.w - pp.w));
                }
                st4(f.w_out + base + q, nx);
                if (f.wbits) {
                    const uint32_t nfm = not_finite(nx.x) | (not_finite(nx.y) << 1) | (not_finite(nx.z) << 2) |
                                         (not_finite(nx.w) << 3);
                    nonfinite |= nfm != 0u;
                    const uint32_t m = ((hb[q >> 5] >> (q & 31)) & 0xfu) | nfm;
                    atomicOr(&wb[q >> 5], m << (q & 31));
                    lm[i] = m;
                    ld[i] = make_float4(nx.x - x.x, nx.y - x.y, nx.z - x.z, nx.w - x.w);
                }
            }
        }
        if (dlr) {
            // one LDS atomic per wavefront for the list positions: the
            // wavefront's prefix of its threads' marked components
            uint32_t mine = 0;
#pragma unroll
            for (int i = 0; i < V; ++i) mine += (uint32_t)__popc(lm[i]);
            const int lane = t & (kWave - 1);
            uint32_t incl = mine;
#pragma unroll
            for (int o = 1; o < kWave; o <<= 1) {
                const uint32_t y = __shfl_up(incl, o, kWave);
                if (lane >= o) incl += y;
            }
            const uint32_t wtotal = __shfl(incl, kWave - 1, kWave);
            uint32_t wbase = 0;
            if (lane == kWave - 1 && wtotal) wbase = atomicAdd(&dl_n, wtotal);
            uint32_t pos = __shfl(wbase, kWave - 1, kWave) + incl - mine;
#pragma unroll
            for (int i = 0; i < V; ++i) {
                const int q = i * (kGroup * 4) + t * 4;
                const float dv[4] = {ld[i].x, ld[i].y, ld[i].z, ld[i].w};
#pragma unroll
                for (int e = 0; e < 4; ++e) {
                    if ((lm[i] >> e) & 1u) {
                        if (pos < dl_cap) dlr[1 + pos] = make_int2(q + e, __float_as_int(dv[e]));
                        ++pos;
                    }
                }
            }
        }
    } else {
        for (int q = t; q < n; q += kGroup) {
            const int64_t j = base + q;
            const float dl = -(s * acc[q]);
            if (f.update) f.update[j] = dl;
            if (kApply && (!sparse || wv[q >> 5])) {
                const float x = f.w_in[j];
                const float wn = next_w(x, dl, f.w_prev, j, f.b);
                f.w_out[j] = wn;
                if (f.wbits && (((hb[q >> 5] >> (q & 31)) & 1u) || not_finite(wn))) {
                    atomicOr(&wb[q >> 5], 1u << (q & 31));
                    if (dlr) list_change(q, wn, x);
                }
                if (f.wbits && not_finite(wn)) nonfinite = true;
            }
        }
    }
    if (kApply && f.wbits) {
        if (nonfinite && f.nf) *f.nf = f.nf_epoch;  // the same value from every writer
        __syncthreads();
        if (t < words) f.wbits[(base >> 5) + t] = wb[t];
        if (dlr && t == 0) dlr[0] = make_int2(dl_n <= dl_cap ? (int32_t)dl_n : -1, 0);
    }
    if (kApply && f.detach) {
        // GMC+: the detached points at the sent components, from w_{t+1}
        // as this workgroup wrote it
        __syncthreads();
        for (int q = t; q < n; q += kGroup) {
            if (!((hb[q >> 5] >> (q & 31)) & 1u)) continue;
            const int64_t j = base + q;
            const float wn = f.w_out[j];
            for (int k = 0; k < K; ++k) f.y[k][j] = detached(wn, f.e[k][j], f.q);
        }
    }
}

hipError_t launch_agg_topk(int32_t K, int32_t d, const int32_t* idx, int64_t idx_row,
                           const float* val, int64_t val_row, const int32_t* rowptr,
                           int32_t n_ranges, const FinishArgs& f, hipStream_t st) {
    // the smaller stage when the messages hold at most 48 entries per range
    // on average (per-tensor top-s of a decoder-sized model: about 33);
    // denser messages keep the larger one, since a range with more entries
    // than the stage reads them worker after worker
    const bool small = (int64_t)K * idx_row <= 48 * (int64_t)n_ranges;
    if (f.w_out && small)
        hipLaunchKernelGGL((agg_topk_kernel<true, kAggTopkStageSmall>), dim3(n_ranges), dim3(kGroup), 0, st, K, d,
                           idx, idx_row, val, val_row, rowptr, n_ranges, f);
    else if (f.w_out)
        hipLaunchKernelGGL((agg_topk_kernel<true, kAggTopkStage>), dim3(n_ranges), dim3(kGroup), 0, st, K, d, idx,
                           idx_row, val, val_row, rowptr, n_ranges, f);
    else if (small)
        hipLaunchKernelGGL((agg_topk_kernel<false, kAggTopkStageSmall>), dim3(n_ranges), dim3(kGroup), 0, st, K, d,
                           idx, idx_row, val, val_row, rowptr, n_ranges, f);
    else
        hipLaunchKernelGGL((agg_topk_kernel<false, kAggTopkStage>), dim3(n_ranges), dim3(kGroup), 0, st, K, d, idx,
                           idx_row, val, val_row, rowptr, n_ranges, f);
    return hipGetLastError();
}

// RBGS: every worker sent the same blocks; block_slot[b] is the position q
// of block b among the step's ascending block ids (-1: not drawn), and a
// component of block b sits at q*B + offset in each message.  The range of
// kAggRange components starting at base.  nf_flag (nullable) is raised when a
// component no worker sent gets a non-finite w_{t+1} (it stays marked, so the
// next sparse server pass visits every range).
struct RbgsLds {
    float acc[kAggRange];
    unsigned char hit[kAggRange];
    uint32_t wb[kAggRange / 32];
    uint32_t wv[kAggRange / 32];
};

template <bool kApply>
__device__ void agg_rbgs_range(int64_t base, int32_t K, int32_t d, int32_t B, const int32_t* block_slot,
                               const float* val, int64_t val_row, const FinishArgs& f, int32_t* nf_flag,
                               RbgsLds& L) {
    float* acc = L.acc;
    unsigned char* hit = L.hit;
    uint32_t* wb = L.wb;
    uint32_t* wv = L.wv;
    const int64_t n = (int64_t)d - base < kAggRange ? (int64_t)d - base : kAggRange;
    const bool sparse = kApply && f.sparse_apply;
    if (threadIdx.x < kAggRange / 32) wb[threadIdx.x] = 0u;
    if (f.wbits) __syncthreads();  // wb cleared before any mark
    const bool vec = n == kAggRange && (B & 3) == 0 && aligned16(val) && (val_row & 3) == 0 &&
                     (f.update == nullptr || aligned16(f.update)) && (!f.detach || f.rows16) &&
                     (!kApply || (aligned16(f.w_in) && aligned16(f.w_out) &&
                                  (f.w_prev == nullptr || aligned16(f.w_prev))));
    if (vec) {
        // two float4 per thread; each lies in one block (B % 4 == 0), whose
        // slot says where its values sit in every message
        const float s = f.s;
        float4 wx[2], pv[2];
        int64_t js[2];
        int32_t slots[2], bs[2];
        bool visit[2];
#pragma unroll
        for (int i = 0; i < 2; ++i) {
            js[i] = base + i * (kGroup * 4) + threadIdx.x * 4;
            bs[i] = (int32_t)(js[i] / B);
            slots[i] = block_slot[bs[i]];
            // sparse apply: the four components need writing where the
            // previous marks fall or the block was sent (j is a multiple of
            // 4, so its four bits sit in one word; flush_marks rewrites the
            // words only after a barrier)
            visit[i] = !sparse || slots[i] >= 0 || ((f.wbits[js[i] >> 5] >> (js[i] & 31)) & 0xfu) != 0u;
            wx[i] = pv[i] = make_float4(0.f, 0.f, 0.f, 0.f);
            if (kApply && visit[i]) {
                wx[i] = ld4(f.w_in + js[i]);
                if (f.w_prev) pv[i] = ld4(f.w_prev + js[i]);
            }
        }
#pragma unroll
        for (int i = 0; i < 2; ++i) {
            const int64_t j = js[i];
            float4 a4 = make_float4(0.f, 0.f, 0.f, 0.f);
            if (slots[i] >= 0) {
                const float* v = val + (int64_t)slots[i] * B + (j - (int64_t)bs[i] * B);
                for (int k = 0; k < K; ++k) {  // worker order
                    const float4 x = ld4(v + (size_t)k * val_row);
                    a4 = make_float4(a4.x + x.x, a4.y + x.y, a4.z + x.z, a4.w + x.w);
                }
            }
            const float4 dl = make_float4(-(s * a4.x), -(s * a4.y), -(s * a4.z), -(s * a4.w));
            if (f.update) st4(f.update + j, dl);
            if (kApply && visit[i]) {
                const float4 x = wx[i];
                float4 nx = make_float4(x.x + dl.x, x.y + dl.y, x.z + dl.z, x.w + dl.w);
                if (f.w_prev) {  // momentum on the server
                    const float4 p = pv[i];
                    const float b = f.b;
                    nx = make_float4(nx.x + b * (x.x - p.x), nx.y + b * (x.y - p.y), nx.z + b * (x.z - p.z),
                                     nx.w + b * (x.w - p.w));
                }
                st4(f.w_out + j, nx);
                if (f.wbits) {
                    const int q = (int)(j - base);
                    const uint32_t nf = not_finite(nx.x) | (not_finite(nx.y) << 1) | (not_finite(nx.z) << 2) |
                                        (not_finite(nx.w) << 3);
                    atomicOr(&wb[q >> 5], ((slots[i] >= 0 ? 0xfu : 0u) | nf) << (q & 31));
                    if (nf_flag && nf && slots[i] < 0) atomicOr(nf_flag, 1);
                }
                if (f.detach && slots[i] >= 0) {  // GMC+: the sent components' detached points
                    const float q = f.q;
                    for (int k0 = 0; k0 < K; k0 += 4) {  // four workers' loads in flight
                        float4 e[4];
#pragma unroll
                        for (int u = 0; u < 4; ++u)
                            if (k0 + u < K) e[u] = ld4(f.e[k0 + u] + j);
#pragma unroll
                        for (int u = 0; u < 4; ++u)
                            if (k0 + u < K)
                                st4(f.y[k0 + u] + j, make_float4(detached(nx.x, e[u].x, q), detached(nx.y, e[u].y, q),
                                                                 detached(nx.z, e[u].z, q), detached(nx.w, e[u].w, q)));
                    }
                }
            }
        }
        if (kApply && f.wbits) flush_marks(wb, base, n, f.wbits);
        return;
    }
    for (int q = threadIdx.x; q < kAggRange; q += kGroup) {
        float a = 0.0f;
        unsigned char sent = 0;
        if (q < n) {
            const int64_t j = base + q;
            const int32_t b = (int32_t)(j / B);
            const int32_t slot = block_slot[b];
            if (slot >= 0) {
                const int64_t vpos = (int64_t)slot * B + (j - (int64_t)b * B);
                for (int k = 0; k < K; ++k) a = a + val[(size_t)k * val_row + vpos];
                sent = 1;
            }
        }
        acc[q] = a;
        hit[q] = sent;
    }
    __syncthreads();
    if (sparse) visit_words(wv, hit, base, n, f.wbits);
    write_update<kApply>(acc, hit, wb, base, n, f, sparse ? wv : nullptr, f.wbits ? nf_flag : nullptr);
    if (kApply && f.wbits) flush_marks(wb, base, n, f.wbits);
    if (kApply && f.detach) finish_detach(hit, base, n, K, f);
}

// The RBGS server pass over the ranges of kAggRange components: one
// workgroup per range, or, for a sparse apply, the visit list the block draw
// built (meta[0] ranges in visit[], ascending; meta[0] < 0: every range),
// each workgroup taking every gridDim-th entry.
template <bool kApply>
__global__ __launch_bounds__(kGroup) void agg_rbgs_kernel(int32_t K, int32_t d, int32_t B, const int32_t* block_slot,
                                                          const float* val, int64_t val_row, FinishArgs f,
                                                          const int32_t* visit, int32_t* meta) {
    __shared__ RbgsLds L;
    const int32_t n_ranges = (int32_t)(((int64_t)d + kAggRange - 1) / kAggRange);
    int32_t count = n_ranges;
    bool list = false;
    if (visit) {
        const int32_t m = meta[0];
        if (m >= 0) {
            count = m;
            list = true;
        }
    }
    for (int32_t vi = blockIdx.x; vi < count; vi += gridDim.x) {
        const int32_t r = list ? visit[vi] : vi;
        agg_rbgs_range<kApply>((int64_t)r * kAggRange, K, d, B, block_slot, val, val_row, f, meta + 1, L);
        __syncthreads();  // the range's LDS is free for the next
    }
}

hipError_t launch_agg_rbgs(int32_t K, int32_t d, int32_t B, int32_t n_sel, const int32_t* block_slot,
                           const float* val, int64_t val_row, const FinishArgs& f, const int32_t* visit,
                           int32_t* meta, hipStream_t st) {
    const int64_t n_ranges = ((int64_t)d + kAggRange - 1) / kAggRange;
    // a sparse apply that writes no dense update visits the drawn list: the
    // ranges of this step's and the last step's blocks
    const bool use_list = f.sparse_apply && f.w_out && !f.update;
    int64_t grid = n_ranges;
    if (use_list) {
        const int64_t per_block = ((int64_t)B + kAggRange - 1) / kAggRange + 1;
        const int64_t want = 2 * (int64_t)n_sel * per_block + 64;
        grid = want < n_ranges ? want : n_ranges;
    }
    const int32_t* vl = use_list ? visit : nullptr;
    if (f.w_out)
        hipLaunchKernelGGL(agg_rbgs_kernel<true>, dim3((unsigned)grid), dim3(kGroup), 0, st, K, d, B, block_slot,
                           val, val_row, f, vl, meta);
    else
        hipLaunchKernelGGL(agg_rbgs_kernel<false>, dim3((unsigned)grid), dim3(kGroup), 0, st, K, d, B, block_slot,
                           val, val_row, f, vl, meta);
    return hipGetLastError();
}

// ============================================================================
// GMC+ detached points, dense: y_k = w - q e_k (Algorithm 2, detach)
// ============================================================================

// One workgroup per (chunk of kChunk components, worker) in the fused pass's
// order: w is read through the cache by the K workgroups of a chunk, e_k and
// y_k are streamed.
__global__ __launch_bounds__(kGroup) void detach_kernel(DetachArgs a, int32_t K) {
    int chunk, k;
    run_order(blockIdx.x, K, 2, &chunk, &k);
    const int64_t start = (int64_t)chunk * kChunk;
    if (start >= a.d) return;  // padding of the run order
    const int64_t len = (int64_t)a.d - start < kChunk ? (int64_t)a.d - start : kChunk;
    const float* e = a.e[k];
    float* y = a.y[k];
    const float q = a.q;
    if (len == kChunk && aligned16(a.w) && aligned16(e) && aligned16(y)) {
#pragma unroll
        for (int i = 0; i < 2; ++i) {
            const int64_t j = start + i * (kGroup * 4) + threadIdx.x * 4;
            const float4 w = ld4(a.w + j), ev = ld4_stream(e + j);
            st4_stream(y + j, make_float4(detached(w.x, ev.x, q), detached(w.y, ev.y, q), detached(w.z, ev.z, q),
                                          detached(w.w, ev.w, q)));
        }
        return;
    }
    for (int64_t o = threadIdx.x; o < len; o += kGroup) y[start + o] = detached(a.w[start + o], e[start + o], q);
}

hipError_t launch_detach(const DetachArgs& a, int32_t K, hipStream_t st) {
    const int64_t chunks = ((int64_t)a.d + kChunk - 1) / kChunk;
    hipLaunchKernelGGL(detach_kernel, dim3((unsigned)run_order_grid(chunks, K, 2)), dim3(kGroup), 0,
                       st, a, K);
    return hipGetLastError();
}

// ============================================================================
// apply
// ============================================================================

__global__ __launch_bounds__(kGroup) void apply_kernel(int32_t d, float* w, float* w_prev_out,
                                                       const float* update) {
    const int64_t j = ((int64_t)blockIdx.x * kGroup + threadIdx.x) * 4;
    if (j >= d) return;
    const bool vec = j + 4 <= d && aligned16(w) && aligned16(update) &&
                     (w_prev_out == nullptr || aligned16(w_prev_out));
    if (vec) {
        const float4 x = ld4(w + j), u = ld4(update + j);
        if (w_prev_out) st4(w_prev_out + j, x);
        st4(w + j, make_float4(x.x + u.x, x.y + u.y, x.z + u.z, x.w + u.w));
        return;
    }
    for (int q = 0; q < 4 && j + q < d; ++q) {
        const float x = w[j + q];
        if (w_prev_out) w_prev_out[j + q] = x;
        w[j + q] = x + update[j + q];
    }
}

hipError_t launch_apply(int32_t d, float* w, float* w_prev_out, const float* update, hipStream_t st) {
    const int64_t threads = ((int64_t)d + 3) / 4;
    const int grid = (int)((threads + kGroup - 1) / kGroup);
    hipLaunchKernelGGL(apply_kernel, dim3(grid), dim3(kGroup), 0, st, d, w, w_prev_out, update);
    return hipGetLastError();
}

// ============================================================================
// plain copy, the reference for memory-counter calibration
// ============================================================================

__global__ __launch_bounds__(kGroup) void calib_copy_kernel(float* dst, const float* src, int64_t n) {
    const int64_t i = ((int64_t)blockIdx.x * kGroup + threadIdx.x) * 4;
    if (i + 4 <= n && aligned16(dst) && aligned16(src)) {
        st4(dst + i, ld4(src + i));
        return;
    }
    for (int64_t q = i; q < i + 4 && q < n; ++q) dst[q] = src[q];
}

hipError_t launch_calib_copy(float* dst, const float* src, int64_t n, hipStream_t st) {
    const int64_t threads = (n + 3) / 4;
    const int grid = (int)((threads + kGroup - 1) / kGroup);
    hipLaunchKernelGGL(calib_copy_kernel, dim3(grid), dim3(kGroup), 0, st, dst, src, n);
    return hipGetLastError();
}

}  // namespace gmc

namespace gmc {

// ============================================================================
// a plain stream in the fused worker pass's shape, the reference for how
// close that pass comes to what the memory system gives its access pattern
// ============================================================================

// e[k][j] = e[k][j] + g[k][j] for K rows of d components (row pitch `pitch`):
// two streamed reads and one streamed write per worker-element, one
// workgroup per (chunk of kChunk components, worker) in the fused pass's
// chunk-major order, 2 float4 per thread per row.
__global__ __launch_bounds__(kGroup) void calib_stream_kernel(float* e, const float* g, int64_t pitch, int32_t K,
                                                              int32_t d) {
    int chunk, k;
    run_order(blockIdx.x, K, 1, &chunk, &k);
    const int64_t start = (int64_t)chunk * kChunk;
    if (start >= d) return;
    const int64_t len = (int64_t)d - start < kChunk ? (int64_t)d - start : kChunk;
    float* ep = e + (int64_t)k * pitch + start;
    const float* gp = g + (int64_t)k * pitch + start;
    if (len == kChunk && aligned16(ep) && aligned16(gp)) {
        const int o0 = threadIdx.x * 4;
        float4 a[2], b[2];
#pragma unroll
        for (int i = 0; i < 2; ++i) {
            a[i] = ld4_stream(ep + o0 + i * (kGroup * 4));
            b[i] = ld4_stream(gp + o0 + i * (kGroup * 4));
        }
#pragma unroll
        for (int i = 0; i < 2; ++i)
            st4_stream(ep + o0 + i * (kGroup * 4),
                       make_float4(a[i].x + b[i].x, a[i].y + b[i].y, a[i].z + b[i].z, a[i].w + b[i].w));
        return;
    }
    for (int64_t o = threadIdx.x; o < len; o += kGroup) ep[o] = ep[o] + gp[o];
}

hipError_t launch_calib_stream(float* e, const float* g, int64_t pitch, int32_t K, int32_t d, hipStream_t st) {
    const int64_t chunks = ((int64_t)d + kChunk - 1) / kChunk;
    hipLaunchKernelGGL(calib_stream_kernel, dim3((unsigned)run_order_grid(chunks, K, 1)), dim3(kGroup), 0, st, e, g,
                       pitch, K, d);
    return hipGetLastError();
}

}  // namespace gmc
