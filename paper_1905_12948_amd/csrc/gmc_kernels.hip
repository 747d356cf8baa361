// HIP kernels of the GMC hot path for CDNA4 (gfx950, wave64).
//
// One iteration of Algorithm 1 (GMC) for K workers resident on one GPU:
//
//   topk_fused   u_k = (e_k + g_k) - c (w_t - w_prev) for every worker, written
//                over e_k; components whose magnitude key reaches the pair's
//                speculative threshold are appended to a candidate list
//   topk_hist    three radix-select passes (11 + 11 + 9 bits of the key) over
//                the candidates, or over all of u when the candidates cannot
//                prove they hold the top k; the last workgroup of each
//                (worker, segment) picks the digit
//   topk_count   per item counts above / at the threshold, then a scan over
//                the segment's items (last workgroup)
//   topk_emit    ordered compaction of the kept components into the message,
//                residual u - u at the kept components
//   rbgs_*       shared block draw and the fused pass that gathers whole blocks
//   agg_*        the server sum over workers in worker order, dense update
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

__device__ __forceinline__ bool aligned16(const void* p) {
    return (reinterpret_cast<uintptr_t>(p) & 15u) == 0;
}

// u = (e + g) - m, two roundings, in this order.
__device__ __forceinline__ float precompress(float e, float g, float m) {
    const float acc = e + g;
    return acc - m;
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

}  // namespace

// ============================================================================
// fused worker pass for top-s
// ============================================================================

// Candidate append of one wavefront-chunk for worker k.  `flags` holds, per
// lane, kIters*kPer bits (iteration-major) of components to append; the
// component of bit (i, q) is element `start + i*kWave*kPer + lane*kPer + q`,
// whose u value has just been stored to e[j] by this lane.
template <int kIters, int kPer, class Flags>
__device__ __forceinline__ void append_candidates(Flags flags, const float* e, int start, int lane,
                                                  const TopkGeometry& g, const TopkScratch& s, int k,
                                                  int chunk, int p) {
    const size_t run_slot = (size_t)k * g.n_chunks + chunk;
    if (ballot(flags != 0) == 0ull) {
        if (lane == 0) {
            s.run_off[run_slot] = 0u;
            s.run_cnt[run_slot] = 0u;
        }
        return;
    }
    // per-iteration exclusive lane prefix and iteration bases
    uint32_t lane_pre[kIters];
    uint32_t base = 0;
#pragma unroll
    for (int i = 0; i < kIters; ++i) {
        const uint32_t bits = (uint32_t)(flags >> (i * kPer)) & ((1u << kPer) - 1u);
        const uint32_t cnt = (uint32_t)__popc(bits);
        uint32_t tot, pre;
        if (kPer == 1) {
            const uint64_t b = ballot(cnt != 0u);
            pre = popc64(b & lanemask_lt());
            tot = popc64(b);
        } else {
            pre = wave_prefix_small(cnt, &tot);
        }
        lane_pre[i] = base + pre;
        base += tot;
    }
    const uint32_t total = base;
    uint32_t off = 0;
    if (lane == 0) off = atomicAdd(&s.pair[p].cand, total);
    off = __shfl(off, 0, kWave);
    if (lane == 0) {
        s.run_off[run_slot] = off;
        s.run_cnt[run_slot] = total;
    }
    const uint32_t cap = (uint32_t)g.pair_cap[p];
    if (off > cap || total > cap - off) return;  // overflow: the selection takes the full-data path
    int32_t* ci = s.cand_idx + g.pair_cand[p];
    float* cv = s.cand_val + g.pair_cand[p];
#pragma unroll
    for (int i = 0; i < kIters; ++i) {
        uint32_t bits = (uint32_t)(flags >> (i * kPer)) & ((1u << kPer) - 1u);
        uint32_t pos = off + lane_pre[i];
        while (bits) {
            const int q = __ffs(bits) - 1;
            bits &= bits - 1u;
            const int j = start + i * (kWave * kPer) + lane * kPer + q;
            ci[pos] = j;
            cv[pos] = e[j];  // re-read of this lane's own store
            ++pos;
        }
    }
}

// Vector path: full chunks whose start is a multiple of 4, workers
// whose g/e rows are 16-byte aligned (bit k of vec_mask), w_t/w_prev aligned.
__global__ __launch_bounds__(kGroup) void topk_fused_vec_kernel(StepArgs a, TopkGeometry g, TopkScratch s,
                                                                uint64_t vec_mask) {
    const int lane = threadIdx.x & (kWave - 1);
    const int wave = threadIdx.x >> 6;
    const int chunk = blockIdx.x * kWavesPerGroup + wave;
    if (chunk >= g.n_chunks) return;  // wave-uniform; no workgroup barrier below
    const int start = g.chunk_start[chunk];
    const int len = g.chunk_len[chunk];
    if ((start & 3) != 0 || len != kChunk) return;  // handled by the element-wise kernel
    const int seg = g.chunk_seg[chunk];
    const float c = a.c;
    const float* wt_p = a.w_t + start + lane * 4;
    const float* wp_p = a.w_prev + start + lane * 4;

    float4 m4[kVecIters];
#pragma unroll
    for (int i = 0; i < kVecIters; ++i) {
        const float4 wt = ld4(wt_p + i * (kWave * 4)), wp = ld4(wp_p + i * (kWave * 4));
        m4[i] = make_float4(c * (wt.x - wp.x), c * (wt.y - wp.y), c * (wt.z - wp.z), c * (wt.w - wp.w));
    }
#pragma unroll 1
    for (int k = 0; k < g.K; ++k) {
        if (!((vec_mask >> k) & 1ull)) continue;
        const int p = k * g.n_seg + seg;
        const uint32_t tau = s.pair[p].tau;
        float* e = a.wp.e[k];
        float* ep = e + start + lane * 4;
        const float* gp = a.wp.g[k] + start + lane * 4;
        float4 ev[kVecIters], gv[kVecIters];
#pragma unroll
        for (int i = 0; i < kVecIters; ++i) {
            ev[i] = ld4(ep + i * (kWave * 4));
            gv[i] = ld4(gp + i * (kWave * 4));
        }
        uint32_t flags = 0;
#pragma unroll
        for (int i = 0; i < kVecIters; ++i) {
            float4 u;
            u.x = precompress(ev[i].x, gv[i].x, m4[i].x);
            u.y = precompress(ev[i].y, gv[i].y, m4[i].y);
            u.z = precompress(ev[i].z, gv[i].z, m4[i].z);
            u.w = precompress(ev[i].w, gv[i].w, m4[i].w);
            st4(ep + i * (kWave * 4), u);
            flags |= (key_of(u.x) >= tau ? 1u : 0u) << (i * 4 + 0);
            flags |= (key_of(u.y) >= tau ? 1u : 0u) << (i * 4 + 1);
            flags |= (key_of(u.z) >= tau ? 1u : 0u) << (i * 4 + 2);
            flags |= (key_of(u.w) >= tau ? 1u : 0u) << (i * 4 + 3);
        }
        append_candidates<kVecIters, 4>(flags, e, start, lane, g, s, k, chunk, p);
    }
}

// Element-wise path for the (chunk, worker) pairs the vector kernel skips:
// partial chunks (a segment's last) and chunks with an unaligned start, and
// workers (or w) whose rows are not 16-byte aligned.  `list` holds the
// chunk ids to visit (NULL: every chunk).
__global__ __launch_bounds__(kGroup) void topk_fused_gen_kernel(StepArgs a, TopkGeometry g, TopkScratch s,
                                                                uint64_t vec_mask, const int32_t* list,
                                                                int32_t n_list) {
    const int lane = threadIdx.x & (kWave - 1);
    const int wave = threadIdx.x >> 6;
    const int li = blockIdx.x * kWavesPerGroup + wave;
    if (li >= n_list) return;
    const int chunk = list ? list[li] : li;
    const int start = g.chunk_start[chunk];
    const int len = g.chunk_len[chunk];
    const bool regular = (start & 3) == 0 && len == kChunk;
    const int seg = g.chunk_seg[chunk];
    const float c = a.c;
    constexpr int kIt = kChunk / kWave;  // 32
    for (int k = 0; k < g.K; ++k) {
        if (regular && ((vec_mask >> k) & 1ull)) continue;  // the vector kernel did this one
        const int p = k * g.n_seg + seg;
        const uint32_t tau = s.pair[p].tau;
        float* e = a.wp.e[k];
        const float* gr = a.wp.g[k];
        uint32_t flags = 0;
#pragma unroll 4
        for (int i = 0; i < kIt; ++i) {
            const int o = i * kWave + lane;
            if (o < len) {
                const int j = start + o;
                const float m = c * (a.w_t[j] - a.w_prev[j]);
                const float u = precompress(e[j], gr[j], m);
                e[j] = u;
                flags |= (key_of(u) >= tau ? 1u : 0u) << i;
            }
        }
        append_candidates<kIt, 1>(flags, e, start, lane, g, s, k, chunk, p);
    }
}

hipError_t launch_topk_fused(const StepArgs& a, const TopkGeometry& g, const TopkScratch& s, uint64_t vec_mask,
                             const int32_t* gen_list, int32_t n_gen, hipStream_t st) {
    if (vec_mask) {
        const int grid = (g.n_chunks + kWavesPerGroup - 1) / kWavesPerGroup;
        hipLaunchKernelGGL(topk_fused_vec_kernel, dim3(grid), dim3(kGroup), 0, st, a, g, s, vec_mask);
        hipError_t e = hipGetLastError();
        if (e != hipSuccess) return e;
    }
    if (n_gen > 0) {
        const int grid = (n_gen + kWavesPerGroup - 1) / kWavesPerGroup;
        hipLaunchKernelGGL(topk_fused_gen_kernel, dim3(grid), dim3(kGroup), 0, st, a, g, s, vec_mask, gen_list,
                           n_gen);
    }
    return hipGetLastError();
}

// ============================================================================
// selection: item iteration helpers
// ============================================================================

namespace {

// The elements of one item in ascending index order: either the candidate
// runs of its chunks (mode 0) or the raw residual range (mode 1).
struct ItemView {
    int mode;
    int32_t total;          // elements in the item
    // mode 0
    const int32_t* cidx;    // candidate region of the pair
    const float* cval;
    // mode 1
    const float* u;         // worker's u (held in e)
    int32_t lo;             // first element index of the item
    int32_t nch;            // chunks in the item
};

// Shared memory for an item's run table (mode 0).
struct ItemShared {
    uint32_t flat[kItemChunks + 1];  // exclusive prefix of run counts
    uint32_t roff[kItemChunks];
    uint32_t wsum[kWavesPerGroup];
};

__device__ ItemView open_item(int mode, int k, int it, int p, const StepArgs& a, const TopkGeometry& g,
                              const TopkScratch& s, ItemShared& sh) {
    ItemView v;
    v.mode = mode;
    const int clo = g.item_chunk_lo[it], chi = g.item_chunk_hi[it];
    v.nch = chi - clo;
    if (mode == 0) {
        v.cidx = s.cand_idx + g.pair_cand[p];
        v.cval = s.cand_val + g.pair_cand[p];
        v.u = nullptr;
        v.lo = 0;
        if (threadIdx.x < kWave) {
            const int lane = threadIdx.x;
            uint32_t cnt = 0, off = 0;
            if (lane < v.nch) {
                const size_t slot = (size_t)k * g.n_chunks + clo + lane;
                cnt = s.run_cnt[slot];
                off = s.run_off[slot];
            }
            uint32_t x = cnt;
#pragma unroll
            for (int o = 1; o < kWave; o <<= 1) {
                const uint32_t y = __shfl_up(x, o, kWave);
                if (lane >= o) x += y;
            }
            if (lane < v.nch) {
                sh.flat[lane] = x - cnt;
                sh.roff[lane] = off;
            }
            if (lane == v.nch - 1) sh.flat[v.nch] = x;
        }
        __syncthreads();
        v.total = (int32_t)sh.flat[v.nch];
    } else {
        v.cidx = nullptr;
        v.cval = nullptr;
        v.u = a.wp.e[k];
        v.lo = g.chunk_start[clo];
        v.total = g.chunk_start[chi - 1] + g.chunk_len[chi - 1] - v.lo;
    }
    return v;
}

// Element at flat position pos (< total): value and global index.
__device__ __forceinline__ float item_get(const ItemView& v, const ItemShared& sh, int32_t pos, int32_t* j) {
    if (v.mode == 1) {
        *j = v.lo + pos;
        return v.u[v.lo + pos];
    }
    // largest c with flat[c] <= pos
    int lo = 0, hi = v.nch - 1;
    while (lo < hi) {
        const int mid = (lo + hi + 1) >> 1;
        if (sh.flat[mid] <= (uint32_t)pos) lo = mid; else hi = mid - 1;
    }
    const uint32_t cpos = sh.roff[lo] + ((uint32_t)pos - sh.flat[lo]);
    *j = v.cidx[cpos];
    return v.cval[cpos];
}

// Finds the bin b (scanning from the top) with above(b) < need <= above(b) +
// h[b], where above(b) = sum of bins above b.  h is in shared memory with
// nbins entries (a multiple of kGroup).  Returns b and *above (all threads).
__device__ int find_bin(const uint32_t* h, int nbins, uint32_t need, uint32_t* above_out,
                        uint32_t* sh_scan, int* sh_res) {
    const int per = nbins / kGroup;
    // thread t owns bins [t*per, (t+1)*per); suffix order: thread 255 first
    const int t = threadIdx.x;
    uint32_t mine = 0;
    for (int q = 0; q < per; ++q) mine += h[t * per + q];
    // exclusive scan in reverse thread order
    const int rt = kGroup - 1 - t;
    // scan over reversed index: use LDS array
    sh_scan[rt] = mine;
    __syncthreads();
    if (t == 0) {
        uint32_t run = 0;
        for (int i = 0; i < kGroup; ++i) {
            const uint32_t x = sh_scan[i];
            sh_scan[i] = run;
            run += x;
        }
    }
    __syncthreads();
    uint32_t above = sh_scan[rt];
    if (t == 0) sh_res[0] = -1;
    __syncthreads();
    for (int q = per - 1; q >= 0; --q) {
        const uint32_t hb = h[t * per + q];
        if (above < need && need <= above + hb) {
            sh_res[0] = t * per + q;
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

}  // namespace

// ============================================================================
// selection: histogram passes
// ============================================================================

template <int PASS>
__global__ __launch_bounds__(kGroup) void topk_hist_kernel(StepArgs a, TopkGeometry g, TopkScratch s,
                                                           int force_full, int margin) {
    constexpr int nbins = PASS == 3 ? 512 : kBins;
    __shared__ uint32_t h[kBins];
    __shared__ ItemShared ish;
    __shared__ uint32_t sh_scan[kGroup];
    __shared__ int sh_res[2];
    __shared__ int sh_last;

    const int k = blockIdx.x / g.n_items;
    const int it = blockIdx.x % g.n_items;
    const int seg = g.item_seg[it];
    const int p = k * g.n_seg + seg;
    PairState* ps = &s.pair[p];
    const int kp = g.pair_k[p];

    int mode;
    uint32_t cand = 0;
    if (PASS == 1) {
        cand = ps->cand;
        mode = (force_full || cand < (uint32_t)kp || cand > (uint32_t)g.pair_cap[p]) ? 1 : 0;
    } else {
        mode = ps->mode;
    }
    const uint32_t prefix = PASS == 1 ? 0u : ps->prefix;

    for (int b = threadIdx.x; b < nbins; b += kGroup) h[b] = 0u;
    ItemView v = open_item(mode, k, it, p, a, g, s, ish);  // contains a barrier
    __syncthreads();

    for (int32_t pos = threadIdx.x; pos < v.total; pos += kGroup) {
        int32_t j;
        const uint32_t key = key_of(item_get(v, ish, pos, &j));
        if (PASS == 1) {
            atomicAdd(&h[key >> kShift1], 1u);
        } else if (PASS == 2) {
            if ((key >> kShift1) == prefix) atomicAdd(&h[(key >> kShift2) & (kBins - 1)], 1u);
        } else {
            if ((key >> kShift2) == prefix) atomicAdd(&h[key & 511u], 1u);
        }
    }
    __syncthreads();

    uint32_t* gh = s.hist + (size_t)p * kBins;
    for (int b = threadIdx.x; b < nbins; b += kGroup)
        if (h[b]) atomicAdd(&gh[b], h[b]);
    __threadfence();
    __syncthreads();
    if (threadIdx.x == 0) {
        const uint32_t prev = atomicAdd(&ps->done, 1u);
        sh_last = prev == (uint32_t)g.seg_items[seg] - 1u;
    }
    __syncthreads();
    if (!sh_last) return;
    __threadfence();

    // last workgroup of this (worker, segment): read and clear the histogram
    for (int b = threadIdx.x; b < nbins; b += kGroup) {
        h[b] = __hip_atomic_load(&gh[b], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        __hip_atomic_store(&gh[b], 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    }
    __syncthreads();
    const uint32_t need = PASS == 1 ? (uint32_t)kp : (uint32_t)ps->need;
    uint32_t above = 0;
    const int bin = find_bin(h, nbins, need, &above, sh_scan, sh_res);

    if (PASS == 1) {
        // speculative threshold for the next step: the lowest bin down to
        // which at least margin*k components were counted this step
        uint32_t total = 0;
        for (int b = threadIdx.x; b < nbins; b += kGroup) total += h[b];
        // reduce total across the block (reuse sh_scan)
        sh_scan[threadIdx.x] = total;
        __syncthreads();
        if (threadIdx.x == 0) {
            uint32_t t = 0;
            for (int i = 0; i < kGroup; ++i) t += sh_scan[i];
            sh_scan[0] = t;
        }
        __syncthreads();
        total = sh_scan[0];
        __syncthreads();
        const uint64_t want64 = (uint64_t)margin * (uint64_t)kp;
        const uint32_t want = (uint32_t)(want64 < total ? want64 : total);
        uint32_t ab2 = 0;
        int tb = find_bin(h, nbins, want, &ab2, sh_scan, sh_res);
        if (threadIdx.x == 0) {
            if (want64 > total && tb > 0) --tb;  // too few counted: widen by one bin
            if (tb < 0) tb = 0;
            ps->tau = (uint32_t)tb << kShift1;
            ps->mode = mode;
            ps->cand = 0u;
            atomicAdd((unsigned long long*)&s.stats[mode == 0 ? 1 : 2], 1ull);
            if (mode == 0) atomicAdd((unsigned long long*)&s.stats[3], (unsigned long long)cand);
        }
    }
    if (threadIdx.x == 0) {
        if (bin < 0) {
            atomicAdd((unsigned long long*)&s.stats[4], 1ull);  // cannot happen for valid counts
        }
        const uint32_t b = bin < 0 ? 0u : (uint32_t)bin;
        if (PASS == 1) {
            ps->prefix = b;
            ps->need = (int32_t)(need - above);
        } else if (PASS == 2) {
            ps->prefix = (prefix << 11) | b;
            ps->need = (int32_t)(need - above);
        } else {
            ps->T = (prefix << 9) | b;
            ps->r = (int32_t)(need - above);
        }
        __hip_atomic_store(&ps->done, 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    }
}

hipError_t launch_topk_hist(int pass, const StepArgs& a, const TopkGeometry& g,
                            const TopkScratch& s, int force_full, int margin, hipStream_t st) {
    const int grid = g.K * g.n_items;
    if (pass == 1)
        hipLaunchKernelGGL(topk_hist_kernel<1>, dim3(grid), dim3(kGroup), 0, st, a, g, s, force_full, margin);
    else if (pass == 2)
        hipLaunchKernelGGL(topk_hist_kernel<2>, dim3(grid), dim3(kGroup), 0, st, a, g, s, force_full, margin);
    else
        hipLaunchKernelGGL(topk_hist_kernel<3>, dim3(grid), dim3(kGroup), 0, st, a, g, s, force_full, margin);
    return hipGetLastError();
}

// ============================================================================
// selection: per-item counts and the scan over a segment's items
// ============================================================================

__global__ __launch_bounds__(kGroup) void topk_count_kernel(StepArgs a, TopkGeometry g, TopkScratch s,
                                                            int64_t* msg_len, int64_t msg_total) {
    __shared__ ItemShared ish;
    __shared__ uint32_t red[2][kWavesPerGroup];
    __shared__ int sh_last;
    __shared__ uint32_t carry[3];

    const int k = blockIdx.x / g.n_items;
    const int it = blockIdx.x % g.n_items;
    const int seg = g.item_seg[it];
    const int p = k * g.n_seg + seg;
    PairState* ps = &s.pair[p];
    const int mode = ps->mode;
    const uint32_t T = ps->T;

    ItemView v = open_item(mode, k, it, p, a, g, s, ish);
    uint32_t above = 0, ties = 0;
    for (int32_t pos = threadIdx.x; pos < v.total; pos += kGroup) {
        int32_t j;
        const uint32_t key = key_of(item_get(v, ish, pos, &j));
        above += key > T;
        ties += key == T;
    }
    // block reduce
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
    const size_t slot = (size_t)k * g.n_items + it;
    if (threadIdx.x == 0) {
        uint32_t A = 0, Ti = 0;
        for (int w = 0; w < kWavesPerGroup; ++w) {
            A += red[0][w];
            Ti += red[1][w];
        }
        s.item_above[slot] = A;
        s.item_ties[slot] = Ti;
    }
    __threadfence();
    __syncthreads();
    if (threadIdx.x == 0) {
        const uint32_t prev = atomicAdd(&ps->done, 1u);
        sh_last = prev == (uint32_t)g.seg_items[seg] - 1u;
    }
    __syncthreads();
    if (!sh_last) return;
    __threadfence();

    // last workgroup of the pair: scan the segment's items in index order
    const int n = g.seg_items[seg];
    const size_t base = (size_t)k * g.n_items + g.seg_item_lo[seg];
    const int32_t r = ps->r;
    if (threadIdx.x == 0) {
        carry[0] = 0;  // ties before
        carry[1] = 0;  // selected before
        carry[2] = 0;
    }
    __syncthreads();
    __shared__ uint32_t wsum[kWavesPerGroup];
    for (int c0 = 0; c0 < n; c0 += kGroup) {
        const int i = c0 + threadIdx.x;
        uint32_t A = 0, Ti = 0;
        if (i < n) {
            A = __hip_atomic_load(&s.item_above[base + i], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
            Ti = __hip_atomic_load(&s.item_ties[base + i], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        }
        uint32_t tot_t;
        const uint32_t tie_pre = carry[0] + block_scan_excl(Ti, &tot_t, wsum);
        int64_t take = (int64_t)r - (int64_t)tie_pre;
        if (take < 0) take = 0;
        if (take > (int64_t)Ti) take = Ti;
        const uint32_t sel = A + (uint32_t)take;
        uint32_t tot_s;
        const uint32_t sel_pre = carry[1] + block_scan_excl(sel, &tot_s, wsum);
        if (i < n) {
            s.item_tiebase[base + i] = tie_pre;
            s.item_out[base + i] = sel_pre;
        }
        __syncthreads();
        if (threadIdx.x == 0) {
            carry[0] += tot_t;
            carry[1] += tot_s;
        }
        __syncthreads();
    }
    if (threadIdx.x == 0) {
        if (carry[1] != (uint32_t)g.pair_k[p]) atomicAdd((unsigned long long*)&s.stats[4], 1ull);
        if (seg == 0) msg_len[k] = msg_total;
        __hip_atomic_store(&ps->done, 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    }
}

hipError_t launch_topk_count(const StepArgs& a, const TopkGeometry& g, const TopkScratch& s,
                             int64_t* msg_len, int64_t msg_total, hipStream_t st) {
    hipLaunchKernelGGL(topk_count_kernel, dim3(g.K * g.n_items), dim3(kGroup), 0, st, a, g, s,
                       msg_len, msg_total);
    return hipGetLastError();
}

// ============================================================================
// selection: ordered emission of the kept components
// ============================================================================

__global__ __launch_bounds__(kGroup) void topk_emit_kernel(StepArgs a, TopkGeometry g, TopkScratch s,
                                                           int32_t* idx, float* val, int64_t row_len) {
    __shared__ ItemShared ish;
    __shared__ uint32_t wcnt[2][kWavesPerGroup];

    const int k = blockIdx.x / g.n_items;
    const int it = blockIdx.x % g.n_items;
    const int seg = g.item_seg[it];
    const int p = k * g.n_seg + seg;
    const PairState* ps = &s.pair[p];
    const int mode = ps->mode;
    const uint32_t T = ps->T;
    const int64_t r = ps->r;
    const size_t slot = (size_t)k * g.n_items + it;
    const uint32_t out0 = s.item_out[slot];
    const int64_t tiebase = s.item_tiebase[slot];
    int64_t ties_quota = r - tiebase;
    if (ties_quota < 0) ties_quota = 0;

    const uint32_t kseg = (uint32_t)g.pair_k[p];
    int32_t* irow = idx + (size_t)k * row_len + g.seg_out[seg];
    float* vrow = val + (size_t)k * row_len + g.seg_out[seg];
    float* e = a.wp.e[k];

    ItemView v = open_item(mode, k, it, p, a, g, s, ish);
    const int lane = threadIdx.x & (kWave - 1), wave = threadIdx.x >> 6;
    uint32_t run_above = 0, run_ties = 0;
    for (int32_t b0 = 0; b0 < v.total; b0 += kGroup) {
        const int32_t pos = b0 + threadIdx.x;
        bool is_above = false, is_tie = false;
        int32_t j = 0;
        float x = 0.0f;
        if (pos < v.total) {
            x = item_get(v, ish, pos, &j);
            const uint32_t key = key_of(x);
            is_above = key > T;
            is_tie = key == T;
        }
        const uint64_t am = ballot(is_above), tm = ballot(is_tie);
        if (lane == 0) {
            wcnt[0][wave] = popc64(am);
            wcnt[1][wave] = popc64(tm);
        }
        __syncthreads();
        uint32_t a_before = run_above + popc64(am & lanemask_lt());
        uint32_t t_before = run_ties + popc64(tm & lanemask_lt());
        uint32_t a_tot = 0, t_tot = 0;
#pragma unroll
        for (int w = 0; w < kWavesPerGroup; ++w) {
            if (w < wave) {
                a_before += wcnt[0][w];
                t_before += wcnt[1][w];
            }
            a_tot += wcnt[0][w];
            t_tot += wcnt[1][w];
        }
        __syncthreads();
        const bool take = is_above || (is_tie && (int64_t)t_before < ties_quota);
        if (take) {
            const int64_t taken_ties = (int64_t)t_before < ties_quota ? (int64_t)t_before : ties_quota;
            const uint32_t o = out0 + a_before + (uint32_t)taken_ties;
            if (o < kseg) {  // always true when the counts are consistent
                irow[o] = j;
                vrow[o] = x;
                e[j] = x - x;  // residual u - C(u) at a kept component
            }
        }
        run_above += a_tot;
        run_ties += t_tot;
    }
}

hipError_t launch_topk_emit(const StepArgs& a, const TopkGeometry& g, const TopkScratch& s,
                            int32_t* idx, float* val, int64_t row_len, hipStream_t st) {
    hipLaunchKernelGGL(topk_emit_kernel, dim3(g.K * g.n_items), dim3(kGroup), 0, st, a, g, s, idx, val,
                       row_len);
    return hipGetLastError();
}

// ============================================================================
// RBGS: block draw shared by all workers, fused gather pass
// ============================================================================

namespace {

__device__ __forceinline__ uint64_t splitmix64_mix(uint64_t z) {
    z = (z ^ (z >> 30)) * 0xbf58476d1ce4e5b9ull;
    z = (z ^ (z >> 27)) * 0x94d049bb133111ebull;
    return z ^ (z >> 31);
}

constexpr int kLdsBitmapWords = 8192;  // 262144 blocks

}  // namespace

// One workgroup.  Floyd's algorithm (one lane; the draws are sequential by
// definition) marks n_sel of nb blocks in a bitmap; the workgroup then
// compacts the bitmap into the ascending block list and the block -> slot map.
__global__ __launch_bounds__(kGroup) void rbgs_sample_kernel(uint64_t seed, uint64_t t, int32_t nb,
                                                             int32_t n_sel, int32_t d, int32_t B,
                                                             int32_t K, uint32_t* gbitmap,
                                                             int32_t* blocks, int32_t* block_slot,
                                                             int32_t* idx, int64_t idx_row,
                                                             int64_t* msg_len) {
    __shared__ uint32_t lbits[kLdsBitmapWords];
    __shared__ uint32_t wsum[kWavesPerGroup];
    __shared__ uint32_t carry;
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
    __threadfence();
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
}

hipError_t launch_rbgs_sample(uint64_t seed, uint64_t t, int32_t nb, int32_t n_sel, int32_t d,
                              int32_t B, int32_t K, uint32_t* bitmap, int32_t* blocks,
                              int32_t* block_slot, int32_t* idx, int64_t idx_row,
                              int64_t* msg_len, hipStream_t st) {
    hipLaunchKernelGGL(rbgs_sample_kernel, dim3(1), dim3(kGroup), 0, st, seed, t, nb, n_sel, d, B, K,
                       bitmap, blocks, block_slot, idx, idx_row, msg_len);
    return hipGetLastError();
}

// Each thread owns 4 consecutive elements per iteration; a selected block's
// components are copied to the message at slot*B + offset (every selected
// block but the last is full, so this is the concatenation in block order).
__global__ __launch_bounds__(kGroup) void rbgs_fused_kernel(StepArgs a, int32_t K, int32_t B,
                                                            const int32_t* block_slot, float* val,
                                                            int64_t val_row) {
    const int32_t d = a.d;
    const int64_t j0 = ((int64_t)blockIdx.x * kGroup + threadIdx.x) * 4;
    if (j0 >= d) return;
    const float c = a.c;
    const bool full = j0 + 4 <= d;
    const bool vec = full && (B & 3) == 0 && aligned16(a.w_t) && aligned16(a.w_prev) && aligned16(val) &&
                     (val_row & 3) == 0;
    if (vec) {
        const int32_t j = (int32_t)j0;
        const int32_t b = j / B;
        const int32_t slot = block_slot[b];
        const float4 wt = ld4(a.w_t + j), wp = ld4(a.w_prev + j);
        const float4 m = make_float4(c * (wt.x - wp.x), c * (wt.y - wp.y), c * (wt.z - wp.z), c * (wt.w - wp.w));
        const int64_t vpos = (int64_t)slot * B + (j - (int64_t)b * B);
        for (int k = 0; k < K; ++k) {
            float* e = a.wp.e[k];
            const float* gr = a.wp.g[k];
            if (aligned16(e) && aligned16(gr)) {
                const float4 ev = ld4(e + j), gv = ld4(gr + j);
                float4 u;
                u.x = precompress(ev.x, gv.x, m.x);
                u.y = precompress(ev.y, gv.y, m.y);
                u.z = precompress(ev.z, gv.z, m.z);
                u.w = precompress(ev.w, gv.w, m.w);
                if (slot >= 0) {
                    st4(val + (size_t)k * val_row + vpos, u);
                    st4(e + j, make_float4(u.x - u.x, u.y - u.y, u.z - u.z, u.w - u.w));
                } else {
                    st4(e + j, u);
                }
            } else {
                const float mm[4] = {m.x, m.y, m.z, m.w};
                for (int q = 0; q < 4; ++q) {
                    const float u = precompress(e[j + q], gr[j + q], mm[q]);
                    if (slot >= 0) {
                        val[(size_t)k * val_row + vpos + q] = u;
                        e[j + q] = u - u;
                    } else {
                        e[j + q] = u;
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
        const float m = c * (a.w_t[j] - a.w_prev[j]);
        const int64_t vpos = (int64_t)slot * B + (j - (int64_t)b * B);
        for (int k = 0; k < K; ++k) {
            float* e = a.wp.e[k];
            const float u = precompress(e[j], a.wp.g[k][j], m);
            if (slot >= 0) {
                val[(size_t)k * val_row + vpos] = u;
                e[j] = u - u;
            } else {
                e[j] = u;
            }
        }
    }
}

hipError_t launch_rbgs_fused(const StepArgs& a, int32_t K, int32_t B, const int32_t* block_slot,
                             float* val, int64_t val_row, hipStream_t st) {
    const int64_t threads = ((int64_t)a.d + 3) / 4;
    const int grid = (int)((threads + kGroup - 1) / kGroup);
    hipLaunchKernelGGL(rbgs_fused_kernel, dim3(grid), dim3(kGroup), 0, st, a, K, B, block_slot, val, val_row);
    return hipGetLastError();
}

// ============================================================================
// server: sum over workers in worker order, dense update
// ============================================================================

// rowptr[k][r] = first message position of worker k whose index falls in
// range r (ranges of kAggRange elements); rowptr[k][n_ranges] = length.
// Out-of-range or non-ascending indices cannot make it write outside rowptr.
__global__ __launch_bounds__(kGroup) void agg_rowptr_kernel(int32_t K, int32_t d, const int32_t* idx,
                                                            int64_t idx_row, const int64_t* msg_len,
                                                            int32_t* rowptr, int32_t n_ranges) {
    const int k = blockIdx.y;
    const int64_t i = (int64_t)blockIdx.x * kGroup + threadIdx.x;
    int64_t L = msg_len[k];
    if (L < 0) L = 0;
    if (L > idx_row) L = idx_row;
    int32_t* rp = rowptr + (size_t)k * (n_ranges + 1);
    auto range_of = [&](int64_t q) -> int64_t {
        int64_t x = idx[(size_t)k * idx_row + q];
        if (x < 0) x = 0;
        if (x >= d) x = d - 1;
        return x / kAggRange;
    };
    if (L == 0) {
        if (i == 0)
            for (int32_t rr = 0; rr <= n_ranges; ++rr) rp[rr] = 0;
        return;
    }
    if (i >= L) return;
    const int64_t rc = range_of(i);
    const int64_t rprev = i == 0 ? -1 : range_of(i - 1);
    for (int64_t rr = rprev + 1; rr <= rc; ++rr) rp[rr] = (int32_t)i;
    if (i == L - 1)
        for (int64_t rr = (rc > rprev ? rc : rprev) + 1; rr <= n_ranges; ++rr) rp[rr] = (int32_t)L;
}

hipError_t launch_agg_rowptr(int32_t K, int32_t d, const int32_t* idx, int64_t idx_row,
                             const int64_t* msg_len, int32_t* rowptr, int32_t n_ranges,
                             hipStream_t st) {
    const int gx = (int)((idx_row + kGroup - 1) / kGroup);
    hipLaunchKernelGGL(agg_rowptr_kernel, dim3(gx > 0 ? gx : 1, K), dim3(kGroup), 0, st, K, d, idx, idx_row,
                       msg_len, rowptr, n_ranges);
    return hipGetLastError();
}

__global__ __launch_bounds__(kGroup) void agg_topk_kernel(int32_t K, int32_t d, float s, const int32_t* idx,
                                                          int64_t idx_row, const float* val, int64_t val_row,
                                                          const int32_t* rowptr, int32_t n_ranges,
                                                          float* update) {
    __shared__ float acc[kAggRange];
    const int r = blockIdx.x;
    const int64_t base = (int64_t)r * kAggRange;
    for (int q = threadIdx.x; q < kAggRange; q += kGroup) acc[q] = 0.0f;
    __syncthreads();
    for (int k = 0; k < K; ++k) {
        const int32_t* rp = rowptr + (size_t)k * (n_ranges + 1);
        int32_t lo = rp[r], hi = rp[r + 1];
        for (int32_t i = lo + threadIdx.x; i < hi; i += kGroup) {
            const int64_t j = (int64_t)idx[(size_t)k * idx_row + i] - base;
            if (j >= 0 && j < kAggRange) acc[j] = acc[j] + val[(size_t)k * val_row + i];
        }
        __syncthreads();  // worker k's additions land before worker k+1's
    }
    const int64_t n = (int64_t)d - base < kAggRange ? (int64_t)d - base : kAggRange;
    if (n == kAggRange && aligned16(update) && (base & 3) == 0) {
        for (int q = threadIdx.x * 4; q < kAggRange; q += kGroup * 4)
            st4(update + base + q, make_float4(-(s * acc[q]), -(s * acc[q + 1]), -(s * acc[q + 2]), -(s * acc[q + 3])));
    } else {
        for (int q = threadIdx.x; q < n; q += kGroup) update[base + q] = -(s * acc[q]);
    }
}

hipError_t launch_agg_topk(int32_t K, int32_t d, float s, const int32_t* idx, int64_t idx_row,
                           const float* val, int64_t val_row, const int32_t* rowptr,
                           int32_t n_ranges, float* update, hipStream_t st) {
    hipLaunchKernelGGL(agg_topk_kernel, dim3(n_ranges), dim3(kGroup), 0, st, K, d, s, idx, idx_row, val,
                       val_row, rowptr, n_ranges, update);
    return hipGetLastError();
}

// RBGS: every worker sent the same blocks (ascending ids in blocks[0..n_sel));
// a component of block blocks[q] sits at q*B + offset in each message.
__global__ __launch_bounds__(kGroup) void agg_rbgs_kernel(int32_t K, int32_t d, int32_t B, float s,
                                                          const int32_t* blocks, int32_t n_sel,
                                                          const float* val, int64_t val_row,
                                                          float* update) {
    const int64_t j = (int64_t)blockIdx.x * kGroup + threadIdx.x;
    if (j >= d) return;
    const int32_t b = (int32_t)(j / B);
    // binary search for b among the ascending block ids
    int lo = 0, hi = n_sel - 1, slot = -1;
    while (lo <= hi) {
        const int mid = (lo + hi) >> 1;
        const int32_t x = blocks[mid];
        if (x == b) {
            slot = mid;
            break;
        }
        if (x < b) lo = mid + 1; else hi = mid - 1;
    }
    float acc = 0.0f;
    if (slot >= 0) {
        const int64_t vpos = (int64_t)slot * B + (j - (int64_t)b * B);
        for (int k = 0; k < K; ++k) acc = acc + val[(size_t)k * val_row + vpos];
    }
    update[j] = -(s * acc);
}

hipError_t launch_agg_rbgs(int32_t K, int32_t d, int32_t B, float s, const int32_t* blocks,
                           int32_t n_sel, const float* val, int64_t val_row, float* update,
                           hipStream_t st) {
    const int grid = (int)(((int64_t)d + kGroup - 1) / kGroup);
    hipLaunchKernelGGL(agg_rbgs_kernel, dim3(grid), dim3(kGroup), 0, st, K, d, B, s, blocks, n_sel, val, val_row,
                       update);
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

}  // namespace gmc
