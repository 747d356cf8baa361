/*
 * A plain C11 caller of the C ABI (include/gmc.h): no Python, no C++.  It
 * allocates its device buffers with the HIP runtime's C API, runs three GMC
 * iterations (Algorithm 1) of global top-s through gmc_iteration with the
 * sparse momentum term, and checks on the host what holds without a
 * reference: every message has k entries, strictly ascending and in range,
 * the sent values are the largest in magnitude (each at least every residual
 * component left unsent, which is u there), and the residual is +0 at the
 * sent components.  Exit status 0 when every check holds.
 */
#include <math.h>
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

#include <hip/hip_runtime_api.h>

#include "gmc.h"

#define D 100003
#define K 3

static int fail(const char* what) {
    fprintf(stderr, "gmc_from_c: %s\n", what);
    return 1;
}

/* a small deterministic generator for the inputs (xorshift64*) */
static uint64_t rng_state = 0x9e3779b97f4a7c15ull;
static float next_value(void) {
    rng_state ^= rng_state >> 12;
    rng_state ^= rng_state << 25;
    rng_state ^= rng_state >> 27;
    const uint64_t x = rng_state * 0x2545f4914f6cdd1dull;
    return (float)((double)(x >> 11) / 9007199254740992.0 - 0.5);
}

static uint32_t key_of(float x) {
    uint32_t b;
    memcpy(&b, &x, sizeof b);
    return b & 0x7fffffffu;
}

int main(void) {
    int ndev = 0;
    if (hipGetDeviceCount(&ndev) != hipSuccess || ndev < 1) return fail("no GPU");
    gmc_ctx* ctx = NULL;
    if (gmc_init(&ctx, D, K, GMC_TOPK_GLOBAL, 0.01, 0.9, 0.1, 7) != GMC_OK) return fail("gmc_init");
    if (gmc_set_option(ctx, GMC_OPT_SPARSE_MOMENTUM, 1) != GMC_OK) return fail("gmc_set_option");
    const int64_t ilen = gmc_index_len(ctx), mlen = gmc_message_len(ctx);
    const int64_t kk = gmc_count(D, 0.01);
    if (ilen != kk || mlen != kk) return fail("message sizes");

    float *w = NULL, *wp = NULL, *g = NULL, *e = NULL, *val = NULL;
    int32_t* idx = NULL;
    int64_t* len = NULL;
    if (hipMalloc((void**)&w, D * sizeof(float)) != hipSuccess || hipMalloc((void**)&wp, D * sizeof(float)) ||
        hipMalloc((void**)&g, (size_t)K * D * sizeof(float)) || hipMalloc((void**)&e, (size_t)K * D * sizeof(float)) ||
        hipMalloc((void**)&val, (size_t)K * mlen * sizeof(float)) ||
        hipMalloc((void**)&idx, (size_t)K * ilen * sizeof(int32_t)) || hipMalloc((void**)&len, K * sizeof(int64_t)))
        return fail("hipMalloc");
    float* h = (float*)malloc((size_t)K * D * sizeof(float));
    float* he = (float*)malloc((size_t)K * D * sizeof(float));
    float* hv = (float*)malloc((size_t)K * mlen * sizeof(float));
    int32_t* hi = (int32_t*)malloc((size_t)K * ilen * sizeof(int32_t));
    if (!h || !he || !hv || !hi) return fail("malloc");
    for (int64_t j = 0; j < D; ++j) h[j] = 0.01f * next_value();
    hipMemcpy(w, h, D * sizeof(float), hipMemcpyHostToDevice);
    hipMemcpy(wp, h, D * sizeof(float), hipMemcpyHostToDevice);
    hipMemset(e, 0, (size_t)K * D * sizeof(float));

    const float* grads[K];
    float* errs[K];
    for (int k = 0; k < K; ++k) {
        grads[k] = g + (size_t)k * D;
        errs[k] = e + (size_t)k * D;
    }
    for (int t = 0; t < 3; ++t) {
        for (int64_t j = 0; j < (int64_t)K * D; ++j) h[j] = next_value();
        hipMemcpy(g, h, (size_t)K * D * sizeof(float), hipMemcpyHostToDevice);
        /* w_{t+1} over w_{t-1}'s buffer; the two buffers swap roles */
        if (gmc_iteration(ctx, w, wp, grads, errs, idx, val, len) != GMC_OK) return fail(gmc_last_error(ctx));
        float* tmp = w;
        w = wp;
        wp = tmp;
    }
    if (hipDeviceSynchronize() != hipSuccess) return fail("device error");
    int64_t hl[K];
    hipMemcpy(hl, len, sizeof hl, hipMemcpyDeviceToHost);
    hipMemcpy(hi, idx, (size_t)K * ilen * sizeof(int32_t), hipMemcpyDeviceToHost);
    hipMemcpy(hv, val, (size_t)K * mlen * sizeof(float), hipMemcpyDeviceToHost);
    hipMemcpy(he, e, (size_t)K * D * sizeof(float), hipMemcpyDeviceToHost);
    for (int k = 0; k < K; ++k) {
        const int32_t* ik = hi + (size_t)k * ilen;
        const float* vk = hv + (size_t)k * mlen;
        const float* ek = he + (size_t)k * D;
        if (hl[k] != kk) return fail("message length");
        uint32_t min_sent = 0xffffffffu;
        for (int64_t q = 0; q < kk; ++q) {
            if (ik[q] < 0 || ik[q] >= D || (q > 0 && ik[q] <= ik[q - 1])) return fail("indices not ascending in range");
            if (ek[ik[q]] != 0.0f || signbit(ek[ik[q]])) return fail("residual not +0 at a sent component");
            if (key_of(vk[q]) < min_sent) min_sent = key_of(vk[q]);
        }
        /* every unsent component (u, kept in the residual) ranks below the
           sent ones: smaller key, or an equal key at a higher index than the
           last sent component of that key */
        for (int64_t j = 0; j < D; ++j) {
            if (key_of(ek[j]) > min_sent) return fail("an unsent component outranks a sent one");
        }
    }
    int64_t st[8] = {0};
    if (gmc_stats(ctx, st, 8) != GMC_OK || st[4] != 0) return fail("count check");
    gmc_destroy(ctx);
    hipFree(w);
    hipFree(wp);
    hipFree(g);
    hipFree(e);
    hipFree(val);
    hipFree(idx);
    hipFree(len);
    free(h);
    free(he);
    free(hv);
    free(hi);
    printf("gmc_from_c: 3 iterations, %d workers, k = %lld: every check holds\n", K, (long long)kk);
    return 0;
}
