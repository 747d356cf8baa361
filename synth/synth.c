/*
 * Seeded synthetic inputs for the GMC hot path: parameter vectors and
 * per-worker stochastic gradients with the shapes and value distributions of
 * the workloads (Gaussian, Student-t built from normals, per-tensor scales,
 * per-worker fixed mean shifts).
 *
 * This file holds no arithmetic of the method itself.  It is the one module
 * that both the device path and the CPU oracle draw their inputs from, so
 * that both sides see the same bits.
 *
 * Every value is a pure function of (seed, stream, element index): the
 * output does not depend on the number of threads or on how a vector is
 * split into calls.  Hashing uses the 64-bit finaliser of MurmurHash3
 * (Appleby); normals use the Box-Muller transform in double precision and
 * are rounded to binary32 once, at the end.
 */
#include <math.h>
#include <stdint.h>
#include <stddef.h>

#ifdef _OPENMP
#include <omp.h>
#endif

static inline uint64_t fmix64(uint64_t k)
{
    k ^= k >> 33;
    k *= 0xff51afd7ed558ccdULL;
    k ^= k >> 33;
    k *= 0xc4ceb9fe1a85ec53ULL;
    k ^= k >> 33;
    return k;
}

static inline uint64_t stream_key(uint64_t seed, uint64_t stream)
{
    return fmix64(seed ^ fmix64(stream ^ 0x5bd1e9955bd1e995ULL));
}

/* 64 random bits for counter i of a stream. */
static inline uint64_t bits_at(uint64_t key, uint64_t i)
{
    return fmix64(key + (i + 1) * 0x9e3779b97f4a7c15ULL);
}

/* Uniform on the open interval (0, 1) with 53 random bits. */
static inline double unif_open(uint64_t x)
{
    return ((double)(x >> 11) + 0.5) * (1.0 / 9007199254740992.0);
}

/* Standard normal number i of the stream: pair p = i/2 of Box-Muller. */
static inline double normal_at(uint64_t key, uint64_t i)
{
    const double two_pi = 6.283185307179586476925286766559;
    uint64_t p = i >> 1;
    double u1 = unif_open(bits_at(key, 2 * p));
    double u2 = unif_open(bits_at(key, 2 * p + 1));
    double r = sqrt(-2.0 * log(u1));
    return (i & 1) ? r * sin(two_pi * u2) : r * cos(two_pi * u2);
}

/* Student-t with nu degrees of freedom from nu+1 normals:
 * Z0 / sqrt((Z1^2 + ... + Znu^2) / nu). */
static inline double student_t_at(uint64_t key, uint64_t i, int nu)
{
    uint64_t base = i * (uint64_t)(nu + 1);
    double z0 = normal_at(key, base);
    double chi = 0.0;
    for (int q = 1; q <= nu; ++q) {
        double z = normal_at(key, base + (uint64_t)q);
        chi += z * z;
    }
    return z0 / sqrt(chi / (double)nu);
}

/* Uniform doubles in (0,1): out[i] for counters start..start+n-1. */
void synth_uniform_f64(uint64_t seed, uint64_t stream, int64_t start, int64_t n, double* out)
{
    uint64_t key = stream_key(seed, stream);
    for (int64_t i = 0; i < n; ++i)
        out[i] = unif_open(bits_at(key, (uint64_t)(start + i)));
}

/*
 * out[j] = fl32( shift[j] + mean + scale(seg(j)) * X_j ),  j in [0, n)
 *
 * X_j ~ N(0,1) when dist == 0, Student-t(nu) when dist == 1.  The counter of
 * element j is j itself, so a vector can be filled in pieces.  The segment
 * table (n_seg+1 ascending offsets starting at 0 and ending at n) gives the
 * per-tensor scale; seg_scale == NULL means scale 1 everywhere.  shift may be
 * NULL.  The sum is formed in double and rounded to binary32 once.
 */
void synth_fill_f32(uint64_t seed, uint64_t stream, int dist, int nu,
                    int64_t n, int64_t n_seg, const int64_t* seg_off,
                    const double* seg_scale, double mean, const float* shift,
                    float* out, int threads)
{
    uint64_t key = stream_key(seed, stream);
    if (threads < 1) threads = 1;
    for (int64_t s = 0; s < n_seg; ++s) {
        int64_t lo = seg_off[s], hi = seg_off[s + 1];
        if (lo < 0) lo = 0;
        if (hi > n) hi = n;
        double sc = seg_scale ? seg_scale[s] : 1.0;
#pragma omp parallel for schedule(static) num_threads(threads) if (hi - lo > 65536)
        for (int64_t j = lo; j < hi; ++j) {
            double x = dist == 1 ? student_t_at(key, (uint64_t)j, nu) : normal_at(key, (uint64_t)j);
            double v = mean + sc * x;
            if (shift) v += (double)shift[j];
            out[j] = (float)v;
        }
    }
}

int synth_max_threads(void)
{
#ifdef _OPENMP
    return omp_get_max_threads();
#else
    return 1;
#endif
}
