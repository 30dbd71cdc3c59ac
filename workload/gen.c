/*
 * gen.c -- seeded, counter-based generator of synthetic KV-cache workloads.
 *
 * Serves both the GPU library's tests/benchmark and the CPU oracle's tests
 * with identical inputs.  It holds none of the conversion's arithmetic: it
 * draws random numbers only.
 *
 * Random stream: splitmix64 (Steele, Lea, Flood, "Fast splittable
 * pseudorandom number generators", OOPSLA 2014) in counter form.  Word i of
 * stream k under seed s is  mix((s ^ (k << 56)) + (i + 1) * golden)  with
 * golden = 0x9E3779B97F4A7C15 and mix the splitmix64 output function, so any
 * index range can be produced independently and in parallel.
 * Uniforms: (word >> 11) * 2^-53 in [0, 1).
 * Normals: Box-Muller on the uniform pair (2k, 2k+1); element 2k takes the
 * cosine branch and 2k+1 the sine branch.
 */
#define _GNU_SOURCE
#include <math.h>
#include <pthread.h>
#include <stdint.h>
#include <stdlib.h>

static inline uint64_t mix64(uint64_t z)
{
    z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ULL;
    z = (z ^ (z >> 27)) * 0x94D049BB133111EBULL;
    return z ^ (z >> 31);
}

uint64_t wl_word(uint64_t seed, uint32_t stream, uint64_t i)
{
    return mix64((seed ^ ((uint64_t)stream << 56)) + (i + 1) * 0x9E3779B97F4A7C15ULL);
}

double wl_uniform(uint64_t seed, uint32_t stream, uint64_t i)
{
    return (double)(wl_word(seed, stream, i) >> 11) * 0x1.0p-53;
}


/* One pair (2k, 2k+1) of the normal stream: Box-Muller, radius from 1 - u1
 * in (0, 1]. */
static inline void normal_pair(uint64_t seed, uint32_t stream, uint64_t k, double *z0, double *z1)
{
    double u1 = wl_uniform(seed, stream, 2 * k);
    double u2 = wl_uniform(seed, stream, 2 * k + 1);
    double rad = sqrt(-2.0 * log(1.0 - u1));
    double sn, cs;
    sincos(6.283185307179586476925286766559 * u2, &sn, &cs);
    *z0 = rad * cs;
    *z1 = rad * sn;
}

/* out[k] = sigma * normal(first + k) for k in [lo, hi) of a run */
static void fill_run(uint64_t seed, uint32_t stream, uint64_t first, int64_t lo, int64_t hi,
                     double sigma, float *out)
{
    int64_t k = lo;
    double z0, z1;
    if (k < hi && ((first + (uint64_t)k) & 1)) {
        normal_pair(seed, stream, (first + (uint64_t)k) >> 1, &z0, &z1);
        out[k] = (float)(sigma * z1);
        ++k;
    }
    for (; k + 1 < hi; k += 2) {
        normal_pair(seed, stream, (first + (uint64_t)k) >> 1, &z0, &z1);
        out[k] = (float)(sigma * z0);
        out[k + 1] = (float)(sigma * z1);
    }
    if (k < hi) {
        normal_pair(seed, stream, (first + (uint64_t)k) >> 1, &z0, &z1);
        out[k] = (float)(sigma * z0);
    }
}

typedef struct {
    uint64_t seed;
    uint32_t stream;
    const uint64_t *starts;  /* first draw index of each block */
    int64_t block_len;
    int64_t lo, hi;          /* flat output range of this thread */
    double sigma;
    float *out;
} fill_job;

static void *fill_worker(void *arg)
{
    fill_job *j = (fill_job *)arg;
    int64_t k = j->lo;
    while (k < j->hi) {
        int64_t b = k / j->block_len, in = k - b * j->block_len;
        int64_t end = (b + 1) * j->block_len < j->hi ? (b + 1) * j->block_len : j->hi;
        fill_run(j->seed, j->stream, j->starts[b], in, in + (end - k), j->sigma,
                 j->out + b * j->block_len);
        k = end;
    }
    return NULL;
}

/* out[b*block_len + k] = sigma * normal(starts[b] + k), b < nblocks, k < block_len */
void wl_fill_normal_blocks(uint64_t seed, uint32_t stream, const uint64_t *starts, int64_t nblocks,
                           int64_t block_len, double sigma, float *out, int nthreads)
{
    int64_t n = nblocks * block_len;
    if (nthreads > 64) nthreads = 64;
    if (nthreads > n / 65536) nthreads = (int)(n / 65536); /* at least 64Ki draws per thread */
    if (nthreads < 1) nthreads = 1;
    pthread_t th[64];
    fill_job jobs[64];
    int64_t per = (n + nthreads - 1) / nthreads;
    for (int t = 0; t < nthreads; ++t) {
        jobs[t].seed = seed; jobs[t].stream = stream; jobs[t].starts = starts;
        jobs[t].block_len = block_len;
        jobs[t].lo = t * per < n ? t * per : n;
        jobs[t].hi = (t + 1) * per < n ? (t + 1) * per : n;
        jobs[t].sigma = sigma; jobs[t].out = out;
    }
    if (nthreads == 1) { fill_worker(&jobs[0]); return; }
    for (int t = 0; t < nthreads; ++t) pthread_create(&th[t], NULL, fill_worker, &jobs[t]);
    for (int t = 0; t < nthreads; ++t) pthread_join(th[t], NULL);
}

double wl_normal(uint64_t seed, uint32_t stream, uint64_t i)
{
    double z0, z1;
    normal_pair(seed, stream, i >> 1, &z0, &z1);
    return (i & 1) ? z1 : z0;
}

/* out[k] = sigma * normal(first + k), k in [0, n) */
void wl_fill_normal(uint64_t seed, uint32_t stream, uint64_t first, int64_t n, double sigma,
                    float *out, int nthreads)
{
    wl_fill_normal_blocks(seed, stream, &first, 1, n, sigma, out, nthreads);
}

/* out[k] = uniform(stream, first + k) */
void wl_fill_uniform(uint64_t seed, uint32_t stream, uint64_t first, int64_t n, double *out)
{
    for (int64_t k = 0; k < n; ++k) out[k] = wl_uniform(seed, stream, first + (uint64_t)k);
}

/* Indices k in [0, n) with uniform(stream, first + k) < p, written to idx;
 * returns their count. */
int64_t wl_select(uint64_t seed, uint32_t stream, uint64_t first, int64_t n, double p,
                  int64_t *idx)
{
    int64_t c = 0;
    for (int64_t k = 0; k < n; ++k)
        if (wl_uniform(seed, stream, first + (uint64_t)k) < p) idx[c++] = k;
    return c;
}

/* Fisher-Yates shuffle of 0..n-1: for i = n-1 down to 1 swap out[i] with
 * out[floor(u_i * (i + 1))], u_i = uniform(stream, i). */
void wl_permutation(uint64_t seed, uint32_t stream, int64_t n, int32_t *out)
{
    for (int64_t i = 0; i < n; ++i) out[i] = (int32_t)i;
    for (int64_t i = n - 1; i >= 1; --i) {
        int64_t j = (int64_t)(wl_uniform(seed, stream, (uint64_t)i) * (double)(i + 1));
        if (j > i) j = i;
        int32_t tmp = out[i]; out[i] = out[j]; out[j] = tmp;
    }
}
