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

double wl_normal(uint64_t seed, uint32_t stream, uint64_t i)
{
    uint64_t k = i >> 1;
    double u1 = wl_uniform(seed, stream, 2 * k);
    double u2 = wl_uniform(seed, stream, 2 * k + 1);
    double rad = sqrt(-2.0 * log(1.0 - u1)); /* 1 - u1 in (0, 1] */
    double ang = 6.283185307179586476925286766559 * u2;
    return (i & 1) ? rad * sin(ang) : rad * cos(ang);
}

typedef struct {
    uint64_t seed;
    uint32_t stream;
    uint64_t first;
    int64_t lo, hi;
    double sigma;
    float *out;
} fill_job;

static void *fill_normal_worker(void *arg)
{
    fill_job *j = (fill_job *)arg;
    int64_t k = j->lo;
    /* leading odd element */
    if (k < j->hi && ((j->first + (uint64_t)k) & 1)) {
        j->out[k] = (float)(j->sigma * wl_normal(j->seed, j->stream, j->first + (uint64_t)k));
        ++k;
    }
    for (; k + 1 < j->hi; k += 2) { /* both branches of one Box-Muller pair */
        uint64_t i = j->first + (uint64_t)k;
        double u1 = wl_uniform(j->seed, j->stream, i);
        double u2 = wl_uniform(j->seed, j->stream, i + 1);
        double rad = sqrt(-2.0 * log(1.0 - u1));
        double ang = 6.283185307179586476925286766559 * u2;
        j->out[k] = (float)(j->sigma * rad * cos(ang));
        j->out[k + 1] = (float)(j->sigma * rad * sin(ang));
    }
    if (k < j->hi)
        j->out[k] = (float)(j->sigma * wl_normal(j->seed, j->stream, j->first + (uint64_t)k));
    return NULL;
}

/* out[k] = sigma * normal(stream, first + k), k in [0, n) */
void wl_fill_normal(uint64_t seed, uint32_t stream, uint64_t first, int64_t n, double sigma,
                    float *out, int nthreads)
{
    if (nthreads < 1) nthreads = 1;
    if (nthreads > 64) nthreads = 64;
    if (n < (int64_t)1 << 20) nthreads = 1;
    pthread_t th[64];
    fill_job jobs[64];
    int64_t per = (n + nthreads - 1) / nthreads;
    per = (per + 1) & ~(int64_t)1;
    for (int t = 0; t < nthreads; ++t) {
        jobs[t].seed = seed; jobs[t].stream = stream; jobs[t].first = first;
        jobs[t].lo = t * per < n ? t * per : n;
        jobs[t].hi = (t + 1) * per < n ? (t + 1) * per : n;
        jobs[t].sigma = sigma; jobs[t].out = out;
    }
    if (nthreads == 1) { fill_normal_worker(&jobs[0]); return; }
    for (int t = 0; t < nthreads; ++t) pthread_create(&th[t], NULL, fill_normal_worker, &jobs[t]);
    for (int t = 0; t < nthreads; ++t) pthread_join(th[t], NULL);
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
