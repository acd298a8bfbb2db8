/*
 * Fast kernels for the synthetic workload generator (data drawing only; no
 * factorisation arithmetic).  Built with gcc -O2 -fopenmp into libgen.so.
 *
 * Random numbers: every user (or rating) has its own stream derived from
 * (seed, index) with the SplitMix64 mixer (Steele, Lea, Flood, "Fast
 * splittable pseudorandom number generators", OOPSLA 2014), so results do
 * not depend on the number of threads.
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

static inline uint64_t splitmix64(uint64_t *state)
{
    uint64_t z = (*state += 0x9E3779B97F4A7C15ull);
    z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
    z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
    return z ^ (z >> 31);
}

static inline uint64_t stream_seed(uint64_t seed, uint64_t index)
{
    uint64_t s = seed * 0xD1B54A32D192ED03ull + index * 0x9E3779B97F4A7C15ull + 0x632BE59BD9B4E019ull;
    (void)splitmix64(&s);
    return s;
}

/* uniform double in (0, 1) */
static inline double uniform01(uint64_t *state)
{
    return ((double)(splitmix64(state) >> 11) + 0.5) * (1.0 / 9007199254740992.0);
}

/* index r with cdf[r-1] <= u < cdf[r] (cdf ascending, cdf[m-1] == 1) */
static inline int64_t sample_cdf(const double *cdf, int64_t m, double u)
{
    int64_t lo = 0, hi = m - 1;
    while (lo < hi) {
        int64_t mid = (lo + hi) >> 1;
        if (cdf[mid] > u) hi = mid; else lo = mid + 1;
    }
    return lo;
}

typedef struct { double key; int32_t item; } keyed_t;

static int cmp_keyed(const void *a, const void *b)
{
    double x = ((const keyed_t *)a)->key, y = ((const keyed_t *)b)->key;
    if (x < y) return -1;
    if (x > y) return 1;
    return ((const keyed_t *)a)->item - ((const keyed_t *)b)->item;
}

/*
 * Distinct items for every user by successive weighted sampling without
 * replacement: user i draws items from the item distribution (cdf over
 * ranks, mapped to ids by item_of_rank) and keeps each item the first time
 * it appears, until it holds deg[i] items.  Users whose degree exceeds a
 * quarter of m use the equivalent exponential-key form (each item gets key
 * E_j / w_j, E_j ~ Exp(1); the deg[i] smallest keys are kept), which avoids
 * the coupon-collector tail.
 *
 * Output: cols_out[offset[i] .. offset[i] + deg[i]) for user i, where
 * offset is the exclusive prefix sum of deg (passed in).  Returns 0, or -1
 * on allocation failure.
 */
int gen_user_items(int64_t n, int64_t m, const int64_t *deg, const int64_t *offset,
                   const double *cdf, const double *weight_of_rank,
                   const int32_t *item_of_rank, uint64_t seed, int32_t *cols_out)
{
    int failed = 0;
#pragma omp parallel
    {
        uint64_t *seen = (uint64_t *)calloc((size_t)((m + 63) / 64), sizeof(uint64_t));
        keyed_t *keys = NULL;
        if (!seen) {
#pragma omp atomic write
            failed = 1;
        }
#pragma omp for schedule(dynamic, 256)
        for (int64_t i = 0; i < n; ++i) {
            if (!seen) continue;
            int64_t d = deg[i];
            int32_t *out = cols_out + offset[i];
            uint64_t st = stream_seed(seed, (uint64_t)i);
            if (d <= 0) continue;
            if (d * 4 > m) {
                if (!keys) keys = (keyed_t *)malloc(sizeof(keyed_t) * (size_t)m);
                if (!keys) {
#pragma omp atomic write
                    failed = 1;
                    continue;
                }
                for (int64_t r = 0; r < m; ++r) {
                    keys[r].key = -log(uniform01(&st)) / weight_of_rank[r];
                    keys[r].item = item_of_rank[r];
                }
                if (d < m) qsort(keys, (size_t)m, sizeof(keyed_t), cmp_keyed);
                for (int64_t t = 0; t < d; ++t) out[t] = keys[t].item;
                continue;
            }
            int64_t got = 0;
            while (got < d) {
                int32_t item = item_of_rank[sample_cdf(cdf, m, uniform01(&st))];
                uint64_t bit = 1ull << (item & 63);
                if (seen[item >> 6] & bit) continue;
                seen[item >> 6] |= bit;
                out[got++] = item;
            }
            for (int64_t t = 0; t < d; ++t) seen[out[t] >> 6] = 0; /* clear touched words */
        }
        free(seen);
        free(keys);
    }
    return failed ? -1 : 0;
}

/* z[e] = sum_r us[rows[e], r] * vs[cols[e], r] in fp64 (planted model). */
void gen_planted_dot(int64_t nnz, int32_t rank, const int32_t *rows, const int32_t *cols,
                     const float *us, const float *vs, double *z)
{
#pragma omp parallel for schedule(static)
    for (int64_t e = 0; e < nnz; ++e) {
        const float *a = us + (int64_t)rows[e] * rank;
        const float *b = vs + (int64_t)cols[e] * rank;
        double acc = 0.0;
        for (int r = 0; r < rank; ++r) acc += (double)a[r] * (double)b[r];
        z[e] = acc;
    }
}

/* Standard normal draws, one stream per index (Box-Muller). */
void gen_normal(int64_t count, uint64_t seed, double *out)
{
#pragma omp parallel for schedule(static)
    for (int64_t e = 0; e < count; ++e) {
        uint64_t st = stream_seed(seed, (uint64_t)e);
        double u1 = uniform01(&st), u2 = uniform01(&st);
        out[e] = sqrt(-2.0 * log(u1)) * cos(6.283185307179586 * u2);
    }
}

/*
 * Uniformly random permutation of 0..count-1 that does not depend on the
 * number of threads.  Every index draws a bucket label from its own stream
 * (seed, index); the indices are grouped by label (in ascending index order
 * inside a bucket), and each bucket is then shuffled by Fisher-Yates with
 * its own stream (seed, count + bucket).  Independent uniform labels plus a
 * uniform order inside every bucket make every permutation equally likely
 * (all indices are exchangeable).  The grouping runs over a fixed number of
 * index chunks so that its result is the same for any thread count.
 * Returns 0, or -1 on allocation failure.
 */
#define PERM_BUCKETS 16384
#define PERM_CHUNKS 256

static inline uint32_t perm_bucket(uint64_t seed, int64_t i)
{
    uint64_t st = stream_seed(seed, (uint64_t)i);
    return (uint32_t)(splitmix64(&st) >> 50);  /* top 14 bits: 0 .. 16383 */
}

int gen_permutation(int64_t count, uint64_t seed, int64_t *perm)
{
    int64_t *cnt = (int64_t *)calloc((size_t)PERM_CHUNKS * PERM_BUCKETS, sizeof(int64_t));
    int64_t *start = (int64_t *)malloc(sizeof(int64_t) * (PERM_BUCKETS + 1));
    if (!cnt || !start) {
        free(cnt);
        free(start);
        return -1;
    }
    const int64_t per = (count + PERM_CHUNKS - 1) / PERM_CHUNKS;
#pragma omp parallel for schedule(dynamic, 1)
    for (int c = 0; c < PERM_CHUNKS; ++c) {
        int64_t *h = cnt + (int64_t)c * PERM_BUCKETS;
        const int64_t lo = (int64_t)c * per, hi = lo + per < count ? lo + per : count;
        for (int64_t i = lo; i < hi; ++i) h[perm_bucket(seed, i)] += 1;
    }
    /* exclusive offsets in (bucket, chunk) order */
    int64_t run = 0;
    for (int b = 0; b < PERM_BUCKETS; ++b) {
        start[b] = run;
        for (int c = 0; c < PERM_CHUNKS; ++c) {
            int64_t v = cnt[(int64_t)c * PERM_BUCKETS + b];
            cnt[(int64_t)c * PERM_BUCKETS + b] = run;
            run += v;
        }
    }
    start[PERM_BUCKETS] = run;
#pragma omp parallel for schedule(dynamic, 1)
    for (int c = 0; c < PERM_CHUNKS; ++c) {
        int64_t *h = cnt + (int64_t)c * PERM_BUCKETS;
        const int64_t lo = (int64_t)c * per, hi = lo + per < count ? lo + per : count;
        for (int64_t i = lo; i < hi; ++i) perm[h[perm_bucket(seed, i)]++] = i;
    }
#pragma omp parallel for schedule(dynamic, 16)
    for (int b = 0; b < PERM_BUCKETS; ++b) {
        uint64_t st = stream_seed(seed, (uint64_t)count + (uint64_t)b);
        int64_t *a = perm + start[b];
        for (int64_t j = start[b + 1] - start[b] - 1; j > 0; --j) {
            int64_t r = (int64_t)(uniform01(&st) * (double)(j + 1));
            if (r > j) r = j;
            int64_t t = a[j];
            a[j] = a[r];
            a[r] = t;
        }
    }
    free(cnt);
    free(start);
    return 0;
}

/* dst[e] = src[perm[e]] for 4-byte elements (int32 or float32). */
void gen_gather32(int64_t count, const int64_t *perm, const uint32_t *src, uint32_t *dst)
{
#pragma omp parallel for schedule(static)
    for (int64_t e = 0; e < count; ++e) dst[e] = src[perm[e]];
}
