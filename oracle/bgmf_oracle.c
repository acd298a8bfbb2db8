/*
 * CPU oracle for blocked SGD matrix factorisation (BGMF).
 *
 * TEST INFRASTRUCTURE ONLY.  This file is the slow, plain, obviously correct
 * statement of what the GPU path computes.  Only the tests, the smoke check
 * and the benchmark's CPU-baseline leg may load it.  It shares no code,
 * header, table or helper with the HIP library, and the HIP library never
 * calls it.
 *
 * Build: gcc -O2 -ffp-contract=off -fno-fast-math -shared -fPIC -pthread
 *   -ffp-contract=off: every product and sum below is rounded separately
 *   (IEEE binary32, round-to-nearest-even), exactly in the written order.
 *
 * Notation (paper, Section 1):
 *   X in R^{n x m} observed at entries x_ij; U in R^{n x k}, V in R^{m x k};
 *   u_i is row i of U, v_j is row j of V (both row-major, fp32).
 *   Learning rate alpha, regularisation beta.
 *
 * Update form used throughout (no factor 2):
 *   e = x - u.v ;  u' = u + alpha (e v - beta u) ;  v' = v + alpha (e u - beta v)
 * where both right-hand sides use the OLD u and v (Eq. 2-3 update u and v
 * simultaneously from the same e).  The paper prints the same update with
 * 2e and step alpha_p; the two coincide for alpha = 2 alpha_p,
 * beta = beta_p / 2.
 */
#include <math.h>
#include <pthread.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

/* ---------------------------------------------------------------------- */
/* Block grid (Eq. 4; Algorithm 1's I x J split with I = J = p).           */
/* Row i lies in row-block R(i) = floor(i p / n); column j in              */
/* C(j) = floor(j p / m).  Blocks have equal size up to one row/column.    */
/* ---------------------------------------------------------------------- */

static int64_t row_block(int64_t i, int64_t n, int64_t p) { return (i * p) / n; }
static int64_t col_block(int64_t j, int64_t m, int64_t p) { return (j * p) / m; }

/* Stratum of block (R, C): blocks (b, (b + s) mod p), b = 0..p-1, form
 * stratum s; they share no row-block and no column-block, so they are
 * mutually independent (Section 1.1).  Slot q = s p + R orders the blocks
 * stratum by stratum. */
static int64_t slot_of(int64_t i, int64_t j, int64_t n, int64_t m, int64_t p)
{
    int64_t R = row_block(i, n, p);
    int64_t C = col_block(j, m, p);
    int64_t s = ((C - R) % p + p) % p;
    return s * p + R;
}

/* Bucketing.
 * block_ptr[q] = number of ratings whose slot is < q, for q = 0..p*p
 * (so block_ptr[p*p] = nnz).
 * perm = the rating indices e sorted by the key (slot, row), ties kept in
 * ascending e (a stable sort).
 *
 * The stable sort is done as two stable counting sorts: first by row i,
 * then by slot q.  A stable sort by the minor key followed by a stable sort
 * by the major key is a stable sort by the pair (major, minor).
 * Returns 0, or -1 if memory runs out. */
int oracle_bucket(int64_t n, int64_t m, int64_t p, int64_t nnz,
                  const int32_t *rows, const int32_t *cols,
                  int64_t *block_ptr, int32_t *perm)
{
    int64_t nslots = p * p;
    int64_t *row_count = (int64_t *)calloc((size_t)n + 1, sizeof(int64_t));
    int32_t *by_row = (int32_t *)malloc((size_t)(nnz > 0 ? nnz : 1) * sizeof(int32_t));
    int64_t *slot_pos = (int64_t *)calloc((size_t)nslots + 1, sizeof(int64_t));
    if (!row_count || !by_row || !slot_pos) {
        free(row_count); free(by_row); free(slot_pos);
        return -1;
    }

    /* pass 1: stable counting sort by row */
    for (int64_t e = 0; e < nnz; ++e) row_count[rows[e] + 1] += 1;
    for (int64_t i = 0; i < n; ++i) row_count[i + 1] += row_count[i];
    for (int64_t e = 0; e < nnz; ++e) by_row[row_count[rows[e]]++] = (int32_t)e;

    /* pass 2: stable counting sort by slot, reading in pass-1 order */
    for (int64_t q = 0; q <= nslots; ++q) block_ptr[q] = 0;
    for (int64_t e = 0; e < nnz; ++e)
        block_ptr[slot_of(rows[e], cols[e], n, m, p) + 1] += 1;
    for (int64_t q = 0; q < nslots; ++q) block_ptr[q + 1] += block_ptr[q];
    for (int64_t q = 0; q < nslots; ++q) slot_pos[q] = block_ptr[q];
    for (int64_t t = 0; t < nnz; ++t) {
        int32_t e = by_row[t];
        int64_t q = slot_of(rows[e], cols[e], n, m, p);
        perm[slot_pos[q]++] = e;
    }

    free(row_count); free(by_row); free(slot_pos);
    return 0;
}

/* Bucketing with given block boundaries (unequal blocks, the extension the
 * paper suggests in Section 3): row-block R holds rows
 * [row_cuts[R], row_cuts[R+1]), column-block C columns
 * [col_cuts[C], col_cuts[C+1]); strata and slots as above.  With
 * row_cuts[R] = ceil(R n / p) (and the same for columns) this is
 * oracle_bucket. */
static int64_t block_of_cut(const int64_t *cut, int64_t p, int64_t i)
{
    int64_t lo = 0, hi = p - 1;   /* the last R with cut[R] <= i */
    while (lo < hi) {
        int64_t mid = (lo + hi + 1) / 2;
        if (cut[mid] <= i) lo = mid; else hi = mid - 1;
    }
    return lo;
}

static int64_t slot_of_cuts(int64_t i, int64_t j, int64_t p,
                            const int64_t *row_cuts, const int64_t *col_cuts)
{
    int64_t R = block_of_cut(row_cuts, p, i);
    int64_t C = block_of_cut(col_cuts, p, j);
    int64_t s = ((C - R) % p + p) % p;
    return s * p + R;
}

int oracle_bucket_cuts(int64_t n, int64_t m, int64_t p, const int64_t *row_cuts,
                       const int64_t *col_cuts, int64_t nnz, const int32_t *rows,
                       const int32_t *cols, int64_t *block_ptr, int32_t *perm)
{
    (void)m;
    int64_t nslots = p * p;
    int64_t *row_count = (int64_t *)calloc((size_t)n + 1, sizeof(int64_t));
    int32_t *by_row = (int32_t *)malloc((size_t)(nnz > 0 ? nnz : 1) * sizeof(int32_t));
    int64_t *slot_pos = (int64_t *)calloc((size_t)nslots + 1, sizeof(int64_t));
    if (!row_count || !by_row || !slot_pos) {
        free(row_count); free(by_row); free(slot_pos);
        return -1;
    }
    for (int64_t e = 0; e < nnz; ++e) row_count[rows[e] + 1] += 1;
    for (int64_t i = 0; i < n; ++i) row_count[i + 1] += row_count[i];
    for (int64_t e = 0; e < nnz; ++e) by_row[row_count[rows[e]]++] = (int32_t)e;
    for (int64_t q = 0; q <= nslots; ++q) block_ptr[q] = 0;
    for (int64_t e = 0; e < nnz; ++e)
        block_ptr[slot_of_cuts(rows[e], cols[e], p, row_cuts, col_cuts) + 1] += 1;
    for (int64_t q = 0; q < nslots; ++q) block_ptr[q + 1] += block_ptr[q];
    for (int64_t q = 0; q < nslots; ++q) slot_pos[q] = block_ptr[q];
    for (int64_t t = 0; t < nnz; ++t) {
        int32_t e = by_row[t];
        perm[slot_pos[slot_of_cuts(rows[e], cols[e], p, row_cuts, col_cuts)]++] = e;
    }
    free(row_count); free(by_row); free(slot_pos);
    return 0;
}

/* ---------------------------------------------------------------------- */
/* One SGD step on one rating (Eq. 2-3; Eq. 14-15 per element).            */
/* ---------------------------------------------------------------------- */

static float dot_f32(int k, const float *u, const float *v)
{
    float acc = 0.0f;
    for (int g = 0; g < k; ++g) acc = acc + u[g] * v[g];
    return acc;
}

static void sgd_step(int k, float *u, float *v, float x, float alpha, float beta)
{
    float err = x - dot_f32(k, u, v);
    for (int g = 0; g < k; ++g) {
        float uo = u[g];
        float vo = v[g];
        u[g] = uo + alpha * ((err * vo) - (beta * uo));
        v[g] = vo + alpha * ((err * uo) - (beta * vo));
    }
}

void oracle_sgd_update(int32_t k, float *u, float *v, float x, float alpha, float beta)
{
    sgd_step(k, u, v, x, alpha, beta);
}

/* The same step carried out in binary64 (factors held in double): the
 * reference against which the rounding of the binary32 schedule is
 * measured.  x, alpha and beta are the binary32 inputs, widened exactly. */
static void sgd_step_f64(int k, double *u, double *v, double x, double alpha, double beta)
{
    double acc = 0.0;
    for (int g = 0; g < k; ++g) acc = acc + u[g] * v[g];
    double err = x - acc;
    for (int g = 0; g < k; ++g) {
        double uo = u[g];
        double vo = v[g];
        u[g] = uo + alpha * ((err * vo) - (beta * uo));
        v[g] = vo + alpha * ((err * uo) - (beta * vo));
    }
}

void oracle_sgd_update_f64(int32_t k, double *u, double *v, float x, float alpha, float beta)
{
    sgd_step_f64(k, u, v, x, alpha, beta);
}

/* ---------------------------------------------------------------------- */
/* One epoch: strata s = 0..p-1 in ascending order; inside a stratum the   */
/* blocks b = 0..p-1 (any order gives the same bits because the blocks of  */
/* a stratum touch disjoint rows of U and V); inside a block the ratings in */
/* bucketed order.  Each rating is visited once per epoch (Section 1: each */
/* element once per iteration; one pass per block is the exact scheme of   */
/* Section 1.3).                                                           */
/* ---------------------------------------------------------------------- */

static void run_block(int32_t k, int64_t q, const int32_t *rows, const int32_t *cols,
                      const float *vals, const int64_t *block_ptr, const int32_t *perm,
                      float *U, float *V, float alpha, float beta)
{
    for (int64_t t = block_ptr[q]; t < block_ptr[q + 1]; ++t) {
        int32_t e = perm[t];
        sgd_step(k, U + (int64_t)rows[e] * k, V + (int64_t)cols[e] * k, vals[e], alpha, beta);
    }
}

static void run_block_f64(int32_t k, int64_t q, const int32_t *rows, const int32_t *cols,
                          const float *vals, const int64_t *block_ptr, const int32_t *perm,
                          double *U, double *V, float alpha, float beta)
{
    for (int64_t t = block_ptr[q]; t < block_ptr[q + 1]; ++t) {
        int32_t e = perm[t];
        sgd_step_f64(k, U + (int64_t)rows[e] * k, V + (int64_t)cols[e] * k, vals[e], alpha, beta);
    }
}

void oracle_epoch(int64_t p, int32_t k, const int32_t *rows, const int32_t *cols,
                  const float *vals, const int64_t *block_ptr, const int32_t *perm,
                  float *U, float *V, float alpha, float beta)
{
    for (int64_t s = 0; s < p; ++s)
        for (int64_t b = 0; b < p; ++b)
            run_block(k, s * p + b, rows, cols, vals, block_ptr, perm, U, V, alpha, beta);
}

/* The epoch with GPU_STEPS = passes (Algorithm 1; Section 1.3): each block
 * is factorised passes times in a row, its ratings in the same order every
 * time, before the next block of the row-block's sequence. */
void oracle_epoch_passes(int64_t p, int32_t k, const int32_t *rows, const int32_t *cols,
                         const float *vals, const int64_t *block_ptr, const int32_t *perm,
                         float *U, float *V, float alpha, float beta, int32_t passes)
{
    for (int64_t s = 0; s < p; ++s)
        for (int64_t b = 0; b < p; ++b)
            for (int32_t g = 0; g < passes; ++g)
                run_block(k, s * p + b, rows, cols, vals, block_ptr, perm, U, V, alpha, beta);
}

/* Same epoch with the blocks of each stratum visited in a caller-given
 * order (order[s * p + idx] = b).  Used to show that the blocks of a
 * stratum commute. */
void oracle_epoch_ordered(int64_t p, int32_t k, const int32_t *rows, const int32_t *cols,
                          const float *vals, const int64_t *block_ptr, const int32_t *perm,
                          float *U, float *V, float alpha, float beta, const int32_t *order)
{
    for (int64_t s = 0; s < p; ++s)
        for (int64_t idx = 0; idx < p; ++idx)
            run_block(k, s * p + order[s * p + idx], rows, cols, vals, block_ptr, perm,
                      U, V, alpha, beta);
}

/* Multithreaded epoch: the p blocks of a stratum are split over T threads,
 * with a barrier after every stratum.  Bit-identical to oracle_epoch
 * because the blocks of one stratum are independent.  Worker threads wait
 * at a start gate until the caller knows how many of them started; if any
 * failed to start, the started ones leave without work and the epoch runs
 * on the calling thread. */
struct mt_ctx {
    int64_t p; int32_t k; int nthreads;
    const int32_t *rows, *cols; const float *vals;
    const int64_t *block_ptr; const int32_t *perm;
    float *U, *V; float alpha, beta;
    double *U64, *V64;  /* non-NULL: the binary64 schedule */
    int32_t passes;     /* GPU_STEPS: passes over each block */
    pthread_barrier_t barrier;
    pthread_mutex_t gate_mu; pthread_cond_t gate_cv; int gate; /* 0 wait, 1 go, -1 abort */
};
struct mt_arg { struct mt_ctx *c; int tid; };

static void *mt_worker(void *arg_)
{
    struct mt_arg *a = (struct mt_arg *)arg_;
    struct mt_ctx *c = a->c;
    pthread_mutex_lock(&c->gate_mu);
    while (c->gate == 0) pthread_cond_wait(&c->gate_cv, &c->gate_mu);
    int go = c->gate;
    pthread_mutex_unlock(&c->gate_mu);
    if (go < 0) return NULL;
    for (int64_t s = 0; s < c->p; ++s) {
        for (int64_t b = a->tid; b < c->p; b += c->nthreads) {
            for (int32_t g = 0; g < c->passes; ++g) {
                if (c->U64)
                    run_block_f64(c->k, s * c->p + b, c->rows, c->cols, c->vals, c->block_ptr,
                                  c->perm, c->U64, c->V64, c->alpha, c->beta);
                else
                    run_block(c->k, s * c->p + b, c->rows, c->cols, c->vals, c->block_ptr,
                              c->perm, c->U, c->V, c->alpha, c->beta);
            }
        }
        pthread_barrier_wait(&c->barrier);
    }
    return NULL;
}

static void epoch_seq(int64_t p, int32_t k, const int32_t *rows, const int32_t *cols,
                      const float *vals, const int64_t *block_ptr, const int32_t *perm,
                      float *U, float *V, double *U64, double *V64, float alpha, float beta,
                      int32_t passes)
{
    if (!U64) {
        oracle_epoch_passes(p, k, rows, cols, vals, block_ptr, perm, U, V, alpha, beta, passes);
        return;
    }
    for (int64_t s = 0; s < p; ++s)
        for (int64_t b = 0; b < p; ++b)
            for (int32_t g = 0; g < passes; ++g)
                run_block_f64(k, s * p + b, rows, cols, vals, block_ptr, perm, U64, V64, alpha,
                              beta);
}

static int epoch_mt(int64_t p, int32_t k, const int32_t *rows, const int32_t *cols,
                    const float *vals, const int64_t *block_ptr, const int32_t *perm,
                    float *U, float *V, double *U64, double *V64, float alpha, float beta,
                    int32_t passes, int32_t nthreads)
{
    if (nthreads <= 1) {
        epoch_seq(p, k, rows, cols, vals, block_ptr, perm, U, V, U64, V64, alpha, beta, passes);
        return 1;
    }
    struct mt_ctx *c = (struct mt_ctx *)calloc(1, sizeof(struct mt_ctx));
    pthread_t *th = (pthread_t *)malloc(sizeof(pthread_t) * (size_t)nthreads);
    struct mt_arg *args = (struct mt_arg *)malloc(sizeof(struct mt_arg) * (size_t)nthreads);
    if (!c || !th || !args) {
        free(c); free(th); free(args);
        epoch_seq(p, k, rows, cols, vals, block_ptr, perm, U, V, U64, V64, alpha, beta, passes);
        return 1;
    }
    c->p = p; c->k = k; c->nthreads = nthreads;
    c->rows = rows; c->cols = cols; c->vals = vals;
    c->block_ptr = block_ptr; c->perm = perm;
    c->U = U; c->V = V; c->alpha = alpha; c->beta = beta;
    c->U64 = U64; c->V64 = V64; c->passes = passes;
    pthread_barrier_init(&c->barrier, NULL, (unsigned)nthreads);
    pthread_mutex_init(&c->gate_mu, NULL);
    pthread_cond_init(&c->gate_cv, NULL);
    c->gate = 0;
    int started = 0;
    for (int t = 0; t < nthreads; ++t) {
        args[t].c = c; args[t].tid = t;
        if (pthread_create(&th[t], NULL, mt_worker, &args[t]) != 0) break;
        ++started;
    }
    pthread_mutex_lock(&c->gate_mu);
    c->gate = (started == nthreads) ? 1 : -1;
    pthread_cond_broadcast(&c->gate_cv);
    pthread_mutex_unlock(&c->gate_mu);
    for (int t = 0; t < started; ++t) pthread_join(th[t], NULL);
    int used = nthreads;
    if (started != nthreads) {
        epoch_seq(p, k, rows, cols, vals, block_ptr, perm, U, V, U64, V64, alpha, beta, passes);
        used = 1;
    }
    pthread_barrier_destroy(&c->barrier);
    pthread_mutex_destroy(&c->gate_mu);
    pthread_cond_destroy(&c->gate_cv);
    free(c); free(th); free(args);
    return used; /* number of threads that did the work */
}

int oracle_epoch_mt(int64_t p, int32_t k, const int32_t *rows, const int32_t *cols,
                    const float *vals, const int64_t *block_ptr, const int32_t *perm,
                    float *U, float *V, float alpha, float beta, int32_t nthreads)
{
    return epoch_mt(p, k, rows, cols, vals, block_ptr, perm, U, V, NULL, NULL, alpha, beta, 1,
                    nthreads);
}

/* Multithreaded epoch with GPU_STEPS = passes (see oracle_epoch_passes). */
int oracle_epoch_mt_passes(int64_t p, int32_t k, const int32_t *rows, const int32_t *cols,
                           const float *vals, const int64_t *block_ptr, const int32_t *perm,
                           float *U, float *V, float alpha, float beta, int32_t passes,
                           int32_t nthreads)
{
    return epoch_mt(p, k, rows, cols, vals, block_ptr, perm, U, V, NULL, NULL, alpha, beta,
                    passes, nthreads);
}

/* The epoch in binary64: same schedule and operation order, factors held in
 * double (U64, V64), ratings and the step sizes widened exactly from their
 * binary32 values.  nthreads <= 1 runs it on the calling thread. */
int oracle_epoch_mt_f64(int64_t p, int32_t k, const int32_t *rows, const int32_t *cols,
                        const float *vals, const int64_t *block_ptr, const int32_t *perm,
                        double *U64, double *V64, float alpha, float beta, int32_t nthreads)
{
    return epoch_mt(p, k, rows, cols, vals, block_ptr, perm, NULL, NULL, U64, V64, alpha, beta, 1,
                    nthreads);
}

/* ---------------------------------------------------------------------- */
/* RMSE over all loaded ratings (Algorithm 1's termination test uses the   */
/* RMSE of the whole matrix): fp32 dot as in the update, squared residuals */
/* accumulated in fp64 in input order.                                     */
/* ---------------------------------------------------------------------- */

double oracle_rmse(int32_t k, int64_t nnz, const int32_t *rows, const int32_t *cols,
                   const float *vals, const float *U, const float *V)
{
    double sq = 0.0;
    for (int64_t e = 0; e < nnz; ++e) {
        float d = vals[e] - dot_f32(k, U + (int64_t)rows[e] * k, V + (int64_t)cols[e] * k);
        sq += (double)d * (double)d;
    }
    return nnz > 0 ? sqrt(sq / (double)nnz) : 0.0;
}

/* Objective of Eq. 1 in fp64: sum over observed entries of
 * (x - u.v)^2 + beta (|u|^2 + |v|^2).  The regulariser is counted once per
 * observed entry, as Eq. 1 writes it inside the sum. */
double oracle_loss(int32_t k, int64_t nnz, const int32_t *rows, const int32_t *cols,
                   const float *vals, const float *U, const float *V, double beta)
{
    double total = 0.0;
    for (int64_t e = 0; e < nnz; ++e) {
        const float *u = U + (int64_t)rows[e] * k;
        const float *v = V + (int64_t)cols[e] * k;
        double dot = 0.0, uu = 0.0, vv = 0.0;
        for (int g = 0; g < k; ++g) {
            dot += (double)u[g] * (double)v[g];
            uu += (double)u[g] * (double)u[g];
            vv += (double)v[g] * (double)v[g];
        }
        double r = (double)vals[e] - dot;
        total += r * r + beta * (uu + vv);
    }
    return total;
}
