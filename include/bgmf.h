/*
 * bgmf.h — C ABI of the MI355X (gfx950) blocked SGD matrix factorisation
 * library (BGMF: block-based GPU matrix factorisation).
 *
 * Problem (paper, Section 1, Eq. 1): a sparse matrix X in R^{n x m} is
 * observed at entries x_ij; find U in R^{n x k}, V in R^{m x k} with
 * X ~ U V^T by stochastic gradient descent on
 *     sum over observed x_ij of (x_ij - u_i.v_j)^2 + beta (|u_i|^2 + |v_j|^2).
 *
 * Method (Eq. 4, Section 1.1, Algorithm 1): X is cut into a p x p grid of
 * blocks; row-block R holds rows [ceil(R n/p), ceil((R+1) n/p)), column-block
 * C holds columns [ceil(C m/p), ceil((C+1) m/p)); equivalently row i is in
 * row-block floor(i p / n).  Stratum s is the set of blocks (b, (b+s) mod p),
 * b = 0..p-1; its blocks share no row and no column, so they run in
 * parallel.  One epoch visits strata s = 0, 1, ..., p-1 in that order, and in
 * each block applies, rating by rating, the update of Eq. 2-3:
 *     e  = x_ij - u_i.v_j
 *     u_i <- u_i + alpha (e v_j - beta u_i)
 *     v_j <- v_j + alpha (e u_i - beta v_j)      (old u_i on the right)
 * This is the paper's update with its factor 2 folded into the step:
 * alpha = 2 alpha_paper, beta = beta_paper / 2.
 *
 * Inside a block, ratings are taken in ascending row, ties in ascending
 * input position (the order the caller passed them to bgmf_load_coo).  The
 * per-block pass count (GPU_STEPS) is one by default (Section 1.3: one pass
 * per block is the exact scheme) and can be raised with
 * BGMF_OPT_BLOCK_PASSES.
 *
 * Conventions for every call:
 *   - Return value: BGMF_OK (0) or a negative BGMF_E_* code; the message is
 *     available from bgmf_last_error(handle).  Nothing aborts the process.
 *   - On error the handle keeps its previous valid state, except that a
 *     failed bgmf_load_coo leaves no ratings loaded.
 *   - Host pointers are read (or written) only during the call; the library
 *     keeps no caller pointer after returning.
 *   - A handle is not thread-safe.  All device work is ordered on the
 *     handle's stream (see bgmf_set_stream).  bgmf_epoch returns without
 *     waiting; bgmf_rmse, bgmf_get_factors, bgmf_get_layout, bgmf_sync and
 *     bgmf_get_timing wait for the stream.
 *   - All floating point is IEEE binary32 except where stated.
 */
#ifndef BGMF_H
#define BGMF_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* Status codes. */
#define BGMF_OK            0
#define BGMF_E_ARG        -1  /* invalid argument (size, null pointer, alpha/beta) */
#define BGMF_E_STATE      -2  /* call not valid in the handle's current state */
#define BGMF_E_RANGE      -3  /* a rating index outside [0,n) x [0,m) */
#define BGMF_E_NONFINITE  -4  /* a rating value that is NaN or infinite */
#define BGMF_E_NOMEM      -5  /* device or host allocation failed */
#define BGMF_E_BUDGET     -6  /* the ratings budget, a bound workspace or a bound host
                                 arena is too small for the loaded ratings */
#define BGMF_E_HIP        -7  /* a HIP runtime call failed */
#define BGMF_E_UNSUPPORTED -8 /* shape the kernels do not handle */
#define BGMF_E_TIMEOUT    -9  /* a device-side wait between strata exceeded its limit */

typedef struct bgmf bgmf_t; /* opaque handle */

/* Create a handle for an n x m matrix, factor width k and a p x p grid
 * (Algorithm 1's I = J = p).  Allocates U (n x k) and V (m x k) on the
 * current HIP device.
 *   1 <= n, m < 2^31;  k a multiple of 16 in [16, 256];
 *   1 <= p <= min(n, m, 8192);  ceil(n/p) <= 65536;  ceil(m/p) <= 65536.
 * Returns NULL on error; the reason is bgmf_last_error(NULL) (per thread). */
bgmf_t *bgmf_create(int64_t n, int64_t m, int32_t k, int32_t p);

/* Release every resource of the handle (waits for its stream first).
 * NULL is ignored. */
void bgmf_destroy(bgmf_t *h);

/* Message of the last failed call on h, or of the last failed bgmf_create on
 * this thread when h is NULL.  Owned by the library; valid until the next
 * call on the same handle (or thread). */
const char *bgmf_last_error(const bgmf_t *h);

/* Order all later device work of h on a caller-owned hipStream_t (for
 * example PyTorch's current stream).  NULL selects the handle's own stream.
 * The caller keeps ownership; the stream must outlive its use by h. */
int bgmf_set_stream(bgmf_t *h, void *hip_stream);

/* Memory a caller provides for a handle (bgmf_bind), for nnz ratings:
 *   *factor_bytes    = bytes of U (n x k) plus V (m x k), fp32;
 *   *incore_ws_bytes = a workspace that keeps every rating on the device:
 *                      the block tables, 8-byte records (+256 of padding),
 *                      perm, and the one-pass bucketing's temporaries (the
 *                      COO arrays and the radix sort's scratch), about
 *                      48 bytes per rating;
 *   *min_ws_bytes    = a lower bound below which no load of nnz ratings can
 *                      stream (the block tables, the bucketing of an average
 *                      block and a ring of two average strata); the real
 *                      need depends on the largest block and stratum, which
 *                      bgmf_load_coo checks (BGMF_E_BUDGET);
 *   *pinned_bytes    = a pinned host arena for streamed ratings (records and
 *                      perm, 12 bytes per rating).
 * Any output may be NULL.  The sizes follow the Problem of Section 1 (U,
 * V) and Eq. 4 (the p x p block tables). */
int bgmf_query_sizes(const bgmf_t *h, int64_t nnz, size_t *factor_bytes, size_t *min_ws_bytes,
                     size_t *incore_ws_bytes, size_t *pinned_bytes);

/* Bind caller-owned memory (for example PyTorch tensors) to the handle,
 * before any ratings are loaded (else BGMF_E_STATE):
 *   U_dev, V_dev  device memory of n x k and m x k fp32, row-major; from
 *                 now on they ARE the factors (Algorithm 1's inputs and
 *                 outputs): the handle's own U and V are freed, whatever
 *                 the buffers hold counts as set factors, and
 *                 bgmf_set_factors / bgmf_get_factors copy into / out of
 *                 them;
 *   ws_dev, ws_bytes  device workspace for the block tables and the
 *                 ratings.  bgmf_load_coo keeps every rating on the device
 *                 when ws_bytes >= incore_ws_bytes (bgmf_query_sizes) and
 *                 BGMF_OPT_RATINGS_BUDGET allows it; otherwise the ratings
 *                 stream, with ws_bytes minus the tables (or the budget
 *                 option, if smaller) as their device budget;
 *   pinned_host, pinned_bytes  pinned host memory (hipHostMalloc, or a
 *                 PyTorch pin_memory tensor) for streamed ratings; NULL if
 *                 the ratings will not stream;
 *   hip_stream    as bgmf_set_stream (NULL: the handle's own stream).
 * Every pointer must start on a 256-byte boundary; U, V and the workspace
 * must be device memory of the handle's device (BGMF_E_ARG otherwise).  A
 * workspace smaller than the tables -> BGMF_E_BUDGET.  The caller keeps
 * ownership; the buffers must outlive their use by the handle and must not
 * be used by the caller while the handle's work on them is in flight.  After
 * binding, bgmf_load_coo, bgmf_epoch and bgmf_rmse allocate no memory
 * (BGMF_OPT_ALLOC_COUNT does not move); the handle still allocates its
 * small fixed tables at bgmf_create, the block trace when BGMF_OPT_TRACE is
 * set, and bgmf_rmse_coo's temporaries. */
int bgmf_bind(bgmf_t *h, float *U_dev, float *V_dev, void *ws_dev, size_t ws_bytes,
              void *pinned_host, size_t pinned_bytes, void *hip_stream);

/* Copy initial factors from host memory: U is n x k, V is m x k, row-major
 * fp32 (u_i = U[i*k .. i*k+k)).  Algorithm 1 starts from random factors;
 * the caller draws them.  Synchronous. */
int bgmf_set_factors(bgmf_t *h, const float *U, const float *V);

/* Load nnz ratings given as host COO arrays (rows[e], cols[e], vals[e]),
 * e = 0..nnz-1, and bucket them into the p x p grid (Eq. 4) on the device.
 *   1 <= nnz < 2^31.  Indices outside [0,n) x [0,m) -> BGMF_E_RANGE;
 *   non-finite values -> BGMF_E_NONFINITE.  Duplicate (i, j) pairs are
 *   separate ratings.  Replaces any earlier ratings.  Synchronous. */
int bgmf_load_coo(bgmf_t *h, const int32_t *rows, const int32_t *cols, const float *vals,
                  int64_t nnz);

/* One epoch (one CPU step of Algorithm 1): strata s = 0..p-1 in order, every
 * loaded rating updated once per block pass (Eq. 2-3; one pass unless
 * BGMF_OPT_BLOCK_PASSES says otherwise).
 * alpha > 0 and beta >= 0, both finite.  Needs factors and ratings.
 * Asynchronous on the handle's stream; a device-side failure is reported by
 * the next synchronising call. */
int bgmf_epoch(bgmf_t *h, float alpha, float beta);

/* Root-mean-square error over all loaded ratings with the current factors:
 * sqrt((1/nnz) sum_e (x_e - u_i.v_j)^2), dots in fp32, sum in fp64 (the
 * whole-matrix RMSE of Algorithm 1's termination test).  Waits for the
 * stream. */
int bgmf_rmse(bgmf_t *h, double *out);

/* Block boundaries.  By default the grid has the paper's equal blocks
 * (Eq. 4): row-block R holds rows [ceil(R n/p), ceil((R+1) n/p)), and the
 * same for columns.  bgmf_set_cuts replaces them by caller-given cut points
 * (row_cuts, col_cuts: p + 1 values each, host memory, strictly increasing
 * from 0 to n, resp. m; row-blocks at most 65536 rows, column-blocks at most
 * 65536 columns wide, else BGMF_E_ARG): row i is then in the block R with
 * row_cuts[R] <= i < row_cuts[R+1].  Strata, the order inside a block and
 * the update are unchanged.  Blocks of unequal size are the paper's
 * suggested extension (Section 3); balanced blocks shorten the serial
 * chains of skewed data.  Drops any loaded ratings (load them again).
 * bgmf_get_cuts copies the cut points in effect (either pointer may be NULL). */
int bgmf_set_cuts(bgmf_t *h, const int64_t *row_cuts, const int64_t *col_cuts);
int bgmf_get_cuts(const bgmf_t *h, int64_t *row_cuts, int64_t *col_cuts);

/* Cut points that balance the ratings over the blocks, from host COO arrays
 * (no handle needed): for each dimension, block b (b = 0..p-2) ends at the
 * first index where the running count of ratings reaches ceil(remaining /
 * blocks left) — or just before that index if it alone holds that many, so
 * that heavy rows and columns get blocks of their own — within 1 ..
 * max_rows (max_cols) indices and leaving every later block at least one
 * index and at most max_rows (max_cols).  Writes
 * p + 1 values to each output.  Exact integer arithmetic.  BGMF_E_ARG if no
 * such cuts exist (p > min(n, m), or p * max_rows < n, or p * max_cols < m);
 * BGMF_E_RANGE for a rating outside the matrix.  Errors are reported by
 * bgmf_last_error(NULL). */
int bgmf_balanced_cuts(int64_t n, int64_t m, int32_t p, const int32_t *rows, const int32_t *cols,
                       int64_t nnz, int64_t max_rows, int64_t max_cols, int64_t *row_cuts,
                       int64_t *col_cuts);

/* Data re-ordering (the extension Section 3 names beside variable block
 * sizes), from host COO arrays (no handle needed): a relabelling of user and
 * item ids that keeps the paper's equal-dimension blocks (Eq. 4) but spreads
 * the heavy rows and columns over them.  For each dimension, the indices in
 * descending number of ratings (ties: ascending index) are dealt one by one
 * to the block with the smallest number of ratings so far that still has a
 * free place (ties: lowest block); inside a block, new ids are given in the
 * order of dealing.  Writes row_newid[i] (n values) and col_newid[j] (m
 * values), each a permutation; the caller renames its ratings (and initial
 * factor rows) with them and loads the renamed matrix, on which the method
 * runs unchanged.  Exact integer arithmetic.  BGMF_E_ARG for p outside
 * [1, min(n, m)]; BGMF_E_RANGE for a rating outside the matrix.  Errors are
 * reported by bgmf_last_error(NULL). */
int bgmf_reorder_ids(int64_t n, int64_t m, int32_t p, const int32_t *rows, const int32_t *cols,
                     int64_t nnz, int32_t *row_newid, int32_t *col_newid);

/* RMSE of the current factors over nnz caller-given ratings in host COO
 * arrays (for example a held-out split, the paper's Table 2 "test RMSE"):
 * sqrt((1/nnz) sum_e (vals[e] - u_rows[e].v_cols[e])^2), dots in fp32, sum
 * in fp64.  The ratings need not be loaded and are not kept.  Index and
 * value checks as in bgmf_load_coo.  Needs factors.  Allocates temporary
 * device memory for the ratings.  Waits for the stream. */
int bgmf_rmse_coo(bgmf_t *h, const int32_t *rows, const int32_t *cols, const float *vals,
                  int64_t nnz, double *out);

/* bgmf_rmse_coo for callers that cannot allocate memory (code under HIP
 * graph capture, tight serving loops, harnesses that forbid hipMalloc):
 * the same RMSE, from the same kernel with the same fixed reduction order
 * (so the same bits), over nnz ratings already in device memory:
 *   rows_dev, cols_dev: int32 device arrays, vals_dev: fp32 device array,
 *   nnz entries each, owned by the caller and read during the call;
 *   out: host double receiving the RMSE.
 * It allocates nothing: the reduction's partial sums, its result and an
 * error word live in a static device array of (4096 + 2) * 8 = 32,784
 * bytes, one per GPU, held until the process ends.  Every call on a GPU
 * shares that GPU's array, so calls that overlap on one GPU (other
 * threads, other handles, other streams) race and their results are
 * undefined; serialise them.  nnz outside [1, 2^31) -> BGMF_E_ARG (the
 * largest input the array's fixed-grid reduction serves); needs factors
 * (BGMF_E_STATE).  Indices and values are checked on the device: a rating
 * outside the matrix -> BGMF_E_RANGE, a non-finite value ->
 * BGMF_E_NONFINITE (such ratings are never used to read factors), and
 * *out is not written.  Waits for the handle's stream. */
int bgmf_rmse_coo_dev(bgmf_t *h, const int32_t *rows_dev, const int32_t *cols_dev,
                      const float *vals_dev, int64_t nnz, double *out);

/* Algorithm 1's outer loop (CPU_STEPS = max_epochs, termination deviation
 * delta): RMSE of the initial factors, then up to max_epochs times one epoch
 * and its RMSE pass, stopping after the first epoch whose RMSE differs from
 * the previous one by less than delta (Section 1.3).
 *   *epochs_run receives the number of epochs run;
 *   rmse_history, if not NULL, must hold max_epochs + 1 doubles and receives
 *     the initial RMSE and the RMSE after each epoch run.
 * max_epochs >= 1, delta >= 0 and finite; alpha, beta as for bgmf_epoch.
 * BGMF_E_NONFINITE if an RMSE is not finite (the step diverges; the history
 * up to that epoch is written).  Waits for the stream after every epoch. */
int bgmf_fit(bgmf_t *h, float alpha, float beta, int32_t max_epochs, double delta,
             int32_t *epochs_run, double *rmse_history);

/* Copy the current factors to host memory (row-major n x k and m x k):
 * the U and V that Algorithm 1 returns.  Either pointer may be NULL to
 * skip it.  Waits for the stream. */
int bgmf_get_factors(bgmf_t *h, float *U, float *V);

/* Bucketing result, for bit-exact checks:
 *   block_ptr[q], q = 0..p*p: number of ratings in slots < q, where slot
 *     q = s*p + R is block (R, (R+s) mod p) of stratum s;
 *   perm[t], t = 0..nnz-1: input position of the t-th rating in slot order,
 *     each slot sorted by (row, input position).
 * Either pointer may be NULL.  Waits for the stream. */
int bgmf_get_layout(bgmf_t *h, int64_t *block_ptr, int32_t *perm);

/* Wait for all work on the handle's stream and report any device-side
 * failure of earlier asynchronous calls. */
int bgmf_sync(bgmf_t *h);

/* Device pointers of U (n x k) and V (m x k), row-major fp32: the handle's
 * own (valid until bgmf_destroy) or the caller's bound ones.  Either output
 * may be NULL. */
int bgmf_factor_ptrs(bgmf_t *h, float **U_dev, float **V_dev);

/* Options (bgmf_set_option / bgmf_get_option). */
#define BGMF_OPT_SCHEDULE      1 /* 0 (default): automatic, one persistent launch per
                                    epoch whose waves hand column-blocks over with
                                    device-side flags when V is staged in LDS and all
                                    p waves fit on the device at once, else one
                                    launch per stratum; 1: one launch per stratum;
                                    2: persistent whenever the waves fit (with V in
                                    global memory every V access is then
                                    device-scope, which is slower) */
#define BGMF_OPT_WAIT_LIMIT_US 2 /* limit of one device-side wait, microseconds
                                    (default 10,000,000) */
#define BGMF_OPT_XCD_REMAP     3 /* 1 (default): place neighbouring row-blocks on
                                    the same XCD; 0: plain workgroup order */
#define BGMF_OPT_RATINGS_BUDGET 4 /* device bytes the ratings may occupy, at load
                                    and during epochs; 0 (default) = no limit.
                                    Takes effect at the next bgmf_load_coo.  If
                                    the one-pass bucketing (about 48 bytes per
                                    rating, see bgmf_query_sizes) does not fit,
                                    the ratings are kept in pinned host memory in
                                    stratum order, bucketed group by group (each
                                    group of whole blocks gathered from the input,
                                    sorted on the device within the budget, and
                                    copied out; the largest block must fit, else
                                    BGMF_E_BUDGET).  The budget is
                                    then split into a ring of 3 (else 2) device
                                    slots and a resident region: the first strata
                                    of the epoch stay resident (copied once, at
                                    load), the others stream through the ring in
                                    chunks of consecutive strata, each copied on a
                                    side stream while earlier strata are swept.  A
                                    slot must hold the widest stratum plus 256
                                    records (else BGMF_E_BUDGET); U and V stay
                                    resident.  This applies the paper's point that
                                    a block-based sweep only needs the blocks in
                                    flight on the device (Sections 1.2 and 2.2).
                                    Results are bit-identical to the in-core sweep. */
#define BGMF_OPT_STREAM_SLOTS  5 /* read-only: number of ring slots when the
                                    loaded ratings stream from host memory, else 0 */
#define BGMF_OPT_V_STAGING     6 /* where a wave keeps the column slice of V it
                                    works on: 0 (default) automatic, 1 staged in
                                    LDS (BGMF_E_UNSUPPORTED if (ceil(m/p) + 1) x k'
                                    floats, k' = k rounded up to a power of two,
                                    exceed the LDS of a workgroup), 2 global
                                    memory.  Automatic picks LDS when the slice
                                    fits with all p waves resident at once.
                                    Results are bit-identical either way. */
#define BGMF_OPT_PLACEMENT     7 /* read-only: how the next epoch runs, bits:
                                    1 = V slice in LDS, 2 = V in global memory,
                                    4 = one persistent launch (else one launch per
                                    stratum) */
#define BGMF_OPT_STREAM_CHUNKS 8 /* read-only: chunks of strata streamed per epoch
                                    when the ratings stream from host memory, else 0 */
#define BGMF_OPT_RESIDENT_STRATA 9 /* read-only: strata whose ratings stay on the
                                    device (all p unless they stream) */
#define BGMF_OPT_BLOCK_PASSES 10 /* GPU_STEPS of Algorithm 1 (Section 1.3, Table 3):
                                    passes of the SGD sweep over each block, its
                                    ratings in the same order every pass, before the
                                    block's column slice moves on; 1 (default) to
                                    1024.  An epoch then makes passes x nnz updates.
                                    Takes effect at the next bgmf_epoch, so a caller
                                    can vary it from epoch to epoch (the paper's
                                    variable block iterations). */
#define BGMF_OPT_SINGLE_COLUMN 11 /* 1 (default): with V staged in LDS, a block
                                    whose ratings all lie on one column (always so
                                    when its column-block is one column wide, as a
                                    heavy item given a column-block of its own
                                    through bgmf_set_cuts; often so for a heavy
                                    item's blocks after bgmf_reorder_ids) and
                                    whose consecutive ratings never share a row
                                    keeps that column's v in
                                    registers from its first rating to its last
                                    and forms each rating's partial products
                                    before the previous error is known (a shorter
                                    dependency chain); 0: such blocks take the
                                    general step.  The stored updates are the same
                                    formula, the next dot product rounds
                                    differently, so results differ in the last
                                    bits (both match the exact sequential
                                    schedule within the parity tolerance). */
#define BGMF_OPT_LDS_HANDOVER 12 /* 1 (default): with V staged in LDS and one
                                    persistent launch, the waves of a workgroup
                                    (consecutive row-blocks) pass column slices
                                    to each other through LDS; only slices that
                                    enter or leave the workgroup, and all of them
                                    after a launch, go through global memory.
                                    Used when the larger LDS ring still lets every
                                    wave be resident.  0: every hand-over goes
                                    through global memory.  Same arithmetic, so
                                    the results are bit-identical. */
#define BGMF_OPT_TRACE 13        /* 1: each bgmf_epoch records a block trace
                                    (bgmf_get_trace); the handle holds 16 p^2
                                    bytes of device memory for it while on.
                                    0 (default): off, and that memory is
                                    freed.  The results do not change. */
#define BGMF_OPT_ALLOC_COUNT 14  /* read-only: device and pinned host allocations
                                    the handle has made since bgmf_create */
#define BGMF_OPT_LOAD_PEAK 15    /* read-only: device bytes the last bgmf_load_coo
                                    used for ratings at its peak (records, perm,
                                    bucketing temporaries, stream slots and
                                    resident strata; block tables not counted);
                                    within the ratings budget when one is set, or
                                    within the bytes needed to bucket the largest
                                    block if those are more (a handle that owns
                                    its memory; a bound one stays within its
                                    workspace or fails with BGMF_E_BUDGET) */
#define BGMF_OPT_LOAD_GROUPS 16  /* read-only: groups of blocks the last streamed
                                    bgmf_load_coo gathered and sorted one at a
                                    time (0 for an in-core load) */
int bgmf_set_option(bgmf_t *h, int32_t option, int64_t value);
int bgmf_get_option(const bgmf_t *h, int32_t option, int64_t *value);

/* Timing of the most recent bgmf_epoch and bgmf_rmse, measured with HIP
 * events on the handle's stream around their kernels, in milliseconds
 * (NaN if not run yet).  Waits for the stream. */
int bgmf_get_timing(bgmf_t *h, double *epoch_ms, double *rmse_ms);

/* Block trace of the most recent bgmf_epoch (with BGMF_OPT_TRACE on), a
 * tool for checking and analysing the stratum schedule of Section 1.1
 * (Algorithm 1's inner loop): for block slot q = s*p + b (the block
 * (b, (b+s) mod p) of stratum s),
 *   begin[q] = device clock when the block starts, after its waits for the
 *              previous holder of its column-block (a neighbour's progress
 *              or, with one launch per stratum, the launch boundary);
 *   end[q]   = device clock when the block hands its results on, before its
 *              progress word moves.
 * A block that no launch of the epoch visited (an empty stratum of a
 * streamed epoch) has begin = end = 0.  Values are ticks of the device's
 * constant-rate clock, *ticks_per_s per second.  begin and end are host
 * arrays of p*p values each, owned by the caller.  Waits for the stream.
 * BGMF_E_STATE if no epoch was traced since the option was set. */
int bgmf_get_trace(bgmf_t *h, int64_t *begin, int64_t *end, int64_t *ticks_per_s);

/* Serial-chain statistics of the loaded ratings, from the block sizes:
 *   out[0] = largest column-block total  (max_C sum_R nnz(R, C))
 *   out[1] = largest row-block total     (max_R sum_C nnz(R, C))
 *   out[2] = sum over strata of the largest block of the stratum
 *   out[3] = number of non-empty blocks
 * Needs ratings. */
int bgmf_chain_stats(bgmf_t *h, int64_t out[4]);

#ifdef __cplusplus
}
#endif

#endif /* BGMF_H */
