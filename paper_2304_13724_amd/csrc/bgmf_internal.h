// Internal declarations shared by the HIP sources of libbgmf (gfx950 only).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace bgmfk {

// ---------------------------------------------------------------------------
// Rating record (8 bytes), stored contiguously per row-block ("wave stream"):
//   .x = local row (16 bits) | local column << 16 (16 bits)
//   .y = rating value (fp32 bits)
// Local indices are relative to the block's first row / first column.
// ---------------------------------------------------------------------------
constexpr int kRowBits = 16;
constexpr int kColShift = 16;
constexpr int kColBits = 16;
constexpr uint32_t kRowMask = (1u << kRowBits) - 1u;
constexpr uint32_t kColMask = (1u << kColBits) - 1u;
#ifndef BGMF_PREFETCH
#define BGMF_PREFETCH 16
#endif
constexpr int kPrefetch = BGMF_PREFETCH;     // prefetch distance of factor rows (ratings)
constexpr int kRecPad = 256;                 // padding records after the last stream

// Block geometry of the p x p grid, as cut points: row-block R holds rows
// [rcut[R], rcut[R+1]), column-block C columns [ccut[C], ccut[C+1]) (p + 1
// strictly increasing values from 0 to n, resp. m, in device memory).  The
// paper's equal blocks (Eq. 4) are rcut[R] = ceil(R n / p), i.e. row i in
// block floor(i p / n); other cut points give blocks of unequal size.
__host__ __device__ __forceinline__ int64_t equal_cut(int64_t R, int64_t n, int32_t p) {
  return (R * n + p - 1) / p;
}

__device__ __forceinline__ int32_t block_of(const int64_t *cut, int32_t p, int64_t i) {
  int32_t lo = 0, hi = p - 1;  // the last R with cut[R] <= i
  while (lo < hi) {
    const int32_t mid = (lo + hi + 1) >> 1;
    if (cut[mid] <= i) lo = mid;
    else hi = mid - 1;
  }
  return lo;
}

struct Grid {
  int64_t n, m;
  int32_t p;
  const int64_t *rcut, *ccut;
  __device__ __forceinline__ int64_t row_start(int64_t R) const { return rcut[R]; }
  __device__ __forceinline__ int64_t col_start(int64_t C) const { return ccut[C]; }
  __device__ __forceinline__ int32_t row_block(int64_t i) const { return block_of(rcut, p, i); }
  __device__ __forceinline__ int32_t col_block(int64_t j) const { return block_of(ccut, p, j); }
};

// Arguments of the SGD sweep kernels.
struct SgdParams {
  float *U;                  // n x k, plus one spare row (index n)
  float *V;                  // m x k
  const uint2 *rec;          // rating records (+ kRecPad readable past the last one used)
  const int64_t *blk;        // block offsets: block (b, s) is records
                             // [blk[x], blk[x + 1]) with x = b*stride_b + s*stride_s
  int64_t stride_b, stride_s;
  int64_t rec_origin;        // record of offset blk[x] is rec[blk[x] - rec_origin]
  int64_t *flags;            // [p * kFlagStride]: strata completed by each row-block
  int32_t *err;              // device error word (0 = ok)
  int64_t n, m;
  const int64_t *rcut, *ccut;  // block cut points (see Grid)
  int32_t k, p;
  int32_t cols_max;          // largest column-block width
  int32_t s_begin, s_end;    // strata of this launch
  int64_t g_base;            // global stratum index of stratum 0 of this epoch
  int64_t wait_ticks;        // wait limit in ticks of the constant clock (s_memrealtime)
  float alpha, beta;
  int32_t xcd_remap;
  int32_t passes;            // sweeps of each block before the next (GPU_STEPS >= 1)
  int32_t single_col;        // 1: blocks whose ratings are all on one column keep v in
                             // registers (the folded one-column step)
  const uint8_t *nofold;     // [p * p], slot s*p + b: 1 if the block cannot take the folded
                             // step (a row repeats in consecutive ratings, or two columns)
  int32_t lds_ring;          // LDS sweep, persistent launches: areas in the workgroup's
                             // hand-over ring (0: each wave its own area, global hand-over)
  int64_t *trace;            // null, or [2 p p]: per block slot s*p + b, the clock when the
                             // block starts and when it hands its results on
  int32_t wpg;               // waves per workgroup (set by launch_sgd; a kernel argument
                             // arrives with the others, blockDim from the dispatch packet
                             // would cost a memory round trip at every launch)
};
constexpr int kFlagStride = 16;  // int64 words per flag (one 128-byte line)
constexpr int kWavesPerGroup = 4;
constexpr int kErrTimeout = 1;
constexpr int kErrLayout = 2;  // a bucketing write fell outside its array

// Where the sweep keeps the column slice of V it is working on.
constexpr int kVLds = 0;             // staged in LDS, (cols_max + 1) x kp floats per wave
constexpr int kVGlobal = 1;          // global memory, plain cached accesses (one stratum per launch)
constexpr int kVGlobalCoherent = 2;  // global memory, device-scope accesses (persistent launch)

// Launchers (defined in the .hip files); all enqueue on `stream`.
// One wave per row-block; a workgroup holds waves_per_group (1, 2 or 4)
// row-blocks, each with its own LDS area: the column slice (kVLds) or the
// ring of recent results, sgd_gv_lds_per_wave(kp) bytes (global V).
hipError_t launch_sgd(const SgdParams &P, int kp, int vmode, int waves_per_group, bool cooperative,
                      size_t lds_bytes, hipStream_t stream);
hipError_t sgd_occupancy(int kp, bool mask, int vmode, int waves_per_group, size_t lds_bytes,
                         int *groups_per_cu);
hipError_t sgd_set_lds_limit(int kp, bool mask, int vmode, size_t lds_bytes);
size_t sgd_gv_lds_per_wave(int kp);
// LDS of one area of the LDS sweep: cols_max + 1 column slots.  A workgroup
// of w waves needs sgd_lds_bytes(kp, cols_max, w, ring): w areas (ring = 0)
// or a hand-over ring of `ring` areas, and one progress word per wave.
size_t sgd_lds_per_wave(int kp, int cols_max);
size_t sgd_lds_bytes(int kp, int cols_max, int waves_per_group, int ring);

hipError_t launch_rmse(const uint2 *rec, const int64_t *wblock_ptr, const float *U,
                       const float *V, const Grid &G, int64_t rows_max, int32_t k, int64_t nnz,
                       double *partials, double *out, size_t lds_limit, hipStream_t stream);
// Out-of-core pieces of the RMSE pass: zero the partial sums
// (kRmseStrataGroups per row-block), add the squared errors of strata
// [s0, s1) (records of block (b, s) at rec[block_ptr[s*p + b] - rec_origin]),
// and finish.
constexpr int kRmseStrataGroups = 16;
hipError_t rmse_stratum_begin(double *partials, int32_t p, hipStream_t stream);
hipError_t rmse_stratum_add(const uint2 *rec, int64_t rec_origin, const int64_t *block_ptr,
                            int32_t s0, int32_t s1, const float *U, const float *V,
                            const Grid &G, int32_t k, double *partials, hipStream_t stream);
hipError_t rmse_stratum_end(const double *partials, int32_t p, int64_t nnz, double *out,
                            hipStream_t stream);
size_t rmse_partials_count(int32_t p);
// RMSE over caller-given COO ratings already on the device (rows, cols,
// vals of nnz ratings); partials must hold rmse_coo_partials_count() doubles.
// *bad is cleared first (by a kernel), then receives bit 1 for a rating
// outside the n x m matrix and bit 2 for a non-finite value (such ratings
// are skipped without reading factors).
constexpr int kRmseCooGroups = 1024;
size_t rmse_coo_partials_count();
hipError_t launch_rmse_coo(const int32_t *rows, const int32_t *cols, const float *vals,
                           int64_t nnz, const float *U, const float *V, int32_t k, int64_t n,
                           int64_t m, double *partials, double *out, int32_t *bad,
                           hipStream_t stream);

// Batched bucketing (ratings that are never all on the device at once).
// Slot counts accumulate over batches (slot_count: p*p + 1 int64, zeroed by
// the caller); bucket_offsets turns them into block_ptr (exclusive prefix,
// total appended) using scan_scratch_bytes(p*p) of scratch.  A group of
// whole blocks, slots [q0, q1), is gathered in input order by
// bucket_select_batch over the same batches (flag and pos: cnt + 1 int64
// each; fill: device counter of ratings gathered so far, zeroed per group),
// then sorted by bucket() as a load of its own; bucket_map_perm turns the
// group-local positions of its perm into input positions.
struct GroupArrays {
  int32_t *rows, *cols;
  float *vals;
  int32_t *e;   // input position of each gathered rating
  int64_t cap;  // capacity of each array
};
size_t scan_scratch_bytes(int64_t len);
hipError_t bucket_count_batch(const int32_t *rows, const int32_t *cols, int64_t cnt,
                              const Grid &G, int64_t *slot_count, hipStream_t stream);
hipError_t bucket_offsets(const int64_t *slot_count, int64_t slots, int64_t *block_ptr,
                          void *scratch, size_t scratch_bytes, hipStream_t stream);
hipError_t bucket_select_batch(const int32_t *rows, const int32_t *cols, const float *vals,
                               int64_t cnt, int64_t e0, const Grid &G, int64_t q0, int64_t q1,
                               int64_t *flag, int64_t *pos, void *scratch, size_t scratch_bytes,
                               int64_t *fill, const GroupArrays &g, int32_t *err,
                               hipStream_t stream);
hipError_t bucket_map_perm(int32_t *perm, const int32_t *g_e, int64_t cnt, int32_t *err,
                           hipStream_t stream);

// Bucketing: from device COO to the block layout.  Scratch buffers are
// allocated by the caller (see bucket_scratch_bytes).
struct BucketOut {
  int64_t *block_ptr;   // [p*p + 1] stratum-major slot starts
  int64_t *wblock_ptr;  // [p*p + 1] wave-major block starts
  int32_t *perm;        // [nnz] input position of each slot-ordered rating
  uint2 *rec;           // [nnz + kRecPad] wave-major records
  uint8_t *nofold;      // [p*p] slot q: 1 if two consecutive ratings of the block share a
                        // row or differ in column (set here; zeroed by the caller)
};
// Scratch of a bucketing of nnz ratings over nq slots.
size_t bucket_scratch_bytes(int64_t nnz, int64_t nq);
// Sorts ratings whose slots all lie in [q0, q0 + nq) (any rating outside
// raises kErrLayout).  out.block_ptr receives nq + 1 offsets relative to
// slot q0; perm the positions in the given arrays; nofold is indexed by the
// global slot.  stratum_major: records in slot order; otherwise (only for
// the whole grid, q0 = 0 and nq = p*p) records in wave-major order, with
// out.wblock_ptr.
// rows_max: the widest row-block (sets the key width).
hipError_t bucket(const int32_t *rows, const int32_t *cols, const float *vals, int64_t nnz,
                  const Grid &G, int64_t rows_max, int64_t q0, int64_t nq, bool stratum_major,
                  void *scratch, size_t scratch_bytes, const BucketOut &out, int32_t *err,
                  hipStream_t stream);

}  // namespace bgmfk
