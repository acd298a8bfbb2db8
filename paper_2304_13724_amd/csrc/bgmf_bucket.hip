// Bucketing of COO ratings into the p x p block grid (Eq. 4) and the strata
// of Section 1.1, on the device, bit-exact:
//   slot q = s*p + R for the block (R, C = (R + s) mod p) of stratum s;
//   inside a slot, ascending row, ties in ascending input position.
//
// The order is produced by a stable LSD radix sort (8-bit digits) of the
// composite key (q, local row) with the input position as the value; a
// stable sort keeps equal keys in input order, which is the tie rule.
// Every pass is three kernels: per-tile digit histograms, an exclusive
// scan of the digit-major histogram table, and a scatter that ranks each
// element among the equal digits of its tile with wave ballots.  Nothing
// depends on the order in which atomics or workgroups run.
//
// The result is written twice: perm/block_ptr in slot order (stratum-major,
// for callers and tests) and the rating records in wave-major order (all
// blocks of row-block b, strata 0..p-1, contiguously), which is the order in
// which one wave of the SGD sweep consumes them.
#include "bgmf_internal.h"

namespace bgmfk {
namespace {

constexpr int kThreads = 256;
constexpr int kItems = 16;
constexpr int kTile = kThreads * kItems;  // elements per radix tile
constexpr int kBins = 256;
constexpr int kScanItems = 8;
constexpr int kScanTile = kThreads * kScanItems;

__device__ __forceinline__ int64_t gid() {
  return (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
}

// ----------------------------------------------------------------- keys

// Key of a rating: (slot - q0, local row).  Every rating's slot lies in
// [q0, q0 + nq); a slot outside it gets the key nq (past every table) and
// raises the layout error.
__global__ void k_make_keys(const int32_t *__restrict__ rows, const int32_t *__restrict__ cols,
                            int64_t nnz, Grid G, int rbits, int64_t q0, int64_t nq,
                            uint64_t *__restrict__ keys, int32_t *__restrict__ idx, int32_t *err) {
  for (int64_t e = gid(); e < nnz; e += (int64_t)gridDim.x * blockDim.x) {
    const int64_t i = rows[e], j = cols[e];
    const int64_t R = G.row_block(i);
    const int64_t C = G.col_block(j);
    int64_t s = C - R;
    if (s < 0) s += G.p;
    int64_t q = s * G.p + R - q0;
    if (q < 0 || q >= nq) {
      atomicOr(err, kErrLayout);
      q = nq;
    }
    keys[e] = ((uint64_t)q << rbits) | (uint64_t)(i - G.row_start(R));
    idx[e] = (int32_t)e;
  }
}

// ----------------------------------------------------------------- scan
// Exclusive scan of int64 values with the total appended: out[0..len].

__device__ int64_t block_exclusive_scan(int64_t v, int64_t *sh, int64_t *total) {
  const int t = threadIdx.x;
  sh[t] = v;
  __syncthreads();
  for (int off = 1; off < kThreads; off <<= 1) {
    int64_t add = (t >= off) ? sh[t - off] : 0;
    __syncthreads();
    sh[t] += add;
    __syncthreads();
  }
  const int64_t incl = sh[t];
  *total = sh[kThreads - 1];
  __syncthreads();
  return incl - v;
}

__global__ void __launch_bounds__(kThreads)
k_scan_tile(const int64_t *__restrict__ in, int64_t len, int64_t *__restrict__ out,
            int64_t *__restrict__ tile_sums) {
  __shared__ int64_t sh[kThreads];
  const int64_t base = (int64_t)blockIdx.x * kScanTile + (int64_t)threadIdx.x * kScanItems;
  int64_t v[kScanItems];
  int64_t run = 0;
#pragma unroll
  for (int i = 0; i < kScanItems; ++i) {
    v[i] = (base + i < len) ? in[base + i] : 0;
    run += v[i];
  }
  int64_t total;
  int64_t pre = block_exclusive_scan(run, sh, &total);
#pragma unroll
  for (int i = 0; i < kScanItems; ++i) {
    if (base + i < len) out[base + i] = pre;
    pre += v[i];
  }
  if (threadIdx.x == 0) tile_sums[blockIdx.x] = total;
}

__global__ void k_scan_add(int64_t *__restrict__ out, int64_t len,
                           const int64_t *__restrict__ tile_off) {
  for (int64_t i = gid(); i < len; i += (int64_t)gridDim.x * blockDim.x)
    out[i] += tile_off[i / kScanTile];
}

__global__ void k_copy1(const int64_t *src, int64_t *dst) { *dst = *src; }

// Bump allocator over the caller's scratch buffer.
struct Arena {
  char *base;
  size_t size, used;
  template <class T>
  T *take(size_t count) {
    size_t off = (used + 255) & ~(size_t)255;
    size_t bytes = count * sizeof(T);
    if (off + bytes > size) return nullptr;
    used = off + bytes;
    return reinterpret_cast<T *>(base + off);
  }
};

int grid_for(int64_t count, int threads, int cap = 65536) {
  int64_t g = (count + threads - 1) / threads;
  if (g < 1) g = 1;
  if (g > cap) g = cap;
  return (int)g;
}

size_t scan_scratch_count(int64_t len) {
  size_t total = 0;
  while (true) {
    int64_t tiles = (len + kScanTile - 1) / kScanTile;
    if (tiles < 1) tiles = 1;
    total += (size_t)tiles + (size_t)tiles + 1 + 64;
    if (tiles == 1) break;
    len = tiles;
  }
  return total;
}

hipError_t scan_exclusive(const int64_t *in, int64_t len, int64_t *out, Arena &ar,
                          hipStream_t st) {
  int64_t tiles = (len + kScanTile - 1) / kScanTile;
  if (tiles < 1) tiles = 1;
  int64_t *sums = ar.take<int64_t>((size_t)tiles);
  if (!sums) return hipErrorOutOfMemory;
  hipLaunchKernelGGL(k_scan_tile, dim3((unsigned)tiles), dim3(kThreads), 0, st, in, len, out,
                     sums);
  if (tiles == 1) {
    hipLaunchKernelGGL(k_copy1, dim3(1), dim3(1), 0, st, sums, out + len);
    return hipGetLastError();
  }
  int64_t *off = ar.take<int64_t>((size_t)tiles + 1);
  if (!off) return hipErrorOutOfMemory;
  hipError_t e = scan_exclusive(sums, tiles, off, ar, st);
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(k_scan_add, dim3(grid_for(len, kThreads)), dim3(kThreads), 0, st, out,
                     len, off);
  hipLaunchKernelGGL(k_copy1, dim3(1), dim3(1), 0, st, off + tiles, out + len);
  return hipGetLastError();
}

// ----------------------------------------------------------------- radix sort
// Element order inside a tile: index = tile*kTile + i*kThreads + thread, for
// i = 0..kItems-1.  The histogram and the scatter use the same order.

__global__ void __launch_bounds__(kThreads)
k_radix_hist(const uint64_t *__restrict__ keys, int64_t nnz, int shift, int64_t tiles,
             int64_t *__restrict__ counts) {
  __shared__ int hist[kBins];
  hist[threadIdx.x] = 0;
  __syncthreads();
  const int64_t base = (int64_t)blockIdx.x * kTile + threadIdx.x;
#pragma unroll
  for (int i = 0; i < kItems; ++i) {
    const int64_t e = base + (int64_t)i * kThreads;
    if (e < nnz) atomicAdd(&hist[(keys[e] >> shift) & (kBins - 1)], 1);
  }
  __syncthreads();
  counts[(int64_t)threadIdx.x * tiles + blockIdx.x] = hist[threadIdx.x];
}

__global__ void __launch_bounds__(kThreads)
k_radix_scatter(const uint64_t *__restrict__ kin, const int32_t *__restrict__ vin,
                uint64_t *__restrict__ kout, int32_t *__restrict__ vout, int64_t nnz, int shift,
                int64_t tiles, const int64_t *__restrict__ offsets, int32_t *err) {
  __shared__ int cnt[kWavesPerGroup][kBins];
  __shared__ int run[kBins];
  const int t = threadIdx.x;
  const int lane = t & 63;
  const int wave = t >> 6;
  for (int w = 0; w < kWavesPerGroup; ++w) cnt[w][t] = 0;
  run[t] = 0;
  __syncthreads();
  const int64_t base = (int64_t)blockIdx.x * kTile + t;
  const uint64_t lt_mask = (lane == 0) ? 0ull : (~0ull >> (64 - lane));
  for (int i = 0; i < kItems; ++i) {
    const int64_t e = base + (int64_t)i * kThreads;
    const bool valid = e < nnz;
    uint64_t key = valid ? kin[e] : 0;
    const int32_t val = valid ? vin[e] : 0;
    const int digit = (int)((key >> shift) & (kBins - 1));
    // lanes holding the same digit
    uint64_t peers = __ballot(valid);
#pragma unroll
    for (int bit = 0; bit < 8; ++bit) {
      const bool set = (digit >> bit) & 1;
      const uint64_t b = __ballot(set);
      peers &= set ? b : ~b;
    }
    const int rank = __popcll(peers & lt_mask);
    if (valid && rank == 0) cnt[wave][digit] = __popcll(peers);
    __syncthreads();
    if (valid) {
      int off = run[digit];
      for (int w = 0; w < wave; ++w) off += cnt[w][digit];
      const int64_t dst = offsets[(int64_t)digit * tiles + blockIdx.x] + off + rank;
      if (dst >= 0 && dst < nnz) {
        kout[dst] = key;
        vout[dst] = val;
      } else {
        atomicOr(err, kErrLayout);
      }
    }
    __syncthreads();
    int add = 0;
    for (int w = 0; w < kWavesPerGroup; ++w) {
      add += cnt[w][t];
      cnt[w][t] = 0;
    }
    run[t] += add;
    __syncthreads();
  }
}

// ----------------------------------------------------------------- layout

// Ratings per slot, from the sorted keys: a slot's ratings are the run
// [start, end) of equal slots, so the first rating of each run subtracts its
// position from its slot's count and adds it to the count of the run before
// (whose end it is), and the last rating adds nnz: two atomics per occupied
// slot instead of one per rating (counts start at 0; the arithmetic wraps
// modulo 2^64 and ends at end - start).  Keys of out-of-range slots sort
// last and raise the layout error.
__global__ void k_slot_count(const uint64_t *__restrict__ keys, int64_t nnz, int rbits,
                             int64_t slots, unsigned long long *__restrict__ count, int32_t *err) {
  for (int64_t t = gid(); t < nnz; t += (int64_t)gridDim.x * blockDim.x) {
    const uint64_t q = keys[t] >> rbits;
    if (q >= (uint64_t)slots) {
      atomicOr(err, kErrLayout);
      continue;
    }
    const uint64_t qp = t > 0 ? keys[t - 1] >> rbits : ~0ull;
    if (q != qp) {
      atomicAdd(&count[q], 0ull - (unsigned long long)t);
      if (qp < (uint64_t)slots) atomicAdd(&count[qp], (unsigned long long)t);
    }
    if (t == nnz - 1) atomicAdd(&count[q], (unsigned long long)nnz);
  }
}

// count_w[b*p + s] = count[s*p + b]
__global__ void k_transpose(const int64_t *__restrict__ count, int32_t p,
                            int64_t *__restrict__ count_w) {
  const int64_t total = (int64_t)p * p;
  for (int64_t x = gid(); x < total; x += (int64_t)gridDim.x * blockDim.x) {
    const int64_t b = x / p, s = x - b * p;
    count_w[x] = count[s * p + b];
  }
}

__global__ void k_gather(const uint64_t *__restrict__ skeys, const int32_t *__restrict__ perm,
                         const int32_t *__restrict__ cols, const float *__restrict__ vals,
                         int64_t nnz, Grid G, int rbits, int64_t q0, int64_t nq,
                         const int64_t *__restrict__ block_ptr,
                         const int64_t *__restrict__ wblock_ptr, bool stratum_major,
                         uint2 *__restrict__ rec, uint8_t *__restrict__ nofold, int32_t *err) {
  const uint64_t rmask = (rbits == 0) ? 0ull : ((1ull << rbits) - 1ull);
  const int lane = threadIdx.x & 63;
  const int64_t stride = (int64_t)gridDim.x * blockDim.x;
  // t0 is the same for the 64 lanes of a wave (lane l takes t0 + l), so the
  // previous rating's column comes from the lane before (one read per wave
  // for lane 0) instead of a second random read of the input
  for (int64_t t0 = gid() - lane; t0 < nnz; t0 += stride) {
    const int64_t t = t0 + lane;
    const bool in = t < nnz;
    const int32_t e = in ? perm[t] : 0;
    const bool e_ok = in && e >= 0 && e < nnz;
    const int32_t j = e_ok ? cols[e] : -1;
    int32_t jprev = __shfl_up(j, 1);
    if (lane == 0 && in && t > 0) {
      const int32_t ep = perm[t - 1];
      jprev = (ep >= 0 && ep < nnz) ? cols[ep] : -1;
    }
    if (!in) continue;
    if (!e_ok) {
      atomicOr(err, kErrLayout);
      continue;
    }
    const uint64_t key = skeys[t];
    const int64_t ql = (int64_t)(key >> rbits);  // slot relative to q0
    if (ql >= nq) {
      atomicOr(err, kErrLayout);
      continue;
    }
    const int64_t q = q0 + ql;
    const uint32_t lrow = (uint32_t)(key & rmask);
    // the folded one-column step needs every rating of the block on one
    // column and no row twice in a row: equal sorted keys are the same block
    // and row (rows ascend inside a block, so equal rows are adjacent), and
    // a column that differs from the previous rating's in the same block
    // means more than one column
    if (t > 0 && (skeys[t - 1] >> rbits) == (key >> rbits) &&
        (skeys[t - 1] == key || jprev != j))
      nofold[q] = 1;
    const int64_t s = q / G.p, b = q - s * G.p;
    const int64_t C = (b + s) % G.p;
    const uint32_t lcol = (uint32_t)(j - G.col_start(C));
    const int64_t beg = block_ptr[ql];
    const int64_t pos = stratum_major ? t : wblock_ptr[b * G.p + s] + (t - beg);
    if (pos >= 0 && pos < nnz && t >= beg && t < block_ptr[ql + 1])
      rec[pos] = make_uint2(lrow | (lcol << kColShift), __float_as_uint(vals[e]));
    else
      atomicOr(err, kErrLayout);
  }
}

__global__ void k_fill_rec(uint2 *rec, int64_t count) {
  for (int64_t t = gid(); t < count; t += (int64_t)gridDim.x * blockDim.x)
    rec[t] = make_uint2(0u, 0u);
}

int bits_for(uint64_t values) {  // bits needed to hold 0..values-1
  int b = 0;
  while (b < 64 && (values - 1) >> b) ++b;
  return b;
}

// ----------------------------------------------------------------- batched load
// Pieces of a bucketing that never holds all ratings on the device: slot
// counts accumulated over batches of the input, and the selection, in input
// order, of the ratings whose slot lies in a range [q0, q1) (a group of whole
// blocks, sorted afterwards by bucket() like a load of its own).

__device__ __forceinline__ int64_t slot_of(const Grid &G, int64_t i, int64_t j) {
  const int64_t R = G.row_block(i);
  int64_t s = (int64_t)G.col_block(j) - R;
  if (s < 0) s += G.p;
  return s * G.p + R;
}

__global__ void k_slot_count_coo(const int32_t *__restrict__ rows,
                                 const int32_t *__restrict__ cols, int64_t cnt, Grid G,
                                 unsigned long long *__restrict__ count) {
  for (int64_t e = gid(); e < cnt; e += (int64_t)gridDim.x * blockDim.x)
    atomicAdd(&count[slot_of(G, rows[e], cols[e])], 1ull);
}

__global__ void k_select_flags(const int32_t *__restrict__ rows, const int32_t *__restrict__ cols,
                               int64_t cnt, Grid G, int64_t q0, int64_t q1,
                               int64_t *__restrict__ flag) {
  for (int64_t e = gid(); e < cnt; e += (int64_t)gridDim.x * blockDim.x) {
    const int64_t q = slot_of(G, rows[e], cols[e]);
    flag[e] = (q >= q0 && q < q1) ? 1 : 0;
  }
}

// pos[0..cnt]: exclusive prefix of the flags, pos[cnt] the batch total.
// Selected rating e goes to position *fill + pos[e] of the group arrays, so
// the group keeps input order; a one-thread kernel then advances *fill by
// the batch total for the next batch (all on one stream, no host wait).
__global__ void k_select_compact(const int32_t *__restrict__ rows,
                                 const int32_t *__restrict__ cols,
                                 const float *__restrict__ vals, int64_t cnt, int64_t e0, Grid G,
                                 int64_t q0, int64_t q1, const int64_t *__restrict__ pos,
                                 const int64_t *__restrict__ fill, int64_t cap,
                                 int32_t *__restrict__ g_rows, int32_t *__restrict__ g_cols,
                                 float *__restrict__ g_vals, int32_t *__restrict__ g_e,
                                 int32_t *err) {
  const int64_t base = *fill;
  for (int64_t e = gid(); e < cnt; e += (int64_t)gridDim.x * blockDim.x) {
    const int64_t q = slot_of(G, rows[e], cols[e]);
    if (q < q0 || q >= q1) continue;
    const int64_t d = base + pos[e];
    if (d < 0 || d >= cap) {
      atomicOr(err, kErrLayout);
      continue;
    }
    g_rows[d] = rows[e];
    g_cols[d] = cols[e];
    g_vals[d] = vals[e];
    g_e[d] = (int32_t)(e0 + e);
  }
}

__global__ void k_advance(int64_t *fill, const int64_t *total) { *fill += *total; }

__global__ void k_map_perm(int32_t *__restrict__ perm, const int32_t *__restrict__ g_e,
                           int64_t cnt, int32_t *err) {
  for (int64_t t = gid(); t < cnt; t += (int64_t)gridDim.x * blockDim.x) {
    const int32_t x = perm[t];
    if (x < 0 || x >= cnt) {
      atomicOr(err, kErrLayout);
      continue;
    }
    perm[t] = g_e[x];
  }
}

}  // namespace

size_t scan_scratch_bytes(int64_t len) {
  return scan_scratch_count(len) * sizeof(int64_t) + 64 * 256;
}

hipError_t bucket_count_batch(const int32_t *rows, const int32_t *cols, int64_t cnt,
                              const Grid &G, int64_t *slot_count, hipStream_t st) {
  if (cnt <= 0) return hipSuccess;
  hipLaunchKernelGGL(k_slot_count_coo, dim3(grid_for(cnt, kThreads)), dim3(kThreads), 0, st,
                     rows, cols, cnt, G, reinterpret_cast<unsigned long long *>(slot_count));
  return hipGetLastError();
}

hipError_t bucket_offsets(const int64_t *slot_count, int64_t slots, int64_t *block_ptr,
                          void *scratch, size_t scratch_bytes, hipStream_t st) {
  Arena ar{static_cast<char *>(scratch), scratch_bytes, 0};
  return scan_exclusive(slot_count, slots, block_ptr, ar, st);
}

hipError_t bucket_select_batch(const int32_t *rows, const int32_t *cols, const float *vals,
                               int64_t cnt, int64_t e0, const Grid &G, int64_t q0, int64_t q1,
                               int64_t *flag, int64_t *pos, void *scratch, size_t scratch_bytes,
                               int64_t *fill, const GroupArrays &g, int32_t *err,
                               hipStream_t st) {
  if (cnt <= 0) return hipSuccess;
  const int grid = grid_for(cnt, kThreads);
  hipLaunchKernelGGL(k_select_flags, dim3(grid), dim3(kThreads), 0, st, rows, cols, cnt, G, q0,
                     q1, flag);
  Arena ar{static_cast<char *>(scratch), scratch_bytes, 0};
  hipError_t e = scan_exclusive(flag, cnt, pos, ar, st);
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(k_select_compact, dim3(grid), dim3(kThreads), 0, st, rows, cols, vals, cnt,
                     e0, G, q0, q1, pos, fill, g.cap, g.rows, g.cols, g.vals, g.e, err);
  hipLaunchKernelGGL(k_advance, dim3(1), dim3(1), 0, st, fill, pos + cnt);
  return hipGetLastError();
}

hipError_t bucket_map_perm(int32_t *perm, const int32_t *g_e, int64_t cnt, int32_t *err,
                           hipStream_t st) {
  if (cnt <= 0) return hipSuccess;
  hipLaunchKernelGGL(k_map_perm, dim3(grid_for(cnt, kThreads)), dim3(kThreads), 0, st, perm, g_e,
                     cnt, err);
  return hipGetLastError();
}

size_t bucket_scratch_bytes(int64_t nnz, int64_t nq) {
  const int64_t tiles = (nnz + kTile - 1) / kTile;
  size_t b = 0;
  b += 2 * (size_t)nnz * sizeof(uint64_t) + 2 * (size_t)nnz * sizeof(int32_t);  // ping-pong
  b += (size_t)kBins * tiles * sizeof(int64_t) * 2;                             // counts, offsets
  b += scan_scratch_count((int64_t)kBins * tiles) * sizeof(int64_t);
  b += 2 * (size_t)(nq + 1) * sizeof(int64_t);                                  // slot counts
  b += scan_scratch_count(nq) * sizeof(int64_t);
  b += 64 * 256;                                                                // alignment
  return b;
}

hipError_t bucket(const int32_t *rows, const int32_t *cols, const float *vals, int64_t nnz,
                  const Grid &G, int64_t rows_max, int64_t q0, int64_t nq, bool stratum_major,
                  void *scratch, size_t scratch_bytes, const BucketOut &out, int32_t *err,
                  hipStream_t st) {
  const int32_t p = G.p;
  const int64_t slots = nq;
  if (!stratum_major && (q0 != 0 || nq != (int64_t)p * p)) return hipErrorInvalidValue;
  const int rbits = bits_for((uint64_t)(rows_max < 1 ? 1 : rows_max));
  const int qbits = bits_for((uint64_t)slots + 1);
  const int total_bits = rbits + qbits;
  const int passes = total_bits <= 0 ? 1 : (total_bits + 7) / 8;
  const int64_t tiles = (nnz + kTile - 1) / kTile;

  Arena ar{static_cast<char *>(scratch), scratch_bytes, 0};
  uint64_t *k0 = ar.take<uint64_t>((size_t)nnz), *k1 = ar.take<uint64_t>((size_t)nnz);
  int32_t *v0 = ar.take<int32_t>((size_t)nnz), *v1 = ar.take<int32_t>((size_t)nnz);
  int64_t *counts = ar.take<int64_t>((size_t)kBins * tiles);
  int64_t *offsets = ar.take<int64_t>((size_t)kBins * tiles + 1);
  int64_t *slot_count = ar.take<int64_t>((size_t)slots + 1);
  int64_t *slot_count_w = ar.take<int64_t>((size_t)slots + 1);
  if (!k0 || !k1 || !v0 || !v1 || !counts || !offsets || !slot_count || !slot_count_w)
    return hipErrorOutOfMemory;

  const int g = grid_for(nnz, kThreads);
  hipLaunchKernelGGL(k_make_keys, dim3(g), dim3(kThreads), 0, st, rows, cols, nnz, G, rbits, q0,
                     nq, k0, v0, err);
  uint64_t *kin = k0, *kout = k1;
  int32_t *vin = v0, *vout = v1;
  for (int pass = 0; pass < passes; ++pass) {
    const int shift = pass * 8;
    hipLaunchKernelGGL(k_radix_hist, dim3((unsigned)tiles), dim3(kThreads), 0, st, kin, nnz,
                       shift, tiles, counts);
    Arena scan_ar = ar;
    hipError_t e = scan_exclusive(counts, (int64_t)kBins * tiles, offsets, scan_ar, st);
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL(k_radix_scatter, dim3((unsigned)tiles), dim3(kThreads), 0, st, kin, vin,
                       kout, vout, nnz, shift, tiles, offsets, err);
    uint64_t *tk = kin; kin = kout; kout = tk;
    int32_t *tv = vin; vin = vout; vout = tv;
  }
  // kin / vin hold the sorted keys and input positions
  hipError_t e = hipMemcpyAsync(out.perm, vin, (size_t)nnz * sizeof(int32_t),
                                hipMemcpyDeviceToDevice, st);
  if (e != hipSuccess) return e;
  e = hipMemsetAsync(slot_count, 0, (size_t)(slots + 1) * sizeof(int64_t), st);
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(k_slot_count, dim3(g), dim3(kThreads), 0, st, kin, nnz, rbits, slots,
                     reinterpret_cast<unsigned long long *>(slot_count), err);
  {
    Arena scan_ar = ar;
    e = scan_exclusive(slot_count, slots, out.block_ptr, scan_ar, st);
    if (e != hipSuccess) return e;
  }
  if (!stratum_major) {
    hipLaunchKernelGGL(k_transpose, dim3(grid_for(slots, kThreads)), dim3(kThreads), 0, st,
                       slot_count, p, slot_count_w);
    Arena scan_ar = ar;
    e = scan_exclusive(slot_count_w, slots, out.wblock_ptr, scan_ar, st);
    if (e != hipSuccess) return e;
  }
  hipLaunchKernelGGL(k_fill_rec, dim3(1), dim3(kThreads), 0, st, out.rec + nnz,
                     (int64_t)kRecPad);
  hipLaunchKernelGGL(k_gather, dim3(g), dim3(kThreads), 0, st, kin, vin, cols, vals, nnz, G,
                     rbits, q0, nq, out.block_ptr, out.wblock_ptr, stratum_major, out.rec,
                     out.nofold, err);
  return hipGetLastError();
}

}  // namespace bgmfk
