// Whole-matrix RMSE over the loaded ratings (Algorithm 1's termination
// test): sqrt((1/nnz) sum (x - u_i.v_j)^2), dot products in fp32, squares
// summed in fp64.  Reads the wave-major records.  With the row-block's U
// rows in LDS (k_rmse_lds) a workgroup covers one row-block; otherwise
// (k_rmse_partial) a workgroup covers one row-block and a group of
// column-blocks, its wave w every fourth of them from w.  A group of lanes
// shares one rating and loads 16-byte slices of u_i and v_j.  Per-wave sums
// are combined in a fixed order by a second kernel, so the result does not
// depend on scheduling.
#include <algorithm>

#include "bgmf_internal.h"

namespace bgmfk {
namespace {

// Column-blocks per workgroup of k_rmse_partial.  Workgroups are numbered
// group-major (all row-blocks of column-blocks 0..63, then 64..127, ...), so
// the workgroups resident at one time read the V rows of about 64
// column-blocks, which stay in the caches, instead of all of V.
constexpr int kRmseColGroup = 64;

template <int CTRL>
__device__ __forceinline__ float dpp_mov(float x) {
  return __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(x), CTRL, 0xF, 0xF, false));
}

// Lanes per rating: from k = 32 up, each lane holds four float4 slices of
// u_i and of v_j (KP/16 lanes per rating), which keeps the cross-lane levels
// and the per-rating index work per wave step low; at k = 16 four lanes
// hold one slice each.  Wave steps whose loads are in flight together: two
// at four slices per lane, eight at one.
template <int KP>
constexpr int rmse_lanes() { return KP >= 32 ? KP / 16 : KP / 4; }
template <int KP>
constexpr int rmse_unroll() { return KP >= 32 ? 2 : 8; }

// KP: padded k; L lanes per rating; each lane covers the float4 slices
// q = g, g + L, ... of the row.
template <int KP>
__global__ void __launch_bounds__(256)
k_rmse_partial(const uint2 *__restrict__ rec, const int64_t *__restrict__ wblock_ptr,
               const float *__restrict__ U, const float *__restrict__ V, Grid G, int32_t k,
               double *__restrict__ partials) {
  const int32_t p = G.p;
  constexpr int L = rmse_lanes<KP>();  // lanes per rating
  constexpr int RPS = 64 / L;                // ratings per wave step
  constexpr int Q = KP / 4;                  // float4 slices per padded row
  constexpr int QL = (Q + L - 1) / L;        // slices per lane
  constexpr int UNR = rmse_unroll<KP>();  // wave steps whose loads are in flight together
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int gl = lane % L, grp = lane / L;
  const int b = blockIdx.x % p;    // row-block
  const int cg = blockIdx.x / p;   // group of column-blocks
  const int c_end = min(p, (cg + 1) * kRmseColGroup);
  const float *Ub = U + G.row_start(b) * k;
  const uint32_t rmax = (uint32_t)(G.row_start(b + 1) - G.row_start(b)) - 1u;
  const int kq = k / 4;
  double acc = 0.0;
  for (int c = cg * kRmseColGroup + wave; c < c_end; c += kWavesPerGroup) {
    const int s = (c - b + p) % p;  // block (b, c) is in stratum s
    const int64_t beg = wblock_ptr[(int64_t)b * p + s];
    const int64_t end = wblock_ptr[(int64_t)b * p + s + 1];
    if (beg == end) continue;
    const int C = (b + s) % p;
    const float *Vb = V + G.col_start(C) * k;
    const uint32_t cmax = (uint32_t)(G.col_start(C + 1) - G.col_start(C)) - 1u;
    // records of the next iteration are loaded one iteration ahead, so the
    // factor-row loads never wait for a record load
    uint2 rn[UNR];
#pragma unroll
    for (int u = 0; u < UNR; ++u) {
      const int64_t t = beg + u * RPS + grp;
      rn[u] = rec[t < end ? t : beg];
    }
    for (int64_t t0 = beg; t0 < end; t0 += RPS * UNR) {
      float4 a[UNR][QL], c[UNR][QL];
      float x[UNR];
      bool ok[UNR];
      uint2 r[UNR];
#pragma unroll
      for (int u = 0; u < UNR; ++u) {
        r[u] = rn[u];
        const int64_t t = t0 + RPS * UNR + u * RPS + grp;
        rn[u] = rec[t < end ? t : beg];
      }
#pragma unroll
      for (int u = 0; u < UNR; ++u) {
        const int64_t t = t0 + u * RPS + grp;
        ok[u] = t < end;
        x[u] = __uint_as_float(r[u].y);
        const uint32_t row = min(r[u].x & kRowMask, rmax);
        const uint32_t col = min((r[u].x >> kColShift) & kColMask, cmax);
        const float4 *up = reinterpret_cast<const float4 *>(Ub + (int64_t)row * k);
        const float4 *vp = reinterpret_cast<const float4 *>(Vb + (int64_t)col * k);
#pragma unroll
        for (int i = 0; i < QL; ++i) {
          // branch-free: slices past k read slice 0 and are zeroed after
          const int q = gl + i * L;
          const bool in = q < kq;
          const int qc = in ? q : 0;
          a[u][i] = up[qc];
          c[u][i] = vp[qc];
          if (!in) a[u][i] = make_float4(0.f, 0.f, 0.f, 0.f);
        }
      }
#pragma unroll
      for (int u = 0; u < UNR; ++u) {
        float part = 0.0f;
#pragma unroll
        for (int i = 0; i < QL; ++i) {
          part = fmaf(a[u][i].x, c[u][i].x, part);
          part = fmaf(a[u][i].y, c[u][i].y, part);
          part = fmaf(a[u][i].z, c[u][i].z, part);
          part = fmaf(a[u][i].w, c[u][i].w, part);
        }
        part += dpp_mov<0xB1>(part);
        if constexpr (L > 2) part += dpp_mov<0x4E>(part);
        if constexpr (L > 4) part += dpp_mov<0x141>(part);
        if constexpr (L > 8) part += dpp_mov<0x140>(part);
        const float d = (ok[u] && gl == 0) ? x[u] - part : 0.0f;
        acc = fma((double)d, (double)d, acc);
      }
    }
  }
  for (int off = 32; off > 0; off >>= 1) acc += __shfl_xor(acc, off);
  if (lane == 0) partials[(int64_t)blockIdx.x * kWavesPerGroup + wave] = acc;
}

// Out-of-core RMSE over the strata [s0, s1) held in one device slot: the
// wave of row-block b and grid row y adds the squared errors of blocks
// (b, s), s = s0 + y, s0 + y + gridDim.y, ..., to partials[y p + b] (each
// partial is owned by one wave per launch, and launches are ordered on the
// stream).
template <int KP>
__global__ void __launch_bounds__(256)
k_rmse_stratum(const uint2 *__restrict__ rec, int64_t rec_origin,
               const int64_t *__restrict__ block_ptr, int32_t s0, int32_t s1,
               const float *__restrict__ U, const float *__restrict__ V, Grid G, int32_t k,
               double *__restrict__ partials) {
  const int32_t p = G.p;
  constexpr int L = rmse_lanes<KP>();
  constexpr int RPS = 64 / L;
  constexpr int Q = KP / 4;
  constexpr int QL = (Q + L - 1) / L;
  constexpr int UNR = rmse_unroll<KP>();
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int gl = lane % L, grp = lane / L;
  const int b = blockIdx.x * kWavesPerGroup + wave;
  if (b >= p) return;
  const float *Ub = U + G.row_start(b) * k;
  const uint32_t rmax = (uint32_t)(G.row_start(b + 1) - G.row_start(b)) - 1u;
  const int kq = k / 4;
  double acc = 0.0;
  for (int32_t s = s0 + (int32_t)blockIdx.y; s < s1; s += (int32_t)gridDim.y) {
  const int64_t beg = block_ptr[(int64_t)s * p + b] - rec_origin;
  const int64_t end = block_ptr[(int64_t)s * p + b + 1] - rec_origin;
  const int C = (b + s) % p;
  const float *Vb = V + G.col_start(C) * k;
  const uint32_t cmax = (uint32_t)(G.col_start(C + 1) - G.col_start(C)) - 1u;
  for (int64_t t0 = beg; t0 < end; t0 += RPS * UNR) {
    float4 a[UNR][QL], c[UNR][QL];
    float x[UNR];
    bool ok[UNR];
#pragma unroll
    for (int u = 0; u < UNR; ++u) {
      const int64_t t = t0 + u * RPS + grp;
      ok[u] = t < end;
      const uint2 r = rec[ok[u] ? t : beg];
      x[u] = __uint_as_float(r.y);
      const uint32_t row = min(r.x & kRowMask, rmax);
      const uint32_t col = min((r.x >> kColShift) & kColMask, cmax);
      const float4 *up = reinterpret_cast<const float4 *>(Ub + (int64_t)row * k);
      const float4 *vp = reinterpret_cast<const float4 *>(Vb + (int64_t)col * k);
#pragma unroll
      for (int i = 0; i < QL; ++i) {
        const int q = gl + i * L;
        const bool in = q < kq;
        const int qc = in ? q : 0;
        a[u][i] = up[qc];
        c[u][i] = vp[qc];
        if (!in) a[u][i] = make_float4(0.f, 0.f, 0.f, 0.f);
      }
    }
#pragma unroll
    for (int u = 0; u < UNR; ++u) {
      float part = 0.0f;
#pragma unroll
      for (int i = 0; i < QL; ++i) {
        part = fmaf(a[u][i].x, c[u][i].x, part);
        part = fmaf(a[u][i].y, c[u][i].y, part);
        part = fmaf(a[u][i].z, c[u][i].z, part);
        part = fmaf(a[u][i].w, c[u][i].w, part);
      }
      part += dpp_mov<0xB1>(part);
      if constexpr (L > 2) part += dpp_mov<0x4E>(part);
      if constexpr (L > 4) part += dpp_mov<0x141>(part);
      if constexpr (L > 8) part += dpp_mov<0x140>(part);
      const float d = (ok[u] && gl == 0) ? x[u] - part : 0.0f;
      acc = fma((double)d, (double)d, acc);
    }
  }
  }
  for (int off = 32; off > 0; off >>= 1) acc += __shfl_xor(acc, off);
  if (lane == 0) partials[(int64_t)blockIdx.y * p + b] += acc;
}

// RMSE over caller-given COO ratings (for example a held-out split): the
// same dot products and fp64 squares, with a lane group per rating taken
// from a fixed grid-stride order, and one partial per wave.  A rating whose
// row or column lies outside the matrix, or whose value is not finite, adds
// nothing and sets a bit of *bad (1: index, 2: value); its factor rows are
// not read.
template <int KP>
__global__ void __launch_bounds__(256)
k_rmse_coo(const int32_t *__restrict__ rows, const int32_t *__restrict__ cols,
           const float *__restrict__ vals, int64_t nnz, const float *__restrict__ U,
           const float *__restrict__ V, int32_t k, int64_t n, int64_t m,
           double *__restrict__ partials, int32_t *bad) {
  constexpr int L = rmse_lanes<KP>();
  constexpr int RPS = 64 / L;
  constexpr int Q = KP / 4;
  constexpr int QL = (Q + L - 1) / L;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int gl = lane % L, grp = lane / L;
  const int64_t gw = (int64_t)blockIdx.x * kWavesPerGroup + wave;
  const int64_t stride = (int64_t)gridDim.x * kWavesPerGroup * RPS;
  const int kq = k / 4;
  double acc = 0.0;
  for (int64_t t = gw * RPS + grp; t - grp < nnz; t += stride) {
    bool ok = t < nnz;
    const int64_t e = ok ? t : 0;
    int64_t i = rows[e], j = cols[e];
    const float x = vals[e];
    const bool in = i >= 0 && i < n && j >= 0 && j < m;
    const bool fin = __builtin_isfinite(x);
    if (ok && gl == 0 && !(in && fin)) atomicOr(bad, (in ? 0 : 1) | (fin ? 0 : 2));
    ok = ok && in && fin;
    if (!in) i = j = 0;
    const float4 *up = reinterpret_cast<const float4 *>(U + i * k);
    const float4 *vp = reinterpret_cast<const float4 *>(V + j * k);
    float part = 0.0f;
#pragma unroll
    for (int i = 0; i < QL; ++i) {
      const int q = gl + i * L;
      if (q < kq) {
        const float4 a = up[q], c = vp[q];
        part = fmaf(a.x, c.x, part);
        part = fmaf(a.y, c.y, part);
        part = fmaf(a.z, c.z, part);
        part = fmaf(a.w, c.w, part);
      }
    }
    part += dpp_mov<0xB1>(part);
    if constexpr (L > 2) part += dpp_mov<0x4E>(part);
    if constexpr (L > 4) part += dpp_mov<0x141>(part);
    if constexpr (L > 8) part += dpp_mov<0x140>(part);
    const float d = (ok && gl == 0) ? x - part : 0.0f;
    acc = fma((double)d, (double)d, acc);
  }
  for (int off = 32; off > 0; off >>= 1) acc += __shfl_xor(acc, off);
  if (lane == 0) partials[gw] = acc;
}

__global__ void k_zero_i32(int32_t *x) { *x = 0; }

__global__ void k_zero(double *x, int64_t count) {
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < count;
       i += (int64_t)gridDim.x * blockDim.x)
    x[i] = 0.0;
}

// Variant with the row-block's U rows staged in LDS: one workgroup of 16
// waves per row-block, u_i read from LDS, v_j from global memory.  The
// row-block's records of all strata are contiguous (wave-major), so each
// wave sums one contiguous sixteenth of them as a single stream; a table of
// block starts and column-blocks in LDS gives the block of each rating (a
// lane group steps its block forward as its ratings cross block starts), so
// no block boundary waits for memory.  Used when the rows and the tables
// fit in LDS.
constexpr int kLdsWaves = 16;

template <int KP>
__global__ void __launch_bounds__(1024)
k_rmse_lds(const uint2 *__restrict__ rec, const int64_t *__restrict__ wblock_ptr,
           const float *__restrict__ U, const float *__restrict__ V, Grid G, int32_t k,
           double *__restrict__ partials) {
  const int32_t p = G.p;
  constexpr int L = rmse_lanes<KP>();
  constexpr int RPS = 64 / L;
  constexpr int Q = KP / 4;
  constexpr int QL = (Q + L - 1) / L;
  constexpr int UNR = rmse_unroll<KP>();
  extern __shared__ float4 us[];
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int gl = lane % L, grp = lane / L;
  const int b = blockIdx.x;
  const int64_t r0 = G.row_start(b);
  const uint32_t rows_b = (uint32_t)(G.row_start(b + 1) - r0);
  const uint32_t rmax = rows_b - 1u;
  const int kq = k / 4;
  // after the rows: the start of block (b, s) relative to the row-block's
  // first record (p + 1 entries), then per stratum its column-block's first
  // column and widest local column
  int32_t *bnd = reinterpret_cast<int32_t *>(us + rows_b * (uint32_t)kq);
  int2 *ctab = reinterpret_cast<int2 *>(bnd + ((p + 2) & ~1));
  const int64_t W0 = wblock_ptr[(int64_t)b * p];
  {  // the row-block's rows are contiguous in U
    const float4 *src = reinterpret_cast<const float4 *>(U + r0 * k);
    const uint32_t total = rows_b * (uint32_t)kq;
    for (uint32_t i = threadIdx.x; i < total; i += blockDim.x) us[i] = src[i];
    for (int s = threadIdx.x; s <= p; s += blockDim.x)
      bnd[s] = (int32_t)(wblock_ptr[(int64_t)b * p + s] - W0);
    for (int s = threadIdx.x; s < p; s += blockDim.x) {
      const int C = (b + s) % p;
      const int64_t c0 = G.col_start(C);
      ctab[s] = make_int2((int32_t)c0, (int32_t)(G.col_start(C + 1) - c0 - 1));
    }
  }
  __syncthreads();
  const int32_t T = bnd[p];
  const int32_t tb = (int32_t)((int64_t)T * wave / kLdsWaves);
  const int32_t te = (int32_t)((int64_t)T * (wave + 1) / kLdsWaves);
  double acc = 0.0;
  if (tb < te) {
    // block of the wave's first rating: the last s with bnd[s] <= tb
    int32_t lo = 0, hi = p - 1;
    while (lo < hi) {
      const int32_t mid = (lo + hi + 1) >> 1;
      if (bnd[mid] <= tb) lo = mid;
      else hi = mid - 1;
    }
    int32_t sg = lo;           // block of the lane group's current rating
    int32_t nb = bnd[sg + 1];  // start of the block after it
    int2 ct = ctab[sg];
    const uint2 *rb = rec + W0;
    // records of the next iteration are loaded one iteration ahead, so the
    // factor-row loads never wait for a record load
    uint2 rn[UNR];
#pragma unroll
    for (int u = 0; u < UNR; ++u) {
      const int32_t t = tb + u * RPS + grp;
      rn[u] = rb[t < te ? t : tb];
    }
    for (int32_t t0 = tb; t0 < te; t0 += RPS * UNR) {
      float4 a[UNR][QL], c[UNR][QL];
      float x[UNR];
      bool ok[UNR];
      uint2 r[UNR];
#pragma unroll
      for (int u = 0; u < UNR; ++u) {
        r[u] = rn[u];
        const int32_t t = t0 + RPS * UNR + u * RPS + grp;
        rn[u] = rb[t < te ? t : tb];
      }
#pragma unroll
      for (int u = 0; u < UNR; ++u) {
        const int32_t t = t0 + u * RPS + grp;
        ok[u] = t < te;
        // step to the block of rating t (past empty blocks); t < T = bnd[p]
        while (ok[u] && t >= nb) {
          ++sg;
          nb = bnd[sg + 1];
          ct = ctab[sg];
        }
        x[u] = __uint_as_float(r[u].y);
        const uint32_t row = min(r[u].x & kRowMask, rmax);
        const uint32_t col = min((r[u].x >> kColShift) & kColMask, (uint32_t)ct.y);
        const float4 *vp = reinterpret_cast<const float4 *>(V + ((int64_t)ct.x + col) * k);
#pragma unroll
        for (int i = 0; i < QL; ++i) {
          // branch-free: slices past k read slice 0 and are zeroed after
          const int q = gl + i * L;
          const bool in = q < kq;
          const int qc = in ? q : 0;
          a[u][i] = us[row * kq + qc];
          c[u][i] = vp[qc];
          if (!in) a[u][i] = make_float4(0.f, 0.f, 0.f, 0.f);
        }
      }
#pragma unroll
      for (int u = 0; u < UNR; ++u) {
        float part = 0.0f;
#pragma unroll
        for (int i = 0; i < QL; ++i) {
          part = fmaf(a[u][i].x, c[u][i].x, part);
          part = fmaf(a[u][i].y, c[u][i].y, part);
          part = fmaf(a[u][i].z, c[u][i].z, part);
          part = fmaf(a[u][i].w, c[u][i].w, part);
        }
        part += dpp_mov<0xB1>(part);
        if constexpr (L > 2) part += dpp_mov<0x4E>(part);
        if constexpr (L > 4) part += dpp_mov<0x141>(part);
        if constexpr (L > 8) part += dpp_mov<0x140>(part);
        const float d = (ok[u] && gl == 0) ? x[u] - part : 0.0f;
        acc = fma((double)d, (double)d, acc);
      }
    }
  }
  for (int off = 32; off > 0; off >>= 1) acc += __shfl_xor(acc, off);
  if (lane == 0) partials[(int64_t)b * kLdsWaves + wave] = acc;
}

// Sum of the partials in a fixed order (the result does not depend on
// scheduling): thread t adds partials t, t + 256, ... into eight sums by
// index (eight loads in flight instead of one), combined pairwise, then a
// tree over the threads.
__global__ void __launch_bounds__(256)
k_rmse_final(const double *__restrict__ partials, int64_t count, int64_t nnz, double *out) {
  __shared__ double sh[256];
  constexpr int A = 8;
  double a[A];
#pragma unroll
  for (int u = 0; u < A; ++u) a[u] = 0.0;
  int64_t i = threadIdx.x;
  for (; i + (A - 1) * 256 < count; i += A * 256) {
#pragma unroll
    for (int u = 0; u < A; ++u) a[u] += partials[i + u * 256];
  }
  for (; i < count; i += 256) a[0] += partials[i];
  sh[threadIdx.x] = ((a[0] + a[1]) + (a[2] + a[3])) + ((a[4] + a[5]) + (a[6] + a[7]));
  __syncthreads();
  for (int off = 128; off > 0; off >>= 1) {
    if ((int)threadIdx.x < off) sh[threadIdx.x] += sh[threadIdx.x + off];
    __syncthreads();
  }
  if (threadIdx.x == 0) out[0] = nnz > 0 ? sqrt(sh[0] / (double)nnz) : 0.0;
}

}  // namespace

size_t rmse_partials_count(int32_t p) {
  const int64_t groups = ((int64_t)p + kRmseColGroup - 1) / kRmseColGroup;
  return (size_t)p * (size_t)std::max<int64_t>(groups * kWavesPerGroup, kLdsWaves);
}

namespace {
template <int KP>
hipError_t launch_rmse_kp(const uint2 *rec, const int64_t *wblock_ptr, const float *U,
                          const float *V, const Grid &G, int64_t rows_max, int32_t k,
                          double *partials, size_t lds_limit, int64_t *count,
                          hipStream_t stream) {
  const int32_t p = G.p;
  const size_t lds = (size_t)rows_max * (size_t)k * sizeof(float) +
                     (size_t)((p + 2) & ~1) * sizeof(int32_t) + (size_t)p * sizeof(int2);
  if (lds <= lds_limit) {
    static bool attr_set = false;
    if (!attr_set) {
      hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void *>(&k_rmse_lds<KP>),
                                         hipFuncAttributeMaxDynamicSharedMemorySize,
                                         (int)lds_limit);
      if (e != hipSuccess) return e;
      attr_set = true;
    }
    hipLaunchKernelGGL(k_rmse_lds<KP>, dim3((unsigned)p), dim3(64 * kLdsWaves), lds, stream, rec,
                       wblock_ptr, U, V, G, k, partials);
    *count = (int64_t)p * kLdsWaves;
  } else {
    const int64_t groups = (int64_t)p * ((p + kRmseColGroup - 1) / kRmseColGroup);
    hipLaunchKernelGGL(k_rmse_partial<KP>, dim3((unsigned)groups), dim3(256), 0, stream,
                       rec, wblock_ptr, U, V, G, k, partials);
    *count = groups * kWavesPerGroup;
  }
  return hipGetLastError();
}
}  // namespace

hipError_t rmse_stratum_begin(double *partials, int32_t p, hipStream_t stream) {
  const int64_t count = (int64_t)kRmseStrataGroups * p;
  hipLaunchKernelGGL(k_zero, dim3((unsigned)((count + 255) / 256)), dim3(256), 0, stream, partials,
                     count);
  return hipGetLastError();
}

hipError_t rmse_stratum_add(const uint2 *rec, int64_t rec_origin, const int64_t *block_ptr,
                            int32_t s0, int32_t s1, const float *U, const float *V,
                            const Grid &G, int32_t k, double *partials, hipStream_t stream) {
  const int32_t p = G.p;
  int kp = 16;
  while (kp < k) kp <<= 1;
  const dim3 grid((unsigned)((p + kWavesPerGroup - 1) / kWavesPerGroup),
                  (unsigned)std::min(kRmseStrataGroups, s1 - s0)),
      block(256);
#define BGMF_RS(KPV)                                                                            \
  hipLaunchKernelGGL(k_rmse_stratum<KPV>, grid, block, 0, stream, rec, rec_origin, block_ptr, s0, \
                     s1, U, V, G, k, partials)
  switch (kp) {
    case 16: BGMF_RS(16); break;
    case 32: BGMF_RS(32); break;
    case 64: BGMF_RS(64); break;
    case 128: BGMF_RS(128); break;
    case 256: BGMF_RS(256); break;
    default: return hipErrorInvalidValue;
  }
#undef BGMF_RS
  return hipGetLastError();
}

hipError_t rmse_stratum_end(const double *partials, int32_t p, int64_t nnz, double *out,
                            hipStream_t stream) {
  hipLaunchKernelGGL(k_rmse_final, dim3(1), dim3(256), 0, stream, partials,
                     (int64_t)kRmseStrataGroups * p, nnz, out);
  return hipGetLastError();
}

size_t rmse_coo_partials_count() { return (size_t)kRmseCooGroups * kWavesPerGroup; }

hipError_t launch_rmse_coo(const int32_t *rows, const int32_t *cols, const float *vals,
                           int64_t nnz, const float *U, const float *V, int32_t k, int64_t n,
                           int64_t m, double *partials, double *out, int32_t *bad,
                           hipStream_t stream) {
  int kp = 16;
  while (kp < k) kp <<= 1;
  const dim3 grid(kRmseCooGroups), block(64 * kWavesPerGroup);
  hipLaunchKernelGGL(k_zero_i32, dim3(1), dim3(1), 0, stream, bad);
#define BGMF_RC(KPV)                                                                           \
  hipLaunchKernelGGL(k_rmse_coo<KPV>, grid, block, 0, stream, rows, cols, vals, nnz, U, V, k, \
                     n, m, partials, bad)
  switch (kp) {
    case 16: BGMF_RC(16); break;
    case 32: BGMF_RC(32); break;
    case 64: BGMF_RC(64); break;
    case 128: BGMF_RC(128); break;
    case 256: BGMF_RC(256); break;
    default: return hipErrorInvalidValue;
  }
#undef BGMF_RC
  hipLaunchKernelGGL(k_rmse_final, dim3(1), dim3(256), 0, stream, partials,
                     (int64_t)rmse_coo_partials_count(), nnz, out);
  return hipGetLastError();
}

hipError_t launch_rmse(const uint2 *rec, const int64_t *wblock_ptr, const float *U,
                       const float *V, const Grid &G, int64_t rows_max, int32_t k, int64_t nnz,
                       double *partials, double *out, size_t lds_limit, hipStream_t stream) {
  int kp = 16;
  while (kp < k) kp <<= 1;
  int64_t count = 0;
  hipError_t e;
  switch (kp) {
    case 16: e = launch_rmse_kp<16>(rec, wblock_ptr, U, V, G, rows_max, k, partials, lds_limit, &count, stream); break;
    case 32: e = launch_rmse_kp<32>(rec, wblock_ptr, U, V, G, rows_max, k, partials, lds_limit, &count, stream); break;
    case 64: e = launch_rmse_kp<64>(rec, wblock_ptr, U, V, G, rows_max, k, partials, lds_limit, &count, stream); break;
    case 128: e = launch_rmse_kp<128>(rec, wblock_ptr, U, V, G, rows_max, k, partials, lds_limit, &count, stream); break;
    case 256: e = launch_rmse_kp<256>(rec, wblock_ptr, U, V, G, rows_max, k, partials, lds_limit, &count, stream); break;
    default: return hipErrorInvalidValue;
  }
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(k_rmse_final, dim3(1), dim3(256), 0, stream, partials, count, nnz, out);
  return hipGetLastError();
}

}  // namespace bgmfk
