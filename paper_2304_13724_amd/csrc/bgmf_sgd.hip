// Blocked SGD sweep (Section 1.1, Algorithm 1, Eq. 2-3) for gfx950.
//
// Mapping: one wavefront owns one row-block b for the whole launch.  For
// stratum s it processes block (b, C = (b + s) mod p): the ratings of the
// block in stored order (ascending row, ties by input position), each one a
// dependent SGD step on u_i and v_j.  Between strata the only dependence of
// wave b is column-block C, which wave (b + 1) mod p finished in stratum
// s - 1 (and, across an epoch boundary, in stratum p - 1 of the previous
// epoch).  So instead of a grid-wide barrier every wave waits only for its
// neighbour's progress word (acquire) and publishes its own (release).
//
// Per wave and block:
//   * the block's column slice of V (ncols x k fp32) is copied into LDS after
//     the acquire, updated there, and written back before the release;
//   * U rows are owned by the wave for the whole launch; they are prefetched
//     from HBM kPrefetch ratings ahead into a register ring and stored after
//     every update (a row that repeats at the next rating is forwarded in
//     registers instead of re-read);
//   * ratings are read 64 at a time with one coalesced 512-byte load and
//     broadcast with v_readlane;
//   * k is spread over the 64 lanes (one dimension per lane, or k/64 per
//     lane for k > 64); the dot product is reduced across lanes with DPP row
//     operations and the gfx950 permlane16/32 swaps, so every lane ends with
//     the same sum and the error e needs no broadcast.
// There is no dense contraction here (each rating is a length-k dot product
// on a serial dependency chain), so no MFMA is used.
#include <type_traits>

#include "bgmf_internal.h"

namespace bgmfk {
namespace {

template <int CTRL>
__device__ __forceinline__ float dpp_mov(float x) {
  return __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(x), CTRL, 0xF, 0xF, false));
}

__device__ __forceinline__ uint32_t rl(uint32_t v, int lane) {
  return (uint32_t)__builtin_amdgcn_readlane((int)v, lane);
}

__device__ __forceinline__ int64_t uniform64(int64_t x) {
  const uint32_t lo = (uint32_t)__builtin_amdgcn_readfirstlane((int)(uint32_t)x);
  const uint32_t hi = (uint32_t)__builtin_amdgcn_readfirstlane((int)(uint32_t)((uint64_t)x >> 32));
  return (int64_t)(((uint64_t)hi << 32) | lo);
}

// Hand-over of a column slice between neighbouring waves.
//
// The slice is written back with device-scope (sc1) stores and staged in
// with device-scope (sc1) loads, both coherent across the XCDs' L2 caches.
// The writer waits for its stores to complete (vmcnt(0), the release fence
// at workgroup scope) before it stores its progress word; the reader waits
// for the progress word (and for that load to return) before it issues the
// loads of the slice, and a workgroup-scope acquire fence keeps the compiler
// from moving them earlier.  An agent-scope release/acquire fence would add
// a write-back / invalidation of the whole L2 of the XCD; it is only needed
// to publish or refresh plain cached accesses, and the hand-over uses none.
constexpr int kCoherent = 16;  // cache-policy bits of a device-scope access (sc1)

// Buffer descriptor word 3 for gfx9 (32-bit data format); accesses whose
// VGPR offset is at or past num_records return 0 / are dropped.
constexpr int kBufWord3 = 0x00020000;
constexpr uint32_t kOff = 0x40000000u;  // outside every buffer, even when added twice

__device__ __forceinline__ float buf_ld(__amdgpu_buffer_rsrc_t r, uint32_t voff) {
  return __uint_as_float(__builtin_amdgcn_raw_buffer_load_b32(r, (int)voff, 0, 0));
}
__device__ __forceinline__ void buf_st(float x, __amdgpu_buffer_rsrc_t r, uint32_t voff) {
  __builtin_amdgcn_raw_buffer_store_b32(__float_as_uint(x), r, (int)voff, 0, 0);
}
// Same with a wave-uniform scalar offset added (used only with in-range values).
__device__ __forceinline__ float buf_ld_s(__amdgpu_buffer_rsrc_t r, uint32_t voff, uint32_t soff) {
  return __uint_as_float(__builtin_amdgcn_raw_buffer_load_b32(r, (int)voff, (int)soff, 0));
}
__device__ __forceinline__ void buf_st_s(float x, __amdgpu_buffer_rsrc_t r, uint32_t voff,
                                         uint32_t soff) {
  __builtin_amdgcn_raw_buffer_store_b32(__float_as_uint(x), r, (int)voff, (int)soff, 0);
}

__device__ __forceinline__ float buf_ld_coherent(__amdgpu_buffer_rsrc_t r, uint32_t voff) {
  return __uint_as_float(__builtin_amdgcn_raw_buffer_load_b32(r, (int)voff, 0, kCoherent));
}
__device__ __forceinline__ void buf_st_coherent(float x, __amdgpu_buffer_rsrc_t r, uint32_t voff) {
  __builtin_amdgcn_raw_buffer_store_b32(__float_as_uint(x), r, (int)voff, 0, kCoherent);
}

// Wait until *flag >= target.  Returns false on timeout.
__device__ __forceinline__ bool wait_progress(const int64_t *flag, int64_t target,
                                              int64_t wait_ticks) {
  if (__hip_atomic_load(flag, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) < target) {
    const uint64_t t0 = __builtin_amdgcn_s_memrealtime();
    while (__hip_atomic_load(flag, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) < target) {
      __builtin_amdgcn_s_sleep(1);
      if ((int64_t)(__builtin_amdgcn_s_memrealtime() - t0) > wait_ticks) return false;
    }
  }
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup");
  return true;
}

// Publish progress: all earlier stores of the wave (the column slice) have
// completed before the progress word is written.
__device__ __forceinline__ void publish_progress(int64_t *flag, int64_t value) {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup");
  __hip_atomic_store(flag, value, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// In-row sum (16 lanes) leaving the row's total in every lane of the row.
__device__ __forceinline__ float row_sum(float x) {
#pragma clang fp contract(off)
  x = x + dpp_mov<0xB1>(x);   // quad_perm [1,0,3,2]
  x = x + dpp_mov<0x4E>(x);   // quad_perm [2,3,0,1]
  x = x + dpp_mov<0x141>(x);  // row_half_mirror
  x = x + dpp_mov<0x140>(x);  // row_mirror
  return x;
}

// Sum over the lanes that hold distinct dimensions, returned as a scalar
// (the value of lane 63).  KPL = lanes holding one copy (16, 32 or 64).
// After the in-row sums, row_bcast:15 adds the last lane of each row to the
// next row and row_bcast:31 adds lane 31 to rows 2 and 3 (lanes without a
// source add 0), so lane 63 ends with rows 0 + 1 + 2 + 3; the other rows
// hold partial sums that are not used.
template <int KPL>
__device__ __forceinline__ float lane_total(float x) {
#pragma clang fp contract(off)
  x = row_sum(x);
  if constexpr (KPL >= 32) x = x + dpp_mov<0x142>(x);  // row_bcast:15
  if constexpr (KPL >= 64) x = x + dpp_mov<0x143>(x);  // row_bcast:31
  return __uint_as_float((uint32_t)__builtin_amdgcn_readlane(__float_as_int(x), 63));
}

__device__ __forceinline__ float &lds_at(char *base, uint32_t byte_off) {
  return *reinterpret_cast<float *>(base + byte_off);
}

// KP: k rounded up to a power of two (>= 16).  Lane l holds dimensions
// dim(l) + 64 v, v < NV, where dim(l) = l for KP >= 64 and l mod KP for
// KP < 64 (then the 64/KP lane groups hold identical copies, compute the
// same values and store them to the same addresses).  MASK: k < KP, so the
// dimensions >= k are padding (kept at zero, never stored).
//
// Error term: every lane adds x/KPL to its partial products, so the lane
// total is e = x - u.v directly (x/KPL is an exact power-of-two scaling).
template <int KP, bool MASK>
__global__ void __launch_bounds__(256) k_sgd_lds(SgdParams P) {
  constexpr int NV = KP <= 64 ? 1 : KP / 64;
  constexpr int KPL = KP < 64 ? KP : 64;
  constexpr int D = kPrefetch;
  constexpr int CH = D;  // ratings per unrolled chunk; ring slot = step in chunk
  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);  // wave-uniform
  const int dim = KP >= 64 ? lane : (lane & (KP - 1));
  int grp = blockIdx.x;
  if (P.xcd_remap) {
    // workgroups are dealt round-robin to the 8 XCDs; give each XCD a
    // contiguous range of row-blocks so that most column-block hand-overs
    // stay inside one L2
    const int G = gridDim.x;
    grp = (blockIdx.x & 7) * (G >> 3) + (blockIdx.x >> 3);
  }
  const int b = grp * (int)(blockDim.x >> 6) + wave;
  if (b >= P.p) return;

  extern __shared__ float lds[];
  const Grid G{P.n, P.m, P.p};
  const int k = P.k;
  const uint32_t rowbytes = (uint32_t)k * 4u;
  const uint32_t colbytes = (uint32_t)KP * 4u;
  bool act[NV];
#pragma unroll
  for (int v = 0; v < NV; ++v) act[v] = !MASK || (dim + 64 * v < k);
  // byte offset of this lane's dimension v inside a row; padding
  // dimensions get an out-of-range offset (loads 0, stores dropped)
  uint32_t doff[NV];
#pragma unroll
  for (int v = 0; v < NV; ++v) doff[v] = act[v] ? (uint32_t)(dim + 64 * v) * 4u : kOff;

  // U rows of row-block b (owned by this wave for the whole launch)
  const int64_t r0 = G.row_start(b);
  const uint32_t rows_b = (uint32_t)(G.row_start(b + 1) - r0);
  const __amdgpu_buffer_rsrc_t Ures =
      __builtin_amdgcn_make_buffer_rsrc(P.U + r0 * k, (short)0, (int)(rows_b * rowbytes), kBufWord3);
  // this wave's LDS column slots: cols_max real ones and one spare
  const uint32_t vbase = ((uint32_t)wave * (P.cols_max + 1) * KP + dim) * 4u;
  const uint32_t spare = (uint32_t)P.cols_max * colbytes;
  char *ldsb = reinterpret_cast<char *>(lds);
  const int64_t *blk_b = P.blk + (int64_t)b * P.stride_b;
  // alpha is kept in a VGPR so that alpha * e (e is a scalar) is one instruction
  float alpha;
  asm("v_mov_b32 %0, %1" : "=v"(alpha) : "s"(P.alpha));
  const float shrink = 1.0f - P.alpha * P.beta;  // u + a(e v - b u) = (1 - a b) u + (a e) v
  const float xscale = 1.0f / (float)KPL;

  for (int s = P.s_begin; s < P.s_end; ++s) {
    const int64_t g = P.g_base + s;
    const int C = (b + s) % P.p;
    const int64_t c0 = G.col_start(C);
    const int ncols = (int)(G.col_start(C + 1) - c0);
    const int64_t *bx = blk_b + (int64_t)s * P.stride_s;
    const int64_t beg = uniform64(bx[0]);
    const int32_t len = (int32_t)(uniform64(bx[1]) - beg);
    const uint2 *rp = P.rec + (beg - P.rec_origin);

    // Decoded window of 64 records starting at chunk position c:
    //   wrow = byte offset of the row in U (row 0 past the block end, so the
    //          value is always a valid scalar offset for a prefetch)
    //   wcol = byte offset of the column slot in LDS (spare past the end)
    //   wx   = x / KPL
    uint32_t wrow = 0u, wcol = spare;
    float wx = 0.0f;
    auto decode = [&](uint2 w, int32_t c) {
      const bool ok = c + lane < len;
      wrow = ok ? (w.x & kRowMask) * rowbytes : 0u;
      wcol = ok ? ((w.x >> kColShift) & kColMask) * colbytes : spare;
      wx = __uint_as_float(w.y) * xscale;
    };

    // ratings of the block and the u rows of its first D ratings: these do
    // not depend on V, so they are requested before the wait
    float ring[D][NV];
    uint32_t ringrow[D];
    uint2 Wn1 = make_uint2(0u, 0u);  // raw records of the next chunk
    if (len > 0) {
      decode(rp[lane], 0);
      Wn1 = rp[CH + lane];
#pragma unroll
      for (int j = 0; j < D; ++j) {
        ringrow[j] = rl(wrow, j);
#pragma unroll
        for (int v = 0; v < NV; ++v) ring[j][v] = buf_ld_s(Ures, doff[v], ringrow[j]);
      }
    }
    if (s > P.s_begin) {
      // column-block C was last updated by row-block b+1 in stratum g-1
      const int nb = (b + 1 == P.p) ? 0 : b + 1;
      if (!wait_progress(P.flags + (int64_t)nb * kFlagStride, g, P.wait_ticks)) {
        __hip_atomic_store(P.err, kErrTimeout, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        return;
      }
    }
    if (len > 0) {
      // stage the column slice of V in LDS, 16 columns per round trip
      const __amdgpu_buffer_rsrc_t Vres = __builtin_amdgcn_make_buffer_rsrc(
          P.V + c0 * k, (short)0, (int)((uint32_t)ncols * rowbytes), kBufWord3);
      for (int cb = 0; cb < ncols; cb += 16) {
        float tmp[16][NV];
#pragma unroll
        for (int i = 0; i < 16; ++i)
#pragma unroll
          for (int v = 0; v < NV; ++v)
            tmp[i][v] = buf_ld_coherent(Vres, doff[v] + (uint32_t)(cb + i) * rowbytes);
#pragma unroll
        for (int i = 0; i < 16; ++i) {
          const uint32_t slot = (uint32_t)min(cb + i, P.cols_max);
#pragma unroll
          for (int v = 0; v < NV; ++v)
            lds_at(ldsb, vbase + slot * colbytes + 256u * v) = tmp[i][v];
        }
      }
      uint32_t waddr = vbase + rl(wcol, 0);  // LDS address of the current column
      float vnext[NV];
#pragma unroll
      for (int v = 0; v < NV; ++v) vnext[v] = lds_at(ldsb, waddr + 256u * v);
      uint32_t prev_row = 0xFFFFFFFFu;
      float uprev[NV];
#pragma unroll
      for (int v = 0; v < NV; ++v) uprev[v] = 0.0f;
      // The ring loads were issued before the wait and the V staging, so
      // they have landed; saying so explicitly (vmcnt(0)) lets the compiler
      // count outstanding loads inside the loop from its steady state alone.
      __builtin_amdgcn_s_waitcnt(0x0F70);

      // One chunk of CH ratings, fully unrolled.  In a full chunk every
      // step is a real rating and U is addressed with the row as a scalar
      // offset; the last, partial chunk of a block sends the U store of each
      // step past the end to an out-of-range vector offset (dropped).
      auto chunk = [&](auto tail_tag, int32_t c) {
        constexpr bool TAIL = decltype(tail_tag)::value;
        // records c .. c+63 are decoded and those of chunk c+CH are in
        // flight; fetch the window two chunks ahead now
        const uint2 Wn2 = rp[c + 2 * CH + lane];
        uint32_t ccur = rl(wcol, 0);
#pragma unroll
        for (int j = 0; j < CH; ++j) {
          const float x64 = __uint_as_float(rl(__float_as_uint(wx), j));
          const uint32_t row = ringrow[j];
          const uint32_t col1 = rl(wcol, j + 1);
          const bool same_row = row == prev_row;
          float u[NV], vv[NV];
#pragma unroll
          for (int v = 0; v < NV; ++v) {
            u[v] = same_row ? uprev[v] : ring[j][v];
            vv[v] = vnext[v];
          }
          // read v of the next rating now; if it is the same column the
          // value computed below is forwarded instead
          const uint32_t raddr = vbase + col1;
          float vl[NV];
#pragma unroll
          for (int v = 0; v < NV; ++v) vl[v] = lds_at(ldsb, raddr + 256u * v);

          float tpart = fmaf(-u[0], vv[0], x64);
#pragma unroll
          for (int v = 1; v < NV; ++v) tpart = fmaf(-u[v], vv[v], tpart);
          const float ae = alpha * lane_total<KPL>(tpart);
          float nu[NV], nv[NV];
#pragma unroll
          for (int v = 0; v < NV; ++v) {
            nu[v] = fmaf(ae, vv[v], shrink * u[v]);
            nv[v] = fmaf(ae, u[v], shrink * vv[v]);
          }
          const uint32_t row_st = (!TAIL || c + j < len) ? row : kOff;
#pragma unroll
          for (int v = 0; v < NV; ++v) {
            lds_at(ldsb, waddr + 256u * v) = nv[v];
            if constexpr (TAIL)
              buf_st(nu[v], Ures, doff[v] + row_st);
            else
              buf_st_s(nu[v], Ures, doff[v], row);
            uprev[v] = nu[v];
            vnext[v] = (col1 == ccur) ? nv[v] : vl[v];
          }
          prev_row = row;
          ccur = col1;
          waddr = raddr;
          // prefetch the u row of rating t + D into the slot just freed
          ringrow[j] = rl(wrow, j + D);
#pragma unroll
          for (int v = 0; v < NV; ++v) ring[j][v] = buf_ld_s(Ures, doff[v], ringrow[j]);
        }
        decode(Wn1, c + CH);
        Wn1 = Wn2;
      };
      const int32_t full = len & ~(CH - 1);
      for (int32_t c = 0; c < full; c += CH) chunk(std::false_type{}, c);
      if (full < len) chunk(std::true_type{}, full);
      // publish the column slice, 16 columns per round
      for (int cb = 0; cb < ncols; cb += 16) {
        float tmp[16][NV];
#pragma unroll
        for (int i = 0; i < 16; ++i) {
          const uint32_t slot = (uint32_t)min(cb + i, P.cols_max);
#pragma unroll
          for (int v = 0; v < NV; ++v) tmp[i][v] = lds_at(ldsb, vbase + slot * colbytes + 256u * v);
        }
#pragma unroll
        for (int i = 0; i < 16; ++i)
#pragma unroll
          for (int v = 0; v < NV; ++v)
            buf_st_coherent(tmp[i][v], Vres, doff[v] + (uint32_t)(cb + i) * rowbytes);
      }
    }
    // a launch of one stratum is ordered by the kernel boundary instead;
    // every lane publishes its own stores (all write the same value)
    if (P.s_end - P.s_begin > 1) publish_progress(P.flags + (int64_t)b * kFlagStride, g + 1);
  }
}

template <int KP>
const void *kernel_for(bool mask) {
  return mask ? reinterpret_cast<const void *>(&k_sgd_lds<KP, true>)
              : reinterpret_cast<const void *>(&k_sgd_lds<KP, false>);
}

const void *sgd_kernel(int kp, bool mask) {
  switch (kp) {
    case 16: return kernel_for<16>(mask);
    case 32: return kernel_for<32>(mask);
    case 64: return kernel_for<64>(mask);
    case 128: return kernel_for<128>(mask);
    case 256: return kernel_for<256>(mask);
    default: return nullptr;
  }
}

}  // namespace

hipError_t sgd_set_lds_limit(int kp, bool mask, size_t lds_bytes) {
  const void *f = sgd_kernel(kp, mask);
  if (!f) return hipErrorInvalidValue;
  return hipFuncSetAttribute(f, hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds_bytes);
}

hipError_t sgd_occupancy(int kp, bool mask, int waves_per_group, size_t lds_bytes,
                         int *groups_per_cu) {
  const void *f = sgd_kernel(kp, mask);
  if (!f) return hipErrorInvalidValue;
  return hipOccupancyMaxActiveBlocksPerMultiprocessor(groups_per_cu, f, 64 * waves_per_group,
                                                      lds_bytes);
}

hipError_t launch_sgd(const SgdParams &P, int kp, int waves_per_group, bool cooperative,
                      size_t lds_bytes, hipStream_t stream) {
  const void *f = sgd_kernel(kp, P.k != kp);
  if (!f) return hipErrorInvalidValue;
  const unsigned groups = (unsigned)((P.p + waves_per_group - 1) / waves_per_group);
  const unsigned threads = 64u * (unsigned)waves_per_group;
  SgdParams args = P;
  if (args.xcd_remap && (groups % 8) != 0) args.xcd_remap = 0;
  void *kargs[] = {&args};
  if (cooperative)
    return hipLaunchCooperativeKernel(f, dim3(groups), dim3(threads), kargs, (unsigned)lds_bytes,
                                      stream);
  return hipLaunchKernel(f, dim3(groups), dim3(threads), kargs, lds_bytes, stream);
}

}  // namespace bgmfk
