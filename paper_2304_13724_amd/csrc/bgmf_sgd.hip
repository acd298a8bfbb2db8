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
#include "bgmf_internal.h"

namespace bgmfk {
namespace {

template <int CTRL>
__device__ __forceinline__ float dpp_mov(float x) {
  return __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(x), CTRL, 0xF, 0xF, false));
}

// Sum over the lanes holding dimensions (all 64 for KP >= 64); every lane
// returns the same bits (each step adds two values whose sum is commutative).
template <int KP>
__device__ __forceinline__ float lane_sum(float x) {
#pragma clang fp contract(off)
  x = x + dpp_mov<0xB1>(x);   // quad_perm [1,0,3,2]
  x = x + dpp_mov<0x4E>(x);   // quad_perm [2,3,0,1]
  if constexpr (KP > 4) x = x + dpp_mov<0x141>(x);  // row_half_mirror
  if constexpr (KP > 8) x = x + dpp_mov<0x140>(x);  // row_mirror
  if constexpr (KP > 16) {
    auto r = __builtin_amdgcn_permlane16_swap(__float_as_uint(x), __float_as_uint(x), false,
                                              false);
    x = __uint_as_float(r[0]) + __uint_as_float(r[1]);
  }
  if constexpr (KP > 32) {
    auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false,
                                              false);
    x = __uint_as_float(r[0]) + __uint_as_float(r[1]);
  }
  return x;
}

__device__ __forceinline__ uint32_t rl(uint32_t v, int lane) {
  return (uint32_t)__builtin_amdgcn_readlane((int)v, lane);
}

__device__ __forceinline__ int64_t uniform64(int64_t x) {
  const uint32_t lo = (uint32_t)__builtin_amdgcn_readfirstlane((int)(uint32_t)x);
  const uint32_t hi = (uint32_t)__builtin_amdgcn_readfirstlane((int)(uint32_t)((uint64_t)x >> 32));
  return (int64_t)(((uint64_t)hi << 32) | lo);
}

// Wait until *flag >= target, then acquire.  Returns false on timeout.
__device__ __forceinline__ bool wait_progress(const int64_t *flag, int64_t target,
                                              int64_t wait_ticks) {
  if (__hip_atomic_load(flag, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) < target) {
    const uint64_t t0 = __builtin_amdgcn_s_memrealtime();
    while (__hip_atomic_load(flag, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) < target) {
      __builtin_amdgcn_s_sleep(1);
      if ((int64_t)(__builtin_amdgcn_s_memrealtime() - t0) > wait_ticks) return false;
    }
  }
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "agent");
  return true;
}

// KP: k rounded up to a power of two (>= 16).  Lane l holds dimensions
// dim(l) + 64 v, v < NV, where dim(l) = l for KP >= 64 and l mod KP for
// KP < 64 (then the 64/KP lane groups hold identical copies, compute the
// same values and store them to the same addresses).  MASK: k < KP, so the
// dimensions >= k are padding (kept at zero, never stored).
template <int KP, bool MASK>
__global__ void __launch_bounds__(256) k_sgd_lds(SgdParams P) {
  constexpr int NV = KP <= 64 ? 1 : KP / 64;
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
  // per wave: cols_max + 1 column slots; the last one absorbs padding steps
  float *vblk = lds + (size_t)wave * (P.cols_max + 1) * KP + dim;
  const Grid G{P.n, P.m, P.p};
  const int k = P.k;
  bool act[NV];
#pragma unroll
  for (int v = 0; v < NV; ++v) act[v] = !MASK || (dim + 64 * v < k);
  float *Ub = P.U + G.row_start(b) * k + dim;
  // local rows are < rmax + 1 by construction; the clamps below keep every
  // address inside U even if a record were corrupt
  const uint32_t rmax = (uint32_t)(G.row_start(b + 1) - G.row_start(b)) - 1u;
  float *Udummy = P.U + P.n * (int64_t)k + dim;  // one spare row after U
  const int64_t *wbp = P.wblock_ptr + (int64_t)b * P.p;
  const float alpha = P.alpha, nbeta = -P.beta;
  const uint32_t cmax = (uint32_t)P.cols_max - 1u;
  const uint32_t cdummy = (uint32_t)P.cols_max;

  for (int s = P.s_begin; s < P.s_end; ++s) {
    const int64_t g = P.g_base + s;
    const int C = (b + s) % P.p;
    const int64_t c0 = G.col_start(C);
    const int ncols = (int)(G.col_start(C + 1) - c0);
    const int64_t beg = uniform64(wbp[s]);
    const int32_t len = (int32_t)(uniform64(wbp[s + 1]) - beg);
    const uint2 *rp = P.rec + beg;

    // ratings of the block and the u rows of its first D ratings: these do
    // not depend on V, so they are requested before the wait
    uint2 W = make_uint2(0u, 0u);
    float ring[D][NV];
    if (len > 0) {
      W = rp[lane];
#pragma unroll
      for (int j = 0; j < D; ++j) {
        const uint32_t row = (j < len) ? min(rl(W.x, j) & kRowMask, rmax) : 0u;
#pragma unroll
        for (int v = 0; v < NV; ++v) ring[j][v] = act[v] ? Ub[row * k + 64 * v] : 0.0f;
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
      const float *Vc = P.V + c0 * k + dim;
      for (int c = 0; c < ncols; ++c) {
#pragma unroll
        for (int v = 0; v < NV; ++v)
          vblk[c * KP + 64 * v] = act[v] ? Vc[(int64_t)c * k + 64 * v] : 0.0f;
      }
      uint32_t meta = rl(W.x, 0);
      float vnext[NV];
      {
        const uint32_t cf = min((meta >> kColShift) & kColMask, cmax);
#pragma unroll
        for (int v = 0; v < NV; ++v) vnext[v] = vblk[cf * KP + 64 * v];
      }
      uint32_t prev_row = 0xFFFFFFFFu;
      float uprev[NV];
#pragma unroll
      for (int v = 0; v < NV; ++v) uprev[v] = 0.0f;
      // The ring loads were issued before the wait and the V staging, so
      // they have landed; saying so explicitly (vmcnt(0)) lets the compiler
      // count outstanding loads inside the loop from its steady state alone.
      __builtin_amdgcn_s_waitcnt(0x0F70);

      for (int32_t c = 0; c < len; c += CH) {
        // records c .. c+63 are in W; fetch the next window now
        const uint2 Wn = rp[c + CH + lane];
#pragma unroll
        for (int j = 0; j < CH; ++j) {
          const int32_t t = c + j;
          const bool valid = t < len;  // steps past the end update spare slots
          const float x = __uint_as_float(rl(W.y, j));
          const uint32_t row = min(meta & kRowMask, rmax);
          const uint32_t col = valid ? min((meta >> kColShift) & kColMask, cmax) : cdummy;
          const bool same_row = row == prev_row;
          float u[NV], vv[NV];
#pragma unroll
          for (int v = 0; v < NV; ++v) {
            u[v] = same_row ? uprev[v] : ring[j][v];
            vv[v] = vnext[v];
          }
          // read v of the next rating now; if it is the same column the
          // value computed below is forwarded instead
          const uint32_t meta1 = rl(W.x, j + 1);
          const uint32_t col1 = min((meta1 >> kColShift) & kColMask, cmax);
          float vl[NV];
#pragma unroll
          for (int v = 0; v < NV; ++v) vl[v] = vblk[col1 * KP + 64 * v];

          float pr = u[0] * vv[0];
#pragma unroll
          for (int v = 1; v < NV; ++v) pr = fmaf(u[v], vv[v], pr);
          const float e = x - lane_sum<KP>(pr);
          float nu[NV], nv[NV];
#pragma unroll
          for (int v = 0; v < NV; ++v) {
            nu[v] = fmaf(alpha, fmaf(e, vv[v], nbeta * u[v]), u[v]);
            nv[v] = fmaf(alpha, fmaf(e, u[v], nbeta * vv[v]), vv[v]);
          }
          float *ud = valid ? Ub + row * k : Udummy;
#pragma unroll
          for (int v = 0; v < NV; ++v) {
            vblk[col * KP + 64 * v] = nv[v];
            if (act[v]) ud[64 * v] = nu[v];
            uprev[v] = nu[v];
            vnext[v] = (col1 == col) ? nv[v] : vl[v];
          }
          prev_row = row;
          meta = meta1;
          // prefetch the u row of rating t + D into the slot just freed
          const uint32_t rowD = min(rl(W.x, j + D) & kRowMask, rmax) & (t + D < len ? kRowMask : 0u);
#pragma unroll
          for (int v = 0; v < NV; ++v) ring[j][v] = act[v] ? Ub[rowD * k + 64 * v] : 0.0f;
        }
        W = Wn;
      }
      // publish the column slice
      float *Vw = P.V + c0 * k + dim;
      for (int c = 0; c < ncols; ++c) {
#pragma unroll
        for (int v = 0; v < NV; ++v)
          if (act[v]) Vw[(int64_t)c * k + 64 * v] = vblk[c * KP + 64 * v];
      }
    }
    // every lane releases its own stores (all write the same value)
    __hip_atomic_store(P.flags + (int64_t)b * kFlagStride, g + 1, __ATOMIC_RELEASE,
                       __HIP_MEMORY_SCOPE_AGENT);
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
