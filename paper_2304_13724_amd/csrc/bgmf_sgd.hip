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
//   * V: either the block's column slice (ncols x k fp32) is copied into LDS
//     after the acquire, updated there and written back before the release
//     (k_sgd_lds; when all of a block's ratings are on one column, that
//     column's v instead stays in registers for the whole block, with a
//     shorter dependency chain per rating when no row repeats), or V stays
//     in global memory and each rating's v row is
//     prefetched like the u rows (k_sgd_gv, for slices too wide for LDS);
//   * U rows are owned by the wave for the whole launch; they are prefetched
//     from HBM kPrefetch ratings ahead into a register ring and stored after
//     every update (a row that repeats at the next rating is forwarded in
//     registers instead of re-read);
//   * ratings are read 64 at a time with one coalesced 512-byte load and
//     broadcast with v_readlane;
//   * k is spread over the 64 lanes, each lane holding k/64 consecutive
//     dimensions (one 4-, 8- or 16-byte access per row); the dot product is
//     reduced across lanes with DPP row operations and row broadcasts.
// There is no dense contraction here (each rating is a length-k dot product
// on a serial dependency chain), so no MFMA is used.  (Regrouping a run of
// ratings on one column into Gram matrices of U rows would make one; on
// gfx950 each fp32 MFMA then costs more of the wave's issue time than it
// saves.)
//
// Timing: a lone wave issues in order, one instruction per 4-cycle slot
// (a lane read takes two, and every hazard wait state costs a slot).  Each
// level of the cross-lane reduction must wait two states for the previous
// one, so the LDS sweep places the step's independent instructions (stores,
// lane reads, the ring refill, the next rating's v) in those gaps, and
// scheduling fences keep them there.
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

// Scheduling fence: the compiler keeps the instructions on either side of
// it in program order.
__device__ __forceinline__ void pin() { __builtin_amdgcn_sched_barrier(0); }

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
// VGPR offset is at or past num_records return 0 / are dropped.  The scalar
// offset is not range-checked: it only ever carries in-range values.
constexpr int kBufWord3 = 0x00020000;
constexpr uint32_t kOff = 0x40000000u;  // outside every buffer, even when added twice

// One lane's share of a factor row: NV consecutive floats, one access.
template <int NV, int POL>
__device__ __forceinline__ void ld_row(float (&x)[NV], __amdgpu_buffer_rsrc_t r, uint32_t voff,
                                       uint32_t soff) {
  if constexpr (NV == 1) {
    x[0] = __uint_as_float(__builtin_amdgcn_raw_buffer_load_b32(r, (int)voff, (int)soff, POL));
  } else if constexpr (NV == 2) {
    const auto t = __builtin_amdgcn_raw_buffer_load_b64(r, (int)voff, (int)soff, POL);
    x[0] = __uint_as_float(t[0]);
    x[1] = __uint_as_float(t[1]);
  } else {
    static_assert(NV == 4, "one lane holds 1, 2 or 4 dimensions");
    const auto t = __builtin_amdgcn_raw_buffer_load_b128(r, (int)voff, (int)soff, POL);
#pragma unroll
    for (int v = 0; v < 4; ++v) x[v] = __uint_as_float(t[v]);
  }
}

template <int NV, int POL>
__device__ __forceinline__ void st_row(const float (&x)[NV], __amdgpu_buffer_rsrc_t r,
                                       uint32_t voff, uint32_t soff) {
  if constexpr (NV == 1) {
    __builtin_amdgcn_raw_buffer_store_b32(__float_as_uint(x[0]), r, (int)voff, (int)soff, POL);
  } else if constexpr (NV == 2) {
    __attribute__((ext_vector_type(2))) unsigned t;
    t[0] = __float_as_uint(x[0]);
    t[1] = __float_as_uint(x[1]);
    __builtin_amdgcn_raw_buffer_store_b64(t, r, (int)voff, (int)soff, POL);
  } else {
    __attribute__((ext_vector_type(4))) unsigned t;
#pragma unroll
    for (int v = 0; v < 4; ++v) t[v] = __float_as_uint(x[v]);
    __builtin_amdgcn_raw_buffer_store_b128(t, r, (int)voff, (int)soff, POL);
  }
}

template <int NV>
struct LdsVec;
template <>
struct LdsVec<1> { using T = float; };
template <>
struct LdsVec<2> { using T = float2; };
template <>
struct LdsVec<4> { using T = float4; };

// LDS pointers: an address kept in a register across steps stays an LDS
// address (ds_read / ds_write), which a generic pointer would not.
using lds_char = __attribute__((address_space(3))) char;
template <int NV>
struct LdsRaw { using T = float __attribute__((ext_vector_type(NV))); };
template <>
struct LdsRaw<1> { using T = float; };

// One lane's share of a row in LDS through an LDS pointer.
template <int NV>
__device__ __forceinline__ void lds_ld(float (&x)[NV], const lds_char *p) {
  using T = typename LdsRaw<NV>::T;
  const T t = *reinterpret_cast<const __attribute__((address_space(3))) T *>(p);
  if constexpr (NV == 1) {
    x[0] = t;
  } else {
#pragma unroll
    for (int v = 0; v < NV; ++v) x[v] = t[v];
  }
}

template <int NV>
__device__ __forceinline__ void lds_st(const float (&x)[NV], lds_char *p) {
  using T = typename LdsRaw<NV>::T;
  T t;
  if constexpr (NV == 1) {
    t = x[0];
  } else {
#pragma unroll
    for (int v = 0; v < NV; ++v) t[v] = x[v];
  }
  *reinterpret_cast<__attribute__((address_space(3))) T *>(p) = t;
}

template <int NV>
__device__ __forceinline__ void lds_ld(float (&x)[NV], const char *base, uint32_t off) {
  const auto t = *reinterpret_cast<const typename LdsVec<NV>::T *>(base + off);
  if constexpr (NV == 1) {
    x[0] = t;
  } else {
    const float *f = reinterpret_cast<const float *>(&t);
#pragma unroll
    for (int v = 0; v < NV; ++v) x[v] = f[v];
  }
}

template <int NV>
__device__ __forceinline__ void lds_st(const float (&x)[NV], char *base, uint32_t off) {
  typename LdsVec<NV>::T t;
  if constexpr (NV == 1) {
    t = x[0];
  } else {
    float *f = reinterpret_cast<float *>(&t);
#pragma unroll
    for (int v = 0; v < NV; ++v) f[v] = x[v];
  }
  *reinterpret_cast<typename LdsVec<NV>::T *>(base + off) = t;
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

// Wait until an LDS progress word of this workgroup is >= target.  LDS
// accesses of one wave complete in order and the writer stored the word
// after its slice accesses had completed, so the slice reads that follow
// see the slice.  Returns false on timeout.
__device__ __forceinline__ bool wait_lds_progress(volatile __attribute__((address_space(3))) int64_t *w,
                                                  int64_t target, int64_t wait_ticks) {
  if (*w < target) {
    const uint64_t t0 = __builtin_amdgcn_s_memrealtime();
    while (*w < target) {
      __builtin_amdgcn_s_sleep(1);
      if ((int64_t)(__builtin_amdgcn_s_memrealtime() - t0) > wait_ticks) return false;
    }
  }
  asm volatile("" ::: "memory");
  return true;
}

// Publish progress: all earlier stores of the wave (the column slice) have
// completed before the progress word is written.
__device__ __forceinline__ void publish_progress(int64_t *flag, int64_t value) {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup");
  __hip_atomic_store(flag, value, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// Block trace (off unless the handle asks for it): lane 0 stores the
// device's constant-rate clock with a vector store.  Slot 2q of the trace is
// the time block q = s*p + b starts (after its waits), slot 2q + 1 the time
// it hands its results on (before its progress word moves).
__device__ __forceinline__ void trace_mark(int64_t *trace, int64_t slot, int lane) {
  const int64_t t = (int64_t)__builtin_amdgcn_s_memrealtime();
  if (lane == 0) trace[slot] = t;
}

// Ratings left in a block's last chunk, as a value the compiler cannot see
// through: the per-step exit tests against it then stay inside that chunk
// instead of being computed ahead for every block (and spilled) at its start.
__device__ __forceinline__ int32_t tail_left(int32_t len, int32_t c) {
  int32_t left = len - c;
  asm volatile("" : "+s"(left));
  return left;
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

// Lane layout shared by both sweeps.  KP: k rounded up to a power of two
// (>= 16).  For KP >= 64 lane l holds dimensions [l NV, l NV + NV), NV =
// KP / 64; for KP < 64 lane l holds dimension l mod KP (the 64/KP lane
// groups hold identical copies, compute the same values and store them to
// the same addresses).  MASK: k < KP; a lane whose dimensions are >= k holds
// padding (kept at zero, never stored).  Since k is a multiple of 16, a
// lane's NV dimensions are all real or all padding.
template <int KP, bool MASK>
struct Lanes {
  static constexpr int NV = KP <= 64 ? 1 : KP / 64;
  static constexpr int KPL = KP < 64 ? KP : 64;  // lanes holding one copy
  int lane, first;  // first dimension of the lane
  uint32_t doff;    // byte offset of that dimension in a row, kOff for padding
  __device__ __forceinline__ explicit Lanes(int k) {
    lane = threadIdx.x & 63;
    first = KP >= 64 ? lane * NV : (lane & (KP - 1));
    doff = (!MASK || first < k) ? (uint32_t)first * 4u : kOff;
  }
};

// Row-block of this wave.  Workgroups are dealt round-robin to the 8 XCDs;
// with xcd_remap each XCD holds a contiguous range of row-blocks, so that
// most column-block hand-overs stay inside one L2.
__device__ __forceinline__ int row_block_of_wave(const SgdParams &P, int wave) {
  int grp = blockIdx.x;
  if (P.xcd_remap) {
    const int G = gridDim.x;
    grp = (blockIdx.x & 7) * (G >> 3) + (blockIdx.x >> 3);
  }
  return grp * P.wpg + wave;
}

// Error term: every lane adds x/KPL to its partial products, so the lane
// total is e = x - u.v directly (x/KPL is an exact power-of-two scaling).
template <int KP, bool MASK>
__global__ void __launch_bounds__(256) k_sgd_lds(SgdParams P) {
  using L = Lanes<KP, MASK>;
  constexpr int NV = L::NV;
  constexpr int KPL = L::KPL;
  constexpr int D = kPrefetch;
  constexpr int CH = D;  // ratings per unrolled chunk; ring slot = step in chunk
  static_assert((CH & (CH - 1)) == 0 && CH <= 32,
                "full chunks are counted with a mask; lanes j + D stay in the 64-record window");
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);  // wave-uniform
  const int wpg = P.wpg;
  const int b = row_block_of_wave(P, wave);
  const L ln(P.k);
  const int lane = ln.lane;
  const uint32_t doff = ln.doff;

  extern __shared__ float lds[];
  const Grid G{P.n, P.m, P.p, P.rcut, P.ccut};
  const int k = P.k;
  const uint32_t rowbytes = (uint32_t)k * 4u;
  const uint32_t colbytes = (uint32_t)KP * 4u;
  char *ldsb = reinterpret_cast<char *>(lds);

  // Column slices live in LDS areas of cols_max + 1 slots.  Without the
  // hand-over ring each wave has its own area.  With it (persistent
  // launches), the workgroup's waves, which own consecutive row-blocks,
  // share a ring of R areas: the slice that wave w finishes in stratum s is
  // the one wave w - 1 needs in stratum s + 1, so it stays in its area
  // (index (w + s) mod R, the same along the slice's way through the
  // workgroup) and moves on with an LDS progress word instead of a
  // device-scope write-back, completion wait and reload.  Only the slices
  // entering the workgroup (at its last wave) and leaving it (at wave 0, and
  // every slice after the launch's last stratum) go through global memory.
  const bool lho = P.lds_ring > 0 && P.s_end - P.s_begin > 1;
  const int R = lho ? P.lds_ring : wpg;
  const uint32_t areabytes = (uint32_t)(P.cols_max + 1) * colbytes;
  using lds_i64 = __attribute__((address_space(3))) int64_t;
  volatile lds_i64 *const lprog = (volatile lds_i64 *)((lds_char *)ldsb + (uint32_t)R * areabytes);
  if (lho) {
    // strata completed by each wave, as the global progress words count them
    if (b < P.p && lane == 0) lprog[wave] = P.g_base + P.s_begin;
    __syncthreads();
  }
  if (b >= P.p) return;

  // U rows of row-block b (owned by this wave for the whole launch)
  const int64_t r0 = G.row_start(b);
  const uint32_t rows_b = (uint32_t)(G.row_start(b + 1) - r0);
  const __amdgpu_buffer_rsrc_t Ures =
      __builtin_amdgcn_make_buffer_rsrc(P.U + r0 * k, (short)0, (int)(rows_b * rowbytes), kBufWord3);
  // in an LDS area: cols_max real column slots and one spare
  const uint32_t spare = (uint32_t)P.cols_max * colbytes;
  const int64_t *blk_b = P.blk + (int64_t)b * P.stride_b;
  // alpha is kept in a VGPR so that alpha * e (e is a scalar) is one instruction
  float alpha;
  asm("v_mov_b32 %0, %1" : "=v"(alpha) : "s"(P.alpha));
  // u + a (e v - b u) is evaluated as u + ((a e) v - (a b) u): the small
  // increment first (one fma onto the decay product, which needs only u and
  // so sits off the dependency chain), then a single rounding at the scale
  // of u, as in the plain formula.  Forms that round twice at that scale
  // (u - (a b) u, then + (a e) v, in either order, or a folded factor
  // 1 - a b) drift several times further from the exact result over an
  // epoch; on 250M ratings with k = 128 the difference is 6e-4 against
  // 1.2e-4 of binary64 after one epoch.
  const float nab = -(P.alpha * P.beta);
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
    // every rating of the block on one column, no row twice in a row
    const bool fold = P.single_col &&
                      __builtin_amdgcn_readfirstlane(P.nofold[(int64_t)s * P.p + b]) == 0;
    // this lane's part of the LDS area holding column-block C; whether the
    // slice comes from wave w + 1 of this workgroup (through LDS) and goes
    // on to wave w - 1 (through LDS)
    const int area = lho ? (wave + s) % R : wave;
    const uint32_t vbase = (uint32_t)area * areabytes + ln.first * 4u;
    const bool from_lds = lho && s > P.s_begin && wave + 1 < wpg && b + 1 < P.p;
    const bool to_lds = lho && s + 1 < P.s_end && wave > 0;

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
    auto prime = [&]() {
      decode(rp[lane], 0);
      Wn1 = rp[CH + lane];
#pragma unroll
      for (int j = 0; j < D; ++j) {
        ringrow[j] = rl(wrow, j);
        ld_row<NV, 0>(ring[j], Ures, doff, ringrow[j]);
      }
    };
    if (len > 0) prime();
    const bool stage = !from_lds && (len > 0 || to_lds);
    if (s > P.s_begin) {
      // column-block C was last updated by row-block b+1 in stratum g-1
      bool ok;
      if (from_lds) {
        ok = wait_lds_progress(lprog + wave + 1, g, P.wait_ticks);
      } else {
        const int nb = (b + 1 == P.p) ? 0 : b + 1;
        ok = wait_progress(P.flags + (int64_t)nb * kFlagStride, g, P.wait_ticks);
        // the area's previous slice (position wave + s - R in the ring) must
        // have left the workgroup: wave 0 finished its stratum wave + s - R
        if (ok && lho && stage && wave + s - R >= P.s_begin)
          ok = wait_lds_progress(lprog, g + wave - R + 1, P.wait_ticks);
      }
      if (!ok) {
        __hip_atomic_store(P.err, kErrTimeout, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        return;
      }
    }
    if (P.trace) trace_mark(P.trace, 2 * ((int64_t)s * P.p + b), lane);
    const __amdgpu_buffer_rsrc_t Vres = __builtin_amdgcn_make_buffer_rsrc(
        P.V + c0 * k, (short)0, (int)((uint32_t)ncols * rowbytes), kBufWord3);
    if (stage) {
      // stage the column slice of V in LDS, 16 columns per round trip
      // (columns past the slice read 0 and land in the spare slot)
      for (int cb = 0; cb < ncols; cb += 16) {
        float tmp[16][NV];
#pragma unroll
        for (int i = 0; i < 16; ++i)
          ld_row<NV, kCoherent>(tmp[i], Vres, doff + (uint32_t)(cb + i) * rowbytes, 0);
#pragma unroll
        for (int i = 0; i < 16; ++i)
          lds_st<NV>(tmp[i], ldsb, vbase + (uint32_t)min(cb + i, P.cols_max) * colbytes);
      }
    }
    if (len > 0) {
      // GPU_STEPS passes over the block, its ratings in the same order each
      // time (Section 1.3); a later pass re-reads the U rows this wave
      // stored in the previous one (the hardware keeps a wave's accesses to
      // one address in order)
      for (int pass = 0; pass < P.passes; ++pass) {
      if (pass > 0) prime();
      // operands of the first step: its column, v, x and u
      uint32_t ccur = rl(wcol, 0);  // LDS byte offset of the current column
      lds_char *const vb = (lds_char *)ldsb + vbase;  // this lane's part of the wave's LDS column slots
      lds_char *waddr = vb + ccur;
      float u[NV], vv[NV];
      lds_ld<NV>(vv, waddr);
      uint32_t x64 = rl(__float_as_uint(wx), 0);
      uint32_t ncol = rl(wcol, 1);  // column of the next rating
      lds_char *naddr = vb + ncol;
      // The ring loads were issued before the wait and the V staging, so
      // they have landed; saying so explicitly (vmcnt(0)) lets the compiler
      // count outstanding loads inside the loop from its steady state alone.
      __builtin_amdgcn_s_waitcnt(0x0F70);
#pragma unroll
      for (int v = 0; v < NV; ++v) u[v] = ring[0][v];
      // Results of a step are stored during the next step's reduction; at
      // the start the pending results are rating 0's current u and v,
      // written back unchanged.
      float pnu[NV], pnv[NV];
      uint32_t prow = ringrow[0];
      lds_char *pwaddr = waddr;
#pragma unroll
      for (int v = 0; v < NV; ++v) {
        pnu[v] = u[v];
        pnv[v] = vv[v];
      }

      // One chunk of CH ratings, fully unrolled, U addressed with the row as
      // a scalar offset; the last, partial chunk of a block leaves the loop
      // after the block's last rating (a uniform branch per step), so no
      // step runs on padding.
      //
      // A step is one dependent chain: partial products, six cross-lane
      // levels, the lane read of e, the update, and the choice of the next
      // step's operands.  A lone wave issues in order, so every other
      // instruction of the step (the stores of the previous step's u and
      // v, the next rating's v, the lane reads of later rows, columns and x,
      // the ring refill, the row and column compares, the decay products)
      // is placed between the reduction levels, where the chain leaves
      // issue slots free anyway (each level waits two states for the
      // previous one); the fences keep that order.  The arithmetic is that
      // of the plain order, so the results are the same bits.
      auto chunk = [&](auto tail_tag, int32_t c) {
        constexpr bool TAIL = decltype(tail_tag)::value;
        const int32_t left = TAIL ? tail_left(len, c) : CH;
        // records c .. c+63 are decoded and those of chunk c+CH are in
        // flight; fetch the window two chunks ahead now
        const uint2 Wn2 = rp[c + 2 * CH + lane];
#pragma unroll
        for (int j = 0; j < CH; ++j) {
          const int slot = (j == 0) ? CH - 1 : j - 1;  // ring slot of the previous rating
          const int next = (j + 1) % CH;               // ring slot of the next rating
          float t = fmaf(-u[0], vv[0], __uint_as_float(x64));
#pragma unroll
          for (int v = 1; v < NV; ++v) t = fmaf(-u[v], vv[v], t);
          pin();
          // the previous step's v, then the next rating's v (after that
          // store; if it is this step's column, the new value is forwarded
          // instead)
          float vl[NV];
          lds_st<NV>(pnv, pwaddr);
          lds_ld<NV>(vl, naddr);
          pin();
          t = t + dpp_mov<0xB1>(t);  // quad_perm [1,0,3,2]
          pin();
          // the previous step's u, then the row of the rating D after the
          // previous one, whose ring slot is free again (its value was
          // consumed one step ago); this order is measurably faster than
          // the lane read first
          st_row<NV, 0>(pnu, Ures, doff, prow);
          pin();
          ringrow[slot] = rl(wrow, slot + D - (j == 0 ? CH : 0));
          pin();
          t = t + dpp_mov<0x4E>(t);  // quad_perm [2,3,0,1]
          pin();
          const uint32_t col2 = rl(wcol, j + 2);  // the column after the next one
          float du[NV], dv[NV];
#pragma unroll
          for (int v = 0; v < NV; ++v) du[v] = nab * u[v];
          pin();
          t = t + dpp_mov<0x141>(t);  // row_half_mirror
          pin();
#pragma unroll
          for (int v = 0; v < NV; ++v) dv[v] = nab * vv[v];
          pin();
          ld_row<NV, 0>(ring[slot], Ures, doff, ringrow[slot]);
          pin();
          t = t + dpp_mov<0x140>(t);  // row_mirror
          pin();
          const bool same_row = ringrow[next] == ringrow[j];
          pin();
          if constexpr (KPL >= 32) t = t + dpp_mov<0x142>(t);  // row_bcast:15
          pin();
          const bool same_col = ncol == ccur;
          pin();
          if constexpr (KPL >= 64) t = t + dpp_mov<0x143>(t);  // row_bcast:31
          pin();
          const uint32_t x64n = rl(__float_as_uint(wx), j + 1);  // the next rating's x
          pin();
          const float e = __uint_as_float(rl(__float_as_uint(t), 63));
          pin();
          // LDS address of the column after the next one, computed here;
          // the empty asm keeps the compiler from recomputing it next to
          // its use, where it would take a slot the gaps above need
          lds_char *naddr2 = vb + col2;
          asm volatile("" : "+v"(naddr2));
          pin();
          const float ae = alpha * e;
          float nu[NV], nv[NV];
#pragma unroll
          for (int v = 0; v < NV; ++v) {
            nu[v] = u[v] + fmaf(ae, vv[v], du[v]);
            nv[v] = vv[v] + fmaf(ae, u[v], dv[v]);
          }
          prow = ringrow[j];
          pwaddr = waddr;
#pragma unroll
          for (int v = 0; v < NV; ++v) {
            pnu[v] = nu[v];
            pnv[v] = nv[v];
            u[v] = same_row ? nu[v] : ring[next][v];
            vv[v] = same_col ? nv[v] : vl[v];
          }
          x64 = x64n;
          ccur = ncol;
          waddr = naddr;
          ncol = col2;
          naddr = naddr2;
          pin();
          if constexpr (TAIL) {
            if (j + 1 >= left) break;
          }
        }
        decode(Wn1, c + CH);
        Wn1 = Wn2;
      };

      // Folded step of a block whose ratings all lie on one column and in
      // which no row repeats in consecutive ratings (every block of a heavy
      // item's own column-block, with cut points of unequal blocks, and most
      // blocks of a heavy item's column-block after re-ordering).  The next rating
      // has another row u' and the same column, so its partial products are
      //   x'/KPL - u'.(v + d_v + (a e) u) = [x'/KPL - u'.(v + d_v)] - e [u'.(a u)]
      // with d_v = -(a b) v: both brackets are known before e, and the
      // dependency chain of a rating shrinks to the reduction, the lane read
      // and one fma.  The update of a rating's u and v (exactly the general
      // step's formula) is then off that chain: it is done during the next
      // rating's reduction, in its gaps, together with the store of u and
      // the ring refill.  v stays in registers for the whole block and goes
      // back to its LDS slot at the end; only the rounding of the next dot
      // product differs from the general step.
      //   tcur: partial products of the current rating t
      //   ep, up, vp, dup, dvp, prow: e, u, v, the decay products and the row
      //   of rating t - 1, whose update is still to be applied
      //   uc: u of rating t
      float tcur = 0.0f, ep = 0.0f;
      float up[NV], vp[NV], dup[NV], dvp[NV], uc[NV];
      auto chunk_fold = [&](auto tail_tag, int32_t c) {
        constexpr bool TAIL = decltype(tail_tag)::value;
        const int32_t left = TAIL ? tail_left(len, c) : CH;
        const uint2 Wn2 = rp[c + 2 * CH + lane];
#pragma unroll
        for (int j = 0; j < CH; ++j) {
          const int slot = (j == 0) ? CH - 1 : j - 1;  // ring slot of rating t - 1
          const int next = (j + 1) % CH;               // ring slot of rating t + 1
          // rating t - 1: increments of v and u
          const float ae = alpha * ep;
          float nvx[NV], nux[NV], vc[NV], nu[NV];
#pragma unroll
          for (int v = 0; v < NV; ++v) nvx[v] = fmaf(ae, up[v], dvp[v]);
          pin();
          float t = tcur;
          t = t + dpp_mov<0xB1>(t);  // quad_perm [1,0,3,2]
          pin();
          ringrow[slot] = rl(wrow, slot + D - (j == 0 ? CH : 0));
          // v of rating t (rating t - 1's result)
#pragma unroll
          for (int v = 0; v < NV; ++v) {
            vc[v] = vp[v] + nvx[v];
          }
          pin();
          t = t + dpp_mov<0x4E>(t);  // quad_perm [2,3,0,1]
          pin();
#pragma unroll
          for (int v = 0; v < NV; ++v) nux[v] = fmaf(ae, vp[v], dup[v]);
          const uint32_t x64n = rl(__float_as_uint(wx), j + 1);  // the next rating's x
          pin();
          t = t + dpp_mov<0x141>(t);  // row_half_mirror
          pin();
          float duc[NV], dvc[NV];
#pragma unroll
          for (int v = 0; v < NV; ++v) {
            nu[v] = up[v] + nux[v];
            duc[v] = nab * uc[v];
          }
          pin();
          t = t + dpp_mov<0x140>(t);  // row_mirror
          pin();
          ld_row<NV, 0>(ring[slot], Ures, doff, ringrow[slot]);
#pragma unroll
          for (int v = 0; v < NV; ++v) dvc[v] = nab * vc[v];
          pin();
          if constexpr (KPL >= 32) t = t + dpp_mov<0x142>(t);  // row_bcast:15
          pin();
          // the next rating's partial products before e (A) and the
          // coefficient of -e (B)
          float au[NV];
          float A = __uint_as_float(x64n);
#pragma unroll
          for (int v = 0; v < NV; ++v) {
            au[v] = alpha * uc[v];
            A = fmaf(-ring[next][v], fmaf(nab, vc[v], vc[v]), A);
          }
          pin();
          if constexpr (KPL >= 64) t = t + dpp_mov<0x143>(t);  // row_bcast:31
          pin();
          float B = ring[next][0] * au[0];
#pragma unroll
          for (int v = 1; v < NV; ++v) B = fmaf(ring[next][v], au[v], B);
          pin();
          const float e = __uint_as_float(rl(__float_as_uint(t), 63));
          pin();
          // rating t - 1's u
          st_row<NV, 0>(nu, Ures, doff, prow);
          pin();
          tcur = fmaf(-e, B, A);
          pin();
          ep = e;
#pragma unroll
          for (int v = 0; v < NV; ++v) {
            up[v] = uc[v];
            vp[v] = vc[v];
            dup[v] = duc[v];
            dvp[v] = dvc[v];
            uc[v] = ring[next][v];
          }
          prow = ringrow[j];
          if constexpr (TAIL) {
            if (j + 1 >= left) break;
          }
        }
        decode(Wn1, c + CH);
        Wn1 = Wn2;
      };

      // After the last chunk (a partial one stops right after the block's
      // last rating) that rating's results are still pending.
      const int32_t full = len & ~(CH - 1);
      if (fold) {
        // before rating 0 the pending update is a no-op on the ring's last
        // slot (its current u, stored back unchanged)
        tcur = __uint_as_float(x64);
        ep = 0.0f;
#pragma unroll
        for (int v = 0; v < NV; ++v) {
          tcur = fmaf(-u[v], vv[v], tcur);
          up[v] = ring[D - 1][v];
          vp[v] = vv[v];
          dup[v] = 0.0f;
          dvp[v] = 0.0f;
          uc[v] = u[v];
        }
        prow = ringrow[D - 1];
        for (int32_t c = 0; c < full; c += CH) chunk_fold(std::false_type{}, c);
        if (full < len) chunk_fold(std::true_type{}, full);
        {
          // the block's last rating: its update is still pending
          const float ae = alpha * ep;
#pragma unroll
          for (int v = 0; v < NV; ++v) {
            const float nu = up[v] + fmaf(ae, vp[v], dup[v]);
            vp[v] = vp[v] + fmaf(ae, up[v], dvp[v]);
            up[v] = nu;
          }
          st_row<NV, 0>(up, Ures, doff, prow);
        }
        lds_st<NV>(vp, waddr);
      } else {
        for (int32_t c = 0; c < full; c += CH) chunk(std::false_type{}, c);
        if (full < len) chunk(std::true_type{}, full);
        st_row<NV, 0>(pnu, Ures, doff, prow);
        lds_st<NV>(pnv, pwaddr);
      }
      }
    }
    if (!to_lds && (len > 0 || from_lds)) {
      // write the column slice back, 16 columns per round (stores past the
      // slice are dropped)
      for (int cb = 0; cb < ncols; cb += 16) {
        float tmp[16][NV];
#pragma unroll
        for (int i = 0; i < 16; ++i)
          lds_ld<NV>(tmp[i], ldsb, vbase + (uint32_t)min(cb + i, P.cols_max) * colbytes);
#pragma unroll
        for (int i = 0; i < 16; ++i)
          st_row<NV, kCoherent>(tmp[i], Vres, doff + (uint32_t)(cb + i) * rowbytes, 0);
      }
    }
    if (P.trace) trace_mark(P.trace, 2 * ((int64_t)s * P.p + b) + 1, lane);
    // a launch of one stratum is ordered by the kernel boundary instead;
    // every lane publishes its own stores (all write the same value)
    if (P.s_end - P.s_begin > 1 && !to_lds)
      publish_progress(P.flags + (int64_t)b * kFlagStride, g + 1);
    if (lho) {
      // the slice's LDS writes (or the write-back's LDS reads) are done
      // before the word moves; lane 0 writes it
      asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
      if (lane == 0) lprog[wave] = g + 1;
    }
  }
}

// Variant with V left in global memory, for column slices too wide to stage
// in LDS next to one wave per row-block (or blocks with far fewer ratings
// than columns, where staging the whole slice would dominate).
//
// Each rating's v row is prefetched D ratings ahead into a second register
// ring, like the u rows.  That prefetch misses the updates made to the same
// column by the D - 1 ratings in between.  The decoded window therefore
// starts one chunk early (lane L holds rating c - CH + L), so at every step
// the columns of the previous D - 1 ratings are in the wave: one compare
// across the lanes finds the most recent of them with the next rating's
// column, and its updated row is read back from a per-wave LDS ring that
// keeps the result of each of the last D steps (slot = rating mod D).  The
// previous step's result is forwarded in registers.
//
// COH: V is accessed with device-scope (sc1) loads and stores, for the
// persistent schedule, where a column-block moves between waves (and XCDs)
// inside one launch; a launch of one stratum touches every column from one
// wave only and uses plain cached accesses.
template <int KP, bool MASK, bool COH>
__global__ void __launch_bounds__(256) k_sgd_gv(SgdParams P) {
  using L = Lanes<KP, MASK>;
  constexpr int NV = L::NV;
  constexpr int KPL = L::KPL;
  constexpr int D = kPrefetch;
  constexpr int CH = D;
  static_assert(D == 16, "the window holds the previous chunk, the current one and the next two");
  constexpr int VPOL = COH ? kCoherent : 0;
  constexpr uint32_t kNoCol = 0xFFFFFFFFu;  // column of ratings before the block: matches none
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int b = row_block_of_wave(P, wave);
  if (b >= P.p) return;
  const L ln(P.k);
  const int lane = ln.lane;
  const uint32_t doff = ln.doff;

  extern __shared__ float lds[];
  const Grid G{P.n, P.m, P.p, P.rcut, P.ccut};
  const int k = P.k;
  const uint32_t rowbytes = (uint32_t)k * 4u;
  const uint32_t slotbytes = (uint32_t)KP * 4u;

  const int64_t r0 = G.row_start(b);
  const uint32_t rows_b = (uint32_t)(G.row_start(b + 1) - r0);
  const __amdgpu_buffer_rsrc_t Ures =
      __builtin_amdgcn_make_buffer_rsrc(P.U + r0 * k, (short)0, (int)(rows_b * rowbytes), kBufWord3);
  // this wave's ring of the last D results (D slots of KP floats)
  const uint32_t rbase = ((uint32_t)wave * D * KP + ln.first) * 4u;
  char *ldsb = reinterpret_cast<char *>(lds);
  const int64_t *blk_b = P.blk + (int64_t)b * P.stride_b;
  float alpha;
  asm("v_mov_b32 %0, %1" : "=v"(alpha) : "s"(P.alpha));
  const float nab = -(P.alpha * P.beta);  // update evaluated as in k_sgd_lds
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

    // Decoded window of chunk c: lane L holds rating t = c - CH + L.
    //   wrow = byte offset of the row in U (0 outside the block)
    //   wcol = byte offset of the column in the slice of V (0 past the end,
    //          kNoCol before the start)
    //   wx   = x / KPL
    uint32_t wrow = 0u, wcol = 0u;
    float wx = 0.0f;
    auto decode = [&](uint2 w, int32_t c) {
      const int32_t t = c - CH + lane;
      const bool ok = t >= 0 && t < len;
      wrow = ok ? (w.x & kRowMask) * rowbytes : 0u;
      wcol = ok ? ((w.x >> kColShift) & kColMask) * rowbytes : (t < 0 ? kNoCol : 0u);
      wx = __uint_as_float(w.y) * xscale;
    };

    float ring[D][NV], vring[D][NV];
    uint32_t ringrow[D];
    uint2 Wn1 = make_uint2(0u, 0u);
    auto prime = [&]() {
      decode(rp[lane >= CH ? lane - CH : 0], 0);
      Wn1 = rp[lane];  // window of chunk CH
#pragma unroll
      for (int j = 0; j < D; ++j) {
        ringrow[j] = rl(wrow, CH + j);
        ld_row<NV, 0>(ring[j], Ures, doff, ringrow[j]);
      }
    };
    if (len > 0) prime();
    if (s > P.s_begin) {
      const int nb = (b + 1 == P.p) ? 0 : b + 1;
      if (!wait_progress(P.flags + (int64_t)nb * kFlagStride, g, P.wait_ticks)) {
        __hip_atomic_store(P.err, kErrTimeout, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        return;
      }
    }
    if (P.trace) trace_mark(P.trace, 2 * ((int64_t)s * P.p + b), lane);
    if (len > 0) {
      const __amdgpu_buffer_rsrc_t Vres = __builtin_amdgcn_make_buffer_rsrc(
          P.V + c0 * k, (short)0, (int)((uint32_t)ncols * rowbytes), kBufWord3);
      // GPU_STEPS passes over the block (Section 1.3); each pass re-reads the
      // U and V rows this wave stored in the previous one (the hardware keeps
      // a wave's accesses to one address in order)
      for (int pass = 0; pass < P.passes; ++pass) {
      if (pass > 0) prime();
#pragma unroll
      for (int j = 0; j < D; ++j) ld_row<NV, VPOL>(vring[j], Vres, doff, rl(wcol, CH + j));
      uint32_t prev_row = 0xFFFFFFFFu;
      float uprev[NV], vnext[NV];
      __builtin_amdgcn_s_waitcnt(0x0F70);
#pragma unroll
      for (int v = 0; v < NV; ++v) {
        uprev[v] = 0.0f;
        vnext[v] = vring[0][v];
      }

      auto chunk = [&](auto tail_tag, int32_t c) {
        constexpr bool TAIL = decltype(tail_tag)::value;
        const int32_t left = TAIL ? tail_left(len, c) : CH;
        // window of chunk c + 2 CH (ratings c + CH .. c + CH + 63)
        const uint2 Wn2 = rp[c + CH + lane];
        uint32_t ccur = rl(wcol, CH);
#pragma unroll
        for (int j = 0; j < CH; ++j) {
          const float x64 = __uint_as_float(rl(__float_as_uint(wx), CH + j));
          const uint32_t row = ringrow[j];
          const uint32_t col1 = rl(wcol, CH + j + 1);
          const bool same_row = row == prev_row;
          // latest of ratings t-14 .. t-1 (lanes j+2 .. j+15) with the next
          // rating's column: its result is in LDS slot (lane mod D)
          // (lanes below 32, so the low half of the ballot suffices)
          const uint32_t kMask = ((1u << (D - 2)) - 1u) << (j + 2);  // folded: j is unrolled
          const uint32_t hit = (uint32_t)__builtin_amdgcn_ballot_w64(wcol == col1) & kMask;
          // hit bits are >= 2, so "| 1" leaves the top bit alone and gives
          // slot 0 (a read whose value is not used) when there is no hit
          const uint32_t hslot = (uint32_t)(31 - __builtin_clz(hit | 1u)) & (D - 1);
          float u[NV], vv[NV], vl[NV];
#pragma unroll
          for (int v = 0; v < NV; ++v) {
            u[v] = same_row ? uprev[v] : ring[j][v];
            vv[v] = vnext[v];
          }
          lds_ld<NV>(vl, ldsb, rbase + hslot * slotbytes);
          float tpart = fmaf(-u[0], vv[0], x64);
#pragma unroll
          for (int v = 1; v < NV; ++v) tpart = fmaf(-u[v], vv[v], tpart);
          const float ae = alpha * lane_total<KPL>(tpart);
          float nu[NV], nv[NV];
#pragma unroll
          for (int v = 0; v < NV; ++v) {
            nu[v] = u[v] + fmaf(ae, vv[v], nab * u[v]);
            nv[v] = vv[v] + fmaf(ae, u[v], nab * vv[v]);
          }
          lds_st<NV>(nv, ldsb, rbase + (uint32_t)j * slotbytes);
          st_row<NV, 0>(nu, Ures, doff, row);
          st_row<NV, VPOL>(nv, Vres, doff, ccur);
#pragma unroll
          for (int v = 0; v < NV; ++v) {
            uprev[v] = nu[v];
            vnext[v] = (col1 == ccur) ? nv[v] : (hit ? vl[v] : vring[(j + 1) % D][v]);
          }
          prev_row = row;
          ccur = col1;
          // prefetch u and v of rating t + D (lane j + 2 CH) into slot j
          ringrow[j] = rl(wrow, 2 * CH + j);
          ld_row<NV, 0>(ring[j], Ures, doff, ringrow[j]);
          ld_row<NV, VPOL>(vring[j], Vres, doff, rl(wcol, 2 * CH + j));
          if constexpr (TAIL) {
            if (j + 1 >= left) break;  // the block's last rating is done
          }
        }
        decode(Wn1, c + CH);
        Wn1 = Wn2;
      };
      // One float per lane (k <= 64): the same step with the stores of a
      // rating's results deferred into the next rating's reduction and every
      // independent instruction pinned between the reduction levels, as in
      // the LDS sweep.  A rating's global stores then come after the
      // prefetch issued in its own step (the prefetch of the rating D later),
      // so the lookup reaches one rating further back (ratings t - 15 ..
      // t - 1 of the next one); its LDS ring entry is written, like its
      // stores, at the start of the next step, before that step's lookup.
      // The arithmetic is unchanged: the results are the same bits.  (With
      // two or more floats per lane the extra stores and loads overfill the
      // gaps, and the compiler's order is faster.)
      //   u, vv: operands of the current rating (chosen at the end of the
      //   step before); pnu, pnv, prow, pcol: results of the previous rating
      //   and where they go; x64: x / KPL of the current rating
      float pnu[NV], pnv[NV], u[NV], vv[NV];
      uint32_t prow = ringrow[0], pcol = rl(wcol, CH);
      uint32_t ccur_p = pcol;
      float x64 = __uint_as_float(rl(__float_as_uint(wx), CH));
#pragma unroll
      for (int v = 0; v < NV; ++v) {
        u[v] = ring[0][v];
        vv[v] = vring[0][v];
        pnu[v] = u[v];  // rating 0's current u and v, written back unchanged
        pnv[v] = vv[v];
      }
      auto chunk_pinned = [&](auto tail_tag, int32_t c) {
        constexpr bool TAIL = decltype(tail_tag)::value;
        const int32_t left = TAIL ? tail_left(len, c) : CH;
        const uint2 Wn2 = rp[c + CH + lane];
#pragma unroll
        for (int j = 0; j < CH; ++j) {
          const int next = (j + 1) % D;  // ring slot of the next rating
          const uint32_t row = ringrow[j];
          float vl[NV], du[NV], dv[NV];
          float t = fmaf(-u[0], vv[0], x64);
#pragma unroll
          for (int v = 1; v < NV; ++v) t = fmaf(-u[v], vv[v], t);
          pin();
          st_row<NV, 0>(pnu, Ures, doff, prow);
          pin();
          t = t + dpp_mov<0xB1>(t);  // quad_perm [1,0,3,2]
          pin();
          st_row<NV, VPOL>(pnv, Vres, doff, pcol);
          lds_st<NV>(pnv, ldsb, rbase + (uint32_t)((j + D - 1) % D) * slotbytes);
          pin();
          t = t + dpp_mov<0x4E>(t);  // quad_perm [2,3,0,1]
          pin();
          // the next rating's column and x; the row and column of rating
          // t + D, prefetched below (lane j + 2 CH)
          const uint32_t col1 = rl(wcol, CH + j + 1);
          const float x64n = __uint_as_float(rl(__float_as_uint(wx), CH + j + 1));
          ringrow[j] = rl(wrow, 2 * CH + j);
          const uint32_t pfcol = rl(wcol, 2 * CH + j);
          pin();
          t = t + dpp_mov<0x141>(t);  // row_half_mirror
          pin();
          // latest of ratings t-15 .. t-1 (lanes j+1 .. j+15) with the next
          // rating's column; hit bits are >= 2, so "| 1" gives slot 0 (a
          // read whose value is not used) when there is none
          const uint32_t kMask = ((1u << (D - 1)) - 1u) << (j + 1);
          const uint32_t hit = (uint32_t)__builtin_amdgcn_ballot_w64(wcol == col1) & kMask;
          const uint32_t hslot = (uint32_t)(31 - __builtin_clz(hit | 1u)) & (D - 1);
          pin();
          t = t + dpp_mov<0x140>(t);  // row_mirror
          pin();
          lds_ld<NV>(vl, ldsb, rbase + hslot * slotbytes);
#pragma unroll
          for (int v = 0; v < NV; ++v) {
            du[v] = nab * u[v];
            dv[v] = nab * vv[v];
          }
          pin();
          if constexpr (KPL >= 32) t = t + dpp_mov<0x142>(t);  // row_bcast:15
          pin();
          // prefetch u and v of rating t + D into slot j
          ld_row<NV, 0>(ring[j], Ures, doff, ringrow[j]);
          ld_row<NV, VPOL>(vring[j], Vres, doff, pfcol);
          const bool same_row = ringrow[next] == row;
          const bool same_col = col1 == ccur_p;
          const bool any_hit = hit != 0u;
          pin();
          if constexpr (KPL >= 64) t = t + dpp_mov<0x143>(t);  // row_bcast:31
          pin();
          const float e = __uint_as_float(rl(__float_as_uint(t), 63));
          pin();
          // the next rating's v unless it is this rating's column (in the
          // wait states of the lane read)
          float vc[NV];
#pragma unroll
          for (int v = 0; v < NV; ++v) vc[v] = any_hit ? vl[v] : vring[next][v];
          pin();
          const float ae = alpha * e;
#pragma unroll
          for (int v = 0; v < NV; ++v) {
            const float nu = u[v] + fmaf(ae, vv[v], du[v]);
            const float nv = vv[v] + fmaf(ae, u[v], dv[v]);
            pnu[v] = nu;
            pnv[v] = nv;
            u[v] = same_row ? nu : ring[next][v];
            vv[v] = same_col ? nv : vc[v];
          }
          prow = row;
          pcol = ccur_p;
          ccur_p = col1;
          x64 = x64n;
          pin();
          if constexpr (TAIL) {
            if (j + 1 >= left) break;  // the block's last rating is done
          }
        }
        decode(Wn1, c + CH);
        Wn1 = Wn2;
      };
      const int32_t full = len & ~(CH - 1);
      if constexpr (NV == 1) {
        for (int32_t c = 0; c < full; c += CH) chunk_pinned(std::false_type{}, c);
        if (full < len) chunk_pinned(std::true_type{}, full);
        // the last rating's results
        st_row<NV, 0>(pnu, Ures, doff, prow);
        st_row<NV, VPOL>(pnv, Vres, doff, pcol);
      } else {
        for (int32_t c = 0; c < full; c += CH) chunk(std::false_type{}, c);
        if (full < len) chunk(std::true_type{}, full);
      }
      }
    }
    if (P.trace) trace_mark(P.trace, 2 * ((int64_t)s * P.p + b) + 1, lane);
    if (P.s_end - P.s_begin > 1) publish_progress(P.flags + (int64_t)b * kFlagStride, g + 1);
  }
}

template <int KP>
const void *kernel_for(bool mask, int vmode) {
  if (vmode == kVGlobalCoherent)
    return mask ? reinterpret_cast<const void *>(&k_sgd_gv<KP, true, true>)
                : reinterpret_cast<const void *>(&k_sgd_gv<KP, false, true>);
  if (vmode == kVGlobal)
    return mask ? reinterpret_cast<const void *>(&k_sgd_gv<KP, true, false>)
                : reinterpret_cast<const void *>(&k_sgd_gv<KP, false, false>);
  return mask ? reinterpret_cast<const void *>(&k_sgd_lds<KP, true>)
              : reinterpret_cast<const void *>(&k_sgd_lds<KP, false>);
}

const void *sgd_kernel(int kp, bool mask, int vmode) {
  switch (kp) {
    case 16: return kernel_for<16>(mask, vmode);
    case 32: return kernel_for<32>(mask, vmode);
    case 64: return kernel_for<64>(mask, vmode);
    case 128: return kernel_for<128>(mask, vmode);
    case 256: return kernel_for<256>(mask, vmode);
    default: return nullptr;
  }
}

}  // namespace

size_t sgd_gv_lds_per_wave(int kp) { return (size_t)kPrefetch * kp * sizeof(float); }

size_t sgd_lds_per_wave(int kp, int cols_max) { return (size_t)(cols_max + 1) * kp * sizeof(float); }

size_t sgd_lds_bytes(int kp, int cols_max, int waves_per_group, int ring) {
  const size_t areas = ring > 0 ? (size_t)ring : (size_t)waves_per_group;
  return areas * sgd_lds_per_wave(kp, cols_max) + (size_t)waves_per_group * sizeof(int64_t);
}

hipError_t sgd_set_lds_limit(int kp, bool mask, int vmode, size_t lds_bytes) {
  const void *f = sgd_kernel(kp, mask, vmode);
  if (!f) return hipErrorInvalidValue;
  return hipFuncSetAttribute(f, hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds_bytes);
}

hipError_t sgd_occupancy(int kp, bool mask, int vmode, int waves_per_group, size_t lds_bytes,
                         int *groups_per_cu) {
  const void *f = sgd_kernel(kp, mask, vmode);
  if (!f) return hipErrorInvalidValue;
  return hipOccupancyMaxActiveBlocksPerMultiprocessor(groups_per_cu, f, 64 * waves_per_group,
                                                      lds_bytes);
}

hipError_t launch_sgd(const SgdParams &P, int kp, int vmode, int waves_per_group, bool cooperative,
                      size_t lds_bytes, hipStream_t stream) {
  const void *f = sgd_kernel(kp, P.k != kp, vmode);
  if (!f) return hipErrorInvalidValue;
  const unsigned groups = (unsigned)((P.p + waves_per_group - 1) / waves_per_group);
  const unsigned threads = 64u * (unsigned)waves_per_group;
  SgdParams args = P;
  args.wpg = waves_per_group;
  if (args.xcd_remap && (groups % 8) != 0) args.xcd_remap = 0;
  void *kargs[] = {&args};
  if (cooperative)
    return hipLaunchCooperativeKernel(f, dim3(groups), dim3(threads), kargs, (unsigned)lds_bytes,
                                      stream);
  return hipLaunchKernel(f, dim3(groups), dim3(threads), kargs, lds_bytes, stream);
}

}  // namespace bgmfk
