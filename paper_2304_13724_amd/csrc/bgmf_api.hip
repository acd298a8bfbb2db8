// Host side of the C ABI declared in include/bgmf.h: handle state, argument
// validation, device memory, and the order of kernel launches on the
// handle's stream.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <cstring>
#include <new>
#include <string>
#include <vector>

#include <rocprofiler-sdk-roctx/roctx.h>

#include "../../include/bgmf.h"
#include "bgmf_handle.h"

using namespace bgmfk;

namespace {

// A named range around each call that does device work, for profilers that
// record ROCTx markers (rocprofv3 --marker-trace); no cost when none listens.
struct Range {
  explicit Range(const char *name) { roctxRangePushA(name); }
  ~Range() { roctxRangePop(); }
  Range(const Range &) = delete;
  Range &operator=(const Range &) = delete;
};

}  // namespace

namespace {

thread_local std::string g_create_error;

// Every device and pinned allocation of the library goes through these two,
// which count them (BGMF_OPT_ALLOC_COUNT): a bound handle makes none in
// bgmf_load_coo, bgmf_epoch or bgmf_rmse.
hipError_t dev_alloc(bgmf_t *h, void **ptr, size_t bytes) {
  ++h->alloc_calls;
  return hipMalloc(ptr, bytes);
}

hipError_t pinned_alloc(bgmf_t *h, void **ptr, size_t bytes) {
  ++h->alloc_calls;
  return hipHostMalloc(ptr, bytes, hipHostMallocDefault);
}

constexpr size_t kAlign = 256;
constexpr size_t aligned(size_t bytes) { return (bytes + kAlign - 1) & ~(kAlign - 1); }

// Bump allocation inside one range of memory (a bound workspace or arena, or
// one block the library allocated); every piece starts on a 256-byte
// boundary, so a sequence of pieces fits in the sum of their aligned sizes.
struct Carve {
  char *base = nullptr;
  size_t size = 0, used = 0, high = 0;
  template <class T>
  T *take(size_t count) {
    const size_t off = aligned(used);
    const size_t bytes = count * sizeof(T);
    if (!base || off + bytes > size) return nullptr;
    used = off + bytes;
    high = std::max(high, used);
    return reinterpret_cast<T *>(base + off);
  }
};

// Sizes of a load (bytes).  Tables: block_ptr and, in-core, wblock_ptr
// (p^2 + 1 int64 each) and the per-block row-repeat flags (p^2 bytes).
size_t tables_bytes(int32_t p, bool wave_major) {
  const size_t slots = (size_t)p * p;
  return aligned((slots + 1) * 8) * (wave_major ? 2 : 1) + aligned(slots);
}

// In-core ratings: records and perm (kept), and the one-pass bucketing's
// temporaries (the COO arrays on the device and the radix sort's scratch).
size_t incore_keep_bytes(int64_t nnz) {
  return aligned(((size_t)nnz + kRecPad) * 8) + aligned((size_t)nnz * 4);
}
size_t incore_temp_bytes(int64_t nnz, int32_t p) {
  return 3 * aligned((size_t)nnz * 4) + aligned(bucket_scratch_bytes(nnz, (int64_t)p * p));
}

// Streamed load: the slot-count pass over batches of `batch` ratings ...
size_t count_pass_bytes(int64_t batch, int32_t p) {
  const int64_t slots = (int64_t)p * p;
  return 2 * aligned((size_t)batch * 4) + aligned(((size_t)slots + 1) * 8) +
         aligned(scan_scratch_bytes(slots));
}
// ... and the gathering and sorting of one group of at most `cap` ratings
// in at most `span` consecutive slots.
size_t group_pass_bytes(int64_t batch, int64_t cap, int64_t span) {
  return 3 * aligned((size_t)batch * 4) + 2 * aligned(((size_t)batch + 1) * 8) +
         aligned(scan_scratch_bytes(batch)) + 4 * aligned((size_t)cap * 4) + aligned(8) +
         aligned(bucket_scratch_bytes(cap, span)) + aligned(((size_t)cap + kRecPad) * 8) +
         aligned((size_t)cap * 4) + aligned(((size_t)span + 1) * 8);
}
size_t pinned_need_bytes(int64_t nnz) {
  return aligned((size_t)nnz * 8) + aligned((size_t)nnz * 4);
}

// Zeroes the block trace with a kernel rather than a memset, so that an
// epoch stays a sequence of kernel launches.
__global__ void k_clear_i64(int64_t *x, int64_t count) {
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < count;
       i += (int64_t)gridDim.x * blockDim.x)
    x[i] = 0;
}

hipError_t clear_trace(int64_t *trace, int64_t count, hipStream_t stream) {
  const int64_t blocks = std::max<int64_t>(1, std::min<int64_t>((count + 255) / 256, 4096));
  hipLaunchKernelGGL(k_clear_i64, dim3((unsigned)blocks), dim3(256), 0, stream, trace, count);
  return hipGetLastError();
}

int fail(bgmf_t *h, int code, const char *fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof buf, fmt, ap);
  va_end(ap);
  if (h) h->msg = buf;
  else g_create_error = buf;
  return code;
}

#define HIP_TRY(h, call)                                                                   \
  do {                                                                                     \
    hipError_t e_ = (call);                                                                \
    if (e_ != hipSuccess)                                                                  \
      return fail((h), e_ == hipErrorOutOfMemory ? BGMF_E_NOMEM : BGMF_E_HIP, "%s: %s",    \
                  #call, hipGetErrorString(e_));                                           \
  } while (0)

void free_layout(bgmf_t *h) {
  if (h->side) hipStreamSynchronize(h->side);
  if (h->own_persist) hipFree(h->own_persist);
  if (h->own_region) hipFree(h->own_region);
  if (h->own_host) hipHostFree(h->own_host);
  h->own_persist = nullptr;
  h->own_region = nullptr;
  h->own_host = nullptr;
  for (auto ev : h->ready) hipEventDestroy(ev);
  for (auto ev : h->freed) hipEventDestroy(ev);
  h->ready.clear();
  h->freed.clear();
  h->slot_used.clear();
  h->chunk.clear();
  h->block_ptr = h->wblock_ptr = nullptr;
  h->nofold = nullptr;
  h->perm = nullptr;
  h->rec = h->ring = h->host_rec = h->resident = nullptr;
  h->s_res = 0;
  h->host_perm = nullptr;
  h->nslots = 0;
  h->ooc = false;
  h->nnz = 0;
  h->loaded = false;
}

// Device-side error word: read, report, clear.  After a failed wait the
// progress words no longer describe a completed epoch; they are reset so
// that later epochs start cleanly (the factors hold a partial epoch).
int check_device_error(bgmf_t *h) {
  int32_t e = 0;
  HIP_TRY(h, hipMemcpyAsync(&e, h->err, sizeof e, hipMemcpyDeviceToHost, h->stream));
  HIP_TRY(h, hipStreamSynchronize(h->stream));
  if (e == 0) return BGMF_OK;
  std::vector<int64_t> fl((size_t)h->p * kFlagStride, h->epochs_done * (int64_t)h->p);
  HIP_TRY(h, hipMemcpyAsync(h->flags, fl.data(), fl.size() * sizeof(int64_t),
                            hipMemcpyHostToDevice, h->stream));
  HIP_TRY(h, hipMemsetAsync(h->err, 0, sizeof(int32_t), h->stream));
  HIP_TRY(h, hipStreamSynchronize(h->stream));
  return fail(h, BGMF_E_TIMEOUT,
              "a device-side wait between strata exceeded its limit (%lld us); the last epoch "
              "is incomplete",
              (long long)h->wait_us);
}

int sync_checked(bgmf_t *h) {
  HIP_TRY(h, hipStreamSynchronize(h->stream));
  return check_device_error(h);
}

Grid grid_of(const bgmf_t *h) {
  return Grid{h->n, h->m, h->p, h->d_cuts, h->d_cuts + h->p + 1};
}

// Launch shapes of the sweep for the current widest column-block: the widest
// workgroup (4, 2 or 1 waves) whose LDS column slices fit, whether all p
// waves can be resident at once (persistent schedule) for the LDS and the
// global-memory placements.  The kernels' dynamic-LDS limit is set to the
// device's, the most any handle may ask for.
hipError_t configure_sweep(bgmf_t *h) {
  const bool mask = h->k != h->kp;
  const int64_t p = h->p;
  int per_cu = 0;
  hipError_t e;
  for (int vm : {kVLds, kVGlobal, kVGlobalCoherent})
    if ((e = sgd_set_lds_limit(h->kp, mask, vm, h->lds_limit)) != hipSuccess) return e;
  h->wpg_lds = kWavesPerGroup;
  while (h->wpg_lds > 1 && sgd_lds_bytes(h->kp, h->cols_max, h->wpg_lds, 0) > h->lds_limit)
    h->wpg_lds >>= 1;
  h->lds_ring = 0;
  h->lds_bytes_lds = sgd_lds_bytes(h->kp, h->cols_max, h->wpg_lds, 0);
  h->lds_fits = h->lds_bytes_lds <= h->lds_limit;
  h->coop_lds = false;
  const int64_t groups = (p + h->wpg_lds - 1) / h->wpg_lds;
  if (h->lds_fits) {
    if ((e = sgd_occupancy(h->kp, mask, kVLds, h->wpg_lds, h->lds_bytes_lds, &per_cu)) !=
        hipSuccess)
      return e;
    h->coop_lds = (int64_t)per_cu * h->cus >= groups;
    // hand-over ring of twice the workgroup's waves, if every wave can
    // still be resident with it
    const int ring = 2 * h->wpg_lds;
    const size_t rb = sgd_lds_bytes(h->kp, h->cols_max, h->wpg_lds, ring);
    if (h->coop_lds && h->lds_handover && h->wpg_lds > 1 && rb <= h->lds_limit) {
      if ((e = sgd_occupancy(h->kp, mask, kVLds, h->wpg_lds, rb, &per_cu)) != hipSuccess) return e;
      if ((int64_t)per_cu * h->cus >= groups) {
        h->lds_ring = ring;
        h->lds_bytes_lds = rb;
      }
    }
  }
  h->wpg_gv = kWavesPerGroup;
  h->lds_bytes_gv = h->wpg_gv * sgd_gv_lds_per_wave(h->kp);
  if ((e = sgd_occupancy(h->kp, mask, kVGlobalCoherent, h->wpg_gv, h->lds_bytes_gv, &per_cu)) !=
      hipSuccess)
    return e;
  h->coop_gv = (int64_t)per_cu * h->cus >= (p + h->wpg_gv - 1) / h->wpg_gv;
  if (h->v_staging == 1 && !h->lds_fits) h->v_staging = 0;
  return hipSuccess;
}

// Host check of cut points: p + 1 strictly increasing values from 0 to len,
// each block at most max_width wide.  Returns the widest block, or -1.
int64_t check_cuts(const int64_t *cut, int32_t p, int64_t len, int64_t max_width) {
  if (cut[0] != 0 || cut[p] != len) return -1;
  int64_t widest = 0;
  for (int32_t b = 0; b < p; ++b) {
    const int64_t w = cut[b + 1] - cut[b];
    if (w < 1 || w > max_width) return -1;
    widest = std::max(widest, w);
  }
  return widest;
}

// Serial-chain statistics from the stratum-major block offsets.
void set_chain_stats(bgmf_t *h, const std::vector<int64_t> &bp) {
  const int64_t p = h->p;
  std::vector<int64_t> colsum(p, 0), rowsum(p, 0);
  int64_t barrier = 0, nonempty = 0;
  for (int64_t s = 0; s < p; ++s) {
    int64_t mx = 0;
    for (int64_t R = 0; R < p; ++R) {
      const int64_t c = bp[s * p + R + 1] - bp[s * p + R];
      colsum[(R + s) % p] += c;
      rowsum[R] += c;
      mx = std::max(mx, c);
      nonempty += c > 0;
    }
    barrier += mx;
  }
  h->chain[0] = *std::max_element(colsum.begin(), colsum.end());
  h->chain[1] = *std::max_element(rowsum.begin(), rowsum.end());
  h->chain[2] = barrier;
  h->chain[3] = nonempty;
}

bool offsets_ok(const std::vector<int64_t> &bp, int64_t nnz) {
  if (bp.front() != 0 || bp.back() != nnz) return false;
  for (size_t q = 0; q + 1 < bp.size(); ++q)
    if (bp[q] > bp[q + 1]) return false;
  return true;
}

int layout_error(bgmf_t *h) {
  hipMemset(h->err, 0, sizeof(int32_t));
  free_layout(h);
  return fail(h, BGMF_E_HIP, "internal error: the device bucketing produced an inconsistent layout");
}

// All ratings on the device: one bucketing pass over the whole input, records
// in wave-major order.  Tables, records and perm are kept; the COO arrays and
// the sort's scratch are temporaries (after the kept part of a bound
// workspace, or one allocation freed before returning).
int load_incore(bgmf_t *h, const int32_t *rows, const int32_t *cols, const float *vals,
                int64_t nnz) {
  const int64_t slots = (int64_t)h->p * h->p;
  const size_t keep = tables_bytes(h->p, true) + incore_keep_bytes(nnz);
  const size_t temp = incore_temp_bytes(nnz, h->p);
  const size_t scratch_bytes = bucket_scratch_bytes(nnz, slots);
  void *own_temp = nullptr;
  Carve kc, tc;
  if (h->bound) {
    kc = Carve{h->ws, h->ws_bytes};
  } else {
    HIP_TRY(h, dev_alloc(h, &h->own_persist, keep));
    kc = Carve{static_cast<char *>(h->own_persist), keep};
    const hipError_t e = dev_alloc(h, &own_temp, temp);
    if (e != hipSuccess) {
      free_layout(h);
      return fail(h, e == hipErrorOutOfMemory ? BGMF_E_NOMEM : BGMF_E_HIP,
                  "hipMalloc(%zu bytes of bucketing temporaries): %s", temp, hipGetErrorString(e));
    }
    tc = Carve{static_cast<char *>(own_temp), temp};
  }
  h->block_ptr = kc.take<int64_t>(slots + 1);
  h->wblock_ptr = kc.take<int64_t>(slots + 1);
  h->nofold = kc.take<uint8_t>(slots);
  h->rec = kc.take<uint2>(nnz + kRecPad);
  h->perm = kc.take<int32_t>(nnz);
  if (h->bound) tc = Carve{h->ws, h->ws_bytes, kc.used, kc.used};
  int32_t *d_rows = tc.take<int32_t>(nnz), *d_cols = tc.take<int32_t>(nnz);
  float *d_vals = tc.take<float>(nnz);
  void *scratch = tc.take<char>(scratch_bytes);
  auto done = [&](int rc) {
    if (own_temp) hipFree(own_temp);
    own_temp = nullptr;
    if (rc != BGMF_OK) free_layout(h);
    return rc;
  };
  if (!h->block_ptr || !h->wblock_ptr || !h->nofold || !h->rec || !h->perm || !d_rows ||
      !d_cols || !d_vals || !scratch)
    return done(fail(h, BGMF_E_HIP, "internal error: in-core load does not fit its plan"));
  h->load_peak = (int64_t)(incore_keep_bytes(nnz) + temp);
  h->load_groups = 0;
#define LOAD_TRY(call)                                                                     \
  do {                                                                                     \
    hipError_t e_ = (call);                                                                \
    if (e_ != hipSuccess)                                                                  \
      return done(fail(h, e_ == hipErrorOutOfMemory ? BGMF_E_NOMEM : BGMF_E_HIP, "%s: %s", \
                       #call, hipGetErrorString(e_)));                                     \
  } while (0)
  LOAD_TRY(hipMemcpyAsync(d_rows, rows, (size_t)nnz * sizeof(int32_t), hipMemcpyHostToDevice,
                          h->stream));
  LOAD_TRY(hipMemcpyAsync(d_cols, cols, (size_t)nnz * sizeof(int32_t), hipMemcpyHostToDevice,
                          h->stream));
  LOAD_TRY(hipMemcpyAsync(d_vals, vals, (size_t)nnz * sizeof(float), hipMemcpyHostToDevice,
                          h->stream));
  LOAD_TRY(hipMemsetAsync(h->err, 0, sizeof(int32_t), h->stream));
  LOAD_TRY(hipMemsetAsync(h->nofold, 0, (size_t)slots, h->stream));
  BucketOut out{h->block_ptr, h->wblock_ptr, h->perm, h->rec, h->nofold};
  LOAD_TRY(bucket(d_rows, d_cols, d_vals, nnz, grid_of(h), h->rows_max, 0, slots, false,
                  scratch, scratch_bytes, out, h->err, h->stream));
  LOAD_TRY(hipStreamSynchronize(h->stream));
  done(BGMF_OK);
  int32_t derr = 0;
  std::vector<int64_t> bp((size_t)slots + 1), wbp((size_t)slots + 1);
  LOAD_TRY(hipMemcpy(&derr, h->err, sizeof derr, hipMemcpyDeviceToHost));
  LOAD_TRY(hipMemcpy(bp.data(), h->block_ptr, bp.size() * sizeof(int64_t), hipMemcpyDeviceToHost));
  LOAD_TRY(hipMemcpy(wbp.data(), h->wblock_ptr, wbp.size() * sizeof(int64_t),
                     hipMemcpyDeviceToHost));
#undef LOAD_TRY
  // the sweep trusts these offsets: check them before any epoch may run
  bool ok = derr == 0 && offsets_ok(bp, nnz) && offsets_ok(wbp, nnz);
  for (int64_t b = 0; ok && b < h->p; ++b)
    for (int64_t s2 = 0; ok && s2 < h->p; ++s2)
      ok = wbp[b * h->p + s2 + 1] - wbp[b * h->p + s2] == bp[s2 * h->p + b + 1] - bp[s2 * h->p + b];
  if (!ok) return layout_error(h);
  set_chain_stats(h, bp);
  return BGMF_OK;
}

// Ratings streamed from pinned host memory.  A pass over batches of the
// input counts the ratings of every slot (block_ptr); the slots are then cut
// into groups of whole blocks, and for each group a pass over the input
// gathers its ratings in input order, sorts them on the device as a load of
// its own and copies records and perm to their stratum-major place in
// pinned memory.  (The input crosses the host link once per group, so a
// small budget makes a slow load; the epochs do not depend on it.)  After
// the load the same device region holds the ring of stream slots and the
// resident strata, within `budget` bytes.  The bucketing's temporaries stay
// within the bound workspace (after the tables), or, for a handle that
// allocates its own memory, within max(budget, the bytes needed to bucket
// the largest block).
int load_streamed(bgmf_t *h, const int32_t *rows, const int32_t *cols, const float *vals,
                  int64_t nnz, int64_t budget) {
  const int32_t p = h->p;
  const int64_t slots = (int64_t)p * p;
  const size_t tab = tables_bytes(p, false);
  const size_t hneed = pinned_need_bytes(nnz);
  auto bail = [&](int code, const char *fmt, auto... args) {
    free_layout(h);
    return fail(h, code, fmt, args...);
  };
#define LOAD_TRY(call)                                                                    \
  do {                                                                                    \
    hipError_t e_ = (call);                                                               \
    if (e_ != hipSuccess)                                                                 \
      return bail(e_ == hipErrorOutOfMemory ? BGMF_E_NOMEM : BGMF_E_HIP, "%s: %s", #call, \
                  hipGetErrorString(e_));                                                 \
  } while (0)
  Carve hc;
  if (h->bound) {
    if (!h->pinned || h->pinned_bytes < hneed)
      return fail(h, BGMF_E_BUDGET,
                  "the ratings do not fit the bound workspace, and streaming them needs a pinned "
                  "host arena of %zu bytes (bound: %zu)",
                  hneed, h->pinned ? h->pinned_bytes : (size_t)0);
    hc = Carve{h->pinned, h->pinned_bytes};
  } else {
    LOAD_TRY(pinned_alloc(h, &h->own_host, hneed));
    hc = Carve{static_cast<char *>(h->own_host), hneed};
  }
  h->host_rec = hc.take<uint2>(nnz);
  h->host_perm = hc.take<int32_t>(nnz);
  // block tables: the front of the workspace, or an allocation of their own
  Carve tc;
  if (h->bound) {
    tc = Carve{h->ws, h->ws_bytes};
  } else {
    LOAD_TRY(dev_alloc(h, &h->own_persist, tab));
    tc = Carve{static_cast<char *>(h->own_persist), tab};
  }
  h->block_ptr = tc.take<int64_t>(slots + 1);
  h->nofold = tc.take<uint8_t>(slots);
  h->wblock_ptr = nullptr;
  if (!h->host_rec || !h->host_perm || !h->block_ptr || !h->nofold)
    return bail(BGMF_E_HIP, "internal error: streamed load does not fit its plan");
  // the ratings region: the rest of a bound workspace, or allocated per pass
  const size_t ws_rest = h->bound ? h->ws_bytes - aligned(tc.used) : 0;
  auto region = [&](size_t want, Carve *c) -> int {
    if (h->bound) {
      *c = Carve{h->ws + aligned(tc.used), ws_rest};
      return BGMF_OK;
    }
    if (h->own_region) hipFree(h->own_region);
    h->own_region = nullptr;
    HIP_TRY(h, dev_alloc(h, &h->own_region, want));
    *c = Carve{static_cast<char *>(h->own_region), want};
    return BGMF_OK;
  };
  auto pick_batch = [&](auto bytes_of, size_t limit) {
    int64_t batch = std::min<int64_t>(nnz, (int64_t)1 << 24);
    while (batch > 4096 && bytes_of(batch) > limit) batch >>= 1;
    return batch;
  };
  const Grid G = grid_of(h);
  size_t peak = 0;

  // pass 1: ratings per slot
  {
    const size_t limit =
        h->bound ? ws_rest : std::max((size_t)budget, count_pass_bytes(std::min<int64_t>(nnz, 4096), p));
    const int64_t batch = pick_batch([&](int64_t b) { return count_pass_bytes(b, p); }, limit);
    const size_t want = count_pass_bytes(batch, p);
    if (want > limit)
      return bail(BGMF_E_BUDGET,
                  "the bound workspace cannot hold the slot counts of a %d x %d grid (%zu bytes "
                  "after the tables, %zu needed)",
                  p, p, limit, want);
    Carve c;
    if (region(want, &c) != BGMF_OK) return bail(BGMF_E_NOMEM, "%s", h->msg.c_str());
    int32_t *b_rows = c.take<int32_t>(batch), *b_cols = c.take<int32_t>(batch);
    int64_t *count = c.take<int64_t>(slots + 1);
    const size_t ssb = scan_scratch_bytes(slots);
    void *ss = c.take<char>(ssb);
    if (!b_rows || !b_cols || !count || !ss)
      return bail(BGMF_E_HIP, "internal error: slot-count pass does not fit its plan");
    peak = std::max(peak, c.high);
    LOAD_TRY(hipMemsetAsync(count, 0, ((size_t)slots + 1) * sizeof(int64_t), h->stream));
    for (int64_t e0 = 0; e0 < nnz; e0 += batch) {
      const int64_t cnt = std::min(batch, nnz - e0);
      LOAD_TRY(hipMemcpyAsync(b_rows, rows + e0, (size_t)cnt * 4, hipMemcpyHostToDevice, h->stream));
      LOAD_TRY(hipMemcpyAsync(b_cols, cols + e0, (size_t)cnt * 4, hipMemcpyHostToDevice, h->stream));
      LOAD_TRY(bucket_count_batch(b_rows, b_cols, cnt, G, count, h->stream));
    }
    LOAD_TRY(bucket_offsets(count, slots, h->block_ptr, ss, ssb, h->stream));
    LOAD_TRY(hipStreamSynchronize(h->stream));
  }
  std::vector<int64_t> bp((size_t)slots + 1);
  LOAD_TRY(hipMemcpy(bp.data(), h->block_ptr, bp.size() * sizeof(int64_t), hipMemcpyDeviceToHost));
  if (!offsets_ok(bp, nnz)) return layout_error(h);

  // ring of stream slots and resident strata, within the budget.
  // The budget is split into a ring of 3 (else 2) slots and a resident
  // region.  A slot holds the widest stratum plus the padding, and is made a
  // quarter of the budget when that fits: each chunk of strata in a slot
  // costs one copy and, with the persistent schedule, one launch, whose end
  // is a barrier across all row-blocks, so few large chunks are better.  The
  // resident region keeps the first strata of the epoch on the device for
  // good; the ring streams the others, and their first copies run while the
  // resident strata are swept.
  h->strat.assign((size_t)p + 1, 0);
  int64_t widest = 0;
  for (int64_t s2 = 0; s2 <= p; ++s2) h->strat[s2] = bp[s2 * p];
  for (int64_t s2 = 0; s2 < p; ++s2) widest = std::max(widest, h->strat[s2 + 1] - h->strat[s2]);
  const int64_t need = widest + kRecPad;
  const int64_t budget_recs = budget / (int64_t)sizeof(uint2);
  h->nslots = 0;
  for (int cand : {3, 2}) {
    for (int64_t slot : {std::max(need, budget_recs / 4), need}) {
      if ((int64_t)cand * slot <= budget_recs) {
        h->nslots = cand;
        h->slot_recs = slot;
        break;
      }
    }
    if (h->nslots) break;
  }
  if (h->nslots == 0)
    return bail(BGMF_E_BUDGET,
                "ratings budget of %lld bytes holds fewer than two strata (the widest stratum "
                "needs %lld bytes)",
                (long long)budget, (long long)(need * (int64_t)sizeof(uint2)));
  const size_t ring_bytes = aligned((size_t)h->nslots * (size_t)h->slot_recs * sizeof(uint2));
  const int64_t res_cap =
      (size_t)budget > ring_bytes ? ((int64_t)((size_t)budget - ring_bytes)) / (int64_t)sizeof(uint2) : 0;
  h->s_res = 0;
  while (h->s_res < p && h->strat[h->s_res + 1] + kRecPad <= res_cap) ++h->s_res;
  // chunks of consecutive streamed strata, each as many as fit in a slot
  h->chunk.assign(1, h->s_res);
  for (int32_t s2 = h->s_res; s2 < p; ++s2)
    if (h->strat[s2 + 1] - h->strat[h->chunk.back()] + kRecPad > h->slot_recs)
      h->chunk.push_back(s2);
  if (h->chunk.back() != p) h->chunk.push_back(p);

  // groups of whole blocks whose bucketing fits the region: at most `cap`
  // ratings in at most `span` consecutive slots (the slot tables take up to
  // a quarter of the region)
  int64_t biggest = 1;
  for (int64_t q = 0; q < slots; ++q) biggest = std::max(biggest, bp[q + 1] - bp[q]);
  const int64_t min_batch = std::min<int64_t>(nnz, 4096);
  const size_t limit =
      h->bound ? ws_rest : std::max((size_t)budget, group_pass_bytes(min_batch, biggest, 1));
  int64_t span = std::max<int64_t>(1, std::min<int64_t>(slots, (int64_t)(limit / 4 / 32)));
  while (span > 1 && group_pass_bytes(min_batch, biggest, span) > limit) span >>= 1;
  const int64_t batch =
      pick_batch([&](int64_t b) { return group_pass_bytes(b, biggest, span); }, limit);
  if (group_pass_bytes(batch, biggest, span) > limit)
    return bail(BGMF_E_BUDGET,
                "the largest block (%lld ratings) needs %zu bytes to be bucketed; the bound "
                "workspace has %zu after the tables",
                (long long)biggest, group_pass_bytes(batch, biggest, span), limit);
  int64_t lo = biggest, hi = std::max<int64_t>(biggest, nnz);
  while (lo < hi) {
    const int64_t mid = lo + (hi - lo + 1) / 2;
    if (group_pass_bytes(batch, mid, span) <= limit) lo = mid;
    else hi = mid - 1;
  }
  const int64_t cap = lo;
  std::vector<std::pair<int64_t, int64_t>> groups;
  for (int64_t q0 = 0; q0 < slots;) {
    int64_t q1 = q0 + 1;
    while (q1 < slots && q1 - q0 < span && bp[q1 + 1] - bp[q0] <= cap) ++q1;
    if (bp[q1] > bp[q0]) groups.emplace_back(q0, q1);
    q0 = q1;
  }
  Carve dc;
  if (region(std::max((size_t)budget, group_pass_bytes(batch, cap, span)), &dc) != BGMF_OK)
    return bail(BGMF_E_NOMEM, "%s", h->msg.c_str());
  const size_t mark = 0;
  h->load_groups = (int64_t)groups.size();

  // pass 2: gather, sort and store each group
  {
    Carve c = dc;
    c.used = c.high = mark;
    int32_t *b_rows = c.take<int32_t>(batch), *b_cols = c.take<int32_t>(batch);
    float *b_vals = c.take<float>(batch);
    int64_t *flag = c.take<int64_t>(batch + 1), *pos = c.take<int64_t>(batch + 1);
    const size_t ssb = scan_scratch_bytes(batch);
    void *ss = c.take<char>(ssb);
    GroupArrays g{c.take<int32_t>(cap), c.take<int32_t>(cap), c.take<float>(cap),
                  c.take<int32_t>(cap), cap};
    int64_t *fill = c.take<int64_t>(1);
    const size_t bsb = bucket_scratch_bytes(cap, span);
    void *bs = c.take<char>(bsb);
    uint2 *rec_t = c.take<uint2>(cap + kRecPad);
    int32_t *perm_t = c.take<int32_t>(cap);
    int64_t *bp_t = c.take<int64_t>(span + 1);
    if (!b_rows || !b_cols || !b_vals || !flag || !pos || !ss || !g.rows || !g.cols || !g.vals ||
        !g.e || !fill || !bs || !rec_t || !perm_t || !bp_t)
      return bail(BGMF_E_HIP, "internal error: group pass does not fit its plan");
    peak = std::max(peak, c.high);
    LOAD_TRY(hipMemsetAsync(h->err, 0, sizeof(int32_t), h->stream));
    LOAD_TRY(hipMemsetAsync(h->nofold, 0, (size_t)slots, h->stream));
    std::vector<int64_t> got;
    for (const auto &gr : groups) {
      const int64_t q0 = gr.first, q1 = gr.second, gcnt = bp[q1] - bp[q0];
      LOAD_TRY(hipMemsetAsync(fill, 0, sizeof(int64_t), h->stream));
      for (int64_t e0 = 0; e0 < nnz; e0 += batch) {
        const int64_t cnt = std::min(batch, nnz - e0);
        LOAD_TRY(hipMemcpyAsync(b_rows, rows + e0, (size_t)cnt * 4, hipMemcpyHostToDevice, h->stream));
        LOAD_TRY(hipMemcpyAsync(b_cols, cols + e0, (size_t)cnt * 4, hipMemcpyHostToDevice, h->stream));
        LOAD_TRY(hipMemcpyAsync(b_vals, vals + e0, (size_t)cnt * 4, hipMemcpyHostToDevice, h->stream));
        LOAD_TRY(bucket_select_batch(b_rows, b_cols, b_vals, cnt, e0, G, q0, q1, flag, pos, ss,
                                     ssb, fill, g, h->err, h->stream));
      }
      BucketOut out{bp_t, nullptr, perm_t, rec_t, h->nofold};
      LOAD_TRY(bucket(g.rows, g.cols, g.vals, gcnt, G, h->rows_max, q0, q1 - q0, true, bs, bsb,
                      out, h->err, h->stream));
      LOAD_TRY(bucket_map_perm(perm_t, g.e, gcnt, h->err, h->stream));
      LOAD_TRY(hipMemcpyAsync(h->host_rec + bp[q0], rec_t, (size_t)gcnt * sizeof(uint2),
                              hipMemcpyDeviceToHost, h->stream));
      LOAD_TRY(hipMemcpyAsync(h->host_perm + bp[q0], perm_t, (size_t)gcnt * sizeof(int32_t),
                              hipMemcpyDeviceToHost, h->stream));
      // the group's own offsets must agree with the counting pass
      got.assign((size_t)(q1 - q0) + 2, -1);
      LOAD_TRY(hipMemcpyAsync(got.data(), bp_t, (size_t)(q1 - q0 + 1) * sizeof(int64_t),
                              hipMemcpyDeviceToHost, h->stream));
      LOAD_TRY(hipMemcpyAsync(got.data() + (q1 - q0 + 1), fill, sizeof(int64_t),
                              hipMemcpyDeviceToHost, h->stream));
      LOAD_TRY(hipStreamSynchronize(h->stream));
      bool ok = got[q1 - q0 + 1] == gcnt;
      for (int64_t q = q0; ok && q <= q1; ++q) ok = got[q - q0] - got[0] == bp[q] - bp[q0];
      if (!ok) return layout_error(h);
    }
    int32_t derr = 0;
    LOAD_TRY(hipMemcpy(&derr, h->err, sizeof derr, hipMemcpyDeviceToHost));
    if (derr != 0) return layout_error(h);
  }

  // the region now holds the ring and the resident strata
  {
    Carve c = dc;
    c.used = c.high = mark;
    const int64_t count = h->strat[h->s_res];
    h->ring = c.take<uint2>((size_t)h->nslots * (size_t)h->slot_recs);
    h->resident = h->s_res > 0 ? c.take<uint2>((size_t)count + kRecPad) : nullptr;
    if (!h->ring || (h->s_res > 0 && !h->resident))
      return bail(BGMF_E_HIP, "internal error: stream ring does not fit its plan");
    peak = std::max(peak, c.high);
    if (h->s_res > 0) {
      LOAD_TRY(hipMemcpyAsync(h->resident, h->host_rec, (size_t)count * sizeof(uint2),
                              hipMemcpyHostToDevice, h->stream));
      LOAD_TRY(hipMemsetAsync(h->resident + count, 0, (size_t)kRecPad * sizeof(uint2), h->stream));
    }
    LOAD_TRY(hipMemsetAsync(h->ring, 0, (size_t)h->nslots * (size_t)h->slot_recs * sizeof(uint2),
                            h->stream));
  }
  if (!h->side) LOAD_TRY(hipStreamCreateWithFlags(&h->side, hipStreamNonBlocking));
  h->ready.assign(h->nslots, nullptr);
  h->freed.assign(h->nslots, nullptr);
  h->slot_used.assign(h->nslots, false);
  for (int i = 0; i < h->nslots; ++i) {
    LOAD_TRY(hipEventCreateWithFlags(&h->ready[i], hipEventDisableTiming));
    LOAD_TRY(hipEventCreateWithFlags(&h->freed[i], hipEventDisableTiming));
  }
  LOAD_TRY(hipStreamSynchronize(h->stream));
#undef LOAD_TRY
  h->load_peak = (int64_t)peak;
  h->ooc = true;
  set_chain_stats(h, bp);
  return BGMF_OK;
}

}  // namespace

extern "C" {

bgmf_t *bgmf_create(int64_t n, int64_t m, int32_t k, int32_t p) {
  if (n < 1 || m < 1 || n >= (1ll << 31) || m >= (1ll << 31)) {
    fail(nullptr, BGMF_E_ARG, "n and m must be in [1, 2^31): n=%lld m=%lld", (long long)n,
         (long long)m);
    return nullptr;
  }
  if (k < 16 || k > 256 || k % 16 != 0) {
    fail(nullptr, BGMF_E_ARG, "k must be a multiple of 16 in [16, 256]: k=%d", k);
    return nullptr;
  }
  if (p < 1 || p > 8192 || p > n || p > m) {
    fail(nullptr, BGMF_E_ARG, "p must be in [1, min(n, m, 8192)]: p=%d", p);
    return nullptr;
  }
  if ((n + p - 1) / p > 65536 || (m + p - 1) / p > (1 << kColBits)) {
    fail(nullptr, BGMF_E_ARG, "blocks too large: ceil(n/p)=%lld (max 65536), ceil(m/p)=%lld (max %d)",
         (long long)((n + p - 1) / p), (long long)((m + p - 1) / p), 1 << kColBits);
    return nullptr;
  }
  bgmf_t *h = new (std::nothrow) bgmf();
  if (!h) {
    fail(nullptr, BGMF_E_NOMEM, "out of host memory");
    return nullptr;
  }
  h->n = n;
  h->m = m;
  h->k = k;
  h->p = p;
  h->kp = 16;
  while (h->kp < k) h->kp <<= 1;
  h->rcut.resize((size_t)p + 1);
  h->ccut.resize((size_t)p + 1);
  for (int64_t b = 0; b <= p; ++b) {
    h->rcut[b] = equal_cut(b, n, p);
    h->ccut[b] = equal_cut(b, m, p);
  }
  h->rows_max = check_cuts(h->rcut.data(), p, n, 65536);
  h->cols_max = (int)check_cuts(h->ccut.data(), p, m, 1 << kColBits);

  auto bail = [&](hipError_t e, const char *what) -> bgmf_t * {
    fail(nullptr, e == hipErrorOutOfMemory ? BGMF_E_NOMEM : BGMF_E_HIP, "%s: %s", what,
         hipGetErrorString(e));
    bgmf_destroy(h);
    return nullptr;
  };
  hipError_t e;
  if ((e = hipGetDevice(&h->device)) != hipSuccess) return bail(e, "hipGetDevice");
  int lds_max = 0;
  if ((e = hipDeviceGetAttribute(&lds_max, hipDeviceAttributeMaxSharedMemoryPerBlock, h->device)) !=
      hipSuccess)
    return bail(e, "hipDeviceGetAttribute");
  if ((e = hipDeviceGetAttribute(&h->cus, hipDeviceAttributeMultiprocessorCount, h->device)) !=
      hipSuccess)
    return bail(e, "hipDeviceGetAttribute");
  h->lds_limit = (size_t)lds_max;
  int khz = 0;
  if ((e = hipDeviceGetAttribute(&khz, hipDeviceAttributeWallClockRate, h->device)) != hipSuccess)
    return bail(e, "hipDeviceGetAttribute");
  if (khz > 0) h->clock_khz = khz;
  if ((e = configure_sweep(h)) != hipSuccess) return bail(e, "configure_sweep");
  if ((e = dev_alloc(h, reinterpret_cast<void **>(&h->d_cuts),
                     2 * ((size_t)p + 1) * sizeof(int64_t))) != hipSuccess)
    return bail(e, "hipMalloc(cuts)");
  if ((e = hipMemcpy(h->d_cuts, h->rcut.data(), ((size_t)p + 1) * sizeof(int64_t),
                     hipMemcpyHostToDevice)) != hipSuccess ||
      (e = hipMemcpy(h->d_cuts + p + 1, h->ccut.data(), ((size_t)p + 1) * sizeof(int64_t),
                     hipMemcpyHostToDevice)) != hipSuccess)
    return bail(e, "hipMemcpy(cuts)");
  if ((e = hipStreamCreateWithFlags(&h->own_stream, hipStreamNonBlocking)) != hipSuccess)
    return bail(e, "hipStreamCreate");
  h->stream = h->own_stream;
  for (auto &ev : h->ev)
    if ((e = hipEventCreate(&ev)) != hipSuccess) return bail(e, "hipEventCreate");
  if ((e = dev_alloc(h, reinterpret_cast<void **>(&h->U), (size_t)n * k * sizeof(float))) !=
      hipSuccess)
    return bail(e, "hipMalloc(U)");
  if ((e = dev_alloc(h, reinterpret_cast<void **>(&h->V), (size_t)m * k * sizeof(float))) !=
      hipSuccess)
    return bail(e, "hipMalloc(V)");
  if ((e = dev_alloc(h, reinterpret_cast<void **>(&h->flags),
                     (size_t)p * kFlagStride * sizeof(int64_t))) != hipSuccess)
    return bail(e, "hipMalloc(flags)");
  if ((e = dev_alloc(h, reinterpret_cast<void **>(&h->err), sizeof(int32_t))) != hipSuccess)
    return bail(e, "hipMalloc(err)");
  if ((e = dev_alloc(h, reinterpret_cast<void **>(&h->partials),
                     rmse_partials_count(p) * sizeof(double))) != hipSuccess)
    return bail(e, "hipMalloc(partials)");
  if ((e = dev_alloc(h, reinterpret_cast<void **>(&h->d_rmse), sizeof(double))) != hipSuccess)
    return bail(e, "hipMalloc(rmse)");
  if ((e = hipMemset(h->flags, 0, (size_t)p * kFlagStride * sizeof(int64_t))) != hipSuccess)
    return bail(e, "hipMemset");
  if ((e = hipMemset(h->err, 0, sizeof(int32_t))) != hipSuccess) return bail(e, "hipMemset");
  if ((e = hipMemset(h->U, 0, (size_t)n * k * sizeof(float))) != hipSuccess)
    return bail(e, "hipMemset");
  if ((e = hipMemset(h->V, 0, (size_t)m * k * sizeof(float))) != hipSuccess)
    return bail(e, "hipMemset");
  return h;
}

void bgmf_destroy(bgmf_t *h) {
  if (!h) return;
  if (h->stream) hipStreamSynchronize(h->stream);
  free_layout(h);
  if (h->own_factors) {
    hipFree(h->U);
    hipFree(h->V);
  }
  hipFree(h->flags);
  hipFree(h->err);
  hipFree(h->partials);
  hipFree(h->d_rmse);
  hipFree(h->d_cuts);
  hipFree(h->d_trace);
  for (auto &ev : h->ev)
    if (ev) hipEventDestroy(ev);
  if (h->own_stream) hipStreamDestroy(h->own_stream);
  if (h->side) hipStreamDestroy(h->side);
  delete h;
}

const char *bgmf_last_error(const bgmf_t *h) {
  return h ? h->msg.c_str() : g_create_error.c_str();
}

int bgmf_set_stream(bgmf_t *h, void *hip_stream) {
  if (!h) return BGMF_E_ARG;
  hipStream_t next = hip_stream ? static_cast<hipStream_t>(hip_stream) : h->own_stream;
  if (next != h->stream) {
    // work already queued on the old stream finishes before later work
    HIP_TRY(h, hipStreamSynchronize(h->stream));
    h->stream = next;
  }
  return BGMF_OK;
}

int bgmf_query_sizes(const bgmf_t *h, int64_t nnz, size_t *factor_bytes, size_t *min_ws_bytes,
                     size_t *incore_ws_bytes, size_t *pinned_bytes) {
  if (!h) return BGMF_E_ARG;
  if (nnz < 1 || nnz >= (1ll << 31)) {
    const_cast<bgmf_t *>(h)->msg = "bgmf_query_sizes: nnz must be in [1, 2^31)";
    return BGMF_E_ARG;
  }
  const int32_t p = h->p;
  if (factor_bytes) *factor_bytes = (size_t)(h->n + h->m) * (size_t)h->k * sizeof(float);
  if (incore_ws_bytes)
    *incore_ws_bytes = tables_bytes(p, true) + incore_keep_bytes(nnz) + incore_temp_bytes(nnz, p);
  if (min_ws_bytes) {
    // necessary, not sufficient: the streamed load also needs room to bucket
    // its largest block and a ring of two copies of its widest stratum, which
    // depend on how the ratings fall into the grid
    const int64_t slots = (int64_t)p * p;
    const int64_t per_stratum = (nnz + p - 1) / p, per_block = (nnz + slots - 1) / slots;
    int64_t batch = std::min<int64_t>(nnz, 4096);
    size_t need = std::max(count_pass_bytes(batch, p), group_pass_bytes(batch, per_block, 1));
    need = std::max(need, 2 * aligned(((size_t)per_stratum + kRecPad) * sizeof(uint2)) + 2 * kAlign);
    *min_ws_bytes = tables_bytes(p, false) + need;
  }
  if (pinned_bytes) *pinned_bytes = pinned_need_bytes(nnz);
  return BGMF_OK;
}

int bgmf_bind(bgmf_t *h, float *U_dev, float *V_dev, void *ws_dev, size_t ws_bytes,
              void *pinned_host, size_t pinned_bytes, void *hip_stream) {
  if (!h) return BGMF_E_ARG;
  if (!U_dev || !V_dev || !ws_dev)
    return fail(h, BGMF_E_ARG, "bgmf_bind: U, V and the workspace must be given");
  const uintptr_t bits = reinterpret_cast<uintptr_t>(U_dev) | reinterpret_cast<uintptr_t>(V_dev) |
                         reinterpret_cast<uintptr_t>(ws_dev) |
                         reinterpret_cast<uintptr_t>(pinned_host);
  if (bits & (kAlign - 1))
    return fail(h, BGMF_E_ARG, "bgmf_bind: every buffer must start on a 256-byte boundary");
  if (pinned_host == nullptr) pinned_bytes = 0;
  if (h->loaded) return fail(h, BGMF_E_STATE, "bgmf_bind: bind before loading ratings");
  if (ws_bytes < tables_bytes(h->p, false))
    return fail(h, BGMF_E_BUDGET, "bgmf_bind: a workspace of %zu bytes is smaller than the "
                "block tables (%zu bytes)", ws_bytes, tables_bytes(h->p, false));
  // the buffers must be memory the device can reach: device memory on the
  // handle's device, and pinned host memory for the arena
  for (const void *ptr : {static_cast<const void *>(U_dev), static_cast<const void *>(V_dev),
                          static_cast<const void *>(ws_dev)}) {
    hipPointerAttribute_t a{};
    if (hipPointerGetAttributes(&a, ptr) != hipSuccess || a.type != hipMemoryTypeDevice ||
        a.device != h->device) {
      hipGetLastError();
      return fail(h, BGMF_E_ARG, "bgmf_bind: U, V and the workspace must be device memory on "
                  "device %d", h->device);
    }
  }
  if (pinned_host) {
    hipPointerAttribute_t a{};
    if (hipPointerGetAttributes(&a, pinned_host) != hipSuccess || a.type != hipMemoryTypeHost) {
      hipGetLastError();
      return fail(h, BGMF_E_ARG, "bgmf_bind: the host arena must be pinned host memory");
    }
  }
  int rc = bgmf_set_stream(h, hip_stream);
  if (rc != BGMF_OK) return rc;
  HIP_TRY(h, hipStreamSynchronize(h->stream));
  free_layout(h);
  if (h->own_factors) {
    hipFree(h->U);
    hipFree(h->V);
  }
  h->U = U_dev;
  h->V = V_dev;
  h->own_factors = false;
  h->factors_set = true;  // the caller's buffers hold the factors
  h->bound = true;
  h->ws = static_cast<char *>(ws_dev);
  h->ws_bytes = ws_bytes;
  h->pinned = static_cast<char *>(pinned_host);
  h->pinned_bytes = pinned_bytes;
  return BGMF_OK;
}

int bgmf_set_factors(bgmf_t *h, const float *U, const float *V) {
  if (!h) return BGMF_E_ARG;
  const Range range("bgmf_set_factors");
  if (!U || !V) return fail(h, BGMF_E_ARG, "bgmf_set_factors: null pointer");
  for (int64_t x = 0, cnt = h->n * h->k; x < cnt; ++x)
    if (!std::isfinite(U[x])) return fail(h, BGMF_E_NONFINITE, "U[%lld] is not finite", (long long)x);
  for (int64_t x = 0, cnt = h->m * h->k; x < cnt; ++x)
    if (!std::isfinite(V[x])) return fail(h, BGMF_E_NONFINITE, "V[%lld] is not finite", (long long)x);
  HIP_TRY(h, hipMemcpyAsync(h->U, U, (size_t)h->n * h->k * sizeof(float), hipMemcpyHostToDevice,
                            h->stream));
  HIP_TRY(h, hipMemcpyAsync(h->V, V, (size_t)h->m * h->k * sizeof(float), hipMemcpyHostToDevice,
                            h->stream));
  HIP_TRY(h, hipStreamSynchronize(h->stream));
  h->factors_set = true;
  return BGMF_OK;
}

int bgmf_load_coo(bgmf_t *h, const int32_t *rows, const int32_t *cols, const float *vals,
                  int64_t nnz) {
  if (!h) return BGMF_E_ARG;
  const Range range("bgmf_load_coo");
  if (!rows || !cols || !vals) return fail(h, BGMF_E_ARG, "bgmf_load_coo: null pointer");
  if (nnz < 1 || nnz >= (1ll << 31))
    return fail(h, BGMF_E_ARG, "nnz must be in [1, 2^31): %lld", (long long)nnz);
  for (int64_t e = 0; e < nnz; ++e) {
    if (rows[e] < 0 || rows[e] >= h->n || cols[e] < 0 || cols[e] >= h->m)
      return fail(h, BGMF_E_RANGE, "rating %lld at (%d, %d) is outside the %lld x %lld matrix",
                  (long long)e, rows[e], cols[e], (long long)h->n, (long long)h->m);
    if (!std::isfinite(vals[e]))
      return fail(h, BGMF_E_NONFINITE, "rating %lld has a non-finite value", (long long)e);
  }
  HIP_TRY(h, hipStreamSynchronize(h->stream));
  free_layout(h);
  // In-core when the one-pass bucketing (records, perm and its temporaries)
  // fits the ratings budget -- a bound workspace minus the tables, or the
  // BGMF_OPT_RATINGS_BUDGET option, whichever is smaller -- else streamed.
  const size_t incore = incore_keep_bytes(nnz) + incore_temp_bytes(nnz, h->p);
  int64_t region = h->budget;  // 0: no limit
  bool fits = h->budget == 0 || incore <= (size_t)h->budget;
  if (h->bound) {
    const size_t tab_in = tables_bytes(h->p, true), tab_st = tables_bytes(h->p, false);
    fits = fits && h->ws_bytes >= tab_in + incore;
    if (h->ws_bytes < tab_st)
      return fail(h, BGMF_E_BUDGET, "the bound workspace (%zu bytes) is smaller than the block "
                  "tables (%zu bytes)", h->ws_bytes, tab_st);
    const int64_t avail = (int64_t)(h->ws_bytes - tab_st);
    region = h->budget > 0 ? std::min(h->budget, avail) : avail;
  }
  const int rc = fits ? load_incore(h, rows, cols, vals, nnz)
                      : load_streamed(h, rows, cols, vals, nnz, region);
  if (rc != BGMF_OK) return rc;
  HIP_TRY(h, hipMemsetAsync(h->flags, 0, (size_t)h->p * kFlagStride * sizeof(int64_t), h->stream));
  HIP_TRY(h, hipStreamSynchronize(h->stream));
  h->epochs_done = 0;
  h->nnz = nnz;
  h->loaded = true;
  return BGMF_OK;
}

namespace {

// Out-of-core streaming, one pass over the strata (an epoch or an RMSE
// pass).  Chunk c goes to ring slot c mod nslots.  Its copy runs on the side
// stream once the kernels that last read the slot have finished (the slot's
// freed event); the handle's stream waits for the copy (ready event) just
// before the chunk's kernels, and records freed after them.  The copies of
// the first nslots chunks are queued at the start of the pass, so they run
// while the resident strata are swept.
int queue_copy(bgmf_t *h, size_t c) {
  const int slot = (int)(c % (size_t)h->nslots);
  uint2 *dst = h->ring + (size_t)slot * (size_t)h->slot_recs;
  const int64_t first = h->strat[h->chunk[c]];
  const int64_t count = h->strat[h->chunk[c + 1]] - first;
  if (h->slot_used[slot]) HIP_TRY(h, hipStreamWaitEvent(h->side, h->freed[slot], 0));
  if (count > 0)
    HIP_TRY(h, hipMemcpyAsync(dst, h->host_rec + first, (size_t)count * sizeof(uint2),
                              hipMemcpyHostToDevice, h->side));
  HIP_TRY(h, hipEventRecord(h->ready[slot], h->side));
  return BGMF_OK;
}

int stream_begin(bgmf_t *h) {
  const size_t nch = h->chunk.size() - 1;
  for (h->issued = 0; h->issued < std::min(nch, (size_t)h->nslots); ++h->issued) {
    int rc = queue_copy(h, h->issued);
    if (rc != BGMF_OK) return rc;
  }
  return BGMF_OK;
}

// Make the handle's stream wait for chunk c; returns its device records.
int chunk_ready(bgmf_t *h, size_t c, const uint2 **slot_rec) {
  const int slot = (int)(c % (size_t)h->nslots);
  HIP_TRY(h, hipStreamWaitEvent(h->stream, h->ready[slot], 0));
  *slot_rec = h->ring + (size_t)slot * (size_t)h->slot_recs;
  return BGMF_OK;
}

// The kernels of chunk c are queued: free its slot and queue the next copy.
int chunk_done(bgmf_t *h, size_t c) {
  const int slot = (int)(c % (size_t)h->nslots);
  HIP_TRY(h, hipEventRecord(h->freed[slot], h->stream));
  h->slot_used[slot] = true;
  if (h->issued < h->chunk.size() - 1) {
    int rc = queue_copy(h, h->issued++);
    if (rc != BGMF_OK) return rc;
  }
  return BGMF_OK;
}

// Where the sweep keeps V, and how it is launched.  Automatic placement
// stages the column slice in LDS when it fits with all p waves resident at
// once, and otherwise leaves V in global memory.  The automatic schedule is
// persistent for the LDS placement only: with V in global memory a
// persistent launch needs device-scope V accesses on every update, which
// cost more than one launch per stratum with plain cached accesses.
struct SweepShape {
  bool lds;         // V slice staged in LDS
  bool persistent;  // one launch for all strata
  int vmode, wpg;
  size_t lds_bytes;
};

SweepShape sweep_shape(const bgmf_t *h) {
  SweepShape sh{};
  sh.lds = h->v_staging == 1 || (h->v_staging == 0 && h->lds_fits && h->coop_lds);
  const bool coop = sh.lds ? h->coop_lds : h->coop_gv;
  sh.persistent = coop && (h->schedule == 2 || (h->schedule == 0 && sh.lds));
  sh.vmode = sh.lds ? kVLds : (sh.persistent ? kVGlobalCoherent : kVGlobal);
  sh.wpg = sh.lds ? h->wpg_lds : h->wpg_gv;
  sh.lds_bytes = sh.lds ? h->lds_bytes_lds : h->lds_bytes_gv;
  return sh;
}

}  // namespace

int bgmf_epoch(bgmf_t *h, float alpha, float beta) {
  if (!h) return BGMF_E_ARG;
  const Range range("bgmf_epoch");
  if (!std::isfinite(alpha) || !(alpha > 0.0f) || !std::isfinite(beta) || beta < 0.0f)
    return fail(h, BGMF_E_ARG, "alpha must be finite and > 0, beta finite and >= 0");
  if (!h->loaded) return fail(h, BGMF_E_STATE, "bgmf_epoch: no ratings loaded");
  if (!h->factors_set) return fail(h, BGMF_E_STATE, "bgmf_epoch: factors not set");
  SgdParams P{};
  P.U = h->U;
  P.V = h->V;
  P.rec = h->rec;
  P.blk = h->wblock_ptr;  // wave-major: block (b, s) at b*p + s
  P.stride_b = h->p;
  P.stride_s = 1;
  P.rec_origin = 0;
  P.flags = h->flags;
  P.err = h->err;
  P.n = h->n;
  P.m = h->m;
  P.rcut = h->d_cuts;
  P.ccut = h->d_cuts + h->p + 1;
  P.k = h->k;
  P.p = h->p;
  P.cols_max = h->cols_max;
  P.g_base = h->epochs_done * (int64_t)h->p;
  P.wait_ticks = h->wait_us * h->clock_khz / 1000;  // s_memrealtime ticks
  P.alpha = alpha;
  P.beta = beta;
  P.xcd_remap = (int32_t)h->xcd_remap;
  P.passes = (int32_t)h->passes;
  P.single_col = (int32_t)h->single_col;
  P.nofold = h->nofold;
  const SweepShape sh = sweep_shape(h);
  P.lds_ring = sh.lds ? h->lds_ring : 0;
  if (h->d_trace) {
    // blocks the epoch skips (empty strata of a streamed epoch) keep 0
    h->trace_valid = false;
    HIP_TRY(h, clear_trace(h->d_trace, 2 * (int64_t)h->p * h->p, h->stream));
    P.trace = h->d_trace;
  }
  HIP_TRY(h, hipEventRecord(h->ev[0], h->stream));
  if (h->ooc) {
    // resident strata, then the streamed chunks; each range is one
    // persistent launch or one launch per stratum
    P.blk = h->block_ptr;  // stratum-major: block (b, s) at s*p + b
    P.stride_b = 1;
    P.stride_s = h->p;
    auto sweep_range = [&](const uint2 *rec, int64_t origin, int32_t s0, int32_t s1) -> int {
      P.rec = rec;
      P.rec_origin = origin;
      if (sh.persistent && s1 - s0 > 1) {
        P.s_begin = s0;
        P.s_end = s1;
        HIP_TRY(h, launch_sgd(P, h->kp, sh.vmode, sh.wpg, true, sh.lds_bytes, h->stream));
        return BGMF_OK;
      }
      const int vmode = sh.lds ? kVLds : kVGlobal;
      for (int32_t s2 = s0; s2 < s1; ++s2) {
        if (h->strat[s2 + 1] == h->strat[s2]) continue;
        P.s_begin = s2;
        P.s_end = s2 + 1;
        HIP_TRY(h, launch_sgd(P, h->kp, vmode, sh.wpg, false, sh.lds_bytes, h->stream));
      }
      return BGMF_OK;
    };
    int rc = stream_begin(h);
    if (rc == BGMF_OK && h->s_res > 0) rc = sweep_range(h->resident, 0, 0, h->s_res);
    for (size_t c = 0; rc == BGMF_OK && c + 1 < h->chunk.size(); ++c) {
      const int32_t s0 = h->chunk[c], s1 = h->chunk[c + 1];
      const uint2 *slot_rec = nullptr;
      rc = chunk_ready(h, c, &slot_rec);
      if (rc == BGMF_OK && h->strat[s1] > h->strat[s0])
        rc = sweep_range(slot_rec, h->strat[s0], s0, s1);
      if (rc == BGMF_OK) rc = chunk_done(h, c);
    }
    if (rc != BGMF_OK) return rc;
  } else if (sh.persistent) {
    P.s_begin = 0;
    P.s_end = h->p;
    HIP_TRY(h, launch_sgd(P, h->kp, sh.vmode, sh.wpg, true, sh.lds_bytes, h->stream));
  } else {
    for (int32_t s = 0; s < h->p; ++s) {
      P.s_begin = s;
      P.s_end = s + 1;
      HIP_TRY(h, launch_sgd(P, h->kp, sh.vmode, sh.wpg, false, sh.lds_bytes, h->stream));
    }
  }
  HIP_TRY(h, hipEventRecord(h->ev[1], h->stream));
  h->epoch_timed = true;
  h->epochs_done += 1;
  h->trace_valid = h->d_trace != nullptr;
  return BGMF_OK;
}

int bgmf_rmse(bgmf_t *h, double *out) {
  if (!h) return BGMF_E_ARG;
  const Range range("bgmf_rmse");
  if (!out) return fail(h, BGMF_E_ARG, "bgmf_rmse: null output");
  if (!h->loaded) return fail(h, BGMF_E_STATE, "bgmf_rmse: no ratings loaded");
  if (!h->factors_set) return fail(h, BGMF_E_STATE, "bgmf_rmse: factors not set");
  HIP_TRY(h, hipEventRecord(h->ev[2], h->stream));
  if (h->ooc) {
    HIP_TRY(h, rmse_stratum_begin(h->partials, h->p, h->stream));
    int rc = stream_begin(h);
    if (rc != BGMF_OK) return rc;
    if (h->s_res > 0)
      HIP_TRY(h, rmse_stratum_add(h->resident, 0, h->block_ptr, 0, h->s_res, h->U, h->V,
                                  grid_of(h), h->k, h->partials, h->stream));
    for (size_t c = 0; c + 1 < h->chunk.size(); ++c) {
      const int32_t s0 = h->chunk[c], s1 = h->chunk[c + 1];
      const uint2 *slot_rec = nullptr;
      rc = chunk_ready(h, c, &slot_rec);
      if (rc != BGMF_OK) return rc;
      if (h->strat[s1] > h->strat[s0])
        HIP_TRY(h, rmse_stratum_add(slot_rec, h->strat[s0], h->block_ptr, s0, s1, h->U, h->V,
                                    grid_of(h), h->k, h->partials, h->stream));
      rc = chunk_done(h, c);
      if (rc != BGMF_OK) return rc;
    }
    HIP_TRY(h, rmse_stratum_end(h->partials, h->p, h->nnz, h->d_rmse, h->stream));
  } else {
    HIP_TRY(h, launch_rmse(h->rec, h->wblock_ptr, h->U, h->V, grid_of(h), h->rows_max, h->k,
                           h->nnz, h->partials, h->d_rmse, h->lds_limit, h->stream));
  }
  HIP_TRY(h, hipEventRecord(h->ev[3], h->stream));
  h->rmse_timed = true;
  double r = 0.0;
  HIP_TRY(h, hipMemcpyAsync(&r, h->d_rmse, sizeof r, hipMemcpyDeviceToHost, h->stream));
  int rc = sync_checked(h);
  if (rc != BGMF_OK) return rc;
  *out = r;
  return BGMF_OK;
}

namespace {

// Greedy nnz-balanced cut points over one dimension of length len: block b
// ends at the first index where the running count of ratings reaches its
// share of what is left (ceil(remaining / blocks left)); if that last index
// alone holds a full share, the block ends before it instead, so that heavy
// rows or columns get blocks of their own (one index cannot be split, and
// its ratings form one serial chain).  Blocks stay at least one and at most
// cap wide, leaving every later block at least one index and at most cap.
// Integer arithmetic only, so the result is exact.
bool balanced_dim(const std::vector<int64_t> &deg, int32_t p, int64_t cap, int64_t *cut) {
  const int64_t len = (int64_t)deg.size();
  if (p < 1 || p > len || cap < 1 || cap * p < len) return false;
  std::vector<int64_t> cum((size_t)len + 1, 0);
  for (int64_t i = 0; i < len; ++i) cum[i + 1] = cum[i] + deg[i];
  const int64_t total = cum[len];
  cut[0] = 0;
  for (int32_t b = 1; b < p; ++b) {
    const int64_t prev = cut[b - 1];
    const int64_t left = p - b + 1;  // blocks b-1 .. p-1
    const int64_t target = cum[prev] + (total - cum[prev] + left - 1) / left;
    int64_t c = (int64_t)(std::lower_bound(cum.begin() + prev + 1, cum.end(), target) -
                          cum.begin());
    if (c <= len && c - 1 > prev && deg[c - 1] >= target - cum[prev]) c -= 1;
    c = std::max(c, prev + 1);
    c = std::min(c, prev + cap);
    c = std::min(c, len - (p - b));                      // one index for each later block
    c = std::max(c, len - (int64_t)(p - b) * cap);       // later blocks within the cap
    cut[b] = c;
  }
  cut[p] = len;
  return true;
}

}  // namespace

int bgmf_balanced_cuts(int64_t n, int64_t m, int32_t p, const int32_t *rows, const int32_t *cols,
                       int64_t nnz, int64_t max_rows, int64_t max_cols, int64_t *row_cuts,
                       int64_t *col_cuts) {
  if (!rows || !cols || !row_cuts || !col_cuts || nnz < 0 || n < 1 || m < 1) {
    fail(nullptr, BGMF_E_ARG, "bgmf_balanced_cuts: bad arguments");
    return BGMF_E_ARG;
  }
  max_rows = std::min<int64_t>(max_rows, 65536);
  max_cols = std::min<int64_t>(max_cols, 1 << kColBits);
  std::vector<int64_t> rd((size_t)n, 0), cd((size_t)m, 0);
  for (int64_t e = 0; e < nnz; ++e) {
    if (rows[e] < 0 || rows[e] >= n || cols[e] < 0 || cols[e] >= m) {
      fail(nullptr, BGMF_E_RANGE, "rating %lld at (%d, %d) is outside the %lld x %lld matrix",
           (long long)e, rows[e], cols[e], (long long)n, (long long)m);
      return BGMF_E_RANGE;
    }
    rd[rows[e]] += 1;
    cd[cols[e]] += 1;
  }
  if (!balanced_dim(rd, p, max_rows, row_cuts) || !balanced_dim(cd, p, max_cols, col_cuts)) {
    fail(nullptr, BGMF_E_ARG,
         "no cut points: need 1 <= p <= min(n, m), p * max_rows >= n and p * max_cols >= m");
    return BGMF_E_ARG;
  }
  return BGMF_OK;
}

namespace {

// Degree-aware relabelling of one dimension over p equal blocks (Eq. 4's
// boundaries ceil(b len / p)): indices in descending degree (ties by
// ascending index) are dealt one by one to the block with the smallest load
// so far that still has a free place (ties by block number); inside a block
// the new ids follow the order of dealing.  Block widths stay those of the
// paper's grid, so only the ids change.  newid[old] receives the new id.
void relabel_dim(const std::vector<int64_t> &deg, int32_t p, int32_t *newid) {
  const int64_t len = (int64_t)deg.size();
  std::vector<int64_t> order((size_t)len);
  for (int64_t i = 0; i < len; ++i) order[i] = i;
  std::stable_sort(order.begin(), order.end(),
                   [&](int64_t a, int64_t b) { return deg[a] > deg[b]; });
  std::vector<int64_t> next((size_t)p), end((size_t)p);
  for (int32_t b = 0; b < p; ++b) {
    next[b] = equal_cut(b, len, p);
    end[b] = equal_cut(b + 1, len, p);
  }
  // min-heap of (load, block) over blocks with a free place
  using Entry = std::pair<int64_t, int32_t>;
  std::vector<Entry> heap;
  heap.reserve((size_t)p);
  for (int32_t b = 0; b < p; ++b)
    if (next[b] < end[b]) heap.emplace_back(0, b);
  auto later = [](const Entry &x, const Entry &y) { return x > y; };
  std::make_heap(heap.begin(), heap.end(), later);
  for (int64_t i : order) {
    std::pop_heap(heap.begin(), heap.end(), later);
    Entry e = heap.back();
    heap.pop_back();
    newid[i] = (int32_t)next[e.second]++;
    if (next[e.second] < end[e.second]) {
      heap.emplace_back(e.first + deg[i], e.second);
      std::push_heap(heap.begin(), heap.end(), later);
    }
  }
}

}  // namespace

int bgmf_reorder_ids(int64_t n, int64_t m, int32_t p, const int32_t *rows, const int32_t *cols,
                     int64_t nnz, int32_t *row_newid, int32_t *col_newid) {
  if (!rows || !cols || !row_newid || !col_newid || nnz < 0 || n < 1 || m < 1 ||
      n >= (1ll << 31) || m >= (1ll << 31)) {
    fail(nullptr, BGMF_E_ARG, "bgmf_reorder_ids: bad arguments");
    return BGMF_E_ARG;
  }
  if (p < 1 || p > n || p > m) {
    fail(nullptr, BGMF_E_ARG, "bgmf_reorder_ids: p must be in [1, min(n, m)]: p=%d", p);
    return BGMF_E_ARG;
  }
  std::vector<int64_t> rd((size_t)n, 0), cd((size_t)m, 0);
  for (int64_t e = 0; e < nnz; ++e) {
    if (rows[e] < 0 || rows[e] >= n || cols[e] < 0 || cols[e] >= m) {
      fail(nullptr, BGMF_E_RANGE, "rating %lld at (%d, %d) is outside the %lld x %lld matrix",
           (long long)e, rows[e], cols[e], (long long)n, (long long)m);
      return BGMF_E_RANGE;
    }
    rd[rows[e]] += 1;
    cd[cols[e]] += 1;
  }
  relabel_dim(rd, p, row_newid);
  relabel_dim(cd, p, col_newid);
  return BGMF_OK;
}

int bgmf_set_cuts(bgmf_t *h, const int64_t *row_cuts, const int64_t *col_cuts) {
  if (!h) return BGMF_E_ARG;
  if (!row_cuts || !col_cuts) return fail(h, BGMF_E_ARG, "bgmf_set_cuts: null pointer");
  const int64_t rmax = check_cuts(row_cuts, h->p, h->n, 65536);
  const int64_t cmax = check_cuts(col_cuts, h->p, h->m, 1 << kColBits);
  if (rmax < 0 || cmax < 0)
    return fail(h, BGMF_E_ARG,
                "cut points must rise strictly from 0 to n (rows, blocks at most 65536 wide) and "
                "from 0 to m (columns, blocks at most %d wide)",
                1 << kColBits);
  HIP_TRY(h, hipStreamSynchronize(h->stream));
  free_layout(h);
  h->rcut.assign(row_cuts, row_cuts + h->p + 1);
  h->ccut.assign(col_cuts, col_cuts + h->p + 1);
  h->rows_max = rmax;
  h->cols_max = (int)cmax;
  HIP_TRY(h, configure_sweep(h));
  HIP_TRY(h, hipMemcpy(h->d_cuts, h->rcut.data(), ((size_t)h->p + 1) * sizeof(int64_t),
                       hipMemcpyHostToDevice));
  HIP_TRY(h, hipMemcpy(h->d_cuts + h->p + 1, h->ccut.data(), ((size_t)h->p + 1) * sizeof(int64_t),
                       hipMemcpyHostToDevice));
  return BGMF_OK;
}

int bgmf_get_cuts(const bgmf_t *h, int64_t *row_cuts, int64_t *col_cuts) {
  if (!h) return BGMF_E_ARG;
  if (row_cuts) std::memcpy(row_cuts, h->rcut.data(), ((size_t)h->p + 1) * sizeof(int64_t));
  if (col_cuts) std::memcpy(col_cuts, h->ccut.data(), ((size_t)h->p + 1) * sizeof(int64_t));
  return BGMF_OK;
}

int bgmf_rmse_coo(bgmf_t *h, const int32_t *rows, const int32_t *cols, const float *vals,
                  int64_t nnz, double *out) {
  if (!h) return BGMF_E_ARG;
  if (!rows || !cols || !vals || !out) return fail(h, BGMF_E_ARG, "bgmf_rmse_coo: null pointer");
  if (nnz < 1 || nnz >= (1ll << 31))
    return fail(h, BGMF_E_ARG, "nnz must be in [1, 2^31): %lld", (long long)nnz);
  if (!h->factors_set) return fail(h, BGMF_E_STATE, "bgmf_rmse_coo: factors not set");
  for (int64_t e = 0; e < nnz; ++e) {
    if (rows[e] < 0 || rows[e] >= h->n || cols[e] < 0 || cols[e] >= h->m)
      return fail(h, BGMF_E_RANGE, "rating %lld at (%d, %d) is outside the %lld x %lld matrix",
                  (long long)e, rows[e], cols[e], (long long)h->n, (long long)h->m);
    if (!std::isfinite(vals[e]))
      return fail(h, BGMF_E_NONFINITE, "rating %lld has a non-finite value", (long long)e);
  }
  int32_t *d_rows = nullptr, *d_cols = nullptr;
  float *d_vals = nullptr;
  double *d_part = nullptr;
  auto cleanup = [&]() {
    hipFree(d_rows);
    hipFree(d_cols);
    hipFree(d_vals);
    hipFree(d_part);
  };
  double r = 0.0;
  hipError_t e = hipSuccess;
  const size_t np = rmse_coo_partials_count();
  if ((e = dev_alloc(h, reinterpret_cast<void **>(&d_rows), (size_t)nnz * sizeof(int32_t))) ==
          hipSuccess &&
      (e = dev_alloc(h, reinterpret_cast<void **>(&d_cols), (size_t)nnz * sizeof(int32_t))) ==
          hipSuccess &&
      (e = dev_alloc(h, reinterpret_cast<void **>(&d_vals), (size_t)nnz * sizeof(float))) ==
          hipSuccess &&
      (e = dev_alloc(h, reinterpret_cast<void **>(&d_part), (np + 2) * sizeof(double))) ==
          hipSuccess &&
      (e = hipMemcpyAsync(d_rows, rows, (size_t)nnz * sizeof(int32_t), hipMemcpyHostToDevice,
                          h->stream)) == hipSuccess &&
      (e = hipMemcpyAsync(d_cols, cols, (size_t)nnz * sizeof(int32_t), hipMemcpyHostToDevice,
                          h->stream)) == hipSuccess &&
      (e = hipMemcpyAsync(d_vals, vals, (size_t)nnz * sizeof(float), hipMemcpyHostToDevice,
                          h->stream)) == hipSuccess &&
      (e = launch_rmse_coo(d_rows, d_cols, d_vals, nnz, h->U, h->V, h->k, h->n, h->m, d_part,
                           d_part + np, reinterpret_cast<int32_t *>(d_part + np + 1),
                           h->stream)) == hipSuccess &&
      (e = hipMemcpyAsync(&r, d_part + np, sizeof r, hipMemcpyDeviceToHost, h->stream)) ==
          hipSuccess)
    e = hipStreamSynchronize(h->stream);
  cleanup();
  if (e != hipSuccess)
    return fail(h, e == hipErrorOutOfMemory ? BGMF_E_NOMEM : BGMF_E_HIP, "bgmf_rmse_coo: %s",
                hipGetErrorString(e));
  int rc = check_device_error(h);
  if (rc != BGMF_OK) return rc;
  *out = r;
  return BGMF_OK;
}

int bgmf_fit(bgmf_t *h, float alpha, float beta, int32_t max_epochs, double delta,
             int32_t *epochs_run, double *rmse_history) {
  if (!h) return BGMF_E_ARG;
  const Range range("bgmf_fit");
  if (!epochs_run) return fail(h, BGMF_E_ARG, "bgmf_fit: null epochs_run");
  if (max_epochs < 1) return fail(h, BGMF_E_ARG, "max_epochs must be >= 1");
  if (!std::isfinite(delta) || delta < 0.0) return fail(h, BGMF_E_ARG, "delta must be finite and >= 0");
  *epochs_run = 0;
  double prev = 0.0;
  int rc = bgmf_rmse(h, &prev);
  if (rc != BGMF_OK) return rc;
  if (rmse_history) rmse_history[0] = prev;
  for (int32_t e = 1; e <= max_epochs; ++e) {
    rc = bgmf_epoch(h, alpha, beta);
    if (rc != BGMF_OK) return rc;
    double r = 0.0;
    rc = bgmf_rmse(h, &r);
    if (rc != BGMF_OK) return rc;
    *epochs_run = e;
    if (rmse_history) rmse_history[e] = r;
    if (!std::isfinite(r))
      return fail(h, BGMF_E_NONFINITE,
                  "the RMSE is not finite after epoch %d: the step alpha = %g diverges on these "
                  "ratings",
                  e, (double)alpha);
    if (std::fabs(prev - r) < delta) break;
    prev = r;
  }
  return BGMF_OK;
}

int bgmf_get_factors(bgmf_t *h, float *U, float *V) {
  if (!h) return BGMF_E_ARG;
  const Range range("bgmf_get_factors");
  if (U)
    HIP_TRY(h, hipMemcpyAsync(U, h->U, (size_t)h->n * h->k * sizeof(float), hipMemcpyDeviceToHost,
                              h->stream));
  if (V)
    HIP_TRY(h, hipMemcpyAsync(V, h->V, (size_t)h->m * h->k * sizeof(float), hipMemcpyDeviceToHost,
                              h->stream));
  return sync_checked(h);
}

int bgmf_get_layout(bgmf_t *h, int64_t *block_ptr, int32_t *perm) {
  if (!h) return BGMF_E_ARG;
  if (!h->loaded) return fail(h, BGMF_E_STATE, "bgmf_get_layout: no ratings loaded");
  if (block_ptr)
    HIP_TRY(h, hipMemcpyAsync(block_ptr, h->block_ptr,
                              (size_t)((int64_t)h->p * h->p + 1) * sizeof(int64_t),
                              hipMemcpyDeviceToHost, h->stream));
  if (perm && h->ooc)
    std::memcpy(perm, h->host_perm, (size_t)h->nnz * sizeof(int32_t));
  else if (perm)
    HIP_TRY(h, hipMemcpyAsync(perm, h->perm, (size_t)h->nnz * sizeof(int32_t),
                              hipMemcpyDeviceToHost, h->stream));
  return sync_checked(h);
}

int bgmf_sync(bgmf_t *h) {
  if (!h) return BGMF_E_ARG;
  return sync_checked(h);
}

int bgmf_factor_ptrs(bgmf_t *h, float **U_dev, float **V_dev) {
  if (!h) return BGMF_E_ARG;
  if (U_dev) *U_dev = h->U;
  if (V_dev) *V_dev = h->V;
  return BGMF_OK;
}

int bgmf_set_option(bgmf_t *h, int32_t option, int64_t value) {
  if (!h) return BGMF_E_ARG;
  switch (option) {
    case BGMF_OPT_SCHEDULE:
      if (value < 0 || value > 2) return fail(h, BGMF_E_ARG, "schedule must be 0, 1 or 2");
      h->schedule = value;
      return BGMF_OK;
    case BGMF_OPT_WAIT_LIMIT_US:
      if (value < 0) return fail(h, BGMF_E_ARG, "wait limit must be >= 0");
      h->wait_us = value;
      return BGMF_OK;
    case BGMF_OPT_XCD_REMAP:
      if (value != 0 && value != 1) return fail(h, BGMF_E_ARG, "xcd remap must be 0 or 1");
      h->xcd_remap = value;
      return BGMF_OK;
    case BGMF_OPT_RATINGS_BUDGET:
      if (value < 0) return fail(h, BGMF_E_ARG, "ratings budget must be >= 0");
      h->budget = value;
      return BGMF_OK;
    case BGMF_OPT_STREAM_SLOTS:
      return fail(h, BGMF_E_ARG, "BGMF_OPT_STREAM_SLOTS is read-only");
    case BGMF_OPT_V_STAGING:
      if (value < 0 || value > 2) return fail(h, BGMF_E_ARG, "V staging must be 0, 1 or 2");
      if (value == 1 && !h->lds_fits)
        return fail(h, BGMF_E_UNSUPPORTED,
                    "a column slice of %d x %d floats does not fit in LDS", h->cols_max + 1,
                    h->kp);
      h->v_staging = value;
      return BGMF_OK;
    case BGMF_OPT_PLACEMENT:
      return fail(h, BGMF_E_ARG, "BGMF_OPT_PLACEMENT is read-only");
    case BGMF_OPT_BLOCK_PASSES:
      if (value < 1 || value > 1024) return fail(h, BGMF_E_ARG, "block passes must be in [1, 1024]");
      h->passes = value;
      return BGMF_OK;
    case BGMF_OPT_SINGLE_COLUMN:
      if (value != 0 && value != 1) return fail(h, BGMF_E_ARG, "single column must be 0 or 1");
      h->single_col = value;
      return BGMF_OK;
    case BGMF_OPT_LDS_HANDOVER:
      if (value != 0 && value != 1) return fail(h, BGMF_E_ARG, "LDS hand-over must be 0 or 1");
      h->lds_handover = value;
      HIP_TRY(h, configure_sweep(h));
      return BGMF_OK;
    case BGMF_OPT_STREAM_CHUNKS:
      return fail(h, BGMF_E_ARG, "BGMF_OPT_STREAM_CHUNKS is read-only");
    case BGMF_OPT_RESIDENT_STRATA:
      return fail(h, BGMF_E_ARG, "BGMF_OPT_RESIDENT_STRATA is read-only");
    case BGMF_OPT_ALLOC_COUNT:
      return fail(h, BGMF_E_ARG, "BGMF_OPT_ALLOC_COUNT is read-only");
    case BGMF_OPT_LOAD_PEAK:
      return fail(h, BGMF_E_ARG, "BGMF_OPT_LOAD_PEAK is read-only");
    case BGMF_OPT_LOAD_GROUPS:
      return fail(h, BGMF_E_ARG, "BGMF_OPT_LOAD_GROUPS is read-only");
    case BGMF_OPT_TRACE:
      if (value != 0 && value != 1) return fail(h, BGMF_E_ARG, "trace must be 0 or 1");
      if (value == 1 && !h->d_trace) {
        HIP_TRY(h, hipStreamSynchronize(h->stream));
        HIP_TRY(h, dev_alloc(h, reinterpret_cast<void **>(&h->d_trace),
                             2 * (size_t)h->p * h->p * sizeof(int64_t)));
      } else if (value == 0 && h->d_trace) {
        HIP_TRY(h, hipStreamSynchronize(h->stream));
        HIP_TRY(h, hipFree(h->d_trace));
        h->d_trace = nullptr;
      }
      h->trace_valid = false;
      return BGMF_OK;
    default:
      return fail(h, BGMF_E_ARG, "unknown option %d", option);
  }
}

int bgmf_get_option(const bgmf_t *h, int32_t option, int64_t *value) {
  if (!h || !value) return BGMF_E_ARG;
  switch (option) {
    case BGMF_OPT_SCHEDULE: *value = h->schedule; return BGMF_OK;
    case BGMF_OPT_WAIT_LIMIT_US: *value = h->wait_us; return BGMF_OK;
    case BGMF_OPT_XCD_REMAP: *value = h->xcd_remap; return BGMF_OK;
    case BGMF_OPT_RATINGS_BUDGET: *value = h->budget; return BGMF_OK;
    case BGMF_OPT_STREAM_SLOTS: *value = h->ooc ? h->nslots : 0; return BGMF_OK;
    case BGMF_OPT_V_STAGING: *value = h->v_staging; return BGMF_OK;
    case BGMF_OPT_STREAM_CHUNKS:
      *value = h->ooc ? (int64_t)h->chunk.size() - 1 : 0;
      return BGMF_OK;
    case BGMF_OPT_RESIDENT_STRATA: *value = h->ooc ? h->s_res : h->p; return BGMF_OK;
    case BGMF_OPT_BLOCK_PASSES: *value = h->passes; return BGMF_OK;
    case BGMF_OPT_SINGLE_COLUMN: *value = h->single_col; return BGMF_OK;
    case BGMF_OPT_LDS_HANDOVER: *value = h->lds_handover; return BGMF_OK;
    case BGMF_OPT_TRACE: *value = h->d_trace ? 1 : 0; return BGMF_OK;
    case BGMF_OPT_ALLOC_COUNT: *value = h->alloc_calls; return BGMF_OK;
    case BGMF_OPT_LOAD_PEAK: *value = h->load_peak; return BGMF_OK;
    case BGMF_OPT_LOAD_GROUPS: *value = h->load_groups; return BGMF_OK;
    case BGMF_OPT_PLACEMENT: {
      const SweepShape sh = sweep_shape(h);
      *value = (sh.lds ? 1 : 2) | (sh.persistent ? 4 : 0);
      return BGMF_OK;
    }
    default: return BGMF_E_ARG;
  }
}

int bgmf_get_timing(bgmf_t *h, double *epoch_ms, double *rmse_ms) {
  if (!h) return BGMF_E_ARG;
  int rc = sync_checked(h);
  if (rc != BGMF_OK) return rc;
  float ms = 0.0f;
  if (epoch_ms) {
    *epoch_ms = NAN;
    if (h->epoch_timed) {
      HIP_TRY(h, hipEventElapsedTime(&ms, h->ev[0], h->ev[1]));
      *epoch_ms = ms;
    }
  }
  if (rmse_ms) {
    *rmse_ms = NAN;
    if (h->rmse_timed) {
      HIP_TRY(h, hipEventElapsedTime(&ms, h->ev[2], h->ev[3]));
      *rmse_ms = ms;
    }
  }
  return BGMF_OK;
}

int bgmf_get_trace(bgmf_t *h, int64_t *begin, int64_t *end, int64_t *ticks_per_s) {
  if (!h) return BGMF_E_ARG;
  if (!begin || !end || !ticks_per_s) return fail(h, BGMF_E_ARG, "bgmf_get_trace: null pointer");
  if (!h->trace_valid)
    return fail(h, BGMF_E_STATE, "bgmf_get_trace: no epoch traced since BGMF_OPT_TRACE was set");
  int rc = sync_checked(h);
  if (rc != BGMF_OK) return rc;
  const size_t q = (size_t)h->p * h->p;
  std::vector<int64_t> t(2 * q);
  HIP_TRY(h, hipMemcpy(t.data(), h->d_trace, t.size() * sizeof(int64_t), hipMemcpyDeviceToHost));
  for (size_t i = 0; i < q; ++i) {
    begin[i] = t[2 * i];
    end[i] = t[2 * i + 1];
  }
  *ticks_per_s = h->clock_khz * 1000;
  return BGMF_OK;
}

int bgmf_chain_stats(bgmf_t *h, int64_t out[4]) {
  if (!h || !out) return BGMF_E_ARG;
  if (!h->loaded) return fail(h, BGMF_E_STATE, "bgmf_chain_stats: no ratings loaded");
  for (int i = 0; i < 4; ++i) out[i] = h->chain[i];
  return BGMF_OK;
}

}  // extern "C"
