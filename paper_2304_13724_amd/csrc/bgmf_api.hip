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

#include "../../include/bgmf.h"
#include "bgmf_internal.h"

using namespace bgmfk;

struct bgmf {
  int64_t n = 0, m = 0;
  int32_t k = 0, p = 0, kp = 0;
  int device = 0;
  int cus = 0;
  hipStream_t own_stream = nullptr;
  hipStream_t stream = nullptr;
  float *U = nullptr, *V = nullptr;
  // ratings layout
  int64_t nnz = 0;
  int64_t *block_ptr = nullptr, *wblock_ptr = nullptr;
  uint8_t *rowrep = nullptr;  // [p*p] per block slot: a row repeats in consecutive ratings
  int32_t *perm = nullptr;
  uint2 *rec = nullptr;
  int64_t *flags = nullptr;
  int32_t *err = nullptr;
  double *partials = nullptr, *d_rmse = nullptr;
  int64_t epochs_done = 0;
  bool factors_set = false, loaded = false;
  // block cut points (host copies and device tables, p + 1 each)
  std::vector<int64_t> rcut, ccut;
  int64_t *d_cuts = nullptr;  // rcut then ccut
  int64_t rows_max = 0;
  // launch shapes: V slice staged in LDS (when it fits) and V in global memory
  int cols_max = 0;
  size_t lds_limit = 0;
  bool lds_fits = false;
  int wpg_lds = 1, wpg_gv = kWavesPerGroup;
  int lds_ring = 0;  // areas of the LDS hand-over ring (0: none)
  size_t lds_bytes_lds = 0, lds_bytes_gv = 0;
  bool coop_lds = false, coop_gv = false;
  // options
  int64_t schedule = 0, wait_us = 10000000, xcd_remap = 1, v_staging = 0, passes = 1;
  int64_t single_col = 1, lds_handover = 1;
  // block trace: [2 p p] clock values of the last epoch (see bgmf_get_trace)
  int64_t *d_trace = nullptr;
  bool trace_valid = false;
  // timing
  hipEvent_t ev[4] = {nullptr, nullptr, nullptr, nullptr};
  bool epoch_timed = false, rmse_timed = false;
  int64_t chain[4] = {0, 0, 0, 0};
  std::string msg;
  // out-of-core: records in pinned host memory, streamed per stratum
  int64_t budget = 0;            // device bytes for ratings (0: no limit)
  bool ooc = false;
  uint2 *host_rec = nullptr;     // stratum-major records (pinned)
  int32_t *host_perm = nullptr;  // slot-order input positions (pinned)
  uint2 *resident = nullptr;     // strata [0, s_res), copied once per load
  int32_t s_res = 0;
  uint2 *ring = nullptr;         // device slots of slot_recs records each
  int nslots = 0;
  int64_t slot_recs = 0;
  std::vector<int64_t> strat;    // p + 1 record offsets of the strata
  std::vector<int32_t> chunk;    // chunk c = strata [chunk[c], chunk[c + 1]), one slot each
  size_t issued = 0;             // chunks whose copy has been queued in the current pass
  hipStream_t side = nullptr;    // copies into the ring
  std::vector<hipEvent_t> ready, freed;
  std::vector<bool> slot_used;
};

namespace {

thread_local std::string g_create_error;

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
  hipFree(h->block_ptr);
  hipFree(h->wblock_ptr);
  hipFree(h->rowrep);
  hipFree(h->perm);
  hipFree(h->rec);
  hipFree(h->ring);
  hipFree(h->resident);
  if (h->host_rec) hipHostFree(h->host_rec);
  if (h->host_perm) hipHostFree(h->host_perm);
  for (auto ev : h->ready) hipEventDestroy(ev);
  for (auto ev : h->freed) hipEventDestroy(ev);
  h->ready.clear();
  h->freed.clear();
  h->slot_used.clear();
  h->chunk.clear();
  h->block_ptr = h->wblock_ptr = nullptr;
  h->rowrep = nullptr;
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
  if ((e = configure_sweep(h)) != hipSuccess) return bail(e, "configure_sweep");
  if ((e = hipMalloc(&h->d_cuts, 2 * ((size_t)p + 1) * sizeof(int64_t))) != hipSuccess)
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
  // one spare row after U absorbs the padding steps of the sweep
  if ((e = hipMalloc(&h->U, (size_t)(n + 1) * k * sizeof(float))) != hipSuccess)
    return bail(e, "hipMalloc(U)");
  if ((e = hipMalloc(&h->V, (size_t)m * k * sizeof(float))) != hipSuccess)
    return bail(e, "hipMalloc(V)");
  if ((e = hipMalloc(&h->flags, (size_t)p * kFlagStride * sizeof(int64_t))) != hipSuccess)
    return bail(e, "hipMalloc(flags)");
  if ((e = hipMalloc(&h->err, sizeof(int32_t))) != hipSuccess) return bail(e, "hipMalloc(err)");
  if ((e = hipMalloc(&h->partials, rmse_partials_count(p) * sizeof(double))) != hipSuccess)
    return bail(e, "hipMalloc(partials)");
  if ((e = hipMalloc(&h->d_rmse, sizeof(double))) != hipSuccess)
    return bail(e, "hipMalloc(rmse)");
  if ((e = hipMemset(h->flags, 0, (size_t)p * kFlagStride * sizeof(int64_t))) != hipSuccess)
    return bail(e, "hipMemset");
  if ((e = hipMemset(h->err, 0, sizeof(int32_t))) != hipSuccess) return bail(e, "hipMemset");
  if ((e = hipMemset(h->U, 0, (size_t)(n + 1) * k * sizeof(float))) != hipSuccess)
    return bail(e, "hipMemset");
  if ((e = hipMemset(h->V, 0, (size_t)m * k * sizeof(float))) != hipSuccess)
    return bail(e, "hipMemset");
  return h;
}

void bgmf_destroy(bgmf_t *h) {
  if (!h) return;
  if (h->stream) hipStreamSynchronize(h->stream);
  free_layout(h);
  hipFree(h->U);
  hipFree(h->V);
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

int bgmf_set_factors(bgmf_t *h, const float *U, const float *V) {
  if (!h) return BGMF_E_ARG;
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

  const int64_t slots = (int64_t)h->p * h->p;
  int32_t *d_rows = nullptr, *d_cols = nullptr;
  float *d_vals = nullptr;
  void *scratch = nullptr;
  const size_t scratch_bytes = bucket_scratch_bytes(nnz, h->p);
  int rc = BGMF_OK;
  auto cleanup = [&]() {
    hipFree(d_rows);
    hipFree(d_cols);
    hipFree(d_vals);
    hipFree(scratch);
  };
#define LOAD_TRY(call)                                                                     \
  do {                                                                                     \
    hipError_t e_ = (call);                                                                \
    if (e_ != hipSuccess) {                                                                \
      rc = fail(h, e_ == hipErrorOutOfMemory ? BGMF_E_NOMEM : BGMF_E_HIP, "%s: %s", #call, \
                hipGetErrorString(e_));                                                    \
      cleanup();                                                                           \
      free_layout(h);                                                                      \
      return rc;                                                                           \
    }                                                                                      \
  } while (0)
  LOAD_TRY(hipMalloc(&d_rows, (size_t)nnz * sizeof(int32_t)));
  LOAD_TRY(hipMalloc(&d_cols, (size_t)nnz * sizeof(int32_t)));
  LOAD_TRY(hipMalloc(&d_vals, (size_t)nnz * sizeof(float)));
  LOAD_TRY(hipMalloc(&scratch, scratch_bytes));
  LOAD_TRY(hipMalloc(&h->block_ptr, (size_t)(slots + 1) * sizeof(int64_t)));
  LOAD_TRY(hipMalloc(&h->wblock_ptr, (size_t)(slots + 1) * sizeof(int64_t)));
  LOAD_TRY(hipMalloc(&h->rowrep, (size_t)slots));
  LOAD_TRY(hipMalloc(&h->perm, (size_t)nnz * sizeof(int32_t)));
  LOAD_TRY(hipMalloc(&h->rec, (size_t)(nnz + kRecPad) * sizeof(uint2)));
  LOAD_TRY(hipMemcpyAsync(d_rows, rows, (size_t)nnz * sizeof(int32_t), hipMemcpyHostToDevice,
                          h->stream));
  LOAD_TRY(hipMemcpyAsync(d_cols, cols, (size_t)nnz * sizeof(int32_t), hipMemcpyHostToDevice,
                          h->stream));
  LOAD_TRY(hipMemcpyAsync(d_vals, vals, (size_t)nnz * sizeof(float), hipMemcpyHostToDevice,
                          h->stream));
  BucketOut out{h->block_ptr, h->wblock_ptr, h->perm, h->rec, h->rowrep};
  LOAD_TRY(hipMemsetAsync(h->err, 0, sizeof(int32_t), h->stream));
  LOAD_TRY(hipMemsetAsync(h->rowrep, 0, (size_t)slots, h->stream));
  // ratings that do not fit the budget are kept stratum-major, so that each
  // stratum is one contiguous range to stream
  const bool ooc = h->budget > 0 && (nnz + kRecPad) * (int64_t)sizeof(uint2) > h->budget;
  LOAD_TRY(bucket(d_rows, d_cols, d_vals, nnz, grid_of(h), h->rows_max, ooc, scratch,
                  scratch_bytes, out, h->err, h->stream));
  LOAD_TRY(hipStreamSynchronize(h->stream));
  cleanup();
#undef LOAD_TRY
  int32_t derr = 0;
  HIP_TRY(h, hipMemcpy(&derr, h->err, sizeof derr, hipMemcpyDeviceToHost));

  // serial-chain statistics from the block sizes
  std::vector<int64_t> bp((size_t)slots + 1), wbp((size_t)slots + 1);
  HIP_TRY(h, hipMemcpy(bp.data(), h->block_ptr, bp.size() * sizeof(int64_t),
                       hipMemcpyDeviceToHost));
  HIP_TRY(h, hipMemcpy(wbp.data(), h->wblock_ptr, wbp.size() * sizeof(int64_t),
                       hipMemcpyDeviceToHost));
  // the sweep trusts these offsets: check them before any epoch may run
  bool ok = derr == 0 && bp[0] == 0 && wbp[0] == 0 && bp[slots] == nnz && wbp[slots] == nnz;
  for (int64_t q = 0; ok && q < slots; ++q) ok = bp[q] <= bp[q + 1] && wbp[q] <= wbp[q + 1];
  for (int64_t b = 0; ok && b < h->p; ++b)
    for (int64_t s2 = 0; ok && s2 < h->p; ++s2)
      ok = wbp[b * h->p + s2 + 1] - wbp[b * h->p + s2] == bp[s2 * h->p + b + 1] - bp[s2 * h->p + b];
  if (!ok) {
    hipMemset(h->err, 0, sizeof(int32_t));
    free_layout(h);
    return fail(h, BGMF_E_HIP, "internal error: the device bucketing produced an inconsistent layout");
  }
  std::vector<int64_t> colsum(h->p, 0), rowsum(h->p, 0);
  int64_t barrier = 0, nonempty = 0;
  for (int64_t s = 0; s < h->p; ++s) {
    int64_t mx = 0;
    for (int64_t R = 0; R < h->p; ++R) {
      const int64_t c = bp[s * h->p + R + 1] - bp[s * h->p + R];
      colsum[(R + s) % h->p] += c;
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

  if (ooc) {
    h->strat.assign((size_t)h->p + 1, 0);
    int64_t widest = 0;
    for (int64_t s2 = 0; s2 <= h->p; ++s2) h->strat[s2] = bp[s2 * h->p];
    for (int64_t s2 = 0; s2 < h->p; ++s2) widest = std::max(widest, h->strat[s2 + 1] - h->strat[s2]);
    // The budget is split into a ring of 3 (else 2) slots and a resident
    // region.  A slot holds the widest stratum plus the padding, and is made
    // a quarter of the budget when that fits: each chunk of strata in a slot
    // costs one copy and, with the persistent schedule, one launch, whose
    // end is a barrier across all row-blocks, so few large chunks are
    // better.  The resident region keeps the first strata of the epoch on
    // the device for good; the ring streams the others, and their first
    // copies run while the resident strata are swept.
    const int64_t need = widest + kRecPad;
    const int64_t budget_recs = h->budget / (int64_t)sizeof(uint2);
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
    if (h->nslots == 0) {
      const int64_t slot_bytes = need * (int64_t)sizeof(uint2);
      free_layout(h);
      return fail(h, BGMF_E_BUDGET,
                  "ratings budget of %lld bytes holds fewer than two strata (the widest stratum "
                  "needs %lld bytes)",
                  (long long)h->budget, (long long)slot_bytes);
    }
    const int64_t res_cap = budget_recs - (int64_t)h->nslots * h->slot_recs;
    h->s_res = 0;
    while (h->s_res < h->p && h->strat[h->s_res + 1] + kRecPad <= res_cap) ++h->s_res;
    // chunks of consecutive streamed strata, each as many as fit in a slot
    h->chunk.assign(1, h->s_res);
    for (int32_t s2 = h->s_res; s2 < h->p; ++s2)
      if (h->strat[s2 + 1] - h->strat[h->chunk.back()] + kRecPad > h->slot_recs)
        h->chunk.push_back(s2);
    if (h->chunk.back() != h->p) h->chunk.push_back(h->p);
    const int64_t slot_bytes = h->slot_recs * (int64_t)sizeof(uint2);
    if (!h->side) HIP_TRY(h, hipStreamCreateWithFlags(&h->side, hipStreamNonBlocking));
    HIP_TRY(h, hipHostMalloc(reinterpret_cast<void **>(&h->host_rec),
                             (size_t)nnz * sizeof(uint2), hipHostMallocDefault));
    HIP_TRY(h, hipHostMalloc(reinterpret_cast<void **>(&h->host_perm),
                             (size_t)nnz * sizeof(int32_t), hipHostMallocDefault));
    HIP_TRY(h, hipMemcpy(h->host_rec, h->rec, (size_t)nnz * sizeof(uint2), hipMemcpyDeviceToHost));
    HIP_TRY(h, hipMemcpy(h->host_perm, h->perm, (size_t)nnz * sizeof(int32_t),
                         hipMemcpyDeviceToHost));
    hipFree(h->rec);
    hipFree(h->perm);
    h->rec = nullptr;
    h->perm = nullptr;
    if (h->s_res > 0) {
      const int64_t count = h->strat[h->s_res];
      HIP_TRY(h, hipMalloc(&h->resident, (size_t)(count + kRecPad) * sizeof(uint2)));
      HIP_TRY(h, hipMemcpy(h->resident, h->host_rec, (size_t)count * sizeof(uint2),
                           hipMemcpyHostToDevice));
      HIP_TRY(h, hipMemset(h->resident + count, 0, (size_t)kRecPad * sizeof(uint2)));
    }
    HIP_TRY(h, hipMalloc(&h->ring, (size_t)h->nslots * (size_t)slot_bytes));
    HIP_TRY(h, hipMemset(h->ring, 0, (size_t)h->nslots * (size_t)slot_bytes));
    h->ready.assign(h->nslots, nullptr);
    h->freed.assign(h->nslots, nullptr);
    h->slot_used.assign(h->nslots, false);
    for (int i = 0; i < h->nslots; ++i) {
      HIP_TRY(h, hipEventCreateWithFlags(&h->ready[i], hipEventDisableTiming));
      HIP_TRY(h, hipEventCreateWithFlags(&h->freed[i], hipEventDisableTiming));
    }
    h->ooc = true;
  }

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
  P.wait_ticks = h->wait_us * 100;  // s_memrealtime runs at 100 MHz
  P.alpha = alpha;
  P.beta = beta;
  P.xcd_remap = (int32_t)h->xcd_remap;
  P.passes = (int32_t)h->passes;
  P.single_col = (int32_t)h->single_col;
  P.rowrep = h->rowrep;
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
  if ((e = hipMalloc(&d_rows, (size_t)nnz * sizeof(int32_t))) == hipSuccess &&
      (e = hipMalloc(&d_cols, (size_t)nnz * sizeof(int32_t))) == hipSuccess &&
      (e = hipMalloc(&d_vals, (size_t)nnz * sizeof(float))) == hipSuccess &&
      (e = hipMalloc(&d_part, (np + 1) * sizeof(double))) == hipSuccess &&
      (e = hipMemcpyAsync(d_rows, rows, (size_t)nnz * sizeof(int32_t), hipMemcpyHostToDevice,
                          h->stream)) == hipSuccess &&
      (e = hipMemcpyAsync(d_cols, cols, (size_t)nnz * sizeof(int32_t), hipMemcpyHostToDevice,
                          h->stream)) == hipSuccess &&
      (e = hipMemcpyAsync(d_vals, vals, (size_t)nnz * sizeof(float), hipMemcpyHostToDevice,
                          h->stream)) == hipSuccess &&
      (e = launch_rmse_coo(d_rows, d_cols, d_vals, nnz, h->U, h->V, h->k, d_part, d_part + np,
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
    case BGMF_OPT_TRACE:
      if (value != 0 && value != 1) return fail(h, BGMF_E_ARG, "trace must be 0 or 1");
      if (value == 1 && !h->d_trace) {
        HIP_TRY(h, hipStreamSynchronize(h->stream));
        HIP_TRY(h, hipMalloc(&h->d_trace, 2 * (size_t)h->p * h->p * sizeof(int64_t)));
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
  int khz = 0;
  HIP_TRY(h, hipDeviceGetAttribute(&khz, hipDeviceAttributeWallClockRate, h->device));
  *ticks_per_s = (int64_t)khz * 1000;
  return BGMF_OK;
}

int bgmf_chain_stats(bgmf_t *h, int64_t out[4]) {
  if (!h || !out) return BGMF_E_ARG;
  if (!h->loaded) return fail(h, BGMF_E_STATE, "bgmf_chain_stats: no ratings loaded");
  for (int i = 0; i < 4; ++i) out[i] = h->chain[i];
  return BGMF_OK;
}

}  // extern "C"
