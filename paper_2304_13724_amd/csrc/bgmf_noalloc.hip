// bgmf_rmse_coo_dev: the RMSE of bgmf_rmse_coo over ratings the caller
// already holds in device memory, without allocating anything.  The
// reduction's partial sums, its result and the error word live in a
// file-scope device array (one copy per GPU, for the life of the process)
// instead of memory allocated per call.
#include <hip/hip_runtime.h>

#include <cmath>
#include <cstdio>
#include <mutex>

#include "bgmf_handle.h"

using namespace bgmfk;

namespace {

// Layout of the scratch array: the partial sums of the COO RMSE kernel's
// fixed grid (rmse_coo_partials_count() doubles), the result (one double),
// and the error word (int32, in its own 8-byte slot).
constexpr size_t kPartials = (size_t)kRmseCooGroups * kWavesPerGroup;
constexpr size_t kScratchBytes = (kPartials + 2) * sizeof(double);

static __device__ __align__(256) unsigned char scratch[kScratchBytes];

// Device address of `scratch` on each device.  In host code the array's name
// is only a host-side stand-in; the address the kernels need comes from
// hipGetSymbolAddress, taken once per device with that device current.
constexpr int kMaxDevices = 64;
std::mutex g_mu;
void *g_scratch[kMaxDevices] = {};

int report(bgmf_t *h, int code, const char *msg) {
  h->msg = msg;
  return code;
}

}  // namespace

extern "C" int bgmf_rmse_coo_dev(bgmf_t *h, const int32_t *rows_dev, const int32_t *cols_dev,
                                 const float *vals_dev, int64_t nnz, double *out) {
  if (!h) return BGMF_E_ARG;
  if (!rows_dev || !cols_dev || !vals_dev || !out)
    return report(h, BGMF_E_ARG, "bgmf_rmse_coo_dev: null pointer");
  if (nnz < 1 || nnz >= (1ll << 31))
    return report(h, BGMF_E_ARG, "bgmf_rmse_coo_dev: nnz must be in [1, 2^31)");
  if (!h->factors_set) return report(h, BGMF_E_STATE, "bgmf_rmse_coo_dev: factors not set");
  static_assert(kPartials == (size_t)kRmseCooGroups * kWavesPerGroup, "scratch layout");
  if (rmse_coo_partials_count() != kPartials)
    return report(h, BGMF_E_UNSUPPORTED, "bgmf_rmse_coo_dev: reduction larger than its scratch");
  if (h->device < 0 || h->device >= kMaxDevices)
    return report(h, BGMF_E_UNSUPPORTED, "bgmf_rmse_coo_dev: device index beyond 63");
  void *base = nullptr;
  {
    std::lock_guard<std::mutex> lock(g_mu);
    if (!g_scratch[h->device]) {
      int cur = 0;
      hipError_t e = hipGetDevice(&cur);
      if (e == hipSuccess && cur != h->device) e = hipSetDevice(h->device);
      void *ptr = nullptr;
      if (e == hipSuccess) e = hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch));
      if (cur != h->device) hipSetDevice(cur);
      if (e != hipSuccess || !ptr) {
        char buf[256];
        snprintf(buf, sizeof buf, "bgmf_rmse_coo_dev: hipGetSymbolAddress: %s",
                 hipGetErrorString(e));
        return report(h, BGMF_E_HIP, buf);
      }
      g_scratch[h->device] = ptr;
    }
    base = g_scratch[h->device];
  }
  double *partials = static_cast<double *>(base);
  double *result = partials + kPartials;
  int32_t *bad = reinterpret_cast<int32_t *>(result + 1);
  // the error word is cleared by a kernel inside launch_rmse_coo; the
  // partials and the result are written in full by every call
  hipError_t e = launch_rmse_coo(rows_dev, cols_dev, vals_dev, nnz, h->U, h->V, h->k, h->n, h->m,
                                 partials, result, bad, h->stream);
  double r = 0.0;
  int32_t flags = 0;
  if (e == hipSuccess) e = hipMemcpyAsync(&r, result, sizeof r, hipMemcpyDeviceToHost, h->stream);
  if (e == hipSuccess)
    e = hipMemcpyAsync(&flags, bad, sizeof flags, hipMemcpyDeviceToHost, h->stream);
  if (e == hipSuccess) e = hipStreamSynchronize(h->stream);
  if (e != hipSuccess) {
    char buf[256];
    snprintf(buf, sizeof buf, "bgmf_rmse_coo_dev: %s", hipGetErrorString(e));
    return report(h, BGMF_E_HIP, buf);
  }
  if (flags & 1)
    return report(h, BGMF_E_RANGE, "bgmf_rmse_coo_dev: a rating lies outside the matrix");
  if (flags & 2)
    return report(h, BGMF_E_NONFINITE, "bgmf_rmse_coo_dev: a rating value is not finite");
  *out = r;
  return BGMF_OK;
}
