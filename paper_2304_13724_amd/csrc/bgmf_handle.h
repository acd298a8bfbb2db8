// The handle behind the opaque bgmf_t of include/bgmf.h, shared by the
// host sources of the library (not part of the ABI).
#pragma once

#include <hip/hip_runtime.h>

#include <string>
#include <vector>

#include "../../include/bgmf.h"
#include "bgmf_internal.h"

// fields of one handle (see include/bgmf.h for the calls that use them)
struct bgmf {
  int64_t n = 0, m = 0;
  int32_t k = 0, p = 0, kp = 0;
  int device = 0;
  int cus = 0;
  int64_t clock_khz = 100000;  // rate of the device's constant clock (s_memrealtime)
  hipStream_t own_stream = nullptr;
  hipStream_t stream = nullptr;
  float *U = nullptr, *V = nullptr;
  // ratings layout
  int64_t nnz = 0;
  int64_t *block_ptr = nullptr, *wblock_ptr = nullptr;
  uint8_t *nofold = nullptr;  // [p*p] per block slot: the folded one-column step does not apply
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
  int wpg_lds = 1, wpg_gv = bgmfk::kWavesPerGroup;
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
  // caller-owned memory (bgmf_bind): U, V, a device workspace for the
  // ratings and their tables, and a pinned host arena for streamed records
  bool bound = false;
  bool own_factors = true;       // U and V were allocated by the library
  char *ws = nullptr;
  size_t ws_bytes = 0;
  char *pinned = nullptr;
  size_t pinned_bytes = 0;
  // memory the library allocated for the current load (unbound handles)
  void *own_persist = nullptr;   // device: tables (and in-core records and perm)
  void *own_region = nullptr;    // device: streamed ratings (ring, resident strata, load temporaries)
  void *own_host = nullptr;      // pinned: streamed records and perm
  int64_t alloc_calls = 0;       // device and pinned allocations made by the library
  int64_t load_peak = 0;         // device bytes for ratings at the peak of the last load
  int64_t load_groups = 0;       // groups of blocks the last streamed load bucketed one by one
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
