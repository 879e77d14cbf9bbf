// timing.cpp - per-kernel launch timing with pooled HIP events (favor_timing_*).
#include <hip/hip_runtime.h>

#include <mutex>
#include <vector>

#include "../../include/favor.h"
#include "kernels.hpp"

namespace favor {
namespace {

struct Pending {
  int kernel;
  hipEvent_t begin, end;
};

std::mutex g_mu;
bool g_enabled = false;
std::vector<hipEvent_t> g_pool;
std::vector<Pending> g_pending;
double g_ms[kNumKernels] = {};
int64_t g_count[kNumKernels] = {};

const char *const kNames[kNumKernels] = {"k_orf_draw",   "k_feature_map", "k_kside",
                                         "k_finalize",   "k_qside",       "k_seg_scan",
                                         "k_causal",     "k_sum_splits",  "k_bwd_dq",
                                         "k_kside_agg",  "k_suffix_scan", "k_bwd_dkv"};

hipEvent_t take_event() {
  if (!g_pool.empty()) {
    hipEvent_t e = g_pool.back();
    g_pool.pop_back();
    return e;
  }
  hipEvent_t e = nullptr;
  if (hipEventCreate(&e) != hipSuccess) return nullptr;
  return e;
}

// Waits for every pending pair and folds it into the totals (lock held).
hipError_t drain() {
  hipError_t first = hipSuccess;
  for (const Pending &p : g_pending) {
    hipError_t e = hipEventSynchronize(p.end);
    float ms = 0.f;
    if (e == hipSuccess) e = hipEventElapsedTime(&ms, p.begin, p.end);
    if (e == hipSuccess) {
      g_ms[p.kernel] += ms;
      g_count[p.kernel] += 1;
    } else if (first == hipSuccess) {
      first = e;
    }
    g_pool.push_back(p.begin);
    g_pool.push_back(p.end);
  }
  g_pending.clear();
  return first;
}

}  // namespace

const char *kernel_name(int k) { return (k >= 0 && k < kNumKernels) ? kNames[k] : ""; }

LaunchTimer::LaunchTimer(int kernel, hipStream_t st) : kernel_(kernel), st_(st) {
  std::lock_guard<std::mutex> lk(g_mu);
  if (!g_enabled) return;
  begin_ = take_event();
  if (begin_ && hipEventRecord(begin_, st_) != hipSuccess) {
    g_pool.push_back(begin_);
    begin_ = nullptr;
  }
}

LaunchTimer::~LaunchTimer() {
  if (!begin_) return;
  std::lock_guard<std::mutex> lk(g_mu);
  hipEvent_t end = take_event();
  if (!end || hipEventRecord(end, st_) != hipSuccess) {
    g_pool.push_back(begin_);
    if (end) g_pool.push_back(end);
    return;
  }
  g_pending.push_back({kernel_, begin_, end});
}

}  // namespace favor

extern "C" {

favor_status favor_timing_enable(int on) {
  std::lock_guard<std::mutex> lk(favor::g_mu);
  favor::g_enabled = (on != 0);
  return FAVOR_OK;
}

favor_status favor_timing_reset(void) {
  std::lock_guard<std::mutex> lk(favor::g_mu);
  const hipError_t e = favor::drain();
  for (int k = 0; k < favor::kNumKernels; ++k) {
    favor::g_ms[k] = 0.0;
    favor::g_count[k] = 0;
  }
  return e == hipSuccess ? FAVOR_OK : FAVOR_ERR_DEVICE;
}

int32_t favor_timing_num_kernels(void) { return favor::kNumKernels; }

const char *favor_timing_kernel_name(int32_t k) { return favor::kernel_name(k); }

favor_status favor_timing_read(int32_t k, double *ms, int64_t *count) {
  if (k < 0 || k >= favor::kNumKernels || !ms || !count) return FAVOR_ERR_INVALID_ARGUMENT;
  std::lock_guard<std::mutex> lk(favor::g_mu);
  const hipError_t e = favor::drain();
  *ms = favor::g_ms[k];
  *count = favor::g_count[k];
  return e == hipSuccess ? FAVOR_OK : FAVOR_ERR_DEVICE;
}

}  // extern "C"
