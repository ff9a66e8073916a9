// Per-kernel event timing (see trace.hpp) and its C entry points.
#include "trace.hpp"

#include <vector>

#include "moe.h"

namespace moe {

bool g_trace_on = false;

namespace {

struct Pending {
  int id;
  hipEvent_t start, stop;
};

std::vector<hipEvent_t> g_pool;
std::vector<Pending> g_pending;
hipEvent_t g_open[K_NUM_KERNELS] = {};

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

const char* const kNames[K_NUM_KERNELS] = {
    "router_logits", "topk",         "perm_scatter", "permute_rows",
    "gateup_fwd",    "down_fwd",     "combine",       "combine_bwd",  "down_dgrad_swiglu",
    "down_wgrad",    "gateup_dgrad", "gateup_wgrad",  "dwr_partial",  "dwr_reduce",   "router_dx",
    "offsets_from_counts", "gateup_recompute", "router_loss", "router_dx_dense", "lora_rows", "lora_wgrad",
    "gate_bwd", "wgrad_plan"};

}  // namespace

void trace_record(int id, bool end, hipStream_t s) {
  if (!end) {
    hipEvent_t start = take_event();
    if (start && hipEventRecord(start, s) != hipSuccess) {
      g_pool.push_back(start);
      start = nullptr;
    }
    g_open[id] = start;
    return;
  }
  if (!g_open[id]) return;
  hipEvent_t stop = take_event();
  if (stop && hipEventRecord(stop, s) == hipSuccess) {
    g_pending.push_back({id, g_open[id], stop});
  } else {
    g_pool.push_back(g_open[id]);
    if (stop) g_pool.push_back(stop);
  }
  g_open[id] = nullptr;
}

}  // namespace moe

using namespace moe;

extern "C" {

int moe_trace_enable(int on) {
  g_trace_on = on != 0;
  return MOE_OK;
}

int moe_trace_read(double* total_ms, int32_t* launches, int n) {
  const int m = n < K_NUM_KERNELS ? n : K_NUM_KERNELS;
  for (int i = 0; i < m; ++i) {
    if (total_ms) total_ms[i] = 0.0;
    if (launches) launches[i] = 0;
  }
  int rc = MOE_OK;
  for (const Pending& p : g_pending) {
    float ms = 0.0f;
    if (hipEventSynchronize(p.stop) != hipSuccess || hipEventElapsedTime(&ms, p.start, p.stop) != hipSuccess)
      rc = MOE_ERR_HIP;
    if (p.id < m) {
      if (total_ms) total_ms[p.id] += ms;
      if (launches) launches[p.id] += 1;
    }
    g_pool.push_back(p.start);
    g_pool.push_back(p.stop);
  }
  g_pending.clear();
  return rc == MOE_OK ? K_NUM_KERNELS : rc;
}

const char* moe_trace_name(int id) {
  if (id < 0 || id >= K_NUM_KERNELS) return "";
  return kNames[id];
}

}  // extern "C"
