// Optional per-kernel timing: when enabled, every kernel launch of the
// library is bracketed by two HIP events recorded on the launch stream.  The
// host reads the elapsed times later (moe_trace_read), after the events
// completed; nothing here synchronises at launch time.
#pragma once

#include <hip/hip_runtime.h>

namespace moe {

enum KernelId {
  K_ROUTER_LOGITS,
  K_TOPK,
  K_PERM_SCATTER,
  K_PERMUTE_ROWS,
  K_GATEUP_FWD,
  K_DOWN_FWD,
  K_COMBINE,
  K_COMBINE_BWD,
  K_DOWN_DGRAD,
  K_DOWN_WGRAD,
  K_GATEUP_DGRAD,
  K_GATEUP_WGRAD,
  K_DWR_PARTIAL,
  K_DWR_REDUCE,
  K_ROUTER_DX,
  K_OFFSETS,
  K_GATEUP_RECOMPUTE,
  K_ROUTER_LOSS,
  K_ROUTER_DX_DENSE,
  K_LORA_ROWS,
  K_LORA_WGRAD,
  K_GATE_BWD,
  K_WGRAD_PLAN,
  K_NUM_KERNELS
};

extern bool g_trace_on;
void trace_record(int id, bool end, hipStream_t s);

struct TraceScope {
  int id;
  hipStream_t s;
  TraceScope(int id_, hipStream_t s_) : id(id_), s(s_) {
    if (g_trace_on) trace_record(id, false, s);
  }
  ~TraceScope() {
    if (g_trace_on) trace_record(id, true, s);
  }
};

}  // namespace moe
