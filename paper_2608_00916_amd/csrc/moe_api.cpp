// C ABI of the MoE block (declared in include/moe.h): argument checks,
// carving of the caller's `saved` and workspace buffers, and the launch
// sequence of the forward and backward passes on the caller's stream.
#include <hip/hip_runtime.h>

#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <cstring>
#include <initializer_list>
#include <utility>

#include "launch.hpp"
#include "moe.h"

using namespace moe;

namespace {

thread_local char g_err[512] = "";

int fail(int code, const char* fmt, ...) {
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(g_err, sizeof g_err, fmt, ap);
  va_end(ap);
  return code;
}

int ok() {
  g_err[0] = '\0';
  return MOE_OK;
}

constexpr size_t kAlign = 256;
size_t up(size_t n) { return (n + kAlign - 1) / kAlign * kAlign; }

// Sequential carve-up of a buffer into 256-byte aligned regions.
struct Carve {
  char* base;
  size_t off = 0;
  explicit Carve(void* b) : base(static_cast<char*>(b)) {}
  template <typename T>
  T* take(size_t count) {
    T* p = base ? reinterpret_cast<T*>(base + off) : nullptr;
    off += up(count * sizeof(T));
    return p;
  }
};

bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

int check_dims(const moe_dims* d) {
  if (d == nullptr) return fail(MOE_ERR_ARG, "dims is NULL");
  if (d->T < 1 || d->H < 1 || d->E < 1 || d->F < 1)
    return fail(MOE_ERR_ARG, "T, H, E, F must be positive (T=%d H=%d E=%d F=%d)", d->T, d->H, d->E, d->F);
  if (d->E > MOE_MAX_EXPERTS) return fail(MOE_ERR_ARG, "E=%d exceeds %d", d->E, MOE_MAX_EXPERTS);
  if (d->top_k < 1 || d->top_k > d->E || d->top_k > MOE_MAX_TOPK)
    return fail(MOE_ERR_ARG, "top_k=%d must be in [1, min(E, %d)]", d->top_k, MOE_MAX_TOPK);
  if (d->H % 128 != 0 || d->F % 128 != 0)
    return fail(MOE_ERR_SHAPE, "H=%d and F=%d must be multiples of 128", d->H, d->F);
  if (d->E % 8 != 0) return fail(MOE_ERR_SHAPE, "E=%d must be a multiple of 8", d->E);
  if (static_cast<int64_t>(d->T) * d->top_k > (1ll << 30))
    return fail(MOE_ERR_ARG, "T*top_k=%lld too large", static_cast<long long>(d->T) * d->top_k);
  if (d->flags & ~(MOE_F_MASK | MOE_F_DW_FP32 | MOE_F_RECOMPUTE))
    return fail(MOE_ERR_ARG, "unknown flags 0x%x", d->flags);
  if (!std::isfinite(d->aux_loss_coef) || !std::isfinite(d->z_loss_coef) || d->aux_loss_coef < 0.0f ||
      d->z_loss_coef < 0.0f)
    return fail(MOE_ERR_ARG, "router-loss coefficients must be finite and >= 0 (aux %g, z %g)",
                static_cast<double>(d->aux_loss_coef), static_cast<double>(d->z_loss_coef));
  return MOE_OK;
}

bool router_losses(const moe_dims* d) { return d->aux_loss_coef != 0.0f || d->z_loss_coef != 0.0f; }

int check_experts_dims(const moe_experts_dims* d) {
  if (d == nullptr) return fail(MOE_ERR_ARG, "dims is NULL");
  if (d->rows < 1 || d->H < 1 || d->E < 1 || d->F < 1)
    return fail(MOE_ERR_ARG, "rows, H, E, F must be positive (rows=%d H=%d E=%d F=%d)", d->rows, d->H, d->E,
                d->F);
  if (d->E > MOE_MAX_EXPERTS) return fail(MOE_ERR_ARG, "E=%d exceeds %d", d->E, MOE_MAX_EXPERTS);
  if (d->H % 128 != 0 || d->F % 128 != 0)
    return fail(MOE_ERR_SHAPE, "H=%d and F=%d must be multiples of 128", d->H, d->F);
  if (d->rows > (1 << 30)) return fail(MOE_ERR_ARG, "rows=%d too large", d->rows);
  if (d->flags & ~(MOE_F_DW_FP32 | MOE_F_RECOMPUTE)) return fail(MOE_ERR_ARG, "unknown flags 0x%x", d->flags);
  return MOE_OK;
}

int check_ptrs(std::initializer_list<std::pair<const char*, const void*>> ps) {
  for (const auto& p : ps) {
    if (p.second == nullptr) return fail(MOE_ERR_ARG, "%s is NULL", p.first);
    if (!aligned16(p.second)) return fail(MOE_ERR_ALIGN, "%s is not 16-byte aligned", p.first);
  }
  return MOE_OK;
}

// ---- layout of the block's `saved` buffer
struct Saved {
  float* logits;
  int32_t *topk_idx, *counts, *offsets, *tile_start, *row_token, *row_of;
  int2* tile_desc;
  float* gates;
  bf16_t *xp, *g, *u, *a, *o;
  float* router_loss;
  size_t bytes;
};

Saved saved_layout(const moe_dims* d, void* base) {
  const size_t T = d->T, E = d->E, k = d->top_k, H = d->H, F = d->F, R = T * k;
  Carve c(base);
  Saved s;
  s.logits = c.take<float>(T * E);
  s.topk_idx = c.take<int32_t>(T * k);
  s.gates = c.take<float>(T * k);
  s.counts = c.take<int32_t>(E);
  s.offsets = c.take<int32_t>(E + 1);
  s.tile_start = c.take<int32_t>(E + 1);
  s.tile_desc = c.take<int2>(static_cast<size_t>(max_row_tiles(d->T * d->top_k, d->E)));
  s.row_token = c.take<int32_t>(R);
  s.row_of = c.take<int32_t>(T * k);
  s.xp = c.take<bf16_t>(R * H);
  const bool keep_gu = !(d->flags & MOE_F_RECOMPUTE);
  s.g = keep_gu ? c.take<bf16_t>(R * F) : nullptr;
  s.u = keep_gu ? c.take<bf16_t>(R * F) : nullptr;
  s.a = c.take<bf16_t>(R * F);
  s.o = c.take<bf16_t>(R * H);
  s.router_loss = c.take<float>(2);
  s.bytes = c.off;
  return s;
}

// ---- layout of the forward workspace: permutation scratch, and the router
// losses' partial sums when they are on
struct FwdWs {
  int32_t* perm;
  float* router_part;
  float* loss;
  size_t bytes;
};

FwdWs fwd_layout(const moe_dims* d, void* base) {
  Carve c(base);
  FwdWs w;
  w.perm = c.take<int32_t>(static_cast<size_t>(permute_ws_ints(d->T, d->E)));
  w.router_part = c.take<float>(static_cast<size_t>(router_part_floats(d->T, d->E)));
  w.loss = router_losses(d) ? c.take<float>(static_cast<size_t>(router_loss_ws_floats(d->T, d->E))) : nullptr;
  w.bytes = c.off;
  return w;
}

size_t fwd_ws(const moe_dims* d) { return fwd_layout(d, nullptr).bytes; }

// ---- layout of the backward workspace
struct BwdWs {
  bf16_t* d_o;  // also dXp once dO is dead
  bf16_t *dg, *du, *dz, *w_rt;
  float *dgate, *dz_slot, *dwr_part;
  float* dgate_part;  // <dA, A> per row and column block of the down product's dgrad
  float* dense;  // dz W_r^T (fp32 [T,H]) when the router losses are on
  int32_t* plan;  // the weight gradients' schedule
  size_t bytes;
};

BwdWs bwd_layout(const moe_dims* d, void* base) {
  const size_t T = d->T, E = d->E, k = d->top_k, H = d->H, F = d->F, R = T * k;
  Carve c(base);
  BwdWs w;
  w.d_o = c.take<bf16_t>(R * H);
  w.dg = c.take<bf16_t>(R * F);
  w.du = c.take<bf16_t>(R * F);
  w.dz = c.take<bf16_t>(T * E);
  w.dgate = c.take<float>(T * k);
  w.dz_slot = c.take<float>(T * k);
  w.dgate_part = c.take<float>(R * static_cast<size_t>(dgate_parts(d->F)));
  w.w_rt = c.take<bf16_t>(E * H);
  w.dwr_part = c.take<float>(static_cast<size_t>(dwr_splits(d->T)) * H * E);
  w.dense = router_losses(d) ? c.take<float>(T * H) : nullptr;
  w.plan = c.take<int32_t>(static_cast<size_t>(wgrad_plan_ints(d->E)));
  w.bytes = c.off;
  return w;
}

// ---- layout of the forward-only (serving) workspace: routing, the permuted
// rows only when x is too large to be read through the permutation, A and O.
struct InferWs {
  float* logits;
  float* router_part;
  int32_t *topk_idx, *counts, *offsets, *tile_start, *row_token, *row_of, *perm;
  int2* tile_desc;
  float* gates;
  bf16_t *xp, *a, *o;
  size_t bytes;
};

// The gate/up product reads x through the permutation when a 32-bit buffer
// offset reaches all of x.
bool infer_reads_x(const moe_dims* d) {
  return static_cast<int64_t>(d->T) * d->H * 2 <= 0x7fffffffll;
}

InferWs infer_layout(const moe_dims* d, void* base) {
  const size_t T = d->T, E = d->E, k = d->top_k, H = d->H, F = d->F, R = T * k;
  Carve c(base);
  InferWs w;
  w.logits = c.take<float>(T * E);
  w.router_part = c.take<float>(static_cast<size_t>(router_part_floats(d->T, d->E)));
  w.topk_idx = c.take<int32_t>(T * k);
  w.gates = c.take<float>(T * k);
  w.counts = c.take<int32_t>(E);
  w.offsets = c.take<int32_t>(E + 1);
  w.tile_start = c.take<int32_t>(E + 1);
  w.tile_desc = c.take<int2>(static_cast<size_t>(max_row_tiles(d->T * d->top_k, d->E)));
  w.row_token = c.take<int32_t>(R);
  w.row_of = c.take<int32_t>(T * k);
  w.perm = c.take<int32_t>(static_cast<size_t>(permute_ws_ints(d->T, d->E)));
  w.xp = infer_reads_x(d) ? nullptr : c.take<bf16_t>(R * H);
  w.a = c.take<bf16_t>(R * F);
  w.o = c.take<bf16_t>(R * H);
  w.bytes = c.off;
  return w;
}

struct ExpSaved {
  int32_t *offsets, *tile_start;
  int2* tile_desc;
  bf16_t *g, *u, *a;
  size_t bytes;
};

ExpSaved exp_saved_layout(const moe_experts_dims* d, void* base) {
  const size_t E = d->E, F = d->F, R = d->rows;
  Carve c(base);
  ExpSaved s;
  s.offsets = c.take<int32_t>(E + 1);
  s.tile_start = c.take<int32_t>(E + 1);
  s.tile_desc = c.take<int2>(static_cast<size_t>(max_row_tiles(d->rows, d->E)));
  const bool keep_gu = !(d->flags & MOE_F_RECOMPUTE);
  s.g = keep_gu ? c.take<bf16_t>(R * F) : nullptr;
  s.u = keep_gu ? c.take<bf16_t>(R * F) : nullptr;
  s.a = c.take<bf16_t>(R * F);
  s.bytes = c.off;
  return s;
}

struct ExpWs {
  bf16_t *dg, *du;
  int32_t* plan;  // the weight gradients' schedule
  size_t bytes;
};

ExpWs exp_ws_layout(const moe_experts_dims* d, void* base) {
  const size_t F = d->F, R = d->rows;
  Carve c(base);
  ExpWs w;
  w.dg = c.take<bf16_t>(R * F);
  w.du = c.take<bf16_t>(R * F);
  w.plan = c.take<int32_t>(static_cast<size_t>(wgrad_plan_ints(d->E)));
  w.bytes = c.off;
  return w;
}

int hip_status(hipError_t e, const char* where) {
  if (e != hipSuccess) return fail(MOE_ERR_HIP, "%s: %s", where, hipGetErrorString(e));
  return ok();
}

// MOE_F_RECOMPUTE: the forward kept no G and U.  Recompute them with the
// forward's kernel (same tiles, same summation order: the same bits) into the
// dG / dU workspace, where the down dgrad then overwrites them in place.
int recompute_gu(uint32_t flags, ExpertArgs& a, bf16_t* dg, bf16_t* du, hipStream_t s) {
  if (!(flags & MOE_F_RECOMPUTE)) return MOE_OK;
  ExpertArgs r = a;
  r.g = dg;
  r.u = du;
  r.act = nullptr;
  const hipError_t e = launch_gateup_fwd(r, s, /*recompute=*/true);
  if (e != hipSuccess) return hip_status(e, "gate/up recompute");
  a.g = dg;
  a.u = du;
  return MOE_OK;
}

// ---- expert LoRA: argument checks, the saved buffer (the block's layout,
// then P1 and P2) and the workspace (the larger of the forward's and the
// backward's, the latter followed by Q1 and Q2)
int check_lora(const moe_lora* l) {
  if (l == nullptr) return fail(MOE_ERR_ARG, "lora is NULL");
  if (l->rank < 16 || l->rank > 64 || l->rank % 16 != 0)
    return fail(MOE_ERR_SHAPE, "LoRA rank %d must be 16, 32, 48 or 64", l->rank);
  if (!std::isfinite(l->scale)) return fail(MOE_ERR_ARG, "LoRA scale is not finite");
  return check_ptrs({{"lora.a1", l->a1}, {"lora.b1_gate", l->b1_gate}, {"lora.b1_up", l->b1_up}, {"lora.a2", l->a2},
                     {"lora.b2", l->b2}});
}

bool lora_rank_ok(int32_t rank) { return rank >= 16 && rank <= 64 && rank % 16 == 0; }

struct LoraSaved {
  bf16_t *p1, *p2;
  size_t bytes;
};

LoraSaved lora_saved_layout(const moe_dims* d, int32_t rank, void* base) {
  const size_t R = static_cast<size_t>(d->T) * d->top_k;
  Carve c(base);
  c.off = saved_layout(d, nullptr).bytes;
  LoraSaved s;
  s.p1 = c.take<bf16_t>(R * rank);
  s.p2 = c.take<bf16_t>(R * rank);
  s.bytes = c.off;
  return s;
}

struct LoraWs {
  bf16_t *q1, *q2;
  size_t bytes;
};

LoraWs lora_ws_layout(const moe_dims* d, int32_t rank, void* base) {
  const size_t R = static_cast<size_t>(d->T) * d->top_k;
  Carve c(base);
  c.off = bwd_layout(d, nullptr).bytes;
  LoraWs w;
  w.q1 = c.take<bf16_t>(R * rank);
  w.q2 = c.take<bf16_t>(R * rank);
  w.bytes = c.off > fwd_ws(d) ? c.off : fwd_ws(d);
  return w;
}

LoraArgs lora_args(const moe_lora* l, const LoraSaved& ls) {
  LoraArgs a;
  a.rank = l->rank;
  a.scale = l->scale;
  a.a1 = static_cast<const bf16_t*>(l->a1);
  a.b1_gate = static_cast<const bf16_t*>(l->b1_gate);
  a.b1_up = static_cast<const bf16_t*>(l->b1_up);
  a.a2 = static_cast<const bf16_t*>(l->a2);
  a.b2 = static_cast<const bf16_t*>(l->b2);
  a.p1 = ls.p1;
  a.p2 = ls.p2;
  return a;
}

// The block forward, with the adapters when `lora` is non-null: routing,
// permutation, router losses, the expert products and the combine.
int block_fwd(const moe_dims* d, const void* x, const void* w_r, const void* w_gate, const void* w_up,
              const void* w_down, const moe_lora* lora, const uint8_t* token_mask, void* y, void* saved,
              void* ws, size_t ws_bytes, void* stream) {
  if (int rc = check_dims(d)) return rc;
  if (int rc = check_ptrs({{"x", x}, {"w_r", w_r}, {"w_gate", w_gate}, {"w_up", w_up}, {"w_down", w_down},
                           {"y", y}, {"saved", saved}, {"ws", ws}}))
    return rc;
  if (lora != nullptr)
    if (int rc = check_lora(lora)) return rc;
  const bool masked = d->flags & MOE_F_MASK;
  if (masked && token_mask == nullptr) return fail(MOE_ERR_ARG, "MOE_F_MASK set but token_mask is NULL");
  const FwdWs fw = fwd_layout(d, ws);
  const size_t need = lora != nullptr ? lora_ws_layout(d, lora->rank, nullptr).bytes : fw.bytes;
  if (ws_bytes < need) return fail(MOE_ERR_WORKSPACE, "workspace %zu < %zu bytes", ws_bytes, need);
  hipStream_t s = static_cast<hipStream_t>(stream);
  const Saved sv = saved_layout(d, saved);
  const int T = d->T, H = d->H, E = d->E, F = d->F, k = d->top_k;
  const bf16_t* xb = static_cast<const bf16_t*>(x);
  hipError_t e = launch_router_fwd(xb, static_cast<const bf16_t*>(w_r), masked ? token_mask : nullptr, T, H,
                                   E, k, sv.logits, fw.router_part, sv.topk_idx, sv.gates, fw.loss, fw.perm,
                                   sv.row_token, s);
  if (e != hipSuccess) return hip_status(e, "router");
  e = launch_permute(sv.topk_idx, xb, T, H, E, k, sv.counts, sv.offsets, sv.tile_start, sv.tile_desc, sv.row_token,
                     sv.row_of, sv.xp, fw.perm, s);
  if (e != hipSuccess) return hip_status(e, "permute");
  if (fw.loss != nullptr) {
    e = launch_router_loss(fw.loss, T, E, k, sv.counts, sv.offsets, d->aux_loss_coef, d->z_loss_coef,
                           sv.router_loss, s);
    if (e != hipSuccess) return hip_status(e, "router losses");
  }
  ExpertArgs a{T * k, H, E, F, sv.xp, static_cast<const bf16_t*>(w_gate), static_cast<const bf16_t*>(w_up),
               static_cast<const bf16_t*>(w_down), sv.offsets, sv.tile_start, sv.tile_desc, sv.g, sv.u, sv.a};
  if (lora != nullptr) {
    a.lora = lora_args(lora, lora_saved_layout(d, lora->rank, saved));
    const int r = lora->rank;
    // P1 = scale Xp a1 (a1 [E][H][r]: the B operand MN-contiguous)
    e = launch_lora_rows(a, sv.xp, nullptr, H, a.lora.a1, nullptr, static_cast<int64_t>(H) * r, H, false,
                         a.lora.p1, s);
    if (e != hipSuccess) return hip_status(e, "LoRA P1");
  }
  e = launch_gateup_fwd(a, s);
  if (e != hipSuccess) return hip_status(e, "gate/up");
  if (lora != nullptr) {
    const int r = lora->rank;
    // P2 = scale A a2 (a2 [E][F][r])
    e = launch_lora_rows(a, sv.a, nullptr, F, a.lora.a2, nullptr, static_cast<int64_t>(F) * r, F, false, a.lora.p2,
                         s);
    if (e != hipSuccess) return hip_status(e, "LoRA P2");
  }
  e = launch_down_fwd(a, sv.o, s);
  if (e != hipSuccess) return hip_status(e, "down");
  e = launch_combine(sv.o, sv.gates, sv.row_of, T, H, k, static_cast<bf16_t*>(y), s);
  return hip_status(e, "combine");
}

}  // namespace

extern "C" {

size_t moe_saved_bytes(const moe_dims* d) {
  if (check_dims(d) != MOE_OK) return 0;
  return saved_layout(d, nullptr).bytes;
}

size_t moe_fwd_workspace_bytes(const moe_dims* d) {
  if (check_dims(d) != MOE_OK) return 0;
  return fwd_ws(d);
}

size_t moe_bwd_workspace_bytes(const moe_dims* d) {
  if (check_dims(d) != MOE_OK) return 0;
  return bwd_layout(d, nullptr).bytes;
}

int moe_saved_views(const moe_dims* d, void* saved, moe_saved_view* v) {
  if (int rc = check_dims(d)) return rc;
  if (saved == nullptr || v == nullptr) return fail(MOE_ERR_ARG, "saved or view is NULL");
  const Saved s = saved_layout(d, saved);
  v->logits = s.logits;
  v->topk_idx = s.topk_idx;
  v->gates = s.gates;
  v->counts = s.counts;
  v->offsets = s.offsets;
  v->row_token = s.row_token;
  v->row_of = s.row_of;
  v->xp = s.xp;
  v->g = s.g;
  v->u = s.u;
  v->a = s.a;
  v->o = s.o;
  v->router_loss = s.router_loss;
  return ok();
}

int moe_fwd(const moe_dims* d, const void* x, const void* w_r, const void* w_gate, const void* w_up,
            const void* w_down, const uint8_t* token_mask, void* y, void* saved, void* ws,
            size_t ws_bytes, void* stream) {
  return block_fwd(d, x, w_r, w_gate, w_up, w_down, nullptr, token_mask, y, saved, ws, ws_bytes, stream);
}

int moe_fwd_noalloc(const moe_dims* d, const void* x, const void* w_r, const void* w_gate, const void* w_up,
                    const void* w_down, const uint8_t* token_mask, void* y, void* saved, void* stream) {
  if (int rc = check_dims(d)) return rc;
  const size_t need = fwd_ws(d);
  if (need > MOE_NOALLOC_SCRATCH_BYTES)
    return fail(MOE_ERR_WORKSPACE, "the forward needs %zu bytes of scratch, beyond the %zu of the static array",
                need, static_cast<size_t>(MOE_NOALLOC_SCRATCH_BYTES));
  // the caller's pointers are checked before the runtime is asked for the
  // array's address, so that every argument error comes back with no HIP call
  if (int rc = check_ptrs({{"x", x}, {"w_r", w_r}, {"w_gate", w_gate}, {"w_up", w_up}, {"w_down", w_down},
                           {"y", y}, {"saved", saved}}))
    return rc;
  if ((d->flags & MOE_F_MASK) && token_mask == nullptr)
    return fail(MOE_ERR_ARG, "MOE_F_MASK set but token_mask is NULL");
  void* ws = nullptr;
  size_t ws_bytes = 0;
  const hipError_t e = static_scratch(&ws, &ws_bytes);
  if (e != hipSuccess) return hip_status(e, "static scratch");
  return block_fwd(d, x, w_r, w_gate, w_up, w_down, nullptr, token_mask, y, saved, ws, ws_bytes, stream);
}

int moe_bwd(const moe_dims* d, const void* x, const void* w_r, const void* w_gate, const void* w_up,
            const void* w_down, const void* dy, const void* saved, void* dx, void* dw_r, void* dw_gate,
            void* dw_up, void* dw_down, void* ws, size_t ws_bytes, void* stream) {
  if (int rc = check_dims(d)) return rc;
  if (int rc = check_ptrs({{"x", x}, {"w_r", w_r}, {"w_gate", w_gate}, {"w_up", w_up}, {"w_down", w_down},
                           {"dy", dy}, {"saved", saved}, {"dx", dx}, {"dw_r", dw_r}, {"dw_gate", dw_gate},
                           {"dw_up", dw_up}, {"dw_down", dw_down}, {"ws", ws}}))
    return rc;
  const BwdWs w = bwd_layout(d, ws);
  if (ws_bytes < w.bytes) return fail(MOE_ERR_WORKSPACE, "workspace %zu < %zu bytes", ws_bytes, w.bytes);
  hipStream_t s = static_cast<hipStream_t>(stream);
  const Saved sv = saved_layout(d, const_cast<void*>(saved));
  const int T = d->T, H = d->H, E = d->E, F = d->F, k = d->top_k;
  const bool f32 = d->flags & MOE_F_DW_FP32;
  // the combine backward's extra workgroup also builds the weight gradients' schedule
  hipError_t e = launch_combine_bwd(static_cast<const bf16_t*>(dy), sv.gates, sv.row_of, T, H, k, w.d_o, s,
                                    sv.offsets, E, F, w.plan);
  if (e != hipSuccess) return hip_status(e, "combine bwd");
  ExpertArgs a{T * k, H, E, F, sv.xp, static_cast<const bf16_t*>(w_gate), static_cast<const bf16_t*>(w_up),
               static_cast<const bf16_t*>(w_down), sv.offsets, sv.tile_start, sv.tile_desc, sv.g, sv.u, sv.a};
  a.dgate_part = w.dgate_part;
  a.wgrad_plan = w.plan;
  a.wgrad_plan_built = true;
  if (int rc = recompute_gu(d->flags, a, w.dg, w.du, s)) return rc;
  // dXp reuses dO's memory: the down products that read dO are queued first.
  e = launch_experts_bwd_data(a, w.d_o, w.dg, w.du, /*dxp=*/w.d_o, dw_down, f32, s);
  if (e != hipSuccess) return hip_status(e, "experts bwd");
  // gate gradients and dz from the down dgrad's <dA, A> sums
  e = launch_gate_bwd(w.dgate_part, dgate_parts(F), sv.gates, sv.topk_idx, sv.row_of, T, E, k, w.dgate, w.dz_slot,
                      w.dz, sv.logits, sv.counts, sv.offsets, d->aux_loss_coef, d->z_loss_coef,
                      w.dense == nullptr ? static_cast<const bf16_t*>(w_r) : nullptr, H, w.w_rt, s);
  if (e != hipSuccess) return hip_status(e, "gate bwd");
  // dX right after dXp, while much of dXp is still in the last-level cache.
  e = launch_router_dx(w.dz_slot, sv.topk_idx, static_cast<const bf16_t*>(w_r), w.d_o, sv.row_of, T, H, E, k,
                       w.w_rt, static_cast<bf16_t*>(dx), w.dense != nullptr ? w.dz : nullptr, w.dense, s);
  if (e != hipSuccess) return hip_status(e, "dx");
  e = launch_experts_bwd_gateup_w(a, w.dg, w.du, dw_gate, dw_up, f32, s);
  if (e != hipSuccess) return hip_status(e, "experts bwd");
  e = launch_dwr(static_cast<const bf16_t*>(x), w.dz, T, H, E, w.dwr_part, dw_r, f32, s);
  return hip_status(e, "router weight grad");
}

size_t moe_lora_saved_bytes(const moe_dims* d, int32_t rank) {
  if (check_dims(d) != MOE_OK || !lora_rank_ok(rank)) return 0;
  return lora_saved_layout(d, rank, nullptr).bytes;
}

size_t moe_lora_workspace_bytes(const moe_dims* d, int32_t rank) {
  if (check_dims(d) != MOE_OK || !lora_rank_ok(rank)) return 0;
  return lora_ws_layout(d, rank, nullptr).bytes;
}

int moe_lora_fwd(const moe_dims* d, const void* x, const void* w_r, const void* w_gate, const void* w_up,
                 const void* w_down, const moe_lora* lora, const uint8_t* token_mask, void* y, void* saved,
                 void* ws, size_t ws_bytes, void* stream) {
  if (lora == nullptr) return fail(MOE_ERR_ARG, "lora is NULL");
  return block_fwd(d, x, w_r, w_gate, w_up, w_down, lora, token_mask, y, saved, ws, ws_bytes, stream);
}

int moe_lora_bwd(const moe_dims* d, const void* x, const void* w_r, const void* w_gate, const void* w_up,
                 const void* w_down, const moe_lora* lora, const void* dy, const void* saved, void* dx, void* da1,
                 void* db1_gate, void* db1_up, void* da2, void* db2, void* ws, size_t ws_bytes, void* stream) {
  if (int rc = check_dims(d)) return rc;
  if (int rc = check_ptrs({{"x", x}, {"w_r", w_r}, {"w_gate", w_gate}, {"w_up", w_up}, {"w_down", w_down},
                           {"dy", dy}, {"saved", saved}, {"dx", dx}, {"da1", da1}, {"db1_gate", db1_gate},
                           {"db1_up", db1_up}, {"da2", da2}, {"db2", db2}, {"ws", ws}}))
    return rc;
  if (int rc = check_lora(lora)) return rc;
  const LoraWs lw = lora_ws_layout(d, lora->rank, ws);
  if (ws_bytes < lw.bytes) return fail(MOE_ERR_WORKSPACE, "workspace %zu < %zu bytes", ws_bytes, lw.bytes);
  const BwdWs w = bwd_layout(d, ws);
  hipStream_t s = static_cast<hipStream_t>(stream);
  const Saved sv = saved_layout(d, const_cast<void*>(saved));
  const int T = d->T, H = d->H, E = d->E, F = d->F, k = d->top_k, r = lora->rank;
  const bool f32 = d->flags & MOE_F_DW_FP32;
  hipError_t e = launch_combine_bwd(static_cast<const bf16_t*>(dy), sv.gates, sv.row_of, T, H, k, w.d_o, s);
  if (e != hipSuccess) return hip_status(e, "combine bwd");
  ExpertArgs a{T * k, H, E, F, sv.xp, static_cast<const bf16_t*>(w_gate), static_cast<const bf16_t*>(w_up),
               static_cast<const bf16_t*>(w_down), sv.offsets, sv.tile_start, sv.tile_desc, sv.g, sv.u, sv.a};
  a.lora = lora_args(lora, lora_saved_layout(d, r, const_cast<void*>(saved)));
  a.dgate_part = w.dgate_part;
  if (int rc = recompute_gu(d->flags, a, w.dg, w.du, s)) return rc;
  // Q2 = scale dO b2^T (b2 [E][r][H]: rows q of the B operand, K-contiguous)
  e = launch_lora_rows(a, w.d_o, nullptr, H, a.lora.b2, nullptr, static_cast<int64_t>(r) * H, H, true, lw.q2, s);
  if (e != hipSuccess) return hip_status(e, "LoRA Q2");
  e = launch_down_dgrad(a, w.d_o, w.dg, w.du, lw.q2, s);
  if (e != hipSuccess) return hip_status(e, "down dgrad");
  e = launch_gate_bwd(w.dgate_part, dgate_parts(F), sv.gates, sv.topk_idx, sv.row_of, T, E, k, w.dgate, w.dz_slot,
                      w.dz, sv.logits, sv.counts, sv.offsets, d->aux_loss_coef, d->z_loss_coef,
                      w.dense == nullptr ? static_cast<const bf16_t*>(w_r) : nullptr, H, w.w_rt, s);
  if (e != hipSuccess) return hip_status(e, "gate bwd");
  // d a2 = A^T Q2 ([E][F][r]); d b2 = P2^T dO, formed as (dO^T P2)^T ([E][r][H])
  e = launch_lora_wgrad(a, sv.a, F, F, lw.q2, false, da2, f32, s);
  if (e != hipSuccess) return hip_status(e, "LoRA d a2");
  e = launch_lora_wgrad(a, w.d_o, H, H, a.lora.p2, true, db2, f32, s);
  if (e != hipSuccess) return hip_status(e, "LoRA d b2");
  // Q1 = scale (dG b1_gate^T + dU b1_up^T)
  e = launch_lora_rows(a, w.dg, w.du, F, a.lora.b1_gate, a.lora.b1_up, static_cast<int64_t>(r) * F, F, true, lw.q1,
                       s);
  if (e != hipSuccess) return hip_status(e, "LoRA Q1");
  // dXp (+ Q1 a1^T) into dO's memory: everything that reads dO is queued above
  e = launch_gateup_dgrad(a, w.dg, w.du, w.d_o, lw.q1, s);
  if (e != hipSuccess) return hip_status(e, "gate/up dgrad");
  e = launch_router_dx(w.dz_slot, sv.topk_idx, static_cast<const bf16_t*>(w_r), w.d_o, sv.row_of, T, H, E, k,
                       w.w_rt, static_cast<bf16_t*>(dx), w.dense != nullptr ? w.dz : nullptr, w.dense, s);
  if (e != hipSuccess) return hip_status(e, "dx");
  // d a1 = Xp^T Q1 ([E][H][r]); d b1 = P1^T dG / dU, formed transposed ([E][r][F])
  e = launch_lora_wgrad(a, sv.xp, H, H, lw.q1, false, da1, f32, s);
  if (e != hipSuccess) return hip_status(e, "LoRA d a1");
  e = launch_lora_wgrad(a, w.dg, F, F, a.lora.p1, true, db1_gate, f32, s);
  if (e != hipSuccess) return hip_status(e, "LoRA d b1_gate");
  e = launch_lora_wgrad(a, w.du, F, F, a.lora.p1, true, db1_up, f32, s);
  return hip_status(e, "LoRA d b1_up");
}

size_t moe_infer_workspace_bytes(const moe_dims* d) {
  if (check_dims(d) != MOE_OK) return 0;
  return infer_layout(d, nullptr).bytes;
}

int moe_infer(const moe_dims* d, const void* x, const void* w_r, const void* w_gate, const void* w_up,
              const void* w_down, const uint8_t* token_mask, void* y, void* ws, size_t ws_bytes, void* stream) {
  if (int rc = check_dims(d)) return rc;
  if (int rc = check_ptrs({{"x", x}, {"w_r", w_r}, {"w_gate", w_gate}, {"w_up", w_up}, {"w_down", w_down},
                           {"y", y}, {"ws", ws}}))
    return rc;
  const bool masked = d->flags & MOE_F_MASK;
  if (masked && token_mask == nullptr) return fail(MOE_ERR_ARG, "MOE_F_MASK set but token_mask is NULL");
  const InferWs w = infer_layout(d, ws);
  if (ws_bytes < w.bytes) return fail(MOE_ERR_WORKSPACE, "workspace %zu < %zu bytes", ws_bytes, w.bytes);
  hipStream_t s = static_cast<hipStream_t>(stream);
  const int T = d->T, H = d->H, E = d->E, F = d->F, k = d->top_k;
  const bf16_t* xb = static_cast<const bf16_t*>(x);
  hipError_t e = launch_router_fwd(xb, static_cast<const bf16_t*>(w_r), masked ? token_mask : nullptr, T, H,
                                   E, k, w.logits, w.router_part, w.topk_idx, w.gates, nullptr, w.perm, w.row_token,
                                   s);
  if (e != hipSuccess) return hip_status(e, "router");
  e = launch_permute(w.topk_idx, xb, T, H, E, k, w.counts, w.offsets, w.tile_start, w.tile_desc, w.row_token, w.row_of,
                     w.xp, w.perm, s);
  if (e != hipSuccess) return hip_status(e, "permute");
  ExpertArgs a{T * k, H, E, F, w.xp, static_cast<const bf16_t*>(w_gate), static_cast<const bf16_t*>(w_up),
               static_cast<const bf16_t*>(w_down), w.offsets, w.tile_start, w.tile_desc, nullptr, nullptr, w.a};
  if (w.xp == nullptr) {
    a.xp = xb;
    a.xp_rows = w.row_token;
    a.xp_bytes = static_cast<int64_t>(T) * H * 2;
  }
  e = launch_gateup_fwd(a, s);
  if (e != hipSuccess) return hip_status(e, "gate/up");
  e = launch_down_fwd(a, w.o, s);
  if (e != hipSuccess) return hip_status(e, "down");
  e = launch_combine(w.o, w.gates, w.row_of, T, H, k, static_cast<bf16_t*>(y), s);
  return hip_status(e, "combine");
}

size_t moe_experts_saved_bytes(const moe_experts_dims* d) {
  if (check_experts_dims(d) != MOE_OK) return 0;
  return exp_saved_layout(d, nullptr).bytes;
}

size_t moe_experts_workspace_bytes(const moe_experts_dims* d) {
  if (check_experts_dims(d) != MOE_OK) return 0;
  return exp_ws_layout(d, nullptr).bytes;
}

int moe_experts_saved_views(const moe_experts_dims* d, void* saved, moe_experts_saved_view* v) {
  if (int rc = check_experts_dims(d)) return rc;
  if (saved == nullptr || v == nullptr) return fail(MOE_ERR_ARG, "saved or view is NULL");
  const ExpSaved s = exp_saved_layout(d, saved);
  v->offsets = s.offsets;
  v->g = s.g;
  v->u = s.u;
  v->a = s.a;
  return ok();
}

int moe_experts_fwd(const moe_experts_dims* d, const void* xp, const int32_t* counts, const void* w_gate,
                    const void* w_up, const void* w_down, void* o, void* saved, void* ws, size_t ws_bytes,
                    void* stream) {
  (void)ws;
  (void)ws_bytes;
  if (int rc = check_experts_dims(d)) return rc;
  if (int rc = check_ptrs({{"xp", xp}, {"counts", counts}, {"w_gate", w_gate}, {"w_up", w_up},
                           {"w_down", w_down}, {"o", o}, {"saved", saved}}))
    return rc;
  hipStream_t s = static_cast<hipStream_t>(stream);
  const ExpSaved sv = exp_saved_layout(d, saved);
  hipError_t e = launch_offsets_from_counts(counts, d->E, d->rows, sv.offsets, sv.tile_start, sv.tile_desc, s);
  if (e != hipSuccess) return hip_status(e, "offsets");
  ExpertArgs a{d->rows, d->H, d->E, d->F, static_cast<const bf16_t*>(xp), static_cast<const bf16_t*>(w_gate),
               static_cast<const bf16_t*>(w_up), static_cast<const bf16_t*>(w_down), sv.offsets, sv.tile_start,
               sv.tile_desc, sv.g, sv.u, sv.a};
  e = launch_gateup_fwd(a, s);
  if (e != hipSuccess) return hip_status(e, "gate/up");
  e = launch_down_fwd(a, static_cast<bf16_t*>(o), s);
  return hip_status(e, "down");
}

int moe_experts_bwd(const moe_experts_dims* d, const void* xp, const void* w_gate, const void* w_up,
                    const void* w_down, const void* d_o, const void* saved, void* dxp, void* dw_gate,
                    void* dw_up, void* dw_down, void* ws, size_t ws_bytes, void* stream) {
  if (int rc = check_experts_dims(d)) return rc;
  if (int rc = check_ptrs({{"xp", xp}, {"w_gate", w_gate}, {"w_up", w_up}, {"w_down", w_down}, {"d_o", d_o},
                           {"saved", saved}, {"dxp", dxp}, {"dw_gate", dw_gate}, {"dw_up", dw_up},
                           {"dw_down", dw_down}, {"ws", ws}}))
    return rc;
  const ExpWs w = exp_ws_layout(d, ws);
  if (ws_bytes < w.bytes) return fail(MOE_ERR_WORKSPACE, "workspace %zu < %zu bytes", ws_bytes, w.bytes);
  hipStream_t s = static_cast<hipStream_t>(stream);
  const ExpSaved sv = exp_saved_layout(d, const_cast<void*>(saved));
  ExpertArgs a{d->rows, d->H, d->E, d->F, static_cast<const bf16_t*>(xp), static_cast<const bf16_t*>(w_gate),
               static_cast<const bf16_t*>(w_up), static_cast<const bf16_t*>(w_down), sv.offsets, sv.tile_start,
               sv.tile_desc, sv.g, sv.u, sv.a};
  a.wgrad_plan = w.plan;
  if (int rc = recompute_gu(d->flags, a, w.dg, w.du, s)) return rc;
  hipError_t e = launch_experts_bwd(a, static_cast<const bf16_t*>(d_o), w.dg, w.du, static_cast<bf16_t*>(dxp),
                                    dw_gate, dw_up, dw_down, (d->flags & MOE_F_DW_FP32) != 0, s);
  return hip_status(e, "experts bwd");
}

const char* moe_last_error(void) { return g_err; }

int moe_version(void) { return 200; }

}  // extern "C"
