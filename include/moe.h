/*
 * moe.h -- C ABI of the MI355X (gfx950) mixture-of-experts FFN block.
 *
 * The block is the expert layer of a Qwen3-30B-A3B-style MoE reranker: the
 * paper (§3, Expert-Parallel MoE Training) routes each token to its top-8 of
 * 128 experts and, under expert parallelism, dispatches routed tokens to the
 * ranks that hold their experts (§3, "Expert parallelism and topology").  The
 * operations below are, in order:
 *
 *   forward   z = x W_r (fp32 logits); per valid token the top-k experts
 *             (descending logit, ties to the lower expert index) and gates
 *             g = softmax over the k selected logits; a stable permutation of
 *             the routed (token, slot) pairs into expert-major, token-ascending
 *             rows; Xp[r] = x[row_token[r]]; per expert e on its rows
 *             G = Xp W_gate[e], U = Xp W_up[e], A = silu(G) * U, O = A W_down[e];
 *             Y[t] = sum_j g[t,j] O[row_of[t,j]].
 *   backward  dO = g dY and dg = <dY, O> per routed row; dA = dO W_down^T;
 *             dG = dA U s (1 + G (1 - s)), dU = dA silu(G) with s = sigmoid(G);
 *             dXp = dG W_gate^T + dU W_up^T; dW_down = A^T dO,
 *             dW_gate = Xp^T dG, dW_up = Xp^T dU per expert (zero for experts
 *             with no rows); dz = g (dg - sum_j g dg) on the selected experts;
 *             dW_r = x^T dz; dX[t] = sum_j dXp[row_of[t,j]] + dz[t] W_r^T.
 *
 * The paper does not print these equations; the readings taken where it is
 * silent (selection precision, tie-break, gate placement, padding, dropless
 * routing, auxiliary router losses off unless asked for) are the ones stated
 * above and at moe_dims.
 *
 * Conventions shared by every entry point
 *   - All tensors are row-major and live in device memory owned by the
 *     caller; the library never allocates or frees device memory (the one
 *     static scratch array of moe_fwd_noalloc aside, which the HIP runtime
 *     reserves on each GPU when it loads the library's device code).
 *   - "bf16" tensors are IEEE bfloat16 (2 bytes); accumulation is fp32.
 *   - Every device pointer must be 16-byte aligned.
 *   - Calls are asynchronous on `stream` (a hipStream_t; NULL = the null
 *     stream) and never synchronise the host; counts stay on the device.
 *   - All argument checks happen before any launch: on an error nothing is
 *     launched and an MOE_ERR_* code is returned; moe_last_error() then
 *     describes it (thread-local string, valid until the next call on the
 *     same thread).
 *   - Results are deterministic: two calls with the same inputs produce the
 *     same bits (no atomics decide any floating-point summation order).
 *   - No thread safety is promised for concurrent calls sharing buffers.
 */
#ifndef MOE_MI355X_H
#define MOE_MI355X_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* return codes */
#define MOE_OK 0
#define MOE_ERR_ARG (-1)       /* null pointer, non-positive size, k not in [1, E], E too large,
                                * a router-loss coefficient negative or not finite */
#define MOE_ERR_SHAPE (-2)     /* H or F not a multiple of 128, E not a multiple of 8 */
#define MOE_ERR_ALIGN (-3)     /* a device pointer not 16-byte aligned */
#define MOE_ERR_WORKSPACE (-4) /* workspace smaller than the size query returns */
#define MOE_ERR_HIP (-5)       /* the HIP runtime reported an error on launch */

/* limits */
#define MOE_MAX_EXPERTS 256
#define MOE_MAX_TOPK 32

/* flags (moe_dims.flags, moe_experts_dims.flags) */
#define MOE_F_MASK 1u    /* token_mask is given: tokens with mask 0 are not routed */
#define MOE_F_DW_FP32 2u /* weight gradients (dW_r, dW_gate, dW_up, dW_down) are fp32, else bf16 */
#define MOE_F_RECOMPUTE 4u /* the forward keeps no G and U (their saved views are NULL and the
                            * saved buffer shrinks by 2 * R_cap * F * 2 bytes); the backward
                            * recomputes them from Xp with the forward's own kernel, one more
                            * gate/up product, so every output is bit-identical to a run
                            * without the flag */

/* Sizes of the full block.  T tokens (T >= 1), hidden size H, E experts,
 * expert width F, top_k experts per token.
 *
 * Router losses (the paper is silent on them; 0 = off, the default):
 *   aux_loss_coef  load-balancing loss  L_aux = aux_loss_coef * E * sum_e f_e P_e,
 *                  f_e = rows of expert e / (T_v k), P_e = mean over valid
 *                  tokens of the full softmax of the logits;
 *   z_loss_coef    z-loss  L_z = z_loss_coef * mean over valid tokens of
 *                  (log sum_e exp z[t,e])^2.
 * With either non-zero, moe_fwd writes {L_aux, L_z} (moe_saved_view.router_loss)
 * and moe_bwd adds their gradient (f held constant) to the router-logit
 * gradient, i.e. the losses join the objective with weight 1.  Both must be
 * finite and >= 0. */
typedef struct moe_dims {
  int32_t T, H, E, F, top_k;
  uint32_t flags;
  float aux_loss_coef, z_loss_coef;
} moe_dims;

/* Device pointers into a `saved` buffer filled by moe_fwd (see
 * moe_saved_views).  R_cap = T * top_k rows are reserved; the routed row
 * count R = offsets[E] <= R_cap lives on the device. */
typedef struct moe_saved_view {
  float* logits;      /* [T, E]      fp32 router logits (masked tokens: computed, not used) */
  int32_t* topk_idx;  /* [T, k]      selected experts, descending logit; -1 for masked tokens */
  float* gates;       /* [T, k]      fp32 gates, sum 1 per valid token; 0 for masked tokens */
  int32_t* counts;    /* [E]         rows per expert */
  int32_t* offsets;   /* [E + 1]     exclusive prefix sum of counts; offsets[E] = R */
  int32_t* row_token; /* [R_cap]     token of row r for r < R, -1 beyond */
  int32_t* row_of;    /* [T, k]      row of (token, slot); -1 for masked tokens */
  void* xp;           /* [R_cap, H]  bf16 permuted tokens (rows >= R undefined) */
  void* g;            /* [R_cap, F]  bf16 gate projection G (NULL with MOE_F_RECOMPUTE) */
  void* u;            /* [R_cap, F]  bf16 up projection U (NULL with MOE_F_RECOMPUTE) */
  void* a;            /* [R_cap, F]  bf16 SwiGLU activation A = silu(G) * U */
  void* o;            /* [R_cap, H]  bf16 expert outputs O (ungated) */
  float* router_loss; /* [2]         {L_aux, L_z}, written when a router-loss coefficient is non-zero */
} moe_saved_view;

/* Bytes of the caller-owned `saved` buffer that carries routing and
 * activations from moe_fwd to moe_bwd.  0 if d is invalid. */
size_t moe_saved_bytes(const moe_dims* d);

/* Bytes of scratch each call needs (contents not preserved across calls).
 * 0 if d is invalid. */
size_t moe_fwd_workspace_bytes(const moe_dims* d);
size_t moe_bwd_workspace_bytes(const moe_dims* d);

/* Fill `view` with device pointers into `saved` (no device work).
 * Returns MOE_OK or MOE_ERR_ARG. */
int moe_saved_views(const moe_dims* d, void* saved, moe_saved_view* view);

/* Forward of the block: the top-k router and the expert FFNs of the paper's
 * MoE layer (§3, Expert-Parallel MoE Training), the forward equations in the
 * header above, with the routed rows grouped per expert as expert-parallel
 * dispatch delivers them to an expert's owner (§3, "Expert parallelism and
 * topology").
 *   x          [T, H]  bf16 tokens
 *   w_r        [H, E]  bf16 router weight
 *   w_gate     [E, H, F], w_up [E, H, F], w_down [E, F, H]  bf16 expert weights
 *   token_mask [T] uint8 (nonzero = real token) when d->flags has MOE_F_MASK,
 *              else ignored (may be NULL)
 *   y          [T, H]  bf16 output (masked tokens: 0)
 *   saved      moe_saved_bytes(d) bytes, filled for moe_bwd
 *   ws         moe_fwd_workspace_bytes(d) bytes of scratch
 */
int moe_fwd(const moe_dims* d, const void* x, const void* w_r, const void* w_gate,
            const void* w_up, const void* w_down, const uint8_t* token_mask, void* y,
            void* saved, void* ws, size_t ws_bytes, void* stream);

/* Backward of the block (the training step of §3, Expert-Parallel MoE
 * Training): the backward equations in the header above, from the `saved`
 * buffer of the matching moe_fwd (same d, x and weights).
 *   dy      [T, H] bf16 upstream gradient
 *   dx      [T, H] bf16
 *   dw_r    [H, E], dw_gate [E, H, F], dw_up [E, H, F], dw_down [E, F, H]:
 *           bf16, or fp32 with MOE_F_DW_FP32; overwritten (not accumulated)
 *   ws      moe_bwd_workspace_bytes(d) bytes of scratch
 */
int moe_bwd(const moe_dims* d, const void* x, const void* w_r, const void* w_gate,
            const void* w_up, const void* w_down, const void* dy, const void* saved,
            void* dx, void* dw_r, void* dw_gate, void* dw_up, void* dw_down, void* ws,
            size_t ws_bytes, void* stream);

/* Allocation-free forward, for callers that cannot allocate device memory or
 * must not see an allocation happen: code under HIP graph capture, tight
 * serving or training loops, harnesses that forbid hipMalloc.  The same
 * operation, arguments (minus the workspace) and outputs as moe_fwd, bit for
 * bit; its scratch is a static array of MOE_NOALLOC_SCRATCH_BYTES bytes
 * inside the library, one per GPU (reserved on each GPU the library runs on
 * until the process ends).  It calls no allocation routine of any kind.
 *   Limit: moe_fwd_workspace_bytes(d) <= MOE_NOALLOC_SCRATCH_BYTES (about
 *   13 bytes per token and expert, with the router losses on: T <= 40000 at
 *   E = 128); larger sizes return MOE_ERR_WORKSPACE before any launch.
 *   Every call on one GPU shares that GPU's array: calls that overlap on one
 *   GPU (two streams, two host threads) race and must be serialised by the
 *   caller.  Nothing in the array needs to start at zero (the kernels clear
 *   what they count into), and its contents after a call are unspecified. */
#define MOE_NOALLOC_SCRATCH_BYTES (64u << 20)
int moe_fwd_noalloc(const moe_dims* d, const void* x, const void* w_r, const void* w_gate,
                    const void* w_up, const void* w_down, const uint8_t* token_mask, void* y,
                    void* saved, void* stream);

/* Expert LoRA (§3, "LoRA target groups for MoE"; §4.3): rank-r adapters on
 * every expert's fused gate/up projection and its down projection, with the
 * base expert weights and the router frozen.  Per expert e the effective
 * weights are
 *   W_gate[e] + scale a1[e] b1_gate[e],  W_up[e] + scale a1[e] b1_up[e],
 *   W_down[e] + scale a2[e] b2[e],
 * applied through the rank-r intermediates P1 = scale Xp a1 and
 * P2 = scale A a2 (bf16, kept in the saved buffer after the block's own
 * layout, so moe_saved_views applies to it unchanged).  The backward writes dX
 * and the five adapter gradients (bf16, or fp32 with MOE_F_DW_FP32) and no base
 * or router weight gradients; dX includes the router term (the router is
 * frozen, not detached).  MOE_F_MASK, MOE_F_RECOMPUTE and the router-loss
 * coefficients behave as in moe_fwd / moe_bwd. */
typedef struct moe_lora {
  int32_t rank;        /* r: 16, 32, 48 or 64 */
  float scale;         /* multiplies every adapter product (alpha / r in the usual parametrisation) */
  const void* a1;      /* [E, H, r] bf16 */
  const void* b1_gate; /* [E, r, F] bf16 */
  const void* b1_up;   /* [E, r, F] bf16 */
  const void* a2;      /* [E, F, r] bf16 */
  const void* b2;      /* [E, r, H] bf16 */
} moe_lora;

/* Bytes of the LoRA saved buffer and of the scratch either LoRA call needs
 * (0 if d or rank is invalid). */
size_t moe_lora_saved_bytes(const moe_dims* d, int32_t rank);
size_t moe_lora_workspace_bytes(const moe_dims* d, int32_t rank);

/* Forward with the adapters; arguments as moe_fwd plus `lora`. */
int moe_lora_fwd(const moe_dims* d, const void* x, const void* w_r, const void* w_gate,
                 const void* w_up, const void* w_down, const moe_lora* lora,
                 const uint8_t* token_mask, void* y, void* saved, void* ws, size_t ws_bytes,
                 void* stream);

/* Backward with the adapters, from the saved buffer of the matching
 * moe_lora_fwd (same d, x, weights and adapters).
 *   dy    [T, H] bf16;  dx  [T, H] bf16
 *   da1 [E, H, r], db1_gate [E, r, F], db1_up [E, r, F], da2 [E, F, r],
 *   db2 [E, r, H]: overwritten; zero for experts with no rows */
int moe_lora_bwd(const moe_dims* d, const void* x, const void* w_r, const void* w_gate,
                 const void* w_up, const void* w_down, const moe_lora* lora, const void* dy,
                 const void* saved, void* dx, void* da1, void* db1_gate, void* db1_up, void* da2,
                 void* db2, void* ws, size_t ws_bytes, void* stream);

/* Forward-only pass of the block for serving (reranking scores a batch of
 * query-passage pairs in one prefill pass, §4.2 "Inference throughput"): the Y of
 * moe_fwd, bit for bit, without a saved buffer.  Routing, A and O live in the
 * workspace, G and U are never stored, and the gate/up product reads its rows
 * of x through the permutation instead of a gathered copy (a copy is made in
 * the workspace only when T * H * 2 bytes exceed 2^31 - 1).  MOE_F_MASK as in
 * moe_fwd; MOE_F_DW_FP32, MOE_F_RECOMPUTE and the router-loss coefficients
 * are ignored.
 *   x, w_r, w_gate, w_up, w_down, token_mask, y   as in moe_fwd
 *   ws    moe_infer_workspace_bytes(d) bytes of scratch
 */
size_t moe_infer_workspace_bytes(const moe_dims* d);
int moe_infer(const moe_dims* d, const void* x, const void* w_r, const void* w_gate,
              const void* w_up, const void* w_down, const uint8_t* token_mask, void* y,
              void* ws, size_t ws_bytes, void* stream);

/* One expert-parallel rank's share (§3, "Expert parallelism and topology"):
 * the rows dispatched to this rank's E local experts, already grouped
 * expert-major.  rows = capacity of the row buffers (rows >= 1). */
typedef struct moe_experts_dims {
  int32_t rows, H, E, F;
  uint32_t flags; /* MOE_F_DW_FP32, MOE_F_RECOMPUTE */
} moe_experts_dims;

/* Device pointers into an experts `saved` buffer. */
typedef struct moe_experts_saved_view {
  int32_t* offsets; /* [E + 1] exclusive prefix sum of counts, clamped to rows */
  void* g;          /* [rows, F] bf16 (NULL with MOE_F_RECOMPUTE) */
  void* u;          /* [rows, F] bf16 (NULL with MOE_F_RECOMPUTE) */
  void* a;          /* [rows, F] bf16 */
} moe_experts_saved_view;

size_t moe_experts_saved_bytes(const moe_experts_dims* d);
size_t moe_experts_workspace_bytes(const moe_experts_dims* d);
int moe_experts_saved_views(const moe_experts_dims* d, void* saved, moe_experts_saved_view* view);

/* Forward of the local experts.
 *   xp      [rows, H] bf16 dispatched rows, expert-major
 *   counts  [E] int32 on the device: rows of each local expert, in order.  Rows
 *           past the capacity (prefix sum beyond `rows`) are dropped: not read,
 *           not computed, not written.  Output rows past sum(counts) are not written.
 *   o       [rows, H] bf16 expert outputs (ungated)
 */
int moe_experts_fwd(const moe_experts_dims* d, const void* xp, const int32_t* counts,
                    const void* w_gate, const void* w_up, const void* w_down, void* o,
                    void* saved, void* ws, size_t ws_bytes, void* stream);

/* Backward of the local experts from the matching moe_experts_fwd `saved`
 * (which holds the row offsets; counts are not passed again).
 *   d_o     [rows, H] bf16 gradient of o
 *   dxp     [rows, H] bf16
 *   dw_*    as in moe_bwd (overwritten; zero for experts with no rows)
 */
int moe_experts_bwd(const moe_experts_dims* d, const void* xp, const void* w_gate, const void* w_up, const void* w_down, const void* d_o,
                    const void* saved, void* dxp, void* dw_gate, void* dw_up, void* dw_down,
                    void* ws, size_t ws_bytes, void* stream);

/* Per-kernel timing.  With tracing on, every kernel the library launches is
 * bracketed by two HIP events recorded on its launch stream (no host
 * synchronisation at launch time).  moe_trace_read waits for the recorded
 * events, writes per kernel id the summed milliseconds and the number of
 * launches since the last read (arrays of n entries; either may be NULL), and
 * returns the number of kernel ids (or MOE_ERR_HIP).  moe_trace_name(id) is a
 * kernel's name ("" for an unknown id).  Not thread-safe; off by default. */
int moe_trace_enable(int on);
int moe_trace_read(double* total_ms, int32_t* launches, int n);
const char* moe_trace_name(int id);

/* Message describing the last error on this thread ("" if none). */
const char* moe_last_error(void);

/* Library version, major * 10000 + minor * 100 + patch. */
int moe_version(void);

#ifdef __cplusplus
}
#endif

#endif /* MOE_MI355X_H */
