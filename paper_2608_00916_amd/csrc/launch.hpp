// Internal launchers of the MoE kernels (host side).  Not part of the C ABI.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "common.hpp"
#include "moe.h"

namespace moe {

// Row passes of the one-wave-per-token kernels (combine, its backward, the
// router dX): a pass covers up to 4 KB of each of the token's KT rows, as
// 16-byte chunks per lane 512 columns apart, with at most kBudget row chunks
// held in registers per lane.
template <int KT, int kBudget>
constexpr int row_chunks() {
  return 4 * KT <= kBudget ? 4 : (kBudget / KT > 0 ? kBudget / KT : 1);
}

// Rank-r adapters on every expert's gate/up and down projections (rank 0:
// none): a1 [E,H,r], b1_gate / b1_up [E,r,F], a2 [E,F,r], b2 [E,r,H], and the
// scale-multiplied rank-r intermediates P1 = scale Xp a1, P2 = scale A a2
// ([rows_cap][r], written by the forward, read by the backward).
struct LoraArgs {
  int rank = 0;
  float scale = 0.0f;
  const bf16_t* a1 = nullptr;
  const bf16_t* b1_gate = nullptr;
  const bf16_t* b1_up = nullptr;
  const bf16_t* a2 = nullptr;
  const bf16_t* b2 = nullptr;
  bf16_t* p1 = nullptr;
  bf16_t* p2 = nullptr;
};

// Operands of the grouped expert products.  Rows are grouped expert-major;
// offsets[E+1] and tile_start[E+1] (prefix sums of rows and of 128-row tiles
// per expert) and tile_desc[tile_start[E]] (per 128-row tile: first row,
// expert | rows << 8) are device arrays.
struct ExpertArgs {
  int rows_cap, H, E, F;
  const bf16_t* xp;
  const bf16_t* w_gate;
  const bf16_t* w_up;
  const bf16_t* w_down;
  const int32_t* offsets;
  const int32_t* tile_start;
  const int2* tile_desc;
  bf16_t* g;    // forward writes, backward reads
  bf16_t* u;
  bf16_t* act;  // A = silu(G) * U
  // Gate/up forward only: when non-null, product row r reads row xp_rows[r]
  // of xp (then the unpermuted tokens, xp_bytes < 2^31 bytes in all).
  const int32_t* xp_rows = nullptr;
  int64_t xp_bytes = 0;
  // Down product's dgrad only: when non-null, it also writes
  // dgate_part[r][p] = <dA[r], A[r]> over its column block p
  // (dgate_parts(F) blocks; A = silu(G) U in fp32).
  float* dgate_part = nullptr;
  // Weight gradients only: their schedule, built on the device per backward
  // (wgrad_plan_ints(E) ints); launch_experts_bwd_data builds it unless an
  // earlier kernel of the backward already has (wgrad_plan_built).
  int32_t* wgrad_plan = nullptr;
  bool wgrad_plan_built = false;
  LoraArgs lora;
};

int max_row_tiles(int rows_cap, int E);
// Ints of the weight gradients' schedule (ExpertArgs::wgrad_plan), and the
// tiles per expert of the down and gate/up weight gradients it schedules.
int wgrad_plan_ints(int E);
void wgrad_tiles_per_expert(int H, int F, int& tpe_down, int& tpe_gu);
// Column blocks of the down product's dgrad (the dgate_part row length).
int dgate_parts(int F);

// G, U, A from Xp (gate/up products + SwiGLU); G and U are skipped when
// a.g is null, A when a.act is.  `recompute` only names the launch in traces
// (the backward's recomputation of G and U).
hipError_t launch_gateup_fwd(const ExpertArgs& a, hipStream_t s, bool recompute = false);
// O = A W_down per expert.
hipError_t launch_down_fwd(const ExpertArgs& a, bf16_t* o, hipStream_t s);
// dG, dU, dXp and the three weight gradients from dO.
hipError_t launch_experts_bwd(const ExpertArgs& a, const bf16_t* d_o, bf16_t* dg, bf16_t* du,
                              bf16_t* dxp, void* dw_gate, void* dw_up, void* dw_down, bool dw_f32,
                              hipStream_t s);
// dG, dU (dA += Q2 a2^T with adapters: q2 non-null) and dXp (+= Q1 a1^T: q1).
hipError_t launch_down_dgrad(const ExpertArgs& a, const bf16_t* d_o, bf16_t* dg, bf16_t* du, const bf16_t* q2,
                             hipStream_t s);
hipError_t launch_gateup_dgrad(const ExpertArgs& a, const bf16_t* dg, const bf16_t* du, bf16_t* dxp,
                               const bf16_t* q1, hipStream_t s);
// Rank-r intermediates: out[r][q] = scale sum_s X_s[r] W_s[e](:, q), X_s
// [rows][K] (ld ldx), W_s per expert (estride apart) [K][rank] or, b_kc,
// [rank][K]; x1/w1 a second segment or null.
hipError_t launch_lora_rows(const ExpertArgs& a, const bf16_t* x0, const bf16_t* x1, int64_t ldx,
                            const bf16_t* w0, const bf16_t* w1, int64_t estride, int K, bool b_kc, bf16_t* out,
                            hipStream_t s);
// Adapter gradients out[e] = X_e^T Y_e (X [rows][M], Y [rows][rank]) stored
// [E][M][rank] or, trans, [E][rank][M]; bf16 or fp32.
hipError_t launch_lora_wgrad(const ExpertArgs& a, const bf16_t* x, int64_t ldx, int M, const bf16_t* y, bool trans,
                             void* out, bool f32, hipStream_t s);
// The same in two parts, so that work can be queued between them: dG, dU,
// dW_down and dXp (dxp may alias d_o: it is written last) ...
hipError_t launch_experts_bwd_data(const ExpertArgs& a, const bf16_t* d_o, bf16_t* dg, bf16_t* du,
                                   bf16_t* dxp, void* dw_down, bool dw_f32, hipStream_t s);
// ... then dW_gate and dW_up.
hipError_t launch_experts_bwd_gateup_w(const ExpertArgs& a, const bf16_t* dg, const bf16_t* du, void* dw_gate,
                                       void* dw_up, bool dw_f32, hipStream_t s);

// Tokens per chunk of the permutation's counting sort.
constexpr int kPermChunk = 256;

// ---- static scratch (noalloc.hip)
// Device address of the current device's static scratch array (the
// allocation-free forward's workspace, MOE_NOALLOC_SCRATCH_BYTES bytes),
// looked up on the first call on each device and cached.
hipError_t static_scratch(void** ptr, size_t* bytes);

// ---- routing (router.hip)
// logits[T,E] = x W_r (fp32); then per token the top-k experts and gates.
// `part` (router_part_floats(T, E) floats) holds the partial sums of the
// K-split logits product.  With aux_ws (router_loss_ws_floats(T, E) floats)
// also the per-workgroup partial sums of the router losses.  For the
// permutation it also writes chunk_counts[c][e] (permute_ws_ints(T, E)
// ints: rows of expert e among the tokens of chunk c, kPermChunk tokens per
// chunk; integer atomic adds, so exact in any order) and sets
// row_token[0, T k) to -1.
hipError_t launch_router_fwd(const bf16_t* x, const bf16_t* w_r, const uint8_t* mask, int T, int H,
                             int E, int k, float* logits, float* part, int32_t* topk_idx, float* gates,
                             float* aux_ws, int32_t* chunk_counts, int32_t* row_token, hipStream_t s);
int64_t router_part_floats(int T, int E);
int64_t router_loss_ws_floats(int T, int E);
// out[0..1] = {L_aux, L_z} from those partial sums and the routing counts.
hipError_t launch_router_loss(const float* aux_ws, int T, int E, int k, const int32_t* counts,
                              const int32_t* offsets, float aux_coef, float z_coef, float* out, hipStream_t s);

// ---- permutation (permute.hip)
// Workspace ints the permutation needs for T tokens and E experts.
int64_t permute_ws_ints(int T, int E);
// counts, offsets, tile_start, row_token (-1 beyond R), row_of from topk_idx
// and the chunk counts in ws that launch_router_fwd left (with row_token
// already -1); then xp[r] = x[row_token[r]], written token-major through
// row_of (skipped when xp is null).
hipError_t launch_permute(const int32_t* topk_idx, const bf16_t* x, int T, int H, int E, int k,
                          int32_t* counts, int32_t* offsets, int32_t* tile_start, int2* tile_desc,
                          int32_t* row_token, int32_t* row_of, bf16_t* xp, int32_t* ws, hipStream_t s);
// offsets (clamped to rows), tile_start and tile_desc from device counts
// (experts path).
hipError_t launch_offsets_from_counts(const int32_t* counts, int E, int rows, int32_t* offsets,
                                      int32_t* tile_start, int2* tile_desc, hipStream_t s);

// ---- combine (combine.hip)
// y[t] = sum_j gates[t,j] o[row_of[t,j]] (0 for masked tokens).
hipError_t launch_combine(const bf16_t* o, const float* gates, const int32_t* row_of, int T, int H,
                          int k, bf16_t* y, hipStream_t s);
// dO[row_of[t,j]] = g dY[t] for every routed slot.  With `plan` non-null,
// one more workgroup of the same launch also builds the weight gradients'
// schedule from `offsets` (E experts, tiles per expert of H x F gradients).
hipError_t launch_combine_bwd(const bf16_t* dy, const float* gates, const int32_t* row_of, int T, int H, int k,
                              bf16_t* d_o, hipStream_t s, const int32_t* offsets = nullptr, int E = 0, int F = 0,
                              int32_t* plan = nullptr);
// After the down product's dgrad (which leaves part[r][0..nparts), the inner
// products <dA[r], A[r]> per column block): dg = <dY[t], O[row]> = sum / g,
// dz per slot (fp32 [T,k]) and dense over E (bf16 [T,E]).  With a non-zero
// router-loss coefficient the dense dz also takes the router losses' gradient
// (from the fp32 logits, the counts and offsets); dz per slot stays the gates'
// part.  With w_r non-null the same launch also writes w_rt = W_r^T ([E,H],
// from W_r [H,E]) for the router dX, in workgroups of its own.
hipError_t launch_gate_bwd(const float* part, int nparts, const float* gates, const int32_t* topk_idx,
                           const int32_t* row_of, int T, int E, int k, float* dg, float* dz_slot, bf16_t* dz,
                           const float* logits, const int32_t* counts, const int32_t* offsets, float aux_coef,
                           float z_coef, const bf16_t* w_r, int H, bf16_t* w_rt, hipStream_t s);

// ---- router backward (router_bwd.hip)
int dwr_splits(int T);
// dW_r = x^T dz via `dwr_splits(T)` fp32 partials in ws_f32 ([splits][H][E]).
hipError_t launch_dwr(const bf16_t* x, const bf16_t* dz, int T, int H, int E, float* ws_f32,
                      void* dw_r, bool f32_out, hipStream_t s);
// dX[t] = sum_j (dXp[row_of[t,j]] + dz_j W_r[:, idx_j]), with W_r^T in w_rt
// ([E,H], written by launch_gate_bwd).  With dz_dense (bf16 [T,E]) the router
// term is dz_dense W_r^T instead, formed in `dense` (fp32 [T,H] scratch) by an
// MFMA product from w_r, and w_rt is not read.
hipError_t launch_router_dx(const float* dz_slot, const int32_t* topk_idx, const bf16_t* w_r,
                            const bf16_t* dxp, const int32_t* row_of, int T, int H, int E, int k,
                            const bf16_t* w_rt, bf16_t* dx, const bf16_t* dz_dense, float* dense, hipStream_t s);

}  // namespace moe
