// Weighted combine of the expert outputs, its backward, and the router-logit
// gradient dz.  One wave per token; rows move as 16-byte
// vectors (8 bf16 per lane), sums are fp32 in slot order.
#include "launch.hpp"
#include "trace.hpp"
#include "wgrad_plan.hpp"

namespace moe {

namespace {

__device__ __forceinline__ void unpack8(const uint4& w, float* f) {
  f[0] = lo_bf(w.x);
  f[1] = hi_bf(w.x);
  f[2] = lo_bf(w.y);
  f[3] = hi_bf(w.y);
  f[4] = lo_bf(w.z);
  f[5] = hi_bf(w.z);
  f[6] = lo_bf(w.w);
  f[7] = hi_bf(w.w);
}

__device__ __forceinline__ uint4 pack8(const float* f) {
  return make_uint4(pack_bf16x2(f[0], f[1]), pack_bf16x2(f[2], f[3]), pack_bf16x2(f[4], f[5]),
                    pack_bf16x2(f[6], f[7]));
}

// Slot counts are a compile-time bound KT >= k (a power of two), so every
// lane issues the loads of all of its token's rows before it needs them.

// Chunks per lane per pass: a pass covers kPassCols columns of each row, as
// kU 16-byte chunks per lane 512 columns apart, so a wave asks for up to
// 4 KB of every row at once; at most 32 row chunks stay in registers.
#ifndef MOE_COMBINE_U
#define MOE_COMBINE_U 4
#endif
template <int KT>
constexpr int kChunks = KT * MOE_COMBINE_U <= 32 ? MOE_COMBINE_U : (32 / KT > 0 ? 32 / KT : 1);

// y[t] = sum_j g[t,j] o[row_of[t,j]]  (0 when the token has no rows).  O is
// read once, with non-temporal loads (10% faster than cached ones: the
// stream does not evict the gates and row indices from L2).
template <int KT>
__global__ __launch_bounds__(256) void k_combine(const bf16_t* __restrict__ o, const float* __restrict__ gates,
                                                 const int32_t* __restrict__ row_of, int T, int H, int k,
                                                 bf16_t* __restrict__ y) {
  constexpr int kU = row_chunks<KT, 32>();
  const int lane = threadIdx.x & 63;
  const int t = blockIdx.x * 4 + (threadIdx.x >> 6);
  if (t >= T) return;
  int rows[KT];
  float g[KT];
#pragma unroll
  for (int j = 0; j < KT; ++j) {
    rows[j] = j < k ? row_of[static_cast<int64_t>(t) * k + j] : -1;
    g[j] = j < k ? gates[static_cast<int64_t>(t) * k + j] : 0.0f;
  }
  for (int c0 = lane * 8; c0 < H; c0 += kWave * 8 * kU) {
    uint4 v[KT][kU];
#pragma unroll
    for (int j = 0; j < KT; ++j)
#pragma unroll
      for (int u = 0; u < kU; ++u) {
        const int c = c0 + u * kWave * 8;
        v[j][u] = (rows[j] >= 0 && c < H) ? load_nt(o + static_cast<int64_t>(rows[j]) * H + c) : make_uint4(0, 0, 0, 0);
      }
#pragma unroll
    for (int u = 0; u < kU; ++u) {
      const int c = c0 + u * kWave * 8;
      float acc[8] = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int j = 0; j < KT; ++j) {
        float f[8];
        unpack8(v[j][u], f);
#pragma unroll
        for (int i = 0; i < 8; ++i) acc[i] += g[j] * f[i];
      }
      if (c < H) *reinterpret_cast<uint4*>(y + static_cast<int64_t>(t) * H + c) = pack8(acc);
    }
  }
}

// The weight gradients' schedule, built by one extra workgroup of the
// combine backward (independent work that would cost a launch of its own).
struct PlanArgs {
  const int32_t* offsets = nullptr;
  int E = 0, tpe0 = 0, tpe1 = 0;
  int32_t* plan = nullptr;
};

// dO[r_j] = g_j dY[t] for every routed slot of token t (bf16).
template <int KT>
__global__ __launch_bounds__(256) void k_combine_bwd(const bf16_t* __restrict__ dy, const float* __restrict__ gates,
                                                     const int32_t* __restrict__ row_of, int T, int H, int k,
                                                     bf16_t* __restrict__ d_o, PlanArgs pa) {
  if (static_cast<int>(blockIdx.x) == cdiv(T, 4)) {  // the plan workgroup
    build_wgrad_plan(pa.offsets, pa.E, pa.tpe0, pa.tpe1, pa.plan);
    return;
  }
  constexpr int kU = row_chunks<KT, 32>();
  const int lane = threadIdx.x & 63;
  const int t = blockIdx.x * 4 + (threadIdx.x >> 6);
  if (t >= T) return;
  int rows[KT];
  float g[KT];
#pragma unroll
  for (int j = 0; j < KT; ++j) {
    rows[j] = j < k ? row_of[static_cast<int64_t>(t) * k + j] : -1;
    g[j] = j < k ? gates[static_cast<int64_t>(t) * k + j] : 0.0f;
  }
  if (rows[0] < 0) return;  // a masked token has no rows
  const bf16_t* dyr = dy + static_cast<int64_t>(t) * H;
  for (int c0 = lane * 8; c0 < H; c0 += kWave * 8 * kU) {
    float fy[kU][8];
#pragma unroll
    for (int u = 0; u < kU; ++u) {
      const int c = c0 + u * kWave * 8;
      unpack8(c < H ? *reinterpret_cast<const uint4*>(dyr + c) : make_uint4(0, 0, 0, 0), fy[u]);
    }
#pragma unroll
    for (int j = 0; j < KT; ++j) {
      if (rows[j] < 0) continue;
#pragma unroll
      for (int u = 0; u < kU; ++u) {
        const int c = c0 + u * kWave * 8;
        float out[8];
#pragma unroll
        for (int i = 0; i < 8; ++i) out[i] = g[j] * fy[u][i];
        if (c < H) *reinterpret_cast<uint4*>(d_o + static_cast<int64_t>(rows[j]) * H + c) = pack8(out);
      }
    }
  }
}

// Per token t with rows r_j (one wave per token, lane j holds slot j):
//   dg_j      = <dY[t], O[r_j]>                              (fp32)
//   dz_j      = g_j (dg_j - sum_j' g_j' dg_j')               (fp32, per slot)
//   dz[t, :]  = dz_j at e = idx_j, else 0                    (bf16, all E)
// dg_j comes from the down product's backward instead of a second pass over
// O: with dA = dO W_down^T and dO[r_j] = g_j dY[t], <dA[r_j], A[r_j]> =
// <dO[r_j], A[r_j] W_down> = g_j <dY[t], O[r_j]>.  The down product's dgrad
// writes that inner product per row and column block (part[r][p], p <
// nparts), so dg_j = sum_p part[r_j][p] / g_j, and 0 where g_j = 0 (dz_j is 0
// there either way).
// With the router losses (RouterLossGrad.on) dz[t, :] also takes, for a
// valid token, their gradient with the routing fractions f held constant:
//   aux_coef E / T_v  p_e (f_e - sum_e' f_e' p_e') + z_coef 2 / T_v  lse p_e,
// p the full softmax of the token's fp32 logits, lse their log-normaliser,
// f_e = counts[e] / R, T_v = R / k.
struct RouterLossGrad {
  const float* logits = nullptr;
  const int32_t* counts = nullptr;
  const int32_t* offsets = nullptr;
  float aux_coef = 0.0f, z_coef = 0.0f;
};

constexpr int kMaxPerLane = MOE_MAX_EXPERTS / kWave;

// W_r^T for the router dX, built by extra workgroups of the gate backward
// (independent work; a launch of its own cost more than the copy): tile b
// of (H/32) x (E/32) 32 x 32 tiles, through LDS, w_rt[e][h] = w_r[h][e].
struct WrTranspose {
  const bf16_t* w_r = nullptr;
  bf16_t* w_rt = nullptr;
  int H = 0;
};

__device__ __forceinline__ void transpose_wr_tile(const WrTranspose& tr, int E, int b) {
  __shared__ bf16_t tile[32][33];
  const int th = cdiv(tr.H, 32);
  const int h0 = (b % th) * 32, e0 = (b / th) * 32;
  const int a = threadIdx.x >> 5, c = threadIdx.x & 31;
#pragma unroll
  for (int i = 0; i < 32; i += 8)
    if (h0 + a + i < tr.H && e0 + c < E) tile[a + i][c] = tr.w_r[static_cast<int64_t>(h0 + a + i) * E + e0 + c];
  __syncthreads();
#pragma unroll
  for (int i = 0; i < 32; i += 8)
    if (e0 + a + i < E && h0 + c < tr.H) tr.w_rt[static_cast<int64_t>(e0 + a + i) * tr.H + h0 + c] = tile[c][a + i];
}

template <int KT, bool kAux>
__global__ __launch_bounds__(256) void k_gate_bwd(const float* __restrict__ part, int nparts,
                                                  const float* __restrict__ gates,
                                                  const int32_t* __restrict__ topk_idx,
                                                  const int32_t* __restrict__ row_of, int T, int E, int k,
                                                  float* __restrict__ dg_out, float* __restrict__ dz_slot,
                                                  bf16_t* __restrict__ dz, RouterLossGrad rl, WrTranspose tr) {
  const int gate_blocks = cdiv(T, 4);
  if (static_cast<int>(blockIdx.x) >= gate_blocks) {  // a W_r^T tile (whole workgroup)
    transpose_wr_tile(tr, E, static_cast<int>(blockIdx.x) - gate_blocks);
    return;
  }
  const int lane = threadIdx.x & 63;
  const int t = blockIdx.x * 4 + (threadIdx.x >> 6);
  if (t >= T) return;
  float my_g = 0.0f, my_dg = 0.0f;
  int my_e = -1;
  if (lane < k) {
    const int64_t p = static_cast<int64_t>(t) * k + lane;
    my_g = gates[p];
    my_e = topk_idx[p];
    const int r = row_of[p];
    if (r >= 0) {
      float sum = 0.0f;
      for (int q = 0; q < nparts; ++q) sum += part[static_cast<int64_t>(r) * nparts + q];
      my_dg = my_g != 0.0f ? sum / my_g : 0.0f;
    }
  }
  const bool valid = row_of[static_cast<int64_t>(t) * k] >= 0;  // slot 0 is routed
  const float inner = wave_sum(my_g * my_dg);
  const float my_dz = my_g * (my_dg - inner);
  if (lane < k) {
    dg_out[static_cast<int64_t>(t) * k + lane] = my_dg;
    dz_slot[static_cast<int64_t>(t) * k + lane] = my_dz;
  }
  float extra[kMaxPerLane];
#pragma unroll
  for (int m = 0; m < kMaxPerLane; ++m) extra[m] = 0.0f;
  if constexpr (kAux) {
    if (valid) {
      const float* zr = rl.logits + static_cast<int64_t>(t) * E;
      const int R = rl.offsets[E];
      const float tv = static_cast<float>(R / k);
      float zv[kMaxPerLane], f[kMaxPerLane];
      float mx = -INFINITY;
#pragma unroll
      for (int m = 0; m < kMaxPerLane; ++m) {
        const int e = lane + kWave * m;
        zv[m] = e < E ? zr[e] : -INFINITY;
        f[m] = e < E ? static_cast<float>(rl.counts[e]) / static_cast<float>(R) : 0.0f;
        mx = fmaxf(mx, zv[m]);
      }
      mx = wave_max(mx);
      float p[kMaxPerLane], s = 0.0f;
#pragma unroll
      for (int m = 0; m < kMaxPerLane; ++m) {
        p[m] = lane + kWave * m < E ? expf(zv[m] - mx) : 0.0f;
        s += p[m];
      }
      s = wave_sum(s);
      float fp = 0.0f;
#pragma unroll
      for (int m = 0; m < kMaxPerLane; ++m) {
        p[m] /= s;
        fp += f[m] * p[m];
      }
      fp = wave_sum(fp);
      const float lse = mx + logf(s);
      const float ca = rl.aux_coef * static_cast<float>(E) / tv, cz = rl.z_coef * 2.0f / tv * lse;
#pragma unroll
      for (int m = 0; m < kMaxPerLane; ++m) extra[m] = ca * p[m] * (f[m] - fp) + cz * p[m];
    }
  }
  bf16_t* dzr = dz + static_cast<int64_t>(t) * E;
#pragma unroll
  for (int m = 0; m < kMaxPerLane; ++m) {
    const int e = kWave * m + lane;
    if (kWave * m >= E) break;
    float v = 0.0f;
#pragma unroll
    for (int j = 0; j < KT; ++j) {
      const int ej = __shfl(my_e, j, kWave);
      const float dzj = __shfl(my_dz, j, kWave);
      if (j < k && ej == e) v = dzj;
    }
    if (e < E) dzr[e] = f2bf(v + extra[m]);
  }
}

}  // namespace

#define MOE_SLOT_DISPATCH(KERNEL, k, grid, s, ...)                                        \
  do {                                                                                     \
    if ((k) <= 1) hipLaunchKernelGGL(KERNEL<1>, grid, dim3(256), 0, s, __VA_ARGS__);       \
    else if ((k) <= 2) hipLaunchKernelGGL(KERNEL<2>, grid, dim3(256), 0, s, __VA_ARGS__);  \
    else if ((k) <= 4) hipLaunchKernelGGL(KERNEL<4>, grid, dim3(256), 0, s, __VA_ARGS__);  \
    else if ((k) <= 8) hipLaunchKernelGGL(KERNEL<8>, grid, dim3(256), 0, s, __VA_ARGS__);  \
    else if ((k) <= 16) hipLaunchKernelGGL(KERNEL<16>, grid, dim3(256), 0, s, __VA_ARGS__); \
    else hipLaunchKernelGGL(KERNEL<32>, grid, dim3(256), 0, s, __VA_ARGS__);               \
  } while (0)
#define MOE_SLOT_DISPATCH2(KERNEL, B, k, grid, s, ...)                                               \
  do {                                                                                                \
    if ((k) <= 1) hipLaunchKernelGGL((KERNEL<1, B>), grid, dim3(256), 0, s, __VA_ARGS__);             \
    else if ((k) <= 2) hipLaunchKernelGGL((KERNEL<2, B>), grid, dim3(256), 0, s, __VA_ARGS__);        \
    else if ((k) <= 4) hipLaunchKernelGGL((KERNEL<4, B>), grid, dim3(256), 0, s, __VA_ARGS__);        \
    else if ((k) <= 8) hipLaunchKernelGGL((KERNEL<8, B>), grid, dim3(256), 0, s, __VA_ARGS__);        \
    else if ((k) <= 16) hipLaunchKernelGGL((KERNEL<16, B>), grid, dim3(256), 0, s, __VA_ARGS__);      \
    else hipLaunchKernelGGL((KERNEL<32, B>), grid, dim3(256), 0, s, __VA_ARGS__);                     \
  } while (0)

hipError_t launch_combine(const bf16_t* o, const float* gates, const int32_t* row_of, int T, int H,
                          int k, bf16_t* y, hipStream_t s) {
  {
    TraceScope trace_scope(K_COMBINE, s);
    MOE_SLOT_DISPATCH(k_combine, k, dim3(cdiv(T, 4)), s, o, gates, row_of, T, H, k, y);
  }
  return hipGetLastError();
}

hipError_t launch_combine_bwd(const bf16_t* dy, const float* gates, const int32_t* row_of, int T, int H, int k,
                              bf16_t* d_o, hipStream_t s, const int32_t* offsets, int E, int F, int32_t* plan) {
  PlanArgs pa;
  if (plan != nullptr) {
    pa.offsets = offsets;
    pa.E = E;
    pa.plan = plan;
    wgrad_tiles_per_expert(H, F, pa.tpe0, pa.tpe1);
  }
  {
    TraceScope trace_scope(K_COMBINE_BWD, s);
    MOE_SLOT_DISPATCH(k_combine_bwd, k, dim3(cdiv(T, 4) + (plan != nullptr ? 1 : 0)), s, dy, gates, row_of, T, H, k,
                      d_o, pa);
  }
  return hipGetLastError();
}

hipError_t launch_gate_bwd(const float* part, int nparts, const float* gates, const int32_t* topk_idx,
                           const int32_t* row_of, int T, int E, int k, float* dg, float* dz_slot, bf16_t* dz,
                           const float* logits, const int32_t* counts, const int32_t* offsets, float aux_coef,
                           float z_coef, const bf16_t* w_r, int H, bf16_t* w_rt, hipStream_t s) {
  WrTranspose tr;
  int tr_blocks = 0;
  if (w_r != nullptr) {
    tr.w_r = w_r;
    tr.w_rt = w_rt;
    tr.H = H;
    tr_blocks = cdiv(H, 32) * cdiv(E, 32);
  }
  const dim3 grid(cdiv(T, 4) + tr_blocks);
  RouterLossGrad rl;
  const bool aux = aux_coef != 0.0f || z_coef != 0.0f;
  if (aux) {
    rl.logits = logits;
    rl.counts = counts;
    rl.offsets = offsets;
    rl.aux_coef = aux_coef;
    rl.z_coef = z_coef;
  }
  {
    TraceScope trace_scope(K_GATE_BWD, s);
    if (aux)
      MOE_SLOT_DISPATCH2(k_gate_bwd, true, k, grid, s, part, nparts, gates, topk_idx, row_of, T, E, k, dg, dz_slot, dz,
                         rl, tr);
    else
      MOE_SLOT_DISPATCH2(k_gate_bwd, false, k, grid, s, part, nparts, gates, topk_idx, row_of, T, E, k, dg, dz_slot,
                         dz, rl, tr);
  }
  return hipGetLastError();
}

}  // namespace moe
