// Grouped (per-expert) bf16 MFMA GEMMs of the MoE block, forward and backward.
//
// Rows are grouped expert-major: expert e owns rows [offsets[e], offsets[e+1]).
// Products over the rows of one expert (gate/up, down, and their input
// gradients) walk a device-built table tile_start[E+1] of 128-row tiles, so the
// host never learns the counts: they run as persistent grids (a few workgroups
// per CU) that stride over the tiles the table holds.  Weight gradients
// (K = rows of one expert) have a fixed grid of E x (M/128) x (N/128) tiles;
// experts without rows write zeros.
#include "launch.hpp"
#include "trace.hpp"
#include "gemm_core.hpp"

#include <algorithm>

namespace moe {

namespace {

struct MTile {
  int e, m0, m_lim, n0;
};

// Run body(tile) for every (expert, row tile, column tile) of a grouped
// product with n_ntiles column tiles.  Tile i*gridDim + xcd_tile(block) goes
// to this workgroup in round i, so each XCD works on a contiguous run of tiles.
template <typename Body>
__device__ __forceinline__ void for_each_grouped_tile(const int32_t* offsets, const int32_t* tile_start,
                                                      int E, int n_ntiles, Body&& body) {
  const int total = tile_start[E] * n_ntiles;
  for (int logical = xcd_tile(blockIdx.x, gridDim.x); logical < total; logical += gridDim.x) {
    const int mt = logical / n_ntiles, nt = logical - mt * n_ntiles;
    MTile t;
    t.e = find_group(tile_start, E, mt);
    t.m0 = offsets[t.e] + (mt - tile_start[t.e]) * BM;
    t.m_lim = min(BM, offsets[t.e + 1] - t.m0);
    t.n0 = nt * BN;
    body(t);
  }
}

// G = Xp W_gate[e], U = Xp W_up[e], A = silu(G) * U  (K = H, N = F).
__global__ __launch_bounds__(kThreads) void k_gateup_fwd(const bf16_t* __restrict__ xp,
                                                         const bf16_t* __restrict__ w_gate,
                                                         const bf16_t* __restrict__ w_up,
                                                         const int32_t* __restrict__ offsets,
                                                         const int32_t* __restrict__ tile_start, int E,
                                                         int H, int F, bf16_t* __restrict__ g_out,
                                                         bf16_t* __restrict__ u_out,
                                                         bf16_t* __restrict__ a_out) {
  __shared__ __attribute__((aligned(16))) char smem[mainloop_lds_bytes<2>()];
  for_each_grouped_tile(offsets, tile_start, E, F / BN, [&](const MTile& t) {
  f32x4 acc[2][FM][FN];
  zero_acc<2>(acc);
  const int64_t wofs = static_cast<int64_t>(t.e) * H * F + t.n0;
  const bf16_t* bs[2] = {w_gate + wofs, w_up + wofs};
  gemm_mainloop<true, false, 2>(xp + static_cast<int64_t>(t.m0) * H, H, t.m_lim, bs, F, F - t.n0, H,
                                smem, acc);
  const int lane = threadIdx.x & 63;
#pragma unroll
  for (int mi = 0; mi < FM; ++mi) {
    const int r = frag_row(mi, lane);
    if (r >= t.m_lim) continue;
    const int64_t base = static_cast<int64_t>(t.m0 + r) * F + t.n0;
#pragma unroll
    for (int ni = 0; ni < FN; ++ni) {
      const int c = frag_col(ni, lane);
      const f32x4 gv = acc[0][mi][ni], uv = acc[1][mi][ni];
      f32x4 av;
#pragma unroll
      for (int i = 0; i < 4; ++i) av[i] = silu_f(gv[i]) * uv[i];
      *reinterpret_cast<uint2*>(g_out + base + c) = pack4_bf16(gv);
      *reinterpret_cast<uint2*>(u_out + base + c) = pack4_bf16(uv);
      *reinterpret_cast<uint2*>(a_out + base + c) = pack4_bf16(av);
    }
  }
  });
}

// O = A W_down[e]  (K = F, N = H).
__global__ __launch_bounds__(kThreads) void k_down_fwd(const bf16_t* __restrict__ act,
                                                       const bf16_t* __restrict__ w_down,
                                                       const int32_t* __restrict__ offsets,
                                                       const int32_t* __restrict__ tile_start, int E,
                                                       int H, int F, bf16_t* __restrict__ o_out) {
  __shared__ __attribute__((aligned(16))) char smem[mainloop_lds_bytes<1>()];
  for_each_grouped_tile(offsets, tile_start, E, H / BN, [&](const MTile& t) {
  f32x4 acc[1][FM][FN];
  zero_acc<1>(acc);
  const bf16_t* bs[1] = {w_down + static_cast<int64_t>(t.e) * F * H + t.n0};
  gemm_mainloop<true, false, 1>(act + static_cast<int64_t>(t.m0) * F, F, t.m_lim, bs, H, H - t.n0, F,
                                smem, acc);
  const int lane = threadIdx.x & 63;
#pragma unroll
  for (int mi = 0; mi < FM; ++mi) {
    const int r = frag_row(mi, lane);
    if (r >= t.m_lim) continue;
    const int64_t base = static_cast<int64_t>(t.m0 + r) * H + t.n0;
#pragma unroll
    for (int ni = 0; ni < FN; ++ni)
      *reinterpret_cast<uint2*>(o_out + base + frag_col(ni, lane)) = pack4_bf16(acc[0][mi][ni]);
  }
  });
}

// dA = dO W_down[e]^T (K = H, N = F) fused with the SwiGLU backward:
// s = sigmoid(G); dG = dA U s (1 + G (1 - s)); dU = dA G s.
__global__ __launch_bounds__(kThreads) void k_down_dgrad_swiglu(
    const bf16_t* __restrict__ d_o, const bf16_t* __restrict__ w_down, const bf16_t* __restrict__ g_in,
    const bf16_t* __restrict__ u_in, const int32_t* __restrict__ offsets,
    const int32_t* __restrict__ tile_start, int E, int H, int F, bf16_t* __restrict__ dg_out,
    bf16_t* __restrict__ du_out) {
  __shared__ __attribute__((aligned(16))) char smem[mainloop_lds_bytes<1>()];
  for_each_grouped_tile(offsets, tile_start, E, F / BN, [&](const MTile& t) {
  f32x4 acc[1][FM][FN];
  zero_acc<1>(acc);
  // B(k = h, n = f) = W_down[e][f][h]: K-contiguous rows of W_down.
  const bf16_t* bs[1] = {w_down + static_cast<int64_t>(t.e) * F * H + static_cast<int64_t>(t.n0) * H};
  gemm_mainloop<true, true, 1>(d_o + static_cast<int64_t>(t.m0) * H, H, t.m_lim, bs, H, F - t.n0, H,
                               smem, acc);
  const int lane = threadIdx.x & 63;
#pragma unroll
  for (int mi = 0; mi < FM; ++mi) {
    const int r = frag_row(mi, lane);
    if (r >= t.m_lim) continue;
    const int64_t base = static_cast<int64_t>(t.m0 + r) * F + t.n0;
#pragma unroll
    for (int ni = 0; ni < FN; ++ni) {
      const int c = frag_col(ni, lane);
      const uint2 gw = *reinterpret_cast<const uint2*>(g_in + base + c);
      const uint2 uw = *reinterpret_cast<const uint2*>(u_in + base + c);
      const float gv[4] = {lo_bf(gw.x), hi_bf(gw.x), lo_bf(gw.y), hi_bf(gw.y)};
      const float uv[4] = {lo_bf(uw.x), hi_bf(uw.x), lo_bf(uw.y), hi_bf(uw.y)};
      f32x4 dgv, duv;
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const float da = acc[0][mi][ni][i];
        const float s = sigmoid_f(gv[i]);
        dgv[i] = da * uv[i] * s * (1.0f + gv[i] * (1.0f - s));
        duv[i] = da * gv[i] * s;
      }
      *reinterpret_cast<uint2*>(dg_out + base + c) = pack4_bf16(dgv);
      *reinterpret_cast<uint2*>(du_out + base + c) = pack4_bf16(duv);
    }
  }
  });
}

// dXp = dG W_gate[e]^T + dU W_up[e]^T  (K = 2F in two segments, N = H).
__global__ __launch_bounds__(kThreads) void k_gateup_dgrad(
    const bf16_t* __restrict__ dg_in, const bf16_t* __restrict__ du_in, const bf16_t* __restrict__ w_gate,
    const bf16_t* __restrict__ w_up, const int32_t* __restrict__ offsets,
    const int32_t* __restrict__ tile_start, int E, int H, int F, bf16_t* __restrict__ dxp_out) {
  __shared__ __attribute__((aligned(16))) char smem[mainloop_lds_bytes<1>()];
  for_each_grouped_tile(offsets, tile_start, E, H / BN, [&](const MTile& t) {
  f32x4 acc[1][FM][FN];
  zero_acc<1>(acc);
  // B(k = f, n = h) = W[e][h][f]: K-contiguous rows of W_gate / W_up.
  const int64_t wofs = static_cast<int64_t>(t.e) * H * F + static_cast<int64_t>(t.n0) * F;
  const int64_t aofs = static_cast<int64_t>(t.m0) * F;
  const bf16_t* bg[1] = {w_gate + wofs};
  gemm_mainloop<true, true, 1>(dg_in + aofs, F, t.m_lim, bg, F, H - t.n0, F, smem, acc);
  const bf16_t* bu[1] = {w_up + wofs};
  gemm_mainloop<true, true, 1>(du_in + aofs, F, t.m_lim, bu, F, H - t.n0, F, smem, acc);
  const int lane = threadIdx.x & 63;
#pragma unroll
  for (int mi = 0; mi < FM; ++mi) {
    const int r = frag_row(mi, lane);
    if (r >= t.m_lim) continue;
    const int64_t base = static_cast<int64_t>(t.m0 + r) * H + t.n0;
#pragma unroll
    for (int ni = 0; ni < FN; ++ni)
      *reinterpret_cast<uint2*>(dxp_out + base + frag_col(ni, lane)) = pack4_bf16(acc[0][mi][ni]);
  }
  });
}

template <bool F32>
__device__ __forceinline__ void store4(void* out, int64_t idx, const f32x4& v) {
  if constexpr (F32)
    *reinterpret_cast<float4*>(static_cast<float*>(out) + idx) = make_float4(v[0], v[1], v[2], v[3]);
  else
    *reinterpret_cast<uint2*>(static_cast<bf16_t*>(out) + idx) = pack4_bf16(v);
}

// Weight-gradient tile: expert e, rows [m0, m0+128) of an M x N gradient.
struct WTile {
  int e, m0, n0;
};
__device__ __forceinline__ WTile wgrad_tile(int M, int N) {
  const int logical = xcd_tile(blockIdx.x, gridDim.x);
  const int nm = M / BM, nn = N / BN;
  WTile t;
  t.e = logical / (nm * nn);
  const int rem = logical - t.e * nm * nn;
  t.m0 = (rem / nn) * BM;
  t.n0 = (rem % nn) * BN;
  return t;
}

// dW_down[e] (F x H) = A_e^T dO_e, K = rows of expert e.
template <bool F32>
__global__ __launch_bounds__(kThreads) void k_down_wgrad(const bf16_t* __restrict__ act,
                                                         const bf16_t* __restrict__ d_o,
                                                         const int32_t* __restrict__ offsets, int E,
                                                         int H, int F, void* __restrict__ dw_down) {
  __shared__ __attribute__((aligned(16))) char smem[mainloop_lds_bytes<1>()];
  const WTile t = wgrad_tile(F, H);
  if (t.e >= E) return;
  const int r0 = offsets[t.e], n_rows = offsets[t.e + 1] - r0;
  f32x4 acc[1][FM][FN];
  zero_acc<1>(acc);
  const bf16_t* bs[1] = {d_o + static_cast<int64_t>(r0) * H + t.n0};
  gemm_mainloop<false, false, 1>(act + static_cast<int64_t>(r0) * F + t.m0, F, BM, bs, H, BN, n_rows,
                                 smem, acc);
  const int lane = threadIdx.x & 63;
  const int64_t obase = static_cast<int64_t>(t.e) * F * H;
#pragma unroll
  for (int mi = 0; mi < FM; ++mi) {
    const int64_t row = obase + static_cast<int64_t>(t.m0 + frag_row(mi, lane)) * H + t.n0;
#pragma unroll
    for (int ni = 0; ni < FN; ++ni) store4<F32>(dw_down, row + frag_col(ni, lane), acc[0][mi][ni]);
  }
}

// dW_gate[e] = Xp_e^T dG_e, dW_up[e] = Xp_e^T dU_e  (H x F each, K = rows).
template <bool F32>
__global__ __launch_bounds__(kThreads) void k_gateup_wgrad(const bf16_t* __restrict__ xp,
                                                           const bf16_t* __restrict__ dg_in,
                                                           const bf16_t* __restrict__ du_in,
                                                           const int32_t* __restrict__ offsets, int E,
                                                           int H, int F, void* __restrict__ dw_gate,
                                                           void* __restrict__ dw_up) {
  __shared__ __attribute__((aligned(16))) char smem[mainloop_lds_bytes<2>()];
  const WTile t = wgrad_tile(H, F);
  if (t.e >= E) return;
  const int r0 = offsets[t.e], n_rows = offsets[t.e + 1] - r0;
  f32x4 acc[2][FM][FN];
  zero_acc<2>(acc);
  const int64_t bofs = static_cast<int64_t>(r0) * F + t.n0;
  const bf16_t* bs[2] = {dg_in + bofs, du_in + bofs};
  gemm_mainloop<false, false, 2>(xp + static_cast<int64_t>(r0) * H + t.m0, H, BM, bs, F, BN, n_rows,
                                 smem, acc);
  const int lane = threadIdx.x & 63;
  const int64_t obase = static_cast<int64_t>(t.e) * H * F;
#pragma unroll
  for (int mi = 0; mi < FM; ++mi) {
    const int64_t row = obase + static_cast<int64_t>(t.m0 + frag_row(mi, lane)) * F + t.n0;
#pragma unroll
    for (int ni = 0; ni < FN; ++ni) {
      store4<F32>(dw_gate, row + frag_col(ni, lane), acc[0][mi][ni]);
      store4<F32>(dw_up, row + frag_col(ni, lane), acc[1][mi][ni]);
    }
  }
}

inline int grid8(int64_t n) { return static_cast<int>(cdiv64(n, 8) * 8); }

// Persistent grid: as many workgroups as can be resident on the device at
// once (queried per kernel and device, then cached), rounded down to a
// multiple of 8, and no more than the worst-case tile count needs.
template <typename Kernel>
int persistent_grid(Kernel kernel, int64_t max_tiles) {
  constexpr int kMaxDev = 64;
  static int cached[kMaxDev] = {0};
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDev) dev = 0;
  if (cached[dev] == 0) {
    int cus = 0, per_cu = 0;
    if (hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || cus <= 0)
      cus = 256;
    if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, kernel, kThreads, 0) != hipSuccess ||
        per_cu <= 0)
      per_cu = 1;
    cached[dev] = std::max(8, (cus * per_cu) / 8 * 8);
  }
  return static_cast<int>(std::min<int64_t>(grid8(max_tiles), cached[dev]));
}

}  // namespace

// Upper bound of the number of 128-row tiles over all experts.
int max_row_tiles(int rows_cap, int E) { return cdiv(rows_cap, BM) + E; }

hipError_t launch_gateup_fwd(const ExpertArgs& a, hipStream_t s) {
  const int grid =
      persistent_grid(k_gateup_fwd, static_cast<int64_t>(max_row_tiles(a.rows_cap, a.E)) * (a.F / BN));
  {
    TraceScope trace_scope(K_GATEUP_FWD, s);
    hipLaunchKernelGGL(k_gateup_fwd, dim3(grid), dim3(kThreads), 0, s, a.xp, a.w_gate, a.w_up, a.offsets,
                       a.tile_start, a.E, a.H, a.F, a.g, a.u, a.act);
  }
  return hipGetLastError();
}

hipError_t launch_down_fwd(const ExpertArgs& a, bf16_t* o, hipStream_t s) {
  const int grid =
      persistent_grid(k_down_fwd, static_cast<int64_t>(max_row_tiles(a.rows_cap, a.E)) * (a.H / BN));
  {
    TraceScope trace_scope(K_DOWN_FWD, s);
    hipLaunchKernelGGL(k_down_fwd, dim3(grid), dim3(kThreads), 0, s, a.act, a.w_down, a.offsets,
                       a.tile_start, a.E, a.H, a.F, o);
  }
  return hipGetLastError();
}

hipError_t launch_experts_bwd(const ExpertArgs& a, const bf16_t* d_o, bf16_t* dg, bf16_t* du,
                              bf16_t* dxp, void* dw_gate, void* dw_up, void* dw_down, bool dw_f32,
                              hipStream_t s) {
  const int64_t tiles = max_row_tiles(a.rows_cap, a.E);
  {
    TraceScope trace_scope(K_DOWN_DGRAD, s);
    hipLaunchKernelGGL(k_down_dgrad_swiglu, dim3(persistent_grid(k_down_dgrad_swiglu, tiles * (a.F / BN))),
                       dim3(kThreads), 0, s, d_o, a.w_down, a.g, a.u, a.offsets, a.tile_start, a.E, a.H,
                       a.F, dg, du);
  }
  const int gw_down = grid8(static_cast<int64_t>(a.E) * (a.F / BM) * (a.H / BN));
  if (dw_f32) {
    TraceScope trace_scope(K_DOWN_WGRAD, s);
    hipLaunchKernelGGL(k_down_wgrad<true>, dim3(gw_down), dim3(kThreads), 0, s, a.act, d_o, a.offsets,
                       a.E, a.H, a.F, dw_down);
  } else {
    TraceScope trace_scope(K_DOWN_WGRAD, s);
    hipLaunchKernelGGL(k_down_wgrad<false>, dim3(gw_down), dim3(kThreads), 0, s, a.act, d_o, a.offsets,
                       a.E, a.H, a.F, dw_down);
  }
  {
    TraceScope trace_scope(K_GATEUP_DGRAD, s);
    hipLaunchKernelGGL(k_gateup_dgrad, dim3(persistent_grid(k_gateup_dgrad, tiles * (a.H / BN))),
                       dim3(kThreads), 0, s, dg, du, a.w_gate, a.w_up, a.offsets, a.tile_start, a.E, a.H,
                       a.F, dxp);
  }
  const int gw_gu = grid8(static_cast<int64_t>(a.E) * (a.H / BM) * (a.F / BN));
  if (dw_f32) {
    TraceScope trace_scope(K_GATEUP_WGRAD, s);
    hipLaunchKernelGGL(k_gateup_wgrad<true>, dim3(gw_gu), dim3(kThreads), 0, s, a.xp, dg, du, a.offsets,
                       a.E, a.H, a.F, dw_gate, dw_up);
  } else {
    TraceScope trace_scope(K_GATEUP_WGRAD, s);
    hipLaunchKernelGGL(k_gateup_wgrad<false>, dim3(gw_gu), dim3(kThreads), 0, s, a.xp, dg, du,
                       a.offsets, a.E, a.H, a.F, dw_gate, dw_up);
  }
  return hipGetLastError();
}

}  // namespace moe
