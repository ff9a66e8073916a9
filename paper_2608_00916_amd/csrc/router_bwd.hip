// Router backward of the MoE block: dW_r = x^T dz (split over tokens into
// fp32 partials reduced in a fixed order) and dX = (sum of the permuted-row
// gradients of the token) + dz W_r^T, where dz has only the k selected
// experts non-zero, so its product with W_r^T is k scaled rows of W_r^T.
#include <algorithm>

#include "gemm_core.hpp"
#include "launch.hpp"
#include "trace.hpp"

namespace moe {

namespace {

constexpr int kDwrChunk = 512;  // tokens per split of dW_r
using RTile = Tile<128, 128, 1>;

// partial[s][H][E] = x[t0:t1]^T dz[t0:t1]; grid (splits, H/128, ceil(E/128)).
__global__ __launch_bounds__(RTile::kThreads) void k_dwr_partial(const bf16_t* __restrict__ x,
                                                          const bf16_t* __restrict__ dz, int T, int H,
                                                          int E, float* __restrict__ partial) {
  using C = RTile;
  __shared__ __attribute__((aligned(16))) char smem[C::kLds];
  const int s = blockIdx.x, m0 = blockIdx.y * C::BM, n0 = blockIdx.z * C::BN;
  const int t0 = s * kDwrChunk, nt = min(kDwrChunk, T - t0);
  f32x4 acc[C::FM][C::FN];
  zero_acc<C>(acc);
  // A(m = h, k = t) = x[t][h] and B(n = e, k = t) = dz[t][e]: both MN-contiguous.
  const bf16_t* bs[1] = {dz + static_cast<int64_t>(t0) * E + n0};
  gemm_mainloop<C, false, false>(x + static_cast<int64_t>(t0) * H + m0, H, C::BM, bs, E, E - n0, nt, smem,
                                 acc);
  const int lane = threadIdx.x & 63;
  float* out = partial + static_cast<int64_t>(s) * H * E;
#pragma unroll
  for (int mi = 0; mi < C::FM; ++mi) {
    const int64_t row = static_cast<int64_t>(m0 + frag_row<C>(mi, lane)) * E;
#pragma unroll
    for (int ni = 0; ni < C::FN; ++ni) {
      const int e = n0 + frag_col<C>(ni, lane);
      if (e >= E) continue;
      const f32x4 v = acc[mi][ni];
      *reinterpret_cast<float4*>(out + row + e) = make_float4(v[0], v[1], v[2], v[3]);
    }
  }
}

// dW_r = sum over splits in order.
template <bool F32>
__global__ __launch_bounds__(256) void k_dwr_reduce(const float* __restrict__ partial, int splits,
                                                    int64_t n, void* __restrict__ dw_r) {
  for (int64_t i = static_cast<int64_t>(blockIdx.x) * 256 + threadIdx.x; i < n;
       i += static_cast<int64_t>(gridDim.x) * 256) {
    float v = 0.0f;
    for (int s = 0; s < splits; ++s) v += partial[static_cast<int64_t>(s) * n + i];
    if constexpr (F32)
      static_cast<float*>(dw_r)[i] = v;
    else
      static_cast<bf16_t*>(dw_r)[i] = f2bf(v);
  }
}

// W_rT[E][H] = W_r[H][E] through 32 x 32 LDS tiles (grid H/32 x E/32).
__global__ __launch_bounds__(256) void k_transpose_wr(const bf16_t* __restrict__ w_r, int H, int E,
                                                      bf16_t* __restrict__ w_rt) {
  __shared__ bf16_t tile[32][33];
  const int h0 = blockIdx.x * 32, e0 = blockIdx.y * 32;
  const int a = threadIdx.x >> 5, b = threadIdx.x & 31;
#pragma unroll
  for (int i = 0; i < 32; i += 8)
    if (h0 + a + i < H && e0 + b < E) tile[a + i][b] = w_r[static_cast<int64_t>(h0 + a + i) * E + e0 + b];
  __syncthreads();
#pragma unroll
  for (int i = 0; i < 32; i += 8)
    if (e0 + a + i < E && h0 + b < H) w_rt[static_cast<int64_t>(e0 + a + i) * H + h0 + b] = tile[b][a + i];
}

// dX[t] = sum_j ( dXp[row_of[t,j]] + dz_j W_r[:, idx_j] ): dz is non-zero on
// the k selected experts only, so the router term is k scaled rows of W_r^T
// (L2-resident).  One wave per token, 8 columns per lane per pass.
template <int KT>
__global__ __launch_bounds__(256) void k_router_dx(const float* __restrict__ dz_slot,
                                                   const int32_t* __restrict__ topk_idx,
                                                   const bf16_t* __restrict__ w_rt,
                                                   const bf16_t* __restrict__ dxp,
                                                   const int32_t* __restrict__ row_of, int T, int H, int k,
                                                   bf16_t* __restrict__ dx) {
  const int lane = threadIdx.x & 63;
  const int t = blockIdx.x * 4 + (threadIdx.x >> 6);
  if (t >= T) return;
  int rows[KT], ex[KT];
  float dzs[KT];
#pragma unroll
  for (int j = 0; j < KT; ++j) {
    const int64_t p = static_cast<int64_t>(t) * k + j;
    rows[j] = j < k ? row_of[p] : -1;
    ex[j] = j < k ? topk_idx[p] : -1;
    dzs[j] = j < k ? dz_slot[p] : 0.0f;
  }
  for (int c = lane * 8; c < H; c += kWave * 8) {
    uint4 v[KT], w[KT];
#pragma unroll
    for (int j = 0; j < KT; ++j) {
      const bool on = rows[j] >= 0;
      v[j] = on ? *reinterpret_cast<const uint4*>(dxp + static_cast<int64_t>(rows[j]) * H + c) : make_uint4(0, 0, 0, 0);
      w[j] = on ? *reinterpret_cast<const uint4*>(w_rt + static_cast<int64_t>(ex[j]) * H + c) : make_uint4(0, 0, 0, 0);
    }
    float acc[8] = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int j = 0; j < KT; ++j) {
      const uint32_t* pv = reinterpret_cast<const uint32_t*>(&v[j]);
      const uint32_t* pw = reinterpret_cast<const uint32_t*>(&w[j]);
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        acc[2 * q] += lo_bf(pv[q]) + dzs[j] * lo_bf(pw[q]);
        acc[2 * q + 1] += hi_bf(pv[q]) + dzs[j] * hi_bf(pw[q]);
      }
    }
    *reinterpret_cast<uint4*>(dx + static_cast<int64_t>(t) * H + c) =
        make_uint4(pack_bf16x2(acc[0], acc[1]), pack_bf16x2(acc[2], acc[3]), pack_bf16x2(acc[4], acc[5]),
                   pack_bf16x2(acc[6], acc[7]));
  }
}

}  // namespace

int dwr_splits(int T) { return cdiv(T, kDwrChunk); }

hipError_t launch_dwr(const bf16_t* x, const bf16_t* dz, int T, int H, int E, float* ws_f32,
                      void* dw_r, bool f32_out, hipStream_t s) {
  const int splits = dwr_splits(T);
  {
    TraceScope trace_scope(K_DWR_PARTIAL, s);
    hipLaunchKernelGGL(k_dwr_partial, dim3(splits, H / RTile::BM, cdiv(E, RTile::BN)), dim3(RTile::kThreads), 0, s, x, dz, T, H,
                       E, ws_f32);
  }
  const int64_t n = static_cast<int64_t>(H) * E;
  const int grid = static_cast<int>(std::min<int64_t>(cdiv64(n, 256), 2048));
  if (f32_out) {
    TraceScope trace_scope(K_DWR_REDUCE, s);
    hipLaunchKernelGGL(k_dwr_reduce<true>, dim3(grid), dim3(256), 0, s, ws_f32, splits, n, dw_r);
  } else {
    TraceScope trace_scope(K_DWR_REDUCE, s);
    hipLaunchKernelGGL(k_dwr_reduce<false>, dim3(grid), dim3(256), 0, s, ws_f32, splits, n, dw_r);
  }
  return hipGetLastError();
}

hipError_t launch_router_dx(const float* dz_slot, const int32_t* topk_idx, const bf16_t* w_r,
                            const bf16_t* dxp, const int32_t* row_of, int T, int H, int E, int k,
                            bf16_t* w_rt, bf16_t* dx, hipStream_t s) {
  {
    TraceScope trace_scope(K_TRANSPOSE_WR, s);
    hipLaunchKernelGGL(k_transpose_wr, dim3(cdiv(H, 32), cdiv(E, 32)), dim3(256), 0, s, w_r, H, E, w_rt);
  }
  {
    TraceScope trace_scope(K_ROUTER_DX, s);
    const dim3 grid(cdiv(T, 4));
    if (k <= 1) hipLaunchKernelGGL(k_router_dx<1>, grid, dim3(256), 0, s, dz_slot, topk_idx, w_rt, dxp, row_of, T, H, k, dx);
    else if (k <= 2) hipLaunchKernelGGL(k_router_dx<2>, grid, dim3(256), 0, s, dz_slot, topk_idx, w_rt, dxp, row_of, T, H, k, dx);
    else if (k <= 4) hipLaunchKernelGGL(k_router_dx<4>, grid, dim3(256), 0, s, dz_slot, topk_idx, w_rt, dxp, row_of, T, H, k, dx);
    else if (k <= 8) hipLaunchKernelGGL(k_router_dx<8>, grid, dim3(256), 0, s, dz_slot, topk_idx, w_rt, dxp, row_of, T, H, k, dx);
    else if (k <= 16) hipLaunchKernelGGL(k_router_dx<16>, grid, dim3(256), 0, s, dz_slot, topk_idx, w_rt, dxp, row_of, T, H, k, dx);
    else hipLaunchKernelGGL(k_router_dx<32>, grid, dim3(256), 0, s, dz_slot, topk_idx, w_rt, dxp, row_of, T, H, k, dx);
  }
  return hipGetLastError();
}

}  // namespace moe
