// Router backward of the MoE block: dW_r = x^T dz (split over tokens into
// fp32 partials reduced in a fixed order) and dX = (sum of the permuted-row
// gradients of the token) + dz W_r^T, the latter a K = E MFMA product whose
// epilogue gathers the token's rows.
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

// dX[t][h] = sum_j dXp[row_of[t,j]][h] + sum_e dz[t][e] W_r[h][e];
// tile 128 tokens x 128 hidden, K = E.
__global__ __launch_bounds__(RTile::kThreads) void k_router_dx(const bf16_t* __restrict__ dz,
                                                        const bf16_t* __restrict__ w_r,
                                                        const bf16_t* __restrict__ dxp,
                                                        const int32_t* __restrict__ row_of, int T, int H,
                                                        int E, int k, bf16_t* __restrict__ dx) {
  using C = RTile;
  __shared__ __attribute__((aligned(16))) char smem[C::kLds];
  const int m0 = blockIdx.x * C::BM, n0 = blockIdx.y * C::BN;
  f32x4 acc[C::FM][C::FN];
  zero_acc<C>(acc);
  // B(k = e, n = h) = W_r[h][e]: K-contiguous rows of W_r.
  const bf16_t* bs[1] = {w_r + static_cast<int64_t>(n0) * E};
  gemm_mainloop<C, true, true>(dz + static_cast<int64_t>(m0) * E, E, min(C::BM, T - m0), bs, E, H - n0, E,
                               smem, acc);
  const int lane = threadIdx.x & 63;
#pragma unroll
  for (int mi = 0; mi < C::FM; ++mi) {
    const int t = m0 + frag_row<C>(mi, lane);
    if (t >= T) continue;
    const int32_t* rows = row_of + static_cast<int64_t>(t) * k;
#pragma unroll
    for (int ni = 0; ni < C::FN; ++ni) {
      const int h = n0 + frag_col<C>(ni, lane);
      float s[4] = {0.f, 0.f, 0.f, 0.f};
      for (int j = 0; j < k; ++j) {
        const int r = rows[j];
        if (r < 0) continue;
        const uint2 w = *reinterpret_cast<const uint2*>(dxp + static_cast<int64_t>(r) * H + h);
        s[0] += lo_bf(w.x);
        s[1] += hi_bf(w.x);
        s[2] += lo_bf(w.y);
        s[3] += hi_bf(w.y);
      }
      f32x4 v = acc[mi][ni];
#pragma unroll
      for (int i = 0; i < 4; ++i) v[i] += s[i];
      *reinterpret_cast<uint2*>(dx + static_cast<int64_t>(t) * H + h) = pack4_bf16(v);
    }
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

hipError_t launch_router_dx(const bf16_t* dz, const bf16_t* w_r, const bf16_t* dxp,
                            const int32_t* row_of, int T, int H, int E, int k, bf16_t* dx,
                            hipStream_t s) {
  {
    TraceScope trace_scope(K_ROUTER_DX, s);
    hipLaunchKernelGGL(k_router_dx, dim3(cdiv(T, RTile::BM), H / RTile::BN), dim3(RTile::kThreads), 0, s, dz, w_r, dxp, row_of, T,
                       H, E, k, dx);
  }
  return hipGetLastError();
}

}  // namespace moe
