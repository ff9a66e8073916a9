// Weighted combine of the expert outputs and its backward (which also forms
// the router-logit gradient dz).  One wave per token; rows move as 16-byte
// vectors (8 bf16 per lane), sums are fp32 in slot order.
#include "launch.hpp"
#include "trace.hpp"

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

// y[t] = sum_j g[t,j] o[row_of[t,j]]  (0 when the token has no rows).
__global__ __launch_bounds__(256) void k_combine(const bf16_t* __restrict__ o, const float* __restrict__ gates,
                                                 const int32_t* __restrict__ row_of, int T, int H, int k,
                                                 bf16_t* __restrict__ y) {
  const int lane = threadIdx.x & 63;
  const int t = blockIdx.x * 4 + (threadIdx.x >> 6);
  if (t >= T) return;
  const int32_t* rows = row_of + static_cast<int64_t>(t) * k;
  const float* g = gates + static_cast<int64_t>(t) * k;
  for (int c = lane * 8; c < H; c += kWave * 8) {
    float acc[8] = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
    for (int j = 0; j < k; ++j) {
      const int r = rows[j];
      if (r < 0) continue;
      float f[8];
      unpack8(*reinterpret_cast<const uint4*>(o + static_cast<int64_t>(r) * H + c), f);
      const float gj = g[j];
#pragma unroll
      for (int i = 0; i < 8; ++i) acc[i] += gj * f[i];
    }
    *reinterpret_cast<uint4*>(y + static_cast<int64_t>(t) * H + c) = pack8(acc);
  }
}

// Per token t with rows r_j:
//   dO[r_j] = g_j dY[t]               (bf16)
//   dg_j    = <dY[t], O[r_j]>         (fp32)
//   dz[t,e] = g_j (dg_j - sum_j' g_j' dg_j') for e = idx_j, else 0  (bf16, all E)
__global__ __launch_bounds__(256) void k_combine_bwd(const bf16_t* __restrict__ dy,
                                                     const bf16_t* __restrict__ o,
                                                     const float* __restrict__ gates,
                                                     const int32_t* __restrict__ topk_idx,
                                                     const int32_t* __restrict__ row_of, int T, int H,
                                                     int E, int k, bf16_t* __restrict__ d_o,
                                                     float* __restrict__ dg_out, bf16_t* __restrict__ dz) {
  const int lane = threadIdx.x & 63;
  const int t = blockIdx.x * 4 + (threadIdx.x >> 6);
  if (t >= T) return;
  const int32_t* rows = row_of + static_cast<int64_t>(t) * k;
  const float* g = gates + static_cast<int64_t>(t) * k;
  const bf16_t* dyr = dy + static_cast<int64_t>(t) * H;
  float my_dg = 0.0f;  // lane j keeps dg_j
  for (int j = 0; j < k; ++j) {
    const int r = rows[j];
    if (r < 0) continue;
    const float gj = g[j];
    float part = 0.0f;
    for (int c = lane * 8; c < H; c += kWave * 8) {
      float fy[8], fo[8], out[8];
      unpack8(*reinterpret_cast<const uint4*>(dyr + c), fy);
      unpack8(*reinterpret_cast<const uint4*>(o + static_cast<int64_t>(r) * H + c), fo);
#pragma unroll
      for (int i = 0; i < 8; ++i) {
        part += fy[i] * fo[i];
        out[i] = gj * fy[i];
      }
      *reinterpret_cast<uint4*>(d_o + static_cast<int64_t>(r) * H + c) = pack8(out);
    }
    const float dgj = wave_sum(part);
    if (lane == j) my_dg = dgj;
  }
  const float my_g = lane < k ? g[lane] : 0.0f;
  const int my_e = lane < k ? topk_idx[static_cast<int64_t>(t) * k + lane] : -1;
  const float inner = wave_sum(my_g * my_dg);
  const float my_dz = my_g * (my_dg - inner);
  if (lane < k) dg_out[static_cast<int64_t>(t) * k + lane] = my_dg;
  bf16_t* dzr = dz + static_cast<int64_t>(t) * E;
  for (int e0 = 0; e0 < E; e0 += kWave) {
    const int e = e0 + lane;
    float v = 0.0f;
    for (int j = 0; j < k; ++j) {
      const int ej = __shfl(my_e, j, kWave);
      const float dzj = __shfl(my_dz, j, kWave);
      if (ej == e) v = dzj;
    }
    if (e < E) dzr[e] = f2bf(v);
  }
}

}  // namespace

hipError_t launch_combine(const bf16_t* o, const float* gates, const int32_t* row_of, int T, int H,
                          int k, bf16_t* y, hipStream_t s) {
  {
    TraceScope trace_scope(K_COMBINE, s);
    hipLaunchKernelGGL(k_combine, dim3(cdiv(T, 4)), dim3(256), 0, s, o, gates, row_of, T, H, k, y);
  }
  return hipGetLastError();
}

hipError_t launch_combine_bwd(const bf16_t* dy, const bf16_t* o, const float* gates,
                              const int32_t* topk_idx, const int32_t* row_of, int T, int H, int E,
                              int k, bf16_t* d_o, float* dg, bf16_t* dz, hipStream_t s) {
  {
    TraceScope trace_scope(K_COMBINE_BWD, s);
    hipLaunchKernelGGL(k_combine_bwd, dim3(cdiv(T, 4)), dim3(256), 0, s, dy, o, gates, topk_idx, row_of, T,
                       H, E, k, d_o, dg, dz);
  }
  return hipGetLastError();
}

}  // namespace moe
