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

// dW_r = sum over splits in order.  Four elements per thread (n % 4 == 0,
// as H E is); each group of kGroup splits has its loads issued before its
// adds, which still run in split order.
template <bool F32>
__global__ __launch_bounds__(256) void k_dwr_reduce(const float* __restrict__ partial, int splits,
                                                    int64_t n, void* __restrict__ dw_r) {
  constexpr int kGroup = 8;
  const int64_t n4 = n / 4;
  for (int64_t i = static_cast<int64_t>(blockIdx.x) * 256 + threadIdx.x; i < n4;
       i += static_cast<int64_t>(gridDim.x) * 256) {
    float4 v = make_float4(0.f, 0.f, 0.f, 0.f);
    for (int s0 = 0; s0 < splits; s0 += kGroup) {
      float4 p[kGroup];
#pragma unroll
      for (int g = 0; g < kGroup; ++g)
        p[g] = s0 + g < splits ? reinterpret_cast<const float4*>(partial + static_cast<int64_t>(s0 + g) * n)[i]
                               : make_float4(0.f, 0.f, 0.f, 0.f);
#pragma unroll
      for (int g = 0; g < kGroup; ++g) {
        v.x += p[g].x;
        v.y += p[g].y;
        v.z += p[g].z;
        v.w += p[g].w;
      }
    }
    if constexpr (F32) {
      reinterpret_cast<float4*>(dw_r)[i] = v;
    } else {
      reinterpret_cast<uint2*>(dw_r)[i] = make_uint2(pack_bf16x2(v.x, v.y), pack_bf16x2(v.z, v.w));
    }
  }
}

// dX[t] = sum_j ( dXp[row_of[t,j]] + dz_j W_r[:, idx_j] ): dz is non-zero on
// the k selected experts only, so the router term is k scaled rows of W_r^T
// (L2-resident).  With kDense the router term is instead a precomputed row of
// dz W_r^T (fp32 [T][H]; dz dense over E when the router losses are on).  One
// wave per token; a pass takes row_chunks 16-byte chunks per lane of every row.
template <int KT, bool kDense>
__global__ __launch_bounds__(256) void k_router_dx(const float* __restrict__ dz_slot,
                                                   const int32_t* __restrict__ topk_idx,
                                                   const bf16_t* __restrict__ w_rt,
                                                   const float* __restrict__ dense,
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
  // dXp and W_r^T rows both in registers: at k = 8 one chunk per row ran
  // fastest (two took 186 registers and halved the waves per SIMD).  dXp is
  // read once, with non-temporal loads, so that the W_r^T rows stay in L2
  // (68 to 64 us at the Qwen shape)
  constexpr int kU = row_chunks<KT, 8>();
  for (int c0 = lane * 8; c0 < H; c0 += kWave * 8 * kU) {
    uint4 v[KT][kU], w[KT][kU];
#pragma unroll
    for (int j = 0; j < KT; ++j)
#pragma unroll
      for (int u = 0; u < kU; ++u) {
        const int c = c0 + u * kWave * 8;
        const bool on = rows[j] >= 0 && c < H;
        v[j][u] = on ? load_nt(dxp + static_cast<int64_t>(rows[j]) * H + c) : make_uint4(0, 0, 0, 0);
        if constexpr (!kDense)
          w[j][u] = on ? *reinterpret_cast<const uint4*>(w_rt + static_cast<int64_t>(ex[j]) * H + c)
                       : make_uint4(0, 0, 0, 0);
      }
#pragma unroll
    for (int u = 0; u < kU; ++u) {
      const int c = c0 + u * kWave * 8;
      float acc[8] = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
      if constexpr (kDense) {
        if (rows[0] >= 0 && c < H) {  // a routed token: its dense router term
          const float4 a = *reinterpret_cast<const float4*>(dense + static_cast<int64_t>(t) * H + c);
          const float4 b = *reinterpret_cast<const float4*>(dense + static_cast<int64_t>(t) * H + c + 4);
          acc[0] = a.x, acc[1] = a.y, acc[2] = a.z, acc[3] = a.w;
          acc[4] = b.x, acc[5] = b.y, acc[6] = b.z, acc[7] = b.w;
        }
      }
#pragma unroll
      for (int j = 0; j < KT; ++j) {
        const uint32_t* pv = reinterpret_cast<const uint32_t*>(&v[j][u]);
        const uint32_t* pw = reinterpret_cast<const uint32_t*>(&w[j][u]);
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          if constexpr (kDense) {
            acc[2 * q] += lo_bf(pv[q]);
            acc[2 * q + 1] += hi_bf(pv[q]);
          } else {
            acc[2 * q] += lo_bf(pv[q]) + dzs[j] * lo_bf(pw[q]);
            acc[2 * q + 1] += hi_bf(pv[q]) + dzs[j] * hi_bf(pw[q]);
          }
        }
      }
      if (c < H)
        *reinterpret_cast<uint4*>(dx + static_cast<int64_t>(t) * H + c) =
            make_uint4(pack_bf16x2(acc[0], acc[1]), pack_bf16x2(acc[2], acc[3]), pack_bf16x2(acc[4], acc[5]),
                       pack_bf16x2(acc[6], acc[7]));
    }
  }
}

// dense[T][H] = dz W_r^T (fp32): A(m = t, k = e) = dz[t][e] and
// B(n = h, k = e) = W_r[h][e], both K-contiguous; grid (T/128, H/128).
__global__ __launch_bounds__(RTile::kThreads) void k_router_dx_dense(const bf16_t* __restrict__ dz,
                                                                   const bf16_t* __restrict__ w_r, int T, int H,
                                                                   int E, float* __restrict__ dense) {
  using C = RTile;
  __shared__ __attribute__((aligned(16))) char smem[C::kLds];
  const int m0 = blockIdx.x * C::BM, n0 = blockIdx.y * C::BN;
  f32x4 acc[C::FM][C::FN];
  zero_acc<C>(acc);
  const bf16_t* bs[1] = {w_r + static_cast<int64_t>(n0) * E};
  gemm_mainloop<C, true, true>(dz + static_cast<int64_t>(m0) * E, E, min(C::BM, T - m0), bs, E, H - n0, E, smem,
                               acc);
  const int lane = threadIdx.x & 63;
#pragma unroll
  for (int mi = 0; mi < C::FM; ++mi) {
    const int t = m0 + frag_row<C>(mi, lane);
    if (t >= T) continue;
#pragma unroll
    for (int ni = 0; ni < C::FN; ++ni) {
      const f32x4 v = acc[mi][ni];
      *reinterpret_cast<float4*>(dense + static_cast<int64_t>(t) * H + n0 + frag_col<C>(ni, lane)) =
          make_float4(v[0], v[1], v[2], v[3]);
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
  const int64_t n = static_cast<int64_t>(H) * E;  // a multiple of 4: E % 8 == 0
  const int grid = static_cast<int>(std::min<int64_t>(cdiv64(n / 4, 256), 2048));
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
                            const bf16_t* w_rt, bf16_t* dx, const bf16_t* dz_dense, float* dense, hipStream_t s) {
  const bool use_dense = dz_dense != nullptr;
  if (use_dense) {
    TraceScope trace_scope(K_ROUTER_DX_DENSE, s);
    hipLaunchKernelGGL(k_router_dx_dense, dim3(cdiv(T, RTile::BM), H / RTile::BN), dim3(RTile::kThreads), 0, s,
                       dz_dense, w_r, T, H, E, dense);
  }
  {
    TraceScope trace_scope(K_ROUTER_DX, s);
    const dim3 grid(cdiv(T, 4)), block(256);
#define MOE_RDX(KT)                                                                                              \
  do {                                                                                                           \
    if (use_dense)                                                                                               \
      hipLaunchKernelGGL((k_router_dx<KT, true>), grid, block, 0, s, dz_slot, topk_idx, w_rt, dense, dxp, row_of, \
                         T, H, k, dx);                                                                           \
    else                                                                                                         \
      hipLaunchKernelGGL((k_router_dx<KT, false>), grid, block, 0, s, dz_slot, topk_idx, w_rt, dense, dxp,       \
                         row_of, T, H, k, dx);                                                                   \
  } while (0)
    if (k <= 1) MOE_RDX(1);
    else if (k <= 2) MOE_RDX(2);
    else if (k <= 4) MOE_RDX(4);
    else if (k <= 8) MOE_RDX(8);
    else if (k <= 16) MOE_RDX(16);
    else MOE_RDX(32);
#undef MOE_RDX
  }
  return hipGetLastError();
}

}  // namespace moe
