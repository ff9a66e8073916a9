// Router of the MoE block: logits z = x W_r (bf16 MFMA, fp32 accumulate) and,
// per valid token, the top-k experts by wave-level max/argmax with the
// softmax-over-selection gates.
#include <math.h>

#include "gemm_core.hpp"
#include "launch.hpp"
#include "trace.hpp"

namespace moe {

namespace {

// z[T,E] = x[T,H] W_r[H,E]; tile 128 tokens x 128 experts, K = H.
using RouterTile = Tile<128, 128, 1>;
__global__ __launch_bounds__(RouterTile::kThreads) void k_router_logits(const bf16_t* __restrict__ x,
                                                            const bf16_t* __restrict__ w_r, int T, int H,
                                                            int E, float* __restrict__ logits) {
  using C = RouterTile;
  __shared__ __attribute__((aligned(16))) char smem[C::kLds];
  const int m0 = blockIdx.x * C::BM, n0 = blockIdx.y * C::BN;
  f32x4 acc[C::FM][C::FN];
  zero_acc<C>(acc);
  const bf16_t* bs[1] = {w_r + n0};  // B(k = h, n = e) = W_r[h][e]: E-contiguous
  gemm_mainloop<C, true, false>(x + static_cast<int64_t>(m0) * H, H, min(C::BM, T - m0), bs, E, E - n0, H,
                                smem, acc);
  const int lane = threadIdx.x & 63;
#pragma unroll
  for (int mi = 0; mi < C::FM; ++mi) {
    const int t = m0 + frag_row<C>(mi, lane);
    if (t >= T) continue;
#pragma unroll
    for (int ni = 0; ni < C::FN; ++ni) {
      const int e = n0 + frag_col<C>(ni, lane);
      if (e >= E) continue;  // E % 8 == 0, so e < E covers e..e+3
      const f32x4 v = acc[mi][ni];
      *reinterpret_cast<float4*>(logits + static_cast<int64_t>(t) * E + e) = make_float4(v[0], v[1], v[2], v[3]);
    }
  }
}

// One wave per token.  Each lane holds the logits of experts lane + 64 i.
// k rounds: every lane offers its best untaken (value, expert), the wave
// reduces with "larger value, then lower expert" and the owner marks it taken.
// Gates: g_j = exp(z_j - z_0) / sum_j' exp(z_j' - z_0).
constexpr int kMaxLogitsPerLane = MOE_MAX_EXPERTS / kWave;

__global__ __launch_bounds__(256) void k_topk(const float* __restrict__ logits,
                                              const uint8_t* __restrict__ mask, int T, int E, int k,
                                              int32_t* __restrict__ topk_idx, float* __restrict__ gates) {
  const int lane = threadIdx.x & 63;
  const int t = blockIdx.x * 4 + (threadIdx.x >> 6);
  if (t >= T) return;
  int32_t* idx_row = topk_idx + static_cast<int64_t>(t) * k;
  float* g_row = gates + static_cast<int64_t>(t) * k;
  if (mask != nullptr && mask[t] == 0) {
    for (int j = lane; j < k; j += kWave) {
      idx_row[j] = -1;
      g_row[j] = 0.0f;
    }
    return;
  }
  const float* z = logits + static_cast<int64_t>(t) * E;
  float v[kMaxLogitsPerLane];
  bool live[kMaxLogitsPerLane];
#pragma unroll
  for (int i = 0; i < kMaxLogitsPerLane; ++i) {
    const int e = lane + kWave * i;
    live[i] = e < E;
    v[i] = live[i] ? z[e] : -INFINITY;
  }
  float my_v = 0.0f;
  int my_e = 0;
  for (int j = 0; j < k; ++j) {
    float bv = -INFINITY;
    int be = 0x7fffffff;
#pragma unroll
    for (int i = 0; i < kMaxLogitsPerLane; ++i) {
      const int e = lane + kWave * i;
      if (live[i] && (v[i] > bv || (v[i] == bv && e < be))) {
        bv = v[i];
        be = e;
      }
    }
#pragma unroll
    for (int m = 32; m >= 1; m >>= 1) {
      const float ov = shfl_xor(bv, m);
      const int oe = shfl_xor(be, m);
      if (ov > bv || (ov == bv && oe < be)) {
        bv = ov;
        be = oe;
      }
    }
    if ((be & 63) == lane) {
#pragma unroll
      for (int i = 0; i < kMaxLogitsPerLane; ++i)
        if (i == (be >> 6)) live[i] = false;
    }
    if (j == lane) {
      my_v = bv;
      my_e = be;
    }
  }
  const float top = __shfl(my_v, 0, kWave);
  const float w = lane < k ? expf(my_v - top) : 0.0f;
  const float sum = wave_sum(w);
  if (lane < k) {
    idx_row[lane] = my_e;
    g_row[lane] = w / sum;
  }
}

}  // namespace

hipError_t launch_router_fwd(const bf16_t* x, const bf16_t* w_r, const uint8_t* mask, int T, int H,
                             int E, int k, float* logits, int32_t* topk_idx, float* gates,
                             hipStream_t s) {
  {
    TraceScope trace_scope(K_ROUTER_LOGITS, s);
    hipLaunchKernelGGL(k_router_logits, dim3(cdiv(T, RouterTile::BM), cdiv(E, RouterTile::BN)), dim3(RouterTile::kThreads), 0, s, x, w_r, T, H,
                       E, logits);
  }
  {
    TraceScope trace_scope(K_TOPK, s);
    hipLaunchKernelGGL(k_topk, dim3(cdiv(T, 4)), dim3(256), 0, s, logits, mask, T, E, k, topk_idx, gates);
  }
  return hipGetLastError();
}

}  // namespace moe
