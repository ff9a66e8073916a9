// Router of the MoE block: logits z = x W_r (bf16 MFMA, fp32 accumulate) and,
// per valid token, the top-k experts (an exact radix selection) with the
// softmax-over-selection gates.
#include <math.h>

#include "gemm_core.hpp"
#include "launch.hpp"
#include "trace.hpp"

namespace moe {

namespace {

static_assert(MOE_MAX_EXPERTS <= 4 * kWave, "at most four experts per lane in the top-k");

// Logits z = x W_r, fp32 [T][E]: one workgroup per 32 tokens and all E
// experts (bf16 MFMA, fp32 accumulate, K = H), one 128-expert column tile at
// a time, so T / 32 workgroups share the chip.
using RouterTile = Tile<32, 128, 1, 1, 4>;
constexpr int kRouterTokens = RouterTile::BM;

__global__ __launch_bounds__(RouterTile::kThreads) void k_router_logits(const bf16_t* __restrict__ x,
                                                                        const bf16_t* __restrict__ w_r, int T,
                                                                        int H, int E, float* __restrict__ logits) {
  using C = RouterTile;
  __shared__ __attribute__((aligned(16))) char smem[C::kLds];
  const int t0 = blockIdx.x * kRouterTokens;
  const int rows = min(kRouterTokens, T - t0);
  const int lane = threadIdx.x & 63;
  for (int n0 = 0; n0 < E; n0 += C::BN) {
    f32x4 acc[C::FM][C::FN];
    zero_acc<C>(acc);
    const bf16_t* bs[1] = {w_r + n0};  // B(k = h, n = e) = W_r[h][e]: E-contiguous
    gemm_mainloop<C, true, false>(x + static_cast<int64_t>(t0) * H, H, rows, bs, E, E - n0, H, smem, acc);
#pragma unroll
    for (int mi = 0; mi < C::FM; ++mi) {
      const int r = frag_row<C>(mi, lane);
      if (r >= rows) continue;
#pragma unroll
      for (int ni = 0; ni < C::FN; ++ni) {
        const int e = n0 + frag_col<C>(ni, lane);
        if (e < E) {  // E % 8 == 0, so e < E covers e..e+3
          const f32x4 v = acc[mi][ni];
          *reinterpret_cast<float4*>(logits + static_cast<int64_t>(t0 + r) * E + e) =
              make_float4(v[0], v[1], v[2], v[3]);
        }
      }
    }
  }
}

// Order-preserving key of an fp32 value: a > b  <=>  key(a) > key(b), and
// -0 == +0 share a key.
__device__ __forceinline__ uint32_t order_key(float v) {
  uint32_t u = __float_as_uint(v);
  if (v == 0.0f) u = 0u;
  return (u >> 31) ? ~u : (u | 0x80000000u);
}
__device__ __forceinline__ float key_value(uint32_t key) {
  return __uint_as_float((key >> 31) ? (key & 0x7fffffffu) : ~key);
}

__device__ __forceinline__ int ballot_count(bool p) { return __popcll(__ballot(p)); }

// Top-k of one token per wave; lane l holds experts e = l + 64 m, m < PL.
// Selection: the k largest logits, ties to the lower expert, in slot order
// (descending logit, then ascending expert).  Exact: a radix search for the
// k-th largest order key (each wave-wide count is a ballot and a popcount),
// then the keys equal to it are taken by lower expert index; an entry's slot
// counts the selected keys that beat it, broadcast one by one.  Gates
// g_j = exp(z_j - z_0) / sum_j' exp(z_j' - z_0).  Keys of absent experts are
// 0, below every logit's key, so they never count.  Many waves per SIMD hide
// the latency of the wave-wide counts.
template <int PL>
__global__ __launch_bounds__(256) void k_topk(const float* __restrict__ logits, const uint8_t* __restrict__ mask,
                                              int T, int E, int k, int32_t* __restrict__ topk_idx,
                                              float* __restrict__ gates) {
  const int lane = threadIdx.x & 63;
  const int t = blockIdx.x * 4 + (threadIdx.x >> 6);
  if (t >= T) return;
  int32_t* idx_row = topk_idx + static_cast<int64_t>(t) * k;
  float* g_row = gates + static_cast<int64_t>(t) * k;
  if (mask != nullptr && mask[t] == 0) {
    if (lane < k) {
      idx_row[lane] = -1;
      g_row[lane] = 0.0f;
    }
    return;
  }
  const float* z = logits + static_cast<int64_t>(t) * E;
  uint32_t key[PL];
  float val[PL];
#pragma unroll
  for (int m = 0; m < PL; ++m) {
    const int e = lane + kWave * m;
    val[m] = e < E ? z[e] : 0.0f;
    key[m] = e < E ? order_key(val[m]) : 0u;
  }
  uint32_t kth = 0u;  // largest P with #{key >= P} >= k
  for (int b = 31; b >= 0; --b) {
    const uint32_t cand = kth | (1u << b);
    int cnt = 0;
#pragma unroll
    for (int m = 0; m < PL; ++m) cnt += ballot_count(key[m] >= cand);
    kth = cnt >= k ? cand : kth;
  }
  int above = 0;
#pragma unroll
  for (int m = 0; m < PL; ++m) above += ballot_count(key[m] > kth);
  const int need = k - above;  // entries equal to the k-th key, by lower expert index
  const unsigned long long below = (1ull << lane) - 1ull;
  bool sel[PL];
  unsigned long long selmask[PL];
  int eq_before = 0;
#pragma unroll
  for (int m = 0; m < PL; ++m) {
    const unsigned long long eq = __ballot(key[m] == kth);
    const int rank_eq = eq_before + __popcll(eq & below);
    eq_before += __popcll(eq);
    sel[m] = key[m] > kth || (key[m] == kth && rank_eq < need);
    selmask[m] = __ballot(sel[m]);
  }
  int slot[PL];
#pragma unroll
  for (int m = 0; m < PL; ++m) slot[m] = 0;
  uint32_t kmax = 0u;
#pragma unroll
  for (int mj = 0; mj < PL; ++mj) {
    unsigned long long msk = selmask[mj];
    while (msk != 0ull) {
      const int lj = __builtin_ctzll(msk);
      msk &= msk - 1ull;
      const uint32_t kj = static_cast<uint32_t>(__builtin_amdgcn_readlane(static_cast<int>(key[mj]), lj));
      const int ej = lj + kWave * mj;
      kmax = kj > kmax ? kj : kmax;
#pragma unroll
      for (int m = 0; m < PL; ++m) {
        const int e = lane + kWave * m;
        slot[m] += (sel[m] && (kj > key[m] || (kj == key[m] && ej < e))) ? 1 : 0;
      }
    }
  }
  const float top = key_value(kmax);
  float w = 0.0f;
  float wm[PL];
#pragma unroll
  for (int m = 0; m < PL; ++m) {
    wm[m] = sel[m] ? expf(val[m] - top) : 0.0f;
    w += wm[m];
  }
  const float sum = wave_sum(w);
#pragma unroll
  for (int m = 0; m < PL; ++m)
    if (sel[m]) {
      idx_row[slot[m]] = lane + kWave * m;
      g_row[slot[m]] = wm[m] / sum;
    }
}

}  // namespace

hipError_t launch_router_fwd(const bf16_t* x, const bf16_t* w_r, const uint8_t* mask, int T, int H,
                             int E, int k, float* logits, int32_t* topk_idx, float* gates,
                             hipStream_t s) {
  {
    TraceScope trace_scope(K_ROUTER_LOGITS, s);
    hipLaunchKernelGGL(k_router_logits, dim3(cdiv(T, kRouterTokens)), dim3(RouterTile::kThreads), 0, s, x, w_r,
                       T, H, E, logits);
  }
  {
    TraceScope trace_scope(K_TOPK, s);
    const dim3 grid(cdiv(T, 4)), block(256);
    // experts per lane: 1, 2 or 4 (E <= 256)
    if (E <= kWave)
      hipLaunchKernelGGL(k_topk<1>, grid, block, 0, s, logits, mask, T, E, k, topk_idx, gates);
    else if (E <= 2 * kWave)
      hipLaunchKernelGGL(k_topk<2>, grid, block, 0, s, logits, mask, T, E, k, topk_idx, gates);
    else
      hipLaunchKernelGGL(k_topk<4>, grid, block, 0, s, logits, mask, T, E, k, topk_idx, gates);
  }
  return hipGetLastError();
}

}  // namespace moe
