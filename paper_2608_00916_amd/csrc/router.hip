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

// Logits z = x W_r, fp32 [T][E], split over K: workgroup (i, s) multiplies
// tokens 128 i .. 128 i + 127 by W_r over the s-th of kRouterSplits
// contiguous K ranges (whole 64-deep steps) and writes its partial sums,
// split 0 into `logits` and split s > 0 into part[s - 1] ([T][E] each); the
// top-k kernel adds them in split order.  All E experts per workgroup, one
// 128-expert column tile at a time (bf16 MFMA, fp32 accumulate).  Every
// workgroup streams its K range of W_r (512 KB in all at H = 2048, E = 128)
// through LDS, so the token tile sets how often W_r crosses from L2: 128
// tokens per tile and a 4-way K split keep the grid at T / 32 workgroups
// while W_r is read T / 128 times instead of T / 32.
using RouterTile = Tile<128, 128, 1, 2, 2>;
constexpr int kRouterTokens = RouterTile::BM;
constexpr int kRouterSplits = 4;

__global__ __launch_bounds__(RouterTile::kThreads) void k_router_logits(const bf16_t* __restrict__ x,
                                                                        const bf16_t* __restrict__ w_r, int T,
                                                                        int H, int E, float* __restrict__ logits,
                                                                        float* __restrict__ part,
                                                                        int32_t* __restrict__ zero, int n_zero) {
  using C = RouterTile;
  __shared__ __attribute__((aligned(16))) char smem[C::kLds];
  // the permutation's chunk counts start at zero for the top-k's atomic adds
  if (blockIdx.x == 0 && blockIdx.y == 0)
    for (int i = threadIdx.x; i < n_zero; i += C::kThreads) zero[i] = 0;
  const int t0 = blockIdx.x * kRouterTokens;
  const int rows = min(kRouterTokens, T - t0);
  const int split = blockIdx.y;
  const int kper = cdiv(cdiv(H, kRouterSplits), BK) * BK;
  const int k0 = min(H, split * kper);
  const int kn = min(H, k0 + kper) - k0;  // 0 for an empty split: its partial sums are zeros
  float* out = split == 0 ? logits : part + static_cast<int64_t>(split - 1) * T * E;
  const int lane = threadIdx.x & 63;
  for (int n0 = 0; n0 < E; n0 += C::BN) {
    f32x4 acc[C::FM][C::FN];
    zero_acc<C>(acc);
    const bf16_t* bs[1] = {w_r + static_cast<int64_t>(k0) * E + n0};  // B(k = h, n = e) = W_r[h][e]: E-contiguous
    gemm_mainloop<C, true, false>(x + static_cast<int64_t>(t0) * H + k0, H, rows, bs, E, E - n0, kn, smem, acc);
#pragma unroll
    for (int mi = 0; mi < C::FM; ++mi) {
      const int r = frag_row<C>(mi, lane);
      if (r >= rows) continue;
#pragma unroll
      for (int ni = 0; ni < C::FN; ++ni) {
        const int e = n0 + frag_col<C>(ni, lane);
        if (e < E) {  // E % 8 == 0, so e < E covers e..e+3
          const f32x4 v = acc[mi][ni];
          *reinterpret_cast<float4*>(out + static_cast<int64_t>(t0 + r) * E + e) = make_float4(v[0], v[1], v[2], v[3]);
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

// Top-k of one token, held by a wave: lane l holds the logits of experts
// e = l + 64 m, m < PL (key 0 and value 0 where e >= E).  Selection: the k
// largest logits, ties to the lower expert, in slot order (descending logit,
// then ascending expert).  Exact: a radix search for the k-th largest order
// key (each wave-wide count is a ballot and a popcount), then the keys equal
// to it are taken by lower expert index; an entry's slot counts the selected
// keys that beat it, broadcast one by one.  Gates
// g_j = exp(z_j - z_0) / sum_j' exp(z_j' - z_0).  Keys of absent experts are
// 0, below every logit's key, so they never count.  Returns the largest logit.
template <int PL>
__device__ __forceinline__ float topk_select(const float (&val)[PL], const uint32_t (&key)[PL], int k, int lane,
                                             int32_t* __restrict__ idx_row, float* __restrict__ g_row,
                                             int32_t* __restrict__ cnt_row) {
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
      atomicAdd(cnt_row + lane + kWave * m, 1);
    }
  return top;
}

// One wave per token: the top-k and gates; masked tokens get expert -1 and
// gate 0.  With kAux the workgroup (4 tokens) also writes one row of partial
// sums for the router losses: the full softmax p[t,e] of its valid tokens
// summed over the 4 tokens in order, and in column E the sum of lse_t^2
// (lse_t = log sum_e exp z[t,e]).  Many waves per SIMD hide the latency of
// the wave-wide counts.
template <int PL, bool kAux>
__global__ __launch_bounds__(256) void k_topk(float* __restrict__ logits, const float* __restrict__ part,
                                              const uint8_t* __restrict__ mask, int T, int E, int k,
                                              int32_t* __restrict__ topk_idx, float* __restrict__ gates,
                                              float* __restrict__ aux_part, int32_t* __restrict__ chunk_counts,
                                              int32_t* __restrict__ row_token) {
  const int lane = threadIdx.x & 63, wv = threadIdx.x >> 6;
  const int t = blockIdx.x * 4 + wv;
  if (!kAux && t >= T) return;
  const bool on = t < T && (mask == nullptr || mask[t] != 0);
  float val[PL];
  uint32_t key[PL];
  if (t < T) {
    // z = the K splits' partial sums added in split order, stored back as the logits
    float* z = logits + static_cast<int64_t>(t) * E;
    const int64_t plane = static_cast<int64_t>(T) * E;
#pragma unroll
    for (int m = 0; m < PL; ++m) {
      const int e = lane + kWave * m;
      float v = 0.0f;
      if (e < E) {
        v = z[e];
#pragma unroll
        for (int sp = 0; sp < kRouterSplits - 1; ++sp) v += part[sp * plane + static_cast<int64_t>(t) * E + e];
        z[e] = v;
      }
      val[m] = v;
      // a present expert's key stays above the padding key 0 (only a NaN
      // with every bit set maps to 0), so a padding lane is never selected
      key[m] = e < E ? max(order_key(v), 1u) : 0u;
    }
  }
  if (t < T && lane < k) row_token[static_cast<int64_t>(t) * k + lane] = -1;
  if (on) {
    topk_select<PL>(val, key, k, lane, topk_idx + static_cast<int64_t>(t) * k, gates + static_cast<int64_t>(t) * k,
                    chunk_counts + static_cast<int64_t>(t / kPermChunk) * E);
  } else if (t < T && lane < k) {
    topk_idx[static_cast<int64_t>(t) * k + lane] = -1;
    gates[static_cast<int64_t>(t) * k + lane] = 0.0f;
  }
  if constexpr (kAux) {
    __shared__ float part[4][MOE_MAX_EXPERTS + 1];
    float p[PL];
    float lse = 0.0f;
#pragma unroll
    for (int m = 0; m < PL; ++m) p[m] = 0.0f;
    if (on) {
      float mx = -INFINITY;
#pragma unroll
      for (int m = 0; m < PL; ++m)
        if (lane + kWave * m < E) mx = fmaxf(mx, val[m]);
      mx = wave_max(mx);
      float s = 0.0f;
#pragma unroll
      for (int m = 0; m < PL; ++m) {
        p[m] = lane + kWave * m < E ? expf(val[m] - mx) : 0.0f;
        s += p[m];
      }
      s = wave_sum(s);
#pragma unroll
      for (int m = 0; m < PL; ++m) p[m] /= s;
      lse = mx + logf(s);
    }
#pragma unroll
    for (int m = 0; m < PL; ++m)
      if (lane + kWave * m < E) part[wv][lane + kWave * m] = p[m];
    if (lane == 0) part[wv][E] = lse * lse;
    __syncthreads();
    float* row = aux_part + static_cast<int64_t>(blockIdx.x) * (E + 1);
    for (int c = threadIdx.x; c <= E; c += 256) row[c] = ((part[0][c] + part[1][c]) + part[2][c]) + part[3][c];
  }
}

// Router-loss sums: col[c] = sum of column c over the partial rows (each
// thread sums a fixed set of rows in order, then a fixed tree).
__global__ __launch_bounds__(256) void k_router_loss_cols(const float* __restrict__ part, int nrows, int ncols,
                                                          float* __restrict__ col) {
  __shared__ float red[256];
  const int c = blockIdx.x;
  float s = 0.0f;
  for (int r = threadIdx.x; r < nrows; r += 256) s += part[static_cast<int64_t>(r) * ncols + c];
  red[threadIdx.x] = s;
  __syncthreads();
  for (int w = 128; w > 0; w >>= 1) {
    if (threadIdx.x < w) red[threadIdx.x] += red[threadIdx.x + w];
    __syncthreads();
  }
  if (threadIdx.x == 0) col[c] = red[0];
}

// {L_aux, L_z} from the column sums and the routing counts:
//   L_aux = aux_coef E sum_e f_e P_e = aux_coef E sum_e counts_e col_e / (R T_v),
//   L_z = z_coef col_E / T_v,  R = offsets[E] = T_v k routed rows.
__global__ __launch_bounds__(256) void k_router_loss_final(const float* __restrict__ col,
                                                           const int32_t* __restrict__ counts,
                                                           const int32_t* __restrict__ offsets, int E, int k,
                                                           float aux_coef, float z_coef, float* __restrict__ out) {
  __shared__ float red[256];
  float s = 0.0f;
  for (int e = threadIdx.x; e < E; e += 256) s += static_cast<float>(counts[e]) * col[e];
  red[threadIdx.x] = s;
  __syncthreads();
  for (int w = 128; w > 0; w >>= 1) {
    if (threadIdx.x < w) red[threadIdx.x] += red[threadIdx.x + w];
    __syncthreads();
  }
  if (threadIdx.x == 0) {
    const int R = offsets[E];
    const float tv = static_cast<float>(R / k);
    out[0] = R > 0 ? aux_coef * static_cast<float>(E) * red[0] / (static_cast<float>(R) * tv) : 0.0f;
    out[1] = R > 0 ? z_coef * col[E] / tv : 0.0f;
  }
}

}  // namespace

int64_t router_loss_ws_floats(int T, int E) { return static_cast<int64_t>(cdiv(T, 4)) * (E + 1) + E + 1; }
int64_t router_part_floats(int T, int E) { return static_cast<int64_t>(kRouterSplits - 1) * T * E; }

hipError_t launch_router_fwd(const bf16_t* x, const bf16_t* w_r, const uint8_t* mask, int T, int H,
                             int E, int k, float* logits, float* part, int32_t* topk_idx, float* gates,
                             float* aux_ws, int32_t* chunk_counts, int32_t* row_token, hipStream_t s) {
  {
    TraceScope trace_scope(K_ROUTER_LOGITS, s);
    hipLaunchKernelGGL(k_router_logits, dim3(cdiv(T, kRouterTokens), kRouterSplits), dim3(RouterTile::kThreads), 0,
                       s, x, w_r, T, H, E, logits, part, chunk_counts, static_cast<int>(permute_ws_ints(T, E)));
  }
  {
    TraceScope trace_scope(K_TOPK, s);
    const dim3 grid(cdiv(T, 4)), block(256);
    // experts per lane: 1, 2 or 4 (E <= 256)
#define MOE_TOPK(PL, AUX) \
  hipLaunchKernelGGL((k_topk<PL, AUX>), grid, block, 0, s, logits, part, mask, T, E, k, topk_idx, gates, aux_ws, \
                     chunk_counts, row_token)
    const bool aux = aux_ws != nullptr;
    if (E <= kWave) {
      if (aux) MOE_TOPK(1, true); else MOE_TOPK(1, false);
    } else if (E <= 2 * kWave) {
      if (aux) MOE_TOPK(2, true); else MOE_TOPK(2, false);
    } else {
      if (aux) MOE_TOPK(4, true); else MOE_TOPK(4, false);
    }
#undef MOE_TOPK
  }
  return hipGetLastError();
}

hipError_t launch_router_loss(const float* aux_ws, int T, int E, int k, const int32_t* counts,
                              const int32_t* offsets, float aux_coef, float z_coef, float* out, hipStream_t s) {
  const int nrows = cdiv(T, 4);
  float* col = const_cast<float*>(aux_ws) + static_cast<int64_t>(nrows) * (E + 1);
  {
    TraceScope trace_scope(K_ROUTER_LOSS, s);
    hipLaunchKernelGGL(k_router_loss_cols, dim3(E + 1), dim3(256), 0, s, aux_ws, nrows, E + 1, col);
    hipLaunchKernelGGL(k_router_loss_final, dim3(1), dim3(256), 0, s, col, counts, offsets, E, k, aux_coef, z_coef,
                       out);
  }
  return hipGetLastError();
}

}  // namespace moe
