// Grouped (per-expert) bf16 MFMA GEMMs of the MoE block, forward and backward.
//
// Rows are grouped expert-major: expert e owns rows [offsets[e], offsets[e+1]).
// Products over the rows of one expert (gate/up, down, and their input
// gradients) walk a device-built table of 128-row tiles, so the
// host never learns the counts: they run as persistent grids (a few workgroups
// per CU) that stride over the tiles the table holds.  Weight gradients
// (K = rows of one expert) have a fixed grid of E x (M/128) x (N/128) tiles;
// experts without rows write zeros.
#include "launch.hpp"
#include "trace.hpp"
#include "gemm_core.hpp"
#include "wgrad_plan.hpp"

#include <algorithm>
#include <mutex>

namespace moe {

namespace {

// Rows per tile of the grouped products (the unit of tile_start).
constexpr int kRowTile = 128;

struct MTile {
  int e, m0, m_lim, nt;
};

// Run body(tile) for every (expert, row tile, column tile) of a grouped
// product with n_ntiles column tiles.  Tile i*gridDim + xcd_tile(block) goes
// to this workgroup in round i, so each XCD works on a contiguous run of tiles.
// A tile's row range comes from one load of the tile table, issued a tile
// ahead (always from a valid entry: a select between that load and a
// register would turn it into a flat access, whose pending state makes every
// LDS wait of the K loop a full drain).
template <typename Body>
__device__ __forceinline__ void for_each_grouped_tile(const int32_t* tile_start, const int2* tile_desc, int E,
                                                      int n_ntiles, Body&& body) {
  const int total = tile_start[E] * n_ntiles;
  int logical = xcd_tile(blockIdx.x, gridDim.x);
  if (logical >= total) return;
  int2 d = tile_desc[logical / n_ntiles];
  while (logical < total) {
    const int mt = logical / n_ntiles;
    const int next = logical + gridDim.x;
    const int2 dn = tile_desc[min(next, total - 1) / n_ntiles];
    MTile t;
    t.e = d.y & 0xff;
    t.m_lim = d.y >> 8;
    t.m0 = d.x;
    t.nt = logical - mt * n_ntiles;
    body(t);
    d = dn;
    logical = next;
  }
}

// A rank-r adapter term of a grouped product, one more K segment (K = r):
// A operand `a` [rows][rank] (bf16, K-contiguous), per-expert B operands b0
// (and b1 for gate/up), whose layout each kernel states.
struct LoraSeg {
  const bf16_t* a = nullptr;
  const bf16_t* b0 = nullptr;
  const bf16_t* b1 = nullptr;
  int rank = 0;
};

// Rank-r intermediates of the adapters, row-grouped like the expert products:
//   out[r][q] = scale * sum_s X_s[r][:] W_s[e](:, q),  q < rank (16 per tile)
// with X_s K-contiguous ([rows][K], ld ldx) and W_s per expert (e * estride):
// MN-contiguous [K][rank] (the a matrices) or, with B_KC, K-contiguous rows q
// of length K ([rank][K], the b matrices).  NSEG = 2 sums two segments (dG with
// b1_gate and dU with b1_up).  These stream whole activation matrices through
// a rank-16 product, so they are bound by memory; one wave takes one 64-row
// half of a 128-row tile (64 x 16).
using LoraRows = Tile<64, 16, 1, 1, 1>;
template <bool B_KC, int NSEG>
__global__ __launch_bounds__(LoraRows::kThreads) void k_lora_rows(
    const bf16_t* __restrict__ x0, const bf16_t* __restrict__ x1, int64_t ldx, const bf16_t* __restrict__ w0,
    const bf16_t* __restrict__ w1, int64_t estride, int K, const int32_t* __restrict__ tile_start,
    const int2* __restrict__ tile_desc, int E, int rank, float scale, bf16_t* __restrict__ out) {
  using C = LoraRows;
  constexpr int kHalves = kRowTile / C::BM;
  static_assert(kHalves * C::BM == kRowTile, "a row tile splits into whole halves");
  __shared__ __attribute__((aligned(16))) char smem[C::kLds];
  for_each_grouped_tile(tile_start, tile_desc, E, rank / C::BN * kHalves, [&](const MTile& t) {
    const int half = t.nt % kHalves;
    const int m0 = t.m0 + half * C::BM;
    const int m_lim = min(C::BM, t.m_lim - half * C::BM);
    if (m_lim <= 0) return;  // the empty second half of a short tile (the whole wave)
    f32x4 acc[C::FM][C::FN];
    zero_acc<C>(acc);
    const int q0 = (t.nt / kHalves) * C::BN;
    const int64_t wofs = static_cast<int64_t>(t.e) * estride + (B_KC ? static_cast<int64_t>(q0) * K : q0);
    const int64_t ldw = B_KC ? K : rank;
    const bf16_t* b0[1] = {w0 + wofs};
    gemm_mainloop<C, true, B_KC>(x0 + static_cast<int64_t>(m0) * ldx, ldx, m_lim, b0, ldw, C::BN, K, smem, acc);
    if constexpr (NSEG == 2) {
      const bf16_t* b1[1] = {w1 + wofs};
      gemm_mainloop<C, true, B_KC>(x1 + static_cast<int64_t>(m0) * ldx, ldx, m_lim, b1, ldw, C::BN, K, smem, acc);
    }
    const int lane = threadIdx.x & 63;
#pragma unroll
    for (int mi = 0; mi < C::FM; ++mi) {
      const int r = frag_row<C>(mi, lane);
      if (r >= m_lim) continue;
      f32x4 v = acc[mi][0];
#pragma unroll
      for (int i = 0; i < 4; ++i) v[i] *= scale;
      *reinterpret_cast<uint2*>(out + static_cast<int64_t>(m0 + r) * rank + q0 + frag_col<C>(0, lane)) =
          pack4_bf16(v);
    }
  });
}

using GateUpFwd = Tile<128, 256, 2, 2, 4>;

// G = X W_gate[e], U = X W_up[e], A = silu(G) * U (K = H, N = F) with row r
// of the product read from row xp_rows[r] of xp (the tokens themselves,
// gathered through the permutation; xp_bytes bounds xp): the forward-only
// pass, which skips the permuted copy.  The B tile holds 128 columns of
// W_gate next to the same 128 of W_up; the SwiGLU takes the bf16-rounded G
// and U, as the streamed kernel does.  G and U are stored when g_out is
// non-null, A when a_out is.
__global__ __launch_bounds__(GateUpFwd::kThreads) void k_gateup_fwd_rows(
    const bf16_t* __restrict__ xp, const int32_t* __restrict__ xp_rows, int64_t xp_bytes,
    const bf16_t* __restrict__ w_gate, const bf16_t* __restrict__ w_up, const int32_t* __restrict__ tile_start,
    const int2* __restrict__ tile_desc, int E, int H, int F, bf16_t* __restrict__ g_out, bf16_t* __restrict__ u_out,
    bf16_t* __restrict__ a_out) {
  using C = GateUpFwd;
  static_assert(C::BM == kRowTile, "grouped products tile rows in units of kRowTile");
  __shared__ __attribute__((aligned(16))) char smem[C::kLds];
  for_each_grouped_tile(tile_start, tile_desc, E, F / C::BNS, [&](const MTile& t) {
    f32x4 acc[C::FM][C::FN];
    zero_acc<C>(acc);
    const int n0 = t.nt * C::BNS;
    const int64_t wofs = static_cast<int64_t>(t.e) * H * F + n0;
    const bf16_t* bs[2] = {w_gate + wofs, w_up + wofs};
    gemm_mainloop<C, true, false>(xp, H, t.m_lim, bs, F, F - n0, H, smem, acc, xp_rows + t.m0, xp_bytes);
    const int lane = threadIdx.x & 63;
#pragma unroll
    for (int mi = 0; mi < C::FM; ++mi) {
      const int r = frag_row<C>(mi, lane);
      if (r >= t.m_lim) continue;
      const int64_t base = static_cast<int64_t>(t.m0 + r) * F + n0;
#pragma unroll
      for (int ni = 0; ni < C::FN / 2; ++ni) {
        const int c = frag_col<C>(ni, lane);  // column within the W_gate half
        const uint2 gw = pack4_bf16(acc[mi][ni]), uw = pack4_bf16(acc[mi][ni + C::FN / 2]);
        const float gv[4] = {lo_bf(gw.x), hi_bf(gw.x), lo_bf(gw.y), hi_bf(gw.y)};
        const float uv[4] = {lo_bf(uw.x), hi_bf(uw.x), lo_bf(uw.y), hi_bf(uw.y)};
        f32x4 av;
#pragma unroll
        for (int i = 0; i < 4; ++i) av[i] = silu_f(gv[i]) * uv[i];
        if (g_out != nullptr) {
          *reinterpret_cast<uint2*>(g_out + base + c) = gw;
          *reinterpret_cast<uint2*>(u_out + base + c) = uw;
        }
        if (a_out != nullptr) *reinterpret_cast<uint2*>(a_out + base + c) = pack4_bf16(av);
      }
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

// Weight-gradient schedule.  Every tile of an expert's weight gradient
// reduces over that expert's rows (K = n_e), so under skewed routing tile
// lengths differ by an order of magnitude and equal tile counts per XCD are
// far from equal work.  A plan built on the device from the offsets
// (k_wgrad_plan, one small launch per backward) orders the experts by
// descending rows (ties to the lower index) and numbers the tiles expert by
// expert in that order; XCD x takes the tiles whose cumulative work (K steps
// plus kTileFixed per tile) starts in [x W / 8, (x + 1) W / 8), W the total,
// and the workgroups of an XCD take its tiles round-robin, longest first.
// An expert's tiles stay on one or two XCDs, so its rows are fetched into few
// L2s.  Each tile is still computed whole by one workgroup: the schedule
// changes no result.
// k_wgrad_plan: the plan (wgrad_plan.hpp) as a launch of its own.
__global__ __launch_bounds__(256) void k_wgrad_plan(const int32_t* __restrict__ offsets, int E, int tpe0, int tpe1,
                                                    int32_t* __restrict__ plan) {
  build_wgrad_plan(offsets, E, tpe0, tpe1, plan);
}

// Job i of this workgroup in weight gradient q (expert e, rows [m0, m0+BM),
// columns [n0, n0+BNS) of each of its NB M x N gradients): tile
// first[x] + j + i n of the plan, x this workgroup's XCD, j its index among
// the XCD's n workgroups.
template <class C>
__device__ __forceinline__ bool wgrad_locate(int i, const int32_t* plan, int q, int E, int M, int N, int& e, int& m0,
                                             int& n0) {
  const int nn = N / C::BNS;
  const int tpe = (M / C::BM) * nn;
  const int x = static_cast<int>(blockIdx.x) & (kPlanXcds - 1);
  const int32_t* first = plan + E + q * (kPlanXcds + 1) + x;
  const int t = uniform_load(first) + static_cast<int>(blockIdx.x >> 3) + i * static_cast<int>(gridDim.x >> 3);
  if (t >= uniform_load(first + 1)) return false;
  const int pos = t / tpe, rem = t - pos * tpe;
  e = uniform_load(plan + pos);
  m0 = (rem / nn) * C::BM;
  n0 = (rem % nn) * C::BNS;
  return true;
}

// dW_down[e] (F x H) = A_e^T dO_e.
template <class C_, bool F32>
struct DownWgradJobs : StagedCopyOut<C_, DownWgradJobs<C_, F32>> {
  using C = C_;
  const int32_t* offsets;
  const int32_t* plan;
  const bf16_t *act, *d_o;
  int E, H, F;
  void* dw_down;
  __device__ bool get(int i, Job<C>& j) const {
    int e, m0, n0;
    if (!wgrad_locate<C>(i, plan, 0, E, F, H, e, m0, n0)) return false;
    const int r0 = uniform_load(offsets + e);
    j.a = act + static_cast<int64_t>(r0) * F + m0;
    j.lda = F;
    j.m_lim = C::BM;
    j.b[0] = d_o + static_cast<int64_t>(r0) * H + n0;
    j.ldb = H;
    j.n_lim = C::BN;
    j.K = uniform_load(offsets + e + 1) - r0;
    j.chain = false;
    j.e = e;
    j.m0 = m0;
    j.n0 = n0;
    return true;
  }
  static constexpr bool kStaged = !F32;  // bf16 gradients leave through the LDS staging area
  __device__ void stage_dst(const Job<C>& j, bf16_t* (&dst)[C::NB], int64_t& ld, int& rows) const {
    dst[0] = static_cast<bf16_t*>(dw_down) + static_cast<int64_t>(j.e) * F * H + static_cast<int64_t>(j.m0) * H + j.n0;
    ld = H;
    rows = C::BM;
  }
  __device__ void epilogue(const Job<C>& j, f32x4 (&acc)[C::FM][C::FN]) const {
    const int lane = threadIdx.x & 63;
    const int64_t obase = static_cast<int64_t>(j.e) * F * H;
#pragma unroll
    for (int mi = 0; mi < C::FM; ++mi) {
      const int64_t row = obase + static_cast<int64_t>(j.m0 + frag_row<C>(mi, lane)) * H + j.n0;
#pragma unroll
      for (int ni = 0; ni < C::FN; ++ni) store4<F32>(dw_down, row + frag_col<C>(ni, lane), acc[mi][ni]);
    }
  }
};

// dW_gate[e] = Xp_e^T dG_e, dW_up[e] = Xp_e^T dU_e  (H x F each).
template <class C_, bool F32>
struct GateUpWgradJobs : StagedCopyOut<C_, GateUpWgradJobs<C_, F32>> {
  using C = C_;
  const int32_t* offsets;
  const int32_t* plan;
  const bf16_t *xp, *dg_in, *du_in;
  int E, H, F;
  void *dw_gate, *dw_up;
  __device__ bool get(int i, Job<C>& j) const {
    int e, m0, n0;
    if (!wgrad_locate<C>(i, plan, 1, E, H, F, e, m0, n0)) return false;
    const int r0 = uniform_load(offsets + e);
    const int64_t bofs = static_cast<int64_t>(r0) * F + n0;
    j.a = xp + static_cast<int64_t>(r0) * H + m0;
    j.lda = H;
    j.m_lim = C::BM;
    j.b[0] = dg_in + bofs;
    j.b[1] = du_in + bofs;
    j.ldb = F;
    j.n_lim = C::BNS;
    j.K = uniform_load(offsets + e + 1) - r0;
    j.chain = false;
    j.e = e;
    j.m0 = m0;
    j.n0 = n0;
    return true;
  }
  static constexpr bool kStaged = !F32;
  __device__ void stage_dst(const Job<C>& j, bf16_t* (&dst)[C::NB], int64_t& ld, int& rows) const {
    const int64_t o = static_cast<int64_t>(j.e) * H * F + static_cast<int64_t>(j.m0) * F + j.n0;
    dst[0] = static_cast<bf16_t*>(dw_gate) + o;
    dst[1] = static_cast<bf16_t*>(dw_up) + o;
    ld = F;
    rows = C::BM;
  }
  __device__ void epilogue(const Job<C>& j, f32x4 (&acc)[C::FM][C::FN]) const {
    const int lane = threadIdx.x & 63;
    const int64_t obase = static_cast<int64_t>(j.e) * H * F;
#pragma unroll
    for (int mi = 0; mi < C::FM; ++mi) {
      const int64_t row = obase + static_cast<int64_t>(j.m0 + frag_row<C>(mi, lane)) * F + j.n0;
#pragma unroll
      for (int ni = 0; ni < C::FN / 2; ++ni) {
        store4<F32>(dw_gate, row + frag_col<C>(ni, lane), acc[mi][ni]);
        store4<F32>(dw_up, row + frag_col<C>(ni, lane), acc[mi][ni + C::FN / 2]);
      }
    }
  }
};

// Adapter weight gradients: out[e] = X_e^T Y_e with X [rows][M] (ld ldx) and
// Y [rows][rank], K = rows of expert e, stored [E][M][rank] or, with trans,
// [E][rank][M] (the b matrices): d a1 = Xp^T Q1, d a2 = A^T Q2,
// d b2 = P2^T dO, d b1 = P1^T dG / dU.  Experts with no rows: zeros.
using LoraW = Tile<128, 16, 1, 2, 1>;
template <bool F32>
struct LoraWgradJobs {
  using C = LoraW;
  const int32_t* offsets;
  const bf16_t* x;
  int64_t ldx;
  int M;
  const bf16_t* y;
  int E, rank;
  bool trans;
  void* out;
  __device__ bool get(int i, Job<C>& j) const {
    const int nm = M / C::BM, nq = rank / C::BN;
    const int logical = xcd_tile(blockIdx.x, gridDim.x) + i * gridDim.x;
    if (logical >= E * nm * nq) return false;
    const int e = logical / (nm * nq);
    const int rem = logical - e * nm * nq;
    const int r0 = uniform_load(offsets + e);
    j.m0 = (rem / nq) * C::BM;
    j.n0 = (rem % nq) * C::BN;
    j.a = x + static_cast<int64_t>(r0) * ldx + j.m0;
    j.lda = ldx;
    j.m_lim = C::BM;
    j.b[0] = y + static_cast<int64_t>(r0) * rank + j.n0;
    j.ldb = rank;
    j.n_lim = C::BN;
    j.K = uniform_load(offsets + e + 1) - r0;
    j.chain = false;
    j.e = e;
    return true;
  }
  __device__ void epilogue(const Job<C>& j, f32x4 (&acc)[C::FM][C::FN]) const {
    const int lane = threadIdx.x & 63;
    const int64_t obase = static_cast<int64_t>(j.e) * M * rank;
#pragma unroll
    for (int mi = 0; mi < C::FM; ++mi) {
      const int m = j.m0 + frag_row<C>(mi, lane);
      const int q = j.n0 + frag_col<C>(0, lane);
      if (!trans) {
        store4<F32>(out, obase + static_cast<int64_t>(m) * rank + q, acc[mi][0]);
      } else {
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const int64_t o = obase + static_cast<int64_t>(q + i) * M + m;
          if constexpr (F32) static_cast<float*>(out)[o] = acc[mi][0][i];
          else static_cast<bf16_t*>(out)[o] = f2bf(acc[mi][0][i]);
        }
      }
    }
  }
};

// ---------------------------------------------------------------- row-tile products as job streams
// The products over each expert's rows run as job streams (gemm_stream):
// job i of a workgroup is segment i % NSEG of logical tile
// xcd_run(i / NSEG, .) of the tile_start[E] x n_ntiles tiles (row tile from
// the tile table, column tile nt: each XCD works through a contiguous run of
// row tiles, so an expert's weights are fetched into one L2); the segments of a
// tile (two halves of a K = 2F reduction, an adapter term) chain into one
// accumulator.  The table is read through the scalar cache, and the tiles
// leave through the LDS staging area, so the pipeline runs on across tiles.
template <int NSEG>
__device__ __forceinline__ bool row_job(int i, const int32_t* tile_start, const int2* tile_desc, int E, int n_ntiles,
                                        MTile& t, int& seg) {
  const int total = uniform_load(tile_start + E) * n_ntiles;
  const int ti = i / NSEG;
  const int logical = xcd_tile(blockIdx.x, gridDim.x) + ti * gridDim.x;
  if (logical >= total) return false;
  const int mt = logical / n_ntiles;
  const uint64_t d = uniform_load(reinterpret_cast<const uint64_t*>(tile_desc + mt));  // {x, y}: x in the low half
  const int dy = static_cast<int>(d >> 32);
  t.e = dy & 0xff;
  t.m_lim = dy >> 8;
  t.m0 = static_cast<int>(static_cast<uint32_t>(d));
  t.nt = logical - mt * n_ntiles;
  seg = i - ti * NSEG;
  return true;
}

template <class C>
__device__ __forceinline__ void row_job_fill(Job<C>& j, const MTile& t, int n0, int n_lim) {
  j.m_lim = t.m_lim;
  j.n_lim = n_lim;
  j.e = t.e;
  j.m0 = t.m0;
  j.n0 = n0;
}

// O = A W_down[e]  (K = F, N = H); with kLora a second segment P2 b2[e]
// (P2 = scale A a2, [rows][r]; b2 [E][r][H], MN-contiguous like W_down).
template <class C_, bool kLora>
struct DownFwdJobs : StagedCopyOut<C_, DownFwdJobs<C_, kLora>, /*kKeep=*/true> {  // O: the combine reads it next
  using C = C_;
  const bf16_t *act, *w_down;
  const int32_t* tile_start;
  const int2* tile_desc;
  int E, H, F;
  bf16_t* o;
  LoraSeg lo;
  __device__ bool get(int i, Job<C>& j) const {
    MTile t;
    int seg;
    if (!row_job<kLora ? 2 : 1>(i, tile_start, tile_desc, E, H / C::BN, t, seg)) return false;
    const int n0 = t.nt * C::BN;
    row_job_fill(j, t, n0, H - n0);
    if (seg == 0) {
      j.a = act + static_cast<int64_t>(t.m0) * F;
      j.lda = F;
      j.b[0] = w_down + static_cast<int64_t>(t.e) * F * H + n0;
      j.ldb = H;
      j.K = F;
      j.chain = kLora;
    } else {
      j.a = lo.a + static_cast<int64_t>(t.m0) * lo.rank;
      j.lda = lo.rank;
      j.b[0] = lo.b0 + static_cast<int64_t>(t.e) * lo.rank * H + n0;
      j.ldb = H;
      j.K = lo.rank;
      j.chain = false;
    }
    return true;
  }
  __device__ void stage_dst(const Job<C>& j, bf16_t* (&dst)[C::NB], int64_t& ld, int& rows) const {
    dst[0] = o + static_cast<int64_t>(j.m0) * H + j.n0;
    ld = H;
    rows = j.m_lim;
  }
};

// dXp = dG W_gate[e]^T + dU W_up[e]^T  (K = 2F as two segments, N = H); with
// kLora a third segment Q1 a1[e]^T (Q1 = scale (dG b1_gate^T + dU b1_up^T),
// [rows][r]; a1 [E][H][r]: K-contiguous rows of the B tile).  B(k = f,
// n = h) = W[e][h][f]: K-contiguous rows of W_gate / W_up.
template <class C_, bool kLora>
struct GateUpDgradJobs : StagedCopyOut<C_, GateUpDgradJobs<C_, kLora>, /*kKeep=*/true> {  // dXp: the router dX reads it next
  using C = C_;
  const bf16_t *dg, *du, *w_gate, *w_up;
  const int32_t* tile_start;
  const int2* tile_desc;
  int E, H, F;
  bf16_t* dxp;
  LoraSeg lo;
  __device__ bool get(int i, Job<C>& j) const {
    MTile t;
    int seg;
    if (!row_job<kLora ? 3 : 2>(i, tile_start, tile_desc, E, H / C::BN, t, seg)) return false;
    const int n0 = t.nt * C::BN;
    row_job_fill(j, t, n0, H - n0);
    if (seg < 2) {
      const int64_t wofs = static_cast<int64_t>(t.e) * H * F + static_cast<int64_t>(n0) * F;
      j.a = (seg == 0 ? dg : du) + static_cast<int64_t>(t.m0) * F;
      j.lda = F;
      j.b[0] = (seg == 0 ? w_gate : w_up) + wofs;
      j.ldb = F;
      j.K = F;
      j.chain = seg == 0 || kLora;
    } else {
      j.a = lo.a + static_cast<int64_t>(t.m0) * lo.rank;
      j.lda = lo.rank;
      j.b[0] = lo.b0 + (static_cast<int64_t>(t.e) * H + n0) * lo.rank;
      j.ldb = lo.rank;
      j.K = lo.rank;
      j.chain = false;
    }
    return true;
  }
  __device__ void stage_dst(const Job<C>& j, bf16_t* (&dst)[C::NB], int64_t& ld, int& rows) const {
    dst[0] = dxp + static_cast<int64_t>(j.m0) * H + j.n0;
    ld = H;
    rows = j.m_lim;
  }
};

// Staged-drain unit of the SwiGLU epilogues: 8 consecutive columns of one
// row.  A slice gives every thread one unit: kCpr units per row, lanes
// l / kCpr of a wave on consecutive rows.
template <class C, int kCols>
struct RowUnits {
  static constexpr int kCpr = kCols / 8;
  static constexpr int kRowsPerWave = 64 / kCpr;
  static constexpr int kSliceRows = C::kThreads / 64 * kRowsPerWave;
  static constexpr int kSlices = C::BM / kSliceRows;
  static_assert(64 % kCpr == 0 && kSlices * kSliceRows == C::BM && kSlices % 2 == 0 && kSliceRows % 16 == 0,
                "an even number of slices of 16k rows");
  __device__ static __forceinline__ int row(int sl) {
    return (threadIdx.x >> 6) * kRowsPerWave + (threadIdx.x & 63) / kCpr + sl * kSliceRows;
  }
  __device__ static __forceinline__ int chunk() { return (threadIdx.x & 63) % kCpr; }
};

__device__ __forceinline__ void unpack8(const uint4& w, float (&f)[8]) {
  const uint32_t v[4] = {w.x, w.y, w.z, w.w};
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    f[2 * i] = lo_bf(v[i]);
    f[2 * i + 1] = hi_bf(v[i]);
  }
}
__device__ __forceinline__ uint4 pack8(const float (&f)[8]) {
  return make_uint4(pack_bf16x2(f[0], f[1]), pack_bf16x2(f[2], f[3]), pack_bf16x2(f[4], f[5]),
                    pack_bf16x2(f[6], f[7]));
}

// G, U (gate/up products) and A = silu(G) U per expert, with the SwiGLU on the
// bf16 G and U; G and U are skipped when g_out is null, A when a_out is.
// With kLora a second segment P1 [b1_gate | b1_up][e] (P1 = scale Xp a1,
// [rows][r]; b1 [E][r][F], MN-contiguous like W_gate).
template <bool kLora>
struct GateUpFwdJobs {
  static constexpr bool kOpaqueSetup = kLora;  // short of registers with the adapter segment
  using C = GateUpFwd;
  const bf16_t *xp, *w_gate, *w_up;
  const int32_t* tile_start;
  const int2* tile_desc;
  int E, H, F;
  bf16_t *g_out, *u_out, *a_out;
  LoraSeg lo;
  __device__ bool get(int i, Job<C>& j) const {
    MTile t;
    int seg;
    if (!row_job<kLora ? 2 : 1>(i, tile_start, tile_desc, E, F / C::BNS, t, seg)) return false;
    const int n0 = t.nt * C::BNS;
    row_job_fill(j, t, n0, F - n0);
    if (seg == 0) {
      const int64_t wofs = static_cast<int64_t>(t.e) * H * F + n0;
      j.a = xp + static_cast<int64_t>(t.m0) * H;
      j.lda = H;
      j.b[0] = w_gate + wofs;
      j.b[1] = w_up + wofs;
      j.ldb = F;
      j.K = H;
      j.chain = kLora;
    } else {
      const int64_t lofs = static_cast<int64_t>(t.e) * lo.rank * F + n0;
      j.a = lo.a + static_cast<int64_t>(t.m0) * lo.rank;
      j.lda = lo.rank;
      j.b[0] = lo.b0 + lofs;
      j.b[1] = lo.b1 + lofs;
      j.ldb = F;
      j.K = lo.rank;
      j.chain = false;
    }
    return true;
  }
  // staged drain: one slice per call; unit (row, 8 columns) reads G (gate
  // block) and U (up block) and stores G, U and A
  using Units = RowUnits<C, C::BNS>;
  static constexpr bool kStaged = true;
  static constexpr int kDrainCalls = Units::kSlices;
  struct Drain {
    int64_t base;  // element offset of the tile's (0, 0) in G, U and A
    int rows;
  };
  __device__ __forceinline__ void drain_reset(Drain& d) const {
    d.base = 0;
    d.rows = 0;
  }
  __device__ __forceinline__ void drain_setup(const Job<C>& j, Drain& d) const {
    d.base = static_cast<int64_t>(j.m0) * F + j.n0;
    d.rows = j.m_lim;
  }
  __device__ __forceinline__ void drain(Drain& d, const char* stg, int sl) const {
    const int s = sl < Units::kSlices ? sl : Units::kSlices - 1;
    const int r = Units::row(s), c = Units::chunk();
    const uint4 gw = *reinterpret_cast<const uint4*>(stg + Staged<C>::off(r, c));
    const uint4 uw = *reinterpret_cast<const uint4*>(stg + Staged<C>::off(r, Units::kCpr + c));
    float gv[8], uv[8], av[8];
    unpack8(gw, gv);
    unpack8(uw, uv);
#pragma unroll
    for (int i = 0; i < 8; ++i) av[i] = silu_f(gv[i]) * uv[i];
    const uint32_t off = sl < Units::kSlices ? static_cast<uint32_t>(r * F * 2 + c * 16) : kOob;
    const int rows_gu = g_out != nullptr ? d.rows : 0, rows_a = a_out != nullptr ? d.rows : 0;
    buf_store16(rows_rsrc(g_out + d.base, rows_gu, F * 2, C::BNS * 2), off, gw);
    buf_store16(rows_rsrc(u_out + d.base, rows_gu, F * 2, C::BNS * 2), off, uw);
    buf_store16(rows_rsrc(a_out + d.base, rows_a, F * 2, C::BNS * 2), off, pack8(av));
  }
};

// Sum over aligned groups of N = 16 or 32 lanes with DPP moves (no LDS round
// trips), in a fixed order: pairs, quads, eights, sixteens, and for N = 32
// the two 16-lane rows.  The group total is in every lane of a 16-lane group,
// and for N = 32 in the upper 16 lanes of the group.
template <int kCtrl, int kRowMask>
__device__ __forceinline__ float dpp_f(float x) {
  return __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(0, __builtin_bit_cast(int, x), kCtrl, kRowMask, 0xf,
                                                               false));
}
template <int N>
__device__ __forceinline__ float row_sum_dpp(float v) {
  static_assert(N == 16 || N == 32, "16- or 32-lane groups");
  v += dpp_f<0xB1, 0xf>(v);   // quad_perm [1, 0, 3, 2]: lane ^ 1
  v += dpp_f<0x4E, 0xf>(v);   // quad_perm [2, 3, 0, 1]: lane ^ 2
  v += dpp_f<0x141, 0xf>(v);  // row_half_mirror: the other quad of each 8 lanes
  v += dpp_f<0x140, 0xf>(v);  // row_mirror: the other 8 of each 16 lanes
  if constexpr (N == 32) v += dpp_f<0x142, 0xa>(v);  // row_bcast15 into rows 1 and 3 (rows 0 and 2 add 0)
  return v;
}

// dA = dO W_down[e]^T (K = H, N = F) fused with the SwiGLU backward:
// s = sigmoid(G); dG = dA U s (1 + G (1 - s)); dU = dA G s, with dA the
// bf16 product.  dG and dU may overwrite G and U in place: each element of
// G and U is read by the one thread that later writes the same element of
// dG and dU, and by no one else.  With kLora a second segment Q2 a2[e]^T
// (Q2 = scale dO b2^T, [rows][r]; a2 [E][F][r]: K-contiguous rows of the B
// tile).  B(k = h, n = f) = W_down[e][f][h]: K-contiguous rows of W_down.
template <class C_, bool kLora>
struct DownDgradJobs {
  static constexpr bool kOpaqueSetup = kLora;  // short of registers with the adapter segment
  using C = C_;
  const bf16_t *d_o, *w_down;
  const bf16_t *g_in, *u_in;
  const int32_t* tile_start;
  const int2* tile_desc;
  int E, H, F;
  bf16_t *dg_out, *du_out;
  LoraSeg lo;
  float* part;  // [rows][F / BN]: <dA, A> per row and column block, or null
  __device__ bool get(int i, Job<C>& j) const {
    MTile t;
    int seg;
    if (!row_job<kLora ? 2 : 1>(i, tile_start, tile_desc, E, F / C::BN, t, seg)) return false;
    const int n0 = t.nt * C::BN;
    row_job_fill(j, t, n0, F - n0);
    if (seg == 0) {
      j.a = d_o + static_cast<int64_t>(t.m0) * H;
      j.lda = H;
      j.b[0] = w_down + static_cast<int64_t>(t.e) * F * H + static_cast<int64_t>(n0) * H;
      j.ldb = H;
      j.K = H;
      j.chain = kLora;
    } else {
      j.a = lo.a + static_cast<int64_t>(t.m0) * lo.rank;
      j.lda = lo.rank;
      j.b[0] = lo.b0 + (static_cast<int64_t>(t.e) * F + n0) * lo.rank;
      j.ldb = lo.rank;
      j.K = lo.rank;
      j.chain = false;
    }
    return true;
  }
  // staged drain: one slice per call; unit (row, 8 columns) of dA, whose G
  // and U were loaded by the previous call (or the setup).  With the adapter
  // segment the stream has no registers to spare for that: G and U are then
  // loaded in the call itself (its wait drains the loads in flight, which
  // costs less than the spills the prefetch causes there).  With `part` the
  // call also sums dA A = dU U over each of its rows' BN columns (fp32, the
  // A = silu(G) U of the G and U it holds; a fixed DPP tree over the lanes of
  // a row) for the gate gradient.
  static constexpr bool kPrefetch = !kLora;
  using Units = RowUnits<C, C::BN>;
  static constexpr bool kStaged = true;
  static constexpr bool kDrainLate = true;  // its G and U loads go after the step's operand loads
  static constexpr int kDrainCalls = Units::kSlices;
  struct Drain {
    int64_t base;   // element offset of the tile's (0, 0) in G, U, dG and dU
    int64_t pbase;  // element offset of the tile's first row and column block in part
    int rows;
    uint4 gw, uw;  // G and U of the next call's unit
  };
  __device__ __forceinline__ void drain_reset(Drain& d) const {
    d.base = 0;
    d.pbase = 0;
    d.rows = 0;
    d.gw = d.uw = make_uint4(0, 0, 0, 0);
  }
  __device__ __forceinline__ uint32_t unit_off(int sl) const {
    return sl < Units::kSlices ? static_cast<uint32_t>(Units::row(sl) * F * 2 + Units::chunk() * 16) : kOob;
  }
  __device__ __forceinline__ void prefetch(Drain& d, int sl) const {
    d.gw = buf_load16(rows_rsrc(g_in + d.base, d.rows, F * 2, C::BN * 2), unit_off(sl));
    d.uw = buf_load16(rows_rsrc(u_in + d.base, d.rows, F * 2, C::BN * 2), unit_off(sl));
  }
  __device__ __forceinline__ void drain_setup(const Job<C>& j, Drain& d) const {
    d.base = static_cast<int64_t>(j.m0) * F + j.n0;
    d.pbase = static_cast<int64_t>(j.m0) * (F / C::BN) + j.n0 / C::BN;
    d.rows = j.m_lim;
    if constexpr (kPrefetch) prefetch(d, 0);
  }
  __device__ __forceinline__ void drain(Drain& d, const char* stg, int sl) const {
    const int s = sl < Units::kSlices ? sl : Units::kSlices - 1;
    const int r = Units::row(s), c = Units::chunk();
    if constexpr (!kPrefetch) prefetch(d, sl);
    float da[8], gv[8], uv[8], dgv[8], duv[8];
    unpack8(*reinterpret_cast<const uint4*>(stg + Staged<C>::off(r, c)), da);
    unpack8(d.gw, gv);
    unpack8(d.uw, uv);
    float dot = 0.0f;
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      const float sg = sigmoid_f(gv[i]);
      dgv[i] = da[i] * uv[i] * sg * (1.0f + gv[i] * (1.0f - sg));
      duv[i] = da[i] * gv[i] * sg;
      dot += duv[i] * uv[i];  // dA silu(G) U = dA A
    }
    buf_store16(rows_rsrc(dg_out + d.base, d.rows, F * 2, C::BN * 2), unit_off(sl), pack8(dgv));
    buf_store16(rows_rsrc(du_out + d.base, d.rows, F * 2, C::BN * 2), unit_off(sl), pack8(duv));
    // unconditional (a null `part` gets an empty resource), so the stream's
    // vector-memory count per call is fixed and its waits stay exact
    dot = row_sum_dpp<Units::kCpr>(dot);
    const int np = F / C::BN;
    const bool writer = c == (Units::kCpr == 32 ? 16 : 0);
    const uint32_t poff = (writer && sl < Units::kSlices) ? static_cast<uint32_t>(r * np * 4) : kOob;
    __builtin_amdgcn_raw_buffer_store_b32(__builtin_bit_cast(uint32_t, dot),
                                          rows_rsrc(part != nullptr ? part + d.pbase : nullptr,
                                                    part != nullptr ? d.rows : 0, np * 4, 4),
                                          static_cast<int>(poff), 0, 0);
    if constexpr (kPrefetch) prefetch(d, sl + 1);
  }
};

// One persistent kernel for every product: the job provider decides.
template <class P, bool A_KC, bool B_KC>
__global__ __launch_bounds__(P::C::kThreads) void k_stream(P prov) {
  __shared__ __attribute__((aligned(16))) char smem[stream_lds<P>()];
  gemm_stream<typename P::C, A_KC, B_KC>(prov, smem);
}

inline int grid8(int64_t n) { return static_cast<int>(cdiv64(n, 8) * 8); }

// Persistent grid: as many workgroups as can be resident on the device at
// once (queried per kernel and device, then cached; the cache is shared by
// every host thread, under a lock), rounded down to a multiple of 8, and no
// more than the worst-case tile count needs.
int resident_workgroups(const void* kernel, int threads) {
  struct Entry {
    const void* kernel;
    int dev, blocks;
  };
  static std::mutex lock;
  static Entry cache[64];
  static int used = 0;
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess) dev = 0;
  std::lock_guard<std::mutex> guard(lock);
  for (int i = 0; i < used; ++i)
    if (cache[i].kernel == kernel && cache[i].dev == dev) return cache[i].blocks;
  int cus = 0, per_cu = 0;
  if (hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || cus <= 0)
    cus = 256;
  if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, kernel, threads, 0) != hipSuccess || per_cu <= 0)
    per_cu = 1;
  const int blocks = std::max(8, (cus * per_cu) / 8 * 8);
  if (used < 64) cache[used++] = Entry{kernel, dev, blocks};
  return blocks;
}

template <typename Kernel>
int persistent_grid(Kernel kernel, int threads, int64_t max_tiles) {
  const int resident = resident_workgroups(reinterpret_cast<const void*>(kernel), threads);
  return static_cast<int>(std::min<int64_t>(grid8(max_tiles), resident));
}

}  // namespace

// Upper bound of the number of 128-row tiles over all experts.
int max_row_tiles(int rows_cap, int E) { return cdiv(rows_cap, kRowTile) + E; }

int wgrad_plan_ints(int E) { return E + 2 * (kPlanXcds + 1); }


// The dgrad of the down product runs 256-column tiles when F allows, else 128.
int dgate_parts(int F) { return F % 256 == 0 ? F / 256 : F / 128; }

namespace {

// Tile shapes: 128 rows x 256 columns over 8 waves (2 x 4, 64 x 64 each, two
// waves per SIMD so one's MFMAs cover the other's LDS waits); 128 x 128 over
// 4 waves when a dimension is not a multiple of 256.
using Wide = Tile<128, 256, 1, 2, 4>;
using Narrow = Tile<128, 128, 1, 2, 2>;
using WideGU = Tile<128, 256, 2, 2, 4>;

template <bool A_KC, bool B_KC, class P>
void run_stream(const P& prov, int64_t max_jobs, int kid, hipStream_t s) {
  auto k = k_stream<P, A_KC, B_KC>;
  const int grid = persistent_grid(k, P::C::kThreads, max_jobs);
  TraceScope trace_scope(kid, s);
  hipLaunchKernelGGL(k, dim3(grid), dim3(P::C::kThreads), 0, s, prov);
}

template <class C>
void down_fwd(const ExpertArgs& a, bf16_t* o, hipStream_t s) {
  LoraSeg lo;
  if (a.lora.rank > 0) {
    lo.a = a.lora.p2;
    lo.b0 = a.lora.b2;
    lo.rank = a.lora.rank;
  }
  const int64_t tiles = static_cast<int64_t>(max_row_tiles(a.rows_cap, a.E)) * (a.H / C::BN);
  if (lo.rank > 0)
    run_stream<true, false>(DownFwdJobs<C, true>{{}, a.act, a.w_down, a.tile_start, a.tile_desc, a.E, a.H, a.F, o, lo},
                            tiles, K_DOWN_FWD, s);
  else
    run_stream<true, false>(DownFwdJobs<C, false>{{}, a.act, a.w_down, a.tile_start, a.tile_desc, a.E, a.H, a.F, o, lo},
                            tiles, K_DOWN_FWD, s);
}

template <class C>
void down_dgrad(const ExpertArgs& a, const bf16_t* d_o, bf16_t* dg, bf16_t* du, const bf16_t* q2, hipStream_t s) {
  LoraSeg lo;
  if (q2 != nullptr) {
    lo.a = q2;
    lo.b0 = a.lora.a2;
    lo.rank = a.lora.rank;
  }
  const int64_t tiles = static_cast<int64_t>(max_row_tiles(a.rows_cap, a.E)) * (a.F / C::BN);
  if (lo.rank > 0)
    run_stream<true, true>(DownDgradJobs<C, true>{d_o, a.w_down, a.g, a.u, a.tile_start, a.tile_desc, a.E, a.H, a.F,
                                                  dg, du, lo, a.dgate_part},
                           tiles, K_DOWN_DGRAD, s);
  else
    run_stream<true, true>(DownDgradJobs<C, false>{d_o, a.w_down, a.g, a.u, a.tile_start, a.tile_desc, a.E, a.H, a.F,
                                                   dg, du, lo, a.dgate_part},
                           tiles, K_DOWN_DGRAD, s);
}

template <class C>
void gateup_dgrad(const ExpertArgs& a, const bf16_t* dg, const bf16_t* du, bf16_t* dxp, const bf16_t* q1,
                  hipStream_t s) {
  LoraSeg lo;
  if (q1 != nullptr) {
    lo.a = q1;
    lo.b0 = a.lora.a1;
    lo.rank = a.lora.rank;
  }
  const int64_t tiles = static_cast<int64_t>(max_row_tiles(a.rows_cap, a.E)) * (a.H / C::BN);
  if (lo.rank > 0)
    run_stream<true, true>(GateUpDgradJobs<C, true>{{}, dg, du, a.w_gate, a.w_up, a.tile_start, a.tile_desc, a.E, a.H,
                                                    a.F, dxp, lo},
                           tiles, K_GATEUP_DGRAD, s);
  else
    run_stream<true, true>(GateUpDgradJobs<C, false>{{}, dg, du, a.w_gate, a.w_up, a.tile_start, a.tile_desc, a.E,
                                                     a.H, a.F, dxp, lo},
                           tiles, K_GATEUP_DGRAD, s);
}

template <class C, bool F32>
void down_wgrad(const ExpertArgs& a, const bf16_t* d_o, void* dw_down, hipStream_t s) {
  DownWgradJobs<C, F32> p{{}, a.offsets, a.wgrad_plan, a.act, d_o, a.E, a.H, a.F, dw_down};
  run_stream<false, false>(p, static_cast<int64_t>(a.E) * (a.F / C::BM) * (a.H / C::BNS), K_DOWN_WGRAD, s);
}

template <class C, bool F32>
void gateup_wgrad(const ExpertArgs& a, const bf16_t* dg, const bf16_t* du, void* dw_gate, void* dw_up,
                  hipStream_t s) {
  GateUpWgradJobs<C, F32> p{{}, a.offsets, a.wgrad_plan, a.xp, dg, du, a.E, a.H, a.F, dw_gate, dw_up};
  run_stream<false, false>(p, static_cast<int64_t>(a.E) * (a.H / C::BM) * (a.F / C::BNS), K_GATEUP_WGRAD, s);
}

template <class C>
void down_wgrad_any(const ExpertArgs& a, const bf16_t* d_o, void* dw, bool f32, hipStream_t s) {
  if (f32) down_wgrad<C, true>(a, d_o, dw, s);
  else down_wgrad<C, false>(a, d_o, dw, s);
}

template <class C>
void gateup_wgrad_any(const ExpertArgs& a, const bf16_t* dg, const bf16_t* du, void* dwg, void* dwu, bool f32,
                      hipStream_t s) {
  if (f32) gateup_wgrad<C, true>(a, dg, du, dwg, dwu, s);
  else gateup_wgrad<C, false>(a, dg, du, dwg, dwu, s);
}

}  // namespace

void wgrad_tiles_per_expert(int H, int F, int& tpe_down, int& tpe_gu) {
  tpe_down = H % 256 == 0 ? (F / Wide::BM) * (H / Wide::BNS) : (F / Narrow::BM) * (H / Narrow::BNS);
  tpe_gu = (H / WideGU::BM) * (F / WideGU::BNS);
}

hipError_t launch_gateup_fwd(const ExpertArgs& a, hipStream_t s, bool recompute) {
  using C = GateUpFwd;
  const int64_t tiles = static_cast<int64_t>(max_row_tiles(a.rows_cap, a.E)) * (a.F / C::BNS);
  const int kid = recompute ? K_GATEUP_RECOMPUTE : K_GATEUP_FWD;
  if (a.xp_rows != nullptr) {  // rows read through an index: one pipeline per tile
    auto k = k_gateup_fwd_rows;
    const int grid = persistent_grid(k, C::kThreads, tiles);
    TraceScope trace_scope(kid, s);
    hipLaunchKernelGGL(k, dim3(grid), dim3(C::kThreads), 0, s, a.xp, a.xp_rows, a.xp_bytes, a.w_gate, a.w_up,
                       a.tile_start, a.tile_desc, a.E, a.H, a.F, a.g, a.u, a.act);
    return hipGetLastError();
  }
  LoraSeg lo;
  if (a.lora.rank > 0) {
    lo.a = a.lora.p1;
    lo.b0 = a.lora.b1_gate;
    lo.b1 = a.lora.b1_up;
    lo.rank = a.lora.rank;
  }
  if (lo.rank > 0)
    run_stream<true, false>(GateUpFwdJobs<true>{a.xp, a.w_gate, a.w_up, a.tile_start, a.tile_desc, a.E, a.H, a.F, a.g,
                                                a.u, a.act, lo},
                            tiles, kid, s);
  else
    run_stream<true, false>(GateUpFwdJobs<false>{a.xp, a.w_gate, a.w_up, a.tile_start, a.tile_desc, a.E, a.H, a.F,
                                                 a.g, a.u, a.act, lo},
                            tiles, kid, s);
  return hipGetLastError();
}

hipError_t launch_down_fwd(const ExpertArgs& a, bf16_t* o, hipStream_t s) {
  if (a.H % 256 == 0) down_fwd<Wide>(a, o, s);
  else down_fwd<Narrow>(a, o, s);
  return hipGetLastError();
}

hipError_t launch_down_dgrad(const ExpertArgs& a, const bf16_t* d_o, bf16_t* dg, bf16_t* du, const bf16_t* q2,
                             hipStream_t s) {
  if (a.F % 256 == 0) down_dgrad<Wide>(a, d_o, dg, du, q2, s);
  else down_dgrad<Narrow>(a, d_o, dg, du, q2, s);
  return hipGetLastError();
}

hipError_t launch_gateup_dgrad(const ExpertArgs& a, const bf16_t* dg, const bf16_t* du, bf16_t* dxp,
                               const bf16_t* q1, hipStream_t s) {
  if (a.H % 256 == 0) gateup_dgrad<Wide>(a, dg, du, dxp, q1, s);
  else gateup_dgrad<Narrow>(a, dg, du, dxp, q1, s);
  return hipGetLastError();
}

hipError_t launch_experts_bwd_data(const ExpertArgs& a, const bf16_t* d_o, bf16_t* dg, bf16_t* du,
                                   bf16_t* dxp, void* dw_down, bool dw_f32, hipStream_t s) {
  if (!a.wgrad_plan_built) {
    int tpe_down = 0, tpe_gu = 0;
    wgrad_tiles_per_expert(a.H, a.F, tpe_down, tpe_gu);
    TraceScope trace_scope(K_WGRAD_PLAN, s);
    hipLaunchKernelGGL(k_wgrad_plan, dim3(1), dim3(256), 0, s, a.offsets, a.E, tpe_down, tpe_gu, a.wgrad_plan);
  }
  if (a.F % 256 == 0) down_dgrad<Wide>(a, d_o, dg, du, nullptr, s);
  else down_dgrad<Narrow>(a, d_o, dg, du, nullptr, s);
  if (a.H % 256 == 0) down_wgrad_any<Wide>(a, d_o, dw_down, dw_f32, s);
  else down_wgrad_any<Narrow>(a, d_o, dw_down, dw_f32, s);
  if (a.H % 256 == 0) gateup_dgrad<Wide>(a, dg, du, dxp, nullptr, s);
  else gateup_dgrad<Narrow>(a, dg, du, dxp, nullptr, s);
  return hipGetLastError();
}

hipError_t launch_experts_bwd_gateup_w(const ExpertArgs& a, const bf16_t* dg, const bf16_t* du, void* dw_gate,
                                       void* dw_up, bool dw_f32, hipStream_t s) {
  gateup_wgrad_any<WideGU>(a, dg, du, dw_gate, dw_up, dw_f32, s);
  return hipGetLastError();
}

hipError_t launch_experts_bwd(const ExpertArgs& a, const bf16_t* d_o, bf16_t* dg, bf16_t* du,
                              bf16_t* dxp, void* dw_gate, void* dw_up, void* dw_down, bool dw_f32,
                              hipStream_t s) {
  const hipError_t e = launch_experts_bwd_data(a, d_o, dg, du, dxp, dw_down, dw_f32, s);
  if (e != hipSuccess) return e;
  return launch_experts_bwd_gateup_w(a, dg, du, dw_gate, dw_up, dw_f32, s);
}

hipError_t launch_lora_rows(const ExpertArgs& a, const bf16_t* x0, const bf16_t* x1, int64_t ldx,
                            const bf16_t* w0, const bf16_t* w1, int64_t estride, int K, bool b_kc, bf16_t* out,
                            hipStream_t s) {
  using C = LoraRows;
  const int64_t tiles =
      static_cast<int64_t>(max_row_tiles(a.rows_cap, a.E)) * (a.lora.rank / C::BN) * (kRowTile / C::BM);
  TraceScope trace_scope(K_LORA_ROWS, s);
#define MOE_LORA_ROWS(KC, NS)                                                                                   \
  do {                                                                                                          \
    auto k = k_lora_rows<KC, NS>;                                                                               \
    hipLaunchKernelGGL(k, dim3(persistent_grid(k, C::kThreads, tiles)), dim3(C::kThreads), 0, s, x0, x1, ldx, w0, \
                       w1, estride, K, a.tile_start, a.tile_desc, a.E, a.lora.rank, a.lora.scale, out);         \
  } while (0)
  if (b_kc) {
    if (x1 != nullptr) MOE_LORA_ROWS(true, 2);
    else MOE_LORA_ROWS(true, 1);
  } else {
    MOE_LORA_ROWS(false, 1);
  }
#undef MOE_LORA_ROWS
  return hipGetLastError();
}

hipError_t launch_lora_wgrad(const ExpertArgs& a, const bf16_t* x, int64_t ldx, int M, const bf16_t* y, bool trans,
                             void* out, bool f32, hipStream_t s) {
  const int64_t jobs = static_cast<int64_t>(a.E) * (M / LoraW::BM) * (a.lora.rank / LoraW::BN);
  if (f32) {
    LoraWgradJobs<true> p{a.offsets, x, ldx, M, y, a.E, a.lora.rank, trans, out};
    run_stream<false, false>(p, jobs, K_LORA_WGRAD, s);
  } else {
    LoraWgradJobs<false> p{a.offsets, x, ldx, M, y, a.E, a.lora.rank, trans, out};
    run_stream<false, false>(p, jobs, K_LORA_WGRAD, s);
  }
  return hipGetLastError();
}

}  // namespace moe
