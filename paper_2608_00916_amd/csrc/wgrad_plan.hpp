// Schedule of the weight-gradient products, built on the device per
// backward from the expert offsets.
//
// Every tile of an expert's weight gradient reduces over that expert's rows
// (K = n_e), so under skewed routing tile lengths differ by an order of
// magnitude and equal tile counts per XCD are far from equal work.  The plan
// orders the experts by descending rows (ties to the lower index) and numbers
// the tiles expert by expert in that order; XCD x takes the tiles whose
// cumulative work (K steps plus kTileFixed per tile) starts in
// [x W / 8, (x + 1) W / 8), W the total, and the workgroups of an XCD take its
// tiles round-robin, longest first.  An expert's tiles stay on one or two
// XCDs, so its rows are fetched into few L2s.  Each tile is still computed
// whole by one workgroup: the schedule changes no result.
//
// Layout (wgrad_plan_ints(E) ints): plan[0, E) the expert at each position of
// the order; then, per weight gradient q (0: down, 1: gate/up), the first
// tile of XCD x at plan[E + q (kPlanXcds + 1) + x], x = 0..kPlanXcds.
#pragma once

#include "common.hpp"
#include "moe.h"

namespace moe {

constexpr int kPlanXcds = 8;
constexpr int kPlanBK = 64;    // K steps are 64 rows deep
constexpr int kTileFixed = 2;  // a tile's fixed cost (setup, epilogue) in K steps

// One workgroup of 256 threads (E <= 256) builds the plan; tpe0 / tpe1 are the
// tiles per expert of the down and gate/up weight gradients.
__device__ __forceinline__ void build_wgrad_plan(const int32_t* __restrict__ offsets, int E, int tpe0, int tpe1,
                                                 int32_t* __restrict__ plan) {
  static_assert(MOE_MAX_EXPERTS <= 256, "one thread per expert");
  constexpr int kPairs = 2 * (kPlanXcds + 1);
  __shared__ int rows[MOE_MAX_EXPERTS];
  __shared__ int wave_tot[4];
  __shared__ int64_t bound[kPairs];
  __shared__ int cum_at[MOE_MAX_EXPERTS];
  __shared__ int steps_at[MOE_MAX_EXPERTS];
  __shared__ int cnt[4][kPairs];
  const int tid = threadIdx.x, lane = tid & 63, wv = tid >> 6;
  if (tid < E) rows[tid] = offsets[tid + 1] - offsets[tid];
  __syncthreads();
  // position of expert tid in the order: experts with more rows, or as many
  // and a lower index, come first
  int pos = 0, steps = 0;
  if (tid < E) {
    const int ne = rows[tid];
    int rank = 0;
#pragma unroll 8
    for (int f = 0; f < E; ++f) {
      const int nf = rows[f];
      rank += (nf > ne || (nf == ne && f < tid)) ? 1 : 0;
    }
    pos = rank;
    steps = cdiv(ne, kPlanBK) + kTileFixed;
    plan[pos] = tid;
    steps_at[pos] = steps;
  }
  __syncthreads();
  // exclusive prefix sum of the steps over positions (thread p holds position p)
  int v = tid < E ? steps_at[tid] : 0;
  int incl = v;
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) {
    const int u = __shfl_up(incl, o, 64);
    incl += lane >= o ? u : 0;
  }
  if (lane == 63) wave_tot[wv] = incl;
  __syncthreads();
  int before = 0;
  for (int w = 0; w < wv; ++w) before += wave_tot[w];
  const int cum = before + incl - v;  // work of the positions before tid, per tile of each
  if (tid < E) cum_at[tid] = cum;
  const int total = wave_tot[0] + wave_tot[1] + wave_tot[2] + wave_tot[3];
  if (tid < kPairs) {
    const int q = tid / (kPlanXcds + 1), x = tid % (kPlanXcds + 1);
    const int64_t tpe = q == 0 ? tpe0 : tpe1;
    bound[tid] = x * (tpe * total) / kPlanXcds;  // work before XCD x's first tile
  }
  __syncthreads();
  // for each (q, x): the last position whose first tile starts at or before
  // the bound (positions 0..E-1; cum strictly increases)
#pragma unroll
  for (int i = 0; i < kPairs; ++i) {
    const int64_t tpe = i < kPlanXcds + 1 ? tpe0 : tpe1;
    const bool le = tid < E && tpe * cum <= bound[i];
    const int c = __popcll(__ballot(le));
    if (lane == 0) cnt[wv][i] = c;
  }
  __syncthreads();
  if (tid < kPairs) {
    const int q = tid / (kPlanXcds + 1), x = tid % (kPlanXcds + 1);
    const int64_t tpe = q == 0 ? tpe0 : tpe1;
    int64_t t = static_cast<int64_t>(E) * tpe;
    if (x < kPlanXcds) {
      const int p = cnt[0][tid] + cnt[1][tid] + cnt[2][tid] + cnt[3][tid] - 1;
      // first tile of position p whose start is at or past the bound
      const int64_t local = cdiv64(bound[tid] - tpe * cum_at[p], steps_at[p]);
      t = static_cast<int64_t>(p) * tpe + (local < tpe ? local : tpe);
    }
    plan[E + q * (kPlanXcds + 1) + x] = static_cast<int32_t>(t);
  }
}

}  // namespace moe
