// bf16 MFMA GEMM core shared by every matrix product of the MoE block.
//
// One workgroup (256 threads = 4 waves of 64, arranged 2 x 2) computes a
// BM x BN fp32 tile C = A_tile * B_tile over a K loop in steps of BK:
//   C[m][n] = sum_k A(m, k) B(k, n)
// Operands come from global memory in one of two layouts:
//   K-contiguous   element (r, k) at src[r * ld + k]   (a row-major A, or B^T)
//   MN-contiguous  element (r, k) at src[k * ld + r]   (a row-major B, or A^T)
// Both are staged in LDS as [rows][BK] bf16 with K contiguous (128-byte rows,
// 16-byte chunks XOR-swizzled by row so that the MFMA operand reads and the
// tile writes are free of bank conflicts).  MN-contiguous tiles are read as
// 8 x 8 blocks of 16-byte rows and transposed in registers on the way in.
//
// LDS holds two stages: the global loads of step k+1 are in flight while the
// MFMAs of step k run, with one barrier per step.
//
// MFMA v_mfma_f32_16x16x32_bf16 is fed with the B tile as its first operand
// and the A tile as its second, so that each lane ends up holding four
// consecutive columns of one output row:
//   lane l, fragment (mi, ni), register i  ->  C[mb + mi*16 + l%16][nb + ni*16 + 4*(l/16) + i]
#pragma once

#include "common.hpp"

namespace moe {

constexpr int BM = 128, BN = 128, BK = 64;
constexpr int kThreads = 256;
constexpr int WTM = BM / 2, WTN = BN / 2;  // wave tile 64 x 64
constexpr int FM = WTM / 16, FN = WTN / 16;
constexpr int kTileBytes = 128 * BK * 2;   // one 128-row LDS operand tile (16 KiB)

// Byte offset of 16-byte chunk `chunk` (0..7) of LDS row `row`.
__device__ __forceinline__ int lds_off(int row, int chunk) {
  return row * (BK * 2) + ((chunk ^ ((row ^ (row >> 3)) & 7)) << 4);
}

// K-contiguous 128 x BK tile.  Rows >= r_lim and k >= k_lim read as zero
// (k_lim is a multiple of 8).
struct LoadKc {
  static constexpr int kPer = 128 * (BK / 8) / kThreads;  // 4 chunks per thread
  uint4 v[kPer];
  __device__ __forceinline__ void load(const bf16_t* src, int64_t ld, int r_lim, int k0, int k_lim,
                                       int tid) {
#pragma unroll
    for (int i = 0; i < kPer; ++i) {
      const int q = i * kThreads + tid;
      const int row = q >> 3, k = k0 + ((q & 7) << 3);
      if (row < r_lim && k < k_lim)
        v[i] = *reinterpret_cast<const uint4*>(src + row * ld + k);
      else
        v[i] = make_uint4(0, 0, 0, 0);
    }
  }
  __device__ __forceinline__ void store(char* lds, int tid) const {
#pragma unroll
    for (int i = 0; i < kPer; ++i) {
      const int q = i * kThreads + tid;
      *reinterpret_cast<uint4*>(lds + lds_off(q >> 3, q & 7)) = v[i];
    }
  }
};

// MN-contiguous 128 x BK tile, transposed into the K-contiguous LDS layout.
// Thread tid < 128 owns the 8 x 8 block (rows rb*8.., k kb*8..) with
// rb = tid % 16 and kb = tid / 16, so that 16 neighbouring lanes read 256
// contiguous bytes of one k row.  Rows >= r_lim (a multiple of 8) and
// k >= k_lim read as zero.
struct LoadMNc {
  uint4 v[8];
  __device__ __forceinline__ void load(const bf16_t* src, int64_t ld, int r_lim, int k0, int k_lim,
                                       int tid) {
    if (tid >= 128) return;
    const int rb = tid & 15, kb = tid >> 4;
    const bool rok = rb * 8 < r_lim;
#pragma unroll
    for (int s = 0; s < 8; ++s) {
      const int k = k0 + kb * 8 + s;
      if (rok && k < k_lim)
        v[s] = *reinterpret_cast<const uint4*>(src + static_cast<int64_t>(k) * ld + rb * 8);
      else
        v[s] = make_uint4(0, 0, 0, 0);
    }
  }
  __device__ __forceinline__ void store(char* lds, int tid) const {
    if (tid >= 128) return;
    const int rb = tid & 15, kb = tid >> 4;
    const uint32_t* in = reinterpret_cast<const uint32_t*>(v);  // in[s*4 + w]: k = s, rows 2w, 2w+1
#pragma unroll
    for (int m = 0; m < 8; ++m) {
      uint32_t o[4];
#pragma unroll
      for (int p = 0; p < 4; ++p) {
        const uint32_t a = in[(2 * p) * 4 + (m >> 1)];      // k = 2p
        const uint32_t b = in[(2 * p + 1) * 4 + (m >> 1)];  // k = 2p + 1
        o[p] = (m & 1) ? ((a >> 16) | (b & 0xffff0000u)) : ((a & 0xffffu) | (b << 16));
      }
      *reinterpret_cast<uint4*>(lds + lds_off(rb * 8 + m, kb)) = make_uint4(o[0], o[1], o[2], o[3]);
    }
  }
};

template <bool KC>
struct Loader;
template <>
struct Loader<true> : LoadKc {};
template <>
struct Loader<false> : LoadMNc {};

// Accumulate one BK step of the wave's 64 x 64 sub-tile(s) from LDS.
template <int NB>
__device__ __forceinline__ void mma_step(const char* a_lds, const char* const* b_lds, int wm, int wn,
                                         int lane, f32x4 (&acc)[NB][FM][FN]) {
#pragma unroll
  for (int ks = 0; ks < BK / 32; ++ks) {
    const int chunk = ks * 4 + (lane >> 4);
    uint4 af[FM];
#pragma unroll
    for (int mi = 0; mi < FM; ++mi)
      af[mi] = *reinterpret_cast<const uint4*>(a_lds + lds_off(wm * WTM + mi * 16 + (lane & 15), chunk));
#pragma unroll
    for (int b = 0; b < NB; ++b) {
      uint4 bfr[FN];
#pragma unroll
      for (int ni = 0; ni < FN; ++ni)
        bfr[ni] = *reinterpret_cast<const uint4*>(b_lds[b] + lds_off(wn * WTN + ni * 16 + (lane & 15), chunk));
#pragma unroll
      for (int mi = 0; mi < FM; ++mi)
#pragma unroll
        for (int ni = 0; ni < FN; ++ni) acc[b][mi][ni] = mfma16x16x32(bfr[ni], af[mi], acc[b][mi][ni]);
    }
  }
}

template <int NB>
__device__ __forceinline__ void zero_acc(f32x4 (&acc)[NB][FM][FN]) {
#pragma unroll
  for (int b = 0; b < NB; ++b)
#pragma unroll
    for (int mi = 0; mi < FM; ++mi)
#pragma unroll
      for (int ni = 0; ni < FN; ++ni) acc[b][mi][ni] = f32x4{0.f, 0.f, 0.f, 0.f};
}

// LDS bytes the main loop needs for NB B operands.
template <int NB>
constexpr int mainloop_lds_bytes() {
  return 2 * (1 + NB) * kTileBytes;
}

// acc[b] += A(0:BM, 0:K) * B_b(0:K, 0:BN).
//   a      tile origin: (m0, k = 0) of A, layout per A_KC, leading dim lda
//   m_lim  valid rows of the tile (<= BM); k_lim = K (number of valid k)
//   b[i]   tile origins of the NB B operands, layout per B_KC, leading dim ldb
//   n_lim  valid columns (multiple of 8)
template <bool A_KC, bool B_KC, int NB>
__device__ __forceinline__ void gemm_mainloop(const bf16_t* a, int64_t lda, int m_lim,
                                              const bf16_t* const* b, int64_t ldb, int n_lim, int K,
                                              char* smem, f32x4 (&acc)[NB][FM][FN]) {
  const int tid = threadIdx.x;
  const int lane = tid & 63, wave = tid >> 6;
  const int wm = wave >> 1, wn = wave & 1;
  constexpr int kStage = (1 + NB) * kTileBytes;
  Loader<A_KC> la;
  Loader<B_KC> lb[NB];
  const int nk = cdiv(K, BK);
  if (nk <= 0) return;

  la.load(a, lda, m_lim, 0, K, tid);
#pragma unroll
  for (int i = 0; i < NB; ++i) lb[i].load(b[i], ldb, n_lim, 0, K, tid);
  la.store(smem, tid);
#pragma unroll
  for (int i = 0; i < NB; ++i) lb[i].store(smem + (1 + i) * kTileBytes, tid);
  __syncthreads();

  for (int kt = 0; kt < nk; ++kt) {
    char* cur = smem + (kt & 1) * kStage;
    char* nxt = smem + ((kt + 1) & 1) * kStage;
    const bool more = kt + 1 < nk;
    if (more) {
      la.load(a, lda, m_lim, (kt + 1) * BK, K, tid);
#pragma unroll
      for (int i = 0; i < NB; ++i) lb[i].load(b[i], ldb, n_lim, (kt + 1) * BK, K, tid);
    }
    const char* bl[NB];
#pragma unroll
    for (int i = 0; i < NB; ++i) bl[i] = cur + (1 + i) * kTileBytes;
    mma_step<NB>(cur, bl, wm, wn, lane, acc);
    if (more) {
      la.store(nxt, tid);
#pragma unroll
      for (int i = 0; i < NB; ++i) lb[i].store(nxt + (1 + i) * kTileBytes, tid);
    }
    __syncthreads();
  }
}

// Output coordinates of fragment (mi, ni) for this lane: row, first of 4 columns.
__device__ __forceinline__ int frag_row(int mi, int lane) {
  const int wm = (threadIdx.x >> 6) >> 1;
  return wm * WTM + mi * 16 + (lane & 15);
}
__device__ __forceinline__ int frag_col(int ni, int lane) {
  const int wn = (threadIdx.x >> 6) & 1;
  return wn * WTN + ni * 16 + 4 * (lane >> 4);
}

__device__ __forceinline__ uint2 pack4_bf16(const f32x4& v) {
  return make_uint2(pack_bf16x2(v[0], v[1]), pack_bf16x2(v[2], v[3]));
}

// Blocks are dispatched round-robin over the 8 XCDs (each with its own L2);
// give each XCD a contiguous range of logical tiles so that neighbouring
// tiles (same expert, same operand rows) share an L2.  nblocks % 8 == 0.
__device__ __forceinline__ int xcd_tile(int bid, int nblocks) {
  const int per = nblocks >> 3;
  return (bid & 7) * per + (bid >> 3);
}

// Largest e in [0, E) with tile_start[e] <= mt, or -1 if mt >= tile_start[E].
__device__ __forceinline__ int find_group(const int32_t* tile_start, int E, int mt) {
  if (mt >= tile_start[E]) return -1;
  int lo = 0, hi = E - 1;
  while (lo < hi) {
    const int mid = (lo + hi + 1) >> 1;
    if (tile_start[mid] <= mt) lo = mid;
    else hi = mid - 1;
  }
  return lo;
}

}  // namespace moe
