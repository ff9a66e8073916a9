// Token permutation of the MoE block: a stable counting sort of the routed
// (token, slot) pairs into expert-major, token-ascending rows, then a
// coalesced gather of the token rows.  All integer work is exact and
// deterministic: per-chunk expert membership is a bitmask built with LDS
// atomic ORs (order-independent), and a pair's rank inside its chunk is a
// popcount of the bits of lower tokens.
#include <algorithm>

#include "launch.hpp"
#include "trace.hpp"

namespace moe {

namespace {

constexpr int kChunk = kPermChunk;  // tokens per workgroup (4 waves x 64 lanes)
#ifndef MOE_PERM_SCAN_CHUNKS
#define MOE_PERM_SCAN_CHUNKS 128
#endif
constexpr int kScanChunks = MOE_PERM_SCAN_CHUNKS;  // chunk count above which the counts are scanned first
constexpr int kWords = kChunk / 64;

// bits[e][w] bit l  <=>  token chunk*256 + 64 w + l selected expert e.
__device__ __forceinline__ void build_bits(unsigned long long (*bits)[kWords], const int32_t* topk_idx,
                                           int T, int E, int k, int chunk) {
  for (int i = threadIdx.x; i < E * kWords; i += kChunk) bits[i / kWords][i % kWords] = 0ull;
  __syncthreads();
  const int t = chunk * kChunk + threadIdx.x;
  if (t < T) {
    const unsigned long long bit = 1ull << (threadIdx.x & 63);
    for (int j = 0; j < k; ++j) {
      const int e = topk_idx[static_cast<int64_t>(t) * k + j];
      if (e >= 0) atomicOr(&bits[e][threadIdx.x >> 6], bit);
    }
  }
  __syncthreads();
}

// Exclusive scan of n values held one per thread (n <= blockDim = 256).
__device__ __forceinline__ int block_exclusive_scan(int v, int* tmp) {
  const int tid = threadIdx.x;
  tmp[tid] = v;
  __syncthreads();
  for (int off = 1; off < 256; off <<= 1) {
    const int add = tid >= off ? tmp[tid - off] : 0;
    __syncthreads();
    tmp[tid] += add;
    __syncthreads();
  }
  const int incl = tmp[tid];
  __syncthreads();
  return incl - v;
}

// Row-tile table of the grouped products: expert e's rows split into 128-row
// tiles numbered from tile_start[e]; tile i is (first row, e | rows << 8).
__device__ __forceinline__ void write_tiles(int e, int off, int n, int toff, int2* __restrict__ tile_desc) {
  for (int i = 0; i * 128 < n; ++i) tile_desc[toff + i] = make_int2(off + i * 128, e | (min(128, n - i * 128) << 8));
}

// Per chunk c (one workgroup): expert e's rows in chunks before c and in all
// chunks, the offsets (an exclusive scan over experts), then the chunk's
// pairs go to row offsets[e] + (rows of e in earlier chunks) + (rank inside
// the chunk: a popcount of the lower tokens' bits).  Workgroup 0 also writes
// counts, offsets[E+1], tile_start[E+1] and the tile table.  The per-expert
// sums over chunks come either from the chunk counts themselves (each
// workgroup adds them up in chunk order: O(chunks) per workgroup, so
// quadratic in T overall, cheapest while chunks are few) or, with `scanned`,
// from k_chunk_scan's exclusive prefix per chunk and its totals row.
__global__ __launch_bounds__(kChunk) void k_perm_scatter(const int32_t* __restrict__ topk_idx, int T, int E,
                                                         int k, const int32_t* __restrict__ chunk_counts,
                                                         int nchunks, bool scanned, int32_t* __restrict__ counts,
                                                         int32_t* __restrict__ offsets,
                                                         int32_t* __restrict__ tile_start,
                                                         int2* __restrict__ tile_desc,
                                                         int32_t* __restrict__ row_token,
                                                         int32_t* __restrict__ row_of) {
  __shared__ unsigned long long bits[MOE_MAX_EXPERTS][kWords];
  __shared__ int tmp[256];
  __shared__ int base[MOE_MAX_EXPERTS];  // offsets[e] + rows of e in earlier chunks
  const int chunk = blockIdx.x;
  const int e = threadIdx.x;
  int before = 0, total = 0;
  if (e < E && scanned) {
    before = chunk_counts[static_cast<int64_t>(chunk) * E + e];
    total = chunk_counts[static_cast<int64_t>(nchunks) * E + e];
  } else if (e < E) {
    constexpr int kBatch = 16;  // independent loads in flight per thread
    for (int c0 = 0; c0 < nchunks; c0 += kBatch) {
      int n[kBatch];
#pragma unroll
      for (int i = 0; i < kBatch; ++i)
        n[i] = c0 + i < nchunks ? chunk_counts[static_cast<int64_t>(c0 + i) * E + e] : 0;
#pragma unroll
      for (int i = 0; i < kBatch; ++i) {
        before += c0 + i < chunk ? n[i] : 0;
        total += n[i];
      }
    }
  }
  const int off = block_exclusive_scan(e < E ? total : 0, tmp);
  if (e < E) base[e] = off + before;
  if (chunk == 0) {
    const int tiles = cdiv(total, 128);
    const int toff = block_exclusive_scan(e < E ? tiles : 0, tmp);
    if (e < E) {
      counts[e] = total;
      offsets[e] = off;
      tile_start[e] = toff;
      write_tiles(e, off, total, toff, tile_desc);
    }
    if (e == E - 1) {
      offsets[E] = off + total;
      tile_start[E] = toff + tiles;
    }
  }
  build_bits(bits, topk_idx, T, E, k, chunk);  // its barriers also publish base[]
  const int t = chunk * kChunk + threadIdx.x;
  if (t >= T) return;
  const int w = threadIdx.x >> 6;
  const unsigned long long below = (1ull << (threadIdx.x & 63)) - 1ull;
  for (int j = 0; j < k; ++j) {
    const int64_t p = static_cast<int64_t>(t) * k + j;
    const int ej = topk_idx[p];
    if (ej < 0) {
      row_of[p] = -1;
      continue;
    }
    int rank = __popcll(bits[ej][w] & below);
    for (int ww = 0; ww < w; ++ww) rank += __popcll(bits[ej][ww]);
    const int r = base[ej] + rank;
    row_token[r] = t;
    row_of[p] = r;
  }
}

// Per expert e (one workgroup): the exclusive prefix over chunks of its
// chunk counts, in place (cnt[c][e] becomes the rows of e in chunks before
// c), and its total in row nchunks.  Thread i takes a contiguous run of
// chunks; integer sums, so the result is exact in any order.
__global__ __launch_bounds__(256) void k_chunk_scan(int32_t* __restrict__ cnt, int nchunks, int E) {
  __shared__ int tmp[256];
  const int e = blockIdx.x;
  const int per = cdiv(nchunks, 256);
  const int c0 = min(nchunks, static_cast<int>(threadIdx.x) * per), c1 = min(nchunks, c0 + per);
  int sum = 0;
  for (int c = c0; c < c1; ++c) sum += cnt[static_cast<int64_t>(c) * E + e];
  int run = block_exclusive_scan(sum, tmp);
  for (int c = c0; c < c1; ++c) {
    const int64_t i = static_cast<int64_t>(c) * E + e;
    const int v = cnt[i];
    cnt[i] = run;
    run += v;
  }
  if (threadIdx.x == 255) cnt[static_cast<int64_t>(nchunks) * E + e] = run;
}

// xp[row_of[t,j]] = x[t] for every routed slot (the same rows as
// xp[r] = x[row_token[r]]), token-major: one wave per token reads its row of
// x once, 16 bytes per lane, and writes it to the token's k permuted rows.
// The stores are non-temporal: Xp is next read by the gate/up product, long
// after it would have left the caches.
typedef unsigned int u32x4_t __attribute__((ext_vector_type(4)));

template <int KT>
__global__ __launch_bounds__(256) void k_permute_rows(const bf16_t* __restrict__ x,
                                                      const int32_t* __restrict__ row_of, int T, int H, int k,
                                                      bf16_t* __restrict__ xp) {
  const int lane = threadIdx.x & 63;
  const int64_t nwaves = static_cast<int64_t>(gridDim.x) * 4;
  for (int64_t t = static_cast<int64_t>(blockIdx.x) * 4 + (threadIdx.x >> 6); t < T; t += nwaves) {
    int rows[KT];
#pragma unroll
    for (int j = 0; j < KT; ++j) rows[j] = j < k ? row_of[t * k + j] : -1;
    if (rows[0] < 0) continue;  // a masked token has no rows
    const bf16_t* src = x + t * H;
    for (int c0 = lane * 8; c0 < H; c0 += 4 * kWave * 8) {
      u32x4_t v[4];
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int c = c0 + i * kWave * 8;
        v[i] = c < H ? *reinterpret_cast<const u32x4_t*>(src + c) : u32x4_t{0u, 0u, 0u, 0u};
      }
#pragma unroll
      for (int j = 0; j < KT; ++j) {
        if (rows[j] < 0) continue;
        bf16_t* dst = xp + static_cast<int64_t>(rows[j]) * H;
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const int c = c0 + i * kWave * 8;
          if (c < H) __builtin_nontemporal_store(v[i], reinterpret_cast<u32x4_t*>(dst + c));
        }
      }
    }
  }
}

// Experts path: offsets from device counts, clamped to the row capacity.
__global__ __launch_bounds__(256) void k_offsets_from_counts(const int32_t* __restrict__ counts, int E,
                                                             int rows, int32_t* __restrict__ offsets,
                                                             int32_t* __restrict__ tile_start,
                                                             int2* __restrict__ tile_desc) {
  __shared__ int tmp[256];
  const int e = threadIdx.x;
  const int c = e < E ? max(0, counts[e]) : 0;
  const int off = block_exclusive_scan(c, tmp);
  const int lo = min(off, rows), hi = min(off + c, rows);
  const int n = hi - lo;
  const int tiles = cdiv(n, 128);
  const int toff = block_exclusive_scan(tiles, tmp);
  if (e < E) {
    offsets[e] = lo;
    tile_start[e] = toff;
    write_tiles(e, lo, n, toff, tile_desc);
  }
  if (e == E - 1) {
    offsets[E] = hi;
    tile_start[E] = toff + tiles;
  }
}

}  // namespace

// Chunk counts [chunks][E] and a row of per-expert totals.
int64_t permute_ws_ints(int T, int E) { return static_cast<int64_t>(cdiv(T, kChunk) + 1) * E; }

hipError_t launch_permute(const int32_t* topk_idx, const bf16_t* x, int T, int H, int E, int k,
                          int32_t* counts, int32_t* offsets, int32_t* tile_start, int2* tile_desc,
                          int32_t* row_token, int32_t* row_of, bf16_t* xp, int32_t* ws, hipStream_t s) {
  const int nchunks = cdiv(T, kChunk);
  int32_t* chunk_counts = ws;  // written by the router's top-k
  // Past kScanChunks chunks, one scan per expert replaces each scatter
  // workgroup's own pass over every chunk's counts (linear instead of
  // quadratic in T).
  const bool scanned = nchunks > kScanChunks;
  {
    TraceScope trace_scope(K_PERM_SCATTER, s);
    if (scanned) hipLaunchKernelGGL(k_chunk_scan, dim3(E), dim3(256), 0, s, chunk_counts, nchunks, E);
    hipLaunchKernelGGL(k_perm_scatter, dim3(nchunks), dim3(kChunk), 0, s, topk_idx, T, E, k, chunk_counts, nchunks,
                       scanned, counts, offsets, tile_start, tile_desc, row_token, row_of);
  }
  if (xp == nullptr) return hipGetLastError();
  // a few waves per CU suffice: each token's row is read once and written k times
  const int grid = static_cast<int>(std::min<int64_t>(cdiv64(T, 4), 1024));
  {
    TraceScope trace_scope(K_PERMUTE_ROWS, s);
    if (k <= 1) hipLaunchKernelGGL(k_permute_rows<1>, dim3(grid), dim3(256), 0, s, x, row_of, T, H, k, xp);
    else if (k <= 2) hipLaunchKernelGGL(k_permute_rows<2>, dim3(grid), dim3(256), 0, s, x, row_of, T, H, k, xp);
    else if (k <= 4) hipLaunchKernelGGL(k_permute_rows<4>, dim3(grid), dim3(256), 0, s, x, row_of, T, H, k, xp);
    else if (k <= 8) hipLaunchKernelGGL(k_permute_rows<8>, dim3(grid), dim3(256), 0, s, x, row_of, T, H, k, xp);
    else if (k <= 16) hipLaunchKernelGGL(k_permute_rows<16>, dim3(grid), dim3(256), 0, s, x, row_of, T, H, k, xp);
    else hipLaunchKernelGGL(k_permute_rows<32>, dim3(grid), dim3(256), 0, s, x, row_of, T, H, k, xp);
  }
  return hipGetLastError();
}

hipError_t launch_offsets_from_counts(const int32_t* counts, int E, int rows, int32_t* offsets,
                                      int32_t* tile_start, int2* tile_desc, hipStream_t s) {
  {
    TraceScope trace_scope(K_OFFSETS, s);
    hipLaunchKernelGGL(k_offsets_from_counts, dim3(1), dim3(256), 0, s, counts, E, rows, offsets, tile_start,
                       tile_desc);
  }
  return hipGetLastError();
}

}  // namespace moe
