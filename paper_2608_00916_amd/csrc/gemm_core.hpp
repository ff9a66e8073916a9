// bf16 MFMA GEMM core shared by every matrix product of the MoE block.
//
// One workgroup (WM x WN waves of 64 lanes) computes a BM x BN fp32 tile C = A_tile * B_tile over a K loop in steps of BK = 64:
//   C[m][n] = sum_k A(m, k) B(k, n)
// Operands come from global memory in one of two layouts:
//   K-contiguous   element (r, k) at src[r * ld + k]   (a row-major A, or B^T)
//   MN-contiguous  element (r, k) at src[k * ld + r]   (a row-major B, or A^T)
// Both are copied to LDS untouched (16-byte buffer loads staged through
// registers): a K-contiguous tile as [rows][64] (128-byte rows), an
// MN-contiguous tile as [64][rows].  16-byte units are XOR-swizzled by row so
// that both the tile writes and the MFMA operand reads are free of bank
// conflicts.  The MFMA wants 8 consecutive k per lane: K-contiguous tiles give
// them with one ds_read_b128; MN-contiguous tiles with two
// ds_read_b64_tr_b16, the gfx950 LDS read that transposes 4 x 4 blocks of
// 16-bit elements across groups of four lanes.
//
// Two LDS stages and two register sets: the global loads of step k+2 are in
// flight while the MFMAs of step k run, with one LDS-only barrier per step.
//
// v_mfma_f32_16x16x32_bf16 is fed with the B tile as its first operand and
// the A tile as its second, so that each lane ends up holding four
// consecutive columns of one output row:
//   lane l, fragment (mi, ni), register i -> C[row(mi) + l%16][col(ni) + 4 (l/16) + i]
//
// With NB = 2 the B tile holds two operands side by side (columns [0, BN/2)
// from the first, [BN/2, BN) from the second) and each wave takes matching
// columns of both, so an epilogue can combine them element by element.
#pragma once

#include <type_traits>

#include "common.hpp"

namespace moe {

constexpr int BK = 64;

typedef short v4i16 __attribute__((ext_vector_type(4)));
typedef uint32_t v4u32 __attribute__((ext_vector_type(4)));
#define MOE_LDS __attribute__((address_space(3)))

// BM x BN tile computed by WM x WN waves (each (BM/WM) x (BN/WN)).
template <int BM_, int BN_, int NB_, int WM_ = 2, int WN_ = 2>
struct Tile {
  static constexpr int BM = BM_, BN = BN_, NB = NB_, WM = WM_, WN = WN_;
  static constexpr int kThreads = 64 * WM * WN;
  static constexpr int FM = BM / WM / 16;  // 16-row A fragments per wave
  static constexpr int FN = BN / WN / 16;  // 16-row B fragments per wave
  static constexpr int BNS = BN / NB;      // rows of one B operand in the tile
  static constexpr int kABytes = BM * BK * 2;
  static constexpr int kBBytes = BN * BK * 2;
  static constexpr int kStage = kABytes + kBBytes;
  static constexpr int kLds = 2 * kStage;
};

// ---------------------------------------------------------------- LDS layouts
// K-contiguous tile [rows][64]: byte offset of 16-byte chunk c (0..7) of row r.
__device__ __forceinline__ int kc_off(int r, int c) { return r * 128 + ((c ^ ((r ^ (r >> 3)) & 7)) << 4); }

// MN-contiguous tile [64][ROWS]: byte offset of 16-byte unit u of k-row k.
// The XOR moves 32-byte blocks so that the 16 rows one transposing read
// touches (k = 8 g + j, g, j < 4) land in distinct banks.  It stays inside
// the k-row: narrow tiles (16 columns: two units per k-row) keep only the
// bits of the XOR below their unit count (none for 16 columns, whose 4
// consecutive k-rows of a read already span distinct banks).
template <int ROWS>
__device__ __forceinline__ int mn_off(int k, int u) {
  static_assert(ROWS >= 16 && (ROWS & (ROWS - 1)) == 0, "MN tiles are a power-of-two number of columns >= 16");
  constexpr int kUnitMask = ROWS / 8 - 1;
  const int h = (k & 3) | (((k >> 3) & 1) << 2);
  return k * (ROWS * 2) + ((u ^ ((h << 1) & kUnitMask)) << 4);
}

// ---------------------------------------------------------------- global -> registers -> LDS
// Global loads go through buffer resources: a lane whose byte offset is at or
// beyond the resource's size reads zeros, so ragged rows and K tails need no
// branches.  Each K step moves the resource base by one step; offsets are
// fixed per lane.
constexpr uint32_t kOob = 0x80000000u;  // an offset beyond every resource size

__device__ __forceinline__ __amdgpu_buffer_rsrc_t make_rsrc(const void* base, int64_t bytes) {
  const int n = static_cast<int>(bytes < 0 ? 0 : (bytes > 0x7fffffff ? 0x7fffffff : bytes));
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), 0, n, 0x00020000);
}

__device__ __forceinline__ uint4 buf_load16(__amdgpu_buffer_rsrc_t r, uint32_t off) {
  return __builtin_bit_cast(uint4, __builtin_amdgcn_raw_buffer_load_b128(r, static_cast<int>(off), 0, 0));
}

// K-contiguous operand: ROWS tile rows starting at LDS row `row0`.  Rows
// >= r_lim and k >= K read as zero (K a multiple of 8).
template <int ROWS, int kThreads>
struct LoadKc {
  static constexpr int kPer = ROWS * (BK / 8) / kThreads;
  static_assert(kPer * kThreads == ROWS * (BK / 8), "tile rows must split evenly over the threads");
  const char* base;
  int32_t valid;  // bytes of the valid rows within the tile's ROWS (< 2^31)
  int32_t ld2;    // row pitch in bytes
  uint32_t off[kPer];
  __device__ __forceinline__ void init(const bf16_t* src, int64_t ld, int r_lim, int tid) {
    base = reinterpret_cast<const char*>(src);
    ld2 = static_cast<int32_t>(ld * 2);
    valid = r_lim > 0 ? (r_lim < ROWS ? r_lim : ROWS) * ld2 : 0;
#pragma unroll
    for (int i = 0; i < kPer; ++i) {
      const int q = i * kThreads + tid;
      off[i] = static_cast<uint32_t>((q >> 3) * ld2 + ((q & 7) << 4));
    }
  }
  // Rows through an index: tile row r is row rows[r] of src for r < r_lim;
  // `bytes` (< 2^31) bounds the whole source.
  __device__ __forceinline__ void init_rows(const bf16_t* src, int64_t ld, const int32_t* rows, int r_lim,
                                            int64_t bytes, int tid) {
    base = reinterpret_cast<const char*>(src);
    ld2 = static_cast<int32_t>(ld * 2);
    valid = static_cast<int32_t>(bytes);
#pragma unroll
    for (int i = 0; i < kPer; ++i) {
      const int q = i * kThreads + tid;
      const int r = q >> 3;
      off[i] = r < r_lim ? static_cast<uint32_t>(rows[r] * ld2 + ((q & 7) << 4)) : kOob;
    }
  }
  __device__ __forceinline__ void disable() { valid = 0; }
  __device__ __forceinline__ void load(uint4 (&v)[kPer], int kt, int K, int tid) const {
    const int64_t step = static_cast<int64_t>(kt) * (BK * 2);
    const __amdgpu_buffer_rsrc_t r = make_rsrc(base + step, valid - step);
#pragma unroll
    for (int i = 0; i < kPer; ++i) {
      const int q = i * kThreads + tid;
      const bool kin = kt * BK + ((q & 7) << 3) < K;
      v[i] = buf_load16(r, kin ? off[i] : kOob);
    }
  }
  __device__ __forceinline__ void store(const uint4 (&v)[kPer], char* lds, int row0, int tid) const {
#pragma unroll
    for (int i = 0; i < kPer; ++i) {
      const int q = i * kThreads + tid;
      *reinterpret_cast<uint4*>(lds + kc_off(row0 + (q >> 3), q & 7)) = v[i];
    }
  }
};

// MN-contiguous operand: ROWS columns of the tile's [64][TROWS] LDS layout
// starting at column `col0`.  Columns >= r_lim (a multiple of 8) and k >= K
// read as zero.
template <int ROWS, int TROWS, int kThreads>
struct LoadMn {
  static constexpr int kUnits = ROWS / 8;  // 16-byte units per k-row
  static constexpr int kPer = BK * kUnits / kThreads;
  static_assert(kPer * kThreads == BK * kUnits, "tile columns must split evenly over the threads");
  const char* base;
  int64_t valid;  // bytes of the K valid k-rows
  int32_t ld2;    // row pitch in bytes
  uint32_t off[kPer];
  __device__ __forceinline__ void init(const bf16_t* src, int64_t ld, int r_lim, int K, int tid) {
    base = reinterpret_cast<const char*>(src);
    ld2 = static_cast<int32_t>(ld * 2);
    valid = K > 0 ? static_cast<int64_t>(K) * ld2 : 0;
#pragma unroll
    for (int i = 0; i < kPer; ++i) {
      const int q = i * kThreads + tid;
      const int k = q / kUnits, u = q % kUnits;
      off[i] = u * 8 < r_lim ? static_cast<uint32_t>(k * ld2 + u * 16) : kOob;
    }
  }
  __device__ __forceinline__ void disable() { valid = 0; }
  __device__ __forceinline__ void load(uint4 (&v)[kPer], int kt, int, int) const {
    const int64_t step = static_cast<int64_t>(kt) * BK * ld2;  // 64-bit: K rows can span more than 2^31 bytes
    const __amdgpu_buffer_rsrc_t r = make_rsrc(base + step, valid - step);
#pragma unroll
    for (int i = 0; i < kPer; ++i) v[i] = buf_load16(r, off[i]);
  }
  __device__ __forceinline__ void store(const uint4 (&v)[kPer], char* lds, int col0, int tid) const {
#pragma unroll
    for (int i = 0; i < kPer; ++i) {
      const int q = i * kThreads + tid;
      const int k = q / kUnits, u = q % kUnits;
      *reinterpret_cast<uint4*>(lds + mn_off<TROWS>(k, (col0 >> 3) + u)) = v[i];
    }
  }
};

template <bool KC, int ROWS, int TROWS, int NT>
struct Loader : LoadKc<ROWS, NT> {
  __device__ __forceinline__ void setup(const bf16_t* src, int64_t ld, int r_lim, int, int tid) {
    this->init(src, ld, r_lim, tid);
  }
};
template <int ROWS, int TROWS, int NT>
struct Loader<false, ROWS, TROWS, NT> : LoadMn<ROWS, TROWS, NT> {
  __device__ __forceinline__ void setup(const bf16_t* src, int64_t ld, int r_lim, int K, int tid) {
    this->init(src, ld, r_lim, K, tid);
  }
};

// Barrier for LDS traffic only: waits for this wave's LDS operations, then
// for every wave, without draining global loads still in flight.
__device__ __forceinline__ void lds_barrier() { asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory"); }

// ---------------------------------------------------------------- LDS -> MFMA operands
// 16 x 32 operand fragment (rows rbase..rbase+15, k = ks*32 .. ks*32+31):
// lane l gets row rbase + l%16, k = ks*32 + 8 (l/16) + 0..7.
template <bool KC, int TROWS>
__device__ __forceinline__ uint4 frag(const char* lds, int rbase, int ks, int lane) {
  if constexpr (KC) {
    return *reinterpret_cast<const uint4*>(lds + kc_off(rbase + (lane & 15), ks * 4 + (lane >> 4)));
  } else {
    const int s = lane & 15, g = lane >> 4;
    const int k = ks * 32 + 8 * g + (s >> 2);
    const int n = rbase + 4 * (s & 3);
    const int o = (n & 7) * 2;
    const MOE_LDS char* base = (const MOE_LDS char*)(lds);
    const v4i16 lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
        (MOE_LDS v4i16*)(base + mn_off<TROWS>(k, n >> 3) + o));
    const v4i16 hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
        (MOE_LDS v4i16*)(base + mn_off<TROWS>(k + 4, n >> 3) + o));
    const uint2 a = __builtin_bit_cast(uint2, lo), b = __builtin_bit_cast(uint2, hi);
    return make_uint4(a.x, a.y, b.x, b.y);
  }
}

// First B-tile row of wave column wn's fragment ni.  With NB = 2 the first
// FN/2 fragments come from the first operand's columns, the rest from the
// matching columns of the second.
template <class C>
__device__ __forceinline__ int brow(int wn, int ni) {
  if constexpr (C::NB == 1) {
    return wn * (C::BN / C::WN) + ni * 16;
  } else {
    constexpr int half = C::FN / 2;
    constexpr int span = C::BN / 2 / C::WN;
    return (ni < half) ? wn * span + ni * 16 : C::BN / 2 + wn * span + (ni - half) * 16;
  }
}

// Operand fragments of one 32-deep slice ks of the LDS stage.
template <class C, bool A_KC, bool B_KC>
__device__ __forceinline__ void read_frags(const char* a_lds, const char* b_lds, int wm, int wn, int ks,
                                           int lane, uint4 (&af)[C::FM], uint4 (&bf)[C::FN]) {
#pragma unroll
  for (int mi = 0; mi < C::FM; ++mi) af[mi] = frag<A_KC, C::BM>(a_lds, wm * (C::BM / C::WM) + mi * 16, ks, lane);
#pragma unroll
  for (int ni = 0; ni < C::FN; ++ni) bf[ni] = frag<B_KC, C::BN>(b_lds, brow<C>(wn, ni), ks, lane);
}

template <class C>
__device__ __forceinline__ void mfmas(const uint4 (&af)[C::FM], const uint4 (&bf)[C::FN],
                                      f32x4 (&acc)[C::FM][C::FN]) {
#pragma unroll
  for (int mi = 0; mi < C::FM; ++mi)
#pragma unroll
    for (int ni = 0; ni < C::FN; ++ni) acc[mi][ni] = mfma16x16x32(bf[ni], af[mi], acc[mi][ni]);
}

template <class C>
__device__ __forceinline__ void zero_acc(f32x4 (&acc)[C::FM][C::FN]) {
#pragma unroll
  for (int mi = 0; mi < C::FM; ++mi)
#pragma unroll
    for (int ni = 0; ni < C::FN; ++ni) acc[mi][ni] = f32x4{0.f, 0.f, 0.f, 0.f};
}

// Scheduling: each of the N MFMAs of a region is followed by an even share
// of A instructions of class MA and B instructions of class MB.
__host__ __device__ constexpr int share(int total, int slots, int i) {
  return total * (i + 1) / slots - total * i / slots;
}
template <int N, int A, int MA, int B, int MB, int I = 0>
__device__ __forceinline__ void interleave() {
  if constexpr (I < N) {
    __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
    if constexpr (share(A, N, I) > 0) __builtin_amdgcn_sched_group_barrier(MA, share(A, N, I), 0);
    if constexpr (share(B, N, I) > 0) __builtin_amdgcn_sched_group_barrier(MB, share(B, N, I), 0);
    interleave<N, A, MA, B, MB, I + 1>();
  }
}

// acc += A(0:BM, 0:K) * [B_0 | B_1](0:K, 0:BN).
//   a      tile origin (m0, k = 0) of A in layout A_KC, leading dimension lda
//   m_lim  valid rows of the tile (<= BM); K = number of valid k
//   b[i]   tile origins of the NB B operands in layout B_KC, leading dim ldb
//   n_lim  valid columns of each B operand (multiple of 8)
//   a_rows if non-null (K-contiguous A only), tile row r is row a_rows[r] of
//          the matrix at `a`, whose a_bytes (< 2^31) bound every access
// Software pipeline: global loads run two K steps ahead of the MFMAs in two
// register sets; LDS holds two stages; one LDS barrier per step.
template <class C, bool A_KC, bool B_KC>
__device__ __forceinline__ void gemm_mainloop(const bf16_t* a, int64_t lda, int m_lim,
                                              const bf16_t* const* b, int64_t ldb, int n_lim, int K,
                                              char* smem, f32x4 (&acc)[C::FM][C::FN],
                                              const int32_t* a_rows = nullptr, int64_t a_bytes = 0) {
  using LA = Loader<A_KC, C::BM, C::BM, C::kThreads>;
  using LB = Loader<B_KC, C::BNS, C::BN, C::kThreads>;
  const int tid = threadIdx.x;
  const int lane = tid & 63, wave = tid >> 6;
  const int wm = wave / C::WN, wn = wave % C::WN;
  const int nk = cdiv(K, BK);
  if (nk <= 0) return;
  LA la;
  LB lb[C::NB];
  if constexpr (A_KC) {
    if (a_rows != nullptr) la.init_rows(a, lda, a_rows, m_lim, a_bytes, tid);
    else la.setup(a, lda, m_lim, K, tid);
  } else {
    la.setup(a, lda, m_lim, K, tid);
  }
#pragma unroll
  for (int i = 0; i < C::NB; ++i) lb[i].setup(b[i], ldb, n_lim, K, tid);
  uint4 ra[2][LA::kPer];
  uint4 rb[2][C::NB][LB::kPer];

  auto load = [&](auto set, int kt) {
    constexpr int S = decltype(set)::value;
    la.load(ra[S], kt, K, tid);
#pragma unroll
    for (int i = 0; i < C::NB; ++i) lb[i].load(rb[S][i], kt, K, tid);
  };
  auto store = [&](auto set, char* stage) {
    constexpr int S = decltype(set)::value;
    la.store(ra[S], stage, 0, tid);
#pragma unroll
    for (int i = 0; i < C::NB; ++i) lb[i].store(rb[S][i], stage + C::kABytes, i * C::BNS, tid);
  };
  using S0 = std::integral_constant<int, 0>;
  using S1 = std::integral_constant<int, 1>;
  // Instruction counts of one K step, for the interleaving below.
  constexpr int kReads = C::FM * (A_KC ? 1 : 2) + C::FN * (B_KC ? 1 : 2);  // per 32-deep slice
  constexpr int kMfma = C::FM * C::FN;                                      // per slice
  constexpr int kWrites = LA::kPer + C::NB * LB::kPer;
  constexpr int kLoads = kWrites;
  // Wide tiles alternate one MFMA with one read, write or load; small tiles
  // (more of those than MFMAs) spread them evenly over the MFMAs.
  constexpr bool kOneEach = kReads <= kMfma && kWrites + kLoads <= kMfma;
  // One K step on LDS stage `set`: MFMAs of both 32-deep slices, the refill of
  // the other stage from the other register set (step kt + 1, loaded two steps
  // ago) and the global loads of step kt + 3 into that register set.  Loads
  // past K read zeros without touching memory, so the body has no branches
  // and the scheduler can interleave: slice-0 fragment reads, then slice-0
  // MFMAs alternating with slice-1 fragment reads, then slice-1 MFMAs
  // alternating with the LDS writes and global loads.
  auto step = [&](auto set, int kt) {
    constexpr int S = decltype(set)::value;
    using Other = std::integral_constant<int, 1 - S>;
    const char* cur = smem + S * C::kStage;
    char* nxt = smem + (1 - S) * C::kStage;
    uint4 af0[C::FM], bf0[C::FN], af1[C::FM], bf1[C::FN];
    read_frags<C, A_KC, B_KC>(cur, cur + C::kABytes, wm, wn, 0, lane, af0, bf0);
    read_frags<C, A_KC, B_KC>(cur, cur + C::kABytes, wm, wn, 1, lane, af1, bf1);
    mfmas<C>(af0, bf0, acc);
    mfmas<C>(af1, bf1, acc);
    store(Other{}, nxt);
    load(Other{}, kt + 3);
    __builtin_amdgcn_sched_group_barrier(0x100, kReads, 0);  // slice-0 reads
    if constexpr (kOneEach) {
#pragma unroll
      for (int i = 0; i < kReads; ++i) {
        __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);  // MFMA
        __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);  // slice-1 read
      }
      __builtin_amdgcn_sched_group_barrier(0x008, kMfma - kReads, 0);
#pragma unroll
      for (int i = 0; i < kWrites; ++i) {
        __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);  // MFMA
        __builtin_amdgcn_sched_group_barrier(0x200, 1, 0);  // LDS write
      }
#pragma unroll
      for (int i = 0; i < kLoads; ++i) {
        __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);  // MFMA
        __builtin_amdgcn_sched_group_barrier(0x020, 1, 0);  // global load
      }
      __builtin_amdgcn_sched_group_barrier(0x008, kMfma - kWrites - kLoads, 0);
    } else {
      interleave<kMfma, kReads, 0x100, 0, 0x200>();                 // slice-0 MFMAs + slice-1 reads
      interleave<kMfma, kWrites, 0x200, kLoads, 0x020>();           // slice-1 MFMAs + refill
    }
    lds_barrier();
  };

  load(S0{}, 0);
  load(S1{}, 1);
  store(S0{}, smem);
  lds_barrier();
  load(S0{}, 2);
  for (int kt = 0; kt < nk; kt += 2) {
    step(S0{}, kt);
    if (kt + 1 < nk) step(S1{}, kt + 1);
  }
}

// ---------------------------------------------------------------- persistent stream
// A workgroup's sequence of tile jobs.  A job is one tile's K range of one
// product; `chain` jobs accumulate into the next job's tile (a K range split
// over two operand pairs) instead of ending it.
// Output coordinates of fragment (mi, ni) for this lane: row, first of 4 columns
// (columns index the B tile: [0, BN/2) first operand, [BN/2, BN) second when NB = 2).
template <class C>
__device__ __forceinline__ int frag_row(int mi, int lane) {
  const int wm = (threadIdx.x >> 6) / C::WN;
  return wm * (C::BM / C::WM) + mi * 16 + (lane & 15);
}
template <class C>
__device__ __forceinline__ int frag_col(int ni, int lane) {
  const int wn = (threadIdx.x >> 6) % C::WN;
  return brow<C>(wn, ni) + 4 * (lane >> 4);
}

__device__ __forceinline__ uint2 pack4_bf16(const f32x4& v) {
  return make_uint2(pack_bf16x2(v[0], v[1]), pack_bf16x2(v[2], v[3]));
}

template <class C>
struct Job {
  const bf16_t* a;
  int64_t lda;
  int m_lim;
  const bf16_t* b[C::NB];
  int64_t ldb;
  int n_lim;
  int K;       // valid k; 0 = an empty tile (its epilogue sees zeros)
  bool chain;  // the next job continues this tile
  int e, m0, n0;
};

// ---------------------------------------------------------------- staged output
// A job provider that declares `static constexpr bool kStaged = true` hands
// its finished tiles over as bf16 through LDS instead of storing them from
// the accumulators: after a tile's last K step the workgroup writes the tile
// into an LDS staging area, and the first step of each following pair of K
// steps drains part of it to global memory (P::drain, with any elementwise
// epilogue), so that the stores overlap the next tile's MFMAs.  Stored
// straight from the accumulators they stall every wave at the tile boundary
// until they complete (one counter tracks both loads and stores), which costs
// as much as the tile's MFMAs when the reduction is short (weight gradients
// over one expert's rows).  The provider supplies
//   Drain                          per-thread state of the tile being drained
//   kDrainCalls                    drain calls per tile
//   drain_setup(job, Drain&)       once the tile is staged
//   drain(Drain&, staging, p)      call p (p >= kDrainCalls: no memory effect)
//   drain_reset(Drain&)            a state whose calls touch no memory
// A tile whose successor is shorter than kDrainCalls step pairs is drained
// in full before the successor is staged.
// Staging layout: tile row r (BN bf16, all NB blocks side by side), 16-byte
// chunk q at Staged<C>::off(r, q).
template <class C>
struct Staged {
  static constexpr int kRowBytes = C::BN * 2;                         // one tile row, all NB blocks
  static constexpr int kBytes = C::BM * kRowBytes;                    // LDS staging area
  static constexpr int kXor = (C::BN / 8 < 16 ? C::BN / 8 : 16) - 1;  // rows of 16 hit distinct banks
  static __device__ __forceinline__ int off(int r, int q) { return r * kRowBytes + ((q ^ (r & kXor)) << 4); }
};

template <class P, class = void>
struct staged_provider : std::false_type {};
template <class P>
struct staged_provider<P, std::void_t<decltype(P::kStaged)>> : std::integral_constant<bool, P::kStaged> {};

// A staged provider that declares `static constexpr bool kDrainLate = true`
// gets its drain call at the end of the step (after the step's operand loads)
// instead of at its start.  The vector-memory counter completes in order, so
// a drain that loads from memory (the SwiGLU backward's G and U) delays every
// operand load issued after it; issued after the step's loads, it delays one
// step's fewer.  Plain stores lose by the move (the loads of the next step
// then queue behind them with less time to spare).
template <class P, class = void>
struct drain_late : std::false_type {};
template <class P>
struct drain_late<P, std::void_t<decltype(P::kDrainLate)>> : std::integral_constant<bool, P::kDrainLate> {};

// A provider that declares `static constexpr bool kOpaqueSetup = true` has
// its loaders' per-lane offsets recomputed from the thread index at each job.
// Streams short of registers (the adapter variants, whose jobs carry a second
// operand segment) otherwise keep them live across the whole stream, spill
// them, and each reload's wait drains the operand loads in flight.
template <class P, class = void>
struct opaque_setup : std::false_type {};
template <class P>
struct opaque_setup<P, std::void_t<decltype(P::kOpaqueSetup)>> : std::integral_constant<bool, P::kOpaqueSetup> {};

// LDS bytes gemm_stream needs for provider P.
template <class P>
constexpr int stream_lds() {
  return P::C::kLds + (staged_provider<P>::value ? Staged<typename P::C>::kBytes : 0);
}

// Output stores of the grouped products are non-temporal (streamed past the
// caches, so that they do not evict the operands the next tiles reuse),
// except where a memory-bound kernel reads the output straight back
// (kKeep: it may then still find it in the last-level cache).
template <bool kKeep = false>
__device__ __forceinline__ void buf_store16(__amdgpu_buffer_rsrc_t r, uint32_t off, const uint4& v) {
  constexpr int kNonTemporal = 2;  // the nt cache-policy bit of a buffer store
  __builtin_amdgcn_raw_buffer_store_b128(__builtin_bit_cast(v4u32, v), r, static_cast<int>(off), 0,
                                         kKeep ? 0 : kNonTemporal);
}

// Buffer resource over `rows` rows of `width_bytes` at pitch ld_bytes:
// accesses to rows >= rows fall outside it (stores are dropped, loads read
// zeros).
__device__ __forceinline__ __amdgpu_buffer_rsrc_t rows_rsrc(const void* base, int rows, int64_t ld_bytes,
                                                            int width_bytes) {
  return make_rsrc(base, rows > 0 ? static_cast<int64_t>(rows - 1) * ld_bytes + width_bytes : 0);
}

// Drain that copies the staged tile to NB destinations (element (0, 0) of
// each BM x BNS block, pitch ld elements, `rows` valid rows; whole rows of BNS
// columns are written).  A slice is one 16-byte chunk per thread: wave w
// stores block w % NB, kRowsPerWave rows of it per slice.  kKeep: cached
// stores (see buf_store16).
template <class C, bool kKeep = false>
struct StagedCopy {
  using SO = Staged<C>;
  static constexpr int kCpr = C::BNS * 2 / 16;  // chunks per block row
  static constexpr int kRowsPerWave = 64 / kCpr;
  static constexpr int kSliceRows = C::kThreads / 64 / C::NB * kRowsPerWave;
  static constexpr int kSlices = C::BM / kSliceRows;
  static constexpr int kCalls = kSlices / 2;  // two slices per drain call
  static_assert(64 % kCpr == 0 && (C::kThreads / 64) % C::NB == 0, "a wave stores whole block rows of one block");
  static_assert(kSlices * kSliceRows == C::BM && kSlices % 2 == 0 && kSliceRows % 16 == 0,
                "an even number of slices of 16k rows (the swizzle repeats every 16 rows)");
  struct State {
    __amdgpu_buffer_rsrc_t out;
    uint32_t ld;  // bytes
  };
  __device__ static __forceinline__ void reset(State& d) {
    d.out = make_rsrc(nullptr, 0);
    d.ld = 0;
  }
  __device__ static __forceinline__ void setup(State& d, bf16_t* const (&dst)[C::NB], int64_t ld, int rows) {
    const int h = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6) % C::NB;
    bf16_t* o = dst[0];
#pragma unroll
    for (int i = 1; i < C::NB; ++i) o = h == i ? dst[i] : o;
    d.out = rows_rsrc(o, rows, ld * 2, C::BNS * 2);
    d.ld = static_cast<uint32_t>(ld * 2);
  }
  __device__ static __forceinline__ void slice(const State& d, const char* stg, int sl) {
    const int lane = threadIdx.x & 63, wv = threadIdx.x >> 6;
    const int cq = lane % kCpr;
    const int row0 = (wv / C::NB) * kRowsPerWave + lane / kCpr;  // row within the slice
    const int s = sl < kSlices ? sl : kSlices - 1;
    const uint4 v = *reinterpret_cast<const uint4*>(stg + SO::off(row0, (wv % C::NB) * kCpr + cq) +
                                                    s * (kSliceRows * SO::kRowBytes));
    const uint32_t off = static_cast<uint32_t>(row0 + s * kSliceRows) * d.ld + cq * 16;
    buf_store16<kKeep>(d.out, sl < kSlices ? off : kOob, v);
  }
  __device__ static __forceinline__ void call(const State& d, const char* stg, int p) {  // two slices
    slice(d, stg, 2 * p);
    slice(d, stg, 2 * p + 1);
  }
};

// Mixin for providers whose staged tiles are copied out unchanged; Derived
// supplies stage_dst(job, dst, ld, rows).  kKeep: cached stores, for an
// output the next kernel reads straight back.
template <class C, class Derived, bool kKeep = false>
struct StagedCopyOut {
  using Copy = StagedCopy<C, kKeep>;
  static constexpr bool kStaged = true;
  using Drain = typename Copy::State;
  static constexpr int kDrainCalls = Copy::kCalls;
  __device__ __forceinline__ void drain_setup(const Job<C>& j, Drain& d) const {
    bf16_t* dst[C::NB];
    int64_t ld;
    int rows;
    static_cast<const Derived*>(this)->stage_dst(j, dst, ld, rows);
    Copy::setup(d, dst, ld, rows);
  }
  __device__ __forceinline__ void drain(Drain& d, const char* stg, int p) const { Copy::call(d, stg, p); }
  __device__ __forceinline__ void drain_reset(Drain& d) const { Copy::reset(d); }
};


// The drain interface of a staged provider, or nothing.
template <class P, bool kStaged>
struct DrainOf {
  struct type {};
  static constexpr int kCalls = 0;
};
template <class P>
struct DrainOf<P, true> {
  using type = typename P::Drain;
  static constexpr int kCalls = P::kDrainCalls;
};

// Runs every job of this workgroup (P::get(i, job) fills the i-th, false past
// the end; P::epilogue(job, acc) consumes a finished tile) as one continuous
// pipeline over the K steps of all jobs: the loads of step s + 3 and the LDS
// writes of step s + 1 overlap the MFMAs of step s even across tile
// boundaries, so a tile's first loads are in flight during the previous
// tile's last steps and its epilogue.
template <class C, bool A_KC, bool B_KC, class P>
__device__ __forceinline__ void gemm_stream(const P& prov, char* smem) {
  static_assert(std::is_same<C, typename P::C>::value, "the provider's tile shape");
  constexpr bool kStaged = staged_provider<P>::value;
  using LA = Loader<A_KC, C::BM, C::BM, C::kThreads>;
  using LB = Loader<B_KC, C::BNS, C::BN, C::kThreads>;
  using S0 = std::integral_constant<int, 0>;
  using S1 = std::integral_constant<int, 1>;
  const int tid = threadIdx.x;
  const int lane = tid & 63, wave = tid >> 6;
  const int wm = wave / C::WN, wn = wave % C::WN;
  LA la;
  LB lb[C::NB];
  uint4 ra[2][LA::kPer];
  uint4 rb[2][C::NB][LB::kPer];
  f32x4 acc[C::FM][C::FN];
  zero_acc<C>(acc);

  // load cursor: job li, step lkt.  Loads are issued unconditionally; once the
  // cursor has run past the last job the loaders read zeros without touching
  // memory.
  int li = 0, lkt = 0;
  Job<C> lj;
  bool lok = prov.get(0, lj);
  auto lsettle = [&]() {  // skip empty jobs, then set the loaders up for lj
    while (lok && lj.K <= 0) lok = prov.get(++li, lj);
    if (lok) {
      // kOpaqueSetup: the thread index made opaque here, so that the
      // per-lane offsets are recomputed at each job instead of being held
      // (and spilled) across the whole stream
      int t = tid;
      if constexpr (opaque_setup<P>::value) asm volatile("" : "+v"(t));
      la.setup(lj.a, lj.lda, lj.m_lim, lj.K, t);
#pragma unroll
      for (int i = 0; i < C::NB; ++i) lb[i].setup(lj.b[i], lj.ldb, lj.n_lim, lj.K, t);
    } else {
      la.disable();
#pragma unroll
      for (int i = 0; i < C::NB; ++i) lb[i].disable();
    }
  };
  lsettle();
  auto load = [&](auto set) {
    constexpr int S = decltype(set)::value;
    la.load(ra[S], lkt, lj.K, tid);
#pragma unroll
    for (int i = 0; i < C::NB; ++i) lb[i].load(rb[S][i], lkt, lj.K, tid);
  };
  auto lnext = [&]() {
    if (lok && ++lkt * BK >= lj.K) {
      lkt = 0;
      lok = prov.get(++li, lj);
      lsettle();
    }
  };
  auto store = [&](auto set, char* stage) {
    constexpr int S = decltype(set)::value;
    la.store(ra[S], stage, 0, tid);
#pragma unroll
    for (int i = 0; i < C::NB; ++i) lb[i].store(rb[S][i], stage + C::kABytes, i * C::BNS, tid);
  };

  // staged output (kStaged): the provider's drain state and the next drain
  // call (kCalls: nothing pending)
  char* const stg = smem + C::kLds;
  typename DrainOf<P, kStaged>::type dr;
  if constexpr (kStaged) prov.drain_reset(dr);
  constexpr int kCalls = DrainOf<P, kStaged>::kCalls;
  int d_call = kCalls;
  auto drain_next = [&]() {
    if constexpr (kStaged) prov.drain(dr, stg, d_call);
  };
  auto drain_rest = [&]() {
    if constexpr (kStaged)
      for (; d_call < kCalls; ++d_call) prov.drain(dr, stg, d_call);
  };
  auto finish = [&](const Job<C>& j) {  // a finished tile: epilogue, or into the staging area
    if constexpr (kStaged) {
      if (d_call < kCalls) {  // the previous tile is not fully drained yet (short K)
        drain_rest();
        lds_barrier();
      }
      const int wm_ = (tid >> 6) / C::WN;
#pragma unroll
      for (int mi = 0; mi < C::FM; ++mi) {
        const int r = wm_ * (C::BM / C::WM) + mi * 16 + (lane & 15);
#pragma unroll
        for (int ni = 0; ni < C::FN; ++ni) {
          const int c = frag_col<C>(ni, lane);
          *reinterpret_cast<uint2*>(stg + Staged<C>::off(r, c >> 3) + (c & 7) * 2) = pack4_bf16(acc[mi][ni]);
        }
      }
      prov.drain_setup(j, dr);
      d_call = 0;
      lds_barrier();
    } else {
      prov.epilogue(j, acc);
    }
  };

  // compute cursor: job ci, step ckt
  int ci = 0, ckt = 0;
  Job<C> cj;
  bool cok = prov.get(0, cj);
  auto csettle = [&]() {  // finish empty jobs (their tiles are zero unless chained)
    while (cok && cj.K <= 0) {
      if (!cj.chain) {
        finish(cj);
        zero_acc<C>(acc);
      }
      cok = prov.get(++ci, cj);
    }
  };
  csettle();
  auto cadvance = [&]() {
    if (++ckt * BK >= cj.K) {
      ckt = 0;
      if (!cj.chain) {
        finish(cj);
        zero_acc<C>(acc);
      }
      cok = prov.get(++ci, cj);
      csettle();
    }
  };

  constexpr int kReads = C::FM * (A_KC ? 1 : 2) + C::FN * (B_KC ? 1 : 2);
  constexpr int kMfma = C::FM * C::FN;
  constexpr int kWrites = LA::kPer + C::NB * LB::kPer;
  constexpr int kLoads = kWrites;
  // the interleave spreads reads, writes and loads evenly over the MFMAs,
  // also when a small tile has more of them than MFMAs
  auto step = [&](auto set) {
    constexpr int S = decltype(set)::value;
    using Other = std::integral_constant<int, 1 - S>;
    const char* cur = smem + S * C::kStage;
    char* nxt = smem + (1 - S) * C::kStage;
    uint4 af0[C::FM], bf0[C::FN], af1[C::FM], bf1[C::FN];
    // staged output: one drain call in the first step of each pair while
    // the staged tile lasts, before the step's fragment reads or, kLate,
    // after its operand loads (a fence keeps it out of the interleave, where
    // every register is taken)
    constexpr bool kDrain = kStaged && S == 0;
    constexpr bool kLate = drain_late<P>::value;
    if constexpr (kDrain && !kLate) {
      if (d_call < kCalls) drain_next();
      __builtin_amdgcn_sched_barrier(0);
    }
    read_frags<C, A_KC, B_KC>(cur, cur + C::kABytes, wm, wn, 0, lane, af0, bf0);
    read_frags<C, A_KC, B_KC>(cur, cur + C::kABytes, wm, wn, 1, lane, af1, bf1);
    mfmas<C>(af0, bf0, acc);
    mfmas<C>(af1, bf1, acc);
    store(Other{}, nxt);
    load(Other{});
    __builtin_amdgcn_sched_group_barrier(0x100, kReads, 0);
    interleave<kMfma, kReads, 0x100, 0, 0x200>();
    interleave<kMfma, kWrites, 0x200, kLoads, 0x020>();
    if constexpr (kDrain && kLate) {
      __builtin_amdgcn_sched_barrier(0);
      if (d_call < kCalls) drain_next();
      __builtin_amdgcn_sched_barrier(0);
    }
    if constexpr (kDrain) d_call = d_call < kCalls ? d_call + 1 : kCalls;
    lds_barrier();
    lnext();
  };

  if (!cok) {  // only empty jobs: the last of them may still be staged
    drain_rest();
    return;
  }
  load(S0{});
  lnext();
  load(S1{});
  lnext();
  store(S0{}, smem);
  lds_barrier();
  load(S0{});
  lnext();
  // Steps alternate S0, S1.  When the jobs run out after an S0 step, one more
  // S1 step runs on the disabled loaders (zeros, no memory access) and its
  // accumulation is dropped: every path back to S0 then passes through S1,
  // and the compiler's waits in S0 count S1's loads as in flight (an exit
  // after S0 left an edge to the loop head that skipped S1, and S0 waited
  // for loads issued one step earlier instead of two).
  for (;;) {  // cok holds here (checked above)
    step(S0{});
    cadvance();
    step(S1{});
    if (!cok) break;
    cadvance();
    if (!cok) break;
  }
  drain_rest();
  lds_barrier();  // the workgroup's LDS is free again
}


// Blocks are dispatched round-robin over the 8 XCDs (each with its own L2);
// give each XCD a contiguous range of logical tiles so that neighbouring
// tiles (same expert, same operand rows) share an L2.  nblocks % 8 == 0.
__device__ __forceinline__ int xcd_tile(int bid, int nblocks) {
  const int per = nblocks >> 3;
  return (bid & 7) * per + (bid >> 3);
}

// Tile of job i of this workgroup when each XCD takes one contiguous run of
// the `total` tiles over the whole launch: the n workgroups of XCD x take
// tiles x * per + j + i * n (j their index on the XCD, per = ceil(total / 8)),
// so the operands of neighbouring tiles (one expert's) are fetched into one
// L2 rather than into every XCD's.  -1 past this XCD's run.  nblocks % 8 == 0.
__device__ __forceinline__ int xcd_run(int i, int total) {
  const int n = gridDim.x >> 3;
  const int per = (total + 7) >> 3;
  const int r = static_cast<int>(blockIdx.x >> 3) + i * n;
  if (r >= per) return -1;
  const int t = static_cast<int>(blockIdx.x & 7) * per + r;
  return t < total ? t : -1;
}

}  // namespace moe
