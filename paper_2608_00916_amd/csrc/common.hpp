// Shared device helpers of the gfx950 MoE kernels: bf16 conversion, vector
// types, MFMA wrappers and wave-level reductions.  Wavefronts are 64 lanes.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace moe {

typedef uint16_t bf16_t;  // bfloat16 storage
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));

constexpr int kWave = 64;

__device__ __forceinline__ float bf2f(bf16_t v) {
  return __uint_as_float(static_cast<uint32_t>(v) << 16);
}

// A value every lane reads from the same address, loaded through the scalar
// data cache (constant address space).  Its wait then counts scalar loads
// only: a vector load of it would be followed by a wait for every vector
// load and store in flight.  Only for data that no running kernel writes
// (the scalar cache is invalidated at each kernel start, not during it).
template <class T>
__device__ __forceinline__ T uniform_load(const T* p) {
  return *(const __attribute__((address_space(4))) T*)(p);
}

// 16-byte load with the non-temporal cache policy, for data a kernel streams
// through once.
__device__ __forceinline__ uint4 load_nt(const void* p) {
  typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));
  return __builtin_bit_cast(uint4, __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(p)));
}

// Round to nearest even (v_cvt_pk_bf16_f32 on gfx950).
__device__ __forceinline__ bf16_t f2bf(float v) {
  __bf16 b = static_cast<__bf16>(v);
  return __builtin_bit_cast(bf16_t, b);
}

// Two floats -> one dword holding two bf16 (lo = a, hi = b).
__device__ __forceinline__ uint32_t pack_bf16x2(float a, float b) {
  return static_cast<uint32_t>(f2bf(a)) | (static_cast<uint32_t>(f2bf(b)) << 16);
}

__device__ __forceinline__ float lo_bf(uint32_t w) { return __uint_as_float(w << 16); }
__device__ __forceinline__ float hi_bf(uint32_t w) { return __uint_as_float(w & 0xffff0000u); }

// D(16x16, fp32) += P(16x32) * Q(32x16) with bf16 operands.  Lane l supplies
// P[l % 16][8 (l / 16) + v] and Q[8 (l / 16) + v][l % 16], v = 0..7, and holds
// D[4 (l / 16) + i][l % 16], i = 0..3.
__device__ __forceinline__ f32x4 mfma16x16x32(const uint4& p, const uint4& q, f32x4 acc) {
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, p),
                                                 __builtin_bit_cast(bf16x8, q), acc, 0, 0, 0);
}

template <typename T>
__device__ __forceinline__ T shfl_xor(T v, int mask) {
  return __shfl_xor(v, mask, kWave);
}

__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
  for (int m = 32; m >= 1; m >>= 1) v += shfl_xor(v, m);
  return v;
}

__device__ __forceinline__ float wave_max(float v) {
#pragma unroll
  for (int m = 32; m >= 1; m >>= 1) v = fmaxf(v, shfl_xor(v, m));
  return v;
}

// sigmoid(v) = 1 / (1 + e^-v) with the hardware reciprocal (v_rcp_f32, 1 ulp)
// rather than an IEEE division, which takes ten instructions; the results
// are rounded to bf16 afterwards.  silu(v) = v sigmoid(v).
__device__ __forceinline__ float sigmoid_f(float v) { return __builtin_amdgcn_rcpf(1.0f + __expf(-v)); }
__device__ __forceinline__ float silu_f(float v) { return v * sigmoid_f(v); }

__host__ __device__ constexpr int cdiv(int a, int b) { return (a + b - 1) / b; }
__host__ __device__ constexpr int64_t cdiv64(int64_t a, int64_t b) { return (a + b - 1) / b; }

}  // namespace moe
