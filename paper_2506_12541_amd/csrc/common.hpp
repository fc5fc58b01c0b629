// Device helpers shared by the BSA kernels: storage types, bf16 conversion, wave64
// reductions and the MFMA fragment convention used by every attention kernel.
//
// Fragment convention (16x16 MFMA tiles, wave64). A 16-row operand slice of width D
// (D = 32 or 64 contraction values) is held as D/32 "chunks" per lane: lane L serves
// row (L % 16) and, for chunk c, the 8 consecutive contraction indices
// [32c + 8*(L/16), 32c + 8*(L/16) + 8). Both MFMA operands use the same mapping, so
// the contraction is exact whatever order the hardware pairs the 8 values in.
//   bf16: one chunk = one v_mfma_f32_16x16x32_bf16.
//   f32 : one chunk = eight v_mfma_f32_16x16x4_f32 (value e of each lane per MFMA).
// Accumulator (16x16 f32): lane L holds column (L % 16), rows 4*(L/16) + i, i = 0..3.
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace bsa {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef float f32x8 __attribute__((ext_vector_type(8)));
typedef uint16_t bf16_t;  // storage of one bfloat16

constexpr float kLog2e = 1.4426950408889634f;
constexpr float kLn2 = 0.6931471805599453f;

__device__ __forceinline__ float bf2f(bf16_t h) { return __uint_as_float((uint32_t)h << 16); }

// Round to nearest even (hardware v_cvt_pk_bf16_f32 on gfx950).
__device__ __forceinline__ bf16_t f2bf(float f) { return __builtin_bit_cast(bf16_t, (__bf16)f); }

// Storage traits: element type in memory, and its 8-wide chunk register type.
template <typename T> struct Chunk;
template <> struct Chunk<bf16_t> {
  typedef bf16x8 type;                 // 16 bytes
  static constexpr int bytes = 16;
};
template <> struct Chunk<float> {
  typedef f32x8 type;                  // 32 bytes
  static constexpr int bytes = 32;
};

template <typename T> __device__ __forceinline__ float to_f32(T x);
template <> __device__ __forceinline__ float to_f32<float>(float x) { return x; }
template <> __device__ __forceinline__ float to_f32<bf16_t>(bf16_t x) { return bf2f(x); }

template <typename T> __device__ __forceinline__ T from_f32(float x);
template <> __device__ __forceinline__ float from_f32<float>(float x) { return x; }
template <> __device__ __forceinline__ bf16_t from_f32<bf16_t>(float x) { return f2bf(x); }

// Load one 8-element chunk (16 B for bf16, 32 B for f32) from global or LDS memory.
__device__ __forceinline__ bf16x8 load_chunk(const bf16_t* p) {
  return *reinterpret_cast<const bf16x8*>(p);
}
__device__ __forceinline__ f32x8 load_chunk(const float* p) {
  return *reinterpret_cast<const f32x8*>(p);
}

// Build a chunk from 8 f32 values (rounded to the storage type).
template <typename T> __device__ __forceinline__ typename Chunk<T>::type make_chunk(const float* v);
template <> __device__ __forceinline__ bf16x8 make_chunk<bf16_t>(const float* v) {
  bf16x8 r;
#pragma unroll
  for (int i = 0; i < 8; ++i) r[i] = (__bf16)v[i];
  return r;
}
template <> __device__ __forceinline__ f32x8 make_chunk<float>(const float* v) {
  f32x8 r;
#pragma unroll
  for (int i = 0; i < 8; ++i) r[i] = v[i];
  return r;
}

// Element e of a chunk as its storage bits (e must fold to a constant).
__device__ __forceinline__ bf16_t chunk_elem(const bf16x8& c, int e) {
  const uint4 u = __builtin_bit_cast(uint4, c);
  const uint32_t w = e < 2 ? u.x : (e < 4 ? u.y : (e < 6 ? u.z : u.w));
  return (bf16_t)((w >> (16 * (e & 1))) & 0xFFFFu);
}
__device__ __forceinline__ float chunk_elem(const f32x8& c, int e) { return c[e]; }

__device__ __forceinline__ bf16x8 zero_chunk(bf16x8) { return bf16x8{}; }
__device__ __forceinline__ f32x8 zero_chunk(f32x8) { return f32x8{}; }

// acc += A_chunk x B_chunk over 8 contraction values per lane group (32 per tile).
__device__ __forceinline__ f32x4 mma(bf16x8 a, bf16x8 b, f32x4 c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c, 0, 0, 0);
}
__device__ __forceinline__ f32x4 mma(f32x8 a, f32x8 b, f32x4 c) {
#pragma unroll
  for (int e = 0; e < 8; ++e) c = __builtin_amdgcn_mfma_f32_16x16x4f32(a[e], b[e], c, 0, 0, 0);
  return c;
}

// ---- wave64 reductions ----
__device__ __forceinline__ float wave_max(float x) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) x = fmaxf(x, __shfl_xor(x, o, 64));
  return x;
}
__device__ __forceinline__ float wave_sum(float x) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) x += __shfl_xor(x, o, 64);
  return x;
}
// Reduce across the four lane groups {L, L^16, L^32, L^48} (one accumulator column).
// The exchanges are gfx950's VALU lane swaps rather than LDS permutes: with both operands
// holding x, v_permlane16_swap leaves each lane the values of its 16-lane group and of
// the group next to it (L^16), v_permlane32_swap those of L and L^32. Keeping the
// exchange off the LDS pipe also means it does not wait behind LDS reads in flight.
__device__ __forceinline__ float xor16_pair(float x, float& other) {
  const auto t = __builtin_amdgcn_permlane16_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  other = __uint_as_float(t[1]);
  return __uint_as_float(t[0]);
}
__device__ __forceinline__ float xor32_pair(float x, float& other) {
  const auto t = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  other = __uint_as_float(t[1]);
  return __uint_as_float(t[0]);
}
__device__ __forceinline__ float col_max(float x) {
  float y;
  x = xor16_pair(x, y);
  x = fmaxf(x, y);
  x = xor32_pair(x, y);
  return fmaxf(x, y);
}
__device__ __forceinline__ float col_sum(float x) {
  float y;
  x = xor16_pair(x, y);
  x += y;
  x = xor32_pair(x, y);
  return x + y;
}
// Reduce across the 16 lanes of one lane group (one accumulator row set).
__device__ __forceinline__ float row16_sum(float x) {
#pragma unroll
  for (int o = 8; o > 0; o >>= 1) x += __shfl_xor(x, o, 64);
  return x;
}

// Order this wave's LDS accesses across lanes (data staged by the wave for itself).
// Wait until every global load of this wave has returned (s_waitcnt vmcnt(0)). Placed
// after loop-invariant operands are loaded and before a loop that prefetches its next
// tile: the wait the compiler puts in front of the operands' first use inside the loop
// would otherwise also wait, on every iteration, for that iteration's prefetch.
__device__ __forceinline__ void vm_drain() { __builtin_amdgcn_s_waitcnt(0x0F70); }

__device__ __forceinline__ void wave_sync() {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
}

__device__ __forceinline__ float fast_exp2(float x) { return __builtin_amdgcn_exp2f(x); }
__device__ __forceinline__ float fast_log2(float x) { return __builtin_amdgcn_logf(x); }

}  // namespace bsa
