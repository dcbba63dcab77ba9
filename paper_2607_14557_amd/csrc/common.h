// Device helpers shared by the gfx950 kernels of the Seer layer library.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace seer {

typedef __attribute__((__vector_size__(8 * sizeof(__bf16)))) __bf16 bf16x8_t;
typedef __attribute__((__vector_size__(8 * sizeof(_Float16)))) _Float16 f16x8_t;
typedef __attribute__((__vector_size__(16 * sizeof(float)))) float f32x16_t;
typedef __attribute__((__vector_size__(4 * sizeof(float)))) float f32x4_t;

// 16-byte register type for global <-> LDS staging.  A native vector type
// (not HIP's struct uint4): arrays of it stay in registers after unrolling,
// where struct copies become private-memory memcpys.
typedef unsigned int u32x4_t __attribute__((ext_vector_type(4)));
typedef unsigned int u32x2_t __attribute__((ext_vector_type(2)));

typedef __attribute__((address_space(3))) void lds_void_t;
typedef __attribute__((address_space(3))) uint8_t lds_u8_t;
typedef __attribute__((address_space(1))) void glb_void_t;

constexpr int kWave = 64;

// bf16 <-> fp32.  bf16 values are carried as raw 16-bit patterns.
__device__ __forceinline__ float bf2f(uint16_t h) {
  return __uint_as_float(static_cast<uint32_t>(h) << 16);
}

typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
typedef float f32x2_t __attribute__((ext_vector_type(2)));

// fp32 -> bf16, round to nearest even, NaN stays NaN: one v_cvt_pk_bf16_f32
// on gfx950 for a pair.
__device__ __forceinline__ uint32_t pack_bf2(float lo, float hi) {
  return __builtin_bit_cast(uint32_t, __builtin_convertvector(f32x2_t{lo, hi}, bf16x2_t));
}

__device__ __forceinline__ uint16_t f2bf(float f) {
  return __builtin_bit_cast(uint16_t, static_cast<__bf16>(f));
}

__device__ __forceinline__ bf16x8_t as_bf16x8(uint4 v) {
  return __builtin_bit_cast(bf16x8_t, v);
}

__device__ __forceinline__ f16x8_t as_f16x8(uint4 v) {
  return __builtin_bit_cast(f16x8_t, v);
}

typedef _Float16 f16x2_t __attribute__((ext_vector_type(2)));

// fp32 -> fp16, round to nearest even.
__device__ __forceinline__ uint32_t f2h_bits(float f) {
  return static_cast<uint32_t>(__builtin_bit_cast(uint16_t, static_cast<_Float16>(f)));
}

// A pair in one v_cvt_pk_f16_f32.
__device__ __forceinline__ uint32_t pack_h2(float lo, float hi) {
  return __builtin_bit_cast(uint32_t, __builtin_convertvector(f32x2_t{lo, hi}, f16x2_t));
}

// bf16 bits -> fp16 bits (exact for magnitudes in fp16's normal range).
__device__ __forceinline__ uint32_t bf_to_h_bits(uint32_t bf) {
  return f2h_bits(__uint_as_float(bf << 16));
}

// z * sigmoid(z) with the hardware reciprocal (1 ulp) instead of a division.
__device__ __forceinline__ float silu(float z) {
  return z * __builtin_amdgcn_rcpf(1.0f + __expf(-z));
}

__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) v += __shfl_xor(v, off, kWave);
  return v;
}

__device__ __forceinline__ float wave_max(float v) {
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) v = fmaxf(v, __shfl_xor(v, off, kWave));
  return v;
}

__device__ __forceinline__ int wave_min_int(int v) {
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) v = min(v, __shfl_xor(v, off, kWave));
  return v;
}

// Workgroup ids are dealt round robin over the 8 XCDs.  xcd_remap turns block
// id bid in [0, nblk) into a logical unit id such that each XCD walks a
// contiguous range of logical units (surplus ids past a multiple of 8 map to
// themselves), so units that share operands run on one XCD and its L2.
__device__ __forceinline__ int xcd_remap(int bid, int nblk) {
  const int per = nblk >> 3;
  return bid < (per << 3) ? (bid & 7) * per + (bid >> 3) : bid;
}

// Row count of a packed batch: cu_seqlens[batch] when given, clamped to the
// host-side upper bound that sized the grid.
__device__ __forceinline__ int rows_from(const int* m_ptr, int m_ub) {
  if (m_ptr == nullptr) return m_ub;
  int m = *m_ptr;
  return m < 0 ? 0 : (m > m_ub ? m_ub : m);
}

}  // namespace seer
