// Shared device helpers for the gfx950 kernels: bf16 vector types, MFMA
// wrappers and wavefront reductions.  CDNA4 wavefronts are 64 lanes wide.
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace al {

typedef __attribute__((__vector_size__(8 * sizeof(__bf16)))) __bf16 bf16x8;
typedef __attribute__((__vector_size__(4 * sizeof(__bf16)))) __bf16 bf16x4;
typedef __attribute__((ext_vector_type(2))) __bf16 bf16x2;
typedef __attribute__((__vector_size__(16 * sizeof(float)))) float f32x16;
typedef __attribute__((__vector_size__(4 * sizeof(float)))) float f32x4;
typedef __attribute__((__vector_size__(4 * sizeof(int)))) int i32x4;

constexpr int kWave = 64;

// D[32x32] += A[32x16] * B[16x32] in bf16 with fp32 accumulation.
// Lane l holds A[l%32][8*(l/32) + e], B[8*(l/32) + e][l%32] (e = 0..7) and
// D[8*(r/4) + 4*(l/32) + r%4][l%32] in register r = 0..15.
__device__ __forceinline__ f32x16 mfma32x32x16(bf16x8 a, bf16x8 b, f32x16 c) {
  return __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0);
}

// D[16x16] += A[16x32] * B[32x16] in bf16 with fp32 accumulation.
// Lane l holds A[l%16][8*(l/16) + e], B[8*(l/16) + e][l%16] (e = 0..7) and
// D[4*(l/16) + r][l%16] in register r = 0..3.
__device__ __forceinline__ f32x4 mfma16x16x32(bf16x8 a, bf16x8 b, f32x4 c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c, 0, 0, 0);
}

__device__ __forceinline__ float exp2_fast(float x) { return __builtin_amdgcn_exp2f(x); }

// fp32 -> bf16 round-to-nearest-even (finite inputs).
__device__ __forceinline__ uint16_t f32_to_bf16_bits(float f) {
  uint32_t u = __float_as_uint(f);
  u += 0x7FFFu + ((u >> 16) & 1u);
  return (uint16_t)(u >> 16);
}
__device__ __forceinline__ float bf16_bits_to_f32(uint16_t b) {
  return __uint_as_float(((uint32_t)b) << 16);
}

__device__ __forceinline__ bf16x8 zero_bf16x8() {
  i32x4 z = {0, 0, 0, 0};
  return __builtin_bit_cast(bf16x8, z);
}

__device__ __forceinline__ bf16x8 load_bf16x8(const uint16_t* p) {
  return __builtin_bit_cast(bf16x8, *reinterpret_cast<const i32x4*>(p));
}

// LDS transpose read (ds_read_b64_tr_b16).  Within each group of 16 lanes,
// lane j passes the address of the 4 consecutive elements at row j/4,
// columns 4(j%4)..4(j%4)+3 of a 4 x 16 block of 16-bit elements, and lane i
// of the group receives column i of that block (rows 0..3 in order).  The
// four groups' blocks are independent.
__device__ __forceinline__ bf16x4 lds_read_tr16(const uint16_t* p) {
  typedef __attribute__((address_space(3))) bf16x4 lds_bf16x4;
  return __builtin_amdgcn_ds_read_tr16_b64_v4bf16((lds_bf16x4*)(p));
}
__device__ __forceinline__ bf16x8 cat_bf16x4(bf16x4 a, bf16x4 b) {
  return __builtin_shufflevector(a, b, 0, 1, 2, 3, 4, 5, 6, 7);
}

// s_waitcnt immediate for gfx9-family encodings: wait until at most n vector
// memory loads are outstanding (n <= 63), no wait on the other counters.
constexpr int vmcnt_imm(int n) { return (n & 15) | (7 << 4) | (15 << 8) | ((n >> 4) << 14); }

// Lane exchange with lane l ^ 32 (the other half of the wavefront).
__device__ __forceinline__ float xor32(float v) { return __shfl_xor(v, 32, kWave); }
__device__ __forceinline__ int xor32(int v) { return __shfl_xor(v, 32, kWave); }

// max / sum of v over the lane pair (l, l ^ 32), the same value (and the
// same bits: both operations commute) on both lanes.  One cross-half swap,
// no LDS round trip.
__device__ __forceinline__ float pair_max32(float v) {
  const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(v), __float_as_uint(v), false, false);
  return fmaxf(__uint_as_float(r[0]), __uint_as_float(r[1]));
}
__device__ __forceinline__ float pair_sum32(float v) {
  const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(v), __float_as_uint(v), false, false);
  return __uint_as_float(r[0]) + __uint_as_float(r[1]);
}

}  // namespace al
