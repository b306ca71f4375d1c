// Device helpers shared by the gfx950 kernels: BF16 unpacking, BF16 dot
// products, DPP row reductions and the base-2 exponential.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace fold {

typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef short s16x4 __attribute__((ext_vector_type(4)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));

// C += A . B on a 16x16 tile with K = 32 BF16 (v_mfma_f32_16x16x32_bf16).  Lane l
// holds A[l%16][8(l/16)..+8] and B[8(l/16)..+8][l%16]; C[4(l/16)+i][l%16] in c[i].
__device__ __forceinline__ f32x4 mfma_16x16x32(u32x4 a, u32x4 b, f32x4 c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, a),
                                                 __builtin_bit_cast(bf16x8, b), c, 0, 0, 0);
}

typedef _Float16 f16x8 __attribute__((ext_vector_type(8)));

// The same tile with FP16 operands (v_mfma_f32_16x16x32_f16).
__device__ __forceinline__ f32x4 mfma_16x16x32_f16(u32x4 a, u32x4 b, f32x4 c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_f16(__builtin_bit_cast(f16x8, a),
                                                __builtin_bit_cast(f16x8, b), c, 0, 0, 0);
}

// FP16 bits of x rounded to nearest even (v_cvt_f16_f32; subnormals kept).
__device__ __forceinline__ uint32_t f32_to_f16_bits(float x) {
  return static_cast<uint32_t>(__builtin_bit_cast(uint16_t, static_cast<_Float16>(x)));
}

// C += A . B on a 16x16 tile with K = 16 BF16 (v_mfma_f32_16x16x16_bf16).  Lane l
// holds A[l%16][4(l/16)..+4] and B[4(l/16)..+4][l%16]; C as above.
__device__ __forceinline__ f32x4 mfma_16x16x16(u32x2 a, u32x2 b, f32x4 c) {
  return __builtin_amdgcn_mfma_f32_16x16x16bf16_1k(__builtin_bit_cast(s16x4, a),
                                                   __builtin_bit_cast(s16x4, b), c, 0, 0, 0);
}

// BF16 halves of a 32-bit word (little endian: element 0 in the low half).
__device__ __forceinline__ float bf16_lo(uint32_t w) { return __uint_as_float(w << 16); }
__device__ __forceinline__ float bf16_hi(uint32_t w) { return __uint_as_float(w & 0xffff0000u); }

// Reinterpret a 32-bit word as two BF16 values.  The word must arrive as a
// scalar: clang lowers __builtin_bit_cast applied directly to an ext-vector
// component (v.y, v.z, ...) to a read of component 0.
__device__ __forceinline__ bf16x2 as_bf16x2(uint32_t w) { return __builtin_bit_cast(bf16x2, w); }

// sum_{e<8} k[e] * q[e] + acc over 8 packed BF16 values, FP32 accumulation
// (v_dot2_f32_bf16: two exact BF16 products per instruction).
__device__ __forceinline__ float dot8_bf16(u32x4 k, u32x4 q, float acc) {
  acc = __builtin_amdgcn_fdot2_f32_bf16(as_bf16x2(k.x), as_bf16x2(q.x), acc, false);
  acc = __builtin_amdgcn_fdot2_f32_bf16(as_bf16x2(k.y), as_bf16x2(q.y), acc, false);
  acc = __builtin_amdgcn_fdot2_f32_bf16(as_bf16x2(k.z), as_bf16x2(q.z), acc, false);
  acc = __builtin_amdgcn_fdot2_f32_bf16(as_bf16x2(k.w), as_bf16x2(q.w), acc, false);
  return acc;
}

template <int CTRL>
__device__ __forceinline__ float dpp_f32(float v) {
  return __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), CTRL, 0xF, 0xF, false));
}

// Sum over aligned groups of LANES (8 or 16) consecutive lanes; every lane of
// a group receives the same, bit-identical total (each step adds a value to
// its mirror image, and IEEE addition is commutative).
template <int LANES>
__device__ __forceinline__ float group_sum(float v) {
  static_assert(LANES == 8 || LANES == 16, "group of 8 or 16 lanes");
  v += dpp_f32<0xB1>(v);   // quad_perm [1,0,3,2]
  v += dpp_f32<0x4E>(v);   // quad_perm [2,3,0,1]
  v += dpp_f32<0x141>(v);  // row_half_mirror
  if constexpr (LANES == 16) v += dpp_f32<0x140>(v);  // row_mirror
  return v;
}

// OR over each aligned group of 16 lanes (every lane of a group gets it).
__device__ __forceinline__ uint32_t group_or16(uint32_t v) {
  v |= static_cast<uint32_t>(__builtin_amdgcn_update_dpp(0, static_cast<int>(v), 0xB1, 0xF, 0xF, false));
  v |= static_cast<uint32_t>(__builtin_amdgcn_update_dpp(0, static_cast<int>(v), 0x4E, 0xF, 0xF, false));
  v |= static_cast<uint32_t>(__builtin_amdgcn_update_dpp(0, static_cast<int>(v), 0x141, 0xF, 0xF, false));
  v |= static_cast<uint32_t>(__builtin_amdgcn_update_dpp(0, static_cast<int>(v), 0x140, 0xF, 0xF, false));
  return v;
}

// Base-2 exponential (v_exp_f32).
__device__ __forceinline__ float exp2_fast(float x) { return __builtin_amdgcn_exp2f(x); }
// Base-2 logarithm (v_log_f32).
__device__ __forceinline__ float log2_fast(float x) { return __builtin_amdgcn_logf(x); }

// Wave-wide max / sum without LDS: DPP within each row of 16 lanes, then the
// four row results read with v_readlane.  Every lane gets the same value;
// the order of additions is fixed.
__device__ __forceinline__ float wave_max_dpp(float v) {
  v = fmaxf(v, dpp_f32<0xB1>(v));
  v = fmaxf(v, dpp_f32<0x4E>(v));
  v = fmaxf(v, dpp_f32<0x141>(v));
  v = fmaxf(v, dpp_f32<0x140>(v));
  const float a = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), 0));
  const float b = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), 16));
  const float c = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), 32));
  const float d = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), 48));
  return fmaxf(fmaxf(a, b), fmaxf(c, d));
}

__device__ __forceinline__ float wave_sum_dpp(float v) {
  v = group_sum<16>(v);
  const float a = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), 0));
  const float b = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), 16));
  const float c = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), 32));
  const float d = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), 48));
  return (a + b) + (c + d);
}

__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) v += __shfl_xor(v, off, 64);
  return v;
}

__device__ __forceinline__ float wave_max(float v) {
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) v = fmaxf(v, __shfl_xor(v, off, 64));
  return v;
}

// Two FP32 values rounded to nearest even BF16 and packed, a in the low half
// (v_cvt_pk_bf16_f32).
__device__ __forceinline__ uint32_t pack_bf16_rne(float a, float b) {
  typedef float f32x2 __attribute__((ext_vector_type(2)));
  return __builtin_bit_cast(uint32_t, __builtin_convertvector((f32x2){a, b}, bf16x2));
}

// Round-to-nearest-even FP32 -> BF16 bits (NaN stays a quiet NaN).
__device__ __forceinline__ uint16_t f32_to_bf16_rne(float f) {
  uint32_t u = __float_as_uint(f);
  if ((u & 0x7fffffffu) > 0x7f800000u) return 0x7fc0;
  u += 0x7fffu + ((u >> 16) & 1u);
  return static_cast<uint16_t>(u >> 16);
}

// Read-only metadata (block tables, lengths, row lists) viewed through the
// constant address space: a wave-uniform index then compiles to a scalar load,
// whose completion is tracked apart from the vector loads of K and V.  The
// caller must not modify these arrays while a call is in flight.
typedef __attribute__((address_space(4))) const int32_t const_i32;
__device__ __forceinline__ int32_t ld_uniform(const int32_t* p, size_t i) {
  return ((const const_i32*)p)[i];  // address-space cast (C-style is required)
}

// Clamp a device-supplied sequence length to what the view can address.
__device__ __forceinline__ int clamp_len(int n, int cap) { return n < 0 ? 0 : (n > cap ? cap : n); }

}  // namespace fold
