// Device helpers for the gfx950 kernels of libqlinear.
#pragma once

#include <hip/hip_fp16.h>
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace ql {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

// fp32 -> bf16 bits, round to nearest even (NaN kept quiet).
__device__ __forceinline__ uint16_t f32_to_bf16(float f) {
  uint32_t u = __float_as_uint(f);
  if ((u & 0x7fffffffu) > 0x7f800000u) return (uint16_t)((u >> 16) | 0x0040u);
  u += 0x7fffu + ((u >> 16) & 1u);
  return (uint16_t)(u >> 16);
}

__device__ __forceinline__ float bf16_lo(uint32_t w) { return __uint_as_float(w << 16); }
__device__ __forceinline__ float bf16_hi(uint32_t w) { return __uint_as_float(w & 0xffff0000u); }

// binary16 bits -> fp32 (exact, subnormals included).
__device__ __forceinline__ float f16_to_f32(uint16_t b) {
  return (float)__builtin_bit_cast(_Float16, b);
}

// Order of the 8 k values a lane feeds to the MFMA from one 16-byte chunk.
// The int4 unpack below yields, from one 32-bit word of 8 codes (k0 in the
// low nibble), the pairs (k0,k4) (k1,k5) (k2,k6) (k3,k7); the activation
// chunk is permuted the same way so that both operands agree on k.
//   in  dwords: (x0,x1) (x2,x3) (x4,x5) (x6,x7)
//   out dwords: (x0,x4) (x1,x5) (x2,x6) (x3,x7)
__device__ __forceinline__ u32x4 permute_chunk(u32x4 v) {
  u32x4 o;
  o.x = __builtin_amdgcn_perm(v.z, v.x, 0x05040100u);
  o.y = __builtin_amdgcn_perm(v.z, v.x, 0x07060302u);
  o.z = __builtin_amdgcn_perm(v.w, v.y, 0x05040100u);
  o.w = __builtin_amdgcn_perm(v.w, v.y, 0x07060302u);
  return o;
}

// 8 int4 codes (two's complement) -> 8 bf16 values equal to 136 + q, exactly:
// u = q + 8 = nibble ^ 8 in [0, 15], and the bf16 pattern 0x4300 | u is
// 128 + u.  Both steps fold into one mask and one XOR per dword,
// ((w >> 4i) & 0x000F000F) ^ 0x43084308 (a single v_bitop3 on gfx950).  The
// constant 136 is removed through the correction term that starts every
// MFMA chain (-136 * sum of the activations of the group).
__device__ __forceinline__ bf16x8 unpack_offset_codes(uint32_t w) {
  u32x4 d;
  d.x = (w & 0x000f000fu) ^ 0x43084308u;
  d.y = ((w >> 4) & 0x000f000fu) ^ 0x43084308u;
  d.z = ((w >> 8) & 0x000f000fu) ^ 0x43084308u;
  d.w = ((w >> 12) & 0x000f000fu) ^ 0x43084308u;
  return __builtin_bit_cast(bf16x8, d);
}

// The same 8 codes in natural k order: dword i holds (136 + q[2i], 136 + q[2i+1]),
// matching an activation chunk read as stored.  Byte i of w holds q[2i] (low
// nibble) and q[2i+1] (high nibble); a byte permute places byte i of w in the
// low half and byte i of w >> 4 in the high half, then the mask / XOR of
// unpack_offset_codes applies.
__device__ __forceinline__ bf16x8 unpack_offset_codes_natural(uint32_t w) {
  const uint32_t w4 = w >> 4;
  u32x4 d;
  d.x = (__builtin_amdgcn_perm(w4, w, 0x04040000u) & 0x000f000fu) ^ 0x43084308u;
  d.y = (__builtin_amdgcn_perm(w4, w, 0x05050101u) & 0x000f000fu) ^ 0x43084308u;
  d.z = (__builtin_amdgcn_perm(w4, w, 0x06060202u) & 0x000f000fu) ^ 0x43084308u;
  d.w = (__builtin_amdgcn_perm(w4, w, 0x07070303u) & 0x000f000fu) ^ 0x43084308u;
  return __builtin_bit_cast(bf16x8, d);
}

__device__ __forceinline__ bf16x8 as_bf16x8(u32x4 v) { return __builtin_bit_cast(bf16x8, v); }

// bf16 -136.0 in both halves of every dword.
__device__ __forceinline__ bf16x8 neg136x8() {
  u32x4 d = {0xc308c308u, 0xc308c308u, 0xc308c308u, 0xc308c308u};
  return __builtin_bit_cast(bf16x8, d);
}

__device__ __forceinline__ f32x4 mfma16x16x32(bf16x8 a, bf16x8 b, f32x4 c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c, 0, 0, 0);
}

__device__ __forceinline__ float gelu_erf(float v) {
  return 0.5f * v * (1.0f + erff(v * 0.70710678118654752440f));
}

__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) v += __shfl_xor(v, o, 64);
  return v;
}

__device__ __forceinline__ float sum16(float v) {
#pragma unroll
  for (int o = 8; o >= 1; o >>= 1) v += __shfl_xor(v, o, 64);
  return v;
}

}  // namespace ql
