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

// Direct-to-LDS copies: lane l writes lds + l * BYTES (a 2-byte copy writes
// its value zero-extended into the dword lds + 4 * l).  Written as inline
// assembly, so the compiler does not track these loads: the kernel waits for
// them itself (s_waitcnt vmcnt), and every vector load it issues after them
// may stay in flight while it does.  M0 carries the LDS base (one wait state
// must separate its write from the load that reads it); M0 is a register the
// compiler reserves, so each sequence saves and restores it instead of
// clobbering it.  Addresses are a uniform 64-bit base in scalar registers
// plus a per-lane 32-bit byte offset.
#define QL_LDS_COPY(OP, V, B, L) \
  "s_mov_b32 m0, %[" L "]\n\ts_nop 0\n\t" OP " %[" V "], %[" B "]\n\t"

// one 2- or 4-byte copy
template <int BYTES>
__device__ __forceinline__ void copy_to_lds(const void* base, uint32_t off, const void* lds) {
  const uint32_t l = (uint32_t)reinterpret_cast<uintptr_t>(lds);
  uint32_t saved;
  if constexpr (BYTES == 4) {
    asm volatile("s_mov_b32 %[sv], m0\n\t" QL_LDS_COPY("global_load_lds_dword", "o", "b", "l")
                 "s_mov_b32 m0, %[sv]"
                 : [sv] "=&s"(saved) : [o] "v"(off), [b] "s"(base), [l] "s"(l) : "memory");
  } else {
    static_assert(BYTES == 2, "copy width");
    asm volatile("s_mov_b32 %[sv], m0\n\t" QL_LDS_COPY("global_load_lds_ushort", "o", "b", "l")
                 "s_mov_b32 m0, %[sv]"
                 : [sv] "=&s"(saved) : [o] "v"(off), [b] "s"(base), [l] "s"(l) : "memory");
  }
}

// one 16-byte copy
__device__ __forceinline__ void copy16_to_lds(const void* base, uint32_t off, uint32_t lds) {
  uint32_t saved;
  asm volatile("s_mov_b32 %[sv], m0\n\t" QL_LDS_COPY("global_load_lds_dwordx4", "o", "b", "l")
               "s_mov_b32 m0, %[sv]"
               : [sv] "=&s"(saved) : [o] "v"(off), [b] "s"(base), [l] "s"(lds) : "memory");
}
#undef QL_LDS_COPY

// s_waitcnt immediate (gfx9 layout): vmcnt(n) (0 <= n < 64), lgkmcnt(0),
// expcnt not waited on
constexpr int vmcnt_lgkm0(int n) { return 0x0070 | (n & 15) | ((n >> 4) << 14); }

// Workgroup barrier without the memory fence of __syncthreads (which would
// also wait for every copy in flight).
__device__ __forceinline__ void wg_barrier() {
  asm volatile("" ::: "memory");
  __builtin_amdgcn_s_barrier();
  asm volatile("" ::: "memory");
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

// GELU in its erf form, z Phi(z) = z/2 (1 + erf(z / sqrt 2)).  The normal
// tail Q(|z|) = 1 - Phi(|z|) is evaluated as exp(-z^2/2) s P(s),
// s = 1 / (1 + p |z|) -- the form of Abramowitz & Stegun 26.2.17, with p and
// the seven coefficients of P (1/sqrt(2 pi) folded in) fitted for relative
// error (gelu_fit.py): at most 7e-7 in exact arithmetic and about 1.2e-5
// as evaluated here in fp32 over |z| <= 14 (3.3e-6 for |z| < 6).
// Then Phi(z) = 1 - Q for z >= 0 and Q otherwise, so the negative tail keeps
// its relative accuracy down to the subnormals (1 + erff(z / sqrt 2) cancels
// in fp32 below about z = -4), at half the instructions of erff; rounded to
// bf16, an output is at most one ulp from the correctly rounded GELU.
__device__ __forceinline__ float gelu_erf(float v) {
  const float a = fabsf(v);
  const float s = __builtin_amdgcn_rcpf(fmaf(0.36151701f, a, 1.0f));
  float r = 4.801544920e-02f;
  r = fmaf(r, s, -1.809354275e-01f);
  r = fmaf(r, s, 1.789837331e-01f);
  r = fmaf(r, s, 2.738756500e-02f);
  r = fmaf(r, s, 1.398224235e-01f);
  r = fmaf(r, s, 1.424095929e-01f);
  r = fmaf(r, s, 1.443170309e-01f);
  // Q scaled by 2^24: v_exp_f32 returns no subnormals, so the exponential is
  // taken 24 binades up and the final product, which does, scales back
  const float q = __builtin_amdgcn_exp2f(fmaf(a * a, -0.72134751f, 24.0f)) * (r * s);
  return v >= 0.0f ? v * (1.0f - q * 5.9604645e-08f) : (v * q) * 5.9604645e-08f;
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
