// Packing, dequantization, activation preparation and RMSNorm kernels.
//
// Quantization scheme (the library's reading of the paper's 4-bit
// pre-quantized weights, Sec. 2.2 / 3.1 / 4.1): one fp16 scale per 128
// consecutive K elements of a weight row, s = fp16(fp32(amax / 7)), codes
// q = clamp(rint(fp32(w / s)), -8, 7), zero codes for a zero scale; two
// codes per byte, even k in the low nibble.
#include "ql_device.h"
#include "ql_internal.h"

namespace ql {

// ---------------------------------------------------------------------------
// pack: one wave per (row n, group j); each lane owns 2 consecutive weights.
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(256) void k_pack(const float* __restrict__ w,
                                              uint8_t* __restrict__ qw,
                                              uint16_t* __restrict__ sc, int64_t N, int64_t K,
                                              int32_t* __restrict__ status) {
  const int lane = threadIdx.x & 63;
  const int64_t G = K / kGroup;
  const int64_t gid = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);  // (n, j) flattened
  if (gid >= N * G) return;
  const int64_t n = gid / G, j = gid % G;
  const float2 v = *reinterpret_cast<const float2*>(w + n * K + j * kGroup + 2 * lane);
  const bool finite = __builtin_isfinite(v.x) && __builtin_isfinite(v.y);
  float a = fmaxf(fabsf(v.x), fabsf(v.y));
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) a = fmaxf(a, __shfl_xor(a, o, 64));
  const bool all_finite = __all(finite);
  // IEEE fp32 division (the library is built with correctly rounded divide)
  const float s32 = a / 7.0f;
  const __half s16 = __float2half_rn(s32);
  const float s = __half2float(s16);
  const bool ok = all_finite && !__hisinf(s16);
  uint8_t byte = 0;
  if (ok && s != 0.0f) {
    float q0 = fminf(fmaxf(rintf(v.x / s), -8.0f), 7.0f);
    float q1 = fminf(fmaxf(rintf(v.y / s), -8.0f), 7.0f);
    const int i0 = (int)q0, i1 = (int)q1;
    byte = (uint8_t)((i0 & 0xf) | ((i1 & 0xf) << 4));
  }
  qw[n * (K / 2) + j * (kGroup / 2) + lane] = byte;
  if (lane == 0) {
    sc[n * G + j] = ok ? __half_as_ushort(s16) : (uint16_t)0;
    if (!ok && status) atomicExch(status, 5 /* QL_ERR_RANGE */);
  }
}

hipError_t launch_pack(const float* w, uint8_t* qw, uint16_t* sc, int64_t N, int64_t K,
                       int32_t* status, hipStream_t s) {
  const int64_t groups = N * (K / kGroup);
  const int64_t blocks = (groups + 3) / 4;
  hipLaunchKernelGGL(k_pack, dim3((unsigned)blocks), dim3(256), 0, s, w, qw, sc, N, K, status);
  return hipGetLastError();
}

// ---------------------------------------------------------------------------
// dequant: thread per packed byte -> two exact fp32 products.
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(256) void k_dequant(const uint8_t* __restrict__ qw,
                                                 const uint16_t* __restrict__ sc,
                                                 float* __restrict__ w, int64_t N, int64_t K) {
  const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;  // byte index
  const int64_t H = K / 2;
  if (i >= N * H) return;
  const int64_t n = i / H, b = i % H;
  const int byte = qw[i];
  const int q0 = ((byte & 0xf) ^ 8) - 8;
  const int q1 = ((byte >> 4) ^ 8) - 8;
  const float s = f16_to_f32(sc[n * (K / kGroup) + (2 * b) / kGroup]);
  float2 o;
  o.x = (float)q0 * s;
  o.y = (float)q1 * s;
  *reinterpret_cast<float2*>(w + n * K + 2 * b) = o;
}

hipError_t launch_dequant(const uint8_t* qw, const uint16_t* sc, float* w, int64_t N,
                          int64_t K, hipStream_t s) {
  const int64_t bytes = N * (K / 2);
  hipLaunchKernelGGL(k_dequant, dim3((unsigned)((bytes + 255) / 256)), dim3(256), 0, s, qw, sc,
                     w, N, K);
  return hipGetLastError();
}

// ---------------------------------------------------------------------------
// Code layouts: row-major [N][K/2] <-> tiled, a permutation of 16-byte
// pieces.  Tiled piece t = ((b G + g) 4 + hh) 16 + c holds row-major piece
// (16 b + c) 4 G + 4 g + hh: bytes 16 hh .. 16 hh + 15 of column 16 b + c's
// 64 bytes of group g.  Thread per piece; the tiled side is the coalesced one.
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(256) void k_tile(const u32x4* __restrict__ src,
                                              u32x4* __restrict__ dst, int64_t pieces, int64_t G,
                                              bool to_tiled) {
  const int64_t t = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (t >= pieces) return;
  const int64_t b = t / (G * 64), r = t - b * (G * 64);
  const int64_t g = r >> 6, hh = (r >> 4) & 3, c = r & 15;
  const int64_t rm = (16 * b + c) * (4 * G) + 4 * g + hh;
  if (to_tiled)
    dst[t] = src[rm];
  else
    dst[rm] = src[t];
}

hipError_t launch_tile_codes(const uint8_t* src, uint8_t* dst, int64_t N, int64_t K,
                             bool to_tiled, hipStream_t s) {
  const int64_t pieces = N * K / 32;
  hipLaunchKernelGGL(k_tile, dim3((unsigned)((pieces + 255) / 256)), dim3(256), 0, s,
                     reinterpret_cast<const u32x4*>(src), reinterpret_cast<u32x4*>(dst), pieces,
                     K / kGroup, to_tiled);
  return hipGetLastError();
}

// ---------------------------------------------------------------------------
// prep: thread per 16-byte chunk (8 bf16) of x; 16 consecutive threads form
// one 128-wide group.  Writes the k-permuted copy and the correction terms.
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(256) void k_prep(const uint16_t* __restrict__ x, int64_t ldx,
                                              uint16_t* __restrict__ xp, float* __restrict__ ns,
                                              int64_t K, int64_t Mp) {
  const int64_t m = blockIdx.x;
  const int64_t c = (int64_t)blockIdx.y * 256 + threadIdx.x;  // chunk index in the row
  const int64_t nchunks = K / 8;
  float sum = 0.0f;
  if (c < nchunks) {
    const u32x4 v = *reinterpret_cast<const u32x4*>(x + m * ldx + c * 8);
    sum = ((bf16_lo(v.x) + bf16_hi(v.x)) + (bf16_lo(v.y) + bf16_hi(v.y))) +
          ((bf16_lo(v.z) + bf16_hi(v.z)) + (bf16_lo(v.w) + bf16_hi(v.w)));
    *reinterpret_cast<u32x4*>(xp + m * K + c * 8) = permute_chunk(v);
  }
  sum = sum16(sum);
  if ((threadIdx.x & 15) == 0 && c < nchunks) ns[(c / 16) * Mp + m] = -136.0f * sum;
}

hipError_t launch_prep(const uint16_t* x, int64_t ldx, uint16_t* xp, float* ns, int64_t M,
                       int64_t K, int64_t Mp, hipStream_t s) {
  const int64_t nchunks = K / 8;
  dim3 grid((unsigned)M, (unsigned)((nchunks + 255) / 256));
  hipLaunchKernelGGL(k_prep, grid, dim3(256), 0, s, x, ldx, xp, ns, K, Mp);
  return hipGetLastError();
}

// ---------------------------------------------------------------------------
// RMSNorm (unit gain): one workgroup per row, two passes over the row.
// ---------------------------------------------------------------------------
// One row per 256-thread block: thread t owns chunks t, t + 256, ... (8
// elements each).  The row is held in registers between the sum of squares
// and the scaling when it fits CPT chunks per thread (CPT = 0: re-read it).
// The same chunk order either way, so the result does not depend on CPT.
template <int CPT>
__global__ __launch_bounds__(256) void k_rmsnorm(const float* __restrict__ h,
                                                 uint16_t* __restrict__ a, float* __restrict__ ns,
                                                 int64_t d, int64_t Mp, float eps, int permuted) {
  __shared__ float red[4];
  const int64_t m = blockIdx.x;
  const float* row = h + m * d;
  const int64_t nchunks = d / 8;
  constexpr int R = CPT > 0 ? CPT : 1;
  float4 P[R], Q[R];
  float ss = 0.0f;
  if constexpr (CPT > 0) {
#pragma unroll
    for (int k = 0; k < CPT; ++k) {
      const int64_t c = k * 256 + threadIdx.x;
      if (c < nchunks) {
        P[k] = *reinterpret_cast<const float4*>(row + c * 8);
        Q[k] = *reinterpret_cast<const float4*>(row + c * 8 + 4);
      }
    }
#pragma unroll
    for (int k = 0; k < CPT; ++k) {
      const int64_t c = k * 256 + threadIdx.x;
      if (c < nchunks) {
        const float4 p = P[k], q = Q[k];
        ss += (p.x * p.x + p.y * p.y) + (p.z * p.z + p.w * p.w) + (q.x * q.x + q.y * q.y) +
              (q.z * q.z + q.w * q.w);
      }
    }
  } else {
    for (int64_t c = threadIdx.x; c < nchunks; c += 256) {
      const float4 p = *reinterpret_cast<const float4*>(row + c * 8);
      const float4 q = *reinterpret_cast<const float4*>(row + c * 8 + 4);
      ss += (p.x * p.x + p.y * p.y) + (p.z * p.z + p.w * p.w) + (q.x * q.x + q.y * q.y) +
            (q.z * q.z + q.w * q.w);
    }
  }
  ss = wave_sum(ss);
  if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = ss;
  __syncthreads();
  const float tot = (red[0] + red[1]) + (red[2] + red[3]);
  const float r = 1.0f / sqrtf(tot / (float)d + eps);
  // chunk loop with a trip count uniform across the block (shuffles below)
  auto emit = [&](int64_t c, const float4& p, const float4& q) {
    float sum = 0.0f;
    if (c < nchunks) {
      const uint16_t b0 = f32_to_bf16(p.x * r), b1 = f32_to_bf16(p.y * r);
      const uint16_t b2 = f32_to_bf16(p.z * r), b3 = f32_to_bf16(p.w * r);
      const uint16_t b4 = f32_to_bf16(q.x * r), b5 = f32_to_bf16(q.y * r);
      const uint16_t b6 = f32_to_bf16(q.z * r), b7 = f32_to_bf16(q.w * r);
      u32x4 v;
      v.x = (uint32_t)b0 | ((uint32_t)b1 << 16);
      v.y = (uint32_t)b2 | ((uint32_t)b3 << 16);
      v.z = (uint32_t)b4 | ((uint32_t)b5 << 16);
      v.w = (uint32_t)b6 | ((uint32_t)b7 << 16);
      if (permuted) {
        sum = ((bf16_lo(v.x) + bf16_hi(v.x)) + (bf16_lo(v.y) + bf16_hi(v.y))) +
              ((bf16_lo(v.z) + bf16_hi(v.z)) + (bf16_lo(v.w) + bf16_hi(v.w)));
        v = permute_chunk(v);
      }
      *reinterpret_cast<u32x4*>(a + m * d + c * 8) = v;
    }
    if (permuted) {
      sum = sum16(sum);
      if ((threadIdx.x & 15) == 0 && c < nchunks) ns[(c / 16) * Mp + m] = -136.0f * sum;
    }
  };
  if constexpr (CPT > 0) {
#pragma unroll
    for (int k = 0; k < CPT; ++k) {
      if ((int64_t)k * 256 >= nchunks) break;   // uniform across the block
      emit(k * 256 + threadIdx.x, P[k], Q[k]);
    }
  } else {
    for (int64_t c0 = 0; c0 < nchunks; c0 += 256) {
      const int64_t c = c0 + threadIdx.x;
      float4 p = {0.f, 0.f, 0.f, 0.f}, q = p;
      if (c < nchunks) {
        p = *reinterpret_cast<const float4*>(row + c * 8);
        q = *reinterpret_cast<const float4*>(row + c * 8 + 4);
      }
      emit(c, p, q);
    }
  }
}

hipError_t launch_rmsnorm(const float* h, uint16_t* a, float* ns, int64_t M, int64_t d,
                          int64_t Mp, float eps, bool permuted, hipStream_t s) {
  const int64_t cpt = (d / 8 + 255) / 256;   // chunks per thread
  const dim3 grid((unsigned)M), block(256);
  const int pm = permuted ? 1 : 0;
  if (cpt <= 2) hipLaunchKernelGGL(k_rmsnorm<2>, grid, block, 0, s, h, a, ns, d, Mp, eps, pm);
  else if (cpt <= 4) hipLaunchKernelGGL(k_rmsnorm<4>, grid, block, 0, s, h, a, ns, d, Mp, eps, pm);
  else if (cpt <= 8) hipLaunchKernelGGL(k_rmsnorm<8>, grid, block, 0, s, h, a, ns, d, Mp, eps, pm);
  else hipLaunchKernelGGL(k_rmsnorm<0>, grid, block, 0, s, h, a, ns, d, Mp, eps, pm);
  return hipGetLastError();
}

}  // namespace ql
