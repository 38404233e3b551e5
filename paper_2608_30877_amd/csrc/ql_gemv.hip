// Small-batch (M <= 16) int4-weight projection: weight bytes bound the run.
//
// Each workgroup (4 waves) owns 64 output columns over the full K; wave w
// takes the scale groups g = w, w+4, w+8, ... so the four waves stream
// adjacent 64-byte pieces of the same weight rows.  Per group, each lane
// issues one 16-byte load per 16-column fragment (the lane's 32 codes),
// unpacks them to bf16 136 + q and runs a 16x16x32 MFMA chain against the
// (at most 16) activation rows; the activation rows' group sums come from
// one more MFMA chain against a constant -136 operand, which starts each
// chain so that it yields the exact code dot product.  The partial sums of
// the four waves are then reduced through LDS (the wavefront reduction) and
// the epilogue is applied.
#include "ql_device.h"
#include "ql_internal.h"

namespace ql {

namespace {

struct GemvParams {
  const uint16_t* x;
  const uint8_t* qw;
  const uint16_t* sc;
  void* out;
  int64_t ldx, ldo;
  int M, N, K, G;
};

struct GroupData {
  u32x4 b[4];
  uint16_t s[4];
  u32x4 a[4];
};

__device__ __forceinline__ void load_group(const GemvParams& p, const uint8_t* const (&wrow)[4],
                                           const uint16_t* const (&srow)[4], const uint16_t* xrow,
                                           int g, int h, GroupData& d) {
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    d.b[j] = *reinterpret_cast<const u32x4*>(wrow[j] + (int64_t)g * (kGroup / 2));
    d.s[j] = srow[j][g];
  }
#pragma unroll
  for (int s = 0; s < 4; ++s)
    d.a[s] = *reinterpret_cast<const u32x4*>(xrow + (int64_t)g * kGroup + (h * 4 + s) * 8);
}

__device__ __forceinline__ void compute_group(const GroupData& d, f32x4 (&acc)[4]) {
  const bf16x8 neg = neg136x8();
  bf16x8 a[4];
#pragma unroll
  for (int s = 0; s < 4; ++s) a[s] = as_bf16x8(permute_chunk(d.a[s]));
  f32x4 nc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
  for (int s = 0; s < 4; ++s) nc = mfma16x16x32(a[s], neg, nc);
  f32x4 c[4] = {nc, nc, nc, nc};
#pragma unroll
  for (int s = 0; s < 4; ++s) {
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const uint32_t wv = s == 0 ? d.b[j].x : s == 1 ? d.b[j].y : s == 2 ? d.b[j].z : d.b[j].w;
      c[j] = mfma16x16x32(a[s], unpack_offset_codes(wv), c[j]);
    }
  }
#pragma unroll
  for (int j = 0; j < 4; ++j) acc[j] += c[j] * f16_to_f32(d.s[j]);
}

template <int EPI>
__global__ __launch_bounds__(256) void k_gemv(GemvParams p) {
  __shared__ f32x4 red[3][4][64];
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int h = lane >> 4, lr = lane & 15;
  const int64_t n0 = (int64_t)blockIdx.x * 64;

  // rows past M and columns past N read valid (clamped) memory; their
  // results are never stored
  const uint16_t* xrow = p.x + (int64_t)min(lr, p.M - 1) * p.ldx;
  const uint8_t* wrow[4];
  const uint16_t* srow[4];
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    const int64_t col = min<int64_t>(n0 + j * 16 + lr, p.N - 1);
    wrow[j] = p.qw + col * (p.K / 2) + h * 16;
    srow[j] = p.sc + col * p.G;
  }

  f32x4 acc[4];
#pragma unroll
  for (int j = 0; j < 4; ++j) acc[j] = f32x4{0.f, 0.f, 0.f, 0.f};

  // software pipeline: the loads of the next group are in flight while the
  // current one is unpacked and multiplied
  int g = wave;
  GroupData cur, nxt;
  if (g < p.G) load_group(p, wrow, srow, xrow, g, h, cur);
  while (g < p.G) {
    const int gn = g + 4;
    if (gn < p.G) load_group(p, wrow, srow, xrow, gn, h, nxt);
    compute_group(cur, acc);
    cur = nxt;
    g = gn;
  }

  if (wave > 0) {
#pragma unroll
    for (int j = 0; j < 4; ++j) red[wave - 1][j][lane] = acc[j];
  }
  __syncthreads();
  if (wave != 0) return;
#pragma unroll
  for (int w = 0; w < 3; ++w)
#pragma unroll
    for (int j = 0; j < 4; ++j) acc[j] += red[w][j][lane];

#pragma unroll
  for (int j = 0; j < 4; ++j) {
    const int64_t col = n0 + j * 16 + lr;
    if (col >= p.N) continue;
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const int row = h * 4 + r;
      if (row >= p.M) continue;
      const float v = acc[j][r];
      if constexpr (EPI == 2) {
        float* o = reinterpret_cast<float*>(p.out) + row * p.ldo + col;
        *o = *o + v;
      } else if constexpr (EPI == 1) {
        reinterpret_cast<uint16_t*>(p.out)[row * p.ldo + col] = f32_to_bf16(gelu_erf(v));
      } else {
        reinterpret_cast<uint16_t*>(p.out)[row * p.ldo + col] = f32_to_bf16(v);
      }
    }
  }
}

}  // namespace

hipError_t launch_gemv(const uint16_t* x, int64_t ldx, const uint8_t* qw, const uint16_t* sc,
                       void* out, int64_t ldo, int64_t M, int64_t N, int64_t K, int epilogue,
                       hipStream_t s) {
  GemvParams p;
  p.x = x;
  p.qw = qw;
  p.sc = sc;
  p.out = out;
  p.ldx = ldx;
  p.ldo = ldo;
  p.M = (int)M;
  p.N = (int)N;
  p.K = (int)K;
  p.G = (int)(K / kGroup);
  const dim3 grid((unsigned)((N + 63) / 64));
  switch (epilogue) {
    case 1: hipLaunchKernelGGL(k_gemv<1>, grid, dim3(256), 0, s, p); break;
    case 2: hipLaunchKernelGGL(k_gemv<2>, grid, dim3(256), 0, s, p); break;
    default: hipLaunchKernelGGL(k_gemv<0>, grid, dim3(256), 0, s, p); break;
  }
  return hipGetLastError();
}

}  // namespace ql
