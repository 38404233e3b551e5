// Large-M int4-weight projection on bf16 MFMA (gfx950).
//
// out[m][n] = sum_g s[n][g] * sum_{k in g} x[m][k] * q[n][k]
//
// Each workgroup (4 waves) owns a 128 x 256 output tile; wave w owns the
// 128 x 64 column slice [64w, 64w+64).  The K loop walks one 128-wide scale
// group per step:
//   * the activation tile (128 rows x 128 k, pre-permuted bf16) and the
//     packed weight tile (256 columns x 64 bytes) are copied global -> LDS
//     with direct-to-LDS loads, double-buffered, one group ahead;
//   * each wave unpacks its 64 x 128 int4 codes once into bf16 values
//     136 + q (exact; see unpack_offset_codes) and reuses them for all 8
//     row fragments;
//   * per 16 x 16 output fragment, a chain of four 16x16x32 MFMAs covers the
//     group.  The chain starts from the correction -136 * sum_k x[m][k], so
//     its result is exactly the integer-code dot product sum x*q (fp32), and
//     one fp32 FMA applies the group's scale: acc += chain * s[n][g].
// Scales therefore stay exact fp32 (no bf16 rounding of q*s).
#include "ql_device.h"
#include "ql_internal.h"

namespace ql {

namespace {

constexpr int BM = kGemmBM;            // 128
constexpr int BN = kGemmBN;            // 256
constexpr int A_SLOTS = BM * 16;       // 16-byte slots per stage (32 KB)
constexpr int B_SLOTS = BN * 4;        // 16 KB

struct GemmParams {
  const uint16_t* xp;
  const float* ns;
  const uint8_t* qw;
  const uint16_t* sc;
  void* out;
  int64_t ldo, Mp;
  int M, N, K, G;
  int tiles_m, tiles_n;
};

// LDS slot swizzles (conflict-free 16-byte reads for 32- and 64-bank LDS).
__device__ __forceinline__ int a_phys(int row, int chunk) { return chunk ^ (row & 15); }
__device__ __forceinline__ int b_phys(int col, int h) { return h ^ (((col >> 1) ^ (col >> 2)) & 3); }

__device__ __forceinline__ void issue_stage(const GemmParams& p, int64_t m0, int64_t n0, int g,
                                            u32x4* sA, u32x4* sB, float* sN, int wave, int lane) {
  // activations: 8 wave-instructions of 64 x 16 B
#pragma unroll
  for (int j = 0; j < 8; ++j) {
    const int base = (j * 4 + wave) * 64;
    const int slot = base + lane;
    const int row = slot >> 4;
    const int chunk = (slot & 15) ^ (row & 15);
    const int64_t gm = min<int64_t>(m0 + row, p.M - 1);
    const uint16_t* src = p.xp + gm * p.K + (int64_t)g * kGroup + chunk * 8;
    __builtin_amdgcn_global_load_lds(src, sA + base, 16, 0, 0);
  }
  // packed weights: 4 wave-instructions of 64 x 16 B
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    const int base = (j * 4 + wave) * 64;
    const int slot = base + lane;
    const int col = slot >> 2;
    const int h = (slot & 3) ^ (((col >> 1) ^ (col >> 2)) & 3);
    const int64_t gn = min<int64_t>(n0 + col, p.N - 1);
    const uint8_t* src = p.qw + gn * (p.K / 2) + (int64_t)g * (kGroup / 2) + h * 16;
    __builtin_amdgcn_global_load_lds(src, sB + base, 16, 0, 0);
  }
  // correction terms of the 128 rows
  if (wave == 0) {
#pragma unroll
    for (int j = 0; j < 2; ++j) {
      const float* src = p.ns + (int64_t)g * p.Mp + m0 + j * 64 + lane;
      __builtin_amdgcn_global_load_lds(src, sN + j * 64, 4, 0, 0);
    }
  }
}

template <int EPI>
__device__ __forceinline__ void store_tile(const GemmParams& p, int64_t m0, int64_t n0, int wave,
                                           int lane, const f32x4 (&acc)[8][4]) {
  const int h = lane >> 4, lr = lane & 15;
#pragma unroll
  for (int i = 0; i < 8; ++i) {
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int64_t col = n0 + wave * 64 + j * 16 + lr;
      if (col >= p.N) continue;
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int64_t row = m0 + i * 16 + h * 4 + r;
        if (row >= p.M) continue;
        const float v = acc[i][j][r];
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
}

__device__ __forceinline__ void compute_stage(const u32x4* sA, const u32x4* sB, const float* sN,
                                              const float (&scf)[4], int wave, int lane,
                                              f32x4 (&acc)[8][4]) {
  const int h = lane >> 4, lr = lane & 15;
  bf16x8 bq[4][4];
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    const int col = wave * 64 + j * 16 + lr;
    const u32x4 raw = sB[col * 4 + b_phys(col, h)];
    bq[j][0] = unpack_offset_codes(raw.x);
    bq[j][1] = unpack_offset_codes(raw.y);
    bq[j][2] = unpack_offset_codes(raw.z);
    bq[j][3] = unpack_offset_codes(raw.w);
  }
#pragma unroll
  for (int i = 0; i < 8; ++i) {
    const int row = i * 16 + lr;
    const f32x4 n4 = *reinterpret_cast<const f32x4*>(sN + i * 16 + h * 4);
    bf16x8 a[4];
#pragma unroll
    for (int s = 0; s < 4; ++s) a[s] = as_bf16x8(sA[row * 16 + a_phys(row, h * 4 + s)]);
    f32x4 c[4] = {n4, n4, n4, n4};
#pragma unroll
    for (int s = 0; s < 4; ++s) {
#pragma unroll
      for (int j = 0; j < 4; ++j) c[j] = mfma16x16x32(a[s], bq[j][s], c[j]);
    }
#pragma unroll
    for (int j = 0; j < 4; ++j) acc[i][j] += c[j] * scf[j];
    __builtin_amdgcn_sched_barrier(0);
  }
}

template <int EPI>
__global__ __launch_bounds__(256, 1) void k_gemm(GemmParams p) {
  __shared__ u32x4 sA0[A_SLOTS];
  __shared__ u32x4 sA1[A_SLOTS];
  __shared__ u32x4 sB0[B_SLOTS];
  __shared__ u32x4 sB1[B_SLOTS];
  __shared__ float sN0[BM];
  __shared__ float sN1[BM];

  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63, lr = lane & 15;

  // workgroup -> tile: first spread consecutive tiles over the 8 XCDs'
  // dispatch order so that each XCD sees a contiguous tile range, then walk
  // that range 4 tile-rows at a time so concurrently resident tiles share
  // activation rows and weight columns in the XCD's L2.
  const int T = p.tiles_m * p.tiles_n;
  int bid = blockIdx.x;
  if ((T & 7) == 0) bid = (bid & 7) * (T >> 3) + (bid >> 3);
  constexpr int GM = 4;
  const int per_group = GM * p.tiles_n;
  const int grp = bid / per_group;
  const int first_m = grp * GM;
  const int gm = min(p.tiles_m - first_m, GM);
  const int in_grp = bid - grp * per_group;
  const int64_t m0 = (int64_t)(first_m + in_grp % gm) * BM;
  const int64_t n0 = (int64_t)(in_grp / gm) * BN;

  // scale pointers of this lane's four 16-column fragments
  const uint16_t* srow[4];
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    const int64_t col = min<int64_t>(n0 + wave * 64 + j * 16 + lr, p.N - 1);
    srow[j] = p.sc + col * p.G;
  }

  f32x4 acc[8][4];
#pragma unroll
  for (int i = 0; i < 8; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j) acc[i][j] = f32x4{0.f, 0.f, 0.f, 0.f};

  // scales of the next group stay raw until after the barrier so that the
  // loads overlap the current group's MFMAs
  float scf[4];
  uint16_t scn[4];
  issue_stage(p, m0, n0, 0, sA0, sB0, sN0, wave, lane);
#pragma unroll
  for (int j = 0; j < 4; ++j) scf[j] = f16_to_f32(srow[j][0]);
  __builtin_amdgcn_s_waitcnt(0);
  __syncthreads();

  for (int g = 0; g < p.G; g += 2) {
    // stage 0 holds group g
    if (g + 1 < p.G) {
      issue_stage(p, m0, n0, g + 1, sA1, sB1, sN1, wave, lane);
#pragma unroll
      for (int j = 0; j < 4; ++j) scn[j] = srow[j][g + 1];
    }
    compute_stage(sA0, sB0, sN0, scf, wave, lane, acc);
    __builtin_amdgcn_s_waitcnt(0);
    __syncthreads();
    if (g + 1 >= p.G) break;
#pragma unroll
    for (int j = 0; j < 4; ++j) scf[j] = f16_to_f32(scn[j]);
    // stage 1 holds group g + 1
    if (g + 2 < p.G) {
      issue_stage(p, m0, n0, g + 2, sA0, sB0, sN0, wave, lane);
#pragma unroll
      for (int j = 0; j < 4; ++j) scn[j] = srow[j][g + 2];
    }
    compute_stage(sA1, sB1, sN1, scf, wave, lane, acc);
    __builtin_amdgcn_s_waitcnt(0);
    __syncthreads();
#pragma unroll
    for (int j = 0; j < 4; ++j) scf[j] = f16_to_f32(scn[j]);
  }

  store_tile<EPI>(p, m0, n0, wave, lane, acc);
}

}  // namespace

hipError_t launch_gemm(const uint16_t* xp, const float* ns, int64_t Mp, const uint8_t* qw,
                       const uint16_t* sc, void* out, int64_t ldo, int64_t M, int64_t N,
                       int64_t K, int epilogue, hipStream_t s) {
  GemmParams p;
  p.xp = xp;
  p.ns = ns;
  p.qw = qw;
  p.sc = sc;
  p.out = out;
  p.ldo = ldo;
  p.Mp = Mp;
  p.M = (int)M;
  p.N = (int)N;
  p.K = (int)K;
  p.G = (int)(K / kGroup);
  p.tiles_m = (int)((M + BM - 1) / BM);
  p.tiles_n = (int)((N + BN - 1) / BN);
  const dim3 grid((unsigned)(p.tiles_m * p.tiles_n));
  switch (epilogue) {
    case 1: hipLaunchKernelGGL(k_gemm<1>, grid, dim3(256), 0, s, p); break;
    case 2: hipLaunchKernelGGL(k_gemm<2>, grid, dim3(256), 0, s, p); break;
    default: hipLaunchKernelGGL(k_gemm<0>, grid, dim3(256), 0, s, p); break;
  }
  return hipGetLastError();
}

}  // namespace ql
