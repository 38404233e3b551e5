// Causal sliding-window multi-head attention between the QKV and output
// projections (the paper's decoder uses sliding-window attention, Sec. 1
// contribution 1.1 and Sec. 2).  Each sequence of seq_len tokens (one
// protein-ligand pair) is independent; token i attends to the tokens j of its
// sequence with i - window < j <= i.  Head dimension 128.
//
// One workgroup (4 waves) owns 64 queries of one head; wave w owns 16 of
// them.  Key blocks of 64 are staged in LDS: K row-major, V transposed.  The
// scores are computed transposed, S^T = K Q^T (16x16x32 bf16 MFMAs with K as
// the row operand), so that a lane ends up holding, for its query, exactly
// the keys it feeds as the column operand of O^T += V^T P^T: nothing moves
// between the two products.  Softmax is online in fp32 (base 2); P is
// rounded to bf16 for the second product and the row sums add the rounded
// values, so the weights the product sees sum to one; O stays fp32 until the
// final bf16 store.
#include <algorithm>

#include "ql_device.h"
#include "ql_internal.h"

namespace ql {

namespace {

constexpr int kDh = 128;  // head dimension
constexpr int kBQ = 64;   // queries per workgroup
constexpr int kBK = 64;   // keys per LDS block

struct AttnParams {
  const uint16_t* qkv;
  uint16_t* out;
  int64_t ldq, ldo;
  int d, L, W, heads, nqb, tiles;
  float scale2;  // log2(e) / sqrt(head dim)
};

// K tile: key r keeps its 16-byte chunk c (dims 8c .. 8c+7) at slot
// r * 16 + (c ^ k_msk(r)); the 16-byte reads of one S^T step are then
// conflict-free (same row mask as the projection kernel's activation tile).
__device__ __forceinline__ int k_msk(int r) {
  r &= 15;
  return r ^ ((((r >> 2) ^ (r >> 3)) & 1) << 2);
}
// V^T tile: dim row e holds the block's 64 keys (128 bytes) in the order
// vpos(key); chunk c of row e sits at slot e * 8 + (c ^ v_msk(e)).
__device__ __forceinline__ int v_msk(int e) {
  return (((e >> 1) & 1) | (((e >> 3) & 1) << 1)) << 1;
}
// key = 32 t + 16 f + 4 hh + r  ->  32 t + 8 hh + 4 f + r: the 8 keys that lane
// group hh feeds to one V^T P^T step (fragments 2t and 2t+1 of S^T) are then
// one contiguous chunk, 4t + hh.
__device__ __forceinline__ int vpos(int key) {
  const int t = key >> 5, f = (key >> 4) & 1, hh = (key >> 2) & 3, r = key & 3;
  return 32 * t + 8 * hh + 4 * f + r;
}

__device__ __forceinline__ float max_over_h(float v) {
  v = fmaxf(v, __shfl_xor(v, 16, 64));
  return fmaxf(v, __shfl_xor(v, 32, 64));
}
__device__ __forceinline__ float sum_over_h(float v) {
  v += __shfl_xor(v, 16, 64);
  return v + __shfl_xor(v, 32, 64);
}

__global__ __launch_bounds__(256) void k_attn(AttnParams p) {
  __shared__ u32x4 sK[kBK * 16];  // 16 KB
  __shared__ u32x4 sV[kDh * 8];   // 16 KB
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  const int h = lane >> 4, lr = lane & 15;

  // Workgroup -> tile.  Consecutive workgroup ids go to the 8 XCDs in turn;
  // give each XCD a contiguous tile range so that the query blocks of one
  // (sequence, head) -- which read the same keys and values -- share its L2.
  int t = blockIdx.x;
  {
    const int q = p.tiles >> 3, r = p.tiles & 7, x = t & 7, i = t >> 3;
    t = x < r ? x * (q + 1) + i : r * (q + 1) + (x - r) * q + i;
  }
  // within a (sequence, head) the longest query blocks come first
  const int ph = t / p.nqb, qb = p.nqb - 1 - (t - ph * p.nqb);
  const int pair = ph / p.heads, head = ph - pair * p.heads;
  const int64_t seq0 = (int64_t)pair * p.L;
  const int i0 = qb * kBQ;
  const int64_t qcol = (int64_t)head * kDh, kcol = p.d + qcol, vcol = 2 * (int64_t)p.d + qcol;

  // this lane's query, the column operand of S^T: chunks 4h + s of its row
  const int iq = i0 + wave * 16 + lr;
  const bool qvalid = iq < p.L;
  bf16x8 qf[4];
  {
    const uint16_t* src = p.qkv + (seq0 + min(iq, p.L - 1)) * p.ldq + qcol;
#pragma unroll
    for (int s = 0; s < 4; ++s)
      qf[s] = as_bf16x8(*reinterpret_cast<const u32x4*>(src + (h * 4 + s) * 8));
  }

  f32x4 o[8];
#pragma unroll
  for (int df = 0; df < 8; ++df) o[df] = f32x4{0.f, 0.f, 0.f, 0.f};
  float m = -1e30f;  // running max of the scaled scores (base 2)
  float l = 0.f;     // this lane's part of the running row sum

  const int ilast = min(i0 + kBQ, p.L) - 1;  // last real query of the block
  const int kb_lo = max(0, i0 - p.W + 1) / kBK, kb_hi = ilast / kBK;
  uint2* sV2 = reinterpret_cast<uint2*>(sV);
  for (int kb = kb_lo; kb <= kb_hi; ++kb) {
    const int j0 = kb * kBK;
    __syncthreads();  // the previous block's reads are done
    // K: thread copies chunks tid + 256 k of the 64 x 128 tile (key = c / 16).
    // Keys past the sequence end (last block of a ragged sequence) repeat
    // its last row; causality masks them for every real query.
#pragma unroll
    for (int k = 0; k < 4; ++k) {
      const int c = k * 256 + tid, key = c >> 4, ch = c & 15;
      const int64_t row = seq0 + min(j0 + key, p.L - 1);
      sK[key * 16 + (ch ^ k_msk(key))] =
          *reinterpret_cast<const u32x4*>(p.qkv + row * p.ldq + kcol + ch * 8);
    }
    // V^T: thread takes keys 4a .. 4a+3 of dims 8 ch .. 8 ch+7 and writes,
    // per dim, the 4 keys' values as one 8-byte word (contiguous in vpos
    // order).  Odd chunks write their dims in the order e ^ 1 so that a
    // half-wave's 32 words fall in distinct banks.
    {
      const int a = tid & 15, ch = tid >> 4, odd = ch & 1;
      u32x4 w[4];
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int64_t row = seq0 + min(j0 + 4 * a + r, p.L - 1);
        w[r] = *reinterpret_cast<const u32x4*>(p.qkv + row * p.ldq + vcol + ch * 8);
      }
      uint2 val[8];
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        const uint32_t sel = (e & 1) ? 0x07060302u : 0x05040100u;
        val[e].x = __builtin_amdgcn_perm(w[1][e >> 1], w[0][e >> 1], sel);
        val[e].y = __builtin_amdgcn_perm(w[3][e >> 1], w[2][e >> 1], sel);
      }
      const int pk = vpos(4 * a), pc = pk >> 3, f = (pk >> 2) & 1;
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        const int dim = ch * 8 + (e ^ odd);
        sV2[(dim * 8 + (pc ^ v_msk(dim))) * 2 + f] = odd ? val[e ^ 1] : val[e];
      }
    }
    __syncthreads();

    // S^T, 4 fragments of 16 keys: lane holds keys j0 + 16 kf + 4 h + r of query iq
    f32x4 sc[4];
#pragma unroll
    for (int kf = 0; kf < 4; ++kf) {
      const int key = kf * 16 + lr;
      f32x4 c = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int s = 0; s < 4; ++s)
        c = mfma16x16x32(as_bf16x8(sK[key * 16 + ((h * 4 + s) ^ k_msk(key))]), qf[s], c);
      sc[kf] = c;
    }
    float bmax = -INFINITY;
#pragma unroll
    for (int kf = 0; kf < 4; ++kf)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int j = j0 + kf * 16 + h * 4 + r;
        const bool ok = j <= iq && iq - j < p.W;
        sc[kf][r] = ok ? sc[kf][r] * p.scale2 : -INFINITY;
        bmax = fmaxf(bmax, sc[kf][r]);
      }
    const float mn = fmaxf(m, max_over_h(bmax));
    const float alpha = exp2f(m - mn);
    m = mn;
    l *= alpha;
#pragma unroll
    for (int df = 0; df < 8; ++df) o[df] *= alpha;
    // P^T in bf16 as the column operand of the two 32-key steps: element
    // 4 f + r of step t is key 32 t + 16 f + 4 h + r
    bf16x8 pb[2];
#pragma unroll
    for (int t2 = 0; t2 < 2; ++t2) {
      u32x4 pw;
#pragma unroll
      for (int f = 0; f < 2; ++f)
#pragma unroll
        for (int r = 0; r < 4; r += 2) {
          const uint16_t b0 = f32_to_bf16(exp2f(sc[2 * t2 + f][r] - mn));
          const uint16_t b1 = f32_to_bf16(exp2f(sc[2 * t2 + f][r + 1] - mn));
          l += __uint_as_float((uint32_t)b0 << 16) + __uint_as_float((uint32_t)b1 << 16);
          pw[f * 2 + r / 2] = (uint32_t)b0 | ((uint32_t)b1 << 16);
        }
      pb[t2] = as_bf16x8(pw);
    }
#pragma unroll
    for (int df = 0; df < 8; ++df) {
      const int dim = df * 16 + lr;
#pragma unroll
      for (int t2 = 0; t2 < 2; ++t2)
        o[df] = mfma16x16x32(as_bf16x8(sV[dim * 8 + ((4 * t2 + h) ^ v_msk(dim))]), pb[t2], o[df]);
    }
  }

  // O^T: lane holds query iq (column lr), dims 16 df + 4 h + r
  const float inv = 1.0f / sum_over_h(l);
  if (!qvalid) return;
  uint16_t* dst = p.out + (seq0 + iq) * p.ldo + qcol;
#pragma unroll
  for (int df = 0; df < 8; ++df) {
    const uint32_t lo =
        (uint32_t)f32_to_bf16(o[df][0] * inv) | ((uint32_t)f32_to_bf16(o[df][1] * inv) << 16);
    const uint32_t hi =
        (uint32_t)f32_to_bf16(o[df][2] * inv) | ((uint32_t)f32_to_bf16(o[df][3] * inv) << 16);
    *reinterpret_cast<uint2*>(dst + df * 16 + h * 4) = make_uint2(lo, hi);
  }
}

}  // namespace

int64_t attention_tiles(int64_t M, int heads, int seq_len) {
  return (M / seq_len) * heads * ((seq_len + kBQ - 1) / kBQ);
}

hipError_t launch_attention(const uint16_t* qkv, int64_t ldq, uint16_t* out, int64_t ldo,
                            int64_t M, int d, int heads, int seq_len, int window, hipStream_t s) {
  AttnParams p;
  p.qkv = qkv;
  p.out = out;
  p.ldq = ldq;
  p.ldo = ldo;
  p.d = d;
  p.L = seq_len;
  p.W = window;
  p.heads = heads;
  p.nqb = (seq_len + kBQ - 1) / kBQ;
  p.tiles = (int)attention_tiles(M, heads, seq_len);
  p.scale2 = 1.4426950408889634f / sqrtf((float)kDh);
  hipLaunchKernelGGL(k_attn, dim3((unsigned)p.tiles), dim3(256), 0, s, p);
  return hipGetLastError();
}

}  // namespace ql
