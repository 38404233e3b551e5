// Causal sliding-window multi-head attention between the QKV and output
// projections (the paper's decoder uses sliding-window attention, Sec. 1
// contribution 1.1 and Sec. 2).  Each sequence of seq_len tokens (one
// protein-ligand pair) is independent; token i attends to the tokens j of its
// sequence with i - window < j <= i.  Head dimension 128.
//
// One workgroup (8 waves) owns 128 queries of one head; wave w owns 16 of
// them.  Key blocks of 64 are staged in LDS (K row-major, V transposed), the
// next block's loads in flight while the current one is computed.  The
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
constexpr int kBQ = 128;  // queries per workgroup (8 waves x 16)
constexpr int kThreads = 512;
constexpr int kBK = 64;   // keys per LDS block

struct AttnParams {
  const uint16_t* qkv;
  uint16_t* out;
  const int32_t* cu;  // ragged batch: sequence offsets [n_seqs + 1], else null
  int64_t ldq, ldo;
  int M, d, L, W, heads, nqb, tiles;  // L: the sequence length (uniform) or
                                      // the longest sequence (ragged)
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

// Reductions over the 4 lanes of a query (lanes lr, lr + 16, lr + 32,
// lr + 48).  v_permlane16_swap with both operands equal to v leaves, in each
// lane, its own value and that of the lane 16 away (one in each result);
// v_permlane32_swap does the same for the lane 32 away.
__device__ __forceinline__ float max_over_h(float v) {
  const auto a = __builtin_amdgcn_permlane16_swap(__float_as_uint(v), __float_as_uint(v), false, false);
  const float x = __uint_as_float(a[0]), y = __uint_as_float(a[1]);
  v = x > y ? x : y;
  const auto b = __builtin_amdgcn_permlane32_swap(__float_as_uint(v), __float_as_uint(v), false, false);
  const float z = __uint_as_float(b[0]), w = __uint_as_float(b[1]);
  return z > w ? z : w;
}
__device__ __forceinline__ float sum_over_h(float v) {
  const auto a = __builtin_amdgcn_permlane16_swap(__float_as_uint(v), __float_as_uint(v), false, false);
  v = __uint_as_float(a[0]) + __uint_as_float(a[1]);
  const auto b = __builtin_amdgcn_permlane32_swap(__float_as_uint(v), __float_as_uint(v), false, false);
  return __uint_as_float(b[0]) + __uint_as_float(b[1]);
}

typedef float f32x2 __attribute__((ext_vector_type(2)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
// two fp32 -> packed bf16 pair, round to nearest even (v_cvt_pk_bf16_f32)
__device__ __forceinline__ uint32_t pack_bf16x2(float a, float b) {
  return __builtin_bit_cast(uint32_t, __builtin_convertvector((f32x2{a, b}), bf16x2));
}

// The next key block's K and V, staged in registers while the current block
// is computed.  Thread t holds K chunks t and t + 512 of the 64 x 128 tile
// and V chunk (t >> 5) of keys 2 (t & 31) and 2 (t & 31) + 1.
struct Staged {
  u32x4 k[2];
  u32x4 v[2];
};

__device__ __forceinline__ void load_block(const AttnParams& p, int64_t seq0, int L, int j0,
                                           int tid, int64_t kcol, int64_t vcol, Staged& st) {
  // keys past the sequence end (last block of a ragged sequence) repeat its
  // last row; causality masks them for every real query
#pragma unroll
  for (int k = 0; k < 2; ++k) {
    const int c = k * kThreads + tid, key = c >> 4, ch = c & 15;
    const int64_t row = seq0 + min(j0 + key, L - 1);
    st.k[k] = *reinterpret_cast<const u32x4*>(p.qkv + row * p.ldq + kcol + ch * 8);
  }
  const int a2 = tid & 31, ch = tid >> 5;
#pragma unroll
  for (int r = 0; r < 2; ++r) {
    const int64_t row = seq0 + min(j0 + 2 * a2 + r, L - 1);
    st.v[r] = *reinterpret_cast<const u32x4*>(p.qkv + row * p.ldq + vcol + ch * 8);
  }
}

// K row-major (swizzled); V transposed: per dim, the two keys' values as one
// dword at their (adjacent) vpos positions.  Odd chunks write their dims in
// the order e ^ 1, so that a wave's 64 dwords fall in 64 distinct banks.
__device__ __forceinline__ void store_block(const Staged& st, int tid, u32x4* sK, uint32_t* sV1) {
#pragma unroll
  for (int k = 0; k < 2; ++k) {
    const int c = k * kThreads + tid, key = c >> 4, ch = c & 15;
    sK[key * 16 + (ch ^ k_msk(key))] = st.k[k];
  }
  const int a2 = tid & 31, ch = tid >> 5, odd = ch & 1;
  const int pk = vpos(2 * a2), pc = pk >> 3, q = (pk & 7) >> 1;
  // dim 8 ch + e' sits in half e' & 1 of dword e' >> 1 of both rows; with
  // e' = e ^ odd only the half (the byte selector) depends on the thread
  const uint32_t sel_lo = odd ? 0x07060302u : 0x05040100u;
  const uint32_t sel_hi = odd ? 0x05040100u : 0x07060302u;
#pragma unroll
  for (int e = 0; e < 8; ++e) {
    const int dim = ch * 8 + (e ^ odd);
    sV1[(dim * 8 + (pc ^ v_msk(dim))) * 4 + q] =
        __builtin_amdgcn_perm(st.v[1][e >> 1], st.v[0][e >> 1], (e & 1) ? sel_hi : sel_lo);
  }
}

__global__ __launch_bounds__(kThreads, 4) void k_attn(AttnParams p) {
  __shared__ u32x4 sK[kBK * 16];  // 16 KB
  __shared__ u32x4 sV[kDh * 8];   // 16 KB
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
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
  const int i0 = qb * kBQ;
  // the sequence's first row and length; ragged offsets are clamped into
  // [0, M] and the length to the launch's query blocks, so malformed offsets
  // give wrong results but no access outside the buffers
  int64_t seq0;
  int L;
  if (p.cu) {
    const int a = min(max(p.cu[pair], 0), p.M), b = min(max(p.cu[pair + 1], a), p.M);
    seq0 = a;
    L = min(b - a, p.nqb * kBQ);
  } else {
    seq0 = (int64_t)pair * p.L;
    L = p.L;
  }
  if (i0 >= L) return;  // the whole workgroup, before any barrier
  const int64_t qcol = (int64_t)head * kDh, kcol = p.d + qcol, vcol = 2 * (int64_t)p.d + qcol;

  // this wave's queries qw0 .. qw1 (wave-uniform); the lane's query iq is the
  // column operand of S^T: chunks 4h + s of its row
  const int qw0 = i0 + wave * 16, qw1 = min(qw0 + 15, L - 1);
  const int iq = qw0 + lr;
  bf16x8 qf[4];
  {
    const uint16_t* src = p.qkv + (seq0 + min(iq, L - 1)) * p.ldq + qcol;
#pragma unroll
    for (int s = 0; s < 4; ++s)
      qf[s] = as_bf16x8(*reinterpret_cast<const u32x4*>(src + (h * 4 + s) * 8));
  }

  f32x4 o[8];
#pragma unroll
  for (int df = 0; df < 8; ++df) o[df] = f32x4{0.f, 0.f, 0.f, 0.f};
  // m: the running reference of the scaled scores (base 2); it only moves up
  // when a block's max exceeds it by more than kLazy, so P = 2^(s - m) stays
  // below 2^kLazy and most blocks skip the rescale.  l: this lane's part of
  // the row sum.
  constexpr float kLazy = 8.0f;
  float m = -1e30f, l = 0.f;

  const int ilast = min(i0 + kBQ, L) - 1;  // last real query of the workgroup
  const int kb_lo = max(0, i0 - p.W + 1) / kBK, kb_hi = ilast / kBK;
  uint32_t* sV1 = reinterpret_cast<uint32_t*>(sV);
  Staged st;
  load_block(p, seq0, L, kb_lo * kBK, tid, kcol, vcol, st);
  for (int kb = kb_lo; kb <= kb_hi; ++kb) {
    const int j0 = kb * kBK;
    __syncthreads();  // the previous block's reads are done
    store_block(st, tid, sK, sV1);
    __syncthreads();
    if (kb < kb_hi) load_block(p, seq0, L, j0 + kBK, tid, kcol, vcol, st);

    // skip blocks no query of this wave can see (wave-uniform)
    if (qw0 >= L || j0 > qw1 || qw0 - (j0 + kBK - 1) >= p.W) continue;
    const bool full = j0 + kBK - 1 <= qw0 && qw1 - j0 < p.W;

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
    if (!full) {
      // key j = j0 + 16 kf + 4 h + r is visible iff 16 kf + r <= dq (causal)
      // and 16 kf + r > dq - W (window), dq = iq - j0 - 4 h
      const int dq = iq - j0 - 4 * h;
      if (qw1 - j0 < p.W) {  // the window cuts no key of this block for this wave
#pragma unroll
        for (int kf = 0; kf < 4; ++kf)
#pragma unroll
          for (int r = 0; r < 4; ++r)
            if (kf * 16 + r > dq) sc[kf][r] = -INFINITY;
      } else {
        const int dw = dq - p.W;
#pragma unroll
        for (int kf = 0; kf < 4; ++kf)
#pragma unroll
          for (int r = 0; r < 4; ++r)
            if (kf * 16 + r > dq || kf * 16 + r <= dw) sc[kf][r] = -INFINITY;
      }
    }
    float bmax = sc[0][0];
#pragma unroll
    for (int kf = 0; kf < 4; ++kf)
#pragma unroll
      for (int r = 0; r < 4; ++r) bmax = fmaxf(bmax, sc[kf][r]);
    bmax = max_over_h(bmax) * p.scale2;
    if (__builtin_amdgcn_ballot_w64(bmax > m + kLazy)) {
      const float mn = bmax > m + kLazy ? bmax : m;
      const float alpha = __builtin_amdgcn_exp2f(m - mn);
      m = mn;
      l *= alpha;
#pragma unroll
      for (int df = 0; df < 8; ++df) o[df] *= alpha;
    }
    // P^T in bf16 as the column operand of the two 32-key steps: element
    // 4 f + r of step t2 is key 32 t2 + 16 f + 4 h + r
    bf16x8 pb[2];
#pragma unroll
    for (int t2 = 0; t2 < 2; ++t2) {
      u32x4 pw;
#pragma unroll
      for (int f = 0; f < 2; ++f)
#pragma unroll
        for (int r = 0; r < 4; r += 2) {
          const float e0 = __builtin_amdgcn_exp2f(fmaf(sc[2 * t2 + f][r], p.scale2, -m));
          const float e1 = __builtin_amdgcn_exp2f(fmaf(sc[2 * t2 + f][r + 1], p.scale2, -m));
          const uint32_t w = pack_bf16x2(e0, e1);
          // the row sum adds the rounded values the product sees
          l += bf16_lo(w) + bf16_hi(w);
          pw[f * 2 + r / 2] = w;
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
  if (iq >= L) return;
  uint16_t* dst = p.out + (seq0 + iq) * p.ldo + qcol;
#pragma unroll
  for (int df = 0; df < 8; ++df)
    *reinterpret_cast<uint2*>(dst + df * 16 + h * 4) =
        make_uint2(pack_bf16x2(o[df][0] * inv, o[df][1] * inv),
                   pack_bf16x2(o[df][2] * inv, o[df][3] * inv));
}

}  // namespace

int64_t attention_tiles(int64_t n_seqs, int heads, int max_len) {
  return n_seqs * heads * ((max_len + kBQ - 1) / kBQ);
}

hipError_t launch_attention(const uint16_t* qkv, int64_t ldq, uint16_t* out, int64_t ldo,
                            int64_t M, int d, int heads, int seq_len, int window,
                            const int32_t* cu_seqlens, int n_seqs, hipStream_t s) {
  AttnParams p;
  p.qkv = qkv;
  p.out = out;
  p.cu = cu_seqlens;
  p.ldq = ldq;
  p.ldo = ldo;
  p.M = (int)M;
  p.d = d;
  p.L = seq_len;
  p.W = window;
  p.heads = heads;
  p.nqb = (seq_len + kBQ - 1) / kBQ;
  const int64_t seqs = cu_seqlens ? n_seqs : M / seq_len;
  p.tiles = (int)attention_tiles(seqs, heads, seq_len);
  p.scale2 = 1.4426950408889634f / sqrtf((float)kDh);
  hipLaunchKernelGGL(k_attn, dim3((unsigned)p.tiles), dim3(kThreads), 0, s, p);
  return hipGetLastError();
}

}  // namespace ql
