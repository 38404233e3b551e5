// Causal sliding-window multi-head attention between the QKV and output
// projections (the paper's decoder uses sliding-window attention, Sec. 1
// contribution 1.1 and Sec. 2).  Each sequence of seq_len tokens (one
// protein-ligand pair) is independent; token i attends to the tokens j of its
// sequence with i - window < j <= i.  Head dimension 128.
//
// One workgroup (8 waves) owns 128 queries of one head; wave w owns 16 of
// them.  (16 waves x 256 queries halve the key / value copies but measure
// slower: one workgroup per CU, and 16 waves meet at every barrier.)  Key
// blocks of 64 keys go global -> LDS by direct-to-LDS copies into a
// two-stage ring (K and V both row-major, swizzled), the next block's copies
// in flight while the current one is computed.  The scores are computed
// transposed, S^T = K Q^T (16x16x32 bf16 MFMAs with K as the row operand), so
// that a lane ends up holding, for its query, exactly the keys it feeds as
// the column operand of O^T += V^T P^T: nothing moves between the two
// products.  The V^T operand is read from the row-major V tile with the
// transposing LDS read (ds_read_b64_tr_b16).  Softmax is online in fp32 (base
// 2); P is rounded to bf16 for the second product and the row sums add the
// rounded values, so the weights the product sees sum to one; O stays fp32
// until the final bf16 store.
#include <algorithm>

#include "ql_device.h"
#include "ql_internal.h"

namespace ql {

namespace {

constexpr int kDh = 128;  // head dimension
constexpr int kWaves = 8;                // waves per workgroup, 16 queries each
constexpr int kThreads = kWaves * 64;
constexpr int kBQ = kWaves * 16;         // queries per workgroup
constexpr int kBK = 64;   // keys per LDS block
constexpr int kCopies = kBK * 16 / 64 / kWaves;  // 16-byte copies of K (and of V) per wave per block
static_assert(kCopies >= 1 && kCopies * kWaves * 64 == kBK * 16, "copies cover the tile");

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
// V tile: key r keeps its 16-byte chunk c (dims 8c .. 8c+7) at slot
// r * 16 + (c ^ v_swz(r)).  A transposing read covers 8 keys x 32 bytes per
// half-wave; the swizzle puts those 8 rows' 32-byte pieces in distinct banks.
__device__ __forceinline__ int v_swz(int r) { return (r & 7) << 1; }

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

// One 16-byte direct-to-LDS copy: lane l writes lds + 16 l.  Inline assembly
// so that the compiler does not track it (it would otherwise wait for the
// copy right after issuing it); the kernel waits with an explicit
// s_waitcnt.  M0 carries the LDS base and is saved and restored (the
// compiler reserves it); one wait state separates its write from the load.
__device__ __forceinline__ void copy16_to_lds(const void* src, const void* lds) {
  const uint32_t l = __builtin_amdgcn_readfirstlane((uint32_t)reinterpret_cast<uintptr_t>(lds));
  uint32_t saved;
  asm volatile(
      "s_mov_b32 %[sv], m0\n\t"
      "s_mov_b32 m0, %[l]\n\t"
      "s_nop 0\n\t"
      "global_load_lds_dwordx4 %[a], off\n\t"
      "s_mov_b32 m0, %[sv]"
      : [sv] "=&s"(saved)
      : [a] "v"(src), [l] "s"(l)
      : "memory");
}

// Copies of key block j0 into one stage: wave w issues copies i < kCopies of
// K and of V, copy i covering the 16-byte slots (kWaves i + w) * 64 + lane,
// i.e. keys 4 (kWaves i + w) .. +3.  src[i] is the lane's source for key block 0
// (sequence row key, its swizzled chunk of K; V follows at +d elements);
// whole blocks advance it by j0 rows.  In the last block of a ragged
// sequence, keys past its end repeat its last row; causality masks them for
// every real query.
__device__ __forceinline__ void issue_block(const AttnParams& p,
                                            const uint16_t* const (&src)[kCopies][2],
                                            int L, int j0, int wave, u32x4* sK, u32x4* sV) {
  const int64_t adv = (int64_t)j0 * p.ldq;
#pragma unroll
  for (int i = 0; i < kCopies; ++i) {
    const int key0 = (i * kWaves + wave) * 4;  // first key of the copy (wave-uniform)
    const uint16_t* ks = src[i][0] + adv;
    const uint16_t* vs = src[i][1] + adv;
    if (j0 + key0 + 3 >= L) {  // rare: the copy reaches past the sequence end
      const int key = key0 + ((int)(threadIdx.x & 63) >> 4);
      const int64_t back = (int64_t)(min(j0 + key, L - 1) - (j0 + key)) * p.ldq;
      ks += back;
      vs += back;
    }
    copy16_to_lds(ks, sK + (i * kWaves + wave) * 64);
    copy16_to_lds(vs, sV + (i * kWaves + wave) * 64);
  }
}

typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) bf16x4 lds_bf16x4;

// V^T operand of one 32-key step for dims 16 df .. 16 df + 15: lane (lr, h)
// gets V[32 t2 + 16 f + 4 h + j][16 df + lr] as element 4 f + j.  In a
// transposing read, lane i = 4a + b of a 16-lane group receives element b of
// the 8-byte pieces addressed by lanes a, a + 4, a + 8, a + 12; so lane
// (lr, h) addresses key 32 t2 + 16 f + 4 h + lr / 4, dims 16 df + 4 (lr % 4)
// .. + 3.  With the V swizzle that is byte
//   (32 t2 + 16 f) * 256 + vt_lane(df, h, lr)
// of the stage: the (t2, f) part is a constant offset of the read.
__device__ __forceinline__ uint32_t vt_lane(int df, int h, int lr) {
  const int key = 4 * h + (lr >> 2);  // (mod 8 the same for every t2, f)
  const int chunk = 2 * df + ((lr >> 1) & 1);
  return (uint32_t)(key * 256 + ((chunk ^ v_swz(key)) << 4) + ((lr & 1) << 3));
}
template <int T2>
__device__ __forceinline__ bf16x8 load_vt(uint32_t addr) {
  const bf16x4 a = __builtin_amdgcn_ds_read_tr16_b64_v4bf16(
      reinterpret_cast<lds_bf16x4*>((uintptr_t)(addr + T2 * 32 * 256)));
  const bf16x4 b = __builtin_amdgcn_ds_read_tr16_b64_v4bf16(
      reinterpret_cast<lds_bf16x4*>((uintptr_t)(addr + T2 * 32 * 256 + 16 * 256)));
  return bf16x8{a[0], a[1], a[2], a[3], b[0], b[1], b[2], b[3]};
}

__global__ __launch_bounds__(kThreads, 4) void k_attn(AttnParams p) {
  __shared__ u32x4 sK[2][kBK * 16];  // two stages of 16 KB
  __shared__ u32x4 sV[2][kBK * 16];
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
  const uint16_t* src[kCopies][2];
#pragma unroll
  for (int i = 0; i < kCopies; ++i) {
    const int slot = (i * kWaves + wave) * 64 + lane, key = slot >> 4, ps = slot & 15;
    const uint16_t* row = p.qkv + (seq0 + key) * p.ldq;
    src[i][0] = row + kcol + (ps ^ k_msk(key)) * 8;
    src[i][1] = row + vcol + (ps ^ v_swz(key)) * 8;
  }
  uint32_t vt_addr[8];  // LDS byte address of this lane's V^T reads in stage 0, per df
#pragma unroll
  for (int df = 0; df < 8; ++df)
    vt_addr[df] = (uint32_t)reinterpret_cast<uintptr_t>(sV[0]) + vt_lane(df, h, lr);
  issue_block(p, src, L, kb_lo * kBK, wave, sK[kb_lo & 1], sV[kb_lo & 1]);
  for (int kb = kb_lo; kb <= kb_hi; ++kb) {
    const int j0 = kb * kBK;
    const u32x4* cK = sK[kb & 1];
    const uint32_t vstage = (kb & 1) * (uint32_t)sizeof(sV[0]);  // byte offset of the stage
    // this wave's copies of block kb have landed (they are its only vector
    // memory operations in flight); after the barrier every wave's copies
    // are visible and every read of the other stage (block kb - 1) is done
    __builtin_amdgcn_s_waitcnt(0);
    __syncthreads();
    if (kb < kb_hi)
      issue_block(p, src, L, j0 + kBK, wave, sK[(kb + 1) & 1], sV[(kb + 1) & 1]);

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
        c = mfma16x16x32(as_bf16x8(cK[key * 16 + ((h * 4 + s) ^ k_msk(key))]), qf[s], c);
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
      o[df] = mfma16x16x32(load_vt<0>(vt_addr[df] + vstage), pb[0], o[df]);
      o[df] = mfma16x16x32(load_vt<1>(vt_addr[df] + vstage), pb[1], o[df]);
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
