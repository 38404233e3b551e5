// Small-batch (M <= 16) int4-weight projection: weight bytes bound the run.
//
// Each workgroup (W = 4 waves, or 8 when it is the only one on its CU) owns
// 16 F output columns (F = 3, 4 or 6 column fragments of 16, chosen per N by
// gemv_fragments) over the full K.  Wave w takes the pairs of scale groups
// (2u, 2u+1), u = w, w+W, w+2W, ..., and loads a pair's codes back to back,
// so that each wave reads whole 128-byte lines of its weight rows (with a
// line's halves spread over two waves the same reads stream about 10 %
// slower).  Per group, each lane issues one 16-byte load per 16-column
// fragment (the lane's 32 codes): 16 rows x 64 bytes from row-major codes,
// or, from the tiled layout, one contiguous kilobyte (a pair's two loads
// then read 2 KB in one run, 6-13 % faster).  The group's activations
// (M rows x 256 bytes) come in ceil(M/4) contiguous loads of 4 rows each and
// reach the MFMA operand layout through a wave-private LDS tile, which costs
// far less than four 16-row loads in that layout.  With pair tiles (F = 6, and F = 3 where
// the LDS allows) each wave keeps two tiles and the next pair's activation
// loads fly while a pair is computed; loaded just before use, their L2 round
// trip stalled the wave once per group.  Inside the main loop every load is
// unconditional: the codes of two pairs stay in flight in registers, and
// the compiler's counted waits let them fly while a pair is computed.  The
// wave's last two or three pairs run after the loop and request nothing
// past its last pair, so that no wave waits for loads it never uses before
// the partial sums are exchanged (that wait was 1-2 % of the kernel).
//
// The codes are unpacked to bf16 136 + q and run through a 16x16x32 MFMA
// chain against the (at most 16) activation rows; the rows' group sums come
// from one more MFMA chain against a constant -136 operand, which starts
// each chain so that it yields the exact code dot product.  The workgroup's
// scales (16 F columns x G, one contiguous block of the scale matrix) are
// copied into LDS once at the start (with pair tiles by direct-to-LDS loads
// issued ahead of the first code loads): per-group scale loads would cost as
// many memory instructions as the codes themselves.  The partial sums of the
// W waves are then reduced through LDS (the wavefront reduction) and the
// epilogue is applied.
#include <algorithm>

#include "ql_device.h"
#include "ql_internal.h"

namespace ql {

namespace {

constexpr int kWaves = 4;   // waves per workgroup unless it is alone on its CU
// LDS ahead of the scales: the waves' activation tiles, later the partial
// sums.  F: 16-column fragments per wave; PT (pair tiles): each wave keeps
// two activation tiles (a pair of groups), otherwise one; W: waves.
template <int F, bool PT, int W = kWaves>
constexpr int tile_bytes() {
  return W * 256 * 16 * (PT ? 2 : 1) > (W - 1) * F * 64 * 16 ? W * 256 * 16 * (PT ? 2 : 1)
                                                             : (W - 1) * F * 64 * 16;
}
template <int F, bool PT, int W = kWaves>
size_t lds_bytes(int64_t K) {
  return (size_t)tile_bytes<F, PT, W>() + (size_t)16 * F * (K / kGroup) * 2;
}

struct GemvParams {
  const uint16_t* x;
  const uint8_t* qw;
  const uint16_t* sc;
  void* out;
  int64_t ldx, ldo;
  int64_t qgs;  // bytes from one group's codes to the next: 64 (row-major) or 1024 (tiled)
  int M, N, K, G;
};

// Activation tile of one group in LDS: 16 rows x 16 chunks of 16 bytes, row r
// storing chunk c at slot c ^ x_msk(r) so that the 16-row MFMA operand reads
// are free of bank conflicts.  Chunks are stored already in the codes' k
// order (permute_chunk when written: ceil(M/4) permutes per group and lane
// instead of four when read).
__device__ __forceinline__ int x_msk(int row) {
  row &= 15;
  return row ^ ((((row >> 2) ^ (row >> 3)) & 1) << 2);
}

// codes of a pair of consecutive groups (2 x F column fragments)
template <int F>
struct PairCodes {
  u32x4 b[2][F];
};
// With pair tiles the workgroup's codes are read through one buffer
// resource over the contiguous byte range they occupy (its columns' rows,
// or its 16-column blocks), with that range's length as the record count:
// a lane's address is then a 32-bit offset (half the registers of a
// pointer, which the widest variants need to stay free of spills), and a
// load of a group past the end (the second group of an odd G's last pair,
// or a pair the set-up requests for a wave that has fewer) takes an offset
// beyond that length, for which the hardware's range check returns zeros
// without a memory access.  A range is at most 16 F x K / 2 bytes, a few
// MB, far below kPastEnd.
constexpr int kPastEnd = 0x40000000;
// word 3 of a raw buffer resource: 32-bit data format, no swizzle
constexpr int kRawBufferWord3 = 0x00020000;

struct CodeSrc {
  __amdgpu_buffer_rsrc_t rs;
  const uint8_t* base;  // first byte of the range
  int qgs;              // bytes from one group's codes to the next
  int G;
};

// 16 bytes at lane offset voff of group g: through the resource (BUF: zeros
// past the last group), or as a plain load with g clamped to the last group
// (the single-tile widths, which run three workgroups per CU: there the
// resource's registers pushed the loop into spills)
template <bool BUF>
__device__ __forceinline__ u32x4 load_code(const CodeSrc& c, uint32_t voff, int g) {
  if constexpr (BUF) {
    const int goff = g < c.G ? g * c.qgs : kPastEnd;
    return __builtin_bit_cast(
        u32x4, __builtin_amdgcn_raw_buffer_load_b128(c.rs, (int)voff + goff, 0, 0));
  } else {
    return *reinterpret_cast<const u32x4*>(c.base + voff + (uint32_t)(min(g, c.G - 1) * c.qgs));
  }
}

// The pair's code loads back to back: the wave reads both 64-byte halves of
// each 128-byte line of its 16 weight rows per fragment one right after the
// other.
template <bool BUF, int F>
__device__ __forceinline__ void load_codes(const CodeSrc& c, const uint32_t (&voff)[F], int g,
                                           PairCodes<F>& d) {
#pragma unroll
  for (int j = 0; j < F; ++j)
#pragma unroll
    for (int e = 0; e < 2; ++e) d.b[e][j] = load_code<BUF>(c, voff[j], g + e);
}

// the codes of one group (F column fragments)
template <bool BUF, int F>
__device__ __forceinline__ void load_group(const CodeSrc& c, const uint32_t (&voff)[F], int g,
                                           u32x4 (&d)[F]) {
#pragma unroll
  for (int j = 0; j < F; ++j) d[j] = load_code<BUF>(c, voff[j], g);
}

// One group: its activations (rows 4q + lane/16, chunk lane%16; L2 hits,
// loaded here, their latency covered by the other waves of the CU) go
// through the wave's LDS tile into the operand layout (rows past M hold stale
// values; they only reach output rows that are never stored).
template <int F>
__device__ __forceinline__ void compute_tile(const u32x4 (&b)[F], const u32x4* xt,
                                             const uint16_t* sS, int G, int g, int h, int lr,
                                             f32x4 (&acc)[F]);

template <int XQ, int F>
__device__ __forceinline__ void compute_group(const u32x4 (&b)[F],
                                              const uint16_t* const (&xsrc)[XQ], u32x4* xt,
                                              const int (&xdst)[XQ], const uint16_t* sS, int G,
                                              int g, int h, int lr, f32x4 (&acc)[F]) {
  u32x4 xa[XQ];
#pragma unroll
  for (int q = 0; q < XQ; ++q) xa[q] = *reinterpret_cast<const u32x4*>(xsrc[q] + (int64_t)g * kGroup);
#pragma unroll
  for (int q = 0; q < XQ; ++q) xt[xdst[q]] = permute_chunk(xa[q]);
  compute_tile<F>(b, xt, sS, G, g, h, lr, acc);
}

// A group whose activations are already in the wave's LDS tile xt.
template <int F>
__device__ __forceinline__ void compute_tile(const u32x4 (&b)[F], const u32x4* xt,
                                             const uint16_t* sS, int G, int g, int h, int lr,
                                             f32x4 (&acc)[F]) {
  const bf16x8 neg = neg136x8();
  bf16x8 a[4];
#pragma unroll
  for (int s = 0; s < 4; ++s)
    a[s] = as_bf16x8(xt[lr * 16 + ((h * 4 + s) ^ x_msk(lr))]);
  f32x4 nc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
  for (int s = 0; s < 4; ++s) nc = mfma16x16x32(a[s], neg, nc);
  f32x4 c[F];
#pragma unroll
  for (int j = 0; j < F; ++j) c[j] = nc;
#pragma unroll
  for (int s = 0; s < 4; ++s) {
#pragma unroll
    for (int j = 0; j < F; ++j) {
      const uint32_t wv = s == 0 ? b[j].x : s == 1 ? b[j].y : s == 2 ? b[j].z : b[j].w;
      c[j] = mfma16x16x32(a[s], unpack_offset_codes(wv), c[j]);
    }
  }
#pragma unroll
  for (int j = 0; j < F; ++j) acc[j] += c[j] * f16_to_f32(sS[(j * 16 + lr) * G + g]);
}

// Copy `count` binary16 values from src to LDS dst with all of a thread's
// loads of a batch in flight together (16-byte loads when src is 16-byte
// aligned, which also makes dst's 16-byte slots line up).
template <int W>
__device__ __forceinline__ void copy_scales(const uint16_t* src, uint16_t* dst, int count) {
  const int t = threadIdx.x, nt = W * 64;
  int done = 0;
  if (((uintptr_t)src & 15u) == 0) {
    const int nv = count / 8;
    const u32x4* s = reinterpret_cast<const u32x4*>(src);
    u32x4* d = reinterpret_cast<u32x4*>(dst);
    for (int v0 = 0; v0 < nv; v0 += 4 * nt) {
      u32x4 r[4];
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        const int v = v0 + u * nt + t;
        if (v < nv) r[u] = s[v];
      }
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        const int v = v0 + u * nt + t;
        if (v < nv) d[v] = r[u];
      }
    }
    done = nv * 8;
  }
  for (int i0 = done; i0 < count; i0 += 8 * nt) {
    uint16_t r[8];
#pragma unroll
    for (int u = 0; u < 8; ++u) {
      const int i = i0 + u * nt + t;
      if (i < count) r[u] = src[i];
    }
#pragma unroll
    for (int u = 0; u < 8; ++u) {
      const int i = i0 + u * nt + t;
      if (i < count) dst[i] = r[u];
    }
  }
}

// Workgroups per CU the launch bounds provide for: 12 / F of 4 waves (2 for
// F = 6), but 3 for F = 3 (no shape that picks F = 3 has more per CU; the
// registers then hold the pair tiles' prefetched activations), and 1 of 8.
template <int F, int W>
constexpr int gemv_wgs_per_cu() {
  return W != kWaves ? 1 : F == 3 ? 3 : 12 / F;
}

// EARLY (pair tiles on tiled codes): each group's codes are reloaded for
// the pair after next as soon as that group is computed, instead of both
// after the pair; with row-major codes that splits the two 64-byte halves of
// each 128-byte line apart (10 % slower), with tiled codes every load is a
// whole kilobyte and the earlier requests gain 1-2 %.
template <int EPI, int XQ, int F, bool PT, int W, bool EARLY>
__global__ __launch_bounds__(W * 64, (gemv_wgs_per_cu<F, W>())) void k_gemv(GemvParams p) {
  constexpr int kCols = 16 * F;
  // [W][256 or 512] activation tiles (after the loop: [W-1][F][64] partial
  // sums), then the scales [kCols][G]
  extern __shared__ __align__(16) unsigned char smem[];
  u32x4* xtiles = reinterpret_cast<u32x4*>(smem);
  f32x4* red = reinterpret_cast<f32x4*>(smem);
  uint16_t* sS = reinterpret_cast<uint16_t*>(smem + tile_bytes<F, PT, W>());
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6), lane = threadIdx.x & 63;
  const int h = lane >> 4, lr = lane & 15;
  const int64_t n0 = (int64_t)blockIdx.x * kCols;
  const int G = p.G;

  // rows past M and columns past N read valid (clamped) memory; their
  // results are never stored (nor are the columns whose scales the
  // workgroup's copy leaves unset)
  const bool rows = p.qgs == kGroup / 2;
  const int64_t lo = rows ? n0 * (p.K / 2) : n0 / 16 * G * 1024;
  const int64_t hi = rows ? std::min<int64_t>(n0 + kCols, p.N) * (p.K / 2)
                          : std::min<int64_t>(n0 / 16 + F, p.N / 16) * G * 1024;
  CodeSrc cs;
  cs.rs = __builtin_amdgcn_make_buffer_rsrc(const_cast<uint8_t*>(p.qw + lo), (short)0,
                                            (int)(hi - lo), kRawBufferWord3);
  cs.base = p.qw + lo;
  cs.qgs = (int)p.qgs;
  cs.G = G;
  uint32_t voff[F];
#pragma unroll
  for (int j = 0; j < F; ++j) {
    if (rows) {
      // row-major: the lane's 16 bytes of its column's group
      const int64_t col = std::min<int64_t>(n0 + j * 16 + lr, p.N - 1);
      voff[j] = (uint32_t)((col - n0) * (p.K / 2) + h * 16);
    } else {
      // tiled: the fragment's 16 columns x 64 bytes of a group are one
      // contiguous kilobyte, lane l at 16 l
      const int64_t blk = std::min<int64_t>(n0 / 16 + j, p.N / 16 - 1);
      voff[j] = (uint32_t)((blk - n0 / 16) * G * 1024 + lane * 16);
    }
  }
  const uint16_t* xsrc[XQ];
  int xdst[XQ];
#pragma unroll
  for (int q = 0; q < XQ; ++q) {
    const int row = q * 4 + (lane >> 4), ch = lane & 15;
    xsrc[q] = p.x + (int64_t)min(row, p.M - 1) * p.ldx + ch * 8;
    xdst[q] = row * 16 + (ch ^ x_msk(row));
  }
  u32x4* xt = xtiles + wave * 256 * (PT ? 2 : 1);

  f32x4 acc[F];
#pragma unroll
  for (int j = 0; j < F; ++j) acc[j] = f32x4{0.f, 0.f, 0.f, 0.f};

  // this wave's groups: pairs of consecutive groups (2u, 2u+1) for u = wave,
  // wave + W, ...; the code loads of the next two pairs are in flight while a
  // pair is computed
  const int U = (G + 1) / 2;
  const int TU = U > wave ? (U - wave + W - 1) / W : 0;
  const auto first = [&](int t) { return 2 * (wave + W * t); };
  // the workgroup's scale block goes to LDS by direct-to-LDS copies issued
  // before the code loads, so that waiting for it (below) leaves the codes
  // in flight (copied through registers after them, waiting for the scales
  // had meant waiting for the first two pairs' codes too: 0.5-1.8 us); a
  // block that is not 16-byte aligned, and the single-tile widths (whose
  // registers are tighter), take the register copy
  const int cols = (int)std::min<int64_t>(kCols, p.N - n0);
  const uint16_t* ssrc = p.sc + n0 * G;
  const bool dma = PT && ((uintptr_t)ssrc & 15u) == 0 && (cols * G) % 8 == 0;
  if (dma) {
    const int nv = cols * G / 8;
    for (int v0 = wave * 64; v0 < nv; v0 += W * 64)
      if (v0 + lane < nv)
        copy16_to_lds(ssrc, (uint32_t)(v0 + lane) * 16,
                      (uint32_t)reinterpret_cast<uintptr_t>(sS + v0 * 8));
  }
  PairCodes<F> cb[2];
  load_codes<PT>(cs, voff, first(0), cb[0]);
  load_codes<PT>(cs, voff, first(1), cb[1]);
  // pair tiles: the first pair's activations are requested before the scale
  // copy, so that their round trip overlaps it
  u32x4 xa[2][XQ];
  const auto load_acts = [&](int g) {
#pragma unroll
    for (int e = 0; e < 2; ++e)
#pragma unroll
      for (int q = 0; q < XQ; ++q)
        xa[e][q] = *reinterpret_cast<const u32x4*>(xsrc[q] + (int64_t)min(g + e, G - 1) * kGroup);
  };
  if constexpr (PT) load_acts(first(0));
  if (dma) {
    // the copies have landed once at most the loads issued after them are
    // outstanding
    __builtin_amdgcn_s_waitcnt(vmcnt_lgkm0(4 * F + (PT ? 2 * XQ : 0)));
    wg_barrier();
  } else {
    copy_scales<W>(ssrc, sS, cols * G);
    __syncthreads();
  }

  // Pair t from code buffer c.  acts: request the next pair's activations;
  // reload: request pair t + 2 into c.  The loop runs while both pairs of
  // an iteration have both successors, with the flags constant; the last
  // two or three pairs follow with the flags taken per pair.
  const auto step = [&](int t, PairCodes<F>& c, bool acts, bool reload) {
    const int g = first(t);
    if constexpr (PT) {
#pragma unroll
      for (int e = 0; e < 2; ++e)
#pragma unroll
        for (int q = 0; q < XQ; ++q) xt[e * 256 + xdst[q]] = permute_chunk(xa[e][q]);
      if (acts) load_acts(first(t + 1));
      compute_tile<F>(c.b[0], xt, sS, G, g, h, lr, acc);
      if constexpr (EARLY) {
        if (reload) load_group<PT>(cs, voff, first(t + 2), c.b[0]);
        if (g + 1 < G) compute_tile<F>(c.b[1], xt + 256, sS, G, g + 1, h, lr, acc);
        if (reload) load_group<PT>(cs, voff, first(t + 2) + 1, c.b[1]);
      } else {
        if (g + 1 < G) compute_tile<F>(c.b[1], xt + 256, sS, G, g + 1, h, lr, acc);
        if (reload) load_codes<PT>(cs, voff, first(t + 2), c);
      }
    } else {
      compute_group<XQ, F>(c.b[0], xsrc, xt, xdst, sS, G, g, h, lr, acc);
      if (g + 1 < G) compute_group<XQ, F>(c.b[1], xsrc, xt, xdst, sS, G, g + 1, h, lr, acc);
      if (reload) load_codes<PT>(cs, voff, first(t + 2), c);
    }
  };
  int t0 = 0;
  for (; t0 + 3 < TU; t0 += 2) {
    step(t0, cb[0], true, true);
    step(t0 + 1, cb[1], true, true);
  }
  if (t0 < TU) step(t0, cb[0], t0 + 1 < TU, t0 + 2 < TU);
  if (t0 + 1 < TU) step(t0 + 1, cb[1], t0 + 2 < TU, false);
  if (t0 + 2 < TU) step(t0 + 2, cb[0], false, false);

  // the partial sums reuse the activation tiles' LDS
  __syncthreads();
  if (wave > 0) {
#pragma unroll
    for (int j = 0; j < F; ++j) red[((wave - 1) * F + j) * 64 + lane] = acc[j];
  }
  __syncthreads();
  if (wave != 0) return;
#pragma unroll
  for (int w = 0; w < W - 1; ++w)
#pragma unroll
    for (int j = 0; j < F; ++j) acc[j] += red[(w * F + j) * 64 + lane];
  if constexpr (EPI == 2) {
    // residual update: all old values loaded before the first store (see the
    // MFMA kernel's epilogue)
    float old[F][4];
#pragma unroll
    for (int j = 0; j < F; ++j)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int64_t col = n0 + j * 16 + lr;
        const int row = h * 4 + r;
        old[j][r] = col < p.N && row < p.M ? reinterpret_cast<const float*>(p.out)[row * p.ldo + col]
                                           : 0.f;
      }
#pragma unroll
    for (int j = 0; j < F; ++j)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int64_t col = n0 + j * 16 + lr;
        const int row = h * 4 + r;
        if (col < p.N && row < p.M)
          reinterpret_cast<float*>(p.out)[row * p.ldo + col] = old[j][r] + acc[j][r];
      }
    return;
  }
#pragma unroll
  for (int j = 0; j < F; ++j) {
    const int64_t col = n0 + j * 16 + lr;
    if (col >= p.N) continue;
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const int row = h * 4 + r;
      if (row >= p.M) continue;
      const float v = acc[j][r];
      if constexpr (EPI == 1) {
        reinterpret_cast<uint16_t*>(p.out)[row * p.ldo + col] = f32_to_bf16(gelu_erf(v));
      } else {
        reinterpret_cast<uint16_t*>(p.out)[row * p.ldo + col] = f32_to_bf16(v);
      }
    }
  }
}

}  // namespace

// The 16-column fragments per wave fall back to 4 with single tiles (the
// smallest LDS need of the shapes that balance: 64 columns per workgroup,
// three per CU).
size_t gemv_lds_bytes(int64_t K) { return lds_bytes<4, false>(K); }

// Fragments per wave for N columns.  Every workgroup re-reads the whole
// activation block, so wide workgroups save load instructions, while the
// workgroups must spread evenly over the 256 CUs: with F fragments (16 F
// columns per workgroup, up to 12 / F workgroups resident per CU) the
// busiest CU runs ceil(workgroups / 256) * F fragment-columns.  The
// smallest such load wins, ties going to the wider workgroup; the scale
// block must fit the LDS bound.  N = 49152: 6 (512 workgroups, 2 per CU);
// N = 36864: 3 (768, 3 per CU); N = 12288: 3 (256, 1 per CU).
int gemv_fragments(int64_t N, int64_t K) {
  constexpr int64_t kCUs = 256;
  int best = 4;
  int64_t best_load = -1;
  for (const int F : {6, 4, 3}) {
    const size_t lds = F == 6 ? lds_bytes<6, true>(K)
                       : F == 4 ? lds_bytes<4, false>(K) : lds_bytes<3, false>(K);
    if (lds > kGemvMaxLds) continue;
    const int64_t wgs = (N + 16 * F - 1) / (16 * F);
    const int64_t load = (wgs + kCUs - 1) / kCUs * F;
    if (best_load < 0 || load < best_load) {
      best = F;
      best_load = load;
    }
  }
  return best;
}

hipError_t launch_gemv(const uint16_t* x, int64_t ldx, const uint8_t* qw, const uint16_t* sc,
                       void* out, int64_t ldo, int64_t M, int64_t N, int64_t K, int epilogue,
                       bool tiled, hipStream_t s) {
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
  p.qgs = tiled ? 1024 : kGroup / 2;
  const int F = gemv_fragments(N, K);
  // pair tiles for F = 6 (within the LDS bound by the choice above) and
  // F = 3 when two workgroups still fit a CU's LDS; F = 4 keeps single tiles
  // (its three workgroups per CU leave no registers for the prefetch)
  const bool pt = F == 6 || (F == 3 && lds_bytes<3, true>(K) <= 80 * 1024);
  // one workgroup per CU (F = 3, at most 256 workgroups): eight waves split
  // its groups, so twice the code bytes are in flight per CU
  const bool w8 = F == 3 && pt && (N + 47) / 48 <= 256 && lds_bytes<3, true, 8>(K) <= 160 * 1024;
  const int xq = (int)((M + 3) / 4);   // contiguous 4-row activation loads per group
#define QL_GEMV(E, Q, FF, PP, WW, EE)                                                         \
  hipLaunchKernelGGL((k_gemv<E, Q, FF, PP, WW, EE>),                                          \
                     dim3((unsigned)((N + 16 * FF - 1) / (16 * FF))), dim3(WW * 64),          \
                     (lds_bytes<FF, PP, WW>(K)), s, p)
#define QL_GEMV_PT(E, Q, FF, WW)                        \
  if (tiled) QL_GEMV(E, Q, FF, true, WW, true);         \
  else QL_GEMV(E, Q, FF, true, WW, false);
#define QL_GEMV_F(E, Q)                                 \
  if (F == 6) { QL_GEMV_PT(E, Q, 6, 4) }                \
  else if (F == 3 && w8) { QL_GEMV_PT(E, Q, 3, 8) }     \
  else if (F == 3 && pt) { QL_GEMV_PT(E, Q, 3, 4) }     \
  else if (F == 3) QL_GEMV(E, Q, 3, false, 4, false);   \
  else QL_GEMV(E, Q, 4, false, 4, false);
#define QL_GEMV_Q(E)                     \
  switch (xq) {                          \
    case 1: QL_GEMV_F(E, 1); break;      \
    case 2: QL_GEMV_F(E, 2); break;      \
    case 3: QL_GEMV_F(E, 3); break;      \
    default: QL_GEMV_F(E, 4); break;     \
  }
  switch (epilogue) {
    case 1: QL_GEMV_Q(1); break;
    case 2: QL_GEMV_Q(2); break;
    default: QL_GEMV_Q(0); break;
  }
#undef QL_GEMV_Q
#undef QL_GEMV_F
#undef QL_GEMV_PT
#undef QL_GEMV
  return hipGetLastError();
}

}  // namespace ql
