// Large-M int4-weight projection on bf16 MFMA (gfx950).
//
// out[m][n] = sum_g s[n][g] * sum_{k in g} x[m][k] * q[n][k]
//
// Each workgroup (8 waves, two per SIMD) owns a 128 x 256 output tile; the
// waves form a 2 x 4 grid, so each owns a 64 x 64 slice.  The K loop walks
// one 128-wide scale group per step:
//   * the activation tile (128 rows x 128 k, bf16), the packed weight tile
//     (256 columns x 64 bytes; from row-major codes 16 rows x 64 bytes per
//     copy instruction, from the tiled layout one contiguous kilobyte), the
//     group's 256 scales and 128 correction terms are copied global -> LDS
//     with direct-to-LDS loads into a
//     three-stage ring: while group g is computed, the copies of groups g+1
//     and g+2 are in flight, so each copy has about two steps to land;
//   * a step runs four 32-k phases; in each, a wave reads its activation
//     fragments from LDS, unpacks one 32-bit word of codes per column
//     fragment into bf16 values 136 + q (exact; see unpack_offset_codes) and
//     issues one 16x16x32 MFMA for each of its 4 x 4 output fragments (in
//     the prepared form two consecutive words share their three shifts,
//     done as 64-bit shifts: between MFMAs a 64-bit shift issues at the cost
//     of a 32-bit one);
//   * each fragment's chain of four MFMAs starts from the correction
//     -136 * sum_k x[m][k], so its result is the integer-code dot product
//     sum x*q (fp32), and one fp32 FMA applies the group's scale:
//     acc += chain * s[n][g].
// Scales therefore stay exact fp32 (no bf16 rounding of q*s).
//
// Two operand forms.  Prepared (RAW = false): the activations arrive
// k-permuted in 8-element chunks with their corrections alongside (written
// by launch_prep or by the producing kernel's epilogue).  Raw (RAW = true):
// the activations are read as stored, the codes are unpacked in natural k
// order, and each wave derives the corrections of the 16 rows it copies
// itself -- one more 4-MFMA chain per group against a constant -136
// operand, run on the next group's rows before the step barrier, so the
// call needs no staging buffer at all.
#include <algorithm>

#include <type_traits>

#include "ql_device.h"
#include "ql_internal.h"

namespace ql {

namespace {

constexpr int NW = 8;                  // waves per workgroup
constexpr int BN = 256;                // columns per workgroup tile
constexpr int B_SLOTS = BN * 4;        // 16-byte slots of codes per stage (16 KB)
constexpr int B_PER_WAVE = B_SLOTS / 64 / NW;   // 2 direct-to-LDS loads per wave
static_assert(BN == kGemmBN, "tile width");

// Row extent of a workgroup tile: IF 16-row fragments per wave.  128 rows
// for large M; 64 or 32 for M <= 64, where taller tiles would spend most of
// their MFMA work on padding rows.
template <int IF>
struct TileM {
  static constexpr int BM = 16 * IF;
  static_assert(kGemmBM % BM == 0, "correction rows are padded to kGemmBM");
  static constexpr int A_SLOTS = BM * 16;             // 16-byte slots per stage
  static constexpr int A_PER_WAVE = A_SLOTS / 64 / NW;
  static constexpr int N_SLOTS = BM < 64 ? 64 : BM;   // correction terms (+ clamped copies)
  // Activation and code copies each wave issues per group, after its
  // correction / scale copy if it has one (see issue_copy); once the next
  // group's copies are all issued, waiting until at most this many are
  // outstanding means every copy of the group before has landed.
  static constexpr int kLaterCopies = A_PER_WAVE + B_PER_WAVE;
  static constexpr int kWaitPrevGroup = vmcnt_lgkm0(kLaterCopies);
};

struct GemmParams {
  const uint16_t* xp;  // prepared operand (row stride K), or raw x (row stride ldx)
  const float* ns;     // corrections of the prepared operand (unused when raw)
  const uint8_t* qw;
  const uint16_t* sc;
  void* out;  // may be null when only the prepared copy is wanted
  int64_t ldo, Mp, ldx;
  int64_t qgs;  // bytes from one group's codes to the next: 64 (row-major) or 1024 (tiled)
  int M, N, K, G;
  int tiles_m, tiles_n;
  // prepared copy of output columns >= pcol0 (see GemmPrep)
  uint16_t* pout;
  float* pns;
  int64_t pld;
  int pcol0;
  // 1: the scales are copied eight groups at a time (16 bytes per column;
  // needs G % 8 == 0 and a 16-byte aligned sc)
  int sbatch;
};

template <int CTRL>
__device__ __forceinline__ float dpp_f32(float v) {
  return __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(0, __builtin_bit_cast(int, v), CTRL,
                                                               0xF, 0xF, false));
}

// position of element e of an 8-element chunk in the MFMA operand order
// (x0,x4,x1,x5,x2,x6,x3,x7)
__device__ __forceinline__ int perm8(int e) { return 2 * (e & 3) + (e >> 2); }

// LDS layouts.  gfx950 serves a 16-byte-per-lane LDS read in four cycles; one
// cycle takes the 4-lane quads of a half-wave whose quad index (lane bits
// 2-4) has a given parity, so a pattern is conflict-free when each such set
// of 16 lanes covers all 16 slots of a 256-byte bank row.
//
// Activation tile: 1 KB blocks of 4 rows (64 16-byte slots; one copy fills
// one block from 4 whole 256-byte row segments).  Inside a block, phase s
// (16 slots) comes first, then row r % 4 (4 slots), then the k-quarter h
// (16-byte chunk 4h + s of the row's group), swizzled by bit 3 of the row.
// A fragment read (16 rows, one phase) by lane (h, lr) then differs between
// phases and row fragments only by a constant, and each 16-lane set -- rows
// r % 4 = 0..3 twice, once with bit 3 clear and once set, and two values of
// h -- covers all 16 slots.
__device__ __forceinline__ int a_swz(int row) { return ((row >> 3) & 1) << 1; }
__device__ __forceinline__ int a_slot(int row, int s, int h) {
  return (row >> 2) * 64 + s * 16 + (row & 3) * 4 + (h ^ a_swz(row));
}
// Code tile: column n stores its 16-byte piece h at slot 4n + (h ^ b_swz(n)).
__device__ __forceinline__ int b_swz(int col) { return ((col >> 1) ^ (col >> 2)) & 3; }

// The copies (copy_to_lds, copy16_to_lds: direct-to-LDS loads the compiler
// does not track) are waited for explicitly: kWaitPrevGroup before the step
// barrier, vmcnt(0) before the epilogue; the kernel issues no other vector
// memory load in its loop.  Tracked copies would not do: the compiler's own
// wait insertion cannot tell the three ring stages apart and would wait for
// the copies just issued before every LDS read.

// Anchors the computation of v at this point of the program: an empty
// volatile statement that reads v.  The compiler otherwise moves pure
// arithmetic (the scale FMAs, the code unpacking) across the scheduling
// barriers towards its first use, which bunches it up between steps.
template <class T>
__device__ __forceinline__ void pin(const T& v) {
  static_assert(sizeof(T) == 16 || sizeof(T) == 4, "pinned value size");
  if constexpr (sizeof(T) == 16) {
    const u32x4 u = __builtin_bit_cast(u32x4, v);
    asm volatile("" ::"v"(u));
  } else {
    asm volatile("" ::"v"(__builtin_bit_cast(uint32_t, v)));
  }
}

struct Stage {
  u32x4* A;     // activation tile, A_SLOTS 16-byte slots
  u32x4* B;     // code tile, B_SLOTS 16-byte slots
  float* N;     // BM correction terms
  uint32_t* S;  // BN scales, one zero-extended binary16 per dword
};

template <int IF>
struct Offsets {
  uint32_t a[TileM<IF>::A_PER_WAVE];  // byte offsets into xp of this lane's A slots (group 0)
  uint32_t b[B_PER_WAVE];             // byte offsets into qw of this lane's B slots (group 0)
};

// 64-slot block (4 rows of the activation tile) that copy j of a wave fills:
// interleaved over the waves for the prepared form; for the raw form wave w
// fills rows 16w .. 16w + 15, the row fragment whose corrections it derives.
template <int IF, bool RAW>
__device__ __forceinline__ int a_block(int j, int wave) {
  return RAW ? wave * TileM<IF>::A_PER_WAVE + j : j * NW + wave;
}

// The copies of group g into stage st, as seen by one wave.
template <int IF>
struct CopyJob {
  const GemmParams& p;
  const Offsets<IF>& o;
  int64_t m0;
  int g;
  int64_t n0;
  Stage st;
  uint16_t* sb;  // the two eight-group scale buffers ([2][BN][8])
  int wave, lane;
};

// Copy J of a wave's NCOPY copies of a group (J is a compile-time index).
// J = 0: prepared form, waves 0-1 copy the BM correction terms (rows past BM
// repeat the last one); both forms, waves 2-5 copy the 256 scales.  J = 1 ..
// A_PER_WAVE: the wave's activation copies; the last two: its code copies.
template <int IF>
constexpr int kCopies = TileM<IF>::A_PER_WAVE + B_PER_WAVE + 1;

__device__ __forceinline__ uint32_t scale_copy_offset(const GemmParams& p, int64_t n0, int wave,
                                                      int lane) {
  // 32-bit: a launch chunk keeps every byte offset below 2^31
  return (uint32_t)min((int)n0 + ((wave - 2) & 3) * 64 + lane, p.N - 1) * (uint32_t)p.G;
}
// The lane id from a volatile statement: the scale copy offset derived from it
// where the copy is issued cannot be hoisted out of the loop or kept live
// across steps (a register held through the loop for it had been spilled,
// and its reload waited for every copy in flight).
__device__ __forceinline__ int lane_id_here() {
  uint32_t l;
  asm volatile("v_mbcnt_lo_u32_b32 %0, -1, 0\n\tv_mbcnt_hi_u32_b32 %0, -1, %0" : "=v"(l));
  return (int)l;
}

template <int IF, bool RAW, int J>
__device__ __forceinline__ void issue_copy(const CopyJob<IF>& c) {
  constexpr int BM = TileM<IF>::BM, NA = TileM<IF>::A_PER_WAVE;
  static_assert(B_PER_WAVE == 2 && J < kCopies<IF>, "copy index");
  const int wave = c.wave;
  if constexpr (J == 0) {
    if (!RAW && wave * 64 < BM)
      copy_to_lds<4>(c.p.ns + (size_t)c.g * c.p.Mp + c.m0,
                     (uint32_t)min(wave * 64 + c.lane, BM - 1) * 4, c.st.N + wave * 64);
    else if (wave >= 2 && wave < 6) {
      if (c.p.sbatch) {
        // groups g .. g + 7 of 64 columns, 16 bytes per column, into the
        // buffer of batch g / 8 (read from step g on; the buffer's previous
        // batch was last read eight steps earlier)
        if ((c.g & 7) == 0)
          copy16_to_lds(c.p.sc + c.g, scale_copy_offset(c.p, c.n0, wave, lane_id_here()) * 2,
                        (uint32_t)reinterpret_cast<uintptr_t>(
                            c.sb + ((c.g >> 3) & 1) * (BN * 8) + (wave - 2) * 64 * 8));
      } else {
        copy_to_lds<2>(c.p.sc + c.g, scale_copy_offset(c.p, c.n0, wave, lane_id_here()) * 2,
                       c.st.S + (wave - 2) * 64);
      }
    }
  } else if constexpr (J <= NA) {
    const char* xa = reinterpret_cast<const char*>(c.p.xp) + (size_t)c.g * (kGroup * 2);
    copy16_to_lds(xa, c.o.a[J - 1],
                  (uint32_t)reinterpret_cast<uintptr_t>(c.st.A + a_block<IF, RAW>(J - 1, wave) * 64));
  } else {
    const char* qb = reinterpret_cast<const char*>(c.p.qw) + (size_t)c.g * c.p.qgs;
    copy16_to_lds(qb, c.o.b[J - NA - 1],
                  (uint32_t)reinterpret_cast<uintptr_t>(c.st.B + ((J - NA - 1) * NW + wave) * 64));
  }
}

template <int J, int N, class F>
__device__ __forceinline__ void static_for(const F& f) {
  if constexpr (J < N) {
    f(std::integral_constant<int, J>{});
    static_for<J + 1, N>(f);
  }
}

// all copies of a group at once (the two groups before the loop)
template <int IF, bool RAW>
__device__ __forceinline__ void issue_stage(const CopyJob<IF>& c) {
  static_for<0, kCopies<IF>>([&](auto J) { issue_copy<IF, RAW, decltype(J)::value>(c); });
}

// In the loop, copy J is issued after MFMA slot J * 2 NC / NCOPY of the first
// two phases (NC MFMAs per phase), not in one burst: a burst of 56 16-byte
// copies per workgroup at the top of every step fills the address unit's
// queue, and the waves stall on it in front of their MFMAs.
template <int IF, bool RAW>
__device__ __forceinline__ void issue_copies_at(const CopyJob<IF>& c, int slot) {
  constexpr int NC = (IF / 2) * 4;
  static_for<0, kCopies<IF>>([&](auto J) {
    constexpr int j = decltype(J)::value;
    if (slot == j * 2 * NC / kCopies<IF>) issue_copy<IF, RAW, j>(c);
  });
}

// Wave layout: the 8 waves form a 2 x 4 grid over the 128 x 256 tile; wave
// (wr, wc) owns rows wr * BM / 2 .. + BM / 2 (RF = IF / 2 row fragments of 16)
// and columns 64 wc .. 64 wc + 63 (CF = 4 column fragments of 16).  Compared
// with waves of 128 x 32, each MFMA needs 41 % fewer LDS bytes (the
// activation tile is read by 4 waves instead of 8), which is what bounds the
// loop: every group step reads the stage from LDS at 128 bytes per clock.
constexpr int WC = 4;            // wave columns
constexpr int CF = 4;            // 16-column fragments per wave
static_assert(WC * CF * 16 == BN && NW % WC == 0, "wave grid");

// Epilogue.  EPI 0: bf16 store, 1: GELU then bf16, 2: fp32 residual add.
// With PREP (EPI 0 or 1) the bf16 values of columns >= pcol0 are also written
// as the next projection's operand: k-permuted in 8-element chunks, plus the
// correction ns[g][m] = -136 * (sum of the group's 128 bf16 values of row m),
// whose per-wave row sums meet in LDS (part, [WC][BM]) and are added in a
// fixed order.
template <int EPI, bool PREP, int IF>
__device__ __forceinline__ void store_tile(const GemmParams& p, int64_t m0, int64_t n0, int wave,
                                           int lane, const f32x4 (&acc)[IF / 2][CF],
                                           float* part) {
  constexpr int BM = TileM<IF>::BM, RF = IF / 2;
  if constexpr (PREP) {
    // a tile left of the prepared columns (the Q and K thirds of a QKV
    // projection) is stored plainly, without the row sums and their exchange
    if (n0 + BN <= p.pcol0) {
      store_tile<EPI, false, IF>(p, m0, n0, wave, lane, acc, part);
      return;
    }
  }
  const int h = lane >> 4, lr = lane & 15, wr = wave / WC, wc = wave % WC;
  if constexpr (EPI == 2) {
    // residual update: every old value is loaded before the first store, so
    // the loads fly together (one load after each store would wait for the
    // store, as the compiler cannot rule out that they alias)
    float old[RF][CF][4];
#pragma unroll
    for (int i = 0; i < RF; ++i)
#pragma unroll
      for (int j = 0; j < CF; ++j) {
        const int64_t col = n0 + wc * (CF * 16) + j * 16 + lr;
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const int64_t row = m0 + wr * (BM / 2) + i * 16 + h * 4 + r;
          old[i][j][r] = col < p.N && row < p.M
                             ? reinterpret_cast<const float*>(p.out)[row * p.ldo + col]
                             : 0.f;
        }
      }
#pragma unroll
    for (int i = 0; i < RF; ++i)
#pragma unroll
      for (int j = 0; j < CF; ++j) {
        const int64_t col = n0 + wc * (CF * 16) + j * 16 + lr;
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const int64_t row = m0 + wr * (BM / 2) + i * 16 + h * 4 + r;
          if (col < p.N && row < p.M)
            reinterpret_cast<float*>(p.out)[row * p.ldo + col] = old[i][j][r] + acc[i][j][r];
        }
      }
    return;
  }
  float rs[RF][4];
#pragma unroll
  for (int i = 0; i < RF; ++i)
#pragma unroll
    for (int r = 0; r < 4; ++r) rs[i][r] = 0.f;
#pragma unroll
  for (int i = 0; i < RF; ++i) {
#pragma unroll
    for (int j = 0; j < CF; ++j) {
      const int64_t col = n0 + wc * (CF * 16) + j * 16 + lr;
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int64_t row = m0 + wr * (BM / 2) + i * 16 + h * 4 + r;
        const bool in = col < p.N && row < p.M;
        const float v = acc[i][j][r];
        {
          const uint16_t b = f32_to_bf16(EPI == 1 ? gelu_erf(v) : v);
          if (in && p.out) reinterpret_cast<uint16_t*>(p.out)[row * p.ldo + col] = b;
          if constexpr (PREP) {
            const int64_t c = col - p.pcol0;
            if (in && c >= 0) p.pout[row * p.pld + (c & ~7) + perm8((int)(c & 7))] = b;
            rs[i][r] += __uint_as_float((uint32_t)b << 16);
          }
        }
      }
    }
  }
  if constexpr (PREP) {
    static_assert(EPI != 2, "prepared copy of a residual update");
    // this wave's 64 columns lie in 128-column group wc / 2 of the tile
#pragma unroll
    for (int i = 0; i < RF; ++i)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        // sum over the 16 lanes of a DPP row: quad swaps, then rotations by 4
        // and 8 within the row
        float t = rs[i][r];
        t += dpp_f32<0xB1>(t);    // quad_perm [1,0,3,2]
        t += dpp_f32<0x4E>(t);    // quad_perm [2,3,0,1]
        t += dpp_f32<0x124>(t);   // row_ror:4
        t += dpp_f32<0x128>(t);   // row_ror:8
        if (lr == 0) part[wc * BM + wr * (BM / 2) + i * 16 + h * 4 + r] = t;
      }
    __syncthreads();
    // thread t: group t / BM of the tile, row t % BM
    const int t = threadIdx.x;
    if (t < 2 * BM) {
      const int gg = t / BM, m = t % BM;
      const int64_t c = n0 + gg * kGroup - p.pcol0;
      if (c >= 0 && n0 + gg * kGroup < p.N) {
        const float sum = part[(2 * gg) * BM + m] + part[(2 * gg + 1) * BM + m];
        p.pns[(c / kGroup) * p.Mp + m0 + m] = -136.0f * sum;
      }
    }
  }
}

// Residual update through LDS: each half of the tile (the rows of one wave
// row) goes into a row-major buffer T (row stride BN + 4 words: conflict-free
// writes from the MFMA output layout), then every wave updates whole rows
// of 256 fp32 values, one 16-byte piece per lane, so the read-modify-write
// of the residual runs in 1 KB rows instead of 64-byte pieces of 4 rows.
// Needs out 16-byte aligned and ldo % 4 == 0; T is the (then idle)
// activation ring.
template <int IF>
__device__ __forceinline__ void store_resid_staged(const GemmParams& p, int64_t m0, int64_t n0,
                                                   int wave, int lane,
                                                   const f32x4 (&acc)[IF / 2][CF], float* T) {
  constexpr int BM = TileM<IF>::BM, RF = IF / 2, HR = BM / 2, LD = BN + 4, RW = HR / NW;
  const int h = lane >> 4, lr = lane & 15, wr = wave / WC, wc = wave % WC;
  float* out = reinterpret_cast<float*>(p.out);
  const int64_t col = n0 + 4 * lane;
  const bool full = col + 3 < p.N;
#pragma unroll
  for (int hf = 0; hf < 2; ++hf) {
    __syncthreads();  // the ring (first half) or the previous half is no longer read
    if (wr == hf) {
#pragma unroll
      for (int i = 0; i < RF; ++i)
#pragma unroll
        for (int j = 0; j < CF; ++j)
#pragma unroll
          for (int r = 0; r < 4; ++r)
            T[(i * 16 + h * 4 + r) * LD + wc * (CF * 16) + j * 16 + lr] = acc[i][j][r];
    }
    __syncthreads();
    f32x4 old[RW];
#pragma unroll
    for (int q = 0; q < RW; ++q) {
      const int64_t row = m0 + hf * HR + wave + q * NW;
      old[q] = f32x4{0.f, 0.f, 0.f, 0.f};
      if (row < p.M) {
        const float* o = out + row * p.ldo + col;
        if (full) {
          old[q] = *reinterpret_cast<const f32x4*>(o);
        } else {
#pragma unroll
          for (int e = 0; e < 4; ++e)
            if (col + e < p.N) old[q][e] = o[e];
        }
      }
    }
#pragma unroll
    for (int q = 0; q < RW; ++q) {
      const int rr = wave + q * NW;
      const int64_t row = m0 + hf * HR + rr;
      if (row >= p.M) continue;
      const f32x4 v = old[q] + *reinterpret_cast<const f32x4*>(T + rr * LD + 4 * lane);
      float* o = out + row * p.ldo + col;
      if (full) {
        *reinterpret_cast<f32x4*>(o) = v;
      } else {
#pragma unroll
        for (int e = 0; e < 4; ++e)
          if (col + e < p.N) o[e] = v[e];
      }
    }
  }
}

// activations of phase s for the wave's row fragments
template <int IF>
__device__ __forceinline__ void read_a(const Stage& st, int wr, int s, int h, int lr,
                                       bf16x8 (&a)[IF / 2]) {
  constexpr int BM = TileM<IF>::BM;
#pragma unroll
  for (int i = 0; i < IF / 2; ++i) {
    const int row = wr * (BM / 2) + i * 16 + lr;
    a[i] = as_bf16x8(st.A[a_slot(row, s, h)]);
  }
}

// the group's codes for the wave's column fragments (16 bytes = 32 codes of
// column lr per fragment: word s of it feeds phase s)
__device__ __forceinline__ void read_codes(const Stage& st, int wc, int h, int lr,
                                           u32x4 (&raw)[CF]) {
#pragma unroll
  for (int j = 0; j < CF; ++j) {
    const int col = wc * (CF * 16) + j * 16 + lr;
    raw[j] = st.B[col * 4 + (h ^ b_swz(col))];
  }
}

template <bool RAW>
__device__ __forceinline__ bf16x8 unpack_word(uint32_t w) {
  if constexpr (RAW)
    return unpack_offset_codes_natural(w);
  else
    return unpack_offset_codes(w);
}

// 8 codes from a word and its copies shifted right by 4, 8 and 12 bits
// (the mask / XOR of unpack_offset_codes)
__device__ __forceinline__ bf16x8 codes_from_shifts(uint32_t w0, uint32_t w4, uint32_t w8,
                                                    uint32_t w12) {
  u32x4 d;
  d.x = (w0 & 0x000f000fu) ^ 0x43084308u;
  d.y = (w4 & 0x000f000fu) ^ 0x43084308u;
  d.z = (w8 & 0x000f000fu) ^ 0x43084308u;
  d.w = (w12 & 0x000f000fu) ^ 0x43084308u;
  return __builtin_bit_cast(bf16x8, d);
}

template <int S>
__device__ __forceinline__ uint32_t word(const u32x4& v) {
  if constexpr (S == 0) return v.x;
  else if constexpr (S == 1) return v.y;
  else if constexpr (S == 2) return v.z;
  else return v.w;
}

// corrections (chain starts) and scales of a group for the wave's fragments
// chain starts (the groups' correction terms) of the wave's row fragments
template <int IF>
__device__ __forceinline__ void read_chain_starts(const Stage& st, int wr, int h,
                                                  f32x4 (&n4)[IF / 2]) {
  constexpr int BM = TileM<IF>::BM;
#pragma unroll
  for (int i = 0; i < IF / 2; ++i)
    n4[i] = *reinterpret_cast<const f32x4*>(st.N + wr * (BM / 2) + i * 16 + h * 4);
}

// binary16 scales of group g for the wave's column fragments, kept as bits
// (converted where they are used, so that no instruction waits on the read)
__device__ __forceinline__ void read_scales(const Stage& st, const uint16_t* sb, int g,
                                            bool sbatch, int wc, int lr, uint32_t (&sc)[CF]) {
  if (sbatch) {
    const uint16_t* b = sb + ((g >> 3) & 1) * (BN * 8) + (g & 7);
#pragma unroll
    for (int j = 0; j < CF; ++j) sc[j] = b[(wc * (CF * 16) + j * 16 + lr) * 8];
  } else {
#pragma unroll
    for (int j = 0; j < CF; ++j) sc[j] = st.S[wc * (CF * 16) + j * 16 + lr];
  }
}

// Raw form: corrections -136 * sum_k x[m][k] of the group in stage st for
// the 16 rows of row fragment `wave` (copied by this wave), as a chain of
// four MFMAs against a constant -136 operand (every column of the result
// holds the row's sum).
__device__ __forceinline__ f32x4 row_corrections(const Stage& st, int wave, int h, int lr) {
  const int row = wave * 16 + lr;
  bf16x8 x[4];
#pragma unroll
  for (int s = 0; s < 4; ++s) x[s] = as_bf16x8(st.A[a_slot(row, s, h)]);
  // all four reads in flight before the chain starts
  __builtin_amdgcn_sched_barrier(0);
  const bf16x8 neg = neg136x8();
  f32x4 c = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
  for (int s = 0; s < 4; ++s) c = mfma16x16x32(x[s], neg, c);
  return c;
}

// lanes of column 0 hold rows 4h .. 4h + 3 of the fragment
__device__ __forceinline__ void store_corrections(const Stage& st, int wave, int h, int lr,
                                                  const f32x4& c) {
  if (lr == 0) *reinterpret_cast<f32x4*>(st.N + wave * 16 + h * 4) = c;
}

// State a wave carries from one group step to the next.
template <int IF>
struct Carry {
  static constexpr int RF = IF / 2, NC = RF * CF, HALF = NC / 2;
  f32x4 acc[RF][CF];   // scaled sums
  f32x4 c[RF][CF];     // chains of the current group
  bf16x8 a[RF];        // activations of the next phase
  bf16x8 b[CF];        // unpacked codes of the next phase
  u32x4 raw[CF];       // codes of the current group
  f32x4 n4[RF];        // chain starts of the current group
  uint32_t sc[CF];     // binary16 scales of the current group, one per column fragment
  uint32_t sprev[CF];  // those of the previous group (its second-half chains)
  uint32_t sh[CF][3];  // next odd code word shifted right by 4, 8, 12 (prepared form)
};

// One 32-k phase S of group step g (see compute_step).
// PS: consecutive code words share their shifts (64-bit shifts; see
// codes_from_shifts), at the cost of three registers per column fragment
// held from one phase to the next
template <int IF, bool RAW, int S, bool PS>
__device__ __forceinline__ void compute_phase(const Stage& cur, const Stage& nxt,
                                              const CopyJob<IF>& cj, int g, int wave, int lane,
                                              Carry<IF>& C) {
  constexpr int RF = Carry<IF>::RF, NC = Carry<IF>::NC, HALF = Carry<IF>::HALF;
  const int h = lane >> 4, lr = lane & 15, wr = wave / WC, wc = wave % WC;
  bf16x8 an[RF], nb[CF];
  u32x4 rawn[CF];
  if constexpr (S < 3) {
    read_a<IF>(cur, wr, S + 1, h, lr, an);
  } else {
    __builtin_amdgcn_s_waitcnt(TileM<IF>::kWaitPrevGroup);
    if constexpr (RAW) {
      // chain starts of this wave's rows of group g + 1 (its own copies,
      // landed), stored before the barrier
      store_corrections(nxt, wave, h, lr, row_corrections(nxt, wave, h, lr));
      __builtin_amdgcn_s_waitcnt(TileM<IF>::kWaitPrevGroup);
    }
    wg_barrier();
    // the codes (unpacked from the fourth MFMA on) and the chain starts (the
    // next step's first MFMAs) before the activations (its second phase)
    read_codes(nxt, wc, h, lr, rawn);
    read_chain_starts<IF>(nxt, wr, h, C.n4);
    read_a<IF>(nxt, wr, 0, h, lr, an);
  }
  if constexpr (S == 0) read_scales(cur, cj.sb, g, cj.p.sbatch != 0, wc, lr, C.sc);
  __builtin_amdgcn_sched_barrier(0);
  // The phase's MFMAs one by one, each followed by its share of the VALU
  // work and a scheduling barrier, so that every wave interleaves its MFMAs
  // and VALU evenly: the other wave on the SIMD then finds the matrix core
  // or the VALU free, instead of both waves contending for the same one.
  //   * phase 0: before chain k's first MFMA (k >= HALF), the deferred
  //     scale FMA of the previous group's chain k;
  //   * phase 3: after the MFMA of chain k >= HALF, the scale FMA of chain
  //     k - HALF (its last MFMA issued HALF MFMAs earlier);
  //   * every NC / CF MFMAs: one code word of the next phase unpacked.
  constexpr int PER_WORD = NC / CF;
#pragma unroll
  for (int k = 0; k < NC; ++k) {
    const int i = k / CF, j = k % CF;
    if (S == 0 && k >= HALF) {
      C.acc[i][j] += C.c[i][j] * f16_to_f32((uint16_t)C.sprev[j]);
      pin(C.acc[i][j]);
    }
    C.c[i][j] = mfma16x16x32(C.a[i], C.b[j], S == 0 ? C.n4[i] : C.c[i][j]);
    if (S == 3 && k >= HALF) {
      const int i2 = (k - HALF) / CF, j2 = (k - HALF) % CF;
      C.acc[i2][j2] += C.c[i2][j2] * f16_to_f32((uint16_t)C.sc[j2]);
      pin(C.acc[i2][j2]);
    }
    if (k % PER_WORD == PER_WORD - 1) {
      const int jw = k / PER_WORD;
      // code word of the next phase (the next group's first word in phase 3)
      if constexpr (RAW || !PS) {
        nb[jw] = unpack_word<RAW>(word<(S + 1) & 3>(S < 3 ? C.raw[jw] : rawn[jw]));
      } else if constexpr (S == 1 || S == 3) {
        // even word now, and the shifted copies of the odd word after it
        // (the next phase's) from the same three 64-bit shifts
        const u32x4& src = S < 3 ? C.raw[jw] : rawn[jw];
        const uint64_t q = ((uint64_t)(S == 1 ? src.w : src.y) << 32) | (S == 1 ? src.z : src.x);
        uint64_t q4, q8, q12;
        asm volatile("v_lshrrev_b64 %0, 4, %1" : "=v"(q4) : "v"(q));
        asm volatile("v_lshrrev_b64 %0, 8, %1" : "=v"(q8) : "v"(q));
        asm volatile("v_lshrrev_b64 %0, 12, %1" : "=v"(q12) : "v"(q));
        nb[jw] = codes_from_shifts((uint32_t)q, (uint32_t)q4, (uint32_t)q8, (uint32_t)q12);
        C.sh[jw][0] = (uint32_t)(q4 >> 32);
        C.sh[jw][1] = (uint32_t)(q8 >> 32);
        C.sh[jw][2] = (uint32_t)(q12 >> 32);
      } else {
        nb[jw] = codes_from_shifts(S == 0 ? C.raw[jw].y : C.raw[jw].w, C.sh[jw][0], C.sh[jw][1],
                                   C.sh[jw][2]);
      }
      pin(nb[jw]);
    }
    if constexpr (S < 2) issue_copies_at<IF, RAW>(cj, S * NC + k);
    __builtin_amdgcn_sched_barrier(0);
  }
  if constexpr (S == 3) {
#pragma unroll
    for (int j = 0; j < CF; ++j) C.sprev[j] = C.sc[j];
#pragma unroll
    for (int j = 0; j < CF; ++j) C.raw[j] = rawn[j];
  }
#pragma unroll
  for (int j = 0; j < CF; ++j) C.b[j] = nb[j];
#pragma unroll
  for (int i = 0; i < RF; ++i) C.a[i] = an[i];
  __builtin_amdgcn_sched_barrier(0);
}

// One group step g from stage `cur`, in four 32-k phases.  Each phase runs
// the 4 MFMAs of all RF x CF chains for one 32-k slice, reads the next
// phase's activations from LDS at its top, and unpacks the next phase's code
// words after its MFMAs, so unpacking is spread evenly over the step.  Chain
// k's scale FMA (acc += chain * s) follows its last MFMA: for the first half
// of the chains in phase 3, for the second half in phase 0 of the next step,
// just before the chain is restarted.
//
// Before phase 3 every read of `cur` has been issued, so the wave waits for
// its copies of group g + 1 and joins the step barrier; phase 3 then reads
// group g + 1's first-phase activations and codes from `nxt` (its chain
// starts and scales are read at the top of the next step).  The copies of
// group g + 2 go into the third stage during the first two phases of the
// step, so every copy has about two steps to land.
// Raw form: before the barrier each wave derives the chain starts of its 16
// rows of group g + 1 (its own copies) and stores them.
template <int IF, bool RAW, bool PS>
__device__ __forceinline__ void compute_step(const GemmParams& p, const Offsets<IF>& o,
                                             int64_t m0, int64_t n0, int g, const Stage& cur,
                                             const Stage& nxt, const Stage& fut, uint16_t* sb,
                                             int wave, int lane, Carry<IF>& C) {
  const CopyJob<IF> cj{p, o, m0, min(g + 2, p.G - 1), n0, fut, sb, wave, lane};
  compute_phase<IF, RAW, 0, PS>(cur, nxt, cj, g, wave, lane, C);
  compute_phase<IF, RAW, 1, PS>(cur, nxt, cj, g, wave, lane, C);
  compute_phase<IF, RAW, 2, PS>(cur, nxt, cj, g, wave, lane, C);
  compute_phase<IF, RAW, 3, PS>(cur, nxt, cj, g, wave, lane, C);
}

template <int EPI, bool PREP, int IF, bool RAW>
__global__ __launch_bounds__(NW * 64, 1) void k_gemm(GemmParams p) {
  static_assert(!RAW || (IF == 8 && !PREP), "raw form: 128-row tiles, plain epilogues");
  using TM = TileM<IF>;
  constexpr int BM = TM::BM, RF = IF / 2;
  // the prepared form shares the unpacking's shifts between code words,
  // except with the plain GELU epilogue, whose loop then had no registers
  // left for it (spilled values reloaded inside the loop, each reload
  // waiting for every copy in flight)
  constexpr bool PS = !RAW && !(EPI == 1 && !PREP);
  // each kind of tile of the three stages contiguous, so that one address
  // register with constant offsets reaches the same slot in every stage
  __shared__ u32x4 sA[3][TM::A_SLOTS];
  __shared__ u32x4 sB[3][B_SLOTS];
  __shared__ float sN[3][TM::N_SLOTS];
  __shared__ uint32_t sS[3][BN];
  const Stage S0{sA[0], sB[0], sN[0], sS[0]}, S1{sA[1], sB[1], sN[1], sS[1]},
      S2{sA[2], sB[2], sN[2], sS[2]};
  __shared__ __attribute__((aligned(16))) uint16_t sSB[2 * BN * 8];

  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int lane = threadIdx.x & 63, lr = lane & 15, h = lane >> 4;
  const int wr = wave / WC, wc = wave % WC;

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

  // per-lane source offsets of the direct-to-LDS copies (rows and columns
  // past the matrix edge are clamped: they load valid memory and their
  // results are never stored)
  Offsets<IF> o;
#pragma unroll
  for (int j = 0; j < TM::A_PER_WAVE; ++j) {
    // lane l fills slot l of block a_block: phase l / 16, row l / 4 % 4 of
    // the block, swizzled k-quarter l % 4
    const int row = a_block<IF, RAW>(j, wave) * 4 + ((lane >> 2) & 3);
    const int chunk = ((lane & 3) ^ a_swz(row)) * 4 + (lane >> 4);
    const int64_t r = min<int64_t>(m0 + row, p.M - 1);
    o.a[j] = (uint32_t)((r * (RAW ? p.ldx : (int64_t)p.K) + chunk * 8) * 2);
  }
#pragma unroll
  for (int j = 0; j < B_PER_WAVE; ++j) {
    const int slot = (j * NW + wave) * 64 + lane;
    const int col = slot >> 2;
    const int hh = (slot & 3) ^ b_swz(col);
    const int64_t c = min<int64_t>(n0 + col, p.N - 1);
    // row-major: column c's 64 bytes of a group at c K/2; tiled: piece hh of
    // column c at 16 (64 (c/16) G + 16 hh + c%16) (one contiguous kilobyte
    // per 16 columns and group, so a copy reads 1 KB in one piece)
    o.b[j] = p.qgs == kGroup / 2 ? (uint32_t)(c * (p.K / 2) + hh * 16)
                                 : (uint32_t)(((c >> 4) * p.G * 64 + hh * 16 + (c & 15)) * 16);
  }
  // element index (group 0) of the scale column this lane copies (waves 2-5)

  Carry<IF> C;
#pragma unroll
  for (int i = 0; i < RF; ++i)
#pragma unroll
    for (int j = 0; j < CF; ++j) {
      C.acc[i][j] = f32x4{0.f, 0.f, 0.f, 0.f};
      C.c[i][j] = f32x4{0.f, 0.f, 0.f, 0.f};  // the first step's deferred FMAs add 0 * 0
    }
#pragma unroll
  for (int j = 0; j < CF; ++j) C.sprev[j] = 0;

  // group g lives in stage g % 3; step g issues group g + 2 (clamped to the
  // last group, so every step issues the same copies; the surplus ones land
  // in a stage that is not read again)
  const int G = p.G;
  issue_stage<IF, RAW>(CopyJob<IF>{p, o, m0, 0, n0, S0, sSB, wave, lane});
  issue_stage<IF, RAW>(CopyJob<IF>{p, o, m0, min(1, G - 1), n0, S1, sSB, wave, lane});
  __builtin_amdgcn_s_waitcnt(TM::kWaitPrevGroup);
  if constexpr (RAW) {
    store_corrections(S0, wave, h, lr, row_corrections(S0, wave, h, lr));
    __builtin_amdgcn_s_waitcnt(TM::kWaitPrevGroup);
  }
  wg_barrier();
  read_codes(S0, wc, h, lr, C.raw);
  read_chain_starts<IF>(S0, wr, h, C.n4);
  read_a<IF>(S0, wr, 0, h, lr, C.a);
#pragma unroll
  for (int j = 0; j < CF; ++j) {
    C.b[j] = unpack_word<RAW>(C.raw[j].x);
    if constexpr (PS) {
      C.sh[j][0] = C.raw[j].y >> 4;
      C.sh[j][1] = C.raw[j].y >> 8;
      C.sh[j][2] = C.raw[j].y >> 12;
    }
  }

  if constexpr (RAW) {
    // the raw form holds more registers in its step (the chain starts it
    // derives); rotating the stages at run time, with scalar stage indices,
    // keeps one address register per LDS access pattern instead of one per
    // stage, and the loop free of spills
    const auto stage = [&](int t) { return Stage{sA[t], sB[t], sN[t], sS[t]}; };
    int cur = 0, nxt = 1, fut = 2;
#pragma nounroll
    for (int g = 0; g < G; ++g) {
      compute_step<IF, RAW, PS>(p, o, m0, n0, g, stage(cur), stage(nxt), stage(fut), sSB, wave,
                            lane, C);
      const int t = cur;
      cur = nxt;
      nxt = fut;
      fut = t;
    }
  } else {
    int g = 0;
    for (;;) {
      compute_step<IF, RAW, PS>(p, o, m0, n0, g, S0, S1, S2, sSB, wave, lane, C);
      if (++g >= G) break;
      compute_step<IF, RAW, PS>(p, o, m0, n0, g, S1, S2, S0, sSB, wave, lane, C);
      if (++g >= G) break;
      compute_step<IF, RAW, PS>(p, o, m0, n0, g, S2, S0, S1, sSB, wave, lane, C);
      if (++g >= G) break;
    }
  }
  // no copy may still be writing LDS when the workgroup retires
  __builtin_amdgcn_s_waitcnt(0);
  // the last group's second-half chains
#pragma unroll
  for (int k = Carry<IF>::HALF; k < Carry<IF>::NC; ++k)
    C.acc[k / CF][k % CF] += C.c[k / CF][k % CF] * f16_to_f32((uint16_t)C.sprev[k % CF]);

  if constexpr (PREP) {
    __shared__ float part[WC * BM];
    store_tile<EPI, true, IF>(p, m0, n0, wave, lane, C.acc, part);
  } else if constexpr (EPI == 2) {
    static_assert(TileM<IF>::BM / 2 * (BN + 4) * 4 <= (int)sizeof(sA), "staging buffer");
    if (((uintptr_t)p.out & 15u) == 0 && (p.ldo & 3) == 0)
      store_resid_staged<IF>(p, m0, n0, wave, lane, C.acc, reinterpret_cast<float*>(&sA[0][0]));
    else
      store_tile<EPI, false, IF>(p, m0, n0, wave, lane, C.acc, nullptr);
  } else {
    store_tile<EPI, false, IF>(p, m0, n0, wave, lane, C.acc, nullptr);
  }
}

template <int EPI, bool PREP, int IF, bool RAW = false>
hipError_t launch_if(GemmParams p, hipStream_t s) {
  p.tiles_m = (p.M + TileM<IF>::BM - 1) / TileM<IF>::BM;
  const dim3 grid((unsigned)(p.tiles_m * p.tiles_n));
  hipLaunchKernelGGL((k_gemm<EPI, PREP, IF, RAW>), grid, dim3(NW * 64), 0, s, p);
  return hipGetLastError();
}

// row extent by the whole call's M (every chunk of a split call uses one)
template <int EPI, bool PREP>
hipError_t launch_one(const GemmParams& p, int64_t M, hipStream_t s) {
  if (M <= 32) return launch_if<EPI, PREP, 2>(p, s);
  if (M <= 64) return launch_if<EPI, PREP, 4>(p, s);
  return launch_if<EPI, PREP, 8>(p, s);
}

GemmParams chunk_params(const uint16_t* x, int64_t ldx, const float* ns, int64_t Mp,
                        const uint8_t* qw, const uint16_t* sc, void* out, int64_t ldo,
                        int64_t m_s, int64_t n_s, int64_t mrows, int64_t ncols, int64_t M,
                        int64_t N, int64_t K, size_t esize, bool tiled) {
  GemmParams p;
  p.xp = x + m_s * ldx;
  p.ns = ns ? ns + m_s : nullptr;
  p.qw = qw + n_s * (K / 2);   // both layouts: n_s is a multiple of 16 columns
  p.qgs = tiled ? 1024 : kGroup / 2;
  p.sc = sc + n_s * (K / kGroup);
  p.out = out ? static_cast<char*>(out) + (size_t)(m_s * ldo + n_s) * esize : nullptr;
  p.ldo = ldo;
  p.Mp = Mp;
  p.ldx = ldx;
  p.M = (int)std::min(mrows, M - m_s);
  p.N = (int)std::min(ncols, N - n_s);
  p.K = (int)K;
  p.G = (int)(K / kGroup);
  p.tiles_m = 0;  // set per row extent in launch_if
  p.tiles_n = (p.N + BN - 1) / BN;
  p.pout = nullptr;
  p.pns = nullptr;
  p.pld = 0;
  p.pcol0 = 0;
  p.sbatch = (p.G % 8 == 0 && reinterpret_cast<uintptr_t>(p.sc) % 16 == 0) ? 1 : 0;
  return p;
}

}  // namespace

// The kernels address operands with 32-bit byte offsets; larger problems are
// split here into row / column chunks that each stay below 2^31 bytes.
hipError_t launch_gemm(const uint16_t* xp, const float* ns, int64_t Mp, const uint8_t* qw,
                       const uint16_t* sc, void* out, int64_t ldo, int64_t M, int64_t N,
                       int64_t K, int epilogue, bool tiled, hipStream_t s, const GemmPrep* prep) {
  const int64_t lim = (int64_t)1 << 31;
  const int64_t mrows = std::max<int64_t>(kGemmBM, (lim / (K * 2)) / kGemmBM * kGemmBM);
  const int64_t ncols = std::max<int64_t>(BN, (lim / (K / 2)) / BN * BN);
  const size_t esize = epilogue == 2 ? 4 : 2;
  for (int64_t m_s = 0; m_s < M; m_s += mrows) {
    for (int64_t n_s = 0; n_s < N; n_s += ncols) {
      GemmParams p = chunk_params(xp, K, ns, Mp, qw, sc, out, ldo, m_s, n_s, mrows, ncols, M, N,
                                  K, esize, tiled);
      p.pout = prep ? prep->out + m_s * prep->ld : nullptr;
      p.pns = prep ? prep->ns + m_s : nullptr;
      p.pld = prep ? prep->ld : 0;
      p.pcol0 = prep ? (int)(prep->col0 - n_s) : 0;
      hipError_t e;
      if (prep) {
        switch (epilogue) {
          case 1: e = launch_one<1, true>(p, M, s); break;
          case 2: return hipErrorInvalidValue;
          default: e = launch_one<0, true>(p, M, s); break;
        }
      } else {
        switch (epilogue) {
          case 1: e = launch_one<1, false>(p, M, s); break;
          case 2: e = launch_one<2, false>(p, M, s); break;
          default: e = launch_one<0, false>(p, M, s); break;
        }
      }
      if (e != hipSuccess) return e;
    }
  }
  return hipSuccess;
}

hipError_t launch_gemm_raw(const uint16_t* x, int64_t ldx, const uint8_t* qw, const uint16_t* sc,
                           void* out, int64_t ldo, int64_t M, int64_t N, int64_t K, int epilogue,
                           bool tiled, hipStream_t s) {
  const int64_t lim = (int64_t)1 << 31;
  const int64_t mrows = std::max<int64_t>(kGemmBM, (lim / (ldx * 2)) / kGemmBM * kGemmBM);
  const int64_t ncols = std::max<int64_t>(BN, (lim / (K / 2)) / BN * BN);
  const size_t esize = epilogue == 2 ? 4 : 2;
  for (int64_t m_s = 0; m_s < M; m_s += mrows) {
    for (int64_t n_s = 0; n_s < N; n_s += ncols) {
      const GemmParams p = chunk_params(x, ldx, nullptr, 0, qw, sc, out, ldo, m_s, n_s, mrows,
                                        ncols, M, N, K, esize, tiled);
      hipError_t e;
      switch (epilogue) {
        case 1: e = launch_if<1, false, 8, true>(p, s); break;
        case 2: e = launch_if<2, false, 8, true>(p, s); break;
        default: e = launch_if<0, false, 8, true>(p, s); break;
      }
      if (e != hipSuccess) return e;
    }
  }
  return hipSuccess;
}

}  // namespace ql
