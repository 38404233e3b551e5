// Internal declarations shared by the HIP translation units of libqlinear.
// Not part of the public ABI (see include/qlinear.h).
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

namespace ql {

constexpr int kGroup = 128;          // K elements per scale group
constexpr int kGemmBM = 128;         // MFMA tile kernel: rows per workgroup
constexpr int kGemmBN = 256;         //                   columns per workgroup
constexpr int kSmallM = 16;          // M at or below this runs the small-batch kernel

// Rows of the correction array are padded to this multiple.
inline int64_t padded_rows(int64_t M) { return (M + kGemmBM - 1) / kGemmBM * kGemmBM; }

// Bytes of the internal operand-staging area for an M x K activation:
// the k-permuted bf16 copy [M][K] followed by the correction terms
// fp32 [K/128][padded_rows(M)], each 256-byte aligned.
inline size_t align256(size_t b) { return (b + 255) / 256 * 256; }
inline size_t xp_bytes(int64_t M, int64_t K) { return align256((size_t)M * K * 2); }
inline size_t ns_bytes(int64_t M, int64_t K) {
  return align256((size_t)(K / kGroup) * padded_rows(M) * 4);
}

// ---- launches (all asynchronous on `s`; return hipGetLastError()) ----

hipError_t launch_pack(const float* w, uint8_t* qw, uint16_t* sc, int64_t N, int64_t K,
                       int32_t* status, hipStream_t s);
hipError_t launch_dequant(const uint8_t* qw, const uint16_t* sc, float* w, int64_t N,
                          int64_t K, hipStream_t s);
// codes row-major [N][K/2] -> tiled (to_tiled) or back; N % 16 == 0, src and
// dst distinct and 16-byte aligned
hipError_t launch_tile_codes(const uint8_t* src, uint8_t* dst, int64_t N, int64_t K,
                             bool to_tiled, hipStream_t s);

// x (bf16, row stride ldx) -> xp (k-permuted bf16 [M][K]) and
// ns[g][m] = -136 * sum_{k in group g} x[m][k]   (fp32, row stride Mp)
hipError_t launch_prep(const uint16_t* x, int64_t ldx, uint16_t* xp, float* ns, int64_t M,
                       int64_t K, int64_t Mp, hipStream_t s);

// RMSNorm of fp32 rows; `permuted` selects the MFMA operand layout (+ ns),
// otherwise a plain row-major bf16 output (ns may be null).
hipError_t launch_rmsnorm(const float* h, uint16_t* a, float* ns, int64_t M, int64_t d,
                          int64_t Mp, float eps, bool permuted, hipStream_t s);

// Prepared copy of a projection's output (epilogue 0 or 1): the bf16 values
// of columns col0 .. N-1 (col0 and N - col0 multiples of 128) are also
// written as the next projection's MFMA operand, i.e. what launch_prep would
// make of them: out [M][ld] k-permuted, ns [(N - col0)/128][Mp].
struct GemmPrep {
  uint16_t* out;
  int64_t ld;
  float* ns;
  int64_t col0;
};

// Large-M MFMA kernel on prepared operands.  `out` may be null when `prep`
// is given.
hipError_t launch_gemm(const uint16_t* xp, const float* ns, int64_t Mp, const uint8_t* qw,
                       const uint16_t* sc, void* out, int64_t ldo, int64_t M, int64_t N,
                       int64_t K, int epilogue, bool tiled, hipStream_t s,
                       const GemmPrep* prep = nullptr);

// The MFMA kernel on activations as stored (row stride ldx): it derives the
// corrections itself and needs no staging buffer (128-row tiles).
hipError_t launch_gemm_raw(const uint16_t* x, int64_t ldx, const uint8_t* qw, const uint16_t* sc,
                           void* out, int64_t ldo, int64_t M, int64_t N, int64_t K, int epilogue,
                           bool tiled, hipStream_t s);

// Small-M kernel on raw bf16 activations (M <= kSmallM).  It keeps the
// workgroup's scales in LDS: gemv_lds_bytes(K) must stay within kGemvMaxLds
// (K <= 49152); use_gemv picks it for the shapes it serves.
constexpr size_t kGemvMaxLds = 65536;
size_t gemv_lds_bytes(int64_t K);
inline bool use_gemv(int64_t M, int64_t K) {
  return M <= kSmallM && gemv_lds_bytes(K) <= kGemvMaxLds;
}
hipError_t launch_gemv(const uint16_t* x, int64_t ldx, const uint8_t* qw, const uint16_t* sc,
                       void* out, int64_t ldo, int64_t M, int64_t N, int64_t K, int epilogue,
                       bool tiled, hipStream_t s);

// Causal sliding-window attention over a [Q | K | V] buffer, head dim 128.
// Uniform batch (cu_seqlens null): M = whole sequences of seq_len tokens.
// Ragged batch: n_seqs sequences at the device offsets cu_seqlens[0..n_seqs],
// each at most seq_len tokens.  Launches attention_tiles(...) workgroups.
int64_t attention_tiles(int64_t n_seqs, int heads, int max_len);
hipError_t launch_attention(const uint16_t* qkv, int64_t ldq, uint16_t* out, int64_t ldo,
                            int64_t M, int d, int heads, int seq_len, int window,
                            const int32_t* cu_seqlens, int n_seqs, hipStream_t s);

}  // namespace ql
