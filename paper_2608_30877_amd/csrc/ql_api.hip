// C ABI of libqlinear: argument validation, dispatch between the small-batch
// and MFMA kernels, and the host driver of the 175B-shaped linear stack.
#include "../../include/qlinear.h"
#include "ql_internal.h"

using namespace ql;

namespace {

inline bool aligned16(const void* p) { return ((uintptr_t)p & 15u) == 0; }
inline bool aligned256(const void* p) { return ((uintptr_t)p & 255u) == 0; }

int check_shape(int64_t M, int64_t N, int64_t K, int32_t group) {
  if (M <= 0 || N <= 0 || K <= 0) return QL_ERR_ARG;
  if (group != kGroup) return QL_ERR_UNSUPPORTED;
  if (K % kGroup) return QL_ERR_ARG;
  // 32-bit index arithmetic inside the kernels
  if (M > (1LL << 30) || N > (1LL << 30) || K > (1LL << 30)) return QL_ERR_ARG;
  return QL_OK;
}

inline int hip_status(hipError_t e) { return e == hipSuccess ? QL_OK : QL_ERR_HIP; }

size_t forward_ws_bytes(int64_t M, int64_t K) {
  if (use_gemv(M, K)) return 0;
  return xp_bytes(M, K) + ns_bytes(M, K);
}

// dispatch: small batches run the small-batch kernel; otherwise the MFMA
// kernel on the operand prepared in the workspace, or, without one, on the
// activations as stored.  Workspace already validated.
int run_linear(const uint16_t* x, int64_t ldx, const uint8_t* qw, const uint16_t* sc, void* out,
               int64_t ldo, int64_t M, int64_t N, int64_t K, int epi, bool tl, void* ws,
               hipStream_t s) {
  if (use_gemv(M, K))
    return hip_status(launch_gemv(x, ldx, qw, sc, out, ldo, M, N, K, epi, tl, s));
  if (!ws) return hip_status(launch_gemm_raw(x, ldx, qw, sc, out, ldo, M, N, K, epi, tl, s));
  uint16_t* xp = static_cast<uint16_t*>(ws);
  float* ns = reinterpret_cast<float*>(static_cast<char*>(ws) + xp_bytes(M, K));
  const int64_t Mp = padded_rows(M);
  hipError_t e = launch_prep(x, ldx, xp, ns, M, K, Mp, s);
  if (e != hipSuccess) return QL_ERR_HIP;
  return hip_status(launch_gemm(xp, ns, Mp, qw, sc, out, ldo, M, N, K, epi, tl, s));
}

// ---- stack workspace layout
// Small batches run the row-major kernel chain: a, qkv, u.  Larger ones keep
// every GEMM input in the MFMA operand layout: a (RMSNorm output, with ns0),
// av (the V slice, written by the QKV epilogue with ns1) and u (the GELU
// output, written by the up projection's epilogue with ns1).  No GEMM reads
// and writes the same correction array.
struct StackLayout {
  bool small;  // every projection runs the small-batch kernel
  size_t a, qkv, u, av, ns0, ns1, total;
};

StackLayout stack_layout(int64_t M, int64_t d, int64_t d_ff) {
  StackLayout L;
  L.small = use_gemv(M, d) && use_gemv(M, d_ff);
  const int64_t kmax = d_ff > d ? d_ff : d;
  size_t off = 0;
  L.a = off;
  off += align256((size_t)M * d * 2);
  L.qkv = off;
  off += align256((size_t)M * 3 * d * 2);
  L.u = off;
  off += align256((size_t)M * kmax * 2);  // u, or the attention output [M][d]
  L.av = off;
  off += L.small ? 0 : align256((size_t)M * d * 2);
  L.ns0 = off;
  off += L.small ? 0 : ns_bytes(M, kmax);
  L.ns1 = off;
  off += L.small ? 0 : ns_bytes(M, kmax);
  L.total = off;
  return L;
}

// seq_len: tokens per sequence (uniform, cu_seqlens null) or the longest
// sequence (ragged: n_seqs sequences at the offsets cu_seqlens[0..n_seqs])
int check_attention(int64_t M, int64_t d, int32_t heads, int32_t seq_len, int32_t window,
                    const int32_t* cu_seqlens, int32_t n_seqs) {
  if (M <= 0 || heads <= 0 || seq_len <= 0 || window <= 0) return QL_ERR_ARG;
  if (M > (1LL << 30)) return QL_ERR_ARG;
  if (d != (int64_t)heads * 128) return QL_ERR_UNSUPPORTED;
  int64_t seqs;
  if (cu_seqlens) {
    if (n_seqs <= 0) return QL_ERR_ARG;
    if ((uintptr_t)cu_seqlens & 3u) return QL_ERR_ALIGN;
    seqs = n_seqs;
  } else {
    if (M % seq_len) return QL_ERR_ARG;
    seqs = M / seq_len;
  }
  if (attention_tiles(seqs, heads, seq_len) > 0x7fffffffLL) return QL_ERR_ARG;
  return QL_OK;
}

inline bool overlap(const void* a, size_t na, const void* b, size_t nb) {
  const uintptr_t x = (uintptr_t)a, y = (uintptr_t)b;
  return x < y + nb && y < x + na;
}

// ---- stack driver
struct StackRun {
  float* h;
  int64_t M, d, d_ff, Mp;
  float eps;
  const ql_attention_cfg* attn;  // null: the width-1 stand-in
  bool small;                    // every projection runs the small-batch kernel
  uint16_t *a, *qkv, *u, *av;
  float *ns0, *ns1;
  void* const* events;
  hipStream_t s;
};

int stack_setup(float* h, int64_t M, int64_t d, int64_t d_ff, int32_t group, float eps,
                const ql_attention_cfg* attn, void* workspace, size_t ws_bytes,
                void* const* events, hipStream_t s, StackRun* r) {
  if (!h) return QL_ERR_ARG;
  int rc = check_shape(M, d, d, group);
  if (rc) return rc;
  rc = check_shape(M, d_ff, d_ff, group);
  if (rc) return rc;
  const bool use_attn = attn && attn->heads != 0;
  if (use_attn) {
    rc = check_attention(M, d, attn->heads, attn->seq_len, attn->window, attn->cu_seqlens,
                         attn->n_seqs);
    if (rc) return rc;
  }
  if (!aligned16(h)) return QL_ERR_ALIGN;
  const StackLayout L = stack_layout(M, d, d_ff);
  if (!workspace || ws_bytes < L.total) return QL_ERR_WORKSPACE;
  if (!aligned256(workspace)) return QL_ERR_ALIGN;
  char* ws = static_cast<char*>(workspace);
  *r = StackRun{h, M, d, d_ff, padded_rows(M), eps, use_attn ? attn : nullptr, L.small,
                reinterpret_cast<uint16_t*>(ws + L.a), reinterpret_cast<uint16_t*>(ws + L.qkv),
                reinterpret_cast<uint16_t*>(ws + L.u), reinterpret_cast<uint16_t*>(ws + L.av),
                reinterpret_cast<float*>(ws + L.ns0), reinterpret_cast<float*>(ws + L.ns1),
                events, s};
  return QL_OK;
}

// (every stack matrix has N and K multiples of 128, so either code layout
// applies to it)
int check_layer(const ql_layer& Ly) {
  const ql_qmat* mats[4] = {&Ly.qkv, &Ly.out, &Ly.up, &Ly.down};
  for (const ql_qmat* q : mats) {
    if (!q->qweight || !q->scales) return QL_ERR_ARG;
    if (q->layout != QL_LAYOUT_ROWS && q->layout != QL_LAYOUT_TILED) return QL_ERR_UNSUPPORTED;
    if (!aligned16(q->qweight) || ((uintptr_t)q->scales & 1u)) return QL_ERR_ALIGN;
  }
  return QL_OK;
}

inline bool tiled(const ql_qmat& q) { return q.layout == QL_LAYOUT_TILED; }

// optional timing hook: events[8l + 2j] / [8l + 2j + 1] bracket projection j
inline hipError_t mark(const StackRun& r, int l, int j, int end) {
  if (!r.events) return hipSuccess;
  void* ev = r.events[8 * l + 2 * j + end];
  return ev ? hipEventRecord(static_cast<hipEvent_t>(ev), r.s) : hipSuccess;
}

// One block on the residual stream (asynchronous on r.s).
hipError_t run_block(const StackRun& r, const ql_layer& Ly, int l) {
  const int64_t M = r.M, d = r.d, d_ff = r.d_ff, Mp = r.Mp;
  const ql_attention_cfg* at = r.attn;
  hipStream_t s = r.s;
  hipError_t e = hipSuccess;
#define QL_TRY(call)                  \
  do {                                \
    e = (call);                       \
    if (e != hipSuccess) return e;    \
  } while (0)
  if (r.small) {
    QL_TRY(launch_rmsnorm(r.h, r.a, nullptr, M, d, 0, r.eps, false, s));
    QL_TRY(mark(r, l, 0, 0));
    QL_TRY(launch_gemv(r.a, d, Ly.qkv.qweight, Ly.qkv.scales, r.qkv, 3 * d, M, 3 * d, d, 0,
                       tiled(Ly.qkv), s));
    QL_TRY(mark(r, l, 0, 1));
    const uint16_t* v = r.qkv + 2 * d;
    int64_t ldv = 3 * d;
    if (at) {
      QL_TRY(launch_attention(r.qkv, 3 * d, r.u, d, M, (int)d, at->heads, at->seq_len, at->window,
                              at->cu_seqlens, at->n_seqs, s));
      v = r.u;
      ldv = d;
    }
    QL_TRY(mark(r, l, 1, 0));
    QL_TRY(launch_gemv(v, ldv, Ly.out.qweight, Ly.out.scales, r.h, d, M, d, d, 2, tiled(Ly.out), s));
    QL_TRY(mark(r, l, 1, 1));
    QL_TRY(launch_rmsnorm(r.h, r.a, nullptr, M, d, 0, r.eps, false, s));
    QL_TRY(mark(r, l, 2, 0));
    QL_TRY(launch_gemv(r.a, d, Ly.up.qweight, Ly.up.scales, r.u, d_ff, M, d_ff, d, 1, tiled(Ly.up),
                       s));
    QL_TRY(mark(r, l, 2, 1));
    QL_TRY(mark(r, l, 3, 0));
    QL_TRY(launch_gemv(r.u, d_ff, Ly.down.qweight, Ly.down.scales, r.h, d, M, d, d_ff, 2,
                       tiled(Ly.down), s));
    QL_TRY(mark(r, l, 3, 1));
  } else {
    const GemmPrep vprep{r.av, d, r.ns1, 2 * d};  // V slice -> out-projection operand
    const GemmPrep uprep{r.u, d_ff, r.ns1, 0};    // GELU output -> down-projection operand
    QL_TRY(launch_rmsnorm(r.h, r.a, r.ns0, M, d, Mp, r.eps, true, s));
    QL_TRY(mark(r, l, 0, 0));
    QL_TRY(launch_gemm(r.a, r.ns0, Mp, Ly.qkv.qweight, Ly.qkv.scales, r.qkv, 3 * d, M, 3 * d, d,
                       0, tiled(Ly.qkv), s, at ? nullptr : &vprep));
    QL_TRY(mark(r, l, 0, 1));
    if (at) {
      QL_TRY(launch_attention(r.qkv, 3 * d, r.u, d, M, (int)d, at->heads, at->seq_len, at->window,
                              at->cu_seqlens, at->n_seqs, s));
      QL_TRY(launch_prep(r.u, d, r.av, r.ns1, M, d, Mp, s));
    }
    QL_TRY(mark(r, l, 1, 0));
    QL_TRY(launch_gemm(r.av, r.ns1, Mp, Ly.out.qweight, Ly.out.scales, r.h, d, M, d, d, 2,
                       tiled(Ly.out), s));
    QL_TRY(mark(r, l, 1, 1));
    QL_TRY(launch_rmsnorm(r.h, r.a, r.ns0, M, d, Mp, r.eps, true, s));
    QL_TRY(mark(r, l, 2, 0));
    QL_TRY(launch_gemm(r.a, r.ns0, Mp, Ly.up.qweight, Ly.up.scales, nullptr, d_ff, M, d_ff, d, 1,
                       tiled(Ly.up), s, &uprep));
    QL_TRY(mark(r, l, 2, 1));
    QL_TRY(mark(r, l, 3, 0));
    QL_TRY(launch_gemm(r.u, r.ns1, Mp, Ly.down.qweight, Ly.down.scales, r.h, d, M, d, d_ff, 2,
                       tiled(Ly.down), s));
    QL_TRY(mark(r, l, 3, 1));
  }
#undef QL_TRY
  return hipSuccess;
}

// ---- host-streamed weights: one block's four matrices in a device slot
struct SlotLayout {
  size_t q[4], sc[4], total;  // byte offsets of codes and scales: qkv, out, up, down
  int64_t n[4], k[4];         // matrix shapes
};

SlotLayout slot_layout(int64_t d, int64_t d_ff) {
  SlotLayout S;
  const int64_t n[4] = {3 * d, d, d_ff, d}, k[4] = {d, d, d, d_ff};
  size_t off = 0;
  for (int i = 0; i < 4; ++i) {
    S.n[i] = n[i];
    S.k[i] = k[i];
    S.q[i] = off;
    off += align256((size_t)n[i] * k[i] / 2);
    S.sc[i] = off;
    off += align256((size_t)n[i] * (k[i] / kGroup) * 2);
  }
  S.total = off;
  return S;
}

ql_layer slot_layer(char* base, const SlotLayout& S) {
  ql_qmat m[4];
  for (int i = 0; i < 4; ++i)
    m[i] = ql_qmat{reinterpret_cast<const uint8_t*>(base + S.q[i]),
                   reinterpret_cast<const uint16_t*>(base + S.sc[i]), QL_LAYOUT_ROWS};
  return ql_layer{m[0], m[1], m[2], m[3]};
}

hipError_t copy_matrices(const ql_layer& src, const ql_layer& dst, int64_t d, int64_t d_ff,
                         hipStream_t cs) {
  const SlotLayout S = slot_layout(d, d_ff);
  const ql_qmat* a[4] = {&src.qkv, &src.out, &src.up, &src.down};
  const ql_qmat* b[4] = {&dst.qkv, &dst.out, &dst.up, &dst.down};
  for (int i = 0; i < 4; ++i) {
    hipError_t e = hipMemcpyAsync(const_cast<uint8_t*>(b[i]->qweight), a[i]->qweight,
                                  (size_t)S.n[i] * S.k[i] / 2, hipMemcpyHostToDevice, cs);
    if (e != hipSuccess) return e;
    e = hipMemcpyAsync(const_cast<uint16_t*>(b[i]->scales), a[i]->scales,
                       (size_t)S.n[i] * (S.k[i] / kGroup) * 2, hipMemcpyHostToDevice, cs);
    if (e != hipSuccess) return e;
  }
  return hipSuccess;
}

// true for page-locked host memory (hipHostMalloc), which the copy engines
// read asynchronously
bool pinned_host(const void* p) {
  hipPointerAttribute_t at;
  if (hipPointerGetAttributes(&at, p) != hipSuccess) {
    (void)hipGetLastError();  // pageable memory reports an error; clear it
    return false;
  }
  return at.type == hipMemoryTypeHost;
}

}  // namespace

extern "C" {

const char* qlinear_status_string(int status) {
  switch (status) {
    case QL_OK: return "ok";
    case QL_ERR_ARG: return "invalid argument (null pointer, non-positive size or K % 128 != 0)";
    case QL_ERR_UNSUPPORTED:
      return "unsupported (group size other than 128, unknown epilogue or code layout)";
    case QL_ERR_ALIGN: return "misaligned pointer or row stride (16-byte alignment required)";
    case QL_ERR_HIP: return "HIP runtime error or launch failure";
    case QL_ERR_RANGE: return "non-finite weight or fp16 scale overflow";
    case QL_ERR_WORKSPACE: return "workspace missing or too small";
    case QL_ERR_SCRATCH:
      return "problem needs more than the library's fixed scratch (qlayer_stack_scratch_capacity)";
    default: return "unknown status";
  }
}

int qlinear_pack(const float* w, uint8_t* qweight, uint16_t* scales, int64_t N, int64_t K,
                 int32_t group, int32_t* status, ql_stream_t stream) {
  if (!w || !qweight || !scales) return QL_ERR_ARG;
  int rc = check_shape(1, N, K, group);
  if (rc) return rc;
  if (!aligned16(w) || !aligned16(qweight) || ((uintptr_t)scales & 1u)) return QL_ERR_ALIGN;
  return hip_status(launch_pack(w, qweight, scales, N, K, status, (hipStream_t)stream));
}

int qlinear_dequant(const uint8_t* qweight, const uint16_t* scales, float* w, int64_t N,
                    int64_t K, int32_t group, ql_stream_t stream) {
  if (!w || !qweight || !scales) return QL_ERR_ARG;
  int rc = check_shape(1, N, K, group);
  if (rc) return rc;
  if (!aligned16(w) || !aligned16(qweight) || ((uintptr_t)scales & 1u)) return QL_ERR_ALIGN;
  return hip_status(launch_dequant(qweight, scales, w, N, K, (hipStream_t)stream));
}

static int tile_common(const uint8_t* src, uint8_t* dst, int64_t N, int64_t K, bool to_tiled,
                       hipStream_t s) {
  if (!src || !dst) return QL_ERR_ARG;
  int rc = check_shape(1, N, K, kGroup);
  if (rc) return rc;
  if (N % 16) return QL_ERR_ARG;
  if (!aligned16(src) || !aligned16(dst)) return QL_ERR_ALIGN;
  if (overlap(src, (size_t)N * K / 2, dst, (size_t)N * K / 2)) return QL_ERR_ARG;
  return hip_status(launch_tile_codes(src, dst, N, K, to_tiled, s));
}

int qlinear_tile_codes(const uint8_t* qweight, uint8_t* tiled, int64_t N, int64_t K,
                       ql_stream_t stream) {
  return tile_common(qweight, tiled, N, K, true, (hipStream_t)stream);
}

int qlinear_untile_codes(const uint8_t* tiled, uint8_t* qweight, int64_t N, int64_t K,
                         ql_stream_t stream) {
  return tile_common(tiled, qweight, N, K, false, (hipStream_t)stream);
}

size_t qlinear_workspace_bytes(int64_t M, int64_t K, int32_t group) {
  if (check_shape(M, 1, K, group)) return 0;
  return forward_ws_bytes(M, K);
}

int qlinear_forward_ex(const uint16_t* x, int64_t ldx, const uint8_t* qweight,
                       const uint16_t* scales, void* out, int64_t ldo, int64_t M, int64_t N,
                       int64_t K, int32_t group, int32_t epilogue, void* workspace,
                       size_t ws_bytes, ql_stream_t stream) {
  if (!x || !qweight || !scales || !out) return QL_ERR_ARG;
  int rc = check_shape(M, N, K, group);
  if (rc) return rc;
  const bool tl = (epilogue & QL_EPI_WEIGHTS_TILED) != 0;
  epilogue &= ~QL_EPI_WEIGHTS_TILED;
  if (epilogue < QL_EPI_NONE || epilogue > QL_EPI_RESID_F32) return QL_ERR_UNSUPPORTED;
  if (ldx < K || ldo < N) return QL_ERR_ARG;
  if (tl && N % 16) return QL_ERR_ARG;
  const uintptr_t esize = epilogue == QL_EPI_RESID_F32 ? 4 : 2;
  if (!aligned16(x) || !aligned16(qweight) || ((uintptr_t)out & (esize - 1)) ||
      ((uintptr_t)scales & 1u))
    return QL_ERR_ALIGN;
  if ((ldx * 2) % 16) return QL_ERR_ALIGN;
  const size_t need = forward_ws_bytes(M, K);
  if (!need || !workspace) {
    workspace = nullptr;  // small batch, or the MFMA kernel on x as stored
  } else {
    if (ws_bytes < need) return QL_ERR_WORKSPACE;
    if (!aligned256(workspace)) return QL_ERR_ALIGN;
  }
  return run_linear(x, ldx, qweight, scales, out, ldo, M, N, K, epilogue, tl, workspace,
                    (hipStream_t)stream);
}

int qlinear_forward(const uint16_t* x, const uint8_t* qweight, const uint16_t* scales,
                    uint16_t* out, int64_t M, int64_t N, int64_t K, int32_t group,
                    ql_stream_t stream) {
  if (!x || !qweight || !scales || !out) return QL_ERR_ARG;
  int rc = check_shape(M, N, K, group);
  if (rc) return rc;
  if (!aligned16(x) || !aligned16(qweight) || ((uintptr_t)out & 1u) || ((uintptr_t)scales & 1u))
    return QL_ERR_ALIGN;
  return run_linear(x, K, qweight, scales, out, N, M, N, K, QL_EPI_NONE, false, nullptr,
                    (hipStream_t)stream);
}

size_t qlayer_stack_workspace_bytes(int64_t M, int64_t d, int64_t d_ff, int32_t group) {
  if (check_shape(M, d, d, group) || check_shape(M, d_ff, d_ff, group)) return 0;
  return stack_layout(M, d, d_ff).total;
}

void qlayer_stack_workspace_offsets(int64_t M, int64_t d, int64_t d_ff, int32_t group,
                                    size_t* qkv_off, size_t* u_off) {
  (void)group;
  const StackLayout L = stack_layout(M, d, d_ff);
  if (qkv_off) *qkv_off = L.qkv;
  if (u_off) *u_off = L.u;
}

int qlinear_rmsnorm(const float* h, uint16_t* a, int64_t M, int64_t d, float eps,
                    ql_stream_t stream) {
  if (!h || !a) return QL_ERR_ARG;
  if (M <= 0 || d <= 0 || d % 8) return QL_ERR_ARG;
  if (!aligned16(h) || !aligned16(a)) return QL_ERR_ALIGN;
  return hip_status(launch_rmsnorm(h, a, nullptr, M, d, 0, eps, false, (hipStream_t)stream));
}

static int attention_common(const uint16_t* qkv, int64_t ldqkv, uint16_t* out, int64_t ldo, int64_t M,
                     int64_t d, int32_t heads, int32_t seq_len, int32_t window,
                     const int32_t* cu_seqlens, int32_t n_seqs, hipStream_t stream) {
  if (!qkv || !out) return QL_ERR_ARG;
  int rc = check_attention(M, d, heads, seq_len, window, cu_seqlens, n_seqs);
  if (rc) return rc;
  if (ldqkv < 3 * d || ldo < d) return QL_ERR_ARG;
  if (!aligned16(qkv) || !aligned16(out) || ldqkv % 8 || ldo % 8) return QL_ERR_ALIGN;
  if (overlap(qkv, (size_t)((M - 1) * ldqkv + 3 * d) * 2, out, (size_t)((M - 1) * ldo + d) * 2))
    return QL_ERR_ARG;
  return hip_status(launch_attention(qkv, ldqkv, out, ldo, M, (int)d, heads, seq_len, window,
                                     cu_seqlens, n_seqs, stream));
}

int qlinear_attention(const uint16_t* qkv, int64_t ldqkv, uint16_t* out, int64_t ldo,
                      int64_t M, int64_t d, int32_t heads, int32_t seq_len, int32_t window,
                      ql_stream_t stream) {
  return attention_common(qkv, ldqkv, out, ldo, M, d, heads, seq_len, window, nullptr, 0,
                          (hipStream_t)stream);
}

int qlinear_attention_varlen(const uint16_t* qkv, int64_t ldqkv, uint16_t* out, int64_t ldo,
                             int64_t M, int64_t d, int32_t heads, const int32_t* cu_seqlens,
                             int32_t n_seqs, int32_t max_seq_len, int32_t window,
                             ql_stream_t stream) {
  if (!cu_seqlens) return QL_ERR_ARG;
  return attention_common(qkv, ldqkv, out, ldo, M, d, heads, max_seq_len, window, cu_seqlens,
                          n_seqs, (hipStream_t)stream);
}

int qlayer_stack_forward_attn(const ql_layer* layers, int32_t n_layers, float* h, int64_t M,
                              int64_t d, int64_t d_ff, int32_t group, float eps,
                              const ql_attention_cfg* attn, void* workspace, size_t ws_bytes,
                              void* const* events, ql_stream_t stream) {
  if (!layers || n_layers < 0) return QL_ERR_ARG;
  StackRun r;
  int rc = stack_setup(h, M, d, d_ff, group, eps, attn, workspace, ws_bytes, events,
                       (hipStream_t)stream, &r);
  if (rc) return rc;
  for (int l = 0; l < n_layers; ++l) {
    rc = check_layer(layers[l]);
    if (rc) return rc;
  }
  for (int l = 0; l < n_layers; ++l)
    if (run_block(r, layers[l], l) != hipSuccess) return QL_ERR_HIP;
  return QL_OK;
}

int qlayer_stack_forward_timed(const ql_layer* layers, int32_t n_layers, float* h, int64_t M,
                               int64_t d, int64_t d_ff, int32_t group, float eps, void* workspace,
                               size_t ws_bytes, void* const* events, ql_stream_t stream) {
  return qlayer_stack_forward_attn(layers, n_layers, h, M, d, d_ff, group, eps, nullptr,
                                   workspace, ws_bytes, events, stream);
}

int qlayer_stack_forward(const ql_layer* layers, int32_t n_layers, float* h, int64_t M,
                         int64_t d, int64_t d_ff, int32_t group, float eps, void* workspace,
                         size_t ws_bytes, ql_stream_t stream) {
  return qlayer_stack_forward_attn(layers, n_layers, h, M, d, d_ff, group, eps, nullptr,
                                   workspace, ws_bytes, nullptr, stream);
}

size_t qlayer_stack_slot_bytes(int64_t d, int64_t d_ff, int32_t group) {
  if (check_shape(1, d, d, group) || check_shape(1, d_ff, d_ff, group)) return 0;
  return slot_layout(d, d_ff).total;
}

int qlayer_stack_forward_streamed(const ql_layer* host_layers, int32_t n_layers, float* h,
                                  int64_t M, int64_t d, int64_t d_ff, int32_t group, float eps,
                                  const ql_attention_cfg* attn, void* workspace, size_t ws_bytes,
                                  void* slots, size_t slot_bytes, ql_stream_t stream,
                                  ql_stream_t copy_stream) {
  if (!host_layers || n_layers < 0 || !slots) return QL_ERR_ARG;
  if (copy_stream == stream) return QL_ERR_ARG;
  StackRun r;
  int rc = stack_setup(h, M, d, d_ff, group, eps, attn, workspace, ws_bytes, nullptr,
                       (hipStream_t)stream, &r);
  if (rc) return rc;
  const SlotLayout S = slot_layout(d, d_ff);
  if (slot_bytes < 2 * S.total) return QL_ERR_WORKSPACE;
  if (!aligned256(slots)) return QL_ERR_ALIGN;
  for (int l = 0; l < n_layers; ++l) {
    const ql_qmat* mats[4] = {&host_layers[l].qkv, &host_layers[l].out, &host_layers[l].up,
                              &host_layers[l].down};
    for (const ql_qmat* q : mats) {
      if (!q->qweight || !q->scales) return QL_ERR_ARG;
      if (q->layout != QL_LAYOUT_ROWS && q->layout != QL_LAYOUT_TILED) return QL_ERR_UNSUPPORTED;
      if (!pinned_host(q->qweight) || !pinned_host(q->scales)) return QL_ERR_ARG;
    }
  }
  if (n_layers == 0) return QL_OK;
  hipStream_t s = (hipStream_t)stream, cs = (hipStream_t)copy_stream;
  // slot k's weights as a device-side layer
  ql_layer dev[2];
  for (int k = 0; k < 2; ++k) dev[k] = slot_layer(static_cast<char*>(slots) + k * S.total, S);
  // copied[k]: slot k holds the layer the next block reads; freed[k]: the
  // block that last read slot k has finished; entry: everything enqueued on
  // `stream` before this call (an earlier call's blocks may still read the
  // slots, and the residual stream may still be in flight)
  hipEvent_t copied[2] = {nullptr, nullptr}, freed[2] = {nullptr, nullptr}, entry = nullptr;
  int out = QL_OK;
  for (int k = 0; k < 2 && out == QL_OK; ++k)
    if (hipEventCreateWithFlags(&copied[k], hipEventDisableTiming) != hipSuccess ||
        hipEventCreateWithFlags(&freed[k], hipEventDisableTiming) != hipSuccess)
      out = QL_ERR_HIP;
  if (out == QL_OK && hipEventCreateWithFlags(&entry, hipEventDisableTiming) != hipSuccess)
    out = QL_ERR_HIP;
  auto copy_layer = [&](int l, int k) -> hipError_t {
    hipError_t e = copy_matrices(host_layers[l], dev[k], d, d_ff, cs);
    return e != hipSuccess ? e : hipEventRecord(copied[k], cs);
  };
  // the first copy into the slots waits for the work already on `stream`
  if (out == QL_OK && (hipEventRecord(entry, s) != hipSuccess ||
                       hipStreamWaitEvent(cs, entry, 0) != hipSuccess))
    out = QL_ERR_HIP;
  if (out == QL_OK && copy_layer(0, 0) != hipSuccess) out = QL_ERR_HIP;
  for (int l = 0; l < n_layers && out == QL_OK; ++l) {
    const int k = l & 1, nk = k ^ 1;
    if (l + 1 < n_layers) {
      // the next layer goes into the other slot once block l - 1 is done with it
      if (l >= 1 && hipStreamWaitEvent(cs, freed[nk], 0) != hipSuccess) { out = QL_ERR_HIP; break; }
      if (copy_layer(l + 1, nk) != hipSuccess) { out = QL_ERR_HIP; break; }
    }
    if (hipStreamWaitEvent(s, copied[k], 0) != hipSuccess) { out = QL_ERR_HIP; break; }
    ql_layer Ly = dev[k];  // the slot's copies keep the host matrices' layouts
    Ly.qkv.layout = host_layers[l].qkv.layout;
    Ly.out.layout = host_layers[l].out.layout;
    Ly.up.layout = host_layers[l].up.layout;
    Ly.down.layout = host_layers[l].down.layout;
    if (run_block(r, Ly, l) != hipSuccess) { out = QL_ERR_HIP; break; }
    if (hipEventRecord(freed[k], s) != hipSuccess) { out = QL_ERR_HIP; break; }
  }
  // events may be destroyed while work that records them is still queued:
  // the runtime releases them once they complete
  for (int k = 0; k < 2; ++k) {
    if (copied[k]) (void)hipEventDestroy(copied[k]);
    if (freed[k]) (void)hipEventDestroy(freed[k]);
  }
  if (entry) (void)hipEventDestroy(entry);
  return out;
}

}  // extern "C"
