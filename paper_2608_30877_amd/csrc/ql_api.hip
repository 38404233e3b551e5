// C ABI of libqlinear: argument validation, dispatch between the small-batch
// and MFMA kernels, the library-owned workspaces of qlinear_forward, and the
// host driver of the 175B-shaped linear stack.
#include <map>
#include <mutex>
#include <utility>

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

// dispatch on prepared / raw operands; workspace already validated
int run_linear(const uint16_t* x, int64_t ldx, const uint8_t* qw, const uint16_t* sc, void* out,
               int64_t ldo, int64_t M, int64_t N, int64_t K, int epi, void* ws,
               hipStream_t s) {
  if (use_gemv(M, K)) return hip_status(launch_gemv(x, ldx, qw, sc, out, ldo, M, N, K, epi, s));
  uint16_t* xp = static_cast<uint16_t*>(ws);
  float* ns = reinterpret_cast<float*>(static_cast<char*>(ws) + xp_bytes(M, K));
  const int64_t Mp = padded_rows(M);
  hipError_t e = launch_prep(x, ldx, xp, ns, M, K, Mp, s);
  if (e != hipSuccess) return QL_ERR_HIP;
  return hip_status(launch_gemm(xp, ns, Mp, qw, sc, out, ldo, M, N, K, epi, s));
}

// ---- library-owned workspaces for qlinear_forward: one per (device, stream)
struct OwnedWs {
  void* ptr = nullptr;
  size_t bytes = 0;
};
std::mutex g_ws_mu;
std::map<std::pair<int, hipStream_t>, OwnedWs> g_ws;

int owned_workspace(hipStream_t s, size_t need, void** out) {
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess) return QL_ERR_HIP;
  std::lock_guard<std::mutex> lk(g_ws_mu);
  OwnedWs& w = g_ws[{dev, s}];
  if (w.bytes < need) {
    if (w.ptr) {
      // work already queued on this stream may still read the old buffer
      if (hipStreamSynchronize(s) != hipSuccess) return QL_ERR_HIP;
      if (hipFree(w.ptr) != hipSuccess) return QL_ERR_HIP;
      w.ptr = nullptr;
      w.bytes = 0;
    }
    size_t grow = need + need / 4;
    if (hipMalloc(&w.ptr, grow) != hipSuccess) {
      w.ptr = nullptr;
      return QL_ERR_HIP;
    }
    w.bytes = grow;
  }
  *out = w.ptr;
  return QL_OK;
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

}  // namespace

extern "C" {

const char* qlinear_status_string(int status) {
  switch (status) {
    case QL_OK: return "ok";
    case QL_ERR_ARG: return "invalid argument (null pointer, non-positive size or K % 128 != 0)";
    case QL_ERR_UNSUPPORTED: return "unsupported (group size other than 128, or unknown epilogue)";
    case QL_ERR_ALIGN: return "misaligned pointer or row stride (16-byte alignment required)";
    case QL_ERR_HIP: return "HIP runtime error or launch failure";
    case QL_ERR_RANGE: return "non-finite weight or fp16 scale overflow";
    case QL_ERR_WORKSPACE: return "workspace missing or too small";
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
  if (epilogue < QL_EPI_NONE || epilogue > QL_EPI_RESID_F32) return QL_ERR_UNSUPPORTED;
  if (ldx < K || ldo < N) return QL_ERR_ARG;
  const uintptr_t esize = epilogue == QL_EPI_RESID_F32 ? 4 : 2;
  if (!aligned16(x) || !aligned16(qweight) || ((uintptr_t)out & (esize - 1)) ||
      ((uintptr_t)scales & 1u))
    return QL_ERR_ALIGN;
  if ((ldx * 2) % 16) return QL_ERR_ALIGN;
  const size_t need = forward_ws_bytes(M, K);
  if (need) {
    if (!workspace || ws_bytes < need) return QL_ERR_WORKSPACE;
    if (!aligned256(workspace)) return QL_ERR_ALIGN;
  }
  return run_linear(x, ldx, qweight, scales, out, ldo, M, N, K, epilogue, workspace,
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
  const size_t need = forward_ws_bytes(M, K);
  void* ws = nullptr;
  if (need) {
    rc = owned_workspace((hipStream_t)stream, need, &ws);
    if (rc) return rc;
  }
  return run_linear(x, K, qweight, scales, out, N, M, N, K, QL_EPI_NONE, ws,
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
  if (!layers || !h || n_layers < 0) return QL_ERR_ARG;
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
  for (int l = 0; l < n_layers; ++l) {
    const ql_qmat* mats[4] = {&layers[l].qkv, &layers[l].out, &layers[l].up, &layers[l].down};
    for (const ql_qmat* q : mats) {
      if (!q->qweight || !q->scales) return QL_ERR_ARG;
      if (!aligned16(q->qweight) || ((uintptr_t)q->scales & 1u)) return QL_ERR_ALIGN;
    }
  }
  hipStream_t s = (hipStream_t)stream;
  char* ws = static_cast<char*>(workspace);
  uint16_t* a = reinterpret_cast<uint16_t*>(ws + L.a);
  uint16_t* qkv = reinterpret_cast<uint16_t*>(ws + L.qkv);
  uint16_t* u = reinterpret_cast<uint16_t*>(ws + L.u);
  uint16_t* av = reinterpret_cast<uint16_t*>(ws + L.av);
  float* ns0 = reinterpret_cast<float*>(ws + L.ns0);
  float* ns1 = reinterpret_cast<float*>(ws + L.ns1);
  const int64_t Mp = padded_rows(M);
  const bool small = L.small;
  hipError_t e = hipSuccess;
#define QL_TRY(call)               \
  do {                             \
    e = (call);                    \
    if (e != hipSuccess) return QL_ERR_HIP; \
  } while (0)
  // optional timing hook: events[8l + 2j] / [8l + 2j + 1] bracket projection j
  auto mark = [&](int l, int j, int end) -> hipError_t {
    if (!events) return hipSuccess;
    void* ev = events[8 * l + 2 * j + end];
    return ev ? hipEventRecord(static_cast<hipEvent_t>(ev), s) : hipSuccess;
  };
  for (int l = 0; l < n_layers; ++l) {
    const ql_layer& Ly = layers[l];
    if (small) {
      QL_TRY(launch_rmsnorm(h, a, nullptr, M, d, 0, eps, false, s));
      QL_TRY(mark(l, 0, 0));
      QL_TRY(launch_gemv(a, d, Ly.qkv.qweight, Ly.qkv.scales, qkv, 3 * d, M, 3 * d, d, 0, s));
      QL_TRY(mark(l, 0, 1));
      const uint16_t* v = qkv + 2 * d;
      int64_t ldv = 3 * d;
      if (use_attn) {
        QL_TRY(launch_attention(qkv, 3 * d, u, d, M, (int)d, attn->heads, attn->seq_len,
                                attn->window, attn->cu_seqlens, attn->n_seqs, s));
        v = u;
        ldv = d;
      }
      QL_TRY(mark(l, 1, 0));
      QL_TRY(launch_gemv(v, ldv, Ly.out.qweight, Ly.out.scales, h, d, M, d, d, 2, s));
      QL_TRY(mark(l, 1, 1));
      QL_TRY(launch_rmsnorm(h, a, nullptr, M, d, 0, eps, false, s));
      QL_TRY(mark(l, 2, 0));
      QL_TRY(launch_gemv(a, d, Ly.up.qweight, Ly.up.scales, u, d_ff, M, d_ff, d, 1, s));
      QL_TRY(mark(l, 2, 1));
      QL_TRY(mark(l, 3, 0));
      QL_TRY(launch_gemv(u, d_ff, Ly.down.qweight, Ly.down.scales, h, d, M, d, d_ff, 2, s));
      QL_TRY(mark(l, 3, 1));
    } else {
      const GemmPrep vprep{av, d, ns1, 2 * d};   // V slice -> out-projection operand
      const GemmPrep uprep{u, d_ff, ns1, 0};     // GELU output -> down-projection operand
      QL_TRY(launch_rmsnorm(h, a, ns0, M, d, Mp, eps, true, s));
      QL_TRY(mark(l, 0, 0));
      QL_TRY(launch_gemm(a, ns0, Mp, Ly.qkv.qweight, Ly.qkv.scales, qkv, 3 * d, M, 3 * d, d, 0, s,
                         use_attn ? nullptr : &vprep));
      QL_TRY(mark(l, 0, 1));
      if (use_attn) {
        QL_TRY(launch_attention(qkv, 3 * d, u, d, M, (int)d, attn->heads, attn->seq_len,
                                attn->window, attn->cu_seqlens, attn->n_seqs, s));
        QL_TRY(launch_prep(u, d, av, ns1, M, d, Mp, s));
      }
      QL_TRY(mark(l, 1, 0));
      QL_TRY(launch_gemm(av, ns1, Mp, Ly.out.qweight, Ly.out.scales, h, d, M, d, d, 2, s));
      QL_TRY(mark(l, 1, 1));
      QL_TRY(launch_rmsnorm(h, a, ns0, M, d, Mp, eps, true, s));
      QL_TRY(mark(l, 2, 0));
      QL_TRY(launch_gemm(a, ns0, Mp, Ly.up.qweight, Ly.up.scales, nullptr, d_ff, M, d_ff, d, 1, s,
                         &uprep));
      QL_TRY(mark(l, 2, 1));
      QL_TRY(mark(l, 3, 0));
      QL_TRY(launch_gemm(u, ns1, Mp, Ly.down.qweight, Ly.down.scales, h, d, M, d, d_ff, 2, s));
      QL_TRY(mark(l, 3, 1));
    }
  }
#undef QL_TRY
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

void qlinear_release(void) {
  std::lock_guard<std::mutex> lk(g_ws_mu);
  if (!g_ws.empty()) (void)hipDeviceSynchronize();
  for (auto& kv : g_ws) {
    if (kv.second.ptr) {
      int cur = 0;
      (void)hipGetDevice(&cur);
      (void)hipSetDevice(kv.first.first);
      (void)hipFree(kv.second.ptr);
      (void)hipSetDevice(cur);
    }
  }
  g_ws.clear();
}

}  // extern "C"
