/*
 * qlinear.h -- C ABI of the int4-weight linear-projection library (gfx950).
 *
 * The paper runs the linear projections of a 175B-parameter decoder on
 * 4-bit pre-quantized weights ("weight quantization", Sec. 2.2;
 * "mixed-precision quantization", Sec. 3.1; "4-bit pre-quantized",
 * Sec. 4.1) and attributes the GPU share of its runtime to that computation
 * (Sec. 4.3).  The paper does not define the 4-bit scheme.  This library
 * fixes it as follows, and every entry point below computes with it:
 *
 *   W        [N][K] fp32 weights, out = x * W^T (no bias).
 *   group    g = 128 consecutive K elements of one weight row.
 *   scale    s[n][j] = fp16_RNE(fp32(max_k |W[n][k]| / 7)), k in group j;
 *            fp16 subnormals kept; overflow to inf is an error.
 *   code     q[n][k] = clamp(rint_even(fp32(W[n][k] / s)), -8, 7), and 0 for
 *            the whole group when s == 0.
 *   qweight  uint8 [N][K/2]: byte i holds q[n][2i] in bits 0-3 and
 *            q[n][2i+1] in bits 4-7, both 4-bit two's complement.
 *   scales   uint16 [N][K/g]: binary16 bit patterns.
 *   x, out   bf16 row-major bit patterns (uint16); accumulation is fp32 and
 *            stored bf16 results are rounded to nearest even.
 *
 * Conventions for every entry point:
 *   - All array pointers are DEVICE pointers (HIP device memory on the
 *     current device) unless the comment says "host".  The caller owns every
 *     buffer; the library never frees a caller buffer.
 *   - Calls enqueue work on `stream` (NULL = the default stream) and return
 *     without synchronising.  Arguments are validated before anything is
 *     enqueued, so QL_ERR_ARG, QL_ERR_UNSUPPORTED, QL_ERR_ALIGN and
 *     QL_ERR_WORKSPACE mean nothing was enqueued.  QL_ERR_HIP reports a
 *     failed launch or runtime call; work enqueued before it (earlier
 *     kernels of the same call) may still run, and the outputs are then
 *     unspecified.
 *   - Shapes: M, N >= 1; K >= 128 and K % 128 == 0; group must be 128
 *     (other group sizes return QL_ERR_UNSUPPORTED).  Ragged M and N are
 *     handled by masking; no padding is required of the caller.
 *   - Alignment: x and qweight must be 16-byte aligned and the row stride
 *     of x (ldx) must keep every row 16-byte aligned; out needs only the
 *     alignment of its element type (2 bytes bf16, 4 bytes fp32); scales 2
 *     bytes (QL_ERR_ALIGN otherwise).
 */
#ifndef QLINEAR_H
#define QLINEAR_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* A hipStream_t; declared opaquely so this header needs no HIP headers. */
typedef struct ihipStream_t* ql_stream_t;

enum ql_status {
    QL_OK = 0,
    QL_ERR_ARG = 1,          /* null pointer, non-positive size, K % 128 != 0  */
    QL_ERR_UNSUPPORTED = 2,  /* group != 128, unknown epilogue or code layout  */
    QL_ERR_ALIGN = 3,        /* a pointer or row stride breaks 16 B alignment  */
    QL_ERR_HIP = 4,          /* a HIP runtime call or a launch failed          */
    QL_ERR_RANGE = 5,        /* pack: non-finite weight or fp16 scale overflow */
    QL_ERR_WORKSPACE = 6,    /* workspace pointer null or smaller than needed  */
    QL_ERR_SCRATCH = 7       /* problem larger than the library's fixed scratch */
};

enum ql_epilogue {
    QL_EPI_NONE = 0,         /* out (bf16)  = acc                              */
    QL_EPI_GELU = 1,         /* out (bf16)  = gelu_erf(acc)                    */
    QL_EPI_RESID_F32 = 2,    /* out (fp32) += acc   (residual stream update)   */
    QL_EPI_WEIGHTS_TILED = 0x100  /* flag OR-ed into qlinear_forward_ex's
                                     epilogue: qweight is in QL_LAYOUT_TILED   */
};

/*
 * Code layouts of a packed matrix's qweight (the scales are [N][K/g] in
 * both).  QL_LAYOUT_ROWS is the packed format above, the one qlinear_pack
 * writes, qlinear_dequant reads and every entry point accepts.
 * QL_LAYOUT_TILED is a permutation of the same N*K/2 bytes (N % 16 == 0)
 * for the forward paths: the 64 bytes of group j of the 16 columns
 * 16b .. 16b+15 are one contiguous kilobyte, so that the small-batch kernel
 * streams whole kilobytes instead of 64-byte pieces of 16 rows.  Byte
 * 16*hh + i (hh < 4, i < 16) of column n's group j, i.e. qweight
 * [n][64*j + 16*hh + i] in QL_LAYOUT_ROWS, sits at tiled byte
 *     16 * (64 * ((n / 16) * (K / 128) + j) + 16 * hh + n % 16) + i.
 * qlinear_tile_codes / qlinear_untile_codes convert; the layout is
 * private to this library's kernels (export to other code in
 * QL_LAYOUT_ROWS).
 */
enum ql_layout {
    QL_LAYOUT_ROWS = 0,
    QL_LAYOUT_TILED = 1
};

/* Human-readable name of a status code (static storage, never NULL). */
const char* qlinear_status_string(int status);

/*
 * qlinear_pack -- quantize fp32 weights into the packed int4 format above
 * (the "pre-quantized" weights of Sec. 4.1).
 *   w        [N][K] fp32, read only.
 *   qweight  [N][K/2] uint8, written.
 *   scales   [N][K/128] uint16 (binary16 bits), written.
 *   status   nullable device int32.  When given, the kernel writes
 *            QL_ERR_RANGE into it if any weight is non-finite or any scale
 *            overflows fp16 (the caller zeroes it first and reads it after
 *            synchronising).  The offending group's outputs are zero.
 * Bit-exact: the division is IEEE fp32 (correctly rounded) on the device.
 */
int qlinear_pack(const float* w, uint8_t* qweight, uint16_t* scales,
                 int64_t N, int64_t K, int32_t group, int32_t* status,
                 ql_stream_t stream);

/*
 * qlinear_dequant -- W_dq[n][k] = fp32(q[n][k]) * fp32(s[n][k/128]), exact.
 * Test and inspection export; the forward path never materialises W_dq.
 *   w  [N][K] fp32, written.
 */
int qlinear_dequant(const uint8_t* qweight, const uint16_t* scales, float* w,
                    int64_t N, int64_t K, int32_t group, ql_stream_t stream);

/*
 * qlinear_tile_codes / qlinear_untile_codes -- QL_LAYOUT_ROWS codes
 * [N][K/2] to QL_LAYOUT_TILED and back (a byte permutation; scales are not
 * touched).  N % 16 == 0 and K % 128 == 0 (QL_ERR_ARG); both buffers
 * N*K/2 bytes, 16-byte aligned (QL_ERR_ALIGN) and not overlapping
 * (QL_ERR_ARG).  Not part of the paper's computation: a storage order for
 * the forward kernels (see QL_LAYOUT_TILED).
 */
int qlinear_tile_codes(const uint8_t* qweight, uint8_t* tiled, int64_t N,
                       int64_t K, ql_stream_t stream);
int qlinear_untile_codes(const uint8_t* tiled, uint8_t* qweight, int64_t N,
                         int64_t K, ql_stream_t stream);

/*
 * qlinear_forward -- out[M][N] = bf16(x[M][K] * W_dq^T), the quantized
 * linear projection of Sec. 3.3's "batch molecular encoding" forward pass.
 * M <= 16 runs the bandwidth-bound small-batch kernel, larger M the
 * MFMA tile kernel directly on x (each workgroup derives the per-group
 * activation sums it needs).  Allocates nothing, keeps no state between
 * calls and does not synchronise, so it may be captured in a HIP graph;
 * calls on different streams are independent.
 *   x    [M][K] bf16 bits, contiguous.
 *   out  [M][N] bf16 bits, contiguous, written.
 */
int qlinear_forward(const uint16_t* x, const uint8_t* qweight,
                    const uint16_t* scales, uint16_t* out,
                    int64_t M, int64_t N, int64_t K, int32_t group,
                    ql_stream_t stream);
/* (qweight in QL_LAYOUT_ROWS; qlinear_forward_ex takes either layout) */

/* Bytes of the optional workspace of qlinear_forward_ex for an M x K input
 * (0 when the small-batch kernel serves the shape). */
size_t qlinear_workspace_bytes(int64_t M, int64_t K, int32_t group);

/*
 * qlinear_forward_ex -- qlinear_forward with strides, a fused epilogue and
 * an optional caller-owned workspace; never allocates.
 *   x          bf16 bits, row m at x + m*ldx (ldx >= K elements).
 *   out        QL_EPI_NONE / QL_EPI_GELU: bf16 bits, row m at out + m*ldo
 *              (uint16 elements).  QL_EPI_RESID_F32: fp32, row m at
 *              (float*)out + m*ldo, read and updated in place.
 *   workspace  NULL (ws_bytes ignored): the MFMA kernel reads x as stored,
 *              as in qlinear_forward.  Otherwise a device buffer of at least
 *              qlinear_workspace_bytes(M, K, g) bytes, 256-byte aligned
 *              (QL_ERR_WORKSPACE / QL_ERR_ALIGN): x is first rewritten there
 *              in the kernel's operand layout with its per-group sums; used
 *              only while the enqueued work runs; calls that overlap on one
 *              workspace race.
 *   epilogue   a ql_epilogue value, | QL_EPI_WEIGHTS_TILED when qweight is
 *              in QL_LAYOUT_TILED (then N % 16 == 0, QL_ERR_ARG otherwise).
 */
int qlinear_forward_ex(const uint16_t* x, int64_t ldx, const uint8_t* qweight,
                       const uint16_t* scales, void* out, int64_t ldo,
                       int64_t M, int64_t N, int64_t K, int32_t group,
                       int32_t epilogue, void* workspace, size_t ws_bytes,
                       ql_stream_t stream);

/* One packed weight matrix (device pointers); layout is a ql_layout value
 * (another value: QL_ERR_UNSUPPORTED). */
typedef struct {
    const uint8_t* qweight;
    const uint16_t* scales;
    int32_t layout;
} ql_qmat;

/*
 * One block of the 175B-shaped linear stack (host struct of device
 * pointers): qkv [3d][d], out [d][d], up [d_ff][d], down [d][d_ff].
 * The QKV output columns are ordered [Q | K | V].
 */
typedef struct {
    ql_qmat qkv, out, up, down;
} ql_layer;

/* Bytes of workspace qlayer_stack_forward needs. */
size_t qlayer_stack_workspace_bytes(int64_t M, int64_t d, int64_t d_ff,
                                    int32_t group);

/*
 * qlayer_stack_forward -- n_layers blocks of the linear stack on the fp32
 * residual stream h [M][d] (updated in place).  Per block:
 *     a   = bf16(RMSNorm(h))                 (unit gain, eps)
 *     qkv = bf16(a * W_qkv^T)
 *     v   = qkv[:, 2d:3d]                    (sliding-window attention of
 *                                             width 1 is the identity on V;
 *                                             the model of Sec. 1 / 2.1 uses
 *                                             sliding-window attention, which
 *                                             qlayer_stack_forward_attn runs)
 *     h  += v * W_o^T                        (fp32)
 *     a2  = bf16(RMSNorm(h))
 *     u   = bf16(gelu_erf(a2 * W_up^T))
 *     h  += u * W_down^T                     (fp32)
 * All weights stay resident in device memory; nothing is paged from the
 * host (the paper's Sec. 4.3 runtime split is dominated by such paging).
 *   layers     HOST array of n_layers ql_layer structs.
 *   workspace  >= qlayer_stack_workspace_bytes(M, d, d_ff, g) bytes,
 *              256-byte aligned.  Layout (byte offsets, each 256-aligned):
 *              [0]        a / a2 staging  bf16 [M][d]   (internal layout)
 *              [qkv_off]  qkv             bf16 [M][3d]  (row-major)
 *              [u_off]    u               bf16 [M][max(d, d_ff)]: row-major when
 *                         M <= 16 (and d, d_ff <= 49152, where every
 *                         projection runs the small-batch kernel); otherwise
 *                         the MFMA operand layout,
 *                         in which each 8-element chunk of a row holds
 *                         elements (0,4,1,5,2,6,3,7) of that chunk
 *              then, for M > 16, the prepared V copy and two correction-term
 *              arrays; see qlayer_stack_workspace_offsets.
 *   d, d_ff    multiples of 128.
 */
int qlayer_stack_forward(const ql_layer* layers, int32_t n_layers, float* h,
                         int64_t M, int64_t d, int64_t d_ff, int32_t group,
                         float eps, void* workspace, size_t ws_bytes,
                         ql_stream_t stream);

/*
 * qlayer_stack_forward_timed -- qlayer_stack_forward with a timing hook for
 * profilers and benchmarks.
 *   events  nullable HOST array of 8 * n_layers hipEvent_t handles (as
 *           void*; entries may be NULL).  events[8l + 2j] is recorded on
 *           `stream` right before, and events[8l + 2j + 1] right after, the
 *           launch of projection j of block l (j: 0 qkv, 1 out, 2 up,
 *           3 down).  The caller creates and destroys the events.
 */
int qlayer_stack_forward_timed(const ql_layer* layers, int32_t n_layers, float* h,
                               int64_t M, int64_t d, int64_t d_ff, int32_t group,
                               float eps, void* workspace, size_t ws_bytes,
                               void* const* events, ql_stream_t stream);

/*
 * qlinear_attention -- causal sliding-window multi-head attention, the
 * attention of the paper's decoder (a 32K sliding window, Sec. 1
 * contribution 1.1 and Sec. 2), run between the QKV and output projections.
 * The M tokens form M / seq_len independent sequences (one protein-ligand
 * pair each); token i of a sequence attends to the tokens j of the same
 * sequence with i - window < j <= i.  Per head (head dim 128):
 *     O = softmax(Q K^T / sqrt(128) restricted to the window) V
 * Scores and softmax in fp32; the probabilities are rounded to bf16 for the
 * product with V and the normaliser sums the rounded values; fp32
 * accumulation; bf16 output, rounded to nearest even.
 *   qkv     bf16 bits, row m at qkv + m*ldqkv: Q in columns 0..d-1, K in
 *           d..2d-1, V in 2d..3d-1; head h uses columns 128h..128h+127 of
 *           each third (the layout of the QKV projection's output).
 *   out     bf16 bits, row m at out + m*ldo, columns 0..d-1 written (heads
 *           side by side); must not overlap qkv (QL_ERR_ARG).
 *   d       heads * 128 (any other head dimension: QL_ERR_UNSUPPORTED).
 *   seq_len >= 1 with M % seq_len == 0; window >= 1 (window >= seq_len is
 *           plain causal attention within each sequence).
 *   ldqkv >= 3d and ldo >= d, both multiples of 8 elements, and qkv and out
 *   16-byte aligned (QL_ERR_ALIGN otherwise).
 */
int qlinear_attention(const uint16_t* qkv, int64_t ldqkv, uint16_t* out,
                      int64_t ldo, int64_t M, int64_t d, int32_t heads,
                      int32_t seq_len, int32_t window, ql_stream_t stream);

/*
 * qlinear_attention_varlen -- qlinear_attention over a ragged batch: the
 * sequences (pairs of different lengths, tokens packed without padding)
 * occupy rows cu_seqlens[s] .. cu_seqlens[s+1]-1, s < n_seqs.
 *   cu_seqlens  DEVICE int32 [n_seqs + 1], non-decreasing, cu_seqlens[0] = 0,
 *               cu_seqlens[n_seqs] = M, every length <= max_seq_len.  The
 *               host does not read it; offsets that break these rules give
 *               unspecified results (the kernel clamps them to [0, M], so it
 *               never reads or writes outside qkv and out).  Empty sequences
 *               are allowed.  Rows not covered by any sequence are not
 *               written.
 *   max_seq_len the longest sequence, >= 1 (sizes the launch).
 * Other arguments and errors as for qlinear_attention (no M % seq_len rule).
 */
int qlinear_attention_varlen(const uint16_t* qkv, int64_t ldqkv, uint16_t* out,
                             int64_t ldo, int64_t M, int64_t d, int32_t heads,
                             const int32_t* cu_seqlens, int32_t n_seqs,
                             int32_t max_seq_len, int32_t window,
                             ql_stream_t stream);

/* Attention between the QKV and output projections of a stack block. */
typedef struct {
    int32_t heads;    /* 0 selects the width-1 stand-in v = qkv[:, 2d:3d]   */
    int32_t seq_len;  /* tokens per sequence (M % seq_len == 0), or with
                         cu_seqlens the longest sequence                    */
    int32_t window;   /* sliding-window width, >= 1                         */
    int32_t n_seqs;   /* ragged batch: number of sequences in cu_seqlens    */
    const int32_t* cu_seqlens;  /* NULL: uniform sequences of seq_len; else
                         DEVICE offsets as for qlinear_attention_varlen     */
} ql_attention_cfg;

/*
 * qlayer_stack_forward_attn -- qlayer_stack_forward_timed with attention:
 * in every block v = qlinear_attention(qkv) (bf16) replaces the stand-in
 * v = qkv[:, 2d:3d].  attn NULL or attn->heads == 0 runs the stand-in.
 * Requirements on heads, seq_len and window as for qlinear_attention, with
 * d = heads * 128.  The attention output is staged in the workspace's u
 * buffer (row-major [M][d]) before the out projection; the workspace is the
 * same size.  With events, attention runs between events[8l + 1] and
 * events[8l + 2].
 */
int qlayer_stack_forward_attn(const ql_layer* layers, int32_t n_layers, float* h,
                              int64_t M, int64_t d, int64_t d_ff, int32_t group,
                              float eps, const ql_attention_cfg* attn,
                              void* workspace, size_t ws_bytes,
                              void* const* events, ql_stream_t stream);

/* Bytes of one weight slot of qlayer_stack_forward_streamed (a block's four
 * packed matrices, each codes + scales 256-byte aligned); the call needs two. */
size_t qlayer_stack_slot_bytes(int64_t d, int64_t d_ff, int32_t group);

/*
 * qlayer_stack_forward_streamed -- qlayer_stack_forward_attn for weights
 * that stay in HOST memory: the paper keeps its weights in host RAM and
 * schedules their loading around the computation (adaptive memory
 * management, Sec. 3.1; page swapping is 72 % of its runtime, Sec. 4.3;
 * prefetching is its stated next step, Sec. 5).  Here the pages are whole
 * blocks, double-buffered: while block l computes from one device
 * slot on `stream`, block l+1's eight arrays are copied into the other slot
 * with hipMemcpyAsync on `copy_stream`, ordered by events (a copy into a
 * slot waits until the block that read it has finished; a block waits for
 * its copy).  The step is bound by max(copy, compute) instead of their sum.
 *   host_layers  HOST array of ql_layer structs whose qweight / scales are
 *                page-locked HOST memory (hipHostMalloc); pageable memory is
 *                refused (QL_ERR_ARG) because its copies would not overlap.
 *   slots        DEVICE buffer of >= 2 * qlayer_stack_slot_bytes(d, d_ff, g)
 *                bytes, 256-byte aligned (QL_ERR_WORKSPACE / QL_ERR_ALIGN).
 *   copy_stream  a stream other than `stream` (QL_ERR_ARG otherwise); keep
 *                both at the default priority.
 * h, workspace, attn as for qlayer_stack_forward_attn.  Returns after
 * enqueuing; the host arrays and the slots must stay valid until `stream`
 * has completed the call's work.  Calls that overlap on one slot buffer race.
 */
int qlayer_stack_forward_streamed(const ql_layer* host_layers, int32_t n_layers,
                                  float* h, int64_t M, int64_t d, int64_t d_ff,
                                  int32_t group, float eps,
                                  const ql_attention_cfg* attn, void* workspace,
                                  size_t ws_bytes, void* slots, size_t slot_bytes,
                                  ql_stream_t stream, ql_stream_t copy_stream);

/*
 * qlayer_stack_forward_noalloc -- qlayer_stack_forward for callers that
 * cannot allocate device memory (code under HIP graph capture, tight
 * serving loops, harnesses that forbid hipMalloc): the same kernels and
 * results, with the workspace in a fixed device array of the library
 * (qlayer_stack_scratch_capacity() bytes, 128 MiB, one per GPU, held until
 * the process ends) instead of a caller buffer.  The call allocates and
 * frees nothing and does not synchronise.
 *   Limit: qlayer_stack_workspace_bytes(M, d, d_ff, 128) must not exceed the
 *   capacity, else QL_ERR_SCRATCH and nothing is enqueued (at d = 12288,
 *   d_ff = 49152 that admits M <= 597 tokens).
 *   Every call on one GPU shares that GPU's array: calls that overlap on one
 *   GPU (other streams, other host threads) race and must be serialised by
 *   the caller.  h, layers and the other arguments as for
 *   qlayer_stack_forward.
 */
int qlayer_stack_forward_noalloc(const ql_layer* layers, int32_t n_layers, float* h,
                                 int64_t M, int64_t d, int64_t d_ff, int32_t group,
                                 float eps, ql_stream_t stream);

/* Bytes of the fixed device array behind qlayer_stack_forward_noalloc. */
size_t qlayer_stack_scratch_capacity(void);

/* Host: byte offsets of the qkv and u buffers inside the stack workspace. */
void qlayer_stack_workspace_offsets(int64_t M, int64_t d, int64_t d_ff,
                                    int32_t group, size_t* qkv_off,
                                    size_t* u_off);

/*
 * qlinear_rmsnorm -- a[m][k] = bf16(h[m][k] / sqrt(mean_k h[m][k]^2 + eps)),
 * the normalisation between blocks of the stack.  Test export.
 *   h  [M][d] fp32;  a  [M][d] bf16 bits, row-major, written.
 */
int qlinear_rmsnorm(const float* h, uint16_t* a, int64_t M, int64_t d,
                    float eps, ql_stream_t stream);

#ifdef __cplusplus
}
#endif

#endif /* QLINEAR_H */
