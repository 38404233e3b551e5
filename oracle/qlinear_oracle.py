"""Plain, slow CPU oracle of the int4-weight linear-projection path.

TEST INFRASTRUCTURE.  Nothing in the product library imports, links or runs
this file; only the tests, the smoke check and the bench's CPU-baseline leg
do.  It shares no code with the HIP path (no kernels, headers, tables or
helpers); the two meet only in the seeded input generators of ``synth``.

What is computed.  The paper runs the linear projections of a 175B-parameter
decoder ("batch molecular encoding", Sec. 3.3) on 4-bit pre-quantized weights
(Sec. 2.2 weight quantization, Sec. 3.1 mixed-precision quantization,
Sec. 4.1 "4-bit pre-quantized"), and attributes the GPU share of its runtime
to that computation (Sec. 4.3).  The paper does not define the 4-bit scheme;
this library fixes it, and the functions below are that scheme written out:

  * W is [N, K] (out = x W^T, no bias); groups are 128 consecutive K
    elements of one row;
  * a[n,j]  = max |W[n,k]| over group j, in fp32 (exact);
  * s[n,j]  = fp16_RNE( fp32( a[n,j] / 7 ) ), fp32 IEEE division, fp16
    subnormals kept; an infinite s (overflow) or a non-finite W is an error;
  * q[n,k]  = 0 for the whole group if s == 0, else
              clamp( rint_RNE( fp32( W[n,k] / fp32(s) ) ), -8, 7 );
  * byte i of row n packs q[n,2i] in its low nibble and q[n,2i+1] in its
    high nibble, both 4-bit two's complement; scales are [N][K/g] binary16;
  * W_dq[n,k] = fp32(q) * fp32(s)   (exact in fp32);
  * Y = fp64(x) fp64(W_dq)^T with x the given bf16 values; stored results
    are bf16 (round to nearest even) unless the step keeps fp32.

The transformer-block steps (RMSNorm, GELU, the attention between the QKV
and output projections -- either the width-1 sliding-window stand-in or the
causal sliding-window attention of ``attention_ref`` over uniform or ragged
sequences -- fp32 residual stream) are written out in ``rmsnorm_bf16``,
``gelu``, ``attention_ref`` and ``stack_layer``; ``attention_rows_ref``
evaluates attention_ref's definition for selected query rows only (long
sequences).

Every function here is pinned by CPU tests against something other than
itself: exact rational brute force, closed forms, special cases, library
routines of a different kind (attention_rows_ref against attention_ref,
which closed forms pin).  None is "parity unpinned".
"""
from __future__ import annotations

import numpy as np
from scipy.special import erfc as _erfc

__all__ = [
    "GROUP", "QMAX", "QMIN", "ERR_RANGE", "OracleRangeError",
    "bf16_bits_to_f64", "f64_to_bf16_bits", "f16_bits_to_f32",
    "quantize_pack", "unpack_codes", "dequant", "qlinear_ref",
    "qlinear_ref_cols", "gelu", "rmsnorm_bf16", "attention_ref", "attention_rows_ref",
    "stack_layer",
    "rel_fro",
]

GROUP = 128
QMAX = 7
QMIN = -8
ERR_RANGE = 5


class OracleRangeError(ValueError):
    """Non-finite weight or fp16 scale overflow (the packer refuses these)."""


# --------------------------------------------------------------------------
# number formats
# --------------------------------------------------------------------------

def bf16_bits_to_f64(bits: np.ndarray) -> np.ndarray:
    """bf16 bit patterns (uint16) -> float64 values (exact)."""
    b = np.asarray(bits, dtype=np.uint16).astype(np.uint32) << 16
    return b.view(np.float32).astype(np.float64)


def f64_to_bf16_bits(x: np.ndarray) -> np.ndarray:
    """float64 -> bf16 bits, correctly rounded (nearest, ties to even).

    bf16 keeps 8 significant bits and fp32's exponent range (normal down to
    2^-126, subnormal quantum 2^-133); overflow goes to +-inf.
    """
    x = np.asarray(x, dtype=np.float64)
    out = np.empty(x.shape, dtype=np.float64)
    m, e = np.frexp(x)                     # x = m * 2^e, 0.5 <= |m| < 1
    normal = np.abs(x) >= 2.0 ** -126
    # normal range: 8 significant bits -> quantum 2^(e-8)
    out[normal] = np.ldexp(np.rint(np.ldexp(m[normal], 8)), e[normal] - 8)
    sub = ~normal
    out[sub] = np.rint(np.ldexp(x[sub], 133)) * 2.0 ** -133
    big = np.abs(out) >= 2.0 ** 128
    out[big] = np.copysign(np.inf, x[big])
    nan = np.isnan(x)
    f32 = out.astype(np.float32)           # exact: out has <= 8 significant bits
    bits = (f32.view(np.uint32) >> 16).astype(np.uint16)
    bits[nan] = 0x7FC0
    return bits


def f16_bits_to_f32(bits: np.ndarray) -> np.ndarray:
    """binary16 bit patterns -> float32 values (exact)."""
    return np.asarray(bits, dtype=np.uint16).view(np.float16).astype(np.float32)


# --------------------------------------------------------------------------
# quantization (the library's fixed reading of the paper's 4-bit weights)
# --------------------------------------------------------------------------

def quantize_pack(w: np.ndarray, group: int = GROUP):
    """fp32 W [N, K] -> (qweight uint8 [N, K/2], scales binary16 bits [N, K/g]).

    Follows the scheme in the module docstring step by step.  Raises
    ``OracleRangeError`` on a non-finite weight or an fp16 scale overflow.
    """
    w = np.asarray(w, dtype=np.float32)
    N, K = w.shape
    if group <= 0 or group % 2 or K % group:
        raise ValueError("group must be even and divide K")
    if not np.all(np.isfinite(w)):
        raise OracleRangeError("non-finite weight")
    G = K // group
    wg = w.reshape(N, G, group)
    # step 1: group absolute maximum, fp32 (exact)
    a = np.max(np.abs(wg), axis=2)
    # step 2: fp32 IEEE division by 7, then round to binary16 (RNE, subnormals kept)
    s_f32 = (a / np.float32(QMAX)).astype(np.float32)
    with np.errstate(over="ignore"):
        s16 = s_f32.astype(np.float16)
    if np.any(np.isinf(s16)):
        raise OracleRangeError("fp16 scale overflow")
    s = s16.astype(np.float32)
    # step 3: fp32 division by the scale, round half to even, clamp to [-8, 7];
    # a zero scale zeroes its whole group
    with np.errstate(divide="ignore", invalid="ignore"):
        ratio = (wg / s[:, :, None]).astype(np.float32)
    q = np.clip(np.rint(ratio), QMIN, QMAX)
    q = np.where((s == 0)[:, :, None], 0.0, q).astype(np.int8).reshape(N, K)
    # step 4: two 4-bit two's-complement codes per byte, even k in the low nibble
    nib = (q.astype(np.int16) & 0xF).astype(np.uint8)
    qweight = (nib[:, 0::2] | (nib[:, 1::2] << 4)).astype(np.uint8)
    scales = s16.view(np.uint16).copy()
    return qweight, scales


def unpack_codes(qweight: np.ndarray) -> np.ndarray:
    """qweight uint8 [N, K/2] -> int8 codes [N, K] in [-8, 7]."""
    qw = np.asarray(qweight, dtype=np.uint8)
    lo = (qw & 0xF).astype(np.int8)
    hi = (qw >> 4).astype(np.int8)
    lo = np.where(lo >= 8, lo - 16, lo).astype(np.int8)
    hi = np.where(hi >= 8, hi - 16, hi).astype(np.int8)
    N, H = qw.shape
    q = np.empty((N, 2 * H), dtype=np.int8)
    q[:, 0::2] = lo
    q[:, 1::2] = hi
    return q


def dequant(qweight: np.ndarray, scales: np.ndarray, group: int = GROUP) -> np.ndarray:
    """W_dq [N, K] fp32 = fp32(q) * fp32(s[n, k // g]) (exact in fp32)."""
    q = unpack_codes(qweight).astype(np.float32)
    s = f16_bits_to_f32(scales)
    N, K = q.shape
    return (q.reshape(N, K // group, group) * s[:, :, None]).reshape(N, K).astype(np.float32)


# --------------------------------------------------------------------------
# the projection itself
# --------------------------------------------------------------------------

def qlinear_ref(x_bits: np.ndarray, qweight: np.ndarray, scales: np.ndarray,
                group: int = GROUP) -> np.ndarray:
    """Y [M, N] float64 = x W_dq^T, x given as bf16 bits [M, K]."""
    x = bf16_bits_to_f64(x_bits)
    w = dequant(qweight, scales, group).astype(np.float64)
    return x @ w.T


def qlinear_ref_cols(x_bits: np.ndarray, qweight: np.ndarray, scales: np.ndarray,
                     cols: np.ndarray, group: int = GROUP) -> np.ndarray:
    """Y[:, cols] float64 for a subset of output columns (dequantizes only the
    weight rows it needs; used for samples of full-size problems)."""
    cols = np.asarray(cols)
    x = bf16_bits_to_f64(x_bits)
    w = dequant(np.asarray(qweight)[cols], np.asarray(scales)[cols], group).astype(np.float64)
    return x @ w.T


def gelu(z: np.ndarray) -> np.ndarray:
    """GELU in its exact (erf) form, fp64: z/2 (1 + erf(z / sqrt 2)), evaluated
    as z/2 erfc(-z / sqrt 2), the same function without the cancellation of
    1 + erf for z below about -4 (relative accuracy in the negative tail)."""
    z = np.asarray(z, dtype=np.float64)
    return 0.5 * z * _erfc(-z / np.sqrt(2.0))


def rmsnorm_bf16(h: np.ndarray, eps: float = 1e-5) -> np.ndarray:
    """bf16 bits of h / sqrt(mean_k h^2 + eps) (unit gain), computed in fp64."""
    h = np.asarray(h, dtype=np.float64)
    r = 1.0 / np.sqrt(np.mean(h * h, axis=-1, keepdims=True) + eps)
    return f64_to_bf16_bits(h * r)


def stack_layer(h: np.ndarray, layer: dict, group: int = GROUP, eps: float = 1e-5,
                keep: bool = False, attn=None):
    """One block of the 175B-shaped linear stack on the fp32 residual h [M, d].

    layer = {"qkv": (qw, s), "out": (qw, s), "up": (qw, s), "down": (qw, s)}
    with the QKV projection's output columns ordered [Q | K | V].

    Steps:  a = RMSNorm(h);  qkv = bf16(a W_qkv^T);
            v = qkv[:, 2d:3d] when attn is None (a sliding window of width 1
            makes attention the identity on V), else
            v = bf16(attention_ref(qkv, d, *attn)) with attn = (heads,
            seq_len or the list of sequence lengths, window) (the paper's
            model uses sliding-window attention, Sec. 1 / 2);
            h1 = fp32(h + v W_o^T);  a2 = RMSNorm(h1);
            u = bf16(GELU(a2 W_up^T));  h2 = fp32(h1 + u W_down^T).
    Returns h2 (and the intermediates when keep=True).
    """
    h = np.asarray(h, dtype=np.float32)
    d = h.shape[1]
    a = rmsnorm_bf16(h, eps)
    qkv = f64_to_bf16_bits(qlinear_ref(a, *layer["qkv"], group=group))
    if attn is None:
        v = np.ascontiguousarray(qkv[:, 2 * d:3 * d])
    else:
        v = f64_to_bf16_bits(attention_ref(qkv, d, *attn))
    h1 = (h.astype(np.float64) + qlinear_ref(v, *layer["out"], group=group)).astype(np.float32)
    a2 = rmsnorm_bf16(h1, eps)
    u = f64_to_bf16_bits(gelu(qlinear_ref(a2, *layer["up"], group=group)))
    h2 = (h1.astype(np.float64) + qlinear_ref(u, *layer["down"], group=group)).astype(np.float32)
    if keep:
        return h2, {"a": a, "qkv": qkv, "v": v, "h1": h1, "a2": a2, "u": u}
    return h2


def attention_ref(qkv_bits: np.ndarray, d: int, heads: int, seq_len, window: int) -> np.ndarray:
    """Causal sliding-window multi-head attention of the paper's decoder
    (sliding-window attention with a 32K window, Sec. 1 contribution 1.1 and
    Sec. 2), fp64 from the given bf16 Q, K, V.

    qkv_bits [M, 3d] bf16 bits, columns [Q | K | V]; head h uses columns
    h*dh .. h*dh+dh-1 of each third, dh = d / heads.  The M tokens are
    independent sequences (one protein-ligand pair each), stored one after
    the other: seq_len is either one length (M / seq_len sequences of equal
    length) or the list of the sequences' lengths (a ragged batch, tokens
    packed without padding; the lengths sum to M).  Token i of a sequence
    attends to tokens j of the same sequence with i - window < j <= i.  Per
    head:
        S = Q K^T / sqrt(dh),  P = softmax over the allowed keys (row-wise),
        O = P V.
    Returns O [M, d] (fp64), heads side by side in the column order of Q.
    """
    x = bf16_bits_to_f64(np.asarray(qkv_bits))
    M = x.shape[0]
    dh = d // heads
    if d % heads:
        raise ValueError("d must split into heads")
    if np.ndim(seq_len) == 0:
        if seq_len <= 0 or M % seq_len:
            raise ValueError("M must split into whole sequences")
        lengths = [int(seq_len)] * (M // int(seq_len))
    else:
        lengths = [int(n) for n in seq_len]
        if min(lengths) <= 0 or sum(lengths) != M:
            raise ValueError("sequence lengths must be positive and sum to M")
    out = np.empty((M, d), dtype=np.float64)
    p0 = 0
    for L in lengths:
        i = np.arange(L)[:, None]
        j = np.arange(L)[None, :]
        allowed = (j <= i) & (j > i - window)
        rows = slice(p0, p0 + L)
        for hh in range(heads):
            c = slice(hh * dh, (hh + 1) * dh)
            q = x[rows, c]
            k = x[rows, d + hh * dh:d + (hh + 1) * dh]
            v = x[rows, 2 * d + hh * dh:2 * d + (hh + 1) * dh]
            s = (q @ k.T) / np.sqrt(dh)
            s = np.where(allowed, s, -np.inf)
            e = np.exp(s - s.max(axis=1, keepdims=True))
            out[rows, c] = (e / e.sum(axis=1, keepdims=True)) @ v
        p0 += L
    return out


def attention_rows_ref(qkv_bits: np.ndarray, d: int, heads: int, seq_len: int, window: int,
                       rows) -> np.ndarray:
    """attention_ref's output for the given token rows only (uniform
    sequences of seq_len tokens): the same definition, evaluated for the
    selected queries against the keys each may see, so that long sequences
    (a 32K window) can be checked without the seq_len x seq_len score
    matrix.  Returns [len(rows), d] (fp64)."""
    x = bf16_bits_to_f64(np.asarray(qkv_bits))
    dh = d // heads
    if d % heads or x.shape[0] % seq_len:
        raise ValueError("d must split into heads and M into whole sequences")
    out = np.empty((len(rows), d), dtype=np.float64)
    for n, t in enumerate(rows):
        p0 = (t // seq_len) * seq_len
        i = t - p0
        lo = p0 + max(0, i - window + 1)
        for hh in range(heads):
            c = slice(hh * dh, (hh + 1) * dh)
            q = x[t, c]
            k = x[lo:t + 1, d + hh * dh:d + (hh + 1) * dh]
            v = x[lo:t + 1, 2 * d + hh * dh:2 * d + (hh + 1) * dh]
            s = (k @ q) / np.sqrt(dh)
            e = np.exp(s - s.max())
            out[n, c] = (e / e.sum()) @ v
    return out


def rel_fro(y: np.ndarray, ref: np.ndarray) -> float:
    """Relative Frobenius error ||y - ref|| / ||ref|| in fp64."""
    y = np.asarray(y, dtype=np.float64)
    ref = np.asarray(ref, dtype=np.float64)
    den = np.linalg.norm(ref)
    num = np.linalg.norm(y - ref)
    return float(num / den) if den > 0 else float(num)
