"""Seeded synthetic inputs shared by the tests, the bench and the smoke check.

This module draws random numbers and nothing else: it holds none of the
quantization, matmul or normalisation arithmetic of the method, so both the
oracle side and the HIP side can take their inputs from it without sharing
any computation.

Workload recipe (the paper's screening set is private and absent; these
synthetic tensors stand in for it with the shapes of a 175B-wide decoder):
  * a protein-ligand pair is 512 tokens (about 450 residue and 60 ligand
    tokens, padded), so 4 pairs give M = 2048 rows and 8 pairs M = 4096;
  * weights W [N, K] are N(0, 0.02) fp32 before quantization;
  * activations x [M, K] are N(0, 1) rounded to bf16, optionally with 1 % of
    the K channels (columns) scaled by 20 before rounding (outliers).

bf16 tensors are carried as uint16 bit patterns (numpy has no bf16).
"""
from __future__ import annotations

import numpy as np

TOKENS_PER_PAIR = 512

# seed bases per workload
SEED_TOY, SEED_QKV, SEED_FFN, SEED_GEMV, SEED_STACK = 0, 1, 2, 3, 4


def matrix_seed(workload_seed: int, layer: int, matrix_idx: int) -> int:
    """Seed of one weight matrix: 1000*workload + 4*layer + matrix index
    (0 = qkv, 1 = out, 2 = up, 3 = down)."""
    return 1000 * workload_seed + 4 * layer + matrix_idx


def _rng(seed: int) -> np.random.Generator:
    return np.random.Generator(np.random.PCG64(seed))


def f32_to_bf16_bits(z: np.ndarray) -> np.ndarray:
    """Round fp32 values to bf16 (round-to-nearest-even) via torch's CPU cast,
    returned as uint16 bit patterns.  Used only to build inputs."""
    import torch

    t = torch.from_numpy(np.ascontiguousarray(z, dtype=np.float32)).to(torch.bfloat16)
    return t.view(torch.int16).numpy().view(np.uint16).copy()


def weights_f32(seed: int, N: int, K: int, std: float = 0.02) -> np.ndarray:
    """W [N, K] fp32 ~ N(0, std)."""
    z = _rng(seed).standard_normal((N, K), dtype=np.float32)
    z *= np.float32(std)
    return z


def activations_bf16(seed: int, M: int, K: int, outlier_frac: float = 0.0,
                     outlier_scale: float = 20.0) -> np.ndarray:
    """x [M, K] as bf16 bits: N(0,1); round(outlier_frac*K) distinct columns
    scaled by outlier_scale in fp32 before the bf16 rounding."""
    rng = _rng(seed + 7_000_000)
    z = rng.standard_normal((M, K), dtype=np.float32)
    n_out = int(round(outlier_frac * K))
    if n_out:
        cols = rng.choice(K, n_out, replace=False)
        z[:, cols] *= np.float32(outlier_scale)
    return f32_to_bf16_bits(z)


def ternary_bf16(seed: int, M: int, K: int) -> np.ndarray:
    """x [M, K] with entries in {-1, 0, +1} (exact in bf16), as bf16 bits."""
    v = _rng(seed + 8_000_000).integers(-1, 2, size=(M, K), dtype=np.int8)
    out = np.zeros((M, K), dtype=np.uint16)
    out[v == 1] = 0x3F80
    out[v == -1] = 0xBF80
    return out


def random_packed_bytes(seed: int, N: int, K: int) -> np.ndarray:
    """qweight [N, K/2] of uniform random bytes: every byte holds two 4-bit
    two's-complement codes, so uniform bytes are uniform codes in [-8, 7]."""
    return _rng(seed + 9_000_000).integers(0, 256, size=(N, K // 2), dtype=np.uint8)


def const_f16_bits(N: int, G: int, bits: int) -> np.ndarray:
    """A [N, G] array filled with one binary16 bit pattern."""
    return np.full((N, G), bits, dtype=np.uint16)


def residual_f32(seed: int, M: int, d: int) -> np.ndarray:
    """Initial residual stream h0 = float32(bf16(N(0,1))) [M, d]."""
    bits = activations_bf16(seed + 11_000_000, M, d)
    return (bits.astype(np.uint32) << 16).view(np.float32)


def weights_f32_cuda(seed: int, N: int, K: int, std: float = 0.02, out=None):
    """W [N, K] fp32 ~ N(0, std) drawn on the current CUDA device with torch's
    seeded generator (for matrices too large to stage on the host)."""
    import torch

    g = torch.Generator(device="cuda")
    g.manual_seed(seed)
    if out is None:
        out = torch.empty((N, K), dtype=torch.float32, device="cuda")
    out.normal_(0.0, std, generator=g)
    return out


def ternary_bf16_cuda(seed: int, M: int, K: int):
    """x [M, K] with entries in {-1, 0, 1} as bf16 bit patterns (int16),
    drawn on the current CUDA device with torch's seeded generator."""
    import torch

    g = torch.Generator(device="cuda")
    g.manual_seed(seed)
    t = torch.randint(-1, 2, (M, K), dtype=torch.int16, device="cuda", generator=g)
    # bf16 bits of -1, 0, +1
    return torch.where(t == 0, 0, torch.where(t > 0, 0x3F80, -16512)).to(torch.int16)


def qkv_bf16(seed: int, M: int, d: int, std: float = 2.2) -> np.ndarray:
    """A [Q | K | V] buffer [M, 3d] as bf16 bits, entries N(0, std^2).  The
    default std is that of a QKV projection output at 175B width
    (0.02 * sqrt(12288) for unit-RMS inputs and N(0, 0.02) weights)."""
    z = _rng(seed + 12_000_000).standard_normal((M, 3 * d), dtype=np.float32)
    z *= np.float32(std)
    return f32_to_bf16_bits(z)


def qkv_bf16_cuda(seed: int, M: int, d: int, std: float = 2.2):
    """qkv_bf16's distribution drawn on the current CUDA device with torch's
    seeded generator: [M, 3d] bf16 (not the same numbers as the host draw)."""
    import torch

    g = torch.Generator(device="cuda")
    g.manual_seed(seed)
    t = torch.empty((M, 3 * d), dtype=torch.float32, device="cuda")
    t.normal_(0.0, std, generator=g)
    return t.to(torch.bfloat16)


def pair_lengths(seed: int, n: int, protein=(380, 450), ligand=(40, 62)) -> np.ndarray:
    """Token counts of n protein-ligand pairs for a ragged (unpadded) batch:
    residue tokens uniform in `protein` plus ligand tokens uniform in
    `ligand` (inclusive), so at most 512 with the defaults."""
    rng = _rng(seed + 13_000_000)
    return (rng.integers(protein[0], protein[1] + 1, size=n)
            + rng.integers(ligand[0], ligand[1] + 1, size=n)).astype(np.int64)


def random_packed_bytes_cuda(seed: int, N: int, K: int):
    """Uniform random code bytes [N, K/2] (uint8) on the current CUDA device."""
    import torch

    g = torch.Generator(device="cuda")
    g.manual_seed(seed)
    return torch.randint(0, 256, (N, K // 2), dtype=torch.uint8, device="cuda", generator=g)


def random_scales_f16(seed: int, N: int, G: int, lo: float = 0.004, hi: float = 0.016) -> np.ndarray:
    """[N, G] binary16 bits of scales uniform in [lo, hi] (the range that
    N(0, 0.02) weights give), for packed weights drawn directly as bytes."""
    v = _rng(seed + 10_000_000).uniform(lo, hi, size=(N, G)).astype(np.float32)
    return v.astype(np.float16).view(np.uint16)


def pow2_scales_f16(seed: int, N: int, G: int, e_lo: int = 2, e_hi: int = 6) -> np.ndarray:
    """[N, G] binary16 bits of 2^-e, e drawn uniformly from e_lo..e_hi for
    every (column, group) on its own.  With ternary activations and uniform
    codes every partial sum of the projection stays an exact fp32 value (up
    to K = 49152 for the default range), so outputs are exact in any
    summation order while each group still has a scale of its own."""
    e = _rng(seed + 14_000_000).integers(e_lo, e_hi + 1, size=(N, G))
    return (0x3C00 - (e << 10)).astype(np.uint16)


def pow2_scales_f16_cuda(seed: int, N: int, G: int, e_lo: int = 2, e_hi: int = 6):
    """pow2_scales_f16's distribution drawn on the current CUDA device with
    torch's seeded generator: [N, G] int16 bit patterns."""
    import torch

    g = torch.Generator(device="cuda")
    g.manual_seed(seed)
    e = torch.randint(e_lo, e_hi + 1, (N, G), dtype=torch.int32, device="cuda", generator=g)
    return (0x3C00 - (e << 10)).to(torch.int16)


def random_scales_f16_cuda(seed: int, N: int, G: int, lo: float = 0.004, hi: float = 0.016):
    """random_scales_f16's distribution drawn on the current CUDA device:
    [N, G] int16 bit patterns of fp16 scales uniform in [lo, hi]."""
    import torch

    g = torch.Generator(device="cuda")
    g.manual_seed(seed)
    t = torch.empty((N, G), dtype=torch.float32, device="cuda")
    t.uniform_(lo, hi, generator=g)
    return t.to(torch.float16).view(torch.int16)
