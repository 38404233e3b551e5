"""GPU parity of the HIP path against the CPU oracle, through the C ABI.

Bars: bit-exact for packing and dequantization; bit-exact for the exact-
arithmetic inputs (ternary x, uniform codes, power-of-two scales: every
partial sum is an exact fp32 value in any order); relative Frobenius error
<= 5e-3 for bf16 outputs on workload-like inputs (the tolerance the path is
specified with).  Full-size problems are checked on sampled output columns
that the oracle computes one by one.
"""
import numpy as np
import pytest
import torch

import oracle as O
import synth
from tests.gpu_util import bf16_as_f64, dev, dev_u16, host_u16, say

pytestmark = pytest.mark.gpu

TOL = 5e-3
# Non-exact inputs: the kernels feed 136 + q to the MFMA and remove 136 * sum(x)
# per group, so a group's dot product carries an absolute error of a few fp32
# ulps of 136 * |sum x| (~1e-4 for N(0,1) x), which flips the bf16 rounding of
# a small fraction of outputs by one ulp: ~1e-5 .. 1e-4 relative Frobenius.
OFFSET_TOL = 2e-4


@pytest.fixture(scope="module")
def ql():
    import paper_2608_30877_amd as ql

    return ql


def _pack_gpu(ql, w):
    qw, sc = ql.pack(dev(w))
    torch.cuda.synchronize()
    return qw.cpu().numpy(), host_u16(sc)


# ------------------------------------------------------------------ pack / dequant

@pytest.mark.parametrize("N,K", [(512, 512), (3, 128), (77, 384), (256, 12288)])
def test_pack_bit_exact(ql, N, K):
    say(f"pack N={N} K={K}")
    w = synth.weights_f32(100 + N, N, K)
    qw_ref, sc_ref = O.quantize_pack(w)
    qw, sc = _pack_gpu(ql, w)
    np.testing.assert_array_equal(sc, sc_ref)
    np.testing.assert_array_equal(qw, qw_ref)


def test_pack_edge_groups_bit_exact(ql):
    """Ties, zero groups, subnormal and tiny scales, the largest scale, and
    a coarse subnormal scale that clamps to -8."""
    w = np.zeros((8, 256), dtype=np.float32)
    w[0, :7] = [7.0, 2.5, -2.5, 3.5, 0.5, 1.5, -1.5]
    w[1, 5] = np.float32(7 * 2.0 ** -25)
    w[2, 5] = np.float32(7 * 2.0 ** -25) * np.float32(1.0001)
    w[2, 6] = -w[2, 5]
    a = np.float32(7 * 1.4 * 2.0 ** -24)
    w[3, 0], w[3, 1] = a, -a
    w[4, 3] = np.float32(7 * 65504.0)
    w[5] = synth.weights_f32(5, 1, 256)[0] * np.float32(3e-6)
    w[6] = synth.weights_f32(6, 1, 256)[0] * np.float32(1e3)
    w[7, 128:] = -np.float32(0.75)
    qw_ref, sc_ref = O.quantize_pack(w)
    qw, sc = _pack_gpu(ql, w)
    np.testing.assert_array_equal(sc, sc_ref)
    np.testing.assert_array_equal(qw, qw_ref)


@pytest.mark.parametrize("bad", [np.nan, np.inf, 7 * 65520.0])
def test_pack_range_error(ql, bad):
    w = synth.weights_f32(7, 4, 256)
    w[2, 100] = np.float32(bad)
    with pytest.raises(ql.QLError) as e:
        ql.pack(dev(w))
    assert e.value.code == 5


def test_pack_full_qkv_shape_bit_exact(ql):
    """The QKV projection at 175B width: N = 36864, K = 12288."""
    N, K = 36864, 12288
    say(f"pack full N={N} K={K}")
    w = synth.weights_f32(synth.matrix_seed(synth.SEED_QKV, 0, 0), N, K)
    qw, sc = _pack_gpu(ql, w)
    for r0 in range(0, N, 6144):      # oracle in row blocks to bound host memory
        qr, sr = O.quantize_pack(w[r0:r0 + 6144])
        np.testing.assert_array_equal(sc[r0:r0 + 6144], sr)
        np.testing.assert_array_equal(qw[r0:r0 + 6144], qr)


@pytest.mark.parametrize("N,K", [(512, 512), (96, 1280)])
def test_dequant_bit_exact(ql, N, K):
    qw = synth.random_packed_bytes(N + K, N, K)
    sc = O.quantize_pack(synth.weights_f32(N, N, K))[1]
    w = ql.dequant(dev(qw), dev_u16(sc)).cpu().numpy()
    np.testing.assert_array_equal(w, O.dequant(qw, sc))


# ------------------------------------------------------------------ forward

SHAPES = [  # (M, N, K): small-batch kernel, MFMA kernel (32-, 64- and 128-row tiles), ragged tails
    (1, 64, 128), (5, 250, 384), (8, 512, 512), (16, 512, 512), (16, 1000, 1280),
    (17, 256, 256), (32, 256, 384), (48, 300, 256), (64, 384, 512), (128, 256, 512),
    (200, 500, 640), (300, 1024, 1152),
    # group counts divisible by 8: the MFMA kernel copies scales eight groups
    # at a time (the other MFMA shapes above take the per-group copy)
    (200, 500, 1024), (130, 300, 2048),
    # the largest K whose scales the small-batch kernel keeps in LDS, and the
    # next group up, which a small batch runs on the MFMA kernel instead
    (3, 70, 49152), (8, 96, 49280),
    # small batches whose column count selects workgroups of 6 and 4 column
    # fragments (the shapes above take 3), each with a ragged last workgroup
    (5, 24566, 384), (7, 12304, 640),
    # N = 49152 (512 workgroups of 96 columns) with one group and with ten:
    # some waves get no group and contribute zero partial sums
    (3, 49152, 128), (8, 49152, 1280),
]


def _forward_np(ql, x, qw, sc):
    y = ql.forward(dev_u16(x), dev(qw), dev_u16(sc))
    torch.cuda.synchronize()
    return host_u16(y)


def _forward_ws_np(ql, x, qw, sc):
    """qlinear_forward_ex with a workspace: the MFMA kernel on the operand
    prepared in that workspace (the form the stack uses)."""
    M, K = x.shape
    xd = dev_u16(x)
    out = torch.empty((M, qw.shape[0]), dtype=torch.bfloat16, device="cuda")
    ws = torch.empty(max(ql.workspace_bytes(M, K), 256), dtype=torch.uint8, device="cuda")
    ql.forward_ex(xd, dev(qw), dev_u16(sc), out, ql.EPI_NONE, ws)
    torch.cuda.synchronize()
    return host_u16(out)


@pytest.mark.parametrize("M,N,K", [s for s in SHAPES if s[0] > 16])
def test_forward_prepared_operand_exact_bit_exact(ql, M, N, K):
    """As test_forward_exact_arithmetic_bit_exact, through the prepared
    operand (permuted copy and correction terms in a workspace) instead of x
    as stored."""
    say(f"exact prepared M={M} N={N} K={K}")
    x = synth.ternary_bf16(M * 7 + N + 1, M, K)
    qw = synth.random_packed_bytes(M + N * 3 + 1, N, K)
    sc = synth.pow2_scales_f16(M + N * 5 + 1, N, K // 128)
    ref = O.f64_to_bf16_bits(O.qlinear_ref(x, qw, sc))
    np.testing.assert_array_equal(_forward_ws_np(ql, x, qw, sc), ref)


@pytest.mark.parametrize("M,N,K", [s for s in SHAPES if s[0] > 16])
def test_forward_prepared_operand_workload(ql, M, N, K):
    x = synth.activations_bf16(M + 11 * N + 1, M, K, outlier_frac=0.01)
    qw, sc = O.quantize_pack(synth.weights_f32(N + 13 * M + 1, N, K))
    ref = O.qlinear_ref(x, qw, sc)
    y = bf16_as_f64(_forward_ws_np(ql, x, qw, sc))
    assert O.rel_fro(y, ref) <= TOL
    # the raw and prepared forms differ only in how the per-group sums are
    # formed: both stay within the offset-trick bound of the exact result
    assert O.rel_fro(y, bf16_as_f64(O.f64_to_bf16_bits(ref))) <= OFFSET_TOL
    yr = bf16_as_f64(_forward_np(ql, x, qw, sc))
    assert O.rel_fro(yr, bf16_as_f64(O.f64_to_bf16_bits(ref))) <= OFFSET_TOL


@pytest.mark.parametrize("M,N,K", SHAPES)
def test_forward_exact_arithmetic_bit_exact(ql, M, N, K):
    """x in {-1,0,1}, uniform codes, a power-of-two scale 2^-2 .. 2^-6 of its
    own for every (column, group): every partial sum is exact, so out must
    equal the oracle's bf16 result bit for bit, which pins which scale each
    kernel applies to which column and group, across tile edges and tails."""
    say(f"exact M={M} N={N} K={K}")
    x = synth.ternary_bf16(M * 7 + N, M, K)
    qw = synth.random_packed_bytes(M + N * 3, N, K)
    sc = synth.pow2_scales_f16(M + N * 5, N, K // 128)
    ref = O.f64_to_bf16_bits(O.qlinear_ref(x, qw, sc))
    np.testing.assert_array_equal(_forward_np(ql, x, qw, sc), ref)


@pytest.mark.parametrize("M,N,K", SHAPES)
def test_forward_workload_inputs(ql, M, N, K):
    say(f"forward M={M} N={N} K={K}")
    x = synth.activations_bf16(M + 11 * N, M, K, outlier_frac=0.01)
    qw, sc = O.quantize_pack(synth.weights_f32(N + 13 * M, N, K))
    y = bf16_as_f64(_forward_np(ql, x, qw, sc))
    assert O.rel_fro(y, O.qlinear_ref(x, qw, sc)) <= TOL


def test_small_batch_unaligned_scales(ql):
    """Scales only 2-byte aligned: the small-batch kernel copies them to LDS
    element by element instead of in 16-byte pieces."""
    M, N, K = 11, 200, 1280
    say(f"unaligned scales M={M} N={N} K={K}")
    x = synth.ternary_bf16(5, M, K)
    qw = synth.random_packed_bytes(6, N, K)
    sc = synth.pow2_scales_f16(6, N, K // 128)
    ref = O.f64_to_bf16_bits(O.qlinear_ref(x, qw, sc))
    buf = torch.zeros(N * (K // 128) + 8, dtype=torch.int16, device="cuda")
    sc_view = buf[1:1 + N * (K // 128)].view(N, K // 128)
    sc_view.copy_(dev_u16(sc))
    assert sc_view.data_ptr() % 16 == 2
    y = ql.forward(dev_u16(x), dev(qw), sc_view)
    torch.cuda.synchronize()
    np.testing.assert_array_equal(host_u16(y), ref)


@pytest.mark.parametrize("ws", [False, True])
def test_mfma_unaligned_scales(ql, ws):
    """16 groups (a multiple of 8) but scales only 2-byte aligned: the MFMA
    kernel falls back from eight-group scale copies to per-group copies."""
    M, N, K = 150, 300, 2048
    say(f"mfma unaligned scales M={M} N={N} K={K} ws={ws}")
    x = synth.ternary_bf16(15, M, K)
    qw = synth.random_packed_bytes(16, N, K)
    sc = synth.pow2_scales_f16(16, N, K // 128)
    ref = O.f64_to_bf16_bits(O.qlinear_ref(x, qw, sc))
    buf = torch.zeros(N * (K // 128) + 8, dtype=torch.int16, device="cuda")
    sc_view = buf[1:1 + N * (K // 128)].view(N, K // 128)
    sc_view.copy_(dev_u16(sc))
    assert sc_view.data_ptr() % 16 == 2
    xd = dev_u16(x)
    y = torch.empty((M, N), dtype=torch.bfloat16, device="cuda")
    wsb = torch.empty(ql.workspace_bytes(M, K), dtype=torch.uint8, device="cuda") if ws else None
    ql.forward_ex(xd, dev(qw), sc_view, y, ql.EPI_NONE, wsb)
    torch.cuda.synchronize()
    np.testing.assert_array_equal(host_u16(y), ref)


def test_forward_toy_config(ql):
    """M = 16 tokens, K = N = 512, N(0,0.02) weights, N(0,1) activations."""
    x = synth.activations_bf16(synth.SEED_TOY, 16, 512)
    qw, sc = O.quantize_pack(synth.weights_f32(synth.SEED_TOY, 512, 512))
    y = bf16_as_f64(_forward_np(ql, x, qw, sc))
    assert O.rel_fro(y, O.qlinear_ref(x, qw, sc)) <= TOL


@pytest.mark.parametrize("M", [8, 200])
def test_zero_scales_zero_output(ql, M):
    x = synth.activations_bf16(M, M, 512)
    qw = synth.random_packed_bytes(M, 384, 512)
    sc = synth.const_f16_bits(384, 4, 0)
    assert not _forward_np(ql, x, qw, sc).any()


def _grid_bf16(seed, M, K):
    """x = k/16 with integer k in [-128, 128]: exact in bf16, and every group
    sum of 136*x + q*x is an exact fp32 value."""
    k = np.random.default_rng(seed).integers(-128, 129, (M, K))
    return O.f64_to_bf16_bits(k / 16.0)


@pytest.mark.parametrize("M", [3, 16, 130])
def test_identity_and_permutation(ql, M):
    """q = 1 on a permuted diagonal, s = 1: out == x[:, perm] bit for bit on
    grid-valued x, and within tolerance on N(0,1) x."""
    K = 512
    perm = np.random.default_rng(M).permutation(K)
    q = np.zeros((K, K), dtype=np.int64)
    q[np.arange(K), perm] = 1
    nib = (q & 0xF).astype(np.uint8)
    qw = (nib[:, 0::2] | (nib[:, 1::2] << 4)).astype(np.uint8)
    sc = synth.const_f16_bits(K, K // 128, 0x3C00)
    xg = _grid_bf16(M, M, K)
    np.testing.assert_array_equal(_forward_np(ql, xg, qw, sc), xg[:, perm])
    x = synth.activations_bf16(M + 1, M, K)
    y = bf16_as_f64(_forward_np(ql, x, qw, sc))
    assert O.rel_fro(y, bf16_as_f64(x[:, perm])) <= OFFSET_TOL


@pytest.mark.parametrize("M", [7, 256])
def test_sign_symmetry(ql, M):
    """forward(x, -q) == -forward(x, q) bit for bit on exact-arithmetic inputs
    (codes in [-7, 7] built through the packer's round trip), and to rounding
    on workload inputs."""
    K, N = 640, 320
    rng = np.random.default_rng(M)
    q = rng.integers(-7, 8, (N, K))
    q[:, ::128] = 7
    w = (q * 0.125).astype(np.float32)
    qw, sc = O.quantize_pack(w)
    qn, sn = O.quantize_pack(-w)
    x = synth.ternary_bf16(M + 3, M, K)
    a = _forward_np(ql, x, qw, sc)
    b = _forward_np(ql, x, qn, sn)
    np.testing.assert_array_equal(bf16_as_f64(b), -bf16_as_f64(a))
    xw = synth.activations_bf16(M + 5, M, K)
    qw, sc = O.quantize_pack(synth.weights_f32(M + 4, N, K))
    qn, sn = O.quantize_pack(-synth.weights_f32(M + 4, N, K))
    a = bf16_as_f64(_forward_np(ql, xw, qw, sc))
    b = bf16_as_f64(_forward_np(ql, xw, qn, sn))
    assert O.rel_fro(-b, a) <= OFFSET_TOL


@pytest.mark.parametrize("with_ws", [True, False])
@pytest.mark.parametrize("epi", [1, 2])
@pytest.mark.parametrize("M", [12, 160])
def test_forward_ex_epilogues_and_strides(ql, epi, M, with_ws):
    """GELU (bf16 out) and fp32 residual-add epilogues, strided x and out,
    with a workspace (prepared operand) and without (x read as stored)."""
    K, N = 512, 384
    xfull = synth.activations_bf16(M + epi, M, K + 256)
    x = xfull[:, 64:64 + K]
    qw, sc = O.quantize_pack(synth.weights_f32(M * epi, N, K))
    ref = O.qlinear_ref(np.ascontiguousarray(x), qw, sc)
    xd = dev_u16(xfull)
    xv = xd[:, 64:64 + K]
    ws = (torch.empty(max(ql.workspace_bytes(M, K), 1), dtype=torch.uint8, device="cuda")
          if with_ws else None)
    if epi == 1:
        out = torch.zeros((M, N + 64), dtype=torch.bfloat16, device="cuda")
        ql.forward_ex(xv, dev(qw), dev_u16(sc), out[:, :N], ql.EPI_GELU, ws, ldo=N + 64)
        y = bf16_as_f64(host_u16(out)[:, :N])
        assert O.rel_fro(y, O.gelu(ref)) <= TOL
        assert not host_u16(out)[:, N:].any()
    else:
        h0 = synth.residual_f32(M, M, N + 64)
        hd = dev(h0)
        ql.forward_ex(xv, dev(qw), dev_u16(sc), hd[:, :N], ql.EPI_RESID_F32, ws, ldo=N + 64)
        h = hd.cpu().numpy()
        np.testing.assert_array_equal(h[:, N:], h0[:, N:])
        assert O.rel_fro(h[:, :N] - h0[:, :N], ref) <= 1e-4


@pytest.mark.parametrize("with_ws", [False, True])
@pytest.mark.parametrize("N,ldo", [(390, 392), (390, 393), (260, 264)])
@pytest.mark.parametrize("M", [37, 160])
def test_residual_epilogue_ragged_rows(ql, M, N, ldo, with_ws):
    """fp32 residual update with a column count that ends inside a 16-byte
    piece (N % 4 != 0) or a tile (N % 256 != 0): the MFMA kernel stages the
    tile in LDS and updates whole rows when out and ldo allow 16-byte
    accesses (ldo % 4 == 0), element by element otherwise (ldo = 393); the
    columns past N stay untouched.  Without a workspace the 128-row raw
    form runs, with one the 64- or 128-row prepared form."""
    K = 512
    x = synth.activations_bf16(M + N, M, K)
    qw, sc = O.quantize_pack(synth.weights_f32(M + ldo, N, K))
    ref = O.qlinear_ref(x, qw, sc)
    h0 = synth.residual_f32(M + 1, M, ldo)
    hd = dev(h0)
    ws = (torch.empty(ql.workspace_bytes(M, K), dtype=torch.uint8, device="cuda")
          if with_ws else None)
    ql.forward_ex(dev_u16(x), dev(qw), dev_u16(sc), hd, ql.EPI_RESID_F32, ws, N=N, ldo=ldo)
    h = hd.cpu().numpy()
    np.testing.assert_array_equal(h[:, N:], h0[:, N:])
    assert O.rel_fro(h[:, :N] - h0[:, :N], ref) <= 1e-4


@pytest.mark.parametrize("M,with_ws", [(8, False), (300, False), (300, True)])
def test_gelu_epilogue_per_element(ql, M, with_ws):
    """GELU epilogue on exact-arithmetic inputs (ternary x, uniform codes,
    per-(column, group) power-of-two scales: every accumulator is exact),
    element by element against the oracle's GELU of the exact product rounded
    to bf16: at most one bf16 ulp apart, and at most 0.1 % of the elements
    differ from the exact GELU first rounded to fp32 (the kernels' GELU is
    an fp32 evaluation good to 7e-6 relative, tail included).  The fp32 step
    matters for these inputs: their accumulators are multiples of 2^-6 and
    often lie exactly halfway between two bf16 values, where GELU(z) =
    z (1 - Q(z)) with Q below fp32's resolution of 1 rounds to the tie and
    then to even."""
    K, N = 1024, 4096
    x = synth.ternary_bf16(75, M, K)
    qw = synth.random_packed_bytes(76, N, K)
    sc = synth.pow2_scales_f16(77, N, K // 128)
    ws = (torch.empty(ql.workspace_bytes(M, K), dtype=torch.uint8, device="cuda")
          if with_ws else None)
    y = torch.empty((M, N), dtype=torch.bfloat16, device="cuda")
    ql.forward_ex(dev_u16(x), dev(qw), dev_u16(sc), y, ql.EPI_GELU, ws)
    torch.cuda.synchronize()
    acc = O.qlinear_ref(x, qw, sc)
    g = O.gelu(acc)
    ref = O.f64_to_bf16_bits(g).astype(np.int32)
    ref32 = O.f64_to_bf16_bits(g.astype(np.float32).astype(np.float64)).astype(np.int32)
    got = host_u16(y).astype(np.int32)
    key = lambda b: np.where(b & 0x8000, -(b & 0x7FFF), b & 0x7FFF)   # ordered, +-0 equal
    dist = np.abs(key(got) - key(ref))
    dist32 = np.abs(key(got) - key(ref32))
    say(f"  differing {np.mean(dist > 0):.2e} (via fp32 {np.mean(dist32 > 0):.2e}), max ulp "
        f"{dist.max()}, negative tail (acc < -4): {np.mean(acc < -4):.3f} of the outputs")
    assert dist.max() <= 1
    assert np.mean(dist32 > 0) <= 1e-3


# ------------------------------------------------------------------ full-size configs

def _sampled(N, n, seed):
    return np.sort(np.random.default_rng(seed).choice(N, n, replace=False))


def _full_case(ql, M, N, K, seed, outliers, epi=0, nsamp=96, x=None):
    """Weights drawn on the device by the seeded generator; the sampled rows
    are copied to the host, packed by the oracle (and compared with the
    device packing), and the sampled output columns are recomputed by the
    oracle from the same x."""
    say(f"full M={M} N={N} K={K} epi={epi}")
    if x is None:
        x = synth.activations_bf16(seed, M, K, outlier_frac=0.01 if outliers else 0.0)
    wd = synth.weights_f32_cuda(synth.matrix_seed(seed, 0, 0), N, K)
    qw, sc = ql.pack(wd)
    cols = _sampled(N, nsamp, seed)
    ci = torch.from_numpy(cols).cuda()
    w_rows = wd[ci].cpu().numpy()
    del wd
    xd = dev_u16(x)
    if epi == 0:
        y = ql.forward(xd, qw, sc)
    else:
        ws = torch.empty(max(ql.workspace_bytes(M, K), 1), dtype=torch.uint8, device="cuda")
        y = torch.empty((M, N), dtype=torch.bfloat16, device="cuda")
        ql.forward_ex(xd, qw, sc, y, epi, ws)
    torch.cuda.synchronize()
    qr, sr = O.quantize_pack(w_rows)
    np.testing.assert_array_equal(qw[ci].cpu().numpy(), qr)
    np.testing.assert_array_equal(host_u16(sc[ci]), sr)
    ys = bf16_as_f64(host_u16(y[:, ci]))
    ref = O.qlinear_ref(x, qr, sr)
    if epi == 1:
        ref = O.gelu(ref)
    return O.rel_fro(ys, ref)


def test_full_qkv_prefill(ql):
    """QKV at 175B width, prefill: M = 2048, K = 12288, N = 36864, outliers."""
    assert _full_case(ql, 2048, 36864, 12288, synth.SEED_QKV, True) <= TOL


def test_full_ffn_up_gelu(ql):
    """FFN up-projection with the GELU epilogue: M = 2048, K = 12288, N = 49152."""
    assert _full_case(ql, 2048, 49152, 12288, synth.SEED_FFN, False, epi=1) <= TOL


def test_full_ffn_down(ql):
    """FFN down-projection: M = 2048, K = 49152, N = 12288 (bf16 N(0,1) input
    of the shape of the GELU output)."""
    x = synth.activations_bf16(synth.SEED_FFN + 50, 2048, 49152)
    assert _full_case(ql, 2048, 12288, 49152, synth.SEED_FFN + 1, False, nsamp=48, x=x) <= TOL


def test_full_ffn_pair_down_on_gpu_gelu_output(ql):
    """The FFN pair as the stack runs it, M = 2048: up-projection with the
    GELU epilogue on the GPU, then the down-projection (K = 49152, N = 12288)
    on that bf16 output u.  The oracle takes the same u (copied back) and
    computes the sampled output columns of the down projection, at 5e-3."""
    M, d, dff = 2048, 12288, 49152
    say("full FFN pair: down projection on the GPU's own u")
    x = dev_u16(synth.activations_bf16(synth.SEED_FFN, M, d))
    qu = synth.random_packed_bytes_cuda(synth.matrix_seed(synth.SEED_FFN, 1, 2), dff, d)
    su = synth.random_scales_f16_cuda(synth.matrix_seed(synth.SEED_FFN, 1, 2), dff, d // 128)
    u = torch.empty((M, dff), dtype=torch.bfloat16, device="cuda")
    ws = torch.empty(ql.workspace_bytes(M, d), dtype=torch.uint8, device="cuda")
    ql.forward_ex(x, qu, su, u, ql.EPI_GELU, ws)
    del qu, su, ws
    qd = synth.random_packed_bytes_cuda(synth.matrix_seed(synth.SEED_FFN, 1, 3), d, dff)
    sd = synth.random_scales_f16_cuda(synth.matrix_seed(synth.SEED_FFN, 1, 3), d, dff // 128)
    y = ql.forward(u, qd, sd)
    torch.cuda.synchronize()
    cols = _sampled(d, 48, 77)
    ci = torch.from_numpy(cols).cuda()
    u_h = host_u16(u)
    ref = O.qlinear_ref(u_h, qd[ci].cpu().numpy(), host_u16(sd[ci]))
    err = O.rel_fro(bf16_as_f64(host_u16(y[:, ci])), ref)
    say(f"  down on u: rel err {err:.3e}")
    assert err <= TOL
    del x, u, qd, sd, y
    torch.cuda.empty_cache()


def test_full_small_batch(ql):
    """Bandwidth-bound regime: M = 8, K = 12288, N = 49152."""
    assert _full_case(ql, 8, 49152, 12288, synth.SEED_GEMV, False, nsamp=512) <= TOL


@pytest.mark.parametrize("M,N,K", [(2048, 12288, 49152), (8, 49152, 12288)])
def test_full_exact_arithmetic_bit_exact(ql, M, N, K):
    """Exact-arithmetic inputs at full size with per-(column, group) scales
    2^-2 .. 2^-6.  K = 49152 is the longest reduction: |sum x q| <= 1024 per
    group, so the output stays below 384 * 1024 * 2^4 = 6.3e6 < 2^24 quanta
    of 2^-6 and every partial sum is exact."""
    say(f"full exact M={M} N={N} K={K}")
    x = synth.ternary_bf16(9, M, K)
    qw = synth.random_packed_bytes(9, N, K)
    sc = synth.pow2_scales_f16(9, N, K // 128)
    y = ql.forward(dev_u16(x), dev(qw), dev_u16(sc))
    torch.cuda.synchronize()
    cols = _sampled(N, 64, 9)
    ci = torch.from_numpy(cols).cuda()
    ref = O.f64_to_bf16_bits(O.qlinear_ref(x, qw[cols], sc[cols]))
    np.testing.assert_array_equal(host_u16(y[:, ci]), ref)


@pytest.mark.parametrize("M,N,K", [(90000, 256, 12288), (256, 360000, 12288)])
def test_max_size_launch_split_bit_exact(ql, M, N, K):
    """Operands past 2^31 bytes (activations 2.2 GB, or codes 2.2 GB): the
    MFMA kernel's 32-bit offsets make the host split the launch into row /
    column chunks.  Exact-arithmetic inputs drawn on the device, checked bit
    for bit on rows or columns on both sides of the split."""
    say(f"max-size split M={M} N={N} K={K}")
    x = synth.ternary_bf16_cuda(31, M, K)
    qw = synth.random_packed_bytes_cuda(32, N, K)
    sc = synth.pow2_scales_f16_cuda(33, N, K // 128)
    y = ql.forward(x, qw, sc)
    torch.cuda.synchronize()
    rows_lim = (2 ** 31 // (K * 2)) // 128 * 128      # row chunk of the split
    cols_lim = (2 ** 31 // (K // 2)) // 256 * 256     # column chunk
    rng = np.random.default_rng(M + N)
    if M * K * 2 >= 2 ** 31:
        rows = np.unique(np.r_[0, rows_lim - 1, rows_lim, M - 1, rng.integers(0, M, 12)])
        cols = np.arange(N)
    else:
        rows = np.arange(M)
        cols = np.unique(np.r_[0, cols_lim - 1, cols_lim, N - 1, rng.integers(0, N, 12)])
    ri = torch.from_numpy(rows).cuda()
    ci = torch.from_numpy(cols).cuda()
    xs = host_u16(x[ri])
    ref = O.f64_to_bf16_bits(O.qlinear_ref(xs, qw[ci].cpu().numpy(), host_u16(sc[ci])))
    np.testing.assert_array_equal(host_u16(y[ri][:, ci]), ref)
    del x, qw, sc, y
    torch.cuda.empty_cache()


# ------------------------------------------------------------------ RMSNorm

@pytest.mark.parametrize("M,d", [(3, 256), (64, 12288), (2, 20480)])
def test_rmsnorm(ql, M, d):
    h = synth.residual_f32(M + d, M, d) * np.float32(3.0)
    a = host_u16(ql.rmsnorm(dev(h)))
    ref = O.rmsnorm_bf16(h)
    diff = np.abs(a.astype(np.int32) - ref.astype(np.int32))
    assert diff.max() <= 1                       # at most one bf16 ulp
    assert (diff > 0).mean() < 1e-3
