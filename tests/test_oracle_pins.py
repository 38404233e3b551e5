"""Pins of the CPU oracle against things other than itself (no GPU needed).

Each test names the definition it checks.  The paper prints no worked
example, kernel-level number or error bound for this path, so the pins are
exact rational brute force, closed forms, special cases and library routines
of a different kind (torch's bf16 cast, Python's math.erf).
"""
import math
from fractions import Fraction

import numpy as np
import pytest

import oracle as O
import synth
from tests.rational import rint_even, to_bf16, to_f16, to_f32


def _f16_value(bits):
    return Fraction(float(np.uint16(bits).view(np.float16)))


# ---------------------------------------------------------------- formats

def test_f16_cast_is_rne_with_subnormals():
    """Scale rounding: fp32 -> binary16, nearest-even, subnormals kept."""
    rng = np.random.default_rng(10)
    vals = np.concatenate([
        rng.standard_normal(2000).astype(np.float32) * np.float32(0.01),
        np.float32(2.0) ** rng.integers(-27, 16, 500).astype(np.float32)
        * (1 + rng.random(500).astype(np.float32)),
        # exact ties between f16 neighbours, normal and subnormal
        np.array([1 + 2 ** -11, 1 + 3 * 2 ** -11, 2 ** -24 * 1.5, 2 ** -24 * 2.5,
                  2 ** -25, 2 ** -25 * 1.0000001, 65504.0, 65519.0], dtype=np.float32),
    ]).astype(np.float32)
    got = vals.astype(np.float16)
    for v, g in zip(vals, got):
        want = to_f16(Fraction(float(v)))
        assert want is not None
        assert Fraction(float(g)) == want, (v, g, want)


def test_bf16_helper_rational_and_torch():
    """f64 -> bf16 helper: exact RNE (rational) and torch's fp32->bf16 cast."""
    import torch

    rng = np.random.default_rng(11)
    x64 = np.concatenate([
        rng.standard_normal(3000) * 10.0 ** rng.integers(-6, 6, 3000),
        np.array([0.0, -0.0, 1.0 + 2 ** -8, 1.0 + 3 * 2 ** -8, -(1.0 + 2 ** -8),
                  2.0 ** -130, 2.0 ** -133 * 1.5, 3.3895313892515355e38]),
    ])
    bits = O.f64_to_bf16_bits(x64)
    for v, b in zip(x64, bits):
        want = to_bf16(Fraction(float(v)))
        if want is None:
            assert (b & 0x7FFF) == 0x7F80
            continue
        got = O.bf16_bits_to_f64(np.array([b]))[0]
        assert Fraction(float(got)) == want, (v, hex(b))
    x32 = x64.astype(np.float32)
    tb = torch.from_numpy(x32).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    np.testing.assert_array_equal(O.f64_to_bf16_bits(x32.astype(np.float64)), tb)


# ---------------------------------------------------------------- quantization

def _rational_quantize(w_row_group):
    """Steps 1-3 of the scheme on one group, in exact rationals."""
    a = max(abs(Fraction(float(v))) for v in w_row_group)
    s32 = to_f32(a / 7)
    s = to_f16(s32)
    if s == 0:
        return s, [0] * len(w_row_group)
    q = []
    for v in w_row_group:
        r = to_f32(Fraction(float(v)) / s)
        q.append(max(-8, min(7, rint_even(r))))
    return s, q


def test_quantize_matches_rational_definition():
    rng = np.random.default_rng(12)
    w = (rng.standard_normal((3, 256)) * 0.02).astype(np.float32)
    w[1, :128] *= np.float32(3e-6)      # subnormal fp16 scales
    w[2, 128:] = 0.0                    # zero group
    qw, sc = O.quantize_pack(w)
    q = O.unpack_codes(qw)
    for n in range(3):
        for j in range(2):
            s, qq = _rational_quantize(w[n, 128 * j:128 * (j + 1)])
            assert _f16_value(sc[n, j]) == s
            assert list(q[n, 128 * j:128 * (j + 1)]) == qq


def test_tie_rounds_half_to_even():
    """A group [7, 2.5, -2.5, 3.5, 0.5, 1.5, -1.5, 0...]: amax 7 -> s = 1 exactly,
    and the halves go to the even neighbour (2, -2, 4, 0, 2, -2)."""
    w = np.zeros((1, 128), dtype=np.float32)
    w[0, :7] = [7.0, 2.5, -2.5, 3.5, 0.5, 1.5, -1.5]
    qw, sc = O.quantize_pack(w)
    assert sc[0, 0] == 0x3C00               # 1.0 in binary16
    assert list(O.unpack_codes(qw)[0, :8]) == [7, 2, -2, 4, 0, 2, -2, 0]


def test_nibble_order_and_twos_complement():
    """Byte i holds code 2i in the low nibble and 2i+1 in the high nibble."""
    w = np.zeros((1, 128), dtype=np.float32)
    w[0, :4] = [1.0, -1.0, 7.0, -7.0]       # s = 1: codes 1, -1, 7, -7
    qw, _ = O.quantize_pack(w)
    assert qw[0, 0] == 0xF1 and qw[0, 1] == 0x97
    allb = np.arange(256, dtype=np.uint8).reshape(1, 256)
    q = O.unpack_codes(allb).astype(np.int64)
    lo, hi = q[0, 0::2], q[0, 1::2]
    assert lo.min() == -8 and hi.max() == 7
    np.testing.assert_array_equal((lo % 16) + 16 * (hi % 16), np.arange(256))


def test_round_trip_of_representable_codes():
    """q in [-7, 7] with a +-7 in every group and normal fp16 scales:
    pack(q*s) == (q, s) and dequant(pack(q*s)) == q*s bit for bit."""
    rng = np.random.default_rng(13)
    N, K = 16, 512
    G = K // 128
    q = rng.integers(-7, 8, (N, K))
    for n in range(N):
        for j in range(G):
            q[n, 128 * j + rng.integers(0, 128)] = 7 * rng.choice([-1, 1])
    e = rng.integers(-10, 5, (N, G))
    mant = rng.integers(0, 1024, (N, G))
    s = ((1 + mant / 1024.0) * 2.0 ** e).astype(np.float16).astype(np.float32)
    w = (q.reshape(N, G, 128) * s[:, :, None]).reshape(N, K).astype(np.float32)
    qw, sc = O.quantize_pack(w)
    np.testing.assert_array_equal(O.unpack_codes(qw), q)
    np.testing.assert_array_equal(O.f16_bits_to_f32(sc), s)
    np.testing.assert_array_equal(O.dequant(qw, sc), w)


def test_zero_and_underflow_groups():
    """Scale threshold: a/7 <= 2^-25 rounds to a zero scale (tie to even),
    just above it to the smallest subnormal 2^-24; zero scale zeroes the group."""
    w = np.zeros((3, 128), dtype=np.float32)
    w[0, 5] = np.float32(7 * 2.0 ** -25)                     # a/7 == 2^-25 exactly
    w[1, 5] = np.float32(7 * 2.0 ** -25) * np.float32(1.0001)
    w[1, 6] = -w[1, 5]
    qw, sc = O.quantize_pack(w)
    assert list(sc[:, 0]) == [0, 1, 0]
    q = O.unpack_codes(qw)
    assert not q[0].any() and not q[2].any()
    # w/s = 7*1.0001*2^-25 / 2^-24 = 3.50035 -> 4 (and -4)
    assert q[1, 5] == 4 and q[1, 6] == -4
    np.testing.assert_array_equal(O.dequant(qw, sc)[2], 0.0)


def test_subnormal_scale_clamps_to_code_range():
    """With a coarse subnormal scale w/s can exceed 7.5: codes clamp to [-8, 7]."""
    w = np.zeros((1, 128), dtype=np.float32)
    a = np.float32(7 * 1.4 * 2.0 ** -24)                      # a/7 -> s = 2^-24
    w[0, 0], w[0, 1] = a, -a
    qw, sc = O.quantize_pack(w)
    assert sc[0, 0] == 1
    q = O.unpack_codes(qw)
    assert q[0, 0] == 7 and q[0, 1] == -8


def test_range_errors():
    w = np.zeros((1, 128), dtype=np.float32)
    w[0, 3] = np.nan
    with pytest.raises(O.OracleRangeError):
        O.quantize_pack(w)
    w[0, 3] = np.inf
    with pytest.raises(O.OracleRangeError):
        O.quantize_pack(w)
    w[0, 3] = np.float32(7 * 65520.0)                        # a/7 rounds to f16 inf
    with pytest.raises(O.OracleRangeError):
        O.quantize_pack(w)
    w[0, 3] = np.float32(7 * 65504.0)                        # largest finite scale
    _, sc = O.quantize_pack(w)
    assert sc[0, 0] == 0x7BFF


def test_sign_symmetry_of_pack():
    w = synth.weights_f32(14, 8, 256)
    qw, sc = O.quantize_pack(w)
    qn, sn = O.quantize_pack(-w)
    np.testing.assert_array_equal(sn, sc)
    np.testing.assert_array_equal(O.unpack_codes(qn), -O.unpack_codes(qw).astype(np.int16))


def test_scale_range_of_workload_weights():
    """N(0, 0.02) weights give normal fp16 scales and never the code -8."""
    w = synth.weights_f32(15, 256, 1024)
    qw, sc = O.quantize_pack(w)
    s = O.f16_bits_to_f32(sc)
    assert s.min() > 2.0 ** -14 and s.max() < 0.05
    q = O.unpack_codes(qw)
    assert q.min() >= -7 and q.max() <= 7


# ---------------------------------------------------------------- matmul

def test_matmul_brute_force_rational():
    """M = N = 4, K = 128: every output as an exact rational sum."""
    x = synth.activations_bf16(16, 4, 128)
    w = synth.weights_f32(16, 4, 128)
    qw, sc = O.quantize_pack(w)
    y = O.qlinear_ref(x, qw, sc)
    xv = O.bf16_bits_to_f64(x)
    q = O.unpack_codes(qw)
    for m in range(4):
        for n in range(4):
            s = _f16_value(sc[n, 0])
            exact = sum(Fraction(float(xv[m, k])) * int(q[n, k]) * s for k in range(128))
            assert abs(float(exact) - y[m, n]) <= 1e-12 * max(1.0, abs(float(exact)))


def test_exact_arithmetic_case_matches_integer_matmul():
    """x in {-1,0,1}, uniform codes, s = 2^-3: Y = (x q^T) * 2^-3 exactly."""
    M, N, K = 32, 48, 1024
    x = synth.ternary_bf16(17, M, K)
    qw = synth.random_packed_bytes(17, N, K)
    sc = synth.const_f16_bits(N, K // 128, 0x3000)       # 2^-3
    y = O.qlinear_ref(x, qw, sc)
    xi = np.rint(O.bf16_bits_to_f64(x)).astype(np.int64)
    qi = O.unpack_codes(qw).astype(np.int64)
    np.testing.assert_array_equal(y, (xi @ qi.T).astype(np.float64) / 8.0)


def test_identity_and_permutation_weights():
    """q = 1 on a permuted diagonal with s = 1 gives out == permuted x; via
    pack, 7*I gives s = 1 and codes 7, i.e. out == 7x."""
    K = 256
    x = synth.activations_bf16(18, 5, K)
    perm = np.random.default_rng(18).permutation(K)
    q = np.zeros((K, K), dtype=np.int64)
    q[np.arange(K), perm] = 1
    nib = (q & 0xF).astype(np.uint8)
    qw = (nib[:, 0::2] | (nib[:, 1::2] << 4)).astype(np.uint8)
    sc = synth.const_f16_bits(K, K // 128, 0x3C00)
    y = O.qlinear_ref(x, qw, sc)
    np.testing.assert_array_equal(y, O.bf16_bits_to_f64(x)[:, perm])
    qw7, sc7 = O.quantize_pack(7 * np.eye(K, dtype=np.float32))
    diag_group = (np.arange(K)[:, None] // 128) == np.arange(K // 128)[None, :]
    np.testing.assert_array_equal(sc7, np.where(diag_group, 0x3C00, 0))
    np.testing.assert_array_equal(O.qlinear_ref(x, qw7, sc7), 7 * O.bf16_bits_to_f64(x))


def test_zero_scales_give_zero_output():
    x = synth.activations_bf16(19, 8, 512)
    qw = synth.random_packed_bytes(19, 64, 512)
    sc = synth.const_f16_bits(64, 4, 0)
    assert not O.qlinear_ref(x, qw, sc).any()


def test_cols_subset_matches_full():
    x = synth.activations_bf16(20, 6, 384)
    qw, sc = O.quantize_pack(synth.weights_f32(20, 40, 384))
    cols = np.array([0, 7, 39, 12])
    np.testing.assert_array_equal(O.qlinear_ref_cols(x, qw, sc, cols),
                                  O.qlinear_ref(x, qw, sc)[:, cols])


# ---------------------------------------------------------------- GELU, RMSNorm

def test_gelu_closed_forms():
    z = np.linspace(-9, 9, 721)
    g = O.gelu(z)
    assert O.gelu(np.array([0.0]))[0] == 0.0
    np.testing.assert_allclose(g - O.gelu(-z), z, rtol=0, atol=1e-14)   # gelu(z)-gelu(-z) = z
    big = z[z >= 6]
    np.testing.assert_allclose(O.gelu(big), big, rtol=1e-8)
    for v in [-3.0, -1.0, -0.25, 0.5, 1.0, 2.0, 4.5]:                 # Python's own erf
        assert abs(O.gelu(np.array([v]))[0] - 0.5 * v * (1 + math.erf(v / math.sqrt(2)))) < 1e-15
    # Phi(1) = 0.8413447460685429 (standard normal CDF at 1, textbook value)
    assert abs(O.gelu(np.array([1.0]))[0] - 0.8413447460685429) < 1e-15


def test_rmsnorm_closed_forms():
    c = 3.0
    h = np.full((2, 512), c, dtype=np.float32)
    h[1] = -c
    out = O.bf16_bits_to_f64(O.rmsnorm_bf16(h, 1e-5))
    want = to_bf16(Fraction(c) / Fraction(math.sqrt(c * c + 1e-5)))
    assert Fraction(float(out[0, 0])) == want and (out[0] == out[0, 0]).all()
    np.testing.assert_array_equal(out[1], -out[0])
    hr = synth.residual_f32(21, 4, 1024)
    y = O.bf16_bits_to_f64(O.rmsnorm_bf16(hr, 0.0))
    np.testing.assert_allclose(np.mean(y * y, axis=1), 1.0, rtol=2e-3)


# ---------------------------------------------------------------- one stack layer

def _direct_pack(q):
    nib = (np.asarray(q, dtype=np.int64) & 0xF).astype(np.uint8)
    return (nib[:, 0::2] | (nib[:, 1::2] << 4)).astype(np.uint8)


def _layer_of(qkv, out, up, down):
    return {"qkv": qkv, "out": out, "up": up, "down": down}


def test_stack_layer_zero_weights_leave_h():
    d, dff = 256, 512
    h = synth.residual_f32(22, 3, d)
    z = lambda n, k: (np.zeros((n, k // 2), np.uint8), synth.const_f16_bits(n, k // 128, 0))
    layer = _layer_of(z(3 * d, d), z(d, d), z(dff, d), z(d, dff))
    np.testing.assert_array_equal(O.stack_layer(h, layer), h)


def test_stack_layer_v_slice_and_gelu_placement():
    """W_qkv has only its V block = 7I (via pack), W_o = I (q=1, s=1), and
    W_up / W_down pass the first d channels: then
    h1 = h + bf16(7 a) and h2 = h1 + bf16(gelu(rmsnorm(h1))) on those channels.
    A wrong V offset, a missing residual or GELU in the wrong place fails."""
    d, dff = 256, 512
    h = synth.residual_f32(23, 4, d)
    wqkv = np.zeros((3 * d, d), np.float32)
    wqkv[2 * d:, :] = 7 * np.eye(d, dtype=np.float32)
    qkv = O.quantize_pack(wqkv)
    one = synth.const_f16_bits
    out = (_direct_pack(np.eye(d, dtype=np.int64)), one(d, d // 128, 0x3C00))
    up_q = np.zeros((dff, d), np.int64)
    up_q[:d, :] = np.eye(d, dtype=np.int64)
    dn_q = np.zeros((d, dff), np.int64)
    dn_q[:, :d] = np.eye(d, dtype=np.int64)
    up = (_direct_pack(up_q), one(dff, d // 128, 0x3C00))
    down = (_direct_pack(dn_q), one(d, dff // 128, 0x3C00))
    h2, mid = O.stack_layer(h, _layer_of(qkv, out, up, down), keep=True)
    a = O.bf16_bits_to_f64(O.rmsnorm_bf16(h))
    v = O.bf16_bits_to_f64(O.f64_to_bf16_bits(7 * a))
    h1 = (h.astype(np.float64) + v).astype(np.float32)
    np.testing.assert_array_equal(mid["h1"], h1)
    a2 = O.bf16_bits_to_f64(O.rmsnorm_bf16(h1))
    g = O.bf16_bits_to_f64(O.f64_to_bf16_bits(
        0.5 * a2 * (1 + np.vectorize(math.erf)(a2 / math.sqrt(2)))))
    np.testing.assert_array_equal(h2, (h1.astype(np.float64) + g).astype(np.float32))


# ------------------------------------------------------------------ attention

def _qkv(q, k, v):
    """bf16 bit patterns of [Q | K | V] from fp64 blocks (values are rounded
    to bf16 first; the pins below compute their expectations from the rounded
    values)."""
    return O.f64_to_bf16_bits(np.concatenate([q, k, v], axis=1))


def test_attention_zero_keys_is_causal_running_mean():
    """K = 0: every allowed score is 0, so token i averages V over
    max(0, i - window + 1) .. i of its own sequence (closed form)."""
    rng = np.random.default_rng(5)
    d, heads, L, window = 8, 2, 6, 4
    M = 2 * L
    q = rng.standard_normal((M, d))
    v = rng.standard_normal((M, d))
    bits = _qkv(q, np.zeros((M, d)), v)
    vr = O.bf16_bits_to_f64(bits[:, 2 * d:])
    out = O.attention_ref(bits, d, heads, L, window)
    for p in range(2):
        for i in range(L):
            lo = max(0, i - window + 1)
            ref = vr[p * L + lo:p * L + i + 1].mean(axis=0)
            np.testing.assert_allclose(out[p * L + i], ref, rtol=0, atol=1e-14)


def test_attention_ragged_zero_keys_is_running_mean_per_sequence():
    """Ragged batch (lengths 3, 1, 5, 2 packed without padding), K = 0: each
    token averages V over the visible tokens of its own sequence."""
    rng = np.random.default_rng(15)
    d, heads, lengths, window = 8, 2, [3, 1, 5, 2], 3
    M = sum(lengths)
    bits = _qkv(rng.standard_normal((M, d)), np.zeros((M, d)), rng.standard_normal((M, d)))
    vr = O.bf16_bits_to_f64(bits[:, 2 * d:])
    out = O.attention_ref(bits, d, heads, lengths, window)
    p0 = 0
    for L in lengths:
        for i in range(L):
            lo = max(0, i - window + 1)
            ref = vr[p0 + lo:p0 + i + 1].mean(axis=0)
            np.testing.assert_allclose(out[p0 + i], ref, rtol=0, atol=1e-14)
        p0 += L
    with pytest.raises(ValueError):
        O.attention_ref(bits, d, heads, [3, 1, 5], window)      # lengths must sum to M


def test_attention_ragged_sequences_are_independent():
    """Each sequence of a ragged batch gives the same output as on its own
    (changing one sequence leaves the others bit for bit unchanged)."""
    rng = np.random.default_rng(16)
    d, heads, lengths = 8, 1, [4, 7, 2]
    M = sum(lengths)
    blocks = [rng.standard_normal((M, d)) for _ in range(3)]
    base = O.attention_ref(_qkv(*blocks), d, heads, lengths, 100)
    changed = [b.copy() for b in blocks]
    for b in changed:
        b[4:11] = rng.standard_normal((7, d))   # the middle sequence
    out = O.attention_ref(_qkv(*changed), d, heads, lengths, 100)
    np.testing.assert_array_equal(out[:4], base[:4])
    np.testing.assert_array_equal(out[11:], base[11:])
    assert not np.array_equal(out[4:11], base[4:11])


def test_attention_window_one_is_identity_on_v():
    """A window of one token reduces attention to the V slice: the width-1
    stand-in of the linear stack."""
    rng = np.random.default_rng(6)
    d, M = 16, 10
    bits = _qkv(rng.standard_normal((M, d)), rng.standard_normal((M, d)),
                rng.standard_normal((M, d)))
    out = O.attention_ref(bits, d, 4, 5, 1)
    np.testing.assert_array_equal(out, O.bf16_bits_to_f64(bits[:, 2 * d:]))


def test_attention_two_token_weights_by_hand():
    """One head, dh = 2: token 1 sees keys 0 and 1 with scores s0 = q.k0 /
    sqrt(2) and s1 = 0, so its output is (e^s0 V0 + V1) / (e^s0 + 1); token 0
    sees only itself."""
    d = 2
    k0 = O.bf16_bits_to_f64(O.f64_to_bf16_bits(np.array([math.sqrt(2) * math.log(3.0)])))[0]
    q = np.array([[0.0, 0.0], [1.0, 0.0]])
    k = np.array([[k0, 0.0], [0.0, 0.0]])
    v = np.array([[2.0, -1.0], [6.0, 3.0]])
    out = O.attention_ref(_qkv(q, k, v), d, 1, 2, 8)
    w0 = math.exp(k0 / math.sqrt(2))          # ~ 3
    np.testing.assert_allclose(out[0], v[0], rtol=0, atol=0)
    np.testing.assert_allclose(out[1], (w0 * v[0] + v[1]) / (w0 + 1.0), rtol=1e-14, atol=1e-14)
    assert abs(w0 - 3.0) < 0.02                 # the weights are about 3/4, 1/4


def test_attention_dominant_key_selects_its_value():
    """A score far above the others puts (all but e^-100 of) the weight on one
    key: the output is that key's V row."""
    rng = np.random.default_rng(7)
    d, heads, L = 8, 1, 5
    q = np.zeros((L, d))
    k = np.zeros((L, d))
    v = rng.standard_normal((L, d))
    q[4, 0] = 16.0
    k[2, 0] = 16.0                              # score 256 / sqrt(8) ~ 90.5
    bits = _qkv(q, k, v)
    out = O.attention_ref(bits, d, heads, L, L)
    np.testing.assert_allclose(out[4], O.bf16_bits_to_f64(bits[2, 2 * d:]), rtol=0, atol=1e-30)


def test_attention_causal_and_sequence_local():
    """Changing a later token of a sequence, or another sequence entirely,
    leaves the earlier outputs of the sequence unchanged."""
    rng = np.random.default_rng(8)
    d, heads, L = 8, 2, 6
    M = 2 * L
    blocks = [rng.standard_normal((M, d)) for _ in range(3)]
    base = O.attention_ref(_qkv(*blocks), d, heads, L, L)
    changed = [b.copy() for b in blocks]
    for b in changed:
        b[4] += 3.0                             # token 4 of sequence 0
        b[L:] = rng.standard_normal((L, d))     # all of sequence 1
    out = O.attention_ref(_qkv(*changed), d, heads, L, L)
    np.testing.assert_array_equal(out[:4], base[:4])


def test_stack_layer_with_width_one_attention_matches_stand_in():
    """stack_layer with attention of window 1 is the width-1 stand-in."""
    d, dff, M = 128, 256, 6
    mk = lambda i, n, k: O.quantize_pack(synth.weights_f32(50 + i, n, k))
    layer = {"qkv": mk(0, 3 * d, d), "out": mk(1, d, d), "up": mk(2, dff, d), "down": mk(3, d, dff)}
    h = synth.residual_f32(9, M, d)
    np.testing.assert_array_equal(O.stack_layer(h, layer), O.stack_layer(h, layer, attn=(1, 3, 1)))


def test_attention_rows_match_the_full_attention():
    """The row-sampled form agrees with attention_ref on every row (windows
    shorter and longer than the sequence), to rounding of the fp64 sums."""
    rng = np.random.default_rng(17)
    d, heads, L = 16, 2, 9
    M = 3 * L
    bits = _qkv(*[rng.standard_normal((M, d)) * 2 for _ in range(3)])
    for window in (1, 4, 9, 50):
        full = O.attention_ref(bits, d, heads, L, window)
        rows = list(range(M))
        got = O.attention_rows_ref(bits, d, heads, L, window, rows)
        np.testing.assert_allclose(got, full, rtol=1e-12, atol=1e-12)


# ------------------------------------------------------------------ checker and scale indexing

def test_rel_fro_closed_forms():
    """The relative Frobenius error that every tolerance test uses."""
    from tests.oracle_checks import check_rel_fro

    check_rel_fro(O.rel_fro)


def test_rmsnorm_eps_and_mean_closed_forms():
    """RMSNorm's eps inside the square root, the mean over d, unit gain:
    rows whose bf16 result changes with each of them (exact to 60 digits)."""
    from tests.oracle_checks import check_rmsnorm

    check_rmsnorm(O.rmsnorm_bf16)


def test_per_group_scales_exact():
    """A scale of its own per (column, group): exact rational sums."""
    from tests.oracle_checks import check_per_group_scales

    check_per_group_scales(O.qlinear_ref, O.unpack_codes)
