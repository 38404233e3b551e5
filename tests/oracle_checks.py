"""Pin checks of oracle functions, written against an implementation passed
in as an argument, so that the same check runs on the oracle
(tests/test_oracle_pins.py) and on deliberately wrong variants of it
(tests/test_oracle_mutants.py), which it must reject.

Every expected value here comes from a closed form or exact rational
arithmetic, never from the oracle itself.
"""
from decimal import Decimal, getcontext
from fractions import Fraction

import numpy as np

from tests.rational import floor_log2, to_bf16


# ---------------------------------------------------------------- rel_fro

def check_rel_fro(rel_fro):
    """Relative Frobenius error ||y - ref||_F / ||ref||_F over all elements:
    a 3-4-5 triangle, exact relative perturbations, the zero output, the
    identity, a 2-D case that per-row or max-norm errors would get wrong,
    and the zero-reference branch (the plain norm of y)."""
    # ||(3, -4)|| / ||(0, 4)|| = 5 / 4
    assert rel_fro(np.array([3.0, 0.0]), np.array([0.0, 4.0])) == 1.25
    rng = np.random.default_rng(1)
    ref = rng.standard_normal((7, 9))
    for t in (1e-3, -0.25, 2.0):
        got = rel_fro(ref * (1.0 + t), ref)
        assert abs(got - abs(t)) <= 1e-12 * max(1.0, abs(t)), (t, got)
    assert rel_fro(np.zeros_like(ref), ref) == 1.0
    assert rel_fro(ref, ref) == 0.0
    # Frobenius over the whole matrix: ||[[0,0],[0,-1]]|| / ||I|| = 1/sqrt(2)
    y = np.array([[1.0, 0.0], [0.0, 0.0]])
    r = np.eye(2)
    assert abs(rel_fro(y, r) - 2 ** -0.5) <= 1e-15
    # zero reference: the error is the plain norm of y
    assert rel_fro(np.array([3.0, 4.0]), np.zeros(2)) == 5.0


# ---------------------------------------------------------------- RMSNorm

def _exact_bf16_of(c: float, eps: float, d_nonzero: int, d: int) -> Fraction:
    """bf16 (nearest even) of c / sqrt((d_nonzero * c^2) / d + eps), with c
    and eps the exact binary values given, to 60 significant digits (far
    from any bf16 rounding boundary for the values used below)."""
    getcontext().prec = 60
    cf, ef = Fraction(float(c)), Fraction(float(eps))
    ms = cf * cf * d_nonzero / d + ef
    den = (Decimal(ms.numerator) / Decimal(ms.denominator)).sqrt()
    val = Decimal(cf.numerator) / Decimal(cf.denominator) / den
    v = Fraction(val)
    r = to_bf16(v)
    # the value must not sit near a rounding boundary of bf16 (8 significant
    # bits: the unit in the last place of r is 2^(floor(log2 |r|) - 7))
    ulp = Fraction(2) ** (floor_log2(abs(r)) - 7)
    assert abs(v - r) < ulp * Fraction(45, 100)
    return r


def check_rmsnorm(rmsnorm_bf16):
    """RMSNorm with unit gain, h / sqrt(mean_k h^2 + eps), rounded to bf16:
    constant rows small enough that eps changes the result, a row with one
    non-zero channel (the mean is over d, not a sum), a sign-symmetric pair
    of rows, and eps = 0 giving unit RMS."""
    d = 512
    # c = 1e-3: c / sqrt(c^2 + 1e-5) ~ 0.3015 (1.0 without eps, 0.990 with
    # eps added outside the square root)
    for c, eps in ((1e-3, 1e-5), (0.1, 1e-2), (3e-3, 1e-5)):
        h = np.full((2, d), c, dtype=np.float32)
        h[1] = -h[1]
        out = rmsnorm_bf16(h, eps)
        vals = ((np.asarray(out, np.uint16).astype(np.uint32) << 16).view(np.float32)
                .astype(np.float64))
        want = _exact_bf16_of(np.float32(c), eps, d, d)
        assert Fraction(float(vals[0, 0])) == want, (c, eps, vals[0, 0], float(want))
        assert (vals[0] == vals[0, 0]).all() and (vals[1] == -vals[0]).all()
    # one non-zero channel of d: 1 / sqrt(1/512 + 1e-5) ~ 22.57
    h = np.zeros((1, d), dtype=np.float32)
    h[0, 17] = 1.0
    vals = ((np.asarray(rmsnorm_bf16(h, 1e-5), np.uint16).astype(np.uint32) << 16)
            .view(np.float32).astype(np.float64))
    assert Fraction(float(vals[0, 17])) == _exact_bf16_of(1.0, 1e-5, 1, d)
    assert not np.delete(vals[0], 17).any()
    # eps = 0: unit root mean square, to the bf16 rounding of each element
    rng = np.random.default_rng(2)
    h = (rng.standard_normal((4, 1024)) * 5).astype(np.float32)
    y = ((np.asarray(rmsnorm_bf16(h, 0.0), np.uint16).astype(np.uint32) << 16)
         .view(np.float32).astype(np.float64))
    np.testing.assert_allclose(np.mean(y * y, axis=1), 1.0, rtol=2e-3)


# ---------------------------------------------------------------- per-group scales

def check_per_group_scales(qlinear_ref, unpack_codes):
    """x W_dq^T with a scale of its own for every (column, group): powers of
    two 2^-e[n][g] applied to integer group sums of ternary x and uniform
    codes, summed exactly in rationals.  A scale taken from the wrong column
    or group, or a transposed operand, fails."""
    rng = np.random.default_rng(3)
    M, N, K = 5, 6, 512
    G = K // 128
    xi = rng.integers(-1, 2, (M, K))
    x_bits = np.where(xi == 1, 0x3F80, np.where(xi == -1, 0xBF80, 0)).astype(np.uint16)
    qw = rng.integers(0, 256, (N, K // 2), dtype=np.uint8)
    e = rng.integers(2, 7, (N, G))
    sc = (0x3C00 - (e << 10)).astype(np.uint16)
    # codes straight from the nibbles (two's complement, even k low)
    lo = (qw & 0xF).astype(np.int64)
    hi = (qw >> 4).astype(np.int64)
    q = np.empty((N, K), dtype=np.int64)
    q[:, 0::2] = np.where(lo >= 8, lo - 16, lo)
    q[:, 1::2] = np.where(hi >= 8, hi - 16, hi)
    np.testing.assert_array_equal(unpack_codes(qw), q)
    y = qlinear_ref(x_bits, qw, sc)
    for m in range(M):
        for n in range(N):
            exact = sum(Fraction(int(xi[m, 128 * g:128 * (g + 1)] @ q[n, 128 * g:128 * (g + 1)]),
                                 2 ** int(e[n, g])) for g in range(G))
            assert Fraction(float(y[m, n])) == exact, (m, n)
