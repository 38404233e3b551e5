"""The oracle's pins reject plausible mistakes (CPU only).

Each test plants one mistake in a copy of an oracle function (a dropped
square root, eps in the wrong place, a scale read from the neighbouring
group, swapped nibbles, ...) and checks that the pin check which the real
oracle passes (tests/test_oracle_pins.py) fails on it.
"""
import numpy as np
import pytest

import oracle as O
from tests.oracle_checks import check_per_group_scales, check_rel_fro, check_rmsnorm


# ---------------------------------------------------------------- rel_fro

def _rf_no_sqrt(y, ref):
    y, ref = np.asarray(y, np.float64), np.asarray(ref, np.float64)
    den = np.sum(ref * ref)
    return float(np.sum((y - ref) ** 2) / den) if den > 0 else float(np.sum((y - ref) ** 2))


def _rf_den_of_y(y, ref):
    y, ref = np.asarray(y, np.float64), np.asarray(ref, np.float64)
    den = np.linalg.norm(y)
    return float(np.linalg.norm(y - ref) / den) if den > 0 else float(np.linalg.norm(y - ref))


def _rf_max_norm(y, ref):
    y, ref = np.asarray(y, np.float64), np.asarray(ref, np.float64)
    den = np.abs(ref).max()
    return float(np.abs(y - ref).max() / den) if den > 0 else float(np.abs(y - ref).max())


def _rf_row_mean(y, ref):
    y, ref = np.atleast_2d(np.asarray(y, np.float64)), np.atleast_2d(np.asarray(ref, np.float64))
    num = np.linalg.norm(y - ref, axis=-1)
    den = np.linalg.norm(ref, axis=-1)
    with np.errstate(invalid="ignore", divide="ignore"):
        r = np.where(den > 0, num / np.where(den > 0, den, 1), num)
    return float(r.mean())


def _rf_zero_ref_is_zero(y, ref):
    den = np.linalg.norm(np.asarray(ref, np.float64))
    return O.rel_fro(y, ref) if den > 0 else 0.0


@pytest.mark.parametrize("mutant", [_rf_no_sqrt, _rf_den_of_y, _rf_max_norm, _rf_row_mean,
                                    _rf_zero_ref_is_zero])
def test_rel_fro_pins_reject(mutant):
    with pytest.raises(AssertionError):
        check_rel_fro(mutant)


# ---------------------------------------------------------------- RMSNorm

def _rms(h, eps, how):
    h = np.asarray(h, dtype=np.float64)
    ms = np.mean(h * h, axis=-1, keepdims=True)
    if how == "no_eps":
        r = 1.0 / np.sqrt(ms)
    elif how == "eps_outside":
        r = 1.0 / (np.sqrt(ms) + eps)
    elif how == "sum":
        r = 1.0 / np.sqrt(np.sum(h * h, axis=-1, keepdims=True) + eps)
    elif how == "eps_squared":
        r = 1.0 / np.sqrt(ms + eps * eps)
    elif how == "eps_over_d":
        r = 1.0 / np.sqrt(ms + eps / h.shape[-1])
    else:
        raise ValueError(how)
    with np.errstate(divide="ignore", invalid="ignore"):
        return O.f64_to_bf16_bits(h * r)


@pytest.mark.parametrize("how", ["no_eps", "eps_outside", "sum", "eps_squared", "eps_over_d"])
def test_rmsnorm_pins_reject(how):
    with pytest.raises(AssertionError):
        check_rmsnorm(lambda h, eps: _rms(h, eps, how))


# ---------------------------------------------------------------- scale indexing

def _ref_next_group(x, qw, sc, group=128):
    return O.qlinear_ref(x, qw, np.roll(sc, 1, axis=1), group)


def _ref_next_column(x, qw, sc, group=128):
    return O.qlinear_ref(x, qw, np.roll(sc, 1, axis=0), group)


def _ref_group_of_k_mod(x, qw, sc, group=128):
    """scale index k mod G instead of k // 128"""
    q = O.unpack_codes(qw).astype(np.float64)
    s = O.f16_bits_to_f32(sc).astype(np.float64)
    N, K = q.shape
    G = K // group
    w = q * s[:, np.arange(K) % G]
    return O.bf16_bits_to_f64(x) @ w.T


def _unpack_swapped(qweight):
    q = O.unpack_codes(qweight)
    out = q.copy()
    out[:, 0::2], out[:, 1::2] = q[:, 1::2], q[:, 0::2]
    return out


@pytest.mark.parametrize("mutant", [_ref_next_group, _ref_next_column, _ref_group_of_k_mod])
def test_per_group_scale_pins_reject(mutant):
    with pytest.raises(AssertionError):
        check_per_group_scales(mutant, O.unpack_codes)


def test_nibble_order_pin_rejects_swapped_nibbles():
    with pytest.raises(AssertionError):
        check_per_group_scales(O.qlinear_ref, _unpack_swapped)
