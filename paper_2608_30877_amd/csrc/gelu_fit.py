"""Derivation of the constants of gelu_erf (ql_device.h).

GELU(z) = z Phi(z).  The normal tail Q(x) = 1 - Phi(x), x >= 0, is written in
the form of Abramowitz & Stegun 26.2.17,

    Q(x) = phi(x) * s * (c1 + c2 s + ... + c7 s^6),   s = 1 / (1 + p x),

with phi the normal density.  p and c1..c7 are fitted here to the Mills ratio
Q / phi for RELATIVE error on x in [0, 13.5] (Lawson's iteratively reweighted
least squares towards the minimax fit, p by a 1-D search), so that the tail
keeps its relative accuracy.  1 / sqrt(2 pi) is folded into the printed
coefficients.  The fp32 evaluation the kernels run (v_rcp_f32, Horner,
v_exp_f32 scaled by 2^24) is then emulated and its relative error printed.

Usage: python paper_2608_30877_amd/csrc/gelu_fit.py   (needs numpy, scipy)
"""
import numpy as np
from scipy.optimize import minimize
from scipy.special import erfc

X = np.concatenate([np.linspace(0, 4, 40001), np.linspace(4, 13.5, 20001)])
MILLS = 0.5 * erfc(X / np.sqrt(2)) / (np.exp(-0.5 * X * X) / np.sqrt(2 * np.pi))
N_TERMS = 7


def lawson(p, n, iters):
    s = 1.0 / (1.0 + p * X)
    A = np.stack([s ** (k + 1) for k in range(n)], 1) / MILLS[:, None]
    w = np.full(len(X), 1.0 / len(X))
    for _ in range(iters):
        sw = np.sqrt(w)
        c, *_ = np.linalg.lstsq(A * sw[:, None], sw, rcond=None)
        w = w * np.abs(A @ c - 1)
        w /= w.sum()
    return c, np.abs(A @ c - 1).max()


def gelu_fp32(z, p, coef):
    f = np.float32
    z = z.astype(f)
    a = np.abs(z)
    s = (f(1) / (f(p) * a + f(1))).astype(f)
    r = f(coef[-1])
    for c in coef[-2::-1]:
        r = (r * s + f(c)).astype(f)
    r = (r * s).astype(f)
    e = np.exp2((a * a * f(-0.5 / np.log(2.0)) + f(24)).astype(f)).astype(f)
    e = np.where(e < f(2.0 ** -126), f(0), e)          # the hardware exp2 has no subnormals
    q = (e * r).astype(f)
    pos = (z * (f(1) - (q * f(2.0 ** -24)).astype(f))).astype(f)
    neg = ((z * q).astype(f) * f(2.0 ** -24)).astype(f)
    return np.where(z >= 0, pos, neg)


def main():
    res = minimize(lambda q: lawson(q[0], N_TERMS, 30)[1], [0.33], method="Nelder-Mead",
                   options={"xatol": 1e-6, "fatol": 1e-13, "maxiter": 60})
    p = float(res.x[0])
    c, err = lawson(p, N_TERMS, 120)
    coef = [float(np.float32(v / np.sqrt(2 * np.pi))) for v in c]
    print(f"p = {np.float32(p)!r}, max relative error of the fit {err:.2e}")
    for i, v in enumerate(coef):
        print(f"c{i + 1} = {v:.9e}")
    z = np.linspace(-14, 14, 2_000_001)
    exact = 0.5 * z * erfc(-z / np.sqrt(2))
    got = gelu_fp32(z, p, coef).astype(np.float64)
    m = np.abs(exact) > 1e-30
    rel = np.abs(got - exact)[m] / np.abs(exact[m])
    print(f"fp32 evaluation: max relative error {rel.max():.2e} over |z| <= 14, "
          f"{rel[np.abs(z[m]) < 6].max():.2e} for |z| < 6")


if __name__ == "__main__":
    main()
