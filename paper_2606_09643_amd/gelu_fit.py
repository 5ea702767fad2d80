"""Derivation of the GELU polynomial used for bf16 outputs (gelu_fast in
csrc/vfm_internal.h).

GELU(x) = x Phi(x), Phi the standard normal CDF.  On |x| <= 4 the odd part
Phi(x) - 1/2 is fitted as (x/4) P((x/4)^2), P with 8 terms, by weighted least
squares with Lawson's iterative reweighting (a near-minimax fit) on Chebyshev
nodes; outside the range x is clamped to +-4, where Phi is within 3.2e-5 of
0 or 1.  The kernel uses Q_j = c_j / 4^(2j+1) so that s(x) = x Q(x^2).

Run: ``python -m paper_2606_09643_amd.gelu_fit`` prints the coefficients and
the error bound of the float32 evaluation.
"""
from __future__ import annotations

import numpy as np

CLAMP = 4.0
TERMS = 8


def _phi(x):
    from scipy.special import erf
    return 0.5 * (1.0 + erf(x / np.sqrt(2.0)))


def fit(n: int = TERMS, c: float = CLAMP, iters: int = 200) -> np.ndarray:
    """Coefficients c_j of Phi(x) - 1/2 ~ (x/c) sum_j c_j ((x/c)^2)^j."""
    k = np.arange(20000)
    x = np.abs(np.cos(np.pi * (k + 0.5) / 20000)) * c
    x = x[x > 1e-9]
    u = (x / c) ** 2
    A = np.stack([x / c * u ** j for j in range(n)], 1)
    y = _phi(x) - 0.5
    w = np.ones_like(x)
    coef = None
    for _ in range(iters):
        coef, *_ = np.linalg.lstsq(A * w[:, None], y * w, rcond=None)
        err = np.abs(A @ coef - y)
        w = w * (err / err.max() + 1e-4) ** 0.5
        w /= w.max()
    return coef


def kernel_coefficients(coef: np.ndarray, c: float = CLAMP) -> np.ndarray:
    """Q_j = c_j / c^(2j+1): s(x) = x Q(x^2) with x clamped to [-c, c]."""
    return np.array([coef[j] / c ** (2 * j + 1) for j in range(len(coef))])


if __name__ == "__main__":
    q = kernel_coefficients(fit())
    for j, v in enumerate(q):
        print(f"Q{j} = {np.float32(v)!r}")
