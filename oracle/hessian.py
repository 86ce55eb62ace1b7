"""Calibration Hessian of the layer objective, float64 (test oracle).

TEST INFRASTRUCTURE ONLY: used by the tests and the smoke check; never by the
product path.

The objective eq. (4) is written with the stacked design A = [X~; nu I]
(App. E.1), so its Hessian is the plain definition H = A^T A = X~^T X~ + nu^2 I.
Calibration inputs arrive in chunks of tokens; over chunks X_c the sum
alpha sum_c X_c^T X_c is accumulated, and the finished matrix adds
(damp mean(diag) + nu^2) I.  damp = 0 is the paper's matrix; damp > 0 is the
relative diagonal damping of GPTQ-style pipelines, used by the synthetic
layers (XX^T / n + 0.01 mean(diag) I).
"""

from __future__ import annotations

import numpy as np


def accumulate(Hacc, X, alpha=1.0):
    """Hacc + alpha X^T X in float64 (X [m, d] tokens x channels)."""
    X = np.asarray(X, dtype=np.float64)
    return np.asarray(Hacc, dtype=np.float64) + alpha * (X.T @ X)


def finalize(Hacc, damp=0.0, nu2=0.0):
    """Hacc + (damp mean(diag Hacc) + nu2) I, float64."""
    H = np.array(Hacc, dtype=np.float64, copy=True)
    d = H.shape[0]
    H[np.arange(d), np.arange(d)] += damp * np.mean(np.diag(Hacc)) + nu2
    return H


def hessian(chunks, d, alpha=1.0, damp=0.0, nu2=0.0):
    """finalize(sum over chunks of alpha X_c^T X_c)."""
    Hacc = np.zeros((d, d))
    for X in chunks:
        Hacc = accumulate(Hacc, X, alpha)
    return finalize(Hacc, damp, nu2)


def entry(cols_a, cols_b, alpha=1.0):
    """One entry alpha sum_t x_ta x_tb from the two channel columns."""
    return alpha * float(np.dot(np.asarray(cols_a, np.float64), np.asarray(cols_b, np.float64)))


def fp32_error_bound(absgram, alpha, segment=256):
    """Bound on |H_fp32path - H| entrywise for a path that rounds each product
    to fp32, sums at most `segment` of them in fp32, adds those partial sums in
    float64 and rounds once to fp32: (segment + 1) u |alpha| (|X|^T |X|) plus
    the final rounding, u = 2^-24 (standard recursive-summation bound,
    gamma_n <= n u / (1 - n u))."""
    u = 2.0 ** -24
    n = segment + 1
    return (n * u / (1.0 - n * u)) * abs(alpha) * absgram


__all__ = ["accumulate", "finalize", "hessian", "entry", "fp32_error_bound"]
