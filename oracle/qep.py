"""Propagation-corrected target (App. E.5), float64 (test oracle).

TEST INFRASTRUCTURE ONLY: used by the tests; never by the product path.

The mixed target Y*(mu) = (1 - mu) X W + mu X~ W (eq. (mu-target)) keeps the
design A = [X~; nu I]; its least-squares solution over real matrices is
eq. (w-corr), W_corr = W + (1 - mu) H^{-1} X~^T (X - X~) W with
H = X~^T X~ + nu^2 I, in the paper's orientation (W: input channels x output
channels).  Functions here take W with rows as output channels and return
W_corr the same way.
"""

from __future__ import annotations

import numpy as np


def cross(chunks_q, chunks_x, d, alpha=1.0):
    """alpha sum_c X~_c^T (X_c - X~_c), float64."""
    D = np.zeros((d, d))
    for Xq, X in zip(chunks_q, chunks_x):
        Xq = np.asarray(Xq, np.float64)
        D += alpha * (Xq.T @ (np.asarray(X, np.float64) - Xq))
    return D


def corrected_weights(W, H, D, mu):
    """Eq. (w-corr) with W [rows = output channels, cols = input channels]."""
    Wp = np.asarray(W, np.float64).T                     # the paper's W: cols x rows
    corr = np.linalg.solve(np.asarray(H, np.float64), np.asarray(D, np.float64) @ Wp)
    return (Wp + (1.0 - mu) * corr).T


__all__ = ["cross", "corrected_weights"]
