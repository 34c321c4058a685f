"""Cross-checks that form the interaction matrix explicitly (test
infrastructure only).  This is the O(d^2)-memory route the method avoids
(Sec. 4.1 contrasts it with the implicit products); it serves as an
independent check of ``oracle.power_iteration``.
"""

from __future__ import annotations

import numpy as np


def interaction_matrix(WQ: np.ndarray, WK: np.ndarray) -> np.ndarray:
    """M = W^Q W^{K T} in R^{d x d} (Eq. "bilinear"), float64."""
    return np.asarray(WQ, dtype=np.float64) @ np.asarray(WK, dtype=np.float64).T


def dense_power_iteration(M: np.ndarray, v0: np.ndarray, n_iter: int, tol: float = 0.0):
    """Textbook power iteration for the top singular value of a formed matrix
    (Golub & Van Loan): w = M v, sigma = ||w||, u = w / sigma,
    v = M^T u / ||M^T u||.  Same stopping rule as the implicit oracle.
    Returns (sigma, u, v, iters)."""
    v = np.asarray(v0, dtype=np.float64)
    v = v / np.linalg.norm(v)
    sigma_prev = None
    sigma, u = float("nan"), None
    for k in range(1, n_iter + 1):
        w = M @ v
        sigma = float(np.linalg.norm(w))
        u = w / sigma
        t = M.T @ u
        v = t / np.linalg.norm(t)
        if tol > 0.0 and k >= 2 and abs(sigma - sigma_prev) <= tol * sigma:
            return sigma, u, v, k
        sigma_prev = sigma
    return sigma, u, v, n_iter


def singular_values(M: np.ndarray) -> np.ndarray:
    """All singular values of a formed matrix (LAPACK gesdd), descending."""
    return np.linalg.svd(M, compute_uv=False)


def sigma_max_reduced(WQ: np.ndarray, WK: np.ndarray) -> np.ndarray:
    """Singular values of W^Q W^{K T} without forming it: with thin QR
    W^Q = Q_A R_A and W^K = Q_B R_B, M = Q_A (R_A R_B^T) Q_B^T and the
    orthonormal factors leave the singular values of the d_h x d_h core
    unchanged.  Returns them descending."""
    _, ra = np.linalg.qr(np.asarray(WQ, dtype=np.float64))
    _, rb = np.linalg.qr(np.asarray(WK, dtype=np.float64))
    return np.linalg.svd(ra @ rb.T, compute_uv=False)


def spectral_norm(A: np.ndarray) -> float:
    """||A||_2 of a single factor (for the submultiplicative bound)."""
    return float(np.linalg.svd(np.asarray(A, dtype=np.float64), compute_uv=False)[0])
