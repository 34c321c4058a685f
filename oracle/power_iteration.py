"""The estimator, step by step, in float64 (test infrastructure only).

Notation follows the paper (Sec. 4.1 and App. E): for one attention head the
query and key slices are W^Q, W^K in R^{d x d_h}, the interaction matrix is
M = W^Q W^{K T} in R^{d x d}, and one power-iteration step is

    z  = W^{K T} v          u' = W^Q z  (= M v)        sigma = ||u'||
    u  = u' / sigma
    y  = W^{Q T} u          v' = W^K y  (= M^T u)      v = v' / ||v'||

The returned estimate is the sigma of the last step (taken before v moves).
M is never formed here either; ``oracle.explicit`` forms it for the pins.

Readings of points the paper leaves open (each listed in the design notes):

* Per-head: sigma_h = ||W^Q_h W^{K T}_{g(h)}||_2 for every query head h, with
  g(h) = floor(h / g), g = n_q / n_kv (App. F maps KV block i to query blocks
  (i-1)g+1 .. ig, 1-based).  The per-layer sigma of Eq. "scale" is the
  maximum over the layer's heads, since each head's logits obey the
  interaction bound with its own sigma_h.
* n_iter counts estimates of sigma; the result is the n_iter-th.
* Convergence (tol > 0): stop after step k when k >= 2 and
  |sigma_k - sigma_{k-1}| <= tol * sigma_k, at most n_iter steps.
* Degenerate inputs: a start vector of norm 0 or with a non-finite entry gives
  sigma = NaN, iters = -1, v unchanged; M v = 0 gives sigma = 0, iters = -2,
  v = the normalised start vector; u is zero in both cases.
* Build layout: a layer's weights are stored as ``wq [n_q*d_h, d]``,
  ``wk [n_kv*d_h, d]`` (rows of head h = (W^Q_h)^T); ``head_slices`` turns
  them into the paper's orientation.
"""

from __future__ import annotations

from dataclasses import dataclass, field

import numpy as np


@dataclass
class HeadResult:
    sigma: float
    u: np.ndarray
    v: np.ndarray
    iters: int
    history: list = field(default_factory=list)   # sigma_1 .. sigma_iters


def head_slices(wq_layer, wk_layer, h: int, n_kv: int, head_dim: int):
    """W^Q_h and W^K_{g(h)} in R^{d x d_h} (float64) from build-layout rows."""
    wq_layer = np.asarray(wq_layer)
    wk_layer = np.asarray(wk_layer)
    n_q = wq_layer.shape[0] // head_dim
    g = n_q // n_kv
    j = h // g
    WQ = np.asarray(wq_layer[h * head_dim:(h + 1) * head_dim], dtype=np.float64).T
    WK = np.asarray(wk_layer[j * head_dim:(j + 1) * head_dim], dtype=np.float64).T
    return WQ, WK


def power_iteration(WQ: np.ndarray, WK: np.ndarray, v0: np.ndarray, n_iter: int,
                    tol: float = 0.0) -> HeadResult:
    """Power iteration for ||W^Q W^{K T}||_2 of one head (App. E, first algorithm)."""
    v0 = np.asarray(v0, dtype=np.float64)
    d = WQ.shape[0]
    nv = float(np.linalg.norm(v0))
    if not np.all(np.isfinite(v0)) or nv == 0.0:
        return HeadResult(float("nan"), np.zeros(d), v0.copy(), -1)
    v = v0 / nv
    u = np.zeros(d)
    sigma_prev = None
    sigma = float("nan")
    history = []
    for k in range(1, n_iter + 1):
        z = WK.T @ v
        u_p = WQ @ z
        sigma = float(np.linalg.norm(u_p))
        if sigma == 0.0:
            return HeadResult(0.0, np.zeros(d), v0 / nv, -2, history)
        history.append(sigma)
        u = u_p / sigma
        y = WQ.T @ u
        v_p = WK @ y
        v = v_p / np.linalg.norm(v_p)
        if tol > 0.0 and k >= 2 and abs(sigma - sigma_prev) <= tol * sigma:
            return HeadResult(sigma, u, v, k, history)
        sigma_prev = sigma
    return HeadResult(sigma, u, v, n_iter, history)


def repeat_blocks(z_kv: np.ndarray, g: int, head_dim: int) -> np.ndarray:
    """RepeatBlocks(z, g): each d_h block of z in R^{n_kv d_h} repeated g times."""
    blocks = z_kv.reshape(-1, head_dim)
    return np.repeat(blocks, g, axis=0).reshape(-1)


def sum_groups(y: np.ndarray, g: int, head_dim: int) -> np.ndarray:
    """SumGroups(y, g): sums every run of g consecutive d_h blocks of y."""
    blocks = y.reshape(-1, g, head_dim)
    return blocks.sum(axis=1).reshape(-1)


def power_iteration_layer(WQ: np.ndarray, WK: np.ndarray, v0: np.ndarray, n_iter: int,
                          g: int, head_dim: int) -> HeadResult:
    """The paper-literal layer-level estimator (App. E, "Implicit GQA Power
    Iteration"; g = 1 is the MHA algorithm): W^Q in R^{d x n_q d_h},
    W^K in R^{d x n_kv d_h}, one pair u, v in R^d for the whole layer."""
    v = np.asarray(v0, dtype=np.float64)
    v = v / np.linalg.norm(v)
    sigma = float("nan")
    u = np.zeros_like(v)
    for _ in range(n_iter):
        z_kv = WK.T @ v
        z = repeat_blocks(z_kv, g, head_dim)
        u_p = WQ @ z
        sigma = float(np.linalg.norm(u_p))
        u = u_p / sigma
        y = WQ.T @ u
        y_kv = sum_groups(y, g, head_dim)
        v_p = WK @ y_kv
        v = v_p / np.linalg.norm(v_p)
    return HeadResult(sigma, u, v, n_iter)


def layer_scale(sigma_layer, alpha: float, d: int, head_dim: int, eta_fp8: float = 0.8,
                r_max: float = 448.0):
    """Eq. "scale": alpha * sigma^(l) * (d / sqrt(d_h)) / (eta_fp8 * R_max)."""
    return alpha * np.asarray(sigma_layer, dtype=np.float64) * (d / np.sqrt(head_dim)) / (eta_fp8 * r_max)


def spectral_step(wq_layers, wk_layers, v_in, n_iter: int, *, n_kv: int, head_dim: int,
                  alpha: float, eta_fp8: float = 0.8, r_max: float = 448.0, tol: float = 0.0,
                  heads=None, want_u: bool = False) -> dict:
    """All heads (or the listed (layer, head) pairs) of all layers.

    wq_layers: [L][n_q*d_h, d], wk_layers: [L][n_kv*d_h, d] (any float type,
    bf16 values already widened exactly); v_in: [L, n_q, d].
    Returns sigma [L, n_q], scale [L] (NaN for a layer whose heads were not all
    computed), v [L, n_q, d], u [L, n_q, d] (if want_u), iters [L, n_q].
    """
    v_in = np.asarray(v_in)
    L, n_q, d = v_in.shape
    sigma = np.full((L, n_q), np.nan)
    iters = np.zeros((L, n_q), dtype=np.int64)
    v_out = np.array(v_in, dtype=np.float64, copy=True)
    u_out = np.zeros((L, n_q, d)) if want_u else None
    done = np.zeros((L, n_q), dtype=bool)
    todo = [(l, h) for l in range(L) for h in range(n_q)] if heads is None else list(heads)
    for (l, h) in todo:
        WQ, WK = head_slices(wq_layers[l], wk_layers[l], h, n_kv, head_dim)
        r = power_iteration(WQ, WK, v_in[l, h], n_iter, tol)
        sigma[l, h] = r.sigma
        iters[l, h] = r.iters
        v_out[l, h] = r.v
        if want_u:
            u_out[l, h] = r.u
        done[l, h] = True
    scale = np.full(L, np.nan)
    for l in range(L):
        if done[l].all():
            scale[l] = layer_scale(np.max(sigma[l]) if not np.isnan(sigma[l]).any() else np.nan,
                                   alpha, d, head_dim, eta_fp8, r_max)
    out = {"sigma": sigma, "scale": scale, "v": v_out, "iters": iters}
    if want_u:
        out["u"] = u_out
    return out
