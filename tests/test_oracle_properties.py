"""Property tests of the float64 oracle on random small shapes (hypothesis):
facts that hold for any weights, so a plausible slip in the oracle (a
transposed factor, a wrong head-to-group map, a dropped normalisation)
fails one of them.  CPU only."""

import math

import numpy as np
from hypothesis import given, settings, strategies as st

from oracle import explicit, fp8_consumer
from oracle.power_iteration import power_iteration, power_iteration_layer, spectral_step

SETTINGS = settings(max_examples=60, deadline=None)


def _rng(seed):
    return np.random.default_rng(seed)


@SETTINGS
@given(d=st.integers(2, 48), dh=st.integers(1, 12), n_iter=st.integers(1, 15), seed=st.integers(0, 2**31 - 1))
def test_estimate_is_a_nondecreasing_lower_bound(d, dh, n_iter, seed):
    """sigma_k = ||M v_{k-1}|| is the square root of a Rayleigh quotient of
    M^T M along the power sequence: non-decreasing in k and at most sigma_1
    (App. E); sigma_1 <= ||W^Q|| ||W^K|| (Cor. "Interaction bound is
    tighter")."""
    rng = _rng(seed)
    WQ, WK = rng.standard_normal((d, dh)), rng.standard_normal((d, dh))
    r = power_iteration(WQ, WK, rng.standard_normal(d), n_iter)
    s1 = explicit.singular_values(explicit.interaction_matrix(WQ, WK))[0]
    h = np.asarray(r.history)
    assert len(h) == n_iter and r.iters == n_iter
    assert np.all(np.diff(h) >= -1e-10 * s1)
    assert r.sigma <= s1 * (1 + 1e-10)
    assert s1 <= explicit.spectral_norm(WQ) * explicit.spectral_norm(WK) * (1 + 1e-10)
    # the QR route to sigma_1 agrees with the SVD of the formed matrix
    assert abs(explicit.sigma_max_reduced(WQ, WK)[0] - s1) <= 1e-10 * s1


@SETTINGS
@given(d=st.integers(2, 40), dh=st.integers(1, 8), n_kv=st.integers(1, 3), g=st.integers(1, 4),
       n_iter=st.integers(1, 8), seed=st.integers(0, 2**31 - 1))
def test_grouped_heads_equal_explicit_key_expansion(d, dh, n_kv, g, n_iter, seed):
    """Prop. "Implicit GQA power iteration": query head h with key head
    floor(h / g) gives the very iterates of multi-head attention on the
    key weights repeated per group."""
    rng = _rng(seed)
    n_q = n_kv * g
    wq = rng.standard_normal((2, n_q * dh, d))
    wk = rng.standard_normal((2, n_kv * dh, d))
    wk_exp = np.stack([np.repeat(w.reshape(n_kv, dh, d), g, axis=0).reshape(n_q * dh, d) for w in wk])
    v0 = rng.standard_normal((2, n_q, d))
    a = spectral_step(wq, wk, v0, n_iter, n_kv=n_kv, head_dim=dh, alpha=0.02)
    b = spectral_step(wq, wk_exp, v0, n_iter, n_kv=n_q, head_dim=dh, alpha=0.02)
    np.testing.assert_array_equal(a["sigma"], b["sigma"])
    np.testing.assert_array_equal(a["scale"], b["scale"])


@SETTINGS
@given(d=st.integers(2, 32), dh=st.integers(1, 8), n_tok=st.integers(1, 12), seed=st.integers(0, 2**31 - 1))
def test_logits_obey_the_interaction_bound_with_equality_on_singular_vectors(d, dh, n_tok, seed):
    """Prop. "Interaction bound": |S_ij| <= sigma_1 ||x_i|| ||x_j|| / sqrt(d_h)
    for the consumer's logits, with equality for x_i = u_1, x_j = v_1, the top
    singular pair of the M the estimator iterates on."""
    rng = _rng(seed)
    wq, wk = rng.standard_normal((dh, d)), rng.standard_normal((dh, d))
    M = explicit.interaction_matrix(wq.T, wk.T)
    U, s, Vt = np.linalg.svd(M)
    x = np.vstack([rng.standard_normal((n_tok, d)), U[:, 0], Vt[0]])
    S = fp8_consumer.head_logits(x, wq, wk, 0, 1, dh)
    n = np.linalg.norm(x, axis=1)
    assert np.all(np.abs(S) <= s[0] * np.outer(n, n) / math.sqrt(dh) * (1 + 1e-10) + 1e-300)
    assert abs(S[n_tok, n_tok + 1] - s[0] / math.sqrt(dh)) <= 1e-10 * s[0]
    # and the estimator converges to that sigma_1 when the gap allows it
    r = power_iteration(wq.T, wk.T, Vt[0] + 1e-3 * rng.standard_normal(d), 200, tol=1e-14)
    if len(s) < 2 or s[1] < 0.9 * s[0]:
        assert abs(r.sigma - s[0]) <= 1e-8 * s[0]


@SETTINGS
@given(d=st.integers(2, 40), dh=st.integers(1, 8), a=st.integers(-6, 6), b=st.integers(-6, 6),
       n_iter=st.integers(1, 10), seed=st.integers(0, 2**31 - 1))
def test_power_of_two_scaling_is_exact(d, dh, a, b, n_iter, seed):
    """sigma(2^a W^Q, 2^b W^K) = 2^(a + b) sigma(W^Q, W^K) bit for bit: the
    estimate is homogeneous and carries no hidden state (App. H spike test)."""
    rng = _rng(seed)
    WQ, WK, v0 = rng.standard_normal((d, dh)), rng.standard_normal((d, dh)), rng.standard_normal(d)
    r0 = power_iteration(WQ, WK, v0, n_iter)
    r1 = power_iteration(WQ * 2.0 ** a, WK * 2.0 ** b, v0, n_iter)
    assert r1.sigma == r0.sigma * 2.0 ** (a + b)


@SETTINGS
@given(d=st.integers(2, 40), dh=st.integers(1, 8), n_iter=st.integers(1, 10), seed=st.integers(0, 2**31 - 1))
def test_layer_form_of_one_head_is_the_head_form(d, dh, n_iter, seed):
    """With one query and one key head the layer-level estimator (App. E,
    "Implicit GQA Power Iteration") is the per-head one."""
    rng = _rng(seed)
    WQ, WK, v0 = rng.standard_normal((d, dh)), rng.standard_normal((d, dh)), rng.standard_normal(d)
    a = power_iteration(WQ, WK, v0, n_iter)
    b = power_iteration_layer(WQ, WK, v0, n_iter, 1, dh)
    assert a.sigma == b.sigma
    np.testing.assert_array_equal(a.v, b.v)
