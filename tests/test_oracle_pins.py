"""Pins of the float64 oracle against what the paper and the mathematics fix:
closed forms, textbook routines, printed values and invariants.  CPU only."""

import math

import numpy as np
import pytest
import torch

from conftest import read_golden
from oracle import calibration, e4m3, explicit
from oracle.power_iteration import (
    head_slices,
    layer_scale,
    power_iteration,
    power_iteration_layer,
    spectral_step,
)
from workloads import WORKLOADS, all_weights, bf16_round, layer_weights, planted_singular_values, start_vectors, tokens


def _orth(rng, n, k):
    q, _ = np.linalg.qr(rng.standard_normal((n, k)))
    return q


def _rel(a, b):
    return abs(a - b) / abs(b)


# ---------------------------------------------------------------- P1 planted


def _closed_form_sigma(s, c, k):
    """sigma_est(k) for M = U diag(s) V^T, c = V^T v0:  ||s o c|| at k = 1,
    ||s^(2k-1) o c|| / ||s^(2k-2) o c|| afterwards."""
    if k == 1:
        return np.linalg.norm(s * c)
    t = s / s.max()
    return s.max() * np.linalg.norm(t ** (2 * k - 1) * c) / np.linalg.norm(t ** (2 * k - 2) * c)


@pytest.mark.parametrize("d,dh", [(40, 6), (257, 16)])
def test_planted_spectrum_closed_form(d, dh):
    rng = np.random.default_rng(7)
    U, V = _orth(rng, d, dh), _orth(rng, d, dh)
    s = np.sort(rng.uniform(0.5, 3.0, dh))[::-1]
    WQ, WK = U * s, V.copy()                       # W^Q = U diag(s), W^K = V
    v0 = rng.standard_normal(d)
    v0 /= np.linalg.norm(v0)
    c = V.T @ v0
    for k in (1, 2, 3, 7, 20):
        r = power_iteration(WQ, WK, v0, k)
        assert r.iters == k
        assert _rel(r.sigma, _closed_form_sigma(s, c, k)) < 1e-12
        # v_k is along V (s^(2k) o c)
        vk = V @ (s ** (2 * k) * c)
        assert abs(abs(vk @ r.v) / np.linalg.norm(vk) - 1.0) < 1e-12
        # u_k is along U (s^(2k-1) o c)
        uk = U @ (s ** (2 * k - 1) * c)
        assert abs(abs(uk @ r.u) / np.linalg.norm(uk) - 1.0) < 1e-12


def test_stopping_rule_matches_closed_form_sequence():
    rng = np.random.default_rng(11)
    d, dh = 64, 8
    U, V = _orth(rng, d, dh), _orth(rng, d, dh)
    s = np.array([2.0, 1.9, 1.5, 1.0, 0.7, 0.5, 0.2, 0.1])
    v0 = rng.standard_normal(d)
    v0 /= np.linalg.norm(v0)
    c = V.T @ v0
    tol = 1e-6
    seq = [_closed_form_sigma(s, c, k) for k in range(1, 400)]
    k_expect = next(k for k in range(2, 400) if abs(seq[k - 1] - seq[k - 2]) <= tol * seq[k - 1])
    r = power_iteration(U * s, V, v0, 1000, tol=tol)
    assert r.iters == k_expect
    assert _rel(r.sigma, seq[k_expect - 1]) < 1e-12


@pytest.mark.parametrize("d,dh,nq,nkv", [(32, 8, 4, 2), (256, 16, 4, 1)])
def test_planted_hadamard_is_bf16_exact(d, dh, nq, nkv):
    wl = WORKLOADS["llama2-70b-perstep"].replace(n_layers=1, d_model=d, head_dim=dh, n_q=nq, n_kv=nkv)
    wq, wk = layer_weights(wl, 0)
    wq32, wk32 = wq.float(), wk.float()
    assert torch.equal(bf16_round(wq32), wq32) and torch.equal(bf16_round(wk32), wk32)
    sv = planted_singular_values(wl, 0)
    for h in range(nq):
        WQ, WK = head_slices(wq32.numpy(), wk32.numpy(), h, nkv, dh)
        got = explicit.singular_values(explicit.interaction_matrix(WQ, WK))[:dh]
        np.testing.assert_allclose(got, np.sort(sv[h])[::-1], rtol=1e-12)
        assert sv[h][1] / sv[h][0] == 251.0 / 256.0
        r = power_iteration(WQ, WK, np.ones(d), 20000, tol=1e-15)
        assert _rel(r.sigma, sv[h][0]) < 1e-9


# ----------------------------------------------- implicit vs explicit (textbook)


@pytest.mark.parametrize("d,dh,tol", [(48, 8, 0.0), (200, 16, 0.0), (200, 16, 1e-5)])
def test_implicit_matches_dense_power_iteration(d, dh, tol):
    rng = np.random.default_rng(3)
    WQ, WK = rng.standard_normal((d, dh)) * 0.02, rng.standard_normal((d, dh)) * 0.02
    v0 = rng.standard_normal(d)
    r = power_iteration(WQ, WK, v0, 40, tol)
    s, u, v, it = explicit.dense_power_iteration(explicit.interaction_matrix(WQ, WK), v0, 40, tol)
    assert r.iters == it
    assert _rel(r.sigma, s) < 1e-12
    assert np.max(np.abs(r.v - v)) < 1e-10 and np.max(np.abs(r.u - u)) < 1e-10


# -------------------------------------------------------- P2 submultiplicative


def test_submultiplicative_bound_and_monotone_estimate():
    rng = np.random.default_rng(5)
    d, dh = 160, 16
    for _ in range(5):
        WQ, WK = rng.standard_normal((d, dh)), rng.standard_normal((d, dh))
        s1 = explicit.sigma_max_reduced(WQ, WK)[0]
        naive = explicit.spectral_norm(WQ) * explicit.spectral_norm(WK)
        assert s1 < naive
        v0 = rng.standard_normal(d)
        prev = 0.0
        for k in (1, 2, 4, 8, 16, 32):
            est = power_iteration(WQ, WK, v0, k).sigma
            assert prev <= est * (1 + 1e-13) and est <= s1 * (1 + 1e-12)
            prev = est


def test_interaction_bound_equality_iff_top_right_vectors_coincide():
    rng = np.random.default_rng(9)
    d, dh = 96, 6
    R = _orth(rng, dh, dh)
    UQ, UK = _orth(rng, d, dh), _orth(rng, d, dh)
    a = np.array([5.0, 3.0, 2.0, 1.0, 0.5, 0.2])
    b = np.array([4.0, 2.5, 1.5, 1.0, 0.3, 0.1])
    WQ, WK = (UQ * a) @ R.T, (UK * b) @ R.T       # shared right singular vectors
    s1 = explicit.sigma_max_reduced(WQ, WK)[0]
    assert _rel(s1, explicit.spectral_norm(WQ) * explicit.spectral_norm(WK)) < 1e-12
    WK2 = (UK * b[::-1].copy()) @ R.T              # top right vectors now differ
    s1b = explicit.sigma_max_reduced(WQ, WK2)[0]
    assert s1b < 0.5 * explicit.spectral_norm(WQ) * explicit.spectral_norm(WK2)


# ------------------------------------------------------------- P3 LAPACK checks


def test_qr_reduction_matches_svd_of_formed_matrix():
    rng = np.random.default_rng(13)
    for d, dh in ((30, 5), (128, 16)):
        WQ, WK = rng.standard_normal((d, dh)), rng.standard_normal((d, dh))
        full = explicit.singular_values(explicit.interaction_matrix(WQ, WK))[:dh]
        np.testing.assert_allclose(explicit.sigma_max_reduced(WQ, WK), full, rtol=1e-11)


def test_spiked_heads_converge_to_exact_sigma():
    wl = WORKLOADS["llama2-7b-spiked"].replace(n_layers=1, d_model=256, n_q=4, n_kv=4, head_dim=16)
    wq, wk = layer_weights(wl, 0)
    v = start_vectors(wl)[0].double().numpy()
    for h in range(4):
        WQ, WK = head_slices(wq.float().numpy(), wk.float().numpy(), h, 4, 16)
        exact = explicit.sigma_max_reduced(WQ, WK)
        gap = exact[1] / exact[0]
        assert gap < 0.999
        n = 30 + int(math.ceil(math.log(1e-13) / (2 * math.log(gap))))
        assert _rel(power_iteration(WQ, WK, v[h], n).sigma, exact[0]) < 1e-10


# ------------------------------------------------------ P4 tiny brute force S


def test_tiny_brute_force_logits_obey_interaction_and_naive_bounds():
    wl = WORKLOADS["tiny"]
    wq, wk = layer_weights(wl, 0)
    x = tokens(wl, 16)
    dh = wl.head_dim
    for h in range(wl.n_q):
        WQ, WK = head_slices(wq.numpy(), wk.numpy(), h, wl.n_kv, dh)
        Q, K = x @ WQ, x @ WK                       # Q = X W^Q, K = X W^K
        S = Q @ K.T / math.sqrt(dh)                 # S = Q K^T / sqrt(d_h)
        M = explicit.interaction_matrix(WQ, WK)
        Sb = np.einsum("id,de,je->ij", x, M, x) / math.sqrt(dh)
        np.testing.assert_allclose(S, Sb, rtol=1e-10, atol=1e-15)
        sig = explicit.singular_values(M)[0]
        nx = np.linalg.norm(x, axis=1)
        inter = sig * np.outer(nx, nx) / math.sqrt(dh)
        naive = explicit.spectral_norm(WQ) * explicit.spectral_norm(WK) * np.outer(nx, nx) / math.sqrt(dh)
        assert np.all(np.abs(S) <= inter * (1 + 1e-12))
        assert np.all(inter <= naive * (1 + 1e-12))
        # equality at x_i = u_1, x_j = v_1
        Um, sv, Vt = np.linalg.svd(M)
        assert _rel(abs(Um[:, 0] @ M @ Vt[0]), sv[0]) < 1e-12


# ----------------------------------------------------- P5 E4M3 and the scale


def test_e4m3_codec_fixed_points():
    codes = np.arange(256)
    vals = e4m3.decode(codes)
    assert np.isnan(vals[0x7F]) and np.isnan(vals[0xFF])
    assert np.nanmax(vals) == 448.0 and vals[0x7E] == 448.0
    assert vals[0x01] == 2.0 ** -9 and vals[0x08] == 2.0 ** -6 and vals[0x38] == 1.0
    finite = ~np.isnan(vals)
    np.testing.assert_array_equal(e4m3.encode(vals[finite]), codes[finite])
    # ties to even: 1.0625 lies between 1.0 (mantissa 0) and 1.125 (mantissa 1)
    assert e4m3.decode(e4m3.encode(1.0625)) == 1.0
    assert e4m3.decode(e4m3.encode(1.1875)) == 1.25
    assert e4m3.decode(e4m3.encode(460.0)) == 448.0
    assert np.isnan(e4m3.decode(e4m3.encode(470.0)))
    assert e4m3.decode(e4m3.encode(470.0, saturate=True)) == 448.0
    assert e4m3.decode(e4m3.encode(2.0 ** -10)) == 0.0           # tie to even (0)
    assert e4m3.decode(e4m3.encode(3 * 2.0 ** -10)) == 2 * 2.0 ** -9


def test_scale_equality_case_hits_the_safe_range():
    """With alpha = 1 and tokens of norm sqrt(d) aligned with the top singular
    pair, |S| = B_max exactly, so |S / scale| = eta_fp8 * R_max = 358.4."""
    consts = {k: float(v) for k, v in read_golden("fp8_constants.txt")}
    assert consts["eta_fp8"] * consts["r_max"] == pytest.approx(consts["r_safe"], rel=1e-12)
    rng = np.random.default_rng(17)
    for d, dh in ((32, 8), (256, 64)):
        WQ, WK = rng.standard_normal((d, dh)) * 0.02, rng.standard_normal((d, dh)) * 0.02
        M = explicit.interaction_matrix(WQ, WK)
        Um, sv, Vt = np.linalg.svd(M)
        sigma = sv[0]
        scale = layer_scale(sigma, 1.0, d, dh, consts["eta_fp8"], consts["r_max"])
        xi, xj = math.sqrt(d) * Um[:, 0], math.sqrt(d) * Vt[0]
        s_ij = (xi @ WQ) @ (xj @ WK) / math.sqrt(dh)
        assert _rel(abs(s_ij) / scale, consts["r_safe"]) < 1e-10
        assert scale == pytest.approx(calibration.scale_factor(sigma, 1.0, d, dh), rel=1e-14)


@pytest.mark.parametrize("key,n_tokens", [("tiny", 64), ("gpt2-small", 24)])
def test_no_e4m3_overflow_with_converged_sigma(key, n_tokens):
    wl = WORKLOADS[key].replace(n_layers=1)
    wq, wk = layer_weights(wl, 0)
    v = start_vectors(wl).double().numpy()
    dh, d = wl.head_dim, wl.d_model
    res = spectral_step([wq.numpy()], [wk.numpy()], v, 200, n_kv=wl.n_kv, head_dim=dh, alpha=1.0)
    x = tokens(wl, n_tokens, spherical=True)
    worst = 0.0
    for h in range(wl.n_q):
        WQ, WK = head_slices(wq.numpy(), wk.numpy(), h, wl.n_kv, dh)
        S = (x @ WQ) @ (x @ WK).T / math.sqrt(dh)
        y = S / res["scale"][0]
        assert not e4m3.overflows(y).any()
        assert not np.isnan(e4m3.decode(e4m3.encode(y))).any()
        worst = max(worst, np.abs(y).max())
    assert worst < 358.4


# --------------------------------------------------------- P6 GQA equivalence


def test_implicit_gqa_equals_explicit_key_expansion():
    rng = np.random.default_rng(19)
    d, dh, nq, nkv = 64, 8, 8, 2
    g = nq // nkv
    wq = rng.standard_normal((nq * dh, d))
    wk = rng.standard_normal((nkv * dh, d))
    wk_exp = np.repeat(wk.reshape(nkv, dh, d), g, axis=0).reshape(nq * dh, d)
    v = rng.standard_normal((1, nq, d))
    a = spectral_step([wq], [wk], v, 25, n_kv=nkv, head_dim=dh, alpha=0.1)
    b = spectral_step([wq], [wk_exp], v, 25, n_kv=nq, head_dim=dh, alpha=0.1)
    np.testing.assert_array_equal(a["sigma"], b["sigma"])
    # paper-literal layer form: RepeatBlocks / SumGroups vs the expanded matrix
    WQl, WKl, WKe = wq.T, wk.T, wk_exp.T
    v0 = rng.standard_normal(d)
    r1 = power_iteration_layer(WQl, WKl, v0, 30, g, dh)
    r2 = power_iteration_layer(WQl, WKe, v0, 30, 1, dh)
    s3 = explicit.dense_power_iteration(explicit.interaction_matrix(WQl, WKe), v0, 30)[0]
    assert _rel(r1.sigma, r2.sigma) < 1e-12 and _rel(r1.sigma, s3) < 1e-12


# ------------------------------------------------------ P7 / P8 invariances


def test_homogeneity_matches_spike_response():
    rng = np.random.default_rng(23)
    d, dh = 80, 8
    WQ, WK = rng.standard_normal((d, dh)) * 0.02, rng.standard_normal((d, dh)) * 0.02
    v0 = rng.standard_normal(d)
    s = power_iteration(WQ, WK, v0, 10).sigma
    s4 = power_iteration(4 * WQ, 4 * WK, v0, 10).sigma
    assert s4 == 16 * s
    assert layer_scale(s4, 0.08, d, dh) == pytest.approx(16 * layer_scale(s, 0.08, d, dh), rel=1e-15)
    g = {k: float(v) for k, v in read_golden("spike_response.txt")}
    m = g["weight_multiplier"]
    assert abs(g["scale_after"] / g["scale_before"] / m ** 2 - 1.0) < 0.015


def test_orthogonal_invariance():
    rng = np.random.default_rng(29)
    d, dh = 120, 12
    WQ, WK = rng.standard_normal((d, dh)), rng.standard_normal((d, dh))
    R = _orth(rng, dh, dh)
    v0 = rng.standard_normal(d)
    a = power_iteration(WQ, WK, v0, 15).sigma
    b = power_iteration(WQ @ R, WK @ R, v0, 15).sigma
    assert _rel(a, b) < 1e-12


# ------------------------------------------------------ P9 alpha selection


def test_alpha_min_table():
    for model, d, dh, N, a_printed in read_golden("alpha_selection.txt"):
        a = calibration.alpha_min(int(d), int(dh), int(N), 1024, 1e-6)
        assert abs(a - float(a_printed)) < 6e-4, model


def test_concentration_table():
    for model, d, dh, g_printed, imp in read_golden("concentration.txt"):
        N = {"GPT-2-XL": 1200, "Mistral-7B": 1024, "Llama-2-13B": 1600, "Llama-2-70B": 5120}[model]
        g = calibration.gamma_select(int(dh), N, 1024, 1e-6)
        assert abs(g - float(g_printed)) < 0.02, model
        assert round(calibration.rank_aware_improvement(int(d), int(dh), g)) == int(imp), model


def test_alpha_used_is_alpha_min_rounded_up():
    for model, d, dh, N, a_used in read_golden("alpha_used.txt"):
        a = calibration.alpha_min(int(d), int(dh), int(N), 1024, 1e-6)
        assert math.ceil(a * 100) / 100 == pytest.approx(float(a_used)), model
    for key, N in (("gpt2-small", 144), ("llama2-7b-spiked", 1024), ("gpt2-xl", 1200),
                   ("llama2-70b-gqa", 5120), ("tiny", 4)):
        wl = WORKLOADS[key]
        a = calibration.alpha_min(wl.d_model, wl.head_dim, N, 1024, 1e-6)
        assert min(1.0, math.ceil(a * 100) / 100) == pytest.approx(wl.alpha), key


def test_selection_rule_meets_the_union_bound():
    for model, d, dh, N, _ in read_golden("alpha_selection.txt"):
        d, dh, N = int(d), int(dh), int(N)
        g = calibration.gamma_select(dh, N, 1024, 1e-6)
        a = calibration.alpha_min(d, dh, N, 1024, 1e-6)
        t1, t2 = calibration.overflow_terms(d, dh, 1024, a, g)
        assert N * t1 <= 0.5e-6 * (1 + 1e-9) and N * t2 == pytest.approx(0.5e-6, rel=1e-9)


# ------------------------------------------------------ degenerate inputs


def test_degenerate_inputs():
    rng = np.random.default_rng(31)
    d, dh = 16, 4
    WQ, WK = rng.standard_normal((d, dh)), rng.standard_normal((d, dh))
    r = power_iteration(WQ, WK, np.zeros(d), 5)
    assert np.isnan(r.sigma) and r.iters == -1
    r = power_iteration(WQ, WK, np.full(d, np.nan), 5)
    assert np.isnan(r.sigma) and r.iters == -1
    v0 = rng.standard_normal(d)
    r = power_iteration(WQ, np.zeros((d, dh)), v0, 5)
    assert r.sigma == 0.0 and r.iters == -2
    np.testing.assert_allclose(r.v, v0 / np.linalg.norm(v0), rtol=0, atol=1e-15)
    assert not r.u.any()


# ------------------------------------ per-layer reduction, auto-alpha, slack


def test_layer_scale_takes_the_largest_head_sigma():
    """Eq. "scale" takes sigma^(l) as the largest sigma_h of the layer (each
    head's logits obey the interaction bound with its own sigma_h).  Planted
    heads have exact sigma_h, a power of two apart from head to head; the
    oracle's spectral_step, run to convergence, must give
    scale_l = layer_scale(max_h planted sigma_h), which a mean, a min, a sum
    or the first head's sigma would not."""
    wl = WORKLOADS["llama2-70b-perstep"].replace(key="pin-max", cfg_id=41, n_layers=4, d_model=256, n_q=6,
                                                 n_kv=2, head_dim=16)
    wq, wk = all_weights(wl, "cpu")
    v0 = start_vectors(wl, "cpu").double().numpy()
    res = spectral_step(wq.float().numpy(), wk.float().numpy(), v0, 5000, n_kv=wl.n_kv, head_dim=wl.head_dim,
                        alpha=wl.alpha, tol=1e-13)
    assert res["iters"].max() < 5000
    sig_exact = np.stack([planted_singular_values(wl, l)[:, 0] for l in range(wl.n_layers)])
    np.testing.assert_allclose(res["sigma"], sig_exact, rtol=1e-9)
    want = [layer_scale(sig_exact[l].max(), wl.alpha, wl.d_model, wl.head_dim) for l in range(wl.n_layers)]
    np.testing.assert_allclose(res["scale"], want, rtol=1e-9)
    # the planted layers separate the readings: every other reduction misses some layer by far
    for other in (np.mean, np.min, np.sum, lambda s: s[0], np.median):
        alt = [layer_scale(other(sig_exact[l]), wl.alpha, wl.d_model, wl.head_dim) for l in range(wl.n_layers)]
        assert np.max(np.abs(np.array(alt) / np.array(want) - 1.0)) > 0.1


def test_auto_alpha_order_statistics():
    """App. M, Algorithm "Auto-alpha Calibration": alpha = Quantile_q(R) * kappa.
    Identities any quantile obeys, on the sorted burn-in ratios: q = 0 is the
    smallest, q = 1 the largest, q = 1/2 of an odd count the middle one; a
    position q (n - 1) that falls between two order statistics interpolates
    linearly between them; kappa multiplies; the order of the burn-in does
    not matter; and with 10001 ratios P99.99 is the 10000th smallest."""
    rng = np.random.default_rng(2024)
    r = rng.uniform(7e-5, 3.7e-4, 101)
    srt = sorted(r.tolist())
    assert calibration.auto_alpha(r, 0.0) == srt[0]
    assert calibration.auto_alpha(r, 1.0) == srt[-1]
    assert calibration.auto_alpha(r, 0.5) == srt[50]
    assert calibration.auto_alpha(r, 0.5, kappa=3.0) == pytest.approx(3.0 * srt[50], rel=1e-15)
    assert calibration.auto_alpha(rng.permutation(r), 0.37) == calibration.auto_alpha(r, 0.37)
    assert calibration.auto_alpha([0.0, 10.0], 0.25) == pytest.approx(2.5, rel=1e-15)
    assert calibration.auto_alpha([4.0, 1.0, 2.0], 0.75) == pytest.approx(3.0, rel=1e-15)
    big = rng.uniform(0.0, 1.0, 10001)
    assert calibration.auto_alpha(big, 0.9999) == pytest.approx(sorted(big.tolist())[9999], rel=1e-12)
    # all ratios equal: alpha is that ratio, whatever q
    assert calibration.auto_alpha([3.6e-4] * 57, 0.9999) == pytest.approx(3.6e-4, rel=1e-15)


def test_slack_ratio_is_one_at_the_interaction_bound_equality():
    """Sec. 3.5: r = max|S| / B_max with B_max = sigma * d / sqrt(d_h) (the
    interaction bound at ||x|| = sqrt(d)).  Prop. "Interaction bound" is tight
    at x_i = sqrt(d) u_1, x_j = sqrt(d) v_1 (top singular pair of M), so the
    brute-force logit there gives r = 1 exactly; x_i = sqrt(d) u_2 gives
    sigma_2 / sigma_1; tokens on the sqrt(d)-sphere give r <= 1."""
    rng = np.random.default_rng(77)
    d, dh = 48, 8
    WQ, WK = rng.standard_normal((d, dh)), rng.standard_normal((d, dh))
    M = explicit.interaction_matrix(WQ, WK)
    U, s, Vt = np.linalg.svd(M)
    sq = math.sqrt(d)

    def logit(xi, xj):
        return float(xi @ M @ xj) / math.sqrt(dh)

    assert calibration.slack_ratio(abs(logit(sq * U[:, 0], sq * Vt[0])), s[0], d, dh) == pytest.approx(1.0, rel=1e-12)
    assert calibration.slack_ratio(abs(logit(sq * U[:, 1], sq * Vt[1])), s[0], d, dh) == pytest.approx(
        s[1] / s[0], rel=1e-12)
    x = rng.standard_normal((64, d))
    x *= sq / np.linalg.norm(x, axis=1, keepdims=True)
    S = x @ M @ x.T / math.sqrt(dh)
    r = calibration.slack_ratio(np.abs(S).max(), s[0], d, dh)
    assert 0.0 < r <= 1.0
