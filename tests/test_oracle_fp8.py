"""Pins of the FP8 consumer oracle (stage 3 of the geometry-aware forward
pass, Sec. 3.4) against the explicit bilinear form, explicit key expansion,
the equality case of the interaction bound (Prop. "Interaction bound") and a
rank-one closed form."""

import math

import numpy as np
import pytest

from oracle import calibration, e4m3, explicit, fp8_consumer
from oracle.power_iteration import head_slices
from workloads import WORKLOADS, layer_weights, tokens


def test_logits_equal_the_explicit_bilinear_form():
    """S_ij = x_i^T (W^Q_h W^{K T}_{g(h)}) x_j / sqrt(d_h) (Eq. "bilinear"), with
    the interaction matrix formed explicitly; GQA shape (g = 2)."""
    wl = WORKLOADS["tiny"].replace(n_q=4, n_kv=2)
    wq, wk = layer_weights(wl, 0)
    wq, wk = wq.double().numpy(), wk.double().numpy()
    x = tokens(wl, 12, spherical=True)
    for h in range(wl.n_q):
        WQ, WK = head_slices(wq, wk, h, wl.n_kv, wl.head_dim)
        M = explicit.interaction_matrix(WQ, WK)
        ref = np.einsum("id,de,je->ij", x, M, x) / math.sqrt(wl.head_dim)
        np.testing.assert_allclose(fp8_consumer.head_logits(x, wq, wk, h, wl.n_kv, wl.head_dim), ref,
                                   rtol=1e-12, atol=1e-14)


def test_gqa_logits_equal_explicit_key_expansion():
    """Query head h reads key head floor(h / g): the same logits as multi-head
    attention with every key block repeated g times (Prop. "Implicit GQA")."""
    wl = WORKLOADS["tiny"].replace(n_q=4, n_kv=1)
    wq, wk = layer_weights(wl, 0)
    wq, wk = wq.double().numpy(), wk.double().numpy()
    wk_exp = np.repeat(wk.reshape(wl.n_kv, wl.head_dim, -1), wl.n_q // wl.n_kv, axis=0).reshape(wq.shape)
    x = tokens(wl, 9)
    for h in range(wl.n_q):
        np.testing.assert_array_equal(fp8_consumer.head_logits(x, wq, wk, h, wl.n_kv, wl.head_dim),
                                      fp8_consumer.head_logits(x, wq, wk_exp, h, wl.n_q, wl.head_dim))


@pytest.mark.parametrize("alpha,over", [(1.0, False), (0.5, True)])
def test_equality_case_of_the_interaction_bound(alpha, over):
    """Tokens sqrt(d) u_1 and sqrt(d) v_1 (top singular pair of M_h) reach
    |S| = sigma_1 d / sqrt(d_h) = B_max exactly; with alpha = 1 the scaled
    logit is eta_fp8 * 448 = 358.4 (the safe range of Sec. 5.1), utilisation
    0.8; alpha = 0.5 doubles it past 464: overflow and a NaN code."""
    wl = WORKLOADS["tiny"]
    wq, wk = layer_weights(wl, 0)
    wq, wk = wq.double().numpy(), wk.double().numpy()
    d, dh = wl.d_model, wl.head_dim
    WQ, WK = head_slices(wq, wk, 0, wl.n_kv, dh)
    U, s, Vt = np.linalg.svd(explicit.interaction_matrix(WQ, WK))
    x = np.stack([math.sqrt(d) * U[:, 0], math.sqrt(d) * Vt[0]])
    scale = calibration.scale_factor(s[0], alpha, d, dh)
    out = fp8_consumer.consume_layer(x, wq, wk, scale, wl.n_kv, dh, heads=[0])
    target = 0.8 * 448.0 / alpha
    assert out["scaled"][0][0, 1] == pytest.approx(target, rel=1e-12)
    assert out["max_abs"][0] == pytest.approx(target, rel=1e-12)
    assert (out["n_over"][0] > 0) == over
    if over:
        assert out["codes"][0][0, 1] == e4m3.NAN_CODE
    else:
        assert fp8_consumer.utilization(out["max_abs"][0]) == pytest.approx(0.8, rel=1e-12)
        assert e4m3.decode(out["codes"][0][0, 1]) == 352.0   # 358.4 rounds to 1.375 * 2^8


def test_rank_one_closed_form_counts():
    """W^Q_0 = a e_0, W^K_0 = b e_0 (one nonzero weight each): S~_ij =
    a b x_i0 x_j0 / (sqrt(d_h) scale).  With that factor 55 and x_i0 in
    {-3 .. 3}, exactly the 4 pairs with |x_i0 x_j0| = 9 exceed 448 (at 495,
    past 464: NaN codes); the largest magnitude is 495."""
    d, dh = 16, 8
    wq = np.zeros((dh, d))
    wk = np.zeros((dh, d))
    wq[0, 0], wk[0, 0] = 2.0, 5.0
    x = np.zeros((7, d))
    x[:, 0] = np.arange(-3, 4)
    x[:, 1] = 1.0
    scale = 2.0 * 5.0 / (math.sqrt(dh) * 55.0)
    out = fp8_consumer.consume_layer(x, wq, wk, scale, 1, dh)
    S = out["scaled"][0]
    np.testing.assert_allclose(S, 55.0 * np.outer(x[:, 0], x[:, 0]), rtol=1e-14, atol=1e-12)
    assert out["n_over"][0] == 4
    assert out["max_abs"][0] == pytest.approx(495.0)
    assert np.count_nonzero((out["codes"][0] & 0x7F) == e4m3.NAN_CODE) == 4


def test_non_finite_scaled_logits_count_as_overflows():
    """Sec. 1: an overflow is a logit E4M3 cannot hold, which turns into NaN.
    |x| > 448 is the paper's predicate; NaN and +-inf (e.g. logits scaled by a
    NaN or zero scale) are not representable either, so they count, and their
    codes are the NaN code.  A NaN scale makes every logit of the layer an
    overflow and the largest scaled logit NaN."""
    x = np.array([np.nan, np.inf, -np.inf, 448.0, -448.0, 448.0001, 0.0, -1e9])
    np.testing.assert_array_equal(e4m3.overflows(x), [True, True, True, False, False, True, False, True])
    assert ((e4m3.encode(x[:3]) & 0x7F) == e4m3.NAN_CODE).all()
    wl = WORKLOADS["tiny"].replace(n_q=4, n_kv=2)
    wq, wk = layer_weights(wl, 0)
    xs = tokens(wl, 10, spherical=True)
    r = fp8_consumer.consume_layer(xs, wq.double().numpy(), wk.double().numpy(), float("nan"), wl.n_kv,
                                   wl.head_dim)
    for h in range(wl.n_q):
        assert r["n_over"][h] == 100 and math.isnan(r["max_abs"][h])
        assert ((r["codes"][h] & 0x7F) == e4m3.NAN_CODE).all()
