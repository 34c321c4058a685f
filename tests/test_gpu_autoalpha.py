"""Auto-alpha calibration driven by the FP8 consumer (Sec. 3.5; App. M,
Algorithm "Auto-alpha Calibration"), through the C ABI: a burn-in of warm
one-iteration estimator calls on seeded perturbed weights, each followed by
the E4M3 logit consumer on fresh seeded tokens at the conservative alpha_0;
the slack ratios r = max|S| / B_max and alpha_final = Quantile_q(R) * kappa
against the oracle's own chain (implicit estimator, explicit logits,
oracle.calibration), and the utilisation alpha_final buys on the next step.

The consumer's max|S~| carries at most 2^-14 relative error (hi/lo bf16
products) and sigma about 1e-6, so each ratio, and alpha_final, must agree
to 1e-3."""

import numpy as np
import pytest
import torch

from oracle import calibration, fp8_consumer
from oracle.power_iteration import spectral_step as oracle_step
from workloads import WORKLOADS, all_weights, start_vectors, tokens

pytestmark = pytest.mark.gpu

if not torch.cuda.is_available():  # pragma: no cover - collected on CPU machines, skipped there
    pytest.skip("needs a GPU", allow_module_level=True)

from paper_2602_18851_amd import AutoAlpha, Spectral, fp8_report  # noqa: E402

RTOL = 1e-3


def _tokens(wl, seq, step):
    return torch.stack([torch.from_numpy(tokens(wl, seq, spherical=True, layer=l, step=step)).to(torch.bfloat16)
                        for l in range(wl.n_layers)])


def _oracle_max_logit(wl, x, wq, wk, l):
    """max over heads and (i, j) of |S_ij| of layer l, explicit logits."""
    x64, wq64, wk64 = x[l].double().numpy(), wq[l].double().numpy(), wk[l].double().numpy()
    return max(np.abs(fp8_consumer.head_logits(x64, wq64, wk64, h, wl.n_kv, wl.head_dim)).max()
               for h in range(wl.n_q))


@pytest.mark.parametrize("quantile,kappa", [(0.9999, 1.0), (0.5, 2.0)])
def test_auto_alpha_from_the_consumer_matches_the_oracle_chain(quantile, kappa):
    wl = WORKLOADS["llama2-70b-gqa"].replace(key="autoalpha", cfg_id=51, n_layers=3, d_model=512, n_q=8, n_kv=2,
                                             head_dim=64, std=0.02)
    seq, steps, alpha0 = 160, 6, 0.3
    est = Spectral(wl.n_layers, wl.d_model, wl.n_q, wl.n_kv, wl.head_dim, wl.dtype, alpha0)
    wq0, wk0 = all_weights(wl, "cpu")
    v0 = start_vectors(wl, "cpu")
    v = v0.cuda()
    est.step(wq0.cuda(), wk0.cuda(), v, 5)   # cold start: the paper's five iterations
    v_o = oracle_step(wq0.float().numpy(), wk0.float().numpy(), v0.double().numpy(), 5, n_kv=wl.n_kv,
                      head_dim=wl.head_dim, alpha=alpha0)["v"]
    auto = AutoAlpha(wl.d_model, wl.head_dim, quantile, kappa)
    ratios_ref = []
    for t in range(steps):
        wq, wk = all_weights(wl, "cpu", perturbed=True, step=t)
        x = _tokens(wl, seq, t)
        sigma, scale, _ = est.step(wq.cuda(), wk.cuda(), v, 1)   # one update per forward pass
        max_abs, n_over, _ = est.logits_fp8(x.cuda(), wq.cuda(), wk.cuda(), scale)
        auto.observe(sigma, scale, max_abs)
        ref = oracle_step(wq.float().numpy(), wk.float().numpy(), v_o, 1, n_kv=wl.n_kv, head_dim=wl.head_dim,
                          alpha=alpha0)
        v_o = ref["v"]
        for l in range(wl.n_layers):
            ratios_ref.append(calibration.slack_ratio(_oracle_max_logit(wl, x, wq, wk, l), ref["sigma"][l].max(),
                                                      wl.d_model, wl.head_dim))
    assert len(auto.ratios) == steps * wl.n_layers
    np.testing.assert_allclose(auto.ratios, ratios_ref, rtol=RTOL)
    a_gpu, a_ref = auto.alpha(), calibration.auto_alpha(ratios_ref, quantile, kappa)
    assert abs(a_gpu - a_ref) <= RTOL * a_ref, (a_gpu, a_ref)

    # the next step at alpha_final: utilisation max|S~| / 448 per layer, GPU and oracle
    est.close()
    est = Spectral(wl.n_layers, wl.d_model, wl.n_q, wl.n_kv, wl.head_dim, wl.dtype, a_gpu)
    wq, wk = all_weights(wl, "cpu", perturbed=True, step=steps)
    x = _tokens(wl, seq, steps)
    sigma, scale, _ = est.step(wq.cuda(), wk.cuda(), v, 1)
    max_abs, n_over, _ = est.logits_fp8(x.cuda(), wq.cuda(), wk.cuda(), scale)
    rep = fp8_report(max_abs, n_over)
    ref = oracle_step(wq.float().numpy(), wk.float().numpy(), v_o, 1, n_kv=wl.n_kv, head_dim=wl.head_dim,
                      alpha=a_gpu)
    util_ref = [100.0 * _oracle_max_logit(wl, x, wq, wk, l) / ref["scale"][l] / 448.0 for l in range(wl.n_layers)]
    util_gpu = 100.0 * max_abs.double().cpu().numpy().max(axis=1) / 448.0
    np.testing.assert_allclose(util_gpu, util_ref, rtol=RTOL)
    assert rep["utilization_pct_layers"]["median"] == pytest.approx(np.median(util_ref), rel=RTOL)
    print(f"q={quantile} kappa={kappa}: alpha {alpha0} -> {a_gpu:.3e} (oracle {a_ref:.3e}); utilisation per layer "
          f"{np.round(util_gpu, 1)} % (at alpha_0: {np.round(util_gpu * a_gpu / alpha0, 2)} %)")
    est.close()
