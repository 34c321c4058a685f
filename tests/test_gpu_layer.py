"""Layer-level form (spectral_step_layer) against the float64 oracle's
paper-literal estimator (App. E, "Implicit GQA Power Iteration": one u, v per
layer, RepeatBlocks / SumGroups), through the C ABI.

Bar: relative error <= 1e-3 on every layer's sigma and scale; |cos| >= 1 - 1e-3
between the GPU's and the oracle's unit vectors u and v."""

import numpy as np
import pytest
import torch

from oracle.power_iteration import layer_scale, power_iteration_layer
from workloads import WORKLOADS, all_weights, layer_start_vectors

pytestmark = pytest.mark.gpu

RTOL = 1e-3

if not torch.cuda.is_available():  # pragma: no cover - collected on CPU machines, skipped there
    pytest.skip("needs a GPU", allow_module_level=True)

from paper_2602_18851_amd import SN_FLAG_LAYER, Spectral  # noqa: E402


def _rel(a, b):
    a, b = np.asarray(a, np.float64), np.asarray(b, np.float64)
    return np.abs(a - b) / np.abs(b)


def run_layer(wl, wq, wk, v0, n_iter, want_u=True, ld=0):
    est = Spectral(wl.n_layers, wl.d_model, wl.n_q, wl.n_kv, wl.head_dim, wl.dtype, wl.alpha, ld=ld,
                   flags=SN_FLAG_LAYER)
    v = v0.cuda().contiguous()
    u = torch.empty_like(v) if want_u else None
    sigma, scale = est.step_layer(wq, wk, v, n_iter, u=u)
    torch.cuda.synchronize()
    out = {"sigma": sigma.cpu().double().numpy(), "scale": scale.cpu().double().numpy(),
           "v": v.cpu().double().numpy(), "u": u.cpu().double().numpy() if want_u else None}
    est.close()
    return out


def oracle_layers(wl, wq_cpu, wk_cpu, v0, n_iter, layers=None):
    g = wl.n_q // wl.n_kv
    res = {}
    for l in (range(wl.n_layers) if layers is None else layers):
        # the paper's W^Q in R^{d x n_q d_h} is the transpose of the Linear-layout rows
        r = power_iteration_layer(wq_cpu[l].T, wk_cpu[l].T, v0[l].double().numpy(), n_iter, g, wl.head_dim)
        res[l] = r
    return res


def check(wl, gpu, ref):
    worst = 0.0
    for l, r in ref.items():
        err = float(_rel(gpu["sigma"][l], r.sigma))
        worst = max(worst, err)
        assert err <= RTOL, (l, gpu["sigma"][l], r.sigma)
        assert _rel(gpu["scale"][l], layer_scale(r.sigma, wl.alpha, wl.d_model, wl.head_dim)) <= RTOL
        assert abs(np.dot(gpu["v"][l], r.v)) >= 1 - 1e-3
        assert abs(np.linalg.norm(gpu["v"][l]) - 1) < 1e-5
        if gpu["u"] is not None:
            assert abs(np.dot(gpu["u"][l], r.u)) >= 1 - 1e-3
    print(f"{wl.key}: layer form, {len(ref)} layers, max rel err sigma {worst:.3e}")


CASES = [
    ("mha-f32", dict(n_layers=2, d_model=256, n_q=4, n_kv=4, head_dim=64, dtype="f32"), 0),
    ("gqa8-bf16", dict(n_layers=2, d_model=1024, n_q=16, n_kv=2, head_dim=128, dtype="bf16"), 0),
    ("gqa3-bf16-ragged", dict(n_layers=1, d_model=1001, n_q=6, n_kv=2, head_dim=32, dtype="bf16"), 1008),
    ("mqa-bf16-dh8", dict(n_layers=2, d_model=64, n_q=8, n_kv=1, head_dim=8, dtype="bf16"), 0),
    ("gqa4-f32-ragged-dh16", dict(n_layers=3, d_model=517, n_q=8, n_kv=2, head_dim=16, dtype="f32"), 520),
    # 2 layers x 64 column tiles: the W_Q column sweep splits its 99 row blocks
    # into 50 runs of two (the last run one block), each wave summing its run
    ("gqa33-bf16-row-runs", dict(n_layers=2, d_model=4096, n_q=99, n_kv=3, head_dim=8, dtype="bf16"), 0),
]


def _padded(w, ld, d):
    if not ld:
        return w.cuda()
    p = torch.zeros(w.shape[0], w.shape[1], ld, dtype=w.dtype)
    p[:, :, :d] = w
    return p.cuda()[:, :, :d]


def _random_cases(n=8, seed=933):
    """Seeded random shapes: MHA and GQA, d_h 8..128, fp32 and bf16, ragged
    widths over padded rows."""
    rng = np.random.default_rng(seed)
    out = []
    for i in range(n):
        dt = str(rng.choice(["f32", "bf16"]))
        align = 4 if dt == "f32" else 8
        d = int(rng.integers(8, 1200))
        ld = -(-d // align) * align + align * int(rng.integers(0, 3))
        n_kv = int(rng.integers(1, 4))
        over = dict(n_layers=int(rng.integers(1, 4)), d_model=d, n_kv=n_kv, n_q=n_kv * int(rng.choice([1, 2, 3, 8])),
                    head_dim=int(rng.choice([8, 16, 32, 64, 128])), dtype=dt, cfg_id=200 + i)
        out.append((f"rand{i}-{dt}-d{d}-ld{ld}-q{over['n_q']}kv{n_kv}-dh{over['head_dim']}", over, ld))
    return out


CASES += _random_cases()


@pytest.mark.parametrize("name,over,ld", CASES, ids=[c[0] for c in CASES])
def test_layer_form_against_oracle(name, over, ld):
    wl = WORKLOADS["llama2-70b-gqa"].replace(key=name, n_iter=9, std=0.02, **over)
    wq, wk = all_weights(wl, "cpu")
    v0 = layer_start_vectors(wl)
    gpu = run_layer(wl, _padded(wq, ld, wl.d_model), _padded(wk, ld, wl.d_model), v0, wl.n_iter, ld=ld)
    ref = oracle_layers(wl, wq.float().numpy(), wk.float().numpy(), v0, wl.n_iter)
    check(wl, gpu, ref)


def test_layer_form_one_step_and_warm_start():
    wl = WORKLOADS["gpt2-small"].replace(n_layers=2)
    wq, wk = all_weights(wl, "cpu")
    v0 = layer_start_vectors(wl)
    for n in (1, 2):
        check(wl, run_layer(wl, wq.cuda(), wk.cuda(), v0, n), oracle_layers(wl, wq.numpy(), wk.numpy(), v0, n))
    # two calls of 4 continue one call of 8 (v is the persistent state)
    est = Spectral(wl.n_layers, wl.d_model, wl.n_q, wl.n_kv, wl.head_dim, wl.dtype, wl.alpha, flags=SN_FLAG_LAYER)
    v = v0.cuda()
    est.step_layer(wq.cuda(), wk.cuda(), v, 4)
    sigma, _ = est.step_layer(wq.cuda(), wk.cuda(), v, 4)
    torch.cuda.synchronize()
    ref = oracle_layers(wl, wq.numpy(), wk.numpy(), v0, 8)
    assert max(float(_rel(sigma[l].item(), ref[l].sigma)) for l in ref) <= RTOL
    est.close()


def test_layer_form_degenerate_layers():
    wl = WORKLOADS["llama2-70b-gqa"].replace(key="degenerate", n_layers=3, d_model=256, n_q=4, n_kv=2,
                                             head_dim=32, n_iter=5)
    wq, wk = all_weights(wl, "cpu")
    wk[2] = 0                                 # layer 2: M = 0
    v0 = layer_start_vectors(wl)
    v0[0] = 0.0                               # layer 0: zero start vector
    gpu = run_layer(wl, wq.cuda(), wk.cuda(), v0, wl.n_iter)
    assert np.isnan(gpu["sigma"][0]) and np.isnan(gpu["scale"][0])
    np.testing.assert_array_equal(gpu["v"][0], 0.0)
    assert not gpu["u"][0].any() and not gpu["u"][2].any()
    assert gpu["sigma"][2] == 0 and gpu["scale"][2] == 0
    vn = v0[2].double().numpy()
    np.testing.assert_allclose(gpu["v"][2], vn / np.linalg.norm(vn), atol=1e-6)
    check(wl, gpu, oracle_layers(wl, wq.float().numpy(), wk.float().numpy(), v0, wl.n_iter, layers=[1]))


def test_layer_form_without_flag_is_refused():
    from paper_2602_18851_amd.spectral import SN_ESTATE, SpectralError

    wl = WORKLOADS["gpt2-small"].replace(n_layers=1)
    wq, wk = all_weights(wl, "cuda")
    est = Spectral(wl.n_layers, wl.d_model, wl.n_q, wl.n_kv, wl.head_dim, wl.dtype, wl.alpha)
    with pytest.raises(SpectralError) as e:
        est.step_layer(wq, wk, torch.ones(1, wl.d_model, device="cuda"), 1)
    assert e.value.code == SN_ESTATE
    est.close()


def test_layer_form_full_size_every_layer():
    """Llama-2-70B GQA shape, all 80 layers at the bench's 30 iterations, every
    layer's sigma and scale against the oracle's layer-level estimator (each
    layer's weights widened to float64 on the device, then copied back)."""
    wl = WORKLOADS["llama2-70b-gqa"]
    gq, gk = all_weights(wl, "cuda")
    v0 = layer_start_vectors(wl)
    gpu = run_layer(wl, gq, gk, v0, wl.n_iter, want_u=False)
    assert np.isfinite(gpu["sigma"]).all()
    ref = {}
    for l in range(wl.n_layers):
        wq_l, wk_l = gq[l].double().cpu().numpy(), gk[l].double().cpu().numpy()
        ref[l] = power_iteration_layer(wq_l.T, wk_l.T, v0[l].double().numpy(), wl.n_iter, wl.n_q // wl.n_kv,
                                       wl.head_dim)
    check(wl, gpu, ref)
