"""spectral_step captured into a HIP graph (torch.cuda.CUDAGraph over the
context's stream) and replayed: every replay, with eager work and
synchronisation between replays, gives the bits of the eager call."""

import numpy as np
import pytest
import torch

from workloads import WORKLOADS, all_weights, start_vectors

pytestmark = pytest.mark.gpu

if not torch.cuda.is_available():  # pragma: no cover - collected on CPU machines, skipped there
    pytest.skip("needs a GPU", allow_module_level=True)

from paper_2602_18851_amd import Spectral  # noqa: E402
from paper_2602_18851_amd.spectral import SN_FLAG_GRAM  # noqa: E402


@pytest.mark.parametrize("flags", [0, SN_FLAG_GRAM], ids=["chain", "gram"])
@pytest.mark.parametrize("key", ["gpt2-small", "llama2-70b-gqa"])
def test_step_replays_from_a_graph(key, flags):
    wl = WORKLOADS[key]
    if key == "llama2-70b-gqa":
        wl = wl.replace(n_layers=2)
    n_iter = 7
    gq, gk = all_weights(wl, "cuda")
    v0 = start_vectors(wl, "cuda")
    est = Spectral(wl.n_layers, wl.d_model, wl.n_q, wl.n_kv, wl.head_dim, wl.dtype, wl.alpha, flags=flags)
    L, nq = wl.n_layers, wl.n_q

    def buffers():
        return (v0.clone(), torch.empty_like(v0), torch.empty(L, nq, device="cuda"), torch.empty(L, device="cuda"),
                torch.empty(L, nq, dtype=torch.int32, device="cuda"))

    ve, ue, se, ce, ie = buffers()
    est.step(gq, gk, ve, n_iter, u=ue, sigma=se, scale=ce, iters=ie)  # eager reference (uploads the table)
    torch.cuda.synchronize()
    ref = [t.cpu().numpy() for t in (ve, ue, se, ce, ie)]

    vg, ug, sg, cg, ig = buffers()
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        est.step(gq, gk, vg, n_iter, u=ug, sigma=sg, scale=cg, iters=ig)
    torch.cuda.synchronize()
    for rep in range(4):
        vg.copy_(v0)  # the start vectors, in place (eager, outside the graph)
        for t in (ug, sg, cg):
            t.fill_(float("nan"))
        ig.fill_(-7)
        graph.replay()
        torch.cuda.synchronize()
        got = [t.cpu().numpy() for t in (vg, ug, sg, cg, ig)]
        for name, a, b in zip(("v", "u", "sigma", "scale", "iters"), ref, got):
            np.testing.assert_array_equal(a, b, err_msg=f"replay {rep}: {name}")
        # eager work of the program between replays
        est.step(gq, gk, ve.copy_(v0), n_iter, u=ue, sigma=se, scale=ce, iters=ie)
        torch.cuda.synchronize()
    del graph
    est.close()


@pytest.mark.parametrize("flags", [0, SN_FLAG_GRAM], ids=["chain", "gram"])
def test_tolerance_step_replays_from_a_graph(flags):
    """Tolerance mode never waits on the host, so a call at tol 1e-4 (cap
    1000) captures too: planted per-step shape (2 layers of the 70B GQA
    layout), cold start, so most heads run far past the two full steps into
    the tail.  Between replays the program runs eager calls on other weights
    (doubled, so other pointers and other results); every replay still gives
    the eager bits of the captured call."""
    wl = WORKLOADS["llama2-70b-perstep"].replace(n_layers=2)
    gq, gk = all_weights(wl, "cuda")
    gq2, gk2 = gq * 2, gk * 2
    v0 = start_vectors(wl, "cuda")
    est = Spectral(wl.n_layers, wl.d_model, wl.n_q, wl.n_kv, wl.head_dim, wl.dtype, wl.alpha, tol=wl.tol,
                   flags=flags)
    L, nq = wl.n_layers, wl.n_q

    def buffers():
        return (v0.clone(), torch.empty_like(v0), torch.empty(L, nq, device="cuda"), torch.empty(L, device="cuda"),
                torch.empty(L, nq, dtype=torch.int32, device="cuda"))

    ve, ue, se, ce, ie = buffers()
    est.step(gq, gk, ve, wl.n_iter, u=ue, sigma=se, scale=ce, iters=ie)
    torch.cuda.synchronize()
    ref = [t.cpu().numpy() for t in (ve, ue, se, ce, ie)]
    assert ref[4].min() >= 2 and np.median(ref[4]) > 2  # most heads ran into the tail

    vg, ug, sg, cg, ig = buffers()
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        est.step(gq, gk, vg, wl.n_iter, u=ug, sigma=sg, scale=cg, iters=ig)
    torch.cuda.synchronize()
    for rep in range(3):
        vg.copy_(v0)
        for t in (ug, sg, cg):
            t.fill_(float("nan"))
        ig.fill_(-7)
        graph.replay()
        torch.cuda.synchronize()
        got = [t.cpu().numpy() for t in (vg, ug, sg, cg, ig)]
        for name, a, b in zip(("v", "u", "sigma", "scale", "iters"), ref, got):
            np.testing.assert_array_equal(a, b, err_msg=f"replay {rep}: {name}")
        # eager work on other weights between replays: sigma x4
        s2, _, _ = est.step(gq2, gk2, ve.copy_(v0), wl.n_iter, u=ue)
        torch.cuda.synchronize()
        np.testing.assert_allclose(s2.cpu().numpy(), 4 * ref[2], rtol=1e-3)
    del graph
    est.close()
