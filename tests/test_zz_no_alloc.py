"""spectral_step_noalloc (the allocation-free entry point: workspace in a
static device array) against spectral_step with a context, through the C
ABI: the same kernels, so the same bits.  Two calls in a row on one device,
the second on a smaller shape, in each form and mode that fits the static
scratch; and a shape whose workspace does not fit is refused."""

import numpy as np
import pytest
import torch

from workloads import WORKLOADS, all_weights, start_vectors

pytestmark = pytest.mark.gpu

if not torch.cuda.is_available():  # pragma: no cover - collected on CPU machines, skipped there
    pytest.skip("needs a GPU", allow_module_level=True)

from paper_2602_18851_amd import Spectral  # noqa: E402
from paper_2602_18851_amd import spectral as sp  # noqa: E402

SHAPES = [
    # first call: 2 layers of the 70B GQA layout at d = 1024 (matrix-core W_K sweeps)
    WORKLOADS["llama2-70b-gqa"].replace(key="na-big", n_layers=2, d_model=1024, n_q=16, n_kv=2, n_iter=7),
    # second call, smaller: one layer, d = 520 (a ragged tile), 8 / 2 heads of d_h 64
    WORKLOADS["llama2-70b-gqa"].replace(key="na-small", n_layers=1, d_model=520, n_q=8, n_kv=2, head_dim=64,
                                        n_iter=5),
]
PLANTED = [  # tolerance mode: planted spectra, cold start, d_h 32 (its tail fits the scratch)
    WORKLOADS["llama2-70b-perstep"].replace(key="na-tol-big", n_layers=2, d_model=512, n_q=8, n_kv=2, head_dim=32,
                                            n_iter=300),
    WORKLOADS["llama2-70b-perstep"].replace(key="na-tol-small", n_layers=1, d_model=256, n_q=4, n_kv=2, head_dim=32,
                                            n_iter=300),
]


def _outputs(wl, v0):
    L, nq = wl.n_layers, wl.n_q
    return (v0.clone(), torch.empty_like(v0), torch.empty(L, nq, device="cuda"), torch.empty(L, device="cuda"),
            torch.empty(L, nq, dtype=torch.int32, device="cuda"))


def _reference(wl, gq, gk, v0, flags, tol):
    est = Spectral(wl.n_layers, wl.d_model, wl.n_q, wl.n_kv, wl.head_dim, wl.dtype, wl.alpha, tol=tol, flags=flags)
    v, u, s, c, i = _outputs(wl, v0)
    est.step(gq, gk, v, wl.n_iter, u=u, sigma=s, scale=c, iters=i)
    torch.cuda.synchronize()
    est.close()
    return [t.cpu().numpy() for t in (v, u, s, c, i)]


def _noalloc(wl, gq, gk, v0, flags, tol):
    shape = sp.sn_shape(wl.n_layers, wl.d_model, wl.n_q, wl.n_kv, wl.head_dim,
                        sp.SN_BF16 if wl.dtype == "bf16" else sp.SN_F32, 0)
    params = sp.sn_params(wl.alpha, 0.8, 448.0, tol, 0, 0, flags)
    v, u, s, c, i = _outputs(wl, v0)
    stream = torch.cuda.current_stream().cuda_stream
    sp.spectral_step_noalloc(shape, params, [t.data_ptr() for t in gq.unbind(0)], [t.data_ptr() for t in gk.unbind(0)],
                             v.data_ptr(), u.data_ptr(), wl.n_iter, s.data_ptr(), c.data_ptr(), i.data_ptr(), stream)
    torch.cuda.synchronize()
    return [t.cpu().numpy() for t in (v, u, s, c, i)]


@pytest.mark.parametrize("flags,tol,shapes", [(0, 0.0, SHAPES), (sp.SN_FLAG_GRAM, 0.0, SHAPES), (0, 1e-4, PLANTED)],
                         ids=["chain", "gram", "chain-tol"])
def test_noalloc_matches_the_context_entry_point(flags, tol, shapes):
    for wl in shapes:  # two calls in a row, the second smaller
        gq, gk = all_weights(wl, "cuda")
        v0 = start_vectors(wl, "cuda")
        ref = _reference(wl, gq, gk, v0, flags, tol)
        got = _noalloc(wl, gq, gk, v0, flags, tol)
        for name, a, b in zip(("v", "u", "sigma", "scale", "iters"), ref, got):
            np.testing.assert_array_equal(a, b, err_msg=f"{wl.key}: {name}")
        if tol > 0:
            assert ref[4].max() > 2  # the device tail ran


def test_noalloc_refuses_a_shape_beyond_the_scratch():
    wl = WORKLOADS["llama2-70b-gqa"]
    shape = sp.sn_shape(wl.n_layers, wl.d_model, wl.n_q, wl.n_kv, wl.head_dim, sp.SN_BF16, 0)
    params = sp.sn_params(wl.alpha, 0.8, 448.0, 1e-4, 0, 0, 0)   # tolerance mode: 240 MB of workspace
    one = torch.zeros(4, device="cuda")
    with pytest.raises(sp.SpectralError) as e:
        sp.spectral_step_noalloc(shape, params, [one.data_ptr()] * wl.n_layers, [one.data_ptr()] * wl.n_layers,
                                 one.data_ptr(), 0, 3, one.data_ptr(), one.data_ptr(), 0, 0)
    assert e.value.code == sp.SN_EINVAL and "scratch" in sp.spectral_last_error()
