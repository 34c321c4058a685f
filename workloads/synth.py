"""Seeded synthetic weights, start vectors and tokens.

Layout of every weight tensor is the PyTorch ``Linear`` one: per layer,
``wq`` is ``[n_q * d_h, d]`` and ``wk`` is ``[n_kv * d_h, d]``, row-major, so
head ``h`` is the contiguous row block ``[h*d_h, (h+1)*d_h)``.  That block is
the transpose of the paper's per-head slice of W^Q in R^{d x n_q d_h}
(Sec. 3.1 defines Q = X W^Q).

Seeds come from ``numpy.random.SeedSequence([20260218, cfg_id, layer, stream])``.
Small factors (orthonormal spike directions, Hadamard column subsets, signs)
are always drawn on the CPU so that they are identical whatever device the
bulk Gaussian draws land on.  Bulk Gaussian draws use a torch generator on the
target device; a CPU draw and a GPU draw of the same seed differ, so a parity
check always hands the oracle the very tensors the GPU consumed.

Four weight recipes stand in for the paper's pretrained checkpoints (which are
not used here):

* ``gauss``   -- i.i.d. N(0, std^2) entries.
* ``spiked``  -- Gaussian bulk plus a planted rank-4 spike per head that the
  query and key slices share through one orthonormal d_h x 4 factor R, with
  spike magnitudes 5-20x the bulk spectral edge std*(sqrt(d)+sqrt(d_h)).
* ``planted`` -- every entry is a bf16-exact value +-s_i: the head's query
  slice is D H[:, S] diag(s) (Sylvester-Hadamard columns, random signs), the
  key slice c D' H[:, S'], so sigma_i(M_h) = s_i * c * d holds exactly on the
  stored bits.  s_2/s_1 = 251/256 (a 0.98 gap), the rest geometric.
"""

from __future__ import annotations

import dataclasses
import math
from dataclasses import dataclass

import numpy as np
import torch

SEED_ROOT = 20260218
STREAMS = {"q": 0, "k": 1, "v0": 2, "u0": 3, "perturb": 4, "x": 5, "plant": 6, "v0-layer": 7}


@dataclass(frozen=True)
class Workload:
    key: str
    cfg_id: int
    n_layers: int
    d_model: int
    n_q: int
    n_kv: int
    head_dim: int
    dtype: str          # "f32" or "bf16": storage type of the weights
    n_iter: int         # iterations (tol == 0) or the cap (tol > 0)
    alpha: float        # calibration factor used in the per-layer scale
    weights: str        # "gauss" | "spiked" | "planted"
    std: float = 0.02
    tol: float = 0.0
    warm: bool = False  # per-step recompute: warm start after a perturbation
    description: str = ""

    @property
    def group(self) -> int:
        return self.n_q // self.n_kv

    @property
    def n_heads(self) -> int:
        return self.n_layers * self.n_q

    @property
    def elem_bytes(self) -> int:
        return 4 if self.dtype == "f32" else 2

    @property
    def torch_dtype(self):
        return torch.float32 if self.dtype == "f32" else torch.bfloat16

    def replace(self, **kw) -> "Workload":
        return dataclasses.replace(self, **kw)

    def weight_bytes(self) -> tuple[int, int]:
        """Bytes of all layers' W_Q and W_K."""
        e = self.elem_bytes
        q = self.n_layers * self.n_q * self.head_dim * self.d_model * e
        k = self.n_layers * self.n_kv * self.head_dim * self.d_model * e
        return q, k


# alpha: the paper's values where it gives them (Sec. 3.2 "Selecting alpha in
# practice"); otherwise alpha_min for delta* = 1e-6, L = 1024 rounded up to the
# next 0.01, and clamped to 1 where the rank-aware bound is vacuous.
WORKLOADS: dict[str, Workload] = {
    w.key: w
    for w in [
        Workload("tiny", 0, 1, 32, 4, 4, 8, "f32", 20, 1.0, "gauss", 0.02,
                 description="tiny check: 1 layer, d=32, d_h=8, 4 MHA heads, fp32"),
        Workload("gpt2-small", 1, 12, 768, 12, 12, 64, "f32", 20, 0.15, "gauss", 0.02,
                 description="GPT-2-small shape, fp32, 20 iterations"),
        Workload("gpt2-xl", 2, 48, 1600, 25, 25, 64, "bf16", 30, 0.08, "gauss", 0.02,
                 description="GPT-2-XL shape, bf16, 30 iterations, cold start"),
        Workload("llama2-7b-spiked", 3, 32, 4096, 32, 32, 128, "bf16", 30, 0.04, "spiked", 0.02,
                 description="Llama-2-7B shape, bf16, Gaussian + planted rank-4 spikes, 30 iterations"),
        Workload("llama2-70b-gqa", 4, 80, 8192, 64, 8, 128, "bf16", 30, 0.02, "gauss", 0.015,
                 description="Llama-2-70B GQA shape (64 Q / 8 KV heads), bf16, 30 iterations, cold start"),
        Workload("llama2-70b-perstep", 5, 80, 8192, 64, 8, 128, "bf16", 1000, 0.02, "planted", 0.0,
                 tol=1e-4, warm=True,
                 description="Llama-2-70B GQA shape, bf16, planted 0.98-gap spectra, perturbed, "
                             "warm start, iterate to rel. tol 1e-4"),
    ]
}


def seed_of(cfg_id: int, layer: int, stream: str, step: int | None = None) -> int:
    """Seed of one (config, layer, stream); ``step`` (a burn-in step) extends
    the sequence so that every step draws afresh."""
    key = [SEED_ROOT, int(cfg_id), int(layer), STREAMS[stream]] + ([] if step is None else [int(step)])
    ss = np.random.SeedSequence(key)
    return int(ss.generate_state(1, dtype=np.uint64)[0] & np.uint64((1 << 62) - 1))


def _gen(device, seed: int) -> torch.Generator:
    g = torch.Generator(device=device)
    g.manual_seed(seed)
    return g


def _np_rng(cfg_id: int, layer: int, stream: str, step: int | None = None) -> np.random.Generator:
    key = [SEED_ROOT, int(cfg_id), int(layer), STREAMS[stream]] + ([] if step is None else [int(step)])
    return np.random.default_rng(np.random.SeedSequence(key))


def bf16_round(t: torch.Tensor) -> torch.Tensor:
    """Round to the nearest bf16 (ties to even) and widen back to float32."""
    return t.to(torch.bfloat16).to(torch.float32)


def _orthonormal(rng: np.random.Generator, batch: int, n: int, k: int) -> np.ndarray:
    a = rng.standard_normal((batch, n, k))
    q, _ = np.linalg.qr(a)
    return q


def _hadamard_rows(cols: torch.Tensor, d: int) -> torch.Tensor:
    """Entries H[c, cols[..., i]] of the order-d Sylvester-Hadamard matrix,
    returned as [..., i, c] (float32 +-1): (-1)^popcount(c & col)."""
    c = torch.arange(d, device=cols.device, dtype=torch.int32)
    x = cols.to(torch.int32).unsqueeze(-1) & c
    for sh in (16, 8, 4, 2, 1):
        x = x ^ (x >> sh)
    return (1 - 2 * (x & 1)).to(torch.float32)


def planted_singular_values(wl: Workload, layer: int) -> np.ndarray:
    """Exact singular values sigma_i(M_h) of the planted recipe, [n_q, d_h] float64."""
    s, c_k = _planted_scales(wl, layer)
    return s.astype(np.float64) * c_k * wl.d_model


def _planted_scales(wl: Workload, layer: int):
    dh = wl.head_dim
    rng = _np_rng(wl.cfg_id, layer, "plant")
    r = np.empty(dh, dtype=np.float64)
    r[0] = 1.0
    if dh > 1:
        r[1] = 251.0 / 256.0
    if dh > 2:
        r[2:] = np.geomspace(0.9, 0.01, dh - 2)
    r = bf16_round(torch.from_numpy(r).float()).double().numpy()
    expo = rng.integers(-2, 4, size=wl.n_q)
    base = 2.0 ** -6
    s = (2.0 ** expo)[:, None] * r[None, :] * base      # bf16-exact (power of two times bf16)
    return s, base


def layer_master(wl: Workload, layer: int, device="cpu") -> tuple[torch.Tensor, torch.Tensor]:
    """float32 master weights (wq [n_q*d_h, d], wk [n_kv*d_h, d]) of one layer."""
    d, dh, nq, nkv = wl.d_model, wl.head_dim, wl.n_q, wl.n_kv
    if wl.weights == "planted":
        if d & (d - 1):
            raise ValueError("planted weights need d a power of two")
        rng = _np_rng(wl.cfg_id, layer, "plant")
        rng.integers(-2, 4, size=nq)  # consumed by _planted_scales
        s, c_k = _planted_scales(wl, layer)
        sel_q = np.stack([rng.choice(d, size=dh, replace=False) for _ in range(nq)])
        sel_k = np.stack([rng.choice(d, size=dh, replace=False) for _ in range(nkv)])
        sgn_q = rng.integers(0, 2, size=(nq, d)) * 2 - 1
        sgn_k = rng.integers(0, 2, size=(nkv, d)) * 2 - 1
        hq = _hadamard_rows(torch.from_numpy(sel_q).to(device), d)          # [nq, dh, d]
        hk = _hadamard_rows(torch.from_numpy(sel_k).to(device), d)
        hq *= torch.from_numpy(sgn_q).to(device=device, dtype=torch.float32)[:, None, :]
        hk *= torch.from_numpy(sgn_k).to(device=device, dtype=torch.float32)[:, None, :]
        hq *= torch.from_numpy(s).to(device=device, dtype=torch.float32)[:, :, None]
        hk *= float(c_k)
        return hq.reshape(nq * dh, d), hk.reshape(nkv * dh, d)

    wq = torch.randn(nq * dh, d, generator=_gen(device, seed_of(wl.cfg_id, layer, "q")),
                     device=device, dtype=torch.float32) * wl.std
    wk = torch.randn(nkv * dh, d, generator=_gen(device, seed_of(wl.cfg_id, layer, "k")),
                     device=device, dtype=torch.float32) * wl.std
    if wl.weights == "spiked":
        if nq != nkv:
            raise ValueError("the spiked recipe is defined for MHA shapes")
        rng = _np_rng(wl.cfg_id, layer, "plant")
        rank = 4
        edge = wl.std * (math.sqrt(d) + math.sqrt(dh))
        r_shared = _orthonormal(rng, nq, dh, rank)       # [nq, dh, 4]
        u_q = _orthonormal(rng, nq, d, rank)             # [nq, d, 4]
        u_k = _orthonormal(rng, nq, d, rank)
        a = rng.uniform(5.0, 20.0, size=(nq, rank)) * edge
        b = rng.uniform(5.0, 20.0, size=(nq, rank)) * edge
        # layout rows of head h: (W^Q_h)^T = G^T + R diag(a) U^T
        sq = np.einsum("hik,hk,hck->hic", r_shared, a, u_q)
        sk = np.einsum("hik,hk,hck->hic", r_shared, b, u_k)
        wq += torch.from_numpy(sq.reshape(nq * dh, d)).to(device=device, dtype=torch.float32)
        wk += torch.from_numpy(sk.reshape(nkv * dh, d)).to(device=device, dtype=torch.float32)
    return wq, wk


def _store(t32: torch.Tensor, wl: Workload) -> torch.Tensor:
    return t32.to(wl.torch_dtype)


def perturb_master(wl: Workload, layer: int, wq: torch.Tensor, wk: torch.Tensor, step: int | None = None):
    """W <- W + 1e-3 * N(0,1) * ||W||_F / sqrt(numel), per layer tensor (float32 masters);
    ``step`` draws the perturbation of one burn-in step."""
    out = []
    for which, w in (("q", wq), ("k", wk)):
        g = _gen(w.device, seed_of(wl.cfg_id, layer, "perturb", step) + (0 if which == "q" else 1))
        rms = torch.sqrt(torch.mean(w.double() ** 2)).item()
        out.append(w + torch.randn(w.shape, generator=g, device=w.device, dtype=torch.float32) * (1e-3 * rms))
    return out[0], out[1]


def layer_weights(wl: Workload, layer: int, device="cpu", perturbed: bool = False, step: int | None = None):
    """Storage-dtype weights of one layer; ``perturbed`` adds the seeded
    perturbation (of burn-in step ``step`` if given) to the float32 master."""
    wq, wk = layer_master(wl, layer, device)
    if perturbed:
        wq, wk = perturb_master(wl, layer, wq, wk, step)
    return _store(wq, wl), _store(wk, wl)


def all_weights(wl: Workload, device="cpu", perturbed: bool = False, step: int | None = None):
    """Stacked storage-dtype weights: wq [L, n_q*d_h, d], wk [L, n_kv*d_h, d]."""
    L, d, dh = wl.n_layers, wl.d_model, wl.head_dim
    wq = torch.empty(L, wl.n_q * dh, d, dtype=wl.torch_dtype, device=device)
    wk = torch.empty(L, wl.n_kv * dh, d, dtype=wl.torch_dtype, device=device)
    for layer in range(L):
        q, k = layer_weights(wl, layer, device, perturbed, step)
        wq[layer].copy_(q)
        wk[layer].copy_(k)
        del q, k
    return wq, wk


def start_vectors(wl: Workload, device="cpu") -> torch.Tensor:
    """Random unit start vectors, one per query head: float32 [L, n_q, d].
    Drawn N(0, I) and normalised in float64 before the float32 store."""
    g = _gen(device, seed_of(wl.cfg_id, 0, "v0"))
    v = torch.randn(wl.n_layers, wl.n_q, wl.d_model, generator=g, device=device, dtype=torch.float64)
    v /= torch.linalg.vector_norm(v, dim=-1, keepdim=True)
    return v.to(torch.float32)


def layer_start_vectors(wl: Workload, device="cpu") -> torch.Tensor:
    """Random unit start vectors, one per layer (the layer-level estimator):
    float32 [L, d], drawn and normalised like ``start_vectors``."""
    g = _gen(device, seed_of(wl.cfg_id, 0, "v0-layer"))
    v = torch.randn(wl.n_layers, wl.d_model, generator=g, device=device, dtype=torch.float64)
    v /= torch.linalg.vector_norm(v, dim=-1, keepdim=True)
    return v.to(torch.float32)


def tokens(wl: Workload, n: int, spherical: bool = False, layer: int = 0, step: int | None = None) -> np.ndarray:
    """Token embeddings x_i ~ N(0, I_d) (float64, CPU); ``spherical`` rescales
    every row to norm sqrt(d), the post-normalisation model of Sec. 3.2;
    ``step`` draws the tokens of one burn-in step."""
    x = _np_rng(wl.cfg_id, layer, "x", step).standard_normal((n, wl.d_model))
    if spherical:
        x *= math.sqrt(wl.d_model) / np.linalg.norm(x, axis=1, keepdims=True)
    return x


def device_tokens(wl: Workload, n: int, device, step: int | None = None) -> torch.Tensor:
    """Post-normalisation tokens of every layer drawn on ``device`` (a torch
    generator, so not the draws of ``tokens``): x = sqrt(d) u, u uniform on the
    sphere, bf16 [L, n, d]."""
    out = torch.empty(wl.n_layers, n, wl.d_model, dtype=torch.bfloat16, device=device)
    for layer in range(wl.n_layers):
        x = torch.randn(n, wl.d_model, generator=_gen(device, seed_of(wl.cfg_id, layer, "x", step)), device=device,
                        dtype=torch.float32)
        x *= math.sqrt(wl.d_model) / torch.linalg.vector_norm(x, dim=1, keepdim=True)
        out[layer].copy_(x)
    return out
