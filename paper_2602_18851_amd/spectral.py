"""ctypes binding of ``libspectral.so`` (C ABI declared in include/spectral.h).

The functions named like the C entry points only marshal arguments; all
arithmetic runs in the HIP kernels.  ``Spectral`` wraps them for torch
tensors: torch supplies device memory and the current stream, nothing else.
There is no fallback: if the library is missing, loading raises.
"""

from __future__ import annotations

import ctypes
import os
from typing import Sequence

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libspectral.so")

SN_OK, SN_EINVAL, SN_ENULL, SN_EDTYPE, SN_EHIP, SN_ESTATE = 0, -1, -2, -3, -4, -5
SN_F32, SN_BF16 = 0, 1
SN_FLAG_VALU_K_SWEEP = 1
SN_FLAG_GRAM = 2
SN_FLAG_LAYER = 4
KIND_NAMES = ("k_sweep_first", "q_sweep", "k_sweep", "finalize", "gram_sweep", "gram_iterate", "gram_final_sweeps",
              "layer_row_sweeps", "layer_col_sweeps", "layer_reduce", "logits_projection", "logits_fp8",
              "tail_lists")
SN_PROFILE_KINDS = len(KIND_NAMES)

EXPORTED = (
    "spectral_init",
    "spectral_step",
    "spectral_step_noalloc",
    "spectral_step_layer",
    "spectral_set_stream",
    "spectral_destroy",
    "spectral_last_error",
    "spectral_workspace_bytes",
    "spectral_profile",
    "spectral_profile_read",
    "spectral_alpha_select",
    "spectral_overflow_terms",
    "spectral_auto_alpha",
    "spectral_slack_ratio",
    "spectral_logits_workspace_bytes",
    "spectral_logits_fp8",
)


class sn_shape(ctypes.Structure):
    _fields_ = [
        ("n_layers", ctypes.c_int32),
        ("d_model", ctypes.c_int32),
        ("n_q_heads", ctypes.c_int32),
        ("n_kv_heads", ctypes.c_int32),
        ("head_dim", ctypes.c_int32),
        ("dtype", ctypes.c_int32),
        ("ld", ctypes.c_int64),
    ]


class sn_params(ctypes.Structure):
    _fields_ = [
        ("alpha", ctypes.c_float),
        ("eta_fp8", ctypes.c_float),
        ("r_max", ctypes.c_float),
        ("tol", ctypes.c_float),
        ("q_strips", ctypes.c_int32),
        ("k_strips", ctypes.c_int32),
        ("flags", ctypes.c_int32),
    ]


class SpectralError(RuntimeError):
    def __init__(self, code: int, msg: str):
        super().__init__(f"spectral error {code}: {msg}")
        self.code = code


_lib = None


def load_library(path: str = LIB_PATH) -> ctypes.CDLL:
    """Loads the HIP library (once).  Raises if it has not been built."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(path):
        raise RuntimeError(f"{path} is missing: build it with `python -m paper_2602_18851_amd.build`")
    lib = ctypes.CDLL(path)
    vp, i32, i64 = ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64
    lib.spectral_init.argtypes = [ctypes.POINTER(vp), ctypes.POINTER(sn_shape), ctypes.POINTER(sn_params), vp]
    lib.spectral_init.restype = ctypes.c_int
    lib.spectral_step.argtypes = [vp, ctypes.POINTER(vp), ctypes.POINTER(vp), vp, vp, i32, vp, vp, vp]
    lib.spectral_step.restype = ctypes.c_int
    lib.spectral_step_noalloc.argtypes = [ctypes.POINTER(sn_shape), ctypes.POINTER(sn_params), ctypes.POINTER(vp),
                                          ctypes.POINTER(vp), vp, vp, i32, vp, vp, vp, vp]
    lib.spectral_step_noalloc.restype = ctypes.c_int
    lib.spectral_step_layer.argtypes = [vp, ctypes.POINTER(vp), ctypes.POINTER(vp), vp, vp, i32, vp, vp]
    lib.spectral_step_layer.restype = ctypes.c_int
    lib.spectral_set_stream.argtypes = [vp, vp]
    lib.spectral_set_stream.restype = ctypes.c_int
    lib.spectral_destroy.argtypes = [vp]
    lib.spectral_destroy.restype = None
    lib.spectral_last_error.argtypes = []
    lib.spectral_last_error.restype = ctypes.c_char_p
    lib.spectral_workspace_bytes.argtypes = [ctypes.POINTER(sn_shape), ctypes.POINTER(sn_params),
                                             ctypes.POINTER(i64)]
    lib.spectral_workspace_bytes.restype = ctypes.c_int
    lib.spectral_profile.argtypes = [vp, i32]
    lib.spectral_profile.restype = ctypes.c_int
    lib.spectral_profile_read.argtypes = [vp, ctypes.POINTER(ctypes.c_double), ctypes.POINTER(i64)]
    lib.spectral_profile_read.restype = ctypes.c_int
    dp = ctypes.POINTER(ctypes.c_double)
    lib.spectral_alpha_select.argtypes = [i32, i32, i64, i64, ctypes.c_double, dp, dp]
    lib.spectral_alpha_select.restype = ctypes.c_int
    lib.spectral_overflow_terms.argtypes = [i32, i32, i64, ctypes.c_double, ctypes.c_double, dp, dp]
    lib.spectral_overflow_terms.restype = ctypes.c_int
    lib.spectral_auto_alpha.argtypes = [dp, i64, ctypes.c_double, ctypes.c_double, dp]
    lib.spectral_auto_alpha.restype = ctypes.c_int
    lib.spectral_slack_ratio.argtypes = [ctypes.c_double, ctypes.c_double, i32, i32]
    lib.spectral_slack_ratio.restype = ctypes.c_double
    lib.spectral_logits_workspace_bytes.argtypes = [ctypes.POINTER(sn_shape), i32, ctypes.POINTER(i64)]
    lib.spectral_logits_workspace_bytes.restype = ctypes.c_int
    lib.spectral_logits_fp8.argtypes = [vp, ctypes.POINTER(vp), i64, i32, ctypes.POINTER(vp), ctypes.POINTER(vp), vp,
                                        vp, i64, vp, vp, vp]
    lib.spectral_logits_fp8.restype = ctypes.c_int
    _lib = lib
    return lib


def _check(rc: int):
    if rc != SN_OK:
        raise SpectralError(rc, spectral_last_error())


# ------------------------------------------------ C entry points, same names


def spectral_last_error() -> str:
    return load_library().spectral_last_error().decode()


def spectral_workspace_bytes(shape: sn_shape, params: sn_params) -> int:
    out = ctypes.c_int64(0)
    _check(load_library().spectral_workspace_bytes(ctypes.byref(shape), ctypes.byref(params), ctypes.byref(out)))
    return out.value


def spectral_init(shape: sn_shape, params: sn_params, stream: int = 0) -> int:
    ctx = ctypes.c_void_p()
    _check(load_library().spectral_init(ctypes.byref(ctx), ctypes.byref(shape), ctypes.byref(params),
                                        ctypes.c_void_p(stream)))
    return ctx.value


def spectral_step(ctx: int, wq_ptrs: Sequence[int], wk_ptrs: Sequence[int], v: int, u: int, n_iter: int,
                  sigma: int, scale: int, iters: int) -> None:
    n = len(wq_ptrs)
    wq = (ctypes.c_void_p * n)(*wq_ptrs)
    wk = (ctypes.c_void_p * n)(*wk_ptrs)
    _check(load_library().spectral_step(ctypes.c_void_p(ctx), wq, wk, ctypes.c_void_p(v),
                                        ctypes.c_void_p(u or None), int(n_iter), ctypes.c_void_p(sigma),
                                        ctypes.c_void_p(scale), ctypes.c_void_p(iters or None)))


def spectral_step_noalloc(shape: sn_shape, params: sn_params, wq_ptrs: Sequence[int], wk_ptrs: Sequence[int], v: int,
                          u: int, n_iter: int, sigma: int, scale: int, iters: int, stream: int = 0) -> None:
    n = len(wq_ptrs)
    wq = (ctypes.c_void_p * n)(*wq_ptrs)
    wk = (ctypes.c_void_p * n)(*wk_ptrs)
    _check(load_library().spectral_step_noalloc(ctypes.byref(shape), ctypes.byref(params), wq, wk, ctypes.c_void_p(v),
                                                ctypes.c_void_p(u or None), int(n_iter), ctypes.c_void_p(sigma),
                                                ctypes.c_void_p(scale), ctypes.c_void_p(iters or None),
                                                ctypes.c_void_p(stream)))


def spectral_step_layer(ctx: int, wq_ptrs: Sequence[int], wk_ptrs: Sequence[int], v: int, u: int, n_iter: int,
                        sigma: int, scale: int) -> None:
    n = len(wq_ptrs)
    wq = (ctypes.c_void_p * n)(*wq_ptrs)
    wk = (ctypes.c_void_p * n)(*wk_ptrs)
    _check(load_library().spectral_step_layer(ctypes.c_void_p(ctx), wq, wk, ctypes.c_void_p(v),
                                              ctypes.c_void_p(u or None), int(n_iter), ctypes.c_void_p(sigma),
                                              ctypes.c_void_p(scale)))

def spectral_set_stream(ctx: int, stream: int) -> None:
    _check(load_library().spectral_set_stream(ctypes.c_void_p(ctx), ctypes.c_void_p(stream)))


def spectral_destroy(ctx: int) -> None:
    load_library().spectral_destroy(ctypes.c_void_p(ctx))


def spectral_profile(ctx: int, enable: bool) -> None:
    _check(load_library().spectral_profile(ctypes.c_void_p(ctx), 1 if enable else 0))


def spectral_profile_read(ctx: int) -> dict:
    ms = (ctypes.c_double * SN_PROFILE_KINDS)()
    n = (ctypes.c_int64 * SN_PROFILE_KINDS)()
    _check(load_library().spectral_profile_read(ctypes.c_void_p(ctx), ms, n))
    return {KIND_NAMES[i]: (ms[i], n[i]) for i in range(SN_PROFILE_KINDS)}


# ------------------------------------------------ host calibration helpers


def spectral_alpha_select(d_model: int, head_dim: int, n_heads_total: int, seq_len: int,
                          delta: float) -> tuple[float, float]:
    """(gamma, alpha_min) of the selection rule (Sec. 3.2)."""
    g, a = ctypes.c_double(), ctypes.c_double()
    _check(load_library().spectral_alpha_select(d_model, head_dim, n_heads_total, seq_len, delta,
                                                ctypes.byref(g), ctypes.byref(a)))
    return g.value, a.value


def spectral_overflow_terms(d_model: int, head_dim: int, seq_len: int, alpha: float,
                            gamma: float) -> tuple[float, float]:
    t1, t2 = ctypes.c_double(), ctypes.c_double()
    _check(load_library().spectral_overflow_terms(d_model, head_dim, seq_len, alpha, gamma,
                                                  ctypes.byref(t1), ctypes.byref(t2)))
    return t1.value, t2.value


def spectral_auto_alpha(slack: Sequence[float], quantile: float = 0.9999, kappa: float = 1.0) -> float:
    arr = (ctypes.c_double * len(slack))(*slack)
    out = ctypes.c_double()
    _check(load_library().spectral_auto_alpha(arr, len(slack), quantile, kappa, ctypes.byref(out)))
    return out.value


def spectral_slack_ratio(max_abs_logit: float, sigma_layer: float, d_model: int, head_dim: int) -> float:
    return load_library().spectral_slack_ratio(max_abs_logit, sigma_layer, d_model, head_dim)


def spectral_logits_workspace_bytes(shape: sn_shape, seq_len: int) -> int:
    out = ctypes.c_int64(0)
    _check(load_library().spectral_logits_workspace_bytes(ctypes.byref(shape), int(seq_len), ctypes.byref(out)))
    return out.value


def spectral_logits_fp8(ctx: int, x_ptrs: Sequence[int], ld_x: int, seq_len: int, wq_ptrs: Sequence[int],
                        wk_ptrs: Sequence[int], scale: int, workspace: int, workspace_bytes: int, codes: int,
                        max_abs: int, n_over: int) -> None:
    n = len(wq_ptrs)
    xs = (ctypes.c_void_p * n)(*x_ptrs)
    wq = (ctypes.c_void_p * n)(*wq_ptrs)
    wk = (ctypes.c_void_p * n)(*wk_ptrs)
    _check(load_library().spectral_logits_fp8(ctypes.c_void_p(ctx), xs, int(ld_x), int(seq_len), wq, wk,
                                              ctypes.c_void_p(scale), ctypes.c_void_p(workspace),
                                              int(workspace_bytes), ctypes.c_void_p(codes or None),
                                              ctypes.c_void_p(max_abs), ctypes.c_void_p(n_over)))


# ------------------------------------------- consumer-side calibration


class AutoAlpha:
    """Auto-alpha calibration (Sec. 3.5; App. M, Algorithm "Auto-alpha
    Calibration") driven by the FP8 consumer.  Each burn-in step observes,
    per layer l, the largest logit M = max_h max|S~_h| * scale_l (the
    consumer's max_abs times the scale it divided by) and the bound
    B_max = sigma^(l) d / sqrt(d_h), sigma^(l) = max_h sigma_h of the step's
    estimate, and records r = M / B_max (spectral_slack_ratio).  alpha()
    returns Quantile_q(R) * kappa (spectral_auto_alpha).  Layers whose sigma
    or scale is not finite and positive (degenerate heads) are skipped."""

    def __init__(self, d_model: int, head_dim: int, quantile: float = 0.9999, kappa: float = 1.0):
        self.d_model, self.head_dim = int(d_model), int(head_dim)
        self.quantile, self.kappa = float(quantile), float(kappa)
        self.ratios: list[float] = []

    def observe(self, sigma, scale, max_abs) -> list[float]:
        """sigma [L, n_q], scale [L], max_abs [L, n_q] (tensors or arrays) of
        one step; returns the step's ratios, one per layer."""
        import numpy as np

        def host(t):
            return np.asarray(t.detach().double().cpu().numpy() if hasattr(t, "detach") else t, dtype=np.float64)

        sig, sc, mx = host(sigma), host(scale), host(max_abs)
        out = []
        for l in range(sc.shape[0]):
            s_l, m_l = float(sig[l].max()), float(mx[l].max())
            if not (np.isfinite(s_l) and s_l > 0 and np.isfinite(sc[l]) and sc[l] > 0 and np.isfinite(m_l)):
                continue
            out.append(spectral_slack_ratio(m_l * float(sc[l]), s_l, self.d_model, self.head_dim))
        self.ratios.extend(out)
        return out

    def alpha(self) -> float:
        return spectral_auto_alpha(self.ratios, self.quantile, self.kappa)


def fp8_report(max_abs, n_over, r_max: float = 448.0) -> dict:
    """Statistics of one consumer call in the form of the paper's tables:
    layers with any logit past R_max (Table "pretrained", "Overflow") and the
    largest scaled logit ("Max Scaled"); FP8 range utilisation max|S~| / R_max
    (Sec. 1), per layer (its largest head) and per head, as median, P10 and
    P90 in percent (App. J, Table "utilization_app")."""
    import numpy as np

    mx = np.asarray(max_abs.detach().double().cpu().numpy() if hasattr(max_abs, "detach") else max_abs,
                    dtype=np.float64)
    ov = np.asarray(n_over.detach().cpu().numpy() if hasattr(n_over, "detach") else n_over)
    per_layer = 100.0 * mx.max(axis=1) / r_max
    per_head = 100.0 * mx.reshape(-1) / r_max

    def q(a):
        return {"median": float(np.median(a)), "p10": float(np.percentile(a, 10)), "p90": float(np.percentile(a, 90))}

    return {"overflow_layers": int((ov.reshape(ov.shape[0], -1) > 0).any(axis=1).sum()), "layers": int(mx.shape[0]),
            "overflow_logits": int(ov.sum()), "max_scaled": float(mx.max()),
            "utilization_pct_layers": q(per_layer), "utilization_pct_heads": q(per_head)}


# ----------------------------------------------------------- torch wrapper


class Spectral:
    """One context per model shape.  ``step`` runs the estimator on the
    current torch stream of the tensors' device."""

    def __init__(self, n_layers: int, d_model: int, n_q_heads: int, n_kv_heads: int, head_dim: int,
                 dtype: str, alpha: float, eta_fp8: float = 0.8, r_max: float = 448.0, tol: float = 0.0,
                 ld: int = 0, q_strips: int = 0, k_strips: int = 0, flags: int = 0):
        import torch

        if dtype not in ("f32", "bf16"):
            raise ValueError("dtype must be 'f32' or 'bf16'")
        self.torch_dtype = torch.float32 if dtype == "f32" else torch.bfloat16
        self.shape = sn_shape(n_layers, d_model, n_q_heads, n_kv_heads, head_dim,
                              SN_F32 if dtype == "f32" else SN_BF16, ld)
        self.params = sn_params(alpha, eta_fp8, r_max, tol, q_strips, k_strips, flags)
        self._stream = torch.cuda.current_stream().cuda_stream
        self.ctx = spectral_init(self.shape, self.params, self._stream)

    @property
    def ld(self) -> int:
        return self.shape.ld or self.shape.d_model

    def close(self):
        if getattr(self, "ctx", None):
            spectral_destroy(self.ctx)
            self.ctx = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    def _layer_ptrs(self, w, rows: int) -> list[int]:
        import torch

        if isinstance(w, torch.Tensor) and w.dim() == 3:
            # one stacked tensor: checked once, layer l starts l * stride(0) elements in
            L = self.shape.n_layers
            if w.shape[0] != L:
                raise ValueError(f"expected {L} layers, got {w.shape[0]}")
            if not w.is_cuda or w.dtype != self.torch_dtype:
                raise ValueError(f"weights must be {self.torch_dtype} CUDA tensors")
            if w.shape[1] != rows or w.shape[2] < self.shape.d_model:
                raise ValueError(f"layer weight must be [{rows}, >= {self.shape.d_model}], got {tuple(w.shape[1:])}")
            if w.stride(2) != 1 or w.stride(1) != self.ld:
                raise ValueError(f"layer weight must be row-major with row stride {self.ld}")
            base, step = w.data_ptr(), w.stride(0) * w.element_size()
            return [base + l * step for l in range(L)]
        layers = list(w)
        if len(layers) != self.shape.n_layers:
            raise ValueError(f"expected {self.shape.n_layers} layers, got {len(layers)}")
        ptrs = []
        for t in layers:
            if not t.is_cuda or t.dtype != self.torch_dtype:
                raise ValueError(f"weights must be {self.torch_dtype} CUDA tensors")
            if t.dim() != 2 or t.shape[0] != rows or t.shape[1] < self.shape.d_model:
                raise ValueError(f"layer weight must be [{rows}, >= {self.shape.d_model}], got {tuple(t.shape)}")
            if t.stride(1) != 1 or t.stride(0) != self.ld:
                raise ValueError(f"layer weight must be row-major with row stride {self.ld}")
            ptrs.append(t.data_ptr())
        return ptrs

    def step(self, wq, wk, v, n_iter: int, u=None, sigma=None, scale=None, iters=None):
        """wq: [L, n_q*d_h, d] tensor or list of [n_q*d_h, d]; wk likewise with
        n_kv; v: float32 [L, n_q, d] (in/out).  Returns (sigma, scale, iters)."""
        import torch

        s = self.shape
        L, nq, d = s.n_layers, s.n_q_heads, s.d_model
        wq_p = self._layer_ptrs(wq, nq * s.head_dim)
        wk_p = self._layer_ptrs(wk, s.n_kv_heads * s.head_dim)
        dev = v.device
        for name, t, shp in (("v", v, (L, nq, d)), ("u", u, (L, nq, d))):
            if t is None:
                continue
            if t.dtype != torch.float32 or tuple(t.shape) != shp or not t.is_contiguous() or not t.is_cuda:
                raise ValueError(f"{name} must be a contiguous float32 CUDA tensor of shape {shp}")
        if sigma is None:
            sigma = torch.empty(L, nq, dtype=torch.float32, device=dev)
        if scale is None:
            scale = torch.empty(L, dtype=torch.float32, device=dev)
        if iters is None:
            iters = torch.empty(L, nq, dtype=torch.int32, device=dev)
        stream = torch.cuda.current_stream(dev).cuda_stream
        if stream != self._stream:
            spectral_set_stream(self.ctx, stream)
            self._stream = stream
        spectral_step(self.ctx, wq_p, wk_p, v.data_ptr(), u.data_ptr() if u is not None else 0, n_iter,
                      sigma.data_ptr(), scale.data_ptr(), iters.data_ptr())
        return sigma, scale, iters

    def step_layer(self, wq, wk, v, n_iter: int, u=None, sigma=None, scale=None):
        """Layer-level form (context made with SN_FLAG_LAYER): v, u float32
        [L, d] (v in/out).  Returns (sigma [L], scale [L])."""
        import torch

        s = self.shape
        L, d = s.n_layers, s.d_model
        wq_p = self._layer_ptrs(wq, s.n_q_heads * s.head_dim)
        wk_p = self._layer_ptrs(wk, s.n_kv_heads * s.head_dim)
        for name, t in (("v", v), ("u", u)):
            if t is None:
                continue
            if t.dtype != torch.float32 or tuple(t.shape) != (L, d) or not t.is_contiguous() or not t.is_cuda:
                raise ValueError(f"{name} must be a contiguous float32 CUDA tensor of shape {(L, d)}")
        dev = v.device
        if sigma is None:
            sigma = torch.empty(L, dtype=torch.float32, device=dev)
        if scale is None:
            scale = torch.empty(L, dtype=torch.float32, device=dev)
        stream = torch.cuda.current_stream(dev).cuda_stream
        if stream != self._stream:
            spectral_set_stream(self.ctx, stream)
            self._stream = stream
        spectral_step_layer(self.ctx, wq_p, wk_p, v.data_ptr(), u.data_ptr() if u is not None else 0, n_iter,
                            sigma.data_ptr(), scale.data_ptr())
        return sigma, scale

    def logits_fp8(self, x, wq, wk, scale, want_codes: bool = False, workspace=None):
        """FP8 E4M3 logit consumer.  x: bf16 [L, seq, d] tensor (or list of
        [seq, >= d] row-major layers); scale: float32 [L] on the device.
        Returns (max_abs [L, n_q], n_over [L, n_q], codes [L, n_q, seq, seq]
        uint8 or None)."""
        import torch

        s = self.shape
        L, nq = s.n_layers, s.n_q_heads
        layers = list(x.unbind(0)) if isinstance(x, torch.Tensor) and x.dim() == 3 else list(x)
        if len(layers) != L:
            raise ValueError(f"expected {L} token layers, got {len(layers)}")
        seq, ld_x = layers[0].shape[0], layers[0].stride(0)
        for t in layers:
            if not t.is_cuda or t.dtype != torch.bfloat16 or t.dim() != 2 or t.stride(1) != 1 \
                    or t.shape[0] != seq or t.stride(0) != ld_x or t.shape[1] < s.d_model:
                raise ValueError("token layers must be bf16 CUDA [seq, >= d] row-major with one row stride")
        wq_p = self._layer_ptrs(wq, nq * s.head_dim)
        wk_p = self._layer_ptrs(wk, s.n_kv_heads * s.head_dim)
        if scale.dtype != torch.float32 or tuple(scale.shape) != (L,) or not scale.is_cuda:
            raise ValueError(f"scale must be a float32 CUDA tensor of shape ({L},)")
        dev = scale.device
        need = spectral_logits_workspace_bytes(self.shape, seq)
        if workspace is None or workspace.numel() < need:
            workspace = torch.empty(need, dtype=torch.uint8, device=dev)
        max_abs = torch.empty(L, nq, dtype=torch.float32, device=dev)
        n_over = torch.empty(L, nq, dtype=torch.int32, device=dev)
        codes = torch.empty(L, nq, seq, seq, dtype=torch.uint8, device=dev) if want_codes else None
        stream = torch.cuda.current_stream(dev).cuda_stream
        if stream != self._stream:
            spectral_set_stream(self.ctx, stream)
            self._stream = stream
        spectral_logits_fp8(self.ctx, [t.data_ptr() for t in layers], ld_x, seq, wq_p, wk_p, scale.data_ptr(),
                            workspace.data_ptr(), workspace.numel(), codes.data_ptr() if want_codes else 0,
                            max_abs.data_ptr(), n_over.data_ptr())
        return max_abs, n_over, codes

    def profile(self, enable: bool = True):
        spectral_profile(self.ctx, enable)

    def profile_read(self) -> dict:
        return spectral_profile_read(self.ctx)
