"""Throughput of the per-head spectral-norm path on one MI355X.

One step = one spectral_step call: all layers, all query heads, n_iter
power-iteration steps each (one W_K sweep from v, then per step one fused W_Q
sweep and one fused W_K sweep), plus the per-layer E4M3 scale.  Weights,
start vectors and outputs are resident in HBM before the timed region.

    python bench.py [--gpus 1] [--steps K] [--warmup W] [--workload KEY] [--form chain|gram]

Prints one JSON line.  ``value`` is heads*iterations per second over all
layers; ``roofline`` reports the dominant kernel against the HBM peak (the
W_Q sweep of the default sweep chain; the Gram sweep with ``--form gram``,
which runs the same iterates through d_h x d_h Gram matrices);
``cpu_baseline`` times the float64 oracle on host cores over a bounded sample
of the same workload.
"""

from __future__ import annotations

import argparse
import hashlib
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK_GBPS = 8000.0   # MI355X HBM3E, vendor figure
# what `dtype` ("f32") summarises: the arithmetic of each form's kernels
ARITHMETIC = {
    "chain": "W_Q sweep: fp32 FMA on the weights (bf16 widened exactly); W_K sweep of grouped bf16 heads (3..8 query "
             "heads per key head, d_h 64/128): bf16 matrix-core products of K with each fp32 vector split into hi and "
             "lo bf16 halves (about 16 significant bits), fp32 accumulation; other W_K sweeps fp32 FMA; norms, "
             "normalisation and the scale fp32",
    "gram": "Gram matrices: bf16 (fp32: fp32) matrix-core products, fp32 accumulation; d_h-space iteration, norms "
            "and the scale fp32; final sweeps as in the chain",
    "layer": "fp32 FMA on the weights (bf16 widened exactly), fp32 norms and scale",
}
METRIC = "heads·iters/sec (all layers) and achieved HBM GB/s vs MI355X peak"
TRAFFIC_FILE = os.path.join(ROOT, "profiles", "q_sweep_traffic.json")
KERNEL_DIR = os.path.join(ROOT, "paper_2602_18851_amd", "csrc")


def log(msg: str) -> None:
    """Progress of the run on stderr (the JSON line alone goes to stdout)."""
    print(f"[bench] {msg}", file=sys.stderr, flush=True)


def parse():
    p = argparse.ArgumentParser()
    p.add_argument("--gpus", type=int, default=1)
    # the warm-up and timed-call counts of the paper's protocol (App. "Overhead Measurement")
    p.add_argument("--steps", type=int, default=100)
    p.add_argument("--warmup", type=int, default=10)
    p.add_argument("--workload", default="llama2-70b-gqa")
    p.add_argument("--n-iter", type=int, default=0, help="override the workload's iteration count")
    p.add_argument("--cpu-seconds", type=float, default=15.0, help="budget of the oracle CPU baseline")
    p.add_argument("--no-cpu-baseline", action="store_true")
    p.add_argument("--q-strips", type=int, default=0, help="column strips per head in the W_Q sweep (0 = auto)")
    p.add_argument("--k-strips", type=int, default=0, help="column strips per KV head in the W_K sweep (0 = auto)")
    p.add_argument("--flags", type=int, default=0, help="sn_params.flags (SN_FLAG_* bits)")
    p.add_argument("--form", choices=("chain", "gram", "layer", "fp8"), default="chain",
                   help="gram: the Gram form of the iteration (adds SN_FLAG_GRAM); layer: the paper-literal "
                        "layer-level estimator (one u, v per layer, spectral_step_layer); fp8: the E4M3 logit "
                        "consumer of the scale (spectral_logits_fp8) on --seq tokens per layer")
    p.add_argument("--seq", type=int, default=1024, help="tokens per layer of the fp8 form")
    p.add_argument("--graph", action="store_true",
                   help="chain/gram forms: capture one call into a HIP graph and time its replays")
    p.add_argument("--no-extras", action="store_true",
                   help="chain/gram forms: skip the context lines (one-iteration call, warm per-step call)")
    p.add_argument("--mode", choices=("bench", "copy", "perstep"), default="bench",
                   help="copy: one plain device copy of --copy-bytes, the reference for HBM byte counters; "
                        "perstep: only the per-step recompute scenario (its JSON line), in the --form chosen")
    p.add_argument("--copy-bytes", type=int, default=4 << 30)
    p.add_argument("--flush", action="store_true",
                   help="chain/gram forms: before every timed call write a 1 GiB scratch buffer (evicts L2 and the "
                        "256 MB Infinity Cache), each call timed alone by HIP events")
    p.add_argument("--calib-steps", type=int, default=20, help="fp8 form: auto-alpha burn-in steps")
    return p.parse_args()


def copy_reference(nbytes: int):
    """One device-to-device copy of a known size: its FETCH_SIZE / WRITE_SIZE
    counter readings calibrate the per-dispatch byte counters."""
    import torch

    src = torch.full((nbytes,), 7, dtype=torch.uint8, device="cuda")
    dst = torch.empty_like(src)
    torch.cuda.synchronize()
    dst.copy_(src)
    torch.cuda.synchronize()
    print(json.dumps({"mode": "copy", "bytes_read": nbytes, "bytes_written": nbytes}), flush=True)


def code_tokens(text: str) -> str:
    """C++ source with comments removed and every run of whitespace made one
    space: an edit of a comment or of layout leaves it unchanged."""
    out, i, n = [], 0, len(text)
    while i < n:
        c = text[i]
        if c in "\"'":  # string or character literal, kept whole
            j = i + 1
            while j < n and text[j] != c:
                j += 2 if text[j] == "\\" else 1
            out.append(text[i:j + 1])
            i = j + 1
        elif text.startswith("//", i):
            j = text.find("\n", i)
            i = n if j < 0 else j
            out.append(" ")
        elif text.startswith("/*", i):
            j = text.find("*/", i + 2)
            i = n if j < 0 else j + 2
            out.append(" ")
        else:
            out.append(c)
            i += 1
    return " ".join("".join(out).split())


def source_hash() -> str:
    """Hash of the code (comments and layout aside) of every kernel source and
    header: the counters are void once any of it changes."""
    h = hashlib.sha256()
    for name in sorted(os.listdir(KERNEL_DIR)):
        if name.endswith((".hip", ".h", ".cpp")):
            with open(os.path.join(KERNEL_DIR, name), encoding="utf-8") as f:
                h.update(name.encode() + b"\0" + code_tokens(f.read()).encode())
    return h.hexdigest()[:16]


def measured_traffic(kernel: str = ""):
    """HBM bytes per launch of the W_Q sweep (or of ``kernel``, a sub-entry
    such as "gram_sweep") from the committed rocprofv3 counter summary, if it
    was taken on the current kernel source; else None."""
    try:
        with open(TRAFFIC_FILE) as f:
            t = json.load(f)
    except (OSError, ValueError):
        return None
    if t.get("source_sha256_16") != source_hash():
        return None
    return (t.get(kernel) or {}).get("bytes_per_launch") if kernel else t.get("bytes_per_launch")


def host_info() -> dict:
    """The host the CPU baseline ran on: logical CPUs and the CPU model."""
    model = ""
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    model = line.split(":", 1)[1].strip()
                    break
    except OSError:
        pass
    return {"os_cpu_count": os.cpu_count(), "cpu_model": model}


def cpu_baseline(wl, budget_s: float, n_iter: int):
    """The float64 oracle (per head, the paper's step order) on host cores,
    over as many heads of the workload as fit in the time budget."""
    import numpy as np
    from threadpoolctl import threadpool_info

    from oracle.power_iteration import head_slices, power_iteration
    from workloads import layer_weights, start_vectors

    v0 = start_vectors(wl.replace(n_layers=1), "cpu")[0].double().numpy()
    wq, wk = layer_weights(wl, 0, "cpu")
    wq, wk = wq.float().numpy(), wk.float().numpy()
    heads = 0
    t0 = time.perf_counter()
    while time.perf_counter() - t0 < budget_s:
        h = heads % wl.n_q
        WQ, WK = head_slices(wq, wk, h, wl.n_kv, wl.head_dim)
        power_iteration(WQ, WK, v0[h], n_iter)
        heads += 1
    dt = time.perf_counter() - t0
    threads = max([i.get("num_threads", 1) for i in threadpool_info()] or [1])
    return {
        "value": heads * n_iter / dt,
        "unit": "heads·iters/s",
        "cores": int(threads),
        "kind": "oracle",
        "sample": f"{heads} head estimates cycling over the {wl.n_q} query heads of layer 0, {n_iter} iterations "
                  f"each, float64 numpy (implicit 4-GEMV chain per head), {dt:.1f} s",
        "cores_note": "cores = BLAS threads the oracle ran with",
        **host_info(),
    }


def cpu_explicit_m(wl, budget_s: float, n_iter: int):
    """The route the method avoids, timed beside the baseline: the oracle's
    cross-check that forms M = Q_h^T K_j (d x d, float64) per head and runs
    dense power iteration on it, over at least one head and as many more of
    layer 0 as fit in the budget."""
    import numpy as np

    from oracle.explicit import dense_power_iteration, interaction_matrix
    from oracle.power_iteration import head_slices
    from workloads import layer_weights, start_vectors

    v0 = start_vectors(wl.replace(n_layers=1), "cpu")[0].double().numpy()
    wq, wk = layer_weights(wl, 0, "cpu")
    wq, wk = wq.float().numpy(), wk.float().numpy()
    heads = 0
    t0 = time.perf_counter()
    while heads == 0 or time.perf_counter() - t0 < budget_s:
        h = heads % wl.n_q
        WQ, WK = head_slices(wq, wk, h, wl.n_kv, wl.head_dim)
        dense_power_iteration(interaction_matrix(WQ, WK), v0[h], n_iter)
        heads += 1
    dt = time.perf_counter() - t0
    return {"value": heads * n_iter / dt, "unit": "heads·iters/s",
            "sample": f"{heads} heads of layer 0, M formed ({wl.d_model} x {wl.d_model} float64) and "
                      f"{n_iter} dense iterations each, {dt:.1f} s"}


def cpu_baseline_layer(wl, budget_s: float, n_iter: int):
    """The oracle's paper-literal layer estimator on host cores, layer 0 repeated."""
    from threadpoolctl import threadpool_info

    from oracle.power_iteration import power_iteration_layer
    from workloads import layer_start_vectors, layer_weights

    v0 = layer_start_vectors(wl.replace(n_layers=1), "cpu")[0].double().numpy()
    wq, wk = layer_weights(wl, 0, "cpu")
    wq, wk = wq.double().numpy().T, wk.double().numpy().T
    runs = 0
    t0 = time.perf_counter()
    while time.perf_counter() - t0 < budget_s:
        power_iteration_layer(wq, wk, v0, n_iter, wl.n_q // wl.n_kv, wl.head_dim)
        runs += 1
    dt = time.perf_counter() - t0
    threads = max([i.get("num_threads", 1) for i in threadpool_info()] or [1])
    return {"value": runs * n_iter / dt, "unit": "layers·iters/s", "cores": int(threads), "kind": "oracle",
            "sample": f"{runs} runs of the layer-0 estimator, {n_iter} iterations each, float64 numpy, {dt:.1f} s",
            **host_info()}


def cpu_baseline_fp8(wl, budget_s: float, seq: int):
    """The oracle's E4M3 logit consumer on host cores: heads of layer 0 in turn."""
    import numpy as np
    import torch
    from threadpoolctl import threadpool_info

    from oracle import fp8_consumer
    from workloads import layer_weights, tokens

    wq, wk = layer_weights(wl, 0, "cpu")
    wq, wk = wq.double().numpy(), wk.double().numpy()
    x = torch.from_numpy(tokens(wl, seq, spherical=True, layer=0)).to(torch.bfloat16).double().numpy()
    heads = 0
    t0 = time.perf_counter()
    while time.perf_counter() - t0 < budget_s:
        fp8_consumer.consume_layer(x, wq, wk, 0.05, wl.n_kv, wl.head_dim, heads=[heads % wl.n_q])
        heads += 1
    dt = time.perf_counter() - t0
    threads = max([i.get("num_threads", 1) for i in threadpool_info()] or [1])
    return {"value": heads * seq * seq / dt, "unit": "scaled logits/s", "cores": int(threads), "kind": "oracle",
            "sample": f"{heads} heads of layer 0 ({seq} tokens: projections, logits, E4M3 codes, counts), "
                      f"float64 numpy, {dt:.1f} s", **host_info()}


def context_lines(args, flags: int) -> dict:
    """Calls reported beside the headline (context, not the metric): n_iter
    = 1 from cold vectors (one pure stream of W_K, W_Q, W_K); for the sweep
    chain, the Gram form on the same weights and iteration count; and the
    per-step scenario of Sec. 5.1 (planted 0.98-gap spectra iterated to
    tolerance 1e-4 untimed, weights perturbed, then one timed warm call), in
    the chosen form and, for the chain, in the Gram form too."""
    import torch

    from paper_2602_18851_amd import Spectral
    from workloads import WORKLOADS, all_weights, start_vectors

    dev = torch.device("cuda", 0)
    out = {}
    wl = WORKLOADS[args.workload]
    wq, wk = all_weights(wl, dev)
    est = Spectral(wl.n_layers, wl.d_model, wl.n_q, wl.n_kv, wl.head_dim, wl.dtype, wl.alpha, flags=flags)
    v = start_vectors(wl, dev)
    est.step(wq, wk, v, 1)
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    for _ in range(5):
        est.step(wq, wk, v, 1)
    e1.record()
    torch.cuda.synchronize()
    ms = e0.elapsed_time(e1) / 5
    q_bytes, k_bytes = wl.weight_bytes()
    H = wl.n_layers * wl.n_q
    out["n_iter_1"] = {"ms": ms, "heads_iters_per_s": H / (ms * 1e-3),
                       "effective_GBps": (q_bytes + 2 * k_bytes + 12 * wl.d_model * H) / (ms * 1e-3) / 1e9}
    est.close()

    from paper_2602_18851_amd.spectral import SN_FLAG_GRAM
    if not flags & SN_FLAG_GRAM and wl.head_dim >= 16:
        # the Gram form on the same weights and iteration count: the same
        # iterates through d_h x d_h Gram matrices, weights read about four
        # times per call instead of twice per iteration
        n_iter = args.n_iter or wl.n_iter
        est = Spectral(wl.n_layers, wl.d_model, wl.n_q, wl.n_kv, wl.head_dim, wl.dtype, wl.alpha,
                       flags=flags | SN_FLAG_GRAM)
        v = start_vectors(wl, dev)
        for _ in range(3):
            est.step(wq, wk, v, n_iter)
        torch.cuda.synchronize()
        est.profile(True)
        n = 20
        e0.record()
        for _ in range(n):
            est.step(wq, wk, v, n_iter)
        e1.record()
        torch.cuda.synchronize()
        prof = est.profile_read()
        est.profile(False)
        ms = e0.elapsed_time(e1) / n
        g_ms, g_n = prof["gram_sweep"]
        # every weight read once, the upper-triangle 16 x 16 blocks written once per query / key head
        g_bytes = q_bytes + k_bytes + (H + wl.n_layers * wl.n_kv) * wl.head_dim * (wl.head_dim + 16) // 2 * 4
        out["gram_form"] = {"ms": ms, "heads_iters_per_s": H * n_iter / (ms * 1e-3), "n_iter": n_iter,
                            "gram_sweep_ms": g_ms / g_n,
                            "gram_sweep_GBps": g_bytes / (g_ms / g_n * 1e-3) / 1e9,
                            "gram_sweep_frac_of_peak": g_bytes / (g_ms / g_n * 1e-3) / 1e9 / HBM_PEAK_GBPS,
                            "note": "SN_FLAG_GRAM on the same weights; not the headline, whose iterations each "
                                    "stream the weights"}
        est.close()
    del wq, wk, v
    torch.cuda.empty_cache()

    out["per_step_warm"] = per_step_warm(flags)
    if not flags & SN_FLAG_GRAM:
        out["per_step_warm_gram"] = per_step_warm(flags | SN_FLAG_GRAM)
    return out


def per_step_warm(flags: int) -> dict:
    """The per-step scenario of Sec. 5.1 on the 70B shape: planted 0.98-gap
    spectra iterated to tolerance 1e-4 from cold vectors (untimed), weights
    perturbed, then the same warm call five times from the same vectors, each
    timed by HIP events around it on the stream and by the wall clock from
    the call to the end of a synchronisation after it (the call itself never
    waits on the host)."""
    import numpy as np
    import torch

    from paper_2602_18851_amd import Spectral
    from workloads import WORKLOADS, all_weights, start_vectors

    dev = torch.device("cuda", 0)
    wl = WORKLOADS["llama2-70b-perstep"]
    wq, wk = all_weights(wl, dev)
    est = Spectral(wl.n_layers, wl.d_model, wl.n_q, wl.n_kv, wl.head_dim, wl.dtype, wl.alpha, tol=wl.tol,
                   flags=flags)
    v = start_vectors(wl, dev)
    _, _, it0 = est.step(wq, wk, v, wl.n_iter)
    it0 = it0.cpu().numpy()
    wq1, wk1 = all_weights(wl, dev, perturbed=True)
    v_warm = v.clone()
    torch.cuda.synchronize()
    times, ev_ms = [], []
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    for _ in range(5):   # the same warm call from the same vectors
        v.copy_(v_warm)
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        e0.record()
        _, _, it = est.step(wq1, wk1, v, wl.n_iter)
        e1.record()
        torch.cuda.synchronize()
        times.append((time.perf_counter() - t0) * 1e3)
        ev_ms.append(e0.elapsed_time(e1))
    it = it.cpu().numpy()
    res = {"workload": wl.key, "tol": wl.tol, "cold_iters_median": float(np.median(it0)),
           "cold_iters_max": int(it0.max()), "warm_iters_median": float(np.median(it)),
           "warm_iters_max": int(it.max()), "warm_ms": float(np.median(ev_ms)), "warm_ms_wall": min(times),
           "note": "one warm spectral_step: HIP events on its stream (median of 5), and the wall clock to the end "
                   "of a synchronisation after it (best of 5)"}
    est.close()
    return res


def bench_fp8(args):
    """The E4M3 logit consumer: every layer and query head of the workload on
    --seq post-normalisation tokens per layer, codes written."""
    import numpy as np
    import torch

    from paper_2602_18851_amd import Spectral
    from paper_2602_18851_amd.spectral import SN_FLAG_GRAM
    from workloads import WORKLOADS, all_weights, start_vectors, tokens

    wl = WORKLOADS[args.workload]
    seq = args.seq
    torch.cuda.set_device(0)
    dev = torch.device("cuda", 0)
    wq, wk = all_weights(wl, dev)
    x = torch.stack([torch.from_numpy(tokens(wl, seq, spherical=True, layer=l)).to(torch.bfloat16)
                     for l in range(wl.n_layers)]).to(dev)
    est = Spectral(wl.n_layers, wl.d_model, wl.n_q, wl.n_kv, wl.head_dim, wl.dtype, wl.alpha, flags=SN_FLAG_GRAM)
    _, scale, _ = est.step(wq, wk, start_vectors(wl, dev), wl.n_iter)   # the layer scales the consumer uses
    from paper_2602_18851_amd.spectral import spectral_logits_fp8, spectral_logits_workspace_bytes
    ws = torch.empty(spectral_logits_workspace_bytes(est.shape, seq), dtype=torch.uint8, device=dev)
    codes = torch.empty(wl.n_layers, wl.n_q, seq, seq, dtype=torch.uint8, device=dev)

    # the timed call writes the codes; buffers are allocated once, outside it
    max_abs = torch.empty(wl.n_layers, wl.n_q, dtype=torch.float32, device=dev)
    n_over = torch.empty(wl.n_layers, wl.n_q, dtype=torch.int32, device=dev)
    xs = [t.data_ptr() for t in x.unbind(0)]
    wqs = [t.data_ptr() for t in wq.unbind(0)]
    wks = [t.data_ptr() for t in wk.unbind(0)]

    def step():
        spectral_logits_fp8(est.ctx, xs, wl.d_model, seq, wqs, wks, scale.data_ptr(), ws.data_ptr(), ws.numel(),
                            codes.data_ptr(), max_abs.data_ptr(), n_over.data_ptr())

    log(f"{wl.key} fp8 consumer: warm-up {args.warmup}, then {args.steps} timed calls")
    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    t_wall = time.perf_counter()
    e0.record()
    for _ in range(args.steps):
        step()
    e1.record()
    torch.cuda.synchronize()
    wall_s = time.perf_counter() - t_wall
    ms = e0.elapsed_time(e1) / args.steps
    est.profile(True)
    step()
    prof = est.profile_read()
    est.profile(False)
    p_ms, p_n = prof["logits_projection"]
    l_ms, l_n = prof["logits_fp8"]
    # one launch of each kernel covers every layer
    proj_flops = 2.0 * seq * wl.d_model * (wl.n_q + wl.n_kv) * wl.head_dim * wl.n_layers
    logit_flops = 3 * 2.0 * seq * seq * wl.head_dim * wl.n_q * wl.n_layers   # three bf16 products
    logit_bytes = 4.0 * seq * (wl.n_q + wl.n_kv) * wl.head_dim * wl.n_layers + 1.0 * wl.n_layers * wl.n_q * seq * seq
    tflops = proj_flops / (p_ms / p_n * 1e-3) / 1e12
    logits = wl.n_layers * wl.n_q * seq * seq
    out = {
        "metric": "scaled E4M3 attention logits/sec (all layers and query heads)",
        "value": logits / (ms * 1e-3), "unit": "logits/s", "n_gpus": 1, "steps": args.steps,
        "warmup": args.warmup, "ms_per_step": ms, "higher_is_better": True, "scaling": "weak",
        "vs_baseline": None, "dtype": "bf16", "data": "synthetic",
        "config": {"workload": wl.key + "-fp8-consumer", "n_layers": wl.n_layers, "d_model": wl.d_model,
                   "n_q_heads": wl.n_q, "n_kv_heads": wl.n_kv, "head_dim": wl.head_dim, "seq_len": seq,
                   "tokens": "x = sqrt(d) u, u uniform on the sphere, per layer, bf16",
                   "scale": f"Eq. scale from the estimator, alpha {wl.alpha}", "form": "fp8"},
        "wall_s_timed": wall_s,
        "kernels_ms_per_step": {k: t for k, (t, n) in prof.items() if n},
        "max_abs_scaled": float(max_abs.max()), "overflow_heads": int((n_over > 0).sum()),
        "roofline": {
            "kernel": "logits_projection (Q, K = X W^T, bf16 matrix cores)",
            "bound": "mfma", "achieved": tflops, "peak": 2500.0, "unit": "TFLOP/s", "frac": tflops / 2500.0,
            "traffic": measured_traffic("proj"), "algorithmic_flops_per_launch": proj_flops,
            "avg_launch_ms": p_ms / p_n, "launches": p_n,
            "logits_kernel_TFLOPs": logit_flops / (l_ms * 1e-3) / 1e12,
        },
        # the logit kernel: three bf16 products per logit on the matrix cores, and its HBM
        # stream (the Q, K hi/lo planes read once, one code byte written per logit)
        # (the profiled call's logit kind covers the statistics reset, a few us, and the
        # logit kernel itself: one of each per call)
        "logits_roofline": {
            "kernel": "logits_fp8 (S~ = Q K^T / (sqrt(d_h) scale) -> E4M3 codes, matrix cores)",
            "bound": "mfma", "achieved": logit_flops / (l_ms * 1e-3) / 1e12, "peak": 2500.0,
            "unit": "TFLOP/s", "frac": logit_flops / (l_ms * 1e-3) / 1e12 / 2500.0,
            "traffic": measured_traffic("logits"), "algorithmic_flops_per_launch": logit_flops,
            "algorithmic_bytes_per_launch": logit_bytes, "hbm_GBps": logit_bytes / (l_ms * 1e-3) / 1e9,
            "hbm_frac": logit_bytes / (l_ms * 1e-3) / 1e9 / 8000.0, "avg_launch_ms": l_ms,
            "launches": 1, "note": "time of one call's statistics reset and logit kernel",
        },
    }
    from paper_2602_18851_amd import fp8_report
    out["report"] = dict(fp8_report(max_abs, n_over), scale=f"Eq. scale, alpha {wl.alpha}, {wl.n_iter} cold "
                                                             f"iterations (Gram form)")
    if not args.no_extras:
        out["context"] = {"library_gemm": library_projection(x, wq, wk, proj_flops)}
        del wq, wk, x, codes, ws
        est.close()
        torch.cuda.empty_cache()
        out["context"]["auto_alpha"] = auto_alpha_burnin(wl, seq, args.calib_steps)
        out["context"]["pretrained_analogue"] = pretrained_analogue(seq)
    if not args.no_cpu_baseline:
        log("cpu baseline (oracle)")
        out["cpu_baseline"] = cpu_baseline_fp8(wl, args.cpu_seconds, seq)
    print(json.dumps(out), flush=True)


def auto_alpha_burnin(wl, seq: int, steps: int, quantile: float = 0.9999, kappa: float = 1.0) -> dict:
    """Auto-alpha (Sec. 3.5; App. M, Algorithm "Auto-alpha Calibration") on
    the workload: cold start (five iterations, the paper's count), then
    `steps` burn-in steps, each a seeded perturbation of the weights, one warm
    estimator iteration (the paper's steady state) at the conservative
    alpha_0 = the workload's alpha, and the E4M3 consumer on fresh seeded
    tokens; the slack ratios (one per layer and step) give alpha_final, and
    one more step at alpha_final shows the utilisation it buys."""
    import numpy as np
    import torch

    from paper_2602_18851_amd import AutoAlpha, Spectral, fp8_report
    from paper_2602_18851_amd.spectral import spectral_logits_workspace_bytes
    from workloads import all_weights, device_tokens, start_vectors

    dev = torch.device("cuda", 0)
    est = Spectral(wl.n_layers, wl.d_model, wl.n_q, wl.n_kv, wl.head_dim, wl.dtype, wl.alpha)
    ws = torch.empty(spectral_logits_workspace_bytes(est.shape, seq), dtype=torch.uint8, device=dev)
    wq, wk = all_weights(wl, dev)
    v = start_vectors(wl, dev)
    est.step(wq, wk, v, 5)
    auto = AutoAlpha(wl.d_model, wl.head_dim, quantile, kappa)
    util0 = []
    t0 = time.perf_counter()
    for t in range(steps):
        log(f"auto-alpha burn-in step {t + 1}/{steps}")
        del wq, wk
        wq, wk = all_weights(wl, dev, perturbed=True, step=t)
        x = device_tokens(wl, seq, dev, step=t)
        sigma, scale, _ = est.step(wq, wk, v, 1)
        max_abs, n_over, _ = est.logits_fp8(x, wq, wk, scale, workspace=ws)
        auto.observe(sigma, scale, max_abs)
        util0.append(fp8_report(max_abs, n_over)["utilization_pct_layers"]["median"])
    alpha = auto.alpha()
    est.close()
    est = Spectral(wl.n_layers, wl.d_model, wl.n_q, wl.n_kv, wl.head_dim, wl.dtype, alpha)
    del wq, wk
    wq, wk = all_weights(wl, dev, perturbed=True, step=steps)
    x = device_tokens(wl, seq, dev, step=steps)
    _, scale, _ = est.step(wq, wk, v, 1)
    max_abs, n_over, _ = est.logits_fp8(x, wq, wk, scale, workspace=ws)
    after = fp8_report(max_abs, n_over)
    est.close()
    r = np.asarray(auto.ratios)
    return {"alpha_0": wl.alpha, "burn_in_steps": steps, "quantile": quantile, "kappa": kappa,
            "slack_ratios": {"n": int(r.size), "min": float(r.min()), "max": float(r.max()), "mean": float(r.mean())},
            "alpha_final": alpha, "tightening": wl.alpha / alpha,
            "utilization_pct_median_at_alpha_0": float(np.median(util0)),
            "next_step_at_alpha_final": after, "wall_s": time.perf_counter() - t0,
            "note": "one slack ratio per layer and step: max|S| of the layer's heads over B_max = sigma_l d / sqrt(d_h)"}


def pretrained_analogue(seq: int) -> dict:
    """Table "pretrained" and App. J analogues on the synthetic GPT-2-XL,
    Llama-2-7B and 70B shapes: the estimator's own scale (the workload's
    alpha, its cold iteration count) on the first call, then the E4M3
    consumer on `seq` post-normalisation tokens per layer: layers with an
    overflow, the largest scaled logit, and the utilisation."""
    import torch

    from paper_2602_18851_amd import Spectral, fp8_report
    from paper_2602_18851_amd.spectral import SN_FLAG_GRAM
    from workloads import WORKLOADS, all_weights, device_tokens, start_vectors

    dev = torch.device("cuda", 0)
    out = {}
    for key in ("gpt2-xl", "llama2-7b-spiked", "llama2-70b-gqa"):
        log(f"pretrained analogue: {key}")
        wl = WORKLOADS[key]
        wq, wk = all_weights(wl, dev)
        x = device_tokens(wl, seq, dev)
        est = Spectral(wl.n_layers, wl.d_model, wl.n_q, wl.n_kv, wl.head_dim, wl.dtype, wl.alpha,
                       flags=SN_FLAG_GRAM)
        _, scale, _ = est.step(wq, wk, start_vectors(wl, dev), wl.n_iter)
        max_abs, n_over, _ = est.logits_fp8(x, wq, wk, scale)
        rep = fp8_report(max_abs, n_over)
        out[key] = {"overflow": f"{rep['overflow_layers']}/{rep['layers']}", "max_scaled": rep["max_scaled"],
                    "alpha": wl.alpha, "n_iter": wl.n_iter, **rep}
        est.close()
        del wq, wk, x
        torch.cuda.empty_cache()
    return out


def library_projection(x, wq, wk, flops: float) -> dict:
    """The projections of the consumer as plain library GEMMs (torch linear,
    one per layer and matrix, bf16 in and out, fp32 accumulation), timed the
    same way: a yardstick for the hand-written projection kernel."""
    import torch
    import torch.nn.functional as F

    def run():
        for l in range(x.shape[0]):
            F.linear(x[l], wq[l])
            F.linear(x[l], wk[l])

    run()
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    reps = 5
    e0.record()
    for _ in range(reps):
        run()
    e1.record()
    torch.cuda.synchronize()
    ms = e0.elapsed_time(e1) / reps
    return {"what": "torch.nn.functional.linear per layer for Q and K (hipBLASLt), same shapes, bf16 output",
            "ms": ms, "TFLOPs": flops / (ms * 1e-3) / 1e12}


def main():
    args = parse()
    if args.gpus != 1:
        print(json.dumps({"error": "the estimator runs on one GPU (each GPU would hold its own shard of layers or heads); --gpus must be 1"}))
        sys.exit(2)
    if args.mode == "copy":
        copy_reference(args.copy_bytes)
        return
    if args.mode == "perstep":
        from paper_2602_18851_amd.spectral import SN_FLAG_GRAM
        print(json.dumps({"form": args.form, "per_step_warm": per_step_warm(SN_FLAG_GRAM if args.form == "gram" else 0)}),
              flush=True)
        return
    if args.form == "fp8":
        bench_fp8(args)
        return

    import torch

    from paper_2602_18851_amd import Spectral
    from paper_2602_18851_amd.spectral import SN_FLAG_GRAM, SN_FLAG_LAYER
    from workloads import WORKLOADS, all_weights, layer_start_vectors, start_vectors

    wl = WORKLOADS[args.workload]
    n_iter = args.n_iter or wl.n_iter
    torch.cuda.set_device(0)
    dev = torch.device("cuda", 0)
    wq, wk = all_weights(wl, dev)
    layer = args.form == "layer"
    v0 = layer_start_vectors(wl, dev) if layer else start_vectors(wl, dev)
    v = v0.clone()
    sigma = torch.empty(wl.n_layers, *([] if layer else [wl.n_q]), dtype=torch.float32, device=dev)
    scale = torch.empty(wl.n_layers, dtype=torch.float32, device=dev)
    iters = torch.empty(wl.n_layers, wl.n_q, dtype=torch.int32, device=dev)
    gram = args.form == "gram"
    flags = args.flags | (SN_FLAG_GRAM if gram else 0) | (SN_FLAG_LAYER if layer else 0)
    est = Spectral(wl.n_layers, wl.d_model, wl.n_q, wl.n_kv, wl.head_dim, wl.dtype, wl.alpha, tol=0.0,
                   q_strips=args.q_strips, k_strips=args.k_strips, flags=flags)
    torch.cuda.synchronize()

    def step():
        if layer:
            est.step_layer(wq, wk, v, n_iter, sigma=sigma, scale=scale)
        else:
            est.step(wq, wk, v, n_iter, sigma=sigma, scale=scale, iters=iters)

    log(f"{wl.key} ({args.form}): warm-up {args.warmup}, then {args.steps} timed calls")
    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    timed_step = step
    if args.graph and not layer:
        # the weight pointers are already on the device, so a call queues
        # kernel launches only and can be captured
        graph = torch.cuda.CUDAGraph()
        with torch.cuda.graph(graph):
            step()
        timed_step = graph.replay
        for _ in range(args.warmup):
            timed_step()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    if args.flush:
        # every call starts from cold caches: 1 GiB written first (4x the
        # Infinity Cache), each call timed alone between its own events
        scratch = torch.empty(1 << 30, dtype=torch.uint8, device=dev)
        evs = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(args.steps)]
        t_wall = time.perf_counter()
        for k, (a_, b_) in enumerate(evs):
            scratch.fill_(k & 0xFF)
            a_.record()
            timed_step()
            b_.record()
        torch.cuda.synchronize()
        wall_s = time.perf_counter() - t_wall
        ms = sum(a_.elapsed_time(b_) for a_, b_ in evs) / args.steps
        del scratch
    else:
        t_wall = time.perf_counter()
        e0.record()
        for _ in range(args.steps):
            timed_step()
        e1.record()
        torch.cuda.synchronize()
        wall_s = time.perf_counter() - t_wall
        ms = e0.elapsed_time(e1) / args.steps
    assert bool(torch.isfinite(sigma).all()) and (layer or bool((iters == n_iter).all()))

    # per-kernel durations, HIP events on the launch stream (separate pass)
    est.profile(True)
    step()
    prof = est.profile_read()
    est.profile(False)
    H = wl.n_layers * wl.n_q
    q_bytes, k_bytes = wl.weight_bytes()
    dom_launch_bytes = None
    if layer:
        # per step: row sweeps over W_K and W_Q; column sweeps over W_Q and W_K,
        # which read one d_h-vector per query / key head and write u' and v'
        col_buf = (H + wl.n_layers * wl.n_kv) * wl.head_dim * 4 + 2 * wl.n_layers * wl.d_model * 4
        r_ms, r_n = prof["layer_row_sweeps"]
        c_ms, c_n = prof["layer_col_sweeps"]
        if r_ms >= c_ms:
            dom_name, dom_kind, dom_alg = "layer_row_sweeps (W_K and W_Q, row sums)", "layer_row_sweeps", \
                n_iter * (q_bytes + k_bytes)
        else:
            dom_name, dom_kind, dom_alg = "layer_col_sweeps (W_Q and W_K, column sums)", "layer_col_sweeps", \
                n_iter * (q_bytes + k_bytes + col_buf)
        dom_launch_bytes = dom_alg  # all launches of the kind together
        dom_flops = None
        call_bytes = n_iter * (2 * (q_bytes + k_bytes) + col_buf) + 12 * wl.d_model * wl.n_layers
        H = wl.n_layers  # one estimate per layer
    elif gram:
        # Gram sweep: every weight read once, the upper-triangle 16 x 16 Gram
        # blocks written once per query / key head (d_h (d_h + 16) / 2 floats)
        units = H + wl.n_layers * wl.n_kv
        g_out = units * wl.head_dim * (wl.head_dim + 16) // 2 * 4
        dom_name, dom_kind = "gram_sweep (G = R R^T of every head, matrix cores)", "gram_sweep"
        dom_alg = q_bytes + k_bytes + g_out
        dom_flops = 2.0 * units * wl.head_dim * (wl.head_dim + 16) / 2 * wl.d_model
        # first W_K sweep, Gram sweep, final W_K sweep, Gram blocks read back, vectors
        call_bytes = 3 * k_bytes + q_bytes + 2 * g_out + 12 * wl.d_model * H
    else:
        dom_name, dom_kind = "q_sweep (fused W_Q sweep)", "q_sweep"
        dom_alg = q_bytes + H * 2 * wl.head_dim * 4          # weights + z in + y out, per launch
        dom_flops = None
        call_bytes = n_iter * (q_bytes + k_bytes) + k_bytes + 12 * wl.d_model * H
    dom_ms, dom_n = prof[dom_kind]
    dom_avg_ms = dom_ms / dom_n
    if dom_launch_bytes is not None:
        dom_alg = dom_launch_bytes / dom_n  # average algorithmic bytes per launch of the kind
    achieved = dom_alg / (dom_avg_ms * 1e-3) / 1e9
    heads_iters = H * n_iter
    out = {
        "metric": METRIC,
        "value": heads_iters / (ms * 1e-3),
        "unit": "layers·iters/s" if layer else "heads·iters/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f32",
        "data": "synthetic",
        "config": {
            "workload": wl.key,
            "description": wl.description,
            "n_layers": wl.n_layers, "d_model": wl.d_model, "n_q_heads": wl.n_q, "n_kv_heads": wl.n_kv,
            "head_dim": wl.head_dim, "weights_dtype": wl.dtype, "n_iter": n_iter, "heads": H,
            "start": "cold (seeded unit vectors), state carried across steps",
            "form": args.form,
            "launch": "HIP graph replay" if args.graph and not layer else "eager",
            "cache": "1 GiB written before every timed call, calls timed one by one" if args.flush
                     else "calls back to back, no flush",
        },
        "arithmetic": ARITHMETIC["gram" if gram else "layer" if layer else "chain"],
        "effective_GBps": call_bytes / (ms * 1e-3) / 1e9,
        "effective_frac_of_peak": call_bytes / (ms * 1e-3) / 1e9 / HBM_PEAK_GBPS,
        "call_bytes": call_bytes,
        "wall_s_timed": wall_s,
        "kernels_ms_per_step": {k: t for k, (t, n) in prof.items() if n},
        "roofline": {
            "kernel": dom_name,
            "bound": "hbm",
            "achieved": achieved,
            "peak": HBM_PEAK_GBPS,
            "unit": "GB/s",
            "frac": achieved / HBM_PEAK_GBPS,
            "traffic": None if layer else measured_traffic("gram_sweep" if gram else ""),
            "algorithmic_bytes_per_launch": dom_alg,
            "avg_launch_ms": dom_avg_ms,
            "launches": dom_n,
        },
    }
    if dom_flops:
        out["roofline"]["mfma_TFLOPs"] = dom_flops / (dom_avg_ms * 1e-3) / 1e12
        out["roofline"]["mfma_frac_of_dense_peak"] = out["roofline"]["mfma_TFLOPs"] / (2500.0 if wl.dtype == "bf16"
                                                                                        else 157.3)
    if not layer and not args.no_extras:
        log("context lines")
        del wq, wk
        est.close()
        torch.cuda.empty_cache()
        out["context"] = context_lines(args, flags)
    if not args.no_cpu_baseline:
        log("cpu baseline (oracle)")
        out["cpu_baseline"] = (cpu_baseline_layer if layer else cpu_baseline)(wl, args.cpu_seconds, n_iter)
        if not layer and not gram and not args.no_extras:
            out.setdefault("context", {})["oracle_explicit_M"] = cpu_explicit_m(wl, args.cpu_seconds / 3, n_iter)
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
