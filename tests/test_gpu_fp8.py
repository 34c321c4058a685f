"""FP8 E4M3 logit consumer (spectral_logits_fp8) against the float64 oracle
(oracle.fp8_consumer), through the C ABI.

The GPU forms S~ = (q . k) / (sqrt(d_h) scale) from fp32 projections split
into bf16 hi + lo halves (3 matrix-core products), so |S~_gpu - S~| stays
below err_ij = 2^-14 ||q_i|| ||k_j|| / (sqrt(d_h) scale): the hi/lo split
leaves at most 3 * 2^-16 of sum_r |q_r k_r| <= ||q|| ||k||, and the fp32
sums of the projections add about sqrt(d) 2^-24 (~5e-6) relative.  Codes are
unique away from the rounding points of E4M3; within err of one, either
neighbour is correct.  So every GPU code must decode inside
[dec(enc(S~ - err)), dec(enc(S~ + err))] (NaN allowed where that interval
reaches past +-464), the overflow count must lie between the counts of
|S~| > 448 + err and |S~| > 448 - err, and max |S~| must agree within the
largest err."""

import math

import numpy as np
import pytest
import torch

from oracle import e4m3, fp8_consumer
from workloads import WORKLOADS, all_weights, tokens

pytestmark = pytest.mark.gpu

if not torch.cuda.is_available():  # pragma: no cover - collected on CPU machines, skipped there
    pytest.skip("needs a GPU", allow_module_level=True)

from paper_2602_18851_amd import Spectral, fp8_report  # noqa: E402

TAU = 2.0 ** -14


def layer_tokens(wl, seq, layer):
    """Post-normalisation tokens x = sqrt(d) u (Sec. 3.2), rounded to bf16."""
    return torch.from_numpy(tokens(wl, seq, spherical=True, layer=layer)).to(torch.bfloat16)


def _pad(t, ld):
    if not ld or ld == t.shape[-1]:
        return t.cuda()
    p = torch.zeros(*t.shape[:-1], ld, dtype=t.dtype)
    p[..., :t.shape[-1]] = t
    return p.cuda()[..., :t.shape[-1]]


def _f64(t):
    return t if isinstance(t, np.ndarray) else t.double().numpy()


def check_head(gpu_codes, gpu_max, gpu_over, x, wq, wk, scale, h, n_kv, dh):
    x64, wq64, wk64 = _f64(x), _f64(wq), _f64(wk)
    S = fp8_consumer.head_logits(x64, wq64, wk64, h, n_kv, dh) / scale
    g = (wq64.shape[0] // dh) // n_kv
    qn = np.linalg.norm(x64 @ wq64[h * dh:(h + 1) * dh].T, axis=1)
    kn = np.linalg.norm(x64 @ wk64[(h // g) * dh:(h // g + 1) * dh].T, axis=1)
    err = TAU * np.outer(qn, kn) / (math.sqrt(dh) * scale)
    # band of correct values; an end past -+464 is open (NaN codes there are correct too)
    lo = np.where(S - err < -464.0, -np.inf, e4m3.decode(e4m3.encode(S - err)))
    hi = np.where(S + err > 464.0, np.inf, e4m3.decode(e4m3.encode(S + err)))
    got = e4m3.decode(gpu_codes)
    with np.errstate(invalid="ignore"):
        ok = np.isfinite(got) & (got >= lo) & (got <= hi)
    ok |= np.isnan(got) & ((S + err > 464.0) | (S - err < -464.0))
    assert ok.all(), (h, np.argwhere(~ok)[:5], S[~ok][:5], gpu_codes[~ok][:5])
    exact = (e4m3.encode(S - err) == e4m3.encode(S + err))
    assert (gpu_codes[exact] == e4m3.encode(S)[exact]).all()
    a = np.abs(S)
    assert np.count_nonzero(a > 448.0 + err) <= gpu_over <= np.count_nonzero(a > 448.0 - err)
    assert abs(gpu_max - a.max()) <= err.max()
    return int(np.count_nonzero(~exact)), float(a.max())


CASES = [
    # name, shape overrides, seq, ld (tokens and weights), target max |S~| per layer
    ("gqa4-dh64-seq192", dict(n_layers=2, d_model=512, n_q=8, n_kv=2, head_dim=64), 192, 0, (540.0, 300.0)),
    ("mha-dh128-ragged", dict(n_layers=1, d_model=1001, n_q=2, n_kv=2, head_dim=128), 130, 1008, (470.0,)),
    ("mqa-dh16-seq64", dict(n_layers=1, d_model=256, n_q=8, n_kv=1, head_dim=16), 64, 0, (450.0,)),
    ("gqa3-dh32-seq256", dict(n_layers=2, d_model=384, n_q=6, n_kv=2, head_dim=32), 256, 0, (1000.0, 100.0)),
]


def _random_cases(n=6, seed=2602):
    """Seeded random shapes: 1..3 layers, ragged widths over padded rows,
    1..600 tokens, d_h 16..128, MHA to 8 query heads per key head."""
    rng = np.random.default_rng(seed)
    out = []
    for i in range(n):
        d = int(rng.integers(16, 900))
        ld = -(-d // 8) * 8 + 8 * int(rng.integers(0, 2))
        n_kv = int(rng.integers(1, 4))
        over = dict(n_layers=int(rng.integers(1, 4)), d_model=d, n_kv=n_kv, n_q=n_kv * int(rng.choice([1, 2, 3, 8])),
                    head_dim=int(rng.choice([16, 32, 64, 128])))
        seq = int(rng.integers(1, 601))
        target = tuple(float(x) for x in rng.uniform(200.0, 700.0, over["n_layers"]))
        out.append((f"rand{i}-d{d}-ld{ld}-q{over['n_q']}kv{n_kv}-dh{over['head_dim']}-seq{seq}", over, seq, ld, target))
    return out


CASES += _random_cases()


@pytest.mark.parametrize("name,over,seq,ld,target", CASES, ids=[c[0] for c in CASES])
def test_logits_against_oracle(name, over, seq, ld, target):
    wl = WORKLOADS["llama2-70b-gqa"].replace(key=name, std=0.02, **over)
    wq, wk = all_weights(wl, "cpu")
    xs = [layer_tokens(wl, seq, l) for l in range(wl.n_layers)]
    # scales chosen from the oracle's own logits so that the largest |S~| of
    # every layer is the target (above 448: overflows and NaN codes)
    scales = []
    for l in range(wl.n_layers):
        m = max(np.abs(fp8_consumer.head_logits(xs[l].double().numpy(), wq[l].double().numpy(),
                                                wk[l].double().numpy(), h, wl.n_kv, wl.head_dim)).max()
                for h in range(wl.n_q))
        scales.append(m / target[l])
    est = Spectral(wl.n_layers, wl.d_model, wl.n_q, wl.n_kv, wl.head_dim, wl.dtype, wl.alpha, ld=ld)
    x_dev = _pad(torch.stack(xs), ld)
    scale_dev = torch.tensor(scales, dtype=torch.float32, device="cuda")
    max_abs, n_over, codes = est.logits_fp8(x_dev, _pad(wq, ld), _pad(wk, ld), scale_dev, want_codes=True)
    torch.cuda.synchronize()
    max_abs, n_over, codes = max_abs.cpu().numpy(), n_over.cpu().numpy(), codes.cpu().numpy()
    # the scale the GPU used is the float32 one
    s32 = scale_dev.cpu().double().numpy()
    band = 0
    for l in range(wl.n_layers):
        for h in range(wl.n_q):
            nb, _ = check_head(codes[l, h], max_abs[l, h], n_over[l, h], xs[l], wq[l], wk[l], s32[l], h, wl.n_kv,
                               wl.head_dim)
            band += nb
    if max(target) > 450.0:
        assert n_over.sum() > 0
    print(f"{name}: codes equal the oracle's outside the rounding bands ({band} entries inside one)")
    # statistics without codes are the same
    m2, o2, c2 = est.logits_fp8(x_dev, _pad(wq, ld), _pad(wk, ld), scale_dev, want_codes=False)
    torch.cuda.synchronize()
    assert c2 is None
    np.testing.assert_array_equal(m2.cpu().numpy(), max_abs)
    np.testing.assert_array_equal(o2.cpu().numpy(), n_over)
    est.close()


def test_zero_tokens_give_zero_logits():
    wl = WORKLOADS["llama2-70b-gqa"].replace(n_layers=1, d_model=256, n_q=4, n_kv=2, head_dim=64)
    gq, gk = all_weights(wl, "cuda")
    est = Spectral(wl.n_layers, wl.d_model, wl.n_q, wl.n_kv, wl.head_dim, wl.dtype, wl.alpha)
    x = torch.zeros(1, 100, wl.d_model, dtype=torch.bfloat16, device="cuda")
    max_abs, n_over, codes = est.logits_fp8(x, gq, gk, torch.ones(1, device="cuda"), want_codes=True)
    torch.cuda.synchronize()
    assert not max_abs.any() and not n_over.any() and not codes.any()
    est.close()


def test_non_finite_scale_counts_every_logit_as_overflow():
    """A NaN scale (a layer with a degenerate head) and a zero scale: every
    scaled logit is non-finite, so every one counts as an overflow, every
    code is the NaN code, and max |S~| is not finite (NaN for the NaN scale),
    as the oracle's statistics say."""
    wl = WORKLOADS["llama2-70b-gqa"].replace(key="nan-scale", std=0.02, n_layers=2, d_model=256, n_q=4, n_kv=2,
                                              head_dim=64)
    seq = 70
    wq, wk = all_weights(wl, "cpu")
    xs = [layer_tokens(wl, seq, l) for l in range(wl.n_layers)]
    est = Spectral(wl.n_layers, wl.d_model, wl.n_q, wl.n_kv, wl.head_dim, wl.dtype, wl.alpha)
    scales = [float("nan"), 0.0]
    max_abs, n_over, codes = est.logits_fp8(torch.stack(xs).cuda(), wq.cuda(), wk.cuda(),
                                            torch.tensor(scales, device="cuda"), want_codes=True)
    torch.cuda.synchronize()
    max_abs, n_over, codes = max_abs.cpu().numpy(), n_over.cpu().numpy(), codes.cpu().numpy()
    assert (n_over == seq * seq).all(), n_over
    assert np.isnan(max_abs[0]).all() and not np.isfinite(max_abs[1]).any()
    assert ((codes & 0x7F) == e4m3.NAN_CODE).all()
    with np.errstate(divide="ignore", invalid="ignore"):
        for l in range(wl.n_layers):
            ref = fp8_consumer.consume_layer(xs[l].double().numpy(), wq[l].double().numpy(), wk[l].double().numpy(),
                                             scales[l], wl.n_kv, wl.head_dim, want_codes=False)
            assert [ref["n_over"][h] for h in range(wl.n_q)] == list(n_over[l])
            assert all(not np.isfinite(ref["max_abs"][h]) for h in range(wl.n_q))
    est.close()


def test_refuses_a_layer_weight_beyond_the_buffer_range():
    """One layer's W_Q of 4 GiB or more (n_q d_h rows of ld bf16 elements)
    does not fit the projection's buffer range: the call is refused with
    SN_EINVAL before anything is queued (no weight is read, so the pointers
    need not cover the shape)."""
    from paper_2602_18851_amd.spectral import (SN_EINVAL, SpectralError, spectral_logits_fp8,
                                               spectral_logits_workspace_bytes)
    n_q, dh, ld, seq = 64, 128, 262144, 64   # 8192 rows x 512 KiB = 4 GiB
    est = Spectral(1, 8192, n_q, 8, dh, "bf16", 0.02, ld=ld)
    ws = torch.empty(spectral_logits_workspace_bytes(est.shape, seq), dtype=torch.uint8, device="cuda")
    buf = torch.zeros(4096, dtype=torch.bfloat16, device="cuda")
    max_abs = torch.zeros(n_q, device="cuda")
    n_over = torch.zeros(n_q, dtype=torch.int32, device="cuda")
    scale = torch.ones(1, device="cuda")
    with pytest.raises(SpectralError) as err:
        spectral_logits_fp8(est.ctx, [buf.data_ptr()], 0, seq, [buf.data_ptr()], [buf.data_ptr()], scale.data_ptr(),
                            ws.data_ptr(), ws.numel(), 0, max_abs.data_ptr(), n_over.data_ptr())
    assert err.value.code == SN_EINVAL and "2^32" in str(err.value)
    est.close()


def test_full_size_70b_sampled_heads():
    """Llama-2-70B GQA shape, 1024 tokens per layer, all 80 layers on the GPU;
    against the oracle, every code, max |S~| and overflow count of a seeded
    sample of 147 heads: all 64 heads of the first and the last layer, and
    one head in every fourth layer between.  Per-layer scales are seeded
    synthetic values around the size that puts the largest logit near 448."""
    wl = WORKLOADS["llama2-70b-gqa"]
    seq = 1024
    gq, gk = all_weights(wl, "cuda")
    x = torch.stack([layer_tokens(wl, seq, l) for l in range(wl.n_layers)]).cuda()
    rng = np.random.default_rng(7)
    scales = (0.02 * rng.uniform(0.5, 2.0, wl.n_layers)).astype(np.float32)
    est = Spectral(wl.n_layers, wl.d_model, wl.n_q, wl.n_kv, wl.head_dim, wl.dtype, wl.alpha)
    max_abs, n_over, codes = est.logits_fp8(x, gq, gk, torch.from_numpy(scales).cuda(), want_codes=True)
    torch.cuda.synchronize()
    sample = {0: range(wl.n_q), wl.n_layers - 1: range(wl.n_q)}
    for l in range(4, wl.n_layers - 1, 4):
        sample[l] = [int(rng.integers(wl.n_q))]
    n_heads = 0
    for l, heads in sorted(sample.items()):
        x64, wq64, wk64 = x[l].cpu().double().numpy(), gq[l].cpu().double().numpy(), gk[l].cpu().double().numpy()
        codes_l, max_l, over_l = codes[l].cpu().numpy(), max_abs[l].cpu().numpy(), n_over[l].cpu().numpy()
        for h in heads:
            check_head(codes_l[h], float(max_l[h]), int(over_l[h]), x64, wq64, wk64, float(scales[l]), h, wl.n_kv,
                       wl.head_dim)
            n_heads += 1
    assert n_heads == 2 * wl.n_q + len(range(4, wl.n_layers - 1, 4))
    print(f"70B: {n_heads} heads checked; max |S~| over all heads {max_abs.max().item():.1f}, overflowing heads "
          f"{int((n_over > 0).sum())} of {n_over.numel()}")
    est.close()


def test_separate_layer_buffers_and_several_row_tiles():
    """Layers passed as separately allocated tensors (the device pointer table
    then holds unrelated addresses) give the same bits as one stacked tensor,
    and both match the oracle; 520 tokens span three 256-row projection tiles
    and five 128-row logit tiles, the last ones ragged."""
    wl = WORKLOADS["llama2-70b-gqa"].replace(key="sep-layers", std=0.02, n_layers=3, d_model=320, n_q=4, n_kv=2,
                                              head_dim=64)
    seq = 520
    wq, wk = all_weights(wl, "cpu")
    xs = [layer_tokens(wl, seq, l) for l in range(wl.n_layers)]
    scales = []
    for l in range(wl.n_layers):
        m = max(np.abs(fp8_consumer.head_logits(xs[l].double().numpy(), wq[l].double().numpy(),
                                                wk[l].double().numpy(), h, wl.n_kv, wl.head_dim)).max()
                for h in range(wl.n_q))
        scales.append(m / 500.0)
    scale_dev = torch.tensor(scales, dtype=torch.float32, device="cuda")
    est = Spectral(wl.n_layers, wl.d_model, wl.n_q, wl.n_kv, wl.head_dim, wl.dtype, wl.alpha)
    stacked = est.logits_fp8(torch.stack(xs).cuda(), wq.cuda(), wk.cuda(), scale_dev, want_codes=True)
    # separate allocations in reverse layer order, with gaps between them
    keep, x_l, q_l, k_l = [], [None] * wl.n_layers, [None] * wl.n_layers, [None] * wl.n_layers
    for l in reversed(range(wl.n_layers)):
        x_l[l] = xs[l].cuda()
        keep.append(torch.empty(4097, dtype=torch.uint8, device="cuda"))
        q_l[l] = wq[l].clone().cuda()
        k_l[l] = wk[l].clone().cuda()
    sep = est.logits_fp8(x_l, q_l, k_l, scale_dev, want_codes=True)
    torch.cuda.synchronize()
    for a_, b_ in zip(stacked, sep):
        np.testing.assert_array_equal(a_.cpu().numpy(), b_.cpu().numpy())
    max_abs, n_over, codes = (t.cpu().numpy() for t in sep)
    s32 = scale_dev.cpu().double().numpy()
    for l in range(wl.n_layers):
        for h in range(wl.n_q):
            check_head(codes[l, h], max_abs[l, h], n_over[l, h], xs[l], wq[l], wk[l], s32[l], h, wl.n_kv,
                       wl.head_dim)
    assert n_over.sum() > 0
    est.close()


def test_report_lines_on_the_gpt2_xl_shape_against_the_oracle():
    """Table "pretrained" and App. J analogues on the GPT-2-XL shape: the
    estimator's own scale (alpha 0.08, 30 cold iterations), 1024
    post-normalisation tokens per layer, every layer on the GPU; the per-layer
    utilisation max|S~| / 448 and overflow flag of two seeded layers (all
    heads) against the oracle's logits at the oracle's own scale, and the
    report's fields against the per-layer values they summarise."""
    from oracle.power_iteration import spectral_step as oracle_step
    from workloads import start_vectors
    wl = WORKLOADS["gpt2-xl"]
    seq = 1024
    gq, gk = all_weights(wl, "cuda")
    x = torch.stack([layer_tokens(wl, seq, l) for l in range(wl.n_layers)]).cuda()
    v0 = start_vectors(wl, "cuda")
    est = Spectral(wl.n_layers, wl.d_model, wl.n_q, wl.n_kv, wl.head_dim, wl.dtype, wl.alpha)
    _, scale, _ = est.step(gq, gk, v0.clone(), wl.n_iter)
    max_abs, n_over, _ = est.logits_fp8(x, gq, gk, scale)
    rep = fp8_report(max_abs, n_over)
    mx, ov = max_abs.double().cpu().numpy(), n_over.cpu().numpy()
    util = 100.0 * mx.max(axis=1) / 448.0
    assert rep["layers"] == wl.n_layers and rep["overflow_layers"] == int((ov > 0).any(axis=1).sum())
    assert rep["max_scaled"] == pytest.approx(mx.max())
    assert rep["utilization_pct_layers"]["median"] == pytest.approx(np.median(util))
    assert rep["utilization_pct_layers"]["p10"] <= rep["utilization_pct_layers"]["median"] <= \
        rep["utilization_pct_layers"]["p90"]
    rng = np.random.default_rng(wl.cfg_id)
    v0c = v0.double().cpu().numpy()
    for l in sorted(rng.choice(wl.n_layers, 2, replace=False)):
        wq_l, wk_l, x_l = gq[l].double().cpu().numpy(), gk[l].double().cpu().numpy(), x[l].double().cpu().numpy()
        ref = oracle_step([wq_l], [wk_l], v0c[l:l + 1], wl.n_iter, n_kv=wl.n_kv, head_dim=wl.head_dim,
                          alpha=wl.alpha)
        res = fp8_consumer.consume_layer(x_l, wq_l, wk_l, ref["scale"][0], wl.n_kv, wl.head_dim, want_codes=False)
        u_ref = 100.0 * max(res["max_abs"].values()) / 448.0
        assert abs(util[l] - u_ref) <= 1e-3 * u_ref, (l, util[l], u_ref)
        assert (ov[l] > 0).any() == (max(res["n_over"].values()) > 0)
    print(f"gpt2-xl: overflow layers {rep['overflow_layers']}/{rep['layers']}, max scaled {rep['max_scaled']:.1f}, "
          f"utilisation per layer median {rep['utilization_pct_layers']['median']:.2f} % "
          f"(P10 {rep['utilization_pct_layers']['p10']:.2f}, P90 {rep['utilization_pct_layers']['p90']:.2f})")
    est.close()
