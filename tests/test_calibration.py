"""Host-side calibration helpers of the C library (no GPU needed) against the
oracle and the numbers the paper prints (Tables "alpha_selection",
"concentration", App. M burn-in statistics)."""

import math
import os

import numpy as np
import pytest

from conftest import read_golden
from oracle import calibration as cal
from paper_2602_18851_amd import spectral as sp
from paper_2602_18851_amd.build import LIB_PATH, build_library


@pytest.fixture(scope="module", autouse=True)
def lib():
    if not os.path.exists(LIB_PATH):
        build_library()
    return sp.load_library()


def test_alpha_select_matches_the_printed_tables_and_the_oracle():
    gammas = {m: float(g) for m, _, _, g, _ in read_golden("concentration.txt")}
    for model, d, dh, N, a_printed in read_golden("alpha_selection.txt"):
        g, a = sp.spectral_alpha_select(int(d), int(dh), int(N), 1024, 1e-6)
        assert abs(a - float(a_printed)) < 6e-4, model
        assert abs(g - gammas[model]) < 0.02, model
        assert a == pytest.approx(cal.alpha_min(int(d), int(dh), int(N), 1024, 1e-6), rel=1e-12)
        assert g == pytest.approx(cal.gamma_select(int(dh), int(N), 1024, 1e-6), rel=1e-12)


def test_overflow_terms_meet_the_split_union_bound():
    for model, d, dh, N, _ in read_golden("alpha_selection.txt"):
        d, dh, N = int(d), int(dh), int(N)
        g, a = sp.spectral_alpha_select(d, dh, N, 1024, 1e-6)
        t1, t2 = sp.spectral_overflow_terms(d, dh, 1024, a, g)
        o1, o2 = cal.overflow_terms(d, dh, 1024, a, g)
        assert t1 == pytest.approx(o1, rel=1e-12) and t2 == pytest.approx(o2, rel=1e-12)
        assert N * t1 <= 0.5e-6 * (1 + 1e-9) and N * t2 == pytest.approx(0.5e-6, rel=1e-9)


@pytest.mark.parametrize("n", [1, 2, 7, 100, 4000])
@pytest.mark.parametrize("q", [0.0, 0.5, 0.9999, 1.0])
def test_auto_alpha_is_the_interpolated_quantile(n, q):
    rng = np.random.default_rng(n)
    r = rng.uniform(7e-5, 3.7e-4, n)
    for kappa in (1.0, 2.0, 3.0):
        got = sp.spectral_auto_alpha(list(r), q, kappa)
        assert got == pytest.approx(cal.auto_alpha(r, q, kappa), rel=1e-14, abs=0.0)


def test_auto_alpha_burn_in_statistics():
    g = {k: float(v) for k, v in read_golden("autoalpha_burnin.txt")}
    # kappa = 1 keeps the quantile; the quantile lies in the observed range
    assert g["alpha_calibrated"] == pytest.approx(g["p9999"] * g["kappa"])
    assert g["slack_min"] <= g["p9999"] <= g["slack_max"]
    # "83x tightening" against the conservative alpha
    assert round(g["alpha_conservative"] / g["alpha_calibrated"]) == g["tightening"]
    # utilisation of the conservative scale at the mean slack: r * B_max / (scale * 448)
    # with scale = alpha * B_max / (0.8 * 448) is r * 0.8 / alpha = 0.47% ~ the printed 0.5%
    sigma, d, dh = 1.0, 5120, 128
    b_max = sigma * d / math.sqrt(dh)
    scale = cal.scale_factor(sigma, g["alpha_conservative"], d, dh)
    util = cal.utilization(g["slack_mean"] * b_max, scale)
    assert round(100 * util, 1) == g["utilization_conservative_percent"]
    # a burn-in whose ratios all equal r gives alpha = r (C library)
    assert sp.spectral_auto_alpha([g["p9999"]] * 100, 0.9999, 1.0) == pytest.approx(g["p9999"], rel=1e-15)


def test_slack_ratio():
    for args in ((120.0, 483.9, 1600, 64), (2.5, 463.5, 5120, 128), (1.0, 1786.1, 8192, 128)):
        assert sp.spectral_slack_ratio(*args) == pytest.approx(cal.slack_ratio(*args), rel=1e-15)


@pytest.mark.parametrize("call", [
    lambda: sp.spectral_alpha_select(0, 64, 10, 1024, 1e-6),
    lambda: sp.spectral_alpha_select(1600, 64, 10, 1024, 1.5),
    lambda: sp.spectral_overflow_terms(1600, 64, 1024, 0.05, 1.0),
    lambda: sp.spectral_auto_alpha([0.1, -1.0], 0.5, 1.0),
    lambda: sp.spectral_auto_alpha([0.1], 1.5, 1.0),
    lambda: sp.spectral_auto_alpha([0.1], 0.5, 0.5),
])
def test_bad_arguments(call):
    with pytest.raises(sp.SpectralError) as e:
        call()
    assert e.value.code == sp.SN_EINVAL and sp.spectral_last_error()
