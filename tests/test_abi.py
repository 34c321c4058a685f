"""The C-ABI library loads without a GPU, exports every symbol the header
declares, and rejects bad shapes/parameters before touching the device."""

import ctypes
import os
import re

import pytest

from conftest import ROOT
from paper_2602_18851_amd import spectral as sp
from paper_2602_18851_amd.build import LIB_PATH, build_library

HEADER = os.path.join(ROOT, "include", "spectral.h")


@pytest.fixture(scope="module")
def lib():
    if not os.path.exists(LIB_PATH):
        build_library()
    return sp.load_library()


def declared_symbols():
    text = open(HEADER).read()
    return sorted(set(re.findall(r"SN_API\s+[\w\s\*]+?\b(spectral_\w+)\s*\(", text)))


def test_header_declares_the_binding_names():
    assert declared_symbols() == sorted(sp.EXPORTED)


def test_every_declared_symbol_is_exported(lib):
    for name in declared_symbols():
        assert hasattr(lib, name), name
        assert isinstance(getattr(lib, name), ctypes._CFuncPtr)


def test_only_the_abi_is_exported(lib):
    out = os.popen(f"nm -D --defined-only {LIB_PATH}").read()
    exported = {l.split()[-1] for l in out.splitlines() if " T " in l}
    assert {s for s in exported if s.startswith("spectral_")} == set(declared_symbols())


def _shape(**kw):
    base = dict(n_layers=2, d_model=256, n_q_heads=8, n_kv_heads=2, head_dim=64, dtype=sp.SN_BF16, ld=0)
    base.update(kw)
    return sp.sn_shape(**base)


def _params(**kw):
    base = dict(alpha=0.02, eta_fp8=0.8, r_max=448.0, tol=0.0, q_strips=0, k_strips=0, flags=0)
    base.update(kw)
    return sp.sn_params(**base)


def test_workspace_bytes_for_a_valid_shape(lib):
    assert sp.spectral_workspace_bytes(_shape(), _params()) > 0


@pytest.mark.parametrize("kw,code", [
    (dict(n_kv_heads=3), sp.SN_EINVAL),      # does not divide n_q
    (dict(head_dim=48), sp.SN_EINVAL),       # unsupported head_dim
    (dict(n_layers=0), sp.SN_EINVAL),
    (dict(dtype=7), sp.SN_EDTYPE),
    (dict(ld=100), sp.SN_EINVAL),            # ld < d_model
    (dict(d_model=250, ld=250), sp.SN_EINVAL),  # rows not 16-byte aligned in bf16
])
def test_bad_shapes_are_rejected(lib, kw, code):
    with pytest.raises(sp.SpectralError) as e:
        sp.spectral_workspace_bytes(_shape(**kw), _params())
    assert e.value.code == code
    assert sp.spectral_last_error()


@pytest.mark.parametrize("kw", [dict(alpha=0.0), dict(eta_fp8=-1.0), dict(tol=-1e-3), dict(r_max=float("nan")),
                                dict(q_strips=-1), dict(flags=8)])
def test_bad_params_are_rejected(lib, kw):
    with pytest.raises(sp.SpectralError) as e:
        sp.spectral_workspace_bytes(_shape(), _params(**kw))
    assert e.value.code == sp.SN_EINVAL


def test_null_arguments(lib):
    assert lib.spectral_init(None, None, None, None) == sp.SN_ENULL
    assert lib.spectral_step(None, None, None, None, None, 1, None, None, None) == sp.SN_ENULL
    assert lib.spectral_set_stream(None, None) == sp.SN_ENULL
    lib.spectral_destroy(None)


def test_padded_rows_are_accepted(lib):
    # d = 250 with a padded row stride of 256 elements: rows 512-byte aligned
    assert sp.spectral_workspace_bytes(_shape(d_model=250, ld=256), _params()) > 0


def test_gram_form_workspace_and_limits(lib):
    base = sp.spectral_workspace_bytes(_shape(), _params())
    gram = sp.spectral_workspace_bytes(_shape(), _params(flags=sp.SN_FLAG_GRAM))
    # Gram partials: 2 d_h (d_h + 16) bytes per query / key head and strip, plus the final z, y
    units = 2 * (8 + 2)
    assert gram - base >= units * 2 * 64 * (64 + 16) + 2 * 8 * 2 * 64 * 4
    with pytest.raises(sp.SpectralError) as e:
        sp.spectral_workspace_bytes(_shape(head_dim=8), _params(flags=sp.SN_FLAG_GRAM))
    assert e.value.code == sp.SN_EINVAL and "Gram" in sp.spectral_last_error()


def test_row_block_size_limit(lib):
    # d_h * ld * element size must stay below 2^31 bytes (32-bit buffer offsets)
    with pytest.raises(sp.SpectralError) as e:
        sp.spectral_workspace_bytes(_shape(head_dim=128, d_model=1 << 23, ld=1 << 23), _params())
    assert e.value.code == sp.SN_EINVAL


def test_layer_form_needs_its_flag(lib):
    base = sp.spectral_workspace_bytes(_shape(), _params())
    lay = sp.spectral_workspace_bytes(_shape(), _params(flags=sp.SN_FLAG_LAYER))
    # column buffer of every query head plus u', v' per layer
    assert lay - base >= (2 * 8 * 256 + 2 * 2 * 256) * 4
    assert lib.spectral_step_layer(None, None, None, None, None, 1, None, None) == sp.SN_ENULL


def test_logit_consumer_workspace_holds_every_layer(lib):
    # pointer table of 3 L device pointers padded to 256 bytes, then hi/lo
    # bf16 planes of Q (n_q d_h columns) and K (n_kv d_h columns) per layer
    for L, seq in ((2, 100), (80, 1024)):
        got = sp.spectral_logits_workspace_bytes(_shape(n_layers=L), seq)
        table = (3 * L * 8 + 255) // 256 * 256
        assert got == table + L * seq * (8 + 2) * 64 * 4
    with pytest.raises(sp.SpectralError):
        sp.spectral_logits_workspace_bytes(_shape(), 0)


def test_noalloc_refuses_bad_calls_before_touching_the_device(lib):
    """The allocation-free entry point checks its arguments and the size of
    the workspace against its static scratch on the host, before any HIP call:
    the 70B GQA shape in tolerance mode (240 MB of workspace) does not fit."""
    one = [16] * 80
    shape = _shape(n_layers=80, d_model=8192, n_q_heads=64, n_kv_heads=8, head_dim=128)
    with pytest.raises(sp.SpectralError) as e:
        sp.spectral_step_noalloc(shape, _params(tol=1e-4), one, one, 16, 0, 3, 16, 16, 0)
    assert e.value.code == sp.SN_EINVAL and "scratch" in sp.spectral_last_error()
    with pytest.raises(sp.SpectralError) as e:
        sp.spectral_step_noalloc(_shape(), _params(), [16, 16], [16, 16], 0, 0, 3, 16, 16, 0)
    assert e.value.code == sp.SN_ENULL
    with pytest.raises(sp.SpectralError) as e:
        sp.spectral_step_noalloc(_shape(n_kv_heads=3), _params(), [16, 16], [16, 16], 16, 0, 3, 16, 16, 0)
    assert e.value.code == sp.SN_EINVAL
