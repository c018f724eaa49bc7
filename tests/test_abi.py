"""The C ABI on the CPU: the library loads without a GPU, exports every
function include/sd_api.h declares, and its host-side policy (cost model,
toggle, draft-length controller, tau/alpha) agrees with the oracle."""
import os
import re

import numpy as np
import pytest

import oracle
from paper_2606_18967_amd import sdrl, synth

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def declared_functions():
    src = open(os.path.join(ROOT, "include", "sd_api.h")).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    names = re.findall(r"\b(sd_\w+|kv_\w+)\s*\(", src)
    return sorted(set(names))


def test_every_declared_symbol_is_exported():
    names = declared_functions()
    assert len(names) >= 20
    L = sdrl.lib()
    missing = [n for n in names if not hasattr(L, n)]
    assert not missing, missing
    assert sorted(sdrl.API_SYMBOLS) == names


def _cfgs():
    return [synth.L4_8B, synth.L32_8B, synth.L64_32B, synth.TINY]


@pytest.mark.parametrize("cfg", _cfgs(), ids=lambda c: c["name"])
def test_cost_model_matches_oracle(cfg):
    calib = dict(BW_eff=5.5e12, F_eff=1.3e15, rho_kappa=0.9, eta_D=1.2, c_T=2e-6, c_D=1.5e-6, c_V=3e-6)
    m = sdrl.cost_init(cfg, 2.0, 4.0, 2.0, **calib)
    o = oracle.cost_arch(cfg["n_layers"], cfg["hidden"], cfg["n_q"], cfg["n_kv"], cfg["head_dim"], cfg["ffn"],
                         cfg["vocab"], 2.0, 4.0, 2.0, **calib)
    for f in ("W_T", "W_D", "kappa_th", "C_dense", "C_attn"):
        assert getattr(m, f) == pytest.approx(getattr(o, f), rel=1e-12), f
    rng = np.random.default_rng(0)
    for _ in range(200):
        B, S, g = int(rng.integers(1, 300)), float(rng.uniform(1, 16000)), int(rng.integers(1, 16))
        a = sdrl.cost_times(m, B, S, g)
        b = oracle.cost_times(o, B, S, g)
        assert np.allclose(a, b, rtol=1e-12)
        tau = float(rng.uniform(1, g + 1))
        assert sdrl.toggle(m, B, S, tau, g, 0.05) == oracle.toggle(o, B, S, tau, g, 0.05)
    assert sdrl.toggle(m, 256, 512, 1.0, 4, 0.05, sd_on=1) == 1          # sticky


def test_gamma_controller_matches_oracle():
    rng = np.random.default_rng(1)
    gset = [5, 7, 9, 11]
    for trial in range(50):
        ctl = sdrl.GammaController(gset, P=2, a_up=0.94, a_down=0.85)
        g, hist = gset[0], []
        for t in range(30):
            tau = float(rng.uniform(1, g + 1.5))
            hist.append(tau)
            g = oracle.gamma_next(gset, g, hist, 2, 0.94, 0.85)
            assert ctl.update(tau) == g


def test_tau_alpha_match_oracle():
    for g in (1, 3, 5, 7, 11):
        for a in np.linspace(0, 0.999, 37):
            assert sdrl.tau_from_alpha(a, g) == pytest.approx(oracle.tau_from_alpha(a, g), rel=1e-12)
        for tau in np.linspace(1.0, g + 1.0, 23):
            assert sdrl.alpha_from_tau(tau, g) == pytest.approx(oracle.alpha_from_tau(tau, g), abs=1e-9)


def test_sizes():
    c = sdrl.model_cfg(synth.L4_8B)
    L = sdrl.lib()
    import ctypes as C
    assert L.sd_num_weights(C.byref(c)) == 3 + 6 * 4
    assert L.sd_kv_bytes(C.byref(c), 64, 2100) == 4 * 64 * 8 * 2100 * 128 * 2
    from oracle.parity import drafter_layout
    _, total = drafter_layout(synth.L4_8B)
    assert L.sd_drafter_bytes(C.byref(c)) == total
    for fmt, code in sdrl.DRAFT_FORMATS.items():
        _, total = drafter_layout(synth.L4_8B, fmt)
        assert L.sd_drafter_bytes_fmt(C.byref(c), code) == total, fmt
    assert L.sd_drafter_bytes_fmt(C.byref(c), 3) == 0
    assert L.sd_drafter_bytes_fmt(C.byref(c), -1) == 0
    # host-side argument checks of the refresh need no device
    assert L.sd_refresh_drafter_fmt(None, 1, None, 0, None) == 1      # SD_E_INVAL
    assert L.sd_kv_page_bytes(C.byref(c), 64) == 4 * 8 * 64 * 128 * 2
    assert L.sd_kv_page_bytes(C.byref(c), 0) == 0
    assert L.sd_bind_kv_paged(None, None, None, 4, 64, None, 4, None) == 1
