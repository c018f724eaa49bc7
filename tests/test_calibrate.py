"""The cost-model calibration of App. D.2 (paper_2606_18967_amd/calibrate.py)
on the host: the two-step log-residual fit recovers known parameters from
noisy synthetic times, and validation against exact model times agrees on
every toggle decision."""
import math

import numpy as np
import pytest

from paper_2606_18967_amd import calibrate, sdrl, synth

TRUTH = dict(BW_eff=5.2e12, rho_kappa=0.8, c_T=2e-6, eta_D=1.3, c_D=1.5e-6, c_V=3e-6)


def _samples(base, noise, seed=0):
    rng = np.random.default_rng(seed)
    out = []
    for B in (1, 4, 16, 64, 128, 256):
        for S in (512, 2048, 8192):
            tp, tq, _ = calibrate.model_times(base, TRUTH, B, S, 1)
            out.append(dict(kind="p", B=B, S=S, gamma=1, t=tp * math.exp(noise * rng.standard_normal())))
            out.append(dict(kind="q", B=B, S=S, gamma=1, t=tq * math.exp(noise * rng.standard_normal())))
            for g in (3, 7, 11):
                tv = calibrate.model_times(base, TRUTH, B, S, g)[2]
                out.append(dict(kind="v", B=B, S=S, gamma=g, t=tv * math.exp(noise * rng.standard_normal())))
    return out


def _base():
    base = sdrl.cost_init(synth.L32_8B)
    base.F_eff = 1.6e15
    return base


def test_two_step_fit_recovers_parameters():
    base = _base()
    params, r1, r2 = calibrate.fit(base, _samples(base, 0.01))
    assert r1 < 0.02 and r2 < 0.02
    assert abs(params["BW_eff"] / TRUTH["BW_eff"] - 1) < 0.03
    assert abs(params["rho_kappa"] / TRUTH["rho_kappa"] - 1) < 0.05
    assert abs(params["eta_D"] / TRUTH["eta_D"] - 1) < 0.05
    for k in ("c_T", "c_D", "c_V"):          # overheads are weakly identified next to the bytes terms
        assert 0.5 < params[k] / TRUTH[k] < 2.0, (k, params[k])


def test_stage_one_uses_target_samples_only():
    base = _base()
    s = _samples(base, 0.0)
    p_all, _, _ = calibrate.fit(base, s)
    # corrupting the drafter / verify samples must not move the stage-1 parameters
    s2 = [dict(x, t=x["t"] * (3.0 if x["kind"] != "p" else 1.0)) for x in s]
    p_bad, _, _ = calibrate.fit(base, s2)
    for k in calibrate.FIT_KEYS_TARGET:
        assert p_bad[k] == pytest.approx(p_all[k], rel=1e-6)


def test_validation_agrees_with_exact_times():
    base = _base()
    meas = {}
    for B in (1, 16, 256):
        for S in (512, 8192):
            for g in (3, 7):
                tp, tq, tv = calibrate.model_times(base, TRUTH, B, S, g)
                meas[(B, S, g)] = (tp, tq, tv)
    rows, agree = calibrate.validate(base, TRUTH, meas, taus=[2.0, 4.0, 5.5, 7.5], eps=0.05)
    assert agree == 1.0 and rows
    assert all(r["pred"] == r["meas"] for r in rows)
    # speedup falls as the batch grows at fixed S, gamma, tau (compute-bound large batches)
    for S in (512, 8192):
        sp = [r["pred"] for r in rows if r["S"] == S and r["gamma"] == 3 and r["tau"] == 4.0]
        assert sp == sorted(sp, reverse=True)
