"""The calibration sweep of App. D.2 on the GPU with the engine's own kernels,
small enough to run in seconds: the measured times are positive and ordered
as the roofline model expects, and the fitted model reproduces them."""
import math

import pytest

from paper_2606_18967_amd import calibrate, synth

from gpu_common import say

pytestmark = pytest.mark.gpu

SMALL = dict(name="small-gqa-bf16", n_layers=2, hidden=512, n_q=4, n_kv=2, head_dim=128, ffn=1024, vocab=4096,
             dtype="bf16", rope_theta=10000.0, rms_eps=1e-5)


def test_small_sweep_fits_and_validates():
    say("calibration sweep on a small bf16 model")
    res = calibrate.run(SMALL, Bs=[1, 8, 32], Ss=[128, 1024], gammas=[3], taus=[2.0, 4.0], reps=3, log=say)
    ts = [s["t"] for s in res["samples"]]
    assert all(t > 0 and math.isfinite(t) for t in ts)
    # a verify step over gamma + 1 tokens costs at least one draft step and at most a few target steps
    for (B, S, g), _ in [((s["B"], s["S"], s["gamma"]), None) for s in res["samples"] if s["kind"] == "v"]:
        tp = next(s["t"] for s in res["samples"] if s["kind"] == "p" and s["B"] == B and s["S"] == S)
        tv = next(s["t"] for s in res["samples"] if s["kind"] == "v" and s["B"] == B and s["S"] == S)
        assert 0.5 * tp < tv < 10 * tp
    assert res["F_eff"] > 1e14
    assert res["rms_log_residual"]["target"] < 0.5 and res["rms_log_residual"]["draft_verify"] < 0.5
    assert 0.0 <= res["agreement"] <= 1.0
    assert 1.0 <= res["measured_tau"][3] <= 4.0
