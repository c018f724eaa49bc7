"""Cost-model calibration and toggle-boundary validation of App. D.2 / D.3 on
the GPU, with the engine's own kernels on the 4-layer 8B-shaped decoder
(hidden 4096, 32/8 heads x 128, FFN 14336, vocab 128256), over batch sizes
1-64, contexts 512 and 2048 and the paper's draft lengths 3, 7, 11, 15.

  - the two-stage fit reproduces the measured times (log residuals);
  - the toggle of the fitted model (predicted speedup >= 1 + eps) agrees with
    the decision the measured T_p, T_q, T_V imply at >= 95% of the (B, S,
    gamma, tau) points (eq:empirical_sd_speedup);
  - the library's sd_toggle with the fitted parameters takes exactly the
    oracle's decision at every one of those points."""
import math

import pytest

import oracle
from paper_2606_18967_amd import calibrate, sdrl, synth

from gpu_common import say

pytestmark = pytest.mark.gpu

GAMMAS = [3, 7, 11, 15]
TAUS = [2.0, 3.0, 4.0, 5.5, 7.5, 10.0, 13.0]


def test_l4_8b_sweep_fits_validates_and_toggle_matches_oracle():
    cfg = synth.L4_8B
    say("calibration sweep on the 4-layer 8B shape")
    res = calibrate.run(cfg, Bs=[1, 4, 16, 64], Ss=[512, 2048], gammas=GAMMAS, taus=TAUS, reps=5, log=say)
    ts = [s["t"] for s in res["samples"]]
    assert all(t > 0 and math.isfinite(t) for t in ts)
    assert res["F_eff"] > 1e14
    assert res["rms_log_residual"]["target"] < 0.25 and res["rms_log_residual"]["draft_verify"] < 0.25
    say("agreement", res["agreement"], "points", len(res["validation"]))
    assert res["agreement"] >= 0.95
    # the library's toggle against the oracle's on the same parameters
    lib_m = sdrl.cost_init(cfg, F_eff=res["F_eff"], **res["params"])
    orc = oracle.cost_arch(cfg["n_layers"], cfg["hidden"], cfg["n_q"], cfg["n_kv"], cfg["head_dim"], cfg["ffn"],
                           cfg["vocab"], F_eff=res["F_eff"], **res["params"])
    for f in ("W_T", "W_D", "kappa_th", "C_dense", "C_attn"):
        assert getattr(lib_m, f) == pytest.approx(getattr(orc, f), rel=1e-12)
    n = 0
    for row in res["validation"]:
        B, S, g, tau = row["B"], row["S"], row["gamma"], row["tau"]
        assert sdrl.toggle(lib_m, B, S, tau, g, res["eps"]) == oracle.toggle(orc, B, S, tau, g, res["eps"]), row
        assert sdrl.toggle(lib_m, B, S, tau, g, res["eps"]) == int(row["on_pred"]), row
        n += 1
    assert n == len(res["validation"]) >= 4 * 2 * 4 * 4
