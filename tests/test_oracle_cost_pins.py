"""Hand-worked pins of the oracle's cost model and speedup equation.

The terms are those of Sec. 4.2 (eq:toggle_latencies, eq:sd_speedup_toggle)
and Sec. 3.1 (eq:sd_speedup):

  M_T = (W_T + kappa_eff B S) / BW_eff,  M_D = (eta_D W_D + kappa_eff B S) / BW_eff,
  C   = B (C_dense + S C_attn) / F_eff,
  T_p = max(M_T, C) + c_T B,  T_q = max(M_D, C) + c_D B,
  T_V = max(M_T, (gamma + 1) C) + c_V B,
  speedup = tau T_p / (gamma T_q + T_V).

Every expected value below was worked out by hand from small round numbers
(written next to it), so a slip in the oracle's arithmetic cannot cancel
against the same slip in the test.  The points cover a memory-bound step, a
compute-bound step where verification pays (gamma + 1) C, the crossover of
T_V between its two branches, nonzero c_T, c_D, c_V, and the architecture
terms of a small decoder.  A mutation check then rebuilds the oracle with a
planted mistake in or_cost_times / or_sd_speedup / or_cost_arch (gamma C for
(gamma + 1) C, a dropped overhead, eta_D left out, the wrong C_attn) and
requires these pins to fail on each.
"""
import ctypes as C
import os
import shutil
import subprocess

import pytest

import oracle


def _cost(**kw):
    c = oracle.Cost()
    base = dict(W_T=0.0, W_D=0.0, kappa_th=0.0, C_dense=0.0, C_attn=0.0, BW_eff=1.0, F_eff=1.0,
                rho_kappa=1.0, eta_D=1.0, c_T=0.0, c_D=0.0, c_V=0.0)
    base.update(kw)
    for k, v in base.items():
        setattr(c, k, v)
    return c


def _times(L, c, B, S, gamma):
    tp, tq, tv = C.c_double(), C.c_double(), C.c_double()
    L.or_cost_times(C.byref(c), B, S, gamma, C.byref(tp), C.byref(tq), C.byref(tv))
    return tp.value, tq.value, tv.value


def _close(a, b):
    return abs(a - b) <= 1e-12 * max(1.0, abs(b))


def check_pins(L):
    """Returns the list of pins the library L violates (empty when all hold)."""
    bad = []

    # 1. memory-bound point: W_T 1000, W_D 300, kappa 2 (rho 0.5), B 4, S 10
    #    kv = 0.5*2*4*10 = 40; M_T = 1040/100 = 10.4; M_D = (2*300 + 40)/100 = 6.4
    #    C = 4*(10 + 10*1)/1000 = 0.08
    #    T_p = 10.4 + 0.25*4 = 11.4; T_q = 6.4 + 0.5*4 = 8.4; T_V = max(10.4, 4*0.08) + 1*4 = 14.4
    c1 = _cost(W_T=1000, W_D=300, kappa_th=2, C_dense=10, C_attn=1, BW_eff=100, F_eff=1000, rho_kappa=0.5,
               eta_D=2, c_T=0.25, c_D=0.5, c_V=1.0)
    got = _times(L, c1, 4, 10, 3)
    if not all(_close(g, w) for g, w in zip(got, (11.4, 8.4, 14.4))):
        bad.append(("memory-bound times", got))
    #    speedup at tau 3: 3*11.4/(3*8.4 + 14.4) = 34.2/39.6
    if not _close(L.or_sd_speedup(3.0, *got, 3), 34.2 / 39.6):
        bad.append(("memory-bound speedup", L.or_sd_speedup(3.0, *got, 3)))
    #    toggle with eps 0.05: on iff tau >= 1.05*39.6/11.4 = 3.6473...
    if L.or_toggle(C.byref(c1), 4, 10, 3.7, 3, 0.05) != 1 or L.or_toggle(C.byref(c1), 4, 10, 3.6, 3, 0.05) != 0:
        bad.append(("toggle threshold", None))

    # 2. compute-bound point: W_T 100, W_D 50, kappa 1, C_dense 100, C_attn 2, BW 100, F 100, B 2, S 5
    #    kv = 10; M_T = 1.1; M_D = 0.6; C = 2*(100 + 5*2)/100 = 2.2
    #    T_p = 2.2 + 0.1*2 = 2.4; T_q = 2.2 + 0.2*2 = 2.6; T_V = max(1.1, 5*2.2) + 0.3*2 = 11.6 (gamma 4)
    c2 = _cost(W_T=100, W_D=50, kappa_th=1, C_dense=100, C_attn=2, BW_eff=100, F_eff=100, c_T=0.1, c_D=0.2,
               c_V=0.3)
    got = _times(L, c2, 2, 5, 4)
    if not all(_close(g, w) for g, w in zip(got, (2.4, 2.6, 11.6))):
        bad.append(("compute-bound times", got))
    #    speedup at tau 5: 5*2.4/(4*2.6 + 11.6) = 12/22
    if not _close(L.or_sd_speedup(5.0, *got, 4), 12.0 / 22.0):
        bad.append(("compute-bound speedup", L.or_sd_speedup(5.0, *got, 4)))

    # 3. crossover of T_V: M_T = (500 + 4*25)/100 = 6, C = 4*50/100 = 2, no overheads
    #    T_V = max(6, (gamma+1)*2) = 6, 6, 8, 12 at gamma 1, 2, 3, 5; T_p = 6, T_q = (200 + 100)/100 = 3
    c3 = _cost(W_T=500, W_D=200, kappa_th=1, C_dense=50, BW_eff=100, F_eff=100)
    for gamma, tv in ((1, 6.0), (2, 6.0), (3, 8.0), (5, 12.0)):
        got = _times(L, c3, 4, 25, gamma)
        if not all(_close(g, w) for g, w in zip(got, (6.0, 3.0, tv))):
            bad.append((f"crossover gamma {gamma}", got))

    # 4. the speedup equation alone: tau 5, T_p 10, T_q 2, T_V 15, gamma 4 -> 50/23
    if not _close(L.or_sd_speedup(5.0, 10.0, 2.0, 15.0, 4), 50.0 / 23.0):
        bad.append(("speedup equation", L.or_sd_speedup(5.0, 10.0, 2.0, 15.0, 4)))

    # 5. architecture terms: L 2, H 4, n_q 2, n_kv 1, d 2, F 8, V 10; 2-byte target, 4-bit drafter, 2-byte KV
    #    QKVO = 2*(4*(2+2)*2 + 2*2*4) = 96; FFN = 2*3*4*8 = 192; embed + LM head = 2*10*4 = 80
    #    W_T = 2*(96 + 192 + 80) = 736; W_D = 0.5*288 + 2*80 = 304; kappa = 2*2*1*2*2 = 16
    #    C_dense = 2*(96 + 192 + 40) = 656; C_attn = 4*2*2*2 = 32
    ca = oracle.Cost()
    L.or_cost_arch(2, 4, 2, 1, 2, 8, 10, 2.0, 4.0, 2.0, C.byref(ca))
    want = dict(W_T=736, W_D=304, kappa_th=16, C_dense=656, C_attn=32)
    for k, w in want.items():
        if not _close(getattr(ca, k), w):
            bad.append((f"arch {k}", getattr(ca, k)))
    return bad


def test_cost_model_hand_worked_values():
    assert check_pins(oracle.lib()) == []


def test_speedup_is_throughput_ratio_of_a_simulated_timeline():
    """eq:sd_speedup read as a throughput ratio: SD blocks of gamma drafts and
    one verification, each emitting (accepted drafts + 1) tokens under i.i.d.
    acceptance alpha, against one AR token per T_p.  Simulated token by token."""
    import numpy as np
    rng = np.random.default_rng(5)
    alpha, gamma, Tp, Tq, Tv = 0.8, 4, 3.0, 1.0, 4.0
    n_blocks = 200_000
    acc = rng.random((n_blocks, gamma)) < alpha
    first_rej = np.where(~acc, np.arange(gamma), gamma).min(axis=1)
    tokens = (first_rej + 1).sum()
    sd_rate = tokens / (n_blocks * (gamma * Tq + Tv))
    ar_rate = 1.0 / Tp
    tau = oracle.tau_from_alpha(alpha, gamma)
    assert abs(sd_rate / ar_rate - oracle.sd_speedup(tau, Tp, Tq, Tv, gamma)) < 0.01


MUTATIONS = {
    "gamma C for (gamma+1) C": ("double CV = (gamma + 1) * C;", "double CV = gamma * C;"),
    "c_V B dropped": ("*Tv = (MT > CV ? MT : CV) + c->c_V * B;", "*Tv = (MT > CV ? MT : CV);"),
    "c_T B dropped": ("*Tp = (MT > C ? MT : C) + c->c_T * B;", "*Tp = (MT > C ? MT : C);"),
    "c_D for c_T": ("*Tq = (MD > C ? MD : C) + c->c_D * B;", "*Tq = (MD > C ? MD : C) + c->c_T * B;"),
    "eta_D dropped": ("double MD = (c->eta_D * c->W_D + kv) / c->BW_eff;", "double MD = (c->W_D + kv) / c->BW_eff;"),
    "rho_kappa dropped": ("double kv = c->rho_kappa * c->kappa_th * B * S;", "double kv = c->kappa_th * B * S;"),
    "S C_attn dropped": ("double C = B * (c->C_dense + S * c->C_attn) / c->F_eff;",
                         "double C = B * c->C_dense / c->F_eff;"),
    "speedup gamma T_q dropped": ("return tau * Tp / (gamma * Tq + Tv);\n}\n\n/* ----",
                                  "return tau * Tp / (Tq + Tv);\n}\n\n/* ----"),
    "C_attn with n_kv": ("out->C_attn = 4.0 * L * nq * d;", "out->C_attn = 4.0 * L * nkv * d;"),
}


@pytest.mark.skipif(shutil.which("gcc") is None, reason="needs gcc")
@pytest.mark.parametrize("name", list(MUTATIONS))
def test_planted_cost_model_mistakes_fail_the_pins(name, tmp_path):
    src = open(oracle.SRC).read()
    old, new = MUTATIONS[name]
    assert src.count(old) == 1, f"mutation site for {name!r} not found exactly once"
    mutated = tmp_path / "mut.c"
    mutated.write_text(src.replace(old, new))
    so = tmp_path / "libmut.so"
    subprocess.run(["gcc", "-O2", "-fPIC", "-shared", "-ffp-contract=off", "-o", str(so), str(mutated), "-lm",
                    "-fopenmp"], check=True)
    L = oracle._declare(C.CDLL(os.fspath(so)))
    assert check_pins(L) != [], f"planted mistake {name!r} passed every pin"
