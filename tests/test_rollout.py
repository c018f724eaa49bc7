"""Host logic of the long-tail rollout driver (Algorithm 1): the decode loop's
accounting, the sticky toggle, and the training loop's tau / gamma wiring.
Runs on the CPU with stand-ins for the GPU iterations; the policy functions
are the library's own (host C)."""
import numpy as np
import pytest

from paper_2606_18967_amd import rollout, sdrl, synth


class FakeClock:
    def __init__(self):
        self.t = 0.0

    def __call__(self):
        self.t += 0.5
        return self.t


def fake_fns(n_sd):
    """AR emits 1 per row; SD emits n_sd (a scalar or a function of the live
    batch size); records the live batch size of every call and compactions."""
    log = dict(calls=[], compact=[])
    live = {"B": None}

    def ar_fn():
        log["calls"].append(("ar", live["B"]))
        return np.ones(live["B"], dtype=np.int64)

    def sd_fn(g):
        log["calls"].append(("sd", live["B"], g))
        k = n_sd(live["B"]) if callable(n_sd) else n_sd
        return np.full(live["B"], k, dtype=np.int64)

    def compact_fn(keep):
        log["compact"].append(int(keep.sum()))
        live["B"] = int(keep.sum())

    return live, log, ar_fn, sd_fn, compact_fn


def cost_l32():
    m = sdrl.cost_init(synth.L32_8B)
    m.BW_eff, m.F_eff, m.rho_kappa, m.eta_D = 5.1e12, 7.1e14, 0.93, 0.97
    m.c_T, m.c_D, m.c_V = 2.7e-6, 3.2e-6, 1.6e-5
    return m


def test_response_lengths_seeded_and_clipped():
    a = rollout.response_lengths(4096, 512, 0.894, 16, 4096, 7)
    b = rollout.response_lengths(4096, 512, 0.894, 16, 4096, 7)
    assert (a == b).all()
    assert a.min() >= 16 and a.max() <= 4096
    assert abs(np.median(a) - 512) < 40                     # the log-normal's median
    assert (rollout.response_lengths(100, 512, 0.894, 16, 4096, 8) != a[:100]).any()


def test_ar_rollout_accounting():
    L = np.array([3, 1, 7, 4, 7])
    live, log, ar_fn, sd_fn, compact_fn = fake_fns(3)
    live["B"] = len(L)
    st = rollout.decode(L, 100, "ar", 5, 5.0, None, 0.05, ar_fn, sd_fn, compact_fn, clock=FakeClock())
    assert st["ar_iters"] == L.max() and st["sd_iters"] == 0 and st["tau"] is None
    assert (st["gen"] == L).all()
    # live batch per iteration: all 5, then as the lengths run out
    assert [c[1] for c in log["calls"]] == [5, 4, 4, 3, 2, 2, 2]
    assert log["compact"] == [4, 3, 2]                       # the last drop empties the batch: no compaction call
    assert st["makespan_s"] == pytest.approx(0.5 * st["ar_iters"])
    assert [t[4] for t in st["trace"]] == [c[1] for c in log["calls"]]


def test_sd_rollout_truncates_and_measures_tau():
    L = np.array([5, 12, 1])
    live, log, ar_fn, sd_fn, compact_fn = fake_fns(4)
    live["B"] = len(L)
    st = rollout.decode(L, 10, "sd", 5, 5.0, None, 0.05, ar_fn, sd_fn, compact_fn, clock=FakeClock())
    assert st["ar_iters"] == 0 and st["sd_iters"] == 3           # 12 tokens at 4 per iteration
    assert (st["gen"] >= L).all() and (st["gen"] - L < 4).all()  # the last iteration may overshoot
    assert st["tau"] == pytest.approx(4.0)
    assert all(c[2] == 5 for c in log["calls"])


def test_toggle_switches_once_at_the_predicted_batch_and_stays_on():
    m = cost_l32()
    prompt, tau, gamma, eps = 512, 3.5, 5, 0.05
    rng = np.random.default_rng(0)
    L = rng.integers(1, 200, size=64)
    L[0] = 400                                                   # one long response: the tail
    live, log, ar_fn, sd_fn, compact_fn = fake_fns(1)            # SD emitting 1 keeps the schedule like AR
    live["B"] = len(L)
    st = rollout.decode(L, prompt, "toggle", gamma, tau, m, eps, ar_fn, sd_fn, compact_fn, clock=FakeClock())
    modes = [c[0] for c in log["calls"]]
    k = modes.index("sd")
    assert set(modes[:k]) == {"ar"} and set(modes[k:]) == {"sd"}          # sticky once on
    assert st["switch_iter"] == k and st["switch_B"] == log["calls"][k][1]
    # the switch point is the first iteration whose predicted speedup reaches 1 + eps
    gen = np.zeros(len(L))
    for i in range(k + 1):
        alive = gen < L
        B, S = int(alive.sum()), prompt + float(np.minimum(gen[alive], L[alive]).mean())
        tp, tq, tv = sdrl.cost_times(m, B, S, gamma)
        assert (tau * tp / (gamma * tq + tv) >= 1 + eps) == (i == k)
        gen[alive] += 1
    assert 1 <= st["switch_B"] < 64


def test_toggle_never_on_when_tau_is_low():
    L = np.array([50, 80, 120])
    live, log, ar_fn, sd_fn, compact_fn = fake_fns(2)
    live["B"] = len(L)
    st = rollout.decode(L, 512, "adaptive", 5, 1.0, cost_l32(), 0.05, ar_fn, sd_fn, compact_fn)
    assert st["sd_iters"] == 0 and st["switch_iter"] is None and st["tau"] is None


def test_bad_iterations_are_rejected():
    live, log, ar_fn, sd_fn, compact_fn = fake_fns(0)
    live["B"] = 2
    with pytest.raises(RuntimeError):
        rollout.decode(np.array([3, 3]), 8, "sd", 5, 5.0, None, 0.05, ar_fn, sd_fn, compact_fn)
    with pytest.raises(ValueError):
        rollout.decode(np.array([3, 0]), 8, "ar", 5, 5.0, None, 0.05, ar_fn, sd_fn, compact_fn)
    with pytest.raises(ValueError):
        rollout.decode(np.array([3]), 8, "always", 5, 5.0, None, 0.05, ar_fn, sd_fn, compact_fn)


def scripted_run(taus):
    """run_fn stand-in: the t-th rollout measures taus[t] (None: no SD ran)."""
    calls = []

    def run_fn(policy, gamma, tau_prev, lengths, step):
        calls.append((gamma, tau_prev))
        return rollout.RolloutResult(policy=policy, step=step, gamma=gamma, tau_prev=tau_prev, tau=taus[step],
                                     makespan_s=1.0, prep_ms=0.0, ar_iters=0, sd_iters=1, tokens=0,
                                     switch_iter=0, switch_B=1)
    return run_fn, calls


def test_training_loop_feeds_tau_and_moves_gamma_with_patience():
    taus = [5.8, 5.8, 7.8, 7.8, None, 2.0, 2.0]
    run_fn, calls = scripted_run(taus)
    rs = rollout.train(run_fn, "adaptive", len(taus), lambda t: None)
    # Algorithm 1: gamma_1 = gamma_low = 5, tau_0 = gamma_low
    assert calls[0] == (5, 5.0)
    # after two steps with tau >= 1 + 5 * 0.94 = 5.7 the draft length moves up to 7; 7.8 twice
    # (>= 1 + 7 * 0.94 = 7.58) moves it to 9; a step with no SD keeps tau and gamma; the last
    # two measured taus, 7.8 and 2.0, are both <= 1 + 9 * 0.85 = 8.65, which moves it back to 7
    assert [c[0] for c in calls] == [5, 5, 7, 7, 9, 9, 7]
    assert [r.gamma for r in rs] == [5, 5, 7, 7, 9, 9, 7]
    # Algorithm 1 as written: the toggle gets the last measured tau as it is
    assert [c[1] for c in calls] == [5.0, 5.8, 5.8, 7.8, 7.8, 7.8, 2.0]
    # the carry variant: the last measured tau moved to the new draft length when gamma changed
    run_fn3, calls3 = scripted_run(taus)
    rollout.train(run_fn3, "adaptive", len(taus), lambda t: None, tau_carry=True)
    assert [c[0] for c in calls3] == [5, 5, 7, 7, 9, 9, 7]

    def carried(tau, g0, g1):
        a = sdrl.alpha_from_tau(tau, g0)
        return sum(a ** i for i in range(g1 + 1))
    want = [5.0, 5.8, carried(5.8, 5, 7), 7.8, carried(7.8, 7, 9), carried(7.8, 7, 9), carried(2.0, 9, 7)]
    assert [c[1] for c in calls3] == pytest.approx(want, rel=1e-9)
    assert calls3[2][1] > 5.8 and calls3[6][1] < 2.0
    run_fn2, calls2 = scripted_run(taus)
    rollout.train(run_fn2, "toggle", len(taus), lambda t: None)
    assert {c[0] for c in calls2} == {5}                         # fixed gamma_low without the adaptive policy
    assert [c[1] for c in calls2] == [5.0, 5.8, 5.8, 7.8, 7.8, 7.8, 2.0]


def test_tau_carried_across_draft_lengths():
    for alpha in (0.3, 0.71, 0.98):
        for g0, g1 in ((5, 7), (9, 5), (4, 11)):
            t0 = sum(alpha ** i for i in range(g0 + 1))
            assert rollout.tau_at(t0, g0, g1) == pytest.approx(sum(alpha ** i for i in range(g1 + 1)), rel=1e-9)
    assert rollout.tau_at(3.3, 5, 5) == 3.3
    assert rollout.tau_at(6.0, 5, 9) == pytest.approx(10.0)       # every draft accepted stays so


def test_calibrated_cost_takes_the_fitted_terms():
    calib = dict(F_eff=7.0e14, params=dict(BW_eff=5.0e12, rho_kappa=0.9, eta_D=0.95, c_T=1e-6, c_D=2e-6, c_V=3e-6))
    m = rollout.calibrated_cost(synth.L4_8B, calib)
    base = sdrl.cost_init(synth.L4_8B)
    assert m.F_eff == 7.0e14 and m.BW_eff == 5.0e12 and m.c_V == 3e-6
    assert m.W_T == base.W_T and m.kappa_th == base.kappa_th


def test_buckets_pad_to_multiples():
    assert [rollout.bucket_of(n) for n in (1, 7, 8, 9, 16, 17, 128)] == [8, 8, 8, 16, 16, 24, 128]
    with pytest.raises(ValueError):
        rollout.bucket_of(0)


def test_capture_time_is_kept_out_of_the_makespan():
    """An iteration that returns (tokens, capture seconds) is timed without
    its capture; the capture time is accumulated apart."""
    clock = iter([0.0, 1.0, 1.5, 2.5]).__next__
    outs = [(np.array([2, 3]), 0.75), np.array([3])]

    def sd_fn(g):
        return outs.pop(0)

    st = rollout.decode(np.array([5, 3]), 10, "sd", 4, 5.0, None, 0.05, lambda: None, sd_fn, lambda keep: None,
                        clock=clock)
    assert st["sd_iters"] == 2 and st["capture_s"] == 0.75
    assert st["makespan_s"] == pytest.approx(0.25 + 1.0)
