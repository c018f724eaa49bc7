"""The decision-parity rule of oracle/parity.py, checked on the CPU.

Decisions are judged on the device's own logits, so a correct sampler passes
whatever logit differences (within the tolerance) its forward pass has, and
every planted sampler error is caught: a wrong draft token, wrong q row
statistics, one accept too many or too few, a wrong final token.  The
rounding-level exemptions fire only where they should: an accept test with
|u - p/q| < 1e-3 that flips n_emit, and nothing else."""
import numpy as np
import pytest

import oracle
from oracle.parity import Mismatch, check_accept, check_ar, check_draws, check_step

V, GAMMA, T = 64, 3, 1.0


def _device_step(seed=7, t=0):
    """Logits of one step and the decisions a correct device takes on them
    (the oracle's own sampler stands in for the device)."""
    rng = np.random.default_rng(seed + t)
    q = rng.normal(0, 1.5, (GAMMA, V)).astype(np.float32)
    p = (q[np.r_[0:GAMMA, GAMMA - 1]] + rng.normal(0, 0.3, (GAMMA + 1, V))).astype(np.float32)
    key = (3, t, 5, 100)
    draft = np.array([oracle.sample_row(q[j], T, key[0], key[1], oracle.STREAM_TOKEN, key[2], key[3] + j + 1)[0]
                      for j in range(GAMMA)], np.int32)
    stats = np.array([oracle.row_stats(q[j], T) for j in range(GAMMA)], np.float32)
    n, out, *_ = oracle.accept_seq(draft, q, p, T, *key)
    out[n:] = -1
    return dict(draft=draft, q=q, q_stats=stats, p=p, out=out, n_emit=n), key


def test_correct_device_passes_with_logits_inside_the_tolerance():
    rng = np.random.default_rng(0)
    for t in range(40):
        dev, key = _device_step(t=t)
        # the oracle's teacher-forced logits differ from the device's by up to 1% of the row maximum
        q_ref = dev["q"] + 0.01 * np.abs(dev["q"]).max() * rng.uniform(-1, 1, dev["q"].shape).astype(np.float32)
        p_ref = dev["p"] + 0.01 * np.abs(dev["p"]).max() * rng.uniform(-1, 1, dev["p"].shape).astype(np.float32)
        info = check_step(dev, q_ref, p_ref, 2e-2, T, key)
        assert info["exempt"] == 0


def test_logits_outside_tolerance_are_caught():
    dev, key = _device_step()
    p_ref = dev["p"].copy()
    p_ref[0, 0] += 0.05 * np.abs(p_ref).max()
    with pytest.raises(Mismatch, match="verify logits"):
        check_step(dev, dev["q"], p_ref, 2e-2, T, key)
    q_ref = dev["q"].copy()
    q_ref[1, 5] -= 0.05 * np.abs(q_ref).max()
    with pytest.raises(Mismatch, match="draft logits"):
        check_step(dev, q_ref, dev["p"], 2e-2, T, key)


def test_wrong_draft_token_is_caught():
    dev, key = _device_step()
    bad = dict(dev, draft=dev["draft"].copy())
    bad["draft"][1] = (bad["draft"][1] + 1) % V
    with pytest.raises(Mismatch, match="draft draw 1"):
        check_draws(bad["q"], bad["draft"], T, key)


def test_wrong_q_stats_are_caught():
    dev, key = _device_step()
    st = dev["q_stats"].copy()
    st[2, 1] += 1e-3
    with pytest.raises(Mismatch, match="q_stats"):
        check_draws(dev["q"], dev["draft"], T, key, st)


def _find(pred, tries=3000):
    for t in range(tries):
        dev, key = _device_step(t=t)
        if pred(dev):
            return dev, key
    pytest.fail("no case found")


@pytest.mark.parametrize("plant", ["last_token", "one_more_accept", "one_less_accept"])
def test_planted_accept_errors_are_caught(plant):
    dev, key = _find(lambda d: 2 <= d["n_emit"] <= GAMMA)
    bad = dict(dev)
    out, n = dev["out"].copy(), dev["n_emit"]
    if plant == "last_token":
        out[n - 1] = (out[n - 1] + 1) % V
    elif plant == "one_more_accept":
        out[:n] = dev["draft"][:n]
        out[n] = 0
        n += 1
    else:
        n -= 1
        out[n - 1] = (int(dev["draft"][n - 1]) + 1) % V
        out[n:] = -1
    bad["out"], bad["n_emit"] = out, n
    with pytest.raises(Mismatch):
        check_accept(bad, T, key)


def test_accept_band_exempts_only_a_flip_of_n_emit():
    # a deciding test with u within 1e-3 of p/q: the opposite decision is a rounding-level tie
    for t in range(20000):
        dev, key = _device_step(t=t)
        n_o, out_o, ratio, u, _ = oracle.accept_seq(dev["draft"], dev["q"], dev["p"], T, *key)
        j = n_o if n_o <= GAMMA else GAMMA      # the last examined accept test (1-based)
        if abs(float(u[j - 1]) - float(ratio[j - 1])) < 1e-3:
            break
    else:
        pytest.skip("no near-tie accept test in the sample")
    flipped = dict(dev, out=dev["out"].copy())
    if n_o <= GAMMA:        # the oracle rejected at j: the device accepting it emits one more draft
        flipped["out"][:j] = dev["draft"][:j]
        flipped["out"][j] = 0
        flipped["n_emit"] = j + 1
    else:                   # the oracle accepted every draft: the device rejecting the last one
        flipped["out"][j - 1] = (int(dev["draft"][j - 1]) + 1) % V
        flipped["out"][j:] = -1
        flipped["n_emit"] = j
    status, info = check_accept(flipped, T, key)
    assert status == "exempt" and info["where"] == f"accept {j}"
    # the same n_emit with a different final token is not covered by the band
    same_n = dict(dev, out=dev["out"].copy())
    same_n["out"][n_o - 1] = (int(dev["out"][n_o - 1]) + 1) % V
    with pytest.raises(Mismatch):
        check_accept(same_n, T, key)


def test_ar_token_judged_on_device_logits():
    rng = np.random.default_rng(4)
    p = rng.normal(0, 2, V).astype(np.float32)
    key = (9, 2, 1, 50)
    x, _ = oracle.sample_row(p, T, key[0], key[1], oracle.STREAM_TOKEN, key[2], key[3] + 1)
    ref = p + 0.005 * np.abs(p).max()
    assert check_ar(p, x, ref, 2e-2, T, key)[0] == "ok"
    with pytest.raises(Mismatch, match="AR token"):
        check_ar(p, (x + 1) % V, ref, 2e-2, T, key)
