"""The decision-parity rule of oracle/parity.py, checked on the CPU: a
decision that differs from the oracle's own only through logits within the
tolerance is exempt when the oracle's accept on the device's logits gives the
device's tokens, and a planted sampler error is still caught."""
import numpy as np
import pytest

import oracle
from oracle.parity import Mismatch, compare_step


def _oracle_step(draft, q, p, T, key):
    n, out, ratio, u, fgap = oracle.accept_seq(draft, q, p, T, *key)
    return dict(n_emit=n, draft=draft, q=q, p=p, out=out[:n].copy(), draft_gap=np.full(len(draft), 1e9, np.float32),
                ratio=ratio, u=u, final_gap=fgap)


def _find_flip(V=64, gamma=3, T=1.0, rel=1e-2, tries=4000):
    """Seeded logits whose accept decision flips under a perturbation of at
    most rel * max|p| (inside a 2e-2 tolerance)."""
    rng = np.random.default_rng(7)
    for t in range(tries):
        q = rng.normal(0, 1.5, (gamma, V)).astype(np.float32)
        p = (q[np.r_[0:gamma, gamma - 1]] + rng.normal(0, 0.3, (gamma + 1, V))).astype(np.float32)
        draft = q.argmax(axis=1).astype(np.int32)
        key = (3, t, 5, 100)
        r = _oracle_step(draft, q, p, T, key)
        pd = (p + rel * np.abs(p).max() * rng.uniform(-1, 1, p.shape)).astype(np.float32)
        n2, out2, *_ = oracle.accept_seq(draft, q, pd, T, *key)
        k = min(n2, r["n_emit"])
        if n2 != r["n_emit"] and k <= gamma and abs(float(r["u"][k - 1]) - float(r["ratio"][k - 1])) >= 1e-3:
            return r, dict(draft=draft, q=q, p=pd, out=out2[:n2].copy(), n_emit=n2), key
    pytest.fail("no decision flip found")


def test_flip_within_tolerance_is_exempt_on_identical_logits():
    r, dev, key = _find_flip()
    status, info = compare_step(r, dev, 2e-2, 1.0, key=key)
    assert status == "exempt" and info["note"] == "oracle on device logits agrees", info
    # without the step's key (no identical-logits check) the same flip is a mismatch
    with pytest.raises(Mismatch):
        compare_step(r, dev, 2e-2, 1.0)


@pytest.mark.parametrize("plant", ["last_token", "one_more_accept", "one_less_accept"])
def test_planted_sampler_error_is_caught(plant):
    r, dev, key = _find_flip()
    bad = dict(dev)
    out, n = dev["out"].copy(), dev["n_emit"]
    V = dev["q"].shape[1]
    if plant == "last_token":
        out[n - 1] = (out[n - 1] + 1) % V
    elif plant == "one_more_accept" and n <= len(dev["draft"]):
        out = np.concatenate([dev["draft"][:n], [0]]).astype(np.int32)
        n += 1
    else:
        n = max(1, n - 1)
        out = np.concatenate([dev["draft"][:n - 1], [(int(dev["draft"][n - 1]) + 1) % V]]).astype(np.int32)
    bad["out"], bad["n_emit"] = out, n
    if n == r["n_emit"] and np.array_equal(out, r["out"]):
        pytest.skip("the planted tokens happen to equal the oracle's")
    with pytest.raises(Mismatch):
        compare_step(r, bad, 2e-2, 1.0, key=key)


def test_logits_outside_tolerance_are_caught():
    r, dev, key = _find_flip()
    bad = dict(dev)
    bad["p"] = dev["p"].copy()
    bad["p"][0, 0] += 0.05 * np.abs(r["p"]).max()
    with pytest.raises(Mismatch, match="verify logits"):
        compare_step(r, bad, 2e-2, 1.0, key=key)
