"""Pins of the oracle's sampler and speculative rejection sampler.

Exactness of SD rests on the textbook law the paper relies on (Sec. 3.1,
App. D.1): the emitted token is distributed as p whatever q is, and a draft is
accepted with probability sum_x min(p, q).  These are checked by chi-square
tests over 10^6 draws, for generic, disjoint-support, identical and one-hot
pairs.  The fp16 rounding used for RTN scales is pinned to numpy's float16.
"""
import numpy as np
import pytest
from scipy import stats

import oracle


def softmax(l, T=1.0):
    x = np.asarray(l, dtype=np.float64) / T
    x = x - x.max()
    e = np.exp(x)
    return e / e.sum()


def chi2_p(counts, probs):
    counts = np.asarray(counts, dtype=np.float64)
    n = counts.sum()
    exp = probs * n
    keep = exp > 0
    assert counts[~keep].sum() == 0, "draws fell where the law has zero mass"
    if keep.sum() == 1:                       # a point mass: every draw must land on it
        return 1.0 if counts[keep][0] == n else 0.0
    return stats.chisquare(counts[keep], exp[keep]).pvalue


# ------------------------------------------------------------------ fp16 rounding
def test_f32_to_f16_matches_numpy():
    rng = np.random.default_rng(0)
    xs = np.concatenate([
        rng.standard_normal(20000).astype(np.float32) * 10.0 ** rng.integers(-9, 5, 20000),
        np.array([0.0, -0.0, 1.0, 65504.0, 65519.99, 65520.0, 1e9, 6e-8, 5.96e-8, 2.98e-8, 3e-8,
                  1 + 2**-11, 1 + 3 * 2**-11, 2049.0, 2051.0, np.inf, -np.inf], dtype=np.float32),
    ]).astype(np.float32)
    for x in xs:
        with np.errstate(over="ignore"):
            want = int(np.array([x], dtype=np.float32).astype(np.float16).view(np.uint16)[0])
        assert oracle.f32_to_f16(float(x)) == want, x
    # round trip of every finite fp16 value
    allh = np.arange(0, 0x7C00, dtype=np.uint16)
    vals = allh.view(np.float16).astype(np.float32)
    for h, v in zip(allh[::37], vals[::37]):
        assert oracle.f16_to_f32(int(h)) == v
        assert oracle.f32_to_f16(float(v)) == int(h)


# ------------------------------------------------------------------ exponential race
@pytest.mark.parametrize("T", [1.0, 0.7])
def test_race_law_is_softmax(T):
    rng = np.random.default_rng(1)
    l = rng.standard_normal(8).astype(np.float32) * 2
    n = 1_000_000
    counts = oracle.sample_hist(l, T, seed=11, step=3, n=n)
    assert counts.sum() == n
    assert chi2_p(counts, softmax(l, T)) > 1e-3


def test_race_single_entry_and_ties():
    x, _ = oracle.sample_row(np.array([3.0], np.float32), 1.0, 0, 0, 0, 0, 5)
    assert x == 0
    # a dominant entry always wins; -inf-like entries never do
    l = np.array([-1e4, 0.0, -1e4, -1e4], np.float32)
    for pos in range(50):
        x, gap = oracle.sample_row(l, 1.0, 1, 2, 0, 0, pos)
        assert x == 1 and gap > 100


# ------------------------------------------------------------------ rejection sampling
def _pairs():
    rng = np.random.default_rng(7)
    V = 8
    yield "generic", rng.standard_normal(V) * 1.5, rng.standard_normal(V) * 1.5
    a = np.full(V, -1e4)
    b = np.full(V, -1e4)
    a[:4] = rng.standard_normal(4)
    b[4:] = rng.standard_normal(4)
    yield "disjoint", a, b                      # p, q disjoint: every draft is rejected
    c = rng.standard_normal(V)
    yield "identical", c, c.copy()              # q = p: every draft is accepted
    d = np.full(V, -1e4); d[3] = 0.0
    yield "onehot_p", d, rng.standard_normal(V)
    yield "onehot_q", rng.standard_normal(V), d.copy()


@pytest.mark.parametrize("name,lp,lq", list(_pairs()), ids=[x[0] for x in _pairs()])
def test_rejection_law_and_acceptance(name, lp, lq):
    lp = lp.astype(np.float32)
    lq = lq.astype(np.float32)
    p, q = softmax(lp), softmax(lq)
    p2 = np.roll(lp, 3).astype(np.float32)      # row for the bonus draw
    n = 1_000_000
    counts, nacc = oracle.accept_hist(lq, lp, p2, 1.0, seed=5, step=9, n=n)
    # first emitted token ~ p (exactness of speculative sampling)
    assert chi2_p(counts, p) > 1e-3, (name, counts)
    # acceptance probability = sum min(p, q) = 1 - TV(p, q)
    beta = np.minimum(p, q).sum()
    sd = np.sqrt(max(beta * (1 - beta), 1e-12) / n)
    assert abs(nacc / n - beta) < 5 * sd + 1e-9, (name, nacc / n, beta)
    if name == "identical":
        assert nacc == n
    if name == "disjoint":
        assert nacc == 0


def test_accept_seq_invariants():
    rng = np.random.default_rng(3)
    V, gamma = 16, 5
    for trial in range(300):
        q = (rng.standard_normal((gamma, V)) * 2).astype(np.float32)
        p = (q[0:1].repeat(gamma + 1, 0) + rng.standard_normal((gamma + 1, V)) * 0.5).astype(np.float32)
        d = rng.integers(0, V, gamma).astype(np.int32)
        n, out, ratio, u, gap = oracle.accept_seq(d, q, p, 1.0, 1, trial, 0, 100)
        assert 1 <= n <= gamma + 1
        assert np.array_equal(out[:n - 1], d[:n - 1])    # accepted prefix is a prefix of the draft
        assert 0 <= out[n - 1] < V
        for j in range(n - 1):
            assert u[j] <= ratio[j]
        if n <= gamma:
            assert u[n - 1] > ratio[n - 1]
            assert np.all(np.isnan(ratio[n:]))
