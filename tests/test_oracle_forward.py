"""Pins of the oracle's decoder forward and of its SD step.

  - A torch float64 re-implementation built on library primitives
    (F.rms_norm, F.scaled_dot_product_attention with a causal mask, F.silu)
    must give the same logits (rel 1e-5 of the row maximum).
  - Special cases: with no layers the logits are RMSNorm(E[x]) W_lm; at
    position 0 RoPE is the identity and the cached K/V are the projections of
    the normalised embedding; RoPE keeps the norm of every rotate-half pair.
  - SD invariants (App. D.1): n_emit in [1, gamma+1]; the accepted prefix is a
    prefix of the draft; after rollback the cache equals a fresh prefill of the
    emitted tokens (bit-exact in the oracle); with the drafter equal to the
    target SD reproduces AR token for token under shared uniforms.
  - The law of the first three emitted tokens of SD with a W4 drafter equals
    the target's AR law (chi-square against exact enumeration, V = 8).
"""
import numpy as np
import pytest
import torch
import torch.nn.functional as F
from scipy import stats

import oracle
from paper_2606_18967_amd import synth


def np_weights(cfg, seed, std=0.02):
    c = dict(cfg, dtype="f32")
    return [t.numpy().astype(np.float32) for t in synth.make_weights(c, seed, "cpu", std=std)]


def torch_forward(cfg, W, tokens):
    """Reference decoder in float64 on torch library primitives."""
    Wt = [torch.tensor(w, dtype=torch.float64) for w in W]
    H, nq, nkv, d, Fd = cfg["hidden"], cfg["n_q"], cfg["n_kv"], cfg["head_dim"], cfg["ffn"]
    n = len(tokens)
    pos = torch.arange(n, dtype=torch.float64)
    inv = cfg["rope_theta"] ** (-torch.arange(0, d // 2, dtype=torch.float64) * 2 / d)
    ang = pos[:, None] * inv[None, :]
    cos = torch.cat([ang.cos(), ang.cos()], -1)[:, None, :]
    sin = torch.cat([ang.sin(), ang.sin()], -1)[:, None, :]

    def rope(x):  # x [n, heads, d]
        x1, x2 = x[..., : d // 2], x[..., d // 2:]
        return x * cos + torch.cat([-x2, x1], -1) * sin

    eps = cfg.get("rms_eps", 1e-5)
    h = Wt[0][torch.tensor(tokens)]
    for l in range(cfg["n_layers"]):
        an, wqkv, wo, fn, wgu, wd = Wt[3 + 6 * l: 9 + 6 * l]
        a = F.rms_norm(h, (H,), an, eps)
        qkv = a @ wqkv.T
        q = rope(qkv[:, : nq * d].reshape(n, nq, d))
        k = rope(qkv[:, nq * d: (nq + nkv) * d].reshape(n, nkv, d))
        v = qkv[:, (nq + nkv) * d:].reshape(n, nkv, d)
        k = k.repeat_interleave(nq // nkv, dim=1)
        v = v.repeat_interleave(nq // nkv, dim=1)
        att = F.scaled_dot_product_attention(q.transpose(0, 1), k.transpose(0, 1), v.transpose(0, 1),
                                             is_causal=True)
        h = h + att.transpose(0, 1).reshape(n, nq * d) @ wo.T
        b = F.rms_norm(h, (H,), fn, eps)
        gu = b @ wgu.T
        h = h + (F.silu(gu[:, :Fd]) * gu[:, Fd:]) @ wd.T
    return (F.rms_norm(h, (H,), Wt[1], eps) @ Wt[2].T).numpy()


GQA = dict(name="gqa-test", n_layers=2, hidden=128, n_q=4, n_kv=2, head_dim=32, ffn=256, vocab=96,
           dtype="f32", rope_theta=10000.0, rms_eps=1e-5)


@pytest.mark.parametrize("cfg", [synth.TINY, GQA], ids=["tiny", "gqa"])
def test_forward_matches_torch_float64(cfg):
    W = np_weights(cfg, 3, std=0.05)
    m = oracle.Model(cfg, W, oracle.F32)
    tokens = np.random.default_rng(0).integers(0, cfg["vocab"], 12)
    kv = oracle.KV(cfg, 16)
    got = oracle.forward_seq(m, kv, tokens, 0)
    want = torch_forward(cfg, W, tokens)
    scale = np.abs(want).max(axis=1, keepdims=True)
    assert np.all(np.abs(got - want) <= 1e-5 * scale)


def test_zero_layers_is_norm_then_lm_head():
    cfg = dict(synth.TINY, n_layers=0)
    W = np_weights(cfg, 4, std=0.1)
    m = oracle.Model(cfg, W, oracle.F32)
    tok = [7, 300]
    got = oracle.forward_seq(m, oracle.KV(cfg, 4), tok, 0)
    e = W[0][tok].astype(np.float64)
    a = e / np.sqrt((e * e).mean(axis=1, keepdims=True) + 1e-5)
    assert np.allclose(got, a @ W[2].T.astype(np.float64), rtol=1e-6, atol=1e-7)


def test_position0_cache_and_rope_pair_norms():
    cfg = synth.TINY
    W = np_weights(cfg, 5, std=0.05)
    m = oracle.Model(cfg, W, oracle.F32)
    x = 123
    kv = oracle.KV(cfg, 40)
    oracle.forward_seq(m, kv, [x] * 33, 0, want_logits=False)
    H, nq, nkv, d = cfg["hidden"], cfg["n_q"], cfg["n_kv"], cfg["head_dim"]
    e = W[0][x].astype(np.float64)
    a = e / np.sqrt((e * e).mean() + 1e-5)
    qkv = a @ W[4].T.astype(np.float64)             # layer 0 Wqkv
    k0 = qkv[nq * d:(nq + nkv) * d].reshape(nkv, d)
    v0 = qkv[(nq + nkv) * d:].reshape(nkv, d)
    assert np.allclose(kv.k[0, :, 0, :], k0, rtol=1e-9, atol=1e-12)   # RoPE(0) = identity
    assert np.allclose(kv.v[0, :, 0, :], v0, rtol=1e-9, atol=1e-12)
    for p in (1, 7, 32):
        kp = kv.k[0, :, p, :]
        pn = np.hypot(kp[:, : d // 2], kp[:, d // 2:])
        assert np.allclose(pn, np.hypot(k0[:, : d // 2], k0[:, d // 2:]), rtol=1e-9)
        assert not np.allclose(kp, k0)
        assert np.allclose(kv.v[0, :, p, :], v0)     # values are not rotated


def _tiny_models(seed=0, std=0.02):
    cfg = synth.TINY
    W = np_weights(cfg, seed, std)
    target = oracle.Model(cfg, W, oracle.F32)
    drafter = oracle.make_drafter(cfg, W, oracle.F32)
    return cfg, W, target, drafter


def test_sd_step_invariants_and_rollback_equals_prefill():
    cfg, W, target, drafter = _tiny_models(1, std=0.05)
    rng = np.random.default_rng(1)
    prompt = rng.integers(0, cfg["vocab"], 16).astype(np.int32)
    cap, gamma = 80, 4
    kv = oracle.KV(cfg, cap)
    oracle.forward_seq(target, kv, prompt[:-1], 0, want_logits=False)
    kv_len, last = len(prompt) - 1, int(prompt[-1])
    emitted = list(prompt)
    n_total = 0
    for step in range(8):
        r = oracle.sd_step_seq(target, drafter, kv, kv_len, last, gamma, 1.0, seed=2, step=7, slot=0)
        n = r["n_emit"]
        assert 1 <= n <= gamma + 1
        assert np.array_equal(r["out"][: n - 1], r["draft"][: n - 1])
        emitted += list(r["out"])
        kv_len += n
        last = int(r["out"][-1])
        n_total += n
    fresh = oracle.KV(cfg, cap)
    oracle.forward_seq(target, fresh, np.array(emitted[:-1], np.int32), 0, want_logits=False)
    assert kv_len == len(emitted) - 1
    assert np.array_equal(kv.k[:, :, :kv_len], fresh.k[:, :, :kv_len])
    assert np.array_equal(kv.v[:, :, :kv_len], fresh.v[:, :, :kv_len])
    assert n_total > 8        # some drafts were accepted


def test_sd_with_target_as_drafter_reproduces_ar():
    cfg, W, target, _ = _tiny_models(2, std=0.05)
    rng = np.random.default_rng(2)
    prompt = rng.integers(0, cfg["vocab"], 10).astype(np.int32)
    cap, gamma, seed, step = 64, 3, 9, 4
    kv_a = oracle.KV(cfg, cap)
    oracle.forward_seq(target, kv_a, prompt[:-1], 0, want_logits=False)
    kv_s = kv_a.copy()
    ar, kv_len, last = [], len(prompt) - 1, int(prompt[-1])
    for _ in range(24):
        x, _, _ = oracle.ar_step_seq(target, kv_a, kv_len, last, 1.0, seed, step, 3)
        ar.append(x)
        kv_len += 1
        last = x
    sd, kv_len, last = [], len(prompt) - 1, int(prompt[-1])
    while len(sd) < 24:
        r = oracle.sd_step_seq(target, target, kv_s, kv_len, last, gamma, 1.0, seed, step, 3)
        assert r["n_emit"] == gamma + 1                     # q = p: every draft is accepted
        sd += list(r["out"])
        kv_len += r["n_emit"]
        last = int(r["out"][-1])
    assert sd[:24] == ar


CHAIN = dict(name="chain-v8", n_layers=1, hidden=128, n_q=2, n_kv=1, head_dim=64, ffn=128, vocab=8,
             dtype="f32", rope_theta=10000.0, rms_eps=1e-5)


def test_sd_chain_law_equals_target_ar_law():
    cfg = CHAIN
    W = np_weights(cfg, 11, std=0.35)
    target = oracle.Model(cfg, W, oracle.F32)
    drafter = oracle.make_drafter(cfg, W, oracle.F32)
    prompt = np.array([1, 5], np.int32)
    cap, gamma, K = 16, 3, 3
    base = oracle.KV(cfg, cap)
    oracle.forward_seq(target, base, prompt[:-1], 0, want_logits=False)

    def probs(kv, kv_len, tok):
        lg = oracle.forward_seq(target, kv, [tok], kv_len)[0].astype(np.float64)
        e = np.exp(lg - lg.max())
        return e / e.sum()

    # exact AR law of (x1, x2, x3)
    law = np.zeros((8, 8, 8))
    kv1 = base.copy()
    p1 = probs(kv1, 1, int(prompt[-1]))
    for a in range(8):
        kv2 = kv1.copy()
        p2 = probs(kv2, 2, a)
        for b in range(8):
            kv3 = kv2.copy()
            p3 = probs(kv3, 3, b)
            law[a, b] = p1[a] * p2[b] * p3
    assert abs(law.sum() - 1) < 1e-9

    n = 24_000
    counts = np.zeros((8, 8, 8))
    acc = 0
    for t in range(n):
        kv = base.copy()
        kv_len, last, out = 1, int(prompt[-1]), []
        while len(out) < K:
            r = oracle.sd_step_seq(target, drafter, kv, kv_len, last, gamma, 1.0, seed=77, step=t, slot=0)
            out += list(r["out"])
            acc += r["n_emit"] - 1
            kv_len += r["n_emit"]
            last = int(r["out"][-1])
        counts[out[0], out[1], out[2]] += 1
    assert 0 < acc < n * gamma          # both accept and reject paths were taken
    exp = law.ravel() * n
    obs = counts.ravel()
    big = exp >= 5
    e2 = np.append(exp[big], exp[~big].sum())
    o2 = np.append(obs[big], obs[~big].sum())
    assert stats.chisquare(o2, e2).pvalue > 1e-3
