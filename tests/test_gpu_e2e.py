"""End-to-end GPU parity of the SD step through the C ABI against the oracle.

Every step of every sequence is checked (oracle.parity.check_step): the
device's decisions on its own logits must be the oracle's (draws, q row
statistics, accept tests, residual and bonus draws), and its logits must
match the oracle teacher-forced onto the device's tokens.

  - the tiny fp32 decoder (2 layers, hidden 256, 4x64 MHA, FFN 1024, vocab
    512; B = 4, 64-token prompts grown to 128 tokens, gamma = 4, T = 1): the
    whole rollout, logits within 5e-3 of the row maximum, and the cache after
    the rollout;
  - the plain AR path on the same model;
  - small bf16 decoders with GQA and head_dim 128, from a prefilled prompt and
    from random context spanning several attention chunks and a ragged tail
    (logits within 2e-2 of the row maximum);
  - the same rollouts on a paged cache, through a captured HIP graph, and
    with the discarded-KV poison switched on.
"""
import numpy as np
import pytest
import torch

import oracle
from oracle.parity import check_ar
from paper_2606_18967_amd import synth

from gpu_common import check_cache, host_bits, i32, make_engine, oracle_models, run_rollout, say

pytestmark = pytest.mark.gpu


def test_tiny_fp32_sd_rollout_matches_oracle():
    cfg, run = synth.TINY, synth.TINY_RUN
    say("tiny fp32 SD rollout", run)
    W = synth.make_weights(cfg, run["seed"], "cpu")
    prompt = synth.make_tokens(run["B"], run["prompt"], cfg["vocab"], run["seed"])
    eng, kv, okv, o_len, st = run_rollout(cfg, W, prompt, run["B"], run["context"], run["gamma"], run["T"],
                                          run["seed"], 3, tol=5e-3)
    say("stats", st)
    assert st["exempt"] == 0 and st["checked"] > 10
    assert st["emitted"] / st["checked"] > 1.5       # the drafter is accepted often enough to exercise chains
    check_cache(cfg, kv, okv, o_len, 5e-3)
    eng.close()


@pytest.mark.parametrize("T", [1.0, 0.5, 1.6])
def test_tiny_fp32_ar_matches_oracle(T):
    cfg, run = synth.TINY, synth.TINY_RUN
    say("tiny fp32 AR", T)
    B, P, seed, step = run["B"], run["prompt"], 4, 8
    W = synth.make_weights(cfg, seed, "cpu")
    prompt = synth.make_tokens(B, P, cfg["vocab"], seed)
    eng, k, v, kv_len = make_engine(cfg, [w.cuda() for w in W], B, 128, 4)
    target, _ = oracle_models(cfg, host_bits(W))
    okv = [oracle.KV(cfg, 128) for _ in range(B)]
    eng.prefill(i32(np.arange(B)), prompt[:, :P - 1].cuda())
    for b in range(B):
        oracle.forward_seq(target, okv[b], prompt[b, :P - 1].numpy(), 0, want_logits=False)
    last = [int(x) for x in prompt[:, P - 1]]
    out = torch.zeros(B, dtype=torch.int32, device="cuda")
    pl = torch.zeros((B, cfg["vocab"]), dtype=torch.float32, device="cuda")
    for t in range(40):
        eng.ar_step(i32(np.arange(B)), i32(last), T, seed, step, out, pl)
        eng.sync()
        xo, po = out.cpu().numpy(), pl.cpu().numpy()
        for b in range(B):
            ref = oracle.forward_seq(target, okv[b], [last[b]], P - 1 + t)[0]
            status, rel, own = check_ar(po[b], int(xo[b]), ref, 5e-3, T, (seed, step, b, P - 1 + t))
            assert status == "ok"
            last[b] = int(xo[b])
    assert np.array_equal(kv_len.cpu().numpy(), np.full(B, P - 1 + 40))
    eng.close()


@pytest.mark.parametrize("gamma,T", [(1, 1.0), (7, 1.0), (4, 0.6), (4, 1.7), (2, 0.35)])
def test_tiny_fp32_sd_matches_oracle_over_gamma_and_temperature(gamma, T):
    """The SD path at the shortest draft, a long draft, and away from T = 1
    (logits scaled by 1/T in the draft draws, the accept test, the residual
    and bonus draws): every decision of a short rollout of the tiny fp32 model
    against the oracle."""
    cfg, run = synth.TINY, synth.TINY_RUN
    say("tiny fp32 SD", gamma, T)
    seed = 40 + gamma
    W = synth.make_weights(cfg, seed, "cpu")
    prompt = synth.make_tokens(run["B"], run["prompt"], cfg["vocab"], seed)
    eng, *_, st = run_rollout(cfg, W, prompt, run["B"], run["prompt"] + 24, gamma, T, seed, 5, tol=5e-3, n_steps=8)
    say("stats", st)
    assert st["checked"] >= 3 * run["B"] and st["exempt"] == 0
    eng.close()


SMALL_GQA = dict(name="small-gqa-bf16", n_layers=2, hidden=512, n_q=4, n_kv=2, head_dim=128, ffn=1024,
                 vocab=2048, dtype="bf16", rope_theta=500000.0, rms_eps=1e-5)


@pytest.mark.parametrize("ctx_fill", [0, 300, 1100], ids=["prefill", "random-context", "long-context"])
def test_small_bf16_sd_matches_oracle(ctx_fill):
    cfg = SMALL_GQA
    say("small bf16 SD", ctx_fill)
    B, P, gamma, T, seed = 8, 40, 4, 1.0, 6
    W = synth.make_weights(cfg, seed, "cpu")
    prompt = synth.make_tokens(B, P, cfg["vocab"], seed)
    eng, kv, okv, o_len, st = run_rollout(cfg, W, prompt, B, P + 24, gamma, T, seed, 11, tol=2e-2,
                                          ctx_fill=ctx_fill, n_steps=4)
    say("stats", st)
    assert st["checked"] == 4 * B and st["exempt"] <= 1
    check_cache(cfg, kv, okv, o_len, 2e-2)
    eng.close()


@pytest.mark.parametrize("gamma,T", [(3, 0.7), (6, 1.4)])
def test_small_bf16_sd_matches_oracle_away_from_unit_temperature(gamma, T):
    """The bf16 path (int4 drafter, GQA, head_dim 128) at other draft lengths
    and temperatures, after 300 positions of random context."""
    cfg = SMALL_GQA
    say("small bf16 SD", gamma, T)
    B, P, seed = 8, 40, 16
    W = synth.make_weights(cfg, seed, "cpu")
    prompt = synth.make_tokens(B, P, cfg["vocab"], seed)
    eng, *_, st = run_rollout(cfg, W, prompt, B, P + 24, gamma, T, seed, 13, tol=2e-2, ctx_fill=300, n_steps=3)
    say("stats", st)
    assert st["checked"] >= 2 * B and st["exempt"] <= 1
    eng.close()


@pytest.mark.parametrize("B", [16, 48])
def test_small_bf16_sd_verify_rows_in_one_tile(B):
    """Batches whose verify forward has 64 < B (gamma + 1) <= 320 rows: the
    projections and the LM head take the LDS-tiled GEMMs (split K for the
    narrow ones)."""
    cfg = SMALL_GQA
    say("small bf16 SD, B", B)
    P, gamma, T, seed = 24, 4, 1.0, 12
    W = synth.make_weights(cfg, seed, "cpu")
    prompt = synth.make_tokens(B, P, cfg["vocab"], seed)
    eng, *_, st = run_rollout(cfg, W, prompt, B, P + 12, gamma, T, seed, 5, tol=2e-2, ctx_fill=150, n_steps=2)
    say("stats", st)
    assert st["checked"] == 2 * B and st["exempt"] <= 1
    eng.close()


@pytest.mark.parametrize("B", [96, 130])
def test_small_bf16_sd_batches_past_one_m_tile(B):
    """Batches of more than 64 sequences: the drafter GEMM runs two or three
    64-row m-tiles (a ragged last one at 130), and the verify forward has 480
    and 650 rows, so its GEMMs take several tiles and the LM head of each draft
    step takes the LDS-tiled kernel."""
    cfg = SMALL_GQA
    say("small bf16 SD, B", B)
    P, gamma, T, seed = 24, 4, 1.0, 19
    W = synth.make_weights(cfg, seed, "cpu")
    prompt = synth.make_tokens(B, P, cfg["vocab"], seed)
    eng, *_, st = run_rollout(cfg, W, prompt, B, P + 12, gamma, T, seed, 9, tol=2e-2, ctx_fill=150, n_steps=2)
    say("stats", st)
    assert st["checked"] == 2 * B and st["exempt"] <= 1
    eng.close()


@pytest.mark.parametrize("B,fmt", [(1, "w4"), (3, "w4"), (2, "w4a"), (4, "w8")])
def test_small_bf16_sd_few_sequences(B, fmt):
    """The tail of a batch: a few sequences (drafter GEMMs with one 32-row
    tile mostly empty), in every drafter format."""
    cfg = SMALL_GQA
    say("small bf16 SD, few sequences", B, fmt)
    P, gamma, T, seed = 24, 4, 1.0, 14
    W = synth.make_weights(cfg, seed, "cpu")
    prompt = synth.make_tokens(B, P, cfg["vocab"], seed)
    eng, *_, st = run_rollout(cfg, W, prompt, B, P + 16, gamma, T, seed, 7, tol=2e-2, ctx_fill=260, n_steps=4,
                              fmt=fmt)
    say("stats", st)
    assert st["checked"] >= 2 * B and st["exempt"] <= 1
    eng.close()


@pytest.mark.parametrize("fmt", ["w4a", "w8"])
def test_tiny_fp32_sd_with_other_drafter_formats(fmt):
    """The asymmetric-int4 and int8 drafters: every decision of a short
    rollout of the fp32 decoder."""
    cfg, run = synth.TINY, synth.TINY_RUN
    say("tiny fp32 SD rollout", fmt)
    W = synth.make_weights(cfg, run["seed"], "cpu")
    prompt = synth.make_tokens(run["B"], run["prompt"], cfg["vocab"], run["seed"])
    eng, *_, st = run_rollout(cfg, W, prompt, run["B"], run["prompt"] + 24, run["gamma"], run["T"], run["seed"], 3,
                              tol=5e-3, fmt=fmt)
    say("stats", st)
    assert st["exempt"] == 0 and st["checked"] >= 8
    eng.close()


@pytest.mark.parametrize("fmt", ["w4a", "w8"])
def test_small_bf16_sd_with_other_drafter_formats(fmt):
    """The same for the bf16 GQA decoder over random context (the MFMA
    drafter GEMM with split K)."""
    cfg = SMALL_GQA
    say("small bf16 SD", fmt)
    B, P, gamma, T, seed = 8, 40, 4, 1.0, 6
    W = synth.make_weights(cfg, seed, "cpu")
    prompt = synth.make_tokens(B, P, cfg["vocab"], seed)
    eng, *_, st = run_rollout(cfg, W, prompt, B, P + 24, gamma, T, seed, 11, tol=2e-2, ctx_fill=300, n_steps=4,
                              fmt=fmt)
    say("stats", st)
    assert st["checked"] == 4 * B and st["exempt"] <= 1
    eng.close()


@pytest.mark.parametrize("cfg,page,tol", [(SMALL_GQA, 32, 2e-2), (SMALL_GQA, 64, 2e-2), (synth.TINY, 32, 5e-3)],
                         ids=["bf16-p32", "bf16-p64", "f32-p32"])
def test_paged_cache_rollout_matches_oracle(cfg, page, tol):
    """The whole rollout on a paged cache (pages handed out in shuffled order):
    every step against the oracle, and the cache after the rollout."""
    say("paged SD rollout", cfg["name"], page)
    B, P, gamma, T, seed = 6, 40, 4, 1.0, 23
    W = synth.make_weights(cfg, seed, "cpu")
    prompt = synth.make_tokens(B, P, cfg["vocab"], seed)
    eng, kv, okv, o_len, st = run_rollout(cfg, W, prompt, B, P + 24, gamma, T, seed, 4, tol=tol, ctx_fill=230,
                                          n_steps=4, page=page)
    say("stats", st)
    assert st["checked"] == 4 * B and st["exempt"] <= 1
    check_cache(cfg, kv, okv, o_len, tol)
    eng.close()


@pytest.mark.parametrize("cfg,tol", [(SMALL_GQA, 2e-2), (synth.TINY, 5e-3)], ids=["bf16", "f32"])
def test_graph_replayed_rollout_matches_oracle(cfg, tol):
    """Every step after the first is a replay of one captured HIP graph (the
    step reads its positions from kv_len on the device): each replay against
    the oracle."""
    say("graph SD rollout", cfg["name"])
    B, P, gamma, T, seed = 4, 40, 4, 1.0, 29
    W = synth.make_weights(cfg, seed, "cpu")
    prompt = synth.make_tokens(B, P, cfg["vocab"], seed)
    eng, kv, okv, o_len, st = run_rollout(cfg, W, prompt, B, P + 200, gamma, T, seed, 6, tol=tol, ctx_fill=120,
                                          n_steps=6, graph=True)
    say("stats", st)
    assert st["checked"] == 6 * B and st["exempt"] <= 1
    check_cache(cfg, kv, okv, o_len, tol)
    eng.close()


def test_poisoned_rollback_changes_nothing_but_the_discarded_span():
    """kv_rollback with the debug poison on overwrites the discarded drafts'
    KV with NaN: the rollout must be token for token the one without poison,
    match the oracle at every step, and leave NaN just past kv_len where the
    last step rejected a draft."""
    cfg = SMALL_GQA
    say("poisoned rollback")
    B, P, gamma, T, seed = 6, 40, 4, 1.0, 31
    W = synth.make_weights(cfg, seed, "cpu")
    prompt = synth.make_tokens(B, P, cfg["vocab"], seed)
    runs = {}
    for poison in (False, True):
        eng, kv, okv, o_len, st = run_rollout(cfg, W, prompt, B, P + 24, gamma, T, seed, 8, tol=2e-2,
                                              ctx_fill=100, n_steps=4, poison=poison)
        say("poison", poison, st)
        assert st["checked"] == 4 * B and st["exempt"] <= 1
        kd, vd = kv.dense()
        runs[poison] = (list(o_len), kd.float().cpu(), vd.float().cpu())
        eng.close()
    assert runs[False][0] == runs[True][0]
    for b, n in enumerate(runs[True][0]):
        for t in (1, 2):
            clean, dirty = runs[False][t], runs[True][t]
            assert torch.equal(clean[:, b, :, :n], dirty[:, b, :, :n]), b     # live KV identical
            assert not torch.isnan(clean[:, b, :, n:]).any()
        # the last step wrote gamma + 1 positions from its start; those past the new kv_len are poisoned
        assert torch.isnan(runs[True][1][:, b, :, n]).all(), b


def test_small_bf16_long_prefill_then_ar():
    """One sequence prefilled in chunks of 40 tokens (80 query rows per
    attention work-group slice set), then AR steps: logits, tokens and cache
    against the oracle."""
    cfg = SMALL_GQA
    say("small bf16 long prefill + AR")
    P, T, seed, step = 97, 1.0, 8, 2
    W = synth.make_weights(cfg, seed, "cpu")
    prompt = synth.make_tokens(1, P, cfg["vocab"], seed)
    eng, k, v, kv_len = make_engine(cfg, [w.cuda() for w in W], 8, 160, 4)
    target, _ = oracle_models(cfg, host_bits(W))
    okv = oracle.KV(cfg, 160)
    slot = 5
    eng.prefill(i32([slot]), prompt[:, :P - 1].cuda())
    oracle.forward_seq(target, okv, prompt[0, :P - 1].numpy(), 0, want_logits=False)
    eng.sync()
    kd = k[:, slot, :, : P - 1].float().cpu().numpy()
    vd = v[:, slot, :, : P - 1].float().cpu().numpy()
    assert np.abs(kd - okv.k[:, :, : P - 1]).max() <= 2e-2 * np.abs(okv.k[:, :, : P - 1]).max()
    assert np.abs(vd - okv.v[:, :, : P - 1]).max() <= 2e-2 * np.abs(okv.v[:, :, : P - 1]).max()
    last = int(prompt[0, P - 1])
    out = torch.zeros(1, dtype=torch.int32, device="cuda")
    pl = torch.zeros((1, cfg["vocab"]), dtype=torch.float32, device="cuda")
    for t in range(6):
        eng.ar_step(i32([slot]), i32([last]), T, seed, step, out, pl)
        eng.sync()
        ref = oracle.forward_seq(target, okv, [last], P - 1 + t)[0]
        status, rel, own = check_ar(pl.cpu().numpy()[0], int(out.cpu()[0]), ref, 2e-2, T, (seed, step, slot, P - 1 + t))
        assert status == "ok"
        last = int(out.cpu()[0])
    eng.close()
