"""Full-size parity: the 4-layer 8B-shaped bf16 decoder (hidden 4096, 32/8
heads x 128, FFN 14336, vocab 128256) with B = 64 sequences, 2048 positions
of random KV context and gamma = 4 -- the launch configuration bench.py
times.  The device runs one SD step for all 64 sequences; the oracle redoes
the step for sampled sequences one by one (draft logits, verify logits,
draws and accept decisions), and the engine's invariants are checked for all
64 rows."""
import numpy as np
import pytest
import torch

import oracle
from oracle.parity import compare_step
from paper_2606_18967_amd import sdrl, synth

from gpu_common import host_bits, say

pytestmark = pytest.mark.gpu


def test_l4_8b_sd_step_matches_oracle_on_sampled_sequences():
    cfg, run = synth.L4_8B, synth.L4_8B_RUN
    B, S, gamma, T, seed, step = run["B"], run["context"], run["gamma"], run["T"], run["seed"], 1
    say("8B-shaped SD step: weights")
    dev = torch.device("cuda", 0)
    W = synth.make_weights(cfg, seed, dev)
    cap = S + gamma + 8
    eng = sdrl.Engine(cfg, B, cap, gamma)
    eng.bind_weights(W)
    k, v, kv_len = eng.alloc_kv()
    eng.bind_kv(k, v, kv_len)
    synth.fill_kv_context(k, v, S, seed + 100)
    kv_len.fill_(S)
    eng.refresh_drafter()
    slots = torch.arange(B, dtype=torch.int32, device=dev)
    last = synth.make_tokens(B, 1, cfg["vocab"], seed + 7)[:, 0].to(dev).contiguous()
    torch.cuda.synchronize()
    sample = [0, 37]
    ctx_host = {b: (k[:, b, :, :S].float().cpu().numpy(), v[:, b, :, :S].float().cpu().numpy()) for b in sample}
    say("8B-shaped SD step: device step")
    bufs = sdrl.SDBuffers(eng, B, gamma)
    sdrl.sd_step(eng, bufs, slots, last, T, seed, step)
    eng.sync()
    n_emit = bufs.n_emit.cpu().numpy()
    out = bufs.out_tok.cpu().numpy()
    draft = bufs.draft_tok.cpu().numpy()
    assert np.all((n_emit >= 1) & (n_emit <= gamma + 1))
    for b in range(B):
        assert np.array_equal(out[b, : n_emit[b] - 1], draft[b, : n_emit[b] - 1])
        assert np.all(out[b, n_emit[b]:] == -1)
    assert np.array_equal(kv_len.cpu().numpy(), S + n_emit)
    rows = {b: dict(draft=draft[b], q=bufs.q_logits[b].cpu().numpy(), p=bufs.p_logits[b].cpu().numpy(),
                    out=out[b], n_emit=int(n_emit[b])) for b in sample}
    lastn = last.cpu().numpy()
    del bufs
    say("8B-shaped SD step: oracle")
    Wh = host_bits(W)
    target = oracle.Model(cfg, Wh, oracle.BF16)
    drafter = oracle.make_drafter(cfg, Wh, oracle.BF16)
    for b in sample:
        kvb = oracle.KV(cfg, cap)
        kvb.k[:, :, :S], kvb.v[:, :, :S] = ctx_host[b]
        r = oracle.sd_step_seq(target, drafter, kvb, S, int(lastn[b]), gamma, T, seed, step, b)
        status, info = compare_step(r, rows[b], 2e-2, T, key=(seed, step, b, S))
        say("sequence", b, status, info, "n_emit", r["n_emit"], rows[b]["n_emit"])
        assert status in ("ok", "exempt")
    eng.close()


def test_32b_shaped_two_layer_sd_step_matches_oracle():
    """The 32B shape (hidden 5120, 40 query / 8 KV heads x 128 -- five query
    heads per KV head --, FFN 27648, vocab 152064) at two layers, B = 64,
    512 positions of context: the per-layer shapes of the 64-layer workload,
    checked against the oracle on two sampled sequences."""
    cfg = dict(synth.L64_32B, n_layers=2, name="32B-shape-2L")
    B, S, gamma, T, seed, step = 64, 512, 4, 1.0, 11, 1
    say("32B-shaped 2-layer SD step: weights")
    dev = torch.device("cuda", 0)
    W = synth.make_weights(cfg, seed, dev)
    cap = S + gamma + 8
    eng = sdrl.Engine(cfg, B, cap, gamma)
    eng.bind_weights(W)
    k, v, kv_len = eng.alloc_kv()
    eng.bind_kv(k, v, kv_len)
    synth.fill_kv_context(k, v, S, seed + 100)
    kv_len.fill_(S)
    eng.refresh_drafter()
    slots = torch.arange(B, dtype=torch.int32, device=dev)
    last = synth.make_tokens(B, 1, cfg["vocab"], seed + 7)[:, 0].to(dev).contiguous()
    torch.cuda.synchronize()
    sample = [5, 62]
    ctx_host = {b: (k[:, b, :, :S].float().cpu().numpy(), v[:, b, :, :S].float().cpu().numpy()) for b in sample}
    say("32B-shaped 2-layer SD step: device step")
    bufs = sdrl.SDBuffers(eng, B, gamma)
    sdrl.sd_step(eng, bufs, slots, last, T, seed, step)
    eng.sync()
    n_emit = bufs.n_emit.cpu().numpy()
    out = bufs.out_tok.cpu().numpy()
    draft = bufs.draft_tok.cpu().numpy()
    assert np.all((n_emit >= 1) & (n_emit <= gamma + 1))
    assert np.array_equal(kv_len.cpu().numpy(), S + n_emit)
    rows = {b: dict(draft=draft[b], q=bufs.q_logits[b].cpu().numpy(), p=bufs.p_logits[b].cpu().numpy(),
                    out=out[b], n_emit=int(n_emit[b])) for b in sample}
    lastn = last.cpu().numpy()
    del bufs
    say("32B-shaped 2-layer SD step: oracle")
    Wh = host_bits(W)
    target = oracle.Model(cfg, Wh, oracle.BF16)
    drafter = oracle.make_drafter(cfg, Wh, oracle.BF16)
    for b in sample:
        kvb = oracle.KV(cfg, cap)
        kvb.k[:, :, :S], kvb.v[:, :, :S] = ctx_host[b]
        r = oracle.sd_step_seq(target, drafter, kvb, S, int(lastn[b]), gamma, T, seed, step, b)
        status, info = compare_step(r, rows[b], 2e-2, T, key=(seed, step, b, S))
        say("sequence", b, status, info, "n_emit", r["n_emit"], rows[b]["n_emit"])
        assert status in ("ok", "exempt")
    eng.close()
