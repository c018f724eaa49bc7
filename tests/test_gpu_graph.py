"""A whole SD step captured as a HIP graph (through torch) and replayed:
every replay must give exactly what the same step gives when its calls are
made one by one (same kernels in the same order on the same data), with
eager work and synchronisations between the replays."""
import numpy as np
import pytest
import torch

from paper_2606_18967_amd import sdrl, synth

from gpu_common import make_engine, say

pytestmark = pytest.mark.gpu

CFG = dict(name="graph-bf16", n_layers=2, hidden=512, n_q=4, n_kv=2, head_dim=128, ffn=1024, vocab=2048,
           dtype="bf16", rope_theta=500000.0, rms_eps=1e-5)


def _setup(W, B, S, gamma, seed):
    eng, k, v, kv_len = make_engine(CFG, W, B, S + 8 * (gamma + 1) + 8, gamma)
    synth.fill_kv_context(k, v, S, seed=seed + 100)
    kv_len.fill_(S)
    last = synth.make_tokens(B, 1, CFG["vocab"], seed + 7)[:, 0].cuda().contiguous()
    return eng, k, kv_len, last


@pytest.mark.parametrize("B", [1, 8])
def test_graph_replay_equals_eager_steps(B):
    say("graph replay", B)
    S, gamma, T, seed, step = 300, 4, 1.0, 3, 9
    W = [w.cuda() for w in synth.make_weights(CFG, seed, "cpu")]
    slots = torch.arange(B, dtype=torch.int32, device="cuda").flip(0).contiguous()
    ea, ka, la, lasta = _setup(W, B, S, gamma, seed)
    eb, kb, lb, lastb = _setup(W, B, S, gamma, seed)
    ba, bb = sdrl.SDBuffers(ea, B, gamma), sdrl.SDBuffers(eb, B, gamma)
    # one eager step on both (loads every kernel), then capture on b
    for e, b, last in ((ea, ba, lasta), (eb, bb, lastb)):
        sdrl.sd_step(e, b, slots, last, T, seed, step)
        last.copy_(b.next_tok)
    torch.cuda.synchronize()
    g = sdrl.StepGraph(eb, bb, slots, lastb, T, seed, step)
    torch.cuda.synchronize()
    assert torch.equal(lb, la)                # capturing ran nothing
    for it in range(4):
        sdrl.sd_step(ea, ba, slots, lasta, T, seed, step)
        lasta.copy_(ba.next_tok)
        g.replay()
        _ = torch.ones(1000, device="cuda").sum()                 # eager work between replays
        torch.cuda.synchronize()
        ea.sync()
        eb.sync()
        for name in ("draft_tok", "q_logits", "q_stats", "p_logits", "out_tok", "n_emit", "next_tok"):
            assert torch.equal(getattr(ba, name), getattr(bb, name)), (it, name)
        assert torch.equal(la, lb) and torch.equal(lasta, lastb), it
    assert torch.equal(ka, kb)                                   # same KV written
    ea.close()
    eb.close()
