"""Paged KV cache (pages [L][n_kv][page_size][head_dim] named by a block
table) against the dense cache: with the same weights and the same context
scattered over shuffled pages, SD steps must give bit-identical tokens,
logits and cache contents (the same arithmetic, only the addressing
differs), for the MFMA attention (bf16) and the fp32 path, at page sizes 32
and 64.  A block-table entry outside the pool is skipped on the device and
reported by sd_sync."""
import numpy as np
import pytest
import torch

from paper_2606_18967_amd import sdrl, synth

from gpu_common import say

pytestmark = pytest.mark.gpu

GQA = dict(name="paged-bf16", n_layers=2, hidden=512, n_q=4, n_kv=2, head_dim=128, ffn=1024, vocab=2048,
           dtype="bf16", rope_theta=500000.0, rms_eps=1e-5)


def _engines(cfg, W, B, max_ctx, gamma, page, seed):
    dense = sdrl.Engine(cfg, B, max_ctx, gamma)
    dense.bind_weights(W)
    kd, vd, ld = dense.alloc_kv()
    dense.bind_kv(kd, vd, ld)
    dense.refresh_drafter()
    paged = sdrl.Engine(cfg, B, max_ctx, gamma)
    paged.bind_weights(W)
    pps = (max_ctx + page - 1) // page
    n_pages = B * pps + 3
    rng = np.random.default_rng(seed)
    table = torch.as_tensor(rng.permutation(n_pages)[: B * pps].reshape(B, pps).astype(np.int32), device="cuda")
    kp, vp, lp = paged.alloc_kv_paged(n_pages, page)
    paged.bind_kv_paged(kp, vp, table, lp)
    paged.refresh_drafter()
    return dense, (kd, vd, ld), paged, (kp, vp, lp, table)


def _gather(pool, table, max_ctx):
    """Dense [L][slots][n_kv][max_ctx][d] view of a paged pool."""
    B, pps = table.shape
    P = pool.shape[3]
    g = pool[table.long()]                                 # [B][pps][L][n_kv][P][d]
    g = g.permute(2, 0, 3, 1, 4, 5).reshape(pool.shape[1], B, pool.shape[2], pps * P, pool.shape[4])
    return g[:, :, :, :max_ctx].contiguous()


def _scatter(pool, table, dense):
    B, pps = table.shape
    P = pool.shape[3]
    L, _, H, C, D = dense.shape
    pad = torch.zeros((L, B, H, pps * P, D), dtype=dense.dtype, device=dense.device)
    pad[:, :, :, :C] = dense
    pool[table.long()] = pad.reshape(L, B, H, pps, P, D).permute(1, 3, 0, 2, 4, 5)


@pytest.mark.parametrize("cfg,page", [(GQA, 32), (GQA, 64), (synth.TINY, 32)], ids=["bf16-p32", "bf16-p64", "f32-p32"])
def test_paged_equals_dense(cfg, page):
    say("paged", cfg["name"], page)
    B, S, gamma, T, seed, step = 6, 203, 4, 1.0, 4, 2
    max_ctx = S + 4 * (gamma + 1) + 4
    W = [w.cuda() for w in synth.make_weights(cfg, seed, "cpu")]
    dense, (kd, vd, ld), paged, (kp, vp, lp, table) = _engines(cfg, W, B, max_ctx, gamma, page, seed)
    synth.fill_kv_context(kd, vd, S, seed=seed + 100)
    _scatter(kp, table, kd)
    _scatter(vp, table, vd)
    ld.fill_(S)
    lp.fill_(S)
    assert torch.equal(_gather(kp, table, max_ctx), kd)
    slots = torch.tensor([3, 0, 5, 1, 4, 2][:B], dtype=torch.int32, device="cuda")
    last_d = synth.make_tokens(B, 1, cfg["vocab"], seed + 7)[:, 0].cuda().contiguous()
    last_p = last_d.clone()
    bd, bp = sdrl.SDBuffers(dense, B, gamma), sdrl.SDBuffers(paged, B, gamma)
    for it in range(3):
        sdrl.sd_step(dense, bd, slots, last_d, T, seed, step)
        sdrl.sd_step(paged, bp, slots, last_p, T, seed, step)
        dense.sync()
        paged.sync()
        for name in ("draft_tok", "q_logits", "p_logits", "out_tok", "n_emit"):
            assert torch.equal(getattr(bd, name), getattr(bp, name)), (it, name)
        last_d.copy_(bd.next_tok)
        last_p.copy_(bp.next_tok)
    assert torch.equal(ld, lp)
    assert torch.equal(_gather(kp, table, max_ctx), kd)
    assert torch.equal(_gather(vp, table, max_ctx), vd)
    dense.close()
    paged.close()


def test_bad_block_table_entry_is_reported():
    cfg = GQA
    say("paged bad entry")
    B, S, gamma, seed = 2, 100, 2, 5
    max_ctx = S + 16
    W = [w.cuda() for w in synth.make_weights(cfg, seed, "cpu")]
    eng = sdrl.Engine(cfg, B, max_ctx, gamma)
    eng.bind_weights(W)
    page = 32
    pps = (max_ctx + page - 1) // page
    n_pages = B * pps
    table = torch.arange(n_pages, dtype=torch.int32, device="cuda").reshape(B, pps).contiguous()
    kp, vp, lp = eng.alloc_kv_paged(n_pages, page)
    eng.bind_kv_paged(kp, vp, table, lp)
    eng.refresh_drafter()
    lp.fill_(S)
    table[1, 1] = n_pages + 3                 # a page the pool does not have, inside slot 1's context
    slots = torch.tensor([0, 1], dtype=torch.int32, device="cuda")
    bufs = sdrl.SDBuffers(eng, B, gamma)
    last = torch.tensor([1, 2], dtype=torch.int32, device="cuda")
    eng.draft(slots, last, gamma, 1.0, seed, 1, bufs.draft_tok, bufs.q_logits, bufs.q_stats)
    with pytest.raises(RuntimeError, match="block-table"):
        eng.sync()
    eng.sync()                                 # the flag was cleared by the report
    eng.close()
