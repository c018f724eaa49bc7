"""GPU parity of the paged-cache attention where a wave reads more than 128
blocks of one chunk.

On a paged cache each wave of k_attn_mfma holds the page ids of its next 128
blocks of 32 positions in two registers and reloads them when a block leaves
that window; a missing page of the wave's range is reported (ERR_PAGE) at
the reload.  With 64 sequences and 8 KV heads a launch has 512 work-groups,
so each sequence is one chunk, and its four waves take every fourth block:
a context above 16480 positions makes every wave reload its window once.
A verify over such contexts (page size 32, shuffled pages) must give the
same logits and the same cache bit for bit as the dense cache, match the
oracle on sampled sequences, and report a missing page that only the second
window reaches; with one query head per KV head (one query tile) and with
four (two tiles, whose next block and its page are set up in the middle of
the block).
"""
import numpy as np
import pytest
import torch

import oracle
from paper_2606_18967_amd import sdrl, synth

from gpu_common import DeviceKV, host_bits, i32, oracle_kv_from_device, oracle_models, say
from test_gpu_attention_chunks import _chunk_bounds

pytestmark = pytest.mark.gpu

WIDE = dict(name="wide-kv-bf16", n_layers=2, hidden=1024, n_q=8, n_kv=8, head_dim=128, ffn=1024, vocab=512,
            dtype="bf16", rope_theta=500000.0, rms_eps=1e-5)
# four query heads per KV head: 20 query rows per KV head at gamma 4, two
# 16-row tiles, the kernel whose next block (and page) is set up mid-block
WIDE_G4 = dict(WIDE, name="wide-kv-gqa4-bf16", n_q=32)
PAGE, WINDOW = 32, 128


@pytest.mark.parametrize("cfg", [WIDE, WIDE_G4], ids=["1tile", "2tiles"])
def test_paged_verify_past_the_page_window_matches_dense_and_oracle(cfg):
    gamma, seed, tol = 4, 41, 2e-2
    B = 64
    # ragged: most contexts past the window of every wave, a few short ones
    lens = [3000 + 7 * b if b % 16 == 5 else 16500 + (53 * b) % 190 for b in range(B)]
    max_ctx = max(lens) + gamma + 8
    assert all(not _chunk_bounds(cfg, B, gamma + 1, max_ctx, kl + gamma + 1) for kl in lens)   # one chunk each
    clen = [((kl + gamma + 1) + 31) & ~31 for kl in lens]
    assert sum(c > 96 + 32 * 4 * WINDOW for c in clen) >= B - 4     # wave 3 of these reaches block 128
    say("paged verify past the page window", B, min(lens), max(lens))
    W = [w.cuda() for w in synth.make_weights(cfg, seed, "cpu")]
    engs, kvs = [], []
    for page in (0, PAGE):
        eng = sdrl.Engine(cfg, B, max_ctx, gamma)
        eng.bind_weights(W)
        kv = DeviceKV(eng, max_ctx, page, seed)
        kv.fill_context(max(lens), seed + 100)
        kv.kv_len.copy_(i32(lens))
        eng.refresh_drafter()
        engs.append(eng)
        kvs.append(kv)
    torch.cuda.synchronize()
    kd0, vd0 = kvs[0].dense()
    okv = {b: oracle_kv_from_device(cfg, kd0, vd0, b, lens[b], max_ctx) for b in (3, 21)}
    V = cfg["vocab"]
    toks = synth.make_tokens(B, gamma + 1, V, seed + 1)
    ps = []
    for eng in engs:
        p = torch.zeros((B, gamma + 1, V), dtype=torch.float32, device="cuda")
        eng.verify(i32(range(B)), toks[:, 0].cuda().contiguous(), toks[:, 1:].cuda().contiguous(), gamma, p)
        eng.sync()
        ps.append(p)
    # the same arithmetic over the same values: identical logits and caches
    assert torch.equal(ps[0], ps[1])
    kp, vp = kvs[1].dense()
    assert torch.equal(kp, kvs[0].k) and torch.equal(vp, kvs[0].v)
    del kp, vp
    target, _ = oracle_models(cfg, host_bits(W))
    pd = ps[1].cpu().numpy()
    for b, ob in okv.items():
        ol = oracle.forward_seq(target, ob, toks[b].numpy(), lens[b])
        for j in range(gamma + 1):
            assert np.abs(pd[b, j] - ol[j]).max() <= tol * np.abs(ol[j]).max(), (b, j)
    engs[0].close()

    # a missing page that wave 2 of sequence 3 reaches at its block 128
    eng, kv = engs[1], kvs[1]
    lp = (64 + 32 * 4 * WINDOW) // PAGE
    assert (lp + 1) * PAGE <= lens[3]
    kv.kv_len.copy_(i32(lens))
    kv.table[3, lp] = kv.table.numel() + 5
    p = torch.zeros((B, gamma + 1, V), dtype=torch.float32, device="cuda")
    eng.verify(i32(range(B)), toks[:, 0].cuda().contiguous(), toks[:, 1:].cuda().contiguous(), gamma, p)
    with pytest.raises(RuntimeError, match="block-table"):
        eng.sync()
    eng.sync()                                 # the flag was cleared by the report
    eng.close()
