"""GPU parity of the verify attention over every query-tile count.

The bf16 attention kernel takes a KV head's (n_q / n_kv) * (gamma + 1) query
rows in 16-row tiles, one to four per work-group (k_attn_mfma<D, MQ>), with
two K/V register sets at one and three tiles and one set at two and four
(where the next block's loads, and on a paged cache its page lookup, go out
in the middle of the block).
On a decoder with four query heads per KV head a verify at gamma = 3, 7, 11
and 15 has 16, 32, 48 and 64 query rows per KV head: one, two, three and
four tiles.  Each verify runs after 613-1017 positions of random context
(two or three attention chunks with four sequences); every row's logits and
the new cache rows are checked against the oracle's forward over the same
tokens, on a dense cache and on shuffled pages of 64 positions, at head
sizes 128 and 64.
"""
import numpy as np
import pytest
import torch

import oracle
from paper_2606_18967_amd import sdrl, synth

from gpu_common import DeviceKV, host_bits, i32, oracle_kv_from_device, oracle_models, say

pytestmark = pytest.mark.gpu

# four query heads per KV head at the production head size
GQA4 = dict(name="gqa4-bf16", n_layers=2, hidden=512, n_q=4, n_kv=1, head_dim=128, ffn=1024, vocab=1024,
            dtype="bf16", rope_theta=500000.0, rms_eps=1e-5)
# the same at the other head size the kernel is built for
GQA4_D64 = dict(GQA4, name="gqa4-d64-bf16", head_dim=64)


@pytest.mark.parametrize("cfg", [GQA4, GQA4_D64], ids=["d128", "d64"])
@pytest.mark.parametrize("page", [0, 64], ids=["dense", "paged"])
@pytest.mark.parametrize("gamma", [3, 7, 11, 15], ids=["1tile", "2tiles", "3tiles", "4tiles"])
def test_verify_every_query_tile_count_matches_oracle(gamma, page, cfg):
    seed, tol = 31 + gamma, 2e-2
    B = 4
    lens = [700, 613, 941, 1017]
    max_ctx = max(lens) + gamma + 8
    say("verify query tiles", gamma, (cfg["n_q"] // cfg["n_kv"]) * (gamma + 1), "rows per KV head, page", page)
    W = synth.make_weights(cfg, seed, "cpu")
    eng = sdrl.Engine(cfg, B, max_ctx, gamma)
    eng.bind_weights([w.cuda() for w in W])
    kv = DeviceKV(eng, max_ctx, page, seed)
    kv.fill_context(max(lens), seed + 100)
    kv.kv_len.copy_(i32(lens))
    eng.refresh_drafter()
    torch.cuda.synchronize()
    kd0, vd0 = kv.dense()
    okv = [oracle_kv_from_device(cfg, kd0, vd0, b, lens[b], max_ctx) for b in range(B)]
    V = cfg["vocab"]
    toks = synth.make_tokens(B, gamma + 1, V, seed + 1)
    p = torch.zeros((B, gamma + 1, V), dtype=torch.float32, device="cuda")
    eng.verify(i32(range(B)), toks[:, 0].cuda().contiguous(), toks[:, 1:].cuda().contiguous(), gamma, p)
    eng.sync()
    kd, vd = kv.dense()
    target, _ = oracle_models(cfg, host_bits(W))
    pd = p.cpu().numpy()
    for b, kl in enumerate(lens):
        ol = oracle.forward_seq(target, okv[b], toks[b].numpy(), kl)
        for j in range(gamma + 1):
            assert np.abs(pd[b, j] - ol[j]).max() <= tol * np.abs(ol[j]).max(), (b, j)
        end = kl + gamma + 1
        ok, ov = okv[b].k[:, :, kl:end], okv[b].v[:, :, kl:end]
        assert np.abs(kd[:, b, :, kl:end].float().cpu().numpy() - ok).max() <= tol * np.abs(ok).max(), b
        assert np.abs(vd[:, b, :, kl:end].float().cpu().numpy() - ov).max() <= tol * np.abs(ov).max(), b
    eng.close()
