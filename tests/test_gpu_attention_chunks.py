"""GPU parity of the attention's RoPE and new-row cache write where the new
rows straddle a context chunk.

With a bf16 cache the attention kernel itself rotates its query rows and
writes its KV head's new K (rotated) and V rows of its own context chunk
before reading them (k_attn_mfma).  The new rows are the last of a
sequence's context, and chunks are at least 512 positions long, so they
cross a chunk start only in long contexts whose last chunk is short; here
each sequence's cached length (about 7.7k) puts a chunk start 1, 2, 3 or 4
positions into the gamma + 1 = 5 positions a verify writes: two work-groups
of every KV head each write their part, and the query rows read rows both of
them wrote.  The verify logits of every row and the new cache rows are
checked against the oracle's forward over the same tokens (positions
0 .. kv_len - 1 are the same random context on both sides), on a dense and
on a paged cache.
"""
import numpy as np
import pytest
import torch

import oracle
from paper_2606_18967_amd import sdrl, synth

from gpu_common import DeviceKV, host_bits, i32, oracle_kv_from_device, oracle_models, say
from test_gpu_e2e import SMALL_GQA

pytestmark = pytest.mark.gpu

# the launcher's chunking (kernels_model.hip: about 512 work-groups per launch,
# chunks of at least 512 positions, in multiples of 32)
ATT_TARGET_WGS, ATT_MIN_CHUNK = 512, 512


def _chunk_bounds(cfg, B, n, max_ctx, ctx):
    """Start positions of the chunks after the first for one sequence of
    context length ctx, as the attention launch splits it."""
    QR = cfg["n_q"] // cfg["n_kv"] * n
    MQ = 4 if QR > 48 else (QR + 15) // 16
    zs = -(-QR // (16 * MQ))
    want = -(-ATT_TARGET_WGS // (B * cfg["n_kv"] * zs))
    ch = -(-max_ctx // want)
    ch = (max(ch, ATT_MIN_CHUNK) + 31) & ~31
    nch = -(-ctx // ch)
    clen = (-(-ctx // nch) + 31) & ~31
    return [c * clen for c in range(1, nch) if c * clen < ctx]


def _straddling_lengths(cfg, B, gamma, max_ctx, lo, count):
    """The first `count` cached lengths >= lo whose gamma + 1 new positions
    cross a chunk start, at different offsets from it."""
    out, offsets = [], set()
    for kl in range(lo, max_ctx - gamma - 1):
        for b0 in _chunk_bounds(cfg, B, gamma + 1, max_ctx, kl + gamma + 1):
            off = b0 - kl
            if 0 < off <= gamma and off not in offsets:
                out.append(kl)
                offsets.add(off)
        if len(out) == count:
            return out
    raise AssertionError("no straddling length in range")


@pytest.mark.parametrize("page", [0, 64], ids=["dense", "paged"])
def test_verify_rows_across_a_chunk_boundary_match_oracle(page):
    cfg, gamma, seed, tol = SMALL_GQA, 4, 21, 2e-2
    B, max_ctx = 4, 9000          # chunks of 512 positions: a chunk starts inside the new rows at offsets 1-4
    lens = _straddling_lengths(cfg, B, gamma, max_ctx, 7000, B)
    say("verify across chunk boundaries", page, lens)
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
        kn = kd[:, b, :, kl:end].float().cpu().numpy()
        vn = vd[:, b, :, kl:end].float().cpu().numpy()
        ok, ov = okv[b].k[:, :, kl:end], okv[b].v[:, :, kl:end]
        assert np.abs(kn - ok).max() <= tol * np.abs(ok).max(), b
        assert np.abs(vn - ov).max() <= tol * np.abs(ov).max(), b
        # the cached context before the new rows is untouched
        assert torch.equal(kd[:, b, :, :kl], kd0[:, b, :, :kl]), b
    eng.close()
