"""GPU parity of the ragged prefill (sd_prefill_ragged) through the C ABI.

Prompts of different lengths, including empty and one-token prompts, are
cached in rounds of a common number of positions (the engine's row budget
split over the batch), through a permuted slot list and on top of a few
positions of random context.  Checked per sequence:

  - kv_len grows by exactly the prompt's length;
  - the cached K/V of every layer match the oracle's prefill of that
    sequence alone (within the cache tolerance of the model's precision);
  - positions past the new kv_len keep their previous contents bit for bit
    (padding rows are never cached), and token entries past a prompt's end
    are never read (they hold -1, which would raise a device token error);
  - with equal lengths the ragged prefill equals sd_prefill bit for bit;
  - a length outside [0, ld] is reported by sd_sync and leaves that sequence
    unchanged.
"""
import numpy as np
import pytest
import torch

import oracle
from paper_2606_18967_amd import sdrl, synth

from gpu_common import DeviceKV, host_bits, i32, oracle_kv_from_device, oracle_models, say
from test_gpu_e2e import SMALL_GQA

pytestmark = pytest.mark.gpu

LENS = [37, 1, 64, 0, 50, 13]
SLOTS = [3, 0, 5, 1, 4, 2]
CTX0 = 3                  # positions of random context before the prompts
SENTINEL = 7.0            # exact in bf16 and fp32


def _setup(cfg, seed, max_gamma=3):
    B, ld = len(LENS), max(LENS)
    cap = CTX0 + ld + 8
    W = synth.make_weights(cfg, seed, "cpu")
    eng = sdrl.Engine(cfg, B, cap, max_gamma)        # rows_max = B (max_gamma + 1): rounds of max_gamma + 1 positions
    eng.bind_weights([w.cuda() for w in W])
    kv = DeviceKV(eng, cap)
    kv.fill_context(CTX0, seed + 100)
    kv.k[:, :, :, CTX0:] = SENTINEL
    kv.v[:, :, :, CTX0:] = SENTINEL
    torch.cuda.synchronize()
    tokens = synth.make_tokens(B, ld, cfg["vocab"], seed + 1)
    for b, n in enumerate(LENS):
        tokens[b, n:] = -1                            # never read
    return W, eng, kv, cap, tokens


@pytest.mark.parametrize("cfg,tol", [(synth.TINY, 5e-3), (SMALL_GQA, 2e-2)], ids=["f32", "bf16"])
def test_ragged_prefill_matches_oracle(cfg, tol):
    say("ragged prefill", cfg["name"], LENS)
    W, eng, kv, cap, tokens = _setup(cfg, 12)
    k0 = [kv.k[:, s].clone() for s in SLOTS]
    eng.prefill_ragged(i32(SLOTS), tokens.cuda(), i32(LENS))
    eng.sync()
    kv_len = kv.kv_len.cpu().numpy()
    target, _ = oracle_models(cfg, host_bits(W))
    for b, (s, n) in enumerate(zip(SLOTS, LENS)):
        assert kv_len[s] == CTX0 + n, (b, kv_len[s])
        okv = oracle_kv_from_device(cfg, kv.k, kv.v, s, CTX0, cap)
        if n:
            oracle.forward_seq(target, okv, tokens[b, :n].numpy(), CTX0, want_logits=False)
        end = CTX0 + n
        kd = kv.k[:, s, :, :end].float().cpu().numpy()
        vd = kv.v[:, s, :, :end].float().cpu().numpy()
        assert np.abs(kd - okv.k[:, :, :end]).max() <= tol * np.abs(okv.k[:, :, :end]).max(), b
        assert np.abs(vd - okv.v[:, :, :end]).max() <= tol * np.abs(okv.v[:, :, :end]).max(), b
        assert torch.equal(kv.k[:, s, :, end:], k0[b][:, :, end:]), b
        assert (kv.v[:, s, :, end:] == SENTINEL).all(), b
    eng.close()


def test_ragged_prefill_with_equal_lengths_equals_prefill():
    cfg = SMALL_GQA
    say("ragged prefill, equal lengths")
    B, n, seed = 4, 29, 13
    W = synth.make_weights(cfg, seed, "cpu")
    tokens = synth.make_tokens(B, n, cfg["vocab"], seed).cuda()
    caches = []
    for ragged in (False, True):
        eng = sdrl.Engine(cfg, B, n + 8, 3)
        eng.bind_weights([w.cuda() for w in W])
        kv = DeviceKV(eng, n + 8)
        kv.k.zero_()
        kv.v.zero_()
        kv.kv_len.zero_()
        if ragged:
            eng.prefill_ragged(i32(range(B)), tokens, i32([n] * B))
        else:
            eng.prefill(i32(range(B)), tokens)
        eng.sync()
        caches.append((kv.k.clone(), kv.v.clone(), kv.kv_len.clone()))
        eng.close()
    for a, b in zip(*caches):
        assert torch.equal(a, b)


def test_ragged_prefill_reports_a_length_past_the_row_width():
    cfg = SMALL_GQA
    say("ragged prefill, bad length")
    W, eng, kv, cap, tokens = _setup(cfg, 14)
    ld = tokens.shape[1]
    bad = list(LENS)
    bad[2] = ld + 1
    with pytest.raises(sdrl.SDError, match="prefill length"):
        eng.prefill_ragged(i32(SLOTS), tokens.cuda(), i32(bad))
        eng.sync()
    kv_len = kv.kv_len.cpu().numpy()
    for b, (s, n) in enumerate(zip(SLOTS, bad)):
        assert kv_len[s] == CTX0 + (0 if b == 2 else n), b
    assert (kv.k[:, SLOTS[2], :, CTX0:] == SENTINEL).all()
    eng.close()
