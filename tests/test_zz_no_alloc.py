"""sd_accept_noalloc (the rejection sampler with no engine and no device
allocation, its scratch in the library's static per-GPU array) against the
engine's sd_accept on the same logits, uniforms and cache lengths: tokens,
n_emit and next tokens identical, on two calls in a row, the second smaller
(the static scratch keeps the first call's contents), and sizes beyond the
scratch refused on the host."""
import numpy as np
import pytest
import torch

from paper_2606_18967_amd import sdrl, synth

from gpu_common import i32, make_engine, say

pytestmark = pytest.mark.gpu


def _case(eng_cfg, B, gamma, V, seed):
    rng = np.random.default_rng(seed)
    q = (rng.standard_normal((B, gamma, V)) * 2).astype(np.float32)
    p = np.concatenate([q, q[:, -1:]], 1) + rng.standard_normal((B, gamma + 1, V)).astype(np.float32) * 0.4
    draft = rng.integers(0, V, (B, gamma)).astype(np.int32)
    return q, p.astype(np.float32), draft


@pytest.mark.parametrize("first,second", [((48, 4, 128256), (5, 2, 1024)), ((16, 7, 152064), (3, 1, 64))])
def test_accept_noalloc_equals_accept(first, second):
    max_slots = 64
    outs = []
    for call, (B, gamma, V) in enumerate((first, second)):
        say("accept_noalloc call", call, "B", B, "gamma", gamma, "V", V)
        cfg = dict(name="acc", n_layers=1, hidden=128, n_q=2, n_kv=1, head_dim=64, ffn=128, vocab=V, dtype="f32",
                   rope_theta=10000.0, rms_eps=1e-5)
        W = [w.cuda() for w in synth.make_weights(cfg, 1, "cpu")]
        eng, k, v, kv_len = make_engine(cfg, W, max_slots, 2048, gamma)
        rng = np.random.default_rng(V + B)
        kv_len.copy_(i32(rng.integers(0, 1500, max_slots)))
        slots = i32(rng.permutation(max_slots)[:B])
        q, p, draft = _case(cfg, B, gamma, V, B * 7 + gamma)
        qd, pd, dd = torch.tensor(q, device="cuda"), torch.tensor(p, device="cuda"), i32(draft)
        # q_stats as the sampler records them: (max, lse) of q / T
        T = 0.9
        qs = torch.stack([qd.max(-1).values / T, torch.logsumexp(qd.double() / T, -1).float()], -1).contiguous()
        res = []
        for noalloc in (False, True):
            out = torch.full((B, gamma + 1), 7, dtype=torch.int32, device="cuda")
            n_emit = torch.full((B,), 7, dtype=torch.int32, device="cuda")
            nxt = torch.full((B,), 7, dtype=torch.int32, device="cuda")
            if noalloc:
                sdrl.accept_noalloc(slots, kv_len, dd, qd, qs, pd, gamma, T, 13, 5 + call, out, n_emit, nxt)
            else:
                eng.accept(slots, dd, qd, qs, pd, gamma, T, 13, 5 + call, out, n_emit, nxt)
            torch.cuda.synchronize()
            res.append((out.cpu(), n_emit.cpu(), nxt.cpu()))
        eng.sync()
        for a, b in zip(*res):
            assert torch.equal(a, b), call
        n = res[1][1].numpy()
        assert ((n >= 1) & (n <= gamma + 1)).all()
        outs.append(res[1])
        eng.close()


def test_accept_noalloc_refuses_sizes_beyond_its_scratch():
    """B = 1024 sequences, gamma = 15 and vocab 152064 need about 1.25M
    scratch floats, more than the 2^20 the array holds: refused on the host
    before anything is launched (so one-element buffers stand in)."""
    import ctypes as C
    one_i = torch.zeros(1, dtype=torch.int32, device="cuda")
    one_f = torch.zeros(2, dtype=torch.float32, device="cuda")
    ip, fp = C.c_void_p(one_i.data_ptr()), C.c_void_p(one_f.data_ptr())
    st = sdrl.lib().sd_accept_noalloc(1024, 152064, ip, ip, 1, ip, fp, fp, fp, 15, 1.0, sdrl.Rng(0, 0), ip, ip, ip,
                                      sdrl._stream())
    assert st == sdrl.SD_E_INVAL
    assert "scratch" in sdrl.lib().sd_last_error().decode()
    torch.cuda.synchronize()
