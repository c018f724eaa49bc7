"""Helpers shared by the GPU tests: engine set-up from seeded inputs, the
oracle twin of the same model, and the rollout harness that grows sequences
on the device and checks every step against the oracle."""
from __future__ import annotations

import sys

import numpy as np
import torch

import oracle
from oracle.parity import check_step, forced_step_logits
from paper_2606_18967_amd import sdrl, synth


def say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


def host_bits(tensors):
    return [synth.to_numpy_bits(t) for t in tensors]


def oracle_models(cfg, W_host, fmt="w4"):
    kind = oracle.BF16 if cfg["dtype"] == "bf16" else oracle.F32
    target = oracle.Model(cfg, W_host, kind)
    drafter = oracle.make_drafter(cfg, W_host, kind, fmt=fmt)
    return target, drafter


def make_engine(cfg, W_dev, max_slots, max_ctx, max_gamma, fmt="w4"):
    eng = sdrl.Engine(cfg, max_slots, max_ctx, max_gamma)
    eng.bind_weights(W_dev)
    k, v, kv_len = eng.alloc_kv()
    eng.bind_kv(k, v, kv_len)
    eng.refresh_drafter(fmt=fmt)
    return eng, k, v, kv_len


def i32(x, dev="cuda"):
    return torch.as_tensor(np.asarray(x, dtype=np.int32), device=dev)


def gather_pages(pool, table, max_ctx):
    """Dense [L][slots][n_kv][max_ctx][d] copy of a paged pool."""
    B, pps = table.shape
    P = pool.shape[3]
    g = pool[table.long()]                                 # [B][pps][L][n_kv][P][d]
    g = g.permute(2, 0, 3, 1, 4, 5).reshape(pool.shape[1], B, pool.shape[2], pps * P, pool.shape[4])
    return g[:, :, :, :max_ctx].contiguous()


def scatter_pages(pool, table, dense):
    """Writes a dense [L][slots][n_kv][C][d] cache into the pages of a pool."""
    B, pps = table.shape
    P = pool.shape[3]
    L, _, H, C, D = dense.shape
    pad = torch.zeros((L, B, H, pps * P, D), dtype=dense.dtype, device=dense.device)
    pad[:, :, :, :C] = dense
    pool[table.long()] = pad.reshape(L, B, H, pps, P, D).permute(1, 3, 0, 2, 4, 5)


class DeviceKV:
    """The device cache of an engine, dense or paged (pages of `page`
    positions in shuffled order), with a dense view for the checks."""

    def __init__(self, eng, cap, page=0, seed=0):
        self.eng, self.cap, self.page = eng, cap, page
        if page:
            B = eng.max_slots
            pps = (cap + page - 1) // page
            n_pages = B * pps + 2
            rng = np.random.default_rng(seed + 77)
            self.table = torch.as_tensor(rng.permutation(n_pages)[: B * pps].reshape(B, pps).astype(np.int32),
                                         device="cuda")
            self.k, self.v, self.kv_len = eng.alloc_kv_paged(n_pages, page)
            eng.bind_kv_paged(self.k, self.v, self.table, self.kv_len)
        else:
            self.k, self.v, self.kv_len = eng.alloc_kv()
            eng.bind_kv(self.k, self.v, self.kv_len)

    def fill_context(self, S, seed):
        """Random N(0, 1) context in positions [0, S) of every slot."""
        if not self.page:
            synth.fill_kv_context(self.k, self.v, S, seed=seed)
        else:
            kd = torch.zeros(self.eng.kv_shape(), dtype=self.eng.wdtype, device="cuda")
            vd = torch.zeros_like(kd)
            synth.fill_kv_context(kd, vd, S, seed=seed)
            scatter_pages(self.k, self.table, kd)
            scatter_pages(self.v, self.table, vd)
        self.kv_len.fill_(S)

    def dense(self):
        if not self.page:
            return self.k, self.v
        return gather_pages(self.k, self.table, self.cap), gather_pages(self.v, self.table, self.cap)


def oracle_kv_from_device(cfg, k, v, slot, upto, cap):
    """Oracle cache of one slot holding the device cache's first `upto`
    positions (used only for random context drawn by the seeded generator
    before any kernel ran)."""
    kv = oracle.KV(cfg, cap)
    kk = k[:, slot, :, :upto, :].float().cpu().numpy().astype(np.float64)
    vv = v[:, slot, :, :upto, :].float().cpu().numpy().astype(np.float64)
    kv.k[:, :, :upto, :] = kk
    kv.v[:, :, :upto, :] = vv
    return kv


def step_arrays(bufs, i):
    n = int(bufs["n_emit"][i])
    return dict(draft=bufs["draft"][i], q=bufs["q"][i], q_stats=bufs["q_stats"][i], p=bufs["p"][i],
                out=bufs["out"][i], n_emit=n)


def host_bufs(b: sdrl.SDBuffers):
    return dict(draft=b.draft_tok.cpu().numpy(), q=b.q_logits.cpu().numpy(), q_stats=b.q_stats.cpu().numpy(),
                p=b.p_logits.cpu().numpy(), out=b.out_tok.cpu().numpy(), n_emit=b.n_emit.cpu().numpy())


class Tally:
    """Counts of checked steps, exempt decisions, emitted tokens, the worst
    relative logit error, and how often the oracle's decisions on its own
    logits agreed with the device's."""

    def __init__(self):
        self.d = dict(checked=0, exempt=0, emitted=0, steps=0, worst=0.0, own_draws=0, draws=0, own_accept=0)

    def add(self, info, gamma):
        d = self.d
        d["checked"] += 1
        d["exempt"] += info["exempt"]
        d["worst"] = max(d["worst"], info["worst"])
        d["own_draws"] += info["own_draws"]
        d["draws"] += gamma
        d["own_accept"] += int(info["own_accept"])

    def __getitem__(self, k):
        return self.d[k]

    def __repr__(self):
        return repr(self.d)


def check_invariants(dv, gamma):
    n = dv["n_emit"]
    assert 1 <= n <= gamma + 1
    assert np.array_equal(dv["out"][: n - 1], dv["draft"][: n - 1])    # accepted prefix of the draft
    assert np.all(dv["out"][n:] == -1)


def run_rollout(cfg, W, prompt, B, ctx_target, gamma, T, seed, step, tol, ctx_fill=0, n_steps=None, fmt="w4",
                page=0, graph=False, poison=False, compare=None):
    """Grows B sequences with SD on the device and checks every step of every
    compared sequence (all by default) against the oracle: decisions on the
    device's own logits, logits against the oracle teacher-forced onto the
    device's tokens (oracle.parity.check_step).  No sequence is ever dropped.

    page > 0 binds a paged cache of that page size; graph=True runs every
    step after the first as a replay of one captured HIP graph (all B
    sequences stay active); poison=True turns the discarded-KV poison on."""
    P = prompt.shape[1]
    cap = ctx_fill + ctx_target + gamma + 2
    Wd = [w.cuda() for w in W]
    eng = sdrl.Engine(cfg, B, cap, gamma)
    eng.bind_weights(Wd)
    kv = DeviceKV(eng, cap, page, seed)
    eng.refresh_drafter(fmt=fmt)
    if poison:
        eng.set_debug(poison=True)
    Wh = host_bits(W)
    target, drafter = oracle_models(cfg, Wh, fmt)
    if ctx_fill:
        kv.fill_context(ctx_fill, seed + 100)
        torch.cuda.synchronize()
        kd, vd = kv.dense()
        okv = [oracle_kv_from_device(cfg, kd, vd, b, ctx_fill, cap) for b in range(B)]
    else:
        okv = [oracle.KV(cfg, cap) for _ in range(B)]
    slots_all = i32(np.arange(B))
    eng.prefill(slots_all, prompt[:, :P - 1].cuda())
    for b in range(B):
        oracle.forward_seq(target, okv[b], prompt[b, :P - 1].numpy(), ctx_fill, want_logits=False)
    o_len = [ctx_fill + P - 1] * B
    last = [int(x) for x in prompt[:, P - 1]]
    total = [P] * B
    compare = set(range(B)) if compare is None else set(compare)
    st = Tally()
    it = 0
    g = None
    bufs = sdrl.SDBuffers(eng, B, gamma) if graph else None
    last_dev = i32(last) if graph else None
    while any(t < ctx_target for t in total) and (n_steps is None or it < n_steps):
        it += 1
        active = [b for b in range(B) if total[b] < ctx_target]
        if graph:
            assert len(active) == B, "graph rollouts keep every sequence active"
            if g is None:
                sdrl.sd_step(eng, bufs, slots_all, last_dev, T, seed, step)
                last_dev.copy_(bufs.next_tok)
                torch.cuda.synchronize()
                g = sdrl.StepGraph(eng, bufs, slots_all, last_dev, T, seed, step)
            else:
                g.replay()
        else:
            bufs = sdrl.SDBuffers(eng, len(active), gamma)
            sdrl.sd_step(eng, bufs, i32(active), i32([last[b] for b in active]), T, seed, step)
        eng.sync()
        h = host_bufs(bufs)
        for i, b in enumerate(active):
            dv = step_arrays(h, i)
            check_invariants(dv, gamma)
            n = dv["n_emit"]
            if b in compare:
                q_ref, p_ref = forced_step_logits(target, drafter, okv[b], o_len[b], last[b], dv["draft"])
                info = check_step(dv, q_ref, p_ref, tol, T, (seed, step, b, o_len[b]))
                st.add(info, gamma)
                if info["exempt"]:
                    say("exempt", b, info)
            o_len[b] += n
            last[b] = int(dv["out"][n - 1])
            total[b] += n
            st.d["emitted"] += n
        st.d["steps"] += 1
    kl = kv.kv_len.cpu().numpy()
    for b in range(B):
        assert kl[b] == o_len[b], (b, kl[b], o_len[b])
    return eng, kv, okv, o_len, st


def check_cache(cfg, kv, okv, o_len, tol, slots=None):
    """Clean target KV up to kv_len of each slot against the oracle's."""
    kd, vd = kv.dense()
    for b in (range(len(o_len)) if slots is None else slots):
        n = o_len[b]
        k = kd[:, b, :, :n].float().cpu().numpy()
        v = vd[:, b, :, :n].float().cpu().numpy()
        assert np.abs(k - okv[b].k[:, :, :n]).max() <= tol * np.abs(okv[b].k[:, :, :n]).max(), b
        assert np.abs(v - okv[b].v[:, :, :n]).max() <= tol * np.abs(okv[b].v[:, :, :n]).max(), b
