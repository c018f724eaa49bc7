"""Helpers shared by the GPU tests: engine set-up from seeded inputs and the
oracle twin of the same model."""
from __future__ import annotations

import sys

import numpy as np
import torch

import oracle
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
    return dict(draft=bufs["draft"][i], q=bufs["q"][i], p=bufs["p"][i], out=bufs["out"][i], n_emit=n)


def host_bufs(b: sdrl.SDBuffers):
    return dict(draft=b.draft_tok.cpu().numpy(), q=b.q_logits.cpu().numpy(), p=b.p_logits.cpu().numpy(),
                out=b.out_tok.cpu().numpy(), n_emit=b.n_emit.cpu().numpy())
