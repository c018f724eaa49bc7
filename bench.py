#!/usr/bin/env python3
"""Throughput of the quantized self-speculative decoding step on one MI355X.

Workload: the 8B-shaped decoder (4 layers, hidden 4096, 32 query / 8 KV heads
x 128, SwiGLU FFN 14336, vocab 128256, bf16, random init), int4 group-128
drafter refreshed from it, B = 64 sequences with 2048 positions of random
bf16 KV context each, gamma = 4, temperature 1.0.  One step = gamma draft
forwards + one verify forward over B*(gamma+1) positions + accept + KV
rollback + the host read of n_emit.  The metric is accepted (emitted)
tokens per second.

The JSON line also carries: the GPU's own AR decode rate at the same batch,
per-kernel-class times measured with HIP events on the launch stream, the
roofline record of the dominant kernel class, and the CPU oracle timed on
the host on a bounded sample of the same workload.
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0
BF16_PEAK_TFLOPS = 2500.0


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--ar-steps", type=int, default=20)
    ap.add_argument("--cpu-seqs", type=int, default=2, help="sequences in the oracle's CPU sample")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--quiet", action="store_true")
    return ap.parse_args()


def log(args, *a):
    if not args.quiet:
        print(*a, file=sys.stderr, flush=True)


def kernel_sources_hash():
    h = hashlib.sha256()
    csrc = os.path.join(ROOT, "paper_2606_18967_amd", "csrc")
    for f in sorted(os.listdir(csrc)):
        with open(os.path.join(csrc, f), "rb") as fh:
            h.update(f.encode() + fh.read())
    return h.hexdigest()[:16]


def measured_traffic(kind: str):
    """HBM bytes per launch from committed rocprofv3 counter runs, or None if
    the kernels changed since they were taken."""
    path = os.path.join(ROOT, "profiles", "traffic.json")
    try:
        with open(path) as fh:
            rec = json.load(fh)
    except (OSError, ValueError):
        return None
    if rec.get("sources") != kernel_sources_hash():
        return None
    return rec.get("per_launch_bytes", {}).get(kind)


def main():
    args = parse()
    if args.gpus != 1:
        print("bench.py measures one GPU: this build has no multi-GPU path (each GPU would run its own "
              "sequences independently; see DESIGN.md). Run with --gpus 1.", file=sys.stderr)
        sys.exit(2)
    import numpy as np
    import torch

    from paper_2606_18967_amd import sdrl, synth

    cfg, run = synth.L4_8B, synth.L4_8B_RUN
    B, S, gamma, T, seed = run["B"], run["context"], run["gamma"], run["T"], run["seed"]
    n_steps, n_warm = args.steps, args.warmup
    # every timed SD step can advance a sequence by gamma + 1 positions
    max_ctx = S + (2 * n_steps + n_warm + 2) * (gamma + 1) + args.ar_steps + gamma + 2
    torch.cuda.set_device(0)
    dev = torch.device("cuda", 0)

    log(args, "weights ...")
    W = synth.make_weights(cfg, seed, dev)
    eng = sdrl.Engine(cfg, B, max_ctx, gamma)
    eng.bind_weights(W)
    k, v, kv_len = eng.alloc_kv()
    eng.bind_kv(k, v, kv_len)
    synth.fill_kv_context(k, v, S, seed + 100)
    kv_len.fill_(S)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    qbuf = eng.refresh_drafter()
    torch.cuda.synchronize()
    prep_ms = (time.perf_counter() - t0) * 1e3

    slots = torch.arange(B, dtype=torch.int32, device=dev)
    bufs = sdrl.SDBuffers(eng, B, gamma)
    tok = [synth.make_tokens(B, 1, cfg["vocab"], seed + 7)[:, 0].to(dev).contiguous(),
           torch.zeros(B, dtype=torch.int32, device=dev)]
    state = dict(it=0, emitted=0)

    def sd_iter():
        i = state["it"]
        last, nxt = tok[i % 2], tok[(i + 1) % 2]
        eng.draft(slots, last, gamma, T, seed, 1, bufs.draft_tok, bufs.q_logits, bufs.q_stats)
        eng.verify(slots, last, bufs.draft_tok, gamma, bufs.p_logits)
        eng.accept(slots, bufs.draft_tok, bufs.q_logits, bufs.q_stats, bufs.p_logits, gamma, T, seed, 1,
                   bufs.out_tok, bufs.n_emit, nxt)
        eng.rollback(slots, bufs.n_emit)
        n = bufs.n_emit.cpu()            # the host needs n_emit every step
        state["it"] = i + 1
        return int(n.sum())

    log(args, "warmup ...")
    for _ in range(n_warm):
        sd_iter()
    eng.sync()

    # ---- timed region: K SD steps
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    emitted = 0
    for _ in range(n_steps):
        emitted += sd_iter()
    torch.cuda.synchronize()
    dt = time.perf_counter() - t0
    eng.sync()
    value = emitted / dt
    tau = emitted / (n_steps * B)
    ctx_mean = float(kv_len.float().mean().item())
    log(args, f"SD: {value:.0f} tok/s, {dt / n_steps * 1e3:.3f} ms/step, tau {tau:.3f}")

    # ---- the same steps again with per-kernel-class events on the launch stream
    kv_before = kv_len.float().mean().item()
    eng.timing(True)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(n_steps):
        sd_iter()
    torch.cuda.synchronize()
    dt_prof = time.perf_counter() - t0
    classes = {}
    for c, name in enumerate(sdrl.T_NAMES):
        ms, n = eng.timing_read(c)
        classes[name] = dict(ms_per_step=ms / n_steps, launches_per_step=n / n_steps,
                             us_per_launch=(ms / n * 1e3) if n else 0.0)
    eng.timing(False)
    kv_after = kv_len.float().mean().item()
    eng.sync()

    # ---- AR baseline at the same batch
    kv_len.fill_(S)
    out = torch.zeros(B, dtype=torch.int32, device=dev)
    pl = torch.zeros((B, cfg["vocab"]), dtype=torch.float32, device=dev)
    last = tok[0].clone()
    for _ in range(2):
        eng.ar_step(slots, last, T, seed, 2, out, pl)
        last, out = out, last
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(args.ar_steps):
        eng.ar_step(slots, last, T, seed, 2, out, pl)
        _ = out.cpu()
        last, out = out, last
    torch.cuda.synchronize()
    ar_dt = time.perf_counter() - t0
    eng.sync()
    ar_rate = B * args.ar_steps / ar_dt
    log(args, f"AR: {ar_rate:.0f} tok/s")

    # ---- roofline of the dominant kernel class
    H, V, d, nkv, nq, F, L = (cfg[x] for x in ("hidden", "vocab", "head_dim", "n_kv", "n_q", "ffn", "n_layers"))
    ctx_prof = 0.5 * (kv_before + kv_after)             # mean context during the profiled steps
    dom = max(classes, key=lambda c: classes[c]["ms_per_step"])
    # algorithmic bytes per launch ("Measurement")
    R_d, R_v = B, B * (gamma + 1)
    la = (gamma * L, L)  # attention launches: per draft forward and per verify
    kv_row = nkv * d * 2 * 2                          # K and V bytes per cached position (bf16)
    attn_bytes = B * kv_row * (ctx_prof + (gamma + 1) / 2) + (R_d * gamma + R_v) / sum(la) * (nq * d * 4 + nq * d * 2)
    q4_w = (H * (nq + 2 * nkv) * d + nq * d * H + 3 * H * F)     # weights per layer
    q4_bytes = (q4_w * 0.5 + q4_w / 128 * 2) / 4               # mean per projection launch (4 per layer)
    lm_bytes = V * H * 2 + (gamma * R_d + R_v) / (gamma + 1) * (H * 2 + V * 4)
    proj_flops = 2 * R_v * q4_w / 4
    algo = {"attention": ("hbm", attn_bytes), "int4_proj": ("hbm", q4_bytes), "lm_head": ("hbm", lm_bytes),
            "bf16_proj": ("mfma", proj_flops)}
    bound, amount = algo.get(dom, ("hbm", float("nan")))
    us = classes[dom]["us_per_launch"]
    if bound == "hbm":
        achieved, peak, unit = amount / (us * 1e-6) / 1e9, HBM_PEAK_GBS, "GB/s"
    else:
        achieved, peak, unit = amount / (us * 1e-6) / 1e12, BF16_PEAK_TFLOPS, "TFLOP/s"
    roof = dict(kernel=dom, bound=bound, achieved=round(achieved, 1), peak=peak, unit=unit,
                frac=round(achieved / peak, 4), traffic=measured_traffic(dom),
                algorithmic_per_launch=amount, us_per_launch=round(us, 2))
    others = {}
    for name, (b, amt) in algo.items():
        u = classes[name]["us_per_launch"]
        if u > 0:
            others[name] = round(amt / (u * 1e-6) / (1e9 if b == "hbm" else 1e12), 1)

    # ---- CPU oracle on a bounded sample of the same workload
    cpu = None
    if not args.no_cpu_baseline:
        cpu = cpu_baseline(args, cfg, W, k, v, S, gamma, T, seed)

    rec = {
        "metric": "accepted tokens/s per GPU per SD step",
        "value": round(value, 1),
        "unit": "tokens/s",
        "n_gpus": 1,
        "steps": n_steps,
        "warmup": n_warm,
        "ms_per_step": round(dt / n_steps * 1e3, 3),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic",
        "config": {"workload": "8B-shaped decoder, 4 layers, bf16 target + int4 g128 drafter, B=64, "
                               "KV context 2048 (random N(0,1)), gamma=4, T=1.0",
                   "batch": B, "context": S, "gamma": gamma, "temperature": T, "layers": L, "hidden": H,
                   "heads": f"{nq}q/{nkv}kv x {d}", "ffn": F, "vocab": V},
        "roofline": roof,
        "cpu_baseline": cpu,
        "tau": round(tau, 4),
        "alpha": round(sdrl.alpha_from_tau(tau, gamma), 4),
        "ar_tokens_per_s": round(ar_rate, 1),
        "sd_over_ar": round(value / ar_rate, 4),
        "mean_context": round(ctx_mean, 1),
        "drafter_refresh_ms": round(prep_ms, 2),
        "kernel_classes": classes,
        "achieved_by_class": others,
        "profiled_ms_per_step": round(dt_prof / n_steps * 1e3, 3),
    }
    print(json.dumps(rec), flush=True)


def cpu_baseline(args, cfg, W, k, v, S, gamma, T, seed):
    """The oracle (plain C, OpenMP over projection rows) on the host: one SD
    step for the first `cpu_seqs` sequences of the workload, from the same
    weights and KV context."""
    import numpy as np

    import oracle
    from paper_2606_18967_amd import synth

    log(args, "cpu baseline: copying weights to host ...")
    Wh = [synth.to_numpy_bits(w) for w in W]
    target = oracle.Model(cfg, Wh, oracle.BF16)
    drafter = oracle.make_drafter(cfg, Wh, oracle.BF16)
    cap = S + gamma + 2
    toks = synth.make_tokens(64, 1, cfg["vocab"], seed + 7)[:, 0].numpy()   # the workload's first tokens
    emitted, elapsed = 0, 0.0
    for b in range(args.cpu_seqs):
        kvb = oracle.KV(cfg, cap)
        kvb.k[:, :, :S] = k[:, b, :, :S].float().cpu().numpy()
        kvb.v[:, :, :S] = v[:, b, :, :S].float().cpu().numpy()
        t0 = time.perf_counter()
        r = oracle.sd_step_seq(target, drafter, kvb, S, int(toks[b]), gamma, T, seed, 1, b)
        elapsed += time.perf_counter() - t0
        emitted += r["n_emit"]
    threads = int(os.environ.get("OMP_NUM_THREADS", os.cpu_count() or 1))
    log(args, f"cpu baseline: {emitted} tokens in {elapsed:.2f}s")
    return dict(value=round(emitted / elapsed, 3), unit="tokens/s", cores=threads, kind="oracle",
                sample=f"one SD step (gamma={gamma}: {gamma} draft + {gamma + 1} verify token forwards, "
                       f"accept) for {args.cpu_seqs} of the 64 sequences, same weights and KV context",
                seconds=round(elapsed, 2), tokens=emitted)


if __name__ == "__main__":
    main()
