#!/usr/bin/env python3
"""Throughput of the quantized self-speculative decoding step on one MI355X.

Default workload: the 64-layer 32B-shaped decoder (hidden 5120, 40 query / 8
KV heads x 128, SwiGLU FFN 27648, vocab 152064, bf16, random init) with the
int4 group-128 drafter refreshed from it, B = 64 sequences with 8192
positions of random bf16 KV context each, gamma = 4, temperature 1.0 (the
largest shape that fits one GPU: B = 128 at 8192 positions needs ~360 GB).
--model L4_8B runs the 4-layer 8B-shaped stack at B = 64 and 2048 positions.
One step = gamma draft forwards + one verify forward over B*(gamma+1)
positions + accept + KV rollback + the host read of n_emit.  The metric is
accepted (emitted) tokens per second.

The JSON line also carries: the GPU's own AR decode rate at the same batch,
per-kernel-class times measured with HIP events on the launch stream, the
roofline record of the dominant kernel class, and the CPU oracle timed on
the host on a bounded sample of the same workload and extrapolated over the
layers.
"""
from __future__ import annotations

import argparse
import hashlib
import re
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
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--drafter", choices=("w4", "w4a", "w8"), default="w4",
                    help="drafter format: RTN int4 symmetric (default), int4 asymmetric, int8")
    ap.add_argument("--page-size", type=int, default=0,
                    help="bind a paged KV cache with pages of this many positions, shuffled (0: dense cache)")
    ap.add_argument("--graph", action="store_true",
                    help="time the SD steps as replays of one captured HIP graph")
    ap.add_argument("--batch", type=int, default=0, help="sequences (default: the workload's)")
    ap.add_argument("--context", type=int, default=0, help="cached positions per sequence (default: the workload's)")
    ap.add_argument("--gamma", type=int, default=0, help="draft length (default 4)")
    ap.add_argument("--model", choices=("L64_32B", "L4_8B", "L32_8B"), default="L64_32B",
                    help="decoder: the 32B shape with 64 layers (the default workload: B = 64, 8192 positions), "
                         "or the 8B shape with 4 or 32 layers (B = 64, 2048 positions)")
    ap.add_argument("--quiet", action="store_true")
    ap.add_argument("--copy-calibration", action="store_true",
                    help="only run a plain 1 GiB device copy (counter calibration)")
    ap.add_argument("--ingest-pmc", nargs=4, metavar=("FETCH_CSV", "WRITE_CSV", "COPY_FETCH_CSV", "COPY_WRITE_CSV"),
                    help="write profiles/traffic.json from rocprofv3 --pmc outputs")
    return ap.parse_args()


def log(args, *a):
    if not args.quiet:
        print(*a, file=sys.stderr, flush=True)


# source files each timing class's kernel is built from (a change to any of
# them voids the committed counter readings for that class)
SOURCES_OF_CLASS = {
    "attn_decode": ("common.h", "kernels.h", "kernels_model.hip"),
    "attn_verify": ("common.h", "kernels.h", "kernels_model.hip"),
    "int4_proj": ("common.h", "kernels.h", "kernels_q4.hip"),
    "bf16_proj": ("common.h", "kernels.h", "kernels_gemm.hip"),
    "lm_head": ("common.h", "kernels.h", "kernels_gemm.hip"),
}


def _code_only(text):
    """Source text with comments removed and whitespace collapsed, so that
    only a change to the code itself changes the hash."""
    text = re.sub(r"/\*.*?\*/", " ", text, flags=re.S)
    text = re.sub(r"//[^\n]*", " ", text)
    return " ".join(text.split())


def kernel_sources_hash(files=None):
    h = hashlib.sha256()
    csrc = os.path.join(ROOT, "paper_2606_18967_amd", "csrc")
    for f in sorted(files or os.listdir(csrc)):
        with open(os.path.join(csrc, f), encoding="utf-8") as fh:
            h.update(f.encode() + _code_only(fh.read()).encode())
    return h.hexdigest()[:16]


def workload_key(model, B, S, gamma, drafter, page):
    return f"{model} B={B} S={S} gamma={gamma} {drafter} page={page}"


# the workload the committed counter runs time (bench.py's defaults)
DEFAULT_WORKLOAD = workload_key("L64_32B", 64, 8192, 4, "w4", 0)
METRIC = "accepted tokens/s per GPU per SD step; draft/verify HBM GB/s & MFMA % of peak"
RUNS = {"L4_8B": "L4_8B_RUN", "L32_8B": "L32_8B_RUN", "L64_32B": "L64_32B_RUN"}
WORKLOAD_NAMES = {"L4_8B": "8B-shaped decoder, 4 layers", "L32_8B": "8B-shaped decoder, 32 layers",
                  "L64_32B": "32B-shaped decoder, 64 layers"}

def measured_traffic(kind: str, workload: str = DEFAULT_WORKLOAD):
    """HBM bytes per launch from committed rocprofv3 counter runs, or None if
    they were taken on another workload or the kernel's sources changed since."""
    path = os.path.join(ROOT, "profiles", "traffic.json")
    try:
        with open(path) as fh:
            rec = json.load(fh)
    except (OSError, ValueError):
        return None
    if rec.get("workload") != workload:
        return None
    d = rec.get("detail", {}).get(kind)
    if not d or d.get("sources") != kernel_sources_hash(SOURCES_OF_CLASS[kind]):
        return None
    return d.get("bytes")


# the kernel each timing class brackets (bf16 KV cache, head_dim 128, M = 64 drafter rows, 320 verify rows)
KERNEL_OF_CLASS = {
    "attn_decode": "k_attn_mfma<128, 1, false>",
    "attn_verify": "k_attn_mfma<128, 2, false>",
    "int4_proj": "k_gemm_q4<2, 0, false> (qkv, o, down; gate/up runs unsplit as the SwiGLU variant <2, 0, true> "
                 "where N allows)",
    "bf16_proj": "k_gemm_dma<4, false> (qkv, o, down; gate/up runs as the SwiGLU variant <4, true> where N allows)",
    "lm_head": "k_gemm_dma64<false> (draft rows), k_gemm_dma<4, false> (verify rows)",
}
# the counter ingest keeps, per class, only the dispatches of its kernel
# launched by that class (work-group counts tell the verify LM head, 594
# 320x256 tiles at V = 152064, from the split projections, <= 240)
CLASS_WG_FILTER = {"bf16_proj": lambda wgs: wgs < 500, "lm_head": lambda wgs: wgs >= 500}


# bytes per quantized weight: codes + fp16 scale (+ zero point) per group of 128
DRAFTER_BYTES_PER_WEIGHT = {"w4": 0.5 + 2 / 128, "w4a": 0.5 + 3 / 128, "w8": 1 + 2 / 128}


def algorithmic_per_launch(cfg, B, gamma, ctx, drafter="w4"):
    """Bytes (HBM-bound classes) or FLOPs (MFMA-bound) one launch of each
    timing class must move or do, for a mean cached length ctx (kv_len at the
    start of the step): the sizes of what the operation reads and writes, not
    what the kernels happen to transfer."""
    H, V, d, nkv, nq, F = (cfg[x] for x in ("hidden", "vocab", "head_dim", "n_kv", "n_q", "ffn"))
    kv_pos = nkv * d * 2 * 2                 # K and V bytes per cached position per layer (bf16)
    qkv_row = (nq + 2 * nkv) * d * 4         # fp32 QKV projection row per token (RoPE is part of the attention)
    # draft j (1..gamma) attends kv_len + j positions; verify attends kv_len + gamma + 1 once for all rows;
    # each token's projection row is read and its new K/V row written
    attn_d = B * kv_pos * (ctx + (gamma + 1) / 2) + B * (qkv_row + kv_pos)
    attn_v = B * kv_pos * (ctx + gamma + 1) + B * (gamma + 1) * (qkv_row + kv_pos)
    w_layer = H * (nq + 2 * nkv) * d + nq * d * H + 3 * H * F          # projection weights per layer
    q4 = w_layer * DRAFTER_BYTES_PER_WEIGHT[drafter] / 4                # mean drafter launch (4 per layer)
    rows_v = B * (gamma + 1)
    proj_flops = 2 * rows_v * w_layer / 4                                 # mean verify projection launch
    lm = V * H * 2 + (gamma * B + rows_v) / (gamma + 1) * (H * 2 + V * 4)
    return {"attn_decode": ("hbm", attn_d), "attn_verify": ("hbm", attn_v), "int4_proj": ("hbm", q4),
            "bf16_proj": ("mfma", proj_flops), "lm_head": ("hbm", lm)}


COPY_BYTES = 1 << 30


def copy_calibration(reps: int = 8):
    """A plain device-to-device copy of COPY_BYTES (torch's copy kernel), for
    scaling the FETCH_SIZE / WRITE_SIZE counters to bytes."""
    import torch
    src = torch.ones(COPY_BYTES // 4, dtype=torch.float32, device="cuda")
    dst = torch.empty_like(src)
    for _ in range(reps):
        dst.copy_(src)
    torch.cuda.synchronize()
    print(json.dumps({"copy_bytes_per_launch": COPY_BYTES, "launches": reps}), flush=True)


def kernel_key(name):
    """'(anonymous namespace)::k_foo<128, 1>(args...)' -> 'k_foo<128,1>'."""
    i = name.find("(anonymous namespace)::")
    if i >= 0:
        name = name[i + len("(anonymous namespace)::"):]
    name = name.removeprefix("void ")
    out, depth = [], 0
    for ch in name:
        if ch == "(" and depth == 0:
            break
        depth += ch == "<"
        depth -= ch == ">"
        out.append(ch)
    return "".join(out).replace(" ", "")


def ingest_pmc(fetch_csv, write_csv, copy_fetch_csv, copy_write_csv, out_path):
    """Writes profiles/traffic.json from rocprofv3 --pmc counter_collection.csv
    files: the bench run's FETCH_SIZE and WRITE_SIZE (KiB per dispatch)
    averaged per kernel, scaled by what the same counters read for the
    COPY_BYTES copy (the kernel with the largest reading in the copy runs)."""
    import csv

    def per_kernel(path, counter, keep=None):
        acc = {}
        with open(path) as fh:
            for row in csv.DictReader(fh):
                if row.get("Counter_Name") != counter:
                    continue
                k = kernel_key(row["Kernel_Name"])
                wgs = int(row.get("Grid_Size", 0)) // max(1, int(row.get("Workgroup_Size", 1)))
                if keep and k in keep and not keep[k](wgs):
                    continue
                d = row.get("Dispatch_Id") or row.get("Correlation_Id")
                acc.setdefault(k, {})
                acc[k][d] = acc[k].get(d, 0.0) + float(row["Counter_Value"])
        return {k: (sum(v.values()) / len(v), len(v)) for k, v in acc.items()}

    def copy_factor(path, counter):
        name, (kib, _) = max(per_kernel(path, counter).items(), key=lambda kv: kv[1][0])
        return COPY_BYTES / (kib * 1024.0), name, kib

    ff, fname, fkib = copy_factor(copy_fetch_csv, "FETCH_SIZE")
    wf, wname, wkib = copy_factor(copy_write_csv, "WRITE_SIZE")
    fetch = {c: per_kernel(fetch_csv, "FETCH_SIZE", {kernel_key(KERNEL_OF_CLASS[c]): f})
             for c, f in CLASS_WG_FILTER.items()}
    write = {c: per_kernel(write_csv, "WRITE_SIZE", {kernel_key(KERNEL_OF_CLASS[c]): f})
             for c, f in CLASS_WG_FILTER.items()}
    fetch_all = per_kernel(fetch_csv, "FETCH_SIZE")
    write_all = per_kernel(write_csv, "WRITE_SIZE")
    per = {}
    for cls, kname in KERNEL_OF_CLASS.items():
        k = kernel_key(kname)
        fe, wr = (fetch[cls], write[cls]) if cls in CLASS_WG_FILTER else (fetch_all, write_all)
        if k not in fe or k not in wr:
            continue
        per[cls] = dict(kernel=k, fetch_bytes=fe[k][0] * 1024 * ff, write_bytes=wr[k][0] * 1024 * wf,
                        bytes=fe[k][0] * 1024 * ff + wr[k][0] * 1024 * wf, dispatches=fe[k][1],
                        sources=kernel_sources_hash(SOURCES_OF_CLASS[cls]))
    rec = {
           "workload": DEFAULT_WORKLOAD,
           "copy_calibration": {"bytes": COPY_BYTES, "fetch_kib": fkib, "write_kib": wkib, "fetch_factor": ff,
                                "write_factor": wf, "kernel": fname},
           "per_launch_bytes": {c: v["bytes"] for c, v in per.items()}, "detail": per}
    with open(out_path, "w") as fh:
        json.dump(rec, fh, indent=1)
    print(json.dumps(rec["per_launch_bytes"]))


def main():
    args = parse()
    if args.copy_calibration:
        copy_calibration()
        return
    if args.ingest_pmc:
        ingest_pmc(*args.ingest_pmc, os.path.join(ROOT, "profiles", "traffic.json"))
        return
    if args.gpus != 1:
        print("bench.py measures one GPU: the SD step has no multi-GPU path (data parallelism gives each GPU "
              "its own sequences, target, drafter and KV cache, with nothing exchanged per step). "
              "Run with --gpus 1.", file=sys.stderr)
        sys.exit(2)
    import numpy as np
    import torch

    from paper_2606_18967_amd import sdrl, synth

    cfg, run = getattr(synth, args.model), getattr(synth, RUNS[args.model])
    B, S, gamma, T, seed = run["B"], run["context"], run["gamma"], run["T"], run["seed"]
    B, S, gamma = args.batch or B, args.context or S, args.gamma or gamma
    n_steps, n_warm = args.steps, args.warmup
    # every timed SD step can advance a sequence by gamma + 1 positions
    max_ctx = S + (2 * n_steps + n_warm + 2) * (gamma + 1) + args.ar_steps + gamma + 2
    torch.cuda.set_device(0)
    dev = torch.device("cuda", 0)

    log(args, "weights ...")
    W = synth.make_weights(cfg, seed, dev)
    eng = sdrl.Engine(cfg, B, max_ctx, gamma)
    eng.bind_weights(W)
    if args.page_size:
        # paged cache: every sequence's pages drawn at random from one pool
        P = args.page_size
        pps = (max_ctx + P - 1) // P
        perm = torch.randperm(B * pps, generator=torch.Generator().manual_seed(seed + 3))
        table = perm.to(torch.int32).reshape(B, pps).to(dev).contiguous()
        k, v, kv_len = eng.alloc_kv_paged(B * pps, P)
        eng.bind_kv_paged(k, v, table, kv_len)
        L_, Hk, D_ = cfg["n_layers"], cfg["n_kv"], cfg["head_dim"]
        g = torch.Generator(device=dev).manual_seed(seed + 100)
        for j in range((S + P - 1) // P):           # random N(0, 1) context in the first S positions
            n = min(P, S - j * P)
            for t in (k, v):
                t[table[:, j].long(), :, :, :n] = torch.randn((B, L_, Hk, n, D_), generator=g, device=dev).to(t.dtype)
    else:
        k, v, kv_len = eng.alloc_kv()
        eng.bind_kv(k, v, kv_len)
        synth.fill_kv_context(k, v, S, seed + 100)
    kv_len.fill_(S)
    torch.cuda.synchronize()
    # drafter refresh (the per-training-step Prep): once to load the kernels,
    # then timed with events on the stream it runs on
    qbuf = eng.refresh_drafter(fmt=args.drafter)
    ev0, ev1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    ev0.record()
    eng.refresh_drafter(qbuf, fmt=args.drafter)
    ev1.record()
    torch.cuda.synchronize()
    prep_ms = ev0.elapsed_time(ev1)

    slots = torch.arange(B, dtype=torch.int32, device=dev)
    bufs = sdrl.SDBuffers(eng, B, gamma)
    tok = [synth.make_tokens(B, 1, cfg["vocab"], seed + 7)[:, 0].to(dev).contiguous(),
           torch.zeros(B, dtype=torch.int32, device=dev)]
    first_tok = int(tok[0][0].item())
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
    eager_iter = sd_iter
    if args.graph:
        # the whole step as one HIP graph: fixed token buffer, kv_len advances on the device
        last_g = tok[state["it"] % 2].clone()
        graph = sdrl.StepGraph(eng, bufs, slots, last_g, T, seed, 1)

        def sd_iter():
            graph.replay()
            n = bufs.n_emit.cpu()
            state["it"] += 1
            return int(n.sum())

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
    if args.graph:
        tok[state["it"] % 2].copy_(last_g)
    for _ in range(n_steps):
        eager_iter()
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
    ctx_prof = 0.5 * (kv_before + kv_after)             # mean kv_len at the start of the profiled steps
    dom = max(classes, key=lambda c: classes[c]["ms_per_step"])
    algo = algorithmic_per_launch(cfg, B, gamma, ctx_prof, args.drafter)
    bound, amount = algo.get(dom, ("hbm", float("nan")))
    us = classes[dom]["us_per_launch"]
    if bound == "hbm":
        achieved, peak, unit = amount / (us * 1e-6) / 1e9, HBM_PEAK_GBS, "GB/s"
    else:
        achieved, peak, unit = amount / (us * 1e-6) / 1e12, BF16_PEAK_TFLOPS, "TFLOP/s"
    roof = dict(bound=bound, achieved=round(achieved, 1), peak=peak, unit=unit,
                frac=round(achieved / peak, 4),
                traffic=measured_traffic(dom, workload_key(args.model, B, S, gamma, args.drafter, args.page_size)),
                kernel=KERNEL_OF_CLASS.get(dom, dom), timing_class=dom,
                algorithmic_per_launch=amount, us_per_launch=round(us, 2))
    others = {}
    for name, (b, amt) in algo.items():
        u = classes[name]["us_per_launch"]
        if u > 0:
            others[name] = round(amt / (u * 1e-6) / (1e9 if b == "hbm" else 1e12), 1)

    # ---- CPU oracle on a bounded sample of the same workload
    cpu = None
    if not args.no_cpu_baseline and not args.page_size:
        cpu = cpu_baseline(args, cfg, W, k, v, S, gamma, T, seed, args.drafter, tau, first_tok)

    rec = {
        "metric": METRIC,
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
        "config": {"workload": WORKLOAD_NAMES[args.model] + ", bf16 target + "
                               + {"w4": "int4 g128", "w4a": "asymmetric int4 g128", "w8": "int8 g128"}[args.drafter]
                               + f" drafter, B={B}, KV context {S} (random N(0,1)), gamma={gamma}, T=1.0",
                   "drafter": args.drafter, "hip_graph": bool(args.graph), "kv_page_size": args.page_size,
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


def _cpu_model():
    try:
        with open("/proc/cpuinfo") as fh:
            for line in fh:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def cpu_baseline(args, cfg, W, k, v, S, gamma, T, seed, fmt, tau_gpu, tok):
    """The oracle (plain C, fp64 model arithmetic, OpenMP over projection
    rows) on the host, on a bounded sample of the same workload, extrapolated
    over the layers.

    All cores: one SD step of sequence 0 (gamma drafter forwards, the verify
    forward over gamma + 1 tokens, the accept) with the workload's first one
    and first two layers (same embedding, final norm and LM head, same KV
    context): T(L) = T(1) + (L - 1) (T(2) - T(1)).  One core: the drafter's
    and the target's one-token forwards at one and two layers, extrapolated
    the same way and composed into gamma drafter + (gamma + 1) target token
    forwards.  The value is the GPU's measured tokens per sequence per step
    over T(L): the oracle's throughput on the full model, by extrapolation."""
    import numpy as np

    import oracle
    from paper_2606_18967_amd import synth

    L = cfg["n_layers"]
    log(args, "cpu baseline: host copies of the first two layers ...")
    idx = list(range(3)) + list(range(3, 15))
    Wh = [synth.to_numpy_bits(W[i]) for i in idx]
    models = {}
    for nl in (1, 2):
        c = dict(cfg, n_layers=nl)
        t = oracle.Model(c, Wh[:3 + 6 * nl], oracle.BF16)
        d = oracle.make_drafter(c, Wh[:3 + 6 * nl], oracle.BF16, fmt=fmt)
        models[nl] = (c, t, d)
    cap = S + gamma + 2
    kk = k[:2, 0, :, :S].float().cpu().numpy()
    vv = v[:2, 0, :, :S].float().cpu().numpy()

    def fresh_kv(nl):
        kv = oracle.KV(models[nl][0], cap)
        kv.k[:, :, :S], kv.v[:, :, :S] = kk[:nl], vv[:nl]
        return kv

    oracle.set_threads(0)
    cores = oracle.get_threads()
    t_all = {}
    for nl in (1, 2):
        kv = fresh_kv(nl)
        t0 = time.perf_counter()
        oracle.sd_step_seq(models[nl][1], models[nl][2], kv, S, tok, gamma, T, seed, 1, 0)
        t_all[nl] = time.perf_counter() - t0
    step_all = t_all[1] + (L - 1) * (t_all[2] - t_all[1])
    oracle.set_threads(1)
    t_one = {}
    try:
        for nl in (1, 2):
            for which, m in (("draft", models[nl][2]), ("target", models[nl][1])):
                kv = fresh_kv(nl)
                t0 = time.perf_counter()
                oracle.forward_seq(m, kv, [tok], S)
                t_one[(which, nl)] = time.perf_counter() - t0
    finally:
        oracle.set_threads(0)
    ext = lambda w: t_one[(w, 1)] + (L - 1) * (t_one[(w, 2)] - t_one[(w, 1)])
    step_one = gamma * ext("draft") + (gamma + 1) * ext("target")
    sample_s = sum(t_all.values()) + sum(t_one.values())
    log(args, f"cpu baseline: {step_all:.1f} s per SD step per sequence on {cores} cores, {step_one:.1f} s on one, "
              f"by extrapolation to {L} layers ({sample_s:.1f} s measured)")
    return dict(value=round(tau_gpu / step_all, 5), unit="tokens/s", cores=cores, kind="oracle",
                sample=(f"extrapolation over the layers: one SD step (gamma={gamma}: {gamma} drafter forwards, a "
                        f"{gamma + 1}-token verify forward, accept) of one sequence with the workload's first 1 "
                        f"and 2 layers (same embedding, LM head and {S}-position KV context), "
                        f"T(L) = T(1) + (L-1)(T(2)-T(1)) at L={L}; tokens per step = the GPU's measured tau"),
                extrapolated=True, seconds_per_step=round(step_all, 3), measured_seconds=round(sample_s, 2),
                single_thread=dict(value=round(tau_gpu / step_one, 6), seconds_per_step=round(step_one, 3),
                                   sample="one-token drafter and target forwards at 1 and 2 layers, extrapolated "
                                          f"to {L} layers, composed into {gamma} drafter + {gamma + 1} target "
                                          "token forwards"),
                cpu_model=_cpu_model(), nproc=os.cpu_count())


if __name__ == "__main__":
    main()
