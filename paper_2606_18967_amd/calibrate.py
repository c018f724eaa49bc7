"""Calibration of the roofline cost model (Sec. 4.2) on this GPU and validation
of the SD toggle boundary (App. D.2, App. D.3).

The procedure follows App. D.2 in three stages:

1. F_eff from a dense-GEMM microbenchmark (the library's own bf16 kernels,
   ``sd_dense_gemm_bf16``).
2. A sweep over batch size B and context length S (and draft length gamma for
   verification) that times, with the engine's own kernels,
     - target decoding T_p: one AR step (target forward + sampling),
     - quantized-drafter decoding T_q: one draft step (gamma = 1),
     - verification T_V: the verify forward over gamma + 1 tokens plus the
       accept step and KV rollback,
   so that gamma T_q + T_V is the wall time of one SD step.
3. A two-step least-squares fit on log-time residuals: BW_eff, rho_kappa and
   c_T on the target sweep alone; then, with those fixed, eta_D, c_D and c_V
   on the drafter and verification sweeps.

Validation (App. D.3): for every sweep point and a block efficiency tau, the
model's predicted speedup tau T_p / (gamma T_q + T_V) is set against the one
the measured times give; the toggle's decision (speedup >= 1 + eps) agrees
when both fall on the same side.  tau is a parameter: random-init weights
have a fixed, low acceptance, so the measured tau of the synthetic model is
reported next to the taus the paper reports for trained policies.

Usage (one GPU):  python -m paper_2606_18967_amd.calibrate --out calib.json
"""
from __future__ import annotations

import argparse
import json
import math
import sys
import time

import numpy as np

from . import sdrl, synth

FIT_KEYS_TARGET = ("BW_eff", "rho_kappa", "c_T")
FIT_KEYS_DRAFT = ("eta_D", "c_D", "c_V")


# ----------------------------------------------------------------- fitting
def model_times(base: sdrl.CostModel, params: dict, B, S, gamma):
    """T_p, T_q, T_V of the cost model with `params` overriding base."""
    m = sdrl.CostModel()
    for f, _ in sdrl.CostModel._fields_:
        setattr(m, f, getattr(base, f))
    for k, v in params.items():
        setattr(m, k, v)
    return sdrl.cost_times(m, B, S, gamma)


def _lsq(fun, x0, lo, hi):
    from scipy.optimize import least_squares
    r = least_squares(fun, x0, bounds=(lo, hi), x_scale="jac", max_nfev=4000)
    return r.x, float(np.sqrt(np.mean(r.fun ** 2)))


def fit(base: sdrl.CostModel, samples: list[dict]):
    """Two-step fit of App. D.2 on samples {kind: 'p'|'q'|'v', B, S, gamma, t}.
    Parameters are fitted in log space (all positive); the residual is
    log(model) - log(measured).  Returns (params, rms_log_residual_p,
    rms_log_residual_qv)."""
    sp = [s for s in samples if s["kind"] == "p"]
    sqv = [s for s in samples if s["kind"] in ("q", "v")]
    if not sp or not sqv:
        raise ValueError("need target (p) and drafter/verify (q, v) samples")
    idx = {"p": 0, "q": 1, "v": 2}

    def res(keys, fixed, logx, pts):
        params = dict(fixed)
        params.update({k: math.exp(v) for k, v in zip(keys, logx)})
        out = []
        for s in pts:
            t = model_times(base, params, s["B"], s["S"], s["gamma"])[idx[s["kind"]]]
            out.append(math.log(t) - math.log(s["t"]))
        return np.array(out)

    # stage 1: BW_eff, rho_kappa, c_T from the target sweep
    t0 = min(s["t"] for s in sp)
    x0 = np.log([base.W_T / t0, 1.0, 1e-6])
    lo = np.log([1e9, 1e-3, 1e-12])
    hi = np.log([1e14, 10.0, 1e-1])
    x1, r1 = _lsq(lambda x: res(FIT_KEYS_TARGET, {}, x, sp), x0, lo, hi)
    p1 = {k: math.exp(v) for k, v in zip(FIT_KEYS_TARGET, x1)}
    # stage 2: eta_D, c_D, c_V with stage 1 fixed
    x0 = np.log([1.0, 1e-6, 1e-6])
    lo = np.log([1e-2, 1e-12, 1e-12])
    hi = np.log([100.0, 1e-1, 1e-1])
    x2, r2 = _lsq(lambda x: res(FIT_KEYS_DRAFT, p1, x, sqv), x0, lo, hi)
    p2 = {k: math.exp(v) for k, v in zip(FIT_KEYS_DRAFT, x2)}
    return {**p1, **p2}, r1, r2


def validate(base: sdrl.CostModel, params: dict, meas: dict, taus, eps=0.05):
    """Predicted vs measured speedup at each (B, S, gamma) with T_p, T_q, T_V
    measured and each tau; returns rows and the fraction of agreeing toggle
    decisions."""
    rows, agree, n = [], 0, 0
    for (B, S, gamma), t in sorted(meas.items()):
        tp_m, tq_m, tv_m = t
        tp, tq, tv = model_times(base, params, B, S, gamma)
        for tau in taus:
            if tau > gamma + 1:
                continue
            s_pred = tau * tp / (gamma * tq + tv)
            s_meas = tau * tp_m / (gamma * tq_m + tv_m)
            on_pred, on_meas = s_pred >= 1 + eps, s_meas >= 1 + eps
            agree += on_pred == on_meas
            n += 1
            rows.append(dict(B=B, S=S, gamma=gamma, tau=tau, pred=round(s_pred, 4), meas=round(s_meas, 4),
                             on_pred=bool(on_pred), on_meas=bool(on_meas)))
    return rows, (agree / n if n else float("nan"))


# -------------------------------------------------------------- measuring
def f_eff(n: int = 8192, reps: int = 10) -> float:
    """Effective dense bf16 throughput (FLOP/s) of the library's GEMM."""
    import torch
    dev = torch.device("cuda", 0)
    g = torch.Generator(device=dev).manual_seed(0)
    A = torch.randn(n, n, generator=g, device=dev).to(torch.bfloat16)
    W = torch.randn(n, n, generator=g, device=dev).to(torch.bfloat16)
    C = torch.empty(n, n, device=dev, dtype=torch.float32)
    for _ in range(2):
        sdrl.dense_gemm_bf16(A, W, C)
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    for _ in range(reps):
        sdrl.dense_gemm_bf16(A, W, C)
    e1.record()
    torch.cuda.synchronize()
    return 2.0 * n ** 3 * reps / (e0.elapsed_time(e1) * 1e-3)


class Sweep:
    """Times T_p, T_q, T_V with the engine's kernels on one model over a grid
    of (B, S, gamma).  KV context is random N(0, 1) (synth.fill_kv_context);
    kv_len is reset to S before each measurement."""

    def __init__(self, cfg: dict, Bmax: int, Smax: int, gmax: int, seed: int = 2, fmt: str = "w4"):
        import torch
        self.torch = torch
        self.cfg = cfg
        self.dev = torch.device("cuda", 0)
        self.W = synth.make_weights(cfg, seed, self.dev)
        self.eng = sdrl.Engine(cfg, Bmax, Smax + 12 * (gmax + 1) + 64, gmax)
        self.eng.bind_weights(self.W)
        self.k, self.v, self.kv_len = self.eng.alloc_kv()
        self.eng.bind_kv(self.k, self.v, self.kv_len)
        synth.fill_kv_context(self.k, self.v, Smax, seed + 100)
        self.qbuf = self.eng.refresh_drafter(fmt=fmt)
        self.seed = seed
        self.V = cfg["vocab"]

    def _time(self, fn, S, reps):
        torch = self.torch
        self.kv_len.fill_(S)
        fn()                                   # warm-up
        self.kv_len.fill_(S)
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        for _ in range(reps):
            fn()
        e1.record()
        torch.cuda.synchronize()
        self.eng.sync()
        return e0.elapsed_time(e1) * 1e-3 / reps

    def measure(self, B: int, S: int, gammas, reps: int = 8):
        """Returns {'p': T_p, 'q': T_q, ('v', gamma): T_V} in seconds."""
        torch = self.torch
        dev, V = self.dev, self.V
        slots = torch.arange(B, dtype=torch.int32, device=dev)
        last = synth.make_tokens(B, 1, V, self.seed + 7)[:, 0].to(dev).contiguous()
        out = torch.zeros(B, dtype=torch.int32, device=dev)
        pl = torch.empty((B, V), dtype=torch.float32, device=dev)
        res = {}
        res["p"] = self._time(lambda: self.eng.ar_step(slots, last, 1.0, self.seed, 1, out, pl), S, reps)
        b1 = sdrl.SDBuffers(self.eng, B, 1)
        res["q"] = self._time(lambda: self.eng.draft(slots, last, 1, 1.0, self.seed, 1, b1.draft_tok, b1.q_logits,
                                                     b1.q_stats), S, reps)
        del b1
        for g in gammas:
            bg = sdrl.SDBuffers(self.eng, B, g)
            self.kv_len.fill_(S)
            self.eng.draft(slots, last, g, 1.0, self.seed, 1, bg.draft_tok, bg.q_logits, bg.q_stats)

            def ver():
                self.eng.verify(slots, last, bg.draft_tok, g, bg.p_logits)
                self.eng.accept(slots, bg.draft_tok, bg.q_logits, bg.q_stats, bg.p_logits, g, 1.0, self.seed, 1,
                                bg.out_tok, bg.n_emit, bg.next_tok)
                self.eng.rollback(slots, bg.n_emit)
                self.kv_len.fill_(S)
            res[("v", g)] = self._time(ver, S, reps)
            del bg
        return res

    def measured_tau(self, B: int, S: int, gamma: int, steps: int = 10) -> float:
        """Mean tokens per SD step of the synthetic model at (B, S, gamma)."""
        torch = self.torch
        dev = self.dev
        slots = torch.arange(B, dtype=torch.int32, device=dev)
        last = synth.make_tokens(B, 1, self.V, self.seed + 7)[:, 0].to(dev).contiguous()
        bufs = sdrl.SDBuffers(self.eng, B, gamma)
        self.kv_len.fill_(S)
        emitted = 0
        for i in range(steps):
            sdrl.sd_step(self.eng, bufs, slots, last, 1.0, self.seed, 10 + i)
            last = bufs.next_tok.clone()
            emitted += int(bufs.n_emit.sum())
        self.eng.sync()
        return emitted / (steps * B)

    def set_drafter(self, fmt: str):
        self.qbuf = self.eng.refresh_drafter(fmt=fmt)

    def close(self):
        self.eng.close()


def drafter_tradeoff(cfg: dict, fmts=("w4", "w4a", "w8"), Bs=(1, 16, 64), S=2048, gamma=4, steps=10, reps=8,
                     log=print):
    """Latency against acceptance of the drafter formats (App. B.3, Table 4):
    per format and batch, the measured T_q / T_p, the model's tau and alpha
    at (B, S, gamma), and the SD speedup tau T_p / (gamma T_q + T_V) those
    measurements give; next to them the cost model's idealized T_q / T_p
    from bytes alone (weights at 16 bits, drafter projections at 4 or 8)."""
    sw = Sweep(cfg, max(Bs), S, gamma)
    rows = []
    for fmt in fmts:
        sw.set_drafter(fmt)
        bits = 8.0 if fmt == "w8" else 4.0
        ideal = sdrl.cost_init(cfg, drafter_bits=bits, BW_eff=1.0, F_eff=1e30)
        for B in Bs:
            r = sw.measure(B, S, [gamma], reps)
            tau = sw.measured_tau(B, S, gamma, steps)
            tp, tq, _ = sdrl.cost_times(ideal, B, S, gamma)
            row = dict(fmt=fmt, B=B, S=S, gamma=gamma, T_p=r["p"], T_q=r["q"], T_V=r[("v", gamma)],
                       tq_over_tp=r["q"] / r["p"], tq_over_tp_ideal=tq / tp, tau=tau,
                       alpha=sdrl.alpha_from_tau(min(tau, gamma + 1 - 1e-9), gamma),
                       speedup=tau * r["p"] / (gamma * r["q"] + r[("v", gamma)]))
            log(json.dumps(row))
            rows.append(row)
    sw.close()
    return rows


def run(cfg: dict, Bs, Ss, gammas, taus, eps=0.05, reps=8, log=print, fmt: str = "w4"):
    torch_started = time.time()
    F = f_eff()
    log(f"F_eff {F / 1e12:.0f} TFLOP/s")
    base = sdrl.cost_init(cfg)
    base.F_eff = F
    sw = Sweep(cfg, max(Bs), max(Ss), max(gammas), fmt=fmt)
    samples, meas = [], {}
    for S in Ss:
        for B in Bs:
            r = sw.measure(B, S, gammas, reps)
            samples.append(dict(kind="p", B=B, S=S, gamma=1, t=r["p"]))
            samples.append(dict(kind="q", B=B, S=S, gamma=1, t=r["q"]))
            for g in gammas:
                samples.append(dict(kind="v", B=B, S=S, gamma=g, t=r[("v", g)]))
                meas[(B, S, g)] = (r["p"], r["q"], r[("v", g)])
            log(f"B={B:4d} S={S:6d}  T_p {r['p'] * 1e3:8.3f} ms  T_q {r['q'] * 1e3:8.3f} ms  "
                + "  ".join(f"T_V(g={g}) {r[('v', g)] * 1e3:8.3f} ms" for g in gammas))
    tau_syn = {g: sw.measured_tau(min(64, max(Bs)), Ss[0], g) for g in gammas}
    sw.close()
    params, r1, r2 = fit(base, samples)
    log("fit: " + ", ".join(f"{k} {v:.4g}" for k, v in params.items()) + f"  (rms log residual {r1:.3f} / {r2:.3f})")
    rows, agree = validate(base, params, meas, taus, eps)
    log(f"toggle decisions agreeing with the measured-time speedup: {agree * 100:.1f}% of {len(rows)} points")
    return dict(cfg=cfg["name"], F_eff=F, params=params, rms_log_residual=dict(target=r1, draft_verify=r2),
                samples=samples, validation=rows, agreement=agree, eps=eps, measured_tau=tau_syn,
                seconds=time.time() - torch_started)


def main(argv=None):
    ap = argparse.ArgumentParser(description=__doc__.split("\n")[0])
    ap.add_argument("--model", default="L4_8B", choices=["L4_8B", "L32_8B", "L64_32B", "TINY_BF16"])
    ap.add_argument("--B", default="1,4,16,64,128,256")
    ap.add_argument("--S", default="512,2048,8192")
    ap.add_argument("--gamma", default="3,7,11,15")
    ap.add_argument("--tau", default="2,3,4,5.5,7.5,10,13")
    ap.add_argument("--eps", type=float, default=0.05)
    ap.add_argument("--reps", type=int, default=8)
    ap.add_argument("--out", default="")
    ap.add_argument("--drafter-tradeoff", action="store_true",
                    help="only compare the drafter formats (latency against acceptance) at S = max(--S)")
    a = ap.parse_args(argv)
    cfg = dict(synth.TINY, dtype="bf16", name="tiny-bf16") if a.model == "TINY_BF16" else getattr(synth, a.model)
    ints = lambda s: [int(x) for x in s.split(",") if x]
    if a.drafter_tradeoff:
        rows = drafter_tradeoff(cfg, Bs=ints(a.B), S=max(ints(a.S)), gamma=max(ints(a.gamma)), reps=a.reps,
                                log=lambda *x: print(*x, file=sys.stderr, flush=True))
        txt = json.dumps(rows, indent=1)
        if a.out:
            with open(a.out, "w") as fh:
                fh.write(txt)
        print(txt)
        return
    res = run(cfg, ints(a.B), ints(a.S), ints(a.gamma), [float(x) for x in a.tau.split(",")], a.eps, a.reps,
              log=lambda *x: print(*x, file=sys.stderr, flush=True))
    txt = json.dumps(res, indent=1, default=str)
    if a.out:
        with open(a.out, "w") as fh:
            fh.write(txt)
    print(json.dumps(dict(params=res["params"], F_eff=res["F_eff"], agreement=res["agreement"],
                          rms_log_residual=res["rms_log_residual"], measured_tau=res["measured_tau"])))


if __name__ == "__main__":
    main()
