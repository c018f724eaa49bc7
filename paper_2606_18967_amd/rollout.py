"""Long-tail rollout driver: the EfficientRollout pipeline (Algorithm 1) on
the library's kernels.

One training step of Algorithm 1 refreshes the drafter (RTN int4 of the
current target, Sec. 4.1), then decodes a batch of responses to completion:
autoregressively while the SD toggle of Sec. 4.2 predicts no gain at the
current (live batch B, mean context S) with the previous step's block
efficiency tau_{t-1} and the current draft length gamma_t, and with SD from the
first iteration where it does, for the rest of the rollout (the toggle is
sticky).  After the rollout the step's block efficiency tau_t is measured and
the adaptive policy of Sec. 4.3 picks gamma_{t+1} from the set Gamma with the
patience rule.  Algorithm 1 starts from gamma_1 = gamma_low and
tau_0 = gamma_low.

Four policies share the loop:
  ar        autoregressive decoding throughout (the baseline);
  sd        SD from the first iteration with a fixed gamma = gamma_low;
  toggle    the toggle with a fixed gamma = gamma_low;
  adaptive  the toggle with the adaptive draft length (the full pipeline).

Responses have synthetic lengths with the long tail of RL rollouts: a
log-normal law clipped to [lo, hi] (the paper's responses run to 8k tokens
with means of 620-660; a few long ones set the completion time, Sec. 3.3
and App. A).  A response finishes when it has emitted its length; finished
sequences leave the batch through the slot list (no KV moves), so the live
batch shrinks as in the paper's long tail.  The prompt is a random KV context
of `prompt` positions per sequence (or, with --prefill, `prompt` random
tokens prefilled through the target), the same for every policy, so the
makespan measured is that of the decode phase.

With graphs on, the live batch of each iteration is padded up to a bucket (a
multiple of BUCKET rows; the padding rows run on spare KV slots whose length
is reset before every step) and each (bucket, draft length) SD step and each
AR bucket is captured once as a HIP graph and replayed afterwards, as serving
engines pre-capture graphs per batch size (Sec. 4.1).  The first iteration at
a new bucket runs the padded step eagerly and captures it; capture time is
reported apart from the makespan.
"""
from __future__ import annotations

import argparse
import json
import sys
import time
from dataclasses import asdict, dataclass, field

import numpy as np

from . import sdrl, synth

POLICIES = ("ar", "sd", "toggle", "adaptive")
BUCKET = 8                         # graph buckets: live batches padded to a multiple of this many rows


def bucket_of(n: int, step: int = BUCKET) -> int:
    """The bucket (padded batch size) of a live batch of n rows."""
    if n < 1:
        raise ValueError("a bucket holds at least one row")
    return (n + step - 1) // step * step
GAMMA_SET = (5, 7, 9, 11)          # Gamma, alpha_up, alpha_down, P and eps as the paper sets them (App. E.3)
A_UP, A_DOWN, PATIENCE, EPS = 0.94, 0.85, 2, 0.05


def response_lengths(B: int, median: float, sigma: float, lo: int, hi: int, seed: int) -> np.ndarray:
    """B lengths round(exp(N(ln median, sigma^2))) clipped to [lo, hi]."""
    rng = np.random.default_rng(seed)
    x = np.exp(rng.normal(np.log(median), sigma, size=B))
    return np.clip(np.rint(x), lo, hi).astype(np.int64)


@dataclass
class RolloutResult:
    policy: str
    step: int
    gamma: int
    tau_prev: float
    tau: float | None                   # measured block efficiency (None: no SD iteration ran)
    makespan_s: float
    prep_ms: float
    ar_iters: int
    sd_iters: int
    tokens: int                         # response tokens kept (sum of the lengths)
    switch_iter: int | None             # iteration at which SD switched on
    switch_B: int | None
    trace: list = field(default_factory=list)   # (mode, B, S_mean, ms, emitted) per iteration
    graphs: int = 0                     # HIP graphs captured during the rollout
    capture_s: float = 0.0              # their capture time (outside makespan_s)


def decode(lengths: np.ndarray, prompt: int, policy: str, gamma: int, tau_prev: float, cost, eps: float,
           ar_fn, sd_fn, compact_fn, clock=time.perf_counter, keep_trace: bool = True) -> dict:
    """The decode loop of one rollout (the while loop of Algorithm 1).

    ar_fn() and sd_fn(gamma) run one iteration on the current live rows and
    return the tokens each row emitted (host int array, in row order; SD
    counts n_emit before truncation at the response's end).  compact_fn(keep)
    drops the rows whose keep flag is False.  cost is an sdrl.CostModel for
    the toggle.  Returns the loop's statistics."""
    if policy not in POLICIES:
        raise ValueError(f"unknown policy {policy!r}")
    B0 = len(lengths)
    L = np.asarray(lengths, dtype=np.int64)
    if B0 < 1 or (L < 1).any():
        raise ValueError("every response needs a length >= 1")
    live = np.arange(B0)
    gen = np.zeros(B0, dtype=np.int64)          # tokens emitted, untruncated
    sd_on = 1 if policy == "sd" else 0
    st = dict(ar_iters=0, sd_iters=0, sd_tokens=0, sd_rows=0, switch_iter=None, switch_B=None, trace=[])
    total = 0.0
    it = 0
    while live.size:
        Bl = int(live.size)
        S_mean = prompt + float(np.minimum(gen[live], L[live]).mean())
        if policy in ("toggle", "adaptive") and not sd_on:
            sd_on = sdrl.toggle(cost, Bl, S_mean, tau_prev, gamma, eps, 0)
            if sd_on:
                st["switch_iter"], st["switch_B"] = it, Bl
        t0 = clock()
        if sd_on:
            r = sd_fn(gamma)
        else:
            r = ar_fn()
        # an iteration function may return (tokens, seconds spent capturing a graph)
        n, cap = (r if isinstance(r, tuple) else (r, 0.0))
        n = np.asarray(n, dtype=np.int64)
        if sd_on:
            st["sd_iters"] += 1
            st["sd_tokens"] += int(n.sum())
            st["sd_rows"] += Bl
        else:
            st["ar_iters"] += 1
        dt = clock() - t0 - cap
        st["capture_s"] = st.get("capture_s", 0.0) + cap
        total += dt
        if n.shape != (Bl,) or (n < 1).any():
            raise RuntimeError("a decode iteration must emit at least one token per live row")
        gen[live] += n
        if keep_trace:
            st["trace"].append(("sd" if sd_on else "ar", Bl, round(S_mean, 1), round(dt * 1e3, 3), int(n.sum())))
        keep = gen[live] < L[live]
        if not keep.all():
            live = live[keep]
            if live.size:
                compact_fn(keep)
        it += 1
    st["makespan_s"] = total
    st["tau"] = st["sd_tokens"] / st["sd_rows"] if st["sd_rows"] else None
    st["gen"] = gen
    return st


class Rollout:
    """One model on the GPU with a dense KV cache for B sequences of up to
    prompt + lmax positions, the drafter buffer, and flat device buffers
    viewed at the live batch size and draft length of each iteration."""

    def __init__(self, cfg: dict, B: int, prompt: int, lmax: int, gmax: int = max(GAMMA_SET), seed: int = 3,
                 T: float = 1.0, fmt: str = "w4", graphs: bool = False, padded: bool | None = None,
                 prefill: bool = False):
        import torch
        self.torch = torch
        self.cfg, self.B, self.prompt, self.gmax, self.seed, self.T, self.fmt = cfg, B, prompt, gmax, seed, T, fmt
        # padded: steps run at the bucket size (spare slots B .. B + BUCKET - 2 carry the padding rows);
        # graphs: the padded steps are captured and replayed
        self.graphs = graphs
        self.padded = graphs if padded is None else (padded or graphs)
        self.spare = BUCKET - 1 if self.padded else 0
        self.dev = torch.device("cuda", 0)
        self.eng = sdrl.Engine(cfg, B + self.spare, prompt + lmax + gmax + 2, gmax)
        self.W = synth.make_weights(cfg, seed, self.dev)
        self.eng.bind_weights(self.W)
        self.k, self.v, self.kv_len = self.eng.alloc_kv()
        self.eng.bind_kv(self.k, self.v, self.kv_len)
        self.prefill_s = None
        if prefill:
            # real prompts: `prompt` random tokens per sequence through the target (every slot, spares too)
            nslots = B + self.spare
            toks = synth.make_tokens(nslots, prompt, cfg["vocab"], seed + 5).to(self.dev).contiguous()
            torch.cuda.synchronize()
            t0 = time.perf_counter()
            self.eng.prefill(torch.arange(nslots, dtype=torch.int32, device=self.dev), toks)
            self.eng.sync()
            self.prefill_s = time.perf_counter() - t0
            del toks
        else:
            synth.fill_kv_context(self.k, self.v, prompt, seed + 100)
        self.qbuf = self.eng.refresh_drafter(fmt=fmt)
        V, dev, i32, f32 = cfg["vocab"], self.dev, torch.int32, torch.float32
        B = B + self.spare
        self.flat = dict(draft_tok=torch.zeros(B * gmax, dtype=i32, device=dev),
                         q_logits=torch.zeros(B * gmax * V, dtype=f32, device=dev),
                         q_stats=torch.zeros(B * gmax * 2, dtype=f32, device=dev),
                         p_logits=torch.zeros(B * (gmax + 1) * V, dtype=f32, device=dev),
                         out_tok=torch.zeros(B * (gmax + 1), dtype=i32, device=dev),
                         n_emit=torch.zeros(B, dtype=i32, device=dev),
                         next_tok=torch.zeros(B, dtype=i32, device=dev),
                         ar_out=torch.zeros(B, dtype=i32, device=dev),
                         ar_logits=torch.zeros(B * V, dtype=f32, device=dev))

    def _view(self, name, *shape):
        n = int(np.prod(shape))
        return self.flat[name][:n].view(*shape)

    def run(self, policy: str, gamma: int, tau_prev: float, cost, eps: float, lengths, step: int,
            keep_trace: bool = True) -> tuple[RolloutResult, dict]:
        torch, eng, V = self.torch, self.eng, self.cfg["vocab"]
        if len(lengths) != self.B:
            raise ValueError("one length per sequence")
        if gamma > self.gmax:
            raise ValueError("gamma above the engine's maximum")
        # Prep: the drafter refresh of this training step
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        eng.refresh_drafter(self.qbuf, fmt=self.fmt)
        e1.record()
        torch.cuda.synchronize()
        prep_ms = e0.elapsed_time(e1)
        self.kv_len.fill_(self.prompt)
        state = dict(slots=torch.arange(self.B, dtype=torch.int32, device=self.dev),
                     last=synth.make_tokens(self.B, 1, V, self.seed + 7 + step)[:, 0].to(self.dev).contiguous())
        T, seed = self.T, self.seed
        cache = {}                             # (kind, bucket, gamma) -> padded buffers and captured graph
        spare = torch.arange(self.B, self.B + self.spare, dtype=torch.int32, device=self.dev)

        def padded_entry(kind, Bl, g):
            bk = bucket_of(Bl)
            key = (kind, bk, g)
            ent = cache.get(key)
            if ent is None:
                ent = dict(slots=torch.zeros(bk, dtype=torch.int32, device=self.dev),
                           last=torch.zeros(bk, dtype=torch.int32, device=self.dev), graph=None)
                if kind == "sd":
                    ent["bufs"] = sdrl.SDBuffers(eng, bk, g)
                else:
                    ent["out"] = torch.zeros(bk, dtype=torch.int32, device=self.dev)
                    ent["logits"] = torch.zeros((bk, V), dtype=torch.float32, device=self.dev)
                cache[key] = ent
            # live rows first, then the spare slots; the spare slots restart from the prompt every step
            ent["slots"][:Bl].copy_(state["slots"])
            ent["slots"][Bl:].copy_(spare[:bk - Bl])
            ent["last"][:Bl].copy_(state["last"])
            ent["last"][Bl:].zero_()
            self.kv_len[self.B:].fill_(self.prompt)
            return ent

        def run_padded(ent, eager, capture):
            """Replays the entry's graph, or runs the step eagerly (and captures it)."""
            if ent["graph"] is not None:
                ent["graph"].replay()
                return 0.0
            eager()
            if not capture:
                return 0.0
            torch.cuda.synchronize()
            t0 = time.perf_counter()
            graph = torch.cuda.CUDAGraph()
            side = torch.cuda.Stream(device=self.dev)          # default priority
            side.wait_stream(torch.cuda.current_stream())
            with torch.cuda.graph(graph, stream=side):
                eager()
            torch.cuda.current_stream().wait_stream(side)
            torch.cuda.synchronize()
            ent["graph"] = graph
            return time.perf_counter() - t0

        def ar_padded():
            Bl = state["slots"].numel()
            ent = padded_entry("ar", Bl, 0)

            def eager():
                eng.ar_step(ent["slots"], ent["last"], T, seed, 2 * step, ent["out"], ent["logits"])
                torch.add(ent["out"], 0, out=ent["last"])      # a kernel node, not a copy node
            cap = run_padded(ent, eager, self.graphs)
            state["last"] = ent["last"][:Bl].clone()
            torch.cuda.synchronize()
            return np.ones(Bl, dtype=np.int64), cap

        def sd_padded(g):
            Bl = state["slots"].numel()
            ent = padded_entry("sd", Bl, g)
            bufs = ent["bufs"]

            def eager():
                sdrl.sd_step(eng, bufs, ent["slots"], ent["last"], T, seed, 2 * step + 1)
                torch.add(bufs.next_tok, 0, out=ent["last"])
            cap = run_padded(ent, eager, self.graphs)
            state["last"] = ent["last"][:Bl].clone()
            return bufs.n_emit[:Bl].cpu().numpy(), cap

        def ar_fn():
            Bl = state["slots"].numel()
            out, pl = self._view("ar_out", Bl), self._view("ar_logits", Bl, V)
            eng.ar_step(state["slots"], state["last"], T, seed, 2 * step, out, pl)
            state["last"] = out.clone()
            torch.cuda.synchronize()          # the host learns which sequences ended (one token each here)
            return np.ones(Bl, dtype=np.int64)

        def sd_fn(g):
            Bl = state["slots"].numel()
            dt_, ql, qs = self._view("draft_tok", Bl, g), self._view("q_logits", Bl, g, V), self._view("q_stats", Bl, g, 2)
            pl, ot = self._view("p_logits", Bl, g + 1, V), self._view("out_tok", Bl, g + 1)
            ne, nt = self._view("n_emit", Bl), self._view("next_tok", Bl)
            eng.draft(state["slots"], state["last"], g, T, seed, 2 * step + 1, dt_, ql, qs)
            eng.verify(state["slots"], state["last"], dt_, g, pl)
            eng.accept(state["slots"], dt_, ql, qs, pl, g, T, seed, 2 * step + 1, ot, ne, nt)
            eng.rollback(state["slots"], ne)
            state["last"] = nt.clone()
            return ne.cpu().numpy()           # the host needs n_emit every step

        def compact_fn(keep):
            idx = torch.from_numpy(np.nonzero(keep)[0]).to(self.dev)
            state["slots"] = state["slots"].index_select(0, idx)
            state["last"] = state["last"].index_select(0, idx)

        torch.cuda.synchronize()
        st = decode(lengths, self.prompt, policy, gamma, tau_prev, cost, eps,
                    ar_padded if self.padded else ar_fn, sd_padded if self.padded else sd_fn, compact_fn,
                    keep_trace=keep_trace)
        eng.sync()
        res = RolloutResult(policy=policy, step=step, gamma=gamma, tau_prev=tau_prev, tau=st["tau"],
                            makespan_s=st["makespan_s"], prep_ms=prep_ms, ar_iters=st["ar_iters"],
                            sd_iters=st["sd_iters"], tokens=int(np.asarray(lengths).sum()),
                            switch_iter=st["switch_iter"], switch_B=st["switch_B"], trace=st["trace"],
                            graphs=sum(e["graph"] is not None for e in cache.values()),
                            capture_s=st.get("capture_s", 0.0))
        return res, st

    def close(self):
        self.eng.close()


def tau_at(tau: float, gamma_meas: int, gamma: int) -> float:
    """Block efficiency expected at draft length gamma from one measured at
    gamma_meas, through the acceptance rate: alpha solves
    tau = (1 - alpha^(gamma_meas+1)) / (1 - alpha), and the result is
    (1 - alpha^(gamma+1)) / (1 - alpha), the i.i.d. acceptance relation of
    Sec. 3.1 (inverted the same way in App. E.2)."""
    if gamma == gamma_meas:
        return float(tau)
    return float(sdrl.tau_from_alpha(sdrl.alpha_from_tau(tau, gamma_meas), gamma))


def train(run_fn, policy: str, n_steps: int, lengths_fn, gset=GAMMA_SET, P=PATIENCE, a_up=A_UP, a_down=A_DOWN,
          tau_carry: bool = False):
    """n_steps training steps of Algorithm 1 under one policy: gamma_1 =
    gamma_low and tau_0 = gamma_low; after each rollout the measured tau_t
    becomes the toggle's tau for the next step and (policy 'adaptive')
    drives gamma_{t+1}.  A rollout with no SD iteration measures no tau; the
    previous one is kept and the controller is not stepped.

    By default the toggle of step t gets the measured tau_{t-1} as it is,
    together with gamma_t, as Algorithm 1 writes it.  With tau_carry, a tau
    measured at another draft length is first carried to gamma_t through
    the acceptance rate (tau_at): the speedup of eq:sd_speedup_toggle uses
    the block efficiency at the draft length it prices, and a tau measured
    at a shorter draft understates the longer draft's gain.  The two
    variants differ only in the step after gamma moves.

    run_fn(policy, gamma, tau_prev, lengths, step) returns a RolloutResult."""
    ctl = sdrl.GammaController(gset, P, a_up, a_down)
    gamma, tau_meas, gamma_meas = int(gset[0]), float(gset[0]), int(gset[0])
    out = []
    for t in range(n_steps):
        g = gamma if policy == "adaptive" else int(gset[0])
        tau_prev = tau_at(tau_meas, gamma_meas, g) if tau_carry else tau_meas
        r = run_fn(policy, g, tau_prev, lengths_fn(t), t)
        if r.tau is not None:
            tau_meas, gamma_meas = r.tau, g
            if policy == "adaptive":
                gamma = ctl.update(r.tau)
        out.append(r)
    return out


def calibrated_cost(cfg: dict, calib: dict):
    """The toggle's cost model (Sec. 4.2): the architecture terms of cfg with
    the fitted parameters of calibrate.py (F_eff, BW_eff, rho_kappa, eta_D,
    c_T, c_D, c_V)."""
    m = sdrl.cost_init(cfg)
    m.F_eff = float(calib["F_eff"])
    for k, v in calib["params"].items():
        setattr(m, k, float(v))
    return m


MODELS = {"L4_8B": synth.L4_8B, "L32_8B": synth.L32_8B, "TINY_BF16": dict(synth.TINY, dtype="bf16", name="tiny-bf16")}


def main(argv=None):
    ap = argparse.ArgumentParser(description=__doc__.split("\n")[0])
    ap.add_argument("--model", default="L32_8B", choices=sorted(MODELS))
    ap.add_argument("--B", type=int, default=128)
    ap.add_argument("--prompt", type=int, default=512)
    ap.add_argument("--median", type=float, default=512.0)
    ap.add_argument("--sigma", type=float, default=0.894)
    ap.add_argument("--lmin", type=int, default=16)
    ap.add_argument("--lmax", type=int, default=4096)
    ap.add_argument("--steps", type=int, default=3, help="training steps per policy")
    ap.add_argument("--policies", default=",".join(POLICIES))
    ap.add_argument("--seed", type=int, default=3)
    ap.add_argument("--drafter", default="w4", choices=sorted(sdrl.DRAFT_FORMATS))
    ap.add_argument("--calib", default="", help="calibrate.py --out JSON; default: calibrate now on this model")
    ap.add_argument("--calib-B", default="1,4,16,64,128")
    ap.add_argument("--calib-S", default="512,2048,4096")
    ap.add_argument("--prefill", action="store_true",
                    help="prefill `prompt` random tokens per sequence through the target instead of random KV context")
    ap.add_argument("--graphs", action="store_true",
                    help="pad live batches to buckets of BUCKET rows and replay one captured HIP graph per "
                         "(bucket, draft length) and per AR bucket")
    ap.add_argument("--tau-carry", action="store_true",
                    help="carry the toggle's tau to a new draft length through the acceptance rate "
                         "(default: Algorithm 1 as written, the measured tau as it is)")
    ap.add_argument("--out", default="")
    a = ap.parse_args(argv)
    log = lambda *x: print(*x, file=sys.stderr, flush=True)
    cfg = MODELS[a.model]
    ints = lambda s: [int(x) for x in s.split(",") if x]
    if a.calib:
        with open(a.calib) as fh:
            calib = json.load(fh)
    else:
        from . import calibrate
        log("calibrating the cost model ...")
        calib = calibrate.run(cfg, ints(a.calib_B), ints(a.calib_S), [GAMMA_SET[0]], [2.0, 3.0, 4.0], EPS, 6, log=log,
                              fmt=a.drafter)
        calib = dict(F_eff=calib["F_eff"], params=calib["params"], agreement=calib["agreement"])
    cost = calibrated_cost(cfg, calib)
    log("building the rollout engine ...")
    ro = Rollout(cfg, a.B, a.prompt, a.lmax, seed=a.seed, fmt=a.drafter, graphs=a.graphs, prefill=a.prefill)
    if ro.prefill_s is not None:
        log(f"prefill of {a.B} x {a.prompt} tokens: {ro.prefill_s:.2f} s")
    lengths_fn = lambda t: response_lengths(a.B, a.median, a.sigma, a.lmin, a.lmax, a.seed * 1000 + t)
    # one untimed rollout to load every kernel
    ro.run("sd", GAMMA_SET[0], float(GAMMA_SET[0]), cost, EPS, np.minimum(lengths_fn(0), 64), 99, keep_trace=False)
    def run_and_report(p, g, tp, L, t):
        r = ro.run(p, g, tp, cost, EPS, L, t)[0]
        # one line per training step as soon as it ends (a policy's steps can take minutes in all)
        log(f"{p:9s} step {r.step}: gamma {r.gamma:2d}  tau_prev {r.tau_prev:5.2f}  tau "
            f"{'  -  ' if r.tau is None else f'{r.tau:5.2f}'}  makespan {r.makespan_s:7.3f} s  "
            f"AR iters {r.ar_iters:5d}  SD iters {r.sd_iters:5d}  SD on at B={r.switch_B}  prep {r.prep_ms:.1f} ms"
            f"  graphs {r.graphs} ({r.capture_s:.2f} s to capture)")
        return r

    results = {}
    for pol in a.policies.split(","):
        results[pol] = train(run_and_report, pol, a.steps, lengths_fn, tau_carry=a.tau_carry)
    ro.close()
    L0 = lengths_fn(0)
    summary = dict(model=cfg["name"], drafter=a.drafter, B=a.B, prompt=a.prompt, tau_carry=a.tau_carry,
                   graphs=a.graphs, prefill_s=ro.prefill_s,
                   lengths=dict(median=a.median, sigma=a.sigma, lo=a.lmin, hi=a.lmax, mean_step0=float(L0.mean()),
                                max_step0=int(L0.max())),
                   calib=dict(F_eff=calib["F_eff"], params=calib["params"]),
                   makespan_s={p: [r.makespan_s for r in rs] for p, rs in results.items()},
                   results={p: [asdict(r) for r in rs] for p, rs in results.items()})
    if a.out:
        with open(a.out, "w") as fh:
            json.dump(summary, fh)
    print(json.dumps(dict(model=summary["model"], drafter=a.drafter, B=a.B, tau_carry=a.tau_carry, graphs=a.graphs,
                          makespan_s=summary["makespan_s"],
                          tau={p: [r.tau for r in rs] for p, rs in results.items()},
                          gamma={p: [r.gamma for r in rs] for p, rs in results.items()},
                          switch_B={p: [r.switch_B for r in rs] for p, rs in results.items()})))


if __name__ == "__main__":
    main()
