"""Comparison of device SD / AR steps against the oracle -- TEST INFRASTRUCTURE.

The device side is given as numpy arrays copied back from the library.  Two
separate checks, following the decision-parity protocol (Sec. 3.1, App. D.1
define the rule; decisions and logits are judged apart):

  decisions   on IDENTICAL logits: the oracle's race sampler and rejection
              rule run on the device's own q and p rows with the same Philox
              uniforms and must reproduce the device's draft tokens, q row
              statistics, n_emit and emitted tokens exactly.  The only
              exemptions are rounding-level ones: an accept test with
              |u - p/q| < 1e-3, or a race whose two best keys differ by less
              than 1e-5 * max(1, |key|).
  logits      against the oracle's forward on the device's own tokens
              (teacher forcing): max |dev - oracle| <= tol * max |oracle| per
              row (tol 5e-3 for fp32 models, 2e-2 for bf16).

Because the oracle is teacher-forced onto the device's emitted tokens, a
sequence is never dropped from comparison: an exempt decision is counted and
the comparison goes on from the device's tokens.  The decisions the oracle
takes on its own logits are reported alongside (they may differ from the
device's wherever the logit tolerance moves a decision; that is information,
not a failure).
"""
from __future__ import annotations

import numpy as np

import oracle

BAND_ACCEPT = 1e-3      # |u - p/q| below which an accept test is a rounding-level tie
REL_KEY_GAP = 1e-5      # race-key gap, relative to max(1, |key|), below which two draws tie


class Mismatch(AssertionError):
    pass


def row_tol_ok(dev, ref, tol):
    scale = np.abs(ref).max(axis=-1)
    err = np.abs(dev - ref).max(axis=-1)
    return bool(np.all(err <= tol * scale)), float((err / np.maximum(scale, 1e-30)).max())


def _race_key(logits, x, T, seed, step, stream, slot, pos):
    """The race key l_x/T - ln(-ln u_x) of entry x (a magnitude for the tie
    rule; float64 is plenty)."""
    u = oracle.uniform_row(seed, step, stream, slot, pos, x + 1)[x]
    return float(logits[x]) / T - np.log(-np.log(float(u)))


def _residual_key(lp, lq, x, T, seed, step, slot, pos):
    p = _softmax(lp, T)
    q = _softmax(lq, T)
    r = max(p[x] - q[x], 1e-300)
    u = oracle.uniform_row(seed, step, oracle.STREAM_RESIDUAL, slot, pos, x + 1)[x]
    return float(np.log(r) - np.log(-np.log(float(u))))


def _softmax(l, T):
    z = np.asarray(l, dtype=np.float64) / T
    z = np.exp(z - z.max())
    return z / z.sum()


def draw_tie(gap, key):
    return gap < REL_KEY_GAP * max(1.0, abs(key))


def check_draws(dev_q, dev_draft, T, key, dev_stats=None):
    """Draft draws (and their row statistics) on the device's own q rows.
    key = (seed, step, slot, kv_len).  Returns the number of exempt ties;
    raises Mismatch otherwise."""
    seed, step, slot, kv_len = key
    exempt = 0
    for j in range(len(dev_draft)):
        pos = kv_len + j + 1
        x, gap = oracle.sample_row(dev_q[j], T, seed, step, oracle.STREAM_TOKEN, slot, pos)
        if x != int(dev_draft[j]):
            k = _race_key(dev_q[j], x, T, seed, step, oracle.STREAM_TOKEN, slot, pos)
            if not draw_tie(gap, k):
                raise Mismatch(f"draft draw {j} on the device's logits: dev {int(dev_draft[j])} oracle {x} "
                               f"gap {gap:.3e} key {k:.3f}")
            exempt += 1
        if dev_stats is not None:
            m, lse = oracle.row_stats(dev_q[j], T)
            dm, dl = float(dev_stats[j][0]), float(dev_stats[j][1])
            if abs(dm - m) > 1e-6 * max(1.0, abs(m)) or abs(dl - lse) > 1e-4 + 1e-6 * abs(lse):
                raise Mismatch(f"q_stats row {j}: dev ({dm}, {dl}) oracle ({m}, {lse})")
    return exempt


def check_accept(dev, T, key):
    """The rejection rule on the device's own draft tokens, q and p rows:
    n_emit and the emitted tokens must be the oracle's.  Returns ("ok" |
    "exempt", info); raises Mismatch otherwise."""
    seed, step, slot, kv_len = key
    gamma = len(dev["draft"])
    n_d = int(dev["n_emit"])
    out_d = np.asarray(dev["out"][:n_d])
    n_o, out_o, ratio, u, fgap = oracle.accept_seq(dev["draft"], dev["q"], dev["p"], T, seed, step, slot, kv_len)
    if n_o == n_d and np.array_equal(out_o[:n_o], out_d):
        return "ok", dict(n=n_o)
    if n_o != n_d:
        k = min(n_o, n_d)                  # 1-based position of the first differing accept decision
        if k <= gamma and abs(float(u[k - 1]) - float(ratio[k - 1])) < BAND_ACCEPT:
            return "exempt", dict(where=f"accept {k}", u=float(u[k - 1]), ratio=float(ratio[k - 1]))
        raise Mismatch(f"accept on the device's logits: dev n={n_d} out={out_d.tolist()} oracle n={n_o} "
                       f"out={out_o[:n_o].tolist()} u={u.tolist()} ratio={ratio.tolist()}")
    # same decisions, different final token: the residual or bonus race
    if not np.array_equal(out_o[:n_o - 1], out_d[:n_d - 1]):
        raise Mismatch(f"accepted prefix differs: dev {out_d.tolist()} oracle {out_o[:n_o].tolist()}")
    x = int(out_o[n_o - 1])
    if n_o <= gamma:
        j = n_o
        k = _residual_key(dev["p"][j - 1], dev["q"][j - 1], x, T, seed, step, slot, kv_len + j)
    else:
        k = _race_key(dev["p"][gamma], x, T, seed, step, oracle.STREAM_TOKEN, slot, kv_len + gamma + 1)
    if draw_tie(fgap, k):
        return "exempt", dict(where="final draw", gap=fgap, key=k)
    raise Mismatch(f"final draw on the device's logits: dev {int(out_d[-1])} oracle {x} gap {fgap:.3e} key {k:.3f}")


def forced_step_logits(target, drafter, kv, kv_len, last_tok, draft_tok):
    """The oracle's q and p rows of one SD step on the given draft tokens:
    the drafter runs [last, d_1..d_{gamma-1}] from kv_len (writing its
    provisional KV), then the target runs [last, d_1..d_gamma] from kv_len
    (overwriting it with clean KV), as in App. D.1."""
    d = [int(x) for x in draft_tok]
    q = oracle.forward_seq(drafter, kv, [int(last_tok)] + d[:-1], kv_len)
    p = oracle.forward_seq(target, kv, [int(last_tok)] + d, kv_len)
    return q, p


def check_step(dev, ref_q, ref_p, tol, T, key):
    """Full check of one device SD step of one sequence.

    dev: draft [gamma], q [gamma][V], p [gamma+1][V], out, n_emit and
    optionally q_stats [gamma][2]; ref_q, ref_p: the oracle's logits on the
    device's tokens (forced_step_logits).  Returns info with the count of
    exempt decisions, the worst relative logit error and the agreement of the
    oracle's own-logit decisions; raises Mismatch on a real disagreement."""
    gamma = len(dev["draft"])
    worst = 0.0
    for j in range(gamma):
        ok, rel = row_tol_ok(dev["q"][j], ref_q[j], tol)
        worst = max(worst, rel)
        if not ok:
            raise Mismatch(f"draft logits row {j}: rel err {rel:.3e} > {tol}")
    ok, rel = row_tol_ok(dev["p"], ref_p, tol)
    worst = max(worst, rel)
    if not ok:
        raise Mismatch(f"verify logits: rel err {rel:.3e} > {tol}")
    n = int(dev["n_emit"])
    if not (1 <= n <= gamma + 1):
        raise Mismatch(f"n_emit {n} outside [1, {gamma + 1}]")
    exempt = check_draws(dev["q"], dev["draft"], T, key, dev.get("q_stats"))
    status, info = check_accept(dev, T, key)
    exempt += status == "exempt"
    # the oracle's decisions on its own logits (reported, not required)
    seed, step, slot, kv_len = key
    own_draws = sum(int(oracle.sample_row(ref_q[j], T, seed, step, oracle.STREAM_TOKEN, slot, kv_len + j + 1)[0]
                        == int(dev["draft"][j])) for j in range(gamma))
    n_o, out_o, *_ = oracle.accept_seq(dev["draft"], ref_q, ref_p, T, seed, step, slot, kv_len)
    own_accept = bool(n_o == n and np.array_equal(out_o[:n_o], np.asarray(dev["out"][:n])))
    return dict(exempt=exempt, worst=worst, accept=info, own_draws=own_draws, own_accept=own_accept)


def check_ar(dev_p, dev_x, ref_p, tol, T, key):
    """One AR step of one sequence: the device's token against the oracle's
    race on the device's own logits (exact up to a key tie), the logits
    against the oracle's forward on the same token.  key = (seed, step, slot,
    kv_len).  Returns ("ok" | "exempt", worst rel error, own-logit token)."""
    seed, step, slot, kv_len = key
    ok, rel = row_tol_ok(dev_p, ref_p, tol)
    if not ok:
        raise Mismatch(f"AR logits: rel err {rel:.3e} > {tol}")
    x, gap = oracle.sample_row(dev_p, T, seed, step, oracle.STREAM_TOKEN, slot, kv_len + 1)
    own, _ = oracle.sample_row(ref_p, T, seed, step, oracle.STREAM_TOKEN, slot, kv_len + 1)
    if x == int(dev_x):
        return "ok", rel, own
    k = _race_key(dev_p, x, T, seed, step, oracle.STREAM_TOKEN, slot, kv_len + 1)
    if draw_tie(gap, k):
        return "exempt", rel, own
    raise Mismatch(f"AR token on the device's logits: dev {int(dev_x)} oracle {x} gap {gap:.3e} key {k:.3f}")


def unpack_q4(packed: np.ndarray, scales_bits: np.ndarray, N: int, K: int, fmt: str = "w4"):
    """Codes [N][K] (int8) and scales [N][K/128] (fp16 bits) from the
    library's packed int4 layout (documented in include/sd_api.h): for column
    block nb = n/32 and group g, word (((nb*G + g)*2 + st//4)*64 + l)*4 + st%4
    of lane l = n%32 + 32*h holds codes k = 128g + 16st + 8h + e at nibble
    4*(e//2) + 16*(e%2), stored as q + 8 ("w4") or q ("w4a"); scale
    (nb*G + g)*32 + n%32."""
    G = K // 128
    words = packed.view(np.uint32).reshape(N // 32, G, 2, 64, 4)     # [nb, g, st//4, lane, st%4]
    codes = np.zeros((N, K), dtype=np.int8)
    lanes = np.arange(64)
    cols = (np.arange(N // 32)[:, None] * 32 + (lanes % 32)[None, :])  # [nb, lane]
    h = lanes // 32
    off = 8 if fmt == "w4" else 0
    for st in range(8):
        w = words[:, :, st // 4, :, st % 4]                             # [nb, g, lane]
        for e in range(8):
            nib = ((w >> np.uint32(4 * (e // 2) + 16 * (e % 2))) & np.uint32(15)).astype(np.int16) - off
            for g in range(G):
                ks = g * 128 + 16 * st + 8 * h + e                      # per lane
                codes[cols, ks[None, :]] = nib[:, g, :]
    return codes, _unpack_groupwise(scales_bits.view(np.uint16), N, G)


def unpack_q8(packed: np.ndarray, scales_bits: np.ndarray, N: int, K: int):
    """Codes [N][K] (int8) and scales from the library's packed int8 layout:
    code e of k-step st, lane l = n%32 + 32*h (k = 128g + 16st + 8h + e) is
    byte e%4 of word j = 2*st + e//4 at index (((nb*G + g)*4 + j//4)*64 + l)*4
    + j%4, stored as q + 128."""
    G = K // 128
    words = packed.view(np.uint32).reshape(N // 32, G, 4, 64, 4)     # [nb, g, j//4, lane, j%4]
    codes = np.zeros((N, K), dtype=np.int8)
    lanes = np.arange(64)
    cols = (np.arange(N // 32)[:, None] * 32 + (lanes % 32)[None, :])
    h = lanes // 32
    for j in range(16):
        w = words[:, :, j // 4, :, j % 4]
        st = j // 2
        for b in range(4):
            e = 4 * (j % 2) + b
            byte = ((w >> np.uint32(8 * b)) & np.uint32(255)).astype(np.int16) - 128
            for g in range(G):
                ks = g * 128 + 16 * st + 8 * h + e
                codes[cols, ks[None, :]] = byte[:, g, :]
    return codes, _unpack_groupwise(scales_bits.view(np.uint16), N, G)


def _unpack_groupwise(x: np.ndarray, N: int, G: int):
    """[N][G] from the per-(column, group) layout (nb*G + g)*32 + n%32."""
    return x.reshape(N // 32, G, 32).transpose(0, 2, 1).reshape(N, G)


def unpack_zeros(zero_bytes: np.ndarray, N: int, K: int):
    return _unpack_groupwise(zero_bytes.view(np.uint8), N, K // 128)


def drafter_layout(cfg: dict, fmt: str = "w4"):
    """(layer, which, N, K, code_offset, scale_offset, zero_offset or None) of
    every quantized projection in the drafter buffer (include/sd_api.h), and
    the buffer's size."""
    H, d, F = cfg["hidden"], cfg["head_dim"], cfg["ffn"]
    shapes = [((cfg["n_q"] + 2 * cfg["n_kv"]) * d, H), (H, cfg["n_q"] * d), (2 * F, H), (H, F)]
    a256 = lambda x: (x + 255) // 256 * 256
    out, off = [], 0
    for l in range(cfg["n_layers"]):
        for w, (N, K) in enumerate(shapes):
            cb = a256(N * K // (1 if fmt == "w8" else 2))
            sb = a256(N * (K // 128) * 2)
            zb = a256(N * (K // 128)) if fmt == "w4a" else 0
            out.append((l, w, N, K, off, off + cb, off + cb + sb if zb else None))
            off += cb + sb + zb
    return out, off
