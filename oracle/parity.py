"""Comparison of one device SD step against the oracle -- TEST INFRASTRUCTURE.

The device side is given as numpy arrays copied back from the library; the
oracle runs its own step on its own state (its inputs come only from the
seeded generators and from its own earlier outputs).  Rules:

  logits   max |dev - oracle| <= tol * max |oracle| per row (tol 5e-3 for
           fp32 models, 2e-2 for bf16);
  draws    a token drawn by exponential race must be identical unless the
           oracle's two best keys are closer than twice the largest logit
           difference of that row (then both draws are correct outcomes of
           nearly equal keys and the sequence stops being compared);
  accept   accept / reject decisions must be identical unless
           |u - p/q| < 1e-3 at the deciding position; the final residual or
           bonus draw follows the draw rule.  A decision or draw that still
           differs is judged on identical logits: the oracle's accept (the
           rejection rule of App. D.1) run on the device's own p and q must
           reproduce the device's tokens exactly.  The difference then comes
           only from logit differences within the tolerance, which move p/q
           (an accept test) or the race of the residual max(0, p - q).
"""
from __future__ import annotations

import numpy as np

import oracle


class Mismatch(AssertionError):
    pass


def row_tol_ok(dev, ref, tol):
    scale = np.abs(ref).max(axis=-1)
    err = np.abs(dev - ref).max(axis=-1)
    return bool(np.all(err <= tol * scale)), float((err / np.maximum(scale, 1e-30)).max())


def compare_step(r: dict, dev: dict, tol: float, T: float = 1.0, key=None):
    """r: oracle step (oracle.sd_step_seq); dev: draft, q, p, out, n_emit of
    the same sequence from the device.  key = (seed, step, slot, kv_len) of
    the step, for the residual-draw check below.  Returns ("ok" | "exempt",
    info); raises Mismatch on a real disagreement."""
    gamma = len(r["draft"])
    worst = 0.0
    for j in range(gamma):
        ok, rel = row_tol_ok(dev["q"][j], r["q"][j], tol)
        worst = max(worst, rel)
        if not ok:
            raise Mismatch(f"draft logits row {j}: rel err {rel:.3e} > {tol}")
        if int(dev["draft"][j]) != int(r["draft"][j]):
            delta = float(np.abs(dev["q"][j] - r["q"][j]).max()) / T
            if r["draft_gap"][j] <= 2 * delta + 1e-6:
                return "exempt", dict(where=f"draft {j}", gap=float(r["draft_gap"][j]), delta=delta, worst=worst)
            raise Mismatch(f"draft token {j}: dev {dev['draft'][j]} oracle {r['draft'][j]} "
                           f"gap {r['draft_gap'][j]:.3e} delta {delta:.3e}")
    ok, rel = row_tol_ok(dev["p"], r["p"], tol)
    worst = max(worst, rel)
    if not ok:
        raise Mismatch(f"verify logits: rel err {rel:.3e} > {tol}")
    n_d, n_o = int(dev["n_emit"]), r["n_emit"]
    out_d = np.asarray(dev["out"][:n_d])
    if n_d == n_o and np.array_equal(out_d, r["out"]):
        return "ok", dict(worst=worst)
    # decisions differ: find the deciding position
    k = min(n_d, n_o)               # 1-based position of the first differing decision
    if k <= gamma and abs(float(r["u"][k - 1]) - float(r["ratio"][k - 1])) < 1e-3:
        return "exempt", dict(where=f"accept {k}", u=float(r["u"][k - 1]), ratio=float(r["ratio"][k - 1]))
    if n_d == n_o:
        delta = float(np.abs(dev["p"] - r["p"]).max() + np.abs(dev["q"] - r["q"]).max()) / T
        if r["final_gap"] <= 2 * delta + 1e-6:
            return "exempt", dict(where="final draw", gap=r["final_gap"], delta=delta)
    # Judged on identical logits: the residual max(0, p - q) of the rejection
    # rule (App. D.1) is the difference of two nearly equal distributions
    # wherever the drafter agrees with the target, and p/q of an accept test
    # moves with the logits, so logit differences within the tolerance can
    # change either.  The oracle's accept on the device's own logits must then
    # give the device's tokens exactly.
    if key is not None:
        seed, step, slot, kv_len = key
        n2, out2, *_ = oracle.accept_seq(dev["draft"], dev["q"], dev["p"], T, seed, step, slot, kv_len)
        if n2 == n_d and np.array_equal(out2[:n2], out_d):
            where = "residual draw" if n_d == n_o else f"accept {k}"
            return "exempt", dict(where=where, note="oracle on device logits agrees", u=float(r["u"][k - 1]) if k <= gamma else None,
                                  ratio=float(r["ratio"][k - 1]) if k <= gamma else None)
    raise Mismatch(f"accept: dev n={n_d} out={out_d.tolist()} oracle n={n_o} out={r['out'].tolist()} "
                   f"u={r['u'].tolist()} ratio={r['ratio'].tolist()}")


def compare_ar(x_oracle: int, gap: float, p_oracle, x_dev: int, p_dev, tol: float, T: float = 1.0):
    ok, rel = row_tol_ok(p_dev, p_oracle, tol)
    if not ok:
        raise Mismatch(f"AR logits: rel err {rel:.3e} > {tol}")
    if x_dev == x_oracle:
        return "ok"
    delta = float(np.abs(p_dev - p_oracle).max()) / T
    if gap <= 2 * delta + 1e-6:
        return "exempt"
    raise Mismatch(f"AR token: dev {x_dev} oracle {x_oracle} gap {gap:.3e} delta {delta:.3e}")


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
