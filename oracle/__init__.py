"""CPU oracle for quantized self-speculative decoding -- TEST INFRASTRUCTURE.

Only ``tests/``, ``__graft_entry__.smoke()`` and the ``cpu_baseline`` leg of
``bench.py`` may import this package.  The product path (the HIP library in
``paper_2606_18967_amd``) never imports, links or calls it, and the two share
no source.

The arithmetic lives in ``sd_oracle.c`` (plain C, double-precision model
arithmetic, fp32 decisions); this module only builds it with gcc and marshals
numpy arrays through ctypes.
"""
from __future__ import annotations

import ctypes as C
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
SRC = os.path.join(_HERE, "sd_oracle.c")
LIB_DIR = os.path.join(_HERE, "_build")
LIB_PATH = os.path.join(LIB_DIR, "liboracle.so")

STREAM_TOKEN, STREAM_ACCEPT, STREAM_RESIDUAL = 0, 1, 2
F32, BF16, Q4 = 0, 1, 2


def build(force: bool = True) -> str:
    """Compile the oracle with gcc (no GPU code involved)."""
    if not force and os.path.exists(LIB_PATH) and os.path.getmtime(LIB_PATH) >= os.path.getmtime(SRC):
        return LIB_PATH
    os.makedirs(LIB_DIR, exist_ok=True)
    tmp = LIB_PATH + ".tmp%d" % os.getpid()
    cmd = ["gcc", "-O2", "-fopenmp", "-fPIC", "-shared", "-ffp-contract=off",
           "-Wall", "-o", tmp, SRC, "-lm"]
    subprocess.run(cmd, check=True)
    os.replace(tmp, LIB_PATH)
    return LIB_PATH


_lib = None


def lib():
    global _lib
    if _lib is None:
        build(force=False)
        _lib = _declare(C.CDLL(LIB_PATH))
    return _lib


class Cfg(C.Structure):
    _fields_ = [("n_layers", C.c_int), ("hidden", C.c_int), ("n_q", C.c_int), ("n_kv", C.c_int),
                ("head_dim", C.c_int), ("ffn", C.c_int), ("vocab", C.c_int),
                ("rms_eps", C.c_float), ("rope_theta", C.c_float)]


class Cost(C.Structure):
    _fields_ = [(n, C.c_double) for n in
                ("W_T", "W_D", "kappa_th", "C_dense", "C_attn",
                 "BW_eff", "F_eff", "rho_kappa", "eta_D", "c_T", "c_D", "c_V")]


_P = C.c_void_p
_u64, _u32, _i32, _f, _d, _i = C.c_uint64, C.c_uint32, C.c_int32, C.c_float, C.c_double, C.c_int


def _declare(L):
    sig = {
        "or_f32_to_f16": (C.c_uint16, [_f]),
        "or_f16_to_f32": (_f, [C.c_uint16]),
        "or_philox4x64_10": (None, [_P, _P, _P]),
        "or_uniform": (_f, [_u64, _u64, _u32, _u32, _u32, _u32]),
        "or_uniform_row": (None, [_u64, _u64, _u32, _u32, _u32, _i, _P]),
        "or_row_stats": (None, [_P, _i, _f, _P, _P]),
        "or_sample_row": (_i, [_P, _i, _f, _u64, _u64, _u32, _u32, _u32, _P]),
        "or_accept_seq": (_i, [_i, _i, _f, _P, _P, _P, _u64, _u64, _u32, _u32, _P, _P, _P, _P]),
        "or_quantize_rtn4": (None, [_P, _i, _i, _i, _P, _P]),
        "or_quantize_rtn4_asym": (None, [_P, _i, _i, _i, _P, _P, _P]),
        "or_quantize_rtn8": (None, [_P, _i, _i, _i, _P, _P]),
        "or_model_new": (_P, [_P, _i, _P]),
        "or_model_set_q4": (None, [_P, _i, _i, _P, _P, _i]),
        "or_model_set_quant": (None, [_P, _i, _i, _P, _P, _P, _i]),
        "or_model_free": (None, [_P]),
        "or_forward_seq": (None, [_P, _P, _P, _i, _P, _i, _i, _P]),
        "or_sd_step_seq": (_i, [_P, _P, _P, _P, _i, _i, _i32, _i, _f, _u64, _u64, _u32,
                                _P, _P, _P, _P, _P, _P, _P, _P]),
        "or_ar_step_seq": (_i32, [_P, _P, _P, _i, _i, _i32, _f, _u64, _u64, _u32, _P, _P]),
        "or_tau_from_alpha": (_d, [_d, _i]),
        "or_alpha_from_tau": (_d, [_d, _i]),
        "or_sd_speedup": (_d, [_d, _d, _d, _d, _i]),
        "or_cost_arch": (None, [_i, _i, _i, _i, _i, _i, _i, _d, _d, _d, _P]),
        "or_cost_times": (None, [_P, _d, _d, _i, _P, _P, _P]),
        "or_toggle": (_i, [_P, _d, _d, _d, _i, _d]),
        "or_toggle_sticky": (_i, [_P, _d, _d, _d, _i, _d, _P]),
        "or_gamma_next": (_i, [_P, _i, _i, _P, _i, _i, _d, _d]),
        "or_decode_breakdown": (None, [_i, _i, _i, _i, _i, _i, _i, _d, _d, _d, _d, _d, _d, _P]),
        "or_sample_hist": (None, [_P, _i, _f, _u64, _u64, _i, _P]),
        "or_accept_hist": (None, [_P, _P, _i, _f, _u64, _u64, _i, _P, _P]),
        "or_set_threads": (None, [_i]),
        "or_get_threads": (_i, []),
    }
    for name, (res, args) in sig.items():
        fn = getattr(L, name)
        fn.restype = res
        fn.argtypes = args
    return L


def _ptr(a: np.ndarray | None):
    if a is None:
        return None
    assert a.flags["C_CONTIGUOUS"]
    return a.ctypes.data_as(C.c_void_p)


def set_threads(n: int = 0):
    """Threads of the oracle's parallel loops (n <= 0: every host core)."""
    lib().or_set_threads(int(n))


def get_threads() -> int:
    return int(lib().or_get_threads())


# ---------------------------------------------------------------- scalars
def f32_to_f16(x: float) -> int:
    return int(lib().or_f32_to_f16(float(x)))


def f16_to_f32(h: int) -> float:
    return float(lib().or_f16_to_f32(int(h)))


def philox(ctr, key) -> np.ndarray:
    c = np.ascontiguousarray(np.asarray(ctr, dtype=np.uint64))
    k = np.ascontiguousarray(np.asarray(key, dtype=np.uint64))
    out = np.zeros(4, dtype=np.uint64)
    lib().or_philox4x64_10(_ptr(c), _ptr(k), _ptr(out))
    return out


def uniform_row(seed, step, stream, slot, pos, n) -> np.ndarray:
    u = np.zeros(n, dtype=np.float32)
    lib().or_uniform_row(seed, step, stream, slot, pos, n, _ptr(u))
    return u


def row_stats(logits: np.ndarray, T: float = 1.0):
    l = np.ascontiguousarray(logits, dtype=np.float32)
    m, lse = C.c_float(), C.c_float()
    lib().or_row_stats(_ptr(l), l.size, T, C.byref(m), C.byref(lse))
    return m.value, lse.value


def sample_row(logits, T, seed, step, stream, slot, pos):
    l = np.ascontiguousarray(logits, dtype=np.float32)
    gap = C.c_float()
    x = lib().or_sample_row(_ptr(l), l.size, T, seed, step, stream, slot, pos, C.byref(gap))
    return int(x), gap.value


def accept_seq(draft_tok, q_logits, p_logits, T, seed, step, slot, kv_len):
    """Returns (n_emit, out_tok[gamma+1], ratio[gamma], u[gamma], final_gap)."""
    d = np.ascontiguousarray(draft_tok, dtype=np.int32)
    q = np.ascontiguousarray(q_logits, dtype=np.float32)
    p = np.ascontiguousarray(p_logits, dtype=np.float32)
    gamma, V = q.shape
    assert p.shape == (gamma + 1, V)
    out = np.full(gamma + 1, -1, dtype=np.int32)
    ratio = np.zeros(gamma, dtype=np.float32)
    u = np.zeros(gamma, dtype=np.float32)
    gap = C.c_float()
    n = lib().or_accept_seq(V, gamma, T, _ptr(d), _ptr(q), _ptr(p), seed, step, slot, kv_len,
                            _ptr(out), _ptr(ratio), _ptr(u), C.byref(gap))
    return int(n), out, ratio, u, gap.value


def quantize_rtn4(w: np.ndarray, group: int = 128):
    w = np.ascontiguousarray(w, dtype=np.float32)
    N, K = w.shape
    codes = np.zeros((N, K), dtype=np.int8)
    scales = np.zeros((N, K // group), dtype=np.uint16)
    lib().or_quantize_rtn4(_ptr(w), N, K, group, _ptr(codes), _ptr(scales))
    return codes, scales


def quantize_rtn4_asym(w: np.ndarray, group: int = 128):
    w = np.ascontiguousarray(w, dtype=np.float32)
    N, K = w.shape
    codes = np.zeros((N, K), dtype=np.uint8)
    scales = np.zeros((N, K // group), dtype=np.uint16)
    zeros = np.zeros((N, K // group), dtype=np.uint8)
    lib().or_quantize_rtn4_asym(_ptr(w), N, K, group, _ptr(codes), _ptr(scales), _ptr(zeros))
    return codes, scales, zeros


def quantize_rtn8(w: np.ndarray, group: int = 128):
    w = np.ascontiguousarray(w, dtype=np.float32)
    N, K = w.shape
    codes = np.zeros((N, K), dtype=np.int8)
    scales = np.zeros((N, K // group), dtype=np.uint16)
    lib().or_quantize_rtn8(_ptr(w), N, K, group, _ptr(codes), _ptr(scales))
    return codes, scales


# drafter formats: RTN int4 symmetric (the default), int4 asymmetric, int8 symmetric
DRAFTER_FORMATS = ("w4", "w4a", "w8")


def quantize(w: np.ndarray, fmt: str = "w4", group: int = 128):
    """(codes, scales, zeros or None) of one weight matrix in drafter format fmt."""
    if fmt == "w4":
        return (*quantize_rtn4(w, group), None)
    if fmt == "w4a":
        return quantize_rtn4_asym(w, group)
    if fmt == "w8":
        return (*quantize_rtn8(w, group), None)
    raise ValueError(f"unknown drafter format {fmt!r}")


def f16_bits_to_f32(h: np.ndarray) -> np.ndarray:
    return np.ascontiguousarray(h, dtype=np.uint16).view(np.float16).astype(np.float32)


# ---------------------------------------------------------------- model
class Model:
    """A decoder whose weights live in numpy arrays (fp32 or bf16 bit patterns).

    ``tensors`` follows the library's binding order: embed, final_norm,
    lm_head, then per layer attn_norm, wqkv, wo, ffn_norm, wgu, wdown.
    """

    def __init__(self, cfg: dict, tensors, wkind: int):
        self.cfg = cfg
        self.c = Cfg(cfg["n_layers"], cfg["hidden"], cfg["n_q"], cfg["n_kv"], cfg["head_dim"],
                     cfg["ffn"], cfg["vocab"], cfg.get("rms_eps", 1e-5), cfg["rope_theta"])
        want = np.uint16 if wkind == BF16 else np.float32
        self._keep = [np.ascontiguousarray(t, dtype=want) for t in tensors]
        n = len(self._keep)
        assert n == 3 + 6 * cfg["n_layers"]
        self._ptrs = (C.c_void_p * n)(*[t.ctypes.data for t in self._keep])
        self.h = lib().or_model_new(C.byref(self.c), wkind, self._ptrs)

    def set_q4(self, layer: int, which: int, codes: np.ndarray, scales: np.ndarray, group=128):
        codes = np.ascontiguousarray(codes, dtype=np.int8)
        scales = np.ascontiguousarray(scales, dtype=np.uint16)
        self._keep += [codes, scales]
        lib().or_model_set_q4(self.h, layer, which, _ptr(codes), _ptr(scales), group)

    def set_quant(self, layer: int, which: int, codes: np.ndarray, scales: np.ndarray, zeros=None, group=128):
        codes = np.ascontiguousarray(codes).astype(np.int8)       # asymmetric codes 0..15 fit in int8
        scales = np.ascontiguousarray(scales, dtype=np.uint16)
        zeros = None if zeros is None else np.ascontiguousarray(zeros, dtype=np.uint8)
        self._keep += [codes, scales] + ([zeros] if zeros is not None else [])
        lib().or_model_set_quant(self.h, layer, which, _ptr(codes), _ptr(scales), _ptr(zeros), group)

    def __del__(self):
        try:
            if getattr(self, "h", None):
                lib().or_model_free(self.h)
        except Exception:
            pass

    # the projections quantized for the drafter, in (layer, which, tensor index) order
    def quant_targets(self):
        L = self.cfg["n_layers"]
        out = []
        for l in range(L):
            base = 3 + 6 * l
            out += [(l, 0, base + 1), (l, 1, base + 2), (l, 2, base + 4), (l, 3, base + 5)]
        return out


def tensor_f32(t: np.ndarray, wkind: int) -> np.ndarray:
    if wkind == BF16:
        return (np.ascontiguousarray(t, dtype=np.uint16).astype(np.uint32) << 16).view(np.float32)
    return np.ascontiguousarray(t, dtype=np.float32)


def make_drafter(cfg: dict, tensors, wkind: int, group: int = 128, fmt: str = "w4") -> Model:
    """RTN drafter: the same network with QKVO/FFN projections replaced by
    their group-`group` RTN codes (Sec. 4.1), int4 symmetric by default,
    int4 asymmetric ("w4a") or int8 ("w8") on request."""
    d = Model(cfg, tensors, wkind)
    for l, which, ti in d.quant_targets():
        codes, scales, zeros = quantize(tensor_f32(tensors[ti], wkind), fmt, group)
        if zeros is None and fmt == "w4":
            d.set_q4(l, which, codes, scales, group)
        else:
            d.set_quant(l, which, codes, scales, zeros, group)
    return d


class KV:
    """Per-sequence double-precision cache [L][n_kv][cap][head_dim]."""

    def __init__(self, cfg: dict, cap: int):
        shape = (cfg["n_layers"], cfg["n_kv"], cap, cfg["head_dim"])
        self.cap = cap
        self.k = np.zeros(shape, dtype=np.float64)
        self.v = np.zeros(shape, dtype=np.float64)

    def copy(self) -> "KV":
        o = KV.__new__(KV)
        o.cap, o.k, o.v = self.cap, self.k.copy(), self.v.copy()
        return o


def forward_seq(model: Model, kv: KV, tokens, start_pos: int, want_logits=True):
    tok = np.ascontiguousarray(tokens, dtype=np.int32)
    n = tok.size
    V = model.cfg["vocab"]
    logits = np.zeros((n, V), dtype=np.float32) if want_logits else None
    lib().or_forward_seq(model.h, _ptr(kv.k), _ptr(kv.v), kv.cap, _ptr(tok), start_pos, n, _ptr(logits))
    return logits


def sd_step_seq(target: Model, drafter: Model, kv: KV, kv_len: int, last_tok: int, gamma: int,
                T: float, seed: int, step: int, slot: int):
    V = target.cfg["vocab"]
    draft = np.zeros(gamma, dtype=np.int32)
    q = np.zeros((gamma, V), dtype=np.float32)
    p = np.zeros((gamma + 1, V), dtype=np.float32)
    out = np.full(gamma + 1, -1, dtype=np.int32)
    dgap = np.zeros(gamma, dtype=np.float32)
    ratio = np.zeros(gamma, dtype=np.float32)
    u = np.zeros(gamma, dtype=np.float32)
    fgap = C.c_float()
    n = lib().or_sd_step_seq(target.h, drafter.h, _ptr(kv.k), _ptr(kv.v), kv.cap, kv_len, int(last_tok),
                             gamma, T, seed, step, slot, _ptr(draft), _ptr(q), _ptr(p), _ptr(out),
                             _ptr(dgap), _ptr(ratio), _ptr(u), C.byref(fgap))
    return dict(n_emit=int(n), draft=draft, q=q, p=p, out=out[:n].copy(), out_full=out,
                draft_gap=dgap, ratio=ratio, u=u, final_gap=fgap.value)


def ar_step_seq(target: Model, kv: KV, kv_len: int, last_tok: int, T: float, seed: int, step: int,
                slot: int):
    V = target.cfg["vocab"]
    p = np.zeros(V, dtype=np.float32)
    gap = C.c_float()
    x = lib().or_ar_step_seq(target.h, _ptr(kv.k), _ptr(kv.v), kv.cap, kv_len, int(last_tok), T,
                             seed, step, slot, _ptr(p), C.byref(gap))
    return int(x), p, gap.value


# ---------------------------------------------------------------- host policy
def tau_from_alpha(alpha, gamma):
    return lib().or_tau_from_alpha(alpha, gamma)


def alpha_from_tau(tau, gamma):
    return lib().or_alpha_from_tau(tau, gamma)


def sd_speedup(tau, Tp, Tq, Tv, gamma):
    return lib().or_sd_speedup(tau, Tp, Tq, Tv, gamma)


def cost_arch(L, H, nq, nkv, d, F, V, tbytes=2.0, dbits=4.0, kvbytes=2.0, **calib) -> Cost:
    c = Cost()
    lib().or_cost_arch(L, H, nq, nkv, d, F, V, tbytes, dbits, kvbytes, C.byref(c))
    c.BW_eff = calib.get("BW_eff", 1.0)
    c.F_eff = calib.get("F_eff", 1.0)
    c.rho_kappa = calib.get("rho_kappa", 1.0)
    c.eta_D = calib.get("eta_D", 1.0)
    c.c_T = calib.get("c_T", 0.0)
    c.c_D = calib.get("c_D", 0.0)
    c.c_V = calib.get("c_V", 0.0)
    return c


def cost_times(c: Cost, B, S, gamma):
    tp, tq, tv = C.c_double(), C.c_double(), C.c_double()
    lib().or_cost_times(C.byref(c), B, S, gamma, C.byref(tp), C.byref(tq), C.byref(tv))
    return tp.value, tq.value, tv.value


def toggle(c: Cost, B, S, tau, gamma, eps=0.05) -> int:
    return int(lib().or_toggle(C.byref(c), B, S, tau, gamma, eps))


def toggle_sticky(c: Cost, B, S, tau, gamma, eps, state: list) -> int:
    s = C.c_int(state[0])
    r = lib().or_toggle_sticky(C.byref(c), B, S, tau, gamma, eps, C.byref(s))
    state[0] = s.value
    return int(r)


def gamma_next(gset, gamma, hist, P=2, a_up=0.94, a_down=0.85) -> int:
    s = np.ascontiguousarray(gset, dtype=np.int32)
    h = np.ascontiguousarray(hist, dtype=np.float64)
    return int(lib().or_gamma_next(_ptr(s), s.size, gamma, _ptr(h) if h.size else None, h.size, P,
                                   a_up, a_down))


def decode_breakdown(L, H, nq, nkv, d, F, V, B, S, wbytes=2.0, kvbytes=2.0, flops=312e12,
                     bw=2.039e12) -> np.ndarray:
    out = np.zeros(4, dtype=np.float64)
    lib().or_decode_breakdown(L, H, nq, nkv, d, F, V, wbytes, kvbytes, B, S, flops, bw, _ptr(out))
    return out


def sample_hist(logits, T, seed, step, n) -> np.ndarray:
    l = np.ascontiguousarray(logits, dtype=np.float32)
    counts = np.zeros(l.size, dtype=np.int64)
    lib().or_sample_hist(_ptr(l), l.size, T, seed, step, n, _ptr(counts))
    return counts


def accept_hist(q_row, p1, p2, T, seed, step, n):
    q = np.ascontiguousarray(q_row, dtype=np.float32)
    p12 = np.ascontiguousarray(np.stack([p1, p2]), dtype=np.float32)
    counts = np.zeros(q.size, dtype=np.int64)
    nacc = C.c_int64()
    lib().or_accept_hist(_ptr(q), _ptr(p12), q.size, T, seed, step, n, _ptr(counts), C.byref(nacc))
    return counts, nacc.value
