"""Thin Python binding of the C ABI in ``include/sd_api.h``.

Argument marshalling only: torch supplies device memory and the current
stream; every step of the SD path runs in the library's HIP kernels.  The
binding checks shapes, dtypes, devices and contiguity of every buffer before
handing raw pointers to the library, so a wrongly sized buffer is a Python
error instead of an out-of-bounds write on the GPU.

The library must have been built (``paper_2606_18967_amd/build.py`` or
``__graft_entry__.build()``); there is no fallback path.
"""
from __future__ import annotations

import ctypes as C
import os

import torch

HERE = os.path.dirname(os.path.abspath(__file__))
# SDRL_LIB may name another build of the same library (e.g. one compiled with
# different tile constants); by default the in-tree build is loaded.
LIB_PATH = os.environ.get("SDRL_LIB") or os.path.join(HERE, "_build", "libsdrl.so")

SD_OK, SD_E_INVAL, SD_E_NOMEM, SD_E_HIP, SD_E_STATE, SD_E_UNSUPPORTED = range(6)
SD_DTYPE_F32, SD_DTYPE_BF16 = 0, 1

# The names every build must export (one per declaration in include/sd_api.h).
API_SYMBOLS = (
    "sd_last_error", "sd_create", "sd_destroy", "sd_num_weights", "sd_bind_weights", "sd_kv_bytes",
    "sd_bind_kv", "sd_kv_page_bytes", "sd_bind_kv_paged", "sd_drafter_bytes", "sd_drafter_bytes_fmt", "sd_refresh_drafter", "sd_refresh_drafter_fmt",
    "sd_prefill", "sd_prefill_ragged", "sd_draft", "sd_verify",
    "sd_accept", "kv_rollback", "sd_ar_step", "sd_sync", "sd_set_debug", "sd_cost_init",
    "sd_cost_times", "sd_toggle", "sd_gamma_init", "sd_gamma_next", "sd_tau_from_alpha",
    "sd_alpha_from_tau", "sd_timing", "sd_timing_read", "sd_dense_gemm_bf16", "sd_accept_noalloc",
)

# kernel classes of sd_timing_read
T_ATTN_D, T_ATTN_V, T_Q4, T_PROJ, T_LMHEAD, T_SAMPLE, T_ACCEPT, T_MISC = range(8)

# drafter weight formats (sd_draft_fmt): int4 symmetric, int4 asymmetric, int8
DRAFT_FORMATS = {"w4": 0, "w4a": 1, "w8": 2}
T_NAMES = ("attn_decode", "attn_verify", "int4_proj", "bf16_proj", "lm_head", "sampler", "accept", "misc")


class SDError(RuntimeError):
    def __init__(self, status: int, msg: str):
        super().__init__(f"sd status {status}: {msg}")
        self.status = status


class ModelCfg(C.Structure):
    _fields_ = [("n_layers", C.c_int32), ("hidden", C.c_int32), ("n_q", C.c_int32), ("n_kv", C.c_int32),
                ("head_dim", C.c_int32), ("ffn", C.c_int32), ("vocab", C.c_int32), ("dtype", C.c_int32),
                ("group", C.c_int32), ("rms_eps", C.c_float), ("rope_theta", C.c_float)]


class Rng(C.Structure):
    _fields_ = [("seed", C.c_uint64), ("step", C.c_uint64)]


class CostModel(C.Structure):
    _fields_ = [(n, C.c_double) for n in
                ("W_T", "W_D", "kappa_th", "C_dense", "C_attn",
                 "BW_eff", "F_eff", "rho_kappa", "eta_D", "c_T", "c_D", "c_V")]


class GammaCtl(C.Structure):
    _fields_ = [("set", C.c_int32 * 16), ("n_set", C.c_int32), ("P", C.c_int32), ("gamma", C.c_int32),
                ("n_hist", C.c_int32), ("a_up", C.c_double), ("a_down", C.c_double),
                ("hist", C.c_double * 64)]


_lib = None
_P, _i32, _f, _d, _sz = C.c_void_p, C.c_int32, C.c_float, C.c_double, C.c_size_t


def lib():
    """Loads the built library; raises if it has not been built."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise ImportError(f"{LIB_PATH} is missing: build it with paper_2606_18967_amd/build.py")
        L = C.CDLL(LIB_PATH)
        sig = {
            "sd_last_error": (C.c_char_p, []),
            "sd_create": (_i32, [_P, _i32, _i32, _i32, _P]),
            "sd_destroy": (_i32, [_P]),
            "sd_num_weights": (_i32, [_P]),
            "sd_bind_weights": (_i32, [_P, _P, _i32]),
            "sd_kv_bytes": (_sz, [_P, _i32, _i32]),
            "sd_bind_kv": (_i32, [_P, _P, _P, _P]),
            "sd_drafter_bytes": (_sz, [_P]),
            "sd_refresh_drafter": (_i32, [_P, _P, _sz, _P]),
            "sd_kv_page_bytes": (_sz, [_P, _i32]),
            "sd_bind_kv_paged": (_i32, [_P, _P, _P, _i32, _i32, _P, _i32, _P]),
            "sd_drafter_bytes_fmt": (_sz, [_P, _i32]),
            "sd_refresh_drafter_fmt": (_i32, [_P, _i32, _P, _sz, _P]),
            "sd_prefill": (_i32, [_P, _i32, _P, _P, _i32, _P]),
            "sd_prefill_ragged": (_i32, [_P, _i32, _P, _P, _i32, _P, _P]),
            "sd_draft": (_i32, [_P, _i32, _P, _P, _i32, _f, Rng, _P, _P, _P, _P]),
            "sd_verify": (_i32, [_P, _i32, _P, _P, _P, _i32, _P, _P]),
            "sd_accept": (_i32, [_P, _i32, _P, _P, _P, _P, _P, _i32, _f, Rng, _P, _P, _P, _P]),
            "sd_accept_noalloc": (_i32, [_i32, _i32, _P, _P, _i32, _P, _P, _P, _P, _i32, _f, Rng, _P, _P, _P, _P]),
            "kv_rollback": (_i32, [_P, _i32, _P, _P, _P]),
            "sd_ar_step": (_i32, [_P, _i32, _P, _P, _f, Rng, _P, _P, _P]),
            "sd_sync": (_i32, [_P, _P]),
            "sd_set_debug": (_i32, [_P, _i32]),
            "sd_timing": (_i32, [_P, _i32]),
            "sd_timing_read": (_i32, [_P, _i32, _P, _P]),
            "sd_dense_gemm_bf16": (_i32, [_P, _P, _P, _i32, _i32, _i32, _P]),
            "sd_cost_init": (_i32, [_P, _d, _d, _d, _P]),
            "sd_cost_times": (_i32, [_P, _d, _d, _i32, _P, _P, _P]),
            "sd_toggle": (_i32, [_P, _i32, _d, _d, _i32, _d, _P]),
            "sd_gamma_init": (_i32, [_P, _P, _i32, _i32, _d, _d]),
            "sd_gamma_next": (_i32, [_P, _d, _P]),
            "sd_tau_from_alpha": (_d, [_d, _i32]),
            "sd_alpha_from_tau": (_d, [_d, _i32]),
        }
        for name, (res, args) in sig.items():
            fn = getattr(L, name)
            fn.restype, fn.argtypes = res, args
        _lib = L
    return _lib


def _check(st: int):
    if st != SD_OK:
        raise SDError(st, lib().sd_last_error().decode(errors="replace"))


def model_cfg(cfg: dict) -> ModelCfg:
    dt = SD_DTYPE_BF16 if cfg["dtype"] in ("bf16", SD_DTYPE_BF16) else SD_DTYPE_F32
    return ModelCfg(cfg["n_layers"], cfg["hidden"], cfg["n_q"], cfg["n_kv"], cfg["head_dim"], cfg["ffn"],
                    cfg["vocab"], dt, cfg.get("group", 128), cfg.get("rms_eps", 1e-5), cfg["rope_theta"])


def torch_dtype(cfg: dict):
    return torch.bfloat16 if cfg["dtype"] in ("bf16", SD_DTYPE_BF16) else torch.float32


def _dev(t: torch.Tensor, name: str, dtype=None, shape=None, dev=None):
    if not isinstance(t, torch.Tensor) or not t.is_cuda:
        raise ValueError(f"{name}: expected a device tensor")
    if dtype is not None and t.dtype != dtype:
        raise ValueError(f"{name}: expected {dtype}, got {t.dtype}")
    if shape is not None and tuple(t.shape) != tuple(shape):
        raise ValueError(f"{name}: expected shape {tuple(shape)}, got {tuple(t.shape)}")
    if not t.is_contiguous():
        raise ValueError(f"{name}: must be contiguous")
    if dev is not None and t.device != dev:
        raise ValueError(f"{name}: on {t.device}, engine is on {dev}")
    return C.c_void_p(t.data_ptr())


def _stream():
    return C.c_void_p(torch.cuda.current_stream().cuda_stream)


class Engine:
    """One SD engine on the current device; buffers are torch device tensors."""

    def __init__(self, cfg: dict, max_slots: int, max_ctx: int, max_gamma: int):
        self.cfg = dict(cfg)
        self.c = model_cfg(cfg)
        self.max_slots, self.max_ctx, self.max_gamma = max_slots, max_ctx, max_gamma
        self.device = torch.device("cuda", torch.cuda.current_device())
        self.wdtype = torch_dtype(cfg)
        h = C.c_void_p()
        _check(lib().sd_create(C.byref(self.c), max_slots, max_ctx, max_gamma, C.byref(h)))
        self.h = h
        self._keep = []

    def close(self):
        if getattr(self, "h", None):
            lib().sd_destroy(self.h)
            self.h = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    # ---------------------------------------------------------------- binding
    def weight_shapes(self):
        c = self.cfg
        H, V, d, F = c["hidden"], c["vocab"], c["head_dim"], c["ffn"]
        qkv = (c["n_q"] + 2 * c["n_kv"]) * d
        shapes = [(V, H), (H,), (V, H)]
        for _ in range(c["n_layers"]):
            shapes += [(H,), (qkv, H), (H, c["n_q"] * d), (H,), (2 * F, H), (H, F)]
        return shapes

    def bind_weights(self, tensors):
        shapes = self.weight_shapes()
        if len(tensors) != len(shapes):
            raise ValueError(f"expected {len(shapes)} tensors")
        ptrs = (C.c_void_p * len(tensors))(
            *[_dev(t, f"weight[{i}]", self.wdtype, shapes[i], self.device).value for i, t in enumerate(tensors)])
        _check(lib().sd_bind_weights(self.h, ptrs, len(tensors)))
        self._keep_w = list(tensors)

    def kv_shape(self):
        c = self.cfg
        return (c["n_layers"], self.max_slots, c["n_kv"], self.max_ctx, c["head_dim"])

    def alloc_kv(self):
        k = torch.zeros(self.kv_shape(), dtype=self.wdtype, device=self.device)
        v = torch.zeros_like(k)
        kv_len = torch.zeros(self.max_slots, dtype=torch.int32, device=self.device)
        return k, v, kv_len

    def bind_kv(self, k, v, kv_len):
        shp = self.kv_shape()
        _check(lib().sd_bind_kv(self.h, _dev(k, "k", self.wdtype, shp, self.device),
                                _dev(v, "v", self.wdtype, shp, self.device),
                                _dev(kv_len, "kv_len", torch.int32, (self.max_slots,), self.device)))
        self._keep_kv = (k, v, kv_len)

    def alloc_kv_paged(self, n_pages: int, page_size: int):
        """K and V page pools [n_pages][L][n_kv][page_size][head_dim] and kv_len."""
        c = self.cfg
        shp = (n_pages, c["n_layers"], c["n_kv"], page_size, c["head_dim"])
        k = torch.zeros(shp, dtype=self.wdtype, device=self.device)
        v = torch.zeros(shp, dtype=self.wdtype, device=self.device)
        kv_len = torch.zeros(self.max_slots, dtype=torch.int32, device=self.device)
        return k, v, kv_len

    def bind_kv_paged(self, k, v, block_table, kv_len):
        """Paged cache: pools from alloc_kv_paged and an int32 block table
        [max_slots][pages_per_seq] of page indices (both caller-owned)."""
        n_pages, page_size = k.shape[0], k.shape[3]
        c = self.cfg
        shp = (n_pages, c["n_layers"], c["n_kv"], page_size, c["head_dim"])
        pps = block_table.shape[1]
        _check(lib().sd_bind_kv_paged(self.h, _dev(k, "k", self.wdtype, shp, self.device),
                                      _dev(v, "v", self.wdtype, shp, self.device), n_pages, page_size,
                                      _dev(block_table, "block_table", torch.int32, (self.max_slots, pps), self.device),
                                      pps, _dev(kv_len, "kv_len", torch.int32, (self.max_slots,), self.device)))
        self._keep_kv = (k, v, block_table, kv_len)

    def drafter_bytes(self, fmt: str = "w4") -> int:
        return int(lib().sd_drafter_bytes_fmt(C.byref(self.c), DRAFT_FORMATS[fmt]))

    def refresh_drafter(self, qbuf: torch.Tensor | None = None, fmt: str = "w4") -> torch.Tensor:
        """RTN-quantizes the bound target into the drafter (format "w4", "w4a"
        or "w8"); returns the caller-owned buffer the drafter reads."""
        n = self.drafter_bytes(fmt)
        if qbuf is None:
            qbuf = torch.empty(n, dtype=torch.uint8, device=self.device)
        if qbuf.numel() * qbuf.element_size() < n:
            raise ValueError("qbuf too small")
        _check(lib().sd_refresh_drafter_fmt(self.h, DRAFT_FORMATS[fmt], _dev(qbuf, "qbuf", None, None, self.device),
                                            qbuf.numel() * qbuf.element_size(), _stream()))
        self._keep_q = qbuf
        self.drafter_fmt = fmt
        return qbuf

    def set_debug(self, poison: bool, unfused_swiglu: bool = False, staged_tiles: bool = False):
        _check(lib().sd_set_debug(self.h, (1 if poison else 0) | (2 if unfused_swiglu else 0) |
                                  (4 if staged_tiles else 0)))

    # ---------------------------------------------------------------- steps
    def _slots(self, slots):
        B = slots.numel()
        if B < 1 or B > self.max_slots:
            raise ValueError("bad batch")
        return B, _dev(slots, "slots", torch.int32, (B,), self.device)

    def prefill(self, slots, tokens):
        B, sp = self._slots(slots)
        n = tokens.shape[1]
        _check(lib().sd_prefill(self.h, B, sp, _dev(tokens, "tokens", torch.int32, (B, n), self.device), n,
                                _stream()))

    def prefill_ragged(self, slots, tokens, lens):
        """Caches tokens[b, :lens[b]] of each sequence; tokens is [B][ld], lens [B] (device int32)."""
        B, sp = self._slots(slots)
        ld = tokens.shape[1]
        _check(lib().sd_prefill_ragged(self.h, B, sp, _dev(tokens, "tokens", torch.int32, (B, ld), self.device), ld,
                                       _dev(lens, "lens", torch.int32, (B,), self.device), _stream()))

    def draft(self, slots, last_tok, gamma, T, seed, step, draft_tok, q_logits, q_stats):
        B, sp = self._slots(slots)
        V = self.cfg["vocab"]
        _check(lib().sd_draft(self.h, B, sp, _dev(last_tok, "last_tok", torch.int32, (B,), self.device), gamma,
                              T, Rng(seed, step),
                              _dev(draft_tok, "draft_tok", torch.int32, (B, gamma), self.device),
                              _dev(q_logits, "q_logits", torch.float32, (B, gamma, V), self.device),
                              _dev(q_stats, "q_stats", torch.float32, (B, gamma, 2), self.device), _stream()))

    def verify(self, slots, last_tok, draft_tok, gamma, p_logits):
        B, sp = self._slots(slots)
        V = self.cfg["vocab"]
        _check(lib().sd_verify(self.h, B, sp, _dev(last_tok, "last_tok", torch.int32, (B,), self.device),
                               _dev(draft_tok, "draft_tok", torch.int32, (B, gamma), self.device), gamma,
                               _dev(p_logits, "p_logits", torch.float32, (B, gamma + 1, V), self.device),
                               _stream()))

    def accept(self, slots, draft_tok, q_logits, q_stats, p_logits, gamma, T, seed, step, out_tok, n_emit,
               next_tok=None):
        B, sp = self._slots(slots)
        V = self.cfg["vocab"]
        nt = _dev(next_tok, "next_tok", torch.int32, (B,), self.device) if next_tok is not None else None
        _check(lib().sd_accept(self.h, B, sp, _dev(draft_tok, "draft_tok", torch.int32, (B, gamma), self.device),
                               _dev(q_logits, "q_logits", torch.float32, (B, gamma, V), self.device),
                               _dev(q_stats, "q_stats", torch.float32, (B, gamma, 2), self.device),
                               _dev(p_logits, "p_logits", torch.float32, (B, gamma + 1, V), self.device),
                               gamma, T, Rng(seed, step),
                               _dev(out_tok, "out_tok", torch.int32, (B, gamma + 1), self.device),
                               _dev(n_emit, "n_emit", torch.int32, (B,), self.device), nt, _stream()))

    def rollback(self, slots, n_emit):
        B, sp = self._slots(slots)
        _check(lib().kv_rollback(self.h, B, sp, _dev(n_emit, "n_emit", torch.int32, (B,), self.device), _stream()))

    def ar_step(self, slots, last_tok, T, seed, step, out_tok, p_logits):
        B, sp = self._slots(slots)
        V = self.cfg["vocab"]
        _check(lib().sd_ar_step(self.h, B, sp, _dev(last_tok, "last_tok", torch.int32, (B,), self.device), T,
                                Rng(seed, step), _dev(out_tok, "out_tok", torch.int32, (B,), self.device),
                                _dev(p_logits, "p_logits", torch.float32, (B, V), self.device), _stream()))

    def sync(self):
        _check(lib().sd_sync(self.h, _stream()))

    def timing(self, on: bool):
        _check(lib().sd_timing(self.h, 1 if on else 0))

    def timing_read(self, cls: int):
        ms, n = C.c_double(), C.c_int32()
        _check(lib().sd_timing_read(self.h, cls, C.byref(ms), C.byref(n)))
        return ms.value, n.value


class SDBuffers:
    """Device buffers of one SD step for B sequences and draft length gamma."""

    def __init__(self, eng: Engine, B: int, gamma: int):
        dev, V = eng.device, eng.cfg["vocab"]
        self.B, self.gamma = B, gamma
        self.draft_tok = torch.zeros((B, gamma), dtype=torch.int32, device=dev)
        self.q_logits = torch.zeros((B, gamma, V), dtype=torch.float32, device=dev)
        self.q_stats = torch.zeros((B, gamma, 2), dtype=torch.float32, device=dev)
        self.p_logits = torch.zeros((B, gamma + 1, V), dtype=torch.float32, device=dev)
        self.out_tok = torch.zeros((B, gamma + 1), dtype=torch.int32, device=dev)
        self.n_emit = torch.zeros((B,), dtype=torch.int32, device=dev)
        self.next_tok = torch.zeros((B,), dtype=torch.int32, device=dev)


def sd_step(eng: Engine, bufs: SDBuffers, slots, last_tok, T, seed, step):
    """One SD iteration: gamma drafts, verify, accept, rollback.  Leaves the
    next last token of each sequence in bufs.next_tok."""
    g = bufs.gamma
    eng.draft(slots, last_tok, g, T, seed, step, bufs.draft_tok, bufs.q_logits, bufs.q_stats)
    eng.verify(slots, last_tok, bufs.draft_tok, g, bufs.p_logits)
    eng.accept(slots, bufs.draft_tok, bufs.q_logits, bufs.q_stats, bufs.p_logits, g, T, seed, step,
               bufs.out_tok, bufs.n_emit, bufs.next_tok)
    eng.rollback(slots, bufs.n_emit)


class StepGraph:
    """One SD step for a fixed batch (slots, last_tok, buffers, gamma, T and
    the Philox key), captured once as a HIP graph through torch: draft,
    verify, accept, rollback, then last_tok <- next_tok.  Every launch of the
    step takes its positions from kv_len on the device, so each replay
    advances the sequences exactly as the eager calls would.  Call after at
    least one eager step (kernels loaded); timing must be off while capturing.
    replay() enqueues the step on the current stream; the host still reads
    n_emit from bufs after it."""

    def __init__(self, eng: Engine, bufs: SDBuffers, slots, last_tok, T, seed, step):
        self.eng, self.bufs, self.slots, self.last_tok = eng, bufs, slots, last_tok
        self.graph = torch.cuda.CUDAGraph()
        side = torch.cuda.Stream(device=eng.device)            # default priority
        side.wait_stream(torch.cuda.current_stream())
        with torch.cuda.graph(self.graph, stream=side):
            sd_step(eng, bufs, slots, last_tok, T, seed, step)
            torch.add(bufs.next_tok, 0, out=last_tok)             # a kernel node, not a copy node
        torch.cuda.current_stream().wait_stream(side)

    def replay(self):
        self.graph.replay()


def accept_noalloc(slots, kv_len, draft_tok, q_logits, q_stats, p_logits, gamma, T, seed, step, out_tok, n_emit,
                   next_tok=None):
    """sd_accept_noalloc: the rejection sampler with no engine and no device
    allocation (its scratch is the library's static per-GPU array).  kv_len
    is the caller's int32 [max_slots] cache-length array; the other buffers
    as Engine.accept."""
    B = slots.numel()
    V = q_logits.shape[-1]
    dev = slots.device
    nt = _dev(next_tok, "next_tok", torch.int32, (B,), dev) if next_tok is not None else None
    _check(lib().sd_accept_noalloc(B, V, _dev(slots, "slots", torch.int32, (B,), dev),
                                   _dev(kv_len, "kv_len", torch.int32, None, dev), kv_len.numel(),
                                   _dev(draft_tok, "draft_tok", torch.int32, (B, gamma), dev),
                                   _dev(q_logits, "q_logits", torch.float32, (B, gamma, V), dev),
                                   _dev(q_stats, "q_stats", torch.float32, (B, gamma, 2), dev),
                                   _dev(p_logits, "p_logits", torch.float32, (B, gamma + 1, V), dev),
                                   gamma, T, Rng(seed, step),
                                   _dev(out_tok, "out_tok", torch.int32, (B, gamma + 1), dev),
                                   _dev(n_emit, "n_emit", torch.int32, (B,), dev), nt, _stream()))


def dense_gemm_bf16(A: torch.Tensor, W: torch.Tensor, out: torch.Tensor):
    """out[M][N] (fp32) = A[M][K] W[N][K]^T with the library's bf16 GEMM kernels."""
    M, K = A.shape
    N = W.shape[0]
    _check(lib().sd_dense_gemm_bf16(_dev(A, "A", torch.bfloat16, (M, K)), _dev(W, "W", torch.bfloat16, (N, K)),
                                    _dev(out, "out", torch.float32, (M, N)), M, N, K, _stream()))


# -------------------------------------------------------------------- host policy
def cost_init(cfg: dict, weight_bytes=2.0, drafter_bits=4.0, kv_bytes=2.0, **calib) -> CostModel:
    m = CostModel()
    _check(lib().sd_cost_init(C.byref(model_cfg(cfg)), weight_bytes, drafter_bits, kv_bytes, C.byref(m)))
    for k, v in calib.items():
        setattr(m, k, v)
    return m


def cost_times(m: CostModel, B, S, gamma):
    tp, tq, tv = C.c_double(), C.c_double(), C.c_double()
    _check(lib().sd_cost_times(C.byref(m), B, S, gamma, C.byref(tp), C.byref(tq), C.byref(tv)))
    return tp.value, tq.value, tv.value


def toggle(m: CostModel, B, S, tau, gamma, eps, sd_on: int = 0) -> int:
    s = C.c_int32(sd_on)
    r = lib().sd_toggle(C.byref(m), B, S, tau, gamma, eps, C.byref(s))
    if r < 0:
        raise ValueError("sd_toggle: bad argument")
    return int(r)


class GammaController:
    def __init__(self, gset=(5, 7, 9, 11), P=2, a_up=0.94, a_down=0.85):
        self.c = GammaCtl()
        arr = (C.c_int32 * len(gset))(*gset)
        _check(lib().sd_gamma_init(C.byref(self.c), arr, len(gset), P, a_up, a_down))

    @property
    def gamma(self) -> int:
        return int(self.c.gamma)

    def update(self, tau: float) -> int:
        g = C.c_int32()
        _check(lib().sd_gamma_next(C.byref(self.c), tau, C.byref(g)))
        return int(g.value)


def tau_from_alpha(alpha, gamma):
    return lib().sd_tau_from_alpha(alpha, gamma)


def alpha_from_tau(tau, gamma):
    return lib().sd_alpha_from_tau(tau, gamma)
