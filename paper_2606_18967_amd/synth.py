"""Seeded synthetic inputs shared by the tests, the smoke check and the
benchmark: model shapes, random weights, prompt tokens and random KV context.

This module holds none of the method's arithmetic; it only draws random
tensors.  The paper trains and samples real Qwen2.5 / Llama3.1 checkpoints on
math datasets; here random-init weights of the same decoder family and random
token ids stand in for them.

Recipe: every linear weight and the embedding ~ N(0, 0.02), norm gains = 1,
drawn in the binding order (embed, final_norm, lm_head, then per layer
attn_norm, wqkv, wo, ffn_norm, wgu, wdown) from one torch generator seeded
with `seed` on the target device.  Prompt tokens are uniform in [0, vocab).
Random KV context is N(0, 1) for the keys (taken as post-RoPE) and values.
"""
from __future__ import annotations

import torch

# Llama-style decoders; rope_theta 1e4 for the tiny model, 5e5 for the 8B shape, 1e6 for the 32B shape.
TINY = dict(name="tiny-2L-h256", n_layers=2, hidden=256, n_q=4, n_kv=4, head_dim=64, ffn=1024, vocab=512,
            dtype="f32", rope_theta=10000.0, rms_eps=1e-5)
L4_8B = dict(name="8B-shape-4L", n_layers=4, hidden=4096, n_q=32, n_kv=8, head_dim=128, ffn=14336, vocab=128256,
             dtype="bf16", rope_theta=500000.0, rms_eps=1e-5)
L32_8B = dict(L4_8B, name="8B-shape-32L", n_layers=32)
L64_32B = dict(name="32B-shape-64L", n_layers=64, hidden=5120, n_q=40, n_kv=8, head_dim=128, ffn=27648,
               vocab=152064, dtype="bf16", rope_theta=1000000.0, rms_eps=1e-5)

# Workloads (batch, context, draft length, temperature).
TINY_RUN = dict(B=4, prompt=64, context=128, gamma=4, T=1.0, seed=0)
L4_8B_RUN = dict(B=64, context=2048, gamma=4, T=1.0, seed=1)
L32_8B_RUN = dict(B=64, context=2048, gamma=4, T=1.0, seed=2)
# the 64-layer 32B shape at B = 128 and 8192 positions needs ~360 GB; one GPU
# holds it at B = 64 and 8192 positions (~224 GB with weights and drafter)
L64_32B_RUN = dict(B=64, context=8192, gamma=4, T=1.0, seed=5)


def weight_shapes(cfg: dict):
    H, V, d, F = cfg["hidden"], cfg["vocab"], cfg["head_dim"], cfg["ffn"]
    qkv = (cfg["n_q"] + 2 * cfg["n_kv"]) * d
    shapes = [(V, H), (H,), (V, H)]
    for _ in range(cfg["n_layers"]):
        shapes += [(H,), (qkv, H), (H, cfg["n_q"] * d), (H,), (2 * F, H), (H, F)]
    return shapes


def is_norm(i: int) -> bool:
    return i == 1 or (i >= 3 and (i - 3) % 6 in (0, 3))


def make_weights(cfg: dict, seed: int, device="cpu", std: float = 0.02):
    dtype = torch.bfloat16 if cfg["dtype"] == "bf16" else torch.float32
    g = torch.Generator(device=device).manual_seed(seed)
    out = []
    for i, shp in enumerate(weight_shapes(cfg)):
        if is_norm(i):
            out.append(torch.ones(shp, dtype=dtype, device=device))
        else:
            t = torch.randn(shp, generator=g, device=device, dtype=torch.float32)
            t.mul_(std)
            out.append(t.to(dtype))
            del t
    return out


def make_tokens(B: int, n: int, vocab: int, seed: int) -> torch.Tensor:
    g = torch.Generator().manual_seed(seed)
    return torch.randint(0, vocab, (B, n), generator=g, dtype=torch.int64).to(torch.int32)


def fill_kv_context(k: torch.Tensor, v: torch.Tensor, S: int, seed: int):
    """Fills positions [0, S) of every layer/slot/head of the [L][slots][n_kv]
    [ctx][d] caches with N(0, 1) draws (in place)."""
    g = torch.Generator(device=k.device).manual_seed(seed)
    for t in (k, v):
        for l in range(t.shape[0]):
            src = torch.randn(t[l, :, :, :S, :].shape, generator=g, device=k.device, dtype=torch.float32)
            t[l, :, :, :S, :].copy_(src.to(t.dtype))
            del src


def to_numpy_bits(t: torch.Tensor):
    """Host copy for the oracle: fp32 as float32, bf16 as raw uint16 bits."""
    t = t.detach().cpu().contiguous()
    if t.dtype == torch.bfloat16:
        return t.view(torch.int16).numpy().view("uint16")
    return t.numpy()
