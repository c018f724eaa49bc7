"""GPU parity of single SD stages through the C ABI:
  - the drafter refresh in every format (RTN int4 symmetric and asymmetric,
    int8: codes, fp16 scales and zero points bit-exact with the oracle,
    unpacked from the documented tile layouts);
  - speculative rejection sampling on identical logits (decisions identical
    to the oracle's except at documented near-ties), for one and for many
    vocabulary chunks;
  - device range errors are reported by sd_sync without touching memory out
    of bounds."""
import numpy as np
import pytest
import torch

import oracle
from oracle.parity import check_accept, drafter_layout, unpack_q4, unpack_q8, unpack_zeros
from paper_2606_18967_amd import sdrl, synth

from gpu_common import host_bits, i32, make_engine, say

pytestmark = pytest.mark.gpu

SMALL_BF16 = dict(name="small-bf16", n_layers=2, hidden=256, n_q=4, n_kv=2, head_dim=64, ffn=512, vocab=256,
                  dtype="bf16", rope_theta=500000.0, rms_eps=1e-5)


@pytest.mark.parametrize("fmt", ["w4", "w4a", "w8"])
@pytest.mark.parametrize("cfg", [synth.TINY, SMALL_BF16], ids=["tiny-f32", "small-bf16"])
def test_refresh_drafter_bit_exact(cfg, fmt):
    say("refresh_drafter", cfg["name"], fmt)
    W = synth.make_weights(cfg, 5, "cpu")
    # edge groups: all zero, huge magnitude, tiny magnitude, constant
    W[4][3, 128:256] = 0
    W[4][5, :128] *= 1000
    W[8][1, 0:128] *= 1e-4
    W[8][2, 128:256] = 0.01
    Wd = [w.cuda() for w in W]
    eng, *_ = make_engine(cfg, Wd, 1, 8, 1)
    qbuf = eng.refresh_drafter(fmt=fmt)
    torch.cuda.synchronize()
    host = qbuf.cpu().numpy()
    Wh = host_bits(W)
    kind = oracle.BF16 if cfg["dtype"] == "bf16" else oracle.F32
    layout, total = drafter_layout(cfg, fmt)
    assert total == host.size
    widx = [1, 2, 4, 5]
    for l, w, N, K, co, so, zo in layout:
        nc = N * K // (1 if fmt == "w8" else 2)
        if fmt == "w8":
            codes, sc = unpack_q8(host[co:co + nc], host[so:so + N * (K // 128) * 2], N, K)
        else:
            codes, sc = unpack_q4(host[co:co + nc], host[so:so + N * (K // 128) * 2], N, K, fmt)
        want_c, want_s, want_z = oracle.quantize(oracle.tensor_f32(Wh[3 + 6 * l + widx[w]], kind), fmt)
        assert np.array_equal(codes, want_c.astype(np.int8)), (l, w)
        assert np.array_equal(sc, want_s), (l, w)
        if fmt == "w4a":
            assert np.array_equal(unpack_zeros(host[zo:zo + N * (K // 128)], N, K), want_z), (l, w)
    eng.close()


def _accept_case(V, B, gamma, mode, seed):
    rng = np.random.default_rng(seed)
    q = (rng.standard_normal((B, gamma, V)) * 2).astype(np.float32)
    if mode == "close":
        p = np.concatenate([q, q[:, -1:]], 1) + rng.standard_normal((B, gamma + 1, V)).astype(np.float32) * 0.3
    else:
        p = (rng.standard_normal((B, gamma + 1, V)) * 2).astype(np.float32)
    return q, p.astype(np.float32)


@pytest.mark.parametrize("V,mode", [(1024, "close"), (1024, "indep"), (128256, "close"), (128256, "indep")])
def test_accept_matches_oracle_on_identical_logits(V, mode):
    say("accept", V, mode)
    B, gamma, T, seed, step = 16, 4, 1.0, 21, 5
    cfg = dict(name="acc", n_layers=1, hidden=128, n_q=2, n_kv=1, head_dim=64, ffn=128, vocab=V, dtype="f32",
               rope_theta=10000.0, rms_eps=1e-5)
    W = [w.cuda() for w in synth.make_weights(cfg, 1, "cpu")]
    eng, k, v, kv_len = make_engine(cfg, W, B, 1024, gamma)
    rng = np.random.default_rng(V)
    lens = rng.integers(0, 900, B).astype(np.int32)
    kv_len.copy_(i32(lens))
    slots = np.arange(B, dtype=np.int32)[::-1].copy()       # slot order differs from row order
    q, p = _accept_case(V, B, gamma, mode, V + len(mode))
    draft = np.zeros((B, gamma), np.int32)
    qstats = np.zeros((B, gamma, 2), np.float32)
    for b in range(B):
        s = int(slots[b])
        for j in range(gamma):
            draft[b, j], _ = oracle.sample_row(q[b, j], T, seed, step, oracle.STREAM_TOKEN, s, int(lens[s]) + j + 1)
            qstats[b, j] = oracle.row_stats(q[b, j], T)
    out = torch.zeros((B, gamma + 1), dtype=torch.int32, device="cuda")
    n_emit = torch.zeros(B, dtype=torch.int32, device="cuda")
    nxt = torch.zeros(B, dtype=torch.int32, device="cuda")
    eng.accept(i32(slots), i32(draft), torch.tensor(q, device="cuda"), torch.tensor(qstats, device="cuda"),
               torch.tensor(p, device="cuda"), gamma, T, seed, step, out, n_emit, nxt)
    eng.sync()
    out, n_emit, nxt = out.cpu().numpy(), n_emit.cpu().numpy(), nxt.cpu().numpy()
    exempt, rejections = 0, 0
    for b in range(B):
        s = int(slots[b])
        n = int(n_emit[b])
        dev = dict(draft=draft[b], q=q[b], p=p[b], out=out[b], n_emit=n)
        status, info = check_accept(dev, T, (seed, step, s, int(lens[s])))
        exempt += status == "exempt"
        rejections += n <= gamma
        assert nxt[b] == out[b, n - 1]
        assert np.all(out[b, n:] == -1)
    assert exempt <= 1
    if mode == "indep":
        assert rejections >= B // 2
    eng.close()


# fp32: k_rope_kv raises the position flags; bf16: the attention kernel does
# (RoPE and the new K/V rows are part of it there)
@pytest.mark.parametrize("cfg", [synth.TINY, dict(synth.TINY, dtype="bf16", name="tiny-bf16")], ids=["f32", "bf16"])
def test_device_range_errors_are_reported(cfg):
    say("range errors", cfg["name"])
    W = [w.cuda() for w in synth.make_weights(cfg, 2, "cpu")]
    B, gamma = 4, 2
    eng, k, v, kv_len = make_engine(cfg, W, B, 64, gamma)
    bufs = sdrl.SDBuffers(eng, B, gamma)
    last = i32([1, 2, 3, 4])
    # a slot index beyond max_slots
    sdrl.sd_step(eng, bufs, i32([0, 1, 2, 7]), last, 1.0, 0, 0)
    with pytest.raises(sdrl.SDError, match="slot"):
        eng.sync()
    # a token id beyond the vocabulary
    eng.ar_step(i32([0]), i32([9999]), 1.0, 0, 0, torch.zeros(1, dtype=torch.int32, device="cuda"),
                torch.zeros((1, cfg["vocab"]), dtype=torch.float32, device="cuda"))
    with pytest.raises(sdrl.SDError, match="token"):
        eng.sync()
    # positions past max_ctx
    kv_len.fill_(62)
    sdrl.sd_step(eng, bufs, i32([0, 1, 2, 3]), last, 1.0, 0, 0)
    with pytest.raises(sdrl.SDError, match="max_ctx"):
        eng.sync()
    # host-side argument checks
    with pytest.raises(sdrl.SDError):
        eng.draft(i32([0]), i32([1]), 5, 1.0, 0, 0, torch.zeros((1, 5), dtype=torch.int32, device="cuda"),
                  torch.zeros((1, 5, cfg["vocab"]), device="cuda"), torch.zeros((1, 5, 2), device="cuda"))
    with pytest.raises(ValueError):
        eng.verify(i32([0]), i32([1]), torch.zeros((1, 2), dtype=torch.int32, device="cuda"), 2,
                   torch.zeros((1, 2, cfg["vocab"]), device="cuda"))
    # temperature must be finite and > 0; gamma at least 1
    o1, l1 = torch.zeros(1, dtype=torch.int32, device="cuda"), torch.zeros((1, cfg["vocab"]), device="cuda")
    for bad_T in (0.0, -1.0, float("nan"), float("inf")):
        with pytest.raises(sdrl.SDError, match="temperature"):
            eng.ar_step(i32([0]), i32([1]), bad_T, 0, 0, o1, l1)
        with pytest.raises(sdrl.SDError, match="temperature"):
            eng.draft(i32([0]), i32([1]), 2, bad_T, 0, 0, torch.zeros((1, 2), dtype=torch.int32, device="cuda"),
                      torch.zeros((1, 2, cfg["vocab"]), device="cuda"), torch.zeros((1, 2, 2), device="cuda"))
    with pytest.raises((sdrl.SDError, ValueError)):
        eng.draft(i32([0]), i32([1]), 0, 1.0, 0, 0, torch.zeros((1, 0), dtype=torch.int32, device="cuda"),
                  torch.zeros((1, 0, cfg["vocab"]), device="cuda"), torch.zeros((1, 0, 2), device="cuda"))
    # weights must be 16-byte aligned (a contiguous view one element into a buffer is not)
    buf = torch.zeros(W[1].numel() + 8, dtype=W[1].dtype, device="cuda")
    off = list(W)
    off[1] = buf[1:1 + W[1].numel()].view(W[1].shape)
    with pytest.raises(sdrl.SDError, match="aligned"):
        eng.bind_weights(off)
    eng.bind_weights(W)
    # so must the cache
    kb = torch.zeros(k.numel() + 8, dtype=k.dtype, device="cuda")
    with pytest.raises(sdrl.SDError, match="aligned"):
        eng.bind_kv(kb[1:1 + k.numel()].view(k.shape), v, kv_len)
    eng.bind_kv(k, v, kv_len)
    kv_len.zero_()
    eng.sync()
    eng.close()


@pytest.mark.parametrize("M", [65, 130, 190, 200, 300, 320, 384, 600, 640, 700, 1000, 1536])
def test_dense_gemm_verify_rows(M):
    """The bf16 GEMM at the verify forward's row counts (M > 64: the LDS-tiled
    kernels with 128- to 320-row tiles, ragged last tiles included; 300, 320,
    600, 640, 700, 1000 and 1536 rows take the DMA-fed 320-row tiles, one to
    five of them, 128 columns wide at this N) against torch in fp32 on the
    same bf16 inputs."""
    say("verify-rows gemm", M)
    g = torch.Generator(device="cuda").manual_seed(M)
    N, K = 24576, 1024
    A = torch.randn((M, K), generator=g, device="cuda").to(torch.bfloat16)
    W = torch.randn((N, K), generator=g, device="cuda").to(torch.bfloat16)
    out = torch.empty((M, N), dtype=torch.float32, device="cuda")
    sdrl.dense_gemm_bf16(A, W, out)
    ref = A.float() @ W.float().t()
    torch.cuda.synchronize()
    err = (out - ref).abs().max().item()
    assert err <= 1e-4 * ref.abs().max().item(), err


@pytest.mark.parametrize("N", [24576, 4224])
@pytest.mark.parametrize("M", [1, 5, 16, 33, 64])
def test_dense_gemm_decode_rows(M, N):
    """The bf16 GEMM at the AR step's and draft LM head's row counts (M <= 64):
    the DMA-fed 64-row tiles where N is a multiple of 256 (rows past M repeat
    the last row and are never stored), the register-streaming kernel
    otherwise (N = 4224), against torch in fp32 on the same bf16 inputs."""
    say("decode-rows gemm", M, N)
    g = torch.Generator(device="cuda").manual_seed(1000 + M)
    K = 1024
    A = torch.randn((M, K), generator=g, device="cuda").to(torch.bfloat16)
    W = torch.randn((N, K), generator=g, device="cuda").to(torch.bfloat16)
    out = torch.full((M, N), float("nan"), dtype=torch.float32, device="cuda")
    sdrl.dense_gemm_bf16(A, W, out)
    ref = A.float() @ W.float().t()
    torch.cuda.synchronize()
    err = (out - ref).abs().max().item()
    assert err <= 1e-4 * ref.abs().max().item(), err


@pytest.mark.parametrize("M,N,K", [(1, 256, 128), (64, 512, 384), (17, 768, 640), (64, 256, 27648)])
def test_dense_gemm_decode_rows_edges(M, N, K):
    """The 64-row DMA tiles at their edges: the fewest stages (K = 128), one
    256-column tile, six and ten stages, and one tile over a long K."""
    say("decode-rows gemm edges", M, N, K)
    g = torch.Generator(device="cuda").manual_seed(M * 7 + N + K)
    A = torch.randn((M, K), generator=g, device="cuda").to(torch.bfloat16)
    W = torch.randn((N, K), generator=g, device="cuda").to(torch.bfloat16)
    out = torch.full((M, N), float("nan"), dtype=torch.float32, device="cuda")
    sdrl.dense_gemm_bf16(A, W, out)
    ref = A.float() @ W.float().t()
    torch.cuda.synchronize()
    err = (out - ref).abs().max().item()
    assert err <= 1e-4 * ref.abs().max().item(), err


@pytest.mark.parametrize("M", [300, 320])
def test_dense_gemm_wide_dma_tiles(M):
    """N with at least 256 tiles of 256 columns: the DMA-fed 320 x 256 tiles
    (eight waves), as used by the verify LM head, against torch in fp32."""
    say("wide dma gemm", M)
    g = torch.Generator(device="cuda").manual_seed(M + 1)
    N, K = 65536, 512
    A = torch.randn((M, K), generator=g, device="cuda").to(torch.bfloat16)
    W = torch.randn((N, K), generator=g, device="cuda").to(torch.bfloat16)
    out = torch.empty((M, N), dtype=torch.float32, device="cuda")
    sdrl.dense_gemm_bf16(A, W, out)
    ref = A.float() @ W.float().t()
    torch.cuda.synchronize()
    err = (out - ref).abs().max().item()
    assert err <= 1e-4 * ref.abs().max().item(), err


# FFN wide enough (24576) that the drafter's gate/up projection runs without a
# K split, which is where its SwiGLU epilogue is used
WIDE_FFN = dict(name="wide-ffn-bf16", n_layers=1, hidden=256, n_q=4, n_kv=2, head_dim=64, ffn=24576, vocab=256,
                dtype="bf16", rope_theta=500000.0, rms_eps=1e-5)


@pytest.mark.parametrize("fmt", ["w4", "w4a", "w8"])
@pytest.mark.parametrize("B,cfg", [(3, SMALL_BF16), (16, SMALL_BF16), (64, SMALL_BF16), (20, WIDE_FFN),
                                   (64, WIDE_FFN), (128, WIDE_FFN)], ids=["3", "16", "64", "wide-20", "wide-64",
                                                                          "wide-128"])
def test_fused_swiglu_equals_separate_kernel(B, cfg, fmt):
    """SwiGLU in the gate/up GEMM's epilogue (the int4 drafter GEMM with one or
    two 32-row tiles where it runs unsplit; the tiled bf16 verify GEMM at 80,
    320 and 640 rows) gives the same SD step, bit for bit, as the gate/up GEMM
    followed by the SwiGLU kernel: same fp32 sums, same SiLU."""
    say("fused swiglu", B, cfg["name"], fmt)
    gamma, T, seed, S = 4, 1.0, 31, 48
    W = [w.cuda() for w in synth.make_weights(cfg, 13, "cpu")]
    eng, k, v, kv_len = make_engine(cfg, W, B, S + gamma + 4, gamma, fmt=fmt)
    synth.fill_kv_context(k, v, S, 17)
    slots = torch.arange(B, dtype=torch.int32, device="cuda")
    last = synth.make_tokens(B, 1, cfg["vocab"], 19)[:, 0].cuda().contiguous()
    outs = []
    for unfused in (False, True):
        eng.set_debug(False, unfused_swiglu=unfused)
        kv_len.fill_(S)
        bufs = sdrl.SDBuffers(eng, B, gamma)
        sdrl.sd_step(eng, bufs, slots, last, T, seed, 1)
        eng.sync()
        outs.append([t.cpu() for t in (bufs.draft_tok, bufs.q_logits, bufs.p_logits, bufs.out_tok, bufs.n_emit,
                                       k[:, :, :, S:S + gamma + 1].contiguous(), v[:, :, :, S:S + gamma + 1].contiguous())])
    for a, b in zip(*outs):
        assert torch.equal(a, b)
    with pytest.raises(sdrl.SDError, match="debug flag"):
        sdrl._check(sdrl.lib().sd_set_debug(eng.h, 8))
    eng.close()


@pytest.mark.parametrize("B", [5, 64])
def test_fused_swiglu_equals_separate_kernel_ar_step(B):
    """The AR step's gate/up projection at M <= 64 (the 64-row DMA tiles,
    unsplit at this FFN width) with SwiGLU in its epilogue gives the same
    logits, token and KV, bit for bit, as the projection followed by the
    SwiGLU kernel."""
    say("fused swiglu, AR step", B)
    cfg, T, seed, S = WIDE_FFN, 1.0, 41, 32
    W = [w.cuda() for w in synth.make_weights(cfg, 43, "cpu")]
    eng, k, v, kv_len = make_engine(cfg, W, B, S + 4, 4)
    synth.fill_kv_context(k, v, S, 47)
    slots = torch.arange(B, dtype=torch.int32, device="cuda")
    last = synth.make_tokens(B, 1, cfg["vocab"], 53)[:, 0].cuda().contiguous()
    outs = []
    for unfused in (False, True):
        eng.set_debug(False, unfused_swiglu=unfused)
        kv_len.fill_(S)
        tok = torch.zeros(B, dtype=torch.int32, device="cuda")
        pl = torch.zeros((B, cfg["vocab"]), dtype=torch.float32, device="cuda")
        eng.ar_step(slots, last, T, seed, 1, tok, pl)
        eng.sync()
        outs.append([t.cpu() for t in (pl, tok, k[:, :, :, S].contiguous(), v[:, :, :, S].contiguous())])
    for a, b in zip(*outs):
        assert torch.equal(a, b)
    eng.close()


@pytest.mark.parametrize("fmt", ["w4", "w8"])
@pytest.mark.parametrize("B", [52, 64, 128, 160])
def test_dma_fed_tiles_equal_register_staged_tiles(B, fmt):
    """The verify forward's 320-row GEMM tiles loaded into LDS by DMA (all four
    projections, SwiGLU fused, and the LM head) give the same SD step, bit
    for bit, as the register-staged tiles: the same MFMA operands in the same
    k order.  B = 52 leaves 60 of the 320 rows empty; B = 128 and 160 (640
    and 800 rows) run two and three m-tiles, the last one half empty at 160."""
    say("dma-fed tiles", B, fmt)
    cfg = SMALL_BF16
    gamma, T, seed, S = 4, 1.0, 37, 40
    W = [w.cuda() for w in synth.make_weights(cfg, 23, "cpu")]
    eng, k, v, kv_len = make_engine(cfg, W, B, S + gamma + 4, gamma, fmt=fmt)
    synth.fill_kv_context(k, v, S, 29)
    slots = torch.arange(B, dtype=torch.int32, device="cuda")
    last = synth.make_tokens(B, 1, cfg["vocab"], 31)[:, 0].cuda().contiguous()
    outs = []
    for staged in (False, True):
        for unfused in (False, True):
            eng.set_debug(False, unfused_swiglu=unfused, staged_tiles=staged)
            kv_len.fill_(S)
            bufs = sdrl.SDBuffers(eng, B, gamma)
            sdrl.sd_step(eng, bufs, slots, last, T, seed, 1)
            eng.sync()
            outs.append([t.cpu() for t in (bufs.p_logits, bufs.out_tok, bufs.n_emit,
                                           k[:, :, :, S:S + gamma + 1].contiguous(),
                                           v[:, :, :, S:S + gamma + 1].contiguous())])
    for o in outs[1:]:
        for a, b in zip(outs[0], o):
            assert torch.equal(a, b)
    eng.close()
