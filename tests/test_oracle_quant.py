"""Pins of the oracle's RTN quantizers (Sec. 4.1; App. B.2 for the asymmetric
int4 form, App. B.3 / Table 4 for the 8-bit drafter).  Codes must be the
nearest grid point (brute force over every code), the scale the fp16
rounding of max|w|/7 (or /127, or (max-min)/15) computed by numpy float16,
the extreme elements of each group must land on the grid's ends, and
all-zero groups on 0.  The drafter built from any format must run the same
network as a model whose weights are the dequantized values, computed here
in numpy."""
import numpy as np
import pytest

import oracle
from paper_2606_18967_amd import synth


def _weights(seed=0, N=48, K=512):
    rng = np.random.default_rng(seed)
    w = (rng.standard_normal((N, K)) * 0.02).astype(np.float32)
    w[3, 128:256] = 0.0                                   # an all-zero group
    w[5, :128] *= 1e4                                     # a large-magnitude group
    w[7, 256:384] = rng.standard_normal(128).astype(np.float32) * 1e-6   # tiny (subnormal fp16 scale)
    return w


def test_symmetric_codes_are_nearest_grid_points():
    w = _weights()
    codes, scales = oracle.quantize_rtn4(w)
    N, K = w.shape
    s = oracle.f16_bits_to_f32(scales)                   # [N][K/128]
    assert codes.min() >= -8 and codes.max() <= 7
    grid = np.arange(-8, 8, dtype=np.float64)
    for n in range(N):
        for g in range(K // 128):
            wg = w[n, g * 128:(g + 1) * 128].astype(np.float64)
            cg = codes[n, g * 128:(g + 1) * 128]
            amax = np.abs(w[n, g * 128:(g + 1) * 128]).max()
            want_s = np.float16(np.float32(amax) / np.float32(7.0))
            assert scales[n, g] == np.array(want_s).view(np.uint16), (n, g)
            if amax == 0:
                assert s[n, g] == 0 and np.all(cg == 0)
                continue
            sg = float(s[n, g])
            err = np.abs(wg[:, None] - sg * grid[None, :])
            best = err.min(axis=1)
            mine = np.abs(wg - sg * cg)
            assert np.all(mine <= best + 1e-6 * sg), (n, g)
            assert np.all(mine <= 0.5 * sg * (1 + 1e-6))
            i = np.argmax(np.abs(wg))
            assert abs(int(cg[i])) == 7, (n, g)


def test_asymmetric_codes():
    w = _weights(1)
    codes, scales, zeros = oracle.quantize_rtn4_asym(w)
    s = oracle.f16_bits_to_f32(scales)
    N, K = w.shape
    assert codes.max() <= 15 and zeros.max() <= 15
    for n in range(N):
        for g in range(K // 128):
            sl = slice(g * 128, (g + 1) * 128)
            wg = w[n, sl].astype(np.float64)
            if s[n, g] == 0:
                continue
            deq = float(s[n, g]) * (codes[n, sl].astype(np.float64) - zeros[n, g])
            # the group's range is covered up to half a step (plus fp16 rounding of s and z)
            assert np.all(np.abs(deq - wg) <= 0.5 * s[n, g] + 0.02 * (wg.max() - wg.min()) + 1e-9)


def test_asymmetric_codes_are_nearest_on_the_shifted_grid():
    w = _weights(2)
    codes, scales, zeros = oracle.quantize_rtn4_asym(w)
    s = oracle.f16_bits_to_f32(scales)
    N, K = w.shape
    for n in range(N):
        for g in range(K // 128):
            sl = slice(g * 128, (g + 1) * 128)
            wg = w[n, sl]
            rng32 = np.float32(wg.max()) - np.float32(wg.min())
            assert scales[n, g] == np.array(np.float16(rng32 / np.float32(15.0))).view(np.uint16), (n, g)
            if s[n, g] == 0:
                assert np.all(codes[n, sl] == 0) and zeros[n, g] == 0
                continue
            sg, z = float(s[n, g]), int(zeros[n, g])
            grid = sg * (np.arange(16, dtype=np.float64) - z)
            err = np.abs(wg.astype(np.float64)[:, None] - grid[None, :])
            mine = np.abs(wg.astype(np.float64) - grid[codes[n, sl]])
            assert np.all(mine <= err.min(axis=1) + 1e-6 * sg), (n, g)
            # the group's minimum sits at the bottom of the grid and its maximum at the top
            assert codes[n, sl][np.argmin(wg)] in (0, 1), (n, g)
            assert codes[n, sl][np.argmax(wg)] in (14, 15), (n, g)


def test_int8_codes_are_nearest_grid_points():
    w = _weights(3)
    codes, scales = oracle.quantize_rtn8(w)
    N, K = w.shape
    s = oracle.f16_bits_to_f32(scales)
    grid = np.arange(-128, 128, dtype=np.float64)
    for n in range(N):
        for g in range(K // 128):
            sl = slice(g * 128, (g + 1) * 128)
            wg = w[n, sl].astype(np.float64)
            amax = np.abs(w[n, sl]).max()
            assert scales[n, g] == np.array(np.float16(np.float32(amax) / np.float32(127.0))).view(np.uint16)
            if s[n, g] == 0:                       # all zero, or max|w|/127 below the smallest fp16
                assert amax < 2.0 ** -24 * 127 and np.all(codes[n, sl] == 0)
                continue
            sg = float(s[n, g])
            mine = np.abs(wg - sg * codes[n, sl])
            best = np.abs(wg[:, None] - sg * grid[None, :]).min(axis=1)
            assert np.all(mine <= best + 1e-6 * sg), (n, g)
            assert abs(int(codes[n, sl][np.argmax(np.abs(wg))])) == 127, (n, g)


@pytest.mark.parametrize("fmt", ["w4", "w4a", "w8"])
def test_drafter_runs_the_dequantized_network(fmt):
    """make_drafter(fmt) == the float model whose projections hold s*(q - z)."""
    cfg = dict(name="q", n_layers=2, hidden=256, n_q=4, n_kv=2, head_dim=32, ffn=384, vocab=64, dtype="f32",
               rope_theta=10000.0, rms_eps=1e-5)
    W = [t.numpy().astype(np.float32) for t in synth.make_weights(cfg, 9, "cpu", std=0.05)]
    drafter = oracle.make_drafter(cfg, W, oracle.F32, fmt=fmt)
    Wd = [w.copy() for w in W]
    for l, which, ti in drafter.quant_targets():
        codes, scales, zeros = oracle.quantize(W[ti], fmt)
        sc = np.repeat(oracle.f16_bits_to_f32(scales).astype(np.float64), 128, axis=1)
        z = 0.0 if zeros is None else np.repeat(zeros.astype(np.float64), 128, axis=1)
        Wd[ti] = (sc * (codes.astype(np.float64) - z)).astype(np.float32)   # exact: 11-bit scale x small integer
    ref = oracle.Model(cfg, Wd, oracle.F32)
    tok = np.random.default_rng(1).integers(0, cfg["vocab"], 6)
    a = oracle.forward_seq(drafter, oracle.KV(cfg, 8), tok, 0)
    b = oracle.forward_seq(ref, oracle.KV(cfg, 8), tok, 0)
    assert np.array_equal(a, b)
    # and it is a drafter: close to the target, closer for more bits
    t = oracle.forward_seq(oracle.Model(cfg, W, oracle.F32), oracle.KV(cfg, 8), tok, 0)
    rel = np.abs(a - t).max() / np.abs(t).max()
    assert rel < (0.02 if fmt == "w8" else 0.3)
