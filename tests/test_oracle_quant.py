"""Pins of the oracle's RTN int4 quantizer (Sec. 4.1; App. B.2 for the
asymmetric form).  Codes must be the nearest grid point (brute force over
every code), the scale the fp16 rounding of max|w|/7 (numpy float16), the
extreme element of each group must land on +-7, and all-zero groups on 0."""
import numpy as np

import oracle


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
