"""Pins of the oracle's fp8 key format (OCP E4M3 codes, per-row power-of-two
scale, exact scores of the quantized operands).  Library references: torch's
float8_e4m3fn dtype for decoding and for float32 -> E4M3 rounding; numpy for
the scores; brute force over all codes for rounding of arbitrary doubles."""
import numpy as np
import pytest
import torch

import oracle

CODES = np.arange(256, dtype=np.uint8)


def _torch_decode(codes):
    return torch.from_numpy(np.asarray(codes, np.uint8).copy()).view(torch.float8_e4m3fn).to(torch.float64).numpy()


def test_decode_matches_torch():
    ours = np.array([oracle.e4m3_value(c) for c in CODES])
    ref = _torch_decode(CODES)
    nan = np.isnan(ref)
    assert np.array_equal(np.isnan(ours), nan) and nan.sum() == 2     # 0x7F and 0xFF
    assert np.array_equal(ours[~nan], ref[~nan])
    assert ours[0x7E] == 448.0 and ours[0x01] == 2.0 ** -9


def test_rounding_matches_torch_on_float32():
    rng = np.random.default_rng(0)
    x = np.concatenate([rng.uniform(-448, 448, 20000), rng.uniform(-1, 1, 20000),
                        rng.uniform(-0.02, 0.02, 20000),
                        _torch_decode(CODES[np.r_[0:127, 128:255]])]).astype(np.float32)
    # exact midpoints between neighbouring finite values: ties go to the even code
    vals = np.sort(np.unique(_torch_decode(CODES[np.r_[0:127, 128:255]])))
    mids = ((vals[:-1] + vals[1:]) / 2).astype(np.float32)
    x = np.concatenate([x, mids])
    ours = oracle.e4m3_round(x.astype(np.float64))
    ref = torch.from_numpy(x).to(torch.float8_e4m3fn).view(torch.uint8).numpy()
    # -0 and +0 decode alike; compare values, and codes elsewhere
    same = (ours == ref) | ((_torch_decode(ours) == 0) & (_torch_decode(ref) == 0))
    assert same.all(), x[~same][:10]


def test_rounding_brute_force_on_doubles():
    rng = np.random.default_rng(1)
    finite = CODES[np.r_[0:127, 128:255]]
    values = _torch_decode(finite)
    x = np.concatenate([rng.uniform(-448, 448, 3000), rng.uniform(-0.05, 0.05, 3000)])
    x = x + rng.uniform(-1e-12, 1e-12, x.shape)      # not float32-representable
    got = oracle.e4m3_round(x)
    for v, c in zip(x, got):
        err = np.abs(values - v)
        best = err.min()
        cand = finite[err == best]
        if len(cand) > 1:                             # a tie: the even code (one of +0/-0 if zero)
            cand = cand[cand % 2 == 0]
        assert oracle.e4m3_value(c) in [oracle.e4m3_value(cc) for cc in cand]


def test_quantize_closed_forms():
    d = 64
    raw = np.zeros((4, d), np.float32)
    raw[0, 3] = 5.0                                   # a basis row: 1 * 2^7 = 128
    raw[1, :2] = [3.0, 4.0]                           # (0.6, 0.8): 0.8 * 2^7 = 102.4 -> scale 2^8
    raw[2] = 0.0                                      # zero row
    raw[3] = -1.0                                     # every component -1/8: -0.125 * 2^10 = -128
    codes, inv = oracle.quantize_rows_fp8(raw)
    assert codes[0, 3] == 0x70 and (np.delete(codes[0], 3) == 0).all() and inv[0] == 2.0 ** -7
    assert inv[1] == 2.0 ** -8
    assert oracle.e4m3_value(codes[1, 1]) == 208.0    # 0.8 * 256 = 204.8 -> 208 (spacing 16)
    assert oracle.e4m3_value(codes[1, 0]) == 160.0    # 153.6 -> 160
    assert (codes[2] == 0).all() and inv[2] == 1.0
    assert (codes[3] == 0xF0).all() and inv[3] == 2.0 ** -10


def test_quantize_scale_rule():
    rng = np.random.default_rng(2)
    raw = (rng.standard_normal((300, 200)) * rng.uniform(0.01, 100, (300, 1))).astype(np.float32)
    raw[:50, 7] *= 50                                 # outlier components
    codes, inv = oracle.quantize_rows_fp8(raw)
    vals = _torch_decode(codes)
    top = np.abs(vals).max(1)
    assert np.all((top >= 128) & (top <= 256))
    assert np.all(np.log2(inv) == np.round(np.log2(inv)))
    # dequantized rows are close to the unit rows (3 fraction bits per value)
    unit = raw / np.linalg.norm(raw.astype(np.float64), axis=1, keepdims=True)
    deq = vals * inv[:, None]
    assert np.all(np.abs(deq - unit) <= np.abs(unit) * 2.0 ** -4 + 2.0 ** -9 * inv[:, None] + 1e-12)


def test_scores_match_numpy():
    rng = np.random.default_rng(3)
    k = rng.standard_normal((500, 96)).astype(np.float32)
    q = rng.standard_normal((7, 96)).astype(np.float32)
    kc, ki = oracle.quantize_rows_fp8(k)
    qc, qi = oracle.quantize_rows_fp8(q)
    s = oracle.scores_fp8(kc, ki, qc, qi)
    ref = (_torch_decode(qc) @ _torch_decode(kc).T) * qi[:, None] * ki[None, :]
    assert np.array_equal(s, ref)
    # and they approximate the bf16 cosines
    sb = oracle.scores(oracle.normalize_rows(k), oracle.normalize_rows(q))
    assert np.abs(s - sb).max() < 0.03
