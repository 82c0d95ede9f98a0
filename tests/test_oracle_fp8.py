"""Pins for the oracle's FP8 (OCP E4M3) codec, quantizer and FP8 LM-head score.

The codec follows the format's definition (values in tests/golden/e4m3_values.json);
the quantizer and the score are the surprise score of Eq. (5) on a model whose LM-head
inputs are FP8-quantized (one scale per activation row, one for the weight matrix)."""
import json
import math
import os

import numpy as np
import pytest

from oracle import cc_oracle as O

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def test_spec_values():
    g = json.load(open(os.path.join(GOLDEN, "e4m3_values.json")))
    for code, val in g["pairs"]:
        c = int(code, 16)
        assert O.e4m3_decode([c])[0] == val, code
        assert O.e4m3_encode([val])[0] == c, code
    nz = int(g["negative_zero"], 16)
    assert O.e4m3_encode([-0.0])[0] == nz
    assert O.e4m3_decode([nz])[0] == 0.0 and math.copysign(1.0, O.e4m3_decode([nz])[0]) < 0
    for code in g["nan"]:
        assert np.isnan(O.e4m3_decode([int(code, 16)])[0])
    assert np.isnan(O.e4m3_decode([0x7F])[0]) and O.e4m3_encode([np.nan])[0] == 0x7F


def test_round_trip_every_finite_code():
    codes = np.array([c for c in range(256) if (c & 0x7F) != 0x7F], dtype=np.uint8)
    np.testing.assert_array_equal(O.e4m3_encode(O.e4m3_decode(codes)), codes)
    # 126 distinct positive values strictly increasing after zero
    pos = O.e4m3_decode(np.arange(0x7F))
    assert np.all(np.diff(pos) > 0) and pos[-1] == 448.0


def test_round_to_nearest_even_and_saturation():
    pos = O.e4m3_decode(np.arange(0x7F))
    mids = (pos[:-1] + pos[1:]) / 2
    lo_codes = np.arange(0x7E)
    got = O.e4m3_encode(mids).astype(int)
    want = np.where(lo_codes % 2 == 0, lo_codes, lo_codes + 1)   # the even code of the pair
    np.testing.assert_array_equal(got, want)
    eps = np.diff(pos) * 1e-3
    np.testing.assert_array_equal(O.e4m3_encode(mids - eps[:]), lo_codes)
    np.testing.assert_array_equal(O.e4m3_encode(mids + eps[:]), lo_codes + 1)
    np.testing.assert_array_equal(O.e4m3_encode([448.0, 460.0, 1e6, -1e6]), [0x7E, 0x7E, 0x7E, 0xFE])
    # negative values mirror positive ones
    x = np.linspace(-500, 500, 2001)
    np.testing.assert_array_equal(O.e4m3_encode(-x) & 0x7F, O.e4m3_encode(x) & 0x7F)


def test_quantizer_error_and_extremes():
    r = np.random.default_rng(0)
    x = r.standard_normal((16, 300)).astype(np.float32) * np.logspace(-3, 3, 16, dtype=np.float32)[:, None]
    x[3] = 0.0
    codes, scale = O.quantize_fp8(x, per_row=True)
    deq = O.e4m3_decode(codes) * scale.astype(np.float64)[:, None]
    assert np.all(codes[3] == 0) and scale[3] == 0
    for i in range(16):
        if i == 3:
            continue
        j = np.argmax(np.abs(x[i]))
        assert (codes[i, j] & 0x7F) == 0x7E          # the row's extreme maps to 448
        amax = float(np.abs(x[i]).max())
        big = np.abs(x[i]) >= amax * 2.0 ** -7        # normal range of the scaled row
        err = np.abs(deq[i] - x[i])
        assert np.all(err[big] <= 2.0 ** -4 * np.abs(x[i][big]) * (1 + 1e-6))
        assert np.all(err <= amax * 2.0 ** -10 * (1 + 1e-6) + 2.0 ** -4 * np.abs(x[i]))
    c1, s1 = O.quantize_fp8(x, per_row=False)
    assert s1.shape == (1,) and s1[0] == np.float32(np.abs(x).max()) / np.float32(448)


def _exact_fp8_matrix(r, rows, cols, exp):
    """Rows whose FP8 quantization is exact: decoded codes times 2^exp, with one 448 per row."""
    codes = r.integers(0, 0x7E, (rows, cols)).astype(np.uint8) | (r.integers(0, 2, (rows, cols)) * 0x80).astype(np.uint8)
    codes[:, 0] = 0x7E
    return O.e4m3_decode(codes) * 2.0 ** exp


def test_fp8_scores_equal_plain_scores_when_quantization_is_exact():
    r = np.random.default_rng(5)
    N, D, V = 10, 48, 70
    cu = [0, 4, 10]
    u = _exact_fp8_matrix(r, N, D, -7).astype(np.float32)   # per-row amax 448 * 2^-7 = 3.5
    w = _exact_fp8_matrix(r, V, D, -12).astype(np.float32)
    w[1:, 0] = O.e4m3_decode([0x70])[0] * 2.0 ** -12          # one 448 in the whole matrix
    ids = r.integers(0, V, N)
    wc, ws = O.quantize_fp8(w, per_row=False)
    np.testing.assert_array_equal(O.e4m3_decode(wc) * float(ws[0]), w.astype(np.float64))
    got = O.lmhead_fp8_scores(u, wc, ws[0], ids, cu, n_frozen=1)
    ref, _, _ = O.surprise(u.astype(np.float64), w, ids)
    ref[O.edge_rows(cu, 1)] = np.inf
    np.testing.assert_array_equal(np.isinf(got), np.isinf(ref))
    fin = np.isfinite(ref)
    np.testing.assert_allclose(got[fin], ref[fin], rtol=1e-12, atol=1e-12)


def test_fp8_zero_head_gives_ln_vocab():
    r = np.random.default_rng(6)
    u = r.standard_normal((5, 32)).astype(np.float32)
    V = 1000
    wc, ws = O.quantize_fp8(np.zeros((V, 32), dtype=np.float32), per_row=False)
    s = O.lmhead_fp8_scores(u, wc, ws[0], np.arange(5), [0, 5])
    np.testing.assert_allclose(s[:-1], math.log(V), rtol=0, atol=1e-12)
    assert s[-1] == np.inf
