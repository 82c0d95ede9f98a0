"""Pins for the oracle's counter-causal attention (Eq. (2) with the mask of Sec. 3.1).

Each test checks the oracle against something other than itself: explicit loops
over scalars, a library attention routine, the time-reversal identity with
textbook causal attention, closed forms for uniform keys, and edge rows."""
import math

import numpy as np
import pytest
import torch

from oracle import cc_oracle as O

SHAPES = [(1, 1, 1, 1), (2, 1, 1, 3), (3, 2, 1, 4), (5, 4, 2, 8), (9, 6, 2, 4), (7, 3, 3, 5),
          (12, 4, 1, 8)]  # (n, Hq, Hkv, d)


def _rand(n, hq, hkv, d, seed):
    r = np.random.default_rng(seed)
    return r.standard_normal((n, hq, d)), r.standard_normal((hkv, n, d)), r.standard_normal((hkv, n, d))


def _brute(q, k, v, diag):
    """Scalar loops straight from the definition: softmax over the allowed keys of
    tau * q.k, weights applied to the values; GQA head h reads KV head h // g."""
    n, hq, d = len(q), len(q[0]), len(q[0][0])
    hkv = len(k)
    g = hq // hkv
    tau = 1.0 / math.sqrt(d)
    out = [[[0.0] * d for _ in range(hq)] for _ in range(n)]
    for i in range(n):
        js = [j for j in range(n) if (j > i if diag == "strict" else j >= i)]
        for h in range(hq):
            c = h // g
            if not js:
                continue
            logits = [tau * sum(q[i][h][t] * k[c][j][t] for t in range(d)) for j in js]
            mx = max(logits)
            ws = [math.exp(x - mx) for x in logits]
            tot = sum(ws)
            for t in range(d):
                out[i][h][t] = sum(w * v[c][j][t] for w, j in zip(ws, js)) / tot
    return np.array(out)


@pytest.mark.parametrize("diag", ["strict", "inclusive"])
@pytest.mark.parametrize("shape", SHAPES)
def test_bruteforce(shape, diag):
    q, k, v = _rand(*shape, seed=hash(shape) % 1000)
    got = O.attention_cc(q, k, v, diag)
    want = _brute(q.tolist(), k.tolist(), v.tolist(), diag)
    np.testing.assert_allclose(got, want, rtol=1e-12, atol=1e-12)


def _sdpa_masked(q, k, v, allow):
    """torch fp64 scaled_dot_product_attention with an explicit boolean mask;
    q [n][Hq][d], k/v [Hkv][n][d] expanded to Hq heads."""
    n, hq, d = q.shape
    g = hq // k.shape[0]
    tq = torch.from_numpy(q).permute(1, 0, 2)                    # [Hq][n][d]
    tk = torch.from_numpy(k).repeat_interleave(g, 0)
    tv = torch.from_numpy(v).repeat_interleave(g, 0)
    out = torch.nn.functional.scaled_dot_product_attention(
        tq, tk, tv, attn_mask=torch.from_numpy(allow))
    return out.permute(1, 0, 2).numpy()


@pytest.mark.parametrize("shape", SHAPES[1:])
def test_vs_library_sdpa(shape):
    n = shape[0]
    q, k, v = _rand(*shape, seed=7)
    allow = np.triu(np.ones((n, n), dtype=bool), k=1)            # j > i
    want = _sdpa_masked(q, k, v, allow)
    got = O.attention_cc(q, k, v, "strict")
    np.testing.assert_allclose(got[:-1], want[:-1], rtol=1e-12, atol=1e-12)
    assert np.all(got[-1] == 0.0)


@pytest.mark.parametrize("shape", SHAPES[1:])
def test_time_reversal_equals_causal(shape):
    """Counter-causal attention is textbook causal attention on the reversed
    sequence: CC_inclusive(Q,K,V)[i] = causal(rev Q, rev K, rev V)[n-1-i], and the
    strict mask corresponds to causal attention that excludes the diagonal."""
    n = shape[0]
    q, k, v = _rand(*shape, seed=11)
    rq, rk, rv = q[::-1].copy(), k[:, ::-1].copy(), v[:, ::-1].copy()
    g = q.shape[1] // k.shape[0]
    tq = torch.from_numpy(rq).permute(1, 0, 2)
    tk = torch.from_numpy(rk).repeat_interleave(g, 0)
    tv = torch.from_numpy(rv).repeat_interleave(g, 0)
    causal = torch.nn.functional.scaled_dot_product_attention(tq, tk, tv, is_causal=True)
    causal = causal.permute(1, 0, 2).numpy()[::-1]
    np.testing.assert_allclose(O.attention_cc(q, k, v, "inclusive"), causal, rtol=1e-12, atol=1e-12)
    strict_allow = torch.from_numpy(np.tril(np.ones((n, n), dtype=bool), k=-1))
    cs = torch.nn.functional.scaled_dot_product_attention(tq, tk, tv, attn_mask=strict_allow)
    cs = cs.permute(1, 0, 2).numpy()[::-1]
    got = O.attention_cc(q, k, v, "strict")
    np.testing.assert_allclose(got[:-1], cs[:-1], rtol=1e-12, atol=1e-12)


def _suffix_mean(v, strict=True):
    """mean of v[c, j] over j > i (strict) or j >= i, by reverse cumulative sums."""
    hkv, n, d = v.shape
    cs = np.cumsum(v[:, ::-1], axis=1)[:, ::-1]                  # sum_{j >= i}
    out = np.zeros_like(v)
    for i in range(n):
        if strict:
            cnt = n - 1 - i
            if cnt:
                out[:, i] = cs[:, i + 1] / cnt
        else:
            out[:, i] = cs[:, i] / (n - i)
    return out


@pytest.mark.parametrize("diag", ["strict", "inclusive"])
def test_uniform_keys_give_suffix_means(diag):
    n, hq, hkv, d = 33, 4, 2, 8
    r = np.random.default_rng(3)
    q = r.standard_normal((n, hq, d))
    krow = r.standard_normal((hkv, 1, d))
    k = np.repeat(krow, n, axis=1)
    v = r.standard_normal((hkv, n, d))
    got = O.attention_cc(q, k, v, diag)
    sm = _suffix_mean(v, diag == "strict")
    g = hq // hkv
    for h in range(hq):
        np.testing.assert_allclose(got[:, h], sm[h // g], rtol=1e-12, atol=1e-12)
    # q = 0 gives the same closed form for arbitrary keys
    got0 = O.attention_cc(np.zeros_like(q), r.standard_normal((hkv, n, d)), v, diag)
    for h in range(hq):
        np.testing.assert_allclose(got0[:, h], sm[h // g], rtol=1e-12, atol=1e-12)


def test_constant_values_and_key_shift():
    n, hq, hkv, d = 17, 4, 1, 8
    q, k, v = _rand(n, hq, hkv, d, seed=5)
    cst = np.full_like(v, 1.75)
    got = O.attention_cc(q, k, cst)
    np.testing.assert_allclose(got[:-1], 1.75, rtol=0, atol=1e-13)
    assert np.all(got[-1] == 0)
    shift = np.random.default_rng(9).standard_normal((hkv, 1, d))
    np.testing.assert_allclose(O.attention_cc(q, k + shift, v), O.attention_cc(q, k, v),
                               rtol=1e-10, atol=1e-12)


def test_edge_rows():
    q, k, v = _rand(6, 2, 1, 4, seed=2)
    s = O.attention_cc(q, k, v, "strict")
    assert np.array_equal(s[-2, 0], v[0, -1]) and np.array_equal(s[-2, 1], v[0, -1])
    assert np.all(s[-1] == 0)
    inc = O.attention_cc(q, k, v, "inclusive")
    assert np.array_equal(inc[-1, 0], v[0, -1])
    one = O.attention_cc(q[:1], k[:, :1], v[:, :1], "strict")
    assert one.shape == (1, 2, 4) and np.all(one == 0)
    two = O.attention_cc(q[:2], k[:, :2], v[:, :2], "strict")
    assert np.array_equal(two[0, 0], v[0, 1]) and np.all(two[1] == 0)


def test_gqa_mapping_is_contiguous_groups():
    """With GQA, query head h reads KV head h // g; expanding each KV head to its g
    query heads must give the same result as multi-head attention."""
    n, hq, hkv, d = 10, 6, 2, 4
    q, k, v = _rand(n, hq, hkv, d, seed=21)
    gqa = O.attention_cc(q, k, v)
    mha = O.attention_cc(q, np.repeat(k, 3, axis=0), np.repeat(v, 3, axis=0))
    np.testing.assert_allclose(gqa, mha, rtol=1e-13, atol=1e-13)
    # and not the interleaved mapping h % Hkv
    inter = O.attention_cc(q, np.tile(k, (3, 1, 1)), np.tile(v, (3, 1, 1)))
    assert not np.allclose(gqa, inter)


def test_row_subset_is_exact():
    q, k, v = _rand(20, 4, 2, 8, seed=4)
    full = O.attention_cc(q, k, v)
    rows = [0, 3, 19, 7]
    np.testing.assert_array_equal(O.attention_cc(q, k, v, rows=rows), full[rows])


def test_bf16_widening_is_exact():
    bits = np.array([0x3F80, 0xBF80, 0x0000, 0x8000, 0x7F80, 0x4049], dtype=np.uint16)
    np.testing.assert_array_equal(O.f64(bits), [1.0, -1.0, 0.0, -0.0, np.inf, 3.140625])
