"""Pins for the oracle's surprise score, keep selection, compaction and full pass.

Surprise: Eq. (5) read as -log P(x_i | future) through the LM head's log-softmax
(Sec. 3.1).  Selection/compaction: the memory-refresh procedure of Sec. 3.2.  Full
pass: Sec. 3.1 (fresh queries at the original positions, stored keys/values)."""
import itertools
import json
import math
import os

import numpy as np
import pytest
import scipy.special
import torch

from oracle import cc_oracle as O

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _load(name):
    with open(os.path.join(GOLDEN, name)) as f:
        return json.load(f)


# ---------------------------------------------------------------- worked example

def test_hand_worked_example():
    g = _load("hand_example.json")
    q, k, v = (np.array(g[x], dtype=float) for x in ("q", "k", "v"))
    o = O.attention_cc(q, k, v)
    np.testing.assert_allclose(o[:, 0, 0], g["o"], rtol=0, atol=1e-15)
    s = O.last_layer_scores(q, k, v, np.array(g["w_o"]), np.array(g["w_lm"]), g["ids"],
                            [0, 3])
    want = np.array([float(x) for x in g["scores"]])
    assert s[2] == np.inf
    np.testing.assert_allclose(s[:2], want[:2], rtol=1e-14, atol=1e-15)
    np.testing.assert_array_equal(O.select_keep(s, 2), g["keep_k2"])


# ---------------------------------------------------------------- LM head / LSE

@pytest.mark.parametrize("V", [1, 1024, 128256, 152064])
def test_zero_lm_head_gives_ln_vocab(V):
    want = _load("uniform_lm_head.json")["ln_V"][str(V)]
    D = 8
    u = np.random.default_rng(0).standard_normal((5, D))
    s, lse, zt = O.surprise(u, np.zeros((V, D)), np.arange(5) % V)
    np.testing.assert_allclose(s, want, rtol=0, atol=1e-12)
    assert want == pytest.approx(math.log(V), abs=1e-15)


def test_lse_and_score_vs_library():
    r = np.random.default_rng(1)
    u = r.standard_normal((7, 16))
    w = r.standard_normal((300, 16))
    ids = r.integers(0, 300, 7)
    s, lse, zt = O.surprise(u, w, ids)
    z = u @ w.T
    np.testing.assert_allclose(lse, scipy.special.logsumexp(z, axis=1), rtol=1e-13)
    logp = torch.log_softmax(torch.from_numpy(z), dim=1).numpy()
    np.testing.assert_allclose(s, -logp[np.arange(7), ids], rtol=1e-12, atol=1e-12)
    np.testing.assert_allclose(np.exp(z - lse[:, None]).sum(1), 1.0, rtol=1e-13)
    assert np.all(s >= 0)


def test_lse_is_stable_for_large_logits():
    u = np.array([[1.0]])
    w = np.array([[800.0], [799.0], [-900.0]])
    s, lse, zt = O.surprise(u, w, [1])
    assert np.isfinite(lse).all()
    np.testing.assert_allclose(s, 1.0 + math.log1p(math.exp(-1.0)), rtol=0, atol=1e-12)


def test_vocab_chunking_does_not_change_logits():
    r = np.random.default_rng(2)
    u = r.standard_normal((3, 8))
    w = r.standard_normal((100, 8))
    np.testing.assert_allclose(O.lm_head_logits(u, w, vocab_chunk=7), u @ w.T, rtol=1e-14)


# ---------------------------------------------------------------- score rules

def test_last_entry_and_frozen_prefix_are_infinite():
    cu = [0, 5, 6, 9]
    m = O.edge_rows(cu)
    np.testing.assert_array_equal(np.nonzero(m)[0], [4, 5, 8])
    m2 = O.edge_rows(cu, n_frozen=2)
    np.testing.assert_array_equal(np.nonzero(m2)[0], [0, 1, 4, 5, 6, 7, 8])


def test_ragged_scores_match_per_sequence():
    r = np.random.default_rng(6)
    lens = [4, 1, 7]
    cu = np.concatenate([[0], np.cumsum(lens)])
    N, hq, hkv, d, D, V = int(cu[-1]), 4, 2, 8, 16, 50
    q = r.standard_normal((N, hq, d))
    k = r.standard_normal((hkv, N, d))
    v = r.standard_normal((hkv, N, d))
    wo = r.standard_normal((D, hq * d)) * 0.1
    wl = r.standard_normal((V, D)) * 0.1
    ids = r.integers(0, V, N)
    s = O.last_layer_scores(q, k, v, wo, wl, ids, cu)
    for b in range(3):
        lo, hi = cu[b], cu[b + 1]
        sb = O.last_layer_scores(q[lo:hi], k[:, lo:hi], v[:, lo:hi], wo, wl, ids[lo:hi],
                                 [0, hi - lo])
        np.testing.assert_array_equal(s[lo:hi], sb)
    assert s[cu[1] - 1] == np.inf and s[cu[2] - 1] == np.inf and s[-1] == np.inf
    sub = [0, 5, 9]
    np.testing.assert_array_equal(O.last_layer_scores(q, k, v, wo, wl, ids, cu, rows=sub), s[sub])


def test_fused_weight_scores_equal_the_two_step_chain():
    """With queries given, the fast variant's output processing is the bare W_o, so
    z = W_lm (W_o y) = (W_lm W_o) y: scores through the product weight equal the two-step
    chain's (fp64 rounding only).  D != Hq*d makes a transposed operand unformable; the
    square case (D == Hq*d, the usual shapes) would accept one, and the random W_o below
    would then disagree."""
    r = np.random.default_rng(17)
    lens = [6, 1, 9]
    cu = np.concatenate([[0], np.cumsum(lens)])
    N, hq, hkv, d, V = int(cu[-1]), 4, 2, 8, 60
    q = r.standard_normal((N, hq, d))
    k = r.standard_normal((hkv, N, d))
    v = r.standard_normal((hkv, N, d))
    ids = r.integers(0, V, N)
    for D in (24, hq * d):
        wo = r.standard_normal((D, hq * d)) * 0.2
        wl = r.standard_normal((V, D)) * 0.2
        M = O.fused_lmhead_weight(wl, wo)
        assert M.shape == (V, hq * d)
        ref = O.last_layer_scores(q, k, v, wo, wl, ids, cu, n_frozen=1)
        got = O.last_layer_fused_scores(q, k, v, M, ids, cu, n_frozen=1)
        np.testing.assert_array_equal(np.isinf(got), np.isinf(ref))
        fin = np.isfinite(ref)
        np.testing.assert_allclose(got[fin], ref[fin], rtol=1e-12, atol=1e-12)
    # the product itself, entry by entry on a tiny case
    wl = r.standard_normal((3, 4))
    wo = r.standard_normal((4, 5))
    M = O.fused_lmhead_weight(wl, wo)
    for a in range(3):
        for c in range(5):
            assert M[a, c] == pytest.approx(sum(wl[a, t] * wo[t, c] for t in range(4)), rel=1e-14)


def test_uniform_keys_closed_form_score():
    """Uniform keys make attention a suffix mean, so the whole fast-path score has a
    closed form built from reverse cumulative sums and a library logsumexp."""
    r = np.random.default_rng(8)
    n, hq, hkv, d, D, V = 12, 2, 1, 4, 6, 20
    q = r.standard_normal((n, hq, d))
    k = np.zeros((hkv, n, d))
    v = r.standard_normal((hkv, n, d))
    wo = r.standard_normal((D, hq * d))
    wl = r.standard_normal((V, D))
    ids = r.integers(0, V, n)
    cs = np.cumsum(v[0, ::-1], axis=0)[::-1]
    y = np.zeros((n, hq * d))
    for i in range(n - 1):
        y[i] = np.tile(cs[i + 1] / (n - 1 - i), hq)
    z = y @ wo.T @ wl.T
    want = scipy.special.logsumexp(z, axis=1) - z[np.arange(n), ids]
    got = O.last_layer_scores(q, k, v, wo, wl, ids, [0, n])
    np.testing.assert_allclose(got[:-1], want[:-1], rtol=1e-12)
    assert got[-1] == np.inf


# ---------------------------------------------------------------- selection

def _brute_select(scores, k):
    """The unique k-subset whose every member beats every non-member under
    (score desc with -0 == +0 and NaN lowest, then index asc)."""
    n = len(scores)

    def beats(a, b):
        sa, sb = scores[a], scores[b]
        na, nb = math.isnan(sa), math.isnan(sb)
        if na != nb:
            return nb
        if not na and sa != sb:
            return sa > sb
        return a < b

    found = []
    for sub in itertools.combinations(range(n), k):
        rest = [j for j in range(n) if j not in sub]
        if all(beats(a, b) for a in sub for b in rest):
            found.append(list(sub))
    assert len(found) == 1
    return found[0]


@pytest.mark.parametrize("seed", range(12))
def test_select_bruteforce(seed):
    r = np.random.default_rng(seed)
    n = int(r.integers(1, 10))
    pool = np.array([-0.0, 0.0, 1.0, 1.0, 2.5, -3.0, np.inf, -np.inf, np.nan, 7.0])
    s = pool[r.integers(0, len(pool), n)]
    for k in range(0, n + 1):
        np.testing.assert_array_equal(O.select_keep(s, k), _brute_select(s.tolist(), k))


def test_select_invariants_and_all_ties():
    r = np.random.default_rng(3)
    s = r.standard_normal(500)
    s[-1] = np.inf
    keep = O.select_keep(s, 100)
    assert len(keep) == 100 and np.all(np.diff(keep) > 0) and keep[-1] == 499
    ev = np.setdiff1d(np.arange(500), keep)
    assert s[keep].min() >= s[ev].max()
    ties = np.full(10, math.log(1024.0))
    ties[-1] = np.inf
    np.testing.assert_array_equal(O.select_keep(ties, 4), [0, 1, 2, 9])
    assert len(O.select_keep(s, 0)) == 0
    np.testing.assert_array_equal(O.select_keep(s, 500), np.arange(500))


def test_select_matches_lexsort():
    r = np.random.default_rng(4)
    s = np.round(r.standard_normal(2000), 1)          # many exact ties
    keep = O.select_keep(s, 300)
    order = np.lexsort((np.arange(2000), -s))
    np.testing.assert_array_equal(keep, np.sort(order[:300]))


# ---------------------------------------------------------------- compaction

def test_compact_is_gather():
    r = np.random.default_rng(5)
    rows = r.integers(0, 1 << 16, (40, 3), dtype=np.uint16)
    keep = np.array([2, 3, 10, 39])
    out = O.compact(rows, keep)
    np.testing.assert_array_equal(out, rows[keep])
    np.testing.assert_array_equal(O.compact(rows, np.arange(40)), rows)
    assert out.dtype == np.uint16


# ---------------------------------------------------------------- RoPE / full pass

def test_rope_closed_forms():
    r = np.random.default_rng(9)
    d, theta = 8, 500000.0
    x = r.standard_normal((5, 2, d))
    pos = np.array([0, 1, 7, 100, 8191])
    y = O.rope(x, pos, theta)
    np.testing.assert_allclose(y[0], x[0], rtol=0, atol=0)             # position 0
    # each pair (t, t + d/2) is a complex number turned by pos * theta^(-2t/d)
    for ri, p in enumerate(pos):
        for t in range(d // 2):
            zc = complex(x[ri, 0, t], x[ri, 0, t + d // 2])
            zc *= complex(math.cos(p * theta ** (-2 * t / d)), math.sin(p * theta ** (-2 * t / d)))
            assert y[ri, 0, t] == pytest.approx(zc.real, abs=1e-12)
            assert y[ri, 0, t + d // 2] == pytest.approx(zc.imag, abs=1e-12)
    # relative-position property of the rotated dot product
    a = O.rope(x[:1], [3], theta)[0, 0] @ O.rope(x[1:2], [10], theta)[0, 0]
    b = O.rope(x[:1], [53], theta)[0, 0] @ O.rope(x[1:2], [60], theta)[0, 0]
    assert a == pytest.approx(b, rel=1e-10)


def _tiny_full(seed, L=2, n=9, hq=4, hkv=2, d=8, D=16, F=24, V=40):
    r = np.random.default_rng(seed)
    W = [dict(attn_norm=1 + 0.1 * r.standard_normal(D), wq=0.3 * r.standard_normal((hq * d, D)),
              wo=0.3 * r.standard_normal((D, hq * d)), mlp_norm=1 + 0.1 * r.standard_normal(D),
              w_gate=0.3 * r.standard_normal((F, D)), w_up=0.3 * r.standard_normal((F, D)),
              w_down=0.3 * r.standard_normal((D, F))) for _ in range(L)]
    KV = [(r.standard_normal((hkv, n, d)), r.standard_normal((hkv, n, d))) for _ in range(L)]
    emb = r.standard_normal((V, D))
    fn = 1 + 0.1 * r.standard_normal(D)
    wl = 0.3 * r.standard_normal((V, D))
    ids = r.integers(0, V, n)
    return dict(W=W, KV=KV, emb=emb, fn=fn, wl=wl, ids=ids, L=L, n=n, hq=hq, hkv=hkv, d=d)


def _torch_full(t, theta, eps):
    """The same pass composed from torch library routines (rms_norm, complex-number
    rotary embedding, scaled_dot_product_attention with the j > i mask, silu,
    log_softmax) in float64."""
    F_ = torch.nn.functional
    n, hq, hkv, d = t["n"], t["hq"], t["hkv"], t["d"]
    g = hq // hkv
    T = lambda a: torch.as_tensor(np.asarray(a, dtype=np.float64))
    h = T(t["emb"])[torch.as_tensor(t["ids"])]
    pos = torch.arange(n, dtype=torch.float64)
    inv = theta ** (-2.0 * torch.arange(d // 2, dtype=torch.float64) / d)
    rot = torch.polar(torch.ones(n, d // 2, dtype=torch.float64), pos[:, None] * inv[None])
    allow = torch.triu(torch.ones(n, n, dtype=torch.bool), diagonal=1)
    for l in range(t["L"]):
        W = {k: T(v) for k, v in t["W"][l].items()}
        K, Vv = (T(x) for x in t["KV"][l])
        a = F_.rms_norm(h, (h.shape[-1],), W["attn_norm"], eps)
        q = (a @ W["wq"].T).reshape(n, hq, d)
        qc = torch.complex(q[..., : d // 2], q[..., d // 2:]) * rot[:, None, :]
        q = torch.cat([qc.real, qc.imag], dim=-1)
        o = F_.scaled_dot_product_attention(q.permute(1, 0, 2), K.repeat_interleave(g, 0),
                                            Vv.repeat_interleave(g, 0), attn_mask=allow)
        o = torch.nan_to_num(o.permute(1, 0, 2), nan=0.0)   # empty last row -> 0
        h = h + o.reshape(n, -1) @ W["wo"].T
        b = F_.rms_norm(h, (h.shape[-1],), W["mlp_norm"], eps)
        h = h + (F_.silu(b @ W["w_gate"].T) * (b @ W["w_up"].T)) @ W["w_down"].T
    u = F_.rms_norm(h, (h.shape[-1],), T(t["fn"]), eps)
    logp = torch.log_softmax(u @ T(t["wl"]).T, dim=-1)
    s = -logp[torch.arange(n), torch.as_tensor(t["ids"])].numpy()
    s[-1] = np.inf
    return s


def _oracle_full(t, theta, eps, rows=None):
    return O.full_scores(t["ids"], lambda l: t["KV"][l], lambda l: t["W"][l], t["emb"], t["fn"],
                         t["wl"], [0, t["n"]], t["L"], t["hq"], t["d"], theta, eps, rows=rows)


@pytest.mark.parametrize("L", [1, 3])
def test_full_pass_vs_library_composition(L):
    t = _tiny_full(seed=L, L=L)
    theta, eps = 5e5, 1e-5
    np.testing.assert_allclose(_oracle_full(t, theta, eps), _torch_full(t, theta, eps),
                               rtol=1e-10, atol=1e-10)


def test_full_pass_row_subset_is_exact():
    t = _tiny_full(seed=7, L=2)
    full = _oracle_full(t, 1e4, 1e-5)
    rows = [0, 4, 8]
    np.testing.assert_allclose(_oracle_full(t, 1e4, 1e-5, rows=rows), full[rows], rtol=1e-13)


def test_full_pass_zero_query_weights_reduce_to_suffix_means():
    """W_q = 0 makes every query 0, so each layer's attention is the suffix mean of
    that layer's stored values; with W_o, W_down = 0 except in layer 0's W_o the
    final hidden state is E[x] + W_o^0 (suffix mean), a closed form."""
    t = _tiny_full(seed=3, L=2)
    for l in range(2):
        t["W"][l]["wq"] = np.zeros_like(t["W"][l]["wq"])
        t["W"][l]["w_down"] = np.zeros_like(t["W"][l]["w_down"])
    t["W"][1]["wo"] = np.zeros_like(t["W"][1]["wo"])
    n, hq, hkv, d = t["n"], t["hq"], t["hkv"], t["d"]
    V0 = t["KV"][0][1]
    cs = np.cumsum(V0[:, ::-1], axis=1)[:, ::-1]
    y = np.zeros((n, hq, d))
    for i in range(n - 1):
        for h in range(hq):
            y[i, h] = cs[h // (hq // hkv), i + 1] / (n - 1 - i)
    hfin = t["emb"][t["ids"]] + y.reshape(n, -1) @ t["W"][0]["wo"].T
    u = hfin / np.sqrt((hfin ** 2).mean(-1, keepdims=True) + 1e-5) * t["fn"]
    z = u @ t["wl"].T
    want = scipy.special.logsumexp(z, axis=1) - z[np.arange(n), t["ids"]]
    got = _oracle_full(t, 5e5, 1e-5)
    np.testing.assert_allclose(got[:-1], want[:-1], rtol=1e-12)


# ---------------------------------------------------------------- exact fast variant

def _torch_last_h(t, H, pos, theta, eps):
    """One layer from H composed from torch library routines (as _torch_full), queries
    rotated at the given original positions, then the final norm and log_softmax."""
    F_ = torch.nn.functional
    n, hq, hkv, d = t["n"], t["hq"], t["hkv"], t["d"]
    g = hq // hkv
    T = lambda a: torch.as_tensor(np.asarray(a, dtype=np.float64))
    W = {k: T(v) for k, v in t["W"][-1].items()}
    K, Vv = (T(x) for x in t["KV"][-1])
    h = T(H)
    inv = theta ** (-2.0 * torch.arange(d // 2, dtype=torch.float64) / d)
    rot = torch.polar(torch.ones(n, d // 2, dtype=torch.float64),
                      T(pos)[:, None] * inv[None])
    allow = torch.triu(torch.ones(n, n, dtype=torch.bool), diagonal=1)
    a = F_.rms_norm(h, (h.shape[-1],), W["attn_norm"], eps)
    q = (a @ W["wq"].T).reshape(n, hq, d)
    qc = torch.complex(q[..., : d // 2], q[..., d // 2:]) * rot[:, None, :]
    q = torch.cat([qc.real, qc.imag], dim=-1)
    o = F_.scaled_dot_product_attention(q.permute(1, 0, 2), K.repeat_interleave(g, 0),
                                        Vv.repeat_interleave(g, 0), attn_mask=allow)
    o = torch.nan_to_num(o.permute(1, 0, 2), nan=0.0)
    h = h + o.reshape(n, -1) @ W["wo"].T
    b = F_.rms_norm(h, (h.shape[-1],), W["mlp_norm"], eps)
    h = h + (F_.silu(b @ W["w_gate"].T) * (b @ W["w_up"].T)) @ W["w_down"].T
    u = F_.rms_norm(h, (h.shape[-1],), T(t["fn"]), eps)
    logp = torch.log_softmax(u @ T(t["wl"]).T, dim=-1)
    s = -logp[torch.arange(n), torch.as_tensor(t["ids"])].numpy()
    s[-1] = np.inf
    return s


def _oracle_last_h(t, H, theta, eps, pos_ids=None, rows=None):
    K, V = t["KV"][-1]
    return O.last_layer_h_scores(H, t["ids"], K, V, t["W"][-1], t["fn"], t["wl"], [0, t["n"]],
                                 t["hq"], t["d"], theta, eps, pos_ids=pos_ids, rows=rows)


def test_last_layer_h_vs_library_composition():
    """Stored activations of an arbitrary scale and original positions that are not
    0..n-1 (as after earlier refreshes)."""
    t = _tiny_full(seed=11, L=2)
    r = np.random.default_rng(5)
    H = 3.0 * r.standard_normal((t["n"], t["W"][0]["wq"].shape[1]))
    pos = np.sort(r.choice(200, t["n"], replace=False))
    theta, eps = 5e5, 1e-5
    got = _oracle_last_h(t, H, theta, eps, pos_ids=pos)
    np.testing.assert_allclose(got, _torch_last_h(t, H, pos, theta, eps), rtol=1e-10, atol=1e-10)
    rows = [1, 5, 8]
    np.testing.assert_allclose(_oracle_last_h(t, H, theta, eps, pos_ids=pos, rows=rows), got[rows],
                               rtol=1e-13)


def test_last_layer_h_with_embeddings_is_one_layer_full_pass():
    t = _tiny_full(seed=12, L=1)
    H = t["emb"][t["ids"]]
    np.testing.assert_allclose(_oracle_last_h(t, H, 1e4, 1e-5), _oracle_full(t, 1e4, 1e-5),
                               rtol=1e-13)


def test_last_layer_h_zero_query_weights_closed_form():
    """W_q = 0 gives uniform attention (suffix means of V); with W_down = 0 the final
    hidden state is H + W_o (suffix means), a closed form."""
    t = _tiny_full(seed=13, L=1)
    t["W"][0]["wq"] = np.zeros_like(t["W"][0]["wq"])
    t["W"][0]["w_down"] = np.zeros_like(t["W"][0]["w_down"])
    r = np.random.default_rng(3)
    n, hq, hkv, d = t["n"], t["hq"], t["hkv"], t["d"]
    H = r.standard_normal((n, t["W"][0]["wq"].shape[1]))
    V0 = t["KV"][0][1]
    cs = np.cumsum(V0[:, ::-1], axis=1)[:, ::-1]
    y = np.zeros((n, hq, d))
    for i in range(n - 1):
        for h in range(hq):
            y[i, h] = cs[h // (hq // hkv), i + 1] / (n - 1 - i)
    hfin = H + y.reshape(n, -1) @ t["W"][0]["wo"].T
    u = hfin / np.sqrt((hfin ** 2).mean(-1, keepdims=True) + 1e-5) * t["fn"]
    z = u @ t["wl"].T
    want = scipy.special.logsumexp(z, axis=1) - z[np.arange(n), t["ids"]]
    got = _oracle_last_h(t, H, 5e5, 1e-5)
    np.testing.assert_allclose(got[:-1], want[:-1], rtol=1e-12)
    assert got[-1] == np.inf
