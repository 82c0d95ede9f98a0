"""Plain float64 CPU oracle of the counter-causal refresh-scoring pass.

TEST INFRASTRUCTURE ONLY.  This module is the checker the HIP path is measured
against; only the tests, the smoke check and the benchmark's CPU-baseline leg may
import it.  It shares no code with the HIP path and never calls it.

What it computes (Gould & van den Hengel, "Back from the Future: Key-Value Cache
Management by Counter-Causal Surprise"):

* Counter-causal attention (Sec. 3.1, with Eq. (2)): each cached position i attends
  only to later positions j > i of the same sequence, reusing the stored keys and
  values; with GQA query head h reads KV head floor(h / g).
* The fast single-layer variant (Sec. 3.1, "Fast single-layer approximation"):
  attention in the last layer only, then that layer's output projection and the LM
  head give one distribution per position.
* The full variant (Sec. 3.1): every layer of a pre-norm transformer (RMSNorm, RoPE
  at the original position ids, SwiGLU MLP) runs with fresh queries against the
  stored keys/values of that layer.
* The per-entry surprise score (Eq. (5), and Sec. 3.1 on using the output at the
  cached token): score_i = -log P(x_i | x_{i+1:n}) = logsumexp(z_i) - z_i[x_i],
  a strictly decreasing function of P, so ranking by it equals ranking by
  s_i = 1 - P.  The last entry of each sequence has no future and gets +inf, as do
  frozen sink entries (Sec. 3.2, last paragraph).
* Keep selection and compaction (Sec. 3.2, the memory-refresh procedure): keep the
  k highest-scoring entries, ties to the lower index, stored in ascending original
  order, and gather every per-entry tensor with that list.

Everything is float64; inputs given as bf16 bit patterns (uint16) or fp32 are
widened exactly.  Functions accept ``rows`` to score only a subset of positions:
keys and values are read from the cache, never recomputed, so rows never interact
and any subset is exact on its own.
"""
from __future__ import annotations

import math
from typing import Callable, Optional, Sequence

import numpy as np


# ----------------------------------------------------------------------------------
# storage widening (exact)
# ----------------------------------------------------------------------------------

def f64(a: np.ndarray) -> np.ndarray:
    """Exact float64 copy of a tensor stored as bf16 bit patterns (uint16) or float."""
    a = np.asarray(a)
    if a.dtype == np.uint16:
        return (a.astype(np.uint32) << np.uint32(16)).view(np.float32).astype(np.float64)
    return a.astype(np.float64)


# ----------------------------------------------------------------------------------
# attention (Eq. (2) with the counter-causal mask of Sec. 3.1)
# ----------------------------------------------------------------------------------

def allowed_keys(i: int, n: int, diag: str = "strict") -> range:
    """Cache positions row i may attend to: j > i (the paper's mask), or j >= i."""
    if diag == "strict":
        return range(i + 1, n)
    if diag == "inclusive":
        return range(i, n)
    raise ValueError(diag)


def attention_cc(q, k, v, diag: str = "strict", scale: Optional[float] = None,
                 rows: Optional[Sequence[int]] = None) -> np.ndarray:
    """Counter-causal attention for one sequence.

    q: [n][Hq][d]; k, v: [Hkv][n][d].  Returns o: [len(rows)][Hq][d] (all rows by
    default).  Row i, head h: softmax over j in allowed_keys(i) of
    scale * <q[i,h], k[c,j]> with c = h // (Hq/Hkv), weights applied to v[c,j].
    A row with no allowed key has output 0."""
    q = f64(q)
    k = f64(k)
    v = f64(v)
    n, hq, d = q.shape
    hkv = k.shape[0]
    assert hq % hkv == 0 and k.shape == (hkv, n, d) and v.shape == (hkv, n, d)
    g = hq // hkv
    tau = 1.0 / math.sqrt(d) if scale is None else float(scale)
    rows = range(n) if rows is None else rows
    out = np.zeros((len(rows), hq, d))
    for r, i in enumerate(rows):
        a = allowed_keys(int(i), n, diag)
        if len(a) == 0:
            continue
        js = np.arange(a.start, a.stop)
        for c in range(hkv):
            heads = slice(c * g, (c + 1) * g)
            e = tau * (q[i, heads] @ k[c, js].T)            # [g][|A_i|]
            m = e.max(axis=1, keepdims=True)
            w = np.exp(e - m)
            w /= w.sum(axis=1, keepdims=True)
            out[r, heads] = w @ v[c, js]
    return out


# ----------------------------------------------------------------------------------
# LM head, log-softmax at the cached token, surprise score (Eq. (5), Sec. 3.1)
# ----------------------------------------------------------------------------------

def lm_head_logits(u, w_lm, vocab_chunk: int = 8192) -> np.ndarray:
    """z = u W_lm^T for rows u [R][D], W_lm [V][D] -> [R][V] (float64).

    W_lm is widened in vocabulary slices only to bound memory; each logit is the
    same dot product whatever the slicing."""
    u = f64(u)
    V = w_lm.shape[0]
    z = np.empty((u.shape[0], V))
    for lo in range(0, V, vocab_chunk):
        hi = min(V, lo + vocab_chunk)
        z[:, lo:hi] = u @ f64(w_lm[lo:hi]).T
    return z


def logsumexp_rows(z: np.ndarray) -> np.ndarray:
    m = z.max(axis=1)
    return m + np.log(np.exp(z - m[:, None]).sum(axis=1))


def surprise(u, w_lm, ids, spread: bool = False) -> tuple:
    """Returns (score, lse, z_target) per row: score = lse(z) - z[x] = -log P(x).

    spread=True appends the standard deviation of z over the vocabulary per row.  It is
    not part of the method: the parity tests use it to size the rounding error a score
    can carry, since the score moves with its input u through z."""
    z = lm_head_logits(u, w_lm)
    lse = logsumexp_rows(z)
    zt = z[np.arange(z.shape[0]), np.asarray(ids, dtype=np.int64)]
    if spread:
        return lse - zt, lse, zt, z.std(axis=1)
    return lse - zt, lse, zt


def edge_rows(cu_seqlens, n_frozen: int = 0) -> np.ndarray:
    """Boolean mask over all N rows: True where the score is +inf by rule (the last
    entry of each sequence, and the first n_frozen entries of each sequence)."""
    cu = np.asarray(cu_seqlens, dtype=np.int64)
    mask = np.zeros(int(cu[-1]), dtype=bool)
    for b in range(len(cu) - 1):
        lo, hi = int(cu[b]), int(cu[b + 1])
        if hi > lo:
            mask[hi - 1] = True
            mask[lo:min(hi, lo + max(0, n_frozen))] = True
    return mask


def _rows_by_seq(cu, rows):
    cu = np.asarray(cu, dtype=np.int64)
    rows = np.asarray(rows, dtype=np.int64)
    seq = np.searchsorted(cu, rows, side="right") - 1
    return seq


# ----------------------------------------------------------------------------------
# fast (last-layer) variant
# ----------------------------------------------------------------------------------

def attention_rows(q, k, v, cu_seqlens, diag="strict", scale=None, rows=None) -> np.ndarray:
    """y_i = concat_h(o_{i,h}), the counter-causal attention output of the requested
    global rows, head-major.

    q: [N][Hq][d]; k, v: [Hkv][N][d] (sequences concatenated by cu_seqlens)."""
    cu = np.asarray(cu_seqlens, dtype=np.int64)
    N = int(cu[-1])
    rows = np.arange(N) if rows is None else np.asarray(rows, dtype=np.int64)
    seq = _rows_by_seq(cu, rows)
    hq, d = q.shape[1], q.shape[2]
    y = np.zeros((len(rows), hq * d))
    for b in np.unique(seq):
        lo, hi = int(cu[b]), int(cu[b + 1])
        sel = np.nonzero(seq == b)[0]
        local = rows[sel] - lo
        o = attention_cc(q[lo:hi], k[:, lo:hi], v[:, lo:hi], diag, scale, local)
        y[sel] = o.reshape(len(sel), hq * d)
    return y


def last_layer_hidden(q, k, v, w_o, cu_seqlens, diag="strict", scale=None,
                      rows=None) -> np.ndarray:
    """u_i = W_o concat_h(o_{i,h}) for the requested global rows."""
    return attention_rows(q, k, v, cu_seqlens, diag, scale, rows) @ f64(w_o).T


def last_layer_scores(q, k, v, w_o, w_lm, ids, cu_seqlens, diag="strict", scale=None,
                      n_frozen=0, rows=None, spread: bool = False):
    """Surprise scores of the fast variant for the requested rows (all by default).
    spread=True also returns the per-row logit spread (see surprise)."""
    cu = np.asarray(cu_seqlens, dtype=np.int64)
    N = int(cu[-1])
    rows = np.arange(N) if rows is None else np.asarray(rows, dtype=np.int64)
    u = last_layer_hidden(q, k, v, w_o, cu, diag, scale, rows)
    out = surprise(u, w_lm, np.asarray(ids)[rows], spread=spread)
    s = out[0]
    s[edge_rows(cu, n_frozen)[rows]] = np.inf
    return (s, out[3]) if spread else s


def fused_lmhead_weight(w_lm, w_o) -> np.ndarray:
    """M = W_lm W_o, [V][Hq*d].  With the queries given, the fast variant's output
    processing is the bare projection W_o (Sec. 3.1), so z = W_lm (W_o y) = M y."""
    return f64(w_lm) @ f64(w_o)


def last_layer_fused_scores(q, k, v, w_fused, ids, cu_seqlens, diag="strict", scale=None,
                            n_frozen=0, rows=None, spread: bool = False):
    """Surprise scores of the fast variant with the LM head applied to the attention rows
    through a given product weight w_fused = W_lm W_o [V][Hq*d]."""
    cu = np.asarray(cu_seqlens, dtype=np.int64)
    N = int(cu[-1])
    rows = np.arange(N) if rows is None else np.asarray(rows, dtype=np.int64)
    y = attention_rows(q, k, v, cu, diag, scale, rows)
    out = surprise(y, w_fused, np.asarray(ids)[rows], spread=spread)
    s = out[0]
    s[edge_rows(cu, n_frozen)[rows]] = np.inf
    return (s, out[3]) if spread else s


# ----------------------------------------------------------------------------------
# full variant: pre-norm transformer with fresh queries, stored keys/values
# ----------------------------------------------------------------------------------

def rmsnorm(x, gamma, eps) -> np.ndarray:
    x = np.asarray(x, dtype=np.float64)
    return x / np.sqrt(np.mean(x * x, axis=-1, keepdims=True) + eps) * f64(gamma)


def rope(x, pos, theta) -> np.ndarray:
    """Rotate-half rotary embedding: pairs (t, t + d/2) turned by pos * theta^(-2t/d).

    x: [R][H][d]; pos: [R]."""
    x = np.asarray(x, dtype=np.float64)
    d = x.shape[-1]
    half = d // 2
    inv = float(theta) ** (-2.0 * np.arange(half) / d)
    ang = np.asarray(pos, dtype=np.float64)[:, None] * inv[None, :]   # [R][half]
    c = np.cos(ang)[:, None, :]
    s = np.sin(ang)[:, None, :]
    a, b = x[..., :half], x[..., half:]
    return np.concatenate([a * c - b * s, b * c + a * s], axis=-1)


def silu(x):
    return x / (1.0 + np.exp(-x))


def _layer(h, W, K, V, rows, seq, pos, cu, n_heads_q, head_dim, theta, eps, diag, scale):
    """One pre-norm transformer layer for the requested rows with fresh queries against
    the stored keys/values K, V ([Hkv][N][d], already rotated): RMSNorm, W_q, RoPE at
    `pos`, counter-causal attention (Eq. (2) under the Sec. 3.1 mask), W_o + residual,
    RMSNorm, SwiGLU MLP + residual."""
    R = len(rows)
    a = rmsnorm(h, W["attn_norm"], eps)
    q = (a @ f64(W["wq"]).T).reshape(R, n_heads_q, head_dim)
    q = rope(q, pos, theta)
    y = np.zeros((R, n_heads_q * head_dim))
    for b in np.unique(seq):
        lo, hi = int(cu[b]), int(cu[b + 1])
        sel = np.nonzero(seq == b)[0]
        n = hi - lo
        qfull = np.zeros((n, n_heads_q, head_dim))
        qfull[rows[sel] - lo] = q[sel]
        o = attention_cc(qfull, K[:, lo:hi], V[:, lo:hi], diag, scale, rows[sel] - lo)
        y[sel] = o.reshape(len(sel), -1)
    h = h + y @ f64(W["wo"]).T
    bn = rmsnorm(h, W["mlp_norm"], eps)
    act = silu(bn @ f64(W["w_gate"]).T) * (bn @ f64(W["w_up"]).T)
    return h + act @ f64(W["w_down"]).T


def _rows_pos(cu_seqlens, rows, pos_ids):
    cu = np.asarray(cu_seqlens, dtype=np.int64)
    N = int(cu[-1])
    rows = np.arange(N) if rows is None else np.asarray(rows, dtype=np.int64)
    seq = _rows_by_seq(cu, rows)
    if pos_ids is None:
        pos = rows - cu[seq]
    else:
        pos = np.asarray(pos_ids, dtype=np.int64)[rows]
    return cu, rows, seq, pos


def full_scores(ids, kv_layer: Callable, layer_weights: Callable, embed, final_norm_w,
                w_lm, cu_seqlens, n_layers, n_heads_q, head_dim, theta, eps,
                diag="strict", scale=None, pos_ids=None, n_frozen=0,
                rows=None) -> np.ndarray:
    """Surprise scores of the full L-layer counter-causal pass for the requested rows.

    kv_layer(l) -> (K_l, V_l) as [Hkv][N][d] (already rotated, as stored);
    layer_weights(l) -> dict(attn_norm, wq, wo, mlp_norm, w_gate, w_up, w_down)."""
    cu, rows, seq, pos = _rows_pos(cu_seqlens, rows, pos_ids)
    ids = np.asarray(ids, dtype=np.int64)
    h = f64(embed[ids[rows]])                                        # [R][D]
    for l in range(n_layers):
        K, V = kv_layer(l)
        h = _layer(h, layer_weights(l), K, V, rows, seq, pos, cu, n_heads_q, head_dim, theta,
                   eps, diag, scale)
    u = rmsnorm(h, final_norm_w, eps)
    s, _, _ = surprise(u, w_lm, ids[rows])
    s[edge_rows(cu, n_frozen)[rows]] = np.inf
    return s


def last_layer_h_scores(h_last, ids, K, V, W, final_norm_w, w_lm, cu_seqlens, n_heads_q,
                        head_dim, theta, eps, diag="strict", scale=None, pos_ids=None,
                        n_frozen=0, rows=None) -> np.ndarray:
    """The fast single-layer approximation in its exact form (Sec. 3.1): the stored
    activations H entering the last layer ([N][D]) go through that layer with fresh
    queries (RoPE at the original positions) against the layer's stored K, V, then the
    final RMSNorm and the LM head; scores as in Eq. (5) read as surprisal."""
    cu, rows, seq, pos = _rows_pos(cu_seqlens, rows, pos_ids)
    ids = np.asarray(ids, dtype=np.int64)
    h = _layer(f64(np.asarray(h_last)[rows]), W, K, V, rows, seq, pos, cu, n_heads_q, head_dim,
               theta, eps, diag, scale)
    u = rmsnorm(h, final_norm_w, eps)
    s, _, _ = surprise(u, w_lm, ids[rows])
    s[edge_rows(cu, n_frozen)[rows]] = np.inf
    return s


# ----------------------------------------------------------------------------------
# LM head on an FP8-quantized model (an implementation variant of the surprise score,
# Eq. (5); the paper fixes no precision).  FP8 is the OCP E4M3 ("FN") format: sign,
# 4 exponent bits (bias 7), 3 mantissa bits, subnormals, no infinities, 0x7F / 0xFF NaN,
# largest finite 448.  Activations u get one scale per row, the LM head one scale for the
# whole matrix; both are chosen in fp32 so the largest magnitude maps to 448.
# ----------------------------------------------------------------------------------

E4M3_MAX = 448.0


def e4m3_decode(codes) -> np.ndarray:
    """Value of each E4M3 code (uint8) as float64; NaN for 0x7F / 0xFF."""
    c = np.asarray(codes, dtype=np.int64)
    sign = np.where(c & 0x80, -1.0, 1.0)
    e = (c >> 3) & 0xF
    m = (c & 7).astype(np.float64)
    mag = np.where(e == 0, m * 2.0 ** -9, (1.0 + m / 8.0) * np.exp2(e - 7.0))
    mag = np.where((e == 0xF) & ((c & 7) == 7), np.nan, mag)
    return sign * mag


# the 127 non-negative finite values, code 0x00 .. 0x7E, ascending
_E4M3_POS = e4m3_decode(np.arange(0x7F))


def e4m3_encode(x) -> np.ndarray:
    """Nearest E4M3 code of each value (round to nearest, ties to the even code, i.e. the
    even mantissa); magnitudes above 448 saturate to 448; -0.0 keeps its sign."""
    x = np.asarray(x, dtype=np.float64)
    a = np.abs(x)
    lo = np.clip(np.searchsorted(_E4M3_POS, a, side="right") - 1, 0, 0x7E)   # v[lo] <= a
    hi = np.minimum(lo + 1, 0x7E)
    dlo = a - _E4M3_POS[lo]
    dhi = _E4M3_POS[hi] - a
    take_hi = (dhi < dlo) | ((dhi == dlo) & (hi != lo) & (hi % 2 == 0))
    code = np.where(take_hi, hi, lo)
    code = np.where(a >= E4M3_MAX, 0x7E, code)
    neg = np.signbit(x)
    code = np.where(neg, code | 0x80, code)
    return np.where(np.isnan(x), 0x7F, code).astype(np.uint8)


def quantize_fp8(x, per_row: bool = True, row_chunk: int = 4096):
    """(codes, scale): x ~= decode(codes) * scale.  Per row (or over the whole matrix):
    amax = max |x|, codes = E4M3(x * (448 / amax)), scale = amax / 448, every step in
    fp32 as stored (an all-zero row gets codes 0, scale 0).  Rows are processed in
    slices only to bound memory; each code depends on its element and amax alone."""
    R = x.shape[0]
    amax = np.empty(R, dtype=np.float32)
    for lo in range(0, R, row_chunk):
        amax[lo:lo + row_chunk] = np.abs(f64(x[lo:lo + row_chunk]).astype(np.float32)).max(axis=1)
    if not per_row:
        amax = np.array([amax.max()], dtype=np.float32)
    nz = amax > 0
    inv = np.zeros_like(amax)
    inv[nz] = np.float32(E4M3_MAX) / amax[nz]
    scale = (amax / np.float32(E4M3_MAX)).astype(np.float32)
    codes = np.empty(x.shape, dtype=np.uint8)
    for lo in range(0, R, row_chunk):
        x32 = f64(x[lo:lo + row_chunk]).astype(np.float32)
        f = inv[lo:lo + row_chunk, None] if per_row else inv[0]
        codes[lo:lo + row_chunk] = e4m3_encode((x32 * f).astype(np.float32))
    return codes, scale


def lmhead_fp8_scores(u, w_codes, w_scale, ids, cu_seqlens, n_frozen=0, rows=None,
                      vocab_chunk: int = 8192):
    """Surprise scores (Eq. (5) read as -log P) of rows u [R][D] through an FP8 LM head:
    u is quantized per row as in quantize_fp8, W_lm is given as E4M3 codes [V][D] with one
    fp32 scale, and z = (sum over d of the decoded products) * scale_u * scale_w exactly.
    ``rows`` lists the global row of each u row (all rows by default)."""
    cu = np.asarray(cu_seqlens, dtype=np.int64)
    qu, su = quantize_fp8(u, per_row=True)
    U = e4m3_decode(qu)
    R = U.shape[0]
    rows = np.arange(R) if rows is None else np.asarray(rows, dtype=np.int64)
    V = w_codes.shape[0]
    z = np.empty((R, V))
    for lo in range(0, V, vocab_chunk):
        hi = min(V, lo + vocab_chunk)
        z[:, lo:hi] = U @ e4m3_decode(w_codes[lo:hi]).T
    z *= su.astype(np.float64)[:, None] * float(w_scale)
    lse = logsumexp_rows(z)
    ids = np.asarray(ids, dtype=np.int64)
    s = lse - z[np.arange(R), ids]
    s[edge_rows(cu, n_frozen)[rows]] = np.inf
    return s


# ----------------------------------------------------------------------------------
# keep selection and compaction (Sec. 3.2, memory refresh)
# ----------------------------------------------------------------------------------

def _order_key(score: float, index: int):
    """Sort key for 'keep first': larger score first, NaN after everything, ties by
    lower index.  -0.0 and +0.0 compare equal."""
    s = float(score)
    if math.isnan(s):
        return (1, 0.0, index)
    return (0, -s, index)


def select_keep(scores, k: int) -> np.ndarray:
    """Indices of the k entries kept from one segment, in ascending order."""
    scores = np.asarray(scores)
    n = len(scores)
    if not 0 <= k <= n:
        raise ValueError("k out of range")
    order = sorted(range(n), key=lambda i: _order_key(scores[i], i))
    return np.array(sorted(order[:k]), dtype=np.int32)


def compact(rows, keep) -> np.ndarray:
    """Gather along the entry axis (axis 0): out[j] = rows[keep[j]], a bit copy."""
    rows = np.asarray(rows)
    out = np.empty((len(keep),) + rows.shape[1:], dtype=rows.dtype)
    for j, src in enumerate(keep):
        out[j] = rows[int(src)]
    return out
