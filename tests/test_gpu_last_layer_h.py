"""GPU parity of the exact fast variant (cc_score, mode LAST_LAYER_H) and of the
compaction of per-entry rows (cc_compact_rows) that carries the stored activations H.

Scores are compared with the oracle at small ragged shapes on every row (norm gains
drawn away from 1, original positions not 0..n-1) and at the Llama-3-8B shapes on
sampled rows; row compaction is a bit copy compared byte for byte."""
import numpy as np
import pytest
import torch

from oracle import cc_oracle as O
from synth import configs as C
from synth import gen
from tests.gpu_util import assert_scores_close, bf16_host, dev

pytestmark = pytest.mark.gpu


def _small():
    return C.shrink(C.C2H, seq_lens=(300, 77, 1, 2), n_heads_q=4, n_heads_kv=2, hidden=256,
                    ffn=512, vocab=1000, cache_layers=2, keep=(75, 19, 1, 1))


def _ref(w, rows=None, pos_ids=None, W=None, fn=None):
    cfg, h = w.cfg, w.host
    return O.last_layer_h_scores(h["h_last"], h["ids"], h["k"], h["v"], W or h["layer"],
                                 h["final_norm"] if fn is None else fn, h["w_lm"], cfg.cu_seqlens,
                                 cfg.n_heads_q, cfg.head_dim, cfg.rope_theta, cfg.rms_eps,
                                 pos_ids=pos_ids, rows=rows)


def test_small_ragged_all_rows_with_gains_and_positions():
    from paper_2607_27600_amd import cc
    from paper_2607_27600_amd.workload import Workload
    cfg = _small()
    print(f"[last_layer_h] lens={cfg.seq_lens}", flush=True)
    w = Workload(cfg, keep_host=True)
    r = np.random.default_rng(4)
    # norm gains away from 1 (device and host copies agree bit for bit)
    W = dict(w.host["layer"])
    for name in ("attn_norm", "mlp_norm"):
        g = gen.f32_to_bf16_bits((1 + 0.2 * r.standard_normal(cfg.hidden)).astype(np.float32))
        W[name] = g
        w.layers[0][name].copy_(dev(g))
    fn = gen.f32_to_bf16_bits((1 + 0.2 * r.standard_normal(cfg.hidden)).astype(np.float32))
    w.final_norm.copy_(dev(fn))
    # original positions with gaps, ascending within each sequence
    cu = cfg.cu_seqlens
    pos = np.concatenate([np.sort(r.choice(4 * max(1, n) + 8, n, replace=False))
                          for n in cfg.seq_lens]).astype(np.int32)
    pos_d = torch.from_numpy(pos).cuda()
    inp = cc.inputs(kv=w.kv, token_ids=w.ids, w_lm=w.w_lm, layers=w.layers,
                    final_norm=w.final_norm, h_last=w.h_last, pos_ids=pos_d)
    scores = torch.full((cfg.n_tokens,), float("nan"), device="cuda")
    cc.cc_score(w.problem, inp, scores)
    torch.cuda.synchronize()
    ref = _ref(w, pos_ids=pos, W=W, fn=fn)
    print("[last_layer_h] small", assert_scores_close(scores.cpu().numpy(), ref, "bf16", "small"))
    # last entry of every sequence is +inf, including the length-1 and length-2 ones
    assert np.all(np.isinf(scores.cpu().numpy()[cu[1:] - 1]))


def test_split_k_projections_all_rows():
    """Shapes whose projections are cut along K (their 256 x 256 tiles fill under half the
    chip): W_q in 4 slices (hidden 1024), W_o in 4, W_down in 5 with a short last slice
    (ffn 2944 = 46 k-tiles of 64: four slices of 10 and one of 6), against the oracle on
    every row."""
    from paper_2607_27600_amd import cc
    from paper_2607_27600_amd.workload import Workload
    cfg = C.shrink(C.C2H, seq_lens=(300, 45), n_heads_q=8, n_heads_kv=2, hidden=1024,
                   ffn=2944, vocab=1000, cache_layers=1, keep=(75, 11))
    print(f"[last_layer_h] split-K lens={cfg.seq_lens} D={cfg.hidden} F={cfg.ffn}", flush=True)
    w = Workload(cfg, keep_host=True)
    scores = torch.full((cfg.n_tokens,), float("nan"), device="cuda")
    cc.cc_score(w.problem, w.inputs(), scores)
    torch.cuda.synchronize()
    print("[last_layer_h] split-K", assert_scores_close(scores.cpu().numpy(), _ref(w), "bf16",
                                                        "split-K"))


@pytest.mark.slow
def test_c2h_sampled_rows():
    from paper_2607_27600_amd import cc
    from paper_2607_27600_amd.workload import Workload
    cfg = C.C2H
    print("[last_layer_h] C2H n=4096", flush=True)
    w = Workload(cfg, cache_layers=1, keep_host=True)
    scores = torch.empty(cfg.n_tokens, device="cuda")
    cc.cc_score(w.problem, w.inputs(), scores)
    torch.cuda.synchronize()
    rows = C.sample_rows(cfg, count=48)
    print("[last_layer_h] C2H", assert_scores_close(scores.cpu().numpy()[rows], _ref(w, rows=rows),
                                                    "bf16", "C2H"))


@pytest.mark.parametrize("in_place", [True, False])
@pytest.mark.parametrize("per_head", [0, 1])
def test_compact_rows(in_place, per_head):
    """H rows follow each sequence's (first) keep list, in place or out of place; rows of
    a width that is not a multiple of 256 bytes use narrower column slabs."""
    from paper_2607_27600_amd import cc
    print(f"[compact_rows] in_place={in_place} per_head={per_head}", flush=True)
    lens = (300, 1, 77, 1025)
    hq, hkv = 4, 2
    p = cc.problem(dtype="bf16", cu_seqlens=np.concatenate([[0], np.cumsum(lens)]).tolist(),
                   n_heads_q=hq, n_heads_kv=hkv, head_dim=128, hidden=256, vocab=1000)
    r = np.random.default_rng(8 + per_head)
    lists, ks = [], []
    for n in lens:
        for h in range(hkv if per_head else 1):
            k = int(r.integers(1, n + 1))
            lists.append(np.sort(r.choice(n, k, replace=False)).astype(np.int32))
            ks.append(k)
    keep = torch.from_numpy(np.concatenate(lists)).cuda()
    cu = p.cu_h.numpy()
    for width in (256, 48):                                   # bf16 elements per row
        rows_h = r.integers(0, 1 << 16, (int(cu[-1]), width), dtype=np.uint16)
        rows_d = dev(rows_h)
        out = torch.zeros_like(rows_d) if not in_place else None
        cc.cc_compact_rows(p, rows_d, keep, ks, per_head, out=out)
        torch.cuda.synchronize()
        got = bf16_host(out if out is not None else rows_d)
        for b, n in enumerate(lens):
            lst = lists[b * (hkv if per_head else 1)]
            lo = int(cu[b])
            np.testing.assert_array_equal(got[lo:lo + len(lst)], O.compact(rows_h[lo:lo + n], lst),
                                          err_msg=f"seq {b} width {width}")
            if in_place:   # rows past the kept prefix are untouched
                np.testing.assert_array_equal(got[lo + len(lst):lo + n], rows_h[lo + len(lst):lo + n])
