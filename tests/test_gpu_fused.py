"""GPU parity of the LM head with W_o folded in: the product weight W_lm W_o
(cc_fuse_wo_lmhead) against the fp64 product of the inputs, and the scores of mode
LAST_LAYER_FUSED against the oracle's two-step chain attention -> W_o -> LM head
(Sec. 3.1 fast variant with the queries given; the fusion is associativity, so the
bf16 tolerance only has to cover the one extra rounding of the product weight)."""
import numpy as np
import pytest
import torch

from oracle import cc_oracle as O
from synth import configs as C
from synth import gen
from tests.gpu_util import assert_scores_close, dev, f64

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("dtype,V,D,Q", [("bf16", 1000, 256, 512), ("bf16", 257, 320, 384),
                                         ("f32", 300, 128, 96)])
def test_fuse_weight_matches_product(dtype, V, D, Q):
    from paper_2607_27600_amd import cc
    print(f"[fuse] {dtype} V={V} D={D} Q={Q}", flush=True)
    r = np.random.default_rng(V + D)
    wl = (0.05 * r.standard_normal((V, D))).astype(np.float32)
    wo = (0.05 * r.standard_normal((D, Q))).astype(np.float32)
    if dtype == "bf16":
        wl, wo = gen.f32_to_bf16_bits(wl), gen.f32_to_bf16_bits(wo)
    out = cc.cc_fuse_wo_lmhead(dtype, dev(wl), dev(wo))
    torch.cuda.synchronize()
    assert out.shape == (V, Q)
    ref = O.fused_lmhead_weight(wl, wo)
    if dtype == "bf16":
        # fp32 accumulation of exact products, then one bf16 rounding (2^-9 relative)
        np.testing.assert_allclose(f64(out), ref, rtol=4e-3, atol=1e-5)
    else:
        np.testing.assert_allclose(f64(out), ref, rtol=0, atol=1e-5)


def _fused_case(cfg, rows=None):
    from paper_2607_27600_amd import cc
    from paper_2607_27600_amd.workload import Workload
    print(f"[fused score] {cfg.name} lens={cfg.seq_lens[:8]} dtype={cfg.dtype} paged={cfg.paged}",
          flush=True)
    w = Workload(cfg, cache_layers=1, keep_host=True)
    p = cc.problem(dtype=cfg.dtype, cu_seqlens=cfg.cu_seqlens.tolist(), n_heads_q=cfg.n_heads_q,
                   n_heads_kv=cfg.n_heads_kv, head_dim=cfg.head_dim, hidden=cfg.hidden,
                   vocab=cfg.vocab, mode="last_layer_fused")
    m = cc.cc_fuse_wo_lmhead(cfg.dtype, w.w_lm, w.w_o)
    inp = cc.inputs(kv=w.kv, token_ids=w.ids, w_lm=m, q=w.q)
    scores = torch.full((cfg.n_tokens,), float("nan"), dtype=torch.float32, device="cuda")
    cc.cc_score(p, inp, scores)
    torch.cuda.synchronize()
    h = w.host
    ref, spread = O.last_layer_scores(h["q"], h["k"], h["v"], h["w_o"], h["w_lm"], h["ids"],
                                      cfg.cu_seqlens, rows=rows, spread=True)
    got = scores.cpu().numpy()
    return (got if rows is None else got[rows]), ref, spread


def test_fused_scores_c1_fp32():
    got, ref, _ = _fused_case(C.C1)
    print("C1 fused", assert_scores_close(got, ref, "f32", "C1 fused"))


def test_fused_scores_bf16_small():
    cfg = C.shrink(C.C2, seq_lens=(300,), hidden=256, vocab=1000, cache_layers=1)
    got, ref, spread = _fused_case(cfg)
    print("bf16 fused", assert_scores_close(got, ref, "bf16", "bf16-small fused", spread))


def test_fused_scores_bf16_paged_ragged():
    cfg = C.shrink(C.C5, seq_lens=(33, 1, 150, 64), hidden=512, vocab=3000, cache_layers=1,
                   keep=(1, 1, 1, 1))
    got, ref, spread = _fused_case(cfg)
    print("paged fused", assert_scores_close(got, ref, "bf16", "paged-small fused", spread))


def test_two_step_mode_requires_w_o():
    """The two-step mode still requires W_o (the fused mode, run above, takes none)."""
    from paper_2607_27600_amd import cc
    from paper_2607_27600_amd.workload import Workload
    cfg = C.shrink(C.C2, seq_lens=(64,), hidden=256, vocab=500, cache_layers=1)
    w = Workload(cfg, cache_layers=1)
    scores = torch.empty(cfg.n_tokens, dtype=torch.float32, device="cuda")
    inp = cc.inputs(kv=w.kv, token_ids=w.ids, w_lm=w.w_lm, q=w.q)
    with pytest.raises(cc.CCError):
        cc.cc_score(w.problem, inp, scores)


@pytest.mark.slow
def test_fused_scores_c2_sampled():
    rows = C.sample_rows(C.C2, count=48)
    got, ref, spread = _fused_case(C.C2, rows=rows)
    print("C2 fused", assert_scores_close(got, ref, "bf16", "C2 fused", spread))
