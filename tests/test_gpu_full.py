"""GPU parity of the full L-layer counter-causal pass (cc_score in FULL mode) against the
oracle: fresh queries from the token embeddings through RMSNorm, W_q and RoPE at the
original positions, attention on each layer's stored keys/values, W_o and the SwiGLU
MLP with residuals, final RMSNorm and the LM head."""
import numpy as np
import pytest
import torch

from oracle import cc_oracle as O
from synth import configs as C
from tests.gpu_util import assert_scores_close

pytestmark = pytest.mark.gpu


def _full_case(cfg, rows=None):
    from paper_2607_27600_amd import cc
    from paper_2607_27600_amd.workload import Workload
    print(f"[full] {cfg.name} lens={cfg.seq_lens} L={cfg.n_layers} D={cfg.hidden} F={cfg.ffn}",
          flush=True)
    w = Workload(cfg, keep_host=True)
    scores = torch.full((cfg.n_tokens,), float("nan"), dtype=torch.float32, device="cuda")
    cc.cc_score(w.problem, w.inputs(), scores)
    torch.cuda.synchronize()
    got = scores.cpu().numpy()
    h = w.host
    kvl = h["kv_layers"]
    # the cache holds the generator's layers in order (cache_layers == n_layers here)
    ref = O.full_scores(h["ids"], lambda l: (kvl[l]["k"], kvl[l]["v"]), lambda l: h["layers"][l],
                        h["embed"], h["final_norm"], h["w_lm"], cfg.cu_seqlens, cfg.n_layers,
                        cfg.n_heads_q, cfg.head_dim, cfg.rope_theta, cfg.rms_eps, rows=rows)
    return (got if rows is None else got[rows]), ref


def test_full_small_two_layers_all_rows():
    cfg = C.shrink(C.C4, seq_lens=(300,), n_layers=2, cache_layers=2, hidden=256, ffn=512,
                   vocab=1000, n_heads_q=4, n_heads_kv=2, keep=(75,))
    got, ref = _full_case(cfg)
    print(assert_scores_close(got, ref, "bf16", "full-small"))


def test_full_ragged_batch_gqa_all_rows():
    cfg = C.shrink(C.C4, seq_lens=(70, 1, 200), n_layers=3, cache_layers=3, hidden=512, ffn=1024,
                   vocab=3000, n_heads_q=8, n_heads_kv=2, keep=(10, 1, 50))
    got, ref = _full_case(cfg)
    print(assert_scores_close(got, ref, "bf16", "full-ragged"))


def test_full_paged_pool_all_rows():
    """Every layer's keys/values read from a shuffled paged pool (16-key pages)."""
    cfg = C.shrink(C.C4, seq_lens=(150, 33, 64), n_layers=2, cache_layers=2, hidden=256, ffn=512,
                   vocab=1000, n_heads_q=4, n_heads_kv=2, keep=(30, 7, 12), paged=True,
                   page_size=16)
    got, ref = _full_case(cfg)
    print(assert_scores_close(got, ref, "bf16", "full-paged"))
