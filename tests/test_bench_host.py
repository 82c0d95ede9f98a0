"""Host-side checks of bench.py (no GPU): the one-GPU contract, the default workload list and
the per-row work model by which the oracle's sampled time is extrapolated."""
import os
import subprocess
import sys

import numpy as np

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)


def test_more_than_one_gpu_exits_with_a_message():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"],
                       capture_output=True, text=True, timeout=120)
    assert r.returncode == 2
    assert "one GPU" in r.stderr
    assert r.stdout == ""


def test_default_workloads_exist_and_the_headline_is_largest_by_entries():
    import bench
    from synth import configs as C
    names = bench.DEFAULT_CONFIGS.split(",")
    assert all(n in C.CONFIGS for n in names)
    tokens = {n: C.CONFIGS[n].n_tokens for n in names}
    assert tokens[names[0]] == max(tokens.values())


def test_row_work_model_matches_the_algorithmic_counts():
    """Summed over all rows, the per-row FLOPs equal the whole-pass formulas: attention
    4 d Hq per allowed key, W_o (last layer), one layer's projections and MLP (exact fast
    variant) or all layers' (full pass), and the LM head."""
    import bench
    from synth import configs as C
    for name in ("C2", "C2H", "C4"):
        cfg = C.CONFIGS[name]
        N, hq, d, D, V, F = cfg.n_tokens, cfg.n_heads_q, cfg.head_dim, cfg.hidden, cfg.vocab, cfg.ffn
        att = 2.0 * d * hq * sum(n * (n - 1) for n in cfg.seq_lens)
        lm = 2.0 * N * D * V
        per_layer = 2.0 * N * D * hq * d * 2 + 2.0 * N * D * F * 3
        want = {"last_layer": att + 2.0 * N * D * hq * d + lm,
                "last_layer_h": per_layer + att + lm,
                "full": cfg.n_layers * (per_layer + att) + lm}[cfg.mode]
        got = bench._row_flops(cfg, np.arange(N)).sum()
        assert abs(got - want) <= 1e-9 * want, (name, got, want)
