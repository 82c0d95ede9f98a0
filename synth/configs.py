"""The five synthetic workloads of the refresh-scoring pass, and their inputs.

Shapes follow the model families and cache sizes the paper evaluates (Llama-3-8B
and Qwen2.5-7B shapes, caches of 256 to 32768 entries); values are seeded random
draws (there are no trained weights here).  Every tensor has a fixed id so each
can be drawn on its own, e.g. a single layer of a 32-layer cache.

This module only describes shapes and draws inputs; it computes nothing of the
method itself.
"""
from __future__ import annotations

import dataclasses
from typing import Optional

import numpy as np

from . import gen

# tensor ids (per-layer tensors add the layer index)
T_Q, T_WO, T_WLM, T_IDS, T_LENS, T_PAGES, T_EMBED, T_H = 1, 4, 5, 6, 7, 8, 9, 10
T_K_LAYER, T_V_LAYER = 1000, 2000
T_WQ, T_WO_L, T_WG, T_WU, T_WD = 3000, 4000, 5000, 6000, 7000


@dataclasses.dataclass(frozen=True)
class Config:
    name: str
    dtype: str                 # "f32" or "bf16"
    mode: str                  # "last_layer", "full" or "last_layer_h"
    seq_lens: tuple            # cached tokens per sequence
    n_heads_q: int
    n_heads_kv: int
    head_dim: int
    hidden: int
    vocab: int
    cache_layers: int          # layers held by the cache (compaction covers all)
    keep: tuple                # keep budget per sequence
    per_head_select: bool = False
    paged: bool = False
    page_size: int = 16
    n_layers: int = 1          # FULL: transformer layers run; LAST_LAYER_H: model depth
    ffn: int = 0
    rope_theta: float = 5e5
    rms_eps: float = 1e-5
    w_std: float = 0.02
    seed: int = 0
    description: str = ""

    @property
    def n_seqs(self) -> int:
        return len(self.seq_lens)

    @property
    def n_tokens(self) -> int:
        return int(sum(self.seq_lens))

    @property
    def group(self) -> int:
        return self.n_heads_q // self.n_heads_kv

    @property
    def cu_seqlens(self) -> np.ndarray:
        return np.concatenate([[0], np.cumsum(self.seq_lens)]).astype(np.int32)


def _c5_lengths(seed: int) -> tuple:
    lens = gen.uniform_ints(seed, T_LENS, (8,), 2048, 16385)
    return tuple(int(x) for x in lens)


def _c5_keep(lens) -> tuple:
    return tuple(max(1, min(n, int(np.floor(0.2 * n)))) for n in lens)


C1 = Config("C1", "f32", "last_layer", (256,), 2, 1, 64, 128, 1024, 1, (64,),
            description="tiny last-layer scoring, fp32: n=256, 2q/1kv heads, d=64, "
                        "hidden 128, vocab 1024, keep 64")
C2 = Config("C2", "bf16", "last_layer", (4096,), 32, 8, 128, 4096, 128256, 32, (1024,),
            description="Llama-3-8B shapes, last-layer scoring, bf16: n=4096, 32q/8kv, "
                        "d=128, hidden 4096, vocab 128256, keep 25%, 32-layer cache")
C3 = Config("C3", "bf16", "last_layer", (32768,), 32, 8, 128, 4096, 128256, 32, (4096,),
            per_head_select=True,
            description="Llama-3-8B shapes at n=32768, bf16: last-layer scoring, "
                        "keep 4096 per KV head, 32-layer cache")
C4 = Config("C4", "bf16", "full", (8192,), 32, 8, 128, 4096, 128256, 32, (2048,),
            n_layers=32, ffn=14336,
            description="full 32-layer pass, 8B-shaped random stack, bf16: n=8192, "
                        "SwiGLU 14336, RMSNorm, RoPE theta 5e5, keep 25%")
_C5_LENS = _c5_lengths(0)
C5 = Config("C5", "bf16", "last_layer", _C5_LENS, 28, 4, 128, 3584, 152064, 28,
            _c5_keep(_C5_LENS), paged=True, page_size=16,
            description="ragged batch of 8, lengths U[2048,16384], Qwen2.5-7B shapes "
                        "(28q/4kv, hidden 3584, vocab 152064), paged cache P=16, keep 20%")

C2H = Config("C2H", "bf16", "last_layer_h", (4096,), 32, 8, 128, 4096, 128256, 32, (1024,),
             n_layers=32, ffn=14336,
             description="Llama-3-8B shapes, exact fast variant from the stored activations "
                         "entering the last layer, bf16: n=4096, SwiGLU 14336, keep 25%, "
                         "32-layer cache")

CONFIGS = {c.name: c for c in (C1, C2, C3, C4, C5, C2H)}


def shrink(cfg: Config, **kw) -> Config:
    """A copy of ``cfg`` with some fields replaced (for small test variants)."""
    return dataclasses.replace(cfg, **kw)


# ----------------------------------------------------------------------------------
# input drawing
# ----------------------------------------------------------------------------------

def _normal(cfg: Config, tid: int, shape, std: float):
    if cfg.dtype == "f32":
        return gen.normal_f32(cfg.seed, tid, shape, std)
    return gen.normal_bf16(cfg.seed, tid, shape, std)


def widen(cfg: Config, a: np.ndarray) -> np.ndarray:
    """Exact float64 copy of a stored tensor (bf16 bits or fp32)."""
    if a.dtype == np.uint16:
        return gen.bf16_to_f64(a)
    return a.astype(np.float64)


def draw_q(cfg: Config) -> np.ndarray:
    """Queries [N][Hq][d], N(0,1)."""
    return _normal(cfg, T_Q, (cfg.n_tokens, cfg.n_heads_q, cfg.head_dim), 1.0)


def draw_h_last(cfg: Config) -> np.ndarray:
    """Stored activations entering the last layer [N][D], N(0,1) (RMSNorm makes the
    layer insensitive to their overall scale)."""
    return _normal(cfg, T_H, (cfg.n_tokens, cfg.hidden), 1.0)


def draw_kv_layer(cfg: Config, layer: int, which: str) -> np.ndarray:
    """One cache layer of keys or values, token-major per KV head: [Hkv][N][d], N(0,1).

    For a batch the sequences are concatenated along the token axis (by cu_seqlens)."""
    tid = (T_K_LAYER if which == "k" else T_V_LAYER) + layer
    return _normal(cfg, tid, (cfg.n_heads_kv, cfg.n_tokens, cfg.head_dim), 1.0)


def draw_wo(cfg: Config, layer: Optional[int] = None) -> np.ndarray:
    """Output projection [D][Hq*d], N(0, w_std^2)."""
    tid = T_WO if layer is None else T_WO_L + layer
    return _normal(cfg, tid, (cfg.hidden, cfg.n_heads_q * cfg.head_dim), cfg.w_std)


def draw_wlm(cfg: Config) -> np.ndarray:
    """LM head [V][D], N(0, w_std^2)."""
    return _normal(cfg, T_WLM, (cfg.vocab, cfg.hidden), cfg.w_std)


def draw_ids(cfg: Config) -> np.ndarray:
    """Cached token ids, uniform on [0, V)."""
    return gen.uniform_ints(cfg.seed, T_IDS, (cfg.n_tokens,), 0, cfg.vocab)


def draw_embed(cfg: Config) -> np.ndarray:
    return _normal(cfg, T_EMBED, (cfg.vocab, cfg.hidden), cfg.w_std)


def draw_layer_weights(cfg: Config, layer: int) -> dict:
    """Weights of one transformer layer (FULL mode); norm gains are 1."""
    D, F, Hd = cfg.hidden, cfg.ffn, cfg.n_heads_q * cfg.head_dim
    one = gen.f32_to_bf16_bits(np.ones(D, np.float32)) if cfg.dtype == "bf16" else np.ones(D, np.float32)
    return {
        "attn_norm": one,
        "wq": _normal(cfg, T_WQ + layer, (Hd, D), cfg.w_std),
        "wo": draw_wo(cfg, layer),
        "mlp_norm": one.copy(),
        "w_gate": _normal(cfg, T_WG + layer, (F, D), cfg.w_std),
        "w_up": _normal(cfg, T_WU + layer, (F, D), cfg.w_std),
        "w_down": _normal(cfg, T_WD + layer, (D, F), cfg.w_std),
    }


def final_norm(cfg: Config) -> np.ndarray:
    one = np.ones(cfg.hidden, np.float32)
    return gen.f32_to_bf16_bits(one) if cfg.dtype == "bf16" else one


def page_table(cfg: Config):
    """Paged layout: pages of ``page_size`` slots placed in a shuffled pool.

    Returns (block_table [B][max_pages] int32, n_pages).  Unused entries are -1."""
    P = cfg.page_size
    npg = [(n + P - 1) // P for n in cfg.seq_lens]
    total = int(sum(npg))
    perm = gen.permutation(cfg.seed, T_PAGES, total)
    maxp = max(npg)
    bt = np.full((cfg.n_seqs, maxp), -1, np.int32)
    o = 0
    for b, m in enumerate(npg):
        bt[b, :m] = perm[o:o + m]
        o += m
    return bt, total


def sample_rows(cfg: Config, count: int = 256, seed: int = 12345) -> np.ndarray:
    """A fixed sample of global row indices: per sequence its first and last rows,
    the rest uniform, sorted and unique."""
    rng = np.random.Generator(np.random.Philox(key=np.array([seed, 77], np.uint64)))
    cu = cfg.cu_seqlens
    picks = []
    per = max(2, count // cfg.n_seqs)
    edge = max(1, min(16, per // 16))
    for b in range(cfg.n_seqs):
        lo, hi = int(cu[b]), int(cu[b + 1])
        n = hi - lo
        picks.extend(range(lo, lo + min(edge, n)))
        picks.extend(range(max(lo, hi - edge), hi))
        rest = per - 2 * edge
        if rest > 0 and n > 0:
            picks.extend(rng.integers(lo, hi, size=rest).tolist())
    return np.unique(np.array(picks, dtype=np.int64))
