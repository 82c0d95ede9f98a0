"""Device-resident synthetic workloads for the refresh-scoring pass.

Draws a configuration's inputs with the seeded generator (synth), uploads them once,
and lays the KV cache out as the library expects: contiguous [L][Hkv][cap][d] per
sequence, or paged [L][pages][Hkv][P][d] pools with a shuffled block table.  Host
copies of what was uploaded can be kept for checking.  Nothing here computes any part
of the method.
"""
from __future__ import annotations

from typing import Optional

import numpy as np
import torch

from synth import configs as C

from . import cc


def to_device(a: np.ndarray, device) -> torch.Tensor:
    """Upload a host array; uint16 arrays are bf16 bit patterns."""
    if a.dtype == np.uint16:
        return torch.from_numpy(np.ascontiguousarray(a).view(np.int16)).view(torch.bfloat16).to(device)
    return torch.from_numpy(np.ascontiguousarray(a)).to(device)


class Workload:
    """Inputs of one configuration on the GPU.

    cache_layers: how many cache layers to hold (default: the configuration's).  Only
    the last one is scored in the fast variant; the others exist for compaction.
    keep_host: keep host copies (q, k/v of the scored layer, weights, ids) for checks."""

    def __init__(self, cfg: C.Config, device="cuda", cache_layers: Optional[int] = None,
                 keep_host: bool = False, with_lm_head: bool = True):
        self.cfg = cfg
        self.device = torch.device(device)
        L = cfg.cache_layers if cache_layers is None else cache_layers
        self.cache_layers = L
        d, hkv = cfg.head_dim, cfg.n_heads_kv
        self.host = {}
        self.problem = cc.problem(dtype=cfg.dtype, cu_seqlens=cfg.cu_seqlens.tolist(),
                                  n_heads_q=cfg.n_heads_q, n_heads_kv=hkv, head_dim=d,
                                  hidden=cfg.hidden, vocab=cfg.vocab, device=device,
                                  mode=cfg.mode, n_layers=cfg.n_layers if cfg.mode == "full" else 0,
                                  ffn=cfg.ffn, rope_theta=cfg.rope_theta, rms_eps=cfg.rms_eps)
        ids = C.draw_ids(cfg)
        self.ids = to_device(ids, device)
        if keep_host:
            self.host["ids"] = ids
        if cfg.mode == "last_layer":
            q = C.draw_q(cfg)
            self.q = to_device(q, device)
            wo = C.draw_wo(cfg)
            self.w_o = to_device(wo, device)
            if keep_host:
                self.host.update(q=q, w_o=wo)
        elif cfg.mode == "last_layer_h":
            self.q = None
            self.w_o = None
            hl = C.draw_h_last(cfg)
            self.h_last = to_device(hl, device)
            W = C.draw_layer_weights(cfg, cfg.n_layers - 1)
            self.layers = [{k: to_device(v, device) for k, v in W.items()}]
            fn = C.final_norm(cfg)
            self.final_norm = to_device(fn, device)
            if keep_host:
                self.host.update(h_last=hl, layer=W, final_norm=fn)
        else:
            self.q = None
            self.w_o = None
            emb = C.draw_embed(cfg)
            self.embed = to_device(emb, device)
            fn = C.final_norm(cfg)
            self.final_norm = to_device(fn, device)
            self.layers = []
            host_layers = []
            for l in range(cfg.n_layers):
                W = C.draw_layer_weights(cfg, l)
                self.layers.append({k: to_device(v, device) for k, v in W.items()})
                if keep_host:
                    host_layers.append(W)
            if keep_host:
                self.host.update(embed=emb, final_norm=fn, layers=host_layers)
        if with_lm_head:
            wlm = C.draw_wlm(cfg)
            self.w_lm = to_device(wlm, device)
            if keep_host:
                self.host["w_lm"] = wlm
        else:
            self.w_lm = None
        self._build_cache(L, keep_host)

    # ------------------------------------------------------------------ KV cache
    def _layer_index(self, l: int) -> int:
        """Cache layer l holds generator layer (cfg.cache_layers - L + l): the scored last
        layer is the same tensor whatever number of layers is held."""
        return self.cfg.cache_layers - self.cache_layers + l

    def _build_cache(self, L: int, keep_host: bool) -> None:
        cfg = self.cfg
        d, hkv, N = cfg.head_dim, cfg.n_heads_kv, cfg.n_tokens
        tdt = torch.bfloat16 if cfg.dtype == "bf16" else torch.float32
        cu = cfg.cu_seqlens
        if cfg.paged:
            P = cfg.page_size
            bt, n_pages = C.page_table(cfg)
            self.block_table = torch.from_numpy(bt).to(self.device)
            self.k_cache = torch.empty((L, n_pages, hkv, P, d), dtype=tdt, device=self.device)
            self.v_cache = torch.empty_like(self.k_cache)
            for l in range(L):
                for which, dst in (("k", self.k_cache), ("v", self.v_cache)):
                    src = C.draw_kv_layer(cfg, self._layer_index(l), which)   # [Hkv][N][d]
                    pool = np.zeros((n_pages, hkv, P, d), dtype=src.dtype)
                    for b in range(cfg.n_seqs):
                        n = int(cu[b + 1] - cu[b])
                        for p in range((n + P - 1) // P):
                            lo = int(cu[b]) + p * P
                            hi = min(int(cu[b + 1]), lo + P)
                            pool[bt[b, p], :, : hi - lo] = src[:, lo:hi]
                    dst[l].copy_(to_device(pool, "cpu"))
                    if keep_host and l == L - 1:
                        self.host[which] = src
                    if keep_host and cfg.mode == "full":
                        self.host.setdefault("kv_layers", {}).setdefault(l, {})[which] = src
            self.kv = cc.kv_paged(self.k_cache, self.v_cache, self.block_table, n_layers=L,
                                  layer_stride=n_pages * hkv * P * d, page_stride=hkv * P * d,
                                  head_stride=P * d, tok_stride=d, page_size=P)
        else:
            cap = int(max(cfg.seq_lens))
            B = cfg.n_seqs
            self.k_cache = torch.empty((B, L, hkv, cap, d), dtype=tdt, device=self.device)
            self.v_cache = torch.empty_like(self.k_cache)
            for l in range(L):
                for which, dst in (("k", self.k_cache), ("v", self.v_cache)):
                    src = C.draw_kv_layer(cfg, self._layer_index(l), which)
                    for b in range(B):
                        lo, hi = int(cu[b]), int(cu[b + 1])
                        dst[b, l, :, : hi - lo].copy_(to_device(np.ascontiguousarray(src[:, lo:hi]), "cpu"))
                    if keep_host and l == L - 1:
                        self.host[which] = src
                    if keep_host and cfg.mode == "full":
                        self.host.setdefault("kv_layers", {}).setdefault(l, {})[which] = src
            self.kv = cc.kv_contiguous(self.k_cache, self.v_cache, n_layers=L,
                                       seq_stride=L * hkv * cap * d, layer_stride=hkv * cap * d,
                                       head_stride=cap * d, tok_stride=d)

    def inputs(self, w_lm_packed=None) -> cc.Inputs:
        """cc_score inputs; w_lm_packed (cc_pack_lmhead of w_lm) for a packed problem."""
        if self.cfg.mode == "last_layer_h":
            return cc.inputs(kv=self.kv, token_ids=self.ids, w_lm=self.w_lm, layers=self.layers,
                             final_norm=self.final_norm, h_last=self.h_last,
                             w_lm_packed=w_lm_packed)
        if self.cfg.mode == "full":
            return cc.inputs(kv=self.kv, token_ids=self.ids, w_lm=self.w_lm, embed=self.embed,
                             layers=self.layers, final_norm=self.final_norm,
                             w_lm_packed=w_lm_packed)
        return cc.inputs(q=self.q, kv=self.kv, token_ids=self.ids, w_o=self.w_o, w_lm=self.w_lm,
                         w_lm_packed=w_lm_packed)

    def keep_budget(self) -> list:
        return list(self.cfg.keep)
