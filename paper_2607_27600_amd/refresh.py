"""The cache-managed inference cycle around the refresh pass (Sec. 3.2, algorithm summary).

A sequence's cache holds up to J + h entries: the J kept by the last refresh followed by
the entries appended since.  `append` adds new entries (their keys and values for every
cache layer, token ids, original positions, and the per-entry rows the scoring mode
needs: queries for the given-query fast variant, the activations entering the last
layer for the exact fast variant).  `refresh` runs one memory-refresh cycle: the
counter-causal score of every cached entry, selection of the J highest (kept in their
original order), and compaction of keys, values, ids, positions and rows.  `run_stream`
drives a prompt and a decode phase, refreshing every h tokens (chunked mode) or once at
the end of the prompt (prefill-end mode).

Everything here is orchestration on the caller's stream; every step of the pass runs in
libcc.  Entries keep the absolute positions they were appended with.
"""
from __future__ import annotations

import dataclasses
from typing import Callable, Optional

import torch

from . import cc


@dataclasses.dataclass
class Model:
    """Shapes and weights the scoring pass needs (device tensors in bf16)."""
    mode: str                         # "last_layer" (queries given), "last_layer_fused" (queries
                                      # given, w_lm = W_lm W_o) or "last_layer_h"
    n_layers: int                     # cache layers
    n_heads_q: int
    n_heads_kv: int
    head_dim: int
    hidden: int
    vocab: int
    w_lm: torch.Tensor
    w_o: Optional[torch.Tensor] = None          # last_layer
    layer: Optional[dict] = None                # last_layer_h: the last layer's weights
    final_norm: Optional[torch.Tensor] = None   # last_layer_h
    ffn: int = 0
    rope_theta: float = 5e5
    rms_eps: float = 1e-5
    w_lm_packed: Optional[torch.Tensor] = None  # cc_pack_lmhead(w_lm): the packed LM head

    @property
    def row_width(self) -> int:
        """Elements of the per-entry row the mode scores from (Q or H)."""
        return self.hidden if self.mode == "last_layer_h" else self.n_heads_q * self.head_dim


class RefreshLoop:
    """One sequence's cache under counter-causal memory management."""

    def __init__(self, model: Model, J: int, h: int, device="cuda",
                 capacity: Optional[int] = None):
        if model.mode not in ("last_layer", "last_layer_fused", "last_layer_h"):
            raise ValueError("mode must be last_layer, last_layer_fused or last_layer_h")
        if J < 1 or h < 1:
            raise ValueError("J and h must be positive")
        self.m, self.J, self.h = model, J, h
        self.device = torch.device(device)
        cap = capacity if capacity is not None else J + h   # chunked mode needs J + h
        self.cap = cap
        L, hkv, d = model.n_layers, model.n_heads_kv, model.head_dim
        bf = torch.bfloat16
        self.k = torch.zeros((L, hkv, cap, d), dtype=bf, device=self.device)
        self.v = torch.zeros_like(self.k)
        self.ids = torch.zeros(cap, dtype=torch.int32, device=self.device)
        self.pos = torch.zeros(cap, dtype=torch.int32, device=self.device)
        self.rows = torch.zeros((cap, model.row_width), dtype=bf, device=self.device)
        self.n = 0
        self.kv = cc.kv_contiguous(self.k, self.v, n_layers=L, layer_stride=hkv * cap * d,
                                   head_stride=cap * d, tok_stride=d)
        self.refreshes = 0

    # ---------------------------------------------------------------- inference side
    def append(self, k: torch.Tensor, v: torch.Tensor, ids: torch.Tensor, pos: torch.Tensor,
               rows: torch.Tensor) -> None:
        """Append m entries: k, v [L][Hkv][m][d]; ids, pos [m]; rows [m][row_width]."""
        m = int(ids.shape[0])
        if self.n + m > self.cap:
            raise ValueError(f"cache holds {self.n} of {self.cap}; refresh before appending {m}")
        sl = slice(self.n, self.n + m)
        self.k[:, :, sl].copy_(k)
        self.v[:, :, sl].copy_(v)
        self.ids[sl].copy_(ids)
        self.pos[sl].copy_(pos)
        self.rows[sl].copy_(rows)
        self.n += m

    # ---------------------------------------------------------------- refresh cycle
    def problem(self) -> cc.Problem:
        m = self.m
        return cc.problem(dtype="bf16", cu_seqlens=[0, self.n], n_heads_q=m.n_heads_q,
                          n_heads_kv=m.n_heads_kv, head_dim=m.head_dim, hidden=m.hidden,
                          vocab=m.vocab, device=self.device, mode=m.mode, ffn=m.ffn,
                          rope_theta=m.rope_theta, rms_eps=m.rms_eps,
                          lmhead_packed=m.w_lm_packed is not None)

    def inputs(self) -> cc.Inputs:
        m, n = self.m, self.n
        if m.mode in ("last_layer", "last_layer_fused"):
            return cc.inputs(kv=self.kv, token_ids=self.ids, w_lm=m.w_lm, w_o=m.w_o,
                             q=self.rows[:n], w_lm_packed=m.w_lm_packed)
        return cc.inputs(kv=self.kv, token_ids=self.ids, w_lm=m.w_lm, layers=[m.layer],
                         final_norm=m.final_norm, h_last=self.rows[:n], pos_ids=self.pos,
                         w_lm_packed=m.w_lm_packed)

    def scores(self) -> torch.Tensor:
        """Counter-causal surprise of every cached entry (the last one is +inf)."""
        s = torch.empty(self.n, dtype=torch.float32, device=self.device)
        cc.cc_score(self.problem(), self.inputs(), s)
        return s

    def refresh(self, hook: Optional[Callable] = None) -> torch.Tensor:
        """One memory-refresh cycle; returns the keep list (indices into the entries as
        they were).  `hook(scores, keep)` sees both before the cache is rewritten."""
        if self.n <= self.J:
            return torch.arange(self.n, dtype=torch.int32, device=self.device)
        p = self.problem()
        s = self.scores()
        keep = torch.empty(self.J, dtype=torch.int32, device=self.device)
        cc.cc_select_keep(s, [0], [self.n], [self.J], keep)
        if hook is not None:
            hook(s, keep)
        cc.cc_compact_kv(p, self.kv, keep, [self.J], 0, token_ids=self.ids, pos_ids=self.pos)
        cc.cc_compact_rows(p, self.rows, keep, [self.J], 0)
        self.n = self.J
        self.refreshes += 1
        return keep


def run_stream(loop: RefreshLoop, entry: Callable, T_prompt: int, T_total: int,
               chunked: bool = True, hook: Optional[Callable] = None) -> None:
    """Drive a stream of T_total tokens through the cache.  `entry(t0, t1)` returns the
    (k, v, ids, pos, rows) of tokens t0..t1-1 (the inference cycle's new keys, values,
    token ids, positions and rows).  Chunked mode refreshes whenever the token count
    reaches a multiple of h: the prompt is appended in batches up to each refresh point,
    the decode phase one token at a time.  Prefill-end mode appends the whole prompt,
    refreshes once, then decodes without refreshing (the cache must hold the prompt and
    the decoded tokens)."""
    h = loop.h
    t = 0
    while t < T_prompt:
        t1 = min(T_prompt, (t // h + 1) * h) if chunked else T_prompt
        loop.append(*entry(t, t1))
        t = t1
        if chunked and t % h == 0:
            loop.refresh(hook)
    if not chunked:
        loop.refresh(hook)
    while t < T_total:
        loop.append(*entry(t, t + 1))
        t += 1
        if chunked and t % h == 0:
            loop.refresh(hook)
