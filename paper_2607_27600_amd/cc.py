"""ctypes binding of libcc (include/cc.h): argument marshalling only.

Every function here has the name of the C entry point it calls.  Tensors are torch
tensors on the GPU; the binding passes their data pointers, the current HIP stream and
a workspace tensor it allocates through torch.  All arithmetic runs in libcc's HIP
kernels; there is no fallback: if libcc.so is missing or fails to load, importing this
module raises.
"""
from __future__ import annotations

import ctypes
import os
from dataclasses import dataclass, field
from typing import Optional, Sequence

import numpy as np
import torch

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libcc.so")

(CC_OK, CC_ERR_ARG, CC_ERR_SHAPE, CC_ERR_DTYPE, CC_ERR_WORKSPACE, CC_ERR_UNSUPPORTED, CC_ERR_HIP,
 CC_ERR_SCRATCH) = range(8)
CC_NOALLOC_SCRATCH_BYTES = 32 << 20
CC_F32, CC_BF16 = 0, 1
CC_DIAG_STRICT, CC_DIAG_INCLUSIVE = 0, 1
CC_MODE_LAST_LAYER, CC_MODE_FULL, CC_MODE_LAST_LAYER_H, CC_MODE_LAST_LAYER_FUSED = 0, 1, 2, 3
CC_KV_CONTIGUOUS, CC_KV_PAGED = 0, 1

EXPORTED = [
    "cc_status_str", "cc_version", "cc_score_workspace", "cc_score", "cc_attention_workspace",
    "cc_attention_cc", "cc_lmhead_workspace", "cc_lmhead_score", "cc_linear",
    "cc_select_workspace", "cc_select_keep", "cc_compact_workspace", "cc_compact_kv",
    "cc_compact_rows_workspace", "cc_compact_rows", "cc_fuse_wo_lmhead_workspace",
    "cc_fuse_wo_lmhead", "cc_quantize_fp8_workspace", "cc_quantize_fp8",
    "cc_lmhead_fp8_workspace", "cc_lmhead_score_fp8", "cc_pack_lmhead_bytes", "cc_pack_lmhead",
    "cc_lmhead_score_packed", "cc_lmhead_score_noalloc",
]

_c_void_p = ctypes.c_void_p
_i32 = ctypes.c_int32
_i64 = ctypes.c_int64


class c_kv(ctypes.Structure):
    _fields_ = [("layout", _i32), ("n_layers", _i32), ("k", _c_void_p), ("v", _c_void_p),
                ("seq_stride", _i64), ("layer_stride", _i64), ("head_stride", _i64),
                ("tok_stride", _i64), ("page_stride", _i64), ("block_table", _c_void_p),
                ("page_size", _i32), ("max_pages", _i32)]


class c_problem(ctypes.Structure):
    _fields_ = [("dtype", _i32), ("mode", _i32), ("diag", _i32), ("n_seqs", _i32),
                ("cu_seqlens_h", ctypes.POINTER(_i32)), ("cu_seqlens_d", _c_void_p),
                ("n_heads_q", _i32), ("n_heads_kv", _i32), ("head_dim", _i32),
                ("hidden", _i32), ("vocab", _i32), ("n_layers", _i32), ("ffn", _i32),
                ("softmax_scale", ctypes.c_float), ("rope_theta", ctypes.c_float),
                ("rms_eps", ctypes.c_float), ("n_frozen", _i32), ("lmhead_packed", _i32)]


class c_layer_weights(ctypes.Structure):
    _fields_ = [("attn_norm", _c_void_p), ("wq", _c_void_p), ("wo", _c_void_p),
                ("mlp_norm", _c_void_p), ("w_gate", _c_void_p), ("w_up", _c_void_p),
                ("w_down", _c_void_p)]


class c_inputs(ctypes.Structure):
    _fields_ = [("q", _c_void_p), ("kv", c_kv), ("token_ids", _c_void_p), ("pos_ids", _c_void_p),
                ("w_o", _c_void_p), ("w_lm", _c_void_p), ("embed", _c_void_p),
                ("layers_h", ctypes.POINTER(c_layer_weights)), ("final_norm", _c_void_p),
                ("h_last", _c_void_p), ("w_lm_packed", _c_void_p)]


def _load():
    if not os.path.exists(LIB_PATH):
        raise ImportError(f"libcc.so not built at {LIB_PATH}; run __graft_entry__.build()")
    lib = ctypes.CDLL(LIB_PATH)
    st = _i32
    sz = ctypes.POINTER(ctypes.c_size_t)
    P = ctypes.POINTER
    sig = {
        "cc_status_str": (ctypes.c_char_p, [st]),
        "cc_version": (ctypes.c_char_p, []),
        "cc_score_workspace": (st, [P(c_problem), sz]),
        "cc_score": (st, [P(c_problem), P(c_inputs), _c_void_p, _c_void_p, ctypes.c_size_t,
                          _c_void_p]),
        "cc_attention_workspace": (st, [P(c_problem), sz]),
        "cc_attention_cc": (st, [P(c_problem), _c_void_p, P(c_kv), _i32, _c_void_p, _c_void_p,
                                 ctypes.c_size_t, _c_void_p]),
        "cc_lmhead_workspace": (st, [P(c_problem), sz]),
        "cc_lmhead_score": (st, [P(c_problem), _c_void_p, _c_void_p, _c_void_p, _c_void_p,
                                 _c_void_p, _c_void_p, ctypes.c_size_t, _c_void_p]),
        "cc_lmhead_score_noalloc": (st, [P(c_problem), _c_void_p, _c_void_p, _c_void_p,
                                         _c_void_p, _c_void_p, _c_void_p]),
        "cc_linear": (st, [_i32, _c_void_p, _c_void_p, _c_void_p, _i32, _i32, _i32, _c_void_p]),
        "cc_fuse_wo_lmhead_workspace": (st, [_i32, _i32, _i32, sz]),
        "cc_quantize_fp8_workspace": (st, [_i64, sz]),
        "cc_quantize_fp8": (st, [_i32, _c_void_p, _i64, _i32, _i32, _c_void_p, _c_void_p,
                                 _c_void_p, ctypes.c_size_t, _c_void_p]),
        "cc_lmhead_fp8_workspace": (st, [P(c_problem), sz]),
        "cc_lmhead_score_fp8": (st, [P(c_problem), _c_void_p, _c_void_p, _c_void_p, _c_void_p,
                                     _c_void_p, _c_void_p, _c_void_p, ctypes.c_size_t,
                                     _c_void_p]),
        "cc_pack_lmhead_bytes": (st, [_i64, _i32, sz]),
        "cc_pack_lmhead": (st, [_c_void_p, _i64, _i32, _c_void_p, ctypes.c_size_t, _c_void_p]),
        "cc_lmhead_score_packed": (st, [P(c_problem), _c_void_p, _c_void_p, _c_void_p,
                                        _c_void_p, _c_void_p, _c_void_p, ctypes.c_size_t,
                                        _c_void_p]),
        "cc_fuse_wo_lmhead": (st, [_i32, _c_void_p, _c_void_p, _c_void_p, _i32, _i32, _i32,
                                   _c_void_p, ctypes.c_size_t, _c_void_p]),
        "cc_select_workspace": (st, [_i32, sz]),
        "cc_select_keep": (st, [_c_void_p, _i32, P(_i64), P(_i32), P(_i32), _c_void_p, _c_void_p,
                                ctypes.c_size_t, _c_void_p]),
        "cc_compact_workspace": (st, [P(c_problem), _i32, _i32, sz]),
        "cc_compact_kv": (st, [P(c_problem), P(c_kv), _c_void_p, P(_i32), _i32, _c_void_p,
                               _c_void_p, P(c_kv), _c_void_p, ctypes.c_size_t, _c_void_p]),
        "cc_compact_rows_workspace": (st, [P(c_problem), _i32, _i32, sz]),
        "cc_compact_rows": (st, [P(c_problem), _c_void_p, _i32, _c_void_p, P(_i32), _i32,
                                 _c_void_p, _c_void_p, ctypes.c_size_t, _c_void_p]),
    }
    for name, (res, args) in sig.items():
        f = getattr(lib, name)
        f.restype = res
        f.argtypes = args
    return lib


_lib = _load()


class CCError(RuntimeError):
    def __init__(self, status: int, where: str):
        super().__init__(f"{where}: {_lib.cc_status_str(status).decode()}")
        self.status = status


def _check(status: int, where: str) -> None:
    if status != CC_OK:
        raise CCError(status, where)


def cc_status_str(status: int) -> str:
    return _lib.cc_status_str(status).decode()


def cc_version() -> str:
    return _lib.cc_version().decode()


def _ptr(t: Optional[torch.Tensor]):
    return None if t is None else ctypes.c_void_p(t.data_ptr())


def _stream(stream=None):
    if stream is None:
        stream = torch.cuda.current_stream()
    return ctypes.c_void_p(stream.cuda_stream)


def _workspace(nbytes: int, device) -> torch.Tensor:
    return torch.empty(max(int(nbytes), 1), dtype=torch.uint8, device=device)


# ---------------------------------------------------------------- descriptors

@dataclass
class Problem:
    """A cc_problem plus the tensors it points at (kept alive with it)."""
    struct: c_problem
    cu_h: torch.Tensor
    cu_d: torch.Tensor
    device: torch.device

    @property
    def n_tokens(self) -> int:
        return int(self.cu_h[-1])


def problem(*, dtype: str, cu_seqlens: Sequence[int], n_heads_q: int, n_heads_kv: int,
            head_dim: int, hidden: int, vocab: int, device="cuda", mode: str = "last_layer",
            diag: str = "strict", n_layers: int = 0, ffn: int = 0, softmax_scale: float = 0.0,
            rope_theta: float = 0.0, rms_eps: float = 0.0, n_frozen: int = 0,
            lmhead_packed: bool = False) -> Problem:
    cu_h = torch.as_tensor(list(cu_seqlens), dtype=torch.int32).contiguous()
    cu_d = cu_h.to(device)
    s = c_problem()
    s.dtype = {"f32": CC_F32, "bf16": CC_BF16}[dtype]
    s.mode = {"last_layer": CC_MODE_LAST_LAYER, "full": CC_MODE_FULL,
              "last_layer_h": CC_MODE_LAST_LAYER_H,
              "last_layer_fused": CC_MODE_LAST_LAYER_FUSED}[mode]
    s.diag = {"strict": CC_DIAG_STRICT, "inclusive": CC_DIAG_INCLUSIVE}[diag]
    s.n_seqs = len(cu_h) - 1
    s.cu_seqlens_h = ctypes.cast(cu_h.data_ptr(), ctypes.POINTER(_i32))
    s.cu_seqlens_d = cu_d.data_ptr()
    s.n_heads_q, s.n_heads_kv, s.head_dim = n_heads_q, n_heads_kv, head_dim
    s.hidden, s.vocab, s.n_layers, s.ffn = hidden, vocab, n_layers, ffn
    s.softmax_scale, s.rope_theta, s.rms_eps = softmax_scale, rope_theta, rms_eps
    s.n_frozen = n_frozen
    s.lmhead_packed = int(lmhead_packed)
    return Problem(s, cu_h, cu_d, torch.device(device))


def packed(p: Problem, on: bool = True) -> Problem:
    """The same problem with the packed LM head switched on (or off)."""
    s = c_problem.from_buffer_copy(p.struct)
    s.lmhead_packed = int(on)
    return Problem(s, p.cu_h, p.cu_d, p.device)


@dataclass
class KV:
    """A cc_kv view plus the tensors it points at."""
    struct: c_kv
    keep: list = field(default_factory=list)


def kv_contiguous(k: torch.Tensor, v: torch.Tensor, *, n_layers: int, layer_stride: int,
                  head_stride: int, tok_stride: int, seq_stride: int = 0) -> KV:
    s = c_kv()
    s.layout = CC_KV_CONTIGUOUS
    s.n_layers = n_layers
    s.k, s.v = k.data_ptr(), v.data_ptr()
    s.seq_stride, s.layer_stride, s.head_stride, s.tok_stride = (seq_stride, layer_stride,
                                                                 head_stride, tok_stride)
    s.page_stride, s.block_table, s.page_size, s.max_pages = 0, None, 0, 0
    return KV(s, [k, v])


def kv_paged(k: torch.Tensor, v: torch.Tensor, block_table: torch.Tensor, *, n_layers: int,
             layer_stride: int, page_stride: int, head_stride: int, tok_stride: int,
             page_size: int) -> KV:
    bt = block_table.to(torch.int32).contiguous()
    s = c_kv()
    s.layout = CC_KV_PAGED
    s.n_layers = n_layers
    s.k, s.v = k.data_ptr(), v.data_ptr()
    s.seq_stride, s.layer_stride, s.head_stride, s.tok_stride = 0, layer_stride, head_stride, tok_stride
    s.page_stride, s.block_table = page_stride, bt.data_ptr()
    s.page_size, s.max_pages = page_size, bt.shape[1]
    return KV(s, [k, v, bt])


@dataclass
class Inputs:
    struct: c_inputs
    keep: list = field(default_factory=list)


def inputs(*, kv: KV, token_ids: torch.Tensor, w_lm: Optional[torch.Tensor] = None,
           q: Optional[torch.Tensor] = None,
           w_o: Optional[torch.Tensor] = None, pos_ids: Optional[torch.Tensor] = None,
           embed: Optional[torch.Tensor] = None, layers: Optional[list] = None,
           final_norm: Optional[torch.Tensor] = None,
           h_last: Optional[torch.Tensor] = None,
           w_lm_packed: Optional[torch.Tensor] = None) -> Inputs:
    s = c_inputs()
    s.q = q.data_ptr() if q is not None else None
    s.kv = kv.struct
    s.token_ids = token_ids.data_ptr()
    s.pos_ids = pos_ids.data_ptr() if pos_ids is not None else None
    s.w_o = w_o.data_ptr() if w_o is not None else None
    s.w_lm = w_lm.data_ptr() if w_lm is not None else None
    s.embed = embed.data_ptr() if embed is not None else None
    s.h_last = h_last.data_ptr() if h_last is not None else None
    s.w_lm_packed = w_lm_packed.data_ptr() if w_lm_packed is not None else None
    keep = [kv, token_ids, w_lm, q, w_o, pos_ids, embed, final_norm, h_last, w_lm_packed]
    if layers:
        arr = (c_layer_weights * len(layers))()
        for i, L in enumerate(layers):
            for name in ("attn_norm", "wq", "wo", "mlp_norm", "w_gate", "w_up", "w_down"):
                setattr(arr[i], name, L[name].data_ptr())
        s.layers_h = ctypes.cast(arr, ctypes.POINTER(c_layer_weights))
        keep += [arr, layers]
    s.final_norm = final_norm.data_ptr() if final_norm is not None else None
    return Inputs(s, keep)


# ---------------------------------------------------------------- entry points

def _query(fn, *args) -> int:
    n = ctypes.c_size_t(0)
    _check(fn(*args, ctypes.byref(n)), fn.__name__)
    return n.value


def cc_score_workspace(p: Problem) -> int:
    return _query(_lib.cc_score_workspace, ctypes.byref(p.struct))


def cc_score(p: Problem, inp: Inputs, scores: torch.Tensor, workspace: Optional[torch.Tensor] = None,
             stream=None) -> torch.Tensor:
    need = cc_score_workspace(p)
    if workspace is None:
        workspace = _workspace(need, p.device)
    _check(_lib.cc_score(ctypes.byref(p.struct), ctypes.byref(inp.struct), _ptr(scores),
                         _ptr(workspace), workspace.numel(), _stream(stream)), "cc_score")
    return scores


def cc_attention_workspace(p: Problem) -> int:
    return _query(_lib.cc_attention_workspace, ctypes.byref(p.struct))


def cc_attention_cc(p: Problem, q: torch.Tensor, kv: KV, layer: int, o: torch.Tensor,
                    workspace: Optional[torch.Tensor] = None, stream=None) -> torch.Tensor:
    if workspace is None:
        workspace = _workspace(cc_attention_workspace(p), p.device)
    _check(_lib.cc_attention_cc(ctypes.byref(p.struct), _ptr(q), ctypes.byref(kv.struct), layer,
                                _ptr(o), _ptr(workspace), workspace.numel(), _stream(stream)),
           "cc_attention_cc")
    return o


def cc_lmhead_workspace(p: Problem) -> int:
    return _query(_lib.cc_lmhead_workspace, ctypes.byref(p.struct))


def cc_lmhead_score(p: Problem, u: torch.Tensor, w_lm: torch.Tensor, token_ids: torch.Tensor,
                    scores: torch.Tensor, lse: Optional[torch.Tensor] = None,
                    workspace: Optional[torch.Tensor] = None, stream=None) -> torch.Tensor:
    if workspace is None:
        workspace = _workspace(cc_lmhead_workspace(p), p.device)
    _check(_lib.cc_lmhead_score(ctypes.byref(p.struct), _ptr(u), _ptr(w_lm), _ptr(token_ids),
                                _ptr(scores), _ptr(lse), _ptr(workspace), workspace.numel(),
                                _stream(stream)), "cc_lmhead_score")
    return scores


def cc_lmhead_score_noalloc(p: Problem, u: torch.Tensor, w_lm: torch.Tensor,
                            token_ids: torch.Tensor, scores: torch.Tensor,
                            lse: Optional[torch.Tensor] = None, stream=None) -> torch.Tensor:
    """cc_lmhead_score with its scratch in the library's static device array (no workspace)."""
    _check(_lib.cc_lmhead_score_noalloc(ctypes.byref(p.struct), _ptr(u), _ptr(w_lm),
                                        _ptr(token_ids), _ptr(scores), _ptr(lse),
                                        _stream(stream)), "cc_lmhead_score_noalloc")
    return scores


def cc_pack_lmhead_bytes(rows: int, cols: int) -> int:
    return _query(_lib.cc_pack_lmhead_bytes, rows, cols)


def cc_pack_lmhead(x: torch.Tensor, out: Optional[torch.Tensor] = None, stream=None) -> torch.Tensor:
    """The packed LM-head layout of a bf16 [rows][cols] matrix (uint8 buffer)."""
    rows, cols = x.shape
    need = cc_pack_lmhead_bytes(rows, cols)
    if out is None:
        out = torch.empty(need, dtype=torch.uint8, device=x.device)
    _check(_lib.cc_pack_lmhead(_ptr(x), rows, cols, _ptr(out), out.numel() * out.element_size(),
                               _stream(stream)), "cc_pack_lmhead")
    return out


def cc_lmhead_score_packed(p: Problem, u: torch.Tensor, w_packed: torch.Tensor,
                           token_ids: torch.Tensor, scores: torch.Tensor,
                           lse: Optional[torch.Tensor] = None, workspace=None, stream=None):
    if workspace is None:
        workspace = _workspace(cc_lmhead_workspace(p), p.device)
    _check(_lib.cc_lmhead_score_packed(ctypes.byref(p.struct), _ptr(u), _ptr(w_packed),
                                       _ptr(token_ids), _ptr(scores), _ptr(lse), _ptr(workspace),
                                       workspace.numel(), _stream(stream)),
           "cc_lmhead_score_packed")
    return scores


def cc_fuse_wo_lmhead_workspace(dtype: str, hidden: int, qdim: int) -> int:
    n = ctypes.c_size_t()
    _check(_lib.cc_fuse_wo_lmhead_workspace({"f32": CC_F32, "bf16": CC_BF16}[dtype], hidden, qdim,
                                            ctypes.byref(n)), "cc_fuse_wo_lmhead_workspace")
    return n.value


def cc_fuse_wo_lmhead(dtype: str, w_lm: torch.Tensor, w_o: torch.Tensor,
                      out: Optional[torch.Tensor] = None, workspace=None, stream=None):
    """The LAST_LAYER_FUSED weight W_lm W_o [V][Hq*d] from w_lm [V][D] and w_o [D][Hq*d]."""
    V, D = w_lm.shape
    D2, Q = w_o.shape
    if D2 != D:
        raise ValueError(f"w_o has {D2} rows, w_lm has {D} columns")
    if out is None:
        out = torch.empty((V, Q), dtype=w_lm.dtype, device=w_lm.device)
    if workspace is None:
        workspace = _workspace(cc_fuse_wo_lmhead_workspace(dtype, D, Q), w_lm.device)
    _check(_lib.cc_fuse_wo_lmhead({"f32": CC_F32, "bf16": CC_BF16}[dtype], _ptr(w_lm), _ptr(w_o),
                                  _ptr(out), V, D, Q, _ptr(workspace), workspace.numel(),
                                  _stream(stream)), "cc_fuse_wo_lmhead")
    return out


def cc_quantize_fp8_workspace(rows: int) -> int:
    n = ctypes.c_size_t()
    _check(_lib.cc_quantize_fp8_workspace(rows, ctypes.byref(n)), "cc_quantize_fp8_workspace")
    return n.value


def cc_quantize_fp8(dtype: str, x: torch.Tensor, per_row: bool, codes=None, scale=None,
                    workspace=None, stream=None):
    """E4M3 codes (uint8, x's shape) and fp32 scales ([rows], or [1] for the matrix)."""
    rows, cols = x.shape
    if codes is None:
        codes = torch.empty((rows, cols), dtype=torch.uint8, device=x.device)
    if scale is None:
        scale = torch.empty(rows if per_row else 1, dtype=torch.float32, device=x.device)
    if workspace is None:
        workspace = _workspace(cc_quantize_fp8_workspace(rows), x.device)
    _check(_lib.cc_quantize_fp8({"f32": CC_F32, "bf16": CC_BF16}[dtype], _ptr(x), rows, cols,
                                int(per_row), _ptr(codes), _ptr(scale), _ptr(workspace),
                                workspace.numel(), _stream(stream)), "cc_quantize_fp8")
    return codes, scale


def cc_lmhead_fp8_workspace(p: Problem) -> int:
    return _query(_lib.cc_lmhead_fp8_workspace, ctypes.byref(p.struct))


def cc_lmhead_score_fp8(p: Problem, u: torch.Tensor, w_codes: torch.Tensor, w_scale: torch.Tensor,
                        token_ids: torch.Tensor, scores: torch.Tensor,
                        lse: Optional[torch.Tensor] = None, workspace=None, stream=None):
    if workspace is None:
        workspace = _workspace(cc_lmhead_fp8_workspace(p), p.device)
    _check(_lib.cc_lmhead_score_fp8(ctypes.byref(p.struct), _ptr(u), _ptr(w_codes), _ptr(w_scale),
                                    _ptr(token_ids), _ptr(scores), _ptr(lse), _ptr(workspace),
                                    workspace.numel(), _stream(stream)), "cc_lmhead_score_fp8")
    return scores


def cc_linear(dtype: str, x: torch.Tensor, w: torch.Tensor, y: torch.Tensor, stream=None):
    M, K = x.shape
    N = w.shape[0]
    _check(_lib.cc_linear({"f32": CC_F32, "bf16": CC_BF16}[dtype], _ptr(x), _ptr(w), _ptr(y), M, N,
                          K, _stream(stream)), "cc_linear")
    return y


def cc_select_workspace(n_segs: int) -> int:
    return _query(_lib.cc_select_workspace, n_segs)


def _host_array(x, dtype):
    """A C-contiguous numpy array of the given integer type (no copy if it is one)."""
    return np.ascontiguousarray(np.asarray(x), dtype=dtype)


def cc_select_keep(scores: torch.Tensor, seg_start: Sequence[int], seg_len: Sequence[int],
                   k: Sequence[int], keep_idx: torch.Tensor,
                   workspace: Optional[torch.Tensor] = None, stream=None) -> torch.Tensor:
    """seg_start, seg_len, k: host sequences or numpy arrays (int64, int32, int32 arrays
    are passed without a copy)."""
    st = _host_array(seg_start, np.int64)
    ln = _host_array(seg_len, np.int32)
    kk = _host_array(k, np.int32)
    n = len(ln)
    if workspace is None:
        workspace = _workspace(cc_select_workspace(n), scores.device)
    _check(_lib.cc_select_keep(_ptr(scores), n, st.ctypes.data_as(ctypes.POINTER(_i64)),
                               ln.ctypes.data_as(ctypes.POINTER(_i32)),
                               kk.ctypes.data_as(ctypes.POINTER(_i32)), _ptr(keep_idx),
                               _ptr(workspace), workspace.numel(), _stream(stream)),
           "cc_select_keep")
    return keep_idx


def cc_compact_workspace(p: Problem, cache_layers: int, per_head: int) -> int:
    return _query(_lib.cc_compact_workspace, ctypes.byref(p.struct), cache_layers, per_head)


def cc_compact_kv(p: Problem, kv: KV, keep_idx: torch.Tensor, k: Sequence[int], per_head: int,
                  token_ids: Optional[torch.Tensor] = None, pos_ids: Optional[torch.Tensor] = None,
                  out: Optional[KV] = None, workspace: Optional[torch.Tensor] = None,
                  stream=None) -> None:
    kk = (_i32 * len(k))(*[int(x) for x in k])
    if workspace is None:
        workspace = _workspace(cc_compact_workspace(p, kv.struct.n_layers, per_head), p.device)
    _check(_lib.cc_compact_kv(ctypes.byref(p.struct), ctypes.byref(kv.struct), _ptr(keep_idx), kk,
                              per_head, _ptr(token_ids), _ptr(pos_ids),
                              ctypes.byref(out.struct) if out is not None else None,
                              _ptr(workspace), workspace.numel(), _stream(stream)),
           "cc_compact_kv")


def cc_compact_rows_workspace(p: Problem, row_bytes: int, per_head: int) -> int:
    return _query(_lib.cc_compact_rows_workspace, ctypes.byref(p.struct), row_bytes, per_head)


def cc_compact_rows(p: Problem, rows: torch.Tensor, keep_idx: torch.Tensor, k: Sequence[int],
                    per_head: int, out: Optional[torch.Tensor] = None,
                    workspace: Optional[torch.Tensor] = None, stream=None) -> None:
    """rows: [N][...] token-major; every entry row is compacted with its sequence's keep
    list (in place unless `out` is given)."""
    row_bytes = rows[0].numel() * rows.element_size() if rows.shape[0] else 16
    kk = (_i32 * len(k))(*[int(x) for x in k])
    if workspace is None:
        workspace = _workspace(cc_compact_rows_workspace(p, row_bytes, per_head), p.device)
    _check(_lib.cc_compact_rows(ctypes.byref(p.struct), _ptr(rows), row_bytes, _ptr(keep_idx), kk,
                                per_head, _ptr(out), _ptr(workspace), workspace.numel(),
                                _stream(stream)), "cc_compact_rows")
