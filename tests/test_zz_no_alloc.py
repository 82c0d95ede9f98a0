"""The allocation-free LM head (cc_lmhead_score_noalloc) against the workspace entry point
(cc_lmhead_score) and the oracle, called twice in a row, the second time with fewer
entries and another vocabulary, both in bf16 and fp32: the static scratch keeps the first
call's contents, which the second must not see.  A problem larger than the scratch is
refused on the host before anything runs."""
import ctypes

import numpy as np
import pytest
import torch

from oracle import cc_oracle as O
from synth import gen
from tests.gpu_util import assert_scores_close, dev

pytestmark = pytest.mark.gpu


def _case(dtype, lens, D, V, seed):
    from paper_2607_27600_amd import cc
    print(f"[noalloc] {dtype} lens={lens} D={D} V={V}", flush=True)
    r = np.random.default_rng(seed)
    cu = np.concatenate([[0], np.cumsum(lens)]).astype(np.int32)
    N = int(cu[-1])
    u = r.standard_normal((N, D)).astype(np.float32)
    w = (0.05 * r.standard_normal((V, D))).astype(np.float32)
    ids = r.integers(0, V, N).astype(np.int32)
    if dtype == "bf16":
        u, w = gen.f32_to_bf16_bits(u), gen.f32_to_bf16_bits(w)
    p = cc.problem(dtype=dtype, cu_seqlens=cu.tolist(), n_heads_q=1, n_heads_kv=1,
                   head_dim=128, hidden=D, vocab=V, n_frozen=1)
    ud, wd, idd = dev(u), dev(w), dev(ids)
    s_na = torch.full((N,), float("nan"), dtype=torch.float32, device="cuda")
    l_na = torch.full((N,), float("nan"), dtype=torch.float32, device="cuda")
    cc.cc_lmhead_score_noalloc(p, ud, wd, idd, s_na, l_na)
    s_ws = torch.full((N,), float("nan"), dtype=torch.float32, device="cuda")
    l_ws = torch.full((N,), float("nan"), dtype=torch.float32, device="cuda")
    cc.cc_lmhead_score(p, ud, wd, idd, s_ws, l_ws)
    torch.cuda.synchronize()
    got, ref_ws = s_na.cpu().numpy(), s_ws.cpu().numpy()
    # the same kernels in the same order: identical results
    np.testing.assert_array_equal(got, ref_ws)
    np.testing.assert_array_equal(l_na.cpu().numpy(), l_ws.cpu().numpy())
    s_ref, _, _ = O.surprise(O.f64(u), w, ids)
    s_ref[O.edge_rows(cu, 1)] = np.inf
    print(assert_scores_close(got, s_ref, dtype, f"noalloc {dtype}"))


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
def test_noalloc_lmhead_two_calls_matches_workspace_entry(dtype):
    _case(dtype, [700, 1, 1299], 256, 3000, seed=1)     # 12 vocabulary tiles x 2000 entries
    _case(dtype, [5, 300], 128, 700, seed=2)             # smaller: 3 tiles x 305 entries


def test_noalloc_lmhead_refuses_more_than_the_scratch():
    from paper_2607_27600_amd import cc
    # 4096 entries x 1254 tiles of a 320,000-word vocabulary: 41 MB of partials
    N, D, V = 4096, 128, 320000
    p = cc.problem(dtype="bf16", cu_seqlens=[0, N], n_heads_q=1, n_heads_kv=1, head_dim=128,
                   hidden=D, vocab=V)
    assert cc.cc_lmhead_workspace(p) > cc.CC_NOALLOC_SCRATCH_BYTES
    scores = torch.full((N,), float("nan"), dtype=torch.float32, device="cuda")
    dummy = torch.zeros(16, dtype=torch.bfloat16, device="cuda")
    ids = torch.zeros(N, dtype=torch.int32, device="cuda")
    st = cc._lib.cc_lmhead_score_noalloc(ctypes.byref(p.struct), cc._ptr(dummy), cc._ptr(dummy),
                                         cc._ptr(ids), cc._ptr(scores), None, None)
    assert st == cc.CC_ERR_SCRATCH
    torch.cuda.synchronize()
    assert torch.isnan(scores).all()          # nothing was written
    pk = cc.packed(p)
    assert cc._lib.cc_lmhead_score_noalloc(ctypes.byref(pk.struct), cc._ptr(dummy),
                                           cc._ptr(dummy), cc._ptr(ids), cc._ptr(scores), None,
                                           None) == cc.CC_ERR_ARG
