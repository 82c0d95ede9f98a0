"""The cache-managed inference cycle (paper_2607_27600_amd.refresh) on a synthetic stream.

At every refresh: the scores equal the oracle's on the cache as it stands (all rows,
bf16 tolerance), the keep list equals the oracle's selection on the GPU's own scores,
and afterwards keys, values, ids, positions and per-entry rows are the byte-exact
gather.  Across the stream every cached entry keeps the position and id it was
appended with.  Exact fast variant (from H), given-query variant and its form with W_o
folded into the LM head (scored against the oracle's two-step chain); chunked and
prefill-end modes."""
import numpy as np
import pytest
import torch

from oracle import cc_oracle as O
from synth import gen
from tests.gpu_util import assert_scores_close, bf16_host, dev

pytestmark = pytest.mark.gpu

L, HQ, HKV, D_HEAD, D, F, V = 2, 4, 2, 128, 256, 512, 1000
THETA, EPS = 5e5, 1e-5


def _stream(T, width, seed=3):
    r = np.random.default_rng(seed)
    return dict(k=gen.normal_bf16(seed, 100, (L, HKV, T, D_HEAD)),
                v=gen.normal_bf16(seed, 101, (L, HKV, T, D_HEAD)),
                rows=gen.normal_bf16(seed, 102, (T, width)),
                ids=r.integers(0, V, T).astype(np.int32))


def _model(mode, packed=False):
    from paper_2607_27600_amd.refresh import Model
    w = lambda tid, shape: gen.normal_bf16(7, tid, shape, 0.05)
    host = dict(w_lm=w(1, (V, D)), w_o=w(2, (D, HQ * D_HEAD)),
                layer=dict(attn_norm=gen.f32_to_bf16_bits(np.ones(D, np.float32)),
                           wq=w(3, (HQ * D_HEAD, D)), wo=w(4, (D, HQ * D_HEAD)),
                           mlp_norm=gen.f32_to_bf16_bits(np.ones(D, np.float32)),
                           w_gate=w(5, (F, D)), w_up=w(6, (F, D)), w_down=w(7, (D, F))),
                final_norm=gen.f32_to_bf16_bits(np.ones(D, np.float32)))
    w_lm = dev(host["w_lm"])
    if mode == "last_layer_fused":      # the GPU model holds W_lm W_o; the oracle the two
        from paper_2607_27600_amd import cc
        w_lm = cc.cc_fuse_wo_lmhead("bf16", w_lm, dev(host["w_o"]))
    m = Model(mode=mode, n_layers=L, n_heads_q=HQ, n_heads_kv=HKV, head_dim=D_HEAD, hidden=D,
              vocab=V, w_lm=w_lm, w_o=dev(host["w_o"]),
              layer={k: dev(v) for k, v in host["layer"].items()},
              final_norm=dev(host["final_norm"]), ffn=F, rope_theta=THETA, rms_eps=EPS)
    if packed:
        from paper_2607_27600_amd import cc
        m.w_lm_packed = cc.cc_pack_lmhead(w_lm)
    return m, host


def _oracle_scores(mode, host, st):
    n = st["n"]
    K, Vv = st["k"][-1][:, :n], st["v"][-1][:, :n]
    if mode == "last_layer_h":
        return O.last_layer_h_scores(st["rows"][:n], st["ids"][:n], K, Vv, host["layer"],
                                     host["final_norm"], host["w_lm"], [0, n], HQ, D_HEAD, THETA,
                                     EPS, pos_ids=st["pos"][:n])
    q = st["rows"][:n].reshape(n, HQ, D_HEAD)
    return O.last_layer_scores(q, K, Vv, host["w_o"], host["w_lm"], st["ids"][:n], [0, n])


def _state(loop):
    return dict(n=loop.n, k=bf16_host(loop.k), v=bf16_host(loop.v), rows=bf16_host(loop.rows),
                ids=loop.ids.cpu().numpy().copy(), pos=loop.pos.cpu().numpy().copy())


@pytest.mark.parametrize("mode,chunked,packed", [("last_layer_h", True, False),
                                                 ("last_layer", True, False),
                                                 ("last_layer_h", False, False),
                                                 ("last_layer_fused", True, False),
                                                 ("last_layer_h", True, True),
                                                 ("last_layer_fused", True, True)])
def test_refresh_loop(mode, chunked, packed):
    from paper_2607_27600_amd.refresh import RefreshLoop, run_stream
    print(f"[refresh loop] mode={mode} chunked={chunked} packed={packed}", flush=True)
    J, h, T_prompt, T_total = 40, 16, 100, 170
    m, host = _model(mode, packed)
    cap = None if chunked else T_total
    loop = RefreshLoop(m, J, h, capacity=cap)
    S = _stream(T_total, m.row_width)
    S_d = {k: dev(v) for k, v in S.items()}
    pos_d = torch.arange(T_total, dtype=torch.int32, device="cuda")

    def entry(t0, t1):
        return (S_d["k"][:, :, t0:t1], S_d["v"][:, :, t0:t1], S_d["ids"][t0:t1], pos_d[t0:t1],
                S_d["rows"][t0:t1])

    checks = []

    def hook(scores, keep):
        torch.cuda.synchronize()
        st = _state(loop)
        s = scores.cpu().numpy()
        kk = keep.cpu().numpy()
        assert_scores_close(s, _oracle_scores(mode, host, st), "bf16", f"refresh {len(checks)}")
        np.testing.assert_array_equal(kk, O.select_keep(s, J))
        checks.append((st, kk))

    refresh = loop.refresh

    def checked_refresh(hk=None):
        before = loop.refreshes
        kept = refresh(hook)
        if loop.refreshes > before:           # a cycle ran: check the compacted cache
            torch.cuda.synchronize()
            st, kk = checks[-1]
            after = _state(loop)
            for name in ("k", "v"):
                np.testing.assert_array_equal(after[name][:, :, :J], st[name][:, :, kk])
            for name in ("rows", "ids", "pos"):
                np.testing.assert_array_equal(after[name][:J], st[name][kk])
        return kept

    loop.refresh = checked_refresh
    run_stream(loop, entry, T_prompt, T_total, chunked=chunked)
    torch.cuda.synchronize()
    assert len(checks) == loop.refreshes >= 1
    # every cached entry still carries the position and id it was appended with
    n = loop.n
    pos = loop.pos[:n].cpu().numpy()
    assert np.all(np.diff(pos) > 0) and pos[-1] == T_total - 1
    np.testing.assert_array_equal(loop.ids[:n].cpu().numpy(), S["ids"][pos])
    np.testing.assert_array_equal(bf16_host(loop.rows)[:n], S["rows"][pos])
    np.testing.assert_array_equal(bf16_host(loop.k)[:, :, :n], S["k"][:, :, pos])
