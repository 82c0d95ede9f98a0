"""GPU parity of the packed LM head (cc_pack_lmhead, cc_lmhead_score_packed, and
cc_score with lmhead_packed = 1).

The packing is a pure layout change, so it is compared byte for byte with the layout as
the header defines it (rebuilt here with numpy index arithmetic).  The packed LM head
computes the same Eq. (5) scores as the row-major one, so it takes the same bf16 bar
against the oracle, on shapes with a ragged vocabulary edge, ragged entry counts and
every residue of the k-step count modulo the four pipeline stages."""
import numpy as np
import pytest
import torch

from oracle import cc_oracle as O
from synth import configs as C
from synth import gen
from tests.gpu_util import assert_scores_close, dev

pytestmark = pytest.mark.gpu


def _packed_reference(x: np.ndarray) -> np.ndarray:
    """uint16 [R][K] -> the packed layout as uint16, from its definition: per 256-row tile
    t and 32-column step s a block of 256 rows x 32; row r holds its 8-element chunk c at
    chunk position c ^ ((r >> 1) & 3); rows past R are zero."""
    R, K = x.shape
    T, S = (R + 255) // 256, K // 32
    xp = np.zeros((T * 256, K), dtype=np.uint16)
    xp[:R] = x
    blocks = xp.reshape(T, 256, S, 4, 8)            # [t][r][s][c][e]
    out = np.zeros((T, S, 256, 4, 8), dtype=np.uint16)
    for r in range(256):
        for c in range(4):
            out[:, :, r, c ^ ((r >> 1) & 3), :] = blocks[:, r, :, c, :]
    return out.reshape(-1)


@pytest.mark.parametrize("R,K", [(300, 64), (256, 96), (1, 32), (513, 128)])
def test_pack_layout_matches_definition(R, K):
    from paper_2607_27600_amd import cc
    print(f"[pack] R={R} K={K}", flush=True)
    x = np.random.default_rng(R + K).integers(0, 65535, (R, K), dtype=np.uint16)
    got = cc.cc_pack_lmhead(dev(x))
    torch.cuda.synchronize()
    assert got.numel() == cc.cc_pack_lmhead_bytes(R, K) == ((R + 255) // 256) * 256 * K * 2
    np.testing.assert_array_equal(got.cpu().numpy().view(np.uint16), _packed_reference(x))


def _lmhead_case(lens, D, V, n_frozen, seed):
    from paper_2607_27600_amd import cc
    print(f"[packed lmhead] lens={lens[:4]} D={D} V={V}", flush=True)
    r = np.random.default_rng(seed)
    cu = np.concatenate([[0], np.cumsum(lens)]).astype(np.int32)
    N = int(cu[-1])
    u = gen.f32_to_bf16_bits(r.standard_normal((N, D)).astype(np.float32))
    w = gen.f32_to_bf16_bits((0.05 * r.standard_normal((V, D))).astype(np.float32))
    ids = r.integers(0, V, N).astype(np.int32)
    wd = dev(w)
    wp = cc.cc_pack_lmhead(wd)
    p = cc.problem(dtype="bf16", cu_seqlens=cu.tolist(), n_heads_q=1, n_heads_kv=1,
                   head_dim=128, hidden=D, vocab=V, n_frozen=n_frozen, lmhead_packed=True)
    scores = torch.full((N,), float("nan"), dtype=torch.float32, device="cuda")
    lse = torch.empty(N, dtype=torch.float32, device="cuda")
    cc.cc_lmhead_score_packed(p, dev(u), wp, dev(ids), scores, lse)
    # the row-major kernel on the same inputs, for the summation-order comparison
    p0 = cc.problem(dtype="bf16", cu_seqlens=cu.tolist(), n_heads_q=1, n_heads_kv=1,
                    head_dim=128, hidden=D, vocab=V, n_frozen=n_frozen)
    s_rm = torch.empty(N, dtype=torch.float32, device="cuda")
    cc.cc_lmhead_score(p0, dev(u), wd, dev(ids), s_rm)
    torch.cuda.synchronize()
    s_ref, lse_ref, _ = O.surprise(O.f64(u), w, ids)
    s_ref[O.edge_rows(cu, n_frozen)] = np.inf
    got = scores.cpu().numpy()
    print("packed vs oracle", assert_scores_close(got, s_ref, "bf16", "packed lmhead"))
    fin = np.isfinite(s_ref)
    np.testing.assert_allclose(lse.cpu().numpy()[fin], lse_ref[fin], rtol=0, atol=2e-2)
    rm = s_rm.cpu().numpy()
    np.testing.assert_array_equal(np.isinf(got), np.isinf(rm))
    d = np.abs(got[fin] - rm[fin])
    print(f"packed vs row-major kernel: max {d.max():.3e}", flush=True)
    # both accumulate exact bf16 products in fp32, in different orders
    assert d.max() <= 1e-4 + 1e-5 * np.abs(rm[fin]).max()


@pytest.mark.parametrize("lens,D,V", [
    ([5, 1, 294], 256, 1000),      # 8 k-steps, ragged vocabulary edge, ragged entries
    ([300], 192, 257),             # 6 k-steps: two-step tail; one row past a vocab tile
    ([1, 40, 600], 320, 777),      # 10 k-steps: two full rounds and a tail of two
    ([77], 64, 300),               # 2 k-steps: fewer steps than stages
])
def test_packed_lmhead_matches_oracle(lens, D, V):
    _lmhead_case(lens, D, V, n_frozen=2, seed=D + V)


def test_packed_score_two_step_and_fused():
    """cc_score with lmhead_packed: the two-step mode (packed W_lm, U packed inside) and the
    W_o-folded mode (packed W_lm W_o over the attention output)."""
    from paper_2607_27600_amd import cc
    from paper_2607_27600_amd.workload import Workload
    cfg = C.shrink(C.C2, seq_lens=(300, 45), hidden=256, vocab=1000, cache_layers=1)
    w = Workload(cfg, cache_layers=1, keep_host=True)
    h = w.host
    ref, spread = O.last_layer_scores(h["q"], h["k"], h["v"], h["w_o"], h["w_lm"], h["ids"],
                                      cfg.cu_seqlens, spread=True)
    for mode in ("last_layer", "last_layer_fused"):
        print(f"[packed score] {mode}", flush=True)
        p = cc.problem(dtype="bf16", cu_seqlens=cfg.cu_seqlens.tolist(), n_heads_q=cfg.n_heads_q,
                       n_heads_kv=cfg.n_heads_kv, head_dim=cfg.head_dim, hidden=cfg.hidden,
                       vocab=cfg.vocab, mode=mode, lmhead_packed=True)
        wl = cc.cc_fuse_wo_lmhead("bf16", w.w_lm, w.w_o) if mode == "last_layer_fused" else w.w_lm
        wp = cc.cc_pack_lmhead(wl)
        inp = cc.inputs(kv=w.kv, token_ids=w.ids, w_lm=wl, q=w.q, w_o=w.w_o, w_lm_packed=wp)
        scores = torch.full((cfg.n_tokens,), float("nan"), dtype=torch.float32, device="cuda")
        cc.cc_score(p, inp, scores)
        torch.cuda.synchronize()
        print(mode, assert_scores_close(scores.cpu().numpy(), ref, "bf16", f"packed {mode}",
                                        spread))
        # without the packed weight the call is refused before anything runs
        inp0 = cc.inputs(kv=w.kv, token_ids=w.ids, w_lm=wl, q=w.q, w_o=w.w_o)
        with pytest.raises(cc.CCError):
            cc.cc_score(p, inp0, scores)


def test_packed_zero_head_gives_ln_vocab():
    from paper_2607_27600_amd import cc
    N, D, V = 100, 128, 128256
    u = gen.f32_to_bf16_bits(np.random.default_rng(3).standard_normal((N, D)).astype(np.float32))
    w = torch.zeros((V, D), dtype=torch.bfloat16, device="cuda")
    ids = torch.arange(N, dtype=torch.int32, device="cuda") * 997
    p = cc.problem(dtype="bf16", cu_seqlens=[0, N], n_heads_q=1, n_heads_kv=1, head_dim=128,
                   hidden=D, vocab=V, lmhead_packed=True)
    scores = torch.empty(N, dtype=torch.float32, device="cuda")
    cc.cc_lmhead_score_packed(p, dev(u), cc.cc_pack_lmhead(w), ids, scores)
    torch.cuda.synchronize()
    s = scores.cpu().numpy().astype(np.float64)
    assert s[-1] == np.inf
    np.testing.assert_allclose(s[:-1], np.log(V), rtol=0, atol=2e-5)


@pytest.mark.slow
def test_packed_lmhead_c2_shape_sampled():
    """Llama-3-8B LM head (V 128256, D 4096) over 4096 entries, 48 sampled rows."""
    from paper_2607_27600_amd import cc
    cfg = C.C2
    print("[packed lmhead] C2 shape", flush=True)
    N, D, V = cfg.n_tokens, cfg.hidden, cfg.vocab
    r = np.random.default_rng(23)
    u = gen.f32_to_bf16_bits(r.standard_normal((N, D)).astype(np.float32))
    w = gen.normal_bf16(0, 3, (V, D), 0.02)
    ids = r.integers(0, V, N).astype(np.int32)
    wd = dev(w)
    wp = cc.cc_pack_lmhead(wd)
    p = cc.problem(dtype="bf16", cu_seqlens=[0, N], n_heads_q=1, n_heads_kv=1, head_dim=128,
                   hidden=D, vocab=V, lmhead_packed=True)
    scores = torch.empty(N, dtype=torch.float32, device="cuda")
    cc.cc_lmhead_score_packed(p, dev(u), wp, dev(ids), scores)
    torch.cuda.synchronize()
    rows = C.sample_rows(cfg, count=48)
    s_ref, _, _ = O.surprise(O.f64(u[rows]), w, ids[rows])
    s_ref[rows == N - 1] = np.inf
    print("C2 packed", assert_scores_close(scores.cpu().numpy()[rows], s_ref, "bf16", "C2 packed"))
