"""GPU keep selection and KV compaction: bit-exact against the oracle.

Selection is compared on identical fp32 scores (ties, -0/+0, +/-inf, NaN, ragged
segments, k = 0 and k = len); compaction is a bit copy compared byte for byte, in place
and out of place, contiguous and paged, one list per sequence or per KV head."""
import numpy as np
import pytest
import torch

from oracle import cc_oracle as O
from synth import configs as C
from tests.gpu_util import bf16_host

pytestmark = pytest.mark.gpu


def _gpu_select(scores: np.ndarray, starts, lens, ks):
    from paper_2607_27600_amd import cc
    s = torch.from_numpy(scores.astype(np.float32)).cuda()
    keep = torch.full((max(1, int(sum(ks))),), -7, dtype=torch.int32, device="cuda")
    cc.cc_select_keep(s, starts, lens, ks, keep)
    torch.cuda.synchronize()
    return keep.cpu().numpy()


@pytest.mark.parametrize("seed", range(4))
def test_select_matches_oracle_with_ties(seed):
    print(f"[select] seed={seed}", flush=True)
    r = np.random.default_rng(seed)
    lens = [1, 2, 7, 1000, 1024, 1025, 5000, 32768]
    total = sum(lens)
    pool = np.array([-0.0, 0.0, 1.5, 1.5, 2.0, -3.0, np.inf, -np.inf, np.nan, 11.75],
                    dtype=np.float32)
    s = np.where(r.random(total) < 0.5, pool[r.integers(0, len(pool), total)],
                 np.round(r.standard_normal(total), 2).astype(np.float32)).astype(np.float32)
    starts = np.concatenate([[0], np.cumsum(lens)[:-1]])
    for kfrac in (0.0, 0.25, 0.5, 1.0):
        ks = [int(kfrac * n) for n in lens]
        got = _gpu_select(s, starts, lens, ks)
        off = 0
        for st, n, k in zip(starts, lens, ks):
            ref = O.select_keep(s[st:st + n], k)
            np.testing.assert_array_equal(got[off:off + k], ref, err_msg=f"len={n} k={k}")
            off += k


@pytest.mark.parametrize("lens", [[32769, 40000, 70001], [5, 32768, 33000]])
def test_select_long_segments(lens):
    """Segments longer than the register-resident path holds go through the kernel that
    re-reads the scores at every pass (any segment past 32768 in the launch selects it)."""
    print(f"[select] long lens={lens}", flush=True)
    r = np.random.default_rng(len(lens) + lens[0])
    total = sum(lens)
    pool = np.array([-0.0, 0.0, 1.5, 2.0, np.inf, -np.inf, np.nan], dtype=np.float32)
    s = np.where(r.random(total) < 0.3, pool[r.integers(0, len(pool), total)],
                 r.standard_normal(total).astype(np.float32)).astype(np.float32)
    starts = np.concatenate([[0], np.cumsum(lens)[:-1]])
    for kfrac in (0.2, 0.5):
        ks = [max(1, int(kfrac * n)) for n in lens]
        got = _gpu_select(s, starts, lens, ks)
        off = 0
        for st, n, k in zip(starts, lens, ks):
            np.testing.assert_array_equal(got[off:off + k], O.select_keep(s[st:st + n], k),
                                          err_msg=f"len={n} k={k}")
            off += k


def test_select_score_ranges():
    """Distributions that stress the radix passes on min-relative keys: surprisal-like
    (exponential), a narrow band (few bits of range), huge magnitudes of both signs, and
    scores one ulp apart; segment starts not 16-byte aligned."""
    r = np.random.default_rng(21)
    n = 9001
    base = np.float32(11.76)
    segs = [
        r.exponential(3.0, n).astype(np.float32),
        (base + r.standard_normal(n) * 1e-3).astype(np.float32),
        (r.uniform(-1, 1, n) * 3e38).astype(np.float32),
        np.nextafter(np.full(n, base), np.float32(np.inf)) * (r.random(n) < 0.5) + base * (r.random(n) >= 0.5),
        r.standard_normal(n).astype(np.float32),
    ]
    segs[3] = segs[3].astype(np.float32)
    segs[4][::7] = -np.inf
    segs[4][::11] = np.inf
    s = np.concatenate([np.zeros(3, np.float32)] + segs).astype(np.float32)
    starts = [3 + i * n for i in range(len(segs))]
    for k in (1, 17, n // 4, n - 1):
        got = _gpu_select(s, starts, [n] * len(segs), [k] * len(segs))
        for i, st in enumerate(starts):
            np.testing.assert_array_equal(got[i * k:(i + 1) * k], O.select_keep(s[st:st + n], k),
                                          err_msg=f"segment {i} k={k}")


def test_select_register_path_branches():
    """Segments of 8193..32768 scores (the register-resident kernel) built to take each of
    its branches: +inf keys that fill the budget or only part of it, a threshold bucket
    too full for the candidate list (a narrow band inside a wide range), a range of fewer
    than 256 key units, every finite score equal, and the four-load read (start not
    16-byte aligned, length not divisible by four)."""
    r = np.random.default_rng(77)
    n = 32768
    base = np.float32(11.0)
    half_inf = r.exponential(3.0, n).astype(np.float32)
    half_inf[r.permutation(n)[: n // 2]] = np.inf
    some_inf = r.exponential(3.0, n).astype(np.float32)
    some_inf[r.integers(0, n, 100)] = np.inf
    some_inf[-1] = np.inf
    band = (base + r.uniform(0.0, 1e-4, n)).astype(np.float32)
    band[r.permutation(n)[:2768]] = r.uniform(0.0, 100.0, 2768).astype(np.float32)
    ulps = (np.float32(1.0) + r.integers(0, 200, n).astype(np.float32) * np.float32(2.0 ** -23))
    ulps = ulps.astype(np.float32)
    flat = np.full(n, np.log(128256.0), dtype=np.float32)
    flat[::97] = np.inf
    segs = [half_inf, some_inf, band, ulps, flat]
    s = np.concatenate(segs).astype(np.float32)
    starts = [i * n for i in range(len(segs))]
    for k in (1, 100, 8192, n // 2 + 5, n - 1):
        print(f"[select] register branches k={k}", flush=True)
        got = _gpu_select(s, starts, [n] * len(segs), [k] * len(segs))
        for i, st in enumerate(starts):
            np.testing.assert_array_equal(got[i * k:(i + 1) * k], O.select_keep(s[st:st + n], k),
                                          err_msg=f"segment {i} k={k}")
    # unaligned start, odd length: the four-load read
    m = 30001
    t = np.concatenate([np.zeros(3, np.float32), some_inf[:m], band[:m]]).astype(np.float32)
    for k in (7, 7500, m - 2):
        print(f"[select] unaligned k={k}", flush=True)
        got = _gpu_select(t, [3, 3 + m], [m, m], [k, k])
        for i, st in enumerate([3, 3 + m]):
            np.testing.assert_array_equal(got[i * k:(i + 1) * k], O.select_keep(t[st:st + m], k),
                                          err_msg=f"unaligned segment {i} k={k}")


@pytest.mark.parametrize("long_seg", [False, True])
def test_select_many_segments(long_seg):
    """More segments than travel in the kernel arguments (16): the descriptors go through
    the workspace table; both kernels (longest segment at most 8192, or up to 32768)."""
    r = np.random.default_rng(31 + long_seg)
    lens = [int(x) for x in r.integers(1, 3000, 40)]
    if long_seg:
        lens[17] = 20000
    s = r.exponential(3.0, sum(lens)).astype(np.float32)
    starts = np.concatenate([[0], np.cumsum(lens)[:-1]])
    ks = [int(r.integers(0, n + 1)) for n in lens]
    print(f"[select] {len(lens)} segments, longest {max(lens)}", flush=True)
    got = _gpu_select(s, starts, lens, ks)
    off = 0
    for st, n, k in zip(starts, lens, ks):
        np.testing.assert_array_equal(got[off:off + k], O.select_keep(s[st:st + n], k),
                                      err_msg=f"len={n} k={k}")
        off += k


@pytest.mark.parametrize("stride", [0, 9000, 9004])
def test_select_regular_segments_without_a_table(stride):
    """More than 16 segments of equal length and budget at a fixed stride (0: one per KV
    head over the same scores; the length: a batch of equal sequences; a gap between
    them): the kernels compute every descriptor and nothing is uploaded."""
    r = np.random.default_rng(stride + 5)
    n, n_segs, k = 9000, 40, 2250
    s = r.exponential(3.0, (n_segs - 1) * stride + n + 8).astype(np.float32)
    s[r.integers(0, len(s), 50)] = np.inf
    starts = [i * stride for i in range(n_segs)]
    print(f"[select] regular stride={stride}", flush=True)
    got = _gpu_select(s, starts, [n] * n_segs, [k] * n_segs)
    for i, st in enumerate(starts):
        np.testing.assert_array_equal(got[i * k:(i + 1) * k], O.select_keep(s[st:st + n], k),
                                      err_msg=f"segment {i}")


def test_select_many_long_segments_mixed_branches():
    """More long segments than the GPU has CUs, mixing the distributions and branches of the
    register path (surprisal-like, +inf filling or not the budget, a narrow band inside a
    wide range, ulp-spaced, all equal), k = 0 and k = len, zero-length segments and
    lengths below 8193; budgets over 8192 kept indices leave in several staging windows."""
    r = np.random.default_rng(2024)
    n_segs = 700
    lens = [int(x) for x in r.choice([12288, 32768, 9000 * 4 // 4, 16384, 4096], n_segs)]
    lens[5] = 0
    lens = [n - n % 4 for n in lens]
    segs, ks = [], []
    for i, n in enumerate(lens):
        kind = i % 6
        if kind == 0:
            x = r.exponential(3.0, n)
        elif kind == 1:
            x = r.exponential(3.0, n)
            x[r.permutation(n)[: n // 2]] = np.inf
        elif kind == 2:
            x = 11.0 + r.uniform(0.0, 1e-4, n)
            m = n // 12
            x[r.permutation(n)[:m]] = r.uniform(0.0, 100.0, m)
        elif kind == 3:
            x = 1.0 + r.integers(0, 200, n) * 2.0 ** -23
        elif kind == 4:
            x = np.full(n, np.log(128256.0))
            x[::97] = np.inf
        else:
            x = np.round(r.standard_normal(n), 2)
            x[::13] = -np.inf
        segs.append(np.asarray(x, dtype=np.float32))
        ks.append(int(r.choice([0, 1, max(1, n // 4), n // 2, max(0, n - 1), n])) if n else 0)
    s = np.concatenate(segs).astype(np.float32)
    starts = np.concatenate([[0], np.cumsum(lens)[:-1]])
    print(f"[select] mixed: {n_segs} segments, {len(s)} scores", flush=True)
    got = _gpu_select(s, starts, lens, ks)
    off = 0
    for st, n, k in zip(starts, lens, ks):
        np.testing.assert_array_equal(got[off:off + k], O.select_keep(s[st:st + n], k),
                                      err_msg=f"len={n} k={k}")
        off += k


def test_select_thousands_of_long_segments():
    """Over 2048 long segments (eight workgroups of the register path per CU): unaligned
    starts, lengths not divisible by four, k = 0 and k = len next to ordinary budgets, five
    score distributions.  Every fifth pair of neighbours and the last segment against the
    oracle; every list ascending and inside its segment."""
    r = np.random.default_rng(77)
    n_segs = 2049
    lens = [int(x) for x in r.choice([8196, 9000, 12288, 16384, 32768, 8193, 10001], n_segs)]
    segs, ks, starts, pos = [], [], [], 0
    for i, n in enumerate(lens):
        kind = i % 5
        if kind == 0:
            x = r.exponential(3.0, n)
            x[-1] = np.inf
        elif kind == 1:
            x = 11.0 + r.uniform(0.0, 1e-4, n)
        elif kind == 2:
            x = 1.0 + r.integers(0, 300, n) * 2.0 ** -23
        elif kind == 3:
            x = np.round(r.standard_normal(n), 2)
            x[::17] = -np.inf
        else:
            x = r.exponential(3.0, n)
            x[r.permutation(n)[: n // 3]] = np.inf
        pos += 1 if i % 7 == 3 else 0   # a 4-byte offset: an unaligned start
        starts.append(pos)
        segs.append((pos, np.asarray(x, dtype=np.float32)))
        pos += n
        ks.append(int(r.choice([0, 1, n // 4, n // 4, n // 2, n - 1, n])))
    s = np.zeros(pos, dtype=np.float32)
    for st, x in segs:
        s[st:st + len(x)] = x
    print(f"[select] two per workgroup: {n_segs} segments, {len(s)} scores", flush=True)
    got = _gpu_select(s, starts, lens, ks)
    offs = np.concatenate([[0], np.cumsum(ks)])
    check = sorted({i for w in range(0, n_segs // 2 + 1, 5) for i in (2 * w, 2 * w + 1) if i < n_segs}
                   | {n_segs - 1})
    for i in range(n_segs):
        g = got[offs[i]:offs[i + 1]]
        assert len(g) == 0 or (g[0] >= 0 and g[-1] < lens[i] and np.all(np.diff(g) > 0)), f"segment {i}"
    for i in check:
        st, n, k = starts[i], lens[i], ks[i]
        np.testing.assert_array_equal(got[offs[i]:offs[i + 1]], O.select_keep(s[st:st + n], k),
                                      err_msg=f"segment {i} len={n} k={k}")


def test_select_overlapping_segments_identical_lists():
    r = np.random.default_rng(9)
    s = r.standard_normal(4096).astype(np.float32)
    s[-1] = np.inf
    got = _gpu_select(s, [0] * 8, [4096] * 8, [1024] * 8).reshape(8, 1024)
    ref = O.select_keep(s, 1024)
    for h in range(8):
        np.testing.assert_array_equal(got[h], ref)


def test_select_all_equal_scores():
    s = np.full(3000, np.log(128256.0), dtype=np.float32)
    s[-1] = np.inf
    got = _gpu_select(s, [0], [3000], [700])
    np.testing.assert_array_equal(got, np.r_[np.arange(699), 2999])


def _contig_cache(L, B, hkv, cap, d, seed, dtype=torch.bfloat16):
    g = torch.Generator().manual_seed(seed)
    k = torch.randn((B, L, hkv, cap, d), generator=g).to(dtype).cuda()
    v = torch.randn((B, L, hkv, cap, d), generator=g).to(dtype).cuda()
    return k, v


@pytest.mark.parametrize("in_place", [True, False])
@pytest.mark.parametrize("per_head", [0, 1])
def test_compact_contiguous(in_place, per_head):
    from paper_2607_27600_amd import cc
    print(f"[compact] contiguous in_place={in_place} per_head={per_head}", flush=True)
    L, hkv, d = 3, 4, 128
    lens = [300, 1, 1000]
    B, cap = len(lens), max(lens)
    cu = np.concatenate([[0], np.cumsum(lens)]).astype(np.int32)
    k, v = _contig_cache(L, B, hkv, cap, d, seed=1)
    k0, v0 = k.clone(), v.clone()
    r = np.random.default_rng(3)
    lists, kk = [], []
    for b, n in enumerate(lens):
        for h in range(hkv if per_head else 1):
            kb = max(1, n // 4) if h % 2 == 0 else n // 3
            kb = min(kb, n)
            lists.append(np.sort(r.choice(n, kb, replace=False)).astype(np.int32))
            kk.append(kb)
    keep = torch.from_numpy(np.concatenate(lists)).cuda()
    ids = torch.from_numpy(r.integers(0, 1000, cu[-1]).astype(np.int32)).cuda()
    pos = torch.arange(int(cu[-1]), dtype=torch.int32).cuda()
    ids0, pos0 = ids.clone(), pos.clone()
    p = cc.problem(dtype="bf16", cu_seqlens=cu.tolist(), n_heads_q=hkv, n_heads_kv=hkv, head_dim=d,
                   hidden=128, vocab=1000)
    strides = dict(n_layers=L, seq_stride=L * hkv * cap * d, layer_stride=hkv * cap * d,
                   head_stride=cap * d, tok_stride=d)
    kv = cc.kv_contiguous(k, v, **strides)
    if in_place:
        cc.cc_compact_kv(p, kv, keep, kk, per_head, ids, pos)
        ok, ov = k, v
    else:
        ok, ov = torch.zeros_like(k), torch.zeros_like(v)
        out = cc.kv_contiguous(ok, ov, **strides)
        cc.cc_compact_kv(p, kv, keep, kk, per_head, ids, pos, out=out)
    torch.cuda.synchronize()
    K0, V0 = bf16_host(k0), bf16_host(v0)
    KO, VO = bf16_host(ok), bf16_host(ov)
    li = 0
    for b, n in enumerate(lens):
        for h in range(hkv):
            lst = lists[b * hkv + h] if per_head else lists[b]
            kb = len(lst)
            for l in range(L):
                np.testing.assert_array_equal(KO[b, l, h, :kb], O.compact(K0[b, l, h], lst))
                np.testing.assert_array_equal(VO[b, l, h, :kb], O.compact(V0[b, l, h], lst))
                if in_place:   # entries past k untouched
                    np.testing.assert_array_equal(KO[b, l, h, kb:], K0[b, l, h, kb:])
        first = lists[b * hkv] if per_head else lists[b]
        lo = cu[b]
        np.testing.assert_array_equal(ids.cpu().numpy()[lo:lo + len(first)],
                                      ids0.cpu().numpy()[lo + first])
        np.testing.assert_array_equal(pos.cpu().numpy()[lo:lo + len(first)], lo + first)


def test_compact_paged_in_place_matches_out_of_place():
    from paper_2607_27600_amd import cc
    from paper_2607_27600_amd.workload import Workload
    cfg = C.shrink(C.C5, seq_lens=(40, 300, 17), cache_layers=2, keep=(8, 60, 17), vocab=1000,
                   hidden=256)
    w = Workload(cfg, cache_layers=2, with_lm_head=False)
    r = np.random.default_rng(5)
    lists = [np.sort(r.choice(n, kb, replace=False)).astype(np.int32)
             for n, kb in zip(cfg.seq_lens, cfg.keep)]
    keep = torch.from_numpy(np.concatenate(lists)).cuda()
    k0, v0 = w.k_cache.clone(), w.v_cache.clone()
    ok, ov = torch.zeros_like(k0), torch.zeros_like(v0)
    P = cfg.page_size
    npg, hkv, d = k0.shape[1], cfg.n_heads_kv, cfg.head_dim
    out = cc.kv_paged(ok, ov, w.block_table, n_layers=2, layer_stride=npg * hkv * P * d,
                      page_stride=hkv * P * d, head_stride=P * d, tok_stride=d, page_size=P)
    cc.cc_compact_kv(w.problem, w.kv, keep, list(cfg.keep), 0, out=out)
    cc.cc_compact_kv(w.problem, w.kv, keep, list(cfg.keep), 0)   # in place
    torch.cuda.synchronize()
    bt = w.block_table.cpu().numpy()
    K0, KI, KO = bf16_host(k0), bf16_host(w.k_cache), bf16_host(ok)
    for b, lst in enumerate(lists):
        for j, src in enumerate(lst):
            for l in range(2):
                want = K0[l, bt[b, src // P], :, src % P]
                np.testing.assert_array_equal(KI[l, bt[b, j // P], :, j % P], want)
                np.testing.assert_array_equal(KO[l, bt[b, j // P], :, j % P], want)
