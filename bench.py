"""Benchmark of the counter-causal refresh pass on one MI355X.

One step is one whole refresh of a workload: the counter-causal scoring pass, keep
selection and compaction of every cache layer.  The headline (the JSON line's top-level
fields) is the largest single-GPU workload by cached entries per refresh:

  C5  8 ragged sequences (Qwen2.5-7B shapes, 75,696 cached entries, paged cache of 28
      layers): attention over the last cache layer -> W_o -> LM head (vocab 152064) with
      the fused log-sum-exp and target gather -> keep 20% per sequence -> compaction.

The other workloads are measured in the same run and reported as sub-objects of the same
line under "configs", each with its own roofline and oracle baseline:

  C3  Llama-3-8B shapes at n = 32768 (keep 4096 per KV head, 32-layer cache)
  C4  the full 32-layer pass (random 8B-shaped stack, n = 8192, keep 25%)
  C2  Llama-3-8B shapes at n = 4096 (keep 25%), with the FP8 and W_o-folded LM heads

Inputs are seeded synthetic data resident in HBM before the timed region.  Each step
compacts out of place (every step sees the same cache); the in-place compaction a live
refresh performs is timed on its own, with the Infinity Cache flushed.  Prints one JSON
line.

    python bench.py [--gpus 1] [--steps K] [--warmup W] [--config C5,C3,C4,C2]
                    [--no-cpu-baseline] [--config LOOP] [--pmc-driver]
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

# MI355X published peaks
PEAK_BF16_TFLOPS = 2516.6
PEAK_HBM_GBS = 8000.0
PEAK_FP8_TFLOPS = 5033.2     # dense E4M3 MFMA: 256 CU x 2.4 GHz x 8192 FLOP/clk
METRIC = "cached tokens scored/sec per refresh; attention TFLOP/s as % of bf16 MFMA peak"
DEFAULT_CONFIGS = "C5,C3,C4,C2,C2H"
# rows of the oracle's bounded sample per workload (about 10-30 s of host work each)
CPU_ROWS = {"C2": 512, "C3": 256, "C5": 512, "C4": 12, "C2H": 256}


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=10)
    # the LM-head GEMM speeds up over its first ~10 launches after an idle gap (the clock
    # settles under load)
    ap.add_argument("--warmup", type=int, default=10)
    ap.add_argument("--config", default=DEFAULT_CONFIGS,
                    help="comma-separated workloads; the first is the headline (or LOOP)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--pmc-driver", action="store_true",
                    help="for counter collection: one refresh step of the first workload, then "
                         "a plain 1 GiB device copy whose counters calibrate the byte counts; "
                         "prints nothing")
    return ap.parse_args()


# ------------------------------------------------------------------ host baseline

def host_info() -> dict:
    """Host cores this process may run on and the CPU model."""
    try:
        n_aff = len(os.sched_getaffinity(0))
    except AttributeError:  # pragma: no cover
        n_aff = os.cpu_count() or 1
    model = "unknown"
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    model = line.split(":", 1)[1].strip()
                    break
    except OSError:
        pass
    return {"affinity_cpus": n_aff, "cpu_model": model}


def _blas_threads() -> int:
    from threadpoolctl import threadpool_info
    return max([i.get("num_threads", 1) for i in threadpool_info()] + [1])


def _row_flops(cfg, rows):
    """Algorithmic FLOPs of scoring each row (attention over its allowed keys, the
    projections, the LM head): the unit by which a sampled oracle time is extrapolated."""
    import numpy as np
    cu = cfg.cu_seqlens
    rows = np.asarray(rows, dtype=np.int64)
    seq = np.searchsorted(cu, rows, side="right") - 1
    keys = (cu[seq + 1] - 1 - rows).astype(np.float64)          # strict mask: j > i
    hq, d, D, V = cfg.n_heads_q, cfg.head_dim, cfg.hidden, cfg.vocab
    att = 4.0 * d * hq * keys
    lm = 2.0 * D * V
    if cfg.mode in ("full", "last_layer_h"):
        per_layer = 2.0 * D * hq * d * 2 + 2.0 * D * cfg.ffn * 3
        return (cfg.n_layers if cfg.mode == "full" else 1) * (per_layer + att) + lm
    return att + 2.0 * D * hq * d + lm


def cpu_baseline(w, rows_count: int) -> dict:
    """The oracle (fp64 NumPy) on this host, as it stands: scores of a seeded row sample
    (rows are independent, so each is exact on its own) extrapolated to every row by
    algorithmic work, the oracle's selection over every segment, and the compaction of one
    cache plane scaled to the cache's planes."""
    import numpy as np
    from threadpoolctl import threadpool_limits

    from oracle import cc_oracle as O
    from synth import configs as C

    cfg = w.cfg
    h = w.host
    info = host_info()
    rows = C.sample_rows(cfg, count=rows_count)
    with threadpool_limits(limits=info["affinity_cpus"]):
        threads = _blas_threads()
        t0 = time.perf_counter()
        if cfg.mode == "full":
            kvl = h["kv_layers"]
            s = O.full_scores(h["ids"], lambda l: (kvl[l]["k"], kvl[l]["v"]),
                              lambda l: h["layers"][l], h["embed"], h["final_norm"], h["w_lm"],
                              cfg.cu_seqlens, cfg.n_layers, cfg.n_heads_q, cfg.head_dim,
                              cfg.rope_theta, cfg.rms_eps, rows=rows)
        elif cfg.mode == "last_layer_h":
            s = O.last_layer_h_scores(h["h_last"], h["ids"], h["k"], h["v"], h["layer"],
                                      h["final_norm"], h["w_lm"], cfg.cu_seqlens, cfg.n_heads_q,
                                      cfg.head_dim, cfg.rope_theta, cfg.rms_eps, rows=rows)
        else:
            s = O.last_layer_scores(h["q"], h["k"], h["v"], h["w_o"], h["w_lm"], h["ids"],
                                    cfg.cu_seqlens, rows=rows)
        t_sample = time.perf_counter() - t0
        scale = float(_row_flops(cfg, np.arange(cfg.n_tokens)).sum() /
                      _row_flops(cfg, rows).sum())
        t_score = t_sample * scale
        # selection in full over the real segments (sampled scores in place, the rest a
        # fixed fill: the oracle's sort costs the same whatever the values)
        full = np.linspace(1.0, 20.0, cfg.n_tokens)
        full[rows] = s
        cu = cfg.cu_seqlens
        per = cfg.n_heads_kv if cfg.per_head_select else 1
        t0 = time.perf_counter()
        lists = []
        for b in range(cfg.n_seqs):
            seg = full[cu[b]:cu[b + 1]]
            for _ in range(per):
                lists.append(O.select_keep(seg, int(cfg.keep[b])))
        t_sel = time.perf_counter() - t0
        # compaction: one [n_b][d] plane of the longest sequence, scaled by kept rows to the
        # planes of every sequence (keys and values of every layer and KV head)
        b_max = int(np.argmax(cfg.seq_lens))
        plane = h["k"][0, cu[b_max]:cu[b_max + 1]]
        t0 = time.perf_counter()
        O.compact(plane, lists[b_max * per])
        t_plane = time.perf_counter() - t0
        planes = 2 * w.cache_layers * cfg.n_heads_kv
        t_compact = t_plane * planes * sum(cfg.keep) / max(1, int(cfg.keep[b_max]))
    total = t_score + t_sel + t_compact
    return {"value": cfg.n_tokens / total, "unit": "tokens/s", "cores": int(threads),
            "kind": "oracle",
            "sample": (f"fp64 oracle scores of {len(rows)} of {cfg.n_tokens} rows (first/last "
                       f"rows of each sequence plus uniform picks, {t_sample:.1f} s), time "
                       f"scaled by algorithmic work (x{scale:.1f}); full selection of every "
                       f"segment; compaction of one plane scaled to the {planes} planes of "
                       f"every sequence"),
            "extrapolated": True, "affinity_cpus": info["affinity_cpus"],
            "cpu_model": info["cpu_model"],
            "seconds": {"score_sample": t_sample, "score_extrapolated": t_score,
                        "select": t_sel, "compact_extrapolated": t_compact}}


# ------------------------------------------------------------------ device helpers

def flushed_ms(fn, reps: int, flush) -> float:
    """Mean time of fn() on the current stream with the 256 MB Infinity Cache and the L2s
    flushed before every call: a 1 GiB buffer is read in between (a read leaves the caches
    holding clean lines, so the timed call is not charged for writing back the flush's own
    data)."""
    import torch
    stream = torch.cuda.current_stream()
    ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
          for _ in range(reps)]
    sink = torch.empty(reps, dtype=flush.dtype, device=flush.device)
    for i, (a, b) in enumerate(ev):
        torch.sum(flush, dim=0, out=sink[i])
        a.record(stream)
        fn()
        b.record(stream)
    torch.cuda.synchronize()
    return sum(a.elapsed_time(b) for a, b in ev) / reps


def lmhead_traffic(cfg_name: str):
    """HBM bytes per LM-head launch from the committed counter summary of this workload,
    or None when there is none or the GEMM source has changed since it was taken."""
    import hashlib
    path = os.path.join(ROOT, "profiles", f"lmhead_{cfg_name.lower()}_traffic.json")
    src = os.path.join(ROOT, "paper_2607_27600_amd", "csrc", "gemm.hip")
    try:
        with open(path) as f:
            rec = json.load(f)
        with open(src, "rb") as f:
            digest = hashlib.sha256(f.read()).hexdigest()
    except OSError:
        return None
    return rec.get("bytes_per_launch") if rec.get("gemm_source_sha256") == digest else None


def select_sweep(dev, flush, reps: int = 5) -> dict:
    """Keep selection at a size where it streams from HBM: 4096 segments of 32768 scores
    (512 MB), keep 25% of each.  Scores are drawn like surprisals (exponential, mean 3)."""
    import numpy as np
    import torch
    from paper_2607_27600_amd import cc
    n_segs, seg, k = 4096, 32768, 8192
    g = torch.Generator(device=dev)
    g.manual_seed(0)
    scores = torch.empty(n_segs * seg, dtype=torch.float32, device=dev).exponential_(1 / 3.0, generator=g)
    keep = torch.empty(n_segs * k, dtype=torch.int32, device=dev)
    ws = torch.empty(max(1, cc.cc_select_workspace(n_segs)), dtype=torch.uint8, device=dev)
    # the segment arrays are built once (host-side conversion stays out of the timed calls)
    starts = np.arange(n_segs, dtype=np.int64) * seg
    lens = np.full(n_segs, seg, dtype=np.int32)
    ks = np.full(n_segs, k, dtype=np.int32)
    cc.cc_select_keep(scores, starts, lens, ks, keep, ws)
    ms = flushed_ms(lambda: cc.cc_select_keep(scores, starts, lens, ks, keep, ws), reps, flush)
    nbytes = 4 * n_segs * seg + 4 * n_segs * k
    del scores, keep
    return {"segments": n_segs, "segment_len": seg, "k": k, "ms": ms, "bytes": nbytes,
            "gb_s": nbytes / (ms * 1e-3) / 1e9, "frac_hbm": nbytes / (ms * 1e-3) / 1e9 / PEAK_HBM_GBS,
            "note": "Infinity Cache flushed before each call; bytes = scores read + keep written"}


def _segments(cfg):
    cu = cfg.cu_seqlens
    starts, lens, ks = [], [], []
    for b in range(cfg.n_seqs):
        for _ in range(cfg.n_heads_kv if cfg.per_head_select else 1):
            starts.append(int(cu[b]))
            lens.append(int(cu[b + 1] - cu[b]))
            ks.append(int(cfg.keep[b]))
    return starts, lens, ks


def _out_cache(w):
    """A second cache of the same geometry, the destination of out-of-place compaction."""
    import torch
    from paper_2607_27600_amd import cc
    out_k = torch.empty_like(w.k_cache)
    out_v = torch.empty_like(w.v_cache)
    s = w.kv.struct
    if w.cfg.paged:
        kv = cc.kv_paged(out_k, out_v, w.block_table, n_layers=s.n_layers,
                         layer_stride=s.layer_stride, page_stride=s.page_stride,
                         head_stride=s.head_stride, tok_stride=s.tok_stride,
                         page_size=s.page_size)
    else:
        kv = cc.kv_contiguous(out_k, out_v, n_layers=s.n_layers, seq_stride=s.seq_stride,
                              layer_stride=s.layer_stride, head_stride=s.head_stride,
                              tok_stride=s.tok_stride)
    return kv


# ------------------------------------------------------------------ one workload

def bench_config(args, name: str, dev, with_extras: bool) -> dict:
    """Whole refreshes of one workload.  Last-layer workloads run as the sub-step chain
    (attention -> W_o -> packed LM head -> select -> compaction), checked once to equal
    cc_score bit for bit, so each sub-step has its own HIP-event time; the full pass and
    the exact fast variant (from the stored activations H, which are compacted with the
    cache) run as cc_score."""
    import torch
    from paper_2607_27600_amd import cc
    from paper_2607_27600_amd.workload import Workload
    from synth import configs as C

    cfg = C.CONFIGS[name]
    t_gen = time.perf_counter()
    w = Workload(cfg, device=dev, keep_host=not args.no_cpu_baseline)
    t_gen = time.perf_counter() - t_gen
    p = w.problem
    pp = cc.packed(p)
    N, Hq, d, D, V = cfg.n_tokens, cfg.n_heads_q, cfg.head_dim, cfg.hidden, cfg.vocab
    L, hkv = w.cache_layers, cfg.n_heads_kv
    per_head = int(cfg.per_head_select)
    starts, lens, ks = _segments(cfg)
    stream = torch.cuda.current_stream()

    # per-model preparation, outside the timed region: the packed LM-head weight
    w_packed = cc.cc_pack_lmhead(w.w_lm)
    ev_pk = [torch.cuda.Event(enable_timing=True) for _ in range(2)]
    ev_pk[0].record(stream)
    cc.cc_pack_lmhead(w.w_lm, out=w_packed)
    ev_pk[1].record(stream)
    torch.cuda.synchronize()
    pack_w_ms = ev_pk[0].elapsed_time(ev_pk[1])

    scores = torch.empty(N, dtype=torch.float32, device=dev)
    keep = torch.empty(sum(ks), dtype=torch.int32, device=dev)
    ws_sel = torch.empty(max(1, cc.cc_select_workspace(len(ks))), dtype=torch.uint8, device=dev)
    ws_cmp = torch.empty(max(1, cc.cc_compact_workspace(p, L, per_head)), dtype=torch.uint8,
                         device=dev)
    out_kv = _out_cache(w)
    # the exact fast variant also compacts the stored activations H with the cache
    h_rows = w.h_last if cfg.mode == "last_layer_h" else None
    if h_rows is not None:
        out_h = torch.empty_like(h_rows)
        ws_rows = torch.empty(max(1, cc.cc_compact_rows_workspace(
            p, h_rows[0].numel() * h_rows.element_size(), per_head)), dtype=torch.uint8, device=dev)
    # the full pass and the exact fast variant (from the stored activations H) run as cc_score
    full = cfg.mode in ("full", "last_layer_h")
    o = u = ws_att = None
    if full:
        names = ["score", "select", "compact"]
        ws_score = torch.empty(max(1, cc.cc_score_workspace(pp)), dtype=torch.uint8, device=dev)
        inp = w.inputs(w_packed)
    else:
        names = ["attention", "wo_proj", "lmhead_lse", "select", "compact"]
        o = torch.empty((N, Hq, d), dtype=torch.bfloat16, device=dev)
        u = torch.empty((N, D), dtype=torch.bfloat16, device=dev)
        ws_att = torch.empty(max(1, cc.cc_attention_workspace(p)), dtype=torch.uint8, device=dev)
        ws_lm = torch.empty(max(1, cc.cc_lmhead_workspace(pp)), dtype=torch.uint8, device=dev)

    def step(ev=None):
        def mark(i):
            if ev is not None:
                ev[i].record(stream)
        mark(0)
        if full:
            cc.cc_score(pp, inp, scores, ws_score)
        else:
            cc.cc_attention_cc(p, w.q, w.kv, L - 1, o, ws_att)
            mark(1)
            cc.cc_linear("bf16", o.view(N, Hq * d), w.w_o, u)
            mark(2)
            cc.cc_lmhead_score_packed(pp, u, w_packed, w.ids, scores, workspace=ws_lm)
        mark(len(names) - 2)
        cc.cc_select_keep(scores, starts, lens, ks, keep, ws_sel)
        mark(len(names) - 1)
        cc.cc_compact_kv(p, w.kv, keep, ks, per_head, out=out_kv, workspace=ws_cmp)
        if h_rows is not None:
            cc.cc_compact_rows(p, h_rows, keep, ks, per_head, out=out_h, workspace=ws_rows)
        mark(len(names))

    if args.pmc_driver:
        step()
        src = torch.empty(1 << 30, dtype=torch.uint8, device=dev)
        dst = torch.empty_like(src)
        dst.copy_(src)
        torch.cuda.synchronize()
        return {}

    if not full:
        # the sub-step chain is the same work as cc_score; check once that they agree
        ref_scores = torch.empty_like(scores)
        cc.cc_score(pp, w.inputs(w_packed), ref_scores)
        step()
        torch.cuda.synchronize()
        if not torch.equal(ref_scores, scores):
            raise SystemExit(f"{name}: sub-step chain and cc_score disagree")
        del ref_scores

    # The clock drops in any idle gap and takes about ten LM-head launches to settle again,
    # so the warm-up runs right before the timed steps with only the synchronisation between.
    evs = [[torch.cuda.Event(enable_timing=True) for _ in range(len(names) + 1)]
           for _ in range(args.steps)]
    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for i in range(args.steps):
        step(evs[i])
    torch.cuda.synchronize()
    ms_step = (time.perf_counter() - t0) * 1e3 / args.steps
    part = {n: sum(e[j].elapsed_time(e[j + 1]) for e in evs) / args.steps
            for j, n in enumerate(names)}

    # FLOPs and bytes (algorithmic)
    att_flop = 2.0 * d * Hq * sum(n * (n - 1) for n in cfg.seq_lens)
    lm_flop = 2.0 * N * D * V
    wo_flop = 2.0 * N * D * Hq * d
    per_layer = 2.0 * N * D * (Hq * d) * 2 + 2.0 * N * D * cfg.ffn * 3
    kept_rows = sum(ks) if per_head else sum(ks) * hkv        # (token, KV head) rows per layer
    kv_bytes = cmp_bytes = 2 * (2 * L * kept_rows * d * 2)    # K and V, read + write
    if h_rows is not None:                                     # + the stored activations H
        cmp_bytes += 2 * sum(ks) * h_rows[0].numel() * h_rows.element_size()

    res = {"workload": f"{cfg.name}: {cfg.description}", "n_cached": N, "n_seqs": cfg.n_seqs,
           "cache_layers": L, "paged": bool(cfg.paged), "mode": cfg.mode,
           "value": N / (ms_step * 1e-3), "unit": "tokens/s", "ms_per_step": ms_step,
           "breakdown_ms": part, "input_generation_s": t_gen,
           "lmhead_layout": {"packed": True, "pack_w_lm_ms": pack_w_ms}}
    if full:
        n_pass = cfg.n_layers if cfg.mode == "full" else 1
        score_flop = n_pass * (per_layer + att_flop) + lm_flop
        achieved = score_flop / (part["score"] * 1e-3) / 1e12
        what = ("the whole 32-layer score pass (cc_score, FULL)" if cfg.mode == "full" else
                "the exact fast variant's score pass (cc_score, LAST_LAYER_H: the last layer "
                "from the stored activations, then the LM head)")
        res["roofline"] = {
            "kernel": what + ": every kernel in it is a bf16 MFMA contraction (projections, "
                      "SwiGLU MLP, attention, LM head) or negligible",
            "bound": "mfma", "achieved": achieved, "peak": PEAK_BF16_TFLOPS, "unit": "TFLOP/s",
            "frac": achieved / PEAK_BF16_TFLOPS, "traffic": None, "flop_per_launch": score_flop}
        # attention of one layer at this workload's shape, on its own (synthetic queries)
        qa = torch.randn((N, Hq, d), dtype=torch.bfloat16, device=dev)
        oa = torch.empty_like(qa)
        ws_a = torch.empty(max(1, cc.cc_attention_workspace(p)), dtype=torch.uint8, device=dev)
        for _ in range(3):
            cc.cc_attention_cc(p, qa, w.kv, L - 1, oa, ws_a)
        ea = [torch.cuda.Event(enable_timing=True) for _ in range(2)]
        ea[0].record(stream)
        for _ in range(args.steps):
            cc.cc_attention_cc(p, qa, w.kv, L - 1, oa, ws_a)
        ea[1].record(stream)
        torch.cuda.synchronize()
        att_ms = ea[0].elapsed_time(ea[1]) / args.steps
        del qa, oa, ws_a
        res["score_tflops"] = achieved
    else:
        att_ms = part["attention"]
        lm_tflops = lm_flop / (part["lmhead_lse"] * 1e-3) / 1e12
        res["roofline"] = {
            "kernel": "LM head on packed operands with the fused log-sum-exp and target gather "
                      "(pack_rows of U + gemm_lmhead_packed<EpiLse16> + lse_combine)",
            "bound": "mfma", "achieved": lm_tflops, "peak": PEAK_BF16_TFLOPS, "unit": "TFLOP/s",
            "frac": lm_tflops / PEAK_BF16_TFLOPS, "traffic": lmhead_traffic(name),
            "flop_per_launch": lm_flop}
        res["wo_proj_tflops"] = wo_flop / (part["wo_proj"] * 1e-3) / 1e12
    att_tflops = att_flop / (att_ms * 1e-3) / 1e12
    res["attention"] = {"ms": att_ms, "tflops": att_tflops,
                        "frac_bf16_peak": att_tflops / PEAK_BF16_TFLOPS,
                        "flop_per_launch": att_flop,
                        "note": "one layer, timed on its own" if full else "sub-step of the step"}
    res["select"] = {"ms": part["select"], "segments": len(ks)}
    res["compact"] = {"mode": "out of place (in the step)", "bytes_moved": cmp_bytes,
                      "ms": part["compact"], "gb_s": cmp_bytes / (part["compact"] * 1e-3) / 1e9,
                      "frac_hbm": cmp_bytes / (part["compact"] * 1e-3) / 1e9 / PEAK_HBM_GBS}

    flush = torch.empty(1 << 28, dtype=torch.float32, device=dev)
    if with_extras:
        res["select_sweep"] = select_sweep(dev, flush)
    if with_extras and not full:
        res.update(next4_extras(args, cc, w, p, cfg, o, u, scores, ks, starts, lens, ws_att,
                                ws_sel, ws_cmp, out_kv, stream, ms_step, part["lmhead_lse"]))
    # in-place compaction (what a live refresh does), with and without the cache flushed;
    # every call reads and writes the same rows.  Last: it rewrites the workload's cache.
    cc.cc_compact_kv(p, w.kv, keep, ks, per_head, workspace=ws_cmp)
    ev_ip = [torch.cuda.Event(enable_timing=True) for _ in range(2)]
    torch.cuda.synchronize()
    ev_ip[0].record(stream)
    for _ in range(args.steps):
        cc.cc_compact_kv(p, w.kv, keep, ks, per_head, workspace=ws_cmp)
    ev_ip[1].record(stream)
    torch.cuda.synchronize()
    ip_ms = ev_ip[0].elapsed_time(ev_ip[1]) / args.steps
    ip_fl = flushed_ms(lambda: cc.cc_compact_kv(p, w.kv, keep, ks, per_head, workspace=ws_cmp),
                       5, flush)
    res["compact_in_place"] = {"bytes_moved": kv_bytes, "ms": ip_ms,
                               "gb_s": kv_bytes / (ip_ms * 1e-3) / 1e9,
                               "ms_cache_flushed": ip_fl,
                               "gb_s_cache_flushed": kv_bytes / (ip_fl * 1e-3) / 1e9,
                               "frac_hbm_cache_flushed": kv_bytes / (ip_fl * 1e-3) / 1e9 / PEAK_HBM_GBS}
    del flush, out_kv
    if not args.no_cpu_baseline:
        res["cpu_baseline"] = cpu_baseline(w, CPU_ROWS.get(name, 64))
    return res


def next4_extras(args, cc, w, p, cfg, o, u, scores, ks, seg_start, seg_len, ws_att, ws_sel,
                 ws_cmp, out_kv, stream, ms_two_step, lm_ms_packed) -> dict:
    """Alternatives of the dominant step, measured beside the bf16 headline: the row-major
    LM head on the same rows, the LM head with W_o folded in, and the FP8 LM head."""
    import torch
    N, Hq, d, D, V = cfg.n_tokens, cfg.n_heads_q, cfg.head_dim, cfg.hidden, cfg.vocab
    dev = scores.device
    per_head = int(cfg.per_head_select)
    lm_flop = 2.0 * N * D * V
    fin = torch.isfinite(scores)
    keep = torch.empty(sum(ks), dtype=torch.int32, device=dev)
    out = {}

    # the row-major LM head on the same rows (same warm-up rule)
    ws_rm = torch.empty(max(1, cc.cc_lmhead_workspace(p)), dtype=torch.uint8, device=dev)
    s_rm = torch.empty_like(scores)
    ev = [torch.cuda.Event(enable_timing=True) for _ in range(2)]
    for _ in range(args.warmup):
        cc.cc_lmhead_score(p, u, w.w_lm, w.ids, s_rm, workspace=ws_rm)
    ev[0].record(stream)
    for _ in range(args.steps):
        cc.cc_lmhead_score(p, u, w.w_lm, w.ids, s_rm, workspace=ws_rm)
    ev[1].record(stream)
    torch.cuda.synchronize()
    rm_ms = ev[0].elapsed_time(ev[1]) / args.steps
    rm_diff = float((s_rm[fin] - scores[fin]).abs().max().item()) if bool(fin.any()) else 0.0
    out["lmhead_row_major"] = {"ms": rm_ms, "tflops": lm_flop / (rm_ms * 1e-3) / 1e12,
                               "max_abs_score_diff_vs_packed": rm_diff,
                               "packed_ms": lm_ms_packed}
    del ws_rm, s_rm

    # W_o folded into the LM head (mode LAST_LAYER_FUSED): the product is made and packed once
    # per model; a fused step is attention -> packed LM head on the product -> select -> compact
    pf = cc.problem(dtype="bf16", cu_seqlens=cfg.cu_seqlens.tolist(), n_heads_q=Hq,
                    n_heads_kv=cfg.n_heads_kv, head_dim=d, hidden=D, vocab=V, device=dev,
                    mode="last_layer_fused", lmhead_packed=True)
    m = torch.empty((V, Hq * d), dtype=torch.bfloat16, device=dev)
    ws_fuse = torch.empty(cc.cc_fuse_wo_lmhead_workspace("bf16", D, Hq * d), dtype=torch.uint8,
                          device=dev)
    cc.cc_fuse_wo_lmhead("bf16", w.w_lm, w.w_o, out=m, workspace=ws_fuse)
    ev[0].record(stream)
    cc.cc_fuse_wo_lmhead("bf16", w.w_lm, w.w_o, out=m, workspace=ws_fuse)
    ev[1].record(stream)
    torch.cuda.synchronize()
    fuse_ms = ev[0].elapsed_time(ev[1])
    del ws_fuse
    m_packed = cc.cc_pack_lmhead(m)
    del m
    inp = cc.inputs(kv=w.kv, token_ids=w.ids, q=w.q, w_lm_packed=m_packed)
    ws = torch.empty(cc.cc_score_workspace(pf), dtype=torch.uint8, device=dev)
    s_fused = torch.empty_like(scores)

    def fstep():
        cc.cc_score(pf, inp, s_fused, workspace=ws)
        cc.cc_select_keep(s_fused, seg_start, seg_len, ks, keep, ws_sel)
        cc.cc_compact_kv(pf, w.kv, keep, ks, per_head, out=out_kv, workspace=ws_cmp)

    for _ in range(max(1, args.warmup)):
        fstep()
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(args.steps):
        fstep()
    torch.cuda.synchronize()
    ms = (time.perf_counter() - t0) * 1e3 / args.steps
    diff = float((s_fused[fin] - scores[fin]).abs().max().item()) if bool(fin.any()) else 0.0
    out["fused_wo_lmhead"] = {
        "ms_per_step": ms, "tokens_per_s": N / (ms * 1e-3), "speedup_vs_two_step": ms_two_step / ms,
        "fuse_weight_ms": fuse_ms, "max_abs_score_diff_vs_two_step": diff,
        "note": "W_lm W_o made and packed once per model (fuse_weight_ms, outside the step)"}
    del m_packed, ws, s_fused

    # the LM head on E4M3 codes (one scale for W_lm, one per entry for u, quantized inside
    # the call)
    keep_bf = torch.empty(sum(ks), dtype=torch.int32, device=dev)
    cc.cc_select_keep(scores, seg_start, seg_len, ks, keep_bf, ws_sel)
    wq, wsc = cc.cc_quantize_fp8("bf16", w.w_lm, per_row=False)
    ev[0].record(stream)
    cc.cc_quantize_fp8("bf16", w.w_lm, per_row=False, codes=wq, scale=wsc)
    ev[1].record(stream)
    torch.cuda.synchronize()
    quant_ms = ev[0].elapsed_time(ev[1])
    ws8 = torch.empty(cc.cc_lmhead_fp8_workspace(p), dtype=torch.uint8, device=dev)
    s8 = torch.empty(N, dtype=torch.float32, device=dev)
    keep8 = torch.empty_like(keep_bf)

    def lm8():
        cc.cc_lmhead_score_fp8(p, u, wq, wsc, w.ids, s8, workspace=ws8)

    def step8():
        cc.cc_attention_cc(p, w.q, w.kv, w.cache_layers - 1, o, ws_att)
        cc.cc_linear("bf16", o.view(N, Hq * d), w.w_o, u)
        lm8()
        cc.cc_select_keep(s8, seg_start, seg_len, ks, keep8, ws_sel)
        cc.cc_compact_kv(p, w.kv, keep8, ks, per_head, out=out_kv, workspace=ws_cmp)

    for _ in range(max(1, args.warmup)):
        step8()
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(args.steps):
        step8()
    torch.cuda.synchronize()
    ms = (time.perf_counter() - t0) * 1e3 / args.steps
    ev[0].record(stream)
    for _ in range(args.steps):
        lm8()
    ev[1].record(stream)
    torch.cuda.synchronize()
    lm_ms = ev[0].elapsed_time(ev[1]) / args.steps
    diff = (s8[fin] - scores[fin]).abs()
    a = set(keep_bf.cpu().tolist())
    b = set(keep8.cpu().tolist())
    out["lmhead_fp8"] = {
        "ms_per_step": ms, "tokens_per_s": N / (ms * 1e-3), "speedup_vs_bf16_step": ms_two_step / ms,
        "lmhead_ms": lm_ms, "lmhead_tflops": lm_flop / (lm_ms * 1e-3) / 1e12,
        "lmhead_frac_fp8_peak": lm_flop / (lm_ms * 1e-3) / 1e12 / PEAK_FP8_TFLOPS,
        "quantize_w_ms": quant_ms,
        "score_diff_vs_bf16": {"max_abs": float(diff.max().item()),
                               "mean_abs": float(diff.mean().item())},
        "keep_overlap_vs_bf16": len(a & b) / max(1, len(a)),
        "note": "W_lm quantized once per model (quantize_w_ms, outside the step); u is "
                "quantized per entry inside the LM-head call; lmhead_ms includes that"}
    return out


# ------------------------------------------------------------------ refresh loop

def bench_loop(args, dev) -> dict:
    """The cache-managed inference cycle at the paper's end-to-end setting (cache budget
    J = 512, chunk h = 256) with Qwen2.5-7B shapes (28 cache layers, 28q/4kv, hidden 3584,
    SwiGLU 18944, vocab 152064) in the exact fast variant: a 4096-token prompt appended in
    chunks, then 1024 decoded tokens appended one at a time, a refresh every 256 tokens
    (each scores J + h = 768 entries).  Keys, values, activations and ids of the stream
    are seeded synthetic data; the model forward that produces them lies outside this library, so
    appends are copies of the stream's next entries."""
    import numpy as np
    import torch
    from paper_2607_27600_amd import cc
    from paper_2607_27600_amd.refresh import Model, RefreshLoop, run_stream
    from synth import gen
    L, hq, hkv, d, D, F, V = 28, 28, 4, 128, 3584, 18944, 152064
    J, h, T_prompt, T_total = 512, 256, 4096, 5120
    t_gen = time.perf_counter()
    up = lambda a: torch.from_numpy(a.view(np.int16)).view(torch.bfloat16).to(dev)
    wt = lambda tid, shape: up(gen.normal_bf16(0, 20000 + tid, shape, 0.02))
    ones = up(gen.f32_to_bf16_bits(np.ones(D, np.float32)))
    layer = dict(attn_norm=ones, wq=wt(1, (hq * d, D)), wo=wt(2, (D, hq * d)), mlp_norm=ones,
                 w_gate=wt(3, (F, D)), w_up=wt(4, (F, D)), w_down=wt(5, (D, F)))
    m = Model(mode="last_layer_h", n_layers=L, n_heads_q=hq, n_heads_kv=hkv, head_dim=d,
              hidden=D, vocab=V, w_lm=wt(6, (V, D)), layer=layer, final_norm=ones, ffn=F)
    m.w_lm_packed = cc.cc_pack_lmhead(m.w_lm)      # packed once per model
    S_k = up(gen.normal_bf16(0, 20010, (L, hkv, T_total, d)))
    S_v = up(gen.normal_bf16(0, 20011, (L, hkv, T_total, d)))
    S_h = up(gen.normal_bf16(0, 20012, (T_total, D)))
    S_ids = torch.from_numpy(gen.uniform_ints(0, 20013, (T_total,), 0, V).astype(np.int32)).to(dev)
    pos = torch.arange(T_total, dtype=torch.int32, device=dev)
    t_gen = time.perf_counter() - t_gen

    def entry(t0, t1):
        return S_k[:, :, t0:t1], S_v[:, :, t0:t1], S_ids[t0:t1], pos[t0:t1], S_h[t0:t1]

    def one_run():
        loop = RefreshLoop(m, J, h, device=dev)
        times = []
        inner = loop.refresh

        def timed(hook=None):
            if loop.n <= loop.J:
                return inner(hook)
            a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            a.record()
            kept = inner(hook)
            b.record()
            times.append((a, b))
            return kept
        loop.refresh = timed
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        run_stream(loop, entry, T_prompt, T_total)
        torch.cuda.synchronize()
        wall = time.perf_counter() - t0
        return wall, [a.elapsed_time(b) for a, b in times]

    for _ in range(max(1, args.warmup)):
        one_run()
    wall, ref_ms = one_run()
    return {
        "metric": "refresh cycle latency at J + h cached entries (exact fast variant)",
        "value": float(np.mean(ref_ms)), "unit": "ms", "higher_is_better": False,
        "n_gpus": 1, "dtype": "bf16", "data": "synthetic",
        "config": {"workload": "LOOP: Qwen2.5-7B shapes, exact fast variant, J=512, h=256, "
                               "4096-token prompt + 1024 decoded tokens",
                   "J": J, "h": h, "cache_layers": L, "prompt": T_prompt, "total": T_total,
                   "lmhead": "packed"},
        "refreshes": len(ref_ms), "refresh_ms_min": float(np.min(ref_ms)),
        "refresh_ms_median": float(np.median(ref_ms)),
        "stream_wall_s": wall, "amortised_refresh_us_per_token": float(np.sum(ref_ms)) * 1e3 / T_total,
        "input_generation_s": t_gen,
    }


# ------------------------------------------------------------------ main

def main():
    args = parse()
    if args.gpus != 1:
        print(f"bench.py runs on exactly one GPU (asked for {args.gpus}): the refresh pass is "
              "built and measured on one MI355X; multi-GPU sharding is a design note only.",
              file=sys.stderr)
        sys.exit(2)

    import torch

    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    if args.config == "LOOP":
        print(json.dumps(bench_loop(args, dev)), flush=True)
        return
    names = [c.strip() for c in args.config.split(",") if c.strip()]
    if args.pmc_driver:
        bench_config(args, names[0], dev, with_extras=False)
        return
    results = {}
    for i, name in enumerate(names):
        # the kernel-level extras (select sweep; FP8, fused and row-major LM heads) run with
        # the C2 workload when it is measured, else with the headline
        extras = name == "C2" or ("C2" not in names and i == 0)
        t0 = time.perf_counter()
        results[name] = bench_config(args, name, dev, with_extras=extras)
        torch.cuda.empty_cache()
        print(f"[bench] {name}: {results[name]['value']:.4g} tokens/s, "
              f"{results[name]['ms_per_step']:.3f} ms/step ({time.perf_counter() - t0:.0f} s)",
              file=sys.stderr, flush=True)
    head = results[names[0]]
    line = {
        "metric": METRIC,
        "value": head["value"],
        "unit": "tokens/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": head["ms_per_step"],
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic",
        "config": {"workload": head["workload"], "n_cached": head["n_cached"],
                   "n_seqs": head["n_seqs"], "cache_layers": head["cache_layers"],
                   "paged": head["paged"], "variant": head["mode"], "lmhead": "packed"},
        "roofline": head["roofline"],
        "attention": head["attention"],
    }
    if "cpu_baseline" in head:
        line["cpu_baseline"] = head["cpu_baseline"]
    line["headline"] = {k: v for k, v in head.items()
                        if k not in ("roofline", "attention", "cpu_baseline", "value", "unit",
                                     "ms_per_step", "workload")}
    line["configs"] = {n: results[n] for n in names[1:]}
    print(json.dumps(line), flush=True)


if __name__ == "__main__":
    main()
