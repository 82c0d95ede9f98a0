"""Turn two rocprofv3 counter runs of `bench.py --pmc-driver` into HBM bytes per LM-head launch.

    rocprofv3 --pmc FETCH_SIZE -d <dir_fetch> -o run --output-format csv -- python bench.py --config C5 --pmc-driver
    rocprofv3 --pmc WRITE_SIZE -d <dir_write> -o run --output-format csv -- python bench.py --config C5 --pmc-driver
    python -m paper_2607_27600_amd.pmc_summary <dir_fetch> <dir_write> profiles/lmhead_c5_traffic.json C5

A third mode tabulates matrix-core utilisation per kernel from one run with the SQ/GRBM
counters named in util():

    python -m paper_2607_27600_amd.pmc_summary util <dir>

A fourth merges several counter passes of the same command (dispatch ids line up) into
issue statistics per kernel: see issue().

    python -m paper_2607_27600_amd.pmc_summary issue <dir1> <dir2> ...

FETCH_SIZE / WRITE_SIZE are in KiB per dispatch.  The driver also copies 1 GiB device to
device; each counter is scaled by (1 GiB / what it reads for that copy), so the figures are
calibrated against a transfer of known size.  The record carries the sha256 of gemm.hip;
bench.py reports the traffic only while the source matches.
"""
from __future__ import annotations

import csv
import hashlib
import json
import os
import sys

GIB_KIB = 1 << 20


def _per_dispatch(path: str, counter: str) -> list:
    out = {}
    with open(path) as f:
        for r in csv.DictReader(f):
            if r["Counter_Name"] != counter:
                continue
            key = r["Dispatch_Id"]
            out.setdefault(key, [r["Kernel_Name"], 0.0])
            out[key][1] += float(r["Counter_Value"])
    return list(out.values())


def _find(rows, pred):
    hits = [v for name, v in rows if pred(name)]
    if not hits:
        raise SystemExit("kernel not found in counter file")
    return hits


def main(fetch_dir: str, write_dir: str, out: str, cfg_name: str = "C5") -> None:
    f_rows = _per_dispatch(os.path.join(fetch_dir, "run_counter_collection.csv"), "FETCH_SIZE")
    w_rows = _per_dispatch(os.path.join(write_dir, "run_counter_collection.csv"), "WRITE_SIZE")
    is_lm = lambda n: "gemm_lmhead_packed" in n
    is_copy = lambda n: "copy" in n.lower() and "gemm" not in n and "compact" not in n
    # the copy is the last dispatch of the driver; take the largest copy-like dispatch
    f_copy = max(_find(f_rows, is_copy))
    w_copy = max(_find(w_rows, is_copy))
    f_lm = _find(f_rows, is_lm)[-1]
    w_lm = _find(w_rows, is_lm)[-1]
    kf, kw = GIB_KIB / f_copy, GIB_KIB / w_copy
    here = os.path.dirname(os.path.abspath(__file__))
    with open(os.path.join(here, "csrc", "gemm.hip"), "rb") as fh:
        digest = hashlib.sha256(fh.read()).hexdigest()
    sys.path.insert(0, os.path.dirname(here))
    from synth import configs as C
    cfg = C.CONFIGS[cfg_name]
    N, D, V = cfg.n_tokens, cfg.hidden, cfg.vocab
    vt = (V + 255) // 256
    alg = 2 * V * D + 2 * N * D + 8 * vt * N + 4 * N
    rec = {
        "kernel": f"gemm_lmhead_packed<EpiLse16> (LM head on packed operands + fused "
                  f"log-sum-exp and target gather), {cfg_name} shapes",
        "fetch_kib_raw": f_lm, "write_kib_raw": w_lm,
        "copy_fetch_kib_raw": f_copy, "copy_write_kib_raw": w_copy,
        "fetch_scale": kf, "write_scale": kw,
        "bytes_per_launch": (f_lm * kf + w_lm * kw) * 1024.0,
        "algorithmic_bytes": alg,
        "algorithmic_bytes_note": f"W_lm {V}x{D} bf16 + U {N}x{D} bf16 read (both packed) + "
                                  f"partials {vt}x{N}x8 B and target logits {N}x4 B written",
        "traffic_over_algorithmic": (f_lm * kf + w_lm * kw) * 1024.0 / alg,
        "gemm_source_sha256": digest,
    }
    with open(out, "w") as fh:
        json.dump(rec, fh, indent=1)
    print(json.dumps(rec, indent=1))


def _all_counters(path: str) -> list:
    """Per dispatch: (id, kernel name, {counter: value summed over instances})."""
    out = {}
    with open(path) as f:
        for r in csv.DictReader(f):
            k = int(r["Dispatch_Id"])
            name, vals = out.setdefault(k, (r["Kernel_Name"], {}))
            vals[r["Counter_Name"]] = vals.get(r["Counter_Name"], 0.0) + float(r["Counter_Value"])
    return [(k, *out[k]) for k in sorted(out)]


def util(run_dir: str, n_xcc: int = 8, n_simd: int = 1024, n_cu: int = 256) -> None:
    """Matrix-core utilisation per kernel from a run with SQ_VALU_MFMA_BUSY_CYCLES,
    SQ_INSTS_VALU_MFMA_MOPS_BF16 and GRBM_GUI_ACTIVE.

    GRBM_GUI_ACTIVE sums the eight XCDs' own clocks, so the kernel's cycle count is the sum
    over n_xcc; SQ_VALU_MFMA_BUSY_CYCLES sums busy cycles over every SIMD; each MOPS unit is
    512 FLOP.  Utilisation = busy / (cycles x SIMDs).  SQ_LDS_BANK_CONFLICT counts cycles in
    which a CU's LDS stalls on bank conflicts, reported per CU-cycle as rocprof's own
    LDSBankConflict metric does.
    """
    rows = _all_counters(os.path.join(run_dir, "run_counter_collection.csv"))
    print("| dispatch | kernel | cycles | MFMA FLOP | MFMA busy | VALU active / wave-cycle | LDS bank-conflict stall / CU-cycle |")
    print("|---|---|---|---|---|---|---|")
    for k, name, c in rows:
        busy = c.get("SQ_VALU_MFMA_BUSY_CYCLES", 0.0)
        if busy == 0.0:
            continue
        cyc = c["GRBM_GUI_ACTIVE"] / n_xcc
        short = name.replace("cc::(anonymous namespace)::", "").replace("void ", "").split("(")[0]
        valu = c.get("SQ_ACTIVE_INST_VALU", 0.0) / max(c.get("SQ_WAVE_CYCLES", 1.0), 1.0)
        lds = c.get("SQ_LDS_BANK_CONFLICT", 0.0) / (cyc * n_cu)
        print(f"| {k} | `{short}` | {cyc:.4g} | {c.get('SQ_INSTS_VALU_MFMA_MOPS_BF16', 0.0) * 512:.4g} "
              f"| {100 * busy / (cyc * n_simd):.1f}% | {valu:.2f} | {100 * lds:.1f}% |")


def issue(run_dirs: list, n_xcc: int = 8, n_simd: int = 1024, match: str = "") -> None:
    """Per kernel, from passes holding (between them) SQ_WAVE_CYCLES, SQ_WAIT_ANY,
    SQ_WAIT_INST_ANY, SQ_ACTIVE_INST_VALU, SQ_VALU_MFMA_BUSY_CYCLES,
    SQ_VALU_MFMA_COEXEC_CYCLES, SQ_INSTS_{MFMA,VALU,SALU,LDS} and GRBM_GUI_ACTIVE.

    SQ_WAVE_CYCLES, SQ_WAIT_ANY and SQ_WAIT_INST_ANY count quad-cycles, so their ratios are
    fractions of the waves' resident time.  MFMA busy is per SIMD-cycle of the kernel;
    co-issue is the share of matrix-busy cycles in which another VALU instruction issued.
    Instruction counts are per MFMA instruction (SQ_INSTS_VALU includes the MFMAs).
    """
    merged = {}
    for d in run_dirs:
        for k, name, c in _all_counters(os.path.join(d, "run_counter_collection.csv")):
            m = merged.setdefault(k, [name, {}])
            for key, v in c.items():
                if key == "GRBM_GUI_ACTIVE" and key in m[1]:
                    continue
                m[1][key] = v
    print("| dispatch | kernel | cycles | MFMA busy | co-issue | waiting on anything | waiting to issue "
          "| VALU / MFMA | SALU / MFMA | LDS / MFMA |")
    print("|---|---|---|---|---|---|---|---|---|---|")
    for k in sorted(merged):
        name, c = merged[k]
        mf = c.get("SQ_INSTS_MFMA", 0.0)
        if mf == 0.0 or (match and match not in name):
            continue
        cyc = c["GRBM_GUI_ACTIVE"] / n_xcc
        wc = max(c.get("SQ_WAVE_CYCLES", 1.0), 1.0)
        busy = c.get("SQ_VALU_MFMA_BUSY_CYCLES", 0.0)
        short = name.replace("cc::(anonymous namespace)::", "").replace("void ", "").split("(")[0]
        print(f"| {k} | `{short}` | {cyc:.4g} | {100 * busy / (cyc * n_simd):.1f}% "
              f"| {100 * c.get('SQ_VALU_MFMA_COEXEC_CYCLES', 0.0) / max(busy, 1.0):.0f}% "
              f"| {100 * c.get('SQ_WAIT_ANY', 0.0) / wc:.0f}% | {100 * c.get('SQ_WAIT_INST_ANY', 0.0) / wc:.0f}% "
              f"| {(c.get('SQ_INSTS_VALU', 0.0) - mf) / mf:.2f} | {c.get('SQ_INSTS_SALU', 0.0) / mf:.2f} "
              f"| {c.get('SQ_INSTS_LDS', 0.0) / mf:.2f} |")


if __name__ == "__main__":
    if sys.argv[1] == "util":
        util(sys.argv[2])
    elif sys.argv[1] == "issue":
        issue(sys.argv[2:])
    else:
        main(*sys.argv[1:5])
