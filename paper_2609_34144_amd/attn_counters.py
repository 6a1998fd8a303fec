"""Matrix-core counters of the routed-attention kernel from one rocprofv3 pass.

    rocprofv3 --pmc GRBM_GUI_ACTIVE SQ_VALU_MFMA_BUSY_CYCLES SQ_INSTS_VALU_MFMA_MOPS_BF16 \
        SQ_INSTS_MFMA SQ_INSTS_VALU SQ_ACTIVE_INST_VALU SQ_INSTS_VALU_TRANS_F32 \
        SQ_LDS_BANK_CONFLICT -d D -o run -- python -u bench.py --steps 5 --warmup 2 \
        --no-cpu-baseline --workload NAME
    python -m paper_2609_34144_amd.attn_counters --workload NAME --db D/run_results.db \
        --cmd "..." --out profiles/STEM

Writes STEM.md: the per-dispatch averages of the counters for the attention
kernel and what follows from them:

* MFMA busy: matrix-core busy cycles over (GUI-active cycles x SIMDs);
* the effective shader clock: GUI-active cycles per XCD over the dispatch duration;
* bf16 MFMA FLOPs issued against the algorithmic FLOPs of the routed attention
  (the excess is the masked tail of each sequence and of each routed chunk);
* VALU instructions per MFMA and transcendental instructions per MFMA.
"""
from __future__ import annotations

import argparse
import os
import sqlite3
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
KERNEL = "anchor_attn_kernel"
N_XCD = 8                  # MI355X: 8 accelerator complex dies
N_SIMD = 1024              # 256 CUs x 4 SIMDs
COUNTERS = ["GRBM_GUI_ACTIVE", "SQ_VALU_MFMA_BUSY_CYCLES", "SQ_INSTS_VALU_MFMA_MOPS_BF16",
            "SQ_INSTS_MFMA", "SQ_INSTS_VALU", "SQ_ACTIVE_INST_VALU", "SQ_INSTS_VALU_TRANS_F32",
            "SQ_LDS_BANK_CONFLICT"]


def per_dispatch(db: str) -> tuple[dict, float, int]:
    """Average over the attention dispatches of each counter summed over the chip
    (the database holds one row per XCD / shader-engine instance), the average
    duration in ns, and the dispatch count."""
    con = sqlite3.connect(db)
    rows = con.execute("select dispatch_id, counter_name, sum(counter_value), max(duration) "
                       "from pmc_events where name like ? group by dispatch_id, counter_name",
                       (f"%{KERNEL}%",)).fetchall()
    if not rows:
        raise SystemExit(f"{db}: no {KERNEL} dispatches")
    sums, durs = {}, {}
    for disp, name, v, dur in rows:
        sums.setdefault(name, []).append(v)
        durs[disp] = dur
    vals = {n: sum(x) / len(x) for n, x in sums.items()}
    return vals, sum(durs.values()) / len(durs), len(durs)


def summarize(workload: str, db: str, cmd: str, out_stem: str) -> dict:
    if ROOT not in sys.path:
        sys.path.insert(0, ROOT)
    import gen
    from bench import attn_flops
    w = gen.get(workload)
    algo = attn_flops(w, min(w.topk, w.M))
    v, dur_ns, n = per_dispatch(db)
    cyc = v["GRBM_GUI_ACTIVE"] / N_XCD
    d = {
        "dispatches": n,
        "duration_us (under counters)": dur_ns / 1e3,
        "effective clock GHz": cyc / dur_ns,
        "MFMA busy %": 100.0 * v["SQ_VALU_MFMA_BUSY_CYCLES"] / (cyc * N_SIMD),
        "bf16 MFMA GFLOP issued": v["SQ_INSTS_VALU_MFMA_MOPS_BF16"] * 512 / 1e9,
        "algorithmic GFLOP": algo / 1e9,
        "issued / algorithmic": v["SQ_INSTS_VALU_MFMA_MOPS_BF16"] * 512 / algo,
        "VALU instructions per MFMA": v["SQ_INSTS_VALU"] / v["SQ_INSTS_MFMA"],
        "transcendental per MFMA": v["SQ_INSTS_VALU_TRANS_F32"] / v["SQ_INSTS_MFMA"],
        # SQ_ACTIVE_INST_VALU counts quad-cycles
        "VALU active % (per SIMD)": 100.0 * 4.0 * v["SQ_ACTIVE_INST_VALU"] / (cyc * N_SIMD),
        "LDS bank conflicts per MFMA": v["SQ_LDS_BANK_CONFLICT"] / v["SQ_INSTS_MFMA"],
    }
    with open(out_stem + ".md", "w") as fh:
        fh.write(f"# Matrix-core counters of the routed attention, {workload}\n\n")
        fh.write("One rocprofv3 counter pass over bench.py; averages per dispatch of "
                 f"`{KERNEL}` (counters summed over the chip).\n\nCommand:\n\n```\n{cmd}\n```\n\n")
        fh.write("| counter | per dispatch |\n|---|---|\n")
        for c in COUNTERS:
            fh.write(f"| `{c}` | {v.get(c, float('nan')):.4g} |\n")
        fh.write("\n| derived | value |\n|---|---|\n")
        for k, x in d.items():
            fh.write(f"| {k} | {x:.4g} |\n")
        fh.write(f"\nMFMA busy = SQ_VALU_MFMA_BUSY_CYCLES / (GRBM_GUI_ACTIVE / {N_XCD} x {N_SIMD} SIMDs); "
                 f"VALU active = 4 SQ_ACTIVE_INST_VALU (quad-cycles) / (GRBM_GUI_ACTIVE / {N_XCD} x {N_SIMD}); "
                 f"clock = GRBM_GUI_ACTIVE / {N_XCD} / duration; issued FLOPs = "
                 "SQ_INSTS_VALU_MFMA_MOPS_BF16 x 512.\n")
    return d


def main() -> None:
    ap = argparse.ArgumentParser()
    ap.add_argument("--workload", required=True)
    ap.add_argument("--db", required=True)
    ap.add_argument("--cmd", required=True)
    ap.add_argument("--out", required=True)
    a = ap.parse_args()
    for k, x in summarize(a.workload, a.db, a.cmd, a.out).items():
        print(f"{k}: {x:.4g}")


if __name__ == "__main__":
    main()
