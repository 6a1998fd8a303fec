"""Per-kernel duration table from a rocprofv3 kernel trace.

    rocprofv3 --kernel-trace --stats -d D -o run -- python -u bench.py --steps 10 \
        --warmup 3 --no-cpu-baseline --workload NAME
    python -m paper_2609_34144_amd.kernel_trace --workload NAME --db D/run_results.db \
        --cmd "..." --out profiles/STEM

Writes STEM.md: one row per kernel (calls, average / min / max / total duration
in microseconds), heaviest first, from the dispatch start and end timestamps in
the trace database; with --bench-log, also the traced bench.py run's per-call
times beside the sums of each call's kernel averages.
"""
from __future__ import annotations

import argparse
import collections
import sqlite3


def durations(db: str) -> dict:
    """Kernel name -> list of dispatch durations in microseconds."""
    con = sqlite3.connect(db)
    out = collections.defaultdict(list)
    for name, start, end in con.execute("select name, start, end from kernels"):
        out[name].append((end - start) / 1000.0)
    return out


def _short(name: str) -> str:
    name = name.replace("void ", "").replace("(anonymous namespace)::", "")
    cut = name.find("(")
    return name[:cut] if cut > 0 else name


def _bench_line(log: str) -> dict | None:
    """The JSON line bench.py printed in the traced run (None if absent)."""
    import json
    with open(log) as fh:
        for line in fh:
            if line.startswith('{"metric"'):
                return json.loads(line)
    return None


def summarize(workload: str, db: str, cmd: str, out_stem: str, bench_log: str | None = None) -> None:
    d = durations(db)
    rows = sorted(d.items(), key=lambda kv: -sum(kv[1]))
    avg = {_short(n): sum(v) / len(v) for n, v in d.items()}
    with open(out_stem + ".md", "w") as fh:
        fh.write(f"# rocprofv3 kernel stats: one block step, workload {workload}\n\n")
        fh.write(f"Command (run from the repository root):\n\n```\n{cmd}\n```\n\n")
        fh.write("| kernel | calls | avg us | min us | max us | total us |\n|---|---|---|---|---|---|\n")
        for name, v in rows:
            fh.write(f"| `{_short(name)}` | {len(v)} | {sum(v) / len(v):.2f} | {min(v):.2f} | "
                     f"{max(v):.2f} | {sum(v):.1f} |\n")
        b = _bench_line(bench_log) if bench_log else None
        if b:
            # each call's kernels, summed from the trace averages, beside the call's
            # average duration that bench.py timed with HIP events in the same run
            parts = {"route": ("route_",), "attn": ("anchor_attn", "attn_merge"), "par": ("par_",)}
            fh.write("\nThe same run's bench.py line: per-call averages (HIP events over back-to-back "
                     "calls of one kind) against the sum of that call's kernel averages above.\n\n")
            fh.write("| call | bench.py ms | trace kernels ms |\n|---|---|---|\n")
            for call, keys in parts.items():
                ms = b["per_call_ms"].get(call)
                if not ms:
                    continue
                tr = sum(v for k, v in avg.items() if any(x in k for x in keys)) / 1e3
                fh.write(f"| {call} | {ms:.4f} | {tr:.4f} |\n")
            r = b.get("roofline", {})
            fh.write(f"\nbench.py roofline: {r.get('kernel')} {r.get('achieved', 0):.1f} {r.get('unit')} "
                     f"= {r.get('frac', 0):.4f} of {r.get('peak')}; step {b['ms_per_step']:.4f} ms, "
                     f"{b['value']:.4g} {b['unit']}.\n")


def main() -> None:
    ap = argparse.ArgumentParser()
    ap.add_argument("--workload", required=True)
    ap.add_argument("--db", required=True)
    ap.add_argument("--cmd", required=True)
    ap.add_argument("--out", required=True)
    ap.add_argument("--bench-log", default=None,
                    help="output of the traced bench.py run, for its per-call times")
    a = ap.parse_args()
    summarize(a.workload, a.db, a.cmd, a.out, a.bench_log)


if __name__ == "__main__":
    main()
