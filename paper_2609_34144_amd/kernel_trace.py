"""Per-kernel duration table from a rocprofv3 kernel trace.

    rocprofv3 --kernel-trace --stats -d D -o run -- python -u bench.py --steps 10 \
        --warmup 3 --no-cpu-baseline --workload NAME
    python -m paper_2609_34144_amd.kernel_trace --workload NAME --db D/run_results.db \
        --cmd "..." --out profiles/STEM

Writes STEM.md: one row per kernel (calls, average / min / max / total duration
in microseconds), heaviest first, from the dispatch start and end timestamps in
the trace database.
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


def summarize(workload: str, db: str, cmd: str, out_stem: str) -> None:
    d = durations(db)
    rows = sorted(d.items(), key=lambda kv: -sum(kv[1]))
    with open(out_stem + ".md", "w") as fh:
        fh.write(f"# rocprofv3 kernel stats: one block step, workload {workload}\n\n")
        fh.write(f"Command (run from the repository root):\n\n```\n{cmd}\n```\n\n")
        fh.write("| kernel | calls | avg us | min us | max us | total us |\n|---|---|---|---|---|---|\n")
        for name, v in rows:
            fh.write(f"| `{_short(name)}` | {len(v)} | {sum(v) / len(v):.2f} | {min(v):.2f} | "
                     f"{max(v):.2f} | {sum(v):.1f} |\n")


def main() -> None:
    ap = argparse.ArgumentParser()
    ap.add_argument("--workload", required=True)
    ap.add_argument("--db", required=True)
    ap.add_argument("--cmd", required=True)
    ap.add_argument("--out", required=True)
    a = ap.parse_args()
    summarize(a.workload, a.db, a.cmd, a.out)


if __name__ == "__main__":
    main()
