"""HBM traffic of the hot-path kernels from rocprofv3 counters.

Two counter passes over the same program (FETCH_SIZE, then WRITE_SIZE: one
pass cannot hold both), each also timing a plain device copy of known size so
the counters can be scaled to bytes:

    python -m paper_2609_34144_amd.hbm_traffic run --workload NAME
        (the program, run under rocprofv3 --pmc FETCH_SIZE, then --pmc WRITE_SIZE)
    python -m paper_2609_34144_amd.hbm_traffic summarize --workload NAME \
        --fetch FETCH_DB --write WRITE_DB --cmd "..." --out profiles/STEM

`summarize` writes STEM.md (a short table) and STEM.json, which bench.py reads
for the `traffic` field of its roofline object.  The JSON records a hash of the
kernel sources; bench.py reports null when the sources have changed since.
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import re
import sqlite3
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
COPY_BYTES = 1 << 29          # 512 MiB fp32 copy: larger than the Infinity Cache
COPY_KERNEL = "__amd_rocclr_copyBuffer"   # the HIP runtime's device-to-device copy
CALIB_REPS = 3
KERNEL_SOURCES = {
    "route": ["route_kv.hip"],
    "attn": ["anchor_attn.hip"],
    "par": ["par.hip", "par_device.h", "par_fused.hip", "fft_tile.h"],
}


def sources_hash(part: str) -> str:
    """Hash of the sources that define the part's kernels (the shared header holds
    only declarations and constants and is left out)."""
    h = hashlib.sha256()
    for f in KERNEL_SOURCES[part]:
        with open(os.path.join(HERE, "csrc", f), "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()[:16]


def part_of(kernel: str) -> str | None:
    if "route_" in kernel:
        return "route"
    if "anchor_attn" in kernel or "attn_merge" in kernel:
        return "attn"
    if "par_" in kernel:
        return "par"
    return None


def run(workload: str, reps: int = CALIB_REPS) -> None:
    if ROOT not in sys.path:
        sys.path.insert(0, ROOT)
    import torch

    import gen
    import paper_2609_34144_amd as cast

    cast.load()
    dev = torch.device("cuda:0")
    # calibration: a plain copy of known size (read COPY_BYTES, write COPY_BYTES)
    x = torch.ones(COPY_BYTES // 4, dtype=torch.float32, device=dev)
    y = torch.empty_like(x)
    for _ in range(reps):
        y.copy_(x)
    torch.cuda.synchronize()
    del x, y
    w = gen.get(workload)
    prm = cast.cast_par_params_default(accumulate=1)
    resid_np, _, _ = gen.par_inputs(w, seed=42)
    resid = torch.from_numpy(resid_np).to(dev)
    out = torch.randn(resid.shape, device=dev)
    if w.has_attention:
        q, k, v, _, _ = gen.attn_inputs(w, seed=42, device=dev)
    for _ in range(reps):
        if w.has_attention:
            idx, ke, _ = cast.cast_route_kv(q, k, w.topk, w.scale)
            cast.cast_anchor_attn(q, k, v, idx, ke, w.scale)
        if w.has_par:
            cast.cast_par_reconstruct(resid, w.anchors, prm, out=out)
        torch.cuda.synchronize()
    print("hbm_traffic run done", flush=True)


def _per_kernel(db: str, counter: str) -> dict:
    con = sqlite3.connect(db)
    rows = con.execute("select name, avg(counter_value), count(*) from pmc_events "
                       "where counter_name = ? group by name", (counter,)).fetchall()
    return {n: (v, c) for n, v, c in rows}


def _short(n: str) -> str:
    n = re.sub(r"\((cast::|float|unsigned|at::).*", "", n)
    return n.replace("void ", "").replace("cast::(anonymous namespace)::", "").replace(
        "cast::pardev::", "")


def _calibration(db: str, counter: str, reps: int = CALIB_REPS) -> float:
    """Mean reading of the calibration copies: the first `reps` dispatches of the
    runtime's device-to-device copy kernel (run() issues them before anything else;
    other kernels with "copy" in their name, such as dtype conversions, are not it)."""
    con = sqlite3.connect(db)
    rows = con.execute("select dispatch_id, counter_value from pmc_events where name = ? and "
                       "counter_name = ? order by dispatch_id", (COPY_KERNEL, counter)).fetchall()
    if len(rows) < reps:
        raise SystemExit(f"{db}: expected {reps} calibration copies ({COPY_KERNEL}), "
                         f"found {len(rows)}")
    vals = [v for _, v in rows[:reps]]
    if max(vals) > 1.01 * min(vals):
        raise SystemExit(f"{db}: calibration copies disagree: {vals}")
    return sum(vals) / len(vals)


def summarize(workload: str, fetch_db: str, write_db: str, cmd: str, out_stem: str) -> None:
    fetch = _per_kernel(fetch_db, "FETCH_SIZE")
    write = _per_kernel(write_db, "WRITE_SIZE")
    kib = COPY_BYTES / 1024.0
    copy_f = _calibration(fetch_db, "FETCH_SIZE")
    copy_w = _calibration(write_db, "WRITE_SIZE")
    f_scale = kib / copy_f           # bytes-per-KiB-reading scale: 1.0 when the counter is exact
    w_scale = kib / copy_w
    kernels = {}
    for n in sorted(set(fetch) | set(write)):
        part = part_of(n)
        if part is None or n == COPY_KERNEL:
            continue
        fb = fetch.get(n, (0.0, 0))[0] * f_scale * 1024.0
        wb = write.get(n, (0.0, 0))[0] * w_scale * 1024.0
        kernels[_short(n)] = {"part": part, "fetch_bytes": fb, "write_bytes": wb,
                              "bytes": fb + wb, "dispatches": fetch.get(n, (0, 0))[1]}
    parts = {}
    for k, v in kernels.items():
        p = parts.setdefault(v["part"], {"fetch_bytes": 0.0, "write_bytes": 0.0, "bytes": 0.0})
        for key in ("fetch_bytes", "write_bytes", "bytes"):
            p[key] += v[key]
    doc = {"workload": workload, "copy_bytes": COPY_BYTES,
           "copy_counter_kib": {"FETCH_SIZE": copy_f, "WRITE_SIZE": copy_w},
           "scale": {"FETCH_SIZE": f_scale, "WRITE_SIZE": w_scale},
           "sources": {p: sources_hash(p) for p in KERNEL_SOURCES},
           "kernels": kernels, "per_call_bytes": parts, "command": cmd}
    with open(out_stem + ".json", "w") as fh:
        json.dump(doc, fh, indent=1)
    with open(out_stem + ".md", "w") as fh:
        fh.write(f"# HBM traffic per dispatch, {workload}\n\n")
        fh.write("rocprofv3 counters FETCH_SIZE and WRITE_SIZE (KiB per dispatch), one pass each, "
                 "scaled by the reading for a plain 512 MiB device copy in the same program "
                 f"(FETCH x{f_scale:.4f}, WRITE x{w_scale:.4f}).\n\nCommand:\n\n```\n{cmd}\n```\n\n")
        fh.write("| kernel | fetch MB | write MB | total MB |\n|---|---|---|---|\n")
        for k, v in kernels.items():
            fh.write(f"| `{k}` | {v['fetch_bytes'] / 1e6:.2f} | {v['write_bytes'] / 1e6:.2f} | "
                     f"{v['bytes'] / 1e6:.2f} |\n")
    print(json.dumps(parts))


def main() -> None:
    ap = argparse.ArgumentParser()
    sub = ap.add_subparsers(dest="mode", required=True)
    r = sub.add_parser("run")
    r.add_argument("--workload", required=True)
    s = sub.add_parser("summarize")
    s.add_argument("--workload", required=True)
    s.add_argument("--fetch", required=True)
    s.add_argument("--write", required=True)
    s.add_argument("--cmd", required=True)
    s.add_argument("--out", required=True)
    a = ap.parse_args()
    if a.mode == "run":
        run(a.workload)
    else:
        summarize(a.workload, a.fetch, a.write, a.cmd, a.out)


if __name__ == "__main__":
    main()
