"""Benchmark of one CAST block step on one MI355X.

A step is the whole hot path on one batch of synthetic input, stream-ordered on
torch's current stream:  cast_route_kv -> cast_anchor_attn -> cast_par_reconstruct
(accumulate mode, X_t += R_hat_t).  Inputs are resident in HBM before timing;
the step cycles over several copies of its inputs so that consecutive steps do
not find their inputs in the Infinity Cache.  The timed steps are launched eagerly
(--graph: replayed from one captured HIP graph per input copy); then each call is
timed alone, K launches back to back between one pair of events.

Prints ONE JSON line.  `value` = frame-tokens/s = N_cur * S / step time.
`roofline` describes the dominant call (routed attention: bf16 MFMA; PAR on a
workload without attention); the per-call figures for routing and PAR are
reported beside it.  `cpu_baseline` times the float64 oracle on a bounded sample
of the same workload on this host.  The default workload is the HY-World-like
block, the largest one that runs all three calls.

    python bench.py [--gpus 1] [--steps K] [--warmup W] [--workload NAME] [--step-only]
"""
from __future__ import annotations

import argparse
import json
import math
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

PEAK_BF16_TFLOPS = 2500.0      # MI355X dense bf16 MFMA
PEAK_HBM_GBS = 8000.0          # MI355X HBM3E
N_COPIES = 4                   # input copies cycled through (> Infinity Cache)


def attn_flops(w, k_eff):
    """Useful FLOPs of routed attention: 4 S (n0 + K Bv) dh per (anchor, head)."""
    return 4.0 * w.S * (w.n0 + k_eff * w.Bv) * w.dh * w.H * w.n_a


def route_bytes(w):
    """Algorithmic bytes of routing: one read of K history and of the anchor Q (bf16)."""
    return 2.0 * (w.M * w.Bv + w.n_a * w.S) * w.H * w.dh


def coupled_route_bytes(w):
    """Algorithmic bytes of coupled routing: one read of K and V history and of the
    anchor Q (bf16); the solver's own traffic is negligible."""
    return 2.0 * (2 * w.M * w.Bv + w.n_a * w.S) * w.H * w.dh


def par_bytes(w, accumulate=True):
    """Algorithmic bytes of PAR: anchors read once; skipped frames written, and read
    too when accumulating (fp32)."""
    frame = 4.0 * w.S * w.D
    n_skip = w.n_frames - w.n_a
    return frame * (w.n_a + n_skip * (2 if accumulate else 1))


def block_update_bytes(w):
    """Algorithmic bytes of one residual site's whole block update (PAR with the
    anchor case of eq:block fused in): anchors read once, then X read and written
    for every current frame (fp32)."""
    frame = 4.0 * w.S * w.D
    return frame * (w.n_a + 2 * w.n_frames)


def frame_select_bytes(w):
    """Algorithmic bytes of frame selection: one read of both control branches'
    bf16 updates of every current frame."""
    return 2.0 * 2.0 * w.n_frames * w.S * w.D


def load_traffic(workload):
    """HBM bytes per call (route / attn / par) from the committed counter summary
    profiles/hbm_traffic_<workload>.json (written by paper_2609_34144_amd.hbm_traffic
    from rocprofv3 FETCH_SIZE / WRITE_SIZE passes); a part whose kernel sources
    changed since the counters were taken is left out (reported as null)."""
    path = os.path.join(ROOT, "profiles", f"hbm_traffic_{workload}.json")
    if not os.path.exists(path):
        return {}
    from paper_2609_34144_amd.hbm_traffic import sources_hash
    with open(path) as fh:
        doc = json.load(fh)
    out = {}
    for part, v in doc.get("per_call_bytes", {}).items():
        if doc.get("sources", {}).get(part) == sources_hash(part):
            out[part] = v["bytes"]
    return out


def cpu_baseline(w, seed=42, attn_seconds=10.0, par_targets=16):
    """The oracle as it stands, timed on this host on a bounded sample of the
    workload: full routing, as many of the n_a*H (anchor, head) attention pairs
    as fit in about `attn_seconds` (scaled by the pair count), and PAR statistics of every anchor pair plus
    the reconstruction of up to `par_targets` skipped frames (scaled by the
    skipped-frame count)."""
    import numpy as np
    import torch
    import gen
    from oracle import attn as OA
    from oracle import par as OP
    from oracle import route as OR
    try:
        from threadpoolctl import threadpool_info
        threads = max([i.get("num_threads", 1) for i in threadpool_info()] + [1])
    except Exception:
        threads = 1
    cores = len(os.sched_getaffinity(0))
    t_route = t_attn = t_par = 0.0
    pairs = []
    if w.has_attention and w.M > 0:
        q, k, v, _, _ = gen.attn_inputs(w, seed=seed, device="cpu")
        qn, kn, vn = (t.float().numpy().astype(np.float64) for t in (q, k, v))
        del q, k, v
        t0 = time.perf_counter()
        _, idx, k_eff = OR.route(qn, kn, w.topk, w.scale, decide_dtype=np.float32)
        t_route = time.perf_counter() - t0
        # (anchor, head) pairs one at a time until `attn_seconds` have passed
        all_pairs = [(i, h) for i in range(w.n_a) for h in range(w.H)]
        t0 = time.perf_counter()
        for (i, h) in all_pairs:
            OA.anchor_attention(qn, kn, vn, idx, w.scale, rows=[(i, h, s) for s in range(w.S)])
            pairs.append((i, h))
            if time.perf_counter() - t0 >= attn_seconds:
                break
        t_attn = (time.perf_counter() - t0) * len(all_pairs) / len(pairs)
        del qn, kn, vn
    n_tgt = 0
    comp = []
    if w.has_par:
        # statistics of every anchor pair, then R_hat_t of up to `par_targets`
        # skipped frames added to X_t, scaled to all of them
        resid, x0, _ = gen.par_inputs(w, seed=seed)
        prm = OP.ParParams(accumulate=True)
        comp = OP.composition(w.anchors, w.n_frames)
        sample = comp[:par_targets]
        n_tgt = len(sample)
        t0 = time.perf_counter()
        stats = OP.par_stats(resid, w.anchors, prm)
        t_stats = time.perf_counter() - t0
        t0 = time.perf_counter()
        for (t, a, b, alpha) in sample:
            r = OP.reconstruct_frame(stats[(a, b)], alpha, w.Hg, w.Wg, w.D)
            if x0 is not None:
                r += x0[t]
        t_tgt = time.perf_counter() - t0
        t_par = t_stats + t_tgt * len(comp) / max(n_tgt, 1)
        del resid, x0
    total = t_route + t_attn + t_par
    return {
        "value": w.frame_tokens / total, "unit": "frame-tokens/s", "cores": max(threads, 1),
        "host_cores_visible": cores, "kind": "oracle",
        "sample": (f"{w.name}: "
                   + (f"full routing ({t_route:.2f} s), attention on {len(pairs)} of "
                      f"{w.n_a * w.H} (anchor, head) pairs scaled x{w.n_a * w.H / len(pairs):.2f} "
                      f"({t_attn:.2f} s extrapolated)" if pairs else "no routing / attention")
                   + (f", PAR accumulate: statistics of every pair and {n_tgt} of {len(comp)} "
                      f"skipped frames, scaled ({t_par:.2f} s)" if w.has_par else ", PAR bypassed")
                   + f"; float64 numpy, BLAS threads {threads}"),
        "seconds": {"route": t_route, "attn_extrapolated": t_attn, "par": t_par},
    }


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--workload", default="hy_world_like_16f44x80_d3072")
    ap.add_argument("--seed", type=int, default=42)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--step-only", action="store_true",
                    help="time the block step and its calls only (no coupled routing, block "
                         "update, frame selection or diagnostics), e.g. under a kernel trace")
    ap.add_argument("--graph", action="store_true",
                    help="replay the timed steps as captured HIP graphs instead of launching them")
    args = ap.parse_args()
    if args.gpus != 1:
        print(f"bench.py measures one MI355X only (got --gpus {args.gpus}); the hot path is "
              f"built and measured on one GPU, multi-GPU sharding is not part of it.",
              file=sys.stderr)
        sys.exit(2)

    import numpy as np
    import torch

    import gen
    import paper_2609_34144_amd as cast

    w = gen.get(args.workload)
    cast.load()
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    stream = torch.cuda.current_stream()

    # ---- inputs (resident in HBM), N_COPIES copies at distinct addresses.  The
    # attention inputs of copy c come from seed SEEDS[c] (the base seed, then the
    # timing repeats 0, 1, 2), so the steps cycle over different routings; PAR's
    # work does not depend on the values, and its copies are clones of one draw.
    seeds = [args.seed] + [s for s in (0, 1, 2) if s != args.seed][:N_COPIES - 1]
    resid_np, _, _ = gen.par_inputs(w, seed=args.seed)
    resid = torch.from_numpy(resid_np).to(dev)
    del resid_np
    sets = []
    for c in range(N_COPIES):
        s = {"resid": resid.clone(), "x": torch.randn(resid.shape, device=dev, dtype=torch.float32)}
        if w.has_attention:
            q, k, v, _, _ = gen.attn_inputs(w, seed=seeds[c % len(seeds)], device=dev)
            s.update(q=q, k=k, v=v)
            del q, k, v
        sets.append(s)
    del resid
    prm = cast.cast_par_params_default(accumulate=1)
    k_eff = min(w.topk, w.M) if w.has_attention else 0
    route_ws = par_ws = attn_ws = None
    if w.has_attention and w.M > 0:
        nb = cast.cast_route_kv_workspace_bytes(w.n_a, w.S, w.H, w.dh, w.M, w.Bv)
        route_ws = torch.empty(nb, dtype=torch.uint8, device=dev)
        nb = cast.cast_anchor_attn_workspace_bytes(w.n_a, w.S, w.H, w.dh, k_eff, 0, w.Bv)
        if nb > 0:
            attn_ws = torch.empty(nb, dtype=torch.uint8, device=dev)
    if w.has_par:
        nb = cast.cast_par_workspace_bytes(w.n_frames, w.n_a, w.Hg, w.Wg, w.D, prm)
        par_ws = torch.empty(max(nb, 1), dtype=torch.uint8, device=dev)
    idx = torch.empty((w.n_a, w.H, max(k_eff, 1)), dtype=torch.int32, device=dev)
    attn_out = torch.empty((w.n_a, w.S, w.H, w.dh), dtype=torch.bfloat16, device=dev) \
        if w.has_attention else None

    ev = lambda: torch.cuda.Event(enable_timing=True)

    def step(s):
        # launched on the current stream (torch's stream, or the capture stream
        # while a graph is captured)
        st = torch.cuda.current_stream()
        if w.has_attention:
            _, ke, _ = cast.cast_route_kv(s["q"], s["k"], w.topk, w.scale, idx_out=idx,
                                          workspace=route_ws, stream=st)
            cast.cast_anchor_attn(s["q"], s["k"], s["v"], idx, ke, w.scale, out=attn_out,
                                  workspace=attn_ws, stream=st)
        if w.has_par:
            cast.cast_par_reconstruct(s["resid"], w.anchors, prm, out=s["x"], workspace=par_ws,
                                      stream=st)

    for i in range(args.warmup):
        step(sets[i % N_COPIES])
    torch.cuda.synchronize()

    # --graph: the step of each input copy captured once as a HIP graph (the
    # library allocates nothing and issues no memsets, so a step replays as
    # captured) and the timed loop replays them.  Measured on MI355X this is no
    # faster than launching the seven kernels eagerly (0.301 against 0.294 ms per
    # step on the 8-frame 30x52 workload), so eager launches are the default.
    graphs = []
    if args.graph:
        for c in range(N_COPIES):
            g = torch.cuda.CUDAGraph()
            with torch.cuda.graph(g):
                step(sets[c])
            graphs.append(g)
        for g in graphs:
            g.replay()
        torch.cuda.synchronize()

    # the timed steps: nothing but the steps between the two events
    t_start, t_end = ev(), ev()
    torch.cuda.synchronize()
    t_start.record(stream)
    for i in range(args.steps):
        if graphs:
            graphs[i % N_COPIES].replay()
        else:
            step(sets[i % N_COPIES])
    t_end.record(stream)
    torch.cuda.synchronize()
    ms_total = t_start.elapsed_time(t_end)
    ms_step = ms_total / args.steps
    # the per-call breakdown: each call launched alone `steps` times back to back
    # (cycling over the input copies) between one pair of events on its stream, so
    # a call's average is its kernels' duration plus the launch gaps between them,
    # as a kernel trace sees it; the route indices for attention come from a
    # routing pass per copy before its loop
    def timed_loop(fn):
        a, b = ev(), ev()
        torch.cuda.synchronize()
        a.record(stream)
        for i in range(args.steps):
            fn(sets[i % N_COPIES])
        b.record(stream)
        torch.cuda.synchronize()
        return a.elapsed_time(b) / args.steps

    # the spread: every step (and below, every call) once more, each between its
    # own pair of events; the headline stays the bracketed loop above
    def each_timed(fn, n):
        evs = [(ev(), ev()) for _ in range(n)]
        torch.cuda.synchronize()
        for i, (a, b) in enumerate(evs):
            a.record(stream)
            fn(i)
            b.record(stream)
        torch.cuda.synchronize()
        return [a.elapsed_time(b) for (a, b) in evs]

    step_each = each_timed(lambda i: (graphs[i % N_COPIES].replay() if graphs
                                      else step(sets[i % N_COPIES])), args.steps)

    per_call = {}
    route_ms = attn_ms = 0.0
    if w.has_attention:
        route_ms = timed_loop(lambda s: cast.cast_route_kv(s["q"], s["k"], w.topk, w.scale,
                                                           idx_out=idx, workspace=route_ws,
                                                           stream=stream))
        idx_c = []
        for c in range(N_COPIES):
            ic = torch.empty_like(idx)
            cast.cast_route_kv(sets[c]["q"], sets[c]["k"], w.topk, w.scale, idx_out=ic,
                               workspace=route_ws, stream=stream)
            sets[c]["idx"] = ic
        attn_ms = timed_loop(lambda s: cast.cast_anchor_attn(s["q"], s["k"], s["v"], s["idx"],
                                                             k_eff, w.scale, out=attn_out,
                                                             workspace=attn_ws, stream=stream))
    par_ms = timed_loop(lambda s: cast.cast_par_reconstruct(
        s["resid"], w.anchors, prm, out=s["x"], workspace=par_ws, stream=stream)) if w.has_par else 0.0
    per_call.update(route=route_ms, attn=attn_ms, par=par_ms)
    call_median = {}
    if w.has_attention:
        call_median["route"] = float(np.median(each_timed(lambda i: cast.cast_route_kv(
            sets[i % N_COPIES]["q"], sets[i % N_COPIES]["k"], w.topk, w.scale, idx_out=idx,
            workspace=route_ws, stream=stream), args.steps)))
        call_median["attn"] = float(np.median(each_timed(lambda i: cast.cast_anchor_attn(
            sets[i % N_COPIES]["q"], sets[i % N_COPIES]["k"], sets[i % N_COPIES]["v"],
            sets[i % N_COPIES]["idx"], k_eff, w.scale, out=attn_out, workspace=attn_ws,
            stream=stream), args.steps)))
    if w.has_par:
        call_median["par"] = float(np.median(each_timed(lambda i: cast.cast_par_reconstruct(
            sets[i % N_COPIES]["resid"], w.anchors, prm, out=sets[i % N_COPIES]["x"],
            workspace=par_ws, stream=stream), args.steps)))

    # reconstruction-coupled routing (NEXT-1), timed on its own after the step;
    # the W_O Gram matrices depend on weights only and are prepared once, untimed
    coupled_ms = None
    if w.has_attention and w.M > 0 and not args.step_only:
        gram = cast.cast_wo_gram(gen.wo_weight(w.D, device=dev), w.H, w.dh)
        cprm = cast.cast_coupled_params_default()
        nb = cast.cast_route_coupled_workspace_bytes(w.n_a, w.S, w.H, w.dh, w.M, w.Bv)
        cws = torch.empty(nb, dtype=torch.uint8, device=dev)
        cidx = torch.empty((w.n_a, w.H, k_eff), dtype=torch.int32, device=dev)
        n_frames_c = max(w.n_frames, max(w.anchors) + 1)
        for i in range(args.warmup):
            s = sets[i % N_COPIES]
            cast.cast_route_coupled(s["q"], s["k"], s["v"], gram, w.anchors, n_frames_c, w.topk,
                                    w.scale, params=cprm, idx_out=cidx, workspace=cws, stream=stream)
        cm = [[ev(), ev()] for _ in range(args.steps)]
        torch.cuda.synchronize()
        for i in range(args.steps):
            s = sets[i % N_COPIES]
            cm[i][0].record(stream)
            cast.cast_route_coupled(s["q"], s["k"], s["v"], gram, w.anchors, n_frames_c, w.topk,
                                    w.scale, params=cprm, idx_out=cidx, workspace=cws, stream=stream)
            cm[i][1].record(stream)
        torch.cuda.synchronize()
        per_call["route_coupled"] = [a.elapsed_time(b) for a, b in cm]
        coupled_ms = float(np.mean(per_call["route_coupled"]))

    # the whole update of one residual site (e.g. the FFN site): PAR of the skipped
    # frames with every anchor's own update fused in, timed on its own
    block_ms = None
    if w.has_par and not args.step_only:
        bprm = cast.cast_par_params_default(accumulate=1, update_anchors=1)
        bm = [[ev(), ev()] for _ in range(args.steps)]
        for i in range(args.warmup):
            s = sets[i % N_COPIES]
            cast.cast_par_reconstruct(s["resid"], w.anchors, bprm, out=s["x"], workspace=par_ws,
                                      stream=stream)
        torch.cuda.synchronize()
        for i in range(args.steps):
            s = sets[i % N_COPIES]
            bm[i][0].record(stream)
            cast.cast_par_reconstruct(s["resid"], w.anchors, bprm, out=s["x"], workspace=par_ws,
                                      stream=stream)
            bm[i][1].record(stream)
        torch.cuda.synchronize()
        per_call["par_block_update"] = [a.elapsed_time(b) for a, b in bm]
        block_ms = float(np.mean(per_call["par_block_update"]))

    # control-aware frame selection for the next block (both control branches, bf16),
    # timed on its own
    sel_ms = None
    if w.n_frames >= 2 and not args.step_only:
        ctl = [gen.control_inputs(w, seed=args.seed + c, device=dev) for c in range(N_COPIES)]
        ages = torch.zeros(w.n_frames, dtype=torch.int32, device=dev)
        sel_out = torch.empty(len(w.anchors), dtype=torch.int32, device=dev)
        nb = cast.cast_frame_select_workspace_bytes(w.n_frames, w.S, w.D)
        sel_ws = torch.empty(nb, dtype=torch.uint8, device=dev)
        sm = [[ev(), ev()] for _ in range(args.steps)]
        for i in range(args.warmup):
            cam, act = ctl[i % N_COPIES]
            cast.cast_frame_select(cam, act, w.anchors, len(w.anchors), ages, anchors_out=sel_out,
                                   workspace=sel_ws, stream=stream)
        torch.cuda.synchronize()
        for i in range(args.steps):
            cam, act = ctl[i % N_COPIES]
            sm[i][0].record(stream)
            cast.cast_frame_select(cam, act, w.anchors, len(w.anchors), ages, anchors_out=sel_out,
                                   workspace=sel_ws, stream=stream)
            sm[i][1].record(stream)
        torch.cuda.synchronize()
        per_call["frame_select"] = [a.elapsed_time(b) for a, b in sm]
        sel_ms = float(np.mean(per_call["frame_select"]))
        del ctl

    # spectral diagnostics of the skipped frames (validation, not inference): error
    # ratio, band energies, transport phase error and both oracle corrections
    diag_ms = prog_ms = None
    if w.has_par and not args.step_only:
        s1, _ = cast.par_debug_shapes(w.n_a, w.Hg, w.Wg, prm)
        theta = torch.zeros(s1, device=dev)
        s0 = sets[0]
        cast.cast_par_reconstruct(s0["resid"], w.anchors, cast.cast_par_params_default(),
                                  out=s0["x"], theta_out=theta, workspace=par_ws, stream=stream)
        dws = torch.empty(cast.cast_spectral_diagnostics_workspace_bytes(
            w.n_frames, w.Hg, w.Wg, w.D, cast.cast_diag_params_default()), dtype=torch.uint8, device=dev)
        dm = [ev(), ev()]
        n_diag = 3
        cast.cast_spectral_diagnostics(s0["resid"], s0["x"], w.anchors, theta=theta,
                                       want_corrections=True, workspace=dws, stream=stream)
        torch.cuda.synchronize()
        dm[0].record(stream)
        for _ in range(n_diag):
            cast.cast_spectral_diagnostics(s0["resid"], s0["x"], w.anchors, theta=theta,
                                           want_corrections=True, workspace=dws, stream=stream)
        dm[1].record(stream)
        torch.cuda.synchronize()
        diag_ms = dm[0].elapsed_time(dm[1]) / n_diag
        del dws
        # phase progress of every coefficient over each pair's interior frames
        dprm = cast.cast_diag_params_default()
        n_tiles = -(-w.Hg // dprm.tile_h) * -(-w.Wg // dprm.tile_w)
        pp = torch.empty((w.n_frames, n_tiles, dprm.tile_h * (dprm.tile_w // 2 + 1), w.D),
                         dtype=torch.float32, device=dev)
        cast.cast_phase_progress(s0["resid"], w.anchors, dprm, p_out=pp, stream=stream)
        torch.cuda.synchronize()
        dm[0].record(stream)
        for _ in range(n_diag):
            cast.cast_phase_progress(s0["resid"], w.anchors, dprm, p_out=pp, stream=stream)
        dm[1].record(stream)
        torch.cuda.synchronize()
        prog_ms = dm[0].elapsed_time(dm[1]) / n_diag
        del pp

    value = w.frame_tokens / (ms_step / 1e3)
    res = {
        "metric": "CAST block-step frame-tokens/s (routing + routed anchor attention + PAR)",
        "value": value, "unit": "frame-tokens/s", "n_gpus": 1, "steps": args.steps,
        "warmup": args.warmup, "ms_per_step": ms_step, "higher_is_better": True,
        "scaling": "weak", "vs_baseline": None, "dtype": "bf16+fp32",
        "data": f"synthetic (seeded generator inputs of workload {w.name})",
        "config": {"workload": w.name, "frames": w.n_frames, "grid": f"{w.Hg}x{w.Wg}",
                   "D": w.D, "heads": w.H, "dh": w.dh, "anchors": list(w.anchors),
                   "history_chunks": w.M, "chunk_tokens": w.Bv, "topk": w.topk,
                   "par_mode": "accumulate", "input_copies": N_COPIES,
                   "step_launch": "eager" if not graphs else "hip graph per input copy",
                   "attn_input_seeds": seeds if w.has_attention else None},
        "per_call_ms": {"route": route_ms, "attn": attn_ms, "par": par_ms,
                        "route_coupled": coupled_ms, "par_block_update": block_ms,
                        "frame_select": sel_ms, "spectral_diagnostics": diag_ms,
                        "phase_progress": prog_ms},
        "per_call_ms_median": {**call_median,
                               **{c: float(np.median(v)) for c, v in per_call.items()
                                  if isinstance(v, list)}},
        "ms_per_step_each": {"median": float(np.median(step_each)), "min": float(min(step_each)),
                             "max": float(max(step_each))},
    }
    extra = {}
    traffic = load_traffic(w.name)
    if w.has_attention:
        fl = attn_flops(w, k_eff)
        tf = fl / (attn_ms / 1e3) / 1e12
        # the attention call: anchor_attn_kernel, plus attn_merge_kernel when the
        # units of a last partial round are split along the keys
        kname = f"anchor_attn_kernel<{w.dh}>" + (" + attn_merge_kernel" if attn_ws is not None else "")
        res["roofline"] = {"bound": "mfma", "kernel": kname,
                           "achieved": tf, "peak": PEAK_BF16_TFLOPS, "unit": "TFLOP/s",
                           "frac": tf / PEAK_BF16_TFLOPS, "traffic": traffic.get("attn"),
                           "algorithmic_per_launch": fl}
        extra["attn_mfma_util_pct"] = 100.0 * tf / PEAK_BF16_TFLOPS
        rg = route_bytes(w) / (route_ms / 1e3) / 1e9
        extra["route_hbm_gbps"] = rg
        extra["route_hbm_pct"] = 100.0 * rg / PEAK_HBM_GBS
        extra["route_traffic_bytes"] = traffic.get("route")
        if coupled_ms:
            cg = coupled_route_bytes(w) / (coupled_ms / 1e3) / 1e9
            extra["route_coupled_hbm_gbps"] = cg
            extra["route_coupled_hbm_pct"] = 100.0 * cg / PEAK_HBM_GBS
    if w.has_par:
        pg = par_bytes(w, True) / (par_ms / 1e3) / 1e9
        extra["par_hbm_gbps"] = pg
        extra["par_hbm_pct"] = 100.0 * pg / PEAK_HBM_GBS
        extra["par_traffic_bytes"] = traffic.get("par")
        if block_ms:
            bg = block_update_bytes(w) / (block_ms / 1e3) / 1e9
            extra["par_block_update_hbm_gbps"] = bg
            extra["par_block_update_hbm_pct"] = 100.0 * bg / PEAK_HBM_GBS
        if not w.has_attention:
            res["roofline"] = {"bound": "hbm", "kernel": "par (xspec+gate+recon)",
                               "achieved": pg, "peak": PEAK_HBM_GBS, "unit": "GB/s",
                               "frac": pg / PEAK_HBM_GBS, "traffic": traffic.get("par"),
                               "algorithmic_per_launch": par_bytes(w, True)}
    if sel_ms:
        fg = frame_select_bytes(w) / (sel_ms / 1e3) / 1e9
        extra["frame_select_hbm_gbps"] = fg
        extra["frame_select_hbm_pct"] = 100.0 * fg / PEAK_HBM_GBS
    res.update(extra)
    if not args.no_cpu_baseline:
        try:
            res["cpu_baseline"] = cpu_baseline(w, seed=args.seed)
        except Exception as e:  # reported, never fatal for the GPU measurement
            res["cpu_baseline"] = {"value": None, "error": repr(e)}
    print(json.dumps(res), flush=True)


if __name__ == "__main__":
    main()
