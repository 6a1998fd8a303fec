"""The block step (routing -> routed anchor attention -> PAR in accumulate mode)
captured as a HIP graph and replayed: every replay must reproduce the eager step
bit for bit.

Each input copy's step is captured once.  Between replays the test does eager
work of its own (resets PAR's accumulator, poisons every output with NaN,
synchronizes), so a replay that reused stale results, skipped a kernel or lost a
node would show.  The library allocates nothing and issues no memsets, so its
launches are all a captured step holds.
"""
import numpy as np
import pytest
import torch

import gen
import paper_2609_34144_amd as cast

pytestmark = pytest.mark.gpu


def log(msg):
    print(msg, flush=True)


@pytest.mark.parametrize("name", ["tiny_4f8x8_d64", "matrix_game_like_8f30x52_d1536"])
def test_step_graph_replays_match_eager(cast_lib, name):
    w = gen.get(name)
    dev = torch.device("cuda:0")
    log(f"graph replay: workload {name}")
    prm = cast_lib.cast_par_params_default(accumulate=1)
    k_eff = min(w.topk, w.M)
    resid_np, _, _ = gen.par_inputs(w, seed=3)
    resid = torch.from_numpy(resid_np).to(dev)
    route_ws = torch.empty(cast_lib.cast_route_kv_workspace_bytes(w.n_a, w.S, w.H, w.dh, w.M, w.Bv),
                           dtype=torch.uint8, device=dev)
    par_ws = torch.empty(max(cast_lib.cast_par_workspace_bytes(w.n_frames, w.n_a, w.Hg, w.Wg, w.D, prm), 1),
                         dtype=torch.uint8, device=dev)

    copies = []
    for seed in (11, 12):
        q, k, v, _, _ = gen.attn_inputs(w, seed=seed, device=dev)
        g = torch.Generator(device="cpu").manual_seed(seed)
        x0 = torch.randn(resid.shape, generator=g, dtype=torch.float32).to(dev)
        copies.append({
            "q": q, "k": k, "v": v, "x0": x0, "x": x0.clone(),
            "idx": torch.empty((w.n_a, w.H, k_eff), dtype=torch.int32, device=dev),
            "out": torch.empty((w.n_a, w.S, w.H, w.dh), dtype=torch.bfloat16, device=dev),
        })

    def step(c):
        st = torch.cuda.current_stream()
        _, ke, _ = cast_lib.cast_route_kv(c["q"], c["k"], w.topk, w.scale, idx_out=c["idx"],
                                          workspace=route_ws, stream=st)
        cast_lib.cast_anchor_attn(c["q"], c["k"], c["v"], c["idx"], ke, w.scale, out=c["out"], stream=st)
        cast_lib.cast_par_reconstruct(resid, w.anchors, prm, out=c["x"], workspace=par_ws, stream=st)

    # eager results
    want = []
    for c in copies:
        c["x"].copy_(c["x0"])
        step(c)
        torch.cuda.synchronize()
        want.append({key: c[key].clone() for key in ("idx", "out", "x")})
    for c, wnt in zip(copies, want):
        assert torch.isfinite(wnt["out"].float()).all() and torch.isfinite(wnt["x"]).all()
        assert not torch.equal(wnt["x"], c["x0"]), "PAR wrote nothing"

    graphs = []
    for c in copies:
        gr = torch.cuda.CUDAGraph()
        with torch.cuda.graph(gr):
            step(c)
        graphs.append(gr)
    torch.cuda.synchronize()

    for rep in range(3):
        for ci, (c, gr) in enumerate(zip(copies, graphs)):
            # eager work between replays: reset the accumulator, poison the outputs
            c["x"].copy_(c["x0"])
            c["idx"].fill_(-1)
            c["out"].fill_(float("nan"))
            torch.cuda.synchronize()
            gr.replay()
            torch.cuda.synchronize()
            for key in ("idx", "out", "x"):
                same = torch.equal(c[key], want[ci][key])
                if not same:
                    d = (c[key].float() - want[ci][key].float()).abs()
                    raise AssertionError(f"{name} replay {rep} copy {ci}: {key} differs from the eager "
                                         f"step (max |diff| {float(torch.nan_to_num(d, nan=np.inf).max())})")
            log(f"  replay {rep} copy {ci}: identical to eager")
