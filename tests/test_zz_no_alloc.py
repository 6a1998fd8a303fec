"""The static-scratch PAR entry point (cast_par_reconstruct_noalloc) against
cast_par_reconstruct with a caller workspace, through the C ABI: two calls in a
row on one GPU, the second with a smaller input, both bit-identical to the
workspace entry point (same kernels, same plan) and within the PAR bar of the
oracle."""
import numpy as np
import pytest
import torch

import gen
from gen import workloads as W
from oracle import par as OP

pytestmark = pytest.mark.gpu


def _rel_rms(x, y):
    return float(np.linalg.norm((x - y).ravel()) / max(np.linalg.norm(y.ravel()), 1e-300))


def _run_both(cast_lib, resid_np, anchors, accumulate, x0_np, label):
    dev = "cuda"
    print(f"[noalloc {label}] shape {resid_np.shape} anchors {anchors} acc {accumulate}", flush=True)
    resid = torch.from_numpy(resid_np.astype(np.float32)).to(dev)
    prm = cast_lib.cast_par_params_default(accumulate=int(accumulate))
    x0 = torch.from_numpy(x0_np.astype(np.float32)).to(dev)
    s1, s2 = cast_lib.par_debug_shapes(len(anchors), resid.shape[1], resid.shape[2], prm)
    outs = []
    for fn in ("ws", "static"):
        out = x0.clone()
        th = torch.zeros(s1, device=dev)
        cf = torch.zeros(s2, device=dev)
        if fn == "ws":
            cast_lib.cast_par_reconstruct(resid, anchors, prm, out=out, theta_out=th, conf_out=cf)
        else:
            cast_lib.cast_par_reconstruct_noalloc(resid, anchors, prm, out=out, theta_out=th,
                                                  conf_out=cf)
        torch.cuda.synchronize()
        outs.append((out, th, cf))
    (a, tha, cfa), (b, thb, cfb) = outs
    assert torch.equal(a, b) and torch.equal(tha, thb) and torch.equal(cfa, cfb), label
    ref = OP.par_reconstruct(resid_np.astype(np.float32).astype(np.float64), anchors,
                             OP.ParParams(accumulate=accumulate),
                             out=x0_np.astype(np.float32).astype(np.float64))
    sk = [t for t in range(resid_np.shape[0]) if t not in set(anchors)]
    rr = _rel_rms(b.cpu().numpy().astype(np.float64)[sk], ref[sk])
    print(f"[noalloc {label}] bit-identical to the workspace entry point; rel-RMS {rr:.2e}",
          flush=True)
    assert rr <= 1e-4, (label, rr)
    for t in anchors:
        assert torch.equal(b[t], x0[t]), (label, t)


def test_noalloc_matches_workspace_entry_point(cast_lib):
    rng = np.random.default_rng(3)
    # first call: Matrix-like grid, three anchors, accumulate mode
    w = gen.get(W.MATRIX)
    resid, _, _ = gen.par_inputs(w, seed=42, D=256)
    assert cast_lib.cast_par_workspace_bytes(w.n_frames, len(w.anchors), w.Hg, w.Wg, 256,
                                             cast_lib.cast_par_params_default()) \
        <= cast_lib.cast_par_static_scratch_bytes()
    x0 = rng.standard_normal(resid.shape)
    _run_both(cast_lib, resid, w.anchors, True, x0, "large")
    # second call, smaller: edge tiles, two anchors, boundary extrapolation, write mode
    base = rng.standard_normal((13, 11, 40))
    small = np.zeros((5, 13, 11, 40))
    small[1] = base
    small[3] = np.roll(base, (1, 1), axis=(0, 1)) + 0.2 * rng.standard_normal(base.shape)
    _run_both(cast_lib, small, (1, 3), False, rng.standard_normal(small.shape), "small")
