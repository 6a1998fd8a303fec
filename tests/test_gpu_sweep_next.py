"""GPU parity on seeded random shapes for the steps beside the hot path:
reconstruction-coupled routing (eq:omission, Algorithm 1), control-aware frame
selection (Sec. 4.2) and the spectral diagnostics, each against the float64
oracle with its own suite's checker and bars (test_gpu_coupled.py,
test_gpu_frame_select.py, test_gpu_diagnostics.py).

Each case draws its sizes from its own seed, so a failure names a reproducible
shape: head sizes 32/64/128, anchors with and without boundary frames on either
side, budgets below and above the history, ragged token counts and channel counts
that are not a multiple of the 64-lane blocks, bf16 and fp32 control inputs, one
or both control branches, tilings 8x8 and 2..7."""
import numpy as np
import pytest
import torch

import gen
from gen import workloads as W
from test_gpu_coupled import run_case as coupled_case
from test_gpu_diagnostics import run_case as diag_case
from test_gpu_frame_select import run_schedule
from test_gpu_parity import log

pytestmark = pytest.mark.gpu


def sorted_anchors(rng, n_frames, n_anchor):
    return tuple(sorted(rng.choice(np.arange(n_frames), n_anchor, replace=False).tolist()))


@pytest.mark.parametrize("seed", list(range(10)))
def test_coupled_random_shapes(cast_lib, seed):
    rng = np.random.default_rng(5000 + seed)
    dh = int(rng.choice([32, 64, 128]))
    H = int(rng.integers(1, 4))
    n_frames = int(rng.integers(2, 13))
    n_anchor = int(rng.integers(1, min(4, n_frames) + 1))
    anchors = sorted_anchors(rng, n_frames, n_anchor)
    M = int(rng.integers(2, 41))
    Bv = int(rng.integers(1, 200))
    topk = int(rng.integers(1, M + 3))
    Hg, Wg = int(rng.integers(1, 20)), int(rng.integers(1, 20))
    prm = {} if seed % 3 else {"passes": int(rng.integers(0, 4)), "l_rec": float(rng.choice([0.5, 2.0]))}
    base = gen.get(W.TINY).__dict__
    w = W.Workload(**{**base, "name": f"coupled{seed}", "H": H, "dh": dh, "Hg": Hg, "Wg": Wg,
                      "anchors": anchors, "M": M, "Bv": Bv, "topk": topk, "n_frames": n_frames})
    log(f"[sweep coupled {seed}] dh {dh} H {H} S {Hg * Wg} anchors {anchors} of {n_frames} "
        f"M {M} Bv {Bv} topk {topk} {prm}")
    (exact, loose), idx = coupled_case(cast_lib, w, anchors, n_frames, topk, seed=seed, M=M, Bv=Bv, **prm)
    if topk >= M:
        assert (idx.cpu().numpy() == np.arange(M)).all()


@pytest.mark.parametrize("seed", list(range(8)))
def test_frame_select_random_shapes(cast_lib, seed):
    rng = np.random.default_rng(6000 + seed)
    n_cur = int(rng.integers(1, 25))
    k_f = int(rng.integers(1, n_cur + 1))
    Hg, Wg, D = int(rng.integers(1, 40)), int(rng.integers(1, 40)), int(rng.integers(1, 200))
    dtype = torch.bfloat16 if seed % 2 == 0 else torch.float32
    branches = [(True, True), (True, False), (False, True)][seed % 3]
    blocks = int(rng.integers(2, 4))
    w = W.Workload(**{**gen.get(W.TINY).__dict__, "Hg": Hg, "Wg": Wg, "D_par": D})
    log(f"[sweep select {seed}] n_cur {n_cur} k_f {k_f} S {Hg * Wg} D {D} {dtype} branches {branches}")
    picks = run_schedule(cast_lib, w, n_cur, k_f, blocks, dtype=dtype, branches=branches, seed=seed,
                         label=f"sweep{seed}")
    for p in picks:
        assert len(p) == k_f and p == sorted(set(p)) and all(0 <= a < n_cur for a in p)


@pytest.mark.parametrize("seed", list(range(8)))
def test_diagnostics_random_shapes(cast_lib, seed):
    rng = np.random.default_rng(7000 + seed)
    n = int(rng.integers(3, 9))
    anchors = sorted_anchors(rng, n, int(rng.integers(2, min(4, n - 1) + 1)))
    Hg, Wg, D = int(rng.integers(1, 34)), int(rng.integers(1, 34)), int(rng.integers(1, 130))
    tile = 8 if seed % 2 == 0 else (int(rng.integers(2, 8)), int(rng.integers(2, 8)))
    n_bands = int(rng.integers(1, 5))
    edges = tuple(np.concatenate([[0.0], np.sort(rng.uniform(0.05, 0.95, n_bands - 1)), [1.0]]))
    shift = rng.integers(-2, 3, size=2)
    base = rng.standard_normal((Hg, Wg, D))
    ref = np.stack([np.roll(base, (int(shift[0]) * t, int(shift[1]) * t), axis=(0, 1))
                    + 0.3 * rng.standard_normal((Hg, Wg, D)) for t in range(n)])
    label = f"sweep{seed} {n}x{Hg}x{Wg}x{D} anchors {anchors} tile {tile} bands {n_bands}"
    log(f"[sweep diag {seed}] {label}")
    diag_case(cast_lib, ref, anchors, label, tile=tile, edges=edges)
