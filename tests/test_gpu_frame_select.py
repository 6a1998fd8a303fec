"""GPU parity of control-aware frame selection (cast_frame_select) against the
oracle (oracle/frame_select.py) on the same inputs.

r (the per-frame RMS of a control branch's update) is floating point: rel <= 1e-6
(fp32 partial sums against float64).  The scores follow r through fp32
operations that both sides perform with one rounding each, so they must agree to
1e-6 absolute.  Ages are integers: exact.  The anchors are integer output decided
by fp32 scores: exact wherever the oracle's K-th / (K+1)-th score gap exceeds
1e-5; inside that band the GPU's set must be a valid TopK of its own scores.
Debt-only selection (no control branch) has exactly representable scores on both
sides and must match exactly.  The scores are also held to the float64 definition
(no rounding between steps): within 2e-6, and the anchors exact wherever that
definition's K-th / (K+1)-th gap exceeds 1e-5.  Each scheduling run continues from the GPU's
anchors, so both sides stay in lockstep."""
import numpy as np
import pytest
import torch

import gen
from gen import workloads as W
from oracle import frame_select as FS
from test_gpu_parity import log

pytestmark = pytest.mark.gpu

R_REL, S_ABS, GAP = 1e-6, 1e-6, 1e-5


def to_np(t):
    return None if t is None else t.float().cpu().numpy().astype(np.float64)


def one_step(cast_lib, cam, act, prev, k_f, ages, h_or, label, n_cur=None, lambda_cov=0.5):
    dev = "cuda"
    n = n_cur if n_cur is not None else (cam if cam is not None else act).shape[0]
    r_out = torch.full((2, n), -1.0, device=dev)
    s_out = torch.full((n,), -1.0, device=dev)
    prm = cast_lib.cast_select_params_default(lambda_cov=lambda_cov)
    got = cast_lib.cast_frame_select(cam, act, prev, k_f, ages, params=prm, n_cur=n, r_out=r_out,
                                     score_out=s_out)
    torch.cuda.synchronize()
    a_or, h_or, s_or, rs_or = FS.select_next([to_np(cam), to_np(act)], h_or, prev, k_f, lambda_cov)
    g_anchors = [int(x) for x in got.cpu().numpy()]
    g_ages = ages.cpu().numpy()
    g_s = s_out.cpu().numpy().astype(np.float64)
    assert list(g_ages) == list(h_or), (label, list(g_ages), list(h_or))
    for row, r in enumerate(rs_or):
        if r is None:
            assert torch.all(r_out[row] == -1.0), (label, "absent branch row written")
            continue
        g_r = r_out[row].cpu().numpy().astype(np.float64)
        assert np.max(np.abs(g_r - r) / np.maximum(np.abs(r), 1e-30)) <= R_REL, (label, row)
    assert np.max(np.abs(g_s - s_or)) <= S_ABS, (label, np.max(np.abs(g_s - s_or)))
    # and against the float64 definition: scores within fp32 rounding, the anchors
    # exact wherever the exact K-th / (K+1)-th gap is clear of it
    ex = FS.scores_exact([to_np(cam), to_np(act)], h_or, k_f, lambda_cov)
    assert np.max(np.abs(g_s - ex)) <= 2 * S_ABS, (label, np.max(np.abs(g_s - ex)))
    srt_ex = np.sort(ex)[::-1]
    if k_f == n or srt_ex[k_f - 1] - srt_ex[k_f] > GAP:
        assert g_anchors == sorted(sorted(range(n), key=lambda i: (-ex[i], i))[:k_f]), label
    assert len(g_anchors) == k_f and g_anchors == sorted(set(g_anchors))
    srt = np.sort(s_or.astype(np.float64))[::-1]
    gap = srt[k_f - 1] - srt[k_f] if k_f < n else np.inf
    if gap > GAP:
        assert g_anchors == a_or, (label, g_anchors, a_or)
        exact = True
    else:
        assert g_anchors == FS.topk_frames(s_out.cpu().numpy(), k_f), label
        exact = False
    return g_anchors, h_or, exact


def run_schedule(cast_lib, w, n_cur, k_f, blocks, *, dtype=torch.bfloat16, branches=(True, True),
                 seed=42, label=""):
    ages = torch.zeros(n_cur, dtype=torch.int32, device="cuda")
    prev, h_or = list(range(n_cur)), np.zeros(n_cur, dtype=np.int64)   # a dense first block
    picks, n_exact = [], 0
    for b in range(blocks):
        cam, act = gen.control_inputs(w, seed=seed + b, device="cuda", n_cur=n_cur, dtype=dtype)
        cam = cam if branches[0] else None
        act = act if branches[1] else None
        prev, h_or, exact = one_step(cast_lib, cam, act, prev, k_f, ages, h_or, f"{label} b{b}")
        picks.append(prev)
        n_exact += exact
    log(f"[select {label}] anchors per block {picks}; exact decisions {n_exact}/{blocks}")
    return picks


def test_select_matrix_like_schedule(cast_lib):
    """Matrix-Game-like block (30x52 tokens, D = 1536), 5 of 10 frames, both
    branches in bf16, six blocks after the dense one."""
    run_schedule(cast_lib, gen.get(W.MATRIX), 10, 5, 6, label="matrix 5/10 bf16")


def test_select_hy_like_one_branch_fp32(cast_lib):
    """HY-World-like grid (44x80, D = 3072), 2 of 4 frames, only the action branch
    (the absent camera branch is left out of d), fp32 updates."""
    run_schedule(cast_lib, gen.get(W.HY), 4, 2, 4, dtype=torch.float32, branches=(False, True),
                 label="hy 2/4 fp32 act")


def test_select_debt_only_interleaves(cast_lib):
    """No fresh control response: S = lambda_cov D; the anchors rotate exactly as
    worked by hand for the oracle (N = 10, K_f = 3)."""
    n, k = 10, 3
    ages = torch.zeros(n, dtype=torch.int32, device="cuda")
    prev, h_or, picks = list(range(n)), np.zeros(n, dtype=np.int64), []
    for b in range(5):
        prev, h_or, exact = one_step(cast_lib, None, None, prev, k, ages, h_or, f"debt b{b}", n_cur=n)
        picks.append(prev)
    assert picks == [[0, 1, 2], [3, 4, 5], [6, 7, 8], [0, 1, 9], [2, 3, 4]]


def test_select_scalar_path_and_alignment(cast_lib):
    """Frames whose element count is not a multiple of the 16-byte vector width,
    and a base that is not 16-byte aligned: the scalar scan."""
    w = W.Workload(**{**gen.get(W.TINY).__dict__, "Hg": 37, "Wg": 1, "D_par": 33})
    for dtype in (torch.float32, torch.bfloat16):
        cam, act = gen.control_inputs(w, seed=9, device="cuda", n_cur=7, dtype=dtype)
        buf = torch.empty(cam.numel() + 1, dtype=dtype, device="cuda")
        cam_off = buf[1:].view(cam.shape)
        cam_off.copy_(cam)
        ages = torch.zeros(7, dtype=torch.int32, device="cuda")
        one_step(cast_lib, cam_off, act, list(range(7)), 3, ages, np.zeros(7, dtype=np.int64),
                 f"scalar {dtype}")


def test_select_many_frames_and_all_frames(cast_lib):
    """Thousands of small frames (several frames per thread in the selection
    block), and K_f = N_cur (every frame an anchor)."""
    w = W.Workload(**{**gen.get(W.TINY).__dict__, "Hg": 2, "Wg": 2, "D_par": 16})
    for n, k in ((3000, 700), (9, 9)):
        cam, act = gen.control_inputs(w, seed=n, device="cuda", n_cur=n)
        ages = torch.zeros(n, dtype=torch.int32, device="cuda")
        got, _, _ = one_step(cast_lib, cam, act, list(range(0, n, 3)), k, ages,
                             np.zeros(n, dtype=np.int64), f"n{n} k{k}")
        if k == n:
            assert got == list(range(n))


def test_select_deterministic(cast_lib):
    w = gen.get(W.MATRIX)
    cam, act = gen.control_inputs(w, seed=5, device="cuda", n_cur=10)
    outs = []
    for _ in range(2):
        ages = torch.zeros(10, dtype=torch.int32, device="cuda")
        s = torch.empty(10, device="cuda")
        a = cast_lib.cast_frame_select(cam, act, [0, 4, 9], 5, ages, score_out=s)
        torch.cuda.synchronize()
        outs.append((a.clone(), s.clone(), ages.clone()))
    assert all(torch.equal(x, y) for x, y in zip(outs[0], outs[1]))


def test_select_single_frame_and_single_anchor(cast_lib):
    """N_cur = 1 (the one frame is always the anchor; its normalised response is 0)
    and K_f = 1 of several frames (the strongest response wins)."""
    w = W.Workload(**{**gen.get(W.TINY).__dict__, "Hg": 4, "Wg": 4, "D_par": 8})
    for n, k in ((1, 1), (6, 1)):
        cam, act = gen.control_inputs(w, seed=21 + n, device="cuda", n_cur=n)
        ages = torch.zeros(n, dtype=torch.int32, device="cuda")
        got, _, _ = one_step(cast_lib, cam, act, [0], k, ages, np.zeros(n, dtype=np.int64), f"n{n} k{k}")
        if n == 1:
            assert got == [0]
