"""Float64 oracle for control-aware frame selection.

TEST INFRASTRUCTURE ONLY (see the package docstring).

Sec. 3.1 eq:sensitivity, Sec. 4.2 eq:debt and eq:score, App. A.1
eq:normalization and the scheduling rules:

* r_{i,k} = RMS of the control branch's feature update Delta_{i,k} over frame i's
  spatial and channel coordinates, for each available branch k (camera, action);
* Norm = (r - min_j r) / (max_j r - min_j r + eps) across the current chunk,
  separately per branch; d_i = the mean of Norm over the available branches
  (an absent branch is left out of the mean, not counted as zero);
* refresh age h_i: 0 for the block's anchors, h_i + 1 for every other frame;
  H_cov = ceil(N_cur / K_f); coverage debt D_i = h_i / H_cov;
* score S_i = d_i + lambda_cov D_i with a fresh control response, lambda_cov D_i
  without one (no stale sensitivity is reused);
* anchors of the next block = the K_f largest S_i, ties by increasing frame index,
  neither endpoint mandatory; a dense block is a block whose anchors are all
  frames (it resets every age).

Readings where the paper leaves a choice: eps = 1e-8 (the paper's stabiliser elsewhere;
its value is not given here); the decision is taken in float32, the precision
the kernels compute scores in: r is formed in float64 and rounded to float32,
every later step is float32 arithmetic with one rounding per operation.
"""
from __future__ import annotations

import math

import numpy as np

LAMBDA_COV = 0.5     # Sec. 4.2, tab:config_cast
EPS = 1e-8
F32 = np.float32


def response_rms(delta) -> np.ndarray:
    """r_i = sqrt(mean of Delta_i^2) over all of frame i's coordinates.
    delta [N_cur, ...] (any float dtype) -> float64 [N_cur]."""
    x = np.asarray(delta, dtype=np.float64)
    x = x.reshape(x.shape[0], -1)
    return np.sqrt((x * x).mean(axis=1))


def normalize(r, eps: float = EPS) -> np.ndarray:
    """eq:normalization in float32: (r - min r) / (max r - min r + eps)."""
    r = np.asarray(r, dtype=F32)
    lo, hi = r.min(), r.max()
    den = F32(F32(hi - lo) + F32(eps))
    return ((r - lo) / den).astype(F32)


def sensitivity(rs, eps: float = EPS):
    """eq:sensitivity: d_i = mean over the available branches of Norm(r_{., k});
    None when no branch is available."""
    rs = [r for r in rs if r is not None]
    if not rs:
        return None
    acc = np.zeros(len(rs[0]), dtype=F32)
    for r in rs:
        acc = (acc + normalize(r, eps)).astype(F32)
    return (acc / F32(len(rs))).astype(F32)


def update_ages(h, anchors, n_cur: int) -> np.ndarray:
    """eq:debt, first line: ages after a block with anchor set `anchors`."""
    h = np.zeros(n_cur, dtype=np.int64) if h is None else np.asarray(h, dtype=np.int64).copy()
    keep = set(int(a) for a in anchors)
    return np.array([0 if i in keep else h[i] + 1 for i in range(n_cur)], dtype=np.int64)


def coverage_debt(h, n_cur: int, k_f: int) -> np.ndarray:
    """eq:debt, second line: D_i = h_i / ceil(N_cur / K_f), float32."""
    h_cov = -(-n_cur // k_f)
    return (np.asarray(h, dtype=F32) / F32(h_cov)).astype(F32)


def scores(d, debt, lambda_cov: float = LAMBDA_COV) -> np.ndarray:
    """eq:score in float32 (product rounded, then the sum)."""
    ld = (F32(lambda_cov) * np.asarray(debt, dtype=F32)).astype(F32)
    if d is None:
        return ld
    return (np.asarray(d, dtype=F32) + ld).astype(F32)


def topk_frames(s, k_f: int) -> list[int]:
    """The K_f largest scores, ties by increasing frame index, ascending output."""
    v = [float(x) for x in s]
    order = sorted(range(len(v)), key=lambda i: (-v[i], i))
    return sorted(order[:k_f])


def select_next(deltas, h_prev, anchors_prev, k_f: int, lambda_cov: float = LAMBDA_COV,
                eps: float = EPS):
    """One scheduling step: the block ran with anchors_prev and its control
    branches produced `deltas` (a list with None for an absent branch).
    Returns (anchors_next, ages, scores, r_per_branch (float32 or None))."""
    n_cur = None
    for dl in deltas:
        if dl is not None:
            n_cur = np.asarray(dl).shape[0]
    if n_cur is None:
        n_cur = len(h_prev)
    rs = [None if dl is None else response_rms(dl).astype(F32) for dl in deltas]
    d = sensitivity(rs, eps)
    h = update_ages(h_prev, anchors_prev, n_cur)
    s = scores(d, coverage_debt(h, n_cur, k_f), lambda_cov)
    return topk_frames(s, k_f), h, s, rs


def scores_exact(deltas, h, k_f: int, lambda_cov: float = LAMBDA_COV, eps: float = EPS):
    """The plain definition in float64 with no rounding between steps (r, the
    min-max normalisation, d, D and S of eq:sensitivity, eq:normalization,
    eq:debt, eq:score), for the ages `h` after the block.  The float32 pipeline
    above takes its decision in the kernels' precision; this is the reference it
    is held to."""
    rs = [None if dl is None else response_rms(dl) for dl in deltas]
    n_cur = len(h)
    norms = []
    for r in rs:
        if r is not None:
            norms.append((r - r.min()) / (r.max() - r.min() + eps))
    d = np.mean(norms, axis=0) if norms else None
    debt = np.asarray(h, dtype=np.float64) / float(-(-n_cur // k_f))
    return lambda_cov * debt if d is None else d + lambda_cov * debt


def brute_topk(s, k_f: int) -> list[int]:
    """The K_f-subset with the largest score sum and, among equal sums, the
    lexicographically smallest index set (brute force over all subsets)."""
    import itertools
    best = None
    for sub in itertools.combinations(range(len(s)), k_f):
        tot = math.fsum(float(s[i]) for i in sub)
        key = (-tot, sub)
        if best is None or key < best[0]:
            best = (key, list(sub))
    return best[1]
