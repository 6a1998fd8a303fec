"""Float64 oracle for pooled chunk scoring and fixed-budget TopK routing.

TEST INFRASTRUCTURE ONLY (see the package docstring).

Sec. 4.4 eq:pooled: each head's historical KV is split into M equal blocks;
pooled query q_bar_i (anchor frame i) and pooled key k_bar_m (block m) give the
chunk score s_{i,m} = q_bar_i . k_bar_m * scale (the paper's scale is
1/sqrt(d_h); the scale is a parameter here).  eq:topk / App. B.3: the budget
keeps exactly K_KV = min(topk, M) blocks per anchor (fewer than K_KV blocks:
keep all and report the realised budget).

Readings where the paper leaves a choice: routing is per (anchor frame, head); the pooled
query is the mean over all S tokens of the anchor frame, the pooled key the
mean over the B_v tokens of the block, so q_bar . k_bar equals the mean of
q . k over all token pairs; the TopK order is (score descending, chunk index
ascending) and the selected set is reported in ascending chunk order.
"""
from __future__ import annotations

import numpy as np


def pooled_means(q: np.ndarray, k_hist: np.ndarray):
    """q [n_a, S, H, dh], k_hist [M, Bv, H, dh] -> q_bar [n_a, H, dh], k_bar [M, H, dh]."""
    qb = np.asarray(q, dtype=np.float64).mean(axis=1)
    kb = np.asarray(k_hist, dtype=np.float64).mean(axis=1)
    return qb, kb


def chunk_scores(q: np.ndarray, k_hist: np.ndarray, scale: float = 1.0) -> np.ndarray:
    """eq:pooled scores s[i, h, m] = scale * q_bar[i, h] . k_bar[m, h]."""
    qb, kb = pooled_means(q, k_hist)
    return scores_from_means(qb, kb, scale)


def scores_from_means(qb: np.ndarray, kb: np.ndarray, scale: float = 1.0) -> np.ndarray:
    """eq:pooled score from pooled means q_bar [n_a, H, dh] and k_bar [M, H, dh]."""
    return scale * np.einsum("ihd,mhd->ihm", np.asarray(qb, np.float64), np.asarray(kb, np.float64))


def topk_select(scores_1d, topk: int) -> list[int]:
    """The k_eff = min(topk, M) largest scores under the total order
    (score descending, chunk index ascending), returned in ascending chunk order."""
    s = [float(x) for x in scores_1d]
    order = sorted(range(len(s)), key=lambda m: (-s[m], m))
    k_eff = min(int(topk), len(s))
    return sorted(order[:k_eff])


def route(q: np.ndarray, k_hist: np.ndarray, topk: int, scale: float = 1.0,
          decide_dtype=None):
    """Scores and per-(anchor, head) selected chunk indices.

    If `decide_dtype` is given (np.float32: the paper's precision for pooled
    reductions), the selection is made on the scores rounded to that type.
    Returns (scores float64 [n_a, H, M], idx int32 [n_a, H, k_eff], k_eff).
    """
    s = chunk_scores(q, k_hist, scale)
    n_a, H, M = s.shape
    k_eff = min(int(topk), M)
    sd = s.astype(decide_dtype) if decide_dtype is not None else s
    idx = np.zeros((n_a, H, k_eff), dtype=np.int32)
    for i in range(n_a):
        for h in range(H):
            idx[i, h] = topk_select(sd[i, h], k_eff)
    return s, idx, k_eff
