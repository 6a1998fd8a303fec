"""Float64 oracle for routed block-sparse anchor attention.

TEST INFRASTRUCTURE ONLY (see the package docstring).

Sec. 4.4 and App. B.4: only anchor frames issue queries; each (anchor i,
head h) attends to the always-available current/text segment (N_0 tokens) and
to the K_KV routed historical blocks M_i (B_v tokens each), i.e. to
N_0 + K_KV B_v keys, with softmax(scale Q K^T) V, scale = 1/sqrt(d_h)
(eq:pooled's scaling).  Dense softmax with max subtraction, in float64.
"""
from __future__ import annotations

import numpy as np


def gather_kv(k_hist, v_hist, idx_ih, h, k_cur=None, v_cur=None):
    """Keys/values one (anchor, head) attends to: [current segment ; routed chunks]."""
    dh = k_hist.shape[-1]
    ks, vs = [], []
    if k_cur is not None and k_cur.shape[0] > 0:
        ks.append(np.asarray(k_cur[:, h, :], dtype=np.float64))
        vs.append(np.asarray(v_cur[:, h, :], dtype=np.float64))
    for c in idx_ih:
        ks.append(np.asarray(k_hist[int(c), :, h, :], dtype=np.float64))
        vs.append(np.asarray(v_hist[int(c), :, h, :], dtype=np.float64))
    if not ks:
        return np.zeros((0, dh)), np.zeros((0, dh))
    return np.concatenate(ks, axis=0), np.concatenate(vs, axis=0)


def softmax_attention(Q: np.ndarray, K: np.ndarray, V: np.ndarray, scale: float):
    """O = softmax(scale Q K^T) V and lse = log sum exp(scale Q K^T), per query row."""
    logits = scale * (Q @ K.T)
    mx = logits.max(axis=1, keepdims=True)
    p = np.exp(logits - mx)
    den = p.sum(axis=1, keepdims=True)
    return (p @ V) / den, (mx + np.log(den))[:, 0]


def anchor_attention(q, k_hist, v_hist, idx, scale, k_cur=None, v_cur=None,
                     rows=None, block=256):
    """q [n_a, S, H, dh]; k_hist, v_hist [M, Bv, H, dh]; idx [n_a, H, k_eff];
    k_cur, v_cur [N_0, H, dh] or None.

    Returns (O [n_a, S, H, dh], lse [n_a, H, S]) in float64.  With `rows` =
    list of (i, h, s) only those query rows are computed (others stay zero),
    for sampled checks at sizes where the full oracle is too slow.
    """
    n_a, S, H, dh = q.shape
    O = np.zeros((n_a, S, H, dh), dtype=np.float64)
    L = np.zeros((n_a, H, S), dtype=np.float64)
    if rows is not None:
        want = {}
        for (i, h, s) in rows:
            want.setdefault((int(i), int(h)), []).append(int(s))
    for i in range(n_a):
        for h in range(H):
            if rows is not None and (i, h) not in want:
                continue
            K, V = gather_kv(k_hist, v_hist, idx[i, h], h, k_cur, v_cur)
            srows = np.arange(S) if rows is None else np.array(sorted(set(want[(i, h)])))
            for b0 in range(0, len(srows), block):
                sel = srows[b0:b0 + block]
                Q = np.asarray(q[i, sel, h, :], dtype=np.float64)
                o, lse = softmax_attention(Q, K, V, scale)
                O[i, sel, h, :] = o
                L[i, h, sel] = lse
    return O, L
