"""Float64 oracle for reconstruction-coupled historical routing.

TEST INFRASTRUCTURE ONLY (see the package docstring).

Sec. 4.4 (eq:pooled, eq:omission, eq:abc, eq:risk, eq:objective, eq:topk) and
App. B (eq:omissionexact, eq:abcclosed, eq:boundarycoeff, eq:boundaryrisk,
eq:gain, eq:boundarygain, Algorithm 1, tab:config routing weights / stopping):

* pooled statistics per head: s_{i,m} = scale q_bar_i . k_bar_m,
  pi_{i,.} = softmax over the M blocks, o_bar_i = sum_m pi_{i,m} v_bar_m;
* one-block omission proxy: delta_{i,m} = pi/(1 - pi + eps) (o_bar_i - v_bar_m),
  u_{i,m} = ||P delta_{i,m}||^2 with P = the head's slice of W_O;
* interval coefficients A, B, C of each adjacent anchor pair over the skipped
  frames strictly between them, boundary coefficients A_q, B_q, C_q (absolute
  cross term) for the frames before the first / after the last anchor,
  extrapolated from the first / last pair;
* objective J(x) = l_anc sum (1-x) u + l_rec [sum_pairs R + R_bdry] and the
  retain gains G_{i,m} of one anchor with its neighbours' masks fixed;
* Algorithm 1: masks start as TopK(u); L_s directional passes (forward, then
  backward, ...) replace an anchor's mask by TopK(G) when that lowers J by more
  than tol * max(J, 1e-8); a pass with no change stops early.

Readings where the paper leaves a choice: the optimisation is per head (masks of
different heads never interact), so J and its acceptance threshold are the
head's own; TopK orders (value descending, block index ascending) and reports
ascending block indices; the omission stabiliser eps is 1e-8 unless given; the
candidate sets are all M blocks (tab:config M_c = M).
"""
from __future__ import annotations

import itertools

import numpy as np


# ---------------------------------------------------------------------------
# pooled statistics and the omission proxy (eq:pooled, eq:omission)
# ---------------------------------------------------------------------------
def pooled_stats(qb, kb, vb, scale):
    """qb [n_a, dh], kb, vb [M, dh] (one head) -> s [n_a, M], pi [n_a, M], o_bar [n_a, dh]."""
    qb, kb, vb = (np.asarray(x, dtype=np.float64) for x in (qb, kb, vb))
    s = scale * (qb @ kb.T)
    e = np.exp(s - s.max(axis=1, keepdims=True))
    pi = e / e.sum(axis=1, keepdims=True)
    o_bar = pi @ vb
    return s, pi, o_bar


def omission(qb, kb, vb, P, scale, eps=1e-8):
    """u [n_a, M] and delta [n_a, M, dh] of one head; P [D, dh] maps a head output
    to the residual (the head's columns of W_O)."""
    _, pi, o_bar = pooled_stats(qb, kb, vb, scale)
    vb = np.asarray(vb, dtype=np.float64)
    P = np.asarray(P, dtype=np.float64)
    coef = pi / (1.0 - pi + eps)
    delta = coef[:, :, None] * (o_bar[:, None, :] - vb[None, :, :])
    proj = np.einsum("dk,imk->imd", P, delta)
    u = (proj ** 2).sum(axis=2)
    return u, delta


def drop_block_output(qb, kb, vb, scale, i, m):
    """Pooled output of anchor i with block m removed and the rest renormalised
    (the left side of eq:omissionexact), computed by actually dropping it."""
    s, _, _ = pooled_stats(qb, kb, vb, scale)
    keep = [j for j in range(s.shape[1]) if j != m]
    sk = s[i, keep]
    w = np.exp(sk - sk.max())
    w /= w.sum()
    return w @ np.asarray(vb, dtype=np.float64)[keep]


# ---------------------------------------------------------------------------
# interval and boundary coefficients (eq:abc, eq:boundarycoeff)
# ---------------------------------------------------------------------------
def interval_coeffs(a, b):
    """A, B, C of the pair (a, b) over the skipped frames a < t < b."""
    A = B = C = 0.0
    for t in range(a + 1, b):
        al = (t - a) / (b - a)
        A += (1.0 - al) ** 2
        B += al ** 2
        C += al * (1.0 - al)
    return A, B, C


def boundary_coeffs(anchors, n_frames):
    """{'L': (a, b, A, B, C), 'R': (...)} for the frames before the first anchor
    (pair of the first two anchors) and after the last (pair of the last two);
    a side with no frames is absent."""
    an = [int(x) for x in anchors]
    out = {}
    if len(an) < 2:
        return out
    sides = {"L": (an[0], an[1], range(0, an[0])),
             "R": (an[-2], an[-1], range(an[-1] + 1, n_frames))}
    for q, (a, b, ts) in sides.items():
        ts = list(ts)
        if not ts:
            continue
        A = B = C = 0.0
        for t in ts:
            al = (t - a) / (b - a)
            A += (1.0 - al) ** 2
            B += al ** 2
            C += abs(al * (1.0 - al))
        out[q] = (a, b, A, B, C)
    return out


# ---------------------------------------------------------------------------
# objective and gains (eq:objective, eq:risk, eq:boundaryrisk, eq:gain)
# ---------------------------------------------------------------------------
def objective(x, u, anchors, n_frames, l_anc=1.0, l_rec=1.0):
    """J of one head: x, u [n_a, M] (x binary), anchors = frame index of each row."""
    x = np.asarray(x, dtype=np.float64)
    u = np.asarray(u, dtype=np.float64)
    an = [int(a) for a in anchors]
    om = 1.0 - x
    J = l_anc * float((om * u).sum())
    rec = 0.0
    for j in range(len(an) - 1):
        A, B, C = interval_coeffs(an[j], an[j + 1])
        rec += float((A * om[j] * u[j] + B * om[j + 1] * u[j + 1]
                      + 2.0 * C * om[j] * om[j + 1] * np.sqrt(u[j] * u[j + 1])).sum())
    row = {a: r for r, a in enumerate(an)}
    for (a, b, A, B, C) in boundary_coeffs(an, n_frames).values():
        ia, ib = row[a], row[b]
        rec += float((A * om[ia] * u[ia] + B * om[ib] * u[ib]
                      + 2.0 * C * om[ia] * om[ib] * np.sqrt(u[ia] * u[ib])).sum())
    return J + l_rec * rec


def gains(i, x, u, anchors, n_frames, l_anc=1.0, l_rec=1.0):
    """Retain gains G[i, :] of anchor row i with every other row's mask fixed."""
    x = np.asarray(x, dtype=np.float64)
    u = np.asarray(u, dtype=np.float64)
    an = [int(a) for a in anchors]
    n = len(an)
    G = l_anc * u[i].copy()
    if i > 0:      # right end of the interval (l, i)
        _, B, C = interval_coeffs(an[i - 1], an[i])
        G += l_rec * (B * u[i] + 2.0 * C * (1.0 - x[i - 1]) * np.sqrt(u[i - 1] * u[i]))
    if i < n - 1:  # left end of the interval (i, r)
        A, _, C = interval_coeffs(an[i], an[i + 1])
        G += l_rec * (A * u[i] + 2.0 * C * (1.0 - x[i + 1]) * np.sqrt(u[i] * u[i + 1]))
    row = {a: r for r, a in enumerate(an)}
    for (a, b, A, B, C) in boundary_coeffs(an, n_frames).values():
        ia, ib = row[a], row[b]
        if i == ia:
            G += l_rec * (A * u[i] + 2.0 * C * (1.0 - x[ib]) * np.sqrt(u[i] * u[ib]))
        if i == ib:
            G += l_rec * (B * u[i] + 2.0 * C * (1.0 - x[ia]) * np.sqrt(u[i] * u[ia]))
    return G


def topk_set(values, k):
    """The k largest under (value descending, index ascending), as a sorted list."""
    v = [float(a) for a in values]
    order = sorted(range(len(v)), key=lambda m: (-v[m], m))
    return sorted(order[:k])


# ---------------------------------------------------------------------------
# Algorithm 1
# ---------------------------------------------------------------------------
def refine(u, anchors, n_frames, k, l_anc=1.0, l_rec=1.0, passes=2, tol=1e-6, trace=None):
    """Masks [n_a, M] (0/1) of one head after Algorithm 1; `trace` (a list) gets
    one dict per anchor visit: pass, row, old / new gain sums, J before, accepted."""
    u = np.asarray(u, dtype=np.float64)
    n_a, M = u.shape
    k = min(int(k), M)
    x = np.zeros((n_a, M))
    for i in range(n_a):
        x[i, topk_set(u[i], k)] = 1.0
    for s in range(passes):
        changed = False
        rows = range(n_a) if s % 2 == 0 else range(n_a - 1, -1, -1)
        for i in rows:
            G = gains(i, x, u, anchors, n_frames, l_anc, l_rec)
            new = topk_set(G, k)
            old = [m for m in range(M) if x[i, m] == 1.0]
            g_new = float(sum(G[m] for m in new))
            g_old = float(sum(G[m] for m in old))
            J = objective(x, u, anchors, n_frames, l_anc, l_rec)
            accept = (g_new - g_old) > tol * max(J, 1e-8)
            if trace is not None:
                trace.append({"pass": s, "row": i, "g_old": g_old, "g_new": g_new, "J": J,
                              "accepted": accept, "G": G.copy(), "new": new})
            if accept:
                x[i, :] = 0.0
                x[i, new] = 1.0
                changed = True
        if not changed:
            break
    return x


def route_coupled(q, k_hist, v_hist, w_o, anchors, n_frames, topk, scale, l_anc=1.0,
                  l_rec=1.0, passes=2, tol=1e-6, eps=1e-8):
    """Per head: pooled means (token means, as in route.pooled_means), omission
    proxy with P = W_O[:, h dh:(h+1) dh], Algorithm 1.  Returns (u [n_a,H,M],
    idx int32 [n_a,H,k_eff] ascending, k_eff)."""
    q = np.asarray(q, dtype=np.float64)
    k_hist = np.asarray(k_hist, dtype=np.float64)
    v_hist = np.asarray(v_hist, dtype=np.float64)
    w_o = np.asarray(w_o, dtype=np.float64)
    n_a, _, H, dh = q.shape
    M = k_hist.shape[0]
    k_eff = min(int(topk), M)
    qb = q.mean(axis=1)          # [n_a, H, dh]
    kb = k_hist.mean(axis=1)     # [M, H, dh]
    vb = v_hist.mean(axis=1)
    u = np.zeros((n_a, H, M))
    idx = np.zeros((n_a, H, k_eff), dtype=np.int32)
    for h in range(H):
        P = w_o[:, h * dh:(h + 1) * dh]
        u[:, h, :], _ = omission(qb[:, h], kb[:, h], vb[:, h], P, scale, eps)
        if k_eff == 0:
            continue
        x = refine(u[:, h, :], anchors, n_frames, k_eff, l_anc, l_rec, passes, tol)
        for i in range(n_a):
            idx[i, h] = [m for m in range(M) if x[i, m] == 1.0]
    return u, idx, k_eff


def brute_force_best_row(i, x, u, anchors, n_frames, k, l_anc=1.0, l_rec=1.0):
    """min over every k-subset of anchor row i (others fixed) of J: (J, subset)."""
    x = np.asarray(x, dtype=np.float64)
    M = x.shape[1]
    best = None
    for sub in itertools.combinations(range(M), k):
        y = x.copy()
        y[i, :] = 0.0
        y[i, list(sub)] = 1.0
        J = objective(y, u, anchors, n_frames, l_anc, l_rec)
        if best is None or J < best[0] - 1e-15:
            best = (J, list(sub))
    return best
