"""Pins of the reconstruction-coupled routing oracle (oracle/coupled.py) against
what the paper and the mathematics fix, independently of the oracle's own code
paths: closed-form coefficients (eq:abcclosed), hand-derived boundary sums
(eq:boundarycoeff), the exact single-block omission identity
(eq:omissionexact), the objective / gain identity J = const - sum x G (App. B
retain gains), brute-force single-anchor optimality of TopK(G), strict descent
and termination of Algorithm 1, and a hand-worked coupling example."""
from fractions import Fraction

import math

import numpy as np
import pytest

from oracle import coupled as OC


# ---------------------------------------------------------------------------
# coefficients
# ---------------------------------------------------------------------------
@pytest.mark.parametrize("n", list(range(1, 13)))
def test_interval_coeffs_closed_form(n):
    """eq:abc sums equal the closed forms of eq:abcclosed for integer gaps
    (A = B = (n-1)(2n-1)/(6n), C = (n^2-1)/(6n)); zero for adjacent anchors."""
    A, B, C = OC.interval_coeffs(7, 7 + n)
    assert A == pytest.approx((n - 1) * (2 * n - 1) / (6 * n), abs=1e-13)
    assert B == pytest.approx((n - 1) * (2 * n - 1) / (6 * n), abs=1e-13)
    assert C == pytest.approx((n * n - 1) / (6 * n), abs=1e-13)


def test_boundary_coeffs_hand_example():
    """Anchors {2, 5} in 9 frames.  Left: t = 0, 1 from (2, 5), alpha = -2/3, -1/3;
    right: t = 6, 7, 8 from (2, 5), alpha = 4/3, 5/3, 2 (eq:boundarycoeff, absolute
    cross term).  Values derived by hand as fractions."""
    bc = OC.boundary_coeffs([2, 5], 9)
    a, b, A, B, C = bc["L"]
    assert (a, b) == (2, 5)
    assert A == pytest.approx(float(Fraction(41, 9)))
    assert B == pytest.approx(float(Fraction(5, 9)))
    assert C == pytest.approx(float(Fraction(14, 9)))
    a, b, A, B, C = bc["R"]
    assert (a, b) == (2, 5)
    assert A == pytest.approx(float(Fraction(14, 9)))
    assert B == pytest.approx(float(Fraction(77, 9)))
    assert C == pytest.approx(float(Fraction(32, 9)))


def test_boundary_empty_sides_and_pairs():
    assert OC.boundary_coeffs([0, 3, 7], 8) == {}
    bc = OC.boundary_coeffs([1, 3, 6], 10)
    assert set(bc) == {"L", "R"}
    assert bc["L"][:2] == (1, 3) and bc["R"][:2] == (3, 6)


# ---------------------------------------------------------------------------
# omission proxy
# ---------------------------------------------------------------------------
def _stats(seed, n_a=3, M=6, dh=8, D=12):
    rng = np.random.default_rng(seed)
    qb = rng.standard_normal((n_a, dh))
    kb = rng.standard_normal((M, dh))
    vb = rng.standard_normal((M, dh))
    P = rng.standard_normal((D, dh))
    return qb, kb, vb, P


@pytest.mark.parametrize("seed", [0, 1, 2])
def test_omission_exact_identity(seed):
    """Without the stabiliser, delta_{i,m} is exactly the change of the pooled output
    when block m is dropped and the rest renormalised (eq:omissionexact)."""
    qb, kb, vb, P = _stats(seed)
    scale = 0.7
    _, delta = OC.omission(qb, kb, vb, P, scale, eps=0.0)
    _, _, o_bar = OC.pooled_stats(qb, kb, vb, scale)
    for i in range(qb.shape[0]):
        for m in range(kb.shape[0]):
            want = OC.drop_block_output(qb, kb, vb, scale, i, m) - o_bar[i]
            assert np.allclose(delta[i, m], want, atol=1e-12, rtol=1e-10)


def test_omission_projection_norm():
    """u = ||P delta||^2: columns of P orthonormal -> ||delta||^2; P scaled by 3 -> 9x."""
    qb, kb, vb, _ = _stats(5, D=20)
    rng = np.random.default_rng(9)
    Q, _ = np.linalg.qr(rng.standard_normal((20, 8)))
    u, delta = OC.omission(qb, kb, vb, Q, 1.0)
    assert np.allclose(u, (delta ** 2).sum(axis=2), rtol=1e-12)
    u3, _ = OC.omission(qb, kb, vb, 3.0 * Q, 1.0)
    assert np.allclose(u3, 9.0 * u, rtol=1e-12)


def test_omission_stabiliser_only_scales():
    """delta with eps > 0 is delta(eps = 0) times (1 - pi)/(1 - pi + eps)."""
    qb, kb, vb, P = _stats(3)
    _, pi, _ = OC.pooled_stats(qb, kb, vb, 1.0)
    _, d0 = OC.omission(qb, kb, vb, P, 1.0, eps=0.0)
    _, d1 = OC.omission(qb, kb, vb, P, 1.0, eps=0.05)
    assert np.allclose(d1, d0 * ((1 - pi) / (1 - pi + 0.05))[:, :, None], rtol=1e-12)


# ---------------------------------------------------------------------------
# objective, gains, best responses
# ---------------------------------------------------------------------------
LAYOUTS = [((0, 3), 4), ((2, 5), 9), ((0, 3, 7), 8), ((1, 4, 6, 11), 14), ((0, 1, 5), 9)]


@pytest.mark.parametrize("anchors,n_frames", LAYOUTS)
def test_gain_identity(anchors, n_frames):
    """J(x with row i set to y) = J(x with row i empty) - sum_m y_m G_{i,m} for any
    y, with the other rows fixed: the gains are the objective's exact linear
    coefficients in one anchor's mask (App. B, retain gains)."""
    rng = np.random.default_rng(len(anchors) * 31 + n_frames)
    n_a, M = len(anchors), 7
    u = rng.gamma(1.0, 1.0, (n_a, M))
    for trial in range(6):
        x = (rng.random((n_a, M)) < 0.4).astype(float)
        for i in range(n_a):
            G = OC.gains(i, x, u, anchors, n_frames, l_anc=1.3, l_rec=0.7)
            x0 = x.copy()
            x0[i] = 0.0
            J0 = OC.objective(x0, u, anchors, n_frames, l_anc=1.3, l_rec=0.7)
            y = (rng.random(M) < 0.5).astype(float)
            x1 = x.copy()
            x1[i] = y
            J1 = OC.objective(x1, u, anchors, n_frames, l_anc=1.3, l_rec=0.7)
            assert J1 == pytest.approx(J0 - float((y * G).sum()), rel=1e-12, abs=1e-12)


@pytest.mark.parametrize("anchors,n_frames", LAYOUTS[:4])
def test_topk_gain_is_single_anchor_optimum(anchors, n_frames):
    """TopK(G) minimises J over every K-subset of one anchor's blocks (brute force)."""
    rng = np.random.default_rng(11)
    n_a, M, k = len(anchors), 6, 2
    u = rng.gamma(1.0, 1.0, (n_a, M))
    x = np.zeros((n_a, M))
    for i in range(n_a):
        x[i, rng.choice(M, k, replace=False)] = 1.0
    for i in range(n_a):
        G = OC.gains(i, x, u, anchors, n_frames)
        J_bf, sub = OC.brute_force_best_row(i, x, u, anchors, n_frames, k)
        y = x.copy()
        y[i] = 0.0
        y[i, OC.topk_set(G, k)] = 1.0
        assert OC.objective(y, u, anchors, n_frames) == pytest.approx(J_bf, rel=1e-12)


@pytest.mark.parametrize("seed", [0, 1, 2, 3])
def test_refine_descent_budget_termination(seed):
    """Every accepted change lowers J by exactly the gain difference; every anchor
    keeps exactly K blocks; run to convergence, the masks are coordinate-wise
    optimal (no single-anchor replacement improves J, by brute force)."""
    rng = np.random.default_rng(seed)
    anchors, n_frames = (1, 4, 6, 11), 14
    n_a, M, k = len(anchors), 7, 3
    u = rng.gamma(0.7, 1.0, (n_a, M))
    trace = []
    x = OC.refine(u, anchors, n_frames, k, passes=50, trace=trace)
    assert (x.sum(axis=1) == k).all()
    xs = np.zeros((n_a, M))
    for i in range(n_a):
        xs[i, OC.topk_set(u[i], k)] = 1.0
    J = OC.objective(xs, u, anchors, n_frames)
    for t in trace:
        assert t["J"] == pytest.approx(J, rel=1e-12)
        if t["accepted"]:
            xs[t["row"]] = 0.0
            xs[t["row"], t["new"]] = 1.0
            J_new = OC.objective(xs, u, anchors, n_frames)
            assert J_new == pytest.approx(J - (t["g_new"] - t["g_old"]), rel=1e-12)
            assert J_new < J
            J = J_new
    assert np.array_equal(xs, x)
    assert not any(t["accepted"] for t in trace[-n_a:])   # a full pass without change
    for i in range(n_a):
        J_bf, _ = OC.brute_force_best_row(i, x, u, anchors, n_frames, k)
        assert OC.objective(x, u, anchors, n_frames) <= J_bf * (1 + 1e-9) + 1e-12


def test_refine_zero_passes_is_independent_topk():
    rng = np.random.default_rng(4)
    u = rng.gamma(1.0, 1.0, (3, 9))
    x = OC.refine(u, (0, 3, 7), 8, 2, passes=0)
    for i in range(3):
        assert [m for m in range(9) if x[i, m]] == OC.topk_set(u[i], 2)


def test_coupling_hand_example():
    """Anchors at frames 0 and 3 of 4 (no boundary frames), M = 3, K = 1,
    u_0 = (1, 0.9, 0), u_1 = (0, 0.9, 1); A = B = 5/9, C = 4/9 (gap 3).
    Independent TopK keeps block 0 for anchor 0 and block 2 for anchor 1.  Anchor
    0's gains with anchor 1 on block 2: G = (1 + 5/9, 0.9 + 0.5 + (8/9) 0.9, 0)
    = (1.5556, 2.2, 0): it moves to block 1 (shared evidence with anchor 1's
    second-best block); anchor 1's gains then favour keeping block 2
    (1 + 5/9 > 0.9 + 0.5).  Worked by hand from eq:gain."""
    u = np.array([[1.0, 0.9, 0.0], [0.0, 0.9, 1.0]])
    trace = []
    x = OC.refine(u, (0, 3), 4, 1, passes=2, trace=trace)
    assert x.tolist() == [[0.0, 1.0, 0.0], [0.0, 0.0, 1.0]]
    G0 = trace[0]["G"]
    assert G0 == pytest.approx([1.0 + 5 / 9, 0.9 + 0.5 + 8 / 9 * 0.9, 0.0], abs=1e-12)
    assert [t["accepted"] for t in trace] == [True, False, False, False]
    assert [t["row"] for t in trace] == [0, 1, 1, 0]     # forward, then backward


def test_pooled_softmax_hand_example():
    """eq:omission's pooled attention by hand: q_bar = (1, 0) and (0, 2), k_bar =
    (1, 0) and (0, 1), scale 1/2, so the scores are (1/2, 0) and (0, 1) and
    pi = (e^(1/2), 1) / (e^(1/2) + 1) and (1, e) / (1 + e); o_bar = pi v_bar."""
    qb = np.array([[1.0, 0.0], [0.0, 2.0]])
    kb = np.array([[1.0, 0.0], [0.0, 1.0]])
    vb = np.array([[3.0, -1.0], [0.5, 2.0]])
    s, pi, o_bar = OC.pooled_stats(qb, kb, vb, 0.5)
    e = math.exp(0.5)
    want = np.array([[e / (e + 1.0), 1.0 / (e + 1.0)], [1.0 / (1.0 + math.e), math.e / (1.0 + math.e)]])
    assert s == pytest.approx(np.array([[0.5, 0.0], [0.0, 1.0]]), abs=1e-15)
    assert pi == pytest.approx(want, abs=1e-15)
    assert o_bar == pytest.approx(want @ vb, abs=1e-14)


def _first_visit(x):
    """The hand example with u_0[1] = x: gains, improvement, J and decision of
    Algorithm 1's first row visit (anchor 0)."""
    u = np.array([[1.0, x, 0.0], [0.0, 0.9, 1.0]])
    trace = []
    OC.refine(u, (0, 3), 4, 1, passes=1, trace=trace)
    t = trace[0]
    return t["g_new"] - t["g_old"], t["J"], t["accepted"]


def test_refine_acceptance_threshold():
    """Algorithm 1 accepts a row's new set only when its gain improvement exceeds
    tol * max(J, 1e-8) (tab:config: tol = 1e-6).  u_0[1] is set by bisection so
    that the improvement is 0.5 or 2 times tol * J (J is about 2.8 here, so the
    first also exceeds tol itself): rejected, then accepted."""
    tol = 1e-6
    for factor, want in ((0.5, False), (2.0, True)):
        lo, hi = 0.5, 0.6                        # no improvement at 0.5, 0.03 at 0.6
        for _ in range(80):
            mid = 0.5 * (lo + hi)
            d, J, _ = _first_visit(mid)
            if d > factor * tol * J:
                hi = mid
            else:
                lo = mid
        d, J, accepted = _first_visit(hi)
        assert factor * tol * J < d < 1.01 * factor * tol * J
        assert d > tol                            # an absolute tol would accept both
        assert accepted == want, (factor, d, J)


def test_refine_stops_after_a_pass_without_change():
    """The hand example changes one row in the first pass and none in the second,
    so Algorithm 1 ends there however many passes it may take."""
    u = np.array([[1.0, 0.9, 0.0], [0.0, 0.9, 1.0]])
    trace = []
    OC.refine(u, (0, 3), 4, 1, passes=6, trace=trace)
    assert len(trace) == 4 and [t["accepted"] for t in trace] == [True, False, False, False]


def test_route_coupled_shapes_and_bypass():
    """Per-head routing end to end: indices ascending, exactly k_eff per (anchor, head);
    topk >= M keeps every block."""
    rng = np.random.default_rng(2)
    n_a, S, H, dh, M, Bv, D = 3, 5, 2, 4, 6, 3, 8
    q = rng.standard_normal((n_a, S, H, dh))
    k = rng.standard_normal((M, Bv, H, dh))
    v = rng.standard_normal((M, Bv, H, dh))
    w_o = rng.standard_normal((D, H * dh))
    u, idx, k_eff = OC.route_coupled(q, k, v, w_o, (0, 3, 7), 8, 2, 0.5)
    assert k_eff == 2 and idx.shape == (n_a, H, 2)
    assert (np.diff(idx, axis=2) > 0).all()
    _, idx_all, k_all = OC.route_coupled(q, k, v, w_o, (0, 3, 7), 8, 10, 0.5)
    assert k_all == M and (idx_all == np.arange(M)).all()


# ---------------------------------------------------------------------------
# pins as functions of an oracle module (used by test_oracle_mutations.py)
# ---------------------------------------------------------------------------
def _on(mod, fn, *args):
    global OC
    saved, OC = OC, mod
    try:
        fn(*args)
    finally:
        OC = saved


def pin_closed_form(mod):
    for n in (1, 2, 3, 7):
        _on(mod, test_interval_coeffs_closed_form, n)


def pin_boundary(mod):
    _on(mod, test_boundary_coeffs_hand_example)


def pin_omission(mod):
    _on(mod, test_omission_exact_identity, 0)
    _on(mod, test_omission_projection_norm)
    _on(mod, test_pooled_softmax_hand_example)


def pin_gain_identity(mod):
    for layout in LAYOUTS:
        _on(mod, test_gain_identity, *layout)


def pin_refine(mod):
    _on(mod, test_coupling_hand_example)
    _on(mod, test_refine_descent_budget_termination, 0)
    _on(mod, test_refine_acceptance_threshold)
    _on(mod, test_refine_stops_after_a_pass_without_change)


PINS = [pin_closed_form, pin_boundary, pin_omission, pin_gain_identity, pin_refine]
