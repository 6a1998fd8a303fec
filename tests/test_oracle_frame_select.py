"""Pins for the frame-selection oracle (oracle/frame_select.py) against what the
paper and arithmetic fix: closed-form RMS values, the end points and invariances
of the min-max normalisation (App. A.1), the rule for an absent control branch,
ages and H_cov worked by hand (eq:debt), the coverage interleaving that debt
alone produces (worked by hand), the tie rule (brute force over subsets) and
eq:score's two cases.  The pins are plain functions so that
tests/test_oracle_mutations.py can plant mistakes and show that one catches
each."""
import numpy as np
import pytest

from oracle import frame_select as FS


def rng(seed=0):
    return np.random.default_rng(seed)


def pin_rms_closed_form(mod=FS):
    """A frame holding the constant c has RMS |c|; a frame of +-a has RMS a;
    RMS over spatial and channel coordinates together."""
    x = np.zeros((3, 4, 5, 6))
    x[0] = -2.5
    x[1] = 3.0 * np.where(rng(1).random((4, 5, 6)) < 0.5, -1.0, 1.0)
    x[2, :, :, :3] = 4.0          # half the channels at 4: RMS = 4 / sqrt(2)
    r = mod.response_rms(x)
    assert np.allclose(r, [2.5, 3.0, 4.0 / np.sqrt(2.0)], rtol=0, atol=1e-12)


def pin_normalize(mod=FS):
    """The weakest frame maps to 0 and the strongest to (max-min)/(max-min+eps);
    a constant response contributes zero; positive affine maps of r leave Norm
    unchanged up to the stabiliser."""
    r = np.array([0.7, 2.5, 1.1, 0.3, 2.0], dtype=np.float32)
    n = mod.normalize(r)
    assert n[3] == 0.0 and abs(n[1] - 1.0) < 1e-6
    assert np.all((n >= 0) & (n < 1.0 + 1e-7))
    assert np.allclose(n, (r - 0.3) / (2.2 + 1e-8), rtol=0, atol=1e-6)
    assert np.all(mod.normalize(np.full(4, 3.25, dtype=np.float32)) == 0.0)
    assert np.allclose(mod.normalize(4.0 * r + 7.0), n, rtol=0, atol=1e-6)


def pin_sensitivity_branches(mod=FS):
    """d is the mean of Norm over the branches present; an absent branch is left
    out (one camera branch alone gives its own Norm, not half of it); no branch
    gives no sensitivity."""
    r1 = np.array([1.0, 3.0, 2.0, 5.0], dtype=np.float32)
    r2 = np.array([4.0, 4.5, 1.0, 2.0], dtype=np.float32)
    n1, n2 = mod.normalize(r1), mod.normalize(r2)
    assert np.array_equal(mod.sensitivity([r1, None]), n1)
    assert np.array_equal(mod.sensitivity([None, r2]), n2)
    assert np.allclose(mod.sensitivity([r1, r2]), (n1 + n2) / 2, rtol=0, atol=1e-7)
    assert mod.sensitivity([None, None]) is None
    d = mod.sensitivity([r1, r2])
    assert np.all((d >= 0) & (d <= 1))


def pin_ages_and_hcov(mod=FS):
    """eq:debt by hand: a dense block (all anchors) resets every age; skipped
    frames age by one per block; H_cov = ceil(N_cur / K_f)."""
    h = mod.update_ages(None, range(6), 6)
    assert list(h) == [0] * 6
    h = mod.update_ages(h, [0, 3], 6)
    assert list(h) == [0, 1, 1, 0, 1, 1]
    h = mod.update_ages(h, [1, 5], 6)
    assert list(h) == [1, 0, 2, 1, 2, 0]
    assert np.allclose(mod.coverage_debt([0, 1, 2, 4], 10, 5), [0, 0.5, 1.0, 2.0])
    assert np.allclose(mod.coverage_debt([3, 4], 10, 3), [0.75, 1.0])    # ceil(10/3) = 4
    assert np.allclose(mod.coverage_debt([1, 3], 4, 2), [0.5, 1.5])


def _debt_only_schedule(mod, n, k, blocks):
    h, anchors, out = None, list(range(n)), []
    for _ in range(blocks):
        anchors, h, _, _ = mod.select_next([None, None], h if h is not None else np.zeros(n), anchors, k)
        out.append(anchors)
    return out


def pin_debt_only_interleaves(mod=FS):
    """Without fresh control responses the score is lambda_cov D alone: after the
    dense first block every age is 0 and the tie rule picks the lowest indices;
    the debt then rotates the anchors through the chunk (worked by hand)."""
    assert _debt_only_schedule(mod, 10, 5, 4) == [[0, 1, 2, 3, 4], [5, 6, 7, 8, 9],
                                                   [0, 1, 2, 3, 4], [5, 6, 7, 8, 9]]
    assert _debt_only_schedule(mod, 4, 2, 3) == [[0, 1], [2, 3], [0, 1]]
    # N = 10, K = 3 (H_cov = 4): ages after each block decide the next anchors
    assert _debt_only_schedule(mod, 10, 3, 5) == [[0, 1, 2], [3, 4, 5], [6, 7, 8], [0, 1, 9],
                                                  [2, 3, 4]]


def pin_score_cases(mod=FS):
    """eq:score: with a fresh response S = d + lambda D, without one S = lambda D."""
    d = np.array([0.1, 0.9, 0.4], dtype=np.float32)
    debt = np.array([0.5, 0.0, 1.5], dtype=np.float32)
    assert np.allclose(mod.scores(d, debt, 0.5), [0.35, 0.9, 1.15], rtol=0, atol=1e-7)
    assert np.allclose(mod.scores(None, debt, 0.5), [0.25, 0.0, 0.75], rtol=0, atol=1e-7)
    assert np.allclose(mod.scores(d, debt, 0.0), d, rtol=0, atol=0)


def pin_topk_ties_bruteforce(mod=FS):
    """TopK with ties by increasing frame index equals the brute-force best
    subset with the lexicographically smallest index set among ties."""
    g = rng(7)
    for n, k in ((5, 2), (7, 3), (8, 5), (6, 6)):
        for _ in range(20):
            s = g.integers(0, 4, size=n).astype(np.float32) / 4   # many exact ties
            assert mod.topk_frames(s, k) == mod.brute_topk(s, k), (s, k)


def pin_strong_response_wins(mod=FS):
    """lambda_cov = 0: the anchors are the frames with the strongest control
    response (scaled copies of one field, both branches agreeing)."""
    base = rng(3).standard_normal((4, 4, 8))
    scale = np.array([0.5, 3.0, 1.0, 2.5, 0.2, 4.0])
    delta = scale[:, None, None, None] * base[None]
    a, _, s, _ = mod.select_next([delta, 0.5 * delta], np.zeros(6), range(6), 3, lambda_cov=0.0)
    assert a == [1, 3, 5]
    assert s[5] == max(s) and s[4] == 0.0


def pin_float32_against_exact(mod=FS):
    """The float32 decision pipeline against the float64 definition (no rounding
    between steps): scores within fp32 rounding, and the same anchors wherever the
    exact K-th / (K+1)-th gap is clear of it."""
    rng = np.random.default_rng(77)
    for trial in range(40):
        n_cur = int(rng.integers(2, 12))
        k_f = int(rng.integers(1, n_cur + 1))
        cam = rng.standard_normal((n_cur, 6, 5)) * rng.uniform(0.3, 3.0, (n_cur, 1, 1))
        act = rng.standard_normal((n_cur, 6, 5)) * rng.uniform(0.3, 3.0, (n_cur, 1, 1))
        deltas = [cam, act if trial % 3 else None]
        h_prev = rng.integers(0, 4, n_cur)
        prev = sorted(rng.choice(n_cur, size=max(1, n_cur // 2), replace=False).tolist())
        anchors, h, s32, _ = mod.select_next(deltas, h_prev, prev, k_f)
        ex = FS.scores_exact(deltas, h, k_f)
        assert np.max(np.abs(s32.astype(np.float64) - ex)) <= 1e-6, trial
        srt = np.sort(ex)[::-1]
        if k_f == n_cur or srt[k_f - 1] - srt[k_f] > 1e-5:
            want = sorted(sorted(range(n_cur), key=lambda i: (-ex[i], i))[:k_f])
            assert anchors == want, (trial, anchors, want)


PINS = [pin_float32_against_exact, pin_rms_closed_form, pin_normalize, pin_sensitivity_branches, pin_ages_and_hcov,
        pin_debt_only_interleaves, pin_score_cases, pin_topk_ties_bruteforce,
        pin_strong_response_wins]


@pytest.mark.parametrize("pin", PINS, ids=[p.__name__ for p in PINS])
def test_pin(pin):
    pin()
