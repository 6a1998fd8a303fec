"""Pins for the PAR oracle against what the paper and mathematics fix.

Each pin checks the oracle against something other than itself: a brute-force
double-sum DFT, numpy's FFT (an independent library), Parseval, closed-form
special cases of eq:fcpasm (g = 0 linear interpolation / extrapolation, g = 1
exact translation eq:exacttranslation), the endpoint identity, the
real-valuedness of the reconstruction (App. A.2) and invariances.  The pins are
plain functions so that tests/test_oracle_mutations.py can plant mistakes in
the oracle and show that a pin catches each one.
"""
import math

import numpy as np
import pytest

from oracle import par as P
from gen.workloads import fourier_shift


def rng(seed=0):
    return np.random.default_rng(seed)


def brute_rfft2(x):
    """Double-sum DFT with scalar cos/sin, orthonormal, stored half-spectrum."""
    hp, wp = x.shape[:2]
    out = np.zeros((hp, wp // 2 + 1) + x.shape[2:], dtype=np.complex128)
    for ky in range(hp):
        for kx in range(wp // 2 + 1):
            acc = 0
            for y in range(hp):
                for xx in range(wp):
                    ang = -2 * math.pi * (ky * y / hp + kx * xx / wp)
                    acc = acc + x[y, xx] * complex(math.cos(ang), math.sin(ang))
            out[ky, kx] = acc / math.sqrt(hp * wp)
    return out


# ---------------------------------------------------------------------------
# pins (functions so mutations can be planted)
# ---------------------------------------------------------------------------

def pin_dft_bruteforce(mod=P):
    for (hp, wp) in [(4, 4), (6, 8), (8, 4), (5, 3), (8, 8)]:
        x = rng(hp * 10 + wp).standard_normal((hp, wp, 3))
        np.testing.assert_allclose(mod.rfft2_ortho(x), brute_rfft2(x), rtol=0, atol=1e-12)


def pin_dft_numpy(mod=P):
    for (hp, wp) in [(8, 8), (6, 8), (8, 4), (6, 4), (4, 8), (7, 5), (1, 1), (2, 8)]:
        x = rng(hp + 100 * wp).standard_normal((hp, wp, 4))
        ref = np.fft.rfft2(x, axes=(0, 1), norm="ortho")
        np.testing.assert_allclose(mod.rfft2_ortho(x), ref, rtol=0, atol=1e-12)
        np.testing.assert_allclose(mod.irfft2_ortho(ref, wp),
                                   np.fft.irfft2(ref, s=(hp, wp), axes=(0, 1), norm="ortho"),
                                   rtol=0, atol=1e-12)


def pin_parseval_kappa(mod=P):
    """Orthonormal transform: sum |x|^2 = sum_stored kappa |F|^2 (pins kappa too)."""
    for (hp, wp) in [(8, 8), (6, 8), (8, 4), (7, 5), (4, 6), (3, 1)]:
        x = rng(7 * hp + wp).standard_normal((hp, wp))
        F = mod.rfft2_ortho(x)
        _, _, kappa, _ = mod.bin_tables(hp, wp)
        assert abs((x ** 2).sum() - (kappa * np.abs(F) ** 2).sum()) < 1e-10


def pin_round_trip(mod=P):
    for (hp, wp) in [(8, 8), (6, 8), (8, 4), (7, 5), (1, 3)]:
        x = rng(hp * wp).standard_normal((hp, wp, 2))
        np.testing.assert_allclose(mod.irfft2_ortho(mod.rfft2_ortho(x), wp), x, atol=1e-12)


def pin_bin_kinds(mod=P):
    """Mirror bins are the conjugates of their partners; self-conjugate bins are real."""
    for (hp, wp) in [(8, 8), (6, 8), (8, 4), (7, 6), (5, 5), (4, 2)]:
        x = rng(hp + wp).standard_normal((hp, wp))
        F = mod.rfft2_ortho(x)
        kind, partner, _, nu = mod.bin_tables(hp, wp)
        for ky in range(hp):
            for kx in range(wp // 2 + 1):
                if kind[ky, kx] == mod.MIRROR:
                    py, px = partner[ky, kx]
                    assert kind[py, px] == mod.REP
                    assert abs(F[ky, kx] - np.conj(F[py, px])) < 1e-12
                    assert abs(nu[ky, kx] - nu[py, px]) < 1e-15
                elif kind[ky, kx] == mod.SELF:
                    assert abs(F[ky, kx].imag) < 1e-12
        # self-conjugate points of an even-even tile: (0,0),(H/2,0),(0,W/2),(H/2,W/2)
        n_self = int((kind == mod.SELF).sum())
        assert n_self == (1 + (hp % 2 == 0)) * (1 + (wp % 2 == 0))
        assert abs(nu.max() - 1.0) < 1e-15 or (hp == 1 and wp == 1)


def pin_nu_isotropy(mod=P):
    _, _, _, nu = mod.bin_tables(8, 8)
    for k in range(1, 5):
        assert abs(nu[k, 0] - nu[0, k]) < 1e-15
    assert nu[0, 0] == 0.0
    assert abs(nu[4, 4] - 1.0) < 1e-15


def _two_anchor(hp, wp, D, seed, shift=None, noise=0.0):
    r = rng(seed)
    a = r.standard_normal((hp, wp, D))
    if shift is None:
        b = r.standard_normal((hp, wp, D))
    else:
        b = np.roll(a, shift, axis=(0, 1)) + noise * r.standard_normal((hp, wp, D))
    return a, b


def _recon_single(a, b, alpha, prm):
    """PAR on a 2-frame buffer with anchors {0, 1}; one target with the given alpha
    is realised through a 3-frame buffer placement."""
    Hg, Wg, D = a.shape
    # place anchors so that the single skipped frame t has the requested alpha
    frac = {1 / 3: (0, 3, 1), 2 / 3: (0, 3, 2), -0.5: (2, 4, 1), 1.5: (0, 2, 3),
            0.25: (0, 4, 1), 0.5: (0, 2, 1), 1.25: (0, 4, 5), -1 / 3: (3, 6, 2)}
    key = min(frac, key=lambda k: abs(k - alpha))
    ta, tb, t = frac[key]
    n = max(ta, tb, t) + 1
    buf = np.zeros((n, Hg, Wg, D))
    buf[ta] = a
    buf[tb] = b
    out = P_mod_holder[0].par_reconstruct(buf, (ta, tb), prm)
    return out[t], key


P_mod_holder = [P]


def pin_linear_g0(mod=P):
    """g = 0: eq:fcpasm reduces to (1-alpha) R_a + alpha R_b for any alpha."""
    P_mod_holder[0] = mod
    try:
        prm = mod.ParParams(gate_mode=mod.GATE_ZERO)
        for (Hg, Wg) in [(8, 8), (14, 13), (9, 20)]:
            a, b = _two_anchor(Hg, Wg, 3, Hg * Wg)
            for alpha in (1 / 3, 2 / 3, -0.5, 1.5, 1.25):
                got, al = _recon_single(a, b, alpha, prm)
                np.testing.assert_allclose(got, (1 - al) * a + al * b, atol=1e-12)
    finally:
        P_mod_holder[0] = P


def pin_translation_ramp(mod=P):
    """g = 1 and a coherent sub-token translation (eq:shift, eq:exacttranslation):
    theta(omega) = -omega . d on reliable bins and R_hat_t = shift(R_a, alpha d),
    also for alpha outside [0, 1]."""
    P_mod_holder[0] = mod
    try:
        hp = wp = 8
        D = 5
        r = rng(3)
        F = np.fft.rfft2(r.standard_normal((hp, wp, D)), axes=(0, 1))
        F[hp // 2, :, :] = 0          # band-limit: no Nyquist row / column content
        F[:, wp // 2, :] = 0
        a = np.fft.irfft2(F, s=(hp, wp), axes=(0, 1))
        d = (0.3, -0.4)
        b = fourier_shift(a, d)
        prm = mod.ParParams(gate_mode=mod.GATE_ONE)
        st = mod.par_stats(np.stack([a, b]), (0, 1), prm)[(0, 1)][0][3]
        kind, _, _, _ = mod.bin_tables(hp, wp)
        for ky in range(hp):
            for kx in range(wp // 2 + 1):
                if not st.reliable[ky, kx] or kind[ky, kx] == mod.SELF:
                    continue
                kys = ky if 2 * ky <= hp else ky - hp
                want = -2 * math.pi * (kys * d[0] / hp + kx * d[1] / wp)
                assert abs(st.theta[ky, kx] - want) < 1e-9, (ky, kx)
        for alpha in (1 / 3, 2 / 3, -0.5, 1.5):
            got, al = _recon_single(a, b, alpha, prm)
            want = fourier_shift(a, (al * d[0], al * d[1]))
            np.testing.assert_allclose(got, want, atol=1e-10)
    finally:
        P_mod_holder[0] = P


def pin_endpoints(mod=P):
    """The anchor endpoints are reproduced exactly (alpha = 0 and alpha = 1)."""
    for (Hg, Wg) in [(8, 8), (14, 13)]:
        a, b = _two_anchor(Hg, Wg, 4, 5 + Hg, shift=(1, 2), noise=0.1)
        st = mod.par_stats(np.stack([a, b]), (0, 1), mod.ParParams())[(0, 1)]
        np.testing.assert_allclose(mod.reconstruct_frame(st, 0.0, Hg, Wg, 4), a, atol=1e-12)
        np.testing.assert_allclose(mod.reconstruct_frame(st, 1.0, Hg, Wg, 4), b, atol=1e-12)


def pin_real_valued(mod=P):
    """App. A.2: with mirrors at -theta and U = 1 on self-conjugate bins the
    full-spectrum multiplier preserves real-valuedness."""
    for (Hg, Wg, tile) in [(8, 8, 8), (14, 13, 8), (12, 10, 6)]:
        a, b = _two_anchor(Hg, Wg, 6, Hg + 3 * Wg, shift=(1, 2), noise=0.3)
        prm = mod.ParParams(tile_h=tile, tile_w=tile)
        st = mod.par_stats(np.stack([a, b]), (0, 1), prm)[(0, 1)]
        for alpha in (0.3, 1.7, -0.6):
            for (y0, hp, x0, wp), Fa, Fb, s in st:
                Fh = mod.blend(Fa, Fb, s.theta, s.gate, alpha)
                full = mod.irfft2_ortho_complex(Fh, wp)
                rms = np.sqrt((full.real ** 2).mean()) + 1e-30
                assert np.abs(full.imag).max() <= 1e-12 * max(rms, 1.0), (hp, wp, alpha)


def pin_confidence_bounds(mod=P):
    r = rng(11)
    for D in (1, 4, 64):
        a = r.standard_normal((8, 8, D))
        b = r.standard_normal((8, 8, D))
        s = mod.tile_stats(mod.rfft2_ortho(a), mod.rfft2_ortho(b), 8, 8, mod.ParParams())
        assert 0.0 <= s.conf <= 1.0
        if D == 1:
            assert s.conf > 1 - 1e-6       # one channel: |Z| = W on every bin


def pin_confidence_full_spectrum(mod=P):
    """c_p from the stored half-spectrum with kappa equals the same ratio over the
    full complex spectrum (every bin weight 1, numpy FFT), reliable non-DC bins."""
    for (hp, wp) in [(8, 8), (6, 8), (8, 4), (7, 5)]:
        r = rng(hp * 31 + wp)
        a = r.standard_normal((hp, wp, 16))
        b = np.roll(a, (1, 1), axis=(0, 1)) + 0.8 * r.standard_normal((hp, wp, 16))
        s = mod.tile_stats(mod.rfft2_ortho(a), mod.rfft2_ortho(b), hp, wp, mod.ParParams())
        Fa = np.fft.fft2(a, axes=(0, 1), norm="ortho")
        Fb = np.fft.fft2(b, axes=(0, 1), norm="ortho")
        Z = (Fb * np.conj(Fa)).sum(-1)
        W = (np.abs(Fb) * np.abs(Fa)).sum(-1)
        eta = 1e-6 * W.max() + 1e-8
        rel = (W > eta) & (np.abs(Z) > eta)
        rel[0, 0] = False
        want = np.abs(Z)[rel].sum() / (W[rel].sum() + 1e-8)
        assert abs(s.conf - want) < 1e-12


def pin_coherence_levels(mod=P):
    """Identical anchors: Z = W, theta = 0, c ~ 1 and P_t = R_a for every alpha.
    Coherent translation: c ~ 1.  Independent channels: c small (~ 1/sqrt(D))."""
    a = rng(21).standard_normal((8, 8, 32))
    s = mod.tile_stats(mod.rfft2_ortho(a), mod.rfft2_ortho(a), 8, 8, mod.ParParams())
    assert np.all(np.abs(s.theta) < 1e-14) and s.conf > 1 - 1e-9
    st = mod.par_stats(np.stack([a, a]), (0, 1), mod.ParParams())[(0, 1)]
    for alpha in (0.4, -1.0, 2.5):
        np.testing.assert_allclose(mod.reconstruct_frame(st, alpha, 8, 8, 32), a, atol=1e-12)
    b = fourier_shift(a, (0.7, 0.2))
    s2 = mod.tile_stats(mod.rfft2_ortho(a), mod.rfft2_ortho(b), 8, 8, mod.ParParams())
    assert s2.conf > 1 - 1e-9
    c = rng(22).standard_normal((8, 8, 256))
    d = rng(23).standard_normal((8, 8, 256))
    s3 = mod.tile_stats(mod.rfft2_ortho(c), mod.rfft2_ortho(d), 8, 8, mod.ParParams())
    assert s3.conf < 0.25


def pin_no_reliable_bin(mod=P):
    """Zero anchors: no reliable bin -> c_p = 0 and U = 1 (theta 0); output 0."""
    z = np.zeros((8, 8, 4))
    s = mod.tile_stats(mod.rfft2_ortho(z), mod.rfft2_ortho(z), 8, 8, mod.ParParams())
    assert s.conf == 0.0 and not s.reliable.any() and np.all(s.theta == 0)


def pin_swap_symmetry(mod=P):
    """Swapping (a, b) and alpha -> 1 - alpha gives the same reconstruction off
    the branch cut (eq:cross conjugates, eq:fcpasm exchanges its terms)."""
    a, b = _two_anchor(16, 16, 8, 77, shift=(2, -1), noise=0.5)
    prm = mod.ParParams()
    s_ab = mod.par_stats(np.stack([a, b]), (0, 1), prm)[(0, 1)]
    s_ba = mod.par_stats(np.stack([b, a]), (0, 1), prm)[(0, 1)]
    for (_, _, _, sa), (_, _, _, sb) in zip(s_ab, s_ba):
        assert np.all(np.pi - np.abs(sa.theta) > 1e-6)
    for alpha in (0.3, 1.4, -0.2):
        np.testing.assert_allclose(mod.reconstruct_frame(s_ab, alpha, 16, 16, 8),
                                   mod.reconstruct_frame(s_ba, 1 - alpha, 16, 16, 8), atol=1e-11)


def pin_channel_permutation(mod=P):
    a, b = _two_anchor(8, 8, 10, 5, shift=(0, 3), noise=0.4)
    perm = rng(9).permutation(10)
    st1 = mod.par_stats(np.stack([a, b]), (0, 1))[(0, 1)]
    st2 = mod.par_stats(np.stack([a[..., perm], b[..., perm]]), (0, 1))[(0, 1)]
    np.testing.assert_allclose(mod.reconstruct_frame(st1, 0.4, 8, 8, 10)[..., perm],
                               mod.reconstruct_frame(st2, 0.4, 8, 8, 10), atol=1e-12)


def pin_gate_shape(mod=P):
    """eq:gate consequences: g = 1/2 where c_p = tau(nu); tau(0) = tau_low and
    tau(1) = tau_high; with c_p = 1 the gate stays in [sigma(2.5), sigma(7.5)]."""
    a = rng(31).standard_normal((8, 8, 1))
    s = mod.tile_stats(mod.rfft2_ortho(a), mod.rfft2_ortho(a), 8, 8, mod.ParParams())
    sig = lambda v: 1 / (1 + math.exp(-v))
    assert abs(s.gate[0, 0] - sig((s.conf - 0.25) / 0.1)) < 1e-12
    assert abs(s.gate[4, 4] - sig((s.conf - 0.75) / 0.1)) < 1e-12
    # an interior radius: bin (2, 2) of an 8x8 tile has nu = |(2/8, 2/8)| / |(1/2, 1/2)|
    # = 1/2, so tau = 0.25 + 0.5 (1/2)^q = 0.375 with q = 2
    assert abs(s.nu[2, 2] - 0.5) < 1e-12
    assert abs(s.gate[2, 2] - sig((s.conf - 0.375) / 0.1)) < 1e-12
    assert sig(2.5) - 1e-9 <= s.gate.min() and s.gate.max() <= sig(7.5) + 1e-9
    # g = 1/2 exactly where c = tau: choose tau_low = c
    prm = mod.ParParams(tau_low=s.conf, tau_high=s.conf + 0.5)
    s2 = mod.tile_stats(mod.rfft2_ortho(a), mod.rfft2_ortho(a), 8, 8, prm)
    assert abs(s2.gate[0, 0] - 0.5) < 1e-12
    # monotone: higher frequency needs more confidence
    order = np.argsort(s.nu.ravel())
    assert np.all(np.diff(s.gate.ravel()[order]) <= 1e-15)


def pin_wrap(mod=P):
    assert mod.wrap_arg(complex(-1.0, 0.0)) == math.pi
    assert mod.wrap_arg(complex(-1.0, -0.0)) == math.pi
    assert -math.pi < mod.wrap_arg(complex(-1.0, -1e-9)) < -3.14
    assert abs(mod.wrap_arg(1j) - math.pi / 2) < 1e-15
    assert abs(mod.wrap_arg(-1j) + math.pi / 2) < 1e-15


def pin_anchor_update(mod=P):
    """eq:block, anchor case: an anchor's update is its own residual.  With
    update_anchors every anchor slot becomes x0 + R_a (accumulate) or R_a
    (write) exactly, and every skipped slot is what it is without the option;
    with K_f = N_cur every frame is an anchor."""
    n, hg, wg, d = 7, 8, 8, 3
    r = rng(41).standard_normal((n, hg, wg, d))
    x0 = rng(42).standard_normal((n, hg, wg, d))
    anchors = [1, 3, 6]
    base = mod.par_reconstruct(r, anchors, mod.ParParams(accumulate=True), out=x0)
    upd = mod.par_reconstruct(r, anchors, mod.ParParams(accumulate=True, update_anchors=True), out=x0)
    wr = mod.par_reconstruct(r, anchors, mod.ParParams(update_anchors=True), out=x0)
    for t in range(n):
        if t in anchors:
            assert np.array_equal(upd[t], x0[t] + r[t])
            assert np.array_equal(wr[t], r[t])
            assert np.array_equal(base[t], x0[t])
        else:
            assert np.array_equal(upd[t], base[t])
    allf = mod.par_reconstruct(r, list(range(n)),
                               mod.ParParams(accumulate=True, update_anchors=True), out=x0)
    assert np.array_equal(allf, x0 + r)


def pin_sites_linear_g0(mod=P):
    """With g = 0 each site's reconstruction is linear in its residual
    (eq:fcpasm), so an attention site and an FFN site sharing the anchors add up
    to one site with the summed residuals, anchors included; a skipped frame then
    gets (1 - alpha) R_a + alpha R_b summed over the sites."""
    n, hg, wg, d = 6, 8, 6, 3
    r1 = rng(51).standard_normal((n, hg, wg, d))
    r2 = rng(52).standard_normal((n, hg, wg, d))
    x0 = rng(53).standard_normal((n, hg, wg, d))
    anchors = [1, 4]
    prm = mod.ParParams(gate_mode=mod.GATE_ZERO)
    two = mod.block_sites(x0, [r1, r2], anchors, prm)
    one = mod.block_sites(x0, [r1 + r2], anchors, prm)
    assert np.allclose(two, one, rtol=0, atol=1e-12)
    s = r1 + r2
    for t, alpha in ((2, 1 / 3), (0, -1 / 3), (5, 4 / 3)):
        want = x0[t] + (1 - alpha) * s[1] + alpha * s[4]
        assert np.allclose(two[t], want, rtol=0, atol=1e-12), t
    for a in anchors:
        assert np.allclose(two[a], x0[a] + s[a], rtol=0, atol=1e-14)


def pin_reliability_threshold(mod=P):
    """App. A.2 worked by hand on a designed 8x8 tile (gen.workloads.RELIABILITY_TILE).
    max W = 4 (at DC) gives eta = 4e-6 + 1e-8.  Reliable: DC, (1,1) with
    Z = 1 + e^{i pi/3} (theta pi/6), (2,1) at W = 1.2e-5 (theta -pi/4), the column-0
    representative (2,0) (theta pi/5) and its mirror (6,0) (-pi/5), and the
    self-conjugate Nyquist point (4,0) (U = 1).  Unreliable: (3,1) (W = 3e-6 < eta),
    (1,3) (W = 1.2e-6) and (1,2), whose W = 0.02 passes but whose two channels
    cancel in Z down to 1e-8.  eq:confidence over the reliable non-DC bins:
        c = (2 sqrt(3) + 2(1.2e-5) + 1.2e-5 + 1.2e-5 + 0.25)
            / (2(2) + 2(1.2e-5) + 1.2e-5 + 1.2e-5 + 0.25 + 1e-8).
    At 1e-3 amplitude every W shrinks by 1e-6, eta = 4e-12 + 1e-8 is set by its
    absolute part, and only DC, (1,1) and (4,0) stay reliable:
        c = (2 sqrt(3) + 0.25) 1e-6 / (4.25e-6 + 1e-8)."""
    from gen.workloads import designed_tile_pair
    pi = math.pi
    cases = [
        (1.0, 4e-6 + 1e-8,
         {(0, 0): 0.0, (1, 1): pi / 6, (2, 1): -pi / 4, (2, 0): pi / 5, (6, 0): -pi / 5,
          (4, 0): 0.0},
         (2 * math.sqrt(3) + 0.25 + 4.8e-5) / (4.25 + 4.8e-5 + 1e-8)),
        (1e-3, 4e-12 + 1e-8, {(0, 0): 0.0, (1, 1): pi / 6, (4, 0): 0.0},
         (2 * math.sqrt(3) + 0.25) * 1e-6 / (4.25e-6 + 1e-8)),
    ]
    for scale, eta, rel_theta, conf in cases:
        ta, tb = designed_tile_pair(scale=scale)
        s = mod.tile_stats(mod.rfft2_ortho(ta), mod.rfft2_ortho(tb), 8, 8, mod.ParParams())
        assert abs(s.eta - eta) <= 1e-9 * eta, (scale, s.eta, eta)
        got = {(int(a), int(b)) for a, b in np.argwhere(s.reliable)}
        assert got == set(rel_theta), (scale, sorted(got))
        for ky in range(8):
            for kx in range(5):
                want = rel_theta.get((ky, kx), 0.0)
                assert abs(s.theta[ky, kx] - want) <= 1e-9, (scale, ky, kx, s.theta[ky, kx], want)
        assert abs(s.conf - conf) <= 1e-12, (scale, s.conf, conf)


PINS = [pin_dft_bruteforce, pin_dft_numpy, pin_parseval_kappa, pin_round_trip, pin_bin_kinds,
        pin_nu_isotropy, pin_linear_g0, pin_translation_ramp, pin_endpoints, pin_real_valued,
        pin_confidence_bounds, pin_confidence_full_spectrum, pin_coherence_levels,
        pin_no_reliable_bin, pin_swap_symmetry, pin_channel_permutation, pin_gate_shape,
        pin_wrap, pin_anchor_update, pin_sites_linear_g0, pin_reliability_threshold]


@pytest.mark.parametrize("pin", PINS, ids=[p.__name__ for p in PINS])
def test_pin(pin):
    pin()


# ---------------------------------------------------------------------------
# composition (eq:block) against the hand-derived table in tests/golden
# ---------------------------------------------------------------------------

def load_composition_golden():
    import os
    path = os.path.join(os.path.dirname(__file__), "golden", "composition.txt")
    cases, cur = [], None
    for line in open(path):
        line = line.split("#", 1)[0].strip()
        if not line:
            continue
        if line.startswith("case"):
            _, n, anchors = line.split(None, 2)
            cur = (int(n), tuple(int(x) for x in anchors.split(",")), [])
            cases.append(cur)
        else:
            t, a, b, num, den = (int(x) for x in line.split())
            cur[2].append((t, a, b, num / den))
    return cases


def test_composition_golden():
    cases = load_composition_golden()
    assert len(cases) >= 5
    for n, anchors, rows in cases:
        got = P.composition(anchors, n)
        assert [(t, a, b) for t, a, b, _ in got] == [(t, a, b) for t, a, b, _ in rows]
        for (_, _, _, x), (_, _, _, y) in zip(got, rows):
            assert abs(x - y) < 1e-15


def test_composition_errors():
    assert P.composition((0, 1, 2, 3), 4) == []          # K_f = N_cur: bypass
    with pytest.raises(ValueError):
        P.composition((2,), 4)                           # K_f < 2
    with pytest.raises(ValueError):
        P.composition((0, 0, 3), 4)
    with pytest.raises(ValueError):
        P.composition((0, 4), 4)


def test_tiny_branch_cut_margin():
    """The tiny workload's integer (1, 2) shift puts some bins at true theta = pi;
    the 0.1 noise decides their side.  For the seed used by the parity tests the
    decision must clear the branch cut by far more than rounding."""
    import gen
    w = gen.get(gen.workloads.TINY)
    resid, _, _ = gen.par_inputs(w, seed=42)
    st = P.par_stats(resid.astype(np.float64), w.anchors)
    for (_, _, _, s) in st[(0, 3)]:
        rel = s.reliable & (s.theta != 0)
        assert np.all(np.pi - np.abs(s.theta[rel]) > 1e-4)
