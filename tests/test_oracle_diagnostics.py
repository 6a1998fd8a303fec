"""Pins for the spectral-diagnostics oracle (oracle/diagnostics.py) against what
the paper and the mathematics fix: the error ratio's special cases, Parseval for
the band energy with kappa, single-frequency errors that land in one band, the
translation identity eq:shift (zero transport phase error with the exact phase,
a closed form without transport, phase progress = alpha), and the oracle
corrections' identities (eq:oracles).  Plain functions, so that
tests/test_oracle_mutations.py can plant mistakes and show that a pin catches
each."""
import math

import numpy as np
import pytest

from gen.workloads import fourier_shift
from oracle import diagnostics as DG
from oracle import par as P


def rng(seed=0):
    return np.random.default_rng(seed)


def pin_nrmse(mod=DG):
    r = rng(1).standard_normal((6, 5, 3))
    assert mod.nrmse(r, r) == 0.0
    assert abs(mod.nrmse(r, np.zeros_like(r)) - 1.0) < 1e-8
    assert abs(mod.nrmse(r, 3.0 * r) - 2.0) < 1e-8
    assert abs(mod.nrmse(r, r + 0.5 * r) - 0.5) < 1e-8


def pin_band_parseval(mod=DG):
    """Summed over bands, the kappa-weighted spectral error energy is the spatial
    error energy (orthonormal transform; edge tiles at their own size)."""
    ref = rng(2).standard_normal((13, 11, 4))
    app = rng(3).standard_normal((13, 11, 4))
    fr = mod.band_energy(ref, app, 8, 8, [0.0, 0.25, 0.5, 0.75, 1.0], eps=0.0)
    assert abs(fr.sum() - 1.0) < 1e-12
    # the unnormalised numerator equals ||err||^2: recover it from a one-band split
    err = ref - app
    num = 0.0
    for (y0, hp, x0, wp) in P.tiles(13, 11, 8, 8):
        F = P.rfft2_ortho(err[y0:y0 + hp, x0:x0 + wp])
        _, _, kappa, _ = P.bin_tables(hp, wp)
        num += float((kappa[:, :, None] * np.abs(F) ** 2).sum())
    assert abs(num - float((err ** 2).sum())) < 1e-9 * num


def pin_band_single_frequency(mod=DG):
    """An error that is one spatial frequency of an 8x8 tile lies in that
    frequency's band only; a constant error lies in the lowest band."""
    y, x = np.meshgrid(np.arange(8), np.arange(8), indexing="ij")
    edges = [0.0, 0.3, 0.6, 1.0]
    for (ky, kx) in [(0, 1), (1, 2), (4, 4), (2, 0)]:
        wave = np.cos(2 * math.pi * (ky * y / 8 + kx * x / 8))[:, :, None]
        _, _, _, nu = P.bin_tables(8, 8)
        want = int(np.clip(np.searchsorted(edges, nu[ky, kx], side="right") - 1, 0, 2))
        fr = mod.band_energy(wave, np.zeros_like(wave), 8, 8, edges, eps=0.0)
        assert abs(fr[want] - 1.0) < 1e-12, (ky, kx, fr)
    fr = mod.band_energy(np.full((8, 8, 2), 3.0), np.zeros((8, 8, 2)), 8, 8, edges, eps=0.0)
    assert abs(fr[0] - 1.0) < 1e-12


def pin_band_split(mod=DG):
    """Two cosines of known spatial energy in different bands (one in a column
    the real FFT stores once, one in a column it stores for both signs): the
    fractions are their energy shares, so kappa must weight the stored bins."""
    y, x = np.meshgrid(np.arange(8), np.arange(8), indexing="ij")
    lo = 2.0 * np.cos(2 * math.pi * (1 * y / 8))[:, :, None]          # (ky, kx) = (1, 0)
    hi = 1.0 * np.cos(2 * math.pi * (3 * y / 8 + 3 * x / 8))[:, :, None]   # (3, 3)
    e_lo, e_hi = float((lo ** 2).sum()), float((hi ** 2).sum())
    fr = mod.band_energy(lo + hi, np.zeros_like(lo), 8, 8, [0.0, 0.5, 1.0], eps=0.0)
    assert np.allclose(fr, [e_lo / (e_lo + e_hi), e_hi / (e_lo + e_hi)], rtol=0, atol=1e-12), fr


def pin_band_edge_rule(mod=DG):
    """A bin exactly on an edge belongs to the band above it (edges[k] <= nu <
    edges[k+1]), and nu = 1 to the last band.  On a 1x8 tile nu = 2 kx / 8
    exactly, so a cosine at kx = 2 (nu = 1/2) with edges (0, 1/2, 1) puts all
    of its energy in band 1, and one at kx = 4 (nu = 1) too."""
    x = np.arange(8)[None, :]
    for kx in (2, 4):
        f = np.cos(2 * math.pi * kx * x / 8)[:, :, None]
        fr = mod.band_energy(f, np.zeros_like(f), 1, 8, [0.0, 0.5, 1.0], eps=0.0)
        assert np.allclose(fr, [0.0, 1.0], rtol=0, atol=1e-12), (kx, fr)


def _bandlimit(x):
    """Zero the Nyquist row and column, so fractional translations are exact."""
    X = np.fft.rfft2(x, axes=(0, 1))
    X[x.shape[0] // 2] = 0
    X[:, x.shape[1] // 2] = 0
    return np.fft.irfft2(X, s=x.shape[:2], axes=(0, 1))


def _translation_case(d, alpha):
    """One 16x16 frame as a single periodic tile: R_a random and band-limited,
    R_t and R_b its translations by alpha d and d (eq:shift)."""
    ra = _bandlimit(rng(5).standard_normal((16, 16, 3)))
    return ra, fourier_shift(ra, np.array(d) * alpha), fourier_shift(ra, np.array(d))


def pin_phase_error_translation(mod=DG):
    """eq:shift: with the exact per-bin displacement phase as theta the transport
    phase error vanishes; with no transport (theta = 0) every bin's error is
    |wrap(-alpha w.d)|, so a single-frequency field gives exactly that."""
    d, alpha = (0.4, -0.3), 0.35
    ra, rt, _ = _translation_case(d, alpha)
    hp = wp = 16
    ky = np.arange(hp)
    kys = np.where(2 * ky <= hp, ky, ky - hp)[:, None]
    kx = np.arange(wp // 2 + 1)[None, :]
    wd = 2 * math.pi * (kys * d[0] / hp + kx * d[1] / wp)
    theta = -wd                                      # Arg(F_b conj F_a), |w.d| < pi here
    assert np.abs(wd).max() < math.pi
    assert mod.phase_error(rt, ra, [theta], alpha, 16, 16) < 1e-9
    yy, xx = np.meshgrid(np.arange(16), np.arange(16), indexing="ij")
    one = np.cos(2 * math.pi * (2 * yy / 16 + 3 * xx / 16))[:, :, None]
    ot = fourier_shift(one, np.array(d) * alpha)
    want = abs(alpha * 2 * math.pi * (2 * d[0] / 16 + 3 * d[1] / 16))
    got = mod.phase_error(ot, one, [np.zeros((16, 9))], alpha, 16, 16)
    assert abs(got - want) < 1e-9, (got, want)
    # two frequencies: the errors average with energy weights |F|^2
    two = one + 0.5 * np.cos(2 * math.pi * (1 * yy / 16))[:, :, None]
    tt = fourier_shift(two, np.array(d) * alpha)
    w2 = abs(alpha * 2 * math.pi * (1 * d[0] / 16))
    assert abs(w2 - want) > 1e-3                     # distinct per-bin errors
    want = (1.0 * want + 0.25 * w2) / 1.25
    got = mod.phase_error(tt, two, [np.zeros((16, 9))], alpha, 16, 16)
    assert abs(got - want) < 1e-9, (got, want)


def pin_phase_progress(mod=DG):
    """Constant-velocity translation: the unwrapped phase of every coefficient
    moves linearly, so the progress equals alpha = (t - a)/(b - a) (eq:shift),
    also across the +-pi branch cut."""
    w_d = 2.5                                          # > pi / 2 per frame: wraps
    frames = np.arange(7)
    phases = np.angle(np.exp(-1j * w_d * frames))     # principal values
    p = mod.phase_progress(phases, 1, 5)
    assert np.allclose(p, (frames - 1) / 4.0, rtol=0, atol=1e-12)


def pin_phase_progress_frames(mod=DG):
    """Every 4x4 tile of an 8x12 grid moves circularly by its own integer step per
    frame, so each coefficient turns by the same angle every frame (eq:shift): where
    that angle is not +-pi and the coefficient is nonzero the progress of an
    interior frame t of the pair (a, b) is (t - a)/(b - a), per pair (anchors 0, 3
    and 7), and every other entry is NaN."""
    r = rng(11)
    n, th, tw, D = 9, 4, 4, 3
    steps = [(1, 0), (0, 1), (1, 1), (3, 1), (2, 3), (1, 2)]
    ref = np.zeros((n, 8, 12, D))
    tl = P.tiles(8, 12, th, tw)
    for p, (y0, hp, x0, wp) in enumerate(tl):
        base = r.standard_normal((hp, wp, D))
        for t in range(n):
            ref[t, y0:y0 + hp, x0:x0 + wp] = np.roll(base, (t * steps[p][0], t * steps[p][1]), axis=(0, 1))
    anchors = (0, 3, 7)
    got = mod.phase_progress_frames(ref, anchors, th, tw)
    assert got.shape == (n, len(tl), th, tw // 2 + 1, D)
    ky = np.arange(th)[:, None]
    kx = np.arange(tw // 2 + 1)[None, :]
    checked = 0
    for p, (y0, hp, x0, wp) in enumerate(tl):
        turn = 2 * math.pi * (ky * steps[p][0] / hp + kx * steps[p][1] / wp)
        ok = np.abs(np.abs(DG.wrap_pm_pi(turn)) - math.pi) > 1e-6
        F0 = P.rfft2_ortho(ref[0, y0:y0 + hp, x0:x0 + wp])
        for (a, b) in [(0, 3), (3, 7)]:
            for t in range(a + 1, b):
                sel = ok[:, :, None] & (np.abs(F0) > 1e-9) & (np.abs(DG.wrap_pm_pi(turn)) > 1e-9)[:, :, None]
                g = got[t, p]
                assert np.allclose(g[sel], (t - a) / (b - a), rtol=0, atol=1e-9), (p, t)
                checked += int(sel.sum())
    assert checked > 100
    for t in (0, 3, 7, 8):
        assert np.isnan(got[t]).all(), t


def pin_oracle_corrections(mod=DG):
    """eq:oracles: when the reference is the linear interpolation both
    corrections return it; when the reference has the magnitudes of the linear
    interpolation (a pure phase change), the phase correction returns it."""
    ra = rng(6).standard_normal((12, 10, 3))
    rb = rng(7).standard_normal((12, 10, 3))
    alpha = 0.3
    rl = (1 - alpha) * ra + alpha * rb
    rp, rm = mod.oracle_corrections(rl, ra, rb, alpha, 8, 8)
    assert np.allclose(rp, rl, atol=1e-12) and np.allclose(rm, rl, atol=1e-12)
    # phase-only change, tile by tile: a circular integer shift inside each tile
    ref = np.zeros_like(rl)
    for (y0, hp, x0, wp) in P.tiles(12, 10, 8, 8):
        ref[y0:y0 + hp, x0:x0 + wp] = np.roll(rl[y0:y0 + hp, x0:x0 + wp], (1, 1), axis=(0, 1))
    rp, rm = mod.oracle_corrections(ref, ra, rb, alpha, 8, 8)
    assert np.allclose(rp, ref, atol=1e-10)
    assert not np.allclose(rm, ref, atol=1e-3)


def pin_frame_diagnostics_translation(mod=DG):
    """eq:shift and eq:block together: a band-limited field translated by t d per
    frame, anchors (0, 4), one periodic 16x16 tile per frame.  The cross-spectrum
    phase is then -w.4d per bin (|w.4d| < pi here), so the transport with the
    gate forced to 1 reconstructs every skipped frame exactly, interior (alpha =
    1/4, 1/2, 3/4) and extrapolated (frame 5, alpha = 5/4) alike: the per-frame
    diagnostics must report e_t = 0, no band energy and no transport phase error
    for each of them, which holds only if each frame is paired with its own
    anchors, alpha and theta."""
    d = np.array([0.05, -0.03])
    base = _bandlimit(rng(8).standard_normal((16, 16, 3)))
    ref = np.stack([fourier_shift(base, d * t) for t in range(6)])
    prm = P.ParParams(tile_h=16, tile_w=16, gate_mode=1)
    approx = P.par_reconstruct(ref, (0, 4), prm)
    out = mod.frame_diagnostics(ref, approx, (0, 4), prm, [0.0, 0.5, 1.0])
    assert sorted(out) == [1, 2, 3, 5]
    for t, v in out.items():
        assert v["nrmse"] < 1e-9, (t, v["nrmse"])
        assert v["phase_err"] < 1e-9, (t, v["phase_err"])
        assert np.abs(v["bands"]).max() < 1e-9, (t, v["bands"])


PINS = [pin_nrmse, pin_band_parseval, pin_band_single_frequency, pin_band_split,
        pin_phase_error_translation,
        pin_phase_progress, pin_phase_progress_frames, pin_oracle_corrections,
        pin_frame_diagnostics_translation,
        pin_band_edge_rule]


@pytest.mark.parametrize("pin", PINS, ids=[p.__name__ for p in PINS])
def test_pin(pin):
    pin()
