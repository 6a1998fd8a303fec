"""Float64 oracle for the spectral diagnostics of reconstructed residuals.

TEST INFRASTRUCTURE ONLY (see the package docstring).

App. C (diagnostics) eq:oracles, eq:shift, eq:phase_progress, eq:bandenergy,
eq:phaseerror, and the relative error e_t of Sec. 3.1 eq:sensitivity, with the
tile / FFT conventions of PAR (App. A.2: disjoint tiles at their own size,
orthonormal real 2-D DFT, real-FFT multiplicities kappa, normalised radius nu):

* e_t = ||R_t - R_hat_t|| / (||R_t|| + eps) over the whole frame;
* band error energy: for radial bands B of nu, eta(B) = sum_{p,c,w in B} kappa
  |F_t - F_hat_t|^2 / (sum_{p,c,w} kappa |F_t - F_hat_t|^2 + eps);
* oracle corrections of the linear interpolation F_lin = (1-alpha) F_a + alpha F_b:
  F_phase = |F_lin| e^{i Arg F_t}, F_mag = |F_t| e^{i Arg F_lin}, inverted;
* transport phase error: the circular distance |wrap_[-pi,pi)(phi_t - phi_a -
  alpha theta_p)| averaged with energy weights kappa |F_t|^2 (bins where F_t or
  F_a vanishes carry no phase and no weight);
* phase progress of one coefficient: (phi_t - phi_a) / (phi_b - phi_a) on phases
  unwrapped along the frames; phase_progress_frames takes it for every stored bin
  of every tile and channel over the interior frames of each anchor pair.

Readings where the paper leaves a choice: the bands are given by edges on PAR's nu
(band k holds edges[k] <= nu < edges[k+1], the last band also nu = 1); the energy
weight of the phase error is kappa |F_t|^2; eps = 1e-8.
"""
from __future__ import annotations

import math

import numpy as np

from . import par as P

EPS = 1e-8


def nrmse(ref_t, approx_t, eps: float = EPS) -> float:
    """e_t of eq:sensitivity over one frame."""
    ref = np.asarray(ref_t, dtype=np.float64)
    d = ref - np.asarray(approx_t, dtype=np.float64)
    return float(np.sqrt((d * d).sum()) / (np.sqrt((ref * ref).sum()) + eps))


def band_index(nu, edges) -> np.ndarray:
    """Band of each bin: k with edges[k] <= nu < edges[k+1]; nu = 1 -> last band."""
    e = np.asarray(edges, dtype=np.float64)
    k = np.searchsorted(e, np.asarray(nu, dtype=np.float64), side="right") - 1
    return np.clip(k, 0, len(e) - 2)


def band_energy(ref_t, approx_t, tile_h: int, tile_w: int, edges, eps: float = EPS) -> np.ndarray:
    """eq:bandenergy of the error R_t - R_hat_t: fraction per radial band."""
    ref = np.asarray(ref_t, dtype=np.float64)
    err = ref - np.asarray(approx_t, dtype=np.float64)
    Hg, Wg = ref.shape[:2]
    num = np.zeros(len(edges) - 1)
    for (y0, hp, x0, wp) in P.tiles(Hg, Wg, tile_h, tile_w):
        F = P.rfft2_ortho(err[y0:y0 + hp, x0:x0 + wp])            # [hp, nkx, D]
        _, _, kappa, nu = P.bin_tables(hp, wp)
        e = (kappa[:, :, None] * np.abs(F) ** 2).sum(axis=2)     # summed over channels
        for k, v in zip(band_index(nu, edges).ravel(), e.ravel()):
            num[k] += v
    return num / (num.sum() + eps)


def wrap_pm_pi(x):
    """Wrap to [-pi, pi)."""
    return x - 2.0 * math.pi * np.floor((x + math.pi) / (2.0 * math.pi))


def phase_error(ref_t, anchor_a, theta_tiles, alpha: float, tile_h: int, tile_w: int,
                eps: float = EPS) -> float:
    """eq:phaseerror, energy-weighted over tiles, channels and stored bins;
    theta_tiles[p] is the pair's transport phase [hp, nkx] of tile p."""
    ref = np.asarray(ref_t, dtype=np.float64)
    anc = np.asarray(anchor_a, dtype=np.float64)
    Hg, Wg = ref.shape[:2]
    num = den = 0.0
    for p, (y0, hp, x0, wp) in enumerate(P.tiles(Hg, Wg, tile_h, tile_w)):
        Ft = P.rfft2_ortho(ref[y0:y0 + hp, x0:x0 + wp])
        Fa = P.rfft2_ortho(anc[y0:y0 + hp, x0:x0 + wp])
        _, _, kappa, _ = P.bin_tables(hp, wp)
        w = kappa[:, :, None] * np.abs(Ft) ** 2
        w = np.where((np.abs(Ft) > 0) & (np.abs(Fa) > 0), w, 0.0)
        x = np.angle(Ft) - np.angle(Fa) - alpha * np.asarray(theta_tiles[p])[:, :, None]
        num += float((w * np.abs(wrap_pm_pi(x))).sum())
        den += float(w.sum())
    return num / (den + eps)


def oracle_corrections(ref_t, anchor_a, anchor_b, alpha: float, tile_h: int, tile_w: int):
    """eq:oracles applied to the linear interpolation of the anchor pair:
    (R_phase, R_mag), each assembled from its tiles."""
    ref = np.asarray(ref_t, dtype=np.float64)
    Ra = np.asarray(anchor_a, dtype=np.float64)
    Rb = np.asarray(anchor_b, dtype=np.float64)
    Hg, Wg = ref.shape[:2]
    out_p = np.zeros_like(ref)
    out_m = np.zeros_like(ref)
    for (y0, hp, x0, wp) in P.tiles(Hg, Wg, tile_h, tile_w):
        sl = (slice(y0, y0 + hp), slice(x0, x0 + wp))
        Ft = P.rfft2_ortho(ref[sl])
        Fl = (1.0 - alpha) * P.rfft2_ortho(Ra[sl]) + alpha * P.rfft2_ortho(Rb[sl])
        out_p[sl] = P.irfft2_ortho(np.abs(Fl) * np.exp(1j * np.angle(Ft)), wp)
        out_m[sl] = P.irfft2_ortho(np.abs(Ft) * np.exp(1j * np.angle(Fl)), wp)
    return out_p, out_m


def unwrap_track(phases) -> np.ndarray:
    """Phases of one coefficient along the frames, made continuous: each step is
    the previous value plus the wrapped difference."""
    ph = np.asarray(phases, dtype=np.float64)
    out = ph.copy()
    for i in range(1, len(ph)):
        out[i] = out[i - 1] + wrap_pm_pi(ph[i] - ph[i - 1])
    return out


def phase_progress(phases, ia: int, ib: int) -> np.ndarray:
    """eq:phase_progress for every frame of one coefficient's phase track."""
    u = unwrap_track(phases)
    return (u - u[ia]) / (u[ib] - u[ia])


def phase_progress_frames(ref, anchors, tile_h: int, tile_w: int) -> np.ndarray:
    """eq:phase_progress for every coefficient: tile p, stored bin (ky, kx) of its
    real 2-D DFT, channel c, and every interior frame t of each adjacent anchor
    pair (a, b).  The track of one coefficient is Arg F_t for t = a .. b (the
    orthonormal tile transform of App. A.2, edge tiles at their own size),
    unwrapped along the frames and normalised by its displacement between the two
    anchors.  Returns p [n_frames, n_tiles, tile_h, tile_w // 2 + 1, D]: NaN on
    anchor frames, frames outside [a_0, a_last] and slots past an edge tile's bins
    (and where the displacement vanishes, 0 / 0)."""
    ref = np.asarray(ref, dtype=np.float64)
    n, Hg, Wg, D = ref.shape
    tl = P.tiles(Hg, Wg, tile_h, tile_w)
    out = np.full((n, len(tl), tile_h, tile_w // 2 + 1, D), np.nan)
    for (a, b) in P.anchor_pairs(anchors):
        for p, (y0, hp, x0, wp) in enumerate(tl):
            ph = np.stack([np.angle(P.rfft2_ortho(ref[t, y0:y0 + hp, x0:x0 + wp]))
                           for t in range(a, b + 1)])
            with np.errstate(divide="ignore", invalid="ignore"):
                prog = phase_progress(ph, 0, b - a)
            out[a + 1:b, p, :hp, :wp // 2 + 1, :] = prog[1:-1]
    return out


def frame_diagnostics(ref, approx, anchors, prm: P.ParParams, edges, eps: float = EPS):
    """For every skipped frame t of eq:block: (e_t, band fractions, transport phase
    error with the pair's PAR theta, R_phase, R_mag).  ref holds the reference
    residual of every frame, approx the reconstruction of the skipped ones."""
    ref = np.asarray(ref, dtype=np.float64)
    n, Hg, Wg, _ = ref.shape
    stats = P.par_stats(ref, anchors, prm)
    out = {}
    for (t, a, b, alpha) in P.composition(anchors, n):
        th = [st.theta for (_, _, _, st) in stats[(a, b)]]
        rp, rm = oracle_corrections(ref[t], ref[a], ref[b], alpha, prm.tile_h, prm.tile_w)
        out[t] = dict(nrmse=nrmse(ref[t], approx[t], eps),
                      bands=band_energy(ref[t], approx[t], prm.tile_h, prm.tile_w, edges, eps),
                      phase_err=phase_error(ref[t], ref[a], th, alpha, prm.tile_h, prm.tile_w, eps),
                      r_phase=rp, r_mag=rm)
    return out
