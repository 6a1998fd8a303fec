"""Float64 oracle for Phase-Aware Reconstruction (PAR).

TEST INFRASTRUCTURE ONLY (see the package docstring): never imported by the
product path.

What it computes, in the paper's order and notation:

* Sec. 4.3 "Local phase transport" and App. A.2: residuals are cut into
  disjoint spatial tiles p (default 8x8, smaller tiles at the lower/right
  edges transformed at their own size); every channel c of every tile gets an
  orthonormal 2-D real FFT F_{i,p,c}(omega).
* eq:cross: pooled cross-spectrum Z_p = sum_c F_b conj(F_a) and magnitude
  product W_p = sum_c |F_b||F_a|, summed over all channels.
* App. A.2: reliable bins satisfy W_p > eta_p and |Z_p| > eta_p with
  eta_p = 1e-6 max_omega W_p + 1e-8; theta_p = Arg Z_p on reliable bins and
  U_p = 1 elsewhere; phases live on one representative of each conjugate pair,
  the mirror gets -theta, self-conjugate bins get U_p = 1.
* eq:confidence: c_p = sum_{Omega+} kappa |Z| / (sum_{Omega+} kappa W + eps),
  Omega+ = reliable non-DC bins, kappa the real-FFT multiplicity; c_p = 0 when
  no reliable bin exists.
* eq:gate: tau(nu) = tau_low + (tau_high - tau_low) nu^q,
  g = sigmoid((c_p - tau(nu)) / T), nu the radial frequency normalised by the
  largest represented radius.
* eq:fcpasm: F_hat = (1-alpha) F_a U^{g alpha} + alpha F_b U^{-g (1-alpha)},
  U^beta = exp(i beta theta); inverse real FFT; tiles assembled.
* eq:block: interior skipped frames use the bracketing anchor pair; frames
  before a_0 use (a_0, a_1) with alpha < 0, frames after a_J use
  (a_{J-1}, a_J) with alpha > 1; alpha is never clipped; K_f >= 2.

Readings where the paper leaves a choice:
forward transform sign exp(-2 pi i k n / N) and the halved axis is the last
(x / width) axis; Arg is taken in (-pi, pi] (atan2, then -pi -> pi) on
representatives only; a mirror bin takes the reliability flag and the negated
phase of its representative; Omega+ keeps reliable self-conjugate Nyquist
points (kappa = 1) and drops only DC; kappa = 1 on the stored columns
k_x = 0 and k_x = W_p/2 (even W_p), 2 elsewhere; eta's max runs over every
stored bin of the tile, DC included; nu is the physical radius
||(k_y^s / H_p, k_x / W_p)|| with signed k_y^s, divided by its maximum over
the tile's stored bins; sigma is the logistic function.

The DFTs are explicit exp(-2 pi i k n / N) matrices (no FFT library); numpy's
FFT appears only in the oracle's own self-tests as an independent check.
"""
from __future__ import annotations

import math
from dataclasses import dataclass

import numpy as np

# App. A.2 / tab:config_cast constants.
TAU_LOW, TAU_HIGH, Q_EXP, TEMP = 0.25, 0.75, 2.0, 0.10
ETA_REL, ETA_ABS, EPS = 1e-6, 1e-8, 1e-8

GATE_PAR, GATE_ONE, GATE_ZERO = 0, 1, 2

@dataclass(frozen=True)
class ParParams:
    """PAR settings; defaults are the paper's (tab:config_cast, App. A.2)."""
    tile_h: int = 8
    tile_w: int = 8
    tau_low: float = TAU_LOW
    tau_high: float = TAU_HIGH
    q: float = Q_EXP
    T: float = TEMP
    eta_rel: float = ETA_REL
    eta_abs: float = ETA_ABS
    eps: float = EPS
    gate_mode: int = GATE_PAR   # 0: eq:gate, 1: g == 1 (full transport), 2: g == 0 (linear)
    accumulate: bool = False    # False: out[t] = R_hat_t ; True: out[t] += R_hat_t (eq:block)
    update_anchors: bool = False  # also the anchor case of eq:block: out[a] (+)= R_a

# ----------------------------------------------------------------------------
# Tiles and the 2-D real DFT (App. A.2: disjoint tiles, orthonormal, own size)
# ----------------------------------------------------------------------------

def tile_starts(n: int, tile: int) -> list[tuple[int, int]]:
    """Disjoint tiles along one axis: full tiles of `tile`, then the remainder."""
    out = []
    s = 0
    while s < n:
        out.append((s, min(tile, n - s)))
        s += tile
    return out

def tiles(Hg: int, Wg: int, tile_h: int, tile_w: int) -> list[tuple[int, int, int, int]]:
    """All tiles (y0, Hp, x0, Wp) in row-major tile order."""
    return [(y0, hp, x0, wp) for (y0, hp) in tile_starts(Hg, tile_h)
            for (x0, wp) in tile_starts(Wg, tile_w)]

def dft_matrix(n: int, sign: int) -> np.ndarray:
    """E[k, m] = exp(sign * 2 pi i k m / n)."""
    k = np.arange(n)
    return np.exp(sign * 2j * np.pi * np.outer(k, k) / n)

def rfft2_ortho(x: np.ndarray) -> np.ndarray:
    """Orthonormal forward 2-D real DFT of x[Hp, Wp, ...] (channels trailing).

    F[ky, kx] = (Hp Wp)^-1/2 sum_{y,x} x[y, x] exp(-2 pi i (ky y / Hp + kx x / Wp)),
    for ky in [0, Hp) and kx in [0, Wp//2] (the stored half-spectrum).
    """
    hp, wp = x.shape[0], x.shape[1]
    ey = dft_matrix(hp, -1)
    ex = dft_matrix(wp, -1)[: wp // 2 + 1]
    f = np.tensordot(ey, x.astype(np.float64), axes=(1, 0))          # [ky, x, ...]
    f = np.tensordot(ex, f, axes=(1, 1))                             # [kx, ky, ...]
    return np.swapaxes(f, 0, 1) / math.sqrt(hp * wp)

def hermitian_full(f_half: np.ndarray, wp: int) -> np.ndarray:
    """Extend a stored half-spectrum [Hp, Wp//2+1, ...] to [Hp, Wp, ...] using
    F[ky, kx] = conj(F[-ky mod Hp, Wp - kx]) for the columns kx > Wp//2."""
    hp = f_half.shape[0]
    full = np.zeros((hp, wp) + f_half.shape[2:], dtype=np.complex128)
    nh = wp // 2 + 1
    full[:, :nh] = f_half
    for kx in range(nh, wp):
        for ky in range(hp):
            full[ky, kx] = np.conj(f_half[(-ky) % hp, wp - kx])
    return full

def irfft2_ortho_complex(f_half: np.ndarray, wp: int) -> np.ndarray:
    """Orthonormal inverse 2-D DFT of the Hermitian-extended spectrum; returns the
    complex result (its imaginary part vanishes when the spectrum is Hermitian)."""
    hp = f_half.shape[0]
    full = hermitian_full(f_half, wp)
    ey = dft_matrix(hp, +1)
    ex = dft_matrix(wp, +1)
    r = np.tensordot(ey, full, axes=(1, 0))                          # [y, kx, ...]
    r = np.tensordot(ex, r, axes=(1, 1))                             # [x, y, ...]
    return np.swapaxes(r, 0, 1) / math.sqrt(hp * wp)

def irfft2_ortho(f_half: np.ndarray, wp: int) -> np.ndarray:
    """Real part of the orthonormal inverse (the inverse real FFT)."""
    return irfft2_ortho_complex(f_half, wp).real

# ----------------------------------------------------------------------------
# Bin bookkeeping (App. A.2: representatives, mirrors, self-conjugate, kappa, nu)
# ----------------------------------------------------------------------------

REP, MIRROR, SELF = 0, 1, 2

def bin_tables(hp: int, wp: int):
    """Per stored bin (ky, kx), ky in [0,Hp), kx in [0, Wp//2]:

    kind   REP / MIRROR / SELF (self-conjugate)
    partner stored (ky, kx) of the representative for a MIRROR (else itself)
    kappa  real-FFT multiplicity: 1 on the columns that hold their own
           conjugates (kx = 0, and kx = Wp/2 when Wp is even), 2 elsewhere
    nu     physical radial frequency normalised by its maximum over the tile
    """
    nkx = wp // 2 + 1
    kind = np.zeros((hp, nkx), dtype=np.int64)
    partner = np.zeros((hp, nkx, 2), dtype=np.int64)
    kappa = np.zeros((hp, nkx), dtype=np.float64)
    radius = np.zeros((hp, nkx), dtype=np.float64)
    for ky in range(hp):
        for kx in range(nkx):
            self_col = (kx == 0) or (wp % 2 == 0 and kx == wp // 2)
            kappa[ky, kx] = 1.0 if self_col else 2.0
            partner[ky, kx] = (ky, kx)
            if self_col:
                mky = (-ky) % hp
                if mky == ky:
                    kind[ky, kx] = SELF
                elif 2 * ky < hp:
                    kind[ky, kx] = REP
                else:
                    kind[ky, kx] = MIRROR
                    partner[ky, kx] = (mky, kx)
            else:
                kind[ky, kx] = REP
            kys = ky if 2 * ky <= hp else ky - hp
            radius[ky, kx] = math.hypot(kys / hp, kx / wp)
    rmax = radius.max()
    nu = radius / rmax if rmax > 0 else np.zeros_like(radius)
    return kind, partner, kappa, nu

def wrap_arg(z: complex) -> float:
    """Principal argument in (-pi, pi]: atan2, with -pi mapped to +pi."""
    th = math.atan2(z.imag, z.real)
    if th == -math.pi:
        th = math.pi
    return th

# ----------------------------------------------------------------------------
# Per-(pair, tile) statistics: eq:cross, reliability, theta, eq:confidence, eq:gate
# ----------------------------------------------------------------------------

@dataclass
class TileStats:
    Z: np.ndarray         # [Hp, nkx] complex
    W: np.ndarray         # [Hp, nkx]
    eta: float
    reliable: np.ndarray  # [Hp, nkx] bool
    theta: np.ndarray     # [Hp, nkx] transport phase (0 where U = 1)
    conf: float           # c_p
    nu: np.ndarray        # [Hp, nkx]
    gate: np.ndarray      # [Hp, nkx] g_{p, omega}

def cross_spectrum(Fa: np.ndarray, Fb: np.ndarray):
    """eq:cross over the trailing channel axis."""
    Z = (Fb * np.conj(Fa)).sum(axis=-1)
    W = (np.abs(Fb) * np.abs(Fa)).sum(axis=-1)
    return Z, W

def tile_stats(Fa: np.ndarray, Fb: np.ndarray, hp: int, wp: int, prm: ParParams) -> TileStats:
    Z, W = cross_spectrum(Fa, Fb)
    kind, partner, kappa, nu = bin_tables(hp, wp)
    eta = prm.eta_rel * W.max() + prm.eta_abs
    own_rel = (W > eta) & (np.abs(Z) > eta)
    reliable = own_rel.copy()
    theta = np.zeros(Z.shape, dtype=np.float64)
    nky, nkx = Z.shape
    for ky in range(nky):
        for kx in range(nkx):
            k = kind[ky, kx]
            if k == REP:
                if own_rel[ky, kx]:
                    theta[ky, kx] = wrap_arg(complex(Z[ky, kx]))
            elif k == MIRROR:
                py, px = partner[ky, kx]
                reliable[ky, kx] = own_rel[py, px]
                if own_rel[py, px]:
                    theta[ky, kx] = -wrap_arg(complex(Z[py, px]))
            # SELF: U = 1 (theta 0); reliability stays its own
    omega_plus = reliable.copy()
    omega_plus[0, 0] = False                     # drop DC
    if omega_plus.any():
        num = (kappa * np.abs(Z))[omega_plus].sum()
        den = (kappa * W)[omega_plus].sum() + prm.eps
        conf = float(num / den)
    else:
        conf = 0.0
    if prm.gate_mode == GATE_ONE:
        gate = np.ones_like(nu)
    elif prm.gate_mode == GATE_ZERO:
        gate = np.zeros_like(nu)
    else:
        tau = prm.tau_low + (prm.tau_high - prm.tau_low) * nu ** prm.q
        gate = 1.0 / (1.0 + np.exp(-(conf - tau) / prm.T))
    return TileStats(Z=Z, W=W, eta=float(eta), reliable=reliable, theta=theta,
                     conf=conf, nu=nu, gate=gate)

def blend(Fa: np.ndarray, Fb: np.ndarray, theta: np.ndarray, gate: np.ndarray,
          alpha: float) -> np.ndarray:
    """eq:fcpasm, per channel (trailing axis), with U^beta = exp(i beta theta)."""
    ua = np.exp(1j * gate * alpha * theta)[..., None]
    ub = np.exp(-1j * gate * (1.0 - alpha) * theta)[..., None]
    return (1.0 - alpha) * Fa * ua + alpha * Fb * ub

# ----------------------------------------------------------------------------
# Composition (eq:block) and the full operator
# ----------------------------------------------------------------------------

def composition(anchors, n_frames: int):
    """List of (t, a, b, alpha) for every skipped frame t, per eq:block.

    Raises ValueError for anchors that are not strictly increasing in
    [0, n_frames) or, when reconstruction is needed, fewer than two anchors.
    """
    a = [int(x) for x in anchors]
    if any(x < 0 or x >= n_frames for x in a) or any(a[i] >= a[i + 1] for i in range(len(a) - 1)):
        raise ValueError("anchors must be strictly increasing frame indices")
    if len(a) == n_frames:
        return []                                   # K_f = N_cur: bypass
    if len(a) < 2:
        raise ValueError("PAR needs K_f >= 2 anchors")
    aset = set(a)
    out = []
    for t in range(n_frames):
        if t in aset:
            continue
        if t < a[0]:
            pa, pb = a[0], a[1]
        elif t > a[-1]:
            pa, pb = a[-2], a[-1]
        else:
            j = max(i for i in range(len(a)) if a[i] < t)
            pa, pb = a[j], a[j + 1]
        out.append((t, pa, pb, (t - pa) / (pb - pa)))
    return out

def anchor_pairs(anchors):
    a = [int(x) for x in anchors]
    return [(a[j], a[j + 1]) for j in range(len(a) - 1)]

def par_stats(resid: np.ndarray, anchors, prm: ParParams = ParParams()):
    """Statistics for every adjacent anchor pair and tile.

    resid: [n_frames, Hg, Wg, D]; only the anchor frames are read.
    Returns {(a, b): [(tile, Fa, Fb, TileStats), ...]}.
    """
    _, Hg, Wg, _ = resid.shape
    out = {}
    for (a, b) in anchor_pairs(anchors):
        lst = []
        for (y0, hp, x0, wp) in tiles(Hg, Wg, prm.tile_h, prm.tile_w):
            Fa = rfft2_ortho(resid[a, y0:y0 + hp, x0:x0 + wp, :])
            Fb = rfft2_ortho(resid[b, y0:y0 + hp, x0:x0 + wp, :])
            lst.append(((y0, hp, x0, wp), Fa, Fb, tile_stats(Fa, Fb, hp, wp, prm)))
        out[(a, b)] = lst
    return out

def reconstruct_frame(stats_for_pair, alpha: float, Hg: int, Wg: int, D: int) -> np.ndarray:
    """R_hat_t = P_t(R_a, R_b): blend every tile, inverse-transform, assemble."""
    out = np.zeros((Hg, Wg, D), dtype=np.float64)
    for (y0, hp, x0, wp), Fa, Fb, st in stats_for_pair:
        Fh = blend(Fa, Fb, st.theta, st.gate, alpha)
        out[y0:y0 + hp, x0:x0 + wp, :] = irfft2_ortho(Fh, wp)
    return out

def anchor_update(out: np.ndarray, resid: np.ndarray, anchors, accumulate: bool) -> None:
    """The anchor case of eq:block: an anchor's update is its own directly
    computed residual, R~_a = R_a (in place on `out`)."""
    for a in anchors:
        r = np.asarray(resid[a], dtype=np.float64)
        out[a] = out[a] + r if accumulate else r

def par_reconstruct(resid: np.ndarray, anchors, prm: ParParams = ParParams(),
                    out: np.ndarray | None = None, targets=None) -> np.ndarray:
    """Apply PAR to every skipped frame (or to the listed `targets` only).

    Write mode: out[t] = R_hat_t.  Accumulate mode: out[t] += R_hat_t.
    Anchor slots of `out` are touched only with `update_anchors`, which applies
    the anchor case of eq:block as well (out[a] = R_a, or out[a] += R_a).
    Returns `out` (float64).
    """
    n_frames, Hg, Wg, D = resid.shape
    comp = composition(anchors, n_frames)
    if out is None:
        out = np.zeros(resid.shape, dtype=np.float64)
    else:
        out = np.array(out, dtype=np.float64, copy=True)
    if prm.update_anchors:
        anchor_update(out, resid, anchors, prm.accumulate)
    if not comp:
        return out
    stats = par_stats(resid, anchors, prm)
    for (t, a, b, alpha) in comp:
        if targets is not None and t not in targets:
            continue
        r = reconstruct_frame(stats[(a, b)], alpha, Hg, Wg, D)
        if prm.accumulate:
            out[t] += r
        else:
            out[t] = r
    return out

def block_sites(x: np.ndarray, site_residuals, anchors, prm: ParParams = ParParams()) -> np.ndarray:
    """One transformer block's eligible residual sites (visual attention, then
    FFN) sharing one anchor set (Sec. 4.1): each site's update is added to the
    current-frame hidden state per eq:block, anchors included.  `site_residuals`
    are the residual buffers of the sites in order (only anchor frames read)."""
    p = ParParams(**{**prm.__dict__, "accumulate": True, "update_anchors": True})
    for r in site_residuals:
        x = par_reconstruct(r, anchors, p, out=x)
    return x

def par_reconstruct_targets(resid: np.ndarray, anchors, targets, prm: ParParams = ParParams()):
    """R_hat_t for the listed skipped frames only, as {t: [Hg, Wg, D] float64}.

    Same arithmetic as par_reconstruct (write mode); reads only the anchor frames
    of `resid` (which may be float32) and never materialises the full buffer, for
    sampled checks of large workloads.
    """
    n_frames, Hg, Wg, D = resid.shape
    comp = {t: (a, b, alpha) for (t, a, b, alpha) in composition(anchors, n_frames)}
    stats = par_stats(resid, anchors, prm)
    return {t: reconstruct_frame(stats[comp[t][:2]], comp[t][2], Hg, Wg, D) for t in targets}

def stats_arrays(resid: np.ndarray, anchors, prm: ParParams = ParParams()):
    """theta, gate as [n_pairs, n_tiles, tile_h * (tile_w//2 + 1)] and conf as
    [n_pairs, n_tiles]; bin (ky, kx) of a tile sits at ky*(tile_w//2+1) + kx,
    entries beyond a smaller edge tile's own bins are zero."""
    st = par_stats(resid, anchors, prm)
    pairs = anchor_pairs(anchors)
    _, Hg, Wg, _ = resid.shape
    nt = len(tiles(Hg, Wg, prm.tile_h, prm.tile_w))
    nkx_max = prm.tile_w // 2 + 1
    nb = prm.tile_h * nkx_max
    theta = np.zeros((len(pairs), nt, nb))
    gate = np.zeros((len(pairs), nt, nb))
    conf = np.zeros((len(pairs), nt))
    for j, pr in enumerate(pairs):
        for p, ((y0, hp, x0, wp), _, _, s) in enumerate(st[pr]):
            for ky in range(hp):
                for kx in range(wp // 2 + 1):
                    theta[j, p, ky * nkx_max + kx] = s.theta[ky, kx]
                    gate[j, p, ky * nkx_max + kx] = s.gate[ky, kx]
            conf[j, p] = s.conf
    return theta, gate, conf
