"""Synthetic workloads for one reconstruction-coupled DiT block step.

The paper's workloads are trained Matrix-Game 3.0 / HY-World 1.5 rollouts on
benchmark trajectories; none of that is available, so these seeded generators
stand in for their shapes (Sec. 5 setup, tab:config):

tiny_4f8x8_d64
    4 current frames of 8x8 tokens, D = 64 (2 heads x 32), anchors {0, 3},
    history 4 chunks x 64 tokens, TopK 2.  Q/K/V ~ N(0,1) (rounded to bf16),
    residuals fp32 N(0,1) with frame 3 = frame 0 circularly shifted by (1, 2)
    tokens plus 0.1 N(0,1).
matrix_game_like_8f30x52_d1536
    8 frames of 30x52 tokens, D = 1536 (12 x 128), anchors {0, 3, 7}, history
    16 chunks x 1560 tokens, TopK 4.  Residuals: per-channel periodic fields
    with power ~ 1/f^2 (DC zero, unit RMS), frame t translated by a random
    continuous d_t with |components| <= 4 tokens (Fourier shift).
hy_world_like_16f44x80_d3072
    16 frames of 44x80 tokens, D = 3072 (24 x 128), anchors {0, 4, 8, 12},
    history 32 chunks x 3520 tokens, TopK 8.  Power ~ 1/f^2.5 and per-channel
    coherence w_c ~ U(0,1): channel c = w_c * translated field + sqrt(1 - w_c^2)
    * an independent field of the same spectrum, drawn per frame.
par_stress_66f64x64_d3072
    PAR only: 66 frames of 64x64 tokens, D = 3072, anchors {0, 65}, 64 skipped
    frames.  R_0 a 1/f^2 field; R_65 = R_0 Fourier-shifted by d ~ U(-1,1)^2
    plus 0.2 x N(0,1) noise high-passed to normalised radius > 0.5.
long_history_4f44x80_d3072_k{4,8,16,32}
    4 frames of 44x80, D = 3072 (24 x 128), all four frames anchors (PAR
    bypass), history 128 chunks x 3520 tokens, TopK swept over {4, 8, 16, 32};
    keys ~ N(mu_c, 1) with mu_c ~ N(0, 0.5) per (chunk, head, dim).

Seeds: base seed 42; each tensor gets its own child seed from
numpy.random.SeedSequence(seed).spawn, so changing one tensor's shape does not
change another's values.  Large Q/K/V tensors are drawn with torch's
generator on the target device (CPU or GPU); residual fields are drawn with
numpy on the host.
"""
from __future__ import annotations

import math
from dataclasses import dataclass, field

import numpy as np


@dataclass(frozen=True)
class Workload:
    name: str
    n_frames: int
    Hg: int
    Wg: int
    H: int
    dh: int
    anchors: tuple
    M: int
    Bv: int
    topk: int
    n0: int = 0
    D_par: int = 0                 # PAR channel count when it differs from H*dh
    spectrum: float = 2.0          # residual power-spectrum exponent (power ~ 1/f^spectrum)
    max_shift: float = 4.0         # per-frame translation bound in tokens
    coherence: bool = False        # per-channel coherence w_c ~ U(0,1)
    kind: str = "block"            # block | tiny | par_only | long_history
    has_attention: bool = True
    key_mean_std: float = 0.0      # std of per-(chunk, head, dim) key means
    tags: tuple = field(default_factory=tuple)

    @property
    def S(self) -> int:
        return self.Hg * self.Wg

    @property
    def D(self) -> int:
        return self.D_par if self.D_par else self.H * self.dh

    @property
    def n_a(self) -> int:
        return len(self.anchors)

    @property
    def scale(self) -> float:
        return 1.0 / math.sqrt(self.dh)

    @property
    def has_par(self) -> bool:
        return len(self.anchors) < self.n_frames

    @property
    def frame_tokens(self) -> int:
        """Current-frame tokens advanced by one block step: N_cur * S, or for the
        PAR-only stress case the reconstructed (skipped) frames' tokens."""
        if self.kind == "par_only":
            return (self.n_frames - self.n_a) * self.S
        return self.n_frames * self.S


def _w(**kw) -> Workload:
    return Workload(**kw)


WORKLOADS: dict[str, Workload] = {}
for _wl in [
    _w(name="tiny_4f8x8_d64", n_frames=4, Hg=8, Wg=8, H=2, dh=32, anchors=(0, 3),
       M=4, Bv=64, topk=2, kind="tiny"),
    _w(name="matrix_game_like_8f30x52_d1536", n_frames=8, Hg=30, Wg=52, H=12, dh=128,
       anchors=(0, 3, 7), M=16, Bv=1560, topk=4, spectrum=2.0),
    _w(name="hy_world_like_16f44x80_d3072", n_frames=16, Hg=44, Wg=80, H=24, dh=128,
       anchors=(0, 4, 8, 12), M=32, Bv=3520, topk=8, spectrum=2.5, coherence=True),
    _w(name="par_stress_66f64x64_d3072", n_frames=66, Hg=64, Wg=64, H=24, dh=128,
       anchors=(0, 65), M=0, Bv=4096, topk=0, kind="par_only", has_attention=False),
] + [
    _w(name=f"long_history_4f44x80_d3072_k{k}", n_frames=4, Hg=44, Wg=80, H=24, dh=128,
       anchors=(0, 1, 2, 3), M=128, Bv=3520, topk=k, kind="long_history",
       key_mean_std=0.5)
    for k in (4, 8, 16, 32)
]:
    WORKLOADS[_wl.name] = _wl

TINY = "tiny_4f8x8_d64"
MATRIX = "matrix_game_like_8f30x52_d1536"
HY = "hy_world_like_16f44x80_d3072"
PAR_STRESS = "par_stress_66f64x64_d3072"


def get(name: str) -> Workload:
    return WORKLOADS[name]


def seeds_for(seed: int, n: int) -> list[int]:
    """n independent 63-bit child seeds of `seed`."""
    return [int(c.generate_state(1, dtype=np.uint64)[0]) & ((1 << 63) - 1)
            for c in np.random.SeedSequence(seed).spawn(n)]


# ----------------------------------------------------------------------------
# Q / K / V (bf16)
# ----------------------------------------------------------------------------

def _randn(shape, seed, device):
    import torch
    g = torch.Generator(device=device)
    g.manual_seed(seed)
    return torch.randn(shape, generator=g, device=device, dtype=torch.float32)


def attn_inputs(w: Workload, seed: int = 42, device="cpu", M=None, Bv=None,
                duplicate_chunks=None):
    """Q [n_a, S, H, dh], K_hist and V_hist [M, Bv, H, dh] as bf16 torch tensors,
    plus the current segment K_cur, V_cur [n0, H, dh] (None when n0 == 0).

    duplicate_chunks: optional list of (dst, src) chunk pairs; chunk dst is made a
    byte-identical copy of chunk src (exact score ties for the TopK tie rule).
    """
    import torch
    M = w.M if M is None else M
    Bv = w.Bv if Bv is None else Bv
    sq, sk, sv, smu, skc, svc = seeds_for(seed, 6)
    q = _randn((w.n_a, w.S, w.H, w.dh), sq, device).to(torch.bfloat16)
    k = _randn((M, Bv, w.H, w.dh), sk, device)
    if w.key_mean_std > 0:
        mu = _randn((M, 1, w.H, w.dh), smu, device) * w.key_mean_std
        k = k + mu
    k = k.to(torch.bfloat16)
    v = _randn((M, Bv, w.H, w.dh), sv, device).to(torch.bfloat16)
    if duplicate_chunks:
        for dst, src in duplicate_chunks:
            k[dst].copy_(k[src])
    kc = vc = None
    if w.n0 > 0:
        kc = _randn((w.n0, w.H, w.dh), skc, device).to(torch.bfloat16)
        vc = _randn((w.n0, w.H, w.dh), svc, device).to(torch.bfloat16)
    return q, k, v, kc, vc


def wo_weight(D: int, seed: int = 7, device="cpu"):
    """A synthetic attention output projection W_O, bf16 [D, D] with N(0, 1/D)
    entries (a randomly initialised linear layer; the trained one is unavailable)."""
    import torch
    return (_randn((D, D), seeds_for(seed, 1)[0], device) / float(np.sqrt(D))).to(torch.bfloat16)


def control_inputs(w: Workload, seed: int = 42, device="cpu", n_cur=None, dtype=None):
    """Feature updates of the camera and action control branches, [n_cur, S, D]
    each (bf16 unless `dtype` is given), standing in for the trained branches'
    outputs: N(0, 1) content times a per-frame magnitude.  The camera branch
    peaks around one frame of the chunk (a control event), the action branch
    varies frame to frame; both magnitudes lie in about [0.3, 3]."""
    import torch
    n = w.n_frames if n_cur is None else n_cur
    s_cam, s_act, s_prof = seeds_for(seed, 3)
    rng = np.random.default_rng(s_prof)
    c = rng.uniform(0, n - 1)
    t = np.arange(n)
    mag_cam = 0.3 + 2.5 * np.exp(-((t - c) / 1.5) ** 2)
    mag_act = rng.uniform(0.3, 3.0, size=n)
    dt = torch.bfloat16 if dtype is None else dtype
    out = []
    for sd, mag in ((s_cam, mag_cam), (s_act, mag_act)):
        x = _randn((n, w.S, w.D), sd, device)
        x = x * torch.as_tensor(mag, dtype=torch.float32, device=x.device)[:, None, None]
        out.append(x.to(dt))
    return out[0], out[1]


# ----------------------------------------------------------------------------
# Residual fields (fp32)
# ----------------------------------------------------------------------------

def _freq_grid(Hg, Wg):
    fy = np.fft.fftfreq(Hg)[:, None]
    fx = np.fft.rfftfreq(Wg)[None, :]
    return fy, fx


def power_law_field(Hg, Wg, D, exponent, rng) -> np.ndarray:
    """Per-channel periodic real field [Hg, Wg, D] with power ~ 1/f^exponent,
    zero DC and unit RMS per channel."""
    fy, fx = _freq_grid(Hg, Wg)
    f = np.sqrt(fy ** 2 + fx ** 2)
    amp = np.zeros_like(f)
    amp[f > 0] = f[f > 0] ** (-exponent / 2.0)
    coef = (rng.standard_normal((Hg, Wg // 2 + 1, D)) +
            1j * rng.standard_normal((Hg, Wg // 2 + 1, D))) * amp[:, :, None]
    x = np.fft.irfft2(coef, s=(Hg, Wg), axes=(0, 1))
    x /= np.sqrt((x ** 2).mean(axis=(0, 1), keepdims=True)) + 1e-30
    return x


def fourier_shift(x: np.ndarray, d) -> np.ndarray:
    """Periodic translation of x[Hg, Wg, ...] by the continuous offset d = (dy, dx):
    result(y, x) = x(y - dy, x - dx) for band-limited x."""
    Hg, Wg = x.shape[:2]
    fy, fx = _freq_grid(Hg, Wg)
    ph = np.exp(-2j * np.pi * (fy * d[0] + fx * d[1]))
    X = np.fft.rfft2(x, axes=(0, 1))
    return np.fft.irfft2(X * ph[..., None] if x.ndim == 3 else X * ph, s=(Hg, Wg), axes=(0, 1))


def _highpass_noise(Hg, Wg, D, cutoff, rng):
    n = rng.standard_normal((Hg, Wg, D))
    fy, fx = _freq_grid(Hg, Wg)
    r = np.sqrt(fy ** 2 + fx ** 2)
    keep = (r / r.max()) > cutoff
    X = np.fft.rfft2(n, axes=(0, 1)) * keep[..., None]
    return np.fft.irfft2(X, s=(Hg, Wg), axes=(0, 1))


def par_inputs(w: Workload, seed: int = 42, frames="anchors", D=None, Hg=None, Wg=None):
    """Residual buffer [n_frames, Hg, Wg, D] fp32 (numpy) and the initial hidden
    state X [n_frames, Hg, Wg, D] fp32 for accumulate mode.

    frames="anchors" fills only the anchor frames of the residual buffer (the
    only ones PAR reads) and leaves the others zero; frames="all" also draws the
    ground-truth skipped frames from the same motion model.
    Returns (resid, x0, info) with info holding the drawn translations.
    """
    D = w.D if D is None else D
    Hg = w.Hg if Hg is None else Hg
    Wg = w.Wg if Wg is None else Wg
    n = w.n_frames
    s_base, s_shift, s_coh, s_ind, s_noise, s_x = seeds_for(seed, 6)
    resid = np.zeros((n, Hg, Wg, D), dtype=np.float32)
    want = set(w.anchors) if frames == "anchors" else set(range(n))
    info = {}
    if w.kind == "tiny":
        rng = np.random.default_rng(s_base)
        r0 = rng.standard_normal((Hg, Wg, D))
        noise = np.random.default_rng(s_noise).standard_normal((Hg, Wg, D))
        a0, a1 = w.anchors
        resid[a0] = r0
        resid[a1] = np.roll(r0, (1, 2), axis=(0, 1)) + 0.1 * noise
        info["shift"] = (1, 2)
    elif w.kind == "par_only":
        rng = np.random.default_rng(s_base)
        ra = power_law_field(Hg, Wg, D, w.spectrum, rng)
        d = np.random.default_rng(s_shift).uniform(-1.0, 1.0, size=2)
        noise = 0.2 * _highpass_noise(Hg, Wg, D, 0.5, np.random.default_rng(s_noise))
        a0, a1 = w.anchors[0], w.anchors[-1]
        resid[a0] = ra
        resid[a1] = fourier_shift(ra, d) + noise
        info["shift"] = tuple(d)
        if frames == "all":
            for t in range(n):
                if t not in (a0, a1):
                    resid[t] = fourier_shift(ra, d * (t - a0) / (a1 - a0))
    else:
        rng = np.random.default_rng(s_base)
        base = power_law_field(Hg, Wg, D, w.spectrum, rng)
        shifts = np.random.default_rng(s_shift).uniform(-w.max_shift, w.max_shift, size=(n, 2))
        info["shifts"] = shifts
        if w.coherence:
            wc = np.random.default_rng(s_coh).uniform(0.0, 1.0, size=D)
            info["coherence"] = wc
            ind_seeds = seeds_for(s_ind, n)
        for t in range(n):
            if t not in want:
                continue
            fld = fourier_shift(base, shifts[t])
            if w.coherence:
                ind = power_law_field(Hg, Wg, D, w.spectrum,
                                      np.random.default_rng(ind_seeds[t]))
                fld = wc * fld + np.sqrt(1.0 - wc ** 2) * ind
            resid[t] = fld
    x0 = np.random.default_rng(s_x).standard_normal((n, Hg, Wg, D)).astype(np.float32) \
        if n * Hg * Wg * D <= (1 << 27) else None
    return resid, x0, info


# ---------------------------------------------------------------------------
# Designed-spectrum tiles (input construction for the reliability threshold of
# App. A.2): a real tile whose orthonormal half-spectrum holds prescribed values
# per channel, so that bins fall on either side of the threshold by design.
# ---------------------------------------------------------------------------

def _pol(r, phi):
    return r * complex(math.cos(phi), math.sin(phi))


# Entries (ky, kx, channel, F_a, F_b) of an 8x8 tile, D >= 2; every other stored
# bin is zero.  Column kx = 0 is listed Hermitian-consistent ((2,0) and (6,0)).
# With max W = 4 at DC the threshold is 4e-6 + 1e-8; bin (2,1) sits at about 3x it,
# bin (3,1) at 0.75x, bin (1,3) at 0.3x, and bin (1,2) has W = 0.02 but its two
# channels cancel in Z down to 1e-8.
_S1, _S2, _S3 = math.sqrt(1.2e-5), math.sqrt(3e-6), math.sqrt(1.2e-6)
RELIABILITY_TILE = (
    (0, 0, 0, 2.0, 2.0),
    (1, 1, 0, 1.0, _pol(1.0, math.pi / 3)),
    (1, 1, 1, 1.0, 1.0),
    (2, 1, 0, _S1, _pol(_S1, -math.pi / 4)),
    (3, 1, 0, _S2, _pol(_S2, 2 * math.pi / 5)),
    (1, 3, 0, _S3, _pol(_S3, -2 * math.pi / 3)),
    (1, 2, 0, 0.1, 0.1),
    (1, 2, 1, 0.1, complex(-0.1, 1e-7)),
    (2, 0, 0, _S1, _pol(_S1, math.pi / 5)),
    (6, 0, 0, _S1, _pol(_S1, -math.pi / 5)),
    (4, 0, 0, 0.5, -0.5),
)


def designed_tile_pair(entries=RELIABILITY_TILE, hp=8, wp=8, D=2, channel_map=None, scale=1.0):
    """Two real tiles [hp, wp, D] (float64) whose orthonormal 2-D real DFTs (last
    axis halved) hold `entries` (ky, kx, channel, F_a, F_b) times `scale`.
    `channel_map` relabels the entries' channels (e.g. {1: 66} puts channel 1's
    values into channel 66)."""
    nkx = wp // 2 + 1
    fa = np.zeros((hp, nkx, D), dtype=np.complex128)
    fb = np.zeros((hp, nkx, D), dtype=np.complex128)
    cmap = channel_map or {}
    for ky, kx, c, va, vb in entries:
        c = cmap.get(c, c)
        fa[ky, kx, c] = va * scale
        fb[ky, kx, c] = vb * scale
    for f in (fa, fb):
        for kx in range(nkx):
            if kx == 0 or (wp % 2 == 0 and kx == wp // 2):
                for ky in range(hp):
                    assert abs(f[(-ky) % hp, kx] - np.conj(f[ky, kx])).max() < 1e-15, (ky, kx)
    ta = np.fft.irfft2(fa, s=(hp, wp), axes=(0, 1), norm="ortho")
    tb = np.fft.irfft2(fb, s=(hp, wp), axes=(0, 1), norm="ortho")
    return ta, tb


def band_limited_tile(hp, wp, D, rng):
    """A random real tile whose Nyquist row and column (even edges) are zero in
    every channel, so those bins of any cross-spectrum vanish."""
    f = np.fft.rfft2(rng.standard_normal((hp, wp, D)), axes=(0, 1), norm="ortho")
    if hp % 2 == 0:
        f[hp // 2] = 0
    if wp % 2 == 0:
        f[:, wp // 2] = 0
    return np.fft.irfft2(f, s=(hp, wp), axes=(0, 1), norm="ortho")


def reliability_frames(D=70, seed=5):
    """A 3-frame [3, 16, 24, D] float64 residual stack with anchors {0, 2} and
    skipped frame 1 (zero), laid out as 2 x 3 tiles of 8x8:
      (0,0) the designed tile (channel 1 of the entries moved to channel D-4,
            so the cancelling pair spans two 64-channel blocks);
      (0,1) zero in both anchors;
      (0,2) zero in anchor 0, random in anchor 2;
      (1,0) band-limited random fields (Nyquist row and column zero), anchor 2 a
            circular shift of anchor 0 plus noise;
      (1,1) the designed tile at 1e-3 amplitude (the absolute part of the
            threshold decides there);
      (1,2) random, anchor 2 a shift of anchor 0 plus noise."""
    rng = np.random.default_rng(seed)
    r = np.zeros((3, 16, 24, D))
    ta, tb = designed_tile_pair(D=D, channel_map={1: D - 4})
    r[0, 0:8, 0:8], r[2, 0:8, 0:8] = ta, tb
    r[2, 0:8, 16:24] = rng.standard_normal((8, 8, D))
    bl = band_limited_tile(8, 8, D, rng)
    r[0, 8:16, 0:8] = bl
    r[2, 8:16, 0:8] = np.roll(bl, (1, 2), axis=(0, 1)) + 0.3 * band_limited_tile(8, 8, D, rng)
    ta, tb = designed_tile_pair(D=D, channel_map={1: D - 4}, scale=1e-3)
    r[0, 8:16, 8:16], r[2, 8:16, 8:16] = ta, tb
    x = rng.standard_normal((8, 8, D))
    r[0, 8:16, 16:24] = x
    r[2, 8:16, 16:24] = np.roll(x, (2, 1), axis=(0, 1)) + 0.5 * rng.standard_normal((8, 8, D))
    return r
