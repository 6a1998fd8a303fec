"""GPU parity of the spectral diagnostics (cast_spectral_diagnostics, and
cast_phase_progress at the end) against the oracle (oracle/diagnostics.py) on
identical inputs: generator ground-truth
residuals of every frame as the reference, the GPU PAR reconstruction (write mode)
as the approximation, and each side's own PAR transport phases.

Bars (fp32 tile DFTs of at most 8x8 points and fp32 per-lane sums, against
float64): e_t relative 1e-4; band fractions 1e-5 absolute; transport phase error
1e-4 absolute; oracle corrections rel-RMS 1e-5 over each frame.

The corrections take the phase of one spectrum and the modulus of another, so a
bin whose spectrum lies within fp32 rounding of zero has no phase that fp32 can
determine (on a real bin, its sign).  Tile columns (tile, channel) with a bin
below COND_TAU times the column's spectral norm, in F_t or F_lin (float64), are
compared by what is unique there: the moduli of the returned tile's spectrum,
|F_lin| for R_phase and |F_t| for R_mag; every other column element by element."""
import numpy as np
import pytest
import torch

import gen
from gen import workloads as W
from oracle import diagnostics as DG
from oracle import par as OP
from test_gpu_parity import log, rel_rms

pytestmark = pytest.mark.gpu

NRMSE_REL, BAND_ABS, PHASE_ABS, CORR_RMS = 1e-4, 1e-5, 1e-4, 1e-5
COND_TAU = 1e-4          # a bin below this fraction of its column's norm: phase undetermined
MOD_ABS = 1e-5           # moduli of ill-conditioned columns, relative to the column's norm
MAX_ILL = 0.02           # at most this fraction of the columns may be ill-conditioned


def corrections_check(ref64, got_p, got_m, want_p, want_m, t, a, b, alpha, tile):
    """rel-RMS of the corrections of frame t over its well-conditioned tile
    columns, after checking the spectral moduli of the others."""
    th, tw = (tile, tile) if np.isscalar(tile) else tile
    Hg, Wg, D = ref64.shape[1:]
    well = np.ones((Hg, Wg, D), dtype=bool)
    n_ill = 0
    for (y0, hp, x0, wp) in OP.tiles(Hg, Wg, th, tw):
        sl = (slice(y0, y0 + hp), slice(x0, x0 + wp))
        Ft = OP.rfft2_ortho(ref64[t][sl])
        Fl = (1.0 - alpha) * OP.rfft2_ortho(ref64[a][sl]) + alpha * OP.rfft2_ortho(ref64[b][sl])
        ill = np.zeros(D, dtype=bool)
        for F in (Ft, Fl):
            norm = np.sqrt((np.abs(F) ** 2).sum(axis=(0, 1)))
            ill |= (np.abs(F) < COND_TAU * norm).any(axis=(0, 1))
        if not ill.any():
            continue
        n_ill += int(ill.sum())
        well[y0:y0 + hp, x0:x0 + wp, ill] = False
        for out, F in ((got_p, Fl), (got_m, Ft)):
            G = OP.rfft2_ortho(out[sl][:, :, ill])
            norm = np.sqrt((np.abs(F[:, :, ill]) ** 2).sum(axis=(0, 1)))
            err = np.abs(np.abs(G) - np.abs(F[:, :, ill])).max(axis=(0, 1))
            assert (err <= MOD_ABS * norm).all(), (t, y0, x0, err.max())
    n_cols = len(OP.tiles(Hg, Wg, th, tw)) * D
    assert n_ill <= MAX_ILL * n_cols, (t, n_ill, n_cols)
    r = max(rel_rms(got_p[well], want_p[well]), rel_rms(got_m[well], want_m[well]))
    return r, n_ill


def run_case(cast_lib, ref_np, anchors, label, tile=8, edges=(0.0, 1 / 3, 2 / 3, 1.0), corr=True):
    dev = "cuda"
    th, tw = (tile, tile) if np.isscalar(tile) else tile
    edges = [float(np.float32(e)) for e in edges]      # the values the kernel sees
    ref = torch.from_numpy(ref_np.astype(np.float32)).to(dev)
    prm = cast_lib.cast_par_params_default(tile_h=th, tile_w=tw)
    s1, _ = cast_lib.par_debug_shapes(len(anchors), ref.shape[1], ref.shape[2], prm)
    theta = torch.zeros(s1, device=dev)
    approx = torch.zeros_like(ref)
    cast_lib.cast_par_reconstruct(ref, anchors, prm, out=approx, theta_out=theta)
    dprm = cast_lib.cast_diag_params_default(band_edges=edges, tile_h=th, tile_w=tw)
    got = cast_lib.cast_spectral_diagnostics(ref, approx, anchors, dprm, theta=theta,
                                             want_corrections=corr)
    torch.cuda.synchronize()
    ref64 = ref.cpu().numpy().astype(np.float64)
    app64 = approx.cpu().numpy().astype(np.float64)
    want = DG.frame_diagnostics(ref64, app64, anchors, OP.ParParams(tile_h=th, tile_w=tw), edges)
    nr = got["nrmse"].cpu().numpy()
    bd = got["bands"].cpu().numpy()
    pe = got["phase_err"].cpu().numpy()
    worst = dict(nrmse=0.0, bands=0.0, phase=0.0, corr=0.0)
    n_ill = 0
    pairs = {t: (a, b, alpha) for (t, a, b, alpha) in OP.composition(anchors, ref.shape[0])}
    for t in range(ref.shape[0]):
        if t in anchors:
            assert nr[t] == 0.0 and not bd[t].any() and pe[t] == 0.0
            continue
        w = want[t]
        worst["nrmse"] = max(worst["nrmse"], abs(nr[t] - w["nrmse"]) / max(w["nrmse"], 1e-30))
        worst["bands"] = max(worst["bands"], float(np.abs(bd[t] - w["bands"]).max()))
        worst["phase"] = max(worst["phase"], abs(pe[t] - w["phase_err"]))
        if corr:
            r, k = corrections_check(ref64, got["r_phase"][t].cpu().numpy().astype(np.float64),
                                     got["r_mag"][t].cpu().numpy().astype(np.float64),
                                     w["r_phase"], w["r_mag"], t, *pairs[t], tile)
            worst["corr"] = max(worst["corr"], r)
            n_ill += k
    log(f"[diag {label}] worst: e_t rel {worst['nrmse']:.2e}, bands {worst['bands']:.2e}, "
        f"phase {worst['phase']:.2e}, corrections rel-RMS {worst['corr']:.2e} "
        f"({n_ill} ill-conditioned tile columns checked by modulus); "
        f"e_t {[round(float(nr[t]), 4) for t in range(len(nr)) if t not in anchors]}, "
        f"phase error {[round(float(pe[t]), 4) for t in range(len(pe)) if t not in anchors]}")
    assert worst["nrmse"] <= NRMSE_REL and worst["bands"] <= BAND_ABS
    assert worst["phase"] <= PHASE_ABS and worst["corr"] <= CORR_RMS, worst
    if corr:   # anchor slots of the corrections are not written
        for a in anchors:
            assert not got["r_phase"][a].any() and not got["r_mag"][a].any()
    return got


def test_diag_translation(cast_lib):
    """A coherent constant-velocity translation (eq:shift) over a 32x32 frame with
    8x8 tiles: every frame is R_0 shifted by t d, so PAR's reconstruction is close
    and the transport phase error small; the linear interpolation is the baseline."""
    rng = np.random.default_rng(4)
    from gen.workloads import fourier_shift, power_law_field
    base = power_law_field(32, 32, 48, 2.0, rng)
    d = np.array([0.3, -0.2])
    ref = np.stack([fourier_shift(base, d * t) for t in range(6)])
    got = run_case(cast_lib, ref, (0, 3, 5), "translation")
    assert float(got["nrmse"][1]) < 0.5


def test_diag_edges_and_bands(cast_lib):
    """Edge tiles of every kind, boundary extrapolation on both sides, four bands,
    channels not a multiple of the 64-lane block, a 4x4 tiling."""
    rng = np.random.default_rng(11)
    for (n, Hg, Wg, D, anchors, tile) in [(7, 14, 13, 80, (2, 5), 8), (5, 11, 11, 16, (0, 1, 3), 4)]:
        base = rng.standard_normal((Hg, Wg, D))
        ref = np.stack([np.roll(base, (t, 2 * t), axis=(0, 1)) + 0.3 * rng.standard_normal((Hg, Wg, D))
                        for t in range(n)])
        run_case(cast_lib, ref, anchors, f"{Hg}x{Wg}x{D} tile{tile}", tile=tile,
                 edges=(0.0, 0.25, 0.5, 0.75, 1.0))


def test_diag_matrix_like(cast_lib):
    """The Matrix-Game-like block with the generator's ground-truth skipped frames."""
    w = gen.get(W.MATRIX)
    ref, _, _ = gen.par_inputs(w, seed=42, frames="all")
    run_case(cast_lib, ref, w.anchors, "matrix")


def test_diag_without_theta(cast_lib):
    w = gen.get(W.TINY)
    ref_np, _, _ = gen.par_inputs(w, seed=3, frames="all")
    ref = torch.from_numpy(ref_np.astype(np.float32)).to("cuda")
    approx = torch.zeros_like(ref)
    cast_lib.cast_par_reconstruct(ref, w.anchors, cast_lib.cast_par_params_default(), out=approx)
    got = cast_lib.cast_spectral_diagnostics(ref, approx, w.anchors)
    torch.cuda.synchronize()
    assert got["phase_err"] is None and got["r_phase"] is None
    want = DG.frame_diagnostics(ref.cpu().numpy().astype(np.float64), approx.cpu().numpy().astype(np.float64),
                                w.anchors, OP.ParParams(), [0.0, float(np.float32(1 / 3)),
                                                            float(np.float32(2 / 3)), 1.0])
    for t, v in want.items():
        assert abs(got["nrmse"][t].item() - v["nrmse"]) <= NRMSE_REL * v["nrmse"]


def test_diag_one_and_eight_bands(cast_lib):
    """The band bookkeeping at its limits: one band (all the error) and eight."""
    rng = np.random.default_rng(12)
    base = rng.standard_normal((16, 16, 8))
    ref = np.stack([np.roll(base, (t, -t), axis=(0, 1)) + 0.2 * rng.standard_normal((16, 16, 8))
                    for t in range(4)])
    got = run_case(cast_lib, ref, (0, 3), "one band", edges=(0.0, 1.0), corr=False)
    assert np.allclose(got["bands"][1:3].cpu().numpy(), 1.0, atol=1e-6)
    run_case(cast_lib, ref, (0, 3), "eight bands", edges=tuple(np.linspace(0.0, 1.0, 9)), corr=False)


def test_diag_tile_shapes(cast_lib):
    """Tile shapes with edges 1, 2, 3 and 7 (each shape has its own kernel):
    15x9 with 8x8 tiles gives 8x8, 8x1, 7x8 and 7x1; 5x7 with 2x3 tiles gives
    2x3, 2x1, 1x3 and 1x1."""
    rng = np.random.default_rng(13)
    for (Hg, Wg, D, tile) in [(15, 9, 40, 8), (5, 7, 300, (2, 3))]:
        base = rng.standard_normal((Hg, Wg, D))
        ref = np.stack([np.roll(base, (t, -t), axis=(0, 1)) + 0.3 * rng.standard_normal((Hg, Wg, D))
                        for t in range(5)])
        run_case(cast_lib, ref, (0, 2, 4), f"{Hg}x{Wg}x{D} tile {tile}", tile=tile)


# ---- phase progress (eq:phase_progress)
# A track (one coefficient over the frames a..b of a pair) is compared where float64
# puts it clear of the decisions fp32 cannot follow: |F_t| >= PROG_MAG times its
# tile column's norm at every frame, every wrapped step at least PROG_STEP from
# +-pi, and a displacement |u_b| >= PROG_DEN.  There the bar is the propagated fp32
# error: an 8x8 orthonormal DFT in fp32 is within 16 eps ||column|| of exact per bin,
# so Arg F_s is within e_s = 16 eps ||column_s|| / |F_s| + 3e-7 (atan2), u_t within
# E_t = 2 (e_a + ... + e_t), and p_t = u_t / u_b within (E_t + |p_t| E_b) / |u_b|.
PROG_MAG, PROG_STEP, PROG_DEN = 1e-3, 1e-2, 5e-2
EPS32 = 2.0 ** -24


def progress_case(cast_lib, ref_np, anchors, tile, label, min_frac=0.5):
    dev = "cuda"
    th, tw = (tile, tile) if np.isscalar(tile) else tile
    ref = torch.from_numpy(ref_np.astype(np.float32)).to(dev)
    dprm = cast_lib.cast_diag_params_default(tile_h=th, tile_w=tw)
    got = cast_lib.cast_phase_progress(ref, anchors, dprm)
    torch.cuda.synchronize()
    ref64 = ref.cpu().numpy().astype(np.float64)
    want = DG.phase_progress_frames(ref64, anchors, th, tw)          # [n, tiles, th, nkx, D]
    n, Hg, Wg, D = ref64.shape
    nkx = tw // 2 + 1
    g = got.cpu().numpy().astype(np.float64).reshape(n, -1, th, nkx, D)
    tl = OP.tiles(Hg, Wg, th, tw)
    defined = np.zeros(g.shape, dtype=bool)
    well = np.zeros(g.shape, dtype=bool)
    bound = np.zeros(g.shape)
    for (a, b) in OP.anchor_pairs(anchors):
        for p, (y0, hp, x0, wp) in enumerate(tl):
            defined[a + 1:b, p, :hp, :wp // 2 + 1, :] = True
            F = np.stack([OP.rfft2_ortho(ref64[t, y0:y0 + hp, x0:x0 + wp]) for t in range(a, b + 1)])
            norm = np.sqrt((np.abs(F) ** 2).sum(axis=(1, 2)))[:, None, None, :]
            steps = DG.wrap_pm_pi(np.diff(np.angle(F), axis=0))
            ok = ((np.abs(F) >= PROG_MAG * norm).all(axis=0)
                  & (np.abs(np.abs(steps) - np.pi) > PROG_STEP).all(axis=0)
                  & (np.abs(steps.sum(axis=0)) >= PROG_DEN))
            # (only the well-conditioned entries use the bound; the others may divide by 0)
            with np.errstate(divide="ignore", invalid="ignore"):
                e = 16 * EPS32 * norm / np.abs(F) + 3e-7
                E = 2.0 * np.cumsum(e, axis=0)                        # E_t for t = a .. b
                ub = np.abs(steps.sum(axis=0))
                pw = np.abs(want[a + 1:b, p, :hp, :wp // 2 + 1, :])
                bound[a + 1:b, p, :hp, :wp // 2 + 1, :] = (E[1:-1] + pw * E[-1][None]) / ub[None]
            well[a + 1:b, p, :hp, :wp // 2 + 1, :] = ok[None]
    # the entries the call must leave alone keep the NaN fill
    assert np.isnan(g[~defined]).all(), label
    err = np.abs(g[well] - want[well])
    frac = well.sum() / max(defined.sum(), 1)
    log(f"[progress {label}] max |dp| {err.max():.2e}, max |dp| / bound "
        f"{(err / bound[well]).max():.2f}, over {int(well.sum())} entries ({frac:.1%} of the defined ones)")
    assert frac > min_frac, (label, frac)
    assert (err <= bound[well] + 1e-6).all(), (label, (err / bound[well]).max())
    return g, want, well


def test_phase_progress_translation(cast_lib):
    """Per-tile circular translations by a fixed integer step per frame: every
    coefficient turns by the same angle each frame, so the progress is alpha."""
    rng = np.random.default_rng(31)
    n, th, tw, D = 9, 8, 8, 70
    Hg, Wg = 16, 24
    steps = [(1, 0), (0, 1), (1, 1), (3, 1), (2, 3), (1, 2)]
    ref = np.zeros((n, Hg, Wg, D))
    for p, (y0, hp, x0, wp) in enumerate(OP.tiles(Hg, Wg, th, tw)):
        base = rng.standard_normal((hp, wp, D))
        for t in range(n):
            ref[t, y0:y0 + hp, x0:x0 + wp] = np.roll(base, (t * steps[p][0], t * steps[p][1]), axis=(0, 1))
    g, want, well = progress_case(cast_lib, ref, (0, 3, 7), 8, "translation")
    for (a, b) in ((0, 3), (3, 7)):
        for t in range(a + 1, b):
            # (turns of exactly +-pi are outside `well`: fp32 may wrap them either way)
            sel = well[t] & (np.abs(want[t] - (t - a) / (b - a)) < 1e-9)
            assert sel.sum() > 1000
            assert np.abs(g[t][sel] - (t - a) / (b - a)).max() <= 1e-4, (t,)


@pytest.mark.parametrize("tile", [8, 4, (5, 3)])
def test_phase_progress_moving_field_and_edge_tiles(cast_lib, tile):
    """A 1/f^2 field moved by a sub-token step per frame plus noise, on a grid whose
    edges leave smaller tiles; three anchors (two pairs, one with four interior
    frames), frames before the first and after the last anchor, channels past a
    multiple of 256."""
    rng = np.random.default_rng(5)
    from gen.workloads import fourier_shift, power_law_field
    base = power_law_field(13, 19, 300, 2.0, rng)
    d = np.array([0.35, -0.6])
    ref = np.stack([fourier_shift(base, d * t) + 0.05 * rng.standard_normal(base.shape)
                    for t in range(10)])
    progress_case(cast_lib, ref, (1, 4, 9), tile, f"tile {tile}")


def test_phase_progress_matrix_like(cast_lib):
    """The Matrix-Game-like block with the generator's ground-truth skipped frames."""
    w = gen.get(W.MATRIX)
    ref, _, _ = gen.par_inputs(w, seed=42, frames="all", D=256)
    progress_case(cast_lib, ref, w.anchors, 8, "matrix-like")


def test_phase_progress_tile_shapes(cast_lib):
    """Tile shapes with edges 1, 2, 3 and 7 (each shape has its own kernel), a pair
    with no interior frame (anchors 2, 3), and channels past a multiple of 256:
    15x9 with 8x8 tiles gives 8x8, 8x1, 7x8 and 7x1; 5x7 with 2x3 tiles gives 2x3,
    2x1, 1x3 and 1x1 (whose real bins carry phases 0 or pi only, most of them
    outside the compared tracks)."""
    rng = np.random.default_rng(14)
    for (Hg, Wg, D, tile, min_frac) in [(15, 9, 40, 8, 0.5), (5, 7, 300, (2, 3), 0.2)]:
        base = rng.standard_normal((Hg, Wg, D))
        ref = np.stack([np.roll(base, (t, -t), axis=(0, 1)) + 0.3 * rng.standard_normal((Hg, Wg, D))
                        for t in range(7)])
        progress_case(cast_lib, ref, (0, 2, 3, 6), tile, f"{Hg}x{Wg}x{D} tile {tile}", min_frac)
