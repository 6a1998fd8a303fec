"""GPU parity of the block update at the eligible residual sites (eq:block with
the anchor case, cast_par_params_t.update_anchors) against the float64 oracle.

Anchor slots: one float32 addition per site on both sides, so X_a + R_a must be
bit-identical to the same float32 additions done on the host.  Skipped slots:
rel-RMS <= 1e-4 against oracle/par.py (the PAR bar).  Two sites (visual
attention, then FFN) share one anchor set and update the same hidden state."""
import numpy as np
import pytest
import torch

import gen
from gen import workloads as W
from oracle import par as OP
from test_gpu_parity import log, rel_rms

pytestmark = pytest.mark.gpu

PAR_REL_RMS = 1e-4


def site_update(cast_lib, resid_np, x, anchors, *, accumulate=True, tile=8):
    """One call with update_anchors = 1 on the device hidden state x (in place)."""
    resid = torch.from_numpy(resid_np.astype(np.float32)).to("cuda")
    prm = cast_lib.cast_par_params_default(accumulate=int(accumulate), update_anchors=1,
                                           tile_h=tile, tile_w=tile)
    cast_lib.cast_par_reconstruct(resid, anchors, prm, out=x)
    return x


def check_sites(cast_lib, x0, site_res, anchors, label, tile=8):
    x = torch.from_numpy(x0.astype(np.float32)).to("cuda")
    for r in site_res:
        site_update(cast_lib, r, x, anchors, tile=tile)
    torch.cuda.synchronize()
    got = x.cpu().numpy()
    # anchors: the same float32 additions, in the same order
    want_a = x0.astype(np.float32)
    for r in site_res:
        want_a = want_a + r.astype(np.float32)
    for a in anchors:
        assert np.array_equal(got[a], want_a[a]), (label, a)
    ref = OP.block_sites(x0.astype(np.float64), [r.astype(np.float32).astype(np.float64) for r in site_res],
                         anchors, OP.ParParams(tile_h=tile, tile_w=tile))
    skipped = [t for t in range(x0.shape[0]) if t not in set(anchors)]
    if skipped:
        # the hidden state dominates X_t; measure the error on the summed updates
        upd_ref = ref[skipped] - x0[skipped]
        upd_got = got[skipped].astype(np.float64) - x0[skipped]
        rr = rel_rms(upd_got, upd_ref)
        log(f"[block {label}] {len(site_res)} sites, rel-RMS of the skipped-frame updates {rr:.3e}")
        assert rr <= PAR_REL_RMS, (label, rr)
    return got


def test_block_update_matrix_two_sites(cast_lib):
    w = gen.get(W.MATRIX)
    r_attn, x0, _ = gen.par_inputs(w, seed=42)
    r_ffn, _, _ = gen.par_inputs(w, seed=43)
    check_sites(cast_lib, x0, [r_attn, r_ffn], w.anchors, "matrix attn+ffn")


def test_block_update_edges_and_tilings(cast_lib):
    """Edge tiles (fused 8x8 launch) and a 4x4 tiling (per-class launches), anchors
    on both boundaries and inside."""
    rng = np.random.default_rng(5)
    for (n, Hg, Wg, D, anchors, tile) in [(7, 14, 13, 80, (2, 5), 8), (6, 17, 9, 33, (0, 2, 5), 8),
                                          (5, 11, 11, 16, (0, 1, 3), 4)]:
        sites = []
        for s in range(2):
            base = rng.standard_normal((Hg, Wg, D))
            r = np.zeros((n, Hg, Wg, D))
            for j, a in enumerate(anchors):
                r[a] = np.roll(base, (j, 2 * j + s), axis=(0, 1)) + 0.3 * rng.standard_normal((Hg, Wg, D))
            sites.append(r)
        x0 = rng.standard_normal((n, Hg, Wg, D))
        check_sites(cast_lib, x0, sites, anchors, f"{Hg}x{Wg}x{D} tile{tile}", tile=tile)


def test_block_update_all_anchors_bypass(cast_lib):
    """K_f = N_cur: nothing is reconstructed and every frame gets its own update."""
    rng = np.random.default_rng(6)
    n, Hg, Wg, D = 4, 9, 7, 37
    r = rng.standard_normal((n, Hg, Wg, D))
    x0 = rng.standard_normal((n, Hg, Wg, D))
    got = check_sites(cast_lib, x0, [r], tuple(range(n)), "bypass")
    assert np.array_equal(got, (x0.astype(np.float32) + r.astype(np.float32)))


def test_block_update_write_mode(cast_lib):
    """Write mode with update_anchors: anchor slots hold R_a, skipped slots R_hat_t."""
    w = gen.get(W.TINY)
    r, _, _ = gen.par_inputs(w, seed=42)
    x = torch.full(r.shape, -3.5, device="cuda")
    site_update(cast_lib, r, x, w.anchors, accumulate=False)
    torch.cuda.synchronize()
    got = x.cpu().numpy()
    for a in w.anchors:
        assert np.array_equal(got[a], r[a].astype(np.float32))
    ref = OP.par_reconstruct(r.astype(np.float32).astype(np.float64), w.anchors, OP.ParParams())
    sk = [t for t in range(w.n_frames) if t not in w.anchors]
    assert rel_rms(got[sk], ref[sk]) <= PAR_REL_RMS
