"""C ABI tests that need no GPU: the library loads, exports every symbol that
include/cast.h declares, and each entry point rejects invalid arguments with the
documented status before enqueueing anything (all checks here return before any
HIP call).  Bypass rules of App. A.1 / App. B.3 return OK without work."""
import ctypes

import numpy as np
import os
import re
import subprocess

import pytest

import paper_2609_34144_amd as cast

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "cast.h")

OK, NULL, SHAPE, ANCHORS, UNSUPPORTED, WORKSPACE = 0, 1, 2, 3, 4, 5

# These tests pass fake (never dereferenced) device addresses: every call below has
# at least one argument the validation rejects, so nothing is ever enqueued.  As a
# second guard they only run where no GPU is visible.
try:
    import torch
    _HAS_GPU = torch.cuda.is_available()
except Exception:  # pragma: no cover
    _HAS_GPU = False
pytestmark = pytest.mark.skipif(_HAS_GPU, reason="fake-pointer validation tests run GPU-less only")
A = 1 << 20   # a 256-byte aligned fake address


@pytest.fixture(scope="module")
def lib():
    if not os.path.exists(cast.LIB_PATH):
        pytest.skip("libcast.so not built (run __graft_entry__.build())")
    return cast.load()


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(cast_[a-z_]+)\s*\(", text)))


def test_header_declares_the_boundary():
    names = declared_functions()
    for required in ("cast_route_kv", "cast_anchor_attn", "cast_par_reconstruct"):
        assert required in names
    assert set(names) == set(cast.EXPORTED)


def test_exports_every_declared_symbol(lib):
    out = subprocess.run(["nm", "-D", "--defined-only", cast.LIB_PATH], capture_output=True,
                         text=True, check=True).stdout
    exported = set(re.findall(r" T (cast_[a-z_]+)$", out, flags=re.M))
    for name in declared_functions():
        assert name in exported, name
        assert hasattr(lib, name)


def test_status_strings(lib):
    for code, name in cast.STATUS_NAMES.items():
        assert lib.cast_status_string(code).decode() == name
    assert lib.cast_abi_version() == 2


def test_par_params_default_matches_paper(lib):
    """tab:config_cast: 8x8 tiles, (tau_low, tau_high, q, T) = (0.25, 0.75, 2, 0.10);
    App. A.2: eta = 1e-6 max W + 1e-8, eps = 1e-8."""
    p = cast.cast_par_params_default()
    assert (p.tile_h, p.tile_w) == (8, 8)
    assert abs(p.tau_low - 0.25) < 1e-7 and abs(p.tau_high - 0.75) < 1e-7
    assert abs(p.q - 2.0) < 1e-7 and abs(p.T - 0.10) < 1e-7
    assert abs(p.eta_rel - 1e-6) < 1e-12 and abs(p.eta_abs - 1e-8) < 1e-14
    assert abs(p.eps - 1e-8) < 1e-14
    assert p.gate_mode == 0 and p.accumulate == 0 and p.update_anchors == 0


def _route(lib, *, q=A, k=2 * A, n_a=2, S=64, H=2, dh=32, M=4, Bv=64, topk=2, idx=3 * A, keff=True,
           ws=None, wsb=0):
    k_eff = ctypes.c_int(-7)
    st = lib.cast_route_kv(q, k, n_a, S, H, dh, M, Bv, topk, 1.0, None, idx,
                           ctypes.byref(k_eff) if keff else None, ws, wsb, None)
    return st, k_eff.value


def test_route_validation(lib):
    assert _route(lib, keff=False)[0] == NULL
    assert _route(lib, dh=96)[0] == UNSUPPORTED
    assert _route(lib, M=5000)[0] == UNSUPPORTED
    assert _route(lib, S=0)[0] == SHAPE
    assert _route(lib, topk=0)[0] == SHAPE
    assert _route(lib, q=None)[0] == NULL
    assert _route(lib, idx=None)[0] == NULL
    assert _route(lib, q=A + 8)[0] == SHAPE                       # misaligned
    assert _route(lib, ws=None, wsb=0)[0] == WORKSPACE
    need = lib.cast_route_kv_workspace_bytes(2, 64, 2, 32, 4, 64)
    assert need > 0
    assert _route(lib, ws=4 * A, wsb=need - 1)[0] == WORKSPACE  # too small
    assert _route(lib, ws=4 * A + 8, wsb=need)[0] == WORKSPACE  # misaligned workspace


def test_route_bypass_m0(lib):
    """M == 0: routing is bypassed, k_eff = 0, nothing enqueued (App. B.3)."""
    st, k_eff = _route(lib, q=None, k=None, idx=None, M=0)
    assert st == OK and k_eff == 0
    assert lib.cast_route_kv_workspace_bytes(2, 64, 2, 32, 0, 64) == 0


def _attn(lib, *, q=A, k=2 * A, v=3 * A, idx=4 * A, k_eff=2, kc=None, vc=None, n0=0, n_a=2, S=64, H=2,
          dh=32, M=4, Bv=64, scale=0.5, out=5 * A, ws=None, wsb=0):
    return lib.cast_anchor_attn(q, k, v, idx, k_eff, kc, vc, n0, n_a, S, H, dh, M, Bv, scale,
                                out, None, ws, wsb, None)


def test_attn_validation(lib):
    assert _attn(lib, dh=48) == UNSUPPORTED
    assert _attn(lib, k_eff=5) == SHAPE                  # k_eff > M
    assert _attn(lib, k_eff=0, n0=0) == SHAPE            # nothing to attend to
    assert _attn(lib, scale=0.0) == SHAPE
    assert _attn(lib, scale=float("nan")) == SHAPE
    assert _attn(lib, q=None) == NULL
    assert _attn(lib, idx=None) == NULL
    assert _attn(lib, n0=4) == NULL                      # k_cur / v_cur missing
    assert _attn(lib, ws=6 * A + 8, wsb=1 << 20) == WORKSPACE   # misaligned workspace
    assert lib.cast_anchor_attn_workspace_bytes(2, 64, 2, 48, 2, 0, 64) == 0   # bad dh
    assert lib.cast_anchor_attn_workspace_bytes(2, 64, 2, 32, 0, 0, 64) == 0   # no keys
    assert _attn(lib, out=5 * A + 8) == SHAPE                   # misaligned


def _par(lib, anchors, *, n_frames=4, Hg=8, Wg=8, D=64, resid=A, out=2 * A, ws=None, wsb=0,
         params=None, **pkw):
    p = params if params is not None else cast.cast_par_params_default(**pkw)
    arr = (ctypes.c_int * max(len(anchors), 1))(*anchors)
    return lib.cast_par_reconstruct(resid, arr if anchors is not None else None, len(anchors),
                                    n_frames, Hg, Wg, D, ctypes.byref(p), out, None, None, None,
                                    ws, wsb, None)


def test_par_validation(lib):
    assert _par(lib, [0, 3], n_frames=4, resid=None) == NULL
    assert _par(lib, [3, 0]) == ANCHORS                  # not increasing
    assert _par(lib, [0, 0, 3]) == ANCHORS
    assert _par(lib, [0, 4]) == ANCHORS                  # out of range
    assert _par(lib, [1]) == ANCHORS                     # K_f < 2 (eq:block)
    assert _par(lib, [0, 3], tile_h=9) == UNSUPPORTED
    assert _par(lib, [0, 3], tile_w=0) == UNSUPPORTED
    assert _par(lib, [0, 3], gate_mode=3) == SHAPE
    assert _par(lib, [0, 3], T=0.0) == SHAPE
    assert _par(lib, [0, 3], tau_low=0.8, tau_high=0.7) == SHAPE
    assert _par(lib, [0, 3]) == WORKSPACE
    assert lib.cast_par_reconstruct(A, None, 2, 4, 8, 8, 64,
                                    ctypes.byref(cast.cast_par_params_default()), 2 * A, None,
                                    None, None, None, 0, None) == NULL


def test_par_noalloc_validation(lib):
    """The static-scratch variant validates like cast_par_reconstruct and rejects
    sizes whose scratch exceeds the static array before touching the device."""
    p = cast.cast_par_params_default()
    cap = lib.cast_par_static_scratch_bytes()
    assert cap == 16 << 20
    arr = (ctypes.c_int * 2)(0, 3)
    assert lib.cast_par_reconstruct_noalloc(None, arr, 2, 4, 8, 8, 64, ctypes.byref(p), 2 * A,
                                            None, None, None, None) == NULL
    arr2 = (ctypes.c_int * 2)(3, 0)
    assert lib.cast_par_reconstruct_noalloc(A, arr2, 2, 4, 8, 8, 64, ctypes.byref(p), 2 * A,
                                            None, None, None, None) == ANCHORS
    # 4096 frames of 64x64 tokens x 4096 channels: far more scratch than the array holds
    need = lib.cast_par_workspace_bytes(4096, 2, 64, 64, 4096, ctypes.byref(p))
    assert need > cap
    big = (ctypes.c_int * 2)(0, 4095)
    assert lib.cast_par_reconstruct_noalloc(A, big, 2, 4096, 64, 64, 4096, ctypes.byref(p),
                                            2 * A, None, None, None, None) == WORKSPACE
    assert "static scratch" in lib.cast_last_error_detail().decode()

def test_par_block_update_validation(lib):
    """update_anchors writes anchor slots of out while anchors of resid are read:
    out must not overlap resid; flags are 0 or 1; the bypass then needs buffers."""
    assert _par(lib, [0, 3], update_anchors=2) == SHAPE
    assert _par(lib, [0, 3], accumulate=2) == SHAPE
    assert _par(lib, [0, 3], update_anchors=1, out=A) == SHAPE
    assert _par(lib, [0, 3], update_anchors=1, out=A + 1024) == SHAPE
    assert _par(lib, [0, 3], update_anchors=1, resid=2 * A, out=2 * A - 1024) == SHAPE
    assert _par(lib, [0, 3], update_anchors=1) == WORKSPACE    # no overlap: reaches the workspace check
    assert _par(lib, [0, 1, 2, 3], update_anchors=1, resid=None) == NULL
    assert _par(lib, [0, 1, 2, 3], update_anchors=1, out=A + 4096) == SHAPE


def test_par_bypass_all_anchors(lib):
    """K_f = N_cur: every frame is computed, reconstruction is bypassed (App. A.1)."""
    assert _par(lib, [0, 1, 2, 3], resid=None, out=None) == OK
    assert _par(lib, [0], n_frames=1, resid=None, out=None) == OK
    p = cast.cast_par_params_default()
    assert lib.cast_par_workspace_bytes(4, 4, 8, 8, 64, ctypes.byref(p)) == 0


def test_workspace_queries_grow_with_size(lib):
    p = cast.cast_par_params_default()
    small = lib.cast_par_workspace_bytes(4, 2, 8, 8, 64, ctypes.byref(p))
    big = lib.cast_par_workspace_bytes(66, 2, 64, 64, 3072, ctypes.byref(p))
    assert 0 < small < big
    assert big % 256 == 0


# ---- reconstruction-coupled routing
def test_coupled_params_default_matches_paper(lib):
    """tab:config: (lambda_anc, lambda_rec) = (1, 1), L_s = 2 passes, accept a
    decrease > 1e-6 max(J, 1e-8); stabiliser 1e-8 (reading)."""
    p = cast.cast_coupled_params_default()
    assert (p.l_anc, p.l_rec, p.passes) == (1.0, 1.0, 2)
    assert abs(p.tol - 1e-6) < 1e-12 and abs(p.eps - 1e-8) < 1e-14


def _coupled(lib, *, q=A, k=2 * A, v=3 * A, gram=4 * A, anchors=(0, 3, 7), n_frames=8, S=64, H=2,
             dh=32, M=4, Bv=64, topk=2, idx=5 * A, keff=True, ws=None, wsb=0, params=True, **prm):
    p = cast.cast_coupled_params_default(**prm)
    arr = (ctypes.c_int * max(len(anchors), 1))(*anchors) if anchors is not None else None
    k_eff = ctypes.c_int(-7)
    n_a = len(anchors) if anchors is not None else 3
    st = lib.cast_route_coupled(q, k, v, gram, arr, n_a, n_frames, S, H, dh, M, Bv,
                                topk, 0.5, ctypes.byref(p) if params else None, None, idx,
                                ctypes.byref(k_eff) if keff else None, ws, wsb, None)
    return st, k_eff.value


def test_coupled_validation(lib):
    assert _coupled(lib, keff=False)[0] == NULL
    assert _coupled(lib, params=False)[0] == NULL
    assert _coupled(lib, anchors=None)[0] == NULL
    assert _coupled(lib, anchors=(0, 3, 3))[0] == ANCHORS
    assert _coupled(lib, anchors=(0, 3, 8))[0] == ANCHORS            # outside [0, n_frames)
    assert _coupled(lib, anchors=(2, 1, 5))[0] == ANCHORS
    assert _coupled(lib, n_frames=2)[0] == SHAPE                     # fewer frames than anchors
    assert _coupled(lib, dh=48)[0] == UNSUPPORTED
    assert _coupled(lib, topk=0)[0] == SHAPE
    assert _coupled(lib, l_anc=-1.0)[0] == SHAPE
    assert _coupled(lib, passes=-1)[0] == SHAPE
    assert _coupled(lib, tol=float("nan"))[0] == SHAPE
    assert _coupled(lib, gram=None)[0] == NULL
    assert _coupled(lib, v=None)[0] == NULL
    assert _coupled(lib, v=A + 8)[0] == SHAPE                        # misaligned
    assert _coupled(lib, M=20000, anchors=(0, 1, 2), n_frames=3)[0] == UNSUPPORTED
    assert _coupled(lib, ws=None, wsb=0)[0] == WORKSPACE
    need = lib.cast_route_coupled_workspace_bytes(3, 64, 2, 32, 4, 64)
    assert need > lib.cast_route_kv_workspace_bytes(3, 64, 2, 32, 4, 64)
    assert _coupled(lib, ws=6 * A, wsb=need - 1)[0] == WORKSPACE


def test_coupled_bypass_m0(lib):
    st, k_eff = _coupled(lib, q=None, k=None, v=None, gram=None, idx=None, M=0)
    assert st == OK and k_eff == 0
    assert lib.cast_route_coupled_workspace_bytes(3, 64, 2, 32, 0, 64) == 0


def test_wo_gram_validation(lib):
    assert lib.cast_wo_gram(A, 64, 2, 48, 2 * A, None) == SHAPE      # dh unsupported
    assert lib.cast_wo_gram(A, 60, 2, 32, 2 * A, None) == SHAPE      # D != H * dh
    assert lib.cast_wo_gram(None, 64, 2, 32, 2 * A, None) == NULL
    assert lib.cast_wo_gram(A + 4, 64, 2, 32, 2 * A, None) == SHAPE


# ---- control-aware frame selection
def test_select_params_default_matches_paper(lib):
    """Sec. 4.2 / tab:config_cast: lambda_cov = 0.5; stabiliser 1e-8 (reading)."""
    p = cast.cast_select_params_default()
    assert abs(p.lambda_cov - 0.5) < 1e-7 and abs(p.eps - 1e-8) < 1e-14


def _fsel(lib, *, cam=A, act=2 * A, dtype=1, n_cur=4, S=64, D=64, prev=(0, 3), k_f=2,
          params=None, ages=3 * A, r=None, sc=None, out=4 * A, ws=None, wsb=0, **pkw):
    p = params if params is not None else cast.cast_select_params_default(**pkw)
    arr = (ctypes.c_int * max(len(prev), 1))(*prev) if prev is not None else None
    return lib.cast_frame_select(cam, act, dtype, n_cur, S, D, arr, len(prev or ()), k_f,
                                 ctypes.byref(p), ages, r, sc, out, ws, wsb, None)


def test_frame_select_validation(lib):
    assert _fsel(lib, ages=None) == NULL
    assert _fsel(lib, out=None) == NULL
    assert _fsel(lib, prev=None) == NULL
    assert _fsel(lib, dtype=2) == SHAPE
    assert _fsel(lib, k_f=0) == SHAPE
    assert _fsel(lib, k_f=5) == SHAPE
    assert _fsel(lib, S=0) == SHAPE
    assert _fsel(lib, lambda_cov=-1.0) == SHAPE
    assert _fsel(lib, prev=(3, 0)) == ANCHORS
    assert _fsel(lib, prev=(0, 4)) == ANCHORS
    assert _fsel(lib, prev=(0, 1, 2, 3, 3)) == ANCHORS
    assert _fsel(lib, n_cur=5000) == UNSUPPORTED
    assert _fsel(lib, cam=A + 1) == SHAPE              # bf16 needs 2-byte alignment
    assert _fsel(lib, dtype=0, act=2 * A + 2) == SHAPE  # fp32 needs 4-byte alignment
    assert _fsel(lib) == WORKSPACE
    nb = lib.cast_frame_select_workspace_bytes(4, 64, 64)
    assert nb > 0 and nb % 256 == 0
    assert lib.cast_frame_select_workspace_bytes(0, 64, 64) == 0
    assert lib.cast_frame_select_workspace_bytes(10, 3520, 3072) > nb


# ---- spectral diagnostics
def test_diag_params_default(lib):
    p = cast.cast_diag_params_default()
    assert (p.tile_h, p.tile_w, p.n_bands) == (8, 8, 3)
    assert list(p.band_edges)[:4] == [0.0, np.float32(1 / 3), np.float32(2 / 3), 1.0]
    assert abs(p.eps - 1e-8) < 1e-14


def _diag(lib, *, ref=A, approx=2 * A, theta=None, anchors=(0, 3), n_frames=4, Hg=8, Wg=8, D=64,
          params=None, ws=None, wsb=0, **pkw):
    p = params if params is not None else cast.cast_diag_params_default(**pkw)
    arr = (ctypes.c_int * max(len(anchors), 1))(*anchors)
    return lib.cast_spectral_diagnostics(ref, approx, theta, arr, len(anchors), n_frames, Hg, Wg, D,
                                         ctypes.byref(p), None, None, None, None, None, ws, wsb, None)


def test_diag_validation(lib):
    assert _diag(lib, ref=None) == NULL
    assert _diag(lib, anchors=(1,)) == ANCHORS
    assert _diag(lib, anchors=(3, 1)) == ANCHORS
    assert _diag(lib, anchors=(0, 4)) == ANCHORS
    assert _diag(lib, tile_h=9) == UNSUPPORTED
    assert _diag(lib, n_bands=0) == SHAPE
    assert _diag(lib, band_edges=[0.0, 0.6, 0.5, 1.0]) == SHAPE
    assert _diag(lib, band_edges=[0.1, 1.0]) == SHAPE
    assert _diag(lib, band_edges=[0.0, 0.9]) == SHAPE
    assert _diag(lib, approx=2 * A + 2) == SHAPE
    assert _diag(lib) == WORKSPACE
    p = cast.cast_diag_params_default()
    nb = lib.cast_spectral_diagnostics_workspace_bytes(4, 8, 8, 64, ctypes.byref(p))
    assert nb > 0 and nb % 256 == 0


def _prog(lib, *, ref=A, anchors=(0, 3), n_frames=4, Hg=8, Wg=8, D=64, p_out=2 * A, params=None, **pkw):
    p = params if params is not None else cast.cast_diag_params_default(**pkw)
    arr = (ctypes.c_int * max(len(anchors), 1))(*anchors)
    return lib.cast_phase_progress(ref, arr, len(anchors), n_frames, Hg, Wg, D, ctypes.byref(p),
                                   p_out, None)


def test_phase_progress_validation(lib):
    assert _prog(lib, ref=None) == NULL
    assert _prog(lib, p_out=None) == NULL
    assert lib.cast_phase_progress(A, None, 2, 4, 8, 8, 64, ctypes.byref(cast.cast_diag_params_default()),
                                   2 * A, None) == NULL
    assert lib.cast_phase_progress(A, (ctypes.c_int * 2)(0, 3), 2, 4, 8, 8, 64, None, 2 * A, None) == NULL
    assert _prog(lib, anchors=(1,)) == ANCHORS
    assert _prog(lib, anchors=(3, 1)) == ANCHORS
    assert _prog(lib, anchors=(0, 4)) == ANCHORS
    assert _prog(lib, tile_w=9) == UNSUPPORTED
    assert _prog(lib, n_frames=5000, anchors=(0, 3)) == UNSUPPORTED
    assert _prog(lib, D=0) == SHAPE
    assert _prog(lib, p_out=2 * A + 2) == SHAPE
    assert _prog(lib, ref=A + 1) == SHAPE


def test_binding_wraps_every_entry_point():
    """The Python binding carries every C entry point under its own name."""
    missing = [n for n in cast.EXPORTED
               if n not in ("cast_status_string", "cast_last_error_detail") and not hasattr(cast, n)]
    assert not missing, missing
