"""Python binding of libcast.so (the MI355X hot path of one CAST block step).

Argument marshalling only: every step of routing, anchor attention and PAR runs in
the library's HIP kernels.  Tensors are torch device tensors (torch supplies the
memory and the current HIP stream); the functions carry the C ABI names and
arguments of include/cast.h, plus small conveniences that allocate outputs and
workspaces with torch.

There is no fallback: if libcast.so is missing or fails to load, every call
raises.
"""
from __future__ import annotations

import ctypes
import os

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libcast.so")

CAST_OK = 0
STATUS_NAMES = {0: "CAST_OK", 1: "CAST_ERR_NULL", 2: "CAST_ERR_SHAPE", 3: "CAST_ERR_ANCHORS",
                4: "CAST_ERR_UNSUPPORTED", 5: "CAST_ERR_WORKSPACE", 6: "CAST_ERR_HIP"}

EXPORTED = ["cast_status_string", "cast_last_error_detail", "cast_abi_version",
            "cast_route_kv_workspace_bytes", "cast_route_kv", "cast_anchor_attn_workspace_bytes",
            "cast_anchor_attn",
            "cast_par_params_default", "cast_par_workspace_bytes", "cast_par_reconstruct",
            "cast_par_reconstruct_noalloc", "cast_par_static_scratch_bytes",
            "cast_coupled_params_default", "cast_wo_gram", "cast_route_coupled_workspace_bytes",
            "cast_route_coupled", "cast_select_params_default",
            "cast_frame_select_workspace_bytes", "cast_frame_select", "cast_diag_params_default",
            "cast_spectral_diagnostics_workspace_bytes", "cast_spectral_diagnostics",
            "cast_phase_progress"]


class CastError(RuntimeError):
    def __init__(self, status: int, detail: str):
        super().__init__(f"{STATUS_NAMES.get(status, status)}: {detail}")
        self.status = status
        self.detail = detail


class ParParams(ctypes.Structure):
    """cast_par_params_t."""
    _fields_ = [("tile_h", ctypes.c_int), ("tile_w", ctypes.c_int),
                ("tau_low", ctypes.c_float), ("tau_high", ctypes.c_float),
                ("q", ctypes.c_float), ("T", ctypes.c_float),
                ("eta_rel", ctypes.c_float), ("eta_abs", ctypes.c_float),
                ("eps", ctypes.c_float), ("gate_mode", ctypes.c_int),
                ("accumulate", ctypes.c_int), ("update_anchors", ctypes.c_int)]


class CoupledParams(ctypes.Structure):
    """cast_coupled_params_t (include/cast.h)."""
    _fields_ = [("l_anc", ctypes.c_float), ("l_rec", ctypes.c_float),
                ("passes", ctypes.c_int), ("tol", ctypes.c_float), ("eps", ctypes.c_float)]


class SelectParams(ctypes.Structure):
    """cast_select_params_t (include/cast.h)."""
    _fields_ = [("lambda_cov", ctypes.c_float), ("eps", ctypes.c_float)]


class DiagParams(ctypes.Structure):
    """cast_diag_params_t (include/cast.h)."""
    _fields_ = [("tile_h", ctypes.c_int), ("tile_w", ctypes.c_int), ("n_bands", ctypes.c_int),
                ("band_edges", ctypes.c_float * 9), ("eps", ctypes.c_float)]


_lib = None
_c = ctypes
_vp, _i, _f, _sz = _c.c_void_p, _c.c_int, _c.c_float, _c.c_size_t


def load(path: str = LIB_PATH):
    """Load libcast.so (after torch, so the library binds to torch's HIP runtime)."""
    global _lib
    if _lib is not None:
        return _lib
    import torch  # noqa: F401  (loads the HIP runtime libcast.so must share)
    if not os.path.exists(path):
        raise RuntimeError(f"{path} is not built; run python -m paper_2609_34144_amd.build")
    lib = ctypes.CDLL(path, mode=ctypes.RTLD_LOCAL)
    lib.cast_status_string.restype = _c.c_char_p
    lib.cast_status_string.argtypes = [_i]
    lib.cast_last_error_detail.restype = _c.c_char_p
    lib.cast_last_error_detail.argtypes = []
    lib.cast_abi_version.restype = _i
    lib.cast_route_kv_workspace_bytes.restype = _sz
    lib.cast_route_kv_workspace_bytes.argtypes = [_i] * 6
    lib.cast_route_kv.restype = _i
    lib.cast_route_kv.argtypes = [_vp, _vp, _i, _i, _i, _i, _i, _i, _i, _f, _vp, _vp,
                                  _c.POINTER(_i), _vp, _sz, _vp]
    lib.cast_anchor_attn.restype = _i
    lib.cast_anchor_attn.argtypes = [_vp, _vp, _vp, _vp, _i, _vp, _vp, _i, _i, _i, _i, _i, _i,
                                     _i, _f, _vp, _vp, _vp, _sz, _vp]
    lib.cast_anchor_attn_workspace_bytes.restype = _sz
    lib.cast_anchor_attn_workspace_bytes.argtypes = [_i] * 7
    lib.cast_par_params_default.restype = None
    lib.cast_par_params_default.argtypes = [_c.POINTER(ParParams)]
    lib.cast_par_workspace_bytes.restype = _sz
    lib.cast_par_workspace_bytes.argtypes = [_i, _i, _i, _i, _i, _c.POINTER(ParParams)]
    lib.cast_par_reconstruct.restype = _i
    lib.cast_par_reconstruct.argtypes = [_vp, _c.POINTER(_i), _i, _i, _i, _i, _i,
                                         _c.POINTER(ParParams), _vp, _vp, _vp, _vp, _vp, _sz, _vp]
    lib.cast_par_reconstruct_noalloc.restype = _i
    lib.cast_par_reconstruct_noalloc.argtypes = [_vp, _c.POINTER(_i), _i, _i, _i, _i, _i,
                                                 _c.POINTER(ParParams), _vp, _vp, _vp, _vp, _vp]
    lib.cast_par_static_scratch_bytes.restype = _sz
    lib.cast_par_static_scratch_bytes.argtypes = []
    lib.cast_coupled_params_default.restype = None
    lib.cast_coupled_params_default.argtypes = [_c.POINTER(CoupledParams)]
    lib.cast_wo_gram.restype = _i
    lib.cast_wo_gram.argtypes = [_vp, _i, _i, _i, _vp, _vp]
    lib.cast_route_coupled_workspace_bytes.restype = _sz
    lib.cast_route_coupled_workspace_bytes.argtypes = [_i] * 6
    lib.cast_route_coupled.restype = _i
    lib.cast_route_coupled.argtypes = [_vp, _vp, _vp, _vp, _c.POINTER(_i), _i, _i, _i, _i, _i, _i,
                                       _i, _i, _f, _c.POINTER(CoupledParams), _vp, _vp,
                                       _c.POINTER(_i), _vp, _sz, _vp]
    lib.cast_select_params_default.restype = None
    lib.cast_select_params_default.argtypes = [_c.POINTER(SelectParams)]
    lib.cast_frame_select_workspace_bytes.restype = _sz
    lib.cast_frame_select_workspace_bytes.argtypes = [_i] * 3
    lib.cast_frame_select.restype = _i
    lib.cast_frame_select.argtypes = [_vp, _vp, _i, _i, _i, _i, _c.POINTER(_i), _i, _i,
                                      _c.POINTER(SelectParams), _vp, _vp, _vp, _vp, _vp, _sz, _vp]
    lib.cast_diag_params_default.restype = None
    lib.cast_diag_params_default.argtypes = [_c.POINTER(DiagParams)]
    lib.cast_spectral_diagnostics_workspace_bytes.restype = _sz
    lib.cast_spectral_diagnostics_workspace_bytes.argtypes = [_i, _i, _i, _i, _c.POINTER(DiagParams)]
    lib.cast_spectral_diagnostics.restype = _i
    lib.cast_spectral_diagnostics.argtypes = [_vp, _vp, _vp, _c.POINTER(_i), _i, _i, _i, _i, _i,
                                              _c.POINTER(DiagParams), _vp, _vp, _vp, _vp, _vp,
                                              _vp, _sz, _vp]
    lib.cast_phase_progress.restype = _i
    lib.cast_phase_progress.argtypes = [_vp, _c.POINTER(_i), _i, _i, _i, _i, _i,
                                        _c.POINTER(DiagParams), _vp, _vp]
    _lib = lib
    return lib


def _check(st: int):
    if st != CAST_OK:
        raise CastError(st, _lib.cast_last_error_detail().decode())


def _ptr(t):
    return None if t is None else t.data_ptr()


def _stream(stream):
    import torch
    if stream is None:
        stream = torch.cuda.current_stream()
    return stream.cuda_stream


def _ws(nbytes: int, device, workspace):
    import torch
    if nbytes == 0:
        return None, 0
    if workspace is not None:
        return workspace, workspace.numel() * workspace.element_size()
    # torch's caching allocator returns >= 512-byte aligned blocks
    return torch.empty(nbytes, dtype=torch.uint8, device=device), nbytes


# ---------------------------------------------------------------------------
# C ABI mirrors
# ---------------------------------------------------------------------------

def cast_abi_version() -> int:
    return load().cast_abi_version()


def cast_route_kv_workspace_bytes(n_a, S, H, dh, M, Bv) -> int:
    return load().cast_route_kv_workspace_bytes(n_a, S, H, dh, M, Bv)


def cast_par_workspace_bytes(n_frames, n_anchor, Hg, Wg, D, params: ParParams) -> int:
    return load().cast_par_workspace_bytes(n_frames, n_anchor, Hg, Wg, D, ctypes.byref(params))


def cast_par_params_default(**overrides) -> ParParams:
    p = ParParams()
    load().cast_par_params_default(ctypes.byref(p))
    for k, v in overrides.items():
        setattr(p, k, v)
    return p


def cast_route_kv(q, k_hist, topk: int, scale: float = 1.0, scores_out=None, idx_out=None,
                  workspace=None, stream=None, want_scores: bool = False):
    """q bf16 [n_a, S, H, dh], k_hist bf16 [M, Bv, H, dh] (device).
    Returns (idx int32 [n_a, H, k_eff], k_eff, scores fp32 [n_a, H, M] or None)."""
    import torch
    lib = load()
    n_a, S, H, dh = q.shape
    M, Bv = k_hist.shape[0], k_hist.shape[1]
    k_eff_guess = min(topk, M)
    if idx_out is None and M > 0:
        idx_out = torch.empty((n_a, H, k_eff_guess), dtype=torch.int32, device=q.device)
    if scores_out is None and want_scores and M > 0:
        scores_out = torch.empty((n_a, H, M), dtype=torch.float32, device=q.device)
    ws, wsb = _ws(lib.cast_route_kv_workspace_bytes(n_a, S, H, dh, M, Bv), q.device, workspace)
    k_eff = ctypes.c_int(-1)
    _check(lib.cast_route_kv(_ptr(q), _ptr(k_hist), n_a, S, H, dh, M, Bv, topk, scale,
                             _ptr(scores_out), _ptr(idx_out), ctypes.byref(k_eff), _ptr(ws), wsb,
                             _stream(stream)))
    return idx_out, k_eff.value, scores_out


def cast_coupled_params_default(**overrides) -> CoupledParams:
    p = CoupledParams()
    load().cast_coupled_params_default(ctypes.byref(p))
    for k, v in overrides.items():
        setattr(p, k, v)
    return p


def cast_route_coupled_workspace_bytes(n_a, S, H, dh, M, Bv) -> int:
    return load().cast_route_coupled_workspace_bytes(n_a, S, H, dh, M, Bv)


def cast_wo_gram(w_o, H: int, dh: int, gram_out=None, stream=None):
    """Gram matrices fp32 [H, dh, dh] of the head slices of w_o bf16 [D, D] (device)."""
    import torch
    lib = load()
    D = w_o.shape[0]
    if gram_out is None:
        gram_out = torch.empty((H, dh, dh), dtype=torch.float32, device=w_o.device)
    _check(lib.cast_wo_gram(_ptr(w_o), D, H, dh, _ptr(gram_out), _stream(stream)))
    return gram_out


def cast_route_coupled(q, k_hist, v_hist, gram, anchors, n_frames: int, topk: int,
                       scale: float, params: CoupledParams | None = None, u_out=None,
                       idx_out=None, workspace=None, stream=None, want_u: bool = False):
    """Reconstruction-coupled routing.  q bf16 [n_a, S, H, dh]; k_hist, v_hist bf16
    [M, Bv, H, dh]; gram fp32 [H, dh, dh] (device); `anchors` the host frame index
    of each row of q.  Returns (idx int32 [n_a, H, k_eff], k_eff, u fp32 [n_a, H, M]
    or None)."""
    import torch
    lib = load()
    if params is None:
        params = cast_coupled_params_default()
    n_a, S, H, dh = q.shape
    M, Bv = k_hist.shape[0], k_hist.shape[1]
    if idx_out is None and M > 0:
        idx_out = torch.empty((n_a, H, min(topk, M)), dtype=torch.int32, device=q.device)
    if u_out is None and want_u and M > 0:
        u_out = torch.empty((n_a, H, M), dtype=torch.float32, device=q.device)
    anc = [int(a) for a in anchors]
    arr = (ctypes.c_int * max(len(anc), 1))(*anc)
    ws, wsb = _ws(lib.cast_route_coupled_workspace_bytes(n_a, S, H, dh, M, Bv), q.device, workspace)
    k_eff = ctypes.c_int(-1)
    _check(lib.cast_route_coupled(_ptr(q), _ptr(k_hist), _ptr(v_hist), _ptr(gram), arr, n_a,
                                  n_frames, S, H, dh, M, Bv, topk, scale, ctypes.byref(params),
                                  _ptr(u_out), _ptr(idx_out), ctypes.byref(k_eff), _ptr(ws), wsb,
                                  _stream(stream)))
    return idx_out, k_eff.value, u_out


def cast_select_params_default(**overrides) -> SelectParams:
    p = SelectParams()
    load().cast_select_params_default(ctypes.byref(p))
    for k, v in overrides.items():
        setattr(p, k, v)
    return p


def cast_frame_select_workspace_bytes(n_cur: int, S: int, D: int) -> int:
    return load().cast_frame_select_workspace_bytes(n_cur, S, D)


def cast_frame_select(delta_cam, delta_act, anchors_prev, k_f: int, ages,
                      params: SelectParams | None = None, n_cur: int | None = None,
                      r_out=None, score_out=None, anchors_out=None, workspace=None, stream=None):
    """Control-aware frame selection.  delta_cam / delta_act: device [n_cur, S, D]
    (fp32 or bf16, the same dtype) or None; `anchors_prev` the host anchors the
    block ran with; `ages` device int32 [n_cur], updated in place.  Returns
    anchors_out (device int32 [k_f], ascending)."""
    import torch
    lib = load()
    if params is None:
        params = cast_select_params_default()
    given = [d for d in (delta_cam, delta_act) if d is not None]
    if given:
        n_cur, S, D = given[0].shape[0], given[0].shape[1], given[0].shape[2]
        dtype = 0 if given[0].dtype == torch.float32 else 1
        device = given[0].device
    else:
        n_cur, S, D, dtype, device = int(n_cur if n_cur is not None else ages.shape[0]), 1, 1, 0, ages.device
    if anchors_out is None:
        anchors_out = torch.empty(k_f, dtype=torch.int32, device=device)
    anc = [int(a) for a in anchors_prev]
    arr = (ctypes.c_int * max(len(anc), 1))(*anc)
    nb = lib.cast_frame_select_workspace_bytes(n_cur, S, D) if given else 0
    ws, wsb = _ws(nb, device, workspace)
    _check(lib.cast_frame_select(_ptr(delta_cam), _ptr(delta_act), dtype, n_cur, S, D, arr,
                                 len(anc), k_f, ctypes.byref(params), _ptr(ages), _ptr(r_out),
                                 _ptr(score_out), _ptr(anchors_out), _ptr(ws), wsb,
                                 _stream(stream)))
    return anchors_out


def cast_diag_params_default(band_edges=None, **overrides) -> DiagParams:
    p = DiagParams()
    load().cast_diag_params_default(ctypes.byref(p))
    for k, v in overrides.items():
        setattr(p, k, v)
    if band_edges is not None:
        p.n_bands = len(band_edges) - 1
        for k, e in enumerate(band_edges):
            p.band_edges[k] = float(e)
    return p


def cast_spectral_diagnostics_workspace_bytes(n_frames, Hg, Wg, D, params: DiagParams) -> int:
    return load().cast_spectral_diagnostics_workspace_bytes(n_frames, Hg, Wg, D, ctypes.byref(params))


def cast_spectral_diagnostics(ref, approx, anchors, params: DiagParams | None = None, theta=None,
                              want_corrections: bool = False, workspace=None, stream=None):
    """Spectral diagnostics of the skipped frames.  ref, approx fp32 [n_frames, Hg,
    Wg, D] (device); theta: PAR's theta_out for the same anchors and tiling, or None.
    Returns dict(nrmse [n_frames], bands [n_frames, n_bands], phase_err [n_frames]
    or None, r_phase, r_mag [n_frames, Hg, Wg, D] or None)."""
    import torch
    lib = load()
    if params is None:
        params = cast_diag_params_default()
    n_frames, Hg, Wg, D = ref.shape
    dev = ref.device
    nrmse = torch.zeros(n_frames, dtype=torch.float32, device=dev)
    bands = torch.zeros((n_frames, params.n_bands), dtype=torch.float32, device=dev)
    perr = torch.zeros(n_frames, dtype=torch.float32, device=dev) if theta is not None else None
    rp = torch.zeros_like(ref) if want_corrections else None
    rm = torch.zeros_like(ref) if want_corrections else None
    anc = [int(a) for a in anchors]
    arr = (ctypes.c_int * max(len(anc), 1))(*anc)
    nb = lib.cast_spectral_diagnostics_workspace_bytes(n_frames, Hg, Wg, D, ctypes.byref(params))
    ws, wsb = _ws(nb, dev, workspace)
    _check(lib.cast_spectral_diagnostics(_ptr(ref), _ptr(approx), _ptr(theta), arr, len(anc),
                                         n_frames, Hg, Wg, D, ctypes.byref(params), _ptr(nrmse),
                                         _ptr(bands), _ptr(perr), _ptr(rp), _ptr(rm), _ptr(ws), wsb,
                                         _stream(stream)))
    return {"nrmse": nrmse, "bands": bands, "phase_err": perr, "r_phase": rp, "r_mag": rm}


def cast_phase_progress(ref, anchors, params: DiagParams | None = None, p_out=None, stream=None):
    """Phase progress of every coefficient over the interior frames of each anchor
    pair.  ref fp32 [n_frames, Hg, Wg, D] (device).  Returns p fp32 [n_frames,
    n_tiles, tile_h * (tile_w // 2 + 1), D]; entries the call does not write keep
    p_out's values (NaN when p_out is None)."""
    import torch
    lib = load()
    if params is None:
        params = cast_diag_params_default()
    n_frames, Hg, Wg, D = ref.shape
    nt = -(-Hg // params.tile_h) * -(-Wg // params.tile_w)
    if p_out is None:
        p_out = torch.full((n_frames, nt, params.tile_h * (params.tile_w // 2 + 1), D), float("nan"),
                           dtype=torch.float32, device=ref.device)
    anc = [int(a) for a in anchors]
    arr = (ctypes.c_int * max(len(anc), 1))(*anc)
    _check(lib.cast_phase_progress(_ptr(ref), arr, len(anc), n_frames, Hg, Wg, D,
                                   ctypes.byref(params), _ptr(p_out), _stream(stream)))
    return p_out


def cast_anchor_attn_workspace_bytes(n_a, S, H, dh, k_eff, n0, Bv) -> int:
    return load().cast_anchor_attn_workspace_bytes(n_a, S, H, dh, k_eff, n0, Bv)


def cast_anchor_attn(q, k_hist, v_hist, idx, k_eff: int, scale: float, k_cur=None, v_cur=None,
                     out=None, lse_out=None, want_lse: bool = False, workspace=None,
                     split: bool = True, stream=None):
    """Routed block-sparse attention of the anchor frames; returns (out bf16, lse or None).
    split=True uses `workspace` (allocated here when None) to split the units of a
    last partial round along the keys; split=False runs every unit whole."""
    import torch
    lib = load()
    n_a, S, H, dh = q.shape
    M, Bv = k_hist.shape[0], k_hist.shape[1]
    n0 = 0 if k_cur is None else k_cur.shape[0]
    if out is None:
        out = torch.empty_like(q)
    if lse_out is None and want_lse:
        lse_out = torch.empty((n_a, H, S), dtype=torch.float32, device=q.device)
    ws, wsb = None, 0
    if split:
        ws, wsb = _ws(lib.cast_anchor_attn_workspace_bytes(n_a, S, H, dh, k_eff, n0, Bv), q.device,
                      workspace)
    _check(lib.cast_anchor_attn(_ptr(q), _ptr(k_hist), _ptr(v_hist), _ptr(idx), k_eff,
                                _ptr(k_cur), _ptr(v_cur), n0, n_a, S, H, dh, M, Bv, scale,
                                _ptr(out), _ptr(lse_out), _ptr(ws), wsb, _stream(stream)))
    return out, lse_out


def cast_par_reconstruct(resid, anchors, params: ParParams | None = None, out=None,
                         theta_out=None, gate_out=None, conf_out=None, workspace=None,
                         stream=None):
    """PAR over resid fp32 [n_frames, Hg, Wg, D] (device) with host `anchors`.
    Writes (or accumulates into) the skipped-frame slots of `out` (default: a new
    zero tensor) and returns it."""
    import torch
    lib = load()
    if params is None:
        params = cast_par_params_default()
    n_frames, Hg, Wg, D = resid.shape
    anc = [int(a) for a in anchors]
    arr = (ctypes.c_int * max(len(anc), 1))(*anc)
    if out is None:
        out = torch.zeros_like(resid)
    nbytes = lib.cast_par_workspace_bytes(n_frames, len(anc), Hg, Wg, D, ctypes.byref(params))
    ws, wsb = _ws(nbytes, resid.device, workspace)
    _check(lib.cast_par_reconstruct(_ptr(resid), arr, len(anc), n_frames, Hg, Wg, D,
                                    ctypes.byref(params), _ptr(out), _ptr(theta_out),
                                    _ptr(gate_out), _ptr(conf_out), _ptr(ws), wsb,
                                    _stream(stream)))
    return out


def cast_par_reconstruct_noalloc(resid, anchors, params: ParParams | None = None, out=None,
                                 theta_out=None, gate_out=None, conf_out=None, stream=None):
    """cast_par_reconstruct with the library's static per-GPU scratch instead of a
    workspace (no device allocation in the call; `out` must be given)."""
    lib = load()
    if params is None:
        params = cast_par_params_default()
    n_frames, Hg, Wg, D = resid.shape
    anc = [int(a) for a in anchors]
    arr = (ctypes.c_int * max(len(anc), 1))(*anc)
    _check(lib.cast_par_reconstruct_noalloc(_ptr(resid), arr, len(anc), n_frames, Hg, Wg, D,
                                            ctypes.byref(params), _ptr(out), _ptr(theta_out),
                                            _ptr(gate_out), _ptr(conf_out), _stream(stream)))
    return out


def cast_par_static_scratch_bytes() -> int:
    return load().cast_par_static_scratch_bytes()


def par_debug_shapes(n_anchor, Hg, Wg, params: ParParams):
    """Shapes of the optional theta/gate ([pairs, tiles, bins]) and conf ([pairs, tiles])."""
    nt = -(-Hg // params.tile_h) * -(-Wg // params.tile_w)
    return (n_anchor - 1, nt, params.tile_h * (params.tile_w // 2 + 1)), (n_anchor - 1, nt)
