"""Property tests of the C ABI's argument checks (no GPU): random shapes, each call
with exactly one invalid argument planted into an otherwise valid call, must
return that argument's documented status before anything is enqueued; the
workspace queries return 0 or a positive multiple of 256 for any integers.

Like test_abi.py, these calls pass fake (never dereferenced) device addresses and
run only where no GPU is visible."""
import ctypes

import pytest
from hypothesis import HealthCheck, given, settings
from hypothesis import strategies as st

import paper_2609_34144_amd as cast
from test_abi import _HAS_GPU

pytestmark = pytest.mark.skipif(_HAS_GPU, reason="fake-pointer validation tests run GPU-less only")

OK, NULL, SHAPE, ANCHORS, UNSUPPORTED, WORKSPACE = 0, 1, 2, 3, 4, 5
A = 1 << 20                      # 256-byte aligned fake addresses: A, 2A, ...
FUZZ = settings(max_examples=150, deadline=None, suppress_health_check=[HealthCheck.function_scoped_fixture])


@pytest.fixture(scope="module")
def lib():
    import os
    if not os.path.exists(cast.LIB_PATH):
        pytest.skip("libcast.so not built (run __graft_entry__.build())")
    return cast.load()


ints = st.integers(min_value=-4, max_value=1 << 17)


@FUZZ
@given(n_a=ints, S=ints, H=ints, dh=ints, M=ints, Bv=ints)
def test_route_workspace_query_any_ints(lib, n_a, S, H, dh, M, Bv):
    for q in (lib.cast_route_kv_workspace_bytes, lib.cast_route_coupled_workspace_bytes):
        nb = q(n_a, S, H, dh, M, Bv)
        assert nb >= 0 and nb % 256 == 0


@FUZZ
@given(n_a=ints, S=ints, H=ints, dh=ints, k_eff=ints, n0=ints, Bv=ints)
def test_attn_workspace_query_any_ints(lib, n_a, S, H, dh, k_eff, n0, Bv):
    nb = lib.cast_anchor_attn_workspace_bytes(n_a, S, H, dh, k_eff, n0, Bv)
    assert nb >= 0 and nb % 256 == 0


@FUZZ
@given(n_frames=st.integers(-2, 600), n_anchor=st.integers(-2, 600), Hg=st.integers(-2, 300),
       Wg=st.integers(-2, 300), D=st.integers(-2, 9000), tile=st.integers(0, 9))
def test_par_workspace_query_any_ints(lib, n_frames, n_anchor, Hg, Wg, D, tile):
    p = cast.cast_par_params_default(tile_h=tile, tile_w=tile)
    nb = lib.cast_par_workspace_bytes(n_frames, n_anchor, Hg, Wg, D, ctypes.byref(p))
    assert nb >= 0 and nb % 256 == 0
    d = cast.cast_diag_params_default(tile_h=tile, tile_w=tile)
    nb = lib.cast_spectral_diagnostics_workspace_bytes(n_frames, Hg, Wg, D, ctypes.byref(d))
    assert nb >= 0 and nb % 256 == 0
    nb = lib.cast_frame_select_workspace_bytes(n_frames, Hg * Wg, D)
    assert nb >= 0 and nb % 256 == 0


# ---- routing: one planted fault per call
ROUTE_FAULTS = ["q_null", "k_null", "idx_null", "keff_null", "q_misaligned", "idx_misaligned", "dh",
                "S", "topk", "ws_null", "ws_small", "ws_misaligned"]


@FUZZ
@given(n_a=st.integers(1, 8), S=st.integers(1, 5000), H=st.integers(1, 32),
       dh=st.sampled_from([32, 64, 128]), M=st.integers(1, 4096), Bv=st.integers(1, 5000),
       topk=st.integers(1, 64), fault=st.sampled_from(ROUTE_FAULTS))
def test_route_single_fault(lib, n_a, S, H, dh, M, Bv, topk, fault):
    need = lib.cast_route_kv_workspace_bytes(n_a, S, H, dh, M, Bv)
    assert need > 0
    arg = dict(q=A, k=2 * A, idx=3 * A, keff=True, ws=4 * A, wsb=need, dh=dh, S=S, topk=topk)
    expect = {"q_null": NULL, "k_null": NULL, "idx_null": NULL, "keff_null": NULL,
              "q_misaligned": SHAPE, "idx_misaligned": SHAPE, "dh": UNSUPPORTED, "S": SHAPE,
              "topk": SHAPE, "ws_null": WORKSPACE, "ws_small": WORKSPACE, "ws_misaligned": WORKSPACE}[fault]
    if fault.endswith("_null") and fault != "ws_null" and fault != "keff_null":
        arg[fault[:-5]] = None
    elif fault == "keff_null":
        arg["keff"] = False
    elif fault == "q_misaligned":
        arg["q"] = A + 2
    elif fault == "idx_misaligned":
        arg["idx"] = 3 * A + 2
    elif fault == "dh":
        arg["dh"] = 48
    elif fault == "S":
        arg["S"] = 0
    elif fault == "topk":
        arg["topk"] = 0
    elif fault == "ws_null":
        arg["ws"], arg["wsb"] = None, 0
    elif fault == "ws_small":
        arg["wsb"] = need - 1
    elif fault == "ws_misaligned":
        arg["ws"] = 4 * A + 64
    k_eff = ctypes.c_int(-7)
    stt = lib.cast_route_kv(arg["q"], arg["k"], n_a, arg["S"], H, arg["dh"], M, Bv, arg["topk"], 1.0,
                            None, arg["idx"], ctypes.byref(k_eff) if arg["keff"] else None,
                            arg["ws"], arg["wsb"], None)
    assert stt == expect, (fault, stt, lib.cast_last_error_detail())


# ---- attention: one planted fault per call
ATTN_FAULTS = ["q_null", "k_null", "v_null", "idx_null", "out_null", "out_misaligned", "idx_misaligned",
               "lse_misaligned", "dh", "k_eff_gt_M", "scale0", "scale_nan", "cur_missing", "ws_misaligned"]


@FUZZ
@given(n_a=st.integers(1, 8), S=st.integers(1, 5000), H=st.integers(1, 32),
       dh=st.sampled_from([32, 64, 128]), M=st.integers(1, 512), Bv=st.integers(1, 5000),
       fault=st.sampled_from(ATTN_FAULTS), data=st.data())
def test_attn_single_fault(lib, n_a, S, H, dh, M, Bv, fault, data):
    k_eff = data.draw(st.integers(1, min(M, 1024)))
    if (M * Bv * H * dh * 2) >= (1 << 32):
        return                                   # the history-size limit is its own check
    arg = dict(q=A, k=2 * A, v=3 * A, idx=4 * A, out=5 * A, dh=dh, k_eff=k_eff, scale=0.125,
               kc=None, vc=None, n0=0, ws=None, wsb=0, lse=None)
    expect = {"q_null": NULL, "k_null": NULL, "v_null": NULL, "idx_null": NULL, "out_null": NULL,
              "out_misaligned": SHAPE, "idx_misaligned": SHAPE, "lse_misaligned": SHAPE, "dh": UNSUPPORTED, "k_eff_gt_M": SHAPE, "scale0": SHAPE,
              "scale_nan": SHAPE, "cur_missing": NULL, "ws_misaligned": WORKSPACE}[fault]
    if fault.endswith("_null"):
        arg[fault[:-5]] = None
    elif fault == "out_misaligned":
        arg["out"] = 5 * A + 8
    elif fault == "idx_misaligned":
        arg["idx"] = 4 * A + 2
    elif fault == "lse_misaligned":
        arg["lse"] = 7 * A + 2
    elif fault == "dh":
        arg["dh"] = 96
    elif fault == "k_eff_gt_M":
        arg["k_eff"] = M + 1
    elif fault == "scale0":
        arg["scale"] = 0.0
    elif fault == "scale_nan":
        arg["scale"] = float("nan")
    elif fault == "cur_missing":
        arg["n0"] = 3
    elif fault == "ws_misaligned":
        arg["ws"], arg["wsb"] = 6 * A + 8, 1 << 30
    stt = lib.cast_anchor_attn(arg["q"], arg["k"], arg["v"], arg["idx"], arg["k_eff"], arg["kc"],
                               arg["vc"], arg["n0"], n_a, S, H, arg["dh"], M, Bv, arg["scale"],
                               arg["out"], arg["lse"], arg["ws"], arg["wsb"], None)
    assert stt == expect, (fault, stt, lib.cast_last_error_detail())


# ---- PAR: one planted fault per call
PAR_FAULTS = ["resid_null", "out_null", "anchors_desc", "anchor_dup", "anchor_range", "one_anchor",
              "tile", "gate_mode", "T", "tau_order", "accumulate_flag", "ws_null", "ws_small",
              "theta_misaligned", "conf_misaligned"]


@FUZZ
@given(n_frames=st.integers(3, 80), Hg=st.integers(1, 96), Wg=st.integers(1, 96),
       D=st.integers(1, 4096), fault=st.sampled_from(PAR_FAULTS), data=st.data())
def test_par_single_fault(lib, n_frames, Hg, Wg, D, fault, data):
    n_anchor = data.draw(st.integers(2, min(n_frames - 1, 8)))
    anchors = sorted(data.draw(st.lists(st.integers(0, n_frames - 1), min_size=n_anchor,
                                        max_size=n_anchor, unique=True)))
    prm = {}
    expect = {"resid_null": NULL, "out_null": NULL, "anchors_desc": ANCHORS, "anchor_dup": ANCHORS,
              "anchor_range": ANCHORS, "one_anchor": ANCHORS, "tile": UNSUPPORTED, "gate_mode": SHAPE,
              "T": SHAPE, "tau_order": SHAPE, "accumulate_flag": SHAPE, "ws_null": WORKSPACE,
              "ws_small": WORKSPACE, "theta_misaligned": SHAPE, "conf_misaligned": SHAPE}[fault]
    if fault == "tile":
        prm["tile_h"] = 9
    elif fault == "gate_mode":
        prm["gate_mode"] = 5
    elif fault == "T":
        prm["T"] = -1.0
    elif fault == "tau_order":
        prm["tau_low"], prm["tau_high"] = 0.9, 0.1
    elif fault == "accumulate_flag":
        prm["accumulate"] = 3
    p = cast.cast_par_params_default(**prm)
    need = lib.cast_par_workspace_bytes(n_frames, n_anchor, Hg, Wg, D,
                                        ctypes.byref(cast.cast_par_params_default()))
    assert need > 0
    resid, out, ws, wsb = A, 1 << 40, 1 << 41, need
    if fault == "resid_null":
        resid = None
    elif fault == "out_null":
        out = None
    elif fault == "anchors_desc":
        anchors = anchors[::-1]
    elif fault == "anchor_dup":
        anchors = anchors[:1] + anchors[:-1]
    elif fault == "anchor_range":
        anchors = anchors[:-1] + [n_frames]
    elif fault == "one_anchor":
        anchors = anchors[:1]
    elif fault == "ws_null":
        ws, wsb = None, 0
    elif fault == "ws_small":
        wsb = need - 1
    theta = conf = None
    if fault == "theta_misaligned":
        theta = (3 << 40) + 2
    elif fault == "conf_misaligned":
        conf = (3 << 40) + 6
    arr = (ctypes.c_int * len(anchors))(*anchors)
    stt = lib.cast_par_reconstruct(resid, arr, len(anchors), n_frames, Hg, Wg, D, ctypes.byref(p), out,
                                   theta, None, conf, ws, wsb, None)
    assert stt == expect, (fault, anchors, stt, lib.cast_last_error_detail())
