"""The degenerate sizes of the hot path on the GPU, against the oracle and the
closed forms they reduce to: one query and one key (attention returns that key's
value row), one history chunk of one token, fewer chunks than the budget; PAR on
one-token frames and single channels (a 1x1 tile's DFT is the identity and its one
bin is self-conjugate, so PAR is the linear interpolation / extrapolation of
eq:block), and a pair of adjacent anchors with nothing to reconstruct.  Then the
largest sizes the boundary accepts: 4096 chunks, 1024 routed chunks, 4096 frames
with 512 anchors."""
import math

import numpy as np
import pytest
import torch

from oracle import attn as OA
from oracle import par as OP
from oracle import route as OR
from test_gpu_parity import ATTN_MAX_ABS, ATTN_REL_RMS, PAR_REL_RMS, log, np64, rel_rms

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("dh", [32, 64, 128])
def test_one_query_one_key(cast_lib, dh):
    dev = "cuda"
    torch.manual_seed(dh)
    q = torch.randn(1, 1, 1, dh, device=dev).to(torch.bfloat16)
    k = torch.randn(1, 1, 1, dh, device=dev).to(torch.bfloat16)
    v = torch.randn(1, 1, 1, dh, device=dev).to(torch.bfloat16)
    print(f"[degenerate] one query, one key, dh {dh}", flush=True)
    idx, k_eff, scores = cast_lib.cast_route_kv(q, k, 1, 1.0 / math.sqrt(dh), want_scores=True)
    out, lse = cast_lib.cast_anchor_attn(q, k, v, idx, k_eff, 1.0 / math.sqrt(dh), want_lse=True)
    torch.cuda.synchronize()
    assert k_eff == 1 and int(idx.item()) == 0
    s_or = OR.chunk_scores(np64(q), np64(k), 1.0 / math.sqrt(dh))
    assert abs(float(scores.item()) - float(s_or[0, 0, 0])) <= 1e-4 * abs(float(s_or[0, 0, 0])) + 1e-7
    # the softmax over one key is 1: the output is that key's value row (to the
    # bf16 rounding of the normalised fp32 accumulation), and the log-sum-exp is
    # that key's scaled logit, which is also the pooled score of a one-token chunk
    vv, oo = np64(v).ravel(), np64(out).ravel()
    assert (np.abs(oo - vv) <= 2.0 ** -8 * np.abs(vv)).all()
    s0 = float(s_or[0, 0, 0])
    assert abs(float(lse.item()) - s0) <= 1e-3 * max(1.0, abs(s0))


@pytest.mark.parametrize("M,topk", [(1, 1), (3, 5), (5, 5)])
def test_short_histories(cast_lib, M, topk):
    """One-token chunks, budgets at and above the number of chunks (App. B.3: all
    kept), several anchors and heads, two queries."""
    dev = "cuda"
    torch.manual_seed(40 + M)
    n_a, S, H, dh, Bv = 3, 2, 2, 64, 1
    q = torch.randn(n_a, S, H, dh, device=dev).to(torch.bfloat16)
    k = torch.randn(M, Bv, H, dh, device=dev).to(torch.bfloat16)
    v = torch.randn(M, Bv, H, dh, device=dev).to(torch.bfloat16)
    print(f"[degenerate] M {M} Bv 1 topk {topk}", flush=True)
    idx, k_eff, _ = cast_lib.cast_route_kv(q, k, topk, 0.125)
    out, _ = cast_lib.cast_anchor_attn(q, k, v, idx, k_eff, 0.125)
    torch.cuda.synchronize()
    assert k_eff == min(topk, M)
    if k_eff == M:
        assert np.array_equal(idx.cpu().numpy(), np.tile(np.arange(M), (n_a, H, 1)))
    O, _ = OA.anchor_attention(np64(q), np64(k), np64(v), idx.cpu().numpy(), 0.125)
    got = np64(out)
    assert np.abs(got - O).max() <= ATTN_MAX_ABS and rel_rms(got, O) <= ATTN_REL_RMS


def test_par_one_token_frames(cast_lib):
    """1x1 grid, one and three channels: the reconstruction is (1 - alpha) R_a +
    alpha R_b for interior and extrapolated frames (alpha = -1, 1/2, 2)."""
    dev = "cuda"
    rng = np.random.default_rng(9)
    for D in (1, 3):
        resid = np.zeros((5, 1, 1, D))
        resid[1] = rng.standard_normal((1, 1, D))
        resid[3] = rng.standard_normal((1, 1, D))
        print(f"[degenerate] PAR 1x1 grid, D {D}", flush=True)
        for gate_mode in (0, 1):
            prm = cast_lib.cast_par_params_default(gate_mode=gate_mode)
            out = torch.full(resid.shape, -2.0, device=dev)
            cast_lib.cast_par_reconstruct(torch.from_numpy(resid.astype(np.float32)).to(dev), (1, 3),
                                          prm, out=out)
            torch.cuda.synchronize()
            got = out.cpu().numpy().astype(np.float64)
            ra, rb = resid[1].astype(np.float32).astype(np.float64), resid[3].astype(np.float32).astype(np.float64)
            for t, alpha in ((0, -0.5), (2, 0.5), (4, 1.5)):
                want = (1 - alpha) * ra + alpha * rb
                assert np.abs(got[t] - want).max() <= 1e-6 * (1 + np.abs(want).max()), (D, t)
            assert (got[1] == -2.0).all() and (got[3] == -2.0).all()
            ref = OP.par_reconstruct(resid.astype(np.float32).astype(np.float64), (1, 3),
                                     OP.ParParams(gate_mode=gate_mode))
            assert rel_rms(got[[0, 2, 4]], ref[[0, 2, 4]]) <= PAR_REL_RMS


def test_par_single_channel_and_adjacent_anchors(cast_lib):
    """One channel on an 11x9 grid (edge tiles), and anchors (0, 1) of a two-frame
    block: no skipped frame, so nothing is written."""
    dev = "cuda"
    rng = np.random.default_rng(10)
    base = rng.standard_normal((11, 9, 1))
    resid = np.stack([base, np.zeros_like(base), np.roll(base, (1, 1), axis=(0, 1)), np.zeros_like(base)])
    print("[degenerate] PAR one channel 11x9; adjacent anchors", flush=True)
    out = torch.zeros(resid.shape, device=dev)
    cast_lib.cast_par_reconstruct(torch.from_numpy(resid.astype(np.float32)).to(dev), (0, 2),
                                  cast_lib.cast_par_params_default(), out=out)
    torch.cuda.synchronize()
    ref = OP.par_reconstruct(resid.astype(np.float32).astype(np.float64), (0, 2), OP.ParParams())
    got = out.cpu().numpy().astype(np.float64)
    assert rel_rms(got[[1, 3]], ref[[1, 3]]) <= PAR_REL_RMS
    two = torch.from_numpy(resid[:2].astype(np.float32)).to(dev)
    out2 = torch.full_like(two, 5.0)
    cast_lib.cast_par_reconstruct(two, (0, 1), cast_lib.cast_par_params_default(), out=out2)
    torch.cuda.synchronize()
    assert (out2 == 5.0).all()


# ---- the largest sizes the boundary accepts
def test_route_4096_chunks(cast_lib):
    """M = 4096 chunks (the bitonic selection's whole LDS key array) with exact ties."""
    from test_gpu_parity import check_route
    dev = "cuda"
    torch.manual_seed(4096)
    q = torch.randn(2, 3, 2, 32, device=dev).to(torch.bfloat16)
    k = torch.randn(4096, 2, 2, 32, device=dev).to(torch.bfloat16)
    k[4095] = k[17]
    print("[max sizes] route M 4096", flush=True)
    for topk in (1, 1000, 4096):
        check_route(cast_lib, q, k, topk, 0.2, f"M4096 k{topk}")


def test_attn_1024_routed_chunks(cast_lib):
    """k_eff = 1024 routed chunks (the most the kernel takes) of 3 tokens each, with
    a current segment: 3,104 keys, the general copy mode, the key split."""
    from test_gpu_parity import check_attn
    dev = "cuda"
    torch.manual_seed(1024)
    n_a, S, H, dh, M, Bv, n0 = 1, 40, 1, 64, 1500, 3, 32
    q = torch.randn(n_a, S, H, dh, device=dev).to(torch.bfloat16)
    k = torch.randn(M, Bv, H, dh, device=dev).to(torch.bfloat16)
    v = torch.randn(M, Bv, H, dh, device=dev).to(torch.bfloat16)
    kc = torch.randn(n0, H, dh, device=dev).to(torch.bfloat16)
    vc = torch.randn(n0, H, dh, device=dev).to(torch.bfloat16)
    rng = np.random.default_rng(1024)
    idx = torch.tensor(np.sort(rng.choice(M, size=(n_a, H, 1024), replace=True), axis=-1),
                       dtype=torch.int32, device=dev)
    print("[max sizes] attention k_eff 1024", flush=True)
    check_attn(cast_lib, q, k, v, idx, 1024, 1 / math.sqrt(dh), kc=kc, vc=vc, label="k_eff 1024")


def test_par_4096_frames_512_anchors(cast_lib):
    """n_frames = 4096 and n_anchor = 512 (the largest accepted), 511 pairs with
    frames before the first anchor and after the last, write and accumulate modes."""
    dev = "cuda"
    rng = np.random.default_rng(512)
    n = 4096
    anchors = tuple(range(3, n, 8))[:512]
    resid = np.zeros((n, 2, 3, 2))
    for a in anchors:
        resid[a] = rng.standard_normal((2, 3, 2))
    print(f"[max sizes] PAR {n} frames, {len(anchors)} anchors", flush=True)
    ref = OP.par_reconstruct(resid.astype(np.float32).astype(np.float64), anchors, OP.ParParams())
    out = torch.zeros(resid.shape, device=dev)
    cast_lib.cast_par_reconstruct(torch.from_numpy(resid.astype(np.float32)).to(dev), anchors,
                                  cast_lib.cast_par_params_default(), out=out)
    torch.cuda.synchronize()
    sk = [t for t in range(n) if t not in set(anchors)]
    got = out.cpu().numpy().astype(np.float64)
    assert rel_rms(got[sk], ref[sk]) <= PAR_REL_RMS
    assert (got[list(anchors)] == 0.0).all()
