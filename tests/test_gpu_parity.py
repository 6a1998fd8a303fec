"""GPU parity: the HIP path (through the C ABI) against the float64 oracle on
identical seeded inputs.

Bars (written here, used everywhere below):
  routing indices   bit-exact wherever the oracle's fp32 K-th / (K+1)-th score gap
                    exceeds the fp32 accumulation bound; inside that bound the
                    selection must be a valid TopK of the oracle scores
  attention         max-abs <= 2e-2 and rel-RMS <= 5e-3 over the whole output
  PAR               rel-RMS <= 1e-4 over the written skipped-frame slots; anchor
                    slots of `out` bit-identical to what they held before
rel-RMS = ||x - y||_2 / ||y||_2.
"""
import math

import numpy as np
import pytest
import torch

import gen
from gen import workloads as W
from oracle import attn as OA
from oracle import par as OP
from oracle import route as OR

pytestmark = pytest.mark.gpu

ATTN_MAX_ABS, ATTN_REL_RMS = 2e-2, 5e-3
PAR_REL_RMS = 1e-4


def rel_rms(x, y):
    x = np.asarray(x, np.float64)
    y = np.asarray(y, np.float64)
    return float(np.linalg.norm((x - y).ravel()) / max(np.linalg.norm(y.ravel()), 1e-300))


def log(msg):
    print(msg, flush=True)


def np64(t):
    return t.detach().float().cpu().numpy().astype(np.float64)


# ---------------------------------------------------------------------------
# routing
# ---------------------------------------------------------------------------

def check_route(cast_lib, q, k, topk, scale, label):
    idx, k_eff, scores = cast_lib.cast_route_kv(q, k, topk, scale, want_scores=True)
    torch.cuda.synchronize()
    s_or = OR.chunk_scores(np64(q), np64(k), scale)                 # fp64
    n_a, H, M = s_or.shape
    assert k_eff == min(topk, M)
    s_gpu = scores.cpu().numpy().astype(np.float64)
    smax = np.abs(s_or).max() + 1e-30
    tol = 1e-4 * smax + 1e-7
    assert np.abs(s_gpu - s_or).max() <= tol, (label, np.abs(s_gpu - s_or).max(), tol)
    s32 = s_or.astype(np.float32)
    g = idx.cpu().numpy()
    exact = near = 0
    for i in range(n_a):
        for h in range(H):
            want = OR.topk_select(s32[i, h], k_eff)
            got = [int(x) for x in g[i, h]]
            assert got == sorted(got), "indices must be ascending"
            assert len(set(got)) == k_eff and all(0 <= x < M for x in got)
            order = sorted(range(M), key=lambda m: (-float(s32[i, h, m]), m))
            kth = float(s32[i, h, order[k_eff - 1]])
            nxt = float(s32[i, h, order[k_eff]]) if k_eff < M else -math.inf
            if kth - nxt > 2 * tol:
                assert got == want, (label, i, h, got, want)
                exact += 1
            else:
                near += 1
                sel = set(got)
                for m in range(M):
                    if m in sel:
                        assert s_or[i, h, m] >= kth - 2 * tol
                    else:
                        assert s_or[i, h, m] <= kth + 2 * tol
    log(f"[route {label}] exact rows {exact}, near-tie rows {near}, max|ds| "
        f"{np.abs(s_gpu - s_or).max():.2e}")
    return idx, k_eff


def test_route_tiny(cast_lib):
    w = gen.get(W.TINY)
    q, k, v, _, _ = gen.attn_inputs(w, seed=42, device="cuda")
    check_route(cast_lib, q, k, w.topk, 1.0, "tiny")


def test_route_matrix_like(cast_lib):
    w = gen.get(W.MATRIX)
    q, k, v, _, _ = gen.attn_inputs(w, seed=42, device="cuda")
    check_route(cast_lib, q, k, w.topk, w.scale, "matrix")


def test_route_ties_and_budget(cast_lib):
    """Byte-identical chunks score identically on both sides: the lower index wins
    (exact tie rule); topk >= M keeps every chunk (App. B.3)."""
    w = gen.get(W.TINY)
    q, k, _, _, _ = gen.attn_inputs(w, seed=7, device="cuda", M=9, Bv=40,
                                    duplicate_chunks=[(5, 2), (8, 2), (7, 0)])
    idx, k_eff, scores = cast_lib.cast_route_kv(q, k, 1, 1.0, want_scores=True)
    torch.cuda.synchronize()
    s = scores.cpu().numpy()
    assert np.array_equal(s[:, :, 5], s[:, :, 2]) and np.array_equal(s[:, :, 8], s[:, :, 2])
    g = idx.cpu().numpy()
    for i in range(g.shape[0]):
        for h in range(g.shape[1]):
            best = max(range(9), key=lambda m: (float(s[i, h, m]), -m))
            assert int(g[i, h, 0]) == best
            assert best not in (5, 8, 7)           # a duplicate never beats its lower twin
    idx_all, k_all, _ = cast_lib.cast_route_kv(q, k, 50, 1.0)
    torch.cuda.synchronize()
    assert k_all == 9
    assert np.array_equal(idx_all.cpu().numpy(), np.tile(np.arange(9), (2, 2, 1)))
    check_route(cast_lib, q, k, 4, 0.3, "ties")


@pytest.mark.parametrize("M", [64, 65, 256, 257, 1000])
def test_route_many_chunks(cast_lib, M):
    """Chunk counts around the TopK's paths: rank counting (one wave per 64 chunks,
    up to 256 chunks) and the bitonic sorts above; budgets below, at and above a
    multiple of 64, with byte-identical duplicate chunks for exact ties."""
    torch.manual_seed(500 + M)
    dev = "cuda"
    n_a, S, H, dh, Bv = 2, 40, 3, 64, 24
    q = torch.randn(n_a, S, H, dh, device=dev).to(torch.bfloat16)
    k = torch.randn(M, Bv, H, dh, device=dev).to(torch.bfloat16)
    k[M - 1] = k[3]                                   # exact tie: chunk 3 must win it
    k[M // 2] = k[1]
    for topk in (1, 7, 64, 100):
        check_route(cast_lib, q, k, topk, 0.125, f"M{M} k{topk}")

def test_route_workspace_reuse(cast_lib):
    """One workspace serves consecutive calls of different shapes (channel groups
    of one, two or four heads, a partial last group; rank-count and bitonic
    selection): each call must match a call on a fresh workspace bit for bit, so
    nothing a call leaves in the workspace reaches the next one."""
    dev = "cuda"
    shapes = [  # n_a, S, H, dh, M, Bv, topk
        (3, 100, 12, 128, 16, 70, 4),
        (2, 33, 5, 64, 40, 17, 7),
        (4, 50, 3, 32, 9, 31, 2),
        (1, 64, 6, 32, 256, 8, 30),
        (2, 40, 3, 64, 300, 12, 9),
        (3, 100, 12, 128, 16, 70, 4),
    ]
    nb = max(cast_lib.cast_route_kv_workspace_bytes(*s[:6]) for s in shapes)
    ws = torch.full((nb,), 0x7f, dtype=torch.uint8, device=dev)
    for j, (n_a, S, H, dh, M, Bv, topk) in enumerate(shapes):
        torch.manual_seed(900 + j)
        q = torch.randn(n_a, S, H, dh, device=dev).to(torch.bfloat16)
        k = (torch.randn(M, Bv, H, dh, device=dev)
             + torch.randn(M, 1, H, dh, device=dev)).to(torch.bfloat16)
        for _ in range(2):
            a = cast_lib.cast_route_kv(q, k, topk, 0.2, want_scores=True, workspace=ws)
            b = cast_lib.cast_route_kv(q, k, topk, 0.2, want_scores=True)
            torch.cuda.synchronize()
            assert torch.equal(a[0], b[0]) and torch.equal(a[2], b[2]), (j, n_a, H, dh, M)
        check_route(cast_lib, q, k, topk, 0.2, f"reuse{j}")


def test_route_deterministic(cast_lib):
    w = gen.get(W.MATRIX)
    q, k, _, _, _ = gen.attn_inputs(w, seed=3, device="cuda")
    a = cast_lib.cast_route_kv(q, k, 4, 0.1, want_scores=True)
    b = cast_lib.cast_route_kv(q, k, 4, 0.1, want_scores=True)
    torch.cuda.synchronize()
    assert torch.equal(a[0], b[0]) and torch.equal(a[2], b[2])


# ---------------------------------------------------------------------------
# attention
# ---------------------------------------------------------------------------

def check_attn(cast_lib, q, k, v, idx, k_eff, scale, kc=None, vc=None, rows=None, label="",
               split=True):
    out, lse = cast_lib.cast_anchor_attn(q, k, v, idx, k_eff, scale, k_cur=kc, v_cur=vc,
                                         want_lse=True, split=split)
    torch.cuda.synchronize()
    O, L = OA.anchor_attention(np64(q), np64(k), np64(v), idx.cpu().numpy() if idx is not None
                               else np.zeros((q.shape[0], q.shape[2], 0), np.int32), scale,
                               k_cur=None if kc is None else np64(kc),
                               v_cur=None if vc is None else np64(vc), rows=rows)
    got = np64(out)
    lg = lse.cpu().numpy().astype(np.float64)
    if rows is not None:
        sel = tuple(np.array(r) for r in zip(*[(i, s, h) for (i, h, s) in rows]))
        got, O = got[sel], O[sel]
        lsel = tuple(np.array(r) for r in zip(*[(i, h, s) for (i, h, s) in rows]))
        lg, L = lg[lsel], L[lsel]
    mx = np.abs(got - O).max()
    rr = rel_rms(got, O)
    log(f"[attn {label}] max-abs {mx:.3e} rel-RMS {rr:.3e} lse max-abs {np.abs(lg - L).max():.2e}")
    assert mx <= ATTN_MAX_ABS and rr <= ATTN_REL_RMS, (label, mx, rr)
    assert np.abs(lg - L).max() <= 1e-3 * max(1.0, np.abs(L).max())
    return out


def test_attn_tiny(cast_lib):
    w = gen.get(W.TINY)
    q, k, v, _, _ = gen.attn_inputs(w, seed=42, device="cuda")
    idx, k_eff = check_route(cast_lib, q, k, w.topk, 1.0, "tiny")
    check_attn(cast_lib, q, k, v, idx, k_eff, w.scale, label="tiny")


@pytest.mark.parametrize("dh", [32, 64, 128])
def test_attn_shapes_and_ragged_tails(cast_lib, dh):
    """Several 128-query tiles plus a ragged query tail; a key sequence that is
    not a multiple of the 64-key tile; chunk lengths that straddle tiles; an
    always-attended current segment; routed indices in arbitrary order."""
    torch.manual_seed(dh)
    n_a, S, H, M, Bv, n0 = 2, 300, 3, 7, 45, 19
    dev = "cuda"
    q = torch.randn(n_a, S, H, dh, device=dev).to(torch.bfloat16)
    k = torch.randn(M, Bv, H, dh, device=dev).to(torch.bfloat16)
    v = torch.randn(M, Bv, H, dh, device=dev).to(torch.bfloat16)
    kc = torch.randn(n0, H, dh, device=dev).to(torch.bfloat16)
    vc = torch.randn(n0, H, dh, device=dev).to(torch.bfloat16)
    idx = torch.tensor([[[6, 1, 3], [0, 2, 5], [4, 4, 1]], [[2, 3, 6], [5, 0, 1], [6, 5, 4]]],
                       dtype=torch.int32, device=dev)
    check_attn(cast_lib, q, k, v, idx, 3, 1 / math.sqrt(dh), kc=kc, vc=vc, label=f"ragged dh{dh}")
    # current segment only (k_eff = 0) and history only (n0 = 0)
    check_attn(cast_lib, q, k, v, idx[:, :, :0].contiguous(), 0, 1 / math.sqrt(dh), kc=kc, vc=vc,
               label=f"n0-only dh{dh}")
    check_attn(cast_lib, q, k, v, idx, 3, 1 / math.sqrt(dh), label=f"hist-only dh{dh}")


@pytest.mark.parametrize("dh", [32, 64, 128])
def test_attn_fast_and_aligned_modes(cast_lib, dh):
    """History-only sequences whose chunks have >= 64 rows: chunks that are not a
    multiple of the 64-key tile (tiles straddle two chunks), chunks that are (no
    tile straddles), and a single routed chunk; ragged query tails; routed
    indices in arbitrary order with a repeated chunk."""
    torch.manual_seed(100 + dh)
    dev = "cuda"
    for (S, M, Bv, idx_rows) in [(300, 5, 100, [[4, 0, 2], [1, 1, 3]]),
                                 (270, 6, 128, [[5, 2, 0], [3, 4, 1]]),
                                 (70, 3, 64, [[2], [0]])]:
        n_a, H = 1, 2
        q = torch.randn(n_a, S, H, dh, device=dev).to(torch.bfloat16)
        k = torch.randn(M, Bv, H, dh, device=dev).to(torch.bfloat16)
        v = torch.randn(M, Bv, H, dh, device=dev).to(torch.bfloat16)
        idx = torch.tensor([idx_rows], dtype=torch.int32, device=dev)
        check_attn(cast_lib, q, k, v, idx, idx.shape[2], 1 / math.sqrt(dh),
                   label=f"modes dh{dh} Bv{Bv}")


@pytest.mark.parametrize("dh", [64, 128])
@pytest.mark.parametrize("Bv,k_eff,n0", [
    (64, 1, 0), (64, 2, 0), (64, 3, 0),      # aligned mode: 1, 2, 3 key tiles
    (100, 1, 0), (100, 2, 0), (70, 3, 0),    # fast mode: 2, 4, 4 key tiles, ragged last one
    (30, 0, 70), (30, 2, 70), (20, 1, 5),    # general mode: 2, 3, 1 key tiles
])
def test_attn_short_key_sequences(cast_lib, dh, Bv, k_eff, n0):
    """Key sequences of one to four 64-key tiles in every copy mode: the tiles that
    the first copies fill (K[0], V[0] before the loop, K[1], V[1] with tile 0) and
    the copy cursor held at the last tile."""
    torch.manual_seed(500 + dh + Bv + k_eff + n0)
    dev = "cuda"
    n_a, S, H, M = 2, 140, 2, 4
    q = torch.randn(n_a, S, H, dh, device=dev).to(torch.bfloat16)
    k = torch.randn(M, Bv, H, dh, device=dev).to(torch.bfloat16)
    v = torch.randn(M, Bv, H, dh, device=dev).to(torch.bfloat16)
    kc = torch.randn(n0, H, dh, device=dev).to(torch.bfloat16) if n0 else None
    vc = torch.randn(n0, H, dh, device=dev).to(torch.bfloat16) if n0 else None
    rng = np.random.default_rng(k_eff * 7 + Bv)
    idx = torch.tensor(rng.integers(0, M, size=(n_a, H, k_eff)), dtype=torch.int32, device=dev)
    check_attn(cast_lib, q, k, v, idx, k_eff, 1 / math.sqrt(dh), kc=kc, vc=vc,
               label=f"short dh{dh} Bv{Bv} k{k_eff} n0 {n0}")


@pytest.mark.parametrize("Bv,k_eff,n0", [(64, 96, 0), (72, 70, 0), (40, 80, 13)])
def test_attn_many_routed_chunks(cast_lib, Bv, k_eff, n0):
    """More than 64 routed chunks (the kernel keeps the first 64 chunk indices in a
    register and reads the others from LDS), in the aligned (chunks of 64 rows),
    fast (chunks of >= 64 rows) and general (current segment, short chunks) copy
    modes; routed indices in arbitrary order with repeats."""
    torch.manual_seed(300 + Bv)
    dev = "cuda"
    n_a, S, H, dh, M = 1, 70, 2, 128, 120
    q = torch.randn(n_a, S, H, dh, device=dev).to(torch.bfloat16)
    k = torch.randn(M, Bv, H, dh, device=dev).to(torch.bfloat16)
    v = torch.randn(M, Bv, H, dh, device=dev).to(torch.bfloat16)
    kc = torch.randn(max(n0, 1), H, dh, device=dev).to(torch.bfloat16) if n0 else None
    vc = torch.randn(max(n0, 1), H, dh, device=dev).to(torch.bfloat16) if n0 else None
    rng = np.random.default_rng(Bv)
    idx = torch.tensor(rng.integers(0, M, size=(n_a, H, k_eff)), dtype=torch.int32, device=dev)
    check_attn(cast_lib, q, k, v, idx, k_eff, 1 / math.sqrt(dh), kc=kc, vc=vc,
               label=f"many chunks Bv{Bv} k{k_eff} n0 {n0}")


@pytest.mark.parametrize("dh", [32, 64, 128])
@pytest.mark.parametrize("n_a,S,H,M,Bv,k_eff,n0", [
    (1, 300, 2, 30, 100, 24, 37),    # general copy mode, 2 pieces, ragged key and query tails
    (2, 256, 3, 128, 64, 128, 0),    # aligned mode, 8 pieces
    (1, 70, 2, 64, 72, 60, 0),       # fast mode, 4 pieces, ragged last key tile
    (1, 320, 2, 40, 64, 40, 0),      # last Q tile of exactly two live waves, aligned mode
])
def test_attn_key_split(cast_lib, dh, n_a, S, H, M, Bv, k_eff, n0):
    """Work units of a last partial round split along the keys (pieces merged by
    their log-sum-exps): the split run and the unsplit run (no workspace) both
    meet the oracle's bar, and they agree with each other to bf16 rounding."""
    need = cast_lib.cast_anchor_attn_workspace_bytes(n_a, S, H, dh, k_eff, n0, Bv)
    assert need > 0, "these sizes must take the split path"
    torch.manual_seed(400 + dh + Bv)
    dev = "cuda"
    q = torch.randn(n_a, S, H, dh, device=dev).to(torch.bfloat16)
    k = torch.randn(M, Bv, H, dh, device=dev).to(torch.bfloat16)
    v = torch.randn(M, Bv, H, dh, device=dev).to(torch.bfloat16)
    kc = torch.randn(n0, H, dh, device=dev).to(torch.bfloat16) if n0 else None
    vc = torch.randn(n0, H, dh, device=dev).to(torch.bfloat16) if n0 else None
    rng = np.random.default_rng(dh + Bv)
    idx = torch.tensor(rng.integers(0, M, size=(n_a, H, k_eff)), dtype=torch.int32, device=dev)
    a = check_attn(cast_lib, q, k, v, idx, k_eff, 1 / math.sqrt(dh), kc=kc, vc=vc,
                   label=f"split dh{dh} Bv{Bv}")
    b = check_attn(cast_lib, q, k, v, idx, k_eff, 1 / math.sqrt(dh), kc=kc, vc=vc,
                   label=f"unsplit dh{dh} Bv{Bv}", split=False)
    d = (a.float() - b.float()).abs().max().item()
    log(f"[attn split vs unsplit dh{dh} Bv{Bv}] max-abs {d:.3e} (workspace {need} B)")
    assert d <= 2.0 ** -7 * max(1.0, b.float().abs().max().item())


@pytest.mark.parametrize("dh", [64, 128])
def test_attn_softmax_paths(cast_lib, dh):
    """Logit ranges that drive every branch of the online softmax: history chunks
    whose keys are scaled from 0.05 to 12 in an order that raises the running max
    by far more than its slack several times (exact path, O rescale), tiles far
    below the running max (probabilities that underflow to 0 on the common path),
    a first tile much larger than the rest, and ties of whole tiles at the max; in
    the aligned (64-row chunks), fast (96-row chunks) and general (current segment)
    copy modes, split and unsplit."""
    torch.manual_seed(900 + dh)
    dev = "cuda"
    n_a, S, H, M = 1, 300, 2, 10
    gains = [0.1, 0.1, 3.0, 0.05, 6.0, 0.1, 12.0, 0.05, 12.0, 0.2]
    for Bv, n0 in ((64, 0), (96, 0), (64, 9)):
        q = torch.randn(n_a, S, H, dh, device=dev).to(torch.bfloat16)
        k = torch.randn(M, Bv, H, dh, device=dev)
        for c, gn in enumerate(gains):
            k[c] *= gn
        k[8] = k[6]                                   # identical tiles at the max
        k = k.to(torch.bfloat16)
        v = torch.randn(M, Bv, H, dh, device=dev).to(torch.bfloat16)
        kc = (8.0 * torch.randn(n0, H, dh, device=dev)).to(torch.bfloat16) if n0 else None
        vc = torch.randn(n0, H, dh, device=dev).to(torch.bfloat16) if n0 else None
        for order in ([0, 1, 2, 3, 4, 5, 6, 7, 8, 9], [6, 0, 1, 3, 5, 7, 9, 2, 4, 8]):
            idx = torch.tensor([[order, order[::-1]]], dtype=torch.int32, device=dev)
            for split in (True, False):
                check_attn(cast_lib, q, k, v, idx, M, 1 / math.sqrt(dh), kc=kc, vc=vc,
                           label=f"softmax paths dh{dh} Bv{Bv} n0 {n0} {order[0]} split {split}",
                           split=split)

def test_attn_topk_all_equals_dense(cast_lib):
    """topk = M routes every chunk: the result is dense attention over the whole history."""
    w = gen.get(W.TINY)
    q, k, v, _, _ = gen.attn_inputs(w, seed=5, device="cuda")
    idx, k_eff, _ = cast_lib.cast_route_kv(q, k, w.M, 1.0)
    assert k_eff == w.M
    out = check_attn(cast_lib, q, k, v, idx, k_eff, w.scale, label="dense")
    ref = torch.nn.functional.scaled_dot_product_attention(
        q.float().permute(0, 2, 1, 3),
        k.float().permute(2, 0, 1, 3).reshape(1, w.H, w.M * w.Bv, w.dh).expand(w.n_a, -1, -1, -1),
        v.float().permute(2, 0, 1, 3).reshape(1, w.H, w.M * w.Bv, w.dh).expand(w.n_a, -1, -1, -1),
        scale=w.scale).permute(0, 2, 1, 3)
    assert (out.float() - ref).abs().max().item() <= ATTN_MAX_ABS


def test_attn_matrix_like_sampled(cast_lib):
    """Full Matrix-Game-like shapes (3 anchors x 12 heads x 1560 queries over 4 routed
    chunks of 1560 tokens), checked on sampled query rows of every (anchor, head)."""
    w = gen.get(W.MATRIX)
    q, k, v, _, _ = gen.attn_inputs(w, seed=42, device="cuda")
    idx, k_eff = check_route(cast_lib, q, k, w.topk, w.scale, "matrix")
    rng = np.random.default_rng(0)
    rows = [(i, h, int(s)) for i in range(w.n_a) for h in range(w.H)
            for s in list(rng.choice(w.S, 24, replace=False)) + [0, w.S - 1, 1535, 1536]]
    check_attn(cast_lib, q, k, v, idx, k_eff, w.scale, rows=rows, label="matrix sampled")


def test_attn_deterministic(cast_lib):
    w = gen.get(W.TINY)
    q, k, v, _, _ = gen.attn_inputs(w, seed=11, device="cuda")
    idx, k_eff, _ = cast_lib.cast_route_kv(q, k, 2, 1.0)
    a, _ = cast_lib.cast_anchor_attn(q, k, v, idx, k_eff, w.scale)
    b, _ = cast_lib.cast_anchor_attn(q, k, v, idx, k_eff, w.scale)
    torch.cuda.synchronize()
    assert torch.equal(a, b)


# ---------------------------------------------------------------------------
# PAR
# ---------------------------------------------------------------------------

def run_par(cast_lib, resid_np, anchors, *, accumulate=False, gate_mode=0, x0=None, tile=8,
            debug=False):
    dev = "cuda"
    resid = torch.from_numpy(resid_np.astype(np.float32)).to(dev)
    prm = cast_lib.cast_par_params_default(accumulate=int(accumulate), gate_mode=gate_mode,
                                           tile_h=tile, tile_w=tile)
    if x0 is None:
        out = torch.full_like(resid, -7.25)            # sentinel: anchor slots must keep it
    else:
        out = torch.from_numpy(x0.astype(np.float32)).to(dev)
    before = out.clone()
    th = gt = cf = None
    if debug:
        s1, s2 = cast_lib.par_debug_shapes(len(anchors), resid.shape[1], resid.shape[2], prm)
        th = torch.full(s1, 99.0, device=dev)
        gt = torch.full(s1, 99.0, device=dev)
        cf = torch.full(s2, 99.0, device=dev)
    cast_lib.cast_par_reconstruct(resid, anchors, prm, out=out, theta_out=th, gate_out=gt,
                                  conf_out=cf)
    torch.cuda.synchronize()
    return out, before, prm, (th, gt, cf)


def check_par(cast_lib, resid_np, anchors, *, accumulate=False, gate_mode=0, x0=None, tile=8,
              targets=None, label="", debug=False):
    n = resid_np.shape[0]
    out, before, prm, dbg = run_par(cast_lib, resid_np, anchors, accumulate=accumulate,
                                    gate_mode=gate_mode, x0=x0, tile=tile, debug=debug)
    oprm = OP.ParParams(tile_h=tile, tile_w=tile, gate_mode=gate_mode, accumulate=accumulate)
    ref = OP.par_reconstruct(resid_np.astype(np.float64), anchors, oprm,
                             out=None if x0 is None else x0.astype(np.float64), targets=targets)
    got = out.cpu().numpy().astype(np.float64)
    skipped = [t for t in range(n) if t not in set(anchors)]
    check_t = skipped if targets is None else [t for t in skipped if t in targets]
    rr = rel_rms(got[check_t], ref[check_t])
    log(f"[par {label}] rel-RMS {rr:.3e} over {len(check_t)} frames")
    assert rr <= PAR_REL_RMS, (label, rr)
    for a in anchors:
        assert torch.equal(out[a], before[a]), f"anchor slot {a} was written"
    if debug:
        th, gt, cf = (t.cpu().numpy().astype(np.float64) for t in dbg)
        th_o, g_o, c_o = OP.stats_arrays(resid_np.astype(np.float64), anchors, oprm)
        assert np.abs(cf - c_o).max() <= 1e-4, np.abs(cf - c_o).max()
        assert np.abs(gt - g_o).max() <= 1e-3, np.abs(gt - g_o).max()
        dth = np.abs(th - th_o)
        dth = np.minimum(dth, 2 * np.pi - dth)
        assert dth.max() <= 1e-3, dth.max()
    return out


def test_par_workspace_reuse_and_long_target_runs(cast_lib):
    """One workspace serves consecutive PAR calls of different shapes (the fused
    8x8 launches with edge classes, a 4x4 tiling launched per class, several pairs,
    long runs of targets between and beyond the anchors, a pair with no interior
    frame).  Each call matches a call on a fresh workspace bit for bit and the
    oracle within the PAR bar."""
    dev = "cuda"
    rng = np.random.default_rng(77)
    cases = [  # n_frames, Hg, Wg, D, anchors, tile, accumulate
        (45, 13, 19, 64, (2, 40), 8, False),
        (9, 16, 16, 96, (0, 3, 8), 4, True),
        (40, 9, 10, 40, (5, 6, 30), 8, True),
        (45, 13, 19, 64, (2, 40), 8, False),
    ]
    nb = 0
    for (n, hg, wg, d, anc, tile, acc) in cases:
        prm = cast_lib.cast_par_params_default(tile_h=tile, tile_w=tile)
        nb = max(nb, cast_lib.cast_par_workspace_bytes(n, len(anc), hg, wg, d, prm))
    ws = torch.full((nb,), 0x7f, dtype=torch.uint8, device=dev)
    for j, (n, hg, wg, d, anc, tile, acc) in enumerate(cases):
        base = rng.standard_normal((hg, wg, d))
        resid_np = np.zeros((n, hg, wg, d))
        for m, f in enumerate(anc):
            resid_np[f] = np.roll(base, (m, 2 * m), axis=(0, 1)) + 0.2 * rng.standard_normal(base.shape)
        x0 = rng.standard_normal(resid_np.shape)
        resid = torch.from_numpy(resid_np.astype(np.float32)).to(dev)
        prm = cast_lib.cast_par_params_default(accumulate=int(acc), tile_h=tile, tile_w=tile)
        outs = []
        for use_ws in (True, False):
            out = torch.from_numpy(x0.astype(np.float32)).to(dev)
            cast_lib.cast_par_reconstruct(resid, anc, prm, out=out, workspace=ws if use_ws else None)
            torch.cuda.synchronize()
            outs.append(out)
        assert torch.equal(outs[0], outs[1]), j
        oprm = OP.ParParams(tile_h=tile, tile_w=tile, accumulate=acc)
        ref = OP.par_reconstruct(resid_np.astype(np.float32).astype(np.float64), anc, oprm,
                                 out=x0.astype(np.float32).astype(np.float64))
        sk = [t for t in range(n) if t not in set(anc)]
        rr = rel_rms(outs[0].cpu().numpy().astype(np.float64)[sk], ref[sk])
        log(f"[par reuse {j}] rel-RMS {rr:.3e} over {len(sk)} frames")
        assert rr <= PAR_REL_RMS, (j, rr)


def test_par_gate_inline_and_launched(cast_lib):
    """Reconstruction grids that the chip holds in one round take the gate inside
    the reconstruction blocks; asking for a debug output (conf_out here) takes the
    gate launch instead.  Both must meet the PAR bar and agree with each other to
    fp32 rounding (their channel sums run in different orders), in write and
    accumulate mode, with one and with several anchor pairs."""
    dev = "cuda"
    rng = np.random.default_rng(21)
    for (n, Hg, Wg, D, anchors) in [(8, 30, 52, 192, (0, 3, 7)), (6, 13, 11, 70, (1, 4)),
                                    (9, 16, 16, 64, (0, 2, 5, 8))]:
        base = rng.standard_normal((Hg, Wg, D))
        resid = np.zeros((n, Hg, Wg, D))
        for j, a in enumerate(anchors):
            resid[a] = np.roll(base, (j, -j), axis=(0, 1)) + 0.3 * rng.standard_normal((Hg, Wg, D))
        r = torch.from_numpy(resid.astype(np.float32)).to(dev)
        for acc in (False, True):
            x0 = rng.standard_normal(resid.shape)
            prm = cast_lib.cast_par_params_default(accumulate=int(acc))
            _, s2 = cast_lib.par_debug_shapes(len(anchors), Hg, Wg, prm)
            outs = []
            for launched in (False, True):
                out = torch.from_numpy(x0.astype(np.float32)).to(dev)
                conf = torch.zeros(s2, device=dev) if launched else None
                cast_lib.cast_par_reconstruct(r, anchors, prm, out=out, conf_out=conf)
                torch.cuda.synchronize()
                outs.append(out.cpu().numpy().astype(np.float64))
            ref = OP.par_reconstruct(resid.astype(np.float32).astype(np.float64), anchors,
                                     OP.ParParams(accumulate=acc),
                                     out=x0.astype(np.float32).astype(np.float64) if acc else None)
            sk = [t for t in range(n) if t not in set(anchors)]
            base_t = x0[sk] if acc else 0.0
            for o in outs:
                assert rel_rms(o[sk], ref[sk]) <= PAR_REL_RMS
            d = rel_rms(outs[0][sk] - base_t, outs[1][sk] - base_t)
            log(f"[par gate inline vs launched {Hg}x{Wg}x{D} acc {acc}] rel-RMS {d:.2e}")
            assert d <= 1e-5, d


def test_par_tiny_all_modes(cast_lib):
    w = gen.get(W.TINY)
    resid, x0, _ = gen.par_inputs(w, seed=42)
    for gm in (0, 1, 2):
        check_par(cast_lib, resid, w.anchors, gate_mode=gm, label=f"tiny gate{gm}", debug=True)
    check_par(cast_lib, resid, w.anchors, accumulate=True, x0=x0, label="tiny acc")


def test_par_edge_tiles_and_ragged_channels(cast_lib):
    """Grids whose edges leave 6-, 5-, 3- and 1-wide tiles, channel counts that are not a
    multiple of the 64-lane block, boundary extrapolation on both sides, K_f = 2."""
    rng = np.random.default_rng(1)
    for (n, Hg, Wg, D, anchors) in [(7, 14, 13, 80, (2, 5)), (6, 17, 9, 33, (0, 2, 5)),
                                    (5, 30, 52, 64, (1, 3))]:
        base = rng.standard_normal((Hg, Wg, D))
        resid = np.zeros((n, Hg, Wg, D))
        for j, a in enumerate(anchors):
            resid[a] = np.roll(base, (j, 2 * j), axis=(0, 1)) + 0.3 * rng.standard_normal((Hg, Wg, D))
        check_par(cast_lib, resid, anchors, label=f"edges {Hg}x{Wg}x{D}", debug=True)
        x0 = rng.standard_normal(resid.shape)
        check_par(cast_lib, resid, anchors, accumulate=True, x0=x0, label=f"edges acc {Hg}x{Wg}")


def test_par_small_tiles(cast_lib):
    """Tile parameter other than 8 (4x4 tiles, remainder 3)."""
    rng = np.random.default_rng(2)
    base = rng.standard_normal((11, 11, 16))
    resid = np.stack([base, np.roll(base, (1, 0), axis=(0, 1)), np.zeros_like(base),
                      np.roll(base, (2, 1), axis=(0, 1))])
    check_par(cast_lib, resid, (0, 1, 3), tile=4, label="tile4", debug=True)


def test_par_matrix_like(cast_lib):
    w = gen.get(W.MATRIX)
    resid, _, _ = gen.par_inputs(w, seed=42)
    check_par(cast_lib, resid, w.anchors, label="matrix write", debug=True)


def test_par_reliability_threshold(cast_lib):
    """App. A.2's reliability rule and eq:confidence's no-reliable-bin case on the
    GPU: a designed tile whose bins straddle eta (one at 3x, one at 0.75x, one at
    0.3x, one where two channels in different 64-channel blocks cancel in Z), the
    same tile at 1e-3 amplitude (the absolute part of eta decides), a tile that is
    zero in both anchors, one zero in one anchor, band-limited anchors (Nyquist
    bins zero) and a plain shifted pair.  theta, g and c_p are compared with the
    oracle on every bin, and the designed bins with their hand-derived values."""
    resid = W.reliability_frames(D=70, seed=5)
    anchors = (0, 2)
    for (_, _, _, st) in OP.par_stats(resid.astype(np.float32).astype(np.float64), anchors)[anchors]:
        moved = st.reliable & (st.theta != 0)     # fp32 must not flip a bin across the cut
        assert not moved.any() or math.pi - np.abs(st.theta[moved]).max() > 1e-3
    for gm in (0, 1, 2):
        check_par(cast_lib, resid, anchors, gate_mode=gm, label=f"reliability gate{gm}", debug=True)
    x0 = np.random.default_rng(8).standard_normal(resid.shape)
    check_par(cast_lib, resid, anchors, accumulate=True, x0=x0, label="reliability acc")
    _, _, prm, (th, gt, cf) = run_par(cast_lib, resid, anchors, debug=True)
    th = th.cpu().numpy()[0]
    gt = gt.cpu().numpy()[0]
    cf = cf.cpu().numpy()[0]
    nb = 5                                           # stored columns of an 8-wide tile
    pi = math.pi
    want = {(1, 1): pi / 6, (2, 1): -pi / 4, (2, 0): pi / 5, (6, 0): -pi / 5}
    for ky in range(8):
        for kx in range(nb):
            w_ = want.get((ky, kx), 0.0)
            assert abs(th[0, ky * nb + kx] - w_) <= 1e-4, ("designed tile", ky, kx, th[0, ky * nb + kx])
            w_ = pi / 6 if (ky, kx) == (1, 1) else 0.0
            assert abs(th[4, ky * nb + kx] - w_) <= 1e-4, ("designed tile 1e-3", ky, kx)
    assert abs(cf[0] - (2 * math.sqrt(3) + 0.25 + 4.8e-5) / (4.25 + 4.8e-5 + 1e-8)) <= 1e-5
    assert abs(cf[4] - (2 * math.sqrt(3) + 0.25) * 1e-6 / (4.25e-6 + 1e-8)) <= 1e-4
    # zero in both anchors / in one anchor: no reliable bin, c_p = 0, U = 1, and the
    # gate is sigma(-tau(nu) / T)
    for tile in (1, 2):
        assert cf[tile] == 0.0 and np.all(th[tile] == 0.0), tile
    _, _, _, nu = OP.bin_tables(8, 8)
    g0 = 1.0 / (1.0 + np.exp((0.25 + 0.5 * nu ** 2) / 0.1))
    assert np.abs(gt[1].reshape(8, nb) - g0).max() <= 1e-5
    # band-limited anchors: the Nyquist row and column carry no transport
    t3 = th[3].reshape(8, nb)
    assert np.all(t3[4, :] == 0.0) and np.all(t3[:, 4] == 0.0)


def test_par_deterministic(cast_lib):
    w = gen.get(W.MATRIX)
    resid, _, _ = gen.par_inputs(w, seed=1)
    a, _, _, _ = run_par(cast_lib, resid, w.anchors)
    b, _, _, _ = run_par(cast_lib, resid, w.anchors)
    assert torch.equal(a, b)
