"""GPU parity at the full workload sizes, in the launch configuration bench.py
times, on outputs the oracle can compute one by one: every routing decision
(pooled means computed chunk by chunk), sampled attention query rows of sampled
(anchor, head) pairs, and sampled skipped frames of PAR (interior and
extrapolated).  Bars as in test_gpu_parity.py."""
import numpy as np
import pytest
import torch

import gen
from gen import workloads as W
from oracle import attn as OA
from oracle import par as OP
from oracle import route as OR
from test_gpu_parity import (ATTN_MAX_ABS, ATTN_REL_RMS, PAR_REL_RMS, log, np64, rel_rms)

pytestmark = pytest.mark.gpu


def oracle_scores_chunked(q, k, scale):
    """eq:pooled scores with the pooled means taken one chunk at a time (the
    oracle's pooled_means on slices), so no full float64 copy of K is needed."""
    qb, _ = OR.pooled_means(np64(q), np64(k[:1]))
    kb = np.concatenate([OR.pooled_means(np64(q[:, :1]), np64(k[m:m + 1]))[1]
                         for m in range(k.shape[0])], axis=0)
    return OR.scores_from_means(qb, kb, scale)


def check_idx(idx, s_or, k_eff, tol, label):
    g = idx.cpu().numpy()
    s32 = s_or.astype(np.float32)
    n_a, H, M = s_or.shape
    exact = near = 0
    for i in range(n_a):
        for h in range(H):
            got = [int(x) for x in g[i, h]]
            assert got == sorted(got) and len(set(got)) == k_eff
            order = sorted(range(M), key=lambda m: (-float(s32[i, h, m]), m))
            kth = float(s32[i, h, order[k_eff - 1]])
            nxt = float(s32[i, h, order[k_eff]]) if k_eff < M else -np.inf
            if kth - nxt > 2 * tol:
                assert got == OR.topk_select(s32[i, h], k_eff), (label, i, h)
                exact += 1
            else:
                near += 1
                sel = set(got)
                for m in range(M):
                    assert (s_or[i, h, m] >= kth - 2 * tol) if m in sel else \
                        (s_or[i, h, m] <= kth + 2 * tol)
    log(f"[route {label}] exact rows {exact}, near-tie rows {near}")


def route_and_check(cast_lib, q, k, topk, scale, s_or, label):
    idx, k_eff, scores = cast_lib.cast_route_kv(q, k, topk, scale, want_scores=True)
    torch.cuda.synchronize()
    assert k_eff == min(topk, k.shape[0])
    tol = 1e-4 * np.abs(s_or).max() + 1e-7
    d = np.abs(scores.cpu().numpy().astype(np.float64) - s_or).max()
    assert d <= tol, (label, d, tol)
    check_idx(idx, s_or, k_eff, tol, label)
    return idx, k_eff


def attn_sampled(cast_lib, w, q, k, v, idx, k_eff, pairs, n_rows, label, seed=0, extra_rows=()):
    out, lse = cast_lib.cast_anchor_attn(q, k, v, idx, k_eff, w.scale, want_lse=True)
    torch.cuda.synchronize()
    rng = np.random.default_rng(seed)
    idx_np = idx.cpu().numpy()
    got_all, ref_all = [], []
    for (i, h) in pairs:
        rows = sorted(set(int(s) for s in rng.choice(w.S, n_rows, replace=False)) | {0, w.S - 1}
                      | set(extra_rows))
        # host copies of just this pair's routed chunks (head h), then the oracle's gather
        sel = torch.as_tensor(idx_np[i, h], dtype=torch.long, device=k.device)
        k_sub = np64(k.index_select(0, sel)[:, :, h:h + 1, :])
        v_sub = np64(v.index_select(0, sel)[:, :, h:h + 1, :])
        K, V = OA.gather_kv(k_sub, v_sub, list(range(len(sel))), 0)
        Q = np64(q[i, rows, h, :])
        o, l = OA.softmax_attention(Q, K, V, w.scale)
        got_all.append(np64(out[i, rows, h, :]))
        ref_all.append(o)
        assert np.abs(lse[i, h, rows].cpu().numpy() - l).max() <= 1e-3 * max(1.0, np.abs(l).max())
    got, ref = np.concatenate(got_all), np.concatenate(ref_all)
    mx, rr = np.abs(got - ref).max(), rel_rms(got, ref)
    log(f"[attn {label}] {len(pairs)} pairs, max-abs {mx:.3e} rel-RMS {rr:.3e}")
    assert mx <= ATTN_MAX_ABS and rr <= ATTN_REL_RMS, (label, mx, rr)


def test_route_attn_hy_like(cast_lib):
    w = gen.get(W.HY)
    q, k, v, _, _ = gen.attn_inputs(w, seed=42, device="cuda")
    s_or = oracle_scores_chunked(q, k, w.scale)
    idx, k_eff = route_and_check(cast_lib, q, k, w.topk, w.scale, s_or, "hy")
    pairs = [(0, 0), (1, 7), (2, 13), (3, 23), (3, 5), (0, 19)]
    attn_sampled(cast_lib, w, q, k, v, idx, k_eff, pairs, 24, "hy sampled")


def test_attn_hy_like_every_pair(cast_lib):
    """Every (anchor, head) pair of the HY-like block (96 pairs), among them the
    pairs whose work units form the last, partial round and run as key pieces
    merged afterwards (the last 64 of 1344 units), a few rows each: the first and
    last query, rows at the borders of the last query tile (192 of 256 queries),
    and random rows."""
    w = gen.get(W.HY)
    q, k, v, _, _ = gen.attn_inputs(w, seed=42, device="cuda")
    idx, k_eff, _ = cast_lib.cast_route_kv(q, k, w.topk, w.scale)
    last = (w.S - 1) // 256 * 256
    pairs = [(i, h) for i in range(w.n_a) for h in range(w.H)]
    attn_sampled(cast_lib, w, q, k, v, idx, k_eff, pairs, 3, "hy every pair", seed=1,
                 extra_rows=(last, last + 31, last - 256, last - 1))


def test_route_attn_long_history(cast_lib):
    """All four budgets of the long-history workload share one input; the routing
    decisions are checked for every (anchor, head) at each budget, and attention
    on sampled rows of three (anchor, head) pairs at every budget, of every pair at
    the budget of 8 and of twelve pairs at 32."""
    w = gen.get("long_history_4f44x80_d3072_k32")
    q, k, v, _, _ = gen.attn_inputs(w, seed=42, device="cuda")
    s_or = oracle_scores_chunked(q, k, w.scale)
    for topk in (4, 8, 16, 32):
        idx, k_eff = route_and_check(cast_lib, q, k, topk, w.scale, s_or, f"long k{topk}")
        attn_sampled(cast_lib, w, q, k, v, idx, k_eff, [(0, 3), (2, 17), (3, 23)], 16,
                     f"long k{topk} sampled")
        if topk == 8:
            attn_sampled(cast_lib, w, q, k, v, idx, k_eff,
                         [(i, h) for i in range(w.n_a) for h in range(w.H)], 2,
                         "long k8 every pair", seed=2)
        if topk == 32:
            attn_sampled(cast_lib, w, q, k, v, idx, k_eff,
                         [(i, 2 * j + i % 2) for i in range(w.n_a) for j in range(0, 12, 4)], 4,
                         "long k32 twelve pairs", seed=3)


def par_sampled(cast_lib, w, targets, accumulate, label, debug=False):
    resid_np, _, _ = gen.par_inputs(w, seed=42)
    dev = "cuda"
    resid = torch.from_numpy(resid_np).to(dev)
    prm = cast_lib.cast_par_params_default(accumulate=int(accumulate))
    g = torch.Generator(device=dev)
    g.manual_seed(5)
    x0 = torch.randn(resid.shape, device=dev, generator=g) if accumulate else \
        torch.full_like(resid, -3.5)
    out = x0.clone()
    dbg = [None, None, None]
    if debug:
        s1, s2 = cast_lib.par_debug_shapes(w.n_a, w.Hg, w.Wg, prm)
        dbg = [torch.zeros(s1, device=dev), torch.zeros(s1, device=dev), torch.zeros(s2, device=dev)]
    cast_lib.cast_par_reconstruct(resid, w.anchors, prm, out=out, theta_out=dbg[0],
                                  gate_out=dbg[1], conf_out=dbg[2])
    torch.cuda.synchronize()
    ref = OP.par_reconstruct_targets(resid_np, w.anchors, targets)
    got = np.stack([out[t].cpu().numpy().astype(np.float64) -
                    (x0[t].cpu().numpy().astype(np.float64) if accumulate else 0.0)
                    for t in targets])
    want = np.stack([ref[t] for t in targets])
    rr = rel_rms(got, want)
    log(f"[par {label}] rel-RMS {rr:.3e} over frames {targets}")
    assert rr <= PAR_REL_RMS, (label, rr)
    for a in w.anchors:
        assert torch.equal(out[a], x0[a])
    if debug:
        _, _, c_o = OP.stats_arrays(resid_np, w.anchors)
        assert np.abs(dbg[2].cpu().numpy() - c_o).max() <= 1e-4


def test_par_hy_like(cast_lib):
    w = gen.get(W.HY)
    # interior frames of each pair and the right-extrapolated frames 13..15
    par_sampled(cast_lib, w, [1, 6, 9, 13, 15], True, "hy acc", debug=True)
    par_sampled(cast_lib, w, [2, 14], False, "hy write")


def test_par_stress(cast_lib):
    w = gen.get(W.PAR_STRESS)
    par_sampled(cast_lib, w, [1, 33, 64], True, "stress acc")
