"""Pins for the routing and attention oracles.

Routing (Sec. 4.4 eq:pooled, eq:topk): q_bar . k_bar equals the brute-force mean
of q . k over every token pair; permuting chunks permutes the selection; exact
ties go to the lower chunk index; topk >= M keeps every chunk (App. B.3 bypass).
Attention: with every chunk routed it equals dense attention over the whole
history, checked against torch's scaled_dot_product_attention in float64 (an
independent library); a chunk of identical keys yields the mean of its values.
"""
import math

import numpy as np
import pytest
import torch

from oracle import route as R
from oracle import attn as A


def rng(seed):
    return np.random.default_rng(seed)


def pin_pooled_bruteforce(mod=R):
    r = rng(1)
    q = r.standard_normal((2, 5, 3, 4))
    k = r.standard_normal((3, 6, 3, 4))
    s = mod.chunk_scores(q, k, scale=0.7)
    for i in range(2):
        for h in range(3):
            for m in range(3):
                acc = 0.0
                for a in range(5):
                    for b in range(6):
                        acc += float(np.dot(q[i, a, h], k[m, b, h]))
                assert abs(s[i, h, m] - 0.7 * acc / 30) < 1e-12


def pin_topk_rules(mod=R):
    assert mod.topk_select([0.1, 0.5, 0.5, 0.2], 2) == [1, 2]
    assert mod.topk_select([0.1, 0.5, 0.5, 0.2], 1) == [1]            # tie: lower index
    assert mod.topk_select([0.3, 0.3, 0.3, 0.3], 2) == [0, 1]
    assert mod.topk_select([3.0, -1.0, 2.0], 5) == [0, 1, 2]          # topk >= M: all
    assert mod.topk_select([-1.0, -3.0, -2.0, 0.0], 2) == [0, 3]      # ascending output
    assert mod.topk_select([], 3) == []


def pin_route_permutation(mod=R):
    r = rng(2)
    q = r.standard_normal((2, 7, 2, 8))
    k = r.standard_normal((9, 5, 2, 8))
    _, idx, _ = mod.route(q, k, 3)
    perm = r.permutation(9)
    _, idx_p, _ = mod.route(q, k[perm], 3)
    inv = np.argsort(perm)
    for i in range(2):
        for h in range(2):
            assert sorted(perm[idx_p[i, h]]) == sorted(idx[i, h]) or \
                sorted(inv[idx[i, h]]) == sorted(idx_p[i, h])


def pin_route_duplicate_tie(mod=R):
    r = rng(3)
    q = r.standard_normal((1, 4, 1, 8))
    k = r.standard_normal((6, 4, 1, 8))
    s = mod.chunk_scores(q, k)[0, 0]
    best = int(np.argmax(s))
    k2 = k.copy()
    k2[5] = k[best]
    _, idx, _ = mod.route(q, k2, 1)
    assert list(idx[0, 0]) == [min(best, 5)]
    k3 = k.copy()
    k3[0] = k[best]
    _, idx3, _ = mod.route(q, k3, 1)
    assert list(idx3[0, 0]) == [0]


def pin_route_selection(mod=R):
    """Every (anchor, head) keeps k_eff = min(topk, M) distinct chunks, listed in
    ascending order, and each kept chunk outscores each dropped one, with the
    scores summed by explicit loops over tokens and dims (eq:pooled, eq:topk)."""
    r = rng(9)
    n_a, S, H, dh, M, Bv = 3, 4, 3, 5, 7, 3
    q = r.standard_normal((n_a, S, H, dh))
    k = r.standard_normal((M, Bv, H, dh))
    for topk in (2, 7, 9):
        _, idx, k_eff = mod.route(q, k, topk)
        assert k_eff == min(topk, M) and idx.shape == (n_a, H, k_eff)
        for i in range(n_a):
            for h in range(H):
                b = [sum(float(q[i, a, h, d] * k[m, c, h, d])
                         for a in range(S) for c in range(Bv) for d in range(dh)) for m in range(M)]
                sel = [int(x) for x in idx[i, h]]
                assert sel == sorted(set(sel)) and len(sel) == k_eff
                for m in sel:
                    for n in set(range(M)) - set(sel):
                        assert b[m] > b[n] or (b[m] == b[n] and m < n), (i, h, m, n)


def _sdpa(q, k, v, scale):
    return torch.nn.functional.scaled_dot_product_attention(
        torch.from_numpy(q)[None, None], torch.from_numpy(k)[None, None],
        torch.from_numpy(v)[None, None], scale=scale)[0, 0].numpy()


def pin_attention_dense(mod=A):
    r = rng(4)
    n_a, S, H, dh, M, Bv = 2, 10, 3, 8, 4, 6
    q = r.standard_normal((n_a, S, H, dh))
    k = r.standard_normal((M, Bv, H, dh))
    v = r.standard_normal((M, Bv, H, dh))
    idx = np.tile(np.arange(M, dtype=np.int32), (n_a, H, 1))
    scale = 1 / math.sqrt(dh)
    O, L = mod.anchor_attention(q, k, v, idx, scale)
    for i in range(n_a):
        for h in range(H):
            K = k[:, :, h, :].reshape(M * Bv, dh)
            V = v[:, :, h, :].reshape(M * Bv, dh)
            np.testing.assert_allclose(O[i, :, h], _sdpa(q[i, :, h], K, V, scale), atol=1e-12)
            lse = torch.logsumexp(torch.from_numpy(scale * q[i, :, h] @ K.T), dim=1).numpy()
            np.testing.assert_allclose(L[i, h], lse, atol=1e-12)


def pin_attention_routed_subset(mod=A):
    """Routed attention equals dense attention restricted to the chosen chunks
    (plus the always-available current segment)."""
    r = rng(5)
    n_a, S, H, dh, M, Bv, n0 = 2, 7, 2, 4, 5, 3, 4
    q = r.standard_normal((n_a, S, H, dh))
    k = r.standard_normal((M, Bv, H, dh))
    v = r.standard_normal((M, Bv, H, dh))
    kc = r.standard_normal((n0, H, dh))
    vc = r.standard_normal((n0, H, dh))
    idx = np.array([[[0, 3], [1, 4]], [[2, 3], [0, 1]]], dtype=np.int32)
    O, _ = mod.anchor_attention(q, k, v, idx, 0.5, k_cur=kc, v_cur=vc)
    for i in range(n_a):
        for h in range(H):
            K = np.concatenate([kc[:, h]] + [k[c, :, h] for c in idx[i, h]])
            V = np.concatenate([vc[:, h]] + [v[c, :, h] for c in idx[i, h]])
            np.testing.assert_allclose(O[i, :, h], _sdpa(q[i, :, h], K, V, 0.5), atol=1e-12)


def pin_attention_constant_keys(mod=A):
    r = rng(6)
    q = r.standard_normal((1, 5, 1, 4))
    k = np.ones((2, 8, 1, 4)) * 0.3
    v = r.standard_normal((2, 8, 1, 4))
    idx = np.array([[[1]]], dtype=np.int32)
    O, _ = mod.anchor_attention(q, k, v, idx, 1.0)
    np.testing.assert_allclose(O[0, :, 0], np.broadcast_to(v[1, :, 0].mean(0), (5, 4)), atol=1e-12)


def pin_attention_rows(mod=A):
    """Sampled rows equal the same rows of the full computation."""
    r = rng(7)
    q = r.standard_normal((2, 9, 2, 4))
    k = r.standard_normal((3, 5, 2, 4))
    v = r.standard_normal((3, 5, 2, 4))
    idx = np.array([[[0, 2], [1, 2]], [[0, 1], [2, 0]]], dtype=np.int32)
    O, L = mod.anchor_attention(q, k, v, idx, 0.8)
    rows = [(0, 1, 3), (1, 0, 8), (1, 1, 0)]
    Os, Ls = mod.anchor_attention(q, k, v, idx, 0.8, rows=rows)
    for (i, h, s) in rows:
        np.testing.assert_allclose(Os[i, s, h], O[i, s, h], atol=1e-14)
        assert abs(Ls[i, h, s] - L[i, h, s]) < 1e-14


ROUTE_PINS = [pin_pooled_bruteforce, pin_topk_rules, pin_route_permutation, pin_route_duplicate_tie,
              pin_route_selection]
ATTN_PINS = [pin_attention_dense, pin_attention_routed_subset, pin_attention_constant_keys,
             pin_attention_rows]


@pytest.mark.parametrize("pin", ROUTE_PINS + ATTN_PINS,
                         ids=[p.__name__ for p in ROUTE_PINS + ATTN_PINS])
def test_pin(pin):
    pin()


def test_route_decide_fp32():
    """Selection on fp32-rounded scores: near-equal fp64 scores that round to the
    same fp32 value become an exact tie and go to the lower index."""
    s = np.array([1.0, 1.0 + 1e-12, 0.5])
    assert R.topk_select(s, 1) == [1]
    assert R.topk_select(s.astype(np.float32), 1) == [0]
