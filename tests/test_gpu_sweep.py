"""GPU parity on seeded random shapes: routing + routed attention and PAR against
the float64 oracle, to the bars of test_gpu_parity.py.

Each case draws its sizes from its own seed (the case id), so a failure names a
reproducible shape.  Attention cases cover the three copy modes (aligned chunks of
a multiple of 64 rows, fast chunks of >= 64 rows, and the general path with a
current segment or short chunks), head sizes 32/64/128, ragged query and key
tails, and the key split of a last partial round (long sequences, few units).
PAR cases cover the fused 8x8 tiling and the per-class tilings 4..7, two to four
anchors with and without frames before the first / after the last anchor
(eq:block extrapolation), write and accumulate modes and the three gate modes.
"""
import math
import os

import numpy as np
import pytest
import torch

from test_gpu_parity import check_attn, check_par, check_route

pytestmark = pytest.mark.gpu

# CAST_SWEEP_CASES widens the sweep (default 24 cases of each kind)
_N = int(os.environ.get("CAST_SWEEP_CASES", "24"))
ATTN_CASES = list(range(_N))
PAR_CASES = list(range(_N))


def attn_case(seed):
    rng = np.random.default_rng(1000 + seed)
    dh = int(rng.choice([32, 64, 128]))
    mode = seed % 3                       # 0 aligned, 1 fast, 2 general
    n_a = int(rng.integers(1, 3))
    H = int(rng.integers(1, 3))
    S = int(rng.integers(1, 420))
    if mode == 0:
        Bv = 64 * int(rng.integers(1, 4))
        n0 = 0
    elif mode == 1:
        Bv = int(rng.integers(65, 200))
        n0 = 0
    else:
        Bv = int(rng.integers(1, 90))
        n0 = int(rng.integers(0, 150))
    long_keys = seed % 4 == 2 or seed % 8 == 7    # long sequences, split and unsplit
    M = int(rng.integers(2, 40)) if not long_keys else int(rng.integers(40, 60))
    kmax = min(M, 12) if not long_keys else M
    k_eff = int(rng.integers(1 if n0 == 0 else 0, kmax + 1))
    if long_keys:
        k_eff = max(k_eff, min(M, -(-2100 // Bv)))    # L >= 2048: two or more pieces
    split = seed % 2 == 0
    return dict(dh=dh, n_a=n_a, H=H, S=S, M=M, Bv=Bv, n0=n0, k_eff=k_eff, split=split)


@pytest.mark.parametrize("seed", ATTN_CASES)
def test_route_attn_random_shapes(cast_lib, seed):
    c = attn_case(seed)
    label = "sweep " + " ".join(f"{k}={v}" for k, v in c.items())
    print(label, flush=True)
    torch.manual_seed(2000 + seed)
    dev = "cuda"
    dh, n_a, H, S, M, Bv, n0, k_eff = (c[k] for k in ("dh", "n_a", "H", "S", "M", "Bv", "n0", "k_eff"))
    q = torch.randn(n_a, S, H, dh, device=dev).to(torch.bfloat16)
    k = torch.randn(M, Bv, H, dh, device=dev).to(torch.bfloat16)
    v = torch.randn(M, Bv, H, dh, device=dev).to(torch.bfloat16)
    kc = torch.randn(n0, H, dh, device=dev).to(torch.bfloat16) if n0 else None
    vc = torch.randn(n0, H, dh, device=dev).to(torch.bfloat16) if n0 else None
    scale = 1.0 / math.sqrt(dh)
    if k_eff > 0:
        idx, got_k = check_route(cast_lib, q, k, k_eff, scale, label)
        assert got_k == k_eff
    else:
        idx = torch.zeros((n_a, H, 0), dtype=torch.int32, device=dev)
    check_attn(cast_lib, q, k, v, idx, k_eff, scale, kc=kc, vc=vc, label=label, split=c["split"])


def par_case(seed):
    rng = np.random.default_rng(3000 + seed)
    tile = 8 if seed % 3 != 2 else int(rng.integers(4, 8))
    n_frames = int(rng.integers(3, 11))
    n_anchor = int(rng.integers(2, min(4, n_frames) + 1))
    inner = sorted(rng.choice(np.arange(n_frames), n_anchor, replace=False).tolist())
    Hg = int(rng.integers(1, 34))
    Wg = int(rng.integers(1, 34))
    D = int(rng.integers(1, 150))
    accumulate = bool(seed % 2)
    gate_mode = int(seed % 3)
    return dict(tile=tile, n_frames=n_frames, anchors=inner, Hg=Hg, Wg=Wg, D=D,
                accumulate=accumulate, gate_mode=gate_mode)


@pytest.mark.parametrize("seed", PAR_CASES)
def test_par_random_shapes(cast_lib, seed):
    c = par_case(seed)
    label = "sweep " + " ".join(f"{k}={v}" for k, v in c.items())
    print(label, flush=True)
    rng = np.random.default_rng(4000 + seed)
    resid = rng.standard_normal((c["n_frames"], c["Hg"], c["Wg"], c["D"]))
    x0 = rng.standard_normal(resid.shape) if c["accumulate"] else None
    check_par(cast_lib, resid, c["anchors"], accumulate=c["accumulate"], gate_mode=c["gate_mode"],
              x0=x0, tile=c["tile"], label=label)
