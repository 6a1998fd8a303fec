"""The C ABI used from C: paper_2609_34144_amd/cast_client (built by
__graft_entry__.build() from csrc/cast_client.cpp, linked against libcast.so, no
Python or torch inside) runs one block step -- cast_route_kv, cast_anchor_attn
with its key-split workspace, cast_par_reconstruct in accumulate mode -- on inputs
written to files, in a child process.  Its outputs must equal the Python
binding's on the same inputs bit for bit (same kernels, same launch plans)."""
import os
import subprocess

import numpy as np
import pytest
import torch

import gen
from gen import workloads as W

pytestmark = pytest.mark.gpu

CLIENT = os.path.join(os.path.dirname(os.path.dirname(os.path.abspath(__file__))),
                      "paper_2609_34144_amd", "cast_client")


def bf16_bits(t):
    return t.contiguous().view(torch.int16).cpu().numpy()


def run_client(tmp, q, k, v, resid, x0, anchors, topk, scale):
    n_a, S, H, dh = q.shape
    M, Bv = k.shape[:2]
    n_frames, Hg, Wg, D = resid.shape
    with open(os.path.join(tmp, "meta.txt"), "w") as f:
        f.write(f"{n_a} {S} {H} {dh} {M} {Bv} {topk} {scale!r} {n_frames} {Hg} {Wg} {D} "
                f"{len(anchors)} " + " ".join(str(a) for a in anchors) + "\n")
    for name, t in (("q", q), ("k", k), ("v", v)):
        bf16_bits(t).tofile(os.path.join(tmp, name + ".bin"))
    resid.cpu().numpy().astype(np.float32).tofile(os.path.join(tmp, "resid.bin"))
    x0.cpu().numpy().astype(np.float32).tofile(os.path.join(tmp, "x.bin"))
    print(f"[c client] n_a {n_a} S {S} H {H} dh {dh} M {M} Bv {Bv} topk {topk}; "
          f"PAR {n_frames}x{Hg}x{Wg}x{D} anchors {anchors}", flush=True)
    r = subprocess.run([CLIENT, tmp], capture_output=True, text=True, timeout=120)
    print(r.stdout.strip(), r.stderr.strip(), flush=True)
    assert r.returncode == 0, r.stderr
    k_eff = min(topk, M)
    idx = np.fromfile(os.path.join(tmp, "idx.bin"), dtype=np.int32).reshape(n_a, H, k_eff)
    scores = np.fromfile(os.path.join(tmp, "scores.bin"), dtype=np.float32).reshape(n_a, H, M)
    out = np.fromfile(os.path.join(tmp, "out.bin"), dtype=np.int16).reshape(n_a, S, H, dh)
    x = np.fromfile(os.path.join(tmp, "x_out.bin"), dtype=np.float32).reshape(resid.shape)
    return idx, scores, out, x


@pytest.mark.parametrize("case", ["tiny", "matrix_like_d256"])
def test_c_client_matches_binding(cast_lib, case, tmp_path):
    assert os.path.exists(CLIENT), "cast_client is missing: run __graft_entry__.build()"
    dev = "cuda"
    if case == "tiny":
        w = gen.get(W.TINY)
        q, k, v, _, _ = gen.attn_inputs(w, seed=42, device=dev)
        resid_np, x0_np, _ = gen.par_inputs(w, seed=42)
        topk, scale, anchors = w.topk, w.scale, w.anchors
    else:
        w = gen.get(W.MATRIX)
        torch.manual_seed(8)
        # Matrix-like routing and PAR shapes with fewer heads and channels
        q = torch.randn(3, w.S, 2, 128, device=dev).to(torch.bfloat16)
        k = torch.randn(w.M, w.Bv, 2, 128, device=dev).to(torch.bfloat16)
        v = torch.randn(w.M, w.Bv, 2, 128, device=dev).to(torch.bfloat16)
        resid_np, x0_np, _ = gen.par_inputs(w, seed=42, D=256)
        topk, scale, anchors = w.topk, w.scale, w.anchors
    resid = torch.from_numpy(resid_np.astype(np.float32)).to(dev)
    x0 = torch.from_numpy(x0_np.astype(np.float32)).to(dev)
    c_idx, c_scores, c_out, c_x = run_client(str(tmp_path), q, k, v, resid, x0, anchors, topk, scale)

    idx, k_eff, scores = cast_lib.cast_route_kv(q, k, topk, scale, want_scores=True)
    out, _ = cast_lib.cast_anchor_attn(q, k, v, idx, k_eff, scale)
    x = x0.clone()
    cast_lib.cast_par_reconstruct(resid, anchors, cast_lib.cast_par_params_default(accumulate=1), out=x)
    torch.cuda.synchronize()
    assert np.array_equal(c_idx, idx.cpu().numpy())
    assert np.array_equal(c_scores.view(np.int32), scores.cpu().numpy().view(np.int32))
    assert np.array_equal(c_out, bf16_bits(out))
    assert np.array_equal(c_x.view(np.int32), x.cpu().numpy().view(np.int32))
    print(f"[c client {case}] idx, scores, attention output and PAR update bit-identical "
          f"to the binding", flush=True)
