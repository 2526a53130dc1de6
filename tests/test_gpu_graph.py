"""Calls captured into a HIP graph and replayed give the same bytes as the
same calls launched eagerly: draft and verifier attention (split prefix or
balanced schedule, so a merge kernel runs too) and the commit. Every replay
is checked, with eager work and synchronisations between replays."""

from __future__ import annotations

import pytest
import torch

from gpu_common import assert_close, oracle_call, wrap
from paper_2609_34538_amd import _lib as das
from paper_2609_34538_amd import datagen as dg

pytestmark = pytest.mark.gpu
DEV = "cuda"


@pytest.mark.parametrize("path", ["valu", "mfma", "balanced"])
def test_graph_replay_matches_eager(path):
    pps = 0 if path == "balanced" else 2
    wl = dg.scaled(dg.WORKLOADS[5], batch=5, hq=6, hkv=3, layers=2, prefix=(0, 400))
    torch.manual_seed(0)
    cd = dg.make_cache(wl, DEV, prefix_lens=[0, 65, 200, 333, 400])
    cache, batch = wrap(cd)
    R = wl.depth_R
    qd, kbd, vbd = dg.block_inputs(cd, 8, 2, DEV)
    qv, _, _ = dg.block_inputs(cd, 16, R, DEV)
    k_new, v_new, num_new = dg.commit_inputs(cd, 16, DEV)
    num_new_t = torch.as_tensor(num_new, device=DEV)
    kp, vp = cd.k_plane[R], cd.v_plane[R]
    ws = das.alloc_workspace(cache, batch, wl.hq, 16, path=path, pages_per_split=pps)
    out_d = torch.empty_like(qd)
    out_v = torch.empty_like(qv)
    lse_d = torch.empty((wl.batch, wl.hq, 8), dtype=torch.float32, device=DEV)
    len_out = torch.empty(wl.batch, dtype=torch.int32, device=DEV)
    stream = torch.cuda.Stream()
    torch.cuda.synchronize()
    calls = [
        das.PreparedAttention(cache, batch, 1, 2, R, qd, kbd, vbd, out_d, ws, lse=lse_d,
                              path=path, pages_per_split=pps, stream=stream),
        das.PreparedAttention(cache, batch, 0, R, R, qv, k_new[kp, 0], v_new[vp, 0], out_v, ws,
                              path=path, pages_per_split=pps, stream=stream),
        das.PreparedAppend(cache, batch, k_new, v_new, num_new_t, len_out, stream=stream),
    ]
    k0, v0 = cd.k_pool.clone(), cd.v_pool.clone()
    for c in calls:
        c()
    torch.cuda.synchronize()
    ref = [t.clone() for t in (out_d, lse_d, out_v, len_out, cd.k_pool, cd.v_pool)]
    o_ref, _ = oracle_call(cd, 1, 2, R, qd, kbd, vbd, list(range(wl.batch)))
    assert_close(out_d, o_ref, wl.dtype, f"eager draft {path}")

    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g, stream=stream):
        for c in calls:
            c()
    torch.cuda.synchronize()
    for rep in range(4):
        for t in (out_d, lse_d, out_v, len_out):
            t.fill_(-7)
        cd.k_pool.copy_(k0)
        cd.v_pool.copy_(v0)
        # unrelated eager work between replays
        das.attn_policy(cache, batch, 1, R, R, qv, k_new[kp, 1], v_new[vp, 1], path=path)
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        got = (out_d, lse_d, out_v, len_out, cd.k_pool, cd.v_pool)
        for name, a, b in zip(("draft", "lse", "verify", "len_out", "k_pool", "v_pool"), got, ref):
            assert torch.equal(a, b), f"replay {rep}: {name} differs from the eager call"
