"""Parity of the calls the DAS-Wave decoder makes beyond the benchmark
workloads' own rounds, against the fp64 oracle:

* every read policy of Eq. (4) on the matrix-core path (bf16, GQA);
* the DAS-Wave refinement schedule of Eq. (5) (widths W_j = min(32, 2 + j),
  j = 0..23) with Deep K/V prefix reads;
* the full-depth verifier at every recurrence depth r = 1..R (Aligned (r, r)
  reads of a fully resident cache)."""

from __future__ import annotations

import pytest
import torch

from gpu_common import assert_close, assert_lse_close, oracle_call, wrap
from paper_2609_34538_amd import _lib as das
from paper_2609_34538_amd import datagen as dg

pytestmark = pytest.mark.gpu
DEV = "cuda"


@pytest.fixture(scope="module")
def resident():
    # every depth stored, GQA 2, ragged prefixes across page boundaries
    wl = dg.scaled(dg.WORKLOADS[2], batch=3, hq=8, hkv=4, depth_R=8, layers=2,
                   prefix=(60, 300), draft_depths=(3,), draft_widths=(8,), verify_width=8,
                   paged_random=True)
    torch.manual_seed(0)
    return dg.make_cache(wl, DEV, prefix_lens=[0, 129, 300], spare_tokens=32)


@pytest.mark.parametrize("path", ["valu", "mfma"])
def test_every_read_policy(resident, path):
    cd = resident
    wl = cd.wl
    cache, batch = wrap(cd)
    R, d = wl.depth_R, 3
    q, kb, vb = dg.block_inputs(cd, 8, d, DEV)
    for kappa, nu in ((d, d), (d, R), (R, d), (R, R), (5, 2)):
        lse = torch.empty((wl.batch, wl.hq, 8), dtype=torch.float32, device=DEV)
        out = das.attn_policy(cache, batch, 1, kappa, nu, q, kb, vb, lse=lse, path=path)
        torch.cuda.synchronize()
        ref, ref_lse = oracle_call(cd, 1, kappa, nu, q, kb, vb, range(wl.batch))
        assert_close(out, ref, wl.dtype, f"policy ({kappa},{nu}) {path}")
        assert_lse_close(lse, ref_lse, f"policy ({kappa},{nu}) lse")


def test_das_wave_schedule(resident):
    cd = resident
    wl = cd.wl
    cache, batch = wrap(cd)
    R = wl.depth_R
    for j in range(24):
        w = min(32, 2 + j)
        q, kb, vb = dg.block_inputs(cd, w, R, DEV)
        out = das.attn_policy(cache, batch, j % wl.layers, R, R, q, kb, vb)
        torch.cuda.synchronize()
        ref, _ = oracle_call(cd, j % wl.layers, R, R, q, kb, vb, range(wl.batch))
        assert_close(out, ref, wl.dtype, f"wave round {j} (w={w})")


@pytest.mark.parametrize("path", ["valu", "mfma"])
def test_verifier_at_every_depth(resident, path):
    cd = resident
    wl = cd.wl
    cache, batch = wrap(cd)
    for r in range(1, wl.depth_R + 1):
        q, kb, vb = dg.block_inputs(cd, 8, r, DEV)
        out = das.attn_verify(cache, batch, 0, r, q, kb, vb) if path == "mfma" else \
            das.attn_policy(cache, batch, 0, r, r, q, kb, vb, path="valu")
        torch.cuda.synchronize()
        ref, _ = oracle_call(cd, 0, r, r, q, kb, vb, range(wl.batch))
        assert_close(out, ref, wl.dtype, f"verify depth {r} {path}")
