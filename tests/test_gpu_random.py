"""Seeded random shapes through every kernel family and schedule against the fp64
oracle: batch, GQA group, head dim, block width, read depths, ragged prefix
lengths (empty, page boundaries, ragged tails) and explicit split sizes."""

from __future__ import annotations

import numpy as np
import pytest
import torch

from gpu_common import assert_close, assert_lse_close, oracle_call, wrap
from paper_2609_34538_amd import _lib as das
from paper_2609_34538_amd import datagen as dg

pytestmark = pytest.mark.gpu
DEV = "cuda"


def _case(seed):
    rng = np.random.default_rng(seed)
    dh = int(rng.choice([64, 96, 128]))
    hkv = int(rng.integers(1, 5))
    group = int(rng.choice([1, 2, 4, 8]))
    batch = int(rng.integers(1, 6))
    w = int(rng.choice([1, 3, 8, 16, 17, 31, 32, 33, 48, 64]))
    R = int(rng.integers(2, 7))
    lens = [int(rng.choice([0, 1, 63, 64, 65, 127, 128, 129, int(rng.integers(0, 700))]))
            for _ in range(batch)]
    pps = int(rng.choice([0, 1, 2, 3, 5, 64]))
    wl = dg.scaled(dg.WORKLOADS[3], batch=batch, hq=hkv * group, hkv=hkv, dh=dh, depth_R=R,
                   layers=2, prefix=(0, 700), draft_depths=(1,), draft_widths=(w,),
                   verify_width=w, paged_random=True, residency="full", k_gain=None)
    return wl, lens, pps, rng


@pytest.mark.parametrize("seed", range(128))
def test_random_shapes(seed):
    wl, lens, pps, rng = _case(seed)
    torch.manual_seed(seed)
    cd = dg.make_cache(wl, DEV, prefix_lens=lens)
    cache, batch = wrap(cd)
    R = wl.depth_R
    kappa, nu = int(rng.integers(1, R + 1)), int(rng.integers(1, R + 1))
    w = wl.draft_widths[0]
    q, kb, vb = dg.block_inputs(cd, w, kappa, DEV)
    ref, ref_lse = oracle_call(cd, 1, kappa, nu, q, kb, vb, range(wl.batch))
    paths = ["valu", "mfma"]
    if wl.batch <= 64 and w * wl.group <= (16 if wl.dh == 128 else 32):
        paths.append("balanced")
    for path in paths:
        lse = torch.empty((wl.batch, wl.hq, w), dtype=torch.float32, device=DEV)
        out = das.attn_policy(cache, batch, 1, kappa, nu, q, kb, vb, lse=lse, path=path,
                              pages_per_split=pps)
        torch.cuda.synchronize()
        what = (f"seed {seed} {path}: B={wl.batch} Hkv={wl.hkv} G={wl.group} dh={wl.dh} "
                f"w={w} lens={lens} pps={pps} ({kappa},{nu})")
        assert_close(out, ref, wl.dtype, what)
        assert_lse_close(lse, ref_lse, what)


@pytest.mark.parametrize("seed", range(1000, 1128))
def test_random_shapes_fp32(seed):
    """fp32 caches (vector-ALU kernel only) at every head dim and block width,
    so every row-tile size of that kernel (4, 8, 16, 32 rows) is met."""
    wl, lens, pps, rng = _case(seed)
    wl = dg.scaled(wl, dtype=torch.float32)
    torch.manual_seed(seed)
    cd = dg.make_cache(wl, DEV, prefix_lens=lens)
    cache, batch = wrap(cd)
    R = wl.depth_R
    kappa, nu = int(rng.integers(1, R + 1)), int(rng.integers(1, R + 1))
    w = wl.draft_widths[0]
    q, kb, vb = dg.block_inputs(cd, w, kappa, DEV)
    ref, ref_lse = oracle_call(cd, 1, kappa, nu, q, kb, vb, range(wl.batch))
    lse = torch.empty((wl.batch, wl.hq, w), dtype=torch.float32, device=DEV)
    out = das.attn_policy(cache, batch, 1, kappa, nu, q, kb, vb, lse=lse, pages_per_split=pps)
    torch.cuda.synchronize()
    what = (f"seed {seed} fp32: B={wl.batch} Hkv={wl.hkv} G={wl.group} dh={wl.dh} "
            f"w={w} lens={lens} pps={pps} ({kappa},{nu})")
    assert_close(out, ref, wl.dtype, what)
    assert_lse_close(lse, ref_lse, what)
