"""Logits that grow along the prefix, on the split grid's shared-ring
workgroups (GQA blocks of 33-64 and of more than 64 query rows): a gradual
ramp moves each row's running maximum a little on many tiles, a step moves
it far once (l and O rescaled mid-split, then a near one-hot softmax whose
outputs reach ~5, where bf16's own rounding is ~0.016 of the 0.02 bound).
Both against the fp64 oracle, with lse."""

from __future__ import annotations

import numpy as np
import pytest
import torch

from gpu_common import assert_close, assert_lse_close, oracle_call, wrap
from paper_2609_34538_amd import _lib as das
from paper_2609_34538_amd import datagen as dg

pytestmark = pytest.mark.gpu
DEV = "cuda"


def _key_gain(kind: str, n_pages: int) -> np.ndarray:
    i = np.arange(n_pages, dtype=np.float64)
    if kind == "ramp":  # logits' spread grows by ~1.7x over the prefix
        return 1.0 + 0.7 * i / max(n_pages - 1, 1)
    if kind == "step":  # logits 12x larger in the second half
        return np.where(i < n_pages // 2, 1.0, 12.0)
    return np.ones(n_pages)


@pytest.mark.parametrize("w", [16, 32])
@pytest.mark.parametrize("kind,pps", [("ramp", 0), ("step", 0), ("step", 4), ("none", 4)])
def test_growing_logits_on_shared_ring(kind, pps, w):
    lens = [3000, 1100, 64]
    wl = dg.scaled(dg.WORKLOADS[4], batch=len(lens), hq=8, hkv=2, dh=128, layers=1,
                   prefix=(0, max(lens)), draft_depths=(2,), draft_widths=(w,), verify_width=w,
                   paged_random=True, k_gain=None)
    torch.manual_seed(5)
    cd = dg.make_cache(wl, DEV, prefix_lens=lens)
    # scale every sequence's keys by logical page, through its block table
    k2 = cd.k_plane[2]
    for b, s_len in enumerate(lens):
        n_pages = -(-s_len // dg.PAGE)
        gain = _key_gain(kind, n_pages)
        for i in range(n_pages):
            pg = int(cd.block_table[b, i])
            cd.k_pool[k2, 0, :, pg] = (cd.k_pool[k2, 0, :, pg].float() * gain[i]).to(wl.dtype)
    cache, batch = wrap(cd)
    q, kb, vb = dg.block_inputs(cd, w, 2, DEV)
    lse = torch.empty((wl.batch, wl.hq, w), dtype=torch.float32, device=DEV)
    out = das.attn_policy(cache, batch, 0, 2, wl.depth_R, q, kb, vb, lse=lse, path="mfma",
                          pages_per_split=pps)
    torch.cuda.synchronize()
    ref, ref_lse = oracle_call(cd, 0, 2, wl.depth_R, q, kb, vb, range(wl.batch))
    assert_close(out, ref, wl.dtype, f"{kind} pps={pps} w={w}")
    assert_lse_close(lse, ref_lse, f"{kind} pps={pps} w={w} lse")
