"""The allocation-free attention entry point (das_attn_policy_noalloc):
through the C ABI, two calls in a row (the second on a smaller input) give
exactly the outputs of das_attn_policy with its own workspace, and a request
whose workspace exceeds the fixed scratch is rejected."""

from __future__ import annotations

import numpy as np
import pytest
import torch

from gpu_common import wrap
from paper_2609_34538_amd import _lib as das
from paper_2609_34538_amd import datagen as dg

pytestmark = pytest.mark.gpu
DEV = "cuda"


def _inputs(wl, lens, w, d):
    cd = dg.make_cache(wl, DEV, prefix_lens=lens)
    cache, batch = wrap(cd)
    q, kb, vb = dg.block_inputs(cd, w, d, DEV)
    return cd, cache, batch, q, kb, vb


@pytest.mark.parametrize("dtype,path", [(torch.bfloat16, "mfma"), (torch.bfloat16, "valu"),
                                        (torch.bfloat16, "balanced"), (torch.float32, "valu")])
def test_noalloc_matches_policy_on_two_calls(dtype, path):
    big = dg.scaled(dg.WORKLOADS[5], dtype=dtype, batch=5, hq=8, hkv=4, layers=2,
                    prefix=(0, 0), draft_widths=(16,), verify_width=16)
    small = dg.scaled(big, batch=2, hq=4, hkv=2, layers=1)
    R = big.depth_R
    cases = [(big, [900, 0, 333, 64, 1201], 16, 3, 1),
             (small, [65, 130], 4, 1, 0)]
    prepared = [_inputs(wl, lens, w, d) + (d, layer) for wl, lens, w, d, layer in cases]
    outs, lses = [], []
    for cd, cache, batch, q, kb, vb, d, layer in prepared:  # two calls in a row
        out = torch.full_like(q, float("nan"))
        lse = torch.full((q.shape[0], q.shape[2], q.shape[1]), float("nan"),
                         dtype=torch.float32, device=DEV)
        das.attn_policy_noalloc(cache, batch, layer, d, R, q, kb, vb, out, lse=lse, path=path)
        outs.append(out)
        lses.append(lse)
    torch.cuda.synchronize()
    for (cd, cache, batch, q, kb, vb, d, layer), out, lse in zip(prepared, outs, lses):
        ref_lse = torch.empty_like(lse)
        ref = das.attn_policy(cache, batch, layer, d, R, q, kb, vb, lse=ref_lse, path=path)
        torch.cuda.synchronize()
        assert torch.equal(out.view(torch.int16 if dtype == torch.bfloat16 else torch.int32),
                           ref.view(torch.int16 if dtype == torch.bfloat16 else torch.int32))
        np.testing.assert_array_equal(lse.cpu().numpy(), ref_lse.cpu().numpy())


def test_noalloc_rejects_requests_beyond_the_scratch():
    # 32 sequences x 55 KV heads x 9 splits of 32-row piece records: > 64 MiB
    hkv, dh, w = 55, 96, 32
    k_pool = torch.zeros((1, 1, hkv, 1, 64, dh), dtype=torch.bfloat16, device=DEV)
    v_pool = torch.zeros((1, 1, hkv, 1, 8, dh, 8), dtype=torch.bfloat16, device=DEV)
    cache = das.PagedCache(k_pool, v_pool, 32, {32: 0}, {32: 0})
    batch = das.Batch(torch.zeros(32, dtype=torch.int32, device=DEV),
                      torch.zeros((32, 257), dtype=torch.int32, device=DEV))
    # on the split grid (the balanced schedule's pieces fit)
    assert das.workspace_bytes(cache, batch, hkv, w, path="mfma") > das.NOALLOC_SCRATCH_BYTES
    assert das.workspace_bytes(cache, batch, hkv, w) <= das.NOALLOC_SCRATCH_BYTES
    q = torch.zeros((32, w, hkv, dh), dtype=torch.bfloat16, device=DEV)
    kb = torch.zeros((32, w, hkv, dh), dtype=torch.bfloat16, device=DEV)
    out = torch.empty_like(q)
    with pytest.raises(das.DasError) as e:
        das.attn_policy_noalloc(cache, batch, 0, 32, 32, q, kb, kb, out, path="mfma")
    assert e.value.status == -5  # DAS_ERR_WORKSPACE
