"""The balanced persistent schedule (DAS_PATH_BALANCED): every resident wave
streams an equal share of all sequences' tiles, across unit boundaries.
Cases that stress its work split against the fp64 oracle: one long sequence
shared by many workers (many pieces per unit), many short sequences per
worker, empty prefixes, and the library's choice of it."""

from __future__ import annotations

import pytest
import torch

from gpu_common import assert_close, assert_lse_close, oracle_call, wrap
from paper_2609_34538_amd import _lib as das
from paper_2609_34538_amd import datagen as dg

pytestmark = pytest.mark.gpu
DEV = "cuda"


def _run(lens, hq, hkv, dh, w, d=2, path="balanced", seed=0):
    wl = dg.scaled(dg.WORKLOADS[3], batch=len(lens), hq=hq, hkv=hkv, dh=dh, layers=1,
                   prefix=(0, max(lens)), draft_depths=(d,), draft_widths=(w,), verify_width=w,
                   paged_random=True)
    torch.manual_seed(seed)
    cd = dg.make_cache(wl, DEV, prefix_lens=lens)
    cache, batch = wrap(cd)
    q, kb, vb = dg.block_inputs(cd, w, d, DEV)
    lse = torch.empty((wl.batch, wl.hq, w), dtype=torch.float32, device=DEV)
    out = das.attn_policy(cache, batch, 0, d, wl.depth_R, q, kb, vb, lse=lse, path=path)
    torch.cuda.synchronize()
    return wl, cd, (cache, batch, q, kb, vb), out, lse


@pytest.mark.parametrize("hkv,dh,w", [(1, 96, 32), (3, 128, 16), (2, 64, 7), (1, 64, 32)])
def test_long_sequence_among_short_ones(hkv, dh, w):
    # the 40000-token unit spans dozens of workers: more pieces than the
    # merge loads at once
    lens = [40000, 0, 1, 64, 65, 700]
    wl, cd, (_, _, q, kb, vb), out, lse = _run(lens, hkv, hkv, dh, w)
    ref, ref_lse = oracle_call(cd, 0, 2, wl.depth_R, q, kb, vb, range(wl.batch))
    assert_close(out, ref, wl.dtype, f"long among short hkv={hkv} dh={dh} w={w}")
    assert_lse_close(lse, ref_lse, "long among short lse")


@pytest.mark.parametrize("path,pps", [("balanced", 0), ("mfma", 4)])
@pytest.mark.parametrize("v_scale", [2.0 ** -100, 2.0 ** -20, 2.0 ** 17, 3.0e5, 2.0 ** 100])
def test_piece_scale_over_value_magnitudes(v_scale, path, pps):
    """Pieces (balanced schedule) and split records (split grid) keep O / l
    in fp16 under a per-row power-of-two scale: values far below fp16's
    normal range and far above its largest finite value merge as accurately
    as unit-scale ones (outputs compared after dividing by the value scale;
    lse does not depend on it)."""
    lens = [40000, 64, 700]
    wl = dg.scaled(dg.WORKLOADS[3], batch=len(lens), hq=2, hkv=2, dh=96, layers=1,
                   prefix=(0, max(lens)), draft_depths=(2,), draft_widths=(16,),
                   verify_width=16, paged_random=True)
    torch.manual_seed(3)
    cd = dg.make_cache(wl, DEV, prefix_lens=lens)
    cd.v_pool.mul_(v_scale)
    cache, batch = wrap(cd)
    q, kb, vb = dg.block_inputs(cd, 16, 2, DEV)
    vb = (vb.float() * v_scale).to(vb.dtype)
    lse = torch.empty((wl.batch, wl.hq, 16), dtype=torch.float32, device=DEV)
    out = das.attn_policy(cache, batch, 0, 2, wl.depth_R, q, kb, vb, lse=lse, path=path,
                          pages_per_split=pps)
    torch.cuda.synchronize()
    ref, ref_lse = oracle_call(cd, 0, 2, wl.depth_R, q, kb, vb, range(wl.batch))
    assert_close(out.double() / v_scale, ref / v_scale, wl.dtype,
                 f"{path} value scale {v_scale:g}")
    assert_lse_close(lse, ref_lse, f"value scale {v_scale:g} lse")


def test_many_short_sequences_per_worker():
    # 64 sequences of 0..300 tokens, 4 KV heads of GQA 2, block 16: several
    # units per worker
    lens = [(37 * i) % 301 for i in range(64)]
    wl, cd, (_, _, q, kb, vb), out, lse = _run(lens, 8, 4, 96, 16)
    ref, ref_lse = oracle_call(cd, 0, 2, wl.depth_R, q, kb, vb, range(wl.batch))
    assert_close(out, ref, wl.dtype, "many short sequences")
    assert_lse_close(lse, ref_lse, "many short sequences lse")


def test_all_prefixes_empty():
    lens = [0, 0, 0]
    wl, cd, (_, _, q, kb, vb), out, lse = _run(lens, 4, 4, 96, 5)
    ref, ref_lse = oracle_call(cd, 0, 2, wl.depth_R, q, kb, vb, range(wl.batch))
    assert_close(out, ref, wl.dtype, "empty prefixes")
    assert_lse_close(lse, ref_lse, "empty prefixes lse")


def test_library_choice_and_determinism():
    """The library takes the balanced schedule for a batch of 2..64 sequences
    with more than W / 8 (sequence, KV head) units (bit-identical to asking
    for it), the split grid for fewer units or when a split size is given;
    repeated calls agree bit for bit."""
    lens = [1500, 333, 4096, 0, 2047]
    # 5 x 40 = 200 units > 1280 / 8 at head dim 96
    wl, cd, (cache, batch, q, kb, vb), out, _ = _run(lens, 40, 40, 96, 16)
    auto = das.attn_policy(cache, batch, 0, 2, wl.depth_R, q, kb, vb)
    again = das.attn_policy(cache, batch, 0, 2, wl.depth_R, q, kb, vb, path="balanced")
    grid = das.attn_policy(cache, batch, 0, 2, wl.depth_R, q, kb, vb, pages_per_split=4)
    grid_ref = das.attn_policy(cache, batch, 0, 2, wl.depth_R, q, kb, vb, path="mfma",
                               pages_per_split=4)
    torch.cuda.synchronize()
    assert torch.equal(auto.view(torch.int16), out.view(torch.int16))
    assert torch.equal(again.view(torch.int16), out.view(torch.int16))
    assert torch.equal(grid.view(torch.int16), grid_ref.view(torch.int16))
    # 5 x 4 = 20 units: the split grid with the library's split size
    wl, cd, (cache, batch, q, kb, vb), bal, _ = _run(lens, 4, 4, 96, 16)
    auto = das.attn_policy(cache, batch, 0, 2, wl.depth_R, q, kb, vb)
    grid = das.attn_policy(cache, batch, 0, 2, wl.depth_R, q, kb, vb, path="mfma")
    torch.cuda.synchronize()
    assert torch.equal(auto.view(torch.int16), grid.view(torch.int16))
    ref, _ = oracle_call(cd, 0, 2, wl.depth_R, q, kb, vb, range(wl.batch))
    assert_close(auto, ref, wl.dtype, "library choice, few units")
    assert_close(bal, ref, wl.dtype, "balanced, few units")


def test_unsupported_shapes_are_refused():
    lens = [100, 200]
    wl, cd, (cache, batch, q, kb, vb), _, _ = _run(lens, 4, 4, 96, 16)
    q33, kb33, vb33 = dg.block_inputs(cd, 33, 2, DEV)
    ws = torch.empty(1 << 20, dtype=torch.uint8, device=DEV)
    with pytest.raises(das.DasError) as e:
        das.attn_policy(cache, batch, 0, 2, wl.depth_R, q33, kb33, vb33, path="balanced",
                        workspace=ws)
    assert e.value.status == -7  # DAS_ERR_UNSUPPORTED
