"""GPU parity of the HIP path against the fp64 oracle, through the C ABI.

Small shapes (several pages, ragged tails, empty prefixes, GQA, every head
dim) are compared element by element on every output; the full-size
workloads in test_gpu_fullsize.py compare sampled sequences."""

from __future__ import annotations

import numpy as np
import pytest
import torch

from gpu_common import assert_close, assert_lse_close, oracle_call, wrap
from paper_2609_34538_amd import _lib as das
from paper_2609_34538_amd import datagen as dg

pytestmark = pytest.mark.gpu
DEV = "cuda"
W = dg.WORKLOADS


def small_workloads():
    return {
        "c1": W[1],
        "c2s": dg.scaled(W[2], hq=5, hkv=5, layers=2, prefix=(333, 333), residency="sparse"),
        "c3s": dg.scaled(W[3], batch=6, hq=4, hkv=4, layers=2, prefix=(0, 300)),
        "c4s": dg.scaled(W[4], batch=2, hq=8, hkv=2, layers=2, prefix=(700, 700)),
        "c5s": dg.scaled(W[5], batch=4, hq=3, hkv=3, layers=2, prefix=(100, 400)),
        "gqa8_dh64": dg.scaled(W[4], batch=2, hq=16, hkv=2, dh=64, layers=1, prefix=(130, 190),
                               draft_widths=(5,), verify_width=5, paged_random=True),
        # 32 x 8 = 256 query rows: two workgroups of 4 row tiles per split
        "gqa8_w32": dg.scaled(W[4], batch=2, hq=16, hkv=2, dh=128, layers=1, prefix=(100, 200),
                              draft_widths=(32,), verify_width=32, paged_random=True),
    }


EDGE_LENS = {"c3s": [0, 1, 63, 64, 65, 300]}


# kernel family (and schedule) of a parametrised case
KERNELS = {"valu": dict(path="valu"), "mfma": dict(path="mfma"),
           "balanced": dict(path="balanced")}


def balanced_ok(wl, widths=None, batch=None):
    """The balanced schedule takes up to 64 sequences and blocks of at most
    32 query rows (16 at head dim 128)."""
    widths = widths if widths is not None else list(wl.draft_widths) + [wl.verify_width]
    limit = 16 if wl.dh == 128 else 32
    return ((batch or wl.batch) <= 64 and max(widths) * wl.group <= limit
            and wl.dtype == torch.bfloat16)


def _paths(wl):
    if wl.dtype == torch.float32:
        return ["valu"]
    return ["valu", "mfma"] + (["balanced"] if balanced_ok(wl) else [])


def _cases():
    out = []
    for name, wl in small_workloads().items():
        for path in _paths(wl):
            out.append(pytest.param(name, path, id=f"{name}-{path}"))
    return out


@pytest.fixture(scope="module")
def small_data():
    data = {}
    for name, wl in small_workloads().items():
        torch.manual_seed(0)
        data[name] = dg.make_cache(wl, DEV, prefix_lens=EDGE_LENS.get(name))
    return data


@pytest.mark.parametrize("name,path", _cases())
def test_draft_and_verify_match_oracle(small_data, name, path):
    cd = small_data[name]
    wl = cd.wl
    cache, batch = wrap(cd)
    seqs = list(range(wl.batch))
    layer = wl.layers - 1
    for d, w in zip(wl.draft_depths, wl.draft_widths):
        q, kb, vb = dg.block_inputs(cd, w, d, DEV)
        lse = torch.empty((wl.batch, wl.hq, w), dtype=torch.float32, device=DEV)
        out = das.attn_policy(cache, batch, layer, d, wl.depth_R, q, kb, vb, lse=lse,
                              **KERNELS[path])
        torch.cuda.synchronize()
        ref, ref_lse = oracle_call(cd, layer, d, wl.depth_R, q, kb, vb, seqs)
        assert_close(out, ref, wl.dtype, f"{name} draft d={d} w={w} {path}")
        assert_lse_close(lse, ref_lse, f"{name} draft lse")
    q, kb, vb = dg.block_inputs(cd, wl.verify_width, wl.depth_R, DEV)
    out = das.attn_policy(cache, batch, 0, wl.depth_R, wl.depth_R, q, kb, vb, **KERNELS[path])
    torch.cuda.synchronize()
    ref, _ = oracle_call(cd, 0, wl.depth_R, wl.depth_R, q, kb, vb, seqs)
    assert_close(out, ref, wl.dtype, f"{name} verify {path}")


@pytest.mark.parametrize("path", list(KERNELS))
@pytest.mark.parametrize("pps", [1, 2, 3, 100])
def test_split_sizes_agree_with_oracle(small_data, path, pps):
    cd = small_data["c3s"]
    wl = cd.wl
    cache, batch = wrap(cd)
    q, kb, vb = dg.block_inputs(cd, 16, 2, DEV)
    lse = torch.empty((wl.batch, wl.hq, 16), dtype=torch.float32, device=DEV)
    out = das.attn_policy(cache, batch, 1, 2, wl.depth_R, q, kb, vb, lse=lse, pages_per_split=pps,
                          **KERNELS[path])
    torch.cuda.synchronize()
    ref, ref_lse = oracle_call(cd, 1, 2, wl.depth_R, q, kb, vb, range(wl.batch))
    # pps = 100: one split per sequence, outputs and lse written by the
    # attention kernel itself, no merge kernel
    assert_close(out, ref, wl.dtype, f"pps={pps} {path}")
    assert_lse_close(lse, ref_lse, f"pps={pps} {path} lse")


@pytest.mark.parametrize("path", list(KERNELS))
@pytest.mark.parametrize("w", [1, 2, 3, 7, 17, 32, 33, 64])
def test_block_widths(small_data, w, path):
    cd = small_data["c5s"]
    wl = cd.wl
    if path == "balanced" and not balanced_ok(wl, [w]):
        pytest.skip("blocks of more than 32 query rows take the split grid")
    cache, batch = wrap(cd)
    q, kb, vb = dg.block_inputs(cd, w, 3, DEV)
    out = das.attn_policy(cache, batch, 0, 3, wl.depth_R, q, kb, vb, **KERNELS[path])
    torch.cuda.synchronize()
    ref, _ = oracle_call(cd, 0, 3, wl.depth_R, q, kb, vb, range(wl.batch))
    assert_close(out, ref, wl.dtype, f"w={w} {path}")


def test_entry_points_are_policy_corners(small_data):
    """das_attn_draft_maturev is (d, R) and das_attn_verify is (r, r): same
    kernels, so the results agree bit for bit with the generic entry point;
    a draft at d = R is the verifier's read."""
    cd = small_data["c5s"]
    wl = cd.wl
    cache, batch = wrap(cd)
    q, kb, vb = dg.block_inputs(cd, 8, 2, DEV)
    a = das.attn_draft_maturev(cache, batch, 1, 2, q, kb, vb)
    b = das.attn_policy(cache, batch, 1, 2, wl.depth_R, q, kb, vb)
    q2, kb2, vb2 = dg.block_inputs(cd, 8, wl.depth_R, DEV)
    c = das.attn_verify(cache, batch, 1, wl.depth_R, q2, kb2, vb2)
    d = das.attn_policy(cache, batch, 1, wl.depth_R, wl.depth_R, q2, kb2, vb2)
    e = das.attn_draft_maturev(cache, batch, 1, wl.depth_R, q2, kb2, vb2)
    torch.cuda.synchronize()
    assert torch.equal(a.view(torch.int16), b.view(torch.int16))
    assert torch.equal(c.view(torch.int16), d.view(torch.int16))
    assert torch.equal(c.view(torch.int16), e.view(torch.int16))


@pytest.mark.parametrize("path", list(KERNELS))
def test_deterministic(small_data, path):
    cd = small_data["c4s" if path != "balanced" else "c5s"]
    wl = cd.wl
    cache, batch = wrap(cd)
    q, kb, vb = dg.block_inputs(cd, 32, 3, DEV)
    a = das.attn_policy(cache, batch, 0, 3, wl.depth_R, q, kb, vb, **KERNELS[path])
    b = das.attn_policy(cache, batch, 0, 3, wl.depth_R, q, kb, vb, **KERNELS[path])
    torch.cuda.synchronize()
    assert torch.equal(a.view(torch.int16), b.view(torch.int16)), path


def test_all_read_policies(small_data):
    """The generic entry point serves every read policy of Eq. (4):
    Aligned (d, d), Mature-V (d, R), Deep K (R, d), Deep K/V (R, R)."""
    cd = small_data["c1"]
    wl = cd.wl
    cache, batch = wrap(cd)
    R, d = wl.depth_R, wl.draft_depths[0]
    q, kb, vb = dg.block_inputs(cd, 4, d, DEV)
    for kappa, nu in ((d, d), (d, R), (R, d), (R, R), (2, 3)):
        out = das.attn_policy(cache, batch, 0, kappa, nu, q, kb, vb)
        torch.cuda.synchronize()
        ref, _ = oracle_call(cd, 0, kappa, nu, q, kb, vb, [0])
        assert_close(out, ref, wl.dtype, f"policy ({kappa},{nu})")


@pytest.mark.parametrize("pps", [0, 1, 3, 5, 63, 64, 100])
def test_long_prefix_split_sizes(pps):
    """Splits longer than 64 pages are clamped; a 5000-token prefix spans 79
    pages, so every clamp and the last partial split are exercised. 1, 3 and
    5 pages give 80, 27 and 16 splits: the merge's eager loads of 16 and 32
    splits and its serial tail past 32."""
    wl = dg.scaled(W[5], batch=3, hq=2, hkv=2, layers=1, prefix=(4000, 5000))
    cd = dg.make_cache(wl, DEV, prefix_lens=[5000, 4100, 64 * 64])
    cache, batch = wrap(cd)
    q, kb, vb = dg.block_inputs(cd, 16, 2, DEV)
    out = das.attn_policy(cache, batch, 0, 2, wl.depth_R, q, kb, vb, pages_per_split=pps)
    torch.cuda.synchronize()
    ref, _ = oracle_call(cd, 0, 2, wl.depth_R, q, kb, vb, range(wl.batch))
    assert_close(out, ref, wl.dtype, f"long prefix pps={pps}")


def _poison_past_prefix(cd: dg.CacheData):
    """Fill every cache slot past a sequence's prefix in its last page with
    NaN (keys) and Inf / NaN (values), in every plane and layer."""
    for b, s_len in enumerate(cd.prefix_lens):
        s_len = int(s_len)
        if s_len % dg.PAGE == 0:
            continue
        page = int(cd.block_table[b][s_len // dg.PAGE])
        for t in range(s_len % dg.PAGE, dg.PAGE):
            cd.k_pool[:, :, :, page, t, :] = float("nan")
            cd.v_pool[:, :, :, page, t // 8, :, t % 8] = float("inf") if t % 2 else float("nan")


@pytest.mark.parametrize("name,path", [("c3s", "valu"), ("c3s", "mfma"), ("c1", "valu"),
                                       ("gqa8_w32", "mfma"), ("c5s", "mfma"),
                                       ("c3s", "balanced"), ("c5s", "balanced")])
def test_non_finite_cache_past_the_prefix_is_ignored(name, path):
    """Positions past a sequence's prefix enter the softmax with probability
    0; whatever the cache holds there (here NaN and Inf) must contribute
    nothing, so the output still matches the oracle, which reads only the
    prefix."""
    wl = small_workloads()[name]
    torch.manual_seed(0)
    cd = dg.make_cache(wl, DEV, prefix_lens=EDGE_LENS.get(name))
    _poison_past_prefix(cd)
    cache, batch = wrap(cd)
    d, w = wl.draft_depths[-1], wl.draft_widths[-1]
    q, kb, vb = dg.block_inputs(cd, w, d, DEV)
    out = das.attn_policy(cache, batch, 0, d, wl.depth_R, q, kb, vb, **KERNELS[path])
    torch.cuda.synchronize()
    ref, _ = oracle_call(cd, 0, d, wl.depth_R, q, kb, vb, range(wl.batch))
    assert_close(out, ref, wl.dtype, f"{name} {path} with non-finite cache past the prefix")
