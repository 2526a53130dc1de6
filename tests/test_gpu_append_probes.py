"""Bit-exact GPU checks: the commit into the paged cache, and one-hot probes
that pin page-table resolution, key/value plane selection, core layer, GQA
head map, the prefix-length boundary and the in-block causal mask.

The probes write the cache directly with the layout documented in das.h
(physical page block_table[b][pos // 64], slot pos % 64; keys token-major
[slot][dh], values token-grouped [slot // 8][dh][slot % 8]), independently of
the test data generator."""

from __future__ import annotations

import numpy as np
import pytest
import torch

from gpu_common import wrap
from oracle import das_oracle as orc
from paper_2609_34538_amd import _lib as das
from paper_2609_34538_amd import datagen as dg

pytestmark = pytest.mark.gpu
DEV = "cuda"
W = dg.WORKLOADS


# ----------------------------------------------------------------------------
# Commit (das_kv_append)
# ----------------------------------------------------------------------------
def _expected_after_append(cd, k_before, v_before, k_new, v_new, lens, num_new):
    k_exp, v_exp = k_before.clone(), v_before.clone()
    for b, (s, n) in enumerate(zip(lens, num_new)):
        for t in range(n):
            pos = s + t
            page = int(cd.block_table[b, pos // 64])
            k_exp[:, :, :, page, pos % 64, :] = k_new[:, :, b, t, :, :]
            v_exp[:, :, :, page, (pos % 64) // 8, :, pos % 8] = v_new[:, :, b, t, :, :]
    return k_exp, v_exp


@pytest.mark.parametrize("dtype", [torch.bfloat16, torch.float32])
def test_append_bit_exact_and_nothing_else_changes(dtype):
    wl = dg.scaled(W[5], batch=6, hq=3, hkv=3, layers=2, dtype=dtype)
    lens = [0, 63, 64, 40, 130, 7]
    num_new = [0, 3, 32, 32, 5, 1]  # empty, page crossings, full width
    cd = dg.make_cache(wl, DEV, prefix_lens=lens)
    cache, batch = wrap(cd)
    k_new, v_new, _ = dg.commit_inputs(cd, 32, DEV)
    k_before, v_before = cd.k_pool.clone(), cd.v_pool.clone()
    len_out = torch.full((wl.batch,), -7, dtype=torch.int32, device=DEV)
    err = torch.zeros(1, dtype=torch.int32, device=DEV)
    batch.dev_error = err
    batch.refresh()
    das.kv_append(cache, batch, k_new, v_new,
                  torch.tensor(num_new, dtype=torch.int32, device=DEV), len_out)
    torch.cuda.synchronize()
    k_exp, v_exp = _expected_after_append(cd, k_before, v_before, k_new, v_new, lens, num_new)
    iv = torch.int16 if dtype == torch.bfloat16 else torch.int32
    assert torch.equal(cd.k_pool.view(iv), k_exp.view(iv))
    assert torch.equal(cd.v_pool.view(iv), v_exp.view(iv))
    assert len_out.tolist() == [s + n for s, n in zip(lens, num_new)]
    assert int(err.item()) == 0


def test_append_matches_oracle_commit():
    """After the commit, the logical prefix of every stored plane and layer is
    the oracle's list append of the kept verifier K/V."""
    wl = dg.scaled(W[3], batch=4, hq=2, hkv=2, layers=2)
    lens = [10, 64, 100, 0]
    num_new = [4, 16, 0, 9]
    cd = dg.make_cache(wl, DEV, prefix_lens=lens)
    cache, batch = wrap(cd)
    k_new, v_new, _ = dg.commit_inputs(cd, 16, DEV)
    before = {}
    for b, s in enumerate(lens):
        before[b] = ({r: np.stack([dg.gather_prefix_k(cd, b, p, l, s) for l in range(wl.layers)])
                      for r, p in cd.k_plane.items()},
                     {r: np.stack([dg.gather_prefix_v(cd, b, p, l, s) for l in range(wl.layers)])
                      for r, p in cd.v_plane.items()})
    das.kv_append(cache, batch, k_new, v_new, torch.tensor(num_new, dtype=torch.int32, device=DEV))
    torch.cuda.synchronize()
    for b, (s, n) in enumerate(zip(lens, num_new)):
        nk = {r: k_new[p, :, b].double().cpu().numpy() for r, p in cd.k_plane.items()}
        nv = {r: v_new[p, :, b].double().cpu().numpy() for r, p in cd.v_plane.items()}
        want_k, want_v = orc.commit_append(before[b][0], before[b][1], nk, nv, n)
        for r, p in cd.k_plane.items():
            got = np.stack([dg.gather_prefix_k(cd, b, p, l, s + n) for l in range(wl.layers)])
            np.testing.assert_array_equal(got, want_k[r])
        for r, p in cd.v_plane.items():
            got = np.stack([dg.gather_prefix_v(cd, b, p, l, s + n) for l in range(wl.layers)])
            np.testing.assert_array_equal(got, want_v[r])


def test_append_device_range_checks():
    """Out-of-range commit counts and page ids are reported through the error
    word and skipped; nothing outside the valid rows is written."""
    wl = dg.scaled(W[3], batch=3, hq=2, hkv=2, layers=1)
    lens = [10, 20, 30]
    cd = dg.make_cache(wl, DEV, prefix_lens=lens)
    table = cd.block_table.copy()
    table[2, 0] = 10 ** 6  # sequence 2 writes into page 0 of its table: bad id
    cache, batch = wrap(cd, table=table)
    err = torch.zeros(1, dtype=torch.int32, device=DEV)
    batch.dev_error = err
    batch.refresh()
    k_new, v_new, _ = dg.commit_inputs(cd, 16, DEV)
    k_before, v_before = cd.k_pool.clone(), cd.v_pool.clone()
    num_new = torch.tensor([17, 2, 3], dtype=torch.int32, device=DEV)  # 17 > w_max
    len_out = torch.zeros(3, dtype=torch.int32, device=DEV)
    das.kv_append(cache, batch, k_new, v_new, num_new, len_out)
    torch.cuda.synchronize()
    assert int(err.item()) == das.DEVERR_COMMIT | das.DEVERR_PAGE
    assert len_out.tolist() == [10, 22, 33]
    k_exp, v_exp = _expected_after_append(cd, k_before, v_before, k_new, v_new, [10, 20],
                                          [0, 2])
    assert torch.equal(cd.k_pool.view(torch.int16), k_exp.view(torch.int16))
    assert torch.equal(cd.v_pool.view(torch.int16), v_exp.view(torch.int16))


# ----------------------------------------------------------------------------
# One-hot probes through the attention kernels
# ----------------------------------------------------------------------------
ALPHA = 2048.0  # alpha / sqrt(dh) > 200: every other weight underflows to 0


def _code(pos, depth, layer, head):
    # bf16-exact integers below 256
    return [pos % 128, pos // 128, depth, layer, head]


def _build_probe(path):
    wl = dg.scaled(W[4], batch=3, hq=8, hkv=2, dh=96, depth_R=6, layers=2, prefix=(70, 200),
                   draft_depths=(2,), draft_widths=(6,), verify_width=6, paged_random=True,
                   residency="full", k_gain=None)
    lens = [70, 130, 200]
    cd = dg.make_cache(wl, DEV, prefix_lens=lens)
    R, d, dh, G, w = wl.depth_R, 2, wl.dh, wl.group, 6
    rng = np.random.default_rng(7)
    k = torch.zeros_like(cd.k_pool)
    v = torch.zeros_like(cd.v_pool)
    # value codes at every logical position (including stale tails past S_b)
    for b in range(wl.batch):
        for pg_i, page in enumerate(cd.block_table[b]):
            if page < 0:
                continue
            for slot in range(64):
                pos = pg_i * 64 + slot
                for r, p in cd.v_plane.items():
                    for layer in range(wl.layers):
                        for h in range(wl.hkv):
                            v[p, layer, h, page, slot // 8, :5, slot % 8] = torch.tensor(
                                _code(pos, r, layer, h), dtype=v.dtype)
    # every query row (b, i, h) targets its own coordinate c = i * G + h % G
    # and the prefix position hot[b][g][c] whose key at depth d holds e_c;
    # decoys put e_c at other positions in the other planes and layers.
    targets = {}
    layer = 1
    for b, s in enumerate(lens):
        for g in range(wl.hkv):
            for c in range(w * G):
                t = int(rng.integers(0, s))
                targets[(b, g, c)] = t
                page, slot = int(cd.block_table[b, t // 64]), t % 64
                k[cd.k_plane[d], layer, g, page, slot, c] = 1.0
                for r, p in cd.k_plane.items():
                    if r == d:
                        continue
                    t2 = (t + 1 + r) % s
                    k[p, layer, g, int(cd.block_table[b, t2 // 64]), t2 % 64, c] = 1.0
                t3 = (t + 3) % s
                k[cd.k_plane[d], 0, g, int(cd.block_table[b, t3 // 64]), t3 % 64, c] = 1.0
                # masked decoys twice as hot: a stale position past S_b in the
                # last page, which must stay invisible
                tail = s + 1
                if tail < 64 * int((cd.block_table[b] >= 0).sum()):
                    k[cd.k_plane[d], layer, g, int(cd.block_table[b, tail // 64]), tail % 64, c] = 2.0
    q = torch.zeros((wl.batch, w, wl.hq, dh), dtype=wl.dtype, device=DEV)
    for i in range(w):
        for h in range(wl.hq):
            q[:, i, h, i * G + h % G] = ALPHA
    # block keys: zeros except a twice-as-hot key at block position w-1 for the
    # coordinate of (i = w-1, g' = 0): only the last row may see it.
    kb = torch.zeros((wl.batch, w, wl.hkv, dh), dtype=wl.dtype, device=DEV)
    vb = torch.zeros((wl.batch, w, wl.hkv, dh), dtype=wl.dtype, device=DEV)
    for j in range(w):
        vb[:, j, :, 0] = 250 - j
        vb[:, j, :, 5] = 1
    for i in range(w):
        kb[:, w - 1, :, i * G] = 2.0
    cd.k_pool.copy_(k)
    cd.v_pool.copy_(v)
    return cd, q, kb, vb, targets, layer, d, lens


@pytest.mark.parametrize("path", ["valu", "mfma"])
def test_onehot_probe_is_bit_exact(path):
    cd, q, kb, vb, targets, layer, d, lens = _build_probe(path)
    wl = cd.wl
    cache, batch = wrap(cd)
    G, w, R = wl.group, 6, wl.depth_R
    err = torch.zeros(1, dtype=torch.int32, device=DEV)
    batch.dev_error = err
    batch.refresh()
    out = das.attn_policy(cache, batch, layer, d, R, q, kb, vb, path=path, pages_per_split=1)
    torch.cuda.synchronize()
    got = out.float().cpu().numpy()
    assert int(err.item()) == 0
    for b in range(wl.batch):
        for i in range(w):
            for h in range(wl.hq):
                g = h // G
                want = np.zeros(wl.dh, dtype=np.float32)
                if h % G == 0 and i == w - 1:
                    # the block key at j = w-1 (visible to the last row only)
                    # outweighs the prefix target
                    want[0], want[5] = 250 - (w - 1), 1
                else:
                    t = targets[(b, g, i * G + h % G)]
                    want[:5] = _code(t, R, layer, g)
                np.testing.assert_array_equal(got[b, i, h], want,
                                              err_msg=f"b={b} i={i} h={h} {path}")
