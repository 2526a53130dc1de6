"""On-device greedy verification (das_greedy_accept) against the oracle's
greedy acceptance and commit count, bit for bit, and the device-side chain
acceptance -> commit."""

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
SENTINEL = -12345


def _run(y, yhat, m, with_tested=True, with_emitted=True):
    B, w = y.shape
    emitted = torch.full((B, w), SENTINEL, dtype=torch.int32, device=DEV) if with_emitted else None
    nem = torch.full((B,), SENTINEL, dtype=torch.int32, device=DEV) if with_emitted else None
    err = torch.zeros(1, dtype=torch.int32, device=DEV)
    acc, keep = das.greedy_accept(y, yhat, m if with_tested else None, emitted=emitted,
                                  num_emitted=nem, dev_error=err)
    torch.cuda.synchronize()
    return acc, keep, emitted, nem, int(err.item())


def _check(y, yhat, m, acc, keep, emitted, nem):
    y, yhat = y.cpu().numpy(), yhat.cpu().numpy()
    B, w = y.shape
    for b in range(B):
        mb = int(m[b]) if m is not None else w
        a_ref, em_ref = orc.greedy_accept(y[b].tolist(), yhat[b].tolist(), mb)
        k_ref = orc.commit_count(a_ref, w)
        assert int(acc[b]) == a_ref, (b, mb)
        assert int(keep[b]) == k_ref, (b, mb)
        if emitted is not None:
            n = int(nem[b])
            assert n == len(em_ref)
            row = emitted[b].cpu().numpy()
            assert row[:n].tolist() == em_ref
            assert (row[n:] == SENTINEL).all()  # nothing written past the emitted tokens


@pytest.mark.parametrize("w", [1, 2, 7, 32, 33, 64])
@pytest.mark.parametrize("random_tested", [False, True])
def test_accept_matches_oracle(w, random_tested):
    B = 37  # not a multiple of the sequences per workgroup
    y, yhat, m = dg.accept_inputs(B, w, seed=100 + w, device=DEV, random_tested=random_tested)
    acc, keep, emitted, nem, err = _run(y, yhat, m)
    assert err == 0
    _check(y, yhat, m.cpu().numpy(), acc.cpu().numpy(), keep.cpu().numpy(), emitted, nem.cpu())
    # every acceptance length from 0 to w occurs in the full-test case
    if not random_tested and w <= 7:
        assert set(acc.cpu().numpy().tolist()) == set(range(w + 1))


def test_accept_without_optional_outputs():
    y, yhat, m = dg.accept_inputs(9, 16, seed=7, device=DEV)
    acc, keep, _, _, err = _run(y, yhat, m, with_tested=False, with_emitted=False)
    assert err == 0
    _check(y, yhat, None, acc.cpu().numpy(), keep.cpu().numpy(), None, None)


def test_tested_out_of_range_is_clamped_and_reported():
    y, yhat, _ = dg.accept_inputs(4, 8, seed=9, device=DEV)
    y[:] = yhat  # everything would be accepted
    m = torch.tensor([-3, 11, 8, 5], dtype=torch.int32, device=DEV)
    acc, keep, emitted, nem, err = _run(y, yhat, m)
    assert err == das.DEVERR_TESTED
    assert acc.cpu().tolist() == [0, 8, 8, 5]
    assert keep.cpu().tolist() == [1, 8, 8, 6]
    _check(y, yhat, np.array([0, 8, 8, 5]), acc.cpu().numpy(), keep.cpu().numpy(), emitted,
           nem.cpu())


def test_accept_feeds_commit_on_device():
    """The commit count written by the acceptance is consumed by das_kv_append
    on the same stream, with no host round trip; the cache then holds the
    oracle's list append of min(a + 1, w) verifier inputs."""
    wl = dg.scaled(dg.WORKLOADS[5], batch=6, hq=3, hkv=3, layers=2)
    lens = [0, 63, 64, 100, 130, 7]
    cd = dg.make_cache(wl, DEV, prefix_lens=lens)
    cache, batch = wrap(cd)
    w = 32
    k_new, v_new, _ = dg.commit_inputs(cd, w, DEV)
    y, yhat, m = dg.accept_inputs(wl.batch, w, seed=11, device=DEV, random_tested=True)
    len_out = torch.empty(wl.batch, dtype=torch.int32, device=DEV)
    acc, keep = das.greedy_accept(y, yhat, m)
    das.kv_append(cache, batch, k_new, v_new, keep, len_out)
    torch.cuda.synchronize()
    keep_h = keep.cpu().numpy()
    a_ref = [orc.greedy_accept(y[b].tolist(), yhat[b].tolist(), int(m[b]))[0]
             for b in range(wl.batch)]
    assert keep_h.tolist() == [orc.commit_count(a, w) for a in a_ref]
    assert len_out.cpu().tolist() == [s + int(k) for s, k in zip(lens, keep_h)]
    for b in range(wl.batch):
        s, n = lens[b], int(keep_h[b])
        for layer in range(wl.layers):
            for r, pl in cd.k_plane.items():
                got = dg.gather_prefix_k(cd, b, pl, layer, s + n)[s:]
                np.testing.assert_array_equal(got, k_new[pl, layer, b, :n].double().cpu().numpy())
            for r, pl in cd.v_plane.items():
                got = dg.gather_prefix_v(cd, b, pl, layer, s + n)[s:]
                np.testing.assert_array_equal(got, v_new[pl, layer, b, :n].double().cpu().numpy())
