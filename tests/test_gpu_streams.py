"""Calls that run concurrently on separate streams, each with its own
workspace, give the same bytes as the same calls run one after another: the
balanced schedule and the split grid side by side, enqueued from one host
thread and from two."""

from __future__ import annotations

import threading

import numpy as np
import pytest
import torch

from gpu_common import wrap
from paper_2609_34538_amd import _lib as das
from paper_2609_34538_amd import datagen as dg

pytestmark = pytest.mark.gpu
DEV = "cuda"


def _setup():
    wl = dg.scaled(dg.WORKLOADS[3], batch=6, hq=8, hkv=4, dh=96, layers=2, prefix=(0, 3000),
                   draft_depths=(2,), draft_widths=(8,), verify_width=8, paged_random=True)
    torch.manual_seed(11)
    cd = dg.make_cache(wl, DEV, prefix_lens=[2999, 0, 700, 1500, 64, 2048])
    cache, batch = wrap(cd)
    # the same cache seen as a single sequence (the split grid)
    _, single = wrap(cd, table=cd.block_table[:1], prefix_lens=cd.prefix_lens[:1])
    q, kb, vb = dg.block_inputs(cd, 8, 2, DEV)
    calls = {
        "balanced": (batch, q, kb, vb, "balanced"),
        "split": (single, q[:1].contiguous(), kb[:1].contiguous(), vb[:1].contiguous(), "mfma"),
    }
    return wl, cache, calls


def _run(wl, cache, args, stream, ws, layer):
    batch, q, kb, vb, path = args
    out = torch.empty_like(q)
    das.attn_policy(cache, batch, layer, 2, wl.depth_R, q, kb, vb, out=out, workspace=ws,
                    path=path, stream=stream)
    return out


def test_two_streams_match_sequential_calls():
    wl, cache, calls = _setup()
    ws = {k: das.alloc_workspace(cache, a[0], wl.hq, 8, path=a[4]) for k, a in calls.items()}
    ref = {}
    for layer in range(wl.layers):
        for k, a in calls.items():
            ref[(k, layer)] = _run(wl, cache, a, None, ws[k], layer)
    torch.cuda.synchronize()
    streams = {k: torch.cuda.Stream() for k in calls}
    for rep in range(4):
        got = {}
        for layer in range(wl.layers):
            for k, a in calls.items():  # enqueued back to back, no synchronisation
                got[(k, layer)] = _run(wl, cache, a, streams[k], ws[k], layer)
        torch.cuda.synchronize()
        for key, t in got.items():
            assert torch.equal(t, ref[key]), f"rep {rep} {key}: concurrent result differs"


def test_two_host_threads_match_sequential_calls():
    wl, cache, calls = _setup()
    ws = {k: das.alloc_workspace(cache, a[0], wl.hq, 8, path=a[4]) for k, a in calls.items()}
    ref = {k: _run(wl, cache, a, None, ws[k], 1) for k, a in calls.items()}
    torch.cuda.synchronize()
    streams = {k: torch.cuda.Stream() for k in calls}
    results, errors = {}, []

    def worker(k):
        try:
            outs = []
            for _ in range(6):
                outs.append(_run(wl, cache, calls[k], streams[k], ws[k], 1))
            streams[k].synchronize()
            results[k] = outs
        except Exception as e:  # reported below, in the main thread
            errors.append(f"{k}: {e!r}")

    threads = [threading.Thread(target=worker, args=(k,)) for k in calls]
    for t in threads:
        t.start()
    for t in threads:
        t.join(timeout=120)
    assert not errors, errors
    for k, outs in results.items():
        for i, t in enumerate(outs):
            assert torch.equal(t, ref[k]), f"thread {k} call {i}: result differs"
    assert set(results) == set(calls)
    assert np.all([torch.isfinite(ref[k].float()).all().item() for k in ref])
