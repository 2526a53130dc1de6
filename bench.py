"""Benchmark of the DAS hot path on one MI355X.

A step is one pass of the whole hot path over one batch of synthetic input:
the Mature-V draft attention of every core layer (keys at the draft depth d,
values at the full depth R), the full-depth verifier attention of every core
layer over the same block, and the commit of the accepted block K/V into the
depth-indexed paged cache. Inputs are resident in HBM before timing starts.

Default workload: a single sequence shaped like the paper's looped models
(bf16, 55 query = 55 KV heads, head_dim 96, verified prefix 2048, draft block
8, R = 32, d = 4, 4 core layers, every depth of the cache stored).
Successive steps rotate over disjoint copies of the cache pages so that the
bytes a step reads are not served by the 256 MB last-level cache. Each step
is captured once per cache copy as a HIP graph and replayed (--eager launches
every call from the host instead).

Prints one JSON line: throughput (block tokens per second, HIP events around
the timed steps), the roofline of the dominant kernel (the attention launch =
attention kernel + split combine, HBM bound: algorithmic bytes over the
average launch duration, from HIP events around replays of each step's
attention launches on the same stream right after the timed steps), and the
fp64 oracle timed on the host's cores on a bounded sample.
"""

from __future__ import annotations

import argparse
import json
import math
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--warmup", type=int, default=10)
    ap.add_argument("--config", type=int, default=2, help="workload index (1-5)")
    ap.add_argument("--path", default="auto", choices=["auto", "valu", "mfma"])
    ap.add_argument("--pps", type=int, default=0, help="prefix pages per split (0 = library)")
    ap.add_argument("--rotate-bytes", type=float, default=1.0e9,
                    help="minimum bytes between reuses of a cache copy")
    ap.add_argument("--cpu-seconds", type=float, default=10.0)
    ap.add_argument("--no-cpu", action="store_true")
    ap.add_argument("--attn-only", action="store_true",
                    help="profiling aid: time only the attention launches")
    ap.add_argument("--eager", action="store_true",
                    help="launch every call from the host instead of replaying HIP graphs")
    return ap.parse_args()


def algorithmic_attn_bytes(wl, lens, w):
    """Prefix K at kappa + prefix V at nu (every visible position once) plus
    Q, O, block K and block V."""
    e = 2 if wl.dtype.itemsize == 2 else 4
    prefix = 2 * int(np.sum(lens)) * wl.hkv * wl.dh * e
    block = wl.batch * w * (2 * wl.hq + 2 * wl.hkv) * wl.dh * e
    return prefix + block


def algorithmic_append_bytes(wl, nk, nv, num_new):
    e = 2 if wl.dtype.itemsize == 2 else 4
    return 2 * int(np.sum(num_new)) * (nk + nv) * wl.layers * wl.hkv * wl.dh * e


def cpu_baseline(cd, step_calls, seconds, tokens_per_step):
    """Time the fp64 oracle on the calls of one step (cycled until the time
    budget is used) and scale to tokens per second of a whole step."""
    import torch
    from oracle import das_oracle as orc
    from paper_2609_34538_amd import datagen as dg

    cores = len(os.sched_getaffinity(0))
    torch.set_num_threads(cores)
    prepared = []
    for (layer, kappa, nu, q, kb, vb) in step_calls:
        for b in range(cd.wl.batch):
            s = int(cd.prefix_lens[b])
            prepared.append((q[b].double().cpu().numpy(),
                             dg.gather_prefix_k(cd, b, cd.k_plane[kappa], layer, s),
                             dg.gather_prefix_v(cd, b, cd.v_plane[nu], layer, s),
                             kb[b].double().cpu().numpy(), vb[b].double().cpu().numpy()))
    per_step = len(prepared)
    done = 0
    t0 = time.perf_counter()
    while True:
        args = prepared[done % per_step]
        orc.policy_attention(*args)
        done += 1
        el = time.perf_counter() - t0
        if el >= seconds and done >= per_step:
            break
    steps = done / per_step
    return {"value": tokens_per_step * steps / el, "unit": "tokens/s", "cores": cores,
            "kind": "oracle",
            "sample": (f"{done} fp64 oracle per-sequence attention calls "
                       f"({steps:.2f} steps of {per_step} calls: draft and verify, every layer) "
                       f"in {el:.1f} s; commit not included")}


def main():
    args = parse()
    if args.gpus != 1:
        print(json.dumps({"error": "this build runs on one GPU; --gpus must be 1",
                          "n_gpus": args.gpus}))
        sys.exit(2)
    import torch
    from paper_2609_34538_amd import _lib as das
    from paper_2609_34538_amd import datagen as dg

    dev = "cuda"
    wl = dg.WORKLOADS[args.config]
    rounds = list(zip(wl.draft_depths, wl.draft_widths))
    R = wl.depth_R
    # bytes one step reads, to size the cache rotation
    rng_lens = np.random.default_rng(wl.seed).integers(wl.prefix[0], wl.prefix[1] + 1,
                                                       size=wl.batch)
    step_read = sum(algorithmic_attn_bytes(wl, rng_lens, w) for _, w in rounds) * wl.layers
    step_read += algorithmic_attn_bytes(wl, rng_lens, wl.verify_width) * wl.layers
    copies = max(1, min(16, math.ceil(args.rotate_bytes / max(step_read, 1))))
    cd = dg.make_cache(wl, dev, copies=copies)
    lens = cd.prefix_lens
    cache = das.PagedCache(cd.k_pool, cd.v_pool, R, cd.k_plane, cd.v_plane)
    batches = [das.Batch(torch.as_tensor(lens.astype(np.int32), device=dev),
                         torch.as_tensor(t, device=dev)) for t in cd.tables]
    # per-round block inputs; the verifier's block K/V is the commit source
    draft_in = [dg.block_inputs(cd, w, d, dev) for d, w in rounds]
    qv, _, _ = dg.block_inputs(cd, wl.verify_width, R, dev)
    k_new, v_new, num_new = dg.commit_inputs(cd, wl.verify_width, dev)
    num_new_t = torch.as_tensor(num_new, device=dev)
    kp, vp = cd.k_plane[R], cd.v_plane[R]
    opts = dict(path=args.path, pages_per_split=args.pps)
    wmax = max(w for _, w in rounds + [(R, wl.verify_width)])
    ws = das.alloc_workspace(cache, batches[0], wl.hq, wmax, **opts)
    outs = [torch.empty_like(q) for q, _, _ in draft_in]
    out_v = torch.empty_like(qv)
    len_out = torch.empty(wl.batch, dtype=torch.int32, device=dev)
    # A stream of its own (default priority): graphs cannot be captured on
    # the legacy default stream.
    # Graph replays launch on the current stream, so it is made current.
    stream = torch.cuda.Stream()
    torch.cuda.synchronize()
    torch.cuda.set_stream(stream)

    # Every call of a step, marshalled once per cache copy: the Mature-V
    # draft of each layer (and round), the verifier of each layer, the commit.
    step_calls = []
    for batch in batches:
        seq = []
        for layer in range(wl.layers):
            for r, (d, w) in enumerate(rounds):
                q, kb, vb = draft_in[r]
                seq.append((w, das.PreparedAttention(cache, batch, layer, d, R, q, kb, vb, outs[r],
                                                     ws, stream=stream, **opts)))
        for layer in range(wl.layers):
            seq.append((wl.verify_width,
                        das.PreparedAttention(cache, batch, layer, R, R, qv, k_new[kp, layer],
                                              v_new[vp, layer], out_v, ws, stream=stream,
                                              **opts)))
        if not args.attn_only:
            seq.append((None, das.PreparedAppend(cache, batch, k_new, v_new, num_new_t, len_out,
                                                 stream=stream)))
        step_calls.append(seq)
    n_attn = sum(1 for w, _ in step_calls[0] if w is not None)
    widths = [w for w, _ in step_calls[0] if w is not None]
    ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
          for _ in range(args.steps if not args.eager else n_attn * args.steps)]
    spans = []  # (start event, end event, attention launches covered)

    if args.eager:
        def step(i, timed):
            k = 0
            for w, call in step_calls[i % copies]:
                if timed and w is not None:
                    e0, e1 = ev[(i * n_attn) + k]
                    e0.record(stream)
                    call()
                    e1.record(stream)
                    spans.append((e0, e1, [w]))
                    k += 1
                else:
                    call()
    else:
        # Per cache copy: one graph holding the whole step (every attention
        # launch, then the commit), replayed for the timed steps, and one
        # holding only the step's attention launches, replayed between HIP
        # events afterwards to time the attention launches on their own.
        for seq in step_calls:  # eager pass first: per-device state is set up
            for _, call in seq:
                call()
        torch.cuda.synchronize()
        graphs = []
        for seq in step_calls:
            g_step = torch.cuda.CUDAGraph()
            with torch.cuda.graph(g_step, stream=stream):
                for w, call in seq:
                    if w is not None:
                        call()
                for w, call in seq:
                    if w is None:
                        call()
            g_attn = torch.cuda.CUDAGraph()
            with torch.cuda.graph(g_attn, stream=stream):
                for w, call in seq:
                    if w is not None:
                        call()
            graphs.append((g_step, g_attn))
        torch.cuda.synchronize()

        def step(i, timed):
            graphs[i % copies][0].replay()

    for i in range(args.warmup):
        step(i, False)
    torch.cuda.synchronize()
    t_start = torch.cuda.Event(enable_timing=True)
    t_end = torch.cuda.Event(enable_timing=True)
    t_start.record(stream)
    for i in range(args.steps):
        step(i, True)
    t_end.record(stream)
    torch.cuda.synchronize()
    total_ms = t_start.elapsed_time(t_end)
    ms_step = total_ms / args.steps
    tokens_per_step = wl.batch * wl.verify_width  # block tokens verified per step
    value = tokens_per_step / (ms_step / 1e3)

    if not args.eager:
        # attention launches alone: the same steps' attention graphs between events
        for i in range(args.warmup):
            graphs[i % copies][1].replay()
        for i in range(args.steps):
            e0, e1 = ev[i]
            e0.record(stream)
            graphs[i % copies][1].replay()
            e1.record(stream)
            spans.append((e0, e1, widths))
        torch.cuda.synchronize()

    # dominant kernel: the attention launches
    attn_total_ms = sum(a.elapsed_time(b) for a, b, _ in spans)
    launches = [w for _, _, ws_ in spans for w in ws_]
    attn_ms = attn_total_ms / len(launches)
    bytes_per = float(np.mean([algorithmic_attn_bytes(wl, lens, w) for w in launches]))
    achieved = bytes_per / (attn_ms / 1e3) / 1e9
    step_bytes = (sum(algorithmic_attn_bytes(wl, lens, w) for _, w in rounds) * wl.layers
                  + algorithmic_attn_bytes(wl, lens, wl.verify_width) * wl.layers
                  + (0 if args.attn_only else
                     algorithmic_append_bytes(wl, cd.k_pool.shape[0], cd.v_pool.shape[0],
                                              num_new)))

    result = {
        "metric": "Mature-V draft-block attention tokens/s + achieved HBM GB/s (% of 8 TB/s)",
        "value": value,
        "unit": "tokens/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms_step,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16" if wl.dtype.itemsize == 2 else "f32",
        "data": "synthetic",
        "config": {"workload": wl.name, "batch": wl.batch, "q_heads": wl.hq,
                   "kv_heads": wl.hkv, "head_dim": wl.dh, "prefix_len": [int(lens.min()),
                                                                          int(lens.max())],
                   "draft_blocks": [{"depth": d, "width": w} for d, w in rounds],
                   "verify": {"depth": R, "width": wl.verify_width}, "depth_R": R,
                   "core_layers": wl.layers, "path": args.path,
                   "pages_per_split": args.pps, "cache_copies_rotated": copies,
                   "launch": "eager" if args.eager else "hip_graph",
                   "commit": not args.attn_only},
        "step_hbm_gbs": step_bytes / (ms_step / 1e3) / 1e9,
        "step_frac_of_8tbs": step_bytes / (ms_step / 1e3) / 1e9 / HBM_PEAK_GBS,
        "roofline": {"bound": "hbm", "achieved": achieved, "peak": HBM_PEAK_GBS,
                     "unit": "GB/s", "frac": achieved / HBM_PEAK_GBS, "traffic": None,
                     "kernel": "attention launch (partial + split combine)",
                     "timing": ("HIP events around each attention launch in the timed steps"
                                if args.eager else
                                "HIP events around replays of each step's attention launches, "
                                "run after the timed steps on the same stream"),
                     "avg_launch_us": attn_ms * 1e3, "bytes_per_launch": bytes_per},
    }
    if not args.no_cpu:
        calls = []
        for layer in range(wl.layers):
            for r, (d, w) in enumerate(rounds):
                q, kb, vb = draft_in[r]
                calls.append((layer, d, R, q, kb, vb))
            calls.append((layer, R, R, qv, k_new[kp, layer], v_new[vp, layer]))
        result["cpu_baseline"] = cpu_baseline(cd, calls, args.cpu_seconds, tokens_per_step)
    print(json.dumps(result))


if __name__ == "__main__":
    main()
