"""Helpers shared by the GPU parity tests: oracle evaluation of one attention
call on the logical (unpaged) view of the cache, and the tolerance checks."""

from __future__ import annotations

import numpy as np
import torch

from oracle import das_oracle as orc
from paper_2609_34538_amd import _lib as das
from paper_2609_34538_amd import datagen as dg

# bf16 inputs with fp32 accumulation: max-abs 2e-2 and mean-rel 5e-3;
# fp32 inputs: both 1e-5.
TOL = {torch.bfloat16: (2e-2, 5e-3), torch.float32: (1e-5, 1e-5)}


def wrap(cd: dg.CacheData, table=None, prefix_lens=None, dev_error=None):
    cache = das.PagedCache(cd.k_pool, cd.v_pool, cd.wl.depth_R, cd.k_plane, cd.v_plane)
    table = cd.block_table if table is None else table
    lens = cd.prefix_lens if prefix_lens is None else prefix_lens
    dev = cd.k_pool.device
    batch = das.Batch(torch.as_tensor(np.asarray(lens, dtype=np.int32), device=dev),
                      torch.as_tensor(np.asarray(table, dtype=np.int32), device=dev),
                      dev_error)
    return cache, batch


def oracle_call(cd: dg.CacheData, layer: int, kappa: int, nu: int, q, kb, vb, seqs,
                table=None, prefix_lens=None):
    """fp64 oracle outputs (O [n, w, Hq, dh], lse [n, Hq, w]) of the sequences
    in `seqs`, on exactly the values the GPU read."""
    lens = cd.prefix_lens if prefix_lens is None else prefix_lens
    outs, lses = [], []
    for b in seqs:
        s_len = int(lens[b])
        kc = dg.gather_prefix_k(cd, b, cd.k_plane[kappa], layer, s_len, table)
        vc = dg.gather_prefix_v(cd, b, cd.v_plane[nu], layer, s_len, table)
        o, lse = orc.policy_attention(q[b].double().cpu().numpy(), kc, vc,
                                      kb[b].double().cpu().numpy(),
                                      vb[b].double().cpu().numpy())
        outs.append(o)
        lses.append(lse)
    return np.stack(outs), np.stack(lses)


def error_stats(gpu: np.ndarray, ref: np.ndarray):
    err = np.abs(gpu - ref)
    return float(err.max()), float(err.sum() / max(np.abs(ref).sum(), 1e-300))


def assert_close(gpu: torch.Tensor, ref: np.ndarray, dtype, what: str):
    g = gpu.double().cpu().numpy()
    assert np.isfinite(g).all(), f"{what}: non-finite output"
    max_abs, mean_rel = error_stats(g, ref)
    tol_abs, tol_rel = TOL[dtype]
    assert max_abs <= tol_abs and mean_rel <= tol_rel, (
        f"{what}: max_abs {max_abs:.3e} (tol {tol_abs}) mean_rel {mean_rel:.3e} (tol {tol_rel})")
    return max_abs, mean_rel


def assert_lse_close(gpu_lse: torch.Tensor, ref_lse: np.ndarray, what: str):
    # lse is fp32 arithmetic on fp32 logits: absolute error well below 1e-3
    g = gpu_lse.double().cpu().numpy()
    err = np.abs(g - ref_lse).max()
    assert err <= 1e-3, f"{what}: lse max err {err:.3e}"
