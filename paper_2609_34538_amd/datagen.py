"""Seeded synthetic inputs shaped like the paper's looped-model decode.

This module holds only input generation and the paged-layout bookkeeping
(which physical page holds which logical position). It contains none of the
attention arithmetic, so both the HIP path (through the binding) and the
fp64 oracle (through the tests and the bench's CPU leg) can take their inputs
from it.

Recipe (stand-in for the paper's GSM8K / MATH-500 / HumanEval / MBPP decode
with Huginn / Raven checkpoints, which are not available):

* values: depth-1 planes are N(0, 1); depth r = depth r-1 + sigma * N(0, 1)
  (a random walk over recurrence depth, so depths differ). Only the stored
  depths are drawn: a jump of dr depths adds sigma * sqrt(dr) * N(0, 1),
  which has the walk's distribution exactly.
* queries and block keys/values at depth r are N(0, 1 + (r - 1) sigma^2),
  the walk's marginal at r.
* the long-prefix GQA workload standardises Q and K at each depth to unit
  variance and multiplies K by 3, so logits have standard deviation ~3.
* prefix lengths and commit counts are uniform integers (inclusive bounds)
  drawn from a numpy generator seeded per workload; values come from a torch
  generator on the target device with the same seed.
* paged workloads place each sequence on a seeded random permutation of the
  physical pages; dense ones use consecutive pages.
"""

from __future__ import annotations

import math
from dataclasses import dataclass, field
from typing import Dict, List, Optional, Sequence, Tuple

import numpy as np
import torch

PAGE = 64


@dataclass(frozen=True)
class Workload:
    idx: int
    name: str
    dtype: torch.dtype
    batch: int
    hq: int
    hkv: int
    dh: int
    depth_R: int
    layers: int
    prefix: Tuple[int, int]            # inclusive bounds of S_b
    draft_depths: Tuple[int, ...]      # one per draft round
    draft_widths: Tuple[int, ...]      # block width of each draft round
    verify_width: int
    sigma: float
    k_gain: Optional[float] = None     # standardise Q/K and scale K
    paged_random: bool = False
    append_max: Optional[int] = None   # commit counts ~ U{0..append_max}
    residency: str = "sparse"          # "full": every depth stored

    @property
    def seed(self) -> int:
        return 1000 + self.idx

    @property
    def group(self) -> int:
        return self.hq // self.hkv

    @property
    def w_max(self) -> int:
        return max(max(self.draft_widths), self.verify_width)

    def k_depths(self) -> List[int]:
        if self.residency == "full":
            return list(range(1, self.depth_R + 1))
        return sorted(set(self.draft_depths) | {self.depth_R})

    def v_depths(self) -> List[int]:
        if self.residency == "full":
            return list(range(1, self.depth_R + 1))
        return [self.depth_R]


WORKLOADS: Dict[int, Workload] = {
    1: Workload(1, "tiny-maturev-fp32", torch.float32, 1, 4, 4, 64, 4, 1, (256, 256), (1,), (4,),
                4, 0.3, residency="full"),
    2: Workload(2, "single-seq-looped-bf16", torch.bfloat16, 1, 55, 55, 96, 32, 4, (2048, 2048),
                (4,), (8,), 8, 0.2, residency="full", append_max=8),
    3: Workload(3, "ragged-paged-bf16", torch.bfloat16, 16, 55, 55, 96, 32, 4, (512, 4096), (2,),
                (16,), 16, 0.2, paged_random=True, append_max=16),
    4: Workload(4, "long-prefix-gqa-bf16", torch.bfloat16, 4, 32, 8, 128, 24, 4, (16384, 16384),
                (3,), (32,), 32, 0.15, k_gain=3.0, append_max=32, residency="full"),
    5: Workload(5, "das-wave-step-bf16", torch.bfloat16, 32, 55, 55, 96, 32, 4, (4096, 8192),
                (1, 2, 3, 4), (4, 8, 16, 32), 32, 0.2, paged_random=True, append_max=32),
}


def scaled(wl: Workload, **changes) -> Workload:
    """A copy of a workload with some fields replaced (smaller test shapes)."""
    d = dict(wl.__dict__)
    d.update(changes)
    return Workload(**d)


def depth_std(wl: Workload, depth: int) -> float:
    return math.sqrt(1.0 + (depth - 1) * wl.sigma ** 2)


@dataclass
class CacheData:
    wl: Workload
    prefix_lens: np.ndarray            # [B] int
    block_table: np.ndarray            # [B, max_pages] int32 (-1 = unused)
    pages_of: List[np.ndarray]         # physical pages of each sequence, in order
    k_pool: torch.Tensor               # [nK, L, Hkv, P, 64, dh]
    v_pool: torch.Tensor               # [nV, L, Hkv, P, 8, dh, 8]
    k_plane: Dict[int, int]
    v_plane: Dict[int, int]
    gen: torch.Generator = field(repr=False, default=None)
    np_rng: np.random.Generator = field(repr=False, default=None)


def _np_rng(wl: Workload) -> np.random.Generator:
    return np.random.default_rng(wl.seed)


def make_cache(wl: Workload, device="cuda", prefix_lens: Optional[Sequence[int]] = None,
               copies: int = 1, spare_tokens: Optional[int] = None) -> CacheData:
    """Build the depth-indexed paged pools of a workload.

    Every sequence gets room for its prefix plus ``spare_tokens`` (default:
    the widest block, so a commit fits). ``copies`` > 1 repeats the page
    assignment on disjoint page sets (``block_table`` of copy c is
    ``tables[c]``), which the bench uses to rotate past the last-level cache.
    """
    rng = _np_rng(wl)
    lo, hi = wl.prefix
    if prefix_lens is None:
        prefix_lens = rng.integers(lo, hi + 1, size=wl.batch)
    prefix_lens = np.asarray(prefix_lens, dtype=np.int64)
    spare = wl.w_max if spare_tokens is None else spare_tokens
    n_pages = [max(1, -(-(int(s) + spare) // PAGE)) for s in prefix_lens]
    per_copy = sum(n_pages)
    total = per_copy * copies
    perm = rng.permutation(total) if wl.paged_random else np.arange(total)
    max_pages = max(n_pages)
    tables = []
    pages_of_all = []
    cursor = 0
    for _ in range(copies):
        table = np.full((wl.batch, max_pages), -1, dtype=np.int32)
        pages_of = []
        for b, n in enumerate(n_pages):
            pg = perm[cursor:cursor + n].astype(np.int32)
            cursor += n
            table[b, :n] = pg
            pages_of.append(pg)
        tables.append(table)
        pages_of_all.append(pages_of)

    kd, vd = wl.k_depths(), wl.v_depths()
    k_plane = {d: i for i, d in enumerate(kd)}
    v_plane = {d: i for i, d in enumerate(vd)}
    gen = torch.Generator(device=device)
    gen.manual_seed(wl.seed)
    shape = (wl.hkv, total, PAGE, wl.dh)
    k_pool = torch.empty((len(kd), wl.layers) + shape, dtype=wl.dtype, device=device)
    v_pool = torch.empty((len(vd), wl.layers, wl.hkv, total, PAGE // 8, wl.dh, 8),
                         dtype=wl.dtype, device=device)
    for layer in range(wl.layers):
        for pool, depths, is_v in ((k_pool, kd, False), (v_pool, vd, True)):
            cur = torch.randn(shape, generator=gen, device=device, dtype=torch.float32)
            prev = 1
            for i, d in enumerate(depths):
                if d > prev:
                    cur.add_(torch.randn(shape, generator=gen, device=device,
                                         dtype=torch.float32), alpha=wl.sigma * math.sqrt(d - prev))
                    prev = d
                x = cur
                if wl.k_gain is not None and not is_v:
                    x = cur * (wl.k_gain / depth_std(wl, d))
                if is_v:  # token-grouped value pages [8][dh][8]
                    pool[i, layer].copy_(
                        x.reshape(wl.hkv, total, PAGE // 8, 8, wl.dh).transpose(-1, -2))
                else:
                    pool[i, layer].copy_(x)
            del cur
    cd = CacheData(wl, prefix_lens, tables[0], pages_of_all[0], k_pool, v_pool, k_plane,
                   v_plane, gen, rng)
    cd.tables = tables
    cd.pages_of_all = pages_of_all
    return cd


def block_inputs(cd: CacheData, width: int, depth: int, device="cuda"):
    """Q [B, w, Hq, dh] and draft-side / verifier block K, V [B, w, Hkv, dh]
    at recurrence depth ``depth``."""
    wl = cd.wl
    std = depth_std(wl, depth)
    g = cd.gen
    q = torch.randn((wl.batch, width, wl.hq, wl.dh), generator=g, device=device) * std
    kb = torch.randn((wl.batch, width, wl.hkv, wl.dh), generator=g, device=device) * std
    vb = torch.randn((wl.batch, width, wl.hkv, wl.dh), generator=g, device=device) * std
    if wl.k_gain is not None:
        q = q / std
        kb = kb * (wl.k_gain / std)
    return q.to(wl.dtype), kb.to(wl.dtype), vb.to(wl.dtype)


def commit_inputs(cd: CacheData, width: int, device="cuda"):
    """Verifier K/V of a block for every stored plane ([nK|nV, L, B, w, Hkv, dh])
    and seeded commit counts num_new [B] ~ U{0..append_max}."""
    wl = cd.wl
    nk, nv = cd.k_pool.shape[0], cd.v_pool.shape[0]
    g = cd.gen
    k_new = torch.randn((nk, wl.layers, wl.batch, width, wl.hkv, wl.dh), generator=g,
                        device=device).to(wl.dtype)
    v_new = torch.randn((nv, wl.layers, wl.batch, width, wl.hkv, wl.dh), generator=g,
                        device=device).to(wl.dtype)
    hi = width if wl.append_max is None else min(wl.append_max, width)
    num_new = cd.np_rng.integers(0, hi + 1, size=wl.batch).astype(np.int32)
    return k_new, v_new, num_new


# ---------------------------------------------------------------------------
# Paged layout bookkeeping (physical page of logical position pos of sequence
# b is block_table[b][pos // 64], row pos % 64 of that page).
# ---------------------------------------------------------------------------
def gather_prefix_k(cd: CacheData, b: int, plane: int, layer: int, s_len: int,
                    table: Optional[np.ndarray] = None) -> np.ndarray:
    """Logical prefix keys [S, Hkv, dh] of sequence b (float64 numpy)."""
    table = cd.block_table if table is None else table
    npg = -(-s_len // PAGE)
    pages = torch.as_tensor(table[b, :npg].astype(np.int64), device=cd.k_pool.device)
    t = cd.k_pool[plane, layer].index_select(1, pages)         # [Hkv, npg, 64, dh]
    t = t.permute(1, 2, 0, 3).reshape(npg * PAGE, cd.wl.hkv, cd.wl.dh)[:s_len]
    return t.double().cpu().numpy()


def gather_prefix_v(cd: CacheData, b: int, plane: int, layer: int, s_len: int,
                    table: Optional[np.ndarray] = None) -> np.ndarray:
    """Logical prefix values [S, Hkv, dh] of sequence b (float64 numpy)."""
    table = cd.block_table if table is None else table
    npg = -(-s_len // PAGE)
    pages = torch.as_tensor(table[b, :npg].astype(np.int64), device=cd.v_pool.device)
    t = cd.v_pool[plane, layer].index_select(1, pages)         # [Hkv, npg, 8, dh, 8]
    t = t.permute(1, 2, 4, 0, 3).reshape(npg * PAGE, cd.wl.hkv, cd.wl.dh)[:s_len]
    return t.double().cpu().numpy()


def accept_inputs(batch: int, width: int, seed: int, vocab: int = 65536, device="cuda",
                  random_tested: bool = False):
    """Seeded verifier predictions yhat [B, w], proposals y [B, w] and tested
    counts m [B] (int32). Each sequence's proposals agree with the predictions
    on a leading run of U{0..w} positions and differ at the next one, so every
    acceptance length occurs; m = w unless random_tested (then U{0..w})."""
    rng = np.random.default_rng(seed)
    yhat = rng.integers(0, vocab, size=(batch, width))
    y = rng.integers(0, vocab, size=(batch, width))
    run = rng.integers(0, width + 1, size=batch)
    for b in range(batch):
        y[b, :run[b]] = yhat[b, :run[b]]
        if run[b] < width:
            y[b, run[b]] = (yhat[b, run[b]] + 1 + rng.integers(0, vocab - 1)) % vocab
    m = rng.integers(0, width + 1, size=batch) if random_tested else np.full(batch, width)
    t = lambda x: torch.as_tensor(np.ascontiguousarray(x).astype(np.int32), device=device)
    return t(y), t(yhat), t(m)
