"""fp64 CPU oracle for depth-asynchronous (DAS) policy attention and the
verified-prefix cache commit.

TEST INFRASTRUCTURE ONLY. This module is the plain, slow definition that the
HIP path is checked against. Only ``tests/``, ``__graft_entry__.smoke()`` and
the ``cpu_baseline`` leg of ``bench.py`` may import it; the library and its
Python binding never do, and this module imports nothing from them.

Everything here is written from the paper's statement of the method:

* Eq. (2)  ``[Pi_C, Pi_U] = softmax(Q^{cur} [K_C^kappa ; K_U^{cur}]^T / sqrt(d_h) + M)``
* Eq. (3)  ``O = Pi_C V_C^nu + Pi_U V_U^{cur}``
* Sec. 3.2 text after Eq. (3): M is the causal mask, prefix and draft-side
  positions share one softmax normalisation, and draft-side K/V always come
  from the current draft computation (only the prefix read depths change).
* Eq. (4)  the four read policies: Aligned (r, r), Mature-V / Deep V (r, R),
  Deep K (R, r), Deep K/V (R, R).
* Sec. 3.4 (commit) and App. B.1 (lifetimes): full-depth K/V of accepted,
  materialised inputs are kept, rejected ones are discarded, and provisional
  draft K/V never enter the cache.
* Eq. (5)  the DAS-Wave width schedule ``W_j = min(gamma, W_init + j)``.
* Sec. 3.4  greedy acceptance: accept in order while the proposal equals the
  target argmax; at the first mismatch emit the target prediction.
* Sec. 3.4 / App. B.3  the target prediction is the argmax of each verifier
  conditional; the tie-breaking rule is left to the target, and the reading
  taken here is the lowest index among the maximal entries.

Readings taken where the paper is silent (each one is listed with its
justification in the design notes of the repository):

* mask: every materialised prefix position is visible; block query ``i`` sees
  block keys ``j <= i`` (the standard causal mask over ``[C ; U]`` with the
  block placed after the prefix);
* ``d_h`` is the per-head dimension, so the scale is ``1/sqrt(head_dim)``;
* grouped-query attention: query head ``h`` reads KV head ``h // G`` with
  ``G = Hq / Hkv`` (contiguous groups);
* depths are 1-based, ``1..R``;
* an empty prefix (S = 0) and an empty commit (n = 0) are legal;
* argmax: ties go to the lowest index; NaN entries never win, and a row with
  no non-NaN entry yields index 0.

Pins: this module is checked by ``tests/test_oracle_pins.py`` against a
hand-derived worked example, a library attention routine on a different
formulation, closed forms, invariants and brute force. No function here is
"parity unpinned".
"""

from __future__ import annotations

import math
from typing import Dict, List, Optional, Sequence, Tuple

import numpy as np


def _f64(x) -> np.ndarray:
    return np.asarray(x, dtype=np.float64)


# ---------------------------------------------------------------------------
# Eq. (2)-(3): policy attention over a verified prefix C and the active
# draft-side block U.
# ---------------------------------------------------------------------------
def policy_attention(q, k_prefix, v_prefix, k_block, v_block,
                     return_probs: bool = False):
    """Depth-asynchronous policy attention for one sequence and one core layer.

    Arguments (all converted to float64; exact for fp32/bf16 inputs):
      q        [w, Hq, dh]   queries from the current draft computation
      k_prefix [S, Hkv, dh]  verified-prefix keys read at depth kappa
      v_prefix [S, Hkv, dh]  verified-prefix values read at depth nu
      k_block  [w, Hkv, dh]  draft-side keys at the current depth
      v_block  [w, Hkv, dh]  draft-side values at the current depth

    Returns ``(O [w, Hq, dh], lse [Hq, w])`` where ``lse`` is the natural-log
    softmax normaliser of each row, and with ``return_probs`` also
    ``(Pi_C [Hq, w, S], Pi_U [Hq, w, w])``.
    """
    q = _f64(q)
    kc, vc = _f64(k_prefix), _f64(v_prefix)
    ku, vu = _f64(k_block), _f64(v_block)
    w, hq, dh = q.shape
    s_len = kc.shape[0]
    hkv = ku.shape[1]
    if hq % hkv != 0:
        raise ValueError("query heads must be a multiple of KV heads")
    if kc.shape != (s_len, hkv, dh) or vc.shape != (s_len, hkv, dh):
        raise ValueError("prefix K/V must be [S, Hkv, dh]")
    if ku.shape != (w, hkv, dh) or vu.shape != (w, hkv, dh):
        raise ValueError("block K/V must be [w, Hkv, dh]")
    group = hq // hkv
    scale = 1.0 / math.sqrt(dh)

    # M: prefix always visible; block key j visible to block query i iff j <= i.
    block_visible = np.tril(np.ones((w, w), dtype=bool))

    out = np.zeros((w, hq, dh))
    lse = np.zeros((hq, w))
    pi_c_all = np.zeros((hq, w, s_len))
    pi_u_all = np.zeros((hq, w, w))
    for h in range(hq):
        g = h // group
        # logits against [K_C^kappa ; K_U^cur]
        s_c = (q[:, h, :] @ kc[:, g, :].T) * scale           # [w, S]
        s_u = (q[:, h, :] @ ku[:, g, :].T) * scale           # [w, w]
        s_u = np.where(block_visible, s_u, -np.inf)
        # one softmax over the concatenated positions (shared normaliser)
        m = np.max(np.concatenate([s_c, s_u], axis=1), axis=1, keepdims=True)
        e_c = np.exp(s_c - m)
        e_u = np.exp(s_u - m)
        z = e_c.sum(axis=1, keepdims=True) + e_u.sum(axis=1, keepdims=True)
        pi_c = e_c / z
        pi_u = e_u / z
        # Eq. (3): prefix weights retrieve V at depth nu, block weights the
        # current block values.
        out[:, h, :] = pi_c @ vc[:, g, :] + pi_u @ vu[:, g, :]
        lse[h, :] = (m + np.log(z))[:, 0]
        pi_c_all[h] = pi_c
        pi_u_all[h] = pi_u
    if return_probs:
        return out, lse, pi_c_all, pi_u_all
    return out, lse


# ---------------------------------------------------------------------------
# Eq. (4): read policies over a depth-indexed cache.
# A logical per-sequence cache is a mapping depth r -> array [L, S, Hkv, dh]
# (only the depths that are stored need be present).
# ---------------------------------------------------------------------------
DepthCache = Dict[int, np.ndarray]


def policy_read(cache_k: DepthCache, cache_v: DepthCache, layer: int,
                kappa: int, nu: int, q, k_block, v_block,
                return_probs: bool = False):
    """Generic (kappa, nu) read at core layer ``layer`` (Eq. (2)-(4)).

    The core-layer index is never remapped; only the recurrence depths of the
    prefix K and V change (Sec. 2, depth vs. core-layer indexing)."""
    return policy_attention(q, cache_k[kappa][layer], cache_v[nu][layer],
                            k_block, v_block, return_probs=return_probs)


def draft_maturev(cache_k: DepthCache, cache_v: DepthCache, layer: int,
                  draft_depth: int, full_depth: int, q, k_block, v_block,
                  return_probs: bool = False):
    """Mature-V / Deep V draft read: (kappa, nu) = (d, R)."""
    return policy_read(cache_k, cache_v, layer, draft_depth, full_depth,
                       q, k_block, v_block, return_probs=return_probs)


def verify(cache_k: DepthCache, cache_v: DepthCache, layer: int, depth: int,
           q, k_block, v_block, return_probs: bool = False):
    """The target's ordinary (Aligned) read at depth r: (kappa, nu) = (r, r).

    With r = R this is one core-layer attention of the full-depth verifier."""
    return policy_read(cache_k, cache_v, layer, depth, depth,
                       q, k_block, v_block, return_probs=return_probs)


# ---------------------------------------------------------------------------
# Commit (Sec. 3.4; App. B.1): the verified prefix grows by the accepted,
# materialised inputs, at every stored depth and core layer.
# ---------------------------------------------------------------------------
def commit_append(cache_k: DepthCache, cache_v: DepthCache,
                  new_k: DepthCache, new_v: DepthCache, n_keep: int
                  ) -> Tuple[DepthCache, DepthCache]:
    """Return new caches with the first ``n_keep`` block entries appended.

    ``new_k[r]``/``new_v[r]`` are ``[L, w, Hkv, dh]``: the verifier's K/V of
    the block inputs at depth r. Entries past ``n_keep`` (rejected
    candidates) are discarded. ``n_keep = 0`` leaves the caches unchanged."""
    out_k, out_v = {}, {}
    for store, src, dst in ((cache_k, new_k, out_k), (cache_v, new_v, out_v)):
        for r, plane in store.items():
            n_layers = plane.shape[0]
            rows = []
            for layer in range(n_layers):
                kept: List[np.ndarray] = [plane[layer, s] for s in range(plane.shape[1])]
                for t in range(n_keep):
                    kept.append(src[r][layer, t])
                rows.append(np.stack(kept, axis=0) if kept else
                            np.zeros((0,) + plane.shape[2:], dtype=plane.dtype))
            dst[r] = np.stack(rows, axis=0)
    return out_k, out_v


# ---------------------------------------------------------------------------
# Eq. (5): DAS-Wave active-width schedule.
# ---------------------------------------------------------------------------
def wave_widths(gamma: int, w_init: int, rounds: int) -> List[int]:
    """``W_j = min(gamma, W_init + j)`` for ``j = 0..J-1``."""
    return [min(gamma, w_init + j) for j in range(rounds)]


# ---------------------------------------------------------------------------
# Sec. 3.4: greedy acceptance against the verifier's argmax predictions.
# ---------------------------------------------------------------------------
def greedy_accept(proposals: Sequence[int], target_pred: Sequence[int],
                  tested: Optional[int] = None) -> Tuple[int, List[int]]:
    """Greedy verification of one block.

    ``proposals`` are y_1..y_w; ``target_pred`` are yhat_1..yhat_w (the
    argmax of each verifier conditional p_i). The first ``tested`` proposals
    (m <= w, default w) are checked in order.

    Returns ``(accepted, emitted)``: the number of accepted proposals and the
    tokens emitted by this block (the accepted proposals, then the target
    prediction at the first mismatch, or the bonus prediction when all m
    tested proposals agree and m < w)."""
    w = len(proposals)
    m = w if tested is None else tested
    if len(target_pred) != w or not 0 <= m <= w:
        raise ValueError("bad block")
    accepted = 0
    while accepted < m and proposals[accepted] == target_pred[accepted]:
        accepted += 1
    emitted = list(proposals[:accepted])
    if accepted < m:
        emitted.append(target_pred[accepted])      # correction at first mismatch
    elif m < w:
        emitted.append(target_pred[m])             # unused conditional: bonus
    return accepted, emitted


def commit_count(accepted: int, width: int) -> int:
    """Number of verifier inputs whose full-depth K/V are retained.

    The verifier consumes ``[x_t, y_1..y_{w-1}]`` (Sec. 3.4). The anchor and
    the accepted proposals among those inputs are materialised and valid, so
    ``min(accepted + 1, w)`` entries are kept; the last emitted token becomes
    the next anchor and is materialised by the next verification pass."""
    if not 0 <= accepted <= width or width < 1:
        raise ValueError("bad acceptance count")
    return min(accepted + 1, width)


def argmax_lowest(row) -> int:
    """Target prediction of one verifier conditional (Sec. 3.4: argmax over the
    vocabulary). Ties go to the lowest index; NaN entries are ignored, and a
    row of NaN only yields 0. Values are compared exactly (float64 holds every
    bf16 and fp32 value)."""
    x = _f64(row).ravel()
    best, arg = None, 0
    for v in range(x.shape[0]):
        if np.isnan(x[v]):
            continue
        if best is None or x[v] > best:
            best, arg = x[v], v
    return arg


def greedy_verify(logits, proposals: Sequence[int], tested: Optional[int] = None):
    """Greedy verification of one block from the verifier's outputs.

    ``logits`` [w, V] are the verifier's conditionals p_1..p_w of Eq. (verify
    conditionals) over the vocabulary, ``proposals`` are y_1..y_w and the
    first ``tested`` (default w) are checked (Sec. 3.4). Returns
    ``(target_pred, accepted, emitted, keep)``: the argmax of every row, the
    number of accepted proposals, the emitted tokens, and the number of
    verifier inputs whose full-depth K/V are retained (``commit_count``)."""
    x = _f64(logits)
    w = x.shape[0]
    target_pred = [argmax_lowest(x[i]) for i in range(w)]
    accepted, emitted = greedy_accept(list(proposals), target_pred, tested)
    return target_pred, accepted, emitted, commit_count(accepted, w)
