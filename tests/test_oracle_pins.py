"""Pins for the fp64 oracle, independent of the oracle's own arithmetic.

Each check below ties the oracle to something it does not compute itself:
a hand-derived worked example (tests/golden), a library attention routine
applied to a different formulation, brute force over absolute positions,
closed forms and invariants of Eq. (2)-(3). The mutation test at the end
plants plausible mistakes into a faithful copy of the oracle's steps and
shows that every one of them is caught by at least one pin.
"""

import json
import math
import os

import numpy as np
import pytest
import torch

from oracle import das_oracle as orc

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _rng(seed):
    return np.random.default_rng(seed)


def _rand_case(seed, w, s_len, hq, hkv, dh, scale=1.0):
    r = _rng(seed)
    q = r.standard_normal((w, hq, dh)) * scale
    kc = r.standard_normal((s_len, hkv, dh))
    vc = r.standard_normal((s_len, hkv, dh))
    ku = r.standard_normal((w, hkv, dh))
    vu = r.standard_normal((w, hkv, dh))
    return q, kc, vc, ku, vu


def _oracle_fn(q, kc, vc, ku, vu):
    return orc.policy_attention(q, kc, vc, ku, vu, return_probs=True)


# ----------------------------------------------------------------------------
# Pin checks. Each takes an attention function with the oracle's signature
# (returning O, lse, Pi_C, Pi_U) and raises AssertionError on a mismatch.
# ----------------------------------------------------------------------------
def check_golden(fn):
    """Hand-derived worked example (tests/golden/maturev_worked_example.json)."""
    g = json.load(open(os.path.join(GOLDEN, "maturev_worked_example.json")))
    a = math.log(2.0)
    dh = g["head_dim"]
    w = len(g["q_first_coord_in_ln2"])

    def vec_first(x):
        out = np.zeros((len(x), 1, dh))
        out[:, 0, 0] = x
        return out

    q = vec_first([c * a for c in g["q_first_coord_in_ln2"]])
    k = {name: vec_first(v) for name, v in g["k_prefix_first_coord"].items()}
    v = {name: np.asarray(x, float)[:, None, :] for name, x in g["v_prefix"].items()}
    ku = vec_first(g["k_block_first_coord"])
    vu = np.asarray(g["v_block"], float)[:, None, :]
    policies = {"maturev": ("d", "R"), "aligned": ("d", "d"),
                "deep_kv": ("R", "R"), "deep_k": ("R", "d")}
    for name, (kap, nu) in policies.items():
        o, lse, _, _ = fn(q, k[kap], v[nu], ku, vu)
        exp = g["expected"][name]
        want = np.asarray(exp["num"], float) / np.asarray(exp["den"], float)[:, None]
        np.testing.assert_allclose(o[:, 0, :], want, rtol=0, atol=1e-13, err_msg=name)
        np.testing.assert_allclose(lse[0], np.log(exp["lse_exp"]), rtol=0, atol=1e-13,
                                   err_msg=name + " lse")
    assert w == 2


def _sdpa_reference(q, kc, vc, ku, vu):
    """torch SDPA (fp64, CPU) over the concatenated positions with an explicit
    boolean mask; GQA handled by the library's own grouping."""
    w, hq, dh = q.shape
    s_len, hkv = kc.shape[0], kc.shape[1]
    key = torch.from_numpy(np.concatenate([kc, ku], 0)).permute(1, 0, 2)[None]
    val = torch.from_numpy(np.concatenate([vc, vu], 0)).permute(1, 0, 2)[None]
    qry = torch.from_numpy(np.ascontiguousarray(q)).permute(1, 0, 2)[None]
    mask = torch.zeros((w, s_len + w), dtype=torch.bool)
    mask[:, :s_len] = True
    mask[:, s_len:] = torch.tril(torch.ones((w, w), dtype=torch.bool))
    out = torch.nn.functional.scaled_dot_product_attention(
        qry.contiguous(), key.contiguous(), val.contiguous(), attn_mask=mask,
        enable_gqa=(hq != hkv))
    return out[0].permute(1, 0, 2).numpy()


def check_sdpa(fn):
    """Library cross-check: K and V from different depths are just two tensors
    to the library, so SDPA computes Eq. (2)-(3) as stated."""
    cases = [(1, 3, 5, 2, 2, 8), (2, 4, 0, 2, 1, 8), (3, 5, 9, 4, 2, 6),
             (4, 1, 1, 3, 3, 4), (5, 6, 13, 8, 2, 16), (6, 2, 7, 6, 3, 5)]
    for seed, w, s_len, hq, hkv, dh in cases:
        q, kc, vc, ku, vu = _rand_case(seed, w, s_len, hq, hkv, dh, scale=1.5)
        o, _, _, _ = fn(q, kc, vc, ku, vu)
        np.testing.assert_allclose(o, _sdpa_reference(q, kc, vc, ku, vu),
                                   rtol=0, atol=1e-10, err_msg=str((seed, w, s_len, hq, hkv)))


def _brute_causal(q, kseq, vseq, q_pos, group):
    """Ordinary causal attention written over absolute positions with Python
    loops: query at position p attends keys at positions 0..p."""
    w, hq, dh = q.shape
    out = np.zeros((w, hq, dh))
    lse = np.zeros((hq, w))
    for h in range(hq):
        g = h // group
        for i in range(w):
            p = q_pos[i]
            scores = [sum(q[i, h, c] * kseq[j, g, c] for c in range(dh)) / math.sqrt(dh)
                      for j in range(p + 1)]
            top = max(scores)
            wts = [math.exp(s - top) for s in scores]
            z = sum(wts)
            for c in range(dh):
                out[i, h, c] = sum(wts[j] * vseq[j, g, c] for j in range(p + 1)) / z
            lse[h, i] = top + math.log(z)
    return out, lse


def check_causal_full_depth(fn):
    """d = R: every read is at one depth, so the call must be ordinary causal
    attention of the block appended after the prefix (Eq. (4) with
    kappa = nu = r)."""
    for seed, w, s_len, hq, hkv, dh in [(11, 3, 4, 2, 1, 3), (12, 4, 0, 2, 2, 2),
                                         (13, 2, 5, 3, 3, 4), (14, 5, 2, 4, 2, 3)]:
        q, kc, vc, ku, vu = _rand_case(seed, w, s_len, hq, hkv, dh)
        kseq = np.concatenate([kc, ku], 0)
        vseq = np.concatenate([vc, vu], 0)
        want, want_lse = _brute_causal(q, kseq, vseq, [s_len + i for i in range(w)], hq // hkv)
        o, lse, _, _ = fn(q, kc, vc, ku, vu)
        np.testing.assert_allclose(o, want, rtol=0, atol=1e-12)
        np.testing.assert_allclose(lse, want_lse, rtol=0, atol=1e-12)


def check_rows_sum_to_one(fn):
    """Joint normalisation: Pi_C and Pi_U of a row sum to 1 together, all
    weights are non-negative and masked block weights are exactly zero."""
    for seed, w, s_len, hq, hkv, dh in [(21, 5, 7, 4, 2, 8), (22, 3, 0, 2, 2, 4),
                                         (23, 8, 33, 6, 3, 16)]:
        q, kc, vc, ku, vu = _rand_case(seed, w, s_len, hq, hkv, dh, scale=2.0)
        _, _, pc, pu = fn(q, kc, vc, ku, vu)
        tot = pc.sum(axis=2) + pu.sum(axis=2)
        np.testing.assert_allclose(tot, 1.0, rtol=0, atol=1e-12)
        assert (pc >= 0).all() and (pu >= 0).all()
        upper = np.triu(np.ones((w, w), dtype=bool), k=1)
        assert (pu[:, upper] == 0.0).all()
        # every visible position gets weight (no dropped terms)
        assert (pu[:, ~upper] > 0).all()
        if s_len:
            assert (pc > 0).all()


def check_permutation(fn):
    """Permuting prefix positions jointly in K and V leaves O unchanged;
    permuting V alone must change it (negative control)."""
    for seed, w, s_len, hq, hkv, dh in [(31, 4, 9, 4, 2, 8), (32, 2, 16, 2, 1, 4)]:
        q, kc, vc, ku, vu = _rand_case(seed, w, s_len, hq, hkv, dh)
        perm = _rng(seed + 100).permutation(s_len)
        o, lse, _, _ = fn(q, kc, vc, ku, vu)
        o2, lse2, _, _ = fn(q, kc[perm], vc[perm], ku, vu)
        np.testing.assert_allclose(o2, o, rtol=0, atol=1e-12)
        np.testing.assert_allclose(lse2, lse, rtol=0, atol=1e-12)
        o3, _, _, _ = fn(q, kc, vc[perm], ku, vu)
        assert np.abs(o3 - o).max() > 1e-3


def check_closed_forms(fn):
    """Closed forms of Eq. (2)-(3)."""
    # S = 0, w = 1: the only visible key is the block's own, O = V_U[0].
    q, kc, vc, ku, vu = _rand_case(41, 1, 0, 3, 3, 8)
    o, lse, _, _ = fn(q, kc, vc, ku, vu)
    np.testing.assert_array_equal(o[0], vu[0])
    np.testing.assert_allclose(lse[:, 0], np.einsum("hc,hc->h", q[0], ku[0]) / math.sqrt(8),
                               rtol=0, atol=1e-14)
    # Q = 0: uniform weights over the S + i + 1 visible rows, prefix V at nu
    # and block V at the current depth.
    q, kc, vc, ku, vu = _rand_case(42, 4, 6, 2, 1, 5)
    o, lse, _, _ = fn(np.zeros_like(q), kc, vc, ku, vu)
    for i in range(4):
        want = (vc[:, 0].sum(0) + vu[: i + 1, 0].sum(0)) / (6 + i + 1)
        np.testing.assert_allclose(o[i, 0], want, rtol=0, atol=1e-13)
        np.testing.assert_allclose(lse[:, i], math.log(6 + i + 1), rtol=0, atol=1e-13)
    # Mature-V isolation: V_C^nu = V_C^kappa + c shifts O by c * sum(Pi_C).
    q, kc, vc, ku, vu = _rand_case(43, 5, 11, 4, 2, 6)
    c = np.linspace(-1.0, 2.0, 6)
    o_al, _, pc, _ = fn(q, kc, vc, ku, vu)
    o_mv, _, _, _ = fn(q, kc, vc + c, ku, vu)
    want = o_al + pc.sum(axis=2).T[:, :, None] * c[None, None, :]
    np.testing.assert_allclose(o_mv, want, rtol=0, atol=1e-12)


def check_gqa(fn):
    """GQA equals multi-head attention with each KV head repeated for its
    contiguous group of query heads."""
    q, kc, vc, ku, vu = _rand_case(51, 4, 10, 6, 2, 8)
    o, lse, _, _ = fn(q, kc, vc, ku, vu)
    rep = lambda x: np.repeat(x, 3, axis=1)
    o2, lse2, _, _ = fn(q, rep(kc), rep(vc), rep(ku), rep(vu))
    np.testing.assert_allclose(o2, o, rtol=0, atol=1e-13)
    np.testing.assert_allclose(lse2, lse, rtol=0, atol=1e-13)


def check_split_merge(fn):
    """Log-sum-exp merge of two prefix halves equals the whole: the
    decomposition a split-prefix implementation relies on."""
    q, kc, vc, ku, vu = _rand_case(61, 3, 20, 2, 2, 8, scale=2.0)
    o, lse, _, _ = fn(q, kc, vc, ku, vu)
    oa, la, _, _ = fn(q, kc[:9], vc[:9], ku, vu)
    # second half without block positions: plain softmax attention over the
    # remaining prefix rows, written out directly
    ob = np.zeros_like(o)
    lb = np.zeros_like(lse)
    for h in range(2):
        s = q[:, h] @ kc[9:, h].T / math.sqrt(8)
        m = s.max(1, keepdims=True)
        e = np.exp(s - m)
        ob[:, h] = (e / e.sum(1, keepdims=True)) @ vc[9:, h]
        lb[h] = m[:, 0] + np.log(e.sum(1))
    top = np.maximum(la, lb)
    wa, wb = np.exp(la - top), np.exp(lb - top)
    merged = (oa * wa.T[:, :, None] + ob * wb.T[:, :, None]) / (wa + wb).T[:, :, None]
    np.testing.assert_allclose(merged, o, rtol=0, atol=1e-12)
    np.testing.assert_allclose(top + np.log(wa + wb), lse, rtol=0, atol=1e-12)


PINS = [check_golden, check_sdpa, check_causal_full_depth, check_rows_sum_to_one,
        check_permutation, check_closed_forms, check_gqa, check_split_merge]


@pytest.mark.parametrize("pin", PINS, ids=lambda f: f.__name__)
def test_oracle_pinned(pin):
    pin(_oracle_fn)


# ----------------------------------------------------------------------------
# Depth-indexed policy entry points (Eq. (4)).
# ----------------------------------------------------------------------------
def _depth_cache(seed, depths, n_layers, s_len, hkv, dh):
    r = _rng(seed)
    base_k = r.standard_normal((n_layers, s_len, hkv, dh))
    base_v = r.standard_normal((n_layers, s_len, hkv, dh))
    ck, cv = {}, {}
    for d in depths:
        ck[d] = base_k + 0.3 * d * r.standard_normal(base_k.shape)
        cv[d] = base_v + 0.3 * d * r.standard_normal(base_v.shape)
    return ck, cv


def test_policy_entry_points_select_depths_and_layer():
    ck, cv = _depth_cache(70, [1, 2, 4], 3, 12, 2, 8)
    q, _, _, ku, vu = _rand_case(71, 3, 0, 4, 2, 8)
    o, _ = orc.draft_maturev(ck, cv, 2, 1, 4, q, ku, vu)
    np.testing.assert_allclose(o, _sdpa_reference(q, ck[1][2], cv[4][2], ku, vu), atol=1e-10)
    o, _ = orc.verify(ck, cv, 1, 2, q, ku, vu)
    np.testing.assert_allclose(o, _sdpa_reference(q, ck[2][1], cv[2][1], ku, vu), atol=1e-10)
    o, _ = orc.policy_read(ck, cv, 0, 4, 1, q, ku, vu)
    np.testing.assert_allclose(o, _sdpa_reference(q, ck[4][0], cv[1][0], ku, vu), atol=1e-10)
    # draft with d = R is the verifier's read at R
    a, _ = orc.draft_maturev(ck, cv, 1, 4, 4, q, ku, vu)
    b, _ = orc.verify(ck, cv, 1, 4, q, ku, vu)
    np.testing.assert_array_equal(a, b)


def test_commit_append_is_list_append():
    ck, cv = _depth_cache(80, [1, 3], 2, 5, 2, 4)
    nk, nv = _depth_cache(81, [1, 3], 2, 6, 2, 4)
    for n in (0, 1, 6):
        ok, ov = orc.commit_append(ck, cv, nk, nv, n)
        for r in (1, 3):
            for store, new, out in ((ck, nk, ok), (cv, nv, ov)):
                assert out[r].shape == (2, 5 + n, 2, 4)
                np.testing.assert_array_equal(out[r][:, :5], store[r])
                np.testing.assert_array_equal(out[r][:, 5:], new[r][:, :n])
    # empty starting prefix
    e_k = {1: np.zeros((1, 0, 1, 2))}
    n_k = {1: np.arange(6.0).reshape(1, 3, 1, 2)}
    ok, _ = orc.commit_append(e_k, e_k, n_k, n_k, 2)
    np.testing.assert_array_equal(ok[1], n_k[1][:, :2])


def test_wave_widths_eq5():
    # gamma = 32, W_init = 2, J = 24: widths 2..25, never capped.
    ws = orc.wave_widths(32, 2, 24)
    assert ws == list(range(2, 26)) and sum(ws) == 324
    # the cap binds once W_init + j reaches gamma
    assert orc.wave_widths(4, 2, 5) == [2, 3, 4, 4, 4]
    assert orc.wave_widths(8, 8, 3) == [8, 8, 8]


def test_greedy_accept_rules():
    # the paper's illustration: y1, y2 accepted, y3 mismatches -> yhat3 emitted
    acc, emitted = orc.greedy_accept([5, 6, 7, 8], [5, 6, 9, 1])
    assert acc == 2 and emitted == [5, 6, 9]
    # all tested agree and m = w: no bonus (every conditional used)
    acc, emitted = orc.greedy_accept([1, 2, 3], [1, 2, 3])
    assert acc == 3 and emitted == [1, 2, 3]
    # all m < w tested agree: the unused conditional supplies a bonus token
    acc, emitted = orc.greedy_accept([1, 2, 3], [1, 2, 4], tested=2)
    assert acc == 2 and emitted == [1, 2, 4]
    # first proposal rejected
    acc, emitted = orc.greedy_accept([3, 2], [4, 2])
    assert acc == 0 and emitted == [4]
    # retained verifier inputs: the anchor plus accepted inputs among y_1..y_{w-1}
    assert [orc.commit_count(a, 4) for a in range(5)] == [1, 2, 3, 4, 4]


def test_argmax_matches_numpy_first_occurrence():
    """numpy documents argmax / nanargmax as returning the first occurrence of
    the maximum: an independent routine for the lowest-index tie rule."""
    rng = np.random.default_rng(3)
    for _ in range(50):
        v = int(rng.integers(1, 300))
        row = rng.integers(-4, 5, size=v).astype(np.float64)  # many ties
        assert orc.argmax_lowest(row) == int(np.argmax(row))
        row[rng.random(v) < 0.2] = np.nan
        if np.isnan(row).all():
            assert orc.argmax_lowest(row) == 0
        else:
            assert orc.argmax_lowest(row) == int(np.nanargmax(row))


def test_argmax_special_values():
    assert orc.argmax_lowest([0.0, 3.0, 1.0, 3.0]) == 1           # tie -> lowest index
    assert orc.argmax_lowest([-0.0, 0.0, -1.0]) == 0              # signed zeros tie
    assert orc.argmax_lowest([np.nan, -5.0, np.nan]) == 1         # NaN never wins
    assert orc.argmax_lowest([np.nan, np.nan]) == 0               # no candidate: 0
    assert orc.argmax_lowest([-np.inf, -np.inf]) == 0
    assert orc.argmax_lowest([1.0, np.inf, np.inf]) == 1
    # bf16-representable values compare exactly in float64
    bf = torch.tensor([1.0078125, 1.0, 1.0078125], dtype=torch.bfloat16)
    assert orc.argmax_lowest(bf.float().numpy()) == 0


def test_greedy_verify_from_logits():
    """The paper's illustration through the logits: y1, y2 accepted, y3 is the
    first mismatch, yhat3 is emitted, anchor + 2 accepted inputs kept."""
    V = 11
    logits = np.zeros((4, V))
    for i, t in enumerate([5, 6, 9, 1]):
        logits[i, t] = 2.0
    logits[2, 10] = 2.0                       # tie with 9 at row 3: lowest index wins
    pred, acc, emitted, keep = orc.greedy_verify(logits, [5, 6, 7, 8])
    assert pred == [5, 6, 9, 1] and acc == 2 and emitted == [5, 6, 9] and keep == 3
    pred, acc, emitted, keep = orc.greedy_verify(logits, [5, 6, 9, 1])
    assert acc == 4 and emitted == [5, 6, 9, 1] and keep == 4       # m = w: no bonus
    pred, acc, emitted, keep = orc.greedy_verify(logits, [5, 6, 9, 1], tested=3)
    assert acc == 3 and emitted == [5, 6, 9, 1] and keep == 4       # bonus yhat_4
    pred, acc, emitted, keep = orc.greedy_verify(logits, [0, 6, 9, 1], tested=0)
    assert acc == 0 and emitted == [5] and keep == 1                # nothing tested


# ----------------------------------------------------------------------------
# Mutation test: each plausible mistake in the oracle's steps fails a pin.
# ----------------------------------------------------------------------------
def _mutant(mutation):
    def fn(q, kc, vc, ku, vu):
        w, hq, dh = q.shape
        s_len, hkv = kc.shape[0], ku.shape[1]
        group = hq // hkv
        scale = 1.0 / (dh if mutation == "scale_1_over_dh" else math.sqrt(dh))
        vis = np.tril(np.ones((w, w), dtype=bool), k=-1 if mutation == "mask_no_diag" else 0)
        if mutation == "mask_none":
            vis[:] = True
        out = np.zeros((w, hq, dh))
        lse = np.zeros((hq, w))
        pca = np.zeros((hq, w, s_len))
        pua = np.zeros((hq, w, w))
        for h in range(hq):
            g = (h % hkv) if mutation == "gqa_modulo" else h // group
            kk = vc if mutation == "k_from_v_depth" else kc
            vv = kc if mutation == "v_from_k_plane" else vc
            if mutation == "v_reversed":
                vv = vv[::-1]
            sc = (q[:, h] @ kk[:, g].T) * scale
            su = np.where(vis, (q[:, h] @ ku[:, g].T) * scale, -np.inf)
            if mutation == "mask_no_diag":
                su[0, 0] = (q[0, h] @ ku[0, g]) * scale  # keep row 0 defined
            if mutation == "separate_softmax":
                # prefix and block normalised by their own sums
                mu = su.max(1, keepdims=True)
                eu = np.exp(su - mu)
                pu = eu / eu.sum(1, keepdims=True)
                if s_len:
                    mc = sc.max(1, keepdims=True)
                    ec = np.exp(sc - mc)
                    pc = ec / ec.sum(1, keepdims=True)
                else:
                    mc, pc = mu, np.zeros_like(sc)
                m = np.maximum(mc, mu)
                z = np.ones_like(m)
            else:
                m = np.max(np.concatenate([sc, su], 1), 1, keepdims=True)
                ec, eu = np.exp(sc - m), np.exp(su - m)
                z = ec.sum(1, keepdims=True) + eu.sum(1, keepdims=True)
                pc, pu = ec / z, eu / z
            o = pc @ vv[:, g]
            if mutation != "drop_block_term":
                o = o + pu @ vu[:, g]
            out[:, h] = o
            lse[h] = ((m if mutation != "lse_no_max" else 0.0) + np.log(z))[:, 0]
            pca[h], pua[h] = pc, pu
        return out, lse, pca, pua
    return fn


MUTATIONS = ["scale_1_over_dh", "mask_no_diag", "mask_none", "gqa_modulo", "k_from_v_depth",
             "v_from_k_plane", "v_reversed", "separate_softmax", "drop_block_term", "lse_no_max"]


def test_mutant_harness_is_faithful():
    for seed, w, s_len, hq, hkv, dh in [(91, 4, 7, 4, 2, 8), (92, 2, 0, 2, 1, 4)]:
        args = _rand_case(seed, w, s_len, hq, hkv, dh)
        for a, b in zip(_mutant(None)(*args), _oracle_fn(*args)):
            np.testing.assert_allclose(a, b, rtol=0, atol=1e-14)


@pytest.mark.parametrize("mutation", MUTATIONS)
def test_pins_catch_mutation(mutation):
    fn = _mutant(mutation)
    caught = []
    for pin in PINS:
        try:
            with np.errstate(all="ignore"):
                pin(fn)
        except (AssertionError, ValueError, IndexError):
            caught.append(pin.__name__)
    assert caught, f"no pin detects mutation {mutation}"
