"""Out-of-range page ids: both kernel families report DAS_DEVERR_PAGE, read
nothing out of bounds, and return the attention over the remaining
positions (the fp64 oracle with that page's tokens removed)."""

from __future__ import annotations

import numpy as np
import pytest
import torch

from gpu_common import assert_close, oracle_call  # noqa: F401
from gpu_common import wrap
from oracle import das_oracle as orc
from paper_2609_34538_amd import _lib as das
from paper_2609_34538_amd import datagen as dg

pytestmark = pytest.mark.gpu
DEV = "cuda"


def _case(uniform_low_logits: bool):
    wl = dg.scaled(dg.WORKLOADS[3], batch=3, hq=4, hkv=2, layers=1, prefix=(0, 0),
                   paged_random=True)
    cd = dg.make_cache(wl, DEV, prefix_lens=[700, 300, 130])
    if uniform_low_logits:
        # every key = e0 and every query = -1536 e0: all logits equal, about
        # -226 in base-2 units, so a merge that let an empty split's maximum
        # count as 0 would underflow every weight to 0 (and divide 0 by 0)
        cd.k_pool.zero_()
        cd.k_pool[..., 0] = 1.0
    table = cd.block_table.copy()
    bad = {(0, 3): cd.k_pool.shape[3] + 7,    # past the pool
           (0, 4): -5,                         # negative
           (1, 1): cd.k_pool.shape[3]}         # one past the pool
    for (b, p), v in bad.items():
        table[b, p] = v
    return wl, cd, table, bad


def _expected(cd, wl, layer, kappa, nu, q, kb, vb, bad):
    outs = []
    for b in range(wl.batch):
        s_len = int(cd.prefix_lens[b])
        kc = dg.gather_prefix_k(cd, b, cd.k_plane[kappa], layer, s_len)
        vc = dg.gather_prefix_v(cd, b, cd.v_plane[nu], layer, s_len)
        keep = np.ones(s_len, dtype=bool)
        for (bb, p) in bad:
            if bb == b:
                keep[64 * p:64 * (p + 1)] = False
        o, _ = orc.policy_attention(q[b].double().cpu().numpy(), kc[keep], vc[keep],
                                    kb[b].double().cpu().numpy(), vb[b].double().cpu().numpy())
        outs.append(o)
    return np.stack(outs)


@pytest.mark.parametrize("path,pps", [("valu", 1), ("valu", 2), ("mfma", 2), ("mfma", 3),
                                      ("balanced", 0)])
@pytest.mark.parametrize("low", [False, True], ids=["random", "low-logits"])
def test_bad_page_ids_are_skipped_and_reported(path, pps, low):
    wl, cd, table, bad = _case(low)
    err = torch.zeros(1, dtype=torch.int32, device=DEV)
    cache, batch = wrap(cd, table=table, dev_error=err)
    R, d, w = wl.depth_R, 2, 16
    q, kb, vb = dg.block_inputs(cd, w, d, DEV)
    if low:
        q.zero_()
        q[..., 0] = -1536.0
        kb.zero_()
        kb[..., 0] = 1.0
    out = das.attn_policy(cache, batch, 0, d, R, q, kb, vb, path=path, pages_per_split=pps)
    torch.cuda.synchronize()
    assert int(err.item()) & das.DEVERR_PAGE
    ref = _expected(cd, wl, 0, d, R, q, kb, vb, bad)
    assert_close(out, ref, wl.dtype, f"bad pages {path} pps={pps} low={low}")
