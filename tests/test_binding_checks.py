"""The Python binding rejects badly shaped outputs and commit tensors before
calling the library (argument marshalling only; no compute)."""

import numpy as np
import pytest
import torch

# The checks raise before any library call; with a visible GPU the tensors
# below would be host memory passed as device pointers if a check were
# missing, so these run on GPU-less hosts only.
if torch.cuda.device_count() > 0:
    pytest.skip("binding checks run on GPU-less hosts", allow_module_level=True)

das = pytest.importorskip("paper_2609_34538_amd._lib")


def _setup(B=2, w=3, hq=4, hkv=2, dh=64, L=1, pages=4):
    k_pool = torch.zeros((1, L, hkv, pages, 64, dh), dtype=torch.bfloat16)
    v_pool = torch.zeros((1, L, hkv, pages, 8, dh, 8), dtype=torch.bfloat16)
    cache = das.PagedCache(k_pool, v_pool, 4, {4: 0}, {4: 0})
    batch = das.Batch(torch.zeros(B, dtype=torch.int32),
                      torch.zeros((B, 2), dtype=torch.int32))
    q = torch.zeros((B, w, hq, dh), dtype=torch.bfloat16)
    kb = torch.zeros((B, w, hkv, dh), dtype=torch.bfloat16)
    return cache, batch, q, kb, kb.clone()


@pytest.mark.parametrize("bad", ["out_shape", "out_dtype", "out_noncontig", "lse_shape",
                                 "lse_dtype", "lse_noncontig"])
def test_attention_outputs_checked(bad):
    cache, batch, q, kb, vb = _setup()
    B, w, hq, dh = q.shape
    out, lse = None, None
    if bad == "out_shape":
        out = torch.empty((B, w, hq, dh + 1), dtype=q.dtype)
    elif bad == "out_dtype":
        out = torch.empty(q.shape, dtype=torch.float32)
    elif bad == "out_noncontig":
        out = torch.empty((B, w, dh, hq), dtype=q.dtype).transpose(2, 3)
    elif bad == "lse_shape":
        lse = torch.empty((B, w, hq), dtype=torch.float32)  # transposed layout
    elif bad == "lse_dtype":
        lse = torch.empty((B, hq, w), dtype=torch.bfloat16)
    else:
        lse = torch.empty((B, w, hq), dtype=torch.float32).transpose(1, 2)
    ws = torch.empty(1 << 16, dtype=torch.uint8)
    for fn in (lambda: das.attn_policy(cache, batch, 0, 4, 4, q, kb, vb, out=out, lse=lse,
                                       workspace=ws),
               lambda: das.attn_draft_maturev(cache, batch, 0, 4, q, kb, vb, out=out, lse=lse,
                                              workspace=ws),
               lambda: das.attn_verify(cache, batch, 0, 4, q, kb, vb, out=out, lse=lse,
                                       workspace=ws),
               lambda: das.PreparedAttention(cache, batch, 0, 4, 4, q, kb, vb,
                                             out if out is not None else torch.empty_like(q),
                                             ws, lse=lse)):
        with pytest.raises(ValueError):
            fn()


@pytest.mark.parametrize("bad", ["k_ndim", "v_shape", "num_new_shape", "num_new_dtype",
                                 "len_out_shape"])
def test_commit_tensors_checked(bad):
    cache, batch, _, _, _ = _setup()
    B, w_max = batch.batch, 4
    k_new = torch.zeros((1, 1, B, w_max, 2, 64), dtype=torch.bfloat16)
    v_new = torch.zeros((1, 1, B, w_max, 2, 64), dtype=torch.bfloat16)
    num_new = torch.zeros(B, dtype=torch.int32)
    len_out = None
    if bad == "k_ndim":
        k_new = k_new[0]
    elif bad == "v_shape":
        v_new = torch.zeros((1, 1, B, w_max + 1, 2, 64), dtype=torch.bfloat16)
    elif bad == "num_new_shape":
        num_new = torch.zeros(B + 1, dtype=torch.int32)
    elif bad == "num_new_dtype":
        num_new = torch.zeros(B, dtype=torch.int64)
    else:
        len_out = torch.zeros((B, 1), dtype=torch.int32)
    for fn in (lambda: das.kv_append(cache, batch, k_new, v_new, num_new, len_out),
               lambda: das.PreparedAppend(cache, batch, k_new, v_new, num_new, len_out)):
        with pytest.raises(ValueError):
            fn()
