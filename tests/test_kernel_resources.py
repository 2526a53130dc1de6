"""Every kernel of the library runs without scratch memory (register spills
or private arrays would put per-lane memory traffic on the hot path) and
within the per-workgroup LDS of the part. Reads the compiler's resource
report that the build writes."""

import os

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
REPORT = os.path.join(ROOT, "paper_2609_34538_amd", "_build", "kernel_resources.txt")


def _kernels():
    if not os.path.exists(REPORT):
        pytest.skip("library not built here")
    rows = [line.split() for line in open(REPORT).read().splitlines()[1:] if line.strip()]
    return [(r[0], int(r[1]), int(r[2]), int(r[3]), int(r[4])) for r in rows]


def test_report_covers_every_kernel_family():
    names = " ".join(k[0] for k in _kernels())
    for family in ("attn_mfma_kernel", "attn_valu_kernel", "attn_combine_kernel",
                   "kv_append_kernel", "greedy_accept_kernel"):
        assert family in names, family


def test_no_scratch_and_lds_within_limits():
    for name, vgpr, agpr, scratch, lds in _kernels():
        assert scratch == 0, f"{name} uses {scratch} bytes of scratch per lane"
        assert 0 <= lds <= 160 * 1024, f"{name} uses {lds} bytes of LDS"
        assert 0 <= vgpr <= 512 and 0 <= agpr <= 256, name


def test_attention_kernels_keep_accumulators_in_vgprs():
    """The matrix-core kernel is built for two waves per SIMD, which keeps it
    within 256 registers with no AGPRs: above that budget the MFMAs wrote the
    accumulators to AGPRs and every tile copied them back (64 moves per tile
    at head dim 128)."""
    mfma = [k for k in _kernels() if "attn_mfma_kernel" in k[0]]
    assert mfma
    for name, vgpr, agpr, scratch, lds in mfma:
        assert agpr == 0 and vgpr <= 256, f"{name}: {vgpr} VGPRs, {agpr} AGPRs"
