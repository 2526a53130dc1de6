"""Host-side validation of the C ABI: bad arguments are rejected with the
documented status before any HIP call, so nothing is enqueued."""

import ctypes
import os

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))

import torch  # noqa: E402

# The calls below pass fake device pointers and rely on validation failing
# first; on a host with a visible GPU a validation bug could launch a kernel
# on them, so these checks run on GPU-less hosts only (device_count does not
# initialise the GPU).
if torch.cuda.device_count() > 0:
    pytest.skip("host-validation checks run on GPU-less hosts", allow_module_level=True)

lib_mod = pytest.importorskip("paper_2609_34538_amd._lib")
from paper_2609_34538_amd._lib import (DasBatchC, DasCacheC, DasOptionsC, LIB, MAX_DEPTH)  # noqa: E402

OK, NULL, SHAPE, DEPTH, DTYPE, WS, HIP, UNSUP, ALIGN = 0, -1, -2, -3, -4, -5, -6, -7, -8
FAKE = 0x100000  # never dereferenced: every call below fails validation first


def make_cache(dtype=1, R=32, L=4, hkv=8, dh=128, pages=100, kd=(3, 32), vd=(32,)):
    c = DasCacheC()
    c.dtype, c.num_depths, c.num_layers, c.num_kv_heads = dtype, R, L, hkv
    c.head_dim, c.num_pages = dh, pages
    c.num_k_planes, c.num_v_planes = len(kd), len(vd)
    for r in range(MAX_DEPTH + 1):
        c.k_plane[r] = -1
        c.v_plane[r] = -1
    for i, d in enumerate(kd):
        c.k_plane[d] = i
    for i, d in enumerate(vd):
        c.v_plane[d] = i
    c.k_pool = FAKE
    c.v_pool = FAKE
    return c


def make_batch(B=4, maxp=10):
    b = DasBatchC()
    b.batch, b.max_pages_per_seq = B, maxp
    b.prefix_len, b.block_table, b.dev_error = FAKE, FAKE, None
    return b


def ws_bytes(c, b, hq=32, w=8, opts=None):
    if opts is None:
        return LIB.das_attn_workspace_bytes(ctypes.byref(c), ctypes.byref(b), hq, w)
    return LIB.das_attn_workspace_bytes_ex(ctypes.byref(c), ctypes.byref(b), hq, w,
                                           ctypes.byref(opts))


_AUTO = object()


def draft(c, b, layer=0, d=3, hq=32, w=8, q=FAKE, ws=_AUTO, nbytes=None, ptrs=FAKE):
    if ws is _AUTO:
        ws = FAKE
    if nbytes is None:
        nbytes = ws_bytes(c, b, hq, w)
    return LIB.das_attn_draft_maturev(ctypes.byref(c), ctypes.byref(b), layer, d, hq, w, q,
                                      ptrs, ptrs, ptrs, None, ws, nbytes, None)


def test_workspace_size_formula():
    c, b = make_cache(), make_batch()
    n = ws_bytes(c, b)
    assert n > 0 and n % 256 == 0
    # grows with the number of rows and is zero for rejected shapes
    assert ws_bytes(c, b, hq=32, w=16) > n
    assert ws_bytes(c, b, hq=33) == 0
    assert ws_bytes(c, b, w=0) == 0
    assert ws_bytes(c, b, w=65) == 0
    # explicit split size: nsplit = ceil((maxp + 1) / pps) (the first split also
    # takes the draft block and holds one page less)
    o = DasOptionsC()
    o.path, o.pages_per_split = 1, 1
    rows, hkv, B, maxp, dh = 8 * 4, 8, 4, 10, 128
    per = B * hkv * (maxp + 1) * rows
    al = lambda x: (x + 255) // 256 * 256
    # partial O per split and row; m and l per row with the splits padded to 4
    assert ws_bytes(c, b, opts=o) == al(per * dh * 4) + 2 * al(B * hkv * rows * 12 * 4)
    # the matrix-core kernel: a piece record per (sequence, KV head, split) of
    # fp16 outputs and 16 bytes per row, 256-byte aligned
    o.path = 2
    assert ws_bytes(c, b, opts=o) == B * hkv * (maxp + 1) * al(rows * (dh * 2 + 16))


def _nsplit_default(B, hkv, maxp, path=2, hq=None, w=8):
    c, b = make_cache(hkv=hkv), make_batch(B=B, maxp=maxp)
    hq = hkv if hq is None else hq
    o = DasOptionsC()
    o.path, o.pages_per_split = path, 0
    rows = w * (hq // hkv)
    per_split = B * hkv * rows  # rows of one split
    n = ws_bytes(c, b, hq=hq, w=w, opts=o)
    al = lambda x: (x + 255) // 256 * 256
    for ns in range(1, maxp + 2):
        if path == 2:  # one piece record per (sequence, KV head, split)
            size = B * hkv * ns * al(rows * (128 * 2 + 16))
        else:          # fp32 partials; m and l per row with the splits padded to 4
            size = al(per_split * ns * 128 * 4) + 2 * al(per_split * ((ns + 3) // 4 * 4) * 4)
        if size == n:
            return ns
    raise AssertionError("no split count matches the workspace size")


def test_default_split_rule():
    # splits = max(2, pow2 floor of T / (B * Hkv * row tiles)), 2 <= pps <= 32,
    # T = 512, or 2048 for matrix-core blocks of more than 32 rows (their row
    # tiles share a workgroup); split slots = ceil((maxp + 1) / pps)
    assert _nsplit_default(B=16, hkv=8, maxp=200) == 7                # 128 units: pps 32
    assert _nsplit_default(B=4, hkv=8, maxp=257) == 17                # 32 units: pps 16
    assert _nsplit_default(B=4, hkv=8, maxp=257, hq=32, w=32) == 17   # 4 row tiles: pps 16
    assert _nsplit_default(B=4, hkv=8, maxp=257, hq=16, w=32) == 33   # 2 row tiles: pps 8
    assert _nsplit_default(B=1, hkv=55, maxp=33) == 9                 # 55 units: pps 4
    assert _nsplit_default(B=1, hkv=8, maxp=20) == 11                 # pps 2 (minimum)
    # vector-ALU kernel: the same T = 512, and splits of 1..32 pages
    assert _nsplit_default(B=1, hkv=8, maxp=33, path=1) == 34         # 8 units: pps 1
    assert _nsplit_default(B=1, hkv=55, maxp=32, path=1) == 9         # 55 units: pps 4
    assert _nsplit_default(B=16, hkv=8, maxp=200, path=1) == 7        # 128 units: pps 32
    assert _nsplit_default(B=32, hkv=8, maxp=1000) == 32              # pps 32 (maximum)


@pytest.mark.parametrize("field,value,code", [
    ("dtype", 7, DTYPE), ("num_depths", 0, SHAPE), ("num_depths", MAX_DEPTH + 1, SHAPE),
    ("num_layers", 0, SHAPE), ("num_kv_heads", 0, SHAPE), ("head_dim", 80, SHAPE),
    ("num_pages", 0, SHAPE), ("num_k_planes", 0, SHAPE), ("k_pool", None, NULL),
    ("v_pool", None, NULL), ("k_pool", FAKE + 8, ALIGN), ("v_pool", FAKE + 2, ALIGN),
])
def test_bad_cache_rejected(field, value, code):
    c, b = make_cache(), make_batch()
    nbytes = ws_bytes(c, b)
    setattr(c, field, value)
    assert draft(c, b, ws=FAKE, nbytes=nbytes) == code


def test_bad_plane_map_rejected():
    c, b = make_cache(), make_batch()
    c.k_plane[5] = 7  # beyond num_k_planes
    assert draft(c, b, ws=FAKE, nbytes=1 << 30) == SHAPE


@pytest.mark.parametrize("field,value,code", [
    ("batch", 0, SHAPE), ("max_pages_per_seq", 0, SHAPE), ("prefix_len", None, NULL),
    ("max_pages_per_seq", (1 << 24) + 1, SHAPE), ("batch", 1 << 28, SHAPE), ("batch", 65536, SHAPE),
    ("block_table", None, NULL), ("prefix_len", FAKE + 2, ALIGN),
    ("block_table", FAKE + 1, ALIGN), ("dev_error", FAKE + 2, ALIGN),
])
def test_bad_batch_rejected(field, value, code):
    c, b = make_cache(), make_batch()
    nbytes = ws_bytes(c, b)
    setattr(b, field, value)
    assert draft(c, b, ws=FAKE, nbytes=nbytes) == code


def test_attention_argument_checks():
    c, b = make_cache(), make_batch()
    n = ws_bytes(c, b)
    assert draft(c, b, q=None) == NULL
    assert draft(c, b, ptrs=None) == NULL
    assert draft(c, b, layer=4) == SHAPE
    assert draft(c, b, layer=-1) == SHAPE
    assert draft(c, b, d=0, ws=FAKE, nbytes=n) == DEPTH
    assert draft(c, b, d=33, ws=FAKE, nbytes=n) == DEPTH
    assert draft(c, b, d=2, ws=FAKE, nbytes=n) == DEPTH  # K at depth 2 not stored
    assert draft(c, b, hq=36, ws=FAKE, nbytes=n) == SHAPE  # not a multiple of Hkv
    assert draft(c, b, hq=80, ws=FAKE, nbytes=1 << 30) == UNSUP  # group of 10
    assert draft(c, b, w=0, ws=FAKE, nbytes=n) == SHAPE
    assert draft(c, b, w=65, ws=FAKE, nbytes=n) == SHAPE
    assert draft(c, b, ws=None, nbytes=n) == WS
    assert draft(c, b, ws=FAKE, nbytes=n - 1) == WS
    assert draft(c, b, ws=FAKE + 4, nbytes=n) == WS  # not 256-byte aligned
    assert draft(c, b, q=FAKE + 8) == ALIGN  # rows move in 16-byte pieces
    assert draft(c, b, ptrs=FAKE + 4) == ALIGN
    # V at the full depth must be stored for a Mature-V read
    c2 = make_cache(vd=(31,))
    assert draft(c2, b, ws=FAKE, nbytes=n) == DEPTH


def test_verify_and_policy_checks():
    c, b = make_cache(), make_batch()
    n = ws_bytes(c, b)
    v = LIB.das_attn_verify(ctypes.byref(c), ctypes.byref(b), 0, 3, 32, 8, FAKE, FAKE, FAKE,
                            FAKE, None, FAKE, n, None)
    assert v == DEPTH  # V at depth 3 is not stored
    o = DasOptionsC()
    o.path, o.pages_per_split = 2, 0
    f32 = make_cache(dtype=0)
    assert LIB.das_attn_policy(ctypes.byref(f32), ctypes.byref(b), 0, 32, 32, 32, 8, FAKE, FAKE,
                               FAKE, FAKE, None, FAKE, 1 << 30, ctypes.byref(o), None) == UNSUP
    o.path = 9
    assert LIB.das_attn_policy(ctypes.byref(c), ctypes.byref(b), 0, 32, 32, 32, 8, FAKE, FAKE,
                               FAKE, FAKE, None, FAKE, 1 << 30, ctypes.byref(o), None) == SHAPE
    o.path, o.pages_per_split = 0, -1
    assert LIB.das_attn_policy(ctypes.byref(c), ctypes.byref(b), 0, 32, 32, 32, 8, FAKE, FAKE,
                               FAKE, FAKE, None, FAKE, 1 << 30, ctypes.byref(o), None) == SHAPE


def test_append_argument_checks():
    c, b = make_cache(), make_batch()
    app = lambda k=FAKE, v=FAKE, w=32, n=FAKE, lo=None, cc=c, bb=b: LIB.das_kv_append(
        ctypes.byref(cc), ctypes.byref(bb), k, v, w, n, lo, None)
    assert app(k=None) == NULL
    assert app(v=None) == NULL
    assert app(n=None) == NULL
    assert app(w=0) == SHAPE
    assert app(w=65) == SHAPE
    assert app(lo=FAKE) == SHAPE  # len_out aliases prefix_len
    assert app(k=FAKE + 8) == ALIGN
    assert app(v=FAKE + 4) == ALIGN
    assert app(n=FAKE + 2) == ALIGN
    assert app(lo=FAKE + 0x1002) == ALIGN
    bad = make_cache()
    bad.head_dim = 100
    assert app(cc=bad) == SHAPE
    # the commit's grid: 2 key planes + 1 value plane x L layers x 8 heads in
    # workgroups of 4 waves = 6 L workgroups of 256 threads, at most 2^32 - 1
    # work-items; at the limit validation passes (and the launch fails on a
    # GPU-less host), one layer more is rejected
    limit = (0xffffffff // 256) // 6
    big = make_cache()
    big.num_layers = limit
    assert app(cc=big) == HIP
    big.num_layers = limit + 1
    assert app(cc=big) == SHAPE
    big.num_layers = 1 << 26
    assert app(cc=big) == SHAPE
    nb = make_batch()
    nb.block_table = None
    assert app(bb=nb) == NULL


def test_greedy_accept_argument_checks():
    def acc(B=4, w=8, y=FAKE, yhat=FAKE, m=None, a=FAKE, keep=FAKE, em=None, nem=None, err=None):
        return LIB.das_greedy_accept(B, w, y, yhat, m, a, keep, em, nem, err, None)
    assert acc(y=None) == NULL
    assert acc(yhat=None) == NULL
    assert acc(a=None) == NULL
    assert acc(keep=None) == NULL
    assert acc(B=0) == SHAPE
    assert acc(w=0) == SHAPE
    assert acc(w=65) == SHAPE
    assert acc(y=FAKE + 2) == ALIGN
    assert acc(m=FAKE + 1) == ALIGN
    assert acc(em=FAKE + 2) == ALIGN
    assert acc(err=FAKE + 3) == ALIGN


def test_attention_grid_limits():
    # matrix-core path, 8 query rows (one single-wave workgroup per chunk):
    # 8 KV heads x nsplit chunks x 64 threads <= 2^32 - 1, nsplit = (maxp + 2) / 2
    # at 2 pages per split
    o = DasOptionsC()
    o.path, o.pages_per_split = 2, 2
    c = make_cache(hkv=8)
    at = make_batch(B=1, maxp=2 * 8388607 - 2)
    past = make_batch(B=1, maxp=2 * 8388608 - 2)
    assert ws_bytes(c, at, hq=8, w=8, opts=o) > 0
    assert ws_bytes(c, past, hq=8, w=8, opts=o) == 0
    # vector-ALU path: the split count x 256 threads along x
    o.path, o.pages_per_split = 1, 1
    at = make_batch(B=1, maxp=(0xffffffff // 256) - 1)
    past = make_batch(B=1, maxp=(0xffffffff // 256))
    assert ws_bytes(c, at, hq=8, w=8, opts=o) > 0
    assert ws_bytes(c, past, hq=8, w=8, opts=o) == 0
    # KV heads: at most 65535
    assert ws_bytes(make_cache(hkv=65535), make_batch(B=1, maxp=4), hq=65535, w=1) > 0
    assert ws_bytes(make_cache(hkv=65536), make_batch(B=1, maxp=4), hq=65536, w=1) == 0


def test_balanced_schedule_workspace_and_limits():
    # pieces = sequences x KV heads + workers (256 CUs x 512 / head_dim
    # single-wave workgroups: 5 at head dim 96, 4 at 128)
    o = DasOptionsC()
    o.path, o.pages_per_split = 3, 0
    al = lambda x: (x + 255) // 256 * 256
    c, b = make_cache(hkv=8, dh=96), make_batch(B=4, maxp=10)
    rows = 16 * 2  # w 16, G 2
    # a piece record per piece (fp16 outputs + 16 bytes per row, 256-byte
    # aligned), plus a {first piece, piece count} record per (sequence, KV head)
    pieces = 4 * 8 + 256 * 5
    rec = al(4 * 8 * 8)
    assert ws_bytes(c, b, hq=16, w=16, opts=o) == pieces * al(rows * (96 * 2 + 16)) + rec
    c128 = make_cache(hkv=8, dh=128)
    pieces = 4 * 8 + 256 * 4
    assert ws_bytes(c128, b, hq=8, w=16, opts=o) == pieces * al(16 * (128 * 2 + 16)) + rec
    # odd row counts: records stay 256-byte aligned
    assert ws_bytes(c, b, hq=8, w=3, opts=o) == (4 * 8 + 256 * 5) * al(3 * (96 * 2 + 16)) + rec
    # limits: 64 sequences, 32 query rows (16 at head dim 128)
    assert ws_bytes(c, make_batch(B=64, maxp=10), hq=8, w=32, opts=o) > 0
    assert ws_bytes(c, make_batch(B=65, maxp=10), hq=8, w=32, opts=o) == 0
    assert ws_bytes(c, b, hq=8, w=33, opts=o) == 0
    assert ws_bytes(c128, b, hq=8, w=17, opts=o) == 0
    # library choice: the balanced schedule for 2..64 sequences with more
    # than W / 8 (sequence, KV head) units (W = 1280 workers at head dim 96,
    # 1024 at 128), the split grid otherwise (its workspace is sized per split)
    o.path = 0
    for B, path in ((21, 3), (20, 2), (4, 2), (1, 2)):
        bb = make_batch(B=B, maxp=10)
        assert ws_bytes(c, bb, hq=16, w=16, opts=o) == ws_bytes(c, bb, hq=16, w=16, opts=_opts(path)), B
    for B, path in ((17, 3), (16, 2)):
        bb = make_batch(B=B, maxp=10)
        assert ws_bytes(c128, bb, hq=8, w=16, opts=o) == ws_bytes(c128, bb, hq=8, w=16, opts=_opts(path)), B
    c64 = make_cache(hkv=8, dh=64)  # 1792 workers: more than 224 units
    for B, path in ((29, 3), (28, 2)):
        bb = make_batch(B=B, maxp=10)
        assert ws_bytes(c64, bb, hq=16, w=16, opts=o) == ws_bytes(c64, bb, hq=16, w=16, opts=_opts(path)), B
    o.pages_per_split = 4
    big = make_batch(B=21, maxp=10)
    assert ws_bytes(c, big, hq=16, w=16, opts=o) == ws_bytes(c, big, hq=16, w=16, opts=_opts(2, 4))
    # fp32 caches have no balanced schedule
    assert ws_bytes(make_cache(dtype=0), b, opts=_opts(3)) == 0


def _opts(path, pps=0):
    o = DasOptionsC()
    o.path, o.pages_per_split = path, pps
    return o
