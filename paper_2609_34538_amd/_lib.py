"""ctypes binding of libdas.so (include/das.h).

Argument marshalling only: tensors are checked for device, dtype, shape and
contiguity, their device pointers and the current HIP stream are passed to
the C ABI, and a non-zero status raises DasError. Every computation runs in
the library's HIP kernels; there is no fallback. Importing this module
without a built library raises, so a missing extension fails loudly.
"""

from __future__ import annotations

import ctypes
import os
from ctypes import POINTER, c_char_p, c_int32, c_size_t, c_uint32, c_void_p
from dataclasses import dataclass, field
from typing import Dict, Optional

import torch

_HERE = os.path.dirname(os.path.abspath(__file__))
# DAS_LIBRARY may point at another build of the same library.
LIB_PATH = os.environ.get("DAS_LIBRARY") or os.path.join(_HERE, "libdas.so")

MAX_DEPTH = 64
PAGE_TOKENS = 64
MAX_BLOCK = 64
NOALLOC_SCRATCH_BYTES = 64 << 20  # DAS_NOALLOC_SCRATCH_BYTES

DAS_OK = 0
STATUS_NAMES = {0: "DAS_OK", -1: "DAS_ERR_NULL", -2: "DAS_ERR_SHAPE", -3: "DAS_ERR_DEPTH",
                -4: "DAS_ERR_DTYPE", -5: "DAS_ERR_WORKSPACE", -6: "DAS_ERR_HIP",
                -7: "DAS_ERR_UNSUPPORTED", -8: "DAS_ERR_ALIGN"}
DTYPE_CODES = {torch.float32: 0, torch.bfloat16: 1}
PATHS = {"auto": 0, "valu": 1, "mfma": 2, "balanced": 3}
DEVERR_PAGE, DEVERR_PREFIX, DEVERR_COMMIT, DEVERR_TESTED = 1, 2, 4, 8

EXPORTED = ["das_attn_workspace_bytes", "das_attn_workspace_bytes_ex", "das_attn_draft_maturev",
            "das_attn_verify", "das_attn_policy", "das_attn_policy_noalloc", "das_kv_append",
            "das_greedy_accept",
            "das_status_string", "das_version"]


class DasError(RuntimeError):
    def __init__(self, status: int, what: str):
        self.status = status
        super().__init__(f"{what}: {STATUS_NAMES.get(status, status)} ({status_string(status)})")


class DasCacheC(ctypes.Structure):
    _fields_ = [("dtype", c_int32), ("num_depths", c_int32), ("num_layers", c_int32),
                ("num_kv_heads", c_int32), ("head_dim", c_int32), ("num_pages", c_int32),
                ("num_k_planes", c_int32), ("num_v_planes", c_int32),
                ("k_plane", c_int32 * (MAX_DEPTH + 1)), ("v_plane", c_int32 * (MAX_DEPTH + 1)),
                ("k_pool", c_void_p), ("v_pool", c_void_p)]


class DasBatchC(ctypes.Structure):
    _fields_ = [("batch", c_int32), ("max_pages_per_seq", c_int32), ("prefix_len", c_void_p),
                ("block_table", c_void_p), ("dev_error", c_void_p)]


class DasOptionsC(ctypes.Structure):
    _fields_ = [("path", c_int32), ("pages_per_split", c_int32)]


def _load() -> ctypes.CDLL:
    if not os.path.exists(LIB_PATH):
        raise ImportError(f"libdas.so not built at {LIB_PATH}; run python -m paper_2609_34538_amd.build")
    lib = ctypes.CDLL(LIB_PATH)
    pc, pb, po = POINTER(DasCacheC), POINTER(DasBatchC), POINTER(DasOptionsC)
    attn_args = [pc, pb, c_int32, c_int32, c_int32, c_int32, c_void_p, c_void_p, c_void_p,
                 c_void_p, c_void_p, c_void_p, c_size_t, c_void_p]
    lib.das_attn_workspace_bytes.argtypes = [pc, pb, c_int32, c_int32]
    lib.das_attn_workspace_bytes.restype = c_size_t
    lib.das_attn_workspace_bytes_ex.argtypes = [pc, pb, c_int32, c_int32, po]
    lib.das_attn_workspace_bytes_ex.restype = c_size_t
    lib.das_attn_draft_maturev.argtypes = attn_args
    lib.das_attn_draft_maturev.restype = c_int32
    lib.das_attn_verify.argtypes = attn_args
    lib.das_attn_verify.restype = c_int32
    lib.das_attn_policy.argtypes = [pc, pb, c_int32, c_int32, c_int32, c_int32, c_int32,
                                    c_void_p, c_void_p, c_void_p, c_void_p, c_void_p, c_void_p,
                                    c_size_t, po, c_void_p]
    lib.das_attn_policy.restype = c_int32
    lib.das_attn_policy_noalloc.argtypes = [pc, pb, c_int32, c_int32, c_int32, c_int32,
                                            c_int32, c_void_p, c_void_p, c_void_p, c_void_p,
                                            c_void_p, po, c_void_p]
    lib.das_attn_policy_noalloc.restype = c_int32
    lib.das_kv_append.argtypes = [pc, pb, c_void_p, c_void_p, c_int32, c_void_p, c_void_p,
                                  c_void_p]
    lib.das_kv_append.restype = c_int32
    lib.das_greedy_accept.argtypes = [c_int32, c_int32] + [c_void_p] * 8 + [c_void_p]
    lib.das_greedy_accept.restype = c_int32
    lib.das_status_string.argtypes = [c_int32]
    lib.das_status_string.restype = c_char_p
    lib.das_version.argtypes = []
    lib.das_version.restype = c_int32
    return lib


LIB = _load()


def status_string(status: int) -> str:
    return LIB.das_status_string(status).decode()


def _ptr(t: Optional[torch.Tensor]) -> Optional[int]:
    return None if t is None else t.data_ptr()


def _stream_handle(stream) -> int:
    if stream is None:
        stream = torch.cuda.current_stream()
    return stream.cuda_stream


@dataclass
class PagedCache:
    """Caller-owned depth-indexed paged cache (layouts as in das.h).

    k_pool: [nK, L, Hkv, P, 64, dh]; v_pool: [nV, L, Hkv, P, 8, dh, 8].
    k_plane / v_plane map a depth r (1..R) to its plane index."""
    k_pool: torch.Tensor
    v_pool: torch.Tensor
    num_depths: int
    k_plane: Dict[int, int]
    v_plane: Dict[int, int]
    _c: DasCacheC = field(default=None, repr=False)

    def __post_init__(self):
        self.refresh()

    @property
    def num_layers(self):
        return self.k_pool.shape[1]

    @property
    def num_kv_heads(self):
        return self.k_pool.shape[2]

    @property
    def num_pages(self):
        return self.k_pool.shape[3]

    @property
    def head_dim(self):
        return self.k_pool.shape[5]

    @property
    def dtype(self):
        return self.k_pool.dtype

    def refresh(self):
        k, v = self.k_pool, self.v_pool
        if k.dim() != 6 or v.dim() != 7:
            raise ValueError("k_pool must be 6-d and v_pool 7-d")
        if k.shape[4] != PAGE_TOKENS or v.shape[4] * v.shape[6] != PAGE_TOKENS or v.shape[6] != 8:
            raise ValueError("pages hold 64 tokens (values in 8 groups of 8)")
        if k.shape[1:4] != v.shape[1:4] or k.shape[5] != v.shape[5] or k.dtype != v.dtype:
            raise ValueError("k_pool / v_pool disagree")
        if not (k.is_contiguous() and v.is_contiguous()):
            raise ValueError("pools must be contiguous")
        c = DasCacheC()
        c.dtype = DTYPE_CODES[k.dtype]
        c.num_depths = self.num_depths
        c.num_layers, c.num_kv_heads, c.num_pages = k.shape[1], k.shape[2], k.shape[3]
        c.head_dim = k.shape[5]
        c.num_k_planes, c.num_v_planes = k.shape[0], v.shape[0]
        for r in range(MAX_DEPTH + 1):
            c.k_plane[r] = self.k_plane.get(r, -1)
            c.v_plane[r] = self.v_plane.get(r, -1)
        c.k_pool, c.v_pool = k.data_ptr(), v.data_ptr()
        self._c = c
        return self

    @property
    def c(self) -> DasCacheC:
        return self._c


@dataclass
class Batch:
    """prefix_len [B] int32, block_table [B, max_pages] int32 (device), and an
    optional device error word."""
    prefix_len: torch.Tensor
    block_table: torch.Tensor
    dev_error: Optional[torch.Tensor] = None
    _c: DasBatchC = field(default=None, repr=False)

    def __post_init__(self):
        self.refresh()

    def refresh(self):
        pl, bt = self.prefix_len, self.block_table
        if pl.dtype != torch.int32 or bt.dtype != torch.int32:
            raise ValueError("prefix_len and block_table are int32")
        if bt.dim() != 2 or pl.shape != (bt.shape[0],):
            raise ValueError("block_table must be [B, max_pages] and prefix_len [B]")
        if not (pl.is_contiguous() and bt.is_contiguous()):
            raise ValueError("batch arrays must be contiguous")
        c = DasBatchC()
        c.batch, c.max_pages_per_seq = bt.shape
        c.prefix_len, c.block_table = pl.data_ptr(), bt.data_ptr()
        c.dev_error = _ptr(self.dev_error)
        self._c = c
        return self

    @property
    def batch(self):
        return self.block_table.shape[0]

    @property
    def c(self) -> DasBatchC:
        return self._c


def _options(path: str, pages_per_split: int):
    o = DasOptionsC()
    o.path = PATHS[path]
    o.pages_per_split = pages_per_split
    return o


def workspace_bytes(cache: PagedCache, batch: Batch, num_q_heads: int, block_len: int,
                    path: str = "auto", pages_per_split: int = 0) -> int:
    o = _options(path, pages_per_split)
    return LIB.das_attn_workspace_bytes_ex(ctypes.byref(cache.c), ctypes.byref(batch.c),
                                           num_q_heads, block_len, ctypes.byref(o))


def alloc_workspace(cache: PagedCache, batch: Batch, num_q_heads: int, block_len: int,
                    path: str = "auto", pages_per_split: int = 0) -> torch.Tensor:
    n = workspace_bytes(cache, batch, num_q_heads, block_len, path, pages_per_split)
    if n == 0:
        raise DasError(-2, "workspace query rejected the shapes")
    return torch.empty(n, dtype=torch.uint8, device=cache.k_pool.device)


def _check_block(cache: PagedCache, batch: Batch, q, k_blk, v_blk):
    B, w, hq, dh = q.shape
    if B != batch.batch or dh != cache.head_dim:
        raise ValueError("q must be [B, w, Hq, dh]")
    want = (B, w, cache.num_kv_heads, dh)
    for t in (q, k_blk, v_blk):
        if t.dtype != cache.dtype or not t.is_contiguous() or t.device != cache.k_pool.device:
            raise ValueError("block tensors must be contiguous, on the cache's device and dtype")
    if tuple(k_blk.shape) != want or tuple(v_blk.shape) != want:
        raise ValueError("k_blk / v_blk must be [B, w, Hkv, dh]")
    return w, hq


def _check_outputs(cache: PagedCache, batch: Batch, q, out, lse):
    """out: same shape, dtype and device as q, contiguous; lse: contiguous
    fp32 [B, Hq, w] on the cache's device."""
    if out is not None:
        if (out.shape != q.shape or out.dtype != q.dtype or not out.is_contiguous()
                or out.device != cache.k_pool.device):
            raise ValueError("out must be a contiguous tensor shaped and typed like q")
    if lse is not None:
        B, w, hq, _ = q.shape
        if (lse.dtype != torch.float32 or tuple(lse.shape) != (B, hq, w)
                or not lse.is_contiguous() or lse.device != cache.k_pool.device):
            raise ValueError("lse must be a contiguous float32 tensor [B, Hq, w] on the "
                             "cache's device")


def attn_policy(cache: PagedCache, batch: Batch, layer: int, kappa: int, nu: int,
                q: torch.Tensor, k_blk: torch.Tensor, v_blk: torch.Tensor,
                out: Optional[torch.Tensor] = None, lse: Optional[torch.Tensor] = None,
                workspace: Optional[torch.Tensor] = None, path: str = "auto",
                pages_per_split: int = 0, stream=None) -> torch.Tensor:
    """Eq. (2)-(3) with prefix keys at depth kappa and values at depth nu."""
    w, hq = _check_block(cache, batch, q, k_blk, v_blk)
    _check_outputs(cache, batch, q, out, lse)
    if out is None:
        out = torch.empty_like(q)
    if workspace is None:
        workspace = alloc_workspace(cache, batch, hq, w, path, pages_per_split)
    o = _options(path, pages_per_split)
    st = LIB.das_attn_policy(ctypes.byref(cache.c), ctypes.byref(batch.c), layer, kappa, nu,
                             hq, w, q.data_ptr(), k_blk.data_ptr(), v_blk.data_ptr(),
                             out.data_ptr(), _ptr(lse), workspace.data_ptr(),
                             workspace.numel(), ctypes.byref(o), _stream_handle(stream))
    if st != DAS_OK:
        raise DasError(st, "das_attn_policy")
    return out


def attn_policy_noalloc(cache: PagedCache, batch: Batch, layer: int, kappa: int, nu: int,
                        q: torch.Tensor, k_blk: torch.Tensor, v_blk: torch.Tensor,
                        out: torch.Tensor, lse: Optional[torch.Tensor] = None,
                        path: str = "auto", pages_per_split: int = 0, stream=None) -> torch.Tensor:
    """attn_policy without a workspace: the split partials go to the
    library's fixed per-GPU scratch (das_attn_policy_noalloc). `out` must be
    given, so the call allocates nothing."""
    _check_block(cache, batch, q, k_blk, v_blk)
    if out is None:
        raise ValueError("out is required (the call allocates nothing)")
    _check_outputs(cache, batch, q, out, lse)
    o = _options(path, pages_per_split)
    w, hq = q.shape[1], q.shape[2]
    st = LIB.das_attn_policy_noalloc(ctypes.byref(cache.c), ctypes.byref(batch.c), layer, kappa,
                                     nu, hq, w, q.data_ptr(), k_blk.data_ptr(), v_blk.data_ptr(),
                                     out.data_ptr(), _ptr(lse), ctypes.byref(o),
                                     _stream_handle(stream))
    if st != DAS_OK:
        raise DasError(st, "das_attn_policy_noalloc")
    return out


class PreparedAttention:
    """One attention call with every argument marshalled up front, for loops
    that issue the same call many times (the device buffers it names must
    stay alive). Calling it enqueues the call on the stream captured here."""

    def __init__(self, cache: PagedCache, batch: Batch, layer: int, kappa: int, nu: int,
                 q: torch.Tensor, k_blk: torch.Tensor, v_blk: torch.Tensor,
                 out: torch.Tensor, workspace: torch.Tensor, lse: Optional[torch.Tensor] = None,
                 path: str = "auto", pages_per_split: int = 0, stream=None):
        w, hq = _check_block(cache, batch, q, k_blk, v_blk)
        _check_outputs(cache, batch, q, out, lse)
        self._keep = (cache, batch, q, k_blk, v_blk, out, workspace, lse)
        self._opts = _options(path, pages_per_split)
        self._fn = LIB.das_attn_policy
        self._args = (ctypes.byref(cache.c), ctypes.byref(batch.c), layer, kappa, nu, hq, w,
                      q.data_ptr(), k_blk.data_ptr(), v_blk.data_ptr(), out.data_ptr(),
                      _ptr(lse), workspace.data_ptr(), workspace.numel(),
                      ctypes.byref(self._opts), _stream_handle(stream))

    def __call__(self):
        st = self._fn(*self._args)
        if st != DAS_OK:
            raise DasError(st, "das_attn_policy")


class PreparedAppend:
    """A commit call with its arguments marshalled up front."""

    def __init__(self, cache: PagedCache, batch: Batch, k_new: torch.Tensor, v_new: torch.Tensor,
                 num_new: torch.Tensor, len_out: Optional[torch.Tensor] = None, stream=None):
        w_max = _check_append(cache, batch, k_new, v_new, num_new, len_out)
        self._keep = (cache, batch, k_new, v_new, num_new, len_out)
        self._fn = LIB.das_kv_append
        self._args = (ctypes.byref(cache.c), ctypes.byref(batch.c), k_new.data_ptr(),
                      v_new.data_ptr(), w_max, num_new.data_ptr(), _ptr(len_out),
                      _stream_handle(stream))

    def __call__(self):
        st = self._fn(*self._args)
        if st != DAS_OK:
            raise DasError(st, "das_kv_append")


def attn_draft_maturev(cache: PagedCache, batch: Batch, layer: int, draft_depth: int,
                       q, k_blk, v_blk, out=None, lse=None, workspace=None, stream=None):
    """Mature-V draft read: keys at draft_depth, values at the full depth R."""
    w, hq = _check_block(cache, batch, q, k_blk, v_blk)
    _check_outputs(cache, batch, q, out, lse)
    if out is None:
        out = torch.empty_like(q)
    if workspace is None:
        workspace = alloc_workspace(cache, batch, hq, w)
    st = LIB.das_attn_draft_maturev(ctypes.byref(cache.c), ctypes.byref(batch.c), layer,
                                    draft_depth, hq, w, q.data_ptr(), k_blk.data_ptr(),
                                    v_blk.data_ptr(), out.data_ptr(), _ptr(lse),
                                    workspace.data_ptr(), workspace.numel(),
                                    _stream_handle(stream))
    if st != DAS_OK:
        raise DasError(st, "das_attn_draft_maturev")
    return out


def attn_verify(cache: PagedCache, batch: Batch, layer: int, depth: int, q, k_blk, v_blk,
                out=None, lse=None, workspace=None, stream=None):
    """The target's aligned read at `depth` (the full-depth verifier at R)."""
    w, hq = _check_block(cache, batch, q, k_blk, v_blk)
    _check_outputs(cache, batch, q, out, lse)
    if out is None:
        out = torch.empty_like(q)
    if workspace is None:
        workspace = alloc_workspace(cache, batch, hq, w)
    st = LIB.das_attn_verify(ctypes.byref(cache.c), ctypes.byref(batch.c), layer, depth, hq,
                             w, q.data_ptr(), k_blk.data_ptr(), v_blk.data_ptr(),
                             out.data_ptr(), _ptr(lse), workspace.data_ptr(),
                             workspace.numel(), _stream_handle(stream))
    if st != DAS_OK:
        raise DasError(st, "das_attn_verify")
    return out


def _check_append(cache: PagedCache, batch: Batch, k_new, v_new, num_new, len_out) -> int:
    """Shapes of a commit's tensors; returns w_max."""
    if k_new.dim() != 6:
        raise ValueError("k_new must be [nK, L, B, w_max, Hkv, dh]")
    nk, L, B, w_max, hkv, dh = k_new.shape
    if (nk, L, B, hkv, dh) != (cache.k_pool.shape[0], cache.num_layers, batch.batch,
                               cache.num_kv_heads, cache.head_dim):
        raise ValueError("k_new must be [nK, L, B, w_max, Hkv, dh]")
    if tuple(v_new.shape) != (cache.v_pool.shape[0], L, B, w_max, hkv, dh):
        raise ValueError("v_new must be [nV, L, B, w_max, Hkv, dh]")
    for t in (k_new, v_new):
        if (t.dtype != cache.dtype or not t.is_contiguous()
                or t.device != cache.k_pool.device):
            raise ValueError("k_new / v_new must be contiguous in the cache dtype and device")
    if num_new.dtype != torch.int32 or tuple(num_new.shape) != (B,) or not num_new.is_contiguous():
        raise ValueError("num_new must be a contiguous int32 tensor [B]")
    if len_out is not None and (len_out.dtype != torch.int32 or tuple(len_out.shape) != (B,)
                                or not len_out.is_contiguous()):
        raise ValueError("len_out must be a contiguous int32 tensor [B]")
    return w_max


def kv_append(cache: PagedCache, batch: Batch, k_new: torch.Tensor, v_new: torch.Tensor,
              num_new: torch.Tensor, len_out: Optional[torch.Tensor] = None, stream=None):
    """Commit the first num_new[b] block entries of every plane and layer."""
    w_max = _check_append(cache, batch, k_new, v_new, num_new, len_out)
    st = LIB.das_kv_append(ctypes.byref(cache.c), ctypes.byref(batch.c), k_new.data_ptr(),
                           v_new.data_ptr(), w_max, num_new.data_ptr(), _ptr(len_out),
                           _stream_handle(stream))
    if st != DAS_OK:
        raise DasError(st, "das_kv_append")


def _i32(t: Optional[torch.Tensor], shape, what: str):
    if t is None:
        return None
    if t.dtype != torch.int32 or tuple(t.shape) != tuple(shape) or not t.is_contiguous():
        raise ValueError(f"{what} must be a contiguous int32 tensor of shape {tuple(shape)}")
    return t.data_ptr()


def greedy_accept(proposals: torch.Tensor, target_pred: torch.Tensor,
                  tested: Optional[torch.Tensor] = None, accepted: Optional[torch.Tensor] = None,
                  num_keep: Optional[torch.Tensor] = None, emitted: Optional[torch.Tensor] = None,
                  num_emitted: Optional[torch.Tensor] = None,
                  dev_error: Optional[torch.Tensor] = None, stream=None):
    """Greedy verification of a block on the device (Sec. 3.4). Returns
    (accepted, num_keep); num_keep is das_kv_append's num_new."""
    B, w = proposals.shape
    if accepted is None:
        accepted = torch.empty(B, dtype=torch.int32, device=proposals.device)
    if num_keep is None:
        num_keep = torch.empty(B, dtype=torch.int32, device=proposals.device)
    args = (_i32(proposals, (B, w), "proposals"), _i32(target_pred, (B, w), "target_pred"),
            _i32(tested, (B,), "tested"), _i32(accepted, (B,), "accepted"),
            _i32(num_keep, (B,), "num_keep"), _i32(emitted, (B, w), "emitted"),
            _i32(num_emitted, (B,), "num_emitted"), _ptr(dev_error))
    st = LIB.das_greedy_accept(B, w, *args, _stream_handle(stream))
    if st != DAS_OK:
        raise DasError(st, "das_greedy_accept")
    return accepted, num_keep
