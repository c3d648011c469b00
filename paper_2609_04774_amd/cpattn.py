"""ctypes binding of libcpattn (include/cp_attn.h): argument marshalling only.

Every computation happens in the library's host code and HIP kernels; this
module only turns torch tensors into device pointers, Python ints into C
integers and non-zero statuses into exceptions.  Importing it fails loudly if
the library has not been built (``python -m paper_2609_04774_amd.build``).
"""

from __future__ import annotations

import ctypes
import math
import os
from typing import Optional, Sequence

PKG_DIR = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(PKG_DIR, "libcpattn.so")

CP_OK = 0
CP_ERR_INVALID = -1
CP_ERR_UNSUPPORTED = -2
CP_ERR_HIP = -3
CP_ERR_CAPACITY = -4
CP_ERR_HOST = -5
CP_HEAD_DIM = 128
CP_KV_BLOCK_TOKENS = 16
CP_MAX_MERGE_PARTS = 16
CP_KV_ALL = -1
CP_KV_NONE = -2
CP_OUT_LOCAL = 0
CP_OUT_SEQUENCE = 1
CP_MAX_DEGREE = 64
CP_NOALLOC_SCRATCH_BYTES = 32 << 20

EXPORTED = ("cp_status_string", "cp_last_error", "cp_shard_plan", "cp_shard_inverse",
            "cp_attn_partial_workspace_size", "cp_attn_partial", "cp_set_workgroup_rows",
            "cp_attn_partial_noalloc", "cp_attn_merge",
            "cp_kv_writeback", "cp_repartition", "cp_repartition_all", "cp_kv_gather")


class CpChunk(ctypes.Structure):
    _fields_ = [("chunk_id", ctypes.c_int32), ("reserved", ctypes.c_int32),
                ("q_begin", ctypes.c_int64), ("q_len", ctypes.c_int64),
                ("local_offset", ctypes.c_int64)]


class CpRankPlan(ctypes.Structure):
    _fields_ = [("C", ctypes.c_int32), ("rank", ctypes.c_int32),
                ("prefix_len", ctypes.c_int64), ("new_len", ctypes.c_int64),
                ("padded_len", ctypes.c_int64), ("chunk_len", ctypes.c_int64),
                ("n_rows", ctypes.c_int64), ("chunk", CpChunk * 2),
                ("visible_pairs", ctypes.c_int64)]

    def as_dict(self) -> dict:
        return {
            "C": self.C, "rank": self.rank, "prefix_len": self.prefix_len,
            "new_len": self.new_len, "padded_len": self.padded_len,
            "chunk_len": self.chunk_len, "n_rows": self.n_rows,
            "chunks": [(c.chunk_id, c.q_begin, c.q_len, c.local_offset) for c in self.chunk],
            "visible_pairs": self.visible_pairs,
        }


class CpPartialDesc(ctypes.Structure):
    _fields_ = [("plan", CpRankPlan),
                ("q", ctypes.c_void_p), ("k_new", ctypes.c_void_p), ("v_new", ctypes.c_void_p),
                ("k_cache", ctypes.c_void_p), ("v_cache", ctypes.c_void_p),
                ("block_table", ctypes.c_void_p),
                ("include_prefix", ctypes.c_int32), ("kv_rank", ctypes.c_int32),
                ("o", ctypes.c_void_p), ("lse", ctypes.c_void_p),
                ("n_blocks", ctypes.c_int64),
                ("out_order", ctypes.c_int32), ("reserved", ctypes.c_int32)]


class CpError(RuntimeError):
    def __init__(self, status: int, detail: str):
        super().__init__(f"{detail} [status {status}]")
        self.status = status


def _load():
    if not os.path.exists(LIB_PATH):
        raise ImportError(f"{LIB_PATH} is missing: build it with `python -m paper_2609_04774_amd.build`")
    # torch ships its own HIP runtime (same soname).  Loading torch first makes
    # libcpattn bind to that already-loaded runtime, so the process has one
    # HIP runtime and torch's streams and allocations are valid in the library.
    import torch  # noqa: F401
    lib = ctypes.CDLL(LIB_PATH)
    lib.cp_status_string.restype = ctypes.c_char_p
    lib.cp_status_string.argtypes = [ctypes.c_int]
    lib.cp_last_error.restype = ctypes.c_char_p
    lib.cp_last_error.argtypes = []
    lib.cp_shard_plan.restype = ctypes.c_int
    lib.cp_shard_plan.argtypes = [ctypes.c_int64, ctypes.c_int64, ctypes.c_int32, ctypes.c_int32,
                                  ctypes.POINTER(CpRankPlan), ctypes.c_void_p, ctypes.c_int64]
    lib.cp_shard_inverse.restype = ctypes.c_int
    lib.cp_shard_inverse.argtypes = [ctypes.c_int64, ctypes.c_int64, ctypes.c_int32,
                                     ctypes.c_void_p, ctypes.c_void_p, ctypes.c_int64]
    lib.cp_attn_partial_workspace_size.restype = ctypes.c_size_t
    lib.cp_attn_partial_workspace_size.argtypes = [ctypes.POINTER(CpPartialDesc), ctypes.c_int32,
                                                   ctypes.c_int32, ctypes.c_int32]
    lib.cp_attn_partial.restype = ctypes.c_int
    lib.cp_attn_partial.argtypes = [ctypes.POINTER(CpPartialDesc), ctypes.c_int32, ctypes.c_int32,
                                    ctypes.c_int32, ctypes.c_int32, ctypes.c_float,
                                    ctypes.c_void_p, ctypes.c_size_t, ctypes.c_void_p]
    lib.cp_set_workgroup_rows.restype = ctypes.c_int
    lib.cp_set_workgroup_rows.argtypes = [ctypes.c_int32]
    lib.cp_attn_partial_noalloc.restype = ctypes.c_int
    lib.cp_attn_partial_noalloc.argtypes = [ctypes.POINTER(CpPartialDesc), ctypes.c_int32, ctypes.c_int32,
                                            ctypes.c_int32, ctypes.c_int32, ctypes.c_float, ctypes.c_void_p]
    lib.cp_attn_merge.restype = ctypes.c_int
    lib.cp_attn_merge.argtypes = [ctypes.c_int32, ctypes.POINTER(ctypes.c_void_p),
                                  ctypes.POINTER(ctypes.c_void_p), ctypes.c_int64, ctypes.c_int32,
                                  ctypes.c_int32, ctypes.c_void_p, ctypes.c_int32, ctypes.c_void_p,
                                  ctypes.POINTER(CpRankPlan), ctypes.c_void_p]
    lib.cp_kv_writeback.restype = ctypes.c_int
    lib.cp_kv_writeback.argtypes = [ctypes.POINTER(CpRankPlan), ctypes.c_void_p, ctypes.c_void_p,
                                    ctypes.c_int32, ctypes.c_int32, ctypes.c_void_p, ctypes.c_void_p,
                                    ctypes.c_int64, ctypes.c_void_p, ctypes.c_int64, ctypes.c_void_p]
    lib.cp_repartition.restype = ctypes.c_int
    lib.cp_repartition.argtypes = [ctypes.c_int64, ctypes.c_int64, ctypes.c_int32,
                                   ctypes.POINTER(ctypes.c_void_p), ctypes.c_int32, ctypes.c_int32,
                                   ctypes.c_void_p, ctypes.c_int64, ctypes.c_void_p]
    lib.cp_repartition_all.restype = ctypes.c_int
    lib.cp_repartition_all.argtypes = [ctypes.c_int64, ctypes.c_int64, ctypes.c_int32,
                                       ctypes.POINTER(ctypes.c_void_p), ctypes.c_int32,
                                       ctypes.POINTER(ctypes.c_void_p), ctypes.c_int32, ctypes.c_int64,
                                       ctypes.c_void_p]
    lib.cp_kv_gather.restype = ctypes.c_int
    lib.cp_kv_gather.argtypes = [ctypes.c_void_p, ctypes.c_void_p, ctypes.c_int64, ctypes.c_void_p,
                                 ctypes.c_int64, ctypes.c_int64, ctypes.c_int64, ctypes.c_int32,
                                 ctypes.c_int32, ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p]
    return lib


lib = _load()


def _check(status: int):
    if status != CP_OK:
        raise CpError(status, lib.cp_last_error().decode() or lib.cp_status_string(status).decode())


def status_string(status: int) -> str:
    return lib.cp_status_string(status).decode()


def last_error() -> str:
    return lib.cp_last_error().decode()


# --- plan ---------------------------------------------------------------------

def shard_plan(prefix_len: int, new_len: int, C: int, rank: int, with_rows: bool = True):
    """cp_shard_plan: (CpRankPlan, row_pos as a list of ints or None)."""
    import numpy as np
    plan = CpRankPlan()
    _check(lib.cp_shard_plan(prefix_len, new_len, C, rank, ctypes.byref(plan), None, 0))
    if not with_rows:
        return plan, None
    rows = np.zeros(max(1, plan.n_rows), dtype=np.int64)
    _check(lib.cp_shard_plan(prefix_len, new_len, C, rank, ctypes.byref(plan),
                             rows.ctypes.data_as(ctypes.c_void_p), plan.n_rows))
    return plan, rows[: plan.n_rows]


def shard_inverse(prefix_len: int, new_len: int, C: int):
    """cp_shard_inverse: (rank_of int32[R], row_of int64[R]) as numpy arrays."""
    import numpy as np
    rank_of = np.zeros(max(1, new_len), dtype=np.int32)
    row_of = np.zeros(max(1, new_len), dtype=np.int64)
    _check(lib.cp_shard_inverse(prefix_len, new_len, C, rank_of.ctypes.data_as(ctypes.c_void_p),
                                row_of.ctypes.data_as(ctypes.c_void_p), new_len))
    return rank_of[:new_len], row_of[:new_len]


# --- partial attention ----------------------------------------------------------

def _ptr(t) -> Optional[int]:
    if t is None:
        return None
    return t.data_ptr()


def _dev(t, name: str, dtype=None, rows: Optional[int] = None, tail=None):
    """Checks that a tensor argument is what the C ABI will read or write
    through its pointer: a contiguous GPU tensor of the right element type,
    with at least ``rows`` entries along its first dimension and, if given,
    trailing dimensions ``tail``.  The library sees only the pointer, so a
    tensor that is too small or of another type would be read or written out
    of bounds; these checks turn that into an exception."""
    if t is None:
        return
    if not t.is_cuda:
        raise ValueError(f"{name} must be a GPU tensor")
    if dtype is not None and t.dtype != dtype:
        raise TypeError(f"{name} must be {dtype}, got {t.dtype}")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    if rows is not None and (t.dim() == 0 or t.shape[0] < rows):
        raise ValueError(f"{name} needs at least {rows} rows, has shape {tuple(t.shape)}")
    if tail is not None and tuple(t.shape[1:]) != tuple(tail):
        raise ValueError(f"{name} must have shape [*, {', '.join(map(str, tail))}], has {tuple(t.shape)}")


def make_desc(plan: CpRankPlan, q, k_new, v_new, o, lse, k_cache=None, v_cache=None,
              block_table=None, include_prefix: bool = True, kv_rank: int = CP_KV_ALL,
              out_order: int = CP_OUT_LOCAL) -> CpPartialDesc:
    """A cp_partial_desc over torch device tensors (layouts in include/cp_attn.h).
    With out_order=CP_OUT_SEQUENCE, o and lse have R rows in the original
    suffix order and only this rank's rows are written.  The tensors' head
    counts are checked against n_heads_q / n_heads_kv when the descriptor is
    launched.  The descriptor keeps references to its tensors; keep it until
    the launch has been issued."""
    import torch
    D = CP_HEAD_DIM
    if out_order not in (CP_OUT_LOCAL, CP_OUT_SEQUENCE):
        raise ValueError("out_order must be CP_OUT_LOCAL or CP_OUT_SEQUENCE")
    out_rows = plan.new_len if out_order == CP_OUT_SEQUENCE else plan.n_rows
    _dev(q, "q", torch.bfloat16, plan.n_rows)
    _dev(o, "o", torch.float32, out_rows)
    _dev(lse, "lse", torch.float32, out_rows)
    _dev(k_new, "k_new", torch.bfloat16, plan.new_len)
    _dev(v_new, "v_new", torch.bfloat16, plan.new_len)
    _dev(k_cache, "k_cache", torch.bfloat16)
    _dev(v_cache, "v_cache", torch.bfloat16)
    _dev(block_table, "block_table", torch.int32)
    if include_prefix and plan.prefix_len > 0 and block_table is not None:
        if block_table.numel() < -(-plan.prefix_len // CP_KV_BLOCK_TOKENS):
            raise ValueError("block_table shorter than ceil(P / 16)")
    for name, t in (("q", q), ("o", o), ("k_new", k_new), ("v_new", v_new)):
        if t is not None and (t.dim() != 3 or t.shape[2] != D):
            raise ValueError(f"{name} must have shape [rows, heads, {D}], has {tuple(t.shape)}")
    for name, t in (("k_cache", k_cache), ("v_cache", v_cache)):
        if t is not None and (t.dim() != 4 or t.shape[1] != CP_KV_BLOCK_TOKENS or t.shape[3] != D):
            raise ValueError(f"{name} must have shape [blocks, 16, heads, {D}], has {tuple(t.shape)}")
    if k_cache is not None and v_cache is not None and k_cache.shape[0] != v_cache.shape[0]:
        raise ValueError("k_cache and v_cache differ in blocks")
    d = CpPartialDesc()
    d.plan = plan
    d.q = _ptr(q)
    d.k_new = _ptr(k_new)
    d.v_new = _ptr(v_new)
    d.k_cache = _ptr(k_cache)
    d.v_cache = _ptr(v_cache)
    d.block_table = _ptr(block_table)
    d.include_prefix = 1 if include_prefix else 0
    d.kv_rank = kv_rank
    d.o = _ptr(o)
    d.lse = _ptr(lse)
    d.n_blocks = k_cache.shape[0] if k_cache is not None else 0
    d.out_order = out_order
    d.reserved = 0
    d._heads = (q, o, lse, k_new, v_new, k_cache, v_cache)
    # The descriptor holds only device pointers: keep every tensor it points
    # at alive for as long as the descriptor exists, so that a caller that
    # drops its own reference (say to a block table built per request) before
    # the launch cannot leave the kernel reading freed, reused memory.
    d._keep = (q, k_new, v_new, k_cache, v_cache, block_table, o, lse)
    return d


def _check_heads(descs, n_heads_q: int, n_heads_kv: int):
    for i, d in enumerate(descs):
        held = getattr(d, "_heads", None)
        if held is None:
            continue
        q, o, lse, k_new, v_new, k_cache, v_cache = held
        for name, t, h in (("q", q, n_heads_q), ("o", o, n_heads_q), ("k_new", k_new, n_heads_kv),
                           ("v_new", v_new, n_heads_kv)):
            if t is not None and t.shape[1] != h:
                raise ValueError(f"desc {i}: {name} has {t.shape[1]} heads, expected {h}")
        if lse is not None and (lse.dim() != 2 or lse.shape[1] != n_heads_q):
            raise ValueError(f"desc {i}: lse must have shape [rows, {n_heads_q}], has {tuple(lse.shape)}")
        for name, t in (("k_cache", k_cache), ("v_cache", v_cache)):
            if t is not None and t.shape[2] != n_heads_kv:
                raise ValueError(f"desc {i}: {name} has {t.shape[2]} heads, expected {n_heads_kv}")


def _desc_array(descs: Sequence[CpPartialDesc]):
    arr = (CpPartialDesc * max(1, len(descs)))()
    for i, d in enumerate(descs):
        arr[i] = d
    return arr


def workspace_size(descs: Sequence[CpPartialDesc], n_heads_q: int, n_heads_kv: int) -> int:
    arr = _desc_array(descs)
    n = lib.cp_attn_partial_workspace_size(arr, len(descs), n_heads_q, n_heads_kv)
    if n == 0 and descs and last_error():
        raise CpError(CP_ERR_INVALID, last_error())
    return n


def _stream_handle(stream) -> Optional[int]:
    import torch
    if stream is None:
        stream = torch.cuda.current_stream()
    return stream.cuda_stream


def attn_partial(descs: Sequence[CpPartialDesc], n_heads_q: int, n_heads_kv: int, workspace,
                 head_dim: int = CP_HEAD_DIM, softmax_scale: float = 0.0, stream=None,
                 workspace_bytes: Optional[int] = None):
    """cp_attn_partial on the given (or current torch) stream.

    ``workspace`` is a torch uint8 device tensor of at least
    ``workspace_size(descs, ...)`` bytes.
    """
    _check_heads(descs, n_heads_q, n_heads_kv)
    _dev(workspace, "workspace")
    arr = _desc_array(descs)
    nbytes = workspace.numel() * workspace.element_size() if workspace_bytes is None else workspace_bytes
    _check(lib.cp_attn_partial(arr, len(descs), n_heads_q, n_heads_kv, head_dim,
                               float(softmax_scale), _ptr(workspace), nbytes,
                               _stream_handle(stream)))


def set_workgroup_rows(rows: int) -> None:
    """cp_set_workgroup_rows: 0 lets each launch choose its workgroup size
    (256 or 384 rows); 256 or 384 pins it for the process."""
    _check(lib.cp_set_workgroup_rows(int(rows)))


def attn_partial_noalloc(descs: Sequence[CpPartialDesc], n_heads_q: int, n_heads_kv: int,
                         head_dim: int = CP_HEAD_DIM, softmax_scale: float = 0.0, stream=None):
    """cp_attn_partial_noalloc on the given (or current torch) stream: no
    workspace; the library's own device scratch serves the launch."""
    _check_heads(descs, n_heads_q, n_heads_kv)
    arr = _desc_array(descs)
    _check(lib.cp_attn_partial_noalloc(arr, len(descs), n_heads_q, n_heads_kv, head_dim,
                                       float(softmax_scale), _stream_handle(stream)))


def attn_merge(o_parts, lse_parts, o_out, lse_out=None, restore: Optional[CpRankPlan] = None,
               n_tokens: Optional[int] = None, n_heads: Optional[int] = None,
               head_dim: int = CP_HEAD_DIM, stream=None):
    """cp_attn_merge of torch device tensors; bf16 output when o_out is bf16."""
    import torch
    n = len(o_parts)
    if len(lse_parts) != n:
        raise ValueError("o_parts and lse_parts differ in length")
    rows = o_parts[0].shape[0] if n_tokens is None else n_tokens
    heads = o_parts[0].shape[1] if n_heads is None else n_heads
    for i in range(n):
        _dev(o_parts[i], f"o_parts[{i}]", torch.float32, rows)
        _dev(lse_parts[i], f"lse_parts[{i}]", torch.float32, rows)
        if o_parts[i].numel() < rows * heads * head_dim or lse_parts[i].numel() < rows * heads:
            raise ValueError(f"partial {i} holds fewer than {rows} x {heads} rows")
    out_rows = restore.new_len if restore is not None else rows
    _dev(o_out, "o_out", None, out_rows)
    if o_out.dtype not in (torch.float32, torch.bfloat16):
        raise TypeError("o_out must be float32 or bfloat16")
    _dev(lse_out, "lse_out", torch.float32, out_rows)
    if o_out.numel() < out_rows * heads * head_dim or (lse_out is not None and lse_out.numel() < out_rows * heads):
        raise ValueError(f"outputs hold fewer than {out_rows} x {heads} rows")
    optrs = (ctypes.c_void_p * max(1, n))(*[_ptr(o) for o in o_parts])
    lptrs = (ctypes.c_void_p * max(1, n))(*[_ptr(s) for s in lse_parts])
    if n_tokens is None:
        n_tokens = o_parts[0].shape[0]
    if n_heads is None:
        n_heads = o_parts[0].shape[1]
    out_bf16 = 1 if o_out.dtype == torch.bfloat16 else 0
    _check(lib.cp_attn_merge(n, optrs, lptrs, n_tokens, n_heads, head_dim, _ptr(o_out), out_bf16,
                             _ptr(lse_out), ctypes.byref(restore) if restore is not None else None,
                             _stream_handle(stream)))


def default_scale(head_dim: int = CP_HEAD_DIM) -> float:
    return 1.0 / math.sqrt(head_dim)


def kv_writeback(plan: CpRankPlan, k_rows, v_rows, k_cache, v_cache, block_table, stream=None):
    """cp_kv_writeback of torch device tensors: the rank's rows [n_rows, Hkv, D]
    (plan order) into caches [n_blocks, 16, Hkv, D] through block_table."""
    import torch
    n_blocks, _, Hkv, D = k_cache.shape
    for name, t in (("k_cache", k_cache), ("v_cache", v_cache)):
        _dev(t, name, torch.bfloat16, None, (CP_KV_BLOCK_TOKENS, Hkv, D))
    if v_cache.shape[0] != n_blocks:
        raise ValueError("k_cache and v_cache differ in blocks")
    _dev(k_rows, "k_rows", torch.bfloat16, plan.n_rows, (Hkv, D))
    _dev(v_rows, "v_rows", torch.bfloat16, plan.n_rows, (Hkv, D))
    _dev(block_table, "block_table", torch.int32)
    _check(lib.cp_kv_writeback(ctypes.byref(plan), _ptr(k_rows), _ptr(v_rows), Hkv, D, _ptr(k_cache),
                               _ptr(v_cache), n_blocks, _ptr(block_table), block_table.numel(),
                               _stream_handle(stream)))


def kv_gather(k_cache, v_cache, block_table, pos_begin: int, k_rows, v_rows, stream=None):
    """cp_kv_gather of torch device tensors: positions pos_begin ..
    pos_begin + len(k_rows) - 1 out of caches [n_blocks, 16, Hkv, D] through
    block_table into k_rows, v_rows [n, Hkv, D]."""
    import torch
    n_blocks, _, Hkv, D = k_cache.shape
    for name, t in (("k_cache", k_cache), ("v_cache", v_cache)):
        _dev(t, name, torch.bfloat16, None, (CP_KV_BLOCK_TOKENS, Hkv, D))
    if v_cache.shape[0] != n_blocks:
        raise ValueError("k_cache and v_cache differ in blocks")
    _dev(k_rows, "k_rows", torch.bfloat16, None, (Hkv, D))
    _dev(v_rows, "v_rows", torch.bfloat16, k_rows.shape[0], (Hkv, D))
    _dev(block_table, "block_table", torch.int32)
    _check(lib.cp_kv_gather(_ptr(k_cache), _ptr(v_cache), n_blocks, _ptr(block_table), block_table.numel(),
                            pos_begin, k_rows.shape[0], Hkv, D, _ptr(k_rows), _ptr(v_rows),
                            _stream_handle(stream)))


def repartition(prefix_len: int, new_len: int, src_rows, C_dst: int, dst_rank: int, dst_rows, stream=None):
    """cp_repartition of torch device tensors: src_rows is the list of the C_src
    ranks' row tensors (plan order); dst_rows receives rank dst_rank's rows at
    degree C_dst.  A row is everything after a tensor's first dimension."""
    C_src = len(src_rows)
    dst_plan, _ = shard_plan(prefix_len, new_len, C_dst, dst_rank, with_rows=False)
    _dev(dst_rows, "dst_rows", None, dst_plan.n_rows)
    for r, t in enumerate(src_rows):
        src_plan, _ = shard_plan(prefix_len, new_len, C_src, r, with_rows=False)
        _dev(t, f"src_rows[{r}]", dst_rows.dtype, src_plan.n_rows, tuple(dst_rows.shape[1:]))
    ptrs = (ctypes.c_void_p * max(1, C_src))(*[_ptr(t) if t.numel() else None for t in src_rows])
    row_bytes = math.prod(dst_rows.shape[1:]) * dst_rows.element_size()
    _check(lib.cp_repartition(prefix_len, new_len, C_src, ptrs, C_dst, dst_rank, _ptr(dst_rows), row_bytes,
                              _stream_handle(stream)))


def repartition_all(prefix_len: int, new_len: int, src_sets, dst_sets, stream=None):
    """cp_repartition_all of torch device tensors: src_sets[k] is the list of
    the C_src ranks' row tensors of set k (plan order), dst_sets[k] the list of
    the C_dst destination ranks' tensors it fills -- every destination rank of
    up to two sets (K and V) in one launch."""
    n_sets = len(src_sets)
    if n_sets != len(dst_sets) or n_sets not in (1, 2):
        raise ValueError("src_sets and dst_sets must both hold 1 or 2 sets")
    C_src, C_dst = len(src_sets[0]), len(dst_sets[0])
    ref = dst_sets[0][0]
    for k in range(n_sets):
        if len(src_sets[k]) != C_src or len(dst_sets[k]) != C_dst:
            raise ValueError("every set needs C_src sources and C_dst destinations")
        for r, t in enumerate(src_sets[k]):
            pl, _ = shard_plan(prefix_len, new_len, C_src, r, with_rows=False)
            _dev(t, f"src_sets[{k}][{r}]", ref.dtype, pl.n_rows, tuple(ref.shape[1:]))
        for r, t in enumerate(dst_sets[k]):
            pl, _ = shard_plan(prefix_len, new_len, C_dst, r, with_rows=False)
            _dev(t, f"dst_sets[{k}][{r}]", ref.dtype, pl.n_rows, tuple(ref.shape[1:]))
    srcs = (ctypes.c_void_p * (n_sets * C_src))(*[_ptr(t) if t.numel() else None for st in src_sets for t in st])
    dsts = (ctypes.c_void_p * (n_sets * C_dst))(*[_ptr(t) if t.numel() else None for st in dst_sets for t in st])
    row_bytes = math.prod(ref.shape[1:]) * ref.element_size()
    _check(lib.cp_repartition_all(prefix_len, new_len, C_src, srcs, C_dst, dsts, n_sets, row_bytes,
                                  _stream_handle(stream)))
