"""C-ABI checks that need no GPU: exports, plan parity, argument errors.

Every error case here fails host-side validation, which runs before any HIP
call, so nothing touches a device.
"""

import ctypes
import os
import re

import numpy as np
import pytest

from oracle import plan as oplan
from paper_2609_04774_amd import cpattn as cp

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "cp_attn.h")


def _declared_functions():
    with open(HEADER) as f:
        text = f.read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(cp_[a-z_]+)\s*\(", text)))


def test_every_declared_symbol_is_exported():
    declared = _declared_functions()
    assert set(declared) == set(cp.EXPORTED)
    for name in declared:
        assert hasattr(cp.lib, name), name


def _comment_before_each_function():
    """{function: the comment block that precedes its declaration}."""
    with open(HEADER) as f:
        text = f.read()
    out = {}
    for name in _declared_functions():
        m = re.search(r"\n(?!\s*/?\*)[^\n]*\b" + name + r"\s*\(", text)
        assert m, name
        head = text[:m.start()]
        end = head.rstrip().rfind("*/")
        # Only a typedef may sit between the comment and the declaration.
        between = head[end + 2:]
        assert not between.strip() or between.strip().startswith("typedef"), name
        start = head.rfind("/*", 0, end)
        out[name] = " ".join(head[start + 2:end].replace("*", " ").split())
    return out


def test_every_declared_function_names_its_source():
    """Each entry point's comment cites the paper section it implements, or
    says that it is a library utility outside the paper; the variant without
    allocation names the callers it is for instead."""
    comments = _comment_before_each_function()
    assert set(comments) == set(cp.EXPORTED)
    for name, c in comments.items():
        if name == "cp_attn_partial_noalloc":
            assert "callers that cannot allocate" in c, name
            continue
        assert re.search(r"Sec\. \d", c) or "not from the paper" in c, name


def test_status_strings():
    for st in (cp.CP_OK, cp.CP_ERR_INVALID, cp.CP_ERR_UNSUPPORTED, cp.CP_ERR_HIP, cp.CP_ERR_CAPACITY,
               cp.CP_ERR_HOST):
        assert cp.status_string(st) and cp.status_string(st) != "unknown status"
    assert cp.status_string(12345) == "unknown status"


def test_struct_layout_matches_header():
    # 4+4 + 5*8 + 2*(4+4+3*8) + 8 bytes
    assert ctypes.sizeof(cp.CpChunk) == 32
    assert ctypes.sizeof(cp.CpRankPlan) == 8 + 5 * 8 + 2 * 32 + 8
    assert ctypes.sizeof(cp.CpPartialDesc) == ctypes.sizeof(cp.CpRankPlan) + 6 * 8 + 8 + 2 * 8 + 8 + 8


PLAN_SWEEP = [(P, R, C) for P in (0, 16, 48, 49152) for R in (0, 1, 3, 7, 16, 100, 1024, 1000)
              for C in (1, 2, 3, 4, 8)]


@pytest.mark.parametrize("P,R,C", PLAN_SWEEP)
def test_plan_bit_exact_vs_oracle(P, R, C):
    for r in range(C):
        got, rows = cp.shard_plan(P, R, C, r)
        ref = oplan.shard_plan_fast(P, R, C, r) if R > 64 else oplan.shard_plan(P, R, C, r)
        d = got.as_dict()
        for key in ("C", "rank", "prefix_len", "new_len", "padded_len", "chunk_len", "n_rows",
                    "visible_pairs"):
            assert d[key] == ref[key], key
        assert [tuple(c) for c in d["chunks"]] == [tuple(c) for c in ref["chunks"]]
        assert rows.tolist() == ref["row_pos"]


@pytest.mark.parametrize("P,R,C", [(0, 32768, 4), (49152, 16384, 2), (0, 131072, 8), (0, 1024, 2)])
def test_plan_full_size_configs(P, R, C):
    total = 0
    for r in range(C):
        got, rows = cp.shard_plan(P, R, C, r)
        ref = oplan.shard_plan_fast(P, R, C, r)
        assert got.visible_pairs == ref["visible_pairs"]
        assert rows.tolist() == ref["row_pos"]
        total += got.visible_pairs
    assert total == oplan.remaining_workload(R, P)


@pytest.mark.parametrize("P,R,C", [(0, 1024, 2), (16, 37, 8), (0, 3, 4), (32, 100, 3), (0, 0, 2)])
def test_inverse_bit_exact_vs_oracle(P, R, C):
    rank_of, row_of = cp.shard_inverse(P, R, C)
    ref_rank, ref_row = oplan.inverse_map(P, R, C)
    assert rank_of.tolist() == ref_rank
    assert row_of.tolist() == ref_row


def _status(fn, *args):
    return fn(*args)


def test_plan_errors():
    plan = cp.CpRankPlan()
    assert cp.lib.cp_shard_plan(0, 10, 0, 0, ctypes.byref(plan), None, 0) == cp.CP_ERR_INVALID
    assert "C must be" in cp.last_error()
    assert cp.lib.cp_shard_plan(0, 10, 2, 2, ctypes.byref(plan), None, 0) == cp.CP_ERR_INVALID
    assert cp.lib.cp_shard_plan(0, 10, 2, -1, ctypes.byref(plan), None, 0) == cp.CP_ERR_INVALID
    assert cp.lib.cp_shard_plan(-1, 10, 2, 0, ctypes.byref(plan), None, 0) == cp.CP_ERR_INVALID
    assert cp.lib.cp_shard_plan(0, -1, 2, 0, ctypes.byref(plan), None, 0) == cp.CP_ERR_INVALID
    assert cp.lib.cp_shard_plan(0, 10, 2, 0, None, None, 0) == cp.CP_ERR_INVALID
    rows = np.zeros(2, dtype=np.int64)
    assert cp.lib.cp_shard_plan(0, 10, 2, 0, ctypes.byref(plan),
                                rows.ctypes.data_as(ctypes.c_void_p), 2) == cp.CP_ERR_CAPACITY
    a = np.zeros(4, dtype=np.int32)
    b = np.zeros(4, dtype=np.int64)
    assert cp.lib.cp_shard_inverse(0, 10, 2, a.ctypes.data_as(ctypes.c_void_p),
                                   b.ctypes.data_as(ctypes.c_void_p), 4) == cp.CP_ERR_CAPACITY
    assert cp.lib.cp_shard_inverse(0, 10, 2, None, None, 10) == cp.CP_ERR_INVALID
    # A successful call clears the error detail.
    assert cp.lib.cp_shard_plan(0, 10, 2, 0, ctypes.byref(plan), None, 0) == cp.CP_OK
    assert cp.last_error() == ""


def test_plan_degree_limit():
    """C up to CP_MAX_DEGREE is planned (chunk 2C-1-rank exact); beyond it
    every call that takes a degree refuses, instead of wrapping the chunk id."""
    plan = cp.CpRankPlan()
    top = cp.CP_MAX_DEGREE
    assert cp.lib.cp_shard_plan(100, 5 * top, top, 0, ctypes.byref(plan), None, 0) == cp.CP_OK
    assert plan.chunk[1].chunk_id == 2 * top - 1 and plan.chunk[1].q_begin == 100 + (2 * top - 1) * 3
    for C in (top + 1, 2 ** 31 - 1):
        assert cp.lib.cp_shard_plan(100, 5, C, 0, ctypes.byref(plan), None, 0) == cp.CP_ERR_INVALID
        assert "CP_MAX_DEGREE" in cp.last_error()
        a = np.zeros(8, dtype=np.int32)
        b = np.zeros(8, dtype=np.int64)
        assert cp.lib.cp_shard_inverse(100, 5, C, a.ctypes.data_as(ctypes.c_void_p),
                                       b.ctypes.data_as(ctypes.c_void_p), 8) == cp.CP_ERR_INVALID
    # A plan claiming a degree beyond the limit is refused by the merge's restore.
    bad = cp.CpRankPlan()
    bad.C, bad.rank, bad.prefix_len, bad.new_len = 2 ** 31 - 1, 0, 100, 5
    optrs = (ctypes.c_void_p * 1)(FAKE)
    lptrs = (ctypes.c_void_p * 1)(FAKE)
    assert cp.lib.cp_attn_merge(1, optrs, lptrs, 0, 8, 128, FAKE, 0, None, ctypes.byref(bad), None) == \
        cp.CP_ERR_INVALID


def test_plan_length_limit_keeps_visible_pairs_exact():
    """Up to 2^31 cached and 2^31 new tokens the pair count W(R, P) =
    RP + R(R+1)/2 (Sec. 2.2) is exact in 64 bits; longer inputs are refused
    rather than wrapped."""
    plan = cp.CpRankPlan()
    big = 1 << 31
    assert cp.lib.cp_shard_plan(big + 1, 10, 2, 0, ctypes.byref(plan), None, 0) == cp.CP_ERR_INVALID
    assert cp.lib.cp_shard_plan(0, big + 1, 2, 0, ctypes.byref(plan), None, 0) == cp.CP_ERR_INVALID
    assert cp.lib.cp_shard_plan(big, big, 1, 0, ctypes.byref(plan), None, 0) == cp.CP_OK
    assert plan.visible_pairs == big * big + big * (big + 1) // 2
    total = 0
    for r in range(4):
        assert cp.lib.cp_shard_plan(big, big, 4, r, ctypes.byref(plan), None, 0) == cp.CP_OK
        total += plan.visible_pairs
    assert total == big * big + big * (big + 1) // 2


FAKE = 1 << 20          # aligned addresses that are never dereferenced


def _desc(P=0, R=64, C=2, rank=0, **kw):
    plan, _ = cp.shard_plan(P, R, C, rank, with_rows=False)
    d = cp.CpPartialDesc()
    d.plan = plan
    d.q = kw.get("q", FAKE)
    d.k_new = kw.get("k_new", FAKE * 2)
    d.v_new = kw.get("v_new", FAKE * 3)
    d.k_cache = kw.get("k_cache", FAKE * 4)
    d.v_cache = kw.get("v_cache", FAKE * 5)
    d.block_table = kw.get("block_table", FAKE * 6)
    d.include_prefix = kw.get("include_prefix", 1)
    d.kv_rank = kw.get("kv_rank", cp.CP_KV_ALL)
    d.o = kw.get("o", FAKE * 7)
    d.lse = kw.get("lse", FAKE * 8)
    d.n_blocks = kw.get("n_blocks", 8)
    d.out_order = kw.get("out_order", cp.CP_OUT_LOCAL)
    d.reserved = kw.get("reserved", 0)
    return d


def _partial_status(descs, Hq=8, Hkv=2, D=128, ws=FAKE * 16, ws_bytes=1 << 30):
    arr = (cp.CpPartialDesc * max(1, len(descs)))(*descs)
    return cp.lib.cp_attn_partial(arr, len(descs), Hq, Hkv, D, 0.0, ws, ws_bytes, None)


@pytest.mark.parametrize("case,kw,args,status", [
    ("head_dim 64", {}, {"D": 64}, cp.CP_ERR_UNSUPPORTED),
    ("Hq not multiple of Hkv", {}, {"Hq": 6, "Hkv": 4}, cp.CP_ERR_INVALID),
    ("zero heads", {}, {"Hq": 0}, cp.CP_ERR_INVALID),
    ("kv_rank >= C", {"kv_rank": 2}, {}, cp.CP_ERR_INVALID),
    ("kv_rank < -2", {"kv_rank": -3}, {}, cp.CP_ERR_INVALID),
    ("prefix not block multiple", {"P": 40}, {}, cp.CP_ERR_INVALID),
    ("null q", {"q": None}, {}, cp.CP_ERR_INVALID),
    ("null o", {"o": None}, {}, cp.CP_ERR_INVALID),
    ("null k_new", {"k_new": None}, {}, cp.CP_ERR_INVALID),
    ("null block table with prefix", {"P": 32, "block_table": None}, {}, cp.CP_ERR_INVALID),
    ("no cache blocks with prefix", {"P": 32, "n_blocks": 0}, {}, cp.CP_ERR_INVALID),
    ("misaligned q", {"q": FAKE + 2}, {}, cp.CP_ERR_INVALID),
    ("misaligned k_cache", {"P": 32, "k_cache": FAKE + 8}, {}, cp.CP_ERR_INVALID),
    ("include_prefix 2", {"include_prefix": 2}, {}, cp.CP_ERR_INVALID),
    ("out_order 2", {"out_order": 2}, {}, cp.CP_ERR_INVALID),
    ("out_order -1", {"out_order": -1}, {}, cp.CP_ERR_INVALID),
    ("reserved not 0", {"reserved": 1}, {}, cp.CP_ERR_INVALID),
    ("workspace too small", {}, {"ws_bytes": 16}, cp.CP_ERR_CAPACITY),
    ("workspace null", {}, {"ws": None}, cp.CP_ERR_INVALID),
    ("workspace misaligned", {}, {"ws": FAKE + 64}, cp.CP_ERR_INVALID),
    ("sequence beyond 2^30 tokens", {"P": 1 << 30, "R": 64}, {}, cp.CP_ERR_UNSUPPORTED),
])
def test_partial_argument_errors(case, kw, args, status):
    P = kw.pop("P", 0)
    R = kw.pop("R", 64)
    d = _desc(P=P, R=R, **kw)
    assert _partial_status([d], **args) == status, case
    assert cp.last_error() != ""


def test_partial_rejects_a_tampered_plan():
    d = _desc()
    d.plan.n_rows += 1
    assert _partial_status([d]) == cp.CP_ERR_INVALID
    d = _desc()
    d.plan.chunk[1].q_begin += 1
    assert _partial_status([d]) == cp.CP_ERR_INVALID


def test_partial_prefix_pointers_optional_when_unused():
    # Prefix not read: the cache pointers may be NULL; the call then fails only
    # on the (deliberately tiny) workspace, i.e. after every descriptor check.
    d = _desc(P=40, include_prefix=0, k_cache=None, v_cache=None, block_table=None)
    assert _partial_status([d], ws_bytes=16) == cp.CP_ERR_CAPACITY
    d = _desc(kv_rank=cp.CP_KV_NONE, k_new=None, v_new=None, include_prefix=0)
    assert _partial_status([d], ws_bytes=16) == cp.CP_ERR_CAPACITY


def test_partial_empty_work_is_a_no_op():
    assert _partial_status([]) == cp.CP_OK
    # A rank with no rows (R < 2C) launches nothing either.
    d = _desc(R=3, C=4, rank=3, q=None, o=None, lse=None)
    assert d.plan.n_rows == 0
    assert _partial_status([d], ws=None, ws_bytes=0) == cp.CP_OK


def test_workspace_size_grows_with_work():
    small = cp.workspace_size([_desc(R=64)], 8, 2)
    big = cp.workspace_size([_desc(R=4096)], 8, 2)
    assert 0 < small < big
    bad = _desc(kv_rank=5)
    with pytest.raises(cp.CpError):
        cp.workspace_size([bad], 8, 2)


def _piece(rows):
    return rows * 128 * 4 + rows * 4


def test_workspace_holds_piece_slots_for_split_walks():
    """Few query rows over a long cached prefix: the launch has few work items,
    so each item's key walk is split into pieces and the workspace grows by
    one slot (fp32 O and LSE of the workgroup's rows) per piece.  A launch
    whose long items do not fill the 256 compute units evenly has some of
    them cut to balance the schedule; one with many small items is never
    split."""
    try:
        for rows in (256, 384):
            cp.set_workgroup_rows(rows)
            # 64 rows, 4 of 32 query heads per workgroup -> 16 items of
            # 2049-2050 tiles; about 1024 pieces in all: pieces of 33 tiles, 62
            # per item.
            split = cp.workspace_size([_desc(P=65536, R=64, C=1)], 32, 8)
            assert 16 * 62 * _piece(rows) <= split < 16 * 62 * _piece(rows) + (1 << 20)
        # The 32K Llama-3-8B rank-0 shard in 384-row workgroups: 688 items of
        # 96 positions x 4 heads, 344 of them long (chunk 7), 43 for each
        # XCD's 32 compute units; 11 of each XCD's are cut in two, so that
        # every unit ends near the ideal.
        cp.set_workgroup_rows(384)
        balanced = cp.workspace_size([_desc(R=32768, C=4)], 32, 8)
        assert 176 * _piece(384) <= balanced < 176 * _piece(384) + (1 << 20)
        # The 70B shard's eight pass-KV partials: 21888 items of 32 bytes and
        # the descriptors, no pieces.
        many = cp.workspace_size([_desc(R=131072, C=8, kv_rank=s) for s in range(8)], 64, 8)
        assert 21888 * 32 <= many < 21888 * 32 + 8192
        # In 256-row workgroups the 32K shard's 512 long items fill two rounds
        # exactly: nothing is cut.
        cp.set_workgroup_rows(256)
        assert cp.workspace_size([_desc(R=32768, C=4)], 32, 8) < _piece(256)
        # Chosen per launch: the larger shape for the 32K rank-0 shard, the
        # smaller for the few long walks (more, shorter pieces fill the units).
        cp.set_workgroup_rows(0)
        assert cp.workspace_size([_desc(R=32768, C=4)], 32, 8) == balanced
        assert cp.workspace_size([_desc(P=65536, R=64, C=1)], 32, 8) < 16 * 62 * _piece(384)
    finally:
        cp.set_workgroup_rows(0)


def test_workgroup_rows_setting():
    for bad in (1, 128, 255, 512, -1):
        with pytest.raises(cp.CpError):
            cp.set_workgroup_rows(bad)
    for ok in (256, 384, 0):
        cp.set_workgroup_rows(ok)


def _merge_status(n_parts=2, n_tokens=4, H=2, D=128, out=FAKE, lse_out=FAKE * 2, restore=None,
                  parts=None, out_bf16=0):
    o = (ctypes.c_void_p * max(1, n_parts))(*([FAKE * 3] * n_parts if parts is None else parts))
    l = (ctypes.c_void_p * max(1, n_parts))(*([FAKE * 4] * n_parts))
    return cp.lib.cp_attn_merge(n_parts, o, l, n_tokens, H, D, out, out_bf16, lse_out,
                                ctypes.byref(restore) if restore is not None else None, None)


def test_merge_argument_errors():
    assert _merge_status(n_parts=0) == cp.CP_ERR_INVALID
    assert _merge_status(n_parts=17) == cp.CP_ERR_INVALID
    assert _merge_status(D=64) == cp.CP_ERR_UNSUPPORTED
    assert _merge_status(H=0) == cp.CP_ERR_INVALID
    assert _merge_status(n_tokens=-1) == cp.CP_ERR_INVALID
    assert _merge_status(out=None) == cp.CP_ERR_INVALID
    assert _merge_status(out=FAKE + 4) == cp.CP_ERR_INVALID
    assert _merge_status(parts=[FAKE * 3, None]) == cp.CP_ERR_INVALID
    assert _merge_status(out_bf16=3) == cp.CP_ERR_INVALID
    plan, _ = cp.shard_plan(0, 10, 2, 0, with_rows=False)
    assert _merge_status(n_tokens=5, restore=plan) == cp.CP_ERR_INVALID   # n_rows is 4
    plan.chunk[0].q_len = 2
    assert _merge_status(n_tokens=4, restore=plan) == cp.CP_ERR_INVALID   # tampered plan


def _wb_status(P=32, R=40, C=2, rank=0, Hkv=2, D=128, rows=FAKE, cache=FAKE * 2, table=FAKE * 3,
               table_len=None, n_blocks=8, plan=None):
    if plan is None:
        plan, _ = cp.shard_plan(P, R, C, rank, with_rows=False)
    if table_len is None:
        table_len = -(-(P + R) // 16)
    return cp.lib.cp_kv_writeback(ctypes.byref(plan), rows, rows, Hkv, D, cache, cache, n_blocks, table,
                                  table_len, None)


def test_writeback_argument_errors():
    assert _wb_status(P=40) == cp.CP_ERR_INVALID                      # prefix not block aligned
    assert _wb_status(table_len=4) == cp.CP_ERR_INVALID               # 72 tokens need 5 blocks
    assert _wb_status(rows=None) == cp.CP_ERR_INVALID
    assert _wb_status(cache=FAKE + 8) == cp.CP_ERR_INVALID
    assert _wb_status(table=FAKE + 2) == cp.CP_ERR_INVALID
    assert _wb_status(Hkv=0) == cp.CP_ERR_INVALID
    assert _wb_status(D=12) == cp.CP_ERR_INVALID
    assert _wb_status(n_blocks=-1) == cp.CP_ERR_INVALID
    plan, _ = cp.shard_plan(32, 40, 2, 0, with_rows=False)
    plan.n_rows += 1
    assert _wb_status(plan=plan) == cp.CP_ERR_INVALID                  # tampered plan
    assert cp.lib.cp_kv_writeback(None, FAKE, FAKE, 2, 128, FAKE, FAKE, 8, FAKE, 5, None) == cp.CP_ERR_INVALID
    assert cp.last_error() != ""


def _ga_status(cache=FAKE, n_blocks=8, table=FAKE, table_len=5, pos_begin=8, n=70, Hkv=2, D=128, rows=FAKE):
    return cp.lib.cp_kv_gather(cache, cache, n_blocks, table, table_len, pos_begin, n, Hkv, D, rows, rows, None)


def test_gather_argument_errors():
    assert _ga_status(table_len=4) == cp.CP_ERR_INVALID               # positions 8..77 need 5 blocks
    assert _ga_status(rows=None) == cp.CP_ERR_INVALID
    assert _ga_status(cache=None) == cp.CP_ERR_INVALID
    assert _ga_status(cache=FAKE + 8) == cp.CP_ERR_INVALID
    assert _ga_status(table=FAKE + 2) == cp.CP_ERR_INVALID
    assert _ga_status(Hkv=0) == cp.CP_ERR_INVALID
    assert _ga_status(D=12) == cp.CP_ERR_INVALID
    assert _ga_status(n_blocks=-1) == cp.CP_ERR_INVALID
    assert _ga_status(pos_begin=-1) == cp.CP_ERR_INVALID
    assert _ga_status(n=-1) == cp.CP_ERR_INVALID
    assert _ga_status(pos_begin=1 << 31, table_len=1 << 28) == cp.CP_ERR_UNSUPPORTED
    assert cp.last_error() != ""
    # Nothing to copy: no pointer is needed and nothing is launched.
    assert _ga_status(cache=None, table=None, rows=None, n=0, table_len=1) == cp.CP_OK


def _rp_status(P=0, R=64, C_src=2, C_dst=4, dst_rank=0, src=None, dst=FAKE, row_bytes=4096):
    ptrs = (ctypes.c_void_p * max(1, C_src))(*([FAKE * 2] * C_src if src is None else src))
    return cp.lib.cp_repartition(P, R, C_src, ptrs, C_dst, dst_rank, dst, row_bytes, None)


def test_repartition_argument_errors():
    assert _rp_status(C_src=0) == cp.CP_ERR_INVALID
    assert _rp_status(C_dst=65) == cp.CP_ERR_INVALID
    assert _rp_status(dst_rank=4) == cp.CP_ERR_INVALID
    assert _rp_status(dst_rank=-1) == cp.CP_ERR_INVALID
    assert _rp_status(row_bytes=24) == cp.CP_ERR_INVALID
    assert _rp_status(row_bytes=0) == cp.CP_ERR_INVALID
    assert _rp_status(dst=None) == cp.CP_ERR_INVALID
    assert _rp_status(dst=FAKE + 8) == cp.CP_ERR_INVALID
    assert _rp_status(src=[FAKE * 2, None]) == cp.CP_ERR_INVALID      # rank 1 has rows
    assert _rp_status(src=[FAKE * 2, FAKE + 4]) == cp.CP_ERR_INVALID
    assert _rp_status(P=-1) == cp.CP_ERR_INVALID
    assert _rp_status(P=1 << 31, R=64) == cp.CP_ERR_UNSUPPORTED
    assert cp.last_error() != ""


def test_binding_refuses_host_tensors():
    """The binding checks a tensor argument before taking its pointer: host
    memory is refused (the kernels would dereference it on the GPU)."""
    import torch
    plan, _ = cp.shard_plan(0, 64, 2, 0)
    q = torch.zeros((plan.n_rows, 8, 128), dtype=torch.bfloat16)
    with pytest.raises(ValueError, match="GPU tensor"):
        cp.make_desc(plan, q, None, None, None, None, include_prefix=False, kv_rank=cp.CP_KV_NONE)


def _noalloc_status(descs, Hq=8, Hkv=2, D=128, scale=0.0):
    arr = (cp.CpPartialDesc * max(1, len(descs)))(*descs)
    return cp.lib.cp_attn_partial_noalloc(arr, len(descs), Hq, Hkv, D, scale, None)


def test_noalloc_argument_errors():
    """The variant without a workspace refuses what cp_attn_partial refuses,
    before any HIP call, and an empty launch is a no-op."""
    assert _noalloc_status([_desc()], D=64) == cp.CP_ERR_UNSUPPORTED
    assert _noalloc_status([_desc()], scale=float("nan")) == cp.CP_ERR_INVALID
    assert _noalloc_status([_desc(kv_rank=5)]) == cp.CP_ERR_INVALID
    assert _noalloc_status([_desc(q=None)]) == cp.CP_ERR_INVALID
    assert _noalloc_status([_desc(P=32, n_blocks=0)]) == cp.CP_ERR_INVALID
    assert _noalloc_status([_desc(P=1 << 30, R=64)]) == cp.CP_ERR_UNSUPPORTED
    assert _noalloc_status([]) == cp.CP_OK
    assert _noalloc_status([_desc(R=3, C=4, rank=3)]) == cp.CP_OK     # a rank with no rows


def test_noalloc_refuses_tables_beyond_its_scratch():
    """2^29 query rows of one head: 2^21 work items, 64 MiB of tables, beyond
    the 32 MiB scratch -- refused with CP_ERR_CAPACITY before any HIP call."""
    d = _desc(P=0, R=1 << 29, C=1)
    assert _noalloc_status([d], Hq=1, Hkv=1) == cp.CP_ERR_CAPACITY
    assert "scratch" in cp.last_error()


def _rpa_status(P=0, R=64, C_src=2, C_dst=4, n_sets=2, row_bytes=512, src=None, dst=None):
    n_src = max(1, n_sets) * C_src
    n_dst = max(1, n_sets) * C_dst
    s = (ctypes.c_void_p * n_src)(*([FAKE] * n_src if src is None else src))
    d = (ctypes.c_void_p * n_dst)(*([FAKE * 2] * n_dst if dst is None else dst))
    return cp.lib.cp_repartition_all(P, R, C_src, s, C_dst, d, n_sets, row_bytes, None)


def test_repartition_all_argument_errors():
    """Every refusal happens before any HIP call."""
    assert _rpa_status(C_src=0) == cp.CP_ERR_INVALID
    assert _rpa_status(C_dst=65) == cp.CP_ERR_INVALID
    assert _rpa_status(n_sets=3) == cp.CP_ERR_INVALID
    assert _rpa_status(n_sets=0) == cp.CP_ERR_INVALID
    assert _rpa_status(row_bytes=24) == cp.CP_ERR_INVALID
    assert _rpa_status(P=-1) == cp.CP_ERR_INVALID
    assert _rpa_status(P=1 << 31, R=1) == cp.CP_ERR_UNSUPPORTED
    # A rank with rows needs an aligned pointer, in either set.
    assert _rpa_status(src=[FAKE, FAKE, FAKE, None]) == cp.CP_ERR_INVALID
    assert _rpa_status(dst=[FAKE * 2] * 7 + [FAKE + 8]) == cp.CP_ERR_INVALID
    assert "set 1 rank 3" in cp.last_error()
    # R < 2C: ranks without rows may be NULL; R = 0 launches nothing.
    assert _rpa_status(R=0, src=[None] * 4, dst=[None] * 8) == cp.CP_OK


def test_binding_constants_match_the_header():
    """Every #define of include/cp_attn.h that the binding mirrors has the
    header's value."""
    import re
    hdr = open(os.path.join(os.path.dirname(os.path.dirname(os.path.abspath(__file__))), "include",
                            "cp_attn.h")).read()
    found = 0
    for name, val in re.findall(r"^#define (CP_[A-Z0-9_]+) +\(?(-?\d+)\)?(?: |$)", hdr, re.M):
        if hasattr(cp, name):
            assert getattr(cp, name) == int(val), name
            found += 1
    assert found >= 14
    assert cp.CP_NOALLOC_SCRATCH_BYTES == 32 << 20  # (32u << 20) in the header
    assert cp.CP_OUT_LOCAL == 0 and cp.CP_OUT_SEQUENCE == 1
