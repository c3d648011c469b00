"""The oracle against its pins (CPU only)."""

import os

import numpy as np
import pytest

import oracle
from oracle import attention as oatt
from oracle import cache as ocache
from oracle import plan as oplan
import oracle_pins as pins

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def test_oracle_matches_brute_force():
    pins.check_brute(oatt.attend)


def test_oracle_matches_torch_sdpa_float64():
    pins.check_sdpa(oatt.full_causal_attention)


def test_oracle_closed_forms():
    pins.check_closed_forms(oatt.full_causal_attention)


def test_zigzag_restore_equals_single_rank():
    pins.check_zigzag_restore(oatt.full_causal_attention, oatt.rank_partial, oplan.shard_plan)


def test_lse_merge_of_any_partition():
    pins.check_merge(oatt.full_causal_attention, oatt.attend, oatt.lse_merge)


def test_paged_prefix_plus_suffix_equals_recompute():
    pins.check_paged_prefix(oatt.full_causal_attention, oatt.rank_partial, oatt.gather_paged)


def test_plan_rule_and_workload():
    pins.check_plan(oplan.shard_plan, oplan.remaining_workload, oplan.shard_plan_fast)


def _golden_lines(name):
    with open(os.path.join(GOLDEN, name)) as f:
        for line in f:
            line = line.strip()
            if line and not line.startswith("#"):
                yield line.split()


def test_plan_golden_chunk_assignment():
    for C, rank, c0, c1 in ([int(x) for x in t] for t in _golden_lines("zigzag_rule.txt")):
        plan = oplan.shard_plan_fast(0, 4 * C * 3, C, rank)
        assert [c[0] for c in plan["chunks"]] == [c0, c1]


def test_plan_golden_rows():
    for P, R, C, rank, s, n_rows, ranges, pairs in _golden_lines("zigzag_rows.txt"):
        P, R, C, rank, s, n_rows, pairs = map(int, (P, R, C, rank, s, n_rows, pairs))
        plan = oplan.shard_plan_fast(P, R, C, rank)
        assert plan["chunk_len"] == s
        assert plan["n_rows"] == n_rows
        assert plan["visible_pairs"] == pairs
        want = []
        if ranges != "-":
            for r in ranges.split(","):
                lo, hi = map(int, r.split("-"))
                want.extend(range(lo, hi))
        assert plan["row_pos"] == want


def test_inverse_map_is_the_inverse():
    for P, R, C in [(0, 1024, 2), (16, 37, 8), (0, 3, 4)]:
        rank_of, row_of = oplan.inverse_map(P, R, C)
        for i in range(R):
            plan = oplan.shard_plan_fast(P, R, C, rank_of[i])
            assert plan["row_pos"][row_of[i]] == P + i


def test_kv_shards_match_hand_worked_zigzag_shards():
    pins.check_kv_shards(oplan.kv_shard_ranges, oplan.shard_plan_fast)


def test_kv_shards_partition_the_suffix():
    for P, R, C in [(0, 1024, 2), (32, 37, 8), (0, 3, 4)]:
        covered = []
        for s in range(C):
            for lo, hi in oplan.kv_shard_ranges(P, R, C, s):
                covered.extend(range(lo, hi))
        assert sorted(covered) == list(range(P, P + R))


def test_pass_kv_partials_merge_to_allgather_view():
    """A rank's partials against each rank's KV shard, merged, equal its
    attention over all causally visible keys (the all-gathered view)."""
    rng = np.random.default_rng(7)
    P, R, C, Hq, Hkv, D = 32, 45, 4, 4, 2, 16
    L = P + R
    q = rng.standard_normal((L, Hq, D))
    k = rng.standard_normal((L, Hkv, D))
    v = rng.standard_normal((L, Hkv, D))
    B = 16
    nb = P // B
    table = rng.permutation(nb)
    kc = np.zeros((nb, B, Hkv, D)); vc = np.zeros((nb, B, Hkv, D))
    for b in range(nb):
        kc[table[b]] = k[b * B:(b + 1) * B]
        vc[table[b]] = v[b * B:(b + 1) * B]
    for r in range(C):
        plan = oplan.shard_plan_fast(P, R, C, r)
        rows = np.array(plan["row_pos"], dtype=np.int64)
        if rows.size == 0:
            continue
        full = oatt.rank_partial(q[rows], rows, P, k[P:], v[P:], kc, vc, table)
        parts = [oatt.rank_partial(q[rows], rows, P, k[P:], v[P:], kc, vc, table,
                                   include_prefix=True, suffix_ranges=[])]
        for s in range(C):
            parts.append(oatt.rank_partial(q[rows], rows, P, k[P:], v[P:], include_prefix=False,
                                           suffix_ranges=oplan.kv_shard_ranges(P, R, C, s)))
        O, Lse = oatt.lse_merge([p[0] for p in parts], [p[1] for p in parts])
        assert np.max(np.abs(O - full[0])) <= 1e-12
        assert np.max(np.abs(Lse - full[1])) <= 1e-12


def test_plan_rejects_bad_arguments():
    for args in [(0, 10, 0, 0), (0, 10, 2, 2), (0, 10, 2, -1), (-16, 10, 2, 0)]:
        with pytest.raises(ValueError):
            oplan.shard_plan_fast(*args)


def test_paged_writeback_round_trip():
    pins.check_writeback(ocache.write_paged, ocache.rank_writeback, oatt.gather_paged)


def test_paged_read_back():
    pins.check_read_paged(ocache.read_paged, ocache.write_paged)


def test_repartition_between_degrees():
    pins.check_repartition(ocache.repartition)
