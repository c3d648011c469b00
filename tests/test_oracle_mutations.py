"""Plant plausible mistakes in copies of the oracle; the pins must catch each.

Each case rewrites one line of an oracle module's source, executes the copy
as a fresh module (the real oracle is untouched) and runs every pin on it.
At least one pin has to fail, otherwise the pins would let that mistake
through.
"""

import os
import types

import numpy as np
import pytest

import oracle_pins as pins

ORACLE_DIR = os.path.join(os.path.dirname(os.path.dirname(os.path.abspath(__file__))), "oracle")


def _mutant(filename, old, new):
    path = os.path.join(ORACLE_DIR, filename)
    with open(path) as f:
        src = f.read()
    assert src.count(old) == 1, f"mutation anchor not unique in {filename}: {old!r}"
    mod = types.ModuleType("mutant_" + filename[:-3])
    exec(compile(src.replace(old, new), path, "exec"), mod.__dict__)
    return mod


def _all_pins(att, plan, cache=None):
    if cache is None:
        from oracle import cache
    checks = [
        lambda: pins.check_writeback(cache.write_paged, cache.rank_writeback, att.gather_paged),
        lambda: pins.check_repartition(cache.repartition),
        lambda: pins.check_read_paged(cache.read_paged, cache.write_paged),
        lambda: pins.check_brute(att.attend),
        lambda: pins.check_sdpa(att.full_causal_attention),
        lambda: pins.check_closed_forms(att.full_causal_attention),
        lambda: pins.check_zigzag_restore(att.full_causal_attention, att.rank_partial, plan.shard_plan),
        lambda: pins.check_merge(att.full_causal_attention, att.attend, att.lse_merge),
        lambda: pins.check_paged_prefix(att.full_causal_attention, att.rank_partial, att.gather_paged),
        lambda: pins.check_plan(plan.shard_plan, plan.remaining_workload, plan.shard_plan_fast),
        lambda: pins.check_kv_shards(plan.kv_shard_ranges, plan.shard_plan_fast),
    ]
    failed = 0
    for c in checks:
        try:
            c()
        except Exception:
            failed += 1
    return failed


ATTENTION_MUTATIONS = [
    ("strict causal mask", "k_pos[None, :] <= q_pos[b0:b1, None]", "k_pos[None, :] < q_pos[b0:b1, None]"),
    ("wrong softmax scale", "scale = 1.0 / math.sqrt(D)", "scale = 1.0 / D"),
    ("GQA heads interleaved", "g = h // group", "g = h % Hkv"),
    ("V used as keys", "x = (q[b0:b1, h, :] @ kg.T) * scale", "x = (q[b0:b1, h, :] @ vg.T) * scale"),
    ("max dropped from LSE", "lse[idx, h] = mx[live] + np.log(denom)", "lse[idx, h] = np.log(denom)"),
    ("output not normalised", "out_rows = (e @ vg) / denom[:, None]", "out_rows = (e @ vg)"),
    ("merge weight sign", "np.exp(stack - safe_mx)", "np.exp(safe_mx - stack)"),
    ("merge ignores the max", "lse = np.where(live, safe_mx + np.log(", "lse = np.where(live, 0 * safe_mx + np.log("),
    ("block table ignored", "rows.append(cache[blk, j % block_tokens] if", "rows.append(cache[j // block_tokens, j % block_tokens] if"),
    ("gather of a bad entry wraps", "if 0 <= blk < cache.shape[0] else zero)", "if blk < cache.shape[0] else zero)"),
    ("gather of a bad entry is skipped", "if 0 <= blk < cache.shape[0] else zero)",
     "if 0 <= blk < cache.shape[0] else cache[0, 0])"),
    ("suffix off by one", "suffix_ranges = [(P, P + R)]", "suffix_ranges = [(P + 1, P + R)]"),
    ("suffix keys at wrong positions", "ps.append(np.arange(P + lo_i, P + hi_i, dtype=np.int64))",
     "ps.append(np.arange(lo_i, hi_i, dtype=np.int64))"),
]

PLAN_MUTATIONS = [
    ("second chunk off by one", "for chunk_id in (rank, 2 * C - 1 - rank):\n        start = chunk_id * s                      # suffix",
     "for chunk_id in (rank, 2 * C - 2 - rank):\n        start = chunk_id * s                      # suffix"),
    ("no padding", "padded = -(-R // (2 * C)) * (2 * C)", "padded = R"),
    ("W drops the prefix term", "return R * P + R * (R + 1) // 2", "return R * (R + 1) // 2"),
    ("diagonal not counted", "for _key in range(pos + 1):", "for _key in range(pos):"),
    ("pass-KV shard holds chunks s and C+s", "for chunk_id in (shard, 2 * C - 1 - shard):",
     "for chunk_id in (shard, C + shard):"),
    ("pass-KV shard holds its first chunk only", "for chunk_id in (shard, 2 * C - 1 - shard):",
     "for chunk_id in (shard,):"),
    ("pass-KV shard keeps padding keys", "        hi = min(R, lo + s)\n        if hi > lo:\n            out.append((P + lo, P + hi))",
     "        hi = lo + s\n        if hi > lo:\n            out.append((P + lo, P + hi))"),
]


CACHE_MUTATIONS = [
    ("slot off by one", "out[table[int(p) // block_tokens], int(p) % block_tokens] = rows[i]",
     "out[table[int(p) // block_tokens], (int(p) + 1) % block_tokens] = rows[i]"),
    ("write-back ignores the block table", "out[table[int(p) // block_tokens], int(p) % block_tokens] = rows[i]",
     "out[int(p) // block_tokens, int(p) % block_tokens] = rows[i]"),
    ("write-back uses the first chunk only", "return write_paged(cache, block_table, plan[\"row_pos\"], rank_rows, block_tokens)",
     "return write_paged(cache, block_table, plan[\"row_pos\"][:plan[\"chunks\"][0][2]], rank_rows[:plan[\"chunks\"][0][2]], block_tokens)"),
    ("repartition reads the destination's own plan", "plan = shard_plan_fast(P, R, C_src, r)",
     "plan = shard_plan_fast(P, R, C_dst, r) if r < C_dst else shard_plan_fast(P, R, C_src, r)"),
    ("repartition reverses a rank's rows", "where[pos] = (r, t)", "where[pos] = (r, plan[\"n_rows\"] - 1 - t)"),
    ("read-back ignores pos_begin", "p = pos_begin + t", "p = t"),
    ("read-back slot off by one", "out[t] = cache[blk, p % block_tokens]", "out[t] = cache[blk, (p + 1) % block_tokens]"),
    ("read-back of a bad entry wraps", "if 0 <= blk < cache.shape[0]:", "if True:"),
]


@pytest.mark.parametrize("name,old,new", CACHE_MUTATIONS, ids=[m[0] for m in CACHE_MUTATIONS])
def test_cache_mutation_is_caught(name, old, new):
    from oracle import attention, plan
    cache = _mutant("cache.py", old, new)
    assert _all_pins(attention, plan, cache) >= 1, f"no pin catches: {name}"


@pytest.mark.parametrize("name,old,new", ATTENTION_MUTATIONS, ids=[m[0] for m in ATTENTION_MUTATIONS])
def test_attention_mutation_is_caught(name, old, new):
    from oracle import plan
    att = _mutant("attention.py", old, new)
    # A mutant may produce -inf or NaN where the pins subtract: expected here.
    with np.errstate(invalid="ignore"):
        assert _all_pins(att, plan) >= 1, f"no pin catches: {name}"


@pytest.mark.parametrize("name,old,new", PLAN_MUTATIONS, ids=[m[0] for m in PLAN_MUTATIONS])
def test_plan_mutation_is_caught(name, old, new):
    from oracle import attention
    plan = _mutant("plan.py", old, new)
    assert _all_pins(attention, plan) >= 1, f"no pin catches: {name}"


def test_unmutated_oracle_passes_every_pin():
    from oracle import attention, plan
    assert _all_pins(attention, plan) == 0
