"""Checks that pin the oracle to facts other than itself.

Each check takes the oracle functions it exercises as arguments, so that
``test_oracle.py`` runs it on the real oracle and ``test_oracle_mutations.py``
runs it on copies with planted mistakes (which must fail).  Every check
raises AssertionError on failure.

What pins what:
  * brute force (``oracle.brute``: scalar loops, math.fsum) on tiny inputs;
  * a library special case: torch's float64 scaled_dot_product_attention with
    is_causal=True (no prefix, KV heads expanded for grouped queries);
  * closed forms: Q = 0 gives the running mean of V and LSE = ln(p + 1);
    position 0 sees only key 0 (O = v_0, LSE = q_0.k_0 / sqrt(D)); a dominant
    key wins; grouped heads read KV head h // (Hq / Hkv);
  * the paper's statements: restoring the zigzag ranks' outputs equals
    single-rank causal attention (Sec. 2.1); the remaining workload is
    W(R, P) = RP + R(R+1)/2 (Sec. 2.2); the log-sum-exp merge of a partition
    of the keys equals attention over all of them.
"""

from __future__ import annotations

import math

import numpy as np
import torch

from oracle.brute import attention_brute


def _rng(seed):
    return np.random.default_rng(seed)


def check_brute(attend, seed=0):
    rng = _rng(seed)
    # (n queries, m keys, Hq, Hkv, D, first query position)
    for n, m, Hq, Hkv, D, q0 in [(12, 12, 2, 2, 8, 0), (10, 26, 4, 2, 16, 16),
                                  (7, 7, 4, 1, 4, 0), (9, 40, 2, 1, 128, 31)]:
        q = rng.standard_normal((n, Hq, D))
        k = rng.standard_normal((m, Hkv, D))
        v = rng.standard_normal((m, Hkv, D))
        q_pos = np.arange(q0, q0 + n)
        k_pos = np.arange(m)
        O, L = attend(q, q_pos, k, v, k_pos)
        Ob, Lb = attention_brute(q, q_pos, k, v, k_pos)
        Ob = np.array(Ob)
        Lb = np.array(Lb)
        fin = np.isfinite(Lb)
        assert np.array_equal(np.isfinite(L), fin), "visible-key sets differ from brute force"
        assert np.max(np.abs(O - Ob)) <= 1e-12, "O differs from brute force"
        assert np.max(np.abs(L[fin] - Lb[fin])) <= 1e-12, "LSE differs from brute force"


def check_sdpa(full_causal_attention, seed=1):
    rng = _rng(seed)
    for L, Hq, Hkv, D in [(96, 8, 2, 128), (33, 4, 4, 64)]:
        q = rng.standard_normal((L, Hq, D))
        k = rng.standard_normal((L, Hkv, D))
        v = rng.standard_normal((L, Hkv, D))
        O, _ = full_causal_attention(q, k, v)
        G = Hq // Hkv
        tq = torch.from_numpy(q).permute(1, 0, 2)[None]
        tk = torch.from_numpy(k).repeat_interleave(G, dim=1).permute(1, 0, 2)[None]
        tv = torch.from_numpy(v).repeat_interleave(G, dim=1).permute(1, 0, 2)[None]
        ref = torch.nn.functional.scaled_dot_product_attention(tq, tk, tv, is_causal=True)
        ref = ref[0].permute(1, 0, 2).numpy()
        assert np.max(np.abs(O - ref)) <= 1e-12, "O differs from torch float64 SDPA"


def check_closed_forms(full_causal_attention, seed=2):
    rng = _rng(seed)
    L, Hq, Hkv, D = 40, 4, 2, 128
    k = rng.standard_normal((L, Hkv, D))
    v = rng.standard_normal((L, Hkv, D))
    G = Hq // Hkv
    # Q = 0: every visible key has logit 0, so the output is the running mean.
    O, LSE = full_causal_attention(np.zeros((L, Hq, D)), k, v)
    for p in range(L):
        for h in range(Hq):
            mean = v[: p + 1, h // G].mean(axis=0)
            assert np.max(np.abs(O[p, h] - mean)) <= 1e-12, "Q=0 output is not the running mean"
            assert abs(LSE[p, h] - math.log(p + 1)) <= 1e-12, "Q=0 LSE is not ln(p+1)"
    # Position 0 sees exactly key 0 (diagonal included, nothing else).
    q = rng.standard_normal((L, Hq, D))
    O, LSE = full_causal_attention(q, k, v)
    for h in range(Hq):
        assert np.max(np.abs(O[0, h] - v[0, h // G])) <= 1e-12, "row 0 output is not v_0"
        dot = math.fsum(q[0, h, d] * k[0, h // G, d] for d in range(D))
        assert abs(LSE[0, h] - dot / math.sqrt(D)) <= 1e-12, "row 0 LSE is not q.k/sqrt(D)"
    # A dominant key: logit gap >= 50 puts all the weight on it.
    q = np.zeros((L, Hq, D))
    q[:, :, 0] = 1.0
    kd = np.zeros((L, Hkv, D))
    j_star = 17
    kd[j_star, :, 0] = 50.0 * math.sqrt(D) + 1.0
    O, _ = full_causal_attention(q, kd, v)
    for p in range(j_star, L):
        for h in range(Hq):
            assert np.max(np.abs(O[p, h] - v[j_star, h // G])) <= 1e-14, \
                "dominant key does not win"
    # Grouped heads: KV head g holds the constant g + 1, so query head h must
    # return exactly h // G + 1.
    vg = np.zeros((L, Hkv, D))
    for g in range(Hkv):
        vg[:, g, :] = g + 1.0
    O, _ = full_causal_attention(rng.standard_normal((L, Hq, D)), k, vg)
    for h in range(Hq):
        assert np.max(np.abs(O[:, h, :] - (h // G + 1.0))) <= 1e-12, "wrong KV head for a query head"


def check_zigzag_restore(full_causal_attention, rank_partial, shard_plan, seed=3):
    """Sec. 2.1: ranks' outputs restored to original order == single-rank attention."""
    rng = _rng(seed)
    Hq, Hkv, D = 4, 2, 32
    for L, C in [(64, 1), (64, 2), (70, 4), (37, 8), (5, 4)]:
        q = rng.standard_normal((L, Hq, D))
        k = rng.standard_normal((L, Hkv, D))
        v = rng.standard_normal((L, Hkv, D))
        O_full, L_full = full_causal_attention(q, k, v)
        O_rest = np.full_like(O_full, np.nan)
        L_rest = np.full_like(L_full, np.nan)
        for r in range(C):
            plan = shard_plan(0, L, C, r)
            rows = np.array(plan["row_pos"], dtype=np.int64)
            if rows.size == 0:
                continue
            O_r, L_r = rank_partial(q[rows], rows, 0, k, v)
            O_rest[rows] = O_r
            L_rest[rows] = L_r
        assert not np.isnan(O_rest).any(), "restored output misses rows"
        assert np.max(np.abs(O_rest - O_full)) <= 1e-12, "restore(ranks) != full attention"
        assert np.max(np.abs(L_rest - L_full)) <= 1e-12, "restored LSE != full LSE"


def check_merge(full_causal_attention, attend, lse_merge, seed=4):
    """Merging partials over any partition of the keys == attention over all."""
    rng = _rng(seed)
    L, Hq, Hkv, D = 48, 4, 2, 16
    q = rng.standard_normal((L, Hq, D)) * 2.0
    k = rng.standard_normal((L, Hkv, D))
    v = rng.standard_normal((L, Hkv, D))
    pos = np.arange(L)
    O_full, L_full = full_causal_attention(q, k, v)
    label = rng.integers(0, 5, size=L)          # subset 4 may be empty or not
    label[label == 3] = 2                       # subset 3 is empty
    parts = []
    for s in range(5):
        sel = np.nonzero(label == s)[0]
        parts.append(attend(q, pos, k[sel], v[sel], pos[sel]))
    O_m, L_m = lse_merge([p[0] for p in parts], [p[1] for p in parts])
    assert np.max(np.abs(O_m - O_full)) <= 1e-12, "merge(partition) != full output"
    assert np.max(np.abs(L_m - L_full)) <= 1e-12, "merge(partition) != full LSE"
    # Any order and grouping gives the same result.
    a = lse_merge([parts[4][0], parts[0][0]], [parts[4][1], parts[0][1]])
    b = lse_merge([parts[2][0], parts[3][0], parts[1][0]], [parts[2][1], parts[3][1], parts[1][1]])
    O_g, L_g = lse_merge([b[0], a[0]], [b[1], a[1]])
    assert np.max(np.abs(O_g - O_full)) <= 1e-12, "merge is not associative/commutative"
    assert np.max(np.abs(L_g - L_full)) <= 1e-12, "merged LSE depends on grouping"
    # A row with no keys anywhere stays O = 0, LSE = -inf.
    empty = attend(q[:3], pos[:3], k[:0], v[:0], pos[:0])
    O_e, L_e = lse_merge([empty[0], empty[0]], [empty[1], empty[1]])
    assert np.all(O_e == 0.0) and np.all(np.isneginf(L_e)), "empty merge is not (0, -inf)"


def check_paged_prefix(full_causal_attention, rank_partial, gather_paged, seed=5):
    """Prefix K/V read through a permuted block table + the uncached suffix ==
    rows P..L-1 of recomputing the whole sequence (Sec. 2.2)."""
    rng = _rng(seed)
    Hq, Hkv, D, B = 4, 1, 32, 16
    for P, R in [(48, 20), (16, 1), (64, 64)]:
        L = P + R
        q = rng.standard_normal((L, Hq, D))
        k = rng.standard_normal((L, Hkv, D))
        v = rng.standard_normal((L, Hkv, D))
        nb = P // B
        spare = 3
        perm = rng.permutation(nb + spare)
        table = perm[:nb]
        k_cache = rng.standard_normal((nb + spare, B, Hkv, D))
        v_cache = rng.standard_normal((nb + spare, B, Hkv, D))
        for b in range(nb):
            k_cache[table[b]] = k[b * B:(b + 1) * B]
            v_cache[table[b]] = v[b * B:(b + 1) * B]
        assert np.array_equal(gather_paged(k_cache, table, P), k[:P]), "paged gather is wrong"
        O_full, L_full = full_causal_attention(q, k, v)
        rows = np.arange(P, L)
        O_p, L_p = rank_partial(q[P:], rows, P, k[P:], v[P:], k_cache, v_cache, table)
        assert np.max(np.abs(O_p - O_full[P:])) <= 1e-12, "prefix + suffix != recompute"
        assert np.max(np.abs(L_p - L_full[P:])) <= 1e-12, "prefix + suffix LSE != recompute"
    # Entries outside the cache read as zero rows: addressing by hand, then
    # attention through such a table == recomputation with those prefix rows
    # zeroed (keys of logit 0, values 0).
    cache = np.arange(3 * B, dtype=np.float64).reshape(3, B, 1, 1)
    got = gather_paged(cache, [1, -1, 3, 0], 4 * B).reshape(-1)
    assert got[:B].tolist() == list(range(B, 2 * B)), "valid entry before bad ones"
    assert not got[B:3 * B].any(), "entries -1 and n_blocks must read as zeros"
    assert got[3 * B:].tolist() == list(range(B)), "valid entry after bad ones"
    P, R = 64, 24
    q = rng.standard_normal((P + R, Hq, D)) * 2.0
    k = rng.standard_normal((P + R, Hkv, D))
    v = rng.standard_normal((P + R, Hkv, D))
    table = np.array([2, -1, 0, 7])              # 4 cache blocks: entry 7 is past the end
    k_cache = rng.standard_normal((4, B, Hkv, D))
    v_cache = rng.standard_normal((4, B, Hkv, D))
    kz, vz = k.copy(), v.copy()
    for b, blk in enumerate(table):
        if 0 <= blk < 4:
            k_cache[blk] = k[b * B:(b + 1) * B]
            v_cache[blk] = v[b * B:(b + 1) * B]
        else:
            kz[b * B:(b + 1) * B] = 0.0
            vz[b * B:(b + 1) * B] = 0.0
    O_full, L_full = full_causal_attention(q, kz, vz)
    O_p, L_p = rank_partial(q[P:], np.arange(P, P + R), P, k[P:], v[P:], k_cache, v_cache, table)
    assert np.max(np.abs(O_p - O_full[P:])) <= 1e-12, "bad entries are not zero keys and values"
    assert np.max(np.abs(L_p - L_full[P:])) <= 1e-12, "bad entries: LSE"


def check_plan(shard_plan, remaining_workload, shard_plan_fast=None):
    """Sec. 2.1 zigzag rule and Sec. 2.2 W(R, P)."""
    # W(R, P) evaluated by hand from RP + R(R+1)/2.
    for R, P, W in [(1, 0, 1), (4, 0, 10), (2, 3, 9), (16384, 49152, 939_532_288),
                    (32768, 0, 536_887_296)]:
        assert remaining_workload(R, P) == W, "W(R, P) closed form"
    for P, R, C in [(0, 1024, 2), (0, 70, 4), (16, 37, 8), (32, 5, 4), (0, 64, 1), (48, 3, 2)]:
        total = 0
        seen = []
        s = -(-R // (2 * C))
        for r in range(C):
            plan = shard_plan(P, R, C, r)
            ids = [c[0] for c in plan["chunks"]]
            assert ids == [r, 2 * C - 1 - r], "rank k must hold chunks k and 2C-1-k"
            assert plan["chunk_len"] == s and plan["padded_len"] == 2 * C * s
            total += plan["visible_pairs"]
            seen.extend(plan["row_pos"])
            if R % (2 * C) == 0:
                assert plan["visible_pairs"] == 2 * s * P + 2 * C * s * s + s, "zigzag balance"
            if shard_plan_fast is not None:
                assert shard_plan_fast(P, R, C, r) == plan
        assert total == remaining_workload(R, P), "sum over ranks != W(R, P)"
        assert sorted(seen) == list(range(P, P + R)), "rows are not a bijection onto the suffix"


GOLDEN_DIR = __import__("os").path.join(__import__("os").path.dirname(__import__("os").path.abspath(__file__)),
                                        "golden")


def _golden_passkv_shards():
    rows = []
    with open(GOLDEN_DIR + "/passkv_shards.txt") as f:
        for line in f:
            if not line.strip() or line.startswith("#"):
                continue
            P, R, C, s, ids, ranges = line.split()
            rng = [] if ranges == "-" else [tuple(int(x) for x in r.split("-")) for r in ranges.split(",")]
            rows.append((int(P), int(R), int(C), int(s), tuple(int(x) for x in ids.split(",")), rng))
    return rows


def check_kv_shards(kv_shard_ranges, shard_plan):
    """Pass-KV shard s is the suffix K/V rank s holds under the zigzag split
    (Sec. 2.1): its chunks s and 2C-1-s.  Checked against ranges worked by hand
    (tests/golden/passkv_shards.txt), and against the pinned plan: shard s's
    ranges are exactly the contiguous runs of rank s's row positions, and the C
    shards partition the suffix."""
    cases = _golden_passkv_shards()
    assert len(cases) >= 18
    for P, R, C, s, ids, want in cases:
        assert [tuple(r) for r in kv_shard_ranges(P, R, C, s)] == want, (P, R, C, s)
        assert ids == (s, 2 * C - 1 - s)
    for P, R, C in [(0, 1024, 2), (0, 70, 4), (16, 37, 8), (32, 5, 4), (0, 64, 1), (48, 3, 2), (16, 37, 3),
                    (0, 1000, 8)]:
        keys = []
        for s in range(C):
            pos = shard_plan(P, R, C, s)["row_pos"]
            runs = []
            for p in pos:
                if runs and runs[-1][1] == p:
                    runs[-1][1] = p + 1
                else:
                    runs.append([p, p + 1])
            got = [tuple(r) for r in kv_shard_ranges(P, R, C, s)]
            merged = []
            for lo, hi in got:                      # two adjacent chunks form one run
                if merged and merged[-1][1] == lo:
                    merged[-1] = (merged[-1][0], hi)
                else:
                    merged.append((lo, hi))
            assert merged == [tuple(r) for r in runs], (P, R, C, s)
            for lo, hi in got:
                keys.extend(range(lo, hi))
        assert sorted(keys) == list(range(P, P + R)), "shards do not partition the suffix"


def check_read_paged(read_paged, write_paged, seed=12):
    """Paged read-back (Sec. 2.2, 7.1, 7.2): addressing by hand; an identity
    block table reads the cache in storage order (closed form); reading a
    range back after writing it returns the rows written, from any start
    position; entries outside the cache read as zeros."""
    cache = np.arange(5 * 16, dtype=np.float64).reshape(5, 16, 1, 1)
    got = read_paged(cache, [4, 0, 2], 15, 4)                 # positions 15, 16, 17, 18
    assert got.reshape(-1).tolist() == [4 * 16 + 15, 0, 1, 2], "block/slot addressing"
    rng = _rng(seed)
    Hkv, D, B = 2, 4, 16
    nb = 7
    cache = rng.standard_normal((nb, B, Hkv, D))
    assert np.array_equal(read_paged(cache, np.arange(nb), 0, nb * B), cache.reshape(nb * B, Hkv, D)), \
        "identity table must read the cache in order"
    for start, n in [(0, 50), (13, 40), (16, 16), (31, 1), (5, 0)]:
        table = rng.permutation(nb + 3)[:nb]
        x = rng.standard_normal((n, Hkv, D))
        written = write_paged(np.full((nb + 3, B, Hkv, D), np.nan), table, list(range(start, start + n)), x)
        assert np.array_equal(read_paged(written, table, start, n), x), "read-back of written rows"
    bad = np.array([1, -1, 9, 0])
    out = read_paged(cache, bad, 0, 4 * B)
    assert np.array_equal(out[:B], cache[1]) and np.array_equal(out[3 * B:], cache[0]), "valid entries"
    assert not np.any(out[B:3 * B]), "entries outside the cache read as zeros"


def check_writeback(write_paged, rank_writeback, gather_paged, seed=9):
    """Write-back into the paged cache (Sec. 2.2, 7.1, 8): the addressing by
    hand, the round trip through the prefix gather (itself pinned by
    ``check_paged_prefix``), every new token written exactly once by the CP
    ranks together, and nothing else touched."""
    # Addressing worked out by hand: position p -> block table[p // 16], slot p % 16.
    table = [4, 0, 2]
    cache = np.zeros((5, 16, 1, 1))
    out = write_paged(cache, table, [0, 17, 37], np.array([[[1.0]], [[2.0]], [[3.0]]]))
    assert out[4, 0, 0, 0] == 1.0 and out[0, 1, 0, 0] == 2.0 and out[2, 5, 0, 0] == 3.0, "block/slot addressing"
    assert np.count_nonzero(out) == 3, "write touched other slots"
    assert np.count_nonzero(cache) == 0, "write must not modify its input"
    rng = _rng(seed)
    Hkv, D, B = 2, 4, 16
    for P, R, C in [(32, 45, 2), (0, 70, 4), (16, 9, 3), (48, 3, 2), (0, 16, 1)]:
        L = P + R
        nb = -(-L // B)
        spare = 2
        table = rng.permutation(nb + spare)[:nb]
        x = rng.standard_normal((L, Hkv, D))
        cache = np.full((nb + spare, B, Hkv, D), np.nan)
        cache = write_paged(cache, table, list(range(P)), x[:P])          # the cached prefix
        before = cache.copy()
        for r in range(C):
            s = -(-R // (2 * C))
            rows = []
            for chunk in (r, 2 * C - 1 - r):                                # zigzag rows by hand
                lo, hi = P + chunk * s, min(P + (chunk + 1) * s, L)
                rows.extend(range(lo, max(lo, hi)))
            cache = rank_writeback(cache, table, P, R, C, r, x[rows] if rows else x[:0])
        assert np.array_equal(gather_paged(cache, table, L), x), "write-back does not round-trip"
        for pos in range(P):
            b, t = table[pos // B], pos % B
            assert np.array_equal(cache[b, t], before[b, t]), "prefix slots rewritten"
        used = {(int(table[p // B]), p % B) for p in range(L)}
        for b in range(nb + spare):
            for t in range(B):
                if (b, t) not in used:
                    assert np.isnan(cache[b, t]).all(), "slot outside the request written"


def check_repartition(repartition, seed=10):
    """Re-sharding rows between CP degrees (Sec. 6.2, 7.2): every destination
    row is the row of its global position (zigzag rows worked out by hand);
    C -> C is the identity and C -> 2C -> C a round trip; when 4C divides the
    padded length, degree-2C ranks 2k and 2k+1 draw only on degree-C rank k."""
    rng = _rng(seed)

    def rows_of(P, R, C, r):
        s = -(-R // (2 * C))
        out = []
        for chunk in (r, 2 * C - 1 - r):
            lo, hi = P + chunk * s, min(P + (chunk + 1) * s, P + R)
            out.extend(range(lo, max(lo, hi)))
        return out

    for P, R, C_src, C_dst in [(0, 64, 2, 4), (16, 37, 4, 2), (0, 70, 3, 5), (32, 8, 1, 4), (0, 128, 4, 8),
                               (0, 5, 4, 1)]:
        x = rng.standard_normal((R, 3))
        src = [x[np.array(rows_of(P, R, C_src, r), dtype=np.int64) - P] for r in range(C_src)]
        dst = repartition(P, R, C_src, src, C_dst)
        assert len(dst) == C_dst
        for r in range(C_dst):
            want = x[np.array(rows_of(P, R, C_dst, r), dtype=np.int64) - P]
            assert np.array_equal(np.asarray(dst[r]).reshape(want.shape), want), "row of the wrong position"
        same = repartition(P, R, C_src, src, C_src)
        assert all(np.array_equal(a, b) for a, b in zip(same, src)), "C -> C is not the identity"
        back = repartition(P, R, C_dst, dst, C_src)
        assert all(np.array_equal(np.asarray(a).reshape(b.shape), b) for a, b in zip(back, src)), "round trip"
    # Pairwise locality: tag each row with its source rank.
    for C, R in [(2, 64), (4, 256), (1, 8)]:
        tags = [np.full((len(rows_of(0, R, C, r)), 1), float(r)) for r in range(C)]
        dst = repartition(0, R, C, tags, 2 * C)
        for r2 in range(2 * C):
            assert (np.asarray(dst[r2]) == r2 // 2).all(), "degree-2C rank 2k+j must come from rank k"
