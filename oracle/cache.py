"""Oracle: the KV-cache steps around the attention -- writing a request's new
K/V into the paged prefix cache, reading positions back out of it, and
re-sharding rows between CP degrees.

TEST INFRASTRUCTURE ONLY (see ``oracle/__init__.py``).

Definitions followed:

* Write-back (Sec. 2.2: prefill builds the KV states of its input tokens and
  prefix caching keeps them for later requests; Sec. 7.1: one trie node is one
  cache block; Sec. 8: a destination reserves physical blocks and installs the
  KV states in them).  Token position p of a request is stored in physical
  block ``block_table[p // 16]``, slot ``p % 16`` -- the same addressing the
  prefix gather (``attention.gather_paged``) reads.  Every other slot keeps
  what it held.
* Read-back (Sec. 2.2: a prefix hit reuses the cached KV states; Sec. 7.1: one
  trie node is one cache block; Sec. 7.2: replication hands KV states to
  another worker).  The row of position p is the one ``write_paged`` stored at
  ``block_table[p // 16]``, slot ``p % 16``.
* Re-sharding between CP degrees (Sec. 6.2: after a split or merge the
  resident KV blocks are installed under the new CP geometry; Sec. 7.2:
  inter-degree replication repartitions KV states for the destination
  worker).  A rank's rows are the zigzag rows of ``plan.shard_plan``; the
  row a destination rank holds for global position p is the row the source
  rank holding p has for it.

Readings (the paper gives no formula for either step): the block size is 16
tokens (as for the prefix gather); write-back covers the new tokens P..P+R-1
only -- the prefix blocks are already cached -- and each CP rank writes the
rows it holds (its two zigzag chunks), so the ranks together write every new
token exactly once.  Rows are copied, not recomputed: both steps are exact.
"""

from __future__ import annotations

import numpy as np

from oracle.plan import shard_plan_fast

BLOCK_TOKENS = 16


def write_paged(cache, block_table, positions, rows, block_tokens=BLOCK_TOKENS):
    """A copy of ``cache`` with ``rows[i]`` stored at token position
    ``positions[i]``: physical block ``block_table[positions[i] // block_tokens]``,
    slot ``positions[i] % block_tokens``.

    cache: [n_blocks, block_tokens, ...]; rows: [n, ...] with the same
    trailing shape.  Positions must be distinct.
    """
    out = np.array(cache, copy=True)
    table = np.asarray(block_table, dtype=np.int64)
    rows = np.asarray(rows)
    if len(set(int(p) for p in positions)) != len(positions):
        raise ValueError("two rows for one position")
    for i, p in enumerate(positions):
        out[table[int(p) // block_tokens], int(p) % block_tokens] = rows[i]
    return out


def read_paged(cache, block_table, pos_begin, n, block_tokens=BLOCK_TOKENS):
    """Rows of positions pos_begin .. pos_begin + n - 1 read out of a paged
    cache: position p is held in physical block ``block_table[p // block_tokens]``,
    slot ``p % block_tokens`` (the addressing ``write_paged`` stores through).
    A position whose block-table entry lies outside the cache reads as zeros
    (reading: nothing is read through such an entry).

    cache: [n_blocks, block_tokens, ...]; returns [n, ...].
    """
    cache = np.asarray(cache)
    table = np.asarray(block_table, dtype=np.int64)
    out = np.zeros((n,) + cache.shape[2:], dtype=cache.dtype)
    for t in range(n):
        p = pos_begin + t
        blk = table[p // block_tokens]
        if 0 <= blk < cache.shape[0]:
            out[t] = cache[blk, p % block_tokens]
    return out


def rank_writeback(cache, block_table, P, R, C, rank, rank_rows, block_tokens=BLOCK_TOKENS):
    """Write-back of one CP rank: its rows (``rank_rows[t]`` for local row t,
    in plan order) go to their global positions."""
    plan = shard_plan_fast(P, R, C, rank)
    if len(rank_rows) != plan["n_rows"]:
        raise ValueError("rank_rows does not match the plan")
    return write_paged(cache, block_table, plan["row_pos"], rank_rows, block_tokens)


def repartition(P, R, C_src, src_rows, C_dst):
    """Rows of every destination rank (degree C_dst), each taken from the
    source rank (degree C_src) that holds the same global position.

    src_rows: list of C_src arrays, rank r's rows in its plan order.
    Returns a list of C_dst arrays in the destination plans' order.
    """
    where = {}
    for r in range(C_src):
        plan = shard_plan_fast(P, R, C_src, r)
        if len(src_rows[r]) != plan["n_rows"]:
            raise ValueError("source rows do not match the plan")
        for t, pos in enumerate(plan["row_pos"]):
            where[pos] = (r, t)
    out = []
    trailing = np.asarray(src_rows[0]).shape[1:] if C_src else ()
    for r in range(C_dst):
        plan = shard_plan_fast(P, R, C_dst, r)
        rows = [np.asarray(src_rows[where[pos][0]])[where[pos][1]] for pos in plan["row_pos"]]
        out.append(np.stack(rows) if rows else np.zeros((0,) + tuple(trailing)))
    return out
