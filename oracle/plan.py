"""Oracle: the zigzag context-parallel partition, written from its definition.

TEST INFRASTRUCTURE ONLY (see ``oracle/__init__.py``).

Paper, Sec. 2.1 (Context Parallelism): for CP degree C the input is padded,
if needed, to a multiple of 2C and cut into 2C equal contiguous chunks; rank
k (k = 0..C-1) receives chunks k and 2C-1-k; afterwards the ranks' outputs
are put back in the original order and concatenated, which must equal
single-rank causal attention.

Paper, Sec. 2.2 (Prefix Caching under CP): with a prefix hit, L = P + R and
only the R uncached tokens are computed; they attend to the P cached tokens
and to the preceding uncached ones, so the remaining work is
W(R, P) = R*P + R*(R+1)/2 query-key pairs (equation "remaining-attention").

Readings where the paper is silent:

* What is zigzagged under a prefix hit: the R-token uncached suffix only.
  Suffix index i (0 <= i < R) is global position P + i.
* Where the padding goes: at the end of the suffix.  Pad positions are not
  rows of any rank (a rank's rows are compact), and, sitting after every real
  token, they are never causally visible to a real query.
* Order of a rank's two chunks: chunk k's rows first, then chunk 2C-1-k's.
* R < 2C is legal: some chunks, hence some ranks, are empty.

Plain Python integers throughout: every value here is exact.
"""

from __future__ import annotations


def remaining_workload(R: int, P: int) -> int:
    """W(R, P) = R*P + R*(R+1)/2 (Sec. 2.2, equation "remaining-attention")."""
    return R * P + R * (R + 1) // 2


def _chunk_len(R: int, C: int) -> int:
    # Pad R up to a multiple of 2C; every one of the 2C chunks has this length.
    padded = -(-R // (2 * C)) * (2 * C)
    return padded // (2 * C)


def shard_plan(P: int, R: int, C: int, rank: int) -> dict:
    """The rows rank ``rank`` of a degree-C worker computes (Sec. 2.1).

    Returns a dict with
      padded_len   R rounded up to a multiple of 2C
      chunk_len    padded_len / 2C
      chunks       [(chunk_id, q_begin, q_len, local_offset)] for chunk ``rank``
                   then chunk ``2C-1-rank``; q_begin is the global position of
                   the chunk's first token, q_len its number of real tokens.
      n_rows       total real rows of the rank
      row_pos      global position of each local row, in local order
      visible_pairs  query-key pairs the rows see when each row attends to all
                   keys at positions 0..pos (the cached prefix included),
                   counted one pair at a time.
    """
    if C < 1 or not (0 <= rank < C) or R < 0 or P < 0:
        raise ValueError("bad plan arguments")
    s = _chunk_len(R, C)
    chunks = []
    row_pos = []
    for chunk_id in (rank, 2 * C - 1 - rank):
        start = chunk_id * s                      # suffix index of the chunk's first token
        q_len = max(0, min(R - start, s))         # real (unpadded) tokens in the chunk
        chunks.append((chunk_id, P + start, q_len, len(row_pos)))
        for i in range(q_len):
            row_pos.append(P + start + i)
    pairs = 0
    for pos in row_pos:
        for _key in range(pos + 1):               # keys 0..pos are causally visible
            pairs += 1
    return {
        "C": C, "rank": rank, "prefix_len": P, "new_len": R,
        "padded_len": 2 * C * s, "chunk_len": s, "n_rows": len(row_pos),
        "chunks": chunks, "row_pos": row_pos, "visible_pairs": pairs,
    }


def shard_plan_fast(P: int, R: int, C: int, rank: int) -> dict:
    """``shard_plan`` with the pair count summed per row instead of per pair.

    Same definition, used for sizes where counting pairs one at a time would
    take too long; ``tests`` check the two agree on small sizes.
    """
    if C < 1 or not (0 <= rank < C) or R < 0 or P < 0:
        raise ValueError("bad plan arguments")
    s = _chunk_len(R, C)
    chunks = []
    row_pos = []
    for chunk_id in (rank, 2 * C - 1 - rank):
        start = chunk_id * s
        q_len = max(0, min(R - start, s))
        chunks.append((chunk_id, P + start, q_len, len(row_pos)))
        row_pos.extend(range(P + start, P + start + q_len))
    pairs = sum(pos + 1 for pos in row_pos)
    return {
        "C": C, "rank": rank, "prefix_len": P, "new_len": R,
        "padded_len": 2 * C * s, "chunk_len": s, "n_rows": len(row_pos),
        "chunks": chunks, "row_pos": row_pos, "visible_pairs": pairs,
    }


def inverse_map(P: int, R: int, C: int):
    """For each suffix index i (global position P+i): (rank, local row).

    Built by walking every rank's plan, i.e. the restore step of Sec. 2.1
    (outputs put back in original order).
    """
    rank_of = [-1] * R
    row_of = [-1] * R
    for r in range(C):
        plan = shard_plan_fast(P, R, C, r)
        for local, pos in enumerate(plan["row_pos"]):
            i = pos - P
            if rank_of[i] != -1:
                raise AssertionError("two ranks claim one token")
            rank_of[i] = r
            row_of[i] = local
    return rank_of, row_of


def kv_shard_ranges(P: int, R: int, C: int, shard: int):
    """Global key positions of the suffix tokens rank ``shard`` holds.

    Under the zigzag split, rank ``shard`` projects the K/V of exactly its own
    two chunks; pass-KV schemes compute partials against one such shard at a
    time.  Returned as half-open ranges, empty ones dropped.
    """
    s = _chunk_len(R, C)
    out = []
    for chunk_id in (shard, 2 * C - 1 - shard):
        lo = chunk_id * s
        hi = min(R, lo + s)
        if hi > lo:
            out.append((P + lo, P + hi))
    return out
