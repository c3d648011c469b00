"""Oracle: causal attention, partial attention with log-sum-exp, and the merge.

TEST INFRASTRUCTURE ONLY (see ``oracle/__init__.py``).

Definition followed (paper Sec. 2.1, the display equation of causal
self-attention): Attn(Q, K, V) = softmax(Q K^T / sqrt(d_h) + M) V with
M_ij = 0 when key j is at or before query i and -inf otherwise.  Everything
is evaluated in float64 from the exact bf16 inputs (bf16 -> float64 is
exact).  One numpy matmul per (head, row block) is the only library step; no
tiling over keys, no online rescaling, no reordering of the definition.

Readings where the paper is silent (it never splits the softmax):

* A *partial* is the same attention restricted to a subset S of the keys.
  It is reported as the normalised output O = sum_{j in S} e^{x_j - LSE} v_j
  together with LSE = ln sum_{j in S} e^{x_j}, natural log, x_j including the
  1/sqrt(d_h) scale.  A row with no visible key in S has LSE = -inf, O = 0.
* Grouped-query attention (Llama-3 shapes): query head h reads KV head
  floor(h / (Hq / Hkv)).
* The positions of the keys: a cached prefix of P tokens occupies positions
  0..P-1, the uncached suffix P..P+R-1 (Sec. 2.2, L = P + R).
* A paged prefix cache stores the prefix as fixed-size blocks of tokens
  addressed through a block table (Sec. 7.1: a trie node is one cache block;
  Sec. 8: workers keep physical KV blocks); the block size is not given and
  is 16 tokens here.
"""

from __future__ import annotations

import math

import numpy as np

BLOCK_TOKENS = 16


def _f64(x):
    if hasattr(x, "detach"):          # a torch tensor: exact widening to float64
        x = x.detach().to("cpu").double().numpy()
    return np.asarray(x, dtype=np.float64)


def attend(q, q_pos, k, v, k_pos, scale=None):
    """Attention of query rows over a set of keys under the causal rule.

    q: [n, Hq, D]; q_pos: [n] global positions of the queries.
    k, v: [m, Hkv, D]; k_pos: [m] global positions of the keys.
    Row i, head h sees the keys j with k_pos[j] <= q_pos[i] (the mask M of
    Sec. 2.1, diagonal included) and reads KV head h // (Hq // Hkv).
    Returns (O [n, Hq, D], LSE [n, Hq]) in float64; rows that see no key get
    O = 0 and LSE = -inf.
    """
    q = _f64(q)
    k = _f64(k)
    v = _f64(v)
    q_pos = np.asarray(q_pos, dtype=np.int64)
    k_pos = np.asarray(k_pos, dtype=np.int64)
    n, Hq, D = q.shape
    m = k.shape[0]
    Hkv = k.shape[1] if m else max(1, Hq)
    if scale is None:
        scale = 1.0 / math.sqrt(D)
    if m and Hq % Hkv:
        raise ValueError("Hq must be a multiple of Hkv")
    out = np.zeros((n, Hq, D), dtype=np.float64)
    lse = np.full((n, Hq), -np.inf, dtype=np.float64)
    if n == 0 or m == 0:
        return out, lse
    group = Hq // Hkv
    rows_per_block = max(1, min(256, (1 << 22) // max(1, m)))
    for h in range(Hq):
        g = h // group
        kg = k[:, g, :]
        vg = v[:, g, :]
        for b0 in range(0, n, rows_per_block):
            b1 = min(n, b0 + rows_per_block)
            x = (q[b0:b1, h, :] @ kg.T) * scale                    # logits
            visible = k_pos[None, :] <= q_pos[b0:b1, None]          # causal mask
            x = np.where(visible, x, -np.inf)
            mx = x.max(axis=1)
            live = np.isfinite(mx)
            if not live.any():
                continue
            xl = x[live]
            e = np.exp(xl - mx[live, None])                         # softmax numerators
            denom = e.sum(axis=1)
            out_rows = (e @ vg) / denom[:, None]
            idx = np.arange(b0, b1)[live]
            out[idx, h, :] = out_rows
            lse[idx, h] = mx[live] + np.log(denom)
    return out, lse


def full_causal_attention(q, k, v, scale=None):
    """Single-rank causal attention over a whole sequence (Sec. 2.1).

    q: [L, Hq, D]; k, v: [L, Hkv, D]; token t sits at position t.
    """
    L = _f64(q).shape[0]
    pos = np.arange(L, dtype=np.int64)
    return attend(q, pos, k, v, pos, scale)


def lse_merge(outs, lses):
    """Combine partials over disjoint key subsets into the attention over
    their union.

    With S = S_1 u ... u S_n disjoint, sum_{j in S} e^{x_j} = sum_i e^{LSE_i},
    so LSE = ln sum_i e^{LSE_i} and O = sum_i e^{LSE_i - LSE} O_i.  Partials
    with LSE_i = -inf carry no keys and get weight 0; a row with no keys in
    any partial stays O = 0, LSE = -inf.  The largest LSE_i is factored out
    before exponentiating.
    """
    outs = [_f64(o) for o in outs]
    lses = [_f64(s) for s in lses]
    stack = np.stack(lses)                                  # [n, ...]
    mx = stack.max(axis=0)
    live = np.isfinite(mx)
    safe_mx = np.where(live, mx, 0.0)
    w = np.where(np.isfinite(stack), np.exp(stack - safe_mx), 0.0)
    total = w.sum(axis=0)
    lse = np.where(live, safe_mx + np.log(np.where(live, total, 1.0)), -np.inf)
    out = np.zeros_like(outs[0])
    for wi, oi in zip(w, outs):
        coef = np.where(live, wi / np.where(live, total, 1.0), 0.0)
        out += coef[..., None] * oi
    return out, lse


def gather_paged(cache, block_table, length, block_tokens=BLOCK_TOKENS):
    """Logical prefix rows 0..length-1 from a paged cache.

    cache: [n_blocks, block_tokens, Hkv, D]; logical token j lives in physical
    block block_table[j // block_tokens], slot j % block_tokens.

    Reading (the paper says nothing of invalid entries): an entry outside
    [0, n_blocks) names no block of the cache, so nothing is read through it
    and the rows of its tokens are zeros -- in attention, keys of logit 0 and
    values 0.
    """
    cache = _f64(cache)
    table = np.asarray(block_table, dtype=np.int64)
    zero = np.zeros(cache.shape[2:], dtype=np.float64)
    rows = []
    for j in range(length):
        blk = table[j // block_tokens]
        rows.append(cache[blk, j % block_tokens] if 0 <= blk < cache.shape[0] else zero)
    if not rows:
        return np.zeros((0,) + cache.shape[2:], dtype=np.float64)
    return np.stack(rows)


def rank_partial(q, row_pos, P, k_new, v_new, k_cache=None, v_cache=None,
                 block_table=None, include_prefix=True, suffix_ranges=None,
                 scale=None):
    """One rank's partial attention (Sec. 2.1 and 2.2).

    q: [n_rows, Hq, D], the rank's query rows at global positions ``row_pos``.
    k_new, v_new: [R, Hkv, D] suffix K/V in original order (position P + i).
    k_cache, v_cache, block_table: the paged prefix (positions 0..P-1).
    include_prefix: the rows attend to all P prefix keys.
    suffix_ranges: None = every suffix key (the all-gathered view);
      otherwise a list of half-open global-position ranges of suffix keys.
    Returns (O, LSE) over the selected keys under the causal rule.
    """
    k_new = _f64(k_new)
    v_new = _f64(v_new)
    R = k_new.shape[0]
    ks, vs, ps = [], [], []
    if include_prefix and P > 0:
        ks.append(gather_paged(k_cache, block_table, P))
        vs.append(gather_paged(v_cache, block_table, P))
        ps.append(np.arange(P, dtype=np.int64))
    if suffix_ranges is None:
        suffix_ranges = [(P, P + R)]
    for lo, hi in suffix_ranges:
        lo_i = max(lo - P, 0)
        hi_i = min(hi - P, R)
        if hi_i > lo_i:
            ks.append(k_new[lo_i:hi_i])
            vs.append(v_new[lo_i:hi_i])
            ps.append(np.arange(P + lo_i, P + hi_i, dtype=np.int64))
    q = _f64(q)
    if not ks:
        n, Hq, D = q.shape
        return np.zeros((n, Hq, D)), np.full((n, Hq), -np.inf)
    return attend(q, row_pos, np.concatenate(ks), np.concatenate(vs),
                  np.concatenate(ps), scale)
