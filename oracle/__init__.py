"""Oracle for the context-parallel (CP) prefill-attention hot path.

TEST INFRASTRUCTURE ONLY.  Only ``tests/``, ``__graft_entry__.smoke()`` and
``bench.py``'s ``cpu_baseline`` leg may import or call anything in this
package.  The product path (the HIP library and its Python binding) never
imports it, and this package imports nothing from the product.

Everything here is a plain, slow, float64 CPU restatement of what the paper
(arXiv 2609.04774, "Adaptive Context Parallelism for Production LLM
Serving") defines:

* ``attention``  -- causal scaled-dot-product attention (Sec. 2.1, the
  display equation softmax(QK^T/sqrt(d_h) + M)V with M_ij = 0 for j <= i),
  its restriction to a subset of keys (partial attention with log-sum-exp),
  the log-sum-exp merge of partials, and the paged prefix-cache gather
  (Sec. 2.2 and Sec. 7.1: a cached prefix is a sequence of cache blocks).
* ``plan``       -- the zigzag CP partition (Sec. 2.1: pad to a multiple of
  2C, split into 2C contiguous chunks, rank k holds chunks k and 2C-1-k) and
  the remaining-attention workload W(R, P) = RP + R(R+1)/2 (Sec. 2.2,
  equation "remaining-attention").
* ``cache``      -- the KV-cache steps after the attention: writing a
  request's new K/V into the block-16 paged cache (Sec. 2.2, 7.1, 8) and
  re-sharding rows between CP degrees (Sec. 6.2, 7.2).
* ``brute``      -- scalar-loop restatement used only to pin ``attention``
  on tiny inputs.

Readings taken where the paper is silent (it describes no partials, no LSE,
no GQA and no block size) are listed in each module's docstring.
"""

from .attention import (  # noqa: F401
    attend,
    full_causal_attention,
    lse_merge,
    gather_paged,
    rank_partial,
)
from .plan import shard_plan, inverse_map, remaining_workload  # noqa: F401
