"""Seeded synthetic inputs for the CP prefill-attention workloads.

Shared by the tests, ``bench.py`` and the scripts that write stored expected
values.  It only draws and lays out random data (and the per-request shape
recipe of the heterogeneous batch); it computes nothing of the attention,
the zigzag plan or the merge, so the oracle and the HIP path share no
arithmetic through it.

Draw order for one attention problem: Q, then K, then V, then (prefix hit)
prefix K, prefix V, then the block-table permutation; all from one
``torch.Generator`` seeded with the given seed, as float32 N(0, 1) times
``data_scale`` rounded to bf16 (round-to-nearest-even, torch's conversion).
"""

from __future__ import annotations

import math
from dataclasses import dataclass, field

import numpy as np
import torch

BLOCK_TOKENS = 16          # tokens per paged KV-cache block
HEAD_DIM = 128


@dataclass(frozen=True)
class Workload:
    """Shape of one named workload (Llama-3 attention shapes)."""
    name: str
    L: int                  # total context length of the (single) request
    P: int                  # cached prefix length (multiple of BLOCK_TOKENS)
    C: int                  # CP degree
    Hq: int
    Hkv: int
    D: int = HEAD_DIM
    data_scale: float = 1.0  # Q/K/V are N(0,1) * data_scale
    seed: int = 1000
    note: str = field(default="", compare=False)

    @property
    def R(self) -> int:
        return self.L - self.P


WORKLOADS = {
    "tiny_1k_c2": Workload("tiny_1k_c2", L=1024, P=0, C=2, Hq=8, Hkv=2,
                           data_scale=1.0 / math.sqrt(128.0), seed=1001,
                           note="1024 tokens, C=2, 8/2 heads, N(0,1)/sqrt(128) data"),
    "llama3_8b_32k_c4": Workload("llama3_8b_32k_c4", L=32768, P=0, C=4, Hq=32, Hkv=8,
                                 seed=1002, note="Llama-3-8B layer, 32K prompt, C=4"),
    "prefix_hit_64k_c2": Workload("prefix_hit_64k_c2", L=65536, P=49152, C=2, Hq=32,
                                  Hkv=8, seed=1003,
                                  note="48K cached prefix (paged, block 16) + 16K new, C=2"),
    "llama3_70b_128k_c8": Workload("llama3_70b_128k_c8", L=131072, P=0, C=8, Hq=64,
                                   Hkv=8, seed=1004, note="Llama-3-70B layer, 128K prompt, C=8"),
}


def generator(seed: int, device="cpu") -> torch.Generator:
    g = torch.Generator(device=device)
    g.manual_seed(int(seed))
    return g


def randn_bf16(gen, shape, scale=1.0, device="cpu") -> torch.Tensor:
    x = torch.randn(*shape, generator=gen, dtype=torch.float32, device=device)
    if scale != 1.0:
        x = x * scale
    return x.to(torch.bfloat16)


def qkv(gen, n_q, n_kv, Hq, Hkv, D=HEAD_DIM, scale=1.0, device="cpu"):
    """Q [n_q, Hq, D], K and V [n_kv, Hkv, D], bf16, drawn in that order."""
    q = randn_bf16(gen, (n_q, Hq, D), scale, device)
    k = randn_bf16(gen, (n_kv, Hkv, D), scale, device)
    v = randn_bf16(gen, (n_kv, Hkv, D), scale, device)
    return q, k, v


@dataclass
class PagedPrefix:
    k_logical: torch.Tensor   # [P, Hkv, D] prefix keys in token order
    v_logical: torch.Tensor
    block_table: torch.Tensor  # int32 [P / 16], physical block of each logical block
    k_cache: torch.Tensor     # [n_blocks, 16, Hkv, D]
    v_cache: torch.Tensor


def paged_prefix(gen, P, Hkv, D=HEAD_DIM, scale=1.0, spare_blocks=0, device="cpu",
                 pool=None) -> PagedPrefix:
    """A cached prefix of P tokens scattered into a paged pool.

    The physical block of each logical block comes from a seeded random
    permutation of the pool, so the gather through the block table is not an
    identity.  With ``pool=(k_cache, v_cache, free_ids)`` the blocks are taken
    from an existing shared pool (heterogeneous batches) instead.
    """
    if P % BLOCK_TOKENS:
        raise ValueError("prefix length must be a multiple of the block size")
    nb = P // BLOCK_TOKENS
    k_log = randn_bf16(gen, (P, Hkv, D), scale, device)
    v_log = randn_bf16(gen, (P, Hkv, D), scale, device)
    if pool is None:
        total = nb + spare_blocks
        perm = torch.randperm(total, generator=gen, device=device)
        table = perm[:nb].to(torch.int32)
        # Unused pool blocks hold unrelated finite data, never read.
        k_cache = randn_bf16(gen, (total, BLOCK_TOKENS, Hkv, D), scale, device)
        v_cache = randn_bf16(gen, (total, BLOCK_TOKENS, Hkv, D), scale, device)
    else:
        k_cache, v_cache, free_ids = pool
        table = free_ids[:nb].to(torch.int32)
    if nb:
        idx = table.long()
        k_cache[idx] = k_log.view(nb, BLOCK_TOKENS, Hkv, D)
        v_cache[idx] = v_log.view(nb, BLOCK_TOKENS, Hkv, D)
    return PagedPrefix(k_log, v_log, table, k_cache, v_cache)


# --- heterogeneous request mix ---------------------------------------------

HETERO_REQUESTS = 64
HETERO_MEDIAN = 2048
HETERO_SIGMA = 1.16
HETERO_MIN, HETERO_MAX = 256, 131072
HETERO_PREFIXED = 19           # round(0.3 * 64) requests carry a cached prefix
HETERO_TOTAL = 256 * 1024      # the mix's stated total, about 256K tokens
HETERO_LONG = 32768            # a request this long or longer is in the long bucket
# The seed of the mix: the first seed from 1005 on whose draw totals within
# 5% of HETERO_TOTAL and holds at least one request in the long bucket
# (tests/test_synth.py checks the rule against the seeds before it).
HETERO_SEED = 1012


def hetero_requests(seed=HETERO_SEED, n=HETERO_REQUESTS, median=HETERO_MEDIAN,
                    sigma=HETERO_SIGMA, n_prefixed=HETERO_PREFIXED):
    """[(L, P)] for a lognormal length mix; some requests hit a prefix.

    Lengths: round(exp(ln(median) + sigma * z)), clipped to [256, 131072].
    Prefix: P = 16 * floor(u * L / 16), u ~ U(0.2, 0.8), on ``n_prefixed``
    randomly chosen requests.  Each request's CP degree is a policy choice
    made by the caller.
    """
    rng = np.random.default_rng(seed)
    z = rng.standard_normal(n)
    L = np.clip(np.round(np.exp(math.log(median) + sigma * z)), HETERO_MIN, HETERO_MAX).astype(np.int64)
    pref = np.zeros(n, dtype=np.int64)
    chosen = rng.choice(n, size=n_prefixed, replace=False)
    u = rng.uniform(0.2, 0.8, size=n_prefixed)
    for i, ui in zip(chosen, u):
        pref[i] = BLOCK_TOKENS * int(math.floor(ui * int(L[i]) / BLOCK_TOKENS))
    return [(int(L[i]), int(pref[i])) for i in range(n)]
