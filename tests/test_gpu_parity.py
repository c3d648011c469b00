"""GPU parity: the HIP path (through the C ABI) against the fp64 oracle.

Small cases compare every output element; the full-size workloads compare
seeded samples of rows (all heads) that the oracle computes one by one, and
check properties that hold at any size.
"""

import math

import numpy as np
import pytest
import torch

import synth
from oracle import attention as oatt
from oracle import plan as oplan
from paper_2609_04774_amd import cpattn as cp

import gpu_cases as gc
from gpu_cases import Problem, compare, f64, DEV

pytestmark = pytest.mark.gpu


@pytest.fixture(autouse=True, params=[256, 384], ids=["rows256", "rows384"])
def workgroup_rows(request):
    """Every case runs on both attention kernel shapes (two or three 16-row
    blocks per wave), pinned for the test and released after it."""
    cp.set_workgroup_rows(request.param)
    yield request.param
    cp.set_workgroup_rows(0)


def _restore_all_ranks(prob, kv_mode="allgather"):
    """Every rank's partial(s), merged and restored into original order by
    cp_attn_merge; returns (O [R, Hq, D], LSE [R, Hq]) on the GPU."""
    R, Hq = prob.R, prob.Hq
    O = torch.full((R, Hq, 128), float("nan"), dtype=torch.float32, device=DEV)
    LSE = torch.full((R, Hq), float("nan"), dtype=torch.float32, device=DEV)
    for r in range(prob.C):
        if kv_mode == "allgather":
            o, lse, plan, _ = prob.gpu_rank(r)
            parts = [(o, lse)]
        else:
            parts = []
            if prob.P:
                o, lse, plan, _ = prob.gpu_rank(r, kv_rank=cp.CP_KV_NONE, include_prefix=True)
                parts.append((o, lse))
            for s in range(prob.C):
                o, lse, plan, _ = prob.gpu_rank(r, kv_rank=s, include_prefix=False)
                parts.append((o, lse))
        if plan.n_rows == 0:
            continue
        cp.attn_merge([p[0] for p in parts], [p[1] for p in parts], O, LSE, restore=plan)
    torch.cuda.synchronize()
    return O, LSE


def _oracle_full(prob):
    d = prob.np()
    if prob.P:
        kp = oatt.gather_paged(d["kc"], d["bt"], prob.P)
        vp = oatt.gather_paged(d["vc"], d["bt"], prob.P)
        k = np.concatenate([kp, d["k"]])
        v = np.concatenate([vp, d["v"]])
        q = np.concatenate([np.zeros((prob.P,) + d["q"].shape[1:]), d["q"]])
        O, L = oatt.full_causal_attention(q, k, v)
        return O[prob.P:], L[prob.P:]
    return oatt.full_causal_attention(d["q"], d["k"], d["v"])


def test_tiny_workload_both_ranks_restored():
    """1024 tokens, C=2, 8/2 heads, N(0,1)/sqrt(128): both ranks, restored."""
    w = synth.WORKLOADS["tiny_1k_c2"]
    prob = Problem(w.L, w.P, w.C, w.Hq, w.Hkv, w.seed, data_scale=w.data_scale)
    O, L = _restore_all_ranks(prob)
    Or, Lr = _oracle_full(prob)
    compare(f64(O), f64(L), Or, Lr, "tiny allgather restore")


def test_tiny_workload_pass_kv_partials_merged():
    w = synth.WORKLOADS["tiny_1k_c2"]
    prob = Problem(w.L, w.P, w.C, w.Hq, w.Hkv, w.seed, data_scale=w.data_scale)
    O, L = _restore_all_ranks(prob, kv_mode="passkv")
    Or, Lr = _oracle_full(prob)
    compare(f64(O), f64(L), Or, Lr, "tiny pass-KV merge")


# (L, P, C, Hq, Hkv, data_scale, q_scale, seed): ragged suffixes, R < 2C,
# GQA ratios 1/2/4/8/16, prefixes that are not tile multiples, unscaled and
# peaky logits.
SHAPES = [
    (1000, 0, 2, 8, 2, 1.0, 1.0, 11),
    (777, 0, 4, 4, 4, 1.0, 1.0, 12),
    (5, 0, 4, 8, 1, 1.0, 1.0, 13),
    (300, 48, 2, 32, 8, 1.0, 1.0, 14),
    (700, 208, 8, 16, 2, 1.0, 8.0, 15),
    (513, 0, 1, 8, 8, 1.0, 1.0, 16),
    (640, 80, 3, 16, 1, 1.0, 1.0, 17),
    (400, 16, 2, 24, 8, 1.0, 1.0, 18),
    (1025, 0, 2, 64, 8, 1.0, 1.0, 19),
    (333, 0, 2, 6, 2, 1.0 / math.sqrt(128.0), 1.0, 20),
]


@pytest.mark.parametrize("L,P,C,Hq,Hkv,ds,qs,seed", SHAPES)
def test_every_rank_matches_oracle(L, P, C, Hq, Hkv, ds, qs, seed):
    prob = Problem(L, P, C, Hq, Hkv, seed, data_scale=ds, q_scale=qs)
    for r in range(C):
        o, lse, plan, rows = prob.gpu_rank(r)
        ref = oplan.shard_plan_fast(P, L - P, C, r)
        assert rows.tolist() == ref["row_pos"]
        Or, Lr = prob.oracle_rank(r)
        compare(f64(o), f64(lse), Or, Lr, f"rank {r}")


@pytest.mark.parametrize("L,P,C,Hq,Hkv,seed", [(1000, 0, 2, 8, 2, 21), (600, 96, 4, 8, 2, 22),
                                                (131, 32, 8, 4, 1, 23)])
def test_pass_kv_and_prefix_only_partials(L, P, C, Hq, Hkv, seed):
    """Each kv_rank shard (some rows see nothing: LSE = -inf, O = 0) and the
    prefix-only partial match the oracle element by element."""
    prob = Problem(L, P, C, Hq, Hkv, seed)
    for r in range(C):
        for s in range(C):
            o, lse, _, _ = prob.gpu_rank(r, kv_rank=s, include_prefix=(s == 0))
            Or, Lr = prob.oracle_rank(r, kv_rank=s, include_prefix=(s == 0))
            compare(f64(o), f64(lse), Or, Lr, f"rank {r} shard {s}")
        if P:
            o, lse, _, _ = prob.gpu_rank(r, kv_rank=cp.CP_KV_NONE, include_prefix=True)
            Or, Lr = prob.oracle_rank(r, kv_rank=cp.CP_KV_NONE, include_prefix=True)
            compare(f64(o), f64(lse), Or, Lr, f"rank {r} prefix only")


# out_order = CP_OUT_SEQUENCE: each rank's rows are stored at their suffix
# index of one R-row output by the attention itself (the restore of Sec. 2.1,
# no merge).  (8392, 8192) splits its key walks, so the split-merge kernel's
# stores are covered too.
@pytest.mark.parametrize("L,P,C,Hq,Hkv,seed", [(1000, 0, 2, 8, 2, 81), (777, 0, 4, 4, 4, 82),
                                                (640, 80, 3, 16, 1, 83), (8392, 8192, 2, 8, 2, 84),
                                                (5, 0, 4, 8, 1, 85)])
def test_sequence_order_output(L, P, C, Hq, Hkv, seed):
    prob = Problem(L, P, C, Hq, Hkv, seed)
    dv, R = prob.dev(), prob.R
    O, LSE = gc.alloc_out(R, Hq)
    O2, LSE2 = gc.alloc_out(R, Hq)
    together = []
    for r in range(C):
        plan, rows = cp.shard_plan(P, R, C, r)
        if plan.n_rows == 0:
            continue
        q = dv["q"][torch.as_tensor(rows - P, device=DEV)].contiguous()
        # One launch per rank, as its local-order launch: the same work
        # decomposition, so the stored rows must be the same bits.
        d = cp.make_desc(plan, q, dv["k"], dv["v"], O, LSE, dv.get("kc"), dv.get("vc"), dv.get("bt"),
                         out_order=cp.CP_OUT_SEQUENCE)
        gc.run_partials([d], Hq, Hkv)
        o, lse, _, _ = prob.gpu_rank(r)
        at = torch.as_tensor(rows - P, device=DEV)
        assert torch.equal(O[at], o) and torch.equal(LSE[at], lse), f"rank {r}"
        together.append(cp.make_desc(plan, q, dv["k"], dv["v"], O2, LSE2, dv.get("kc"), dv.get("vc"),
                                     dv.get("bt"), out_order=cp.CP_OUT_SEQUENCE))
    # Every rank in one launch, into one output: every row written once, and
    # the whole output is single-rank causal attention (Sec. 2.1).
    gc.run_partials(together, Hq, Hkv)
    Or, Lr = _oracle_full(prob)
    compare(f64(O[:R]), f64(LSE[:R]), Or, Lr, "per-rank launches")
    compare(f64(O2[:R]), f64(LSE2[:R]), Or, Lr, "one launch")


@pytest.mark.parametrize("L,P,C,seed", [(1100, 0, 2, 91), (1300, 256, 2, 92), (900, 0, 1, 93)])
def test_exact_redo_on_every_tile(L, P, C, seed):
    """Logits that rise by more than 2^12 (in base-2 units) from one 32-key
    tile to the next for the query heads of KV head 0: every tile's
    probabilities pass the running max's bound, so each tile is redone
    exactly (O and both row sums rescaled).  KV head 1's logits fall instead
    (the first tile's max holds for the whole walk)."""
    Hq, Hkv = 8, 2
    prob = Problem(L, P, C, Hq, Hkv, seed)
    pos = torch.arange(prob.R, dtype=torch.float32) * 0.125
    k = prob.k.float()
    k[:, 0, 0] = pos
    k[:, 1, 0] = -pos
    q = prob.q.float()
    q[:, :, 0] = 40.0          # 40 * 0.125 * 32 / sqrt(128) * log2(e) = 20.4 per tile
    prob.k = k.to(torch.bfloat16)
    prob.q = q.to(torch.bfloat16)
    # The premise, on the host: for the last query of KV head 0's first
    # query head, each 32-key tile's largest logit exceeds the previous
    # tile's by more than 13 in base-2 units (2^13 > 2^16 / 16 lane keys).
    d = prob.np()
    x = d["k"][:, 0, :] @ d["q"][-1, 0, :] / math.sqrt(128) / math.log(2)
    tmax = np.array([x[i:i + 32].max() for i in range(0, prob.R - 31, 32)])
    assert np.all(np.diff(tmax) > 13.0)
    for r in range(C):
        o, lse, _, _ = prob.gpu_rank(r)
        Or, Lr = prob.oracle_rank(r)
        compare(f64(o), f64(lse), Or, Lr, f"rank {r}")


# Launches with few work items, so the key walks are split into pieces of
# >= 32 tiles whose partials are merged in the workspace: a long cached
# prefix under a short suffix (the prefix-hit case), and a small-head shard
# whose long second chunk spans two suffix ranges.
@pytest.mark.parametrize("L,P,C,Hq,Hkv,seed", [(8392, 8192, 2, 8, 2, 61), (8192, 0, 8, 4, 4, 62),
                                                (4200, 3072, 1, 16, 4, 63)])
def test_split_key_walks_match_oracle(L, P, C, Hq, Hkv, seed):
    prob = Problem(L, P, C, Hq, Hkv, seed)
    for r in range(C):
        o, lse, plan, rows = prob.gpu_rank(r)
        Or, Lr = prob.oracle_rank(r)
        compare(f64(o), f64(lse), Or, Lr, f"rank {r}")
    # Pass-KV shards too: pieces of a walk over one shard's two chunks.
    for s in range(min(C, 2)):
        o, lse, _, _ = prob.gpu_rank(0, kv_rank=s, include_prefix=(s == 0))
        Or, Lr = prob.oracle_rank(0, kv_rank=s, include_prefix=(s == 0))
        compare(f64(o), f64(lse), Or, Lr, f"rank 0 shard {s}")


@pytest.mark.parametrize("L,P,C,Hq,Hkv,seed", [(400, 96, 2, 8, 2, 71), (8392, 8192, 2, 8, 2, 72)])
def test_block_table_entries_outside_the_cache_read_as_zeros(L, P, C, Hq, Hkv, seed):
    """Entries -1, n_blocks and 2^31 - 1 in the prefix's block table: the
    kernel reads nothing through them and their 16 tokens act as zero keys
    and values, as the oracle's paged gather reads them.  (400, 96): one
    walk per item; (8392, 8192): split walks over a long prefix."""
    prob = Problem(L, P, C, Hq, Hkv, seed)
    bt = prob.prefix.block_table
    n_blocks = prob.prefix.k_cache.shape[0]
    nb = P // 16
    for i, bad in zip((1, nb // 2, nb - 1), (-1, n_blocks, 2 ** 31 - 1)):
        bt[i] = bad
    for r in range(C):
        o, lse, _, _ = prob.gpu_rank(r)
        Or, Lr = prob.oracle_rank(r)
        compare(f64(o), f64(lse), Or, Lr, f"rank {r}")
    o, lse, _, _ = prob.gpu_rank(0, kv_rank=cp.CP_KV_NONE, include_prefix=True)
    Or, Lr = prob.oracle_rank(0, kv_rank=cp.CP_KV_NONE, include_prefix=True)
    compare(f64(o), f64(lse), Or, Lr, "prefix only")


def test_explicit_softmax_scale():
    prob = Problem(300, 0, 2, 8, 2, 31)
    o, lse, _, _ = prob.gpu_rank(0, scale=0.05)
    Or, Lr = prob.oracle_rank(0, scale=0.05)
    compare(f64(o), f64(lse), Or, Lr, "scale 0.05")


@pytest.mark.parametrize("n_tok,H", [(300, 6), (301, 3)])
def test_merge_kernel_matches_oracle_merge(n_tok, H):
    # (301, 3): an odd number of rows, so the last two-row group has one row.
    g = torch.Generator().manual_seed(41 + n_tok)
    for n in (1, 2, 3, 8, 16):
        outs = [torch.randn(n_tok, H, 128, generator=g) for _ in range(n)]
        lses = [torch.randn(n_tok, H, generator=g) * 4 for _ in range(n)]
        # Some partials carry no keys, and a few rows carry none anywhere.
        for i in range(0, n, 2):
            mask = torch.rand(n_tok, H, generator=g) < 0.3
            lses[i][mask] = -math.inf
            outs[i][mask] = 0.0
        for i in range(n):
            lses[i][:5] = -math.inf
            outs[i][:5] = 0.0
        Or, Lr = oatt.lse_merge([o.double().numpy() for o in outs], [s.double().numpy() for s in lses])
        od = [o.to(DEV) for o in outs]
        ld = [s.to(DEV) for s in lses]
        O = torch.empty(n_tok, H, 128, device=DEV)
        L = torch.empty(n_tok, H, device=DEV)
        cp.attn_merge(od, ld, O, L)
        Ob = torch.empty(n_tok, H, 128, dtype=torch.bfloat16, device=DEV)
        cp.attn_merge(od, ld, Ob, None)
        torch.cuda.synchronize()
        compare(f64(O), f64(L), Or, Lr, f"merge n={n}")
        # bf16 output: within half an ulp of bf16 at |O| (plus the fp32 error).
        ob = f64(Ob)
        assert np.all(np.abs(ob - Or) <= np.abs(Or) * 2.0 ** -8 + 1e-5)


def test_results_are_deterministic():
    prob = Problem(2000, 32, 2, 32, 8, 51)
    o1, l1, _, _ = prob.gpu_rank(1)
    o2, l2, _, _ = prob.gpu_rank(1)
    assert torch.equal(o1, o2) and torch.equal(l1, l2)


def test_empty_and_degenerate_launches():
    # R = 0: every rank is empty; the call is a no-op.
    plan, _ = cp.shard_plan(0, 0, 2, 0)
    o, lse = gc.alloc_out(1, 8)
    q = torch.zeros((1, 8, 128), dtype=torch.bfloat16, device=o.device)
    desc = cp.make_desc(plan, q, None, None, o, lse)
    gc.run_partials([desc], 8, 2)
    assert torch.isnan(o).all()
    # One token: it sees exactly itself, so O = v_0 and LSE = q.k/sqrt(D).
    prob = Problem(1, 0, 1, 4, 2, 61)
    o, lse, _, _ = prob.gpu_rank(0)
    Or, Lr = prob.oracle_rank(0)
    compare(f64(o), f64(lse), Or, Lr, "single token")
    assert torch.equal(o[0, 0].cpu(), prob.v[0, 0].float())
