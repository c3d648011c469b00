"""GPU parity at the full workload sizes, in both launch configurations that
bench.py times: its default step -- one cp_attn_partial launch of the rank's
rows against every key they see in the all-gathered KV (and the paged
prefix), whose stores put every row at its place in the original order
(CP_OUT_SEQUENCE) -- and its --mode passkv step, one launch with the rank's C
pass-KV partials (plus a prefix-only partial when a prefix is cached), merged
and restored by cp_attn_merge with the rank's plan.

The oracle recomputes seeded samples of rows (every head): the first and
last rows of each chunk, rows on both sides of 64- and 256-row boundaries,
random rows, and one seeded row in every 32-row block of each chunk (every
8th block at the largest size) -- a wave owns 32 or 48 consecutive
positions of one head (256- or 384-row workgroups), so every wave of every
work item of the launch meets the oracle (at the largest size, where an
item holds 32 or 48 positions of eight heads, one item in five to eight).
Both steps' rows are compared with it.
Properties that hold at any size are checked on every row: the two steps
agree, no NaN anywhere, and every restored row is written exactly once.
"""

import os

import numpy as np
import pytest
import torch

import synth
from oracle import attention as oatt
from oracle import plan as oplan
from paper_2609_04774_amd import cpattn as cp
from paper_2609_04774_amd import placement as pl

from gpu_cases import DEV, LSE_TOL, O_TOL, compare, f64

pytestmark = pytest.mark.gpu


def _inputs(w, rank):
    """Rank `rank`'s queries plus the whole suffix K/V (and paged prefix),
    drawn on the GPU from the workload's seed."""
    g = synth.generator(w.seed + 100 * rank, device="cuda")
    plan, rows = cp.shard_plan(w.P, w.R, w.C, rank)
    q = synth.randn_bf16(g, (plan.n_rows, w.Hq, w.D), w.data_scale, device="cuda")
    k = synth.randn_bf16(g, (w.R, w.Hkv, w.D), w.data_scale, device="cuda")
    v = synth.randn_bf16(g, (w.R, w.Hkv, w.D), w.data_scale, device="cuda")
    pre = synth.paged_prefix(g, w.P, w.Hkv, w.D, w.data_scale, spare_blocks=64, device="cuda") if w.P else None
    return plan, rows, q, k, v, pre


def _run_passkv(w, plan, q, k, v, pre):
    """bench.py --mode passkv: pass-KV partials (+ prefix partial) and the merge."""
    n_parts = w.C + (1 if w.P else 0)
    o = torch.empty((n_parts, plan.n_rows, w.Hq, w.D), dtype=torch.float32, device=DEV)
    l = torch.empty((n_parts, plan.n_rows, w.Hq), dtype=torch.float32, device=DEV)
    kc, vc, bt = (pre.k_cache, pre.v_cache, pre.block_table) if pre else (None, None, None)
    descs = []
    i = 0
    if w.P:
        descs.append(cp.make_desc(plan, q, k, v, o[i], l[i], kc, vc, bt, include_prefix=True,
                                  kv_rank=cp.CP_KV_NONE))
        i += 1
    for s in range(w.C):
        descs.append(cp.make_desc(plan, q, k, v, o[i], l[i], kc, vc, bt, include_prefix=False, kv_rank=s))
        i += 1
    ws = torch.empty(max(256, cp.workspace_size(descs, w.Hq, w.Hkv)), dtype=torch.uint8, device=DEV)
    cp.attn_partial(descs, w.Hq, w.Hkv, ws)
    out = torch.full((w.R, w.Hq, w.D), float("nan"), dtype=torch.float32, device=DEV)
    out_lse = torch.full((w.R, w.Hq), float("nan"), dtype=torch.float32, device=DEV)
    cp.attn_merge([o[j] for j in range(n_parts)], [l[j] for j in range(n_parts)], out, out_lse, restore=plan)
    torch.cuda.synchronize()
    return out, out_lse


def _run_allgather(w, plan, q, k, v, pre):
    """bench.py's default step: one partial over all visible keys, its rows
    stored straight into their places in sequence order."""
    kc, vc, bt = (pre.k_cache, pre.v_cache, pre.block_table) if pre else (None, None, None)
    out = torch.full((w.R, w.Hq, w.D), float("nan"), dtype=torch.float32, device=DEV)
    out_lse = torch.full((w.R, w.Hq), float("nan"), dtype=torch.float32, device=DEV)
    d = cp.make_desc(plan, q, k, v, out, out_lse, kc, vc, bt, include_prefix=True, kv_rank=cp.CP_KV_ALL,
                     out_order=cp.CP_OUT_SEQUENCE)
    ws = torch.empty(max(256, cp.workspace_size([d], w.Hq, w.Hkv)), dtype=torch.uint8, device=DEV)
    cp.attn_partial([d], w.Hq, w.Hkv, ws)
    torch.cuda.synchronize()
    return out, out_lse


def _sample_rows(plan, n_random, seed, block_every=1):
    rng = np.random.default_rng(seed)
    picks = set()
    for c in plan.chunk:
        lo, n = c.local_offset, c.q_len
        if n == 0:
            continue
        for r in (0, 1, 63, 64, 255, 256, n - 2, n - 1):
            if 0 <= r < n:
                picks.add(lo + r)
        for b0 in range(0, n, 32 * block_every):
            picks.add(lo + b0 + int(rng.integers(0, min(32, n - b0))))
    picks.update(int(x) for x in rng.choice(plan.n_rows, size=min(n_random, plan.n_rows), replace=False))
    return np.array(sorted(picks), dtype=np.int64)


def _check_workload(name, rank, n_random, block_every=1):
    w = synth.WORKLOADS[name]
    plan, rows, q, k, v, pre = _inputs(w, rank)
    ref_plan = oplan.shard_plan_fast(w.P, w.R, w.C, rank)
    assert rows.tolist() == ref_plan["row_pos"], "C-ABI plan differs from the oracle's"
    out_ag, lse_ag = _run_allgather(w, plan, q, k, v, pre)
    out, out_lse = _run_passkv(w, plan, q, k, v, pre)
    # Every restored row of this rank is written, nothing else is.
    sel = torch.as_tensor(rows - w.P, device=DEV)
    written = torch.zeros(w.R, dtype=torch.bool, device=DEV)
    written[sel] = True
    for o_, l_ in ((out_ag, lse_ag), (out, out_lse)):
        assert not torch.isnan(o_[sel]).any() and not torch.isnan(l_[sel]).any()
        assert torch.isnan(l_[~written]).all(), "merge wrote rows of another rank"
    # Merged pass-KV partials == the all-gathered partial, on every row.
    assert float((out_ag[sel] - out[sel]).abs().max()) <= O_TOL
    assert float((lse_ag[sel] - out_lse[sel]).abs().max()) <= LSE_TOL
    # Sampled rows against the fp64 oracle.
    pick = _sample_rows(plan, n_random, w.seed, block_every)
    print(f"{name} rank {rank}: {len(pick)} of {plan.n_rows} rows checked against the oracle", flush=True)
    pos = rows[pick]
    kk, vv = f64(k), f64(v)
    kc = vc = bt = None
    if pre is not None:
        kc, vc = f64(pre.k_cache), f64(pre.v_cache)
        bt = pre.block_table.cpu().numpy().astype(np.int64)
    qq = f64(q[torch.as_tensor(pick, device=DEV)])
    O_ref, L_ref = oatt.rank_partial(qq, pos, w.P, kk, vv, kc, vc, bt)
    at = torch.as_tensor(pos - w.P, device=DEV)
    compare(f64(out_ag[at]), f64(lse_ag[at]), O_ref, L_ref, f"{name} rank {rank} all-gathered")
    return compare(f64(out[at]), f64(out_lse[at]), O_ref, L_ref, f"{name} rank {rank} pass-KV")


@pytest.fixture(params=[0, 256, 384], ids=["rows_auto", "rows256", "rows384"])
def workgroup_rows(request):
    """The launch's own choice of workgroup shape, then each shape pinned (the
    32K rank-0 shard's work list is cut in 384-row items only; the prefix-hit
    shard's, checked in its own choice of shape, is cut evenly)."""
    cp.set_workgroup_rows(request.param)
    yield request.param
    cp.set_workgroup_rows(0)


def test_llama3_8b_32k_rank0_full_size(workgroup_rows):
    _check_workload("llama3_8b_32k_c4", 0, n_random=24 if workgroup_rows == 0 else 8)


def test_llama3_8b_32k_rank3_full_size(workgroup_rows):
    _check_workload("llama3_8b_32k_c4", 3, n_random=8)


def test_prefix_hit_64k_full_size():
    _check_workload("prefix_hit_64k_c2", 0, n_random=8)
    _check_workload("prefix_hit_64k_c2", 1, n_random=4)


def test_llama3_70b_128k_rank0_full_size():
    _check_workload("llama3_70b_128k_c8", 0, n_random=2, block_every=8)


CALIBRATION = os.path.join(os.path.dirname(os.path.dirname(os.path.abspath(__file__))), "profiles",
                           "calibration_attention_llama3_8b.json")


@pytest.mark.parametrize("wg_rows", [0, 256, 384])
def test_heterogeneous_batch_one_launch(wg_rows):
    """The heterogeneous mix (64 lognormal-length requests, 19 with a cached
    prefix in one shared paged pool) plus two long requests (40K tokens, and
    70K with a 16K cached prefix), each request at the CP degree the placement
    cost prefers over the calibrated prefill-time model: every (request, rank)
    shard in one launch, degrees 1, 2, 4 and 8 mixed."""
    Hq, Hkv, D, B = 32, 8, 128, synth.BLOCK_TOKENS
    model = pl.model_from_calibration(CALIBRATION)
    reqs = synth.hetero_requests() + [(40000, 0), (70000, 16000)]
    degrees = pl.choose_degrees(reqs, "cost", model)
    print("C histogram", {C: degrees.count(C) for C in pl.DEGREES}, flush=True)
    assert set(degrees) == {1, 2, 4, 8}
    total_blocks = sum(P // B for _, P in reqs) + 32
    g = synth.generator(2005, device="cuda")
    k_pool = synth.randn_bf16(g, (total_blocks, B, Hkv, D), device="cuda")
    v_pool = synth.randn_bf16(g, (total_blocks, B, Hkv, D), device="cuda")
    free = torch.randperm(total_blocks, generator=g, device="cuda")
    used = 0
    keep, descs, checks = [], [], []
    for ri, ((L, P), C) in enumerate(zip(reqs, degrees)):
        R = L - P
        q_full, k, v = synth.qkv(g, R, R, Hq, Hkv, D, device="cuda")
        pre = None
        if P:
            pre = synth.paged_prefix(g, P, Hkv, D, device="cuda", pool=(k_pool, v_pool, free[used:used + P // B]))
            used += P // B
        for r in range(C):
            plan, rows = cp.shard_plan(P, R, C, r)
            if plan.n_rows == 0:
                continue
            q = q_full[torch.as_tensor(rows - P, device=DEV)].contiguous()
            o = torch.empty((plan.n_rows, Hq, D), dtype=torch.float32, device=DEV)
            l = torch.empty((plan.n_rows, Hq), dtype=torch.float32, device=DEV)
            descs.append(cp.make_desc(plan, q, k, v, o, l, k_pool, v_pool,
                                      pre.block_table if pre else None, include_prefix=True))
            keep.append((q, o, l))
            checks.append((ri, C, P, R, r, plan, rows, q, k, v, pre, o, l))
    try:
        cp.set_workgroup_rows(wg_rows)
        ws = torch.empty(max(256, cp.workspace_size(descs, Hq, Hkv)), dtype=torch.uint8, device=DEV)
        cp.attn_partial(descs, Hq, Hkv, ws)
        torch.cuda.synchronize()
    finally:
        cp.set_workgroup_rows(0)
    kp, vp = f64(k_pool), f64(v_pool)
    rng = np.random.default_rng(7)
    n_rows = 0
    for ri, C, P, R, r, plan, rows, q, k, v, pre, o, l in checks:
        assert not torch.isnan(o).any() and not torch.isnan(l).any()
        ends = [c.local_offset + e for c in plan.chunk if c.q_len for e in (0, c.q_len - 1)]
        pick = np.unique(np.concatenate([ends, rng.integers(0, plan.n_rows, size=1)]))
        pos = rows[pick]
        bt = pre.block_table.cpu().numpy().astype(np.int64) if pre else None
        sel = torch.as_tensor(pick, device=DEV)
        O_ref, L_ref = oatt.rank_partial(f64(q[sel]), pos, P, f64(k), f64(v), kp if pre else None,
                                         vp if pre else None, bt)
        compare(f64(o[sel]), f64(l[sel]), O_ref, L_ref, f"request {ri} (C={C}) rank {r}")
        n_rows += len(pick)
    print(f"{len(checks)} shards, {n_rows} rows checked against the oracle", flush=True)
