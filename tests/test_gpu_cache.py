"""GPU checks of the KV-cache steps after the attention (cp_kv_writeback,
cp_repartition) against the oracle: both are row copies, so every check is
bit-exact.  The end-to-end case writes one request's K/V with the kernel and
serves a second request's prefix hit from that cache through
cp_attn_partial, compared with the fp64 oracle."""

import numpy as np
import pytest
import torch

import synth
from oracle import attention as oatt
from oracle import cache as ocache
from paper_2609_04774_amd import cpattn as cp

from gpu_cases import DEV, compare, f64

pytestmark = pytest.mark.gpu

B = synth.BLOCK_TOKENS


def _rank_rows(x, P, R, C, r):
    """Rank r's rows of a per-position tensor x [R, ...] (suffix order)."""
    _, rows = cp.shard_plan(P, R, C, r)
    return x[torch.as_tensor(rows - P, device=DEV)].contiguous()


def _request_cache(g, P, R, Hkv, D, spare=5):
    n = -(-(P + R) // B)
    table = torch.randperm(n + spare, generator=g, device=DEV)[:n].to(torch.int32).contiguous()
    kc = synth.randn_bf16(g, (n + spare, B, Hkv, D), device=DEV)
    vc = synth.randn_bf16(g, (n + spare, B, Hkv, D), device=DEV)
    return table, kc, vc


@pytest.mark.parametrize("P,R,C,Hkv", [(32, 45, 2, 2), (0, 70, 4, 1), (16, 9, 3, 8), (0, 16, 1, 2)])
def test_writeback_matches_oracle(P, R, C, Hkv):
    g = synth.generator(3000 + P + R + C, device=DEV)
    D = 128
    table, kc, vc = _request_cache(g, P, R, Hkv, D)
    k = synth.randn_bf16(g, (R, Hkv, D), device=DEV)
    v = synth.randn_bf16(g, (R, Hkv, D), device=DEV)
    want_k, want_v = f64(kc), f64(vc)
    tab = table.cpu().numpy()
    for r in range(C):
        plan, _ = cp.shard_plan(P, R, C, r)
        kr, vr = _rank_rows(k, P, R, C, r), _rank_rows(v, P, R, C, r)
        cp.kv_writeback(plan, kr, vr, kc, vc, table)
        want_k = ocache.rank_writeback(want_k, tab, P, R, C, r, f64(kr))
        want_v = ocache.rank_writeback(want_v, tab, P, R, C, r, f64(vr))
    torch.cuda.synchronize()
    assert np.array_equal(f64(kc), want_k)
    assert np.array_equal(f64(vc), want_v)


def test_writeback_skips_entries_outside_the_cache():
    g = synth.generator(3100, device=DEV)
    P, R, C, Hkv, D = 0, 64, 1, 2, 128
    table, kc, vc = _request_cache(g, P, R, Hkv, D, spare=0)
    n_blocks = kc.shape[0]
    bad = table.clone()
    bad[2] = n_blocks          # logical block 2 (positions 32..47) points past the cache
    bad[3] = -1
    k = synth.randn_bf16(g, (R, Hkv, D), device=DEV)
    before_k, before_v = kc.clone(), vc.clone()
    plan, _ = cp.shard_plan(P, R, C, 0)
    cp.kv_writeback(plan, k, k, kc, vc, bad)
    torch.cuda.synchronize()
    tab = bad.cpu().numpy()
    keep = [p for p in range(R) if 0 <= tab[p // B] < n_blocks]
    want = ocache.write_paged(f64(before_k), tab, keep, f64(k)[keep])
    assert np.array_equal(f64(kc), want)
    assert np.array_equal(f64(vc), ocache.write_paged(f64(before_v), tab, keep, f64(k)[keep]))


def test_prefix_hit_reads_the_written_cache():
    """Request A (3000 tokens, C=2) is prefilled and its K/V written back by
    the kernel; request B reuses A's first 2048 tokens as a cached prefix
    (block aligned) and attends its 500 new tokens over them."""
    g = synth.generator(3200, device=DEV)
    Hq, Hkv, D = 8, 2, 128
    LA, C = 3000, 2
    table_a, kc, vc = _request_cache(g, 0, LA, Hkv, D, spare=40)
    ka = synth.randn_bf16(g, (LA, Hkv, D), device=DEV)
    va = synth.randn_bf16(g, (LA, Hkv, D), device=DEV)
    for r in range(C):
        plan, _ = cp.shard_plan(0, LA, C, r)
        cp.kv_writeback(plan, _rank_rows(ka, 0, LA, C, r), _rank_rows(va, 0, LA, C, r), kc, vc, table_a)
    PB, RB = 2048, 500
    table_b = table_a[:PB // B].contiguous()
    q, kb, vb = synth.qkv(g, RB, RB, Hq, Hkv, D, device=DEV)
    k_ref = torch.cat([ka[:PB], kb])
    v_ref = torch.cat([va[:PB], vb])
    for r in range(C):
        plan, rows = cp.shard_plan(PB, RB, C, r)
        qr = q[torch.as_tensor(rows - PB, device=DEV)].contiguous()
        o = torch.empty((plan.n_rows, Hq, D), dtype=torch.float32, device=DEV)
        l = torch.empty((plan.n_rows, Hq), dtype=torch.float32, device=DEV)
        d = cp.make_desc(plan, qr, kb, vb, o, l, kc, vc, table_b, include_prefix=True)
        ws = torch.empty(max(256, cp.workspace_size([d], Hq, Hkv)), dtype=torch.uint8, device=DEV)
        cp.attn_partial([d], Hq, Hkv, ws)
        torch.cuda.synchronize()
        O_ref, L_ref = oatt.attend(f64(qr), rows, f64(k_ref), f64(v_ref), np.arange(PB + RB))
        compare(f64(o), f64(l), O_ref, L_ref, f"prefix hit from the written cache, rank {r}")


def test_writeback_full_size_round_trip():
    """Every rank of the 32K Llama-3-8B request writes its rows; reading the
    cache back through the block table returns the request's K and V."""
    w = synth.WORKLOADS["llama3_8b_32k_c4"]
    g = synth.generator(3300, device=DEV)
    table, kc, vc = _request_cache(g, 0, w.R, w.Hkv, w.D, spare=16)
    k = synth.randn_bf16(g, (w.R, w.Hkv, w.D), device=DEV)
    v = synth.randn_bf16(g, (w.R, w.Hkv, w.D), device=DEV)
    for r in range(w.C):
        plan, _ = cp.shard_plan(0, w.R, w.C, r)
        cp.kv_writeback(plan, _rank_rows(k, 0, w.R, w.C, r), _rank_rows(v, 0, w.R, w.C, r), kc, vc, table)
    torch.cuda.synchronize()
    pos = torch.arange(w.R, device=DEV)
    idx = table.long()[pos // B] * B + pos % B
    assert torch.equal(kc.reshape(-1, w.Hkv, w.D)[idx], k)
    assert torch.equal(vc.reshape(-1, w.Hkv, w.D)[idx], v)


def _ranks(x, P, R, C):
    return [_rank_rows(x, P, R, C, r) for r in range(C)]


@pytest.mark.parametrize("P,R,C_src,C_dst", [(0, 64, 2, 4), (16, 37, 4, 2), (0, 70, 3, 5), (32, 8, 1, 4),
                                             (0, 5, 4, 1), (0, 4096, 4, 8)])
def test_repartition_matches_oracle(P, R, C_src, C_dst):
    g = synth.generator(3400 + R, device=DEV)
    x = synth.randn_bf16(g, (R, 2, 128), device=DEV)
    src = _ranks(x, P, R, C_src)
    want = ocache.repartition(P, R, C_src, [f64(s) for s in src], C_dst)
    for r in range(C_dst):
        plan, _ = cp.shard_plan(P, R, C_dst, r)
        dst = torch.full((plan.n_rows, 2, 128), float("nan"), dtype=torch.bfloat16, device=DEV)
        cp.repartition(P, R, src, C_dst, r, dst)
        torch.cuda.synchronize()
        assert np.array_equal(f64(dst), np.asarray(want[r]).reshape(f64(dst).shape))


@pytest.mark.parametrize("P,R,C_src,C_dst", [(0, 64, 2, 4), (16, 37, 4, 2), (0, 70, 3, 5), (32, 8, 1, 4),
                                               (0, 1000, 8, 1), (48, 5, 4, 8)])
def test_repartition_all_matches_oracle(P, R, C_src, C_dst):
    """Every destination rank of two row sets (K and V) in one launch, bit for
    bit the oracle's re-shard of each set."""
    g = synth.generator(3450 + R, device=DEV)
    sets = [synth.randn_bf16(g, (R, 2, 128), device=DEV) for _ in range(2)]
    src = [_ranks(x, P, R, C_src) for x in sets]
    dst = [[torch.full((cp.shard_plan(P, R, C_dst, r)[0].n_rows, 2, 128), float("nan"), dtype=torch.bfloat16,
                       device=DEV) for r in range(C_dst)] for _ in range(2)]
    cp.repartition_all(P, R, src, dst)
    torch.cuda.synchronize()
    for k in range(2):
        want = ocache.repartition(P, R, C_src, [f64(t) for t in src[k]], C_dst)
        for r in range(C_dst):
            assert np.array_equal(f64(dst[k][r]), np.asarray(want[r]).reshape(f64(dst[k][r]).shape)), (k, r)


def test_repartition_all_full_size_round_trip():
    """The 32K Llama-3-8B request's K and V, 4 -> 8 -> 4 ranks, one launch each
    way: every degree-8 rank holds its own rows, and the way back restores the
    degree-4 ranks exactly."""
    w = synth.WORKLOADS["llama3_8b_32k_c4"]
    g = synth.generator(3550, device=DEV)
    kv = [synth.randn_bf16(g, (w.R, w.Hkv, w.D), device=DEV) for _ in range(2)]
    src = [_ranks(x, 0, w.R, 4) for x in kv]
    mid = [[torch.empty((cp.shard_plan(0, w.R, 8, r)[0].n_rows, w.Hkv, w.D), dtype=torch.bfloat16, device=DEV)
            for r in range(8)] for _ in range(2)]
    cp.repartition_all(0, w.R, src, mid)
    back = [[torch.empty_like(t) for t in src[k]] for k in range(2)]
    cp.repartition_all(0, w.R, mid, back)
    torch.cuda.synchronize()
    for k in range(2):
        for r in range(8):
            assert torch.equal(mid[k][r], _rank_rows(kv[k], 0, w.R, 8, r))
        for r in range(4):
            assert torch.equal(back[k][r], src[k][r])


def test_repartition_full_size_round_trip():
    """32K Llama-3-8B K rows re-sharded 4 -> 8 -> 4 ranks; degree-8 ranks 2k
    and 2k+1 hold exactly the rows of degree-4 rank k."""
    w = synth.WORKLOADS["llama3_8b_32k_c4"]
    g = synth.generator(3500, device=DEV)
    k = synth.randn_bf16(g, (w.R, w.Hkv, w.D), device=DEV)
    src = _ranks(k, 0, w.R, 4)
    mid = []
    for r in range(8):
        plan, _ = cp.shard_plan(0, w.R, 8, r)
        t = torch.empty((plan.n_rows, w.Hkv, w.D), dtype=torch.bfloat16, device=DEV)
        cp.repartition(0, w.R, src, 8, r, t)
        mid.append(t)
    torch.cuda.synchronize()
    for r in range(8):
        assert torch.equal(mid[r], _rank_rows(k, 0, w.R, 8, r))
    for kk in range(4):
        got = torch.cat([mid[2 * kk], mid[2 * kk + 1]])
        assert torch.equal(torch.sort(got.reshape(got.shape[0], -1)[:, 0])[0],
                           torch.sort(src[kk].reshape(src[kk].shape[0], -1)[:, 0])[0])
    for r in range(4):
        plan, _ = cp.shard_plan(0, w.R, 4, r)
        back = torch.empty((plan.n_rows, w.Hkv, w.D), dtype=torch.bfloat16, device=DEV)
        cp.repartition(0, w.R, mid, 4, r, back)
        torch.cuda.synchronize()
        assert torch.equal(back, src[r])


@pytest.mark.parametrize("pos_begin,n,Hkv", [(0, 100, 2), (37, 70, 1), (16, 16, 8), (5, 1, 4), (0, 0, 2)])
def test_gather_matches_oracle(pos_begin, n, Hkv):
    g = synth.generator(3600 + pos_begin + n, device=DEV)
    D = 128
    table, kc, vc = _request_cache(g, 0, pos_begin + n, Hkv, D, spare=4)
    k = torch.full((n, Hkv, D), float("nan"), dtype=torch.bfloat16, device=DEV)
    v = torch.full((n, Hkv, D), float("nan"), dtype=torch.bfloat16, device=DEV)
    cp.kv_gather(kc, vc, table, pos_begin, k, v)
    torch.cuda.synchronize()
    tab = table.cpu().numpy()
    assert np.array_equal(f64(k), ocache.read_paged(f64(kc), tab, pos_begin, n))
    assert np.array_equal(f64(v), ocache.read_paged(f64(vc), tab, pos_begin, n))


def test_gather_of_entries_outside_the_cache_is_zero():
    g = synth.generator(3700, device=DEV)
    Hkv, D, n = 2, 128, 64
    table, kc, vc = _request_cache(g, 0, n, Hkv, D, spare=0)
    bad = table.clone()
    bad[1] = kc.shape[0]
    bad[2] = -7
    k = torch.full((n, Hkv, D), float("nan"), dtype=torch.bfloat16, device=DEV)
    v = torch.full_like(k, float("nan"))
    cp.kv_gather(kc, vc, bad, 0, k, v)
    torch.cuda.synchronize()
    tab = bad.cpu().numpy()
    assert np.array_equal(f64(k), ocache.read_paged(f64(kc), tab, 0, n))
    assert np.array_equal(f64(v), ocache.read_paged(f64(vc), tab, 0, n))
    assert not torch.any(k[16:48].float()) and not torch.any(v[16:48].float())


def test_gather_full_size_round_trip():
    """The 48K-token prefix of the prefix-hit workload (3072 blocks of 16,
    permuted table, Llama-3-8B KV heads) read back out of the paged cache is
    exactly what the cache holds at those positions."""
    w = synth.WORKLOADS["prefix_hit_64k_c2"]
    g = synth.generator(3800, device=DEV)
    pre = synth.paged_prefix(g, w.P, w.Hkv, w.D, 1.0, spare_blocks=16, device=DEV)
    k = torch.empty((w.P, w.Hkv, w.D), dtype=torch.bfloat16, device=DEV)
    v = torch.empty_like(k)
    cp.kv_gather(pre.k_cache, pre.v_cache, pre.block_table, 0, k, v)
    torch.cuda.synchronize()
    pos = torch.arange(w.P, device=DEV)
    idx = pre.block_table.long()[pos // B] * B + pos % B
    assert torch.equal(k, pre.k_cache.reshape(-1, w.Hkv, w.D)[idx])
    assert torch.equal(v, pre.v_cache.reshape(-1, w.Hkv, w.D)[idx])
