"""Helpers for the GPU parity tests: run the HIP path through the C ABI and
compare with the oracle on the same seeded inputs.

Tolerances: max-abs 1e-2 on the fp32 output O and 1e-3 on the natural-log
LSE, against the fp64 oracle on the same bf16 inputs (bf16 in, fp32
accumulate on the GPU).
"""

from __future__ import annotations

import numpy as np
import torch

import synth
from oracle import attention as oatt
from oracle import plan as oplan
from paper_2609_04774_amd import cpattn as cp

O_TOL = 1e-2
LSE_TOL = 1e-3
DEV = "cuda"


def new_workspace(descs, Hq, Hkv):
    n = cp.workspace_size(descs, Hq, Hkv)
    return torch.empty(max(n, 256), dtype=torch.uint8, device=DEV)


def run_partials(descs, Hq, Hkv, scale=0.0):
    ws = new_workspace(descs, Hq, Hkv)
    cp.attn_partial(descs, Hq, Hkv, ws, softmax_scale=scale)
    torch.cuda.synchronize()
    return ws


def alloc_out(n_rows, Hq, D=128):
    o = torch.full((max(n_rows, 1), Hq, D), float("nan"), dtype=torch.float32, device=DEV)
    lse = torch.full((max(n_rows, 1), Hq), float("nan"), dtype=torch.float32, device=DEV)
    return o, lse


def f64(t):
    return t.detach().to("cpu").double().numpy()


def compare(o_gpu, lse_gpu, o_ref, lse_ref, what=""):
    """Element-wise parity.  Rows whose reference LSE is -inf must be -inf
    with O == 0 exactly on the GPU too."""
    o_gpu = np.asarray(o_gpu, dtype=np.float64)
    lse_gpu = np.asarray(lse_gpu, dtype=np.float64)
    empty = np.isneginf(lse_ref)
    assert np.array_equal(np.isneginf(lse_gpu), empty), f"{what}: -inf LSE rows differ"
    assert not np.isnan(o_gpu).any() and not np.isnan(lse_gpu).any(), f"{what}: NaN in GPU output"
    if empty.any():
        assert np.all(o_gpu[empty] == 0.0), f"{what}: rows without keys must have O == 0"
    live = ~empty
    err_o = float(np.max(np.abs(o_gpu - o_ref))) if o_ref.size else 0.0
    err_l = float(np.max(np.abs(lse_gpu[live] - lse_ref[live]))) if live.any() else 0.0
    assert err_o <= O_TOL, f"{what}: max |dO| = {err_o:.3e} > {O_TOL}"
    assert err_l <= LSE_TOL, f"{what}: max |dLSE| = {err_l:.3e} > {LSE_TOL}"
    return err_o, err_l


class Problem:
    """One request: full-sequence Q/K/V (bf16, CPU) + optional paged prefix."""

    def __init__(self, L, P, C, Hq, Hkv, seed, data_scale=1.0, q_scale=1.0, spare_blocks=3):
        self.L, self.P, self.C, self.Hq, self.Hkv = L, P, C, Hq, Hkv
        self.R = L - P
        g = synth.generator(seed)
        self.q, self.k, self.v = synth.qkv(g, self.R, self.R, Hq, Hkv, scale=data_scale)
        if q_scale != 1.0:
            self.q = (self.q.float() * q_scale).to(torch.bfloat16)
        self.prefix = None
        if P:
            self.prefix = synth.paged_prefix(g, P, Hkv, scale=data_scale, spare_blocks=spare_blocks)
        self._dev = None
        self._f64 = None

    def dev(self):
        if self._dev is None:
            d = {"k": self.k.to(DEV), "v": self.v.to(DEV), "q": self.q.to(DEV)}
            if self.prefix is not None:
                d["kc"] = self.prefix.k_cache.to(DEV)
                d["vc"] = self.prefix.v_cache.to(DEV)
                d["bt"] = self.prefix.block_table.to(DEV)
            self._dev = d
        return self._dev

    def np(self):
        if self._f64 is None:
            d = {"q": f64(self.q), "k": f64(self.k), "v": f64(self.v)}
            if self.prefix is not None:
                d["kc"] = f64(self.prefix.k_cache)
                d["vc"] = f64(self.prefix.v_cache)
                d["bt"] = self.prefix.block_table.numpy().astype(np.int64)
            self._f64 = d
        return self._f64

    def gpu_rank(self, rank, kv_rank=cp.CP_KV_ALL, include_prefix=True, scale=0.0):
        """Rank `rank`'s partial on the GPU: (o, lse, plan, row_pos)."""
        plan, rows = cp.shard_plan(self.P, self.R, self.C, rank)
        dv = self.dev()
        q = dv["q"][torch.as_tensor(rows - self.P, device=DEV)].contiguous() if plan.n_rows else dv["q"][:1]
        o, lse = alloc_out(plan.n_rows, self.Hq)
        desc = cp.make_desc(plan, q, dv["k"], dv["v"], o, lse, dv.get("kc"), dv.get("vc"),
                            dv.get("bt"), include_prefix=include_prefix, kv_rank=kv_rank)
        run_partials([desc], self.Hq, self.Hkv, scale)
        return o[: plan.n_rows], lse[: plan.n_rows], plan, rows

    def oracle_rank(self, rank, kv_rank=cp.CP_KV_ALL, include_prefix=True, rows_subset=None,
                    scale=None):
        """The oracle's partial for the same rank (its own plan)."""
        ref_plan = oplan.shard_plan_fast(self.P, self.R, self.C, rank)
        rows = np.array(ref_plan["row_pos"], dtype=np.int64)
        if rows_subset is not None:
            rows = rows[rows_subset]
        d = self.np()
        if kv_rank == cp.CP_KV_ALL:
            ranges = None
        elif kv_rank == cp.CP_KV_NONE:
            ranges = []
        else:
            ranges = oplan.kv_shard_ranges(self.P, self.R, self.C, kv_rank)
        return oatt.rank_partial(d["q"][rows - self.P], rows, self.P, d["k"], d["v"], d.get("kc"),
                                 d.get("vc"), d.get("bt"), include_prefix=include_prefix,
                                 suffix_ranges=ranges, scale=scale)
