"""cp_attn_partial_noalloc -- the partial attention without a workspace, on
the library's own device scratch -- against cp_attn_partial on the same
descriptors: two calls in a row on one stream with no wait between them, the
second with a smaller input, so the second call's tables overwrite the
scratch the first call's launch used."""

import pytest
import torch

import gpu_cases as gc
from gpu_cases import DEV, Problem, compare, f64
from paper_2609_04774_amd import cpattn as cp

pytestmark = pytest.mark.gpu


def _descs(prob):
    """Every rank's all-gathered partial and its shard-0 pass-KV partial (with
    the prefix): (descs, outputs)."""
    dv = prob.dev()
    descs, outs = [], []
    for r in range(prob.C):
        plan, rows = cp.shard_plan(prob.P, prob.R, prob.C, r)
        if plan.n_rows == 0:
            continue
        q = dv["q"][torch.as_tensor(rows - prob.P, device=DEV)].contiguous()
        for kv in (cp.CP_KV_ALL, 0):
            o, lse = gc.alloc_out(plan.n_rows, prob.Hq)
            outs.append((o[: plan.n_rows], lse[: plan.n_rows], r, kv))
            descs.append(cp.make_desc(plan, q, dv["k"], dv["v"], o, lse, dv.get("kc"), dv.get("vc"),
                                      dv.get("bt"), include_prefix=True, kv_rank=kv))
    return descs, outs


# (L, P, C, Hq, Hkv, seed, same plan as with a workspace)
@pytest.mark.parametrize("first,second", [
    # A larger launch, then a smaller one (no split walks).
    ((3000, 256, 2, 32, 8, 81, True), (500, 0, 1, 8, 2, 82, True)),
    # Split walks over an 8192-token prefix (128 pieces: they fit), then a
    # small launch.
    ((8392, 8192, 2, 8, 2, 83, True), (700, 48, 2, 8, 2, 84, True)),
    # Split walks over a 16384-token prefix: about 960 pieces with a
    # workspace, more than the scratch holds, so fewer, longer pieces (same
    # attention, other decomposition); then a smaller split launch.
    ((16640, 16384, 1, 32, 8, 85, False), (8392, 8192, 2, 8, 2, 86, True)),
])
def test_noalloc_matches_workspace_entry_point(first, second):
    probs = [Problem(*c[:5], seed=c[5]) for c in (first, second)]
    same_plan = [first[6], second[6]]
    ref = [_descs(p) for p in probs]
    na = [_descs(p) for p in probs]
    for p, (descs, _) in zip(probs, ref):
        gc.run_partials(descs, p.Hq, p.Hkv)
    stream = torch.cuda.current_stream()
    for p, (descs, _) in zip(probs, na):
        cp.attn_partial_noalloc(descs, p.Hq, p.Hkv, stream=stream)
    torch.cuda.synchronize()
    for i, p in enumerate(probs):
        for (o_r, l_r, r, kv), (o_n, l_n, _, _) in zip(ref[i][1], na[i][1]):
            what = f"call {i + 1}, rank {r}, kv {kv}"
            print(what, flush=True)
            if same_plan[i]:
                assert torch.equal(o_r, o_n) and torch.equal(l_r, l_n), what + ": differs from cp_attn_partial"
            compare(f64(o_n), f64(l_n), f64(o_r), f64(l_r), what + " vs cp_attn_partial")
            Or, Lr = p.oracle_rank(r, kv_rank=kv, include_prefix=True)
            compare(f64(o_n), f64(l_n), Or, Lr, what + " vs oracle")
