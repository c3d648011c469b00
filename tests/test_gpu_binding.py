"""The Python binding refuses tensors the C ABI would read or write out of
bounds (wrong element type, too few rows, non-contiguous, wrong head count)
before anything is launched."""

import pytest
import torch

from paper_2609_04774_amd import cpattn as cp

pytestmark = pytest.mark.gpu

DEV = torch.device("cuda", 0)


def _bf(*shape):
    return torch.zeros(shape, dtype=torch.bfloat16, device=DEV)


def _f32(*shape):
    return torch.zeros(shape, dtype=torch.float32, device=DEV)


def test_partial_descriptor_checks():
    plan, _ = cp.shard_plan(0, 256, 2, 0)
    n, R, Hq, Hkv = plan.n_rows, 256, 8, 2
    q, k, v, o, lse = _bf(n, Hq, 128), _bf(R, Hkv, 128), _bf(R, Hkv, 128), _f32(n, Hq, 128), _f32(n, Hq)
    d = cp.make_desc(plan, q, k, v, o, lse)
    ws = torch.empty(max(256, cp.workspace_size([d], Hq, Hkv)), dtype=torch.uint8, device=DEV)
    with pytest.raises(TypeError):
        cp.make_desc(plan, q, k, v, _bf(n, Hq, 128), lse)           # O must be fp32
    with pytest.raises(ValueError):
        cp.make_desc(plan, q[: n - 1], k, v, o, lse)                # too few query rows
    with pytest.raises(ValueError):
        cp.make_desc(plan, q, k[: R - 1], v, o, lse)                # too few suffix keys
    with pytest.raises(ValueError):
        cp.make_desc(plan, q.transpose(0, 1), k, v, o, lse)         # not contiguous
    with pytest.raises(ValueError):
        cp.make_desc(plan, q, k, v, o, lse.cpu())                   # host memory
    with pytest.raises(ValueError):
        cp.attn_partial([d], 16, Hkv, ws)                           # q holds 8 heads, not 16
    cp.attn_partial([d], Hq, Hkv, ws)
    torch.cuda.synchronize()


def test_merge_and_cache_checks():
    o, l = _f32(10, 4, 128), _f32(10, 4)
    with pytest.raises(ValueError):
        cp.attn_merge([o], [l], _f32(9, 4, 128), _f32(10, 4))      # output too small
    with pytest.raises(TypeError):
        cp.attn_merge([o], [l.double()], _f32(10, 4, 128))          # LSE must be fp32
    plan, _ = cp.shard_plan(0, 64, 2, 0)
    kc, vc = _bf(8, 16, 2, 128), _bf(8, 16, 2, 128)
    table = torch.arange(8, dtype=torch.int32, device=DEV)
    rows = _bf(plan.n_rows, 2, 128)
    with pytest.raises(ValueError):
        cp.kv_writeback(plan, rows[:-1], rows, kc, vc, table)       # too few rows
    with pytest.raises(TypeError):
        cp.kv_gather(kc, vc, table.long(), 0, _bf(16, 2, 128), _bf(16, 2, 128))
    with pytest.raises(ValueError):
        cp.repartition(0, 64, [rows, rows[:1]], 4, 0, _bf(16, 2, 128))  # a source rank too small


def test_descriptor_keeps_its_tensors_alive():
    """A block table (or any other tensor) handed to make_desc stays allocated
    while the descriptor exists, even when the caller drops its own
    reference: its memory cannot be reused before the launch reads it."""
    import gc
    import weakref
    plan, _ = cp.shard_plan(64, 64, 2, 0)
    q, k, v = _bf(plan.n_rows, 8, 128), _bf(64, 2, 128), _bf(64, 2, 128)
    o, lse = _f32(plan.n_rows, 8, 128), _f32(plan.n_rows, 8)
    kc, vc = _bf(4, 16, 2, 128), _bf(4, 16, 2, 128)
    table = torch.arange(4, dtype=torch.int32, device=DEV)
    ref = weakref.ref(table)
    d = cp.make_desc(plan, q, k, v, o, lse, kc, vc, table, include_prefix=True)
    del table
    gc.collect()
    assert ref() is not None and ref().data_ptr() == d.block_table
    del d
    gc.collect()
    assert ref() is None
