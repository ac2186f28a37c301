"""The allocation-free de-duplication entry point against the one that takes a
workspace: bit-exact uni, inv, u, gathered rows, miss list and miss count on
calls in a row through the C ABI, each later call smaller than the one before
it, so every call finds the previous call's data in the fixed scratch."""
import ctypes

import numpy as np
import pytest
import torch

import paper_2607_05095_amd as fast
from synth import make_batch, make_slot_map, make_table

pytestmark = pytest.mark.gpu


def _announce(msg):
    print(f"[no-alloc] {msg}", flush=True)


def _outputs(n, D, dtype):
    o = dict(uni=torch.full((n,), -7, dtype=torch.int64, device="cuda"),
             inv=torch.full((n,), -7, dtype=torch.int32, device="cuda"),
             nu=torch.full((1,), -7, dtype=torch.int64, device="cuda"),
             miss=torch.full((n,), -7, dtype=torch.int32, device="cuda"),
             nm=torch.full((1,), -7, dtype=torch.int64, device="cuda"))
    # the same fill in both runs: rows of missed ids are left untouched
    o["rows"] = torch.full((n, D), 3.0, dtype=dtype, device="cuda") if D else None
    return o


def _run(noalloc, ids, bound, table, slot):
    n = ids.shape[0]
    D = table.shape[1] if table is not None else 0
    rows_dt = table.dtype if table is not None else torch.float32
    o = _outputs(n, D, rows_dt)
    DT = fast.F32 if rows_dt == torch.float32 else fast.BF16
    trows = table.shape[0] if table is not None else 0
    if noalloc:
        fast.fast_dedup_gather_noalloc(ids, n, bound, table, trows, D, DT, slot, o["uni"], o["inv"],
                                       o["nu"], o["rows"], o["miss"], o["nm"])
    else:
        wsb = fast.fast_dedup_gather_workspace(n, bound)
        ws = torch.full((wsb,), 0xA5, dtype=torch.uint8, device="cuda")
        fast.fast_dedup_gather(ids, n, bound, table, trows, D, DT, slot, o["uni"], o["inv"], o["nu"],
                               o["rows"], o["miss"], o["nm"], ws, wsb)
    torch.cuda.synchronize()
    return o


def _same(a, b, what):
    u = int(a["nu"].item())
    assert u == int(b["nu"].item()), f"{what}: u {u} vs {int(b['nu'].item())}"
    assert torch.equal(a["uni"][:u], b["uni"][:u]), f"{what}: uni differs"
    assert torch.equal(a["inv"], b["inv"]), f"{what}: inv differs"
    m = int(a["nm"].item())
    assert m == int(b["nm"].item()), f"{what}: miss count differs"
    assert torch.equal(a["miss"][:m], b["miss"][:m]), f"{what}: miss list differs"
    if a["rows"] is not None:
        assert torch.equal(a["rows"].view(torch.int16) if a["rows"].dtype == torch.bfloat16
                           else a["rows"].view(torch.int32),
                           b["rows"].view(torch.int16) if b["rows"].dtype == torch.bfloat16
                           else b["rows"].view(torch.int32)), f"{what}: rows differ"
    return u, m


def test_noalloc_dedup_gather_equals_workspace_entry_point():
    torch.cuda.set_device(0)
    big = make_batch(4)
    # 1. edge ids of the 1e7-node / 2e8-edge batch through the cached-row slot
    #    map: the largest scratch the benchmark uses (bucketed marking)
    edge_ids = torch.from_numpy(big.edge_ids).cuda()
    slot = make_slot_map(big, device="cuda")
    cache = make_table(big.edge_cache_rows, big.edge_D, "f32", "cuda", big.seed, 4)
    need = fast.fast_dedup_gather_workspace(edge_ids.shape[0], big.edge_bound)
    assert 0 < need <= fast.NOALLOC_SCRATCH_BYTES
    cases = [("edges n=2.64e6 over 2e8, slot map", edge_ids, big.edge_bound, cache, slot),
             # 2. a smaller batch on the same marking path: stale records of call 1 remain
             ("edges n=2e5 over 2e8, slot map", edge_ids[:200_000].contiguous(), big.edge_bound,
              cache, slot)]
    # 3. smaller still, dense universe (byte map), bf16 rows without a slot map
    mid = make_batch(2)
    node_ids = torch.from_numpy(mid.node_ids).cuda()
    ntab = make_table(mid.node_bound, 64, "bf16", "cuda", mid.seed, 3)
    cases.append(("nodes n=%d over 1e5, bf16 rows" % node_ids.shape[0], node_ids, mid.node_bound,
                  ntab, None))
    # 4. dedup only (no rows), tiny
    cases.append(("ids n=700 over 1e3, no rows", node_ids[:700].remainder(1000).contiguous(), 1000,
                  None, None))
    prev = None
    for what, ids, bound, table, sm in cases:
        _announce(what)
        assert prev is None or ids.shape[0] < prev
        prev = ids.shape[0]
        ref = _run(False, ids, bound, table, sm)
        got = _run(True, ids, bound, table, sm)
        u, m = _same(got, ref, what)
        assert u > 0
        _announce(f"  u = {u}, misses = {m}: equal")
    # a second pass over the first two cases, with the scratch as the last
    # (smallest) call left it
    for what, ids, bound, table, sm in cases[:2]:
        _announce("again: " + what)
        _same(_run(True, ids, bound, table, sm), _run(False, ids, bound, table, sm), what)


def test_noalloc_rejects_problems_beyond_its_scratch():
    """Refused on the host, before anything is enqueued."""
    L = fast.lib()
    FAKE = 0x10000
    one = ctypes.c_void_p(FAKE)
    # a 2^35-id universe needs a 4 GiB bitmap, far beyond the fixed scratch
    assert fast.fast_dedup_gather_workspace(1000, 1 << 35) > fast.NOALLOC_SCRATCH_BYTES
    st = L.fast_dedup_gather_noalloc(one, 1000, 1 << 35, None, 0, 0, fast.F32, None, one, one, one,
                                     None, None, None, None)
    assert st == 2
    assert "scratch" in fast.fast_last_error()
    st = L.fast_dedup_gather_noalloc(one, -1, 10, None, 0, 0, fast.F32, None, one, one, one,
                                     None, None, None, None)
    assert st == 1
