"""GPU parity of SlimCache's greedy cache selection (Alg. 1) through the C
ABI: access counts bit-exact against the oracle, and the hot node / edge
sets and slot maps bit-exact against the oracle's selection (the oracle
returns ids in selection order, the library in ascending id order, so sets
are compared sorted and the slot map is checked against that order).

At the big-dedup universe (1e7 nodes, 2e8 edges) the oracle's sort of 2.1e8
ids is out of reach; there the counts are still compared bit-exactly, and
the selection is checked by properties that fix it at any size: the budget,
the count threshold (everything above taken, nothing below), edges before
nodes and lowest ids first at the threshold, the slot map as the rank in
the hot list, and maximal total count.
"""
import numpy as np
import pytest
import torch

import oracle
import paper_2607_05095_amd as fast
from synth import presampled_ids

pytestmark = pytest.mark.gpu


def _announce(msg):
    print(f"[parity] {msg}", flush=True)


def _count_gpu(batches, bound, freq=None):
    sizes = [b.size for b in batches]
    ids = torch.from_numpy(np.concatenate(batches).astype(np.int64)).cuda()
    offs = np.concatenate([[0], np.cumsum(sizes)]).astype(np.int64)
    f = torch.zeros(bound, dtype=torch.int32, device="cuda") if freq is None else freq
    wsb = fast.fast_access_count_workspace(bound)
    ws = torch.empty(wsb, dtype=torch.uint8, device="cuda")
    fast.fast_access_count(ids, offs, len(batches), bound, f, ws, wsb)
    torch.cuda.synchronize()
    return f


def _select_gpu(fv, fe, max_freq, budget, want_slots=True, slot_offset=0):
    """slot_offset > 0 places both slot maps that many int32 past a 256-byte
    boundary (off the 16-byte grid for 1..3: the element-wise stores)."""
    nv, ne = fv.numel(), fe.numel()
    hv = torch.full((max(min(budget, nv), 1),), -7, dtype=torch.int64, device="cuda")
    he = torch.full((max(min(budget, ne), 1),), -7, dtype=torch.int64, device="cuda")
    nhv = torch.empty(1, dtype=torch.int64, device="cuda")
    nhe = torch.empty(1, dtype=torch.int64, device="cuda")
    o = slot_offset
    sv = torch.empty(nv + o, dtype=torch.int32, device="cuda")[o:] if want_slots else None
    se = torch.empty(ne + o, dtype=torch.int32, device="cuda")[o:] if want_slots else None
    wsb = fast.fast_greedy_hot_set_workspace(nv, ne, max_freq)
    ws = torch.empty(wsb, dtype=torch.uint8, device="cuda")
    fast.fast_greedy_hot_set(fv, nv, fe, ne, max_freq, budget, hv, nhv, sv, he, nhe, se, ws, wsb)
    torch.cuda.synchronize()
    a, b = int(nhv.item()), int(nhe.item())
    return hv[:a].cpu().numpy(), he[:b].cpu().numpy(), sv, se


def _check_slots(slot, hot, n):
    want = np.full(n, -1, dtype=np.int32)
    want[hot] = np.arange(hot.size, dtype=np.int32)
    assert np.array_equal(slot.cpu().numpy(), want)


@pytest.mark.parametrize("cfg,k", [(2, 12), (3, 4), (1, 6), (2, 40)])
def test_access_count_and_selection_vs_oracle(cfg, k):
    """cfg 2's edge ids are counted in the sparse form: 12 batches with batch
    bits in two groups, 40 batches with stamps; the other universes are dense
    (a byte map per batch)."""
    nodes, edges, nb, eb = presampled_ids(cfg, k)
    _announce(f"hot set cfg={cfg} batches={k} |V|={nb} |E|={eb}")
    fv = _count_gpu(nodes, nb)
    fe = _count_gpu(edges, eb)
    rv, re_ = oracle.access_count(nodes, nb), oracle.access_count(edges, eb)
    assert np.array_equal(fv.cpu().numpy(), rv)
    assert np.array_equal(fe.cpu().numpy(), re_)
    for alpha in (0.0, 0.003, 0.01, 0.1, 0.35, 1.0, 1.5):
        B = fast.fast_hot_set_budget(alpha, nb, eb)
        hv, he, sv, se = _select_gpu(fv, fe, k, B)
        ov, oe = oracle.greedy_hot_set(rv, re_, alpha)
        assert hv.size + he.size == B == ov.size + oe.size, alpha
        assert np.array_equal(hv, np.sort(ov)), f"node set alpha={alpha}"
        assert np.array_equal(he, np.sort(oe)), f"edge set alpha={alpha}"
        _check_slots(sv, hv, nb)
        _check_slots(se, he, eb)


@pytest.mark.parametrize("bound", [1000, 40])
def test_access_count_repeats_invalid_ids_and_accumulation(bound):
    # bound 1000 over ~4 ids a batch takes the stamp path, bound 40 the byte map
    _announce(f"access count edge cases bound={bound}")
    top = bound - 1
    batches = [np.array([5, 5, 5, top, 0, -1, bound, 7 << 40], np.int64),
               np.zeros(0, np.int64), np.array([5, 3, 3], np.int64)]
    f = _count_gpu(batches, bound)
    f = _count_gpu([np.array([3, top - 1], np.int64)], bound, freq=f)      # accumulates
    want = oracle.access_count([np.array([3, top - 1])], bound,
                               freq=oracle.access_count(batches, bound))
    assert np.array_equal(f.cpu().numpy(), want)
    assert f[5].item() == 2 and f[3].item() == 2 and f[top].item() == 1


def test_selection_edge_cases():
    _announce("hot set edge cases")
    dev = lambda a: torch.tensor(a, dtype=torch.int32, device="cuda")
    # the hand example of the oracle pins: budget 4 of 7 ids
    hv, he, sv, se = _select_gpu(dev([3, 1, 2]), dev([2, 2, 0, 5]), 5, 4)
    assert hv.tolist() == [0] and he.tolist() == [0, 1, 3]
    assert sv.cpu().tolist() == [0, -1, -1] and se.cpu().tolist() == [0, 1, -1, 2]
    # all counts equal: edges first, lowest ids
    hv, he, _, _ = _select_gpu(dev([1] * 5), dev([1] * 4), 1, 6)
    assert he.tolist() == [0, 1, 2, 3] and hv.tolist() == [0, 1]
    # no nodes; no edges; zero budget; counts above max_freq are clamped
    hv, he, _, _ = _select_gpu(dev([]), dev([0, 9, 2]), 9, 2)
    assert hv.size == 0 and he.tolist() == [1, 2]
    hv, he, _, _ = _select_gpu(dev([4, 0, 4]), dev([]), 4, 2)
    assert hv.tolist() == [0, 2] and he.size == 0
    hv, he, sv, se = _select_gpu(dev([4, 0]), dev([1]), 4, 0)
    assert hv.size == 0 and he.size == 0 and sv.cpu().tolist() == [-1, -1]
    # a budget beyond every id takes everything
    hv, he, _, _ = _select_gpu(dev([0, 0]), dev([0]), 3, 10)
    assert hv.tolist() == [0, 1] and he.tolist() == [0]
    # a wide count range (several 256-count chunks of the threshold search,
    # counts above the LDS-binned range)
    r = np.random.default_rng(1)
    fv_np = r.integers(0, 9000, 20000).astype(np.int32)
    fe_np = r.integers(0, 9000, 30000).astype(np.int32)
    for alpha in (0.001, 0.2, 0.77):
        B = fast.fast_hot_set_budget(alpha, fv_np.size, fe_np.size)
        hv, he, _, _ = _select_gpu(dev(fv_np), dev(fe_np), 9000, B, want_slots=False)
        ov, oe = oracle.greedy_hot_set(fv_np, fe_np, alpha)
        assert np.array_equal(hv, np.sort(ov)) and np.array_equal(he, np.sort(oe))


@pytest.mark.parametrize("max_freq", [63, 64])
def test_selection_both_histogram_paths(max_freq):
    """Counts below 64 are histogrammed per tile of 4096 ids (the tile sums of
    the selection come from those histograms); 64 and above take the plain
    global histogram and a second pass over the counts.  Both against the
    oracle on ragged sizes (a partial last tile), with counts clamped into
    [0, max_freq], a count array that is not 16-byte aligned, and slot maps
    on and off the 16-byte grid."""
    _announce(f"hot set histogram path max_freq={max_freq}")
    r = np.random.default_rng(max_freq)
    nv, ne = 4096 * 7 + 1234, 4096 * 11 + 5
    fv_np = np.minimum(r.zipf(1.3, nv), max_freq + 20).astype(np.int32) - 1
    fe_np = np.minimum(r.zipf(1.4, ne), max_freq + 20).astype(np.int32) - 1
    clamp = lambda a: np.clip(a, 0, max_freq)
    fv_big = torch.tensor(np.concatenate([[7], fv_np]), dtype=torch.int32, device="cuda")
    fv = fv_big[1:]                                   # 4 bytes off the 16-byte grid
    fe = torch.tensor(fe_np, dtype=torch.int32, device="cuda")
    for alpha, off in ((0.0005, 0), (0.02, 1), (0.3, 0), (1.0, 3)):
        B = fast.fast_hot_set_budget(alpha, nv, ne)
        hv, he, sv, se = _select_gpu(fv, fe, max_freq, B, slot_offset=off)
        ov, oe = oracle.greedy_hot_set(clamp(fv_np), clamp(fe_np), alpha)
        assert np.array_equal(hv, np.sort(ov)) and np.array_equal(he, np.sort(oe)), alpha
        _check_slots(sv, hv, nv)
        _check_slots(se, he, ne)


def test_bigdedup_universe_properties():
    k = 4
    nodes, edges, nb, eb = presampled_ids(4, k)
    _announce(f"hot set bigdedup |V|={nb} |E|={eb} batches={k}")
    fv = _count_gpu(nodes, nb)
    fe = _count_gpu(edges, eb)
    rv = oracle.access_count(nodes, nb)
    assert np.array_equal(fv.cpu().numpy(), rv)
    re_ = oracle.access_count(edges, eb)
    assert np.array_equal(fe.cpu().numpy(), re_)
    del nodes, edges
    B = fast.fast_hot_set_budget(0.01, nb, eb)           # ~2.1e6 cached rows
    hv, he, sv, se = _select_gpu(fv, fe, k, B)
    assert hv.size + he.size == B
    # threshold T: every selected count >= T >= every unselected count
    T = min(rv[hv].min() if hv.size else k + 1, re_[he].min() if he.size else k + 1)
    sel_v = np.zeros(nb, bool); sel_v[hv] = True
    sel_e = np.zeros(eb, bool); sel_e[he] = True
    assert np.all(sel_v[rv > T]) and np.all(sel_e[re_ > T])
    assert not np.any(sel_v[rv < T]) and not np.any(sel_e[re_ < T])
    tie_v, tie_e = np.flatnonzero(rv == T), np.flatnonzero(re_ == T)
    nt_v, nt_e = int(sel_v[tie_v].sum()), int(sel_e[tie_e].sum())
    if nt_v:
        assert nt_e == tie_e.size                       # edges before nodes at T
    assert sel_v[tie_v[:nt_v]].all() and sel_e[tie_e[:nt_e]].all()   # lowest ids first
    # maximal total count: the budget's largest counts over both kinds
    hist = np.bincount(rv, minlength=k + 1) + np.bincount(re_, minlength=k + 1)
    best, left = 0, B
    for c in range(k, -1, -1):
        t = min(left, int(hist[c]))
        best += t * c
        left -= t
    assert int(rv[hv].sum()) + int(re_[he].sum()) == best
    assert np.all(np.diff(hv) > 0) and np.all(np.diff(he) > 0)
    _check_slots(sv, hv, nb)
    _check_slots(se, he, eb)


@pytest.mark.parametrize("seed", range(24))
def test_selection_random(seed):
    """Seeded random universes (0 to 300 k nodes and edges), count laws
    (uniform or Zipf-like, clamped at max_freq from 1 to 5000, both sides of
    the one-byte code path at 64) and budgets from 0 to beyond every id,
    with slot maps on and off the 16-byte grid: sets and slot maps equal to
    the oracle's selection."""
    r = np.random.default_rng(8000 + seed)
    max_freq = int(r.choice([1, 2, 7, 63, 64, 300, 5000]))
    nv = int(r.choice([0, int(r.integers(1, 5000)), int(r.integers(5000, 300_001))], p=[0.1, 0.4, 0.5]))
    ne = int(r.choice([0, int(r.integers(1, 5000)), int(r.integers(5000, 300_001))], p=[0.1, 0.4, 0.5]))

    def law(n):
        if r.random() < 0.5:
            return r.integers(0, max_freq + 1, n)
        return np.minimum(r.zipf(float(r.uniform(1.1, 2.5)), n) - 1, max_freq + 3)

    fv_np, fe_np = law(nv).astype(np.int32), law(ne).astype(np.int32)
    alpha = float(r.choice([0.0, float(r.uniform(0, 0.05)), float(r.uniform(0.05, 1.0)), 1.0, 1.7]))
    off = int(r.integers(0, 4))
    _announce(f"hot set random seed={seed}: |V|={nv} |E|={ne} max_freq={max_freq} alpha={alpha:.4f}")
    clamp = lambda a: np.clip(a, 0, max_freq)
    dev = lambda a: torch.tensor(a, dtype=torch.int32, device="cuda")
    B = fast.fast_hot_set_budget(alpha, nv, ne)
    hv, he, sv, se = _select_gpu(dev(fv_np), dev(fe_np), max_freq, B, slot_offset=off)
    ov, oe = oracle.greedy_hot_set(clamp(fv_np), clamp(fe_np), alpha)
    assert hv.size + he.size == B == ov.size + oe.size
    assert np.array_equal(hv, np.sort(ov)) and np.array_equal(he, np.sort(oe))
    _check_slots(sv, hv, nv)
    _check_slots(se, he, ne)
