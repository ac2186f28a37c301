"""The seeded input generators (CPU): shapes, laws and the structural
properties the operators' contracts rely on."""
import numpy as np

from synth import make_batch, make_temporal_graph, presampled_ids, sampler_roots


def test_presampled_batches_share_the_workload_id_maps():
    nodes, edges, nb, eb = presampled_ids(2, 3)
    b = make_batch(2)
    assert nb == b.node_bound and eb == b.edge_bound
    assert [x.size for x in nodes] == [b.node_ids.size] * 3
    assert [x.size for x in edges] == [b.edge_ids.size] * 3
    for x, bound in ((nodes, nb), (edges, eb)):
        assert all(a.min() >= 0 and a.max() < bound for a in x)
    assert not np.array_equal(nodes[0], nodes[1])                 # a fresh draw per batch
    # the hottest id of every pre-sampled batch is the hottest id of the batch (same map)
    top = lambda a: np.bincount(a).argmax()
    assert top(nodes[0]) == top(nodes[1]) == top(b.node_ids)


def test_temporal_graph_is_time_sorted_per_node():
    g = make_temporal_graph(5000, 40000, seed=3)
    assert g.indptr[0] == 0 and g.indptr[-1] == 2 * 40000 and np.all(np.diff(g.indptr) >= 0)
    node = np.repeat(np.arange(g.num_nodes), np.diff(g.indptr))
    # per node, entries in non-decreasing time and, at equal times, event order
    same = node[1:] == node[:-1]
    dt = np.diff(g.ts)
    assert np.all(dt[same] >= 0)
    tie = same & (dt == 0)
    assert np.all(np.diff(g.eid)[tie] >= 0)
    # every event sits under both of its endpoints
    assert np.array_equal(np.sort(g.eid), np.repeat(np.arange(40000), 2))
    src_of = np.zeros(40000, np.int64)
    src_of[g.eid[node == g.ev_src[g.eid]]] = 1
    assert src_of.sum() == 40000
    assert np.all(np.diff(g.ev_t) >= 0)


def test_sampler_roots_come_from_the_stream():
    g = make_temporal_graph(5000, 40000, seed=4)
    roots, rt = sampler_roots(g, 300, seed=4)
    assert roots.shape == rt.shape == (900,)
    assert np.all((roots >= 0) & (roots < g.num_nodes))
    assert np.array_equal(rt[:300], rt[300:600]) and np.array_equal(rt[:300], rt[600:])
    assert np.all(np.diff(rt[:300]) >= 0) and rt.min() >= g.ev_t[int(0.8 * 40000)]


def test_batches_are_reproducible():
    a, b = make_batch(2), make_batch(2)
    assert np.array_equal(a.node_ids, b.node_ids) and np.array_equal(a.blocks[0].edge_t, b.blocks[0].edge_t)
