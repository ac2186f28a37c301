"""Seeded synthetic temporal-subgraph batches.

This module only *draws* inputs: topology (per-destination edge counts), node
and edge ids, timestamps, feature tables and the dense operands Q/K/V/dOut.
It performs none of the operators' arithmetic (no offsets scan, no dedup, no
time encoding, no softmax or aggregation); both the HIP path and the CPU
oracle receive exactly the arrays produced here.

Workload shapes follow the paper's training setting (Sec. 6.1: top-k most
recent temporal neighbours with k=10, 2-layer message passing, TGAT-style
attention with random Fourier time features) and its dataset statistics
(Table 3: 172-wide edge features, 100/128-wide node features; Table 1: high
within-batch id repetition).  The five named workloads are:

  0 tiny     64 destinations x 10 neighbours, ids uniform over 1e3, 1 layer
  1 layer1   1,800 roots x 10 neighbours, ids uniform over 1e4, 1 layer
  2 skewed   1,800 roots, 2 hops, per-node fan-out ~ truncated Zipf(1.5) on
             [1,10] with 5% of nodes forced to zero, ids Zipf(1.2) over 1e5
  3 large    12,000 roots, 2 hops x 20, ids uniform over 1e6, bf16 storage,
             4 heads x 32
  4 bigdedup 24,000 roots, 2 hops x 10, node ids Zipf(1.1) over 1e7 with a
             1e7 x 100 fp32 table, edge ids Zipf(1.1) over 2e8 served from a
             2e6-row 172-wide fp32 edge-feature cache (slot map)

Random streams: numpy ``default_rng([seed, stream])`` with ``seed = 1000 +
config``; stream 0 topology, 1 ids, 2 timestamps; torch generators seeded
``seed*16 + stream`` draw tables (3 node, 4 edge) and operands (5 Q, 6 K,
7 V, 8 dOut; +16 per layer block).
"""
from __future__ import annotations

import math
from dataclasses import dataclass, field
from typing import List, Optional

import numpy as np

__all__ = [
    "CONFIGS", "LayerBlock", "Batch", "make_batch", "make_block_operands",
    "make_table", "make_slot_map", "omega_phi", "tiny_graph",
]

# --------------------------------------------------------------------------
# workload table
# --------------------------------------------------------------------------
CONFIGS = {
    0: dict(name="tiny", roots=64, hops=1, fanout=(10,), deg_law="const",
            node_law=("uniform", 1_000), edge_law=("perm", None),
            H=2, dh=50, d_t=100, dtype="f32", node_D=100, edge_D=172,
            edge_cache_rows=None, root_times="uniform"),
    1: dict(name="layer1", roots=1_800, hops=1, fanout=(10,), deg_law="const",
            node_law=("uniform", 10_000), edge_law=("perm", None),
            H=2, dh=50, d_t=100, dtype="f32", node_D=100, edge_D=172,
            edge_cache_rows=None, root_times="sorted"),
    2: dict(name="skewed", roots=1_800, hops=2, fanout=(10, 10), deg_law="zipf1.5",
            node_law=("zipf", 100_000, 1.2), edge_law=("zipf", 1_000_000, 1.2),
            H=2, dh=50, d_t=100, dtype="f32", node_D=100, edge_D=172,
            edge_cache_rows=None, root_times="sorted"),
    3: dict(name="large", roots=12_000, hops=2, fanout=(20, 20), deg_law="const",
            node_law=("uniform", 1_000_000), edge_law=("uniform", 10_000_000),
            H=4, dh=32, d_t=128, dtype="bf16", node_D=128, edge_D=172,
            edge_cache_rows=None, root_times="sorted"),
    4: dict(name="bigdedup", roots=24_000, hops=2, fanout=(10, 10), deg_law="const",
            node_law=("zipf", 10_000_000, 1.1), edge_law=("zipf", 200_000_000, 1.1),
            H=2, dh=50, d_t=100, dtype="f32", node_D=100, edge_D=172,
            edge_cache_rows=2_000_000, root_times="sorted"),
}

T_MAX = 1.0e4          # root timestamps are drawn in [0, T_MAX)
ZERO_DEG_FRAC = 0.05   # skewed workload: share of nodes forced to degree 0


@dataclass
class LayerBlock:
    """One message-flow block: destinations in CSR order, edges grouped by
    destination (edges of destination v are contiguous and in order)."""
    counts: np.ndarray      # int32 [N]  edges per destination segment
    dst_t: np.ndarray       # float32 [N] destination (query) timestamps
    edge_t: np.ndarray      # float32 [E] edge timestamps, < dst_t of their segment
    src_ids: np.ndarray     # int64 [E]  source node id of each edge
    edge_ids: np.ndarray    # int64 [E]  edge id of each edge

    @property
    def num_dst(self) -> int:
        return int(self.counts.shape[0])

    @property
    def num_edges(self) -> int:
        return int(self.edge_t.shape[0])


@dataclass
class Batch:
    cfg: int
    name: str
    H: int
    dh: int
    d_t: int
    dtype: str                      # storage dtype of operands: "f32" | "bf16"
    blocks: List[LayerBlock]        # blocks[0] = layer-1 (input-most) block
    node_ids: np.ndarray            # int64: roots, hop-1 and hop-2 node ids
    edge_ids: np.ndarray            # int64: hop-1 and hop-2 edge ids
    node_bound: int                 # node ids lie in [0, node_bound)
    edge_bound: int                 # edge ids lie in [0, edge_bound)
    node_D: int
    edge_D: int
    edge_cache_rows: Optional[int]  # None: edge table is indexed by id
    edge_map: Optional[tuple] = None  # (a, b): rank r -> id (a*(r-1)+b) % bound
    seed: int = 0
    node_map: Optional[tuple] = None  # the same for node ids (Zipf laws only)
    extra: dict = field(default_factory=dict)

    @property
    def sampled_edges(self) -> int:
        return sum(b.num_edges for b in self.blocks)


# --------------------------------------------------------------------------
# helpers
# --------------------------------------------------------------------------
def _rng(seed: int, stream: int) -> np.random.Generator:
    return np.random.default_rng([seed, stream])


def _affine(bound: int, rng: np.random.Generator):
    """A seeded bijection of [0, bound): r -> (a*r + b) % bound, gcd(a,bound)=1."""
    while True:
        a = int(rng.integers(bound // 3 + 1, bound)) if bound > 2 else 1
        if math.gcd(a, bound) == 1:
            break
    b = int(rng.integers(0, bound))
    return a, b


def _zipf_ranks(rng, s: float, bound: int, n: int) -> np.ndarray:
    """Ranks 1..bound drawn from Zipf(s), truncated by redrawing values > bound."""
    out = rng.zipf(s, n).astype(np.int64)
    bad = out > bound
    while bad.any():
        out[bad] = rng.zipf(s, int(bad.sum()))
        bad = out > bound
    return out


def _draw_ids(law, n, rng, amap):
    kind = law[0]
    if kind == "uniform":
        return rng.integers(0, law[1], n, dtype=np.int64)
    if kind == "zipf":
        bound, s = law[1], law[2]
        r = _zipf_ranks(rng, s, bound, n)
        a, b = amap
        return (a * (r - 1) + b) % bound
    raise ValueError(kind)


def _degrees(law, fan, n, rng):
    if law == "const":
        return np.full(n, fan, dtype=np.int32)
    if law == "zipf1.5":
        k = np.arange(1, fan + 1, dtype=np.float64)
        p = k ** -1.5
        p /= p.sum()
        deg = rng.choice(np.arange(1, fan + 1), size=n, p=p).astype(np.int32)
        zero = rng.random(n) < ZERO_DEG_FRAC
        deg[zero] = 0
        return deg
    raise ValueError(law)


def _child_times(parent_t: np.ndarray, counts: np.ndarray, rng) -> np.ndarray:
    """Edge times t_e = t_parent * U[0,1), redrawn until strictly below the parent."""
    pt = np.repeat(parent_t, counts).astype(np.float32)
    t = (pt.astype(np.float64) * rng.random(pt.shape[0])).astype(np.float32)
    bad = t >= pt
    while bad.any():
        t[bad] = (pt[bad].astype(np.float64) * rng.random(int(bad.sum()))).astype(np.float32)
        bad = t >= pt
    return t


def omega_phi(d_t: int):
    """Time-encoding frequencies omega_j = 10^(-9 j/(d_t-1)) and phases phi_j = 0,
    as float32 arrays (the same arrays are handed to both implementations)."""
    if d_t == 1:
        om = np.ones(1, dtype=np.float64)
    else:
        om = 10.0 ** (-9.0 * np.arange(d_t, dtype=np.float64) / (d_t - 1))
    return om.astype(np.float32), np.zeros(d_t, dtype=np.float32)


# --------------------------------------------------------------------------
# batches
# --------------------------------------------------------------------------
def make_batch(cfg: int, seed: Optional[int] = None) -> Batch:
    c = CONFIGS[cfg]
    seed = 1000 + cfg if seed is None else seed
    r_top, r_ids, r_t = _rng(seed, 0), _rng(seed, 1), _rng(seed, 2)
    R = c["roots"]
    node_law, edge_law = c["node_law"], c["edge_law"]
    node_bound = node_law[1]
    node_map = _affine(node_bound, r_ids) if node_law[0] == "zipf" else None

    # roots
    root_ids = _draw_ids(node_law, R, r_ids, node_map)
    rt = r_t.random(R) * T_MAX
    while (rt <= 0).any():
        rt[rt <= 0] = r_t.random(int((rt <= 0).sum())) * T_MAX
    if c["root_times"] == "sorted":
        rt = np.sort(rt)
    root_t = rt.astype(np.float32)

    # hop 1
    c1 = _degrees(c["deg_law"], c["fanout"][0], R, r_top)
    E1 = int(c1.sum())
    ids1 = _draw_ids(node_law, E1, r_ids, node_map)
    t1 = _child_times(root_t, c1, r_t)
    hop_counts, hop_ids, hop_t, hop_parent_t = [c1], [ids1], [t1], [root_t]
    if c["hops"] == 2:
        c2 = _degrees(c["deg_law"], c["fanout"][1], E1, r_top)
        E2 = int(c2.sum())
        ids2 = _draw_ids(node_law, E2, r_ids, node_map)
        t2 = _child_times(t1, c2, r_t)
        hop_counts.append(c2); hop_ids.append(ids2); hop_t.append(t2)
        hop_parent_t.append(t1)
    n_edges = sum(int(x.sum()) for x in hop_counts)

    # edge ids
    edge_map = None
    if edge_law[0] == "perm":
        edge_bound = n_edges
        all_eids = r_ids.permutation(n_edges).astype(np.int64)
    else:
        edge_bound = edge_law[1]
        if edge_law[0] == "zipf":
            edge_map = _affine(edge_bound, r_ids)
        all_eids = _draw_ids(edge_law, n_edges, r_ids, edge_map)
    eids = np.split(all_eids, np.cumsum([int(x.sum()) for x in hop_counts])[:-1])

    # layer blocks (TGL message-flow order: roots first, then hop-1 nodes)
    blocks = []
    if c["hops"] == 1:
        blocks.append(LayerBlock(c1.astype(np.int32), root_t, t1, ids1, eids[0]))
    else:
        blocks.append(LayerBlock(
            np.concatenate([c1, hop_counts[1]]).astype(np.int32),
            np.concatenate([root_t, t1]).astype(np.float32),
            np.concatenate([t1, hop_t[1]]).astype(np.float32),
            np.concatenate([ids1, hop_ids[1]]).astype(np.int64),
            np.concatenate([eids[0], eids[1]]).astype(np.int64)))
        blocks.append(LayerBlock(c1.astype(np.int32), root_t, t1, ids1, eids[0]))

    node_ids = np.concatenate([root_ids] + hop_ids).astype(np.int64)
    return Batch(cfg=cfg, name=c["name"], H=c["H"], dh=c["dh"], d_t=c["d_t"],
                 dtype=c["dtype"], blocks=blocks, node_ids=node_ids,
                 edge_ids=all_eids, node_bound=node_bound, edge_bound=edge_bound,
                 node_D=c["node_D"], edge_D=c["edge_D"],
                 edge_cache_rows=c["edge_cache_rows"], edge_map=edge_map, seed=seed,
                 node_map=node_map)


def presampled_ids(cfg: int, num_batches: int, seed: Optional[int] = None):
    """Node and edge ids of `num_batches` pre-sampled batches of one graph:
    the id laws, sizes and rank -> id maps of make_batch(cfg, seed), with a
    fresh draw per batch (stream 100 + k), so that the hot ids agree with
    the batch that make_batch returns.  An edge law that is a per-batch
    permutation becomes uniform over its bound.  Returns (node_batches,
    edge_batches, node_bound, edge_bound)."""
    c = CONFIGS[cfg]
    b = make_batch(cfg, seed)
    nodes, edges = [], []
    node_law, edge_law = c["node_law"], c["edge_law"]
    if edge_law[0] == "perm":
        edge_law = ("uniform", b.edge_bound)
    for k in range(num_batches):
        r = _rng(b.seed, 100 + k)
        nodes.append(_draw_ids(node_law, b.node_ids.size, r, b.node_map))
        edges.append(_draw_ids(edge_law, b.edge_ids.size, r, b.edge_map))
    return nodes, edges, b.node_bound, b.edge_bound


@dataclass
class TemporalGraph:
    """A T-CSR temporal graph: node v's entries are p in [indptr[v],
    indptr[v+1]), each an event of v with neighbour nbr[p] at time ts[p]
    (event id eid[p]), in time order (ties in event order).  `events` holds
    the chronological stream (src, dst, t) the graph was built from."""
    indptr: np.ndarray   # int64 [V+1]
    nbr: np.ndarray      # int64 [M]
    ts: np.ndarray       # float32 [M]
    eid: np.ndarray      # int64 [M]
    ev_src: np.ndarray   # int64 [num_events]
    ev_dst: np.ndarray   # int64 [num_events]
    ev_t: np.ndarray     # float32 [num_events], non-decreasing

    @property
    def num_nodes(self) -> int:
        return self.indptr.shape[0] - 1


def make_temporal_graph(num_nodes: int, num_events: int, seed: int = 0, zipf_s: float = 1.1):
    """Event stream over `num_nodes` nodes: endpoints Zipf(zipf_s) ranks mapped
    by a seeded affine bijection (a few hub nodes hold most events, as in the
    paper's interaction graphs), times sorted U(0, T_MAX).  Every event is
    stored under both endpoints (an undirected temporal graph)."""
    r = _rng(seed, 20)
    amap = _affine(num_nodes, r)
    law = ("zipf", num_nodes, zipf_s)
    src = _draw_ids(law, num_events, r, amap)
    dst = _draw_ids(law, num_events, r, amap)
    t = np.sort(r.random(num_events) * T_MAX).astype(np.float32)
    # each event's two entries side by side in stream order, which is (time,
    # event id) order already; one stable sort by node keeps it within a node
    node = np.empty(2 * num_events, np.int64)
    nbr = np.empty(2 * num_events, np.int64)
    node[0::2], node[1::2] = src, dst
    nbr[0::2], nbr[1::2] = dst, src
    ts = np.repeat(t, 2)
    eid = np.repeat(np.arange(num_events, dtype=np.int64), 2)
    order = np.argsort(node, kind="stable")
    indptr = np.concatenate([[0], np.cumsum(np.bincount(node, minlength=num_nodes))]).astype(np.int64)
    return TemporalGraph(indptr, nbr[order].astype(np.int64), ts[order].astype(np.float32),
                         eid[order], src, dst, t)


def sampler_roots(g: TemporalGraph, num_events: int, seed: int = 0):
    """Roots of one training batch: `num_events` consecutive events from the
    last fifth of the stream, each giving (src, t), (dst, t) and a uniform
    negative destination at t.  Returns (roots int64 [3B], root_t float32 [3B])."""
    r = _rng(seed, 21)
    n = g.ev_t.shape[0]
    lo = int(0.8 * n)
    e0 = int(r.integers(lo, max(lo + 1, n - num_events)))
    sl = slice(e0, e0 + num_events)
    neg = r.integers(0, g.num_nodes, num_events, dtype=np.int64)
    roots = np.concatenate([g.ev_src[sl], g.ev_dst[sl], neg]).astype(np.int64)
    t = g.ev_t[sl]
    return roots, np.concatenate([t, t, t]).astype(np.float32)


def tiny_graph(counts, H=2, dh=4, seed=7):
    """A hand-sized block with the given per-destination edge counts (zeros
    allowed); timestamps and ids drawn like the named workloads."""
    rng = _rng(seed, 0)
    counts = np.asarray(counts, dtype=np.int32)
    N = counts.shape[0]
    dst_t = (rng.random(N) * T_MAX + 1.0).astype(np.float32)
    edge_t = _child_times(dst_t, counts, rng)
    E = edge_t.shape[0]
    src = rng.integers(0, 100, E, dtype=np.int64)
    eid = rng.permutation(E).astype(np.int64)
    return LayerBlock(counts, dst_t, edge_t, src, eid)


# --------------------------------------------------------------------------
# dense operands and tables (torch, so they can be drawn directly in HBM)
# --------------------------------------------------------------------------
def _torch_gen(device, seed):
    import torch
    g = torch.Generator(device=device)
    g.manual_seed(int(seed))
    return g


def _randn(shape, dtype, device, seed):
    import torch
    g = _torch_gen(device, seed)
    x = torch.randn(shape, generator=g, device=device, dtype=torch.float32)
    if dtype == "bf16":
        x = x.to(torch.bfloat16)      # round-to-nearest-even; these values are the inputs
    return x


def make_block_operands(batch_or_shape, block_index=0, device="cpu", seed=None,
                        dtype=None, H=None, dh=None):
    """Q [N,H,dh], K/V [E,H,dh], dOut [N,H,dh], N(0,1) in the storage dtype.

    `batch_or_shape` is a Batch (operands for batch.blocks[block_index]) or an
    (N, E) tuple together with explicit H, dh, dtype, seed."""
    if isinstance(batch_or_shape, Batch):
        b = batch_or_shape
        blk = b.blocks[block_index]
        N, E = blk.num_dst, blk.num_edges
        H, dh, dtype = b.H, b.dh, b.dtype
        seed = b.seed if seed is None else seed
    else:
        N, E = batch_or_shape
        seed = 0 if seed is None else seed
        dtype = dtype or "f32"
    base = int(seed) * 16 + 16 * block_index
    return dict(
        Q=_randn((N, H, dh), dtype, device, base + 5),
        K=_randn((E, H, dh), dtype, device, base + 6),
        V=_randn((E, H, dh), dtype, device, base + 7),
        dO=_randn((N, H, dh), dtype, device, base + 8),
    )


def make_table(rows: int, D: int, dtype: str, device="cpu", seed=0, stream=3):
    """A [rows, D] feature table, N(0,1) in the storage dtype."""
    return _randn((rows, D), dtype, device, int(seed) * 16 + stream)


def make_slot_map(batch: Batch, device="cpu"):
    """Edge-feature cache layout of the big-dedup workload: the cache holds the
    `edge_cache_rows` most frequent ids of the Zipf law (ranks 1..C, which is
    what a frequency-greedy hot set converges to); slot_map[id] = rank-1 for
    cached ids and -1 otherwise.  Returns (slot_map int32 [edge_bound])."""
    import torch
    assert batch.edge_cache_rows is not None and batch.edge_map is not None
    a, b = batch.edge_map
    C = batch.edge_cache_rows
    ranks = torch.arange(C, dtype=torch.int64, device=device)
    ids = (ranks * a + b) % batch.edge_bound
    sm = torch.full((batch.edge_bound,), -1, dtype=torch.int32, device=device)
    sm[ids] = ranks.to(torch.int32)
    return sm
