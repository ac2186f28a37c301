"""The whole-block parity helpers on the CPU: the contiguous segment ranges
cover every segment once, and the oracle run range by range on threads
recomposes the oracle run on the whole block exactly (attention forward and
backward, time encoding, temporal sampling), so the full-size GPU
comparisons check what the oracle computes for the whole block."""
import numpy as np
import pytest

import oracle
from synth import make_batch, make_temporal_graph, omega_phi, sampler_roots
from tests.parity import (check_attention_block_full, check_time_encode_full, oracle_sample_chunks,
                          segment_ranges)


@pytest.mark.parametrize("counts,parts", [([3, 0, 5, 1, 0, 0, 7], 4), ([0, 0, 0], 2), ([4], 8),
                                          ([1] * 100, 7), ([0, 9, 0], 1)])
def test_segment_ranges_cover_every_segment_once(counts, parts):
    off = oracle.csr_offsets(np.asarray(counts, np.int32))
    r = segment_ranges(off, parts)
    assert r[0][0] == 0 and r[-1][1] == len(counts) and len(r) <= parts
    assert all(a < c for a, c in r) and all(r[i][1] == r[i + 1][0] for i in range(len(r) - 1))
    assert segment_ranges(oracle.csr_offsets(np.zeros(0, np.int32)), 3) == []


def test_range_checks_accept_the_whole_block_oracle_and_reject_a_changed_row():
    import torch
    b = make_batch(2)
    blk = b.blocks[0]
    off = oracle.csr_offsets(blk.counts)
    N, E, H, dh = blk.num_dst, blk.num_edges, 2, 6
    r = np.random.default_rng(3)
    ins = {k: torch.from_numpy(r.standard_normal(s).astype(np.float32))
           for k, s in (("Q", (N, H, dh)), ("K", (E, H, dh)), ("V", (E, H, dh)), ("dO", (N, H, dh)))}
    f64 = {k: v.double().numpy() for k, v in ins.items()}
    out, lse, alpha, _ = oracle.edge_attention_fwd(off, f64["Q"], f64["K"], f64["V"], 0.4, 0.2)
    dQ, dK, dV = oracle.edge_attention_bwd(off, f64["Q"], f64["K"], f64["V"], f64["dO"], 0.4, 0.2)
    dalpha, _ = oracle.aggregate_bwd(off, alpha, f64["V"], f64["dO"])
    fused = [torch.from_numpy(x) for x in (out, lse, dQ, dK, dV)]
    unf = [torch.from_numpy(x) for x in (alpha, lse, out, dalpha, dV, dQ, dK)]
    assert check_attention_block_full(off, ins, fused, fused, unf, 0.4, 0.2, "f32", "whole", parts=9) > 1
    bad = [t.clone() for t in fused]
    bad[3][E - 1, 1, 2] += 1e-3                   # the last edge's dK
    with pytest.raises(AssertionError):
        check_attention_block_full(off, ins, bad, None, None, 0.4, 0.2, "f32", "planted", parts=9)
    om, ph = omega_phi(20)
    te = oracle.time_encode(off, blk.dst_t, blk.edge_t, om, ph)
    check_time_encode_full(off, blk.dst_t, blk.edge_t, om, ph, torch.from_numpy(te), "f32", "te", parts=5)
    te[0, 0] += 1e-3
    with pytest.raises(AssertionError):
        check_time_encode_full(off, blk.dst_t, blk.edge_t, om, ph, torch.from_numpy(te), "f32", "te", parts=5)


def test_chunked_sampling_equals_the_whole_batch():
    g = make_temporal_graph(2000, 30000, seed=3)
    roots, rt = sampler_roots(g, 300, seed=3)
    roots[::17] = -1
    want = oracle.sample_recent(g.indptr, g.nbr, g.ts, g.eid, roots, rt, 10)
    for chunk in (1, 7, 256, 5000):
        got = oracle_sample_chunks(g, roots, rt, 10, chunk)
        for x, y in zip(got, want):
            assert x.dtype == y.dtype and np.array_equal(x, y)
