"""GPU parity: every operator through the C ABI against the fp64 CPU oracle.

Every workload is compared in full: the small ones span many workgroups and
end in a ragged tail; the two large ones run at their full size in the
launch configuration the benchmark times, and the oracle checks every
segment of them over contiguous segment ranges on all host threads.
"""
import os

import numpy as np
import pytest
import torch

import oracle
import paper_2607_05095_amd as fast
from synth import make_batch, make_block_operands, make_slot_map, make_table, omega_phi, tiny_graph
from tests.parity import (SLOPE, assert_bwd_close, assert_close, bwd_reference_with_kinks,
                          check_attention_block_full, check_time_encode_full, sub_csr, tdtype,
                          to_dev)

pytestmark = pytest.mark.gpu

DT = {"f32": fast.F32, "bf16": fast.BF16}


def _announce(msg):
    print(f"[parity] {msg}", flush=True)


# ------------------------------------------------------------------ device block
class DevBlock:
    """A layer block on the GPU: offsets from the oracle, timestamps, operands."""

    def __init__(self, counts, dst_t, edge_t, ops, H, dh, dt):
        self.counts = np.asarray(counts, dtype=np.int32)
        self.off = oracle.csr_offsets(self.counts)
        self.N, self.E = self.counts.shape[0], int(self.off[-1])
        self.H, self.dh, self.dt = H, dh, dt
        self.d_off = to_dev(self.off)
        self.d_dst_t = to_dev(np.asarray(dst_t, dtype=np.float32))
        self.d_edge_t = to_dev(np.asarray(edge_t, dtype=np.float32))
        self.ops = {k: v.cuda() for k, v in ops.items()}
        self.g = fast.tcsr(self.d_off, self.E, edge_t=self.d_edge_t, dst_t=self.d_dst_t)
        self.scale = float(np.float32(1.0 / np.sqrt(dh)))

    def empty(self, rows, dtype=None):
        return torch.empty((rows, self.H, self.dh), dtype=dtype or tdtype(self.dt), device="cuda")

    def scalars(self, rows):
        return torch.empty((rows, self.H), dtype=torch.float32, device="cuda")


def _block_from_batch(b, i):
    blk = b.blocks[i]
    ops = make_block_operands(b, i, device="cuda")
    return DevBlock(blk.counts, blk.dst_t, blk.edge_t, ops, b.H, b.dh, b.dtype)


def _host(t):
    return t.detach().float().cpu().double().numpy()


def _run_fused(d, with_lse=True, slope=SLOPE):
    o = d.ops
    out = d.empty(d.N)
    lse = d.scalars(d.N)
    fast.fast_edge_attention_fwd(d.g, d.H, d.dh, DT[d.dt], o["Q"], o["K"], o["V"], d.scale, slope,
                                 out, lse)
    dQ, dK, dV = d.empty(d.N), d.empty(d.E), d.empty(d.E)
    fast.fast_edge_attention_bwd(d.g, d.H, d.dh, DT[d.dt], o["Q"], o["K"], o["V"], d.scale, slope,
                                 lse if with_lse else None, o["dO"], dQ, dK, dV)
    return out, lse, dQ, dK, dV


def _run_fused_packed(d, with_lse=True, slope=SLOPE):
    """The fused pair on packed K|V rows: KV[e] = (K[e], V[e]); the gradients
    come back as dKV[e] = (dK[e], dV[e]), poisoned with NaN beforehand."""
    o = d.ops
    KV = torch.empty((d.E, 2, d.H, d.dh), dtype=tdtype(d.dt), device="cuda")
    KV[:, 0] = o["K"]
    KV[:, 1] = o["V"]
    out = d.empty(d.N)
    lse = d.scalars(d.N)
    fast.fast_edge_attention_fwd_packed(d.g, d.H, d.dh, DT[d.dt], o["Q"], KV if d.E else None,
                                        d.scale, slope, out, lse)
    dQ = d.empty(d.N)
    dKV = torch.full((d.E, 2, d.H, d.dh), float("nan"), dtype=tdtype(d.dt), device="cuda")
    fast.fast_edge_attention_bwd_packed(d.g, d.H, d.dh, DT[d.dt], o["Q"], KV if d.E else None,
                                        d.scale, slope, lse if with_lse else None, o["dO"], dQ,
                                        dKV if d.E else None)
    return out, lse, dQ, dKV[:, 0], dKV[:, 1]


def _run_unfused(d, slope=SLOPE):
    o = d.ops
    alpha, lse = d.scalars(d.E), d.scalars(d.N)
    fast.fast_edge_softmax_fwd(d.g, d.H, d.dh, DT[d.dt], o["Q"], o["K"], d.scale, slope, alpha, lse)
    out = d.empty(d.N)
    fast.fast_temporal_aggregate_fwd(d.g, d.H, d.dh, DT[d.dt], alpha, o["V"], out)
    dalpha, dV = d.scalars(d.E), d.empty(d.E)
    fast.fast_temporal_aggregate_bwd(d.g, d.H, d.dh, DT[d.dt], alpha, o["V"], o["dO"], dalpha, dV)
    dQ, dK = d.empty(d.N), d.empty(d.E)
    fast.fast_edge_softmax_bwd(d.g, d.H, d.dh, DT[d.dt], o["Q"], o["K"], d.scale, slope, alpha,
                               dalpha, dQ, dK)
    return alpha, lse, out, dalpha, dV, dQ, dK


def _check_block(d, segs=None, what="", slope=SLOPE):
    """Fused and unfused operators vs the oracle on all (segs=None) or the
    sampled segments."""
    torch.cuda.synchronize()
    fused = _run_fused(d, with_lse=True, slope=slope)
    fused_nolse = _run_fused(d, with_lse=False, slope=slope)
    unf = _run_unfused(d, slope=slope)
    torch.cuda.synchronize()
    if segs is None:
        segs = np.arange(d.N, dtype=np.int64)
    sub_off, eidx = sub_csr(d.off, segs)
    Q = _host(d.ops["Q"][torch.as_tensor(segs, device="cuda")])
    dO = _host(d.ops["dO"][torch.as_tensor(segs, device="cuda")])
    ei = torch.as_tensor(eidx, device="cuda")
    K = _host(d.ops["K"][ei])
    V = _host(d.ops["V"][ei])
    out, lse, alpha, _ = oracle.edge_attention_fwd(sub_off, Q, K, V, d.scale, slope)
    dalpha, _ = oracle.aggregate_bwd(sub_off, alpha, V, dO)
    dQ, dK, dV, alts = bwd_reference_with_kinks(sub_off, Q, K, V, dO, d.scale, slope)
    sg = torch.as_tensor(segs, device="cuda")
    nz = np.diff(sub_off) > 0
    # forward
    g_out, g_lse, g_dQ, g_dK, g_dV = fused
    assert_close(g_out[sg], out, d.dt, what + " fused out")
    assert_close(_host(g_lse[sg])[nz], lse[nz], "f32", what + " fused lse")
    assert np.all(np.isneginf(_host(g_lse[sg])[~nz])), "empty segment lse must be -inf"
    # fused backward, with and without the saved lse
    for tag, (_, _, bdQ, bdK, bdV) in (("lse", fused), ("nolse", fused_nolse)):
        assert_close(bdV[ei], dV, d.dt, f"{what} fused[{tag}] dV")
        assert_bwd_close(bdQ[sg], bdK[ei], sub_off, dQ, dK, alts, d.dt, f"{what} fused[{tag}]")
    # unfused chain
    u_alpha, u_lse, u_out, u_dalpha, u_dV, u_dQ, u_dK = unf
    assert_close(u_alpha[ei], alpha, "f32", what + " ESM alpha")
    assert_close(_host(u_lse[sg])[nz], lse[nz], "f32", what + " ESM lse")
    assert_close(u_out[sg], out, d.dt, what + " AGG out")
    assert_close(u_dalpha[ei], dalpha, "f32", what + " AGG dalpha")
    assert_close(u_dV[ei], dV, d.dt, what + " AGG dV")
    assert_bwd_close(u_dQ[sg], u_dK[ei], sub_off, dQ, dK, alts, d.dt, what + " ESM-bwd")
    return fused, unf


# ------------------------------------------------------------------ attention: workloads
@pytest.mark.parametrize("cfg", [0, 1, 2])
def test_attention_small_workloads_full(cfg):
    b = make_batch(cfg)
    for i in range(len(b.blocks)):
        _announce(f"attention cfg={cfg} block={i}")
        d = _block_from_batch(b, i)
        _check_block(d, None, f"cfg{cfg}/L{i + 1}")


def _cpu(t):
    return t.detach().cpu() if t is not None else None


@pytest.mark.parametrize("cfg,block", [(3, 0), (3, 1), (4, 0), (4, 1)])
def test_attention_large_workloads_full(cfg, block):
    """The two full-size workloads in the launch configuration the benchmark
    times: every segment of each layer block, fused forward and backward with
    and without the saved lse and the unfused chain, against the oracle run
    over contiguous segment ranges on all host threads."""
    b = make_batch(cfg)
    d = _block_from_batch(b, block)
    _announce(f"attention cfg={cfg} block={block}: N={d.N} E={d.E}, every segment")
    fused = [_cpu(t) for t in _run_fused(d, with_lse=True)]
    fused_nolse = [_cpu(t) for t in _run_fused(d, with_lse=False)]
    unf = [_cpu(t) for t in _run_unfused(d)]
    ins = {k: _cpu(d.ops[k]) for k in ("Q", "K", "V", "dO")}
    torch.cuda.synchronize()
    off = d.off
    del d
    torch.cuda.empty_cache()
    parts = check_attention_block_full(off, ins, fused, fused_nolse, unf, float(np.float32(1.0 / np.sqrt(b.dh))),
                                       SLOPE, b.dtype, f"cfg{cfg}/L{block + 1}")
    _announce(f"  {parts} segment ranges equal to the oracle")


# ------------------------------------------------------------------ attention: edge cases
def _synthetic_block(counts, H, dh, dt, seed=0):
    blk = tiny_graph(counts, H=H, dh=dh, seed=seed + 1)
    ops = make_block_operands((blk.num_dst, blk.num_edges), device="cuda", seed=seed,
                              dtype=dt, H=H, dh=dh)
    return DevBlock(blk.counts, blk.dst_t, blk.edge_t, ops, H, dh, dt)


@pytest.mark.parametrize("name,counts,H,dh,dt", [
    ("single_edge", [1], 2, 50, "f32"),
    ("deg1_everywhere", [1] * 300, 2, 50, "f32"),
    ("all_empty", [0] * 40, 2, 50, "f32"),
    ("empties_mixed", [0, 3, 0, 0, 7, 1, 0, 12, 0], 2, 50, "f32"),
    ("long_segments", [1000, 3, 25, 24, 23, 40, 8, 9, 17], 2, 50, "f32"),
    ("long_bf16", [333, 20, 21, 1, 0, 64], 4, 32, "bf16"),
    ("one_head", [5, 9, 2, 30], 1, 64, "f32"),
    ("odd_dh", [4, 7, 11, 2], 3, 13, "f32"),
    ("wide_dh_P4", [6, 3, 10], 2, 130, "f32"),
    ("wide_dh_P2_bf16", [6, 3, 10], 2, 100, "bf16"),
    ("many_heads", [8, 8, 3, 15], 16, 16, "f32"),
    ("bf16_vec4", [5, 12, 1], 2, 36, "bf16"),
    ("big_block_G", [4, 9], 8, 64, "f32"),
    ("wide_group_512", [3, 7, 1, 12], 5, 130, "f32"),
    ("many_heads_bf16", [6, 2, 9], 64, 16, "bf16"),
])
def test_attention_edge_cases(name, counts, H, dh, dt):
    _announce(f"attention edge case {name}")
    d = _synthetic_block(counts, H, dh, dt, seed=len(counts))
    fused, unf = _check_block(d, None, name)
    if name == "deg1_everywhere":
        # a single-neighbour segment returns its value row exactly
        assert torch.equal(fused[0], d.ops["V"])
        assert torch.equal(unf[0], torch.ones_like(unf[0]))
    if name == "all_empty":
        assert torch.count_nonzero(fused[0]) == 0 and torch.count_nonzero(fused[2]) == 0


@pytest.mark.parametrize("slope", [-0.3, 0.0])
@pytest.mark.parametrize("name,counts,H,dh,dt", [
    ("rowmajor_f32", [10, 1, 0, 7, 30, 10, 25, 3, 12], 2, 50, "f32"),
    ("headmajor_f32", [10, 1, 0, 7, 30, 10, 25, 3, 12], 4, 32, "f32"),
    ("headmajor_bf16", [20, 1, 0, 7, 41, 20, 25, 3, 12], 4, 32, "bf16"),
    ("headmajor_f32_dh50", [10, 2, 0, 29, 10], 3, 50, "f32"),
])
def test_attention_nonpositive_slope(name, counts, H, dh, dt, slope):
    """LeakyReLU slopes of 0 and below: the backward's branch is the sign of
    the pre-activation, which a negative slope hides in the activated logit.
    Segments longer than the backward's register window re-read their rows,
    so both of its paths are covered.  fp32 2 x 50 runs the row-major
    kernels; the other shapes run the head-major ones."""
    _announce(f"attention slope={slope} {name}")
    d = _synthetic_block(counts * 8, H, dh, dt, seed=11 + len(counts))
    _check_block(d, None, f"{name} slope={slope}", slope=slope)


# ------------------------------------------------------------------ attention: packed K|V rows
_PACKED_NAMES = ("out", "lse", "dQ", "dK", "dV")


def _assert_packed_equals_separate(d, what, slope=SLOPE):
    for with_lse in (True, False):
        sep = _run_fused(d, with_lse=with_lse, slope=slope)
        pk = _run_fused_packed(d, with_lse=with_lse, slope=slope)
        torch.cuda.synchronize()
        for n, x, y in zip(_PACKED_NAMES, sep, pk):
            assert torch.equal(x, y), f"{what} lse={with_lse}: packed {n} differs from separate"


def _random_attention_case(seed):
    """A seeded random shape: H in {1..8}, dh in [1, 128], fp32 or bf16, a
    slope of 0.2, 0, -0.3 or 1, and 20-60 segments of mixed degree (empty,
    1-30, and now and then 100-400 edges)."""
    r = np.random.default_rng(4000 + seed)
    H = int(r.choice([1, 2, 3, 4, 5, 8]))
    dh = int(r.integers(1, 129))
    dt = "bf16" if r.random() < 0.4 else "f32"
    slope = float(r.choice([0.2, 0.0, -0.3, 1.0]))
    N = int(r.integers(20, 61))
    counts = r.integers(1, 31, N)
    counts[r.random(N) < 0.1] = 0
    counts[r.random(N) < 0.05] = r.integers(100, 401)
    return [int(c) for c in counts], H, dh, dt, slope


@pytest.mark.parametrize("seed", range(48))
def test_attention_random_shapes(seed):
    """Seeded random head counts, head widths (every vector width and lane
    layout those reach), storage types, slopes and degree mixes: the fused
    operators (with and without the saved lse) and the unfused chain against
    the oracle, and packed K|V rows equal to separate arrays bit for bit."""
    counts, H, dh, dt, slope = _random_attention_case(seed)
    _announce(f"attention random shape seed={seed}: H={H} dh={dh} {dt} slope={slope} "
              f"N={len(counts)} E={sum(counts)}")
    d = _synthetic_block(counts, H, dh, dt, seed=100 + seed)
    _check_block(d, None, f"random seed={seed}", slope=slope)
    _assert_packed_equals_separate(d, f"random seed={seed}", slope=slope)


@pytest.mark.parametrize("cfg", [0, 1, 2, 3, 4])
def test_attention_packed_kv_equals_separate_workloads(cfg):
    """Packed K|V rows run the same kernels with rows 2F apart: every output
    equals the separate-array operator's (itself checked against the oracle in
    full above) bit for bit, on every block of every workload at full size."""
    b = make_batch(cfg)
    for i in range(len(b.blocks)):
        d = _block_from_batch(b, i)
        _announce(f"packed K|V cfg={cfg} block={i}: N={d.N} E={d.E}")
        _assert_packed_equals_separate(d, f"cfg{cfg}/L{i + 1}")
        del d
        torch.cuda.empty_cache()


@pytest.mark.parametrize("name,counts,H,dh,dt,slope", [
    ("long_segments_rowmajor", [1000, 3, 25, 24, 23, 40, 8, 9, 17], 2, 50, "f32", SLOPE),
    ("long_bf16", [333, 20, 21, 1, 0, 64], 4, 32, "bf16", SLOPE),
    ("empties_mixed", [0, 3, 0, 0, 7, 1, 0, 12, 0], 2, 50, "f32", SLOPE),
    ("odd_dh_vec1", [4, 7, 11, 2], 3, 13, "f32", SLOPE),
    ("bf16_vec4", [5, 12, 1], 2, 36, "bf16", SLOPE),
    ("wide_dh_P4", [6, 3, 10], 2, 130, "f32", SLOPE),
    ("many_heads_bf16", [6, 2, 9], 64, 16, "bf16", SLOPE),
    ("rowmajor_negative_slope", [10, 1, 0, 7, 30, 10, 25, 3, 12] * 8, 2, 50, "f32", -0.3),
    ("headmajor_bf16_zero_slope", [20, 1, 0, 7, 41, 20, 25, 3, 12] * 8, 4, 32, "bf16", 0.0),
])
def test_attention_packed_kv_edge_cases(name, counts, H, dh, dt, slope):
    """Both lane layouts, every vector width, segments beyond the backward's
    register window, empty segments, and slopes of 0 and below."""
    _announce(f"packed K|V edge case {name}")
    d = _synthetic_block(counts, H, dh, dt, seed=len(counts) + 3)
    _assert_packed_equals_separate(d, name, slope=slope)


@pytest.mark.parametrize("case", ["cfg1", "long_bf16"])
def test_attention_packed_kv_vs_oracle(case):
    """The packed operators against the oracle directly, element by element."""
    _announce(f"packed K|V vs oracle {case}")
    if case == "cfg1":
        d = _block_from_batch(make_batch(1), 0)
    else:
        d = _synthetic_block([333, 20, 21, 1, 0, 64], 4, 32, "bf16", seed=9)
    out, lse, dQ, dK, dV = _run_fused_packed(d)
    torch.cuda.synchronize()
    Q, K, V, dO = (_host(d.ops[k]) for k in ("Q", "K", "V", "dO"))
    r_out, r_lse, _, _ = oracle.edge_attention_fwd(d.off, Q, K, V, d.scale, SLOPE)
    r_dQ, r_dK, r_dV, alts = bwd_reference_with_kinks(d.off, Q, K, V, dO, d.scale, SLOPE)
    nz = np.diff(d.off) > 0
    assert_close(out, r_out, d.dt, case + " packed out")
    assert_close(_host(lse)[nz], r_lse[nz], "f32", case + " packed lse")
    assert_close(dV, r_dV, d.dt, case + " packed dV")
    assert_bwd_close(dQ, dK, d.off, r_dQ, r_dK, alts, d.dt, case + " packed")


def test_attention_empty_graph_and_zero_edges():
    _announce("attention N=0")
    d0 = torch.zeros(1, dtype=torch.int32, device="cuda")
    g = fast.tcsr(d0, 0)
    fast.fast_edge_attention_fwd(g, 2, 50, fast.F32, None, None, None, 0.1, SLOPE, None, None)
    fast.fast_edge_attention_bwd(g, 2, 50, fast.F32, None, None, None, 0.1, SLOPE, None, None,
                                 None, None, None)
    fast.fast_edge_attention_fwd_packed(g, 2, 50, fast.F32, None, None, 0.1, SLOPE, None, None)
    fast.fast_edge_attention_bwd_packed(g, 2, 50, fast.F32, None, None, 0.1, SLOPE, None, None,
                                        None, None)
    # destinations without edges: no K|V rows at all, every output row 0, lse -inf
    d = _synthetic_block([0, 0, 0], 2, 50, "f32", seed=4)
    out, lse, dQ, _, _ = _run_fused_packed(d)
    torch.cuda.synchronize()
    assert torch.count_nonzero(out) == 0 and torch.count_nonzero(dQ) == 0
    assert torch.all(torch.isneginf(lse))


def test_attention_run_to_run_bitwise_determinism():
    _announce("attention determinism cfg=2")
    b = make_batch(2)
    d = _block_from_batch(b, 0)
    r1 = _run_fused(d)
    r2 = _run_fused(d)
    torch.cuda.synchronize()
    for x, y in zip(r1, r2):
        assert torch.equal(x, y)


def test_fused_equals_unfused_composition():
    _announce("fused vs unfused cfg=1")
    b = make_batch(1)
    d = _block_from_batch(b, 0)
    out, lse, dQ, dK, dV = _run_fused(d)
    _, u_lse, u_out, _, u_dV, u_dQ, u_dK = _run_unfused(d)
    torch.cuda.synchronize()
    for a_, b_, n in ((out, u_out, "out"), (dV, u_dV, "dV"), (dQ, u_dQ, "dQ"), (dK, u_dK, "dK")):
        assert_close(a_, _host(b_), "f32", f"fused vs unfused {n}")


# ------------------------------------------------------------------ offsets (a1)
@pytest.mark.parametrize("case", ["cfg0", "cfg2", "cfg3", "cfg4", "empty", "zeros", "ragged", "big",
                                  "one_tile", "tiles_2048", "tiles_2049"])
def test_csr_offsets_bit_exact(case):
    _announce(f"offsets {case}")
    r = np.random.default_rng(1)
    counts = {
        "cfg0": lambda: make_batch(0).blocks[0].counts,
        "cfg2": lambda: make_batch(2).blocks[0].counts,
        "cfg3": lambda: make_batch(3).blocks[0].counts,
        "cfg4": lambda: make_batch(4).blocks[0].counts,
        "empty": lambda: np.zeros(0, np.int32),
        "zeros": lambda: np.zeros(5000, np.int32),
        "ragged": lambda: r.integers(0, 30, 2049 * 3 + 7).astype(np.int32),
        "big": lambda: r.integers(0, 3, 3_000_001).astype(np.int32),
        # the scan's two launch plans: up to 2048 tiles of 2048 counts each
        # tile adds up the preceding tile sums, beyond that a one-block scan
        "one_tile": lambda: r.integers(0, 50, 2048).astype(np.int32),
        "tiles_2048": lambda: r.integers(0, 5, 2048 * 2048).astype(np.int32),
        "tiles_2049": lambda: r.integers(0, 5, 2048 * 2048 + 1).astype(np.int32),
    }[case]()
    n = counts.shape[0]
    d_counts = to_dev(counts) if n else torch.zeros(1, dtype=torch.int32, device="cuda")
    off = torch.full((n + 1,), -7, dtype=torch.int32, device="cuda")
    wsb = fast.fast_csr_offsets_workspace(n)
    ws = torch.empty(wsb, dtype=torch.uint8, device="cuda")
    fast.fast_csr_offsets(d_counts, n, off, ws, wsb)
    assert np.array_equal(off.cpu().numpy(), oracle.csr_offsets(counts))


def _offsets_batched(counts_list):
    d_counts = [to_dev(np.asarray(c, np.int32)) if len(c) else None for c in counts_list]
    ns = [len(c) for c in counts_list]
    outs = [torch.full((n + 1,), -7, dtype=torch.int32, device="cuda") for n in ns]
    wsb = fast.fast_csr_offsets_batched_workspace(ns)
    ws = torch.empty(wsb, dtype=torch.uint8, device="cuda")
    fast.fast_csr_offsets_batched(d_counts, ns, outs, ws, wsb)
    torch.cuda.synchronize()
    return [o.cpu().numpy() for o in outs]


@pytest.mark.parametrize("case", ["cfg3", "cfg4", "with_empty", "single", "nine_blocks",
                                  "big_block", "all_empty"])
def test_csr_offsets_batched_bit_exact(case):
    """All layer blocks in one pair of launches (with empty blocks, more than
    the 8 blocks of one pair, and a block of more than 2048 tiles, which the
    blocks then take one after another), bit-exact against the oracle."""
    _announce(f"offsets batched {case}")
    r = np.random.default_rng(3)
    ri = lambda hi, n: r.integers(0, hi, n).astype(np.int32)
    lists = {
        "cfg3": lambda: [blk.counts for blk in make_batch(3).blocks],
        "cfg4": lambda: [blk.counts for blk in make_batch(4).blocks],
        "with_empty": lambda: [ri(30, 5000), np.zeros(0, np.int32), ri(5, 2049), np.zeros(0, np.int32),
                               ri(7, 2048)],
        "single": lambda: [ri(30, 777)],
        "nine_blocks": lambda: [ri(20, int(r.integers(1, 9000))) for _ in range(9)],
        "big_block": lambda: [ri(3, 2048 * 2048 + 5), ri(9, 100)],
        "all_empty": lambda: [np.zeros(0, np.int32), np.zeros(0, np.int32)],
    }[case]()
    for k, (got, c) in enumerate(zip(_offsets_batched(lists), lists)):
        assert np.array_equal(got, oracle.csr_offsets(c)), f"block {k}"


@pytest.mark.parametrize("seed", range(16))
def test_csr_offsets_random(seed):
    """Seeded random layer-block sets: 1 to 12 blocks of 0 to 5e6 segments
    (one, two or three scan launches; blocks beyond the 8 of one batched
    launch pair and beyond 2048 tiles), degrees up to 60 with empty
    segments; the batched and the single-block scans bit-exact against the
    oracle."""
    r = np.random.default_rng(9700 + seed)
    k = int(r.integers(1, 13))
    lists = []
    for _ in range(k):
        n = int(r.choice([0, int(r.integers(1, 3000)), int(r.integers(3000, 300_000)),
                          int(r.integers(4_200_000, 5_000_000))], p=[0.1, 0.4, 0.4, 0.1]))
        c = r.integers(0, 61, n).astype(np.int32)
        c[r.random(n) < 0.1] = 0
        lists.append(c)
    _announce(f"offsets random seed={seed}: blocks {[x.size for x in lists]}")
    for i, (got, c) in enumerate(zip(_offsets_batched(lists), lists)):
        assert np.array_equal(got, oracle.csr_offsets(c)), f"batched block {i}"
    for i, c in enumerate(lists[:3]):
        n = c.size
        d_c = to_dev(c) if n else torch.zeros(1, dtype=torch.int32, device="cuda")
        out = torch.full((n + 1,), -7, dtype=torch.int32, device="cuda")
        wsb = fast.fast_csr_offsets_workspace(n)
        ws = torch.empty(wsb, dtype=torch.uint8, device="cuda")
        fast.fast_csr_offsets(d_c, n, out, ws, wsb)
        torch.cuda.synchronize()
        assert np.array_equal(out.cpu().numpy(), oracle.csr_offsets(c)), f"single block {i}"


def _te_block_dev(off, dst_t, edge_t):
    d_off, d_dst, d_e = to_dev(off), to_dev(dst_t), to_dev(edge_t)
    return fast.tcsr(d_off, edge_t.shape[0], edge_t=d_e, dst_t=d_dst), (d_off, d_dst, d_e)


def _te_batched_vs_single(blocks, om, ph, dt, shift=0):
    """blocks: (off, dst_t, edge_t) per block; shift: elements by which every
    output starts past a 256-byte aligned allocation."""
    graphs, keep, outs, singles = [], [], [], []
    for off, dst_t, edge_t in blocks:
        g, k = _te_block_dev(off, dst_t, edge_t)
        graphs.append(g)
        keep.append(k)
        E = edge_t.shape[0]
        big = torch.full((E * om.shape[0] + shift + 1,), float("nan"), dtype=tdtype(dt), device="cuda")
        outs.append(big[shift:shift + E * om.shape[0]].view(E, om.shape[0]) if E else None)
        singles.append(_te_gpu(off, dst_t, edge_t, om, ph, dt) if E else None)
    fast.fast_time_encode_batched(graphs, to_dev(om), to_dev(ph), om.shape[0], outs, DT[dt])
    torch.cuda.synchronize()
    for k, (o, s1) in enumerate(zip(outs, singles)):
        if o is not None:
            assert torch.equal(o, s1), f"block {k}: batched differs from the single-block call"
    return outs


@pytest.mark.parametrize("cfg", [0, 1, 2, 3, 4])
def test_time_encode_batched_equals_single_workloads(cfg):
    """Both layer blocks in one launch write exactly what one call per block
    writes (itself checked against the oracle on every row above)."""
    b = make_batch(cfg)
    _announce(f"time encode batched cfg={cfg}")
    om, ph = omega_phi(b.d_t)
    blocks = [(oracle.csr_offsets(x.counts), x.dst_t, x.edge_t) for x in b.blocks]
    _te_batched_vs_single(blocks, om, ph, b.dtype)


@pytest.mark.parametrize("d_t,dt,shift", [(100, "f32", 0), (100, "f32", 1), (6, "bf16", 0),
                                          (128, "bf16", 3), (7, "f32", 0)])
def test_time_encode_batched_edge_cases(d_t, dt, shift):
    """Nine blocks (two launches), blocks without edges or destinations mixed
    in, outputs off the 16-byte grid (narrower vectors for every block), and
    the oracle on every block."""
    _announce(f"time encode batched d_t={d_t} {dt} shift={shift}")
    r = np.random.default_rng(d_t + shift)
    blocks = []
    for k in range(9):
        counts = [0, 0, 0] if k == 4 else list(r.integers(0, 40, int(r.integers(1, 300))))
        blk = tiny_graph(counts, seed=k + 7)
        blocks.append((oracle.csr_offsets(blk.counts), blk.dst_t, blk.edge_t))
    blocks.insert(2, (np.zeros(1, np.int32), np.zeros(0, np.float32), np.zeros(0, np.float32)))
    om, ph = omega_phi(d_t)
    outs = _te_batched_vs_single(blocks, om, ph, dt, shift)
    for k, (o, (off, dst_t, edge_t)) in enumerate(zip(outs, blocks)):
        if o is not None:
            assert_close(o, oracle.time_encode(off, dst_t, edge_t, om, ph), dt, f"te batched block {k}")


# ------------------------------------------------------------------ subgraph contract check
def _check_gpu(off, E, src=None, src_bound=0, eid=None, edge_bound=0, et=None, dt=None):
    d = lambda a, t: None if a is None else to_dev(np.asarray(a, dtype=t))
    d_off = to_dev(np.asarray(off, np.int32))
    d_src, d_eid = d(src, np.int64), d(eid, np.int64)
    d_et, d_dt = d(et, np.float32), d(dt, np.float32)
    g = fast.tcsr(d_off, E, src_ids=d_src, edge_t=d_et, edge_ids=d_eid, dst_t=d_dt)
    v = torch.full((5,), -3, dtype=torch.int64, device="cuda")
    fast.fast_check_tcsr(g, src_bound, edge_bound, v)
    return v.cpu().numpy()


@pytest.mark.parametrize("cfg", [0, 1, 2, 3, 4])
def test_check_tcsr_workloads_clean(cfg):
    _announce(f"check_tcsr cfg{cfg}")
    b = make_batch(cfg)
    for blk in b.blocks:
        off = oracle.csr_offsets(blk.counts)
        args = (off, blk.num_edges, blk.src_ids, b.node_bound, blk.edge_ids, b.edge_bound,
                blk.edge_t, blk.dst_t)
        got = _check_gpu(*args)
        assert np.array_equal(got, oracle.check_tcsr(*args))
        assert got.tolist() == [0, 0, 0, 0, 0]


@pytest.mark.parametrize("seed", [0, 1, 2])
def test_check_tcsr_malformed_bit_exact(seed):
    _announce(f"check_tcsr malformed seed {seed}")
    r = np.random.default_rng(100 + seed)
    N, E = 3001 + 517 * seed, 4099 + 1031 * seed
    # offsets mostly increasing with random faults, some below 0 or above E
    off = np.sort(r.integers(0, E + 1, N + 1)).astype(np.int32)
    off[0], off[-1] = 0, E
    bad = r.choice(N + 1, 40, replace=False)
    off[bad] = r.integers(-100, E + 100, 40)
    src = r.integers(-5, 1000, E)
    eid = r.integers(0, 2000, E)
    dt = r.uniform(0, 100, N).astype(np.float32)
    et = r.uniform(0, 110, E).astype(np.float32)
    args = (off, E, src, 995, eid, 1990, et, dt)
    want = oracle.check_tcsr(*args)
    assert want.min() >= 0 and want[[0, 2, 3, 4]].min() > 0
    assert np.array_equal(_check_gpu(*args), want)
    # optional arrays absent
    assert np.array_equal(_check_gpu(off, E), oracle.check_tcsr(off, E))


def test_check_tcsr_empty_and_single_offset():
    _announce("check_tcsr empty")
    assert _check_gpu([0], 0).tolist() == [0, 0, 0, 0, 0]
    assert _check_gpu([3], 0).tolist() == [0, 2, 0, 0, 0]
    assert _check_gpu([0, 0, 0], 0, et=[], dt=[1.0, 2.0]).tolist() == [0, 0, 0, 0, 0]


# ------------------------------------------------------------------ dedup + gather (a2, a3)
def _dedup(ids_np, id_bound, table=None, slot_map=None, want_miss=True):
    n = ids_np.shape[0]
    ids = to_dev(ids_np) if n else torch.zeros(1, dtype=torch.int64, device="cuda")
    cap = max(n, 1)
    uni = torch.full((cap,), -5, dtype=torch.int64, device="cuda")
    inv = torch.full((cap,), -5, dtype=torch.int32, device="cuda")
    nu = torch.full((1,), -1, dtype=torch.int64, device="cuda")
    rows = None
    D = 0
    dt = fast.F32
    if table is not None:
        D = table.shape[1]
        dt = fast.dtype_of(table)
        rows = torch.zeros((cap, D), dtype=table.dtype, device="cuda")
    miss = torch.full((cap,), -5, dtype=torch.int32, device="cuda") if want_miss else None
    nm = torch.full((1,), -1, dtype=torch.int64, device="cuda")
    wsb = fast.fast_dedup_gather_workspace(n, id_bound)
    ws = torch.empty(wsb, dtype=torch.uint8, device="cuda")
    fast.fast_dedup_gather(ids, n, id_bound, table, table.shape[0] if table is not None else 0, D,
                           dt, slot_map, uni, inv, nu, rows, miss, nm, ws, wsb)
    torch.cuda.synchronize()
    u = int(nu.item())
    return (uni[:u].cpu().numpy(), inv[:n].cpu().numpy(), u,
            None if rows is None else rows[:u], None if miss is None else miss, int(nm.item()))


def _bits(t):
    """Raw bits of a device float tensor (bf16 via int16 view) as numpy."""
    if t.dtype == torch.bfloat16:
        return t.view(torch.int16).cpu().numpy()
    return t.view(torch.int32).cpu().numpy()


@pytest.mark.parametrize("cfg", [0, 1, 2, 3])
def test_dedup_gather_workloads(cfg):
    b = make_batch(cfg)
    for kind, ids, bound, D, stream in (("node", b.node_ids, b.node_bound, b.node_D, 3),
                                        ("edge", b.edge_ids, b.edge_bound, b.edge_D, 4)):
        _announce(f"dedup cfg={cfg} {kind} n={ids.size} bound={bound}")
        table = make_table(bound, D, b.dtype, device="cuda", seed=b.seed, stream=stream)
        uni, inv, u, rows, miss, nm = _dedup(ids, bound, table)
        ref_uni, ref_inv = oracle.dedup(ids)
        assert u == ref_uni.size
        assert np.array_equal(uni, ref_uni) and np.array_equal(inv, ref_inv)
        assert nm == 0
        ref_rows, hit, _ = oracle.gather(ref_uni, _bits(table))
        assert hit.all()
        assert np.array_equal(_bits(rows), ref_rows), "gathered rows differ"
        del table
        torch.cuda.empty_cache()


def test_dedup_gather_bigdedup_slot_map():
    b = make_batch(4)
    _announce("dedup cfg=4 node ids over 1e7 with a 4 GB table")
    table = make_table(b.node_bound, b.node_D, "f32", device="cuda", seed=b.seed, stream=3)
    uni, inv, u, rows, miss, nm = _dedup(b.node_ids, b.node_bound, table)
    ref_uni, ref_inv = oracle.dedup(b.node_ids)
    assert u == ref_uni.size and np.array_equal(uni, ref_uni) and np.array_equal(inv, ref_inv)
    ref_rows, _, _ = oracle.gather(ref_uni, _bits(table))
    assert np.array_equal(_bits(rows), ref_rows)
    del table, rows
    torch.cuda.empty_cache()
    _announce("dedup cfg=4 edge ids over 2e8 through a 2e6-row cache")
    cache = make_table(b.edge_cache_rows, b.edge_D, "f32", device="cuda", seed=b.seed, stream=4)
    sm = make_slot_map(b, device="cuda")
    uni, inv, u, rows, miss, nm = _dedup(b.edge_ids, b.edge_bound, cache, slot_map=sm)
    ref_uni, ref_inv = oracle.dedup(b.edge_ids)
    assert u == ref_uni.size and np.array_equal(uni, ref_uni) and np.array_equal(inv, ref_inv)
    ref_rows, hit, ref_miss = oracle.gather(ref_uni, _bits(cache), sm.cpu().numpy())
    assert nm == ref_miss.size and np.array_equal(miss[:nm].cpu().numpy(), ref_miss)
    assert 0 < nm < u
    assert np.array_equal(_bits(rows)[hit], ref_rows[hit])


@pytest.mark.parametrize("case", ["empty", "single", "allsame", "top_id", "bound_not_x32",
                                  "bf16_odd_D", "dedup_only", "negative_and_oob"])
def test_dedup_edge_cases(case):
    _announce(f"dedup edge case {case}")
    r = np.random.default_rng(2)
    bound = 1000
    ids = {
        "empty": np.zeros(0, np.int64),
        "single": np.array([17], np.int64),
        "allsame": np.full(5000, 999, np.int64),
        "top_id": np.array([999, 0, 999, 998, 31, 32, 33], np.int64),
        "bound_not_x32": r.integers(0, 1000, 777).astype(np.int64),
        "bf16_odd_D": r.integers(0, 1000, 3000).astype(np.int64),
        "dedup_only": r.integers(0, 1000, 3000).astype(np.int64),
        "negative_and_oob": np.array([5, -1, 7, 1000, 5, 123456, 7], np.int64),
    }[case]
    table = None
    if case == "bf16_odd_D":
        table = make_table(bound, 7, "bf16", device="cuda", seed=9)
    elif case != "dedup_only":
        table = make_table(bound, 12, "f32", device="cuda", seed=9)
    uni, inv, u, rows, miss, nm = _dedup(ids, bound, table)
    valid = (ids >= 0) & (ids < bound)
    ref_uni, ref_inv = oracle.dedup(ids[valid])
    assert u == ref_uni.size and np.array_equal(uni, ref_uni)
    assert np.array_equal(inv[valid], ref_inv) and np.all(inv[~valid] == -1)
    if table is not None:
        ref_rows, _, _ = oracle.gather(ref_uni, _bits(table))
        assert np.array_equal(_bits(rows), ref_rows)
        assert nm == 0
    else:
        # no table: every distinct id is a miss (slot = id lies outside zero table rows)
        assert nm == u and np.array_equal(miss[:nm].cpu().numpy(), np.arange(u))


@pytest.mark.parametrize("bound,n", [(2**29, 3000), (2**31, 3000), (2**31 + 1, 3000), (2**33 + 5, 50_000),
                                     (3 * 10**7 + 13, 300_000), (40_000, 1200), (2**31, 9_000_000)])
def test_dedup_sparse_universes(bound, n):
    """Universes far larger than the batch, on both sides of the largest one
    that bucketed marking takes (2^31 ids: 4096 buckets of 2^19) and up to
    2^33 ids (hashed marking), with Zipf-like hot ids (a few ids repeated in
    every workgroup's share), ids at both ends of the universe, and many
    workgroups; 9 M ids over 2^31 give more (bucket, workgroup) counts than
    the bucketed marking takes (2^24), so they are marked by hashed atomics."""
    _announce(f"dedup sparse universe bound={bound} n={n}")
    r = np.random.default_rng(bound % 1000 + n)
    hot = r.integers(0, bound, 16)
    ids = np.where(r.random(n) < 0.4, hot[r.integers(0, 16, n)], r.integers(0, bound, n)).astype(np.int64)
    ids[:4] = [0, bound - 1, bound - 1, 0]
    uni, inv, u, _, _, nm = _dedup(ids, bound, None)
    ref_uni, ref_inv = oracle.dedup(ids)
    assert u == ref_uni.size and np.array_equal(uni, ref_uni)
    assert np.array_equal(inv, ref_inv)
    torch.cuda.empty_cache()


@pytest.mark.parametrize("D,dt", [(4, "bf16"), (12, "bf16"), (44, "bf16"), (172, "bf16"), (252, "bf16"),
                                  (260, "bf16"), (508, "bf16"), (6, "f32"), (86, "f32"), (126, "f32")])
def test_gather_rows_of_odd_eight_byte_width(D, dt):
    """Rows of 16h + 8 bytes (every other row off the 16-byte grid) are
    copied bit-exactly, directly and through a slot map whose slots mix both
    parities and misses; D = 4 bf16 (8-byte rows) is the narrow case."""
    _announce(f"gather rows D={D} {dt}")
    r = np.random.default_rng(D)
    bound, n = 20_000, 30_000
    ids = r.integers(0, bound, n).astype(np.int64)
    table = make_table(bound, D, dt, device="cuda", seed=D, stream=5)
    uni, inv, u, rows, miss, nm = _dedup(ids, bound, table)
    ref_uni, ref_inv = oracle.dedup(ids)
    assert np.array_equal(uni, ref_uni) and np.array_equal(inv, ref_inv) and nm == 0
    ref_rows, _, _ = oracle.gather(ref_uni, _bits(table))
    assert np.array_equal(_bits(rows), ref_rows)
    cache_rows = 5_001
    sm_np = r.integers(0, cache_rows, bound).astype(np.int32)
    sm_np[r.random(bound) < 0.3] = -1
    cache = make_table(cache_rows, D, dt, device="cuda", seed=D + 1, stream=6)
    uni, inv, u, rows, miss, nm = _dedup(ids, bound, cache, slot_map=to_dev(sm_np))
    ref_rows, hit, ref_miss = oracle.gather(ref_uni, _bits(cache), sm_np)
    assert nm == ref_miss.size and np.array_equal(miss[:nm].cpu().numpy(), ref_miss)
    assert np.array_equal(_bits(rows)[hit], ref_rows[hit])
    assert np.all(_bits(rows)[~hit] == 0), "a miss row must be left untouched"


@pytest.mark.parametrize("seed", range(24))
def test_dedup_gather_random(seed):
    """Seeded random batches: universes from 16 ids to 2^31, 0 to 120 k ids
    (uniform, or Zipf-hot with a few ids in every workgroup's share), some
    ids outside the universe, and rows of random width and storage gathered
    straight from a table or through a slot map into a cache with misses --
    every marking path and row-copy shape, against the oracle."""
    r = np.random.default_rng(5000 + seed)
    bound = int(2 ** r.uniform(4, 31))
    n = int(r.choice([0, 1, int(r.integers(2, 3000)), int(r.integers(3000, 120_001))],
                     p=[0.08, 0.08, 0.42, 0.42]))
    if r.random() < 0.5:
        ids = r.integers(0, bound, n)
    else:
        hot = r.integers(0, bound, 8)
        ids = np.where(r.random(n) < 0.5, hot[r.integers(0, 8, n)], r.integers(0, bound, n))
    ids = ids.astype(np.int64)
    bad = r.random(n) < 0.02
    ids[bad] = r.choice([-1, -7, bound, bound + 5], int(bad.sum()))
    valid = (ids >= 0) & (ids < bound)
    D = int(r.integers(1, 257))          # any width whose row is at most 256 vectors
    dt = "bf16" if r.random() < 0.5 else "f32"
    mode = str(r.choice(["none", "table", "slot"], p=[0.2, 0.4, 0.4]))
    if mode == "table" and bound > 200_000:          # the oracle copies the whole table
        mode = "slot" if bound <= 50_000_000 else "none"
    if mode == "slot" and bound > 50_000_000:
        mode = "none"
    _announce(f"dedup random seed={seed}: n={n} bound={bound} {mode} D={D} {dt}")
    table = sm_np = None
    if mode == "table":
        table = make_table(bound, D, dt, device="cuda", seed=seed, stream=7)
    elif mode == "slot":
        rows = int(r.integers(1, 20_000))
        table = make_table(rows, D, dt, device="cuda", seed=seed, stream=8)
        sm_np = r.integers(0, rows, bound).astype(np.int32)
        sm_np[r.random(bound) < 0.3] = -1
    uni, inv, u, got_rows, miss, nm = _dedup(ids, bound, table,
                                             slot_map=to_dev(sm_np) if sm_np is not None else None)
    ref_uni, ref_inv = oracle.dedup(ids[valid])
    assert u == ref_uni.size and np.array_equal(uni, ref_uni)
    assert np.array_equal(inv[valid], ref_inv) and np.all(inv[~valid] == -1)
    if table is not None:
        ref_rows, hit, ref_miss = oracle.gather(ref_uni, _bits(table), sm_np)
        assert np.array_equal(_bits(got_rows)[hit], ref_rows[hit]), "gathered rows differ"
        assert nm == ref_miss.size and np.array_equal(miss[:nm].cpu().numpy(), ref_miss)
    else:
        assert nm == u and np.array_equal(miss[:nm].cpu().numpy(), np.arange(u))
    del table
    torch.cuda.empty_cache()


# ------------------------------------------------------------------ time encoding (a4)
def _te_gpu(blk_off, dst_t, edge_t, omega, phi, dt="f32"):
    E = edge_t.shape[0]
    d_off, d_dst, d_e = to_dev(blk_off), to_dev(dst_t), to_dev(edge_t)
    g = fast.tcsr(d_off, E, edge_t=d_e, dst_t=d_dst)
    te = torch.empty((max(E, 1), omega.shape[0]), dtype=tdtype(dt), device="cuda")
    fast.fast_time_encode(g, to_dev(omega), to_dev(phi), omega.shape[0], te, DT[dt])
    torch.cuda.synchronize()
    return te[:E]


@pytest.mark.parametrize("cfg", [0, 1, 2, 3, 4])
def test_time_encode_workloads(cfg):
    """Every row of both blocks, the oracle over segment ranges on all host threads."""
    b = make_batch(cfg)
    om, ph = omega_phi(b.d_t)
    for i, blk in enumerate(b.blocks):
        _announce(f"time encode cfg={cfg} block={i} E={blk.num_edges} d_t={b.d_t} {b.dtype}")
        off = oracle.csr_offsets(blk.counts)
        te = _te_gpu(off, blk.dst_t, blk.edge_t, om, ph, b.dtype).cpu()
        check_time_encode_full(off, blk.dst_t, blk.edge_t, om, ph, te, b.dtype, f"te cfg{cfg}/L{i + 1}")
        del te


@pytest.mark.parametrize("d_t,dt", [(1, "f32"), (7, "f32"), (6, "f32"), (100, "bf16"),
                                    (3, "bf16"), (6, "bf16"), (128, "f32")])
def test_time_encode_shapes_and_zero_dt(d_t, dt):
    _announce(f"time encode d_t={d_t} {dt}")
    blk = tiny_graph([0, 3, 0, 70, 1, 0, 130, 2], seed=d_t)
    off = oracle.csr_offsets(blk.counts)
    edge_t = blk.edge_t.copy()
    seg = np.repeat(np.arange(blk.num_dst), blk.counts)
    edge_t[::9] = blk.dst_t[seg[::9]]                  # dt = 0 rows
    om, ph = omega_phi(d_t)
    te = _te_gpu(off, blk.dst_t, edge_t, om, ph, dt)
    ref = oracle.time_encode(off, blk.dst_t, edge_t, om, ph)
    assert_close(te, ref, dt, f"te d_t={d_t}")
    assert torch.all(te[::9].float() == 1.0)


def test_time_encode_no_edges():
    off = np.zeros(6, np.int32)
    te = _te_gpu(off, np.ones(5, np.float32), np.zeros(0, np.float32), *omega_phi(10))
    assert te.shape[0] == 0


@pytest.mark.parametrize("seed", range(16))
def test_time_encode_random(seed):
    """Seeded random blocks: time widths 1-256, fp32 or bf16 output, 1-3000
    segments of degree 0-60, time scales from 1 to 1e4 and phases drawn at
    random; every row against the oracle, and the batched launch over a
    random split of the same segments equal to the single-block calls bit
    for bit."""
    r = np.random.default_rng(6000 + seed)
    d_t = int(r.integers(1, 257))
    dt = "bf16" if r.random() < 0.5 else "f32"
    N = int(r.integers(1, 3001))
    counts = r.integers(0, 61, N)
    counts[r.random(N) < 0.1] = 0
    scale = float(10 ** r.uniform(0, 4))
    off = np.concatenate([[0], np.cumsum(counts)]).astype(np.int32)
    E = int(off[-1])
    dst_t = (r.random(N) * scale + 1.0).astype(np.float32)
    seg = np.repeat(np.arange(N), counts)
    edge_t = (dst_t[seg] * r.random(E)).astype(np.float32)
    om, ph = omega_phi(d_t)
    ph = (r.uniform(-3.0, 3.0, d_t) if r.random() < 0.5 else ph).astype(np.float32)
    _announce(f"time encode random seed={seed}: d_t={d_t} {dt} N={N} E={E} scale={scale:.0f}")
    te = _te_gpu(off, dst_t, edge_t, om, ph, dt)
    check_time_encode_full(off, dst_t, edge_t, om, ph, te.cpu(), dt, f"te random seed={seed}")
    cuts = np.sort(r.choice(np.arange(1, N), min(int(r.integers(0, 4)), N - 1), replace=False)) if N > 1 else []
    bounds = [0] + [int(c) for c in cuts] + [N]
    blocks = []
    for a, c in zip(bounds[:-1], bounds[1:]):
        sub = (off[a:c + 1] - off[a]).astype(np.int32)
        blocks.append((sub, dst_t[a:c], edge_t[off[a]:off[c]]))
    _te_batched_vs_single(blocks, om, ph, dt)


@pytest.mark.parametrize("out", ["f32", "bf16"])
def test_time_encode_cosine_accuracy_sweep(out):
    # one destination per edge with dst_t = dt and edge_t = 0, so dt is exact;
    # omega = 1 makes the argument dt itself (plus a phase-shifted column).
    # bf16 rows take their range check per row: arguments beyond 2^16 there
    # must still reach the fallback.
    _announce(f"time encode cosine sweep {out}")
    r = np.random.default_rng(5)
    n = 400_000
    dt = np.concatenate([r.uniform(0, 1e4, n // 2), r.uniform(1e4, 2e5, n // 4),
                         np.linspace(0, 20, n // 8), r.uniform(65000, 66000, n // 8)]).astype(np.float32)
    off = np.arange(dt.size + 1, dtype=np.int32)
    om = np.array([1.0, 1.0, 0.37], dtype=np.float32)
    ph = np.array([0.0, np.float32(np.pi / 2), -1.25], dtype=np.float32)
    te = _te_gpu(off, dt, np.zeros(dt.size, np.float32), om, ph, out)
    ref = oracle.time_encode(off, dt, np.zeros(dt.size, np.float32), om, ph)
    if out == "f32":
        err = np.abs(te.cpu().numpy().astype(np.float64) - ref)
        assert err.max() <= 1e-6, f"max cosine error {err.max():.3g}"
    else:
        # an fp32 cosine within 1e-6, rounded to bf16: rounding is monotone, so
        # the result lies between the roundings of ref - 1e-6 and ref + 1e-6
        rnd = lambda a: torch.from_numpy(a.astype(np.float32)).to(torch.bfloat16).double().numpy()
        got = te.cpu().double().numpy()
        lo, hi = rnd(ref - 1e-6), rnd(ref + 1e-6)
        bad = (got < lo) | (got > hi)
        assert not bad.any(), f"{int(bad.sum())} bf16 cosines outside the rounding band"
