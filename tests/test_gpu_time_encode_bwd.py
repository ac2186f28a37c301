"""GPU parity of the time-encoding backward (domega, dphi) against the fp64
oracle, through the C ABI.

Every workload runs at its full size in the launch configuration the
benchmark times; each output is a sum over the whole block, so the oracle
adds the whole block too, in chunks of segments (fp64 sums of chunk sums).
Tolerance: |x - r| <= 1e-5 + 1e-5 |r| on the fp32 outputs, for fp32 and
bf16 upstream gradients alike (the bf16 values are exact inputs; the
arithmetic is fp64).
"""
import numpy as np
import pytest
import torch

import oracle
import paper_2607_05095_amd as fast
from synth import _randn, make_batch, omega_phi, tiny_graph
from tests.parity import assert_close, to_dev

pytestmark = pytest.mark.gpu

DT = {"f32": fast.F32, "bf16": fast.BF16}


def _announce(msg):
    print(f"[parity] {msg}", flush=True)


def _tb_gpu(off, dst_t, edge_t, om, ph, dte):
    """dte: device tensor [E, d_t] (fp32 or bf16).  Returns (domega, dphi) on the host."""
    E, d_t = edge_t.shape[0], om.shape[0]
    d_off, d_dst, d_e = to_dev(off), to_dev(dst_t), to_dev(edge_t)
    g = fast.tcsr(d_off, E, edge_t=d_e, dst_t=d_dst)
    wsb = fast.fast_time_encode_bwd_workspace(off.shape[0] - 1, d_t)
    ws = torch.empty(wsb, dtype=torch.uint8, device="cuda")
    dw = torch.full((d_t,), float("nan"), device="cuda")
    dp = torch.full((d_t,), float("nan"), device="cuda")
    dtype = fast.BF16 if dte.dtype == torch.bfloat16 else fast.F32
    fast.fast_time_encode_bwd(g, to_dev(om), to_dev(ph), d_t, dte, dtype, dw, dp, ws, wsb)
    torch.cuda.synchronize()
    return dw.cpu().numpy(), dp.cpu().numpy()


def _oracle_chunked(off, dst_t, edge_t, om, ph, dte, seg_chunk=20000):
    """Oracle sums over consecutive chunks of segments, added in fp64."""
    N = off.shape[0] - 1
    dw, dp = np.zeros(om.size), np.zeros(om.size)
    for s0 in range(0, N, seg_chunk):
        s1 = min(N, s0 + seg_chunk)
        e0, e1 = int(off[s0]), int(off[s1])
        sub = (off[s0:s1 + 1] - off[s0]).astype(np.int32)
        g = dte[e0:e1].double().cpu().numpy()
        w, p = oracle.time_encode_bwd(sub, dst_t[s0:s1], edge_t[e0:e1], om, ph, g)
        dw += w
        dp += p
    return dw, dp


@pytest.mark.parametrize("cfg", [0, 1, 2, 3, 4])
def test_time_encode_bwd_workloads(cfg):
    b = make_batch(cfg)
    om, ph = omega_phi(b.d_t)
    for i, blk in enumerate(b.blocks):
        _announce(f"time encode bwd cfg={cfg} block={i} E={blk.num_edges} d_t={b.d_t} {b.dtype}")
        off = oracle.csr_offsets(blk.counts)
        dte = _randn((blk.num_edges, b.d_t), b.dtype, "cuda", 1000 + 16 * cfg + i)
        got = _tb_gpu(off, blk.dst_t, blk.edge_t, om, ph, dte)
        ref = _oracle_chunked(off, blk.dst_t, blk.edge_t, om, ph, dte)
        assert_close(got[0], ref[0], "f32", f"domega cfg{cfg}/L{i + 1}")
        assert_close(got[1], ref[1], "f32", f"dphi cfg{cfg}/L{i + 1}")
        del dte


def test_time_encode_bwd_is_deterministic():
    _announce("time encode bwd determinism")
    b = make_batch(4)
    blk = b.blocks[0]
    om, ph = omega_phi(b.d_t)
    off = oracle.csr_offsets(blk.counts)
    dte = _randn((blk.num_edges, b.d_t), "f32", "cuda", 77)
    a = _tb_gpu(off, blk.dst_t, blk.edge_t, om, ph, dte)
    c = _tb_gpu(off, blk.dst_t, blk.edge_t, om, ph, dte)
    assert np.array_equal(a[0], c[0]) and np.array_equal(a[1], c[1])


@pytest.mark.parametrize("d_t,dt", [(1, "f32"), (7, "f32"), (6, "bf16"), (3, "bf16"),
                                    (128, "bf16"), (100, "f32"), (1024, "f32"), (2048, "bf16")])
def test_time_encode_bwd_shapes(d_t, dt):
    # ragged degrees with empty segments, dt = 0 rows, and more segments than
    # one workgroup group (32) so several partials are combined
    _announce(f"time encode bwd d_t={d_t} {dt}")
    counts = [0, 3, 0, 70, 1, 0, 130, 2] * 9
    blk = tiny_graph(counts, seed=d_t)
    off = oracle.csr_offsets(blk.counts)
    edge_t = blk.edge_t.copy()
    seg = np.repeat(np.arange(blk.num_dst), blk.counts)
    edge_t[::9] = blk.dst_t[seg[::9]]
    om, ph = omega_phi(d_t)
    ph = np.linspace(-2, 2, d_t).astype(np.float32)
    dte = _randn((blk.num_edges, d_t), dt, "cuda", d_t)
    got = _tb_gpu(off, blk.dst_t, edge_t, om, ph, dte)
    ref = oracle.time_encode_bwd(off, blk.dst_t, edge_t, om, ph, dte.double().cpu().numpy())
    assert_close(got[0], ref[0], "f32", f"domega d_t={d_t}")
    assert_close(got[1], ref[1], "f32", f"dphi d_t={d_t}")


def test_time_encode_bwd_no_edges_writes_zeros():
    _announce("time encode bwd without edges")
    off = np.zeros(6, np.int32)
    om, ph = omega_phi(10)
    dte = torch.empty((1, 10), device="cuda")
    got = _tb_gpu(off, np.ones(5, np.float32), np.zeros(0, np.float32), om, ph, dte[:0])
    assert np.all(got[0] == 0) and np.all(got[1] == 0)


def test_time_encode_bwd_cancelling_column_and_huge_arguments():
    # Pairs of edges with equal dt and opposite upstream gradients cancel
    # exactly, so each sum is carried by a small remainder of uncancelled
    # edges (|sum| ~ 1e-3 of sum |terms|); and a few arguments beyond 2^30 rad
    # take the library sine.
    _announce("time encode bwd cancellation and huge arguments")
    r = np.random.default_rng(3)
    n_pair, n_rest = 200_000, 200
    dt = np.concatenate([np.repeat(r.uniform(0, 1e4, n_pair), 2), r.uniform(0, 1e4, n_rest),
                         np.array([2.0e9, 3.5e9, 1.5e9], np.float64)]).astype(np.float32)
    E = dt.size
    off = np.arange(E + 1, dtype=np.int32)                 # one edge per destination
    om = np.array([1.0, 0.37, 1e-3, 1e-9], dtype=np.float32)
    ph = np.array([0.0, 0.5, -1.0, 0.25], dtype=np.float32)
    g = r.standard_normal((n_pair, om.size))
    dte = np.concatenate([np.stack([g, -g], 1).reshape(2 * n_pair, om.size),
                          1e-3 * r.standard_normal((n_rest + 3, om.size))]).astype(np.float32)
    got = _tb_gpu(off, dt, np.zeros(E, np.float32), om, ph, to_dev(dte))
    ref = oracle.time_encode_bwd(off, dt, np.zeros(E, np.float32), om, ph, dte)
    assert_close(got[0], ref[0], "f32", "domega (cancelling)")
    assert_close(got[1], ref[1], "f32", "dphi (cancelling)")


def test_time_encode_bwd_reduction_range():
    # Rows on both sides of the in-line reduction's range (a row is reduced
    # in-line when fmaf(max|omega|, |dt|, max|phi|) <= 1e6, else it takes the
    # library sine): dt log-uniform over [1e5, 1e8], so that the in-line rows
    # reach the top of the range, where the one-step reduction is least
    # accurate, and the cold rows span 1e6 .. 1e8 rad.  Pairs of equal dt and
    # opposite gradients cancel, so each sum is a small remainder of its terms
    # and an error of the sine shows at full weight.
    _announce("time encode bwd around the reduction's range")
    r = np.random.default_rng(11)
    n_pair, n_rest = 100_000, 300
    dt = np.concatenate([np.repeat(10 ** r.uniform(5, 8, n_pair), 2),
                         10 ** r.uniform(5, 8, n_rest)]).astype(np.float32)
    E = dt.size
    off = np.arange(E + 1, dtype=np.int32)                 # one edge per destination
    om = np.array([1.0, 0.37, 0.05, 1e-3], dtype=np.float32)
    ph = np.array([0.0, -2.5, 3.0, 0.25], dtype=np.float32)
    g = r.standard_normal((n_pair, om.size))
    dte = np.concatenate([np.stack([g, -g], 1).reshape(2 * n_pair, om.size),
                          1e-3 * r.standard_normal((n_rest, om.size))]).astype(np.float32)
    inline = np.abs(dt) * 1.0 + 3.0 <= 1e6
    assert 0.2 < inline.mean() < 0.5                        # both paths well populated
    got = _tb_gpu(off, dt, np.zeros(E, np.float32), om, ph, to_dev(dte))
    ref = oracle.time_encode_bwd(off, dt, np.zeros(E, np.float32), om, ph, dte)
    assert_close(got[0], ref[0], "f32", "domega (reduction range)")
    assert_close(got[1], ref[1], "f32", "dphi (reduction range)")


@pytest.mark.parametrize("seed", range(16))
def test_time_encode_bwd_random(seed):
    """Seeded random blocks: time widths 1-256 (every vector width the
    kernel picks), fp32 or bf16 upstream gradients, 1-6000 segments of degree
    0-60 (a partial last group of segments, more groups than workgroups at
    the top of the range), time scales 1-1e4 and random phases; both outputs
    against the oracle's fp64 sums, and a second call bitwise equal."""
    r = np.random.default_rng(9000 + seed)
    d_t = int(r.integers(1, 257))
    dt = "bf16" if r.random() < 0.5 else "f32"
    N = int(r.integers(1, 6001))
    counts = r.integers(0, 61, N)
    counts[r.random(N) < 0.1] = 0
    scale = float(10 ** r.uniform(0, 4))
    off = np.concatenate([[0], np.cumsum(counts)]).astype(np.int32)
    E = int(off[-1])
    dst_t = (r.random(N) * scale + 1.0).astype(np.float32)
    edge_t = (dst_t[np.repeat(np.arange(N), counts)] * r.random(E)).astype(np.float32)
    om, ph = omega_phi(d_t)
    ph = (r.uniform(-3.0, 3.0, d_t) if r.random() < 0.5 else ph).astype(np.float32)
    _announce(f"time encode bwd random seed={seed}: d_t={d_t} {dt} N={N} E={E} scale={scale:.0f}")
    dte = _randn((max(E, 1), d_t), dt, "cuda", 9100 + seed)[:E]
    got = _tb_gpu(off, dst_t, edge_t, om, ph, dte)
    ref = _oracle_chunked(off, dst_t, edge_t, om, ph, dte)
    assert_close(got[0], ref[0], "f32", f"domega random seed={seed}")
    assert_close(got[1], ref[1], "f32", f"dphi random seed={seed}")
    again = _tb_gpu(off, dst_t, edge_t, om, ph, dte)
    assert np.array_equal(got[0], again[0]) and np.array_equal(got[1], again[1])
