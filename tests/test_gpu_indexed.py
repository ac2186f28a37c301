"""GPU parity of indexed operands through the C ABI: the fused attention
reading K and V through an index into de-duplicated rows (forward and
per-edge backward), the occurrence lists of an index (bit-exact), and the
transposed gather that turns per-edge gradients into row gradients.

Each GPU op is compared with the oracle on the same inputs, every segment
and every row at every workload: the attention against the oracle on the
gathered rows (over segment ranges on all host threads), the occurrence
lists bit-exactly, and the row sums against the oracle's fp64 sums of the
same per-edge rows or coefficients.
"""
import numpy as np
import pytest
import torch

import oracle
import paper_2607_05095_amd as fast
from synth import _randn, make_batch
from tests.parity import (SLOPE, assert_bwd_close, assert_close, bwd_reference_with_kinks,
                          check_attention_block_full, over_ranges, segment_ranges, tdtype, to_dev)

pytestmark = pytest.mark.gpu

DT = {"f32": fast.F32, "bf16": fast.BF16}


def _announce(msg):
    print(f"[parity] {msg}", flush=True)


def _host(t):
    return t.detach().float().cpu().double().numpy()


def _occ_gpu(index_np, num_rows):
    n = index_np.shape[0]
    idx = to_dev(np.ascontiguousarray(index_np, np.int32)) if n else \
        torch.empty(0, dtype=torch.int32, device="cuda")
    off = torch.full((num_rows + 1,), -9, dtype=torch.int32, device="cuda")
    occ = torch.full((max(n, 1),), -9, dtype=torch.int32, device="cuda")
    wsb = fast.fast_occurrence_csr_workspace(n, num_rows)
    ws = torch.empty(wsb, dtype=torch.uint8, device="cuda")
    fast.fast_occurrence_csr(idx, n, num_rows, off, occ, ws, wsb)
    torch.cuda.synchronize()
    return off, occ


def _index_add_gpu(off, occ, n, num_rows, src):
    D = int(np.prod(src.shape[1:])) if src.dim() > 1 else 1
    dst = torch.full((num_rows, D), float("nan"), device="cuda")
    wsb = fast.fast_index_add_rows_workspace(n, num_rows, D)
    ws = torch.empty(wsb, dtype=torch.uint8, device="cuda")
    dt = fast.BF16 if src.dtype == torch.bfloat16 else fast.F32
    fast.fast_index_add_rows(off, occ, n, num_rows, D, dt, src, dst, ws, wsb)
    torch.cuda.synchronize()
    return dst


@pytest.mark.parametrize("n,rows", [(0, 5), (10, 0), (1, 1), (5000, 37), (300_000, 200),
                                    (300_000, 60_000), (2_000_000, 541_000), (5_052_000, 1_000_000)])
def test_occurrence_csr_bit_exact(n, rows):
    _announce(f"occurrence csr n={n} rows={rows}")
    r = np.random.default_rng(n + rows)
    idx = ((r.zipf(1.2, n) - 1) % max(rows, 1)).astype(np.int32) if rows else r.integers(-3, 3, n).astype(np.int32)
    if n > 20:
        idx[::29] = -1                                   # positions outside the row range
        idx[3::31] = rows + 7
    off, occ = _occ_gpu(idx, rows)
    want_off, want_occ = oracle.occurrence_csr(idx, rows)
    assert np.array_equal(off.cpu().numpy(), want_off)
    assert np.array_equal(occ.cpu().numpy()[:want_off[-1]], want_occ)


@pytest.mark.parametrize("D,dt,rows", [(100, "f32", 300), (128, "bf16", 5000), (172, "f32", 40),
                                       (7, "f32", 1000), (50, "bf16", 3), (1, "f32", 100)])
def test_index_add_rows_vs_oracle(D, dt, rows):
    _announce(f"index add D={D} {dt} rows={rows}")
    r = np.random.default_rng(D * 7 + rows)
    n = 200_000
    idx = ((r.zipf(1.3, n) - 1) % rows).astype(np.int32)   # hub rows with tens of thousands of reads
    idx[::97] = -1
    src = _randn((n, D), dt, "cuda", D + rows)
    off, occ = _occ_gpu(idx, rows + 2)                      # two rows nobody reads
    got = _index_add_gpu(off, occ, n, rows + 2, src)
    want = oracle.index_add_rows(idx, rows + 2, _host(src))
    assert_close(got, want, "f32", f"index add D={D}")
    again = _index_add_gpu(off, occ, n, rows + 2, src)
    assert torch.equal(got, again), "index add must be bitwise reproducible"
    assert torch.all(got[rows:] == 0)


@pytest.mark.parametrize("seed", range(24))
def test_occurrence_lists_and_row_sums_random(seed):
    """Seeded random indices: 0 to 400 k positions over 1 to 300 k rows,
    uniform or Zipf with exponents from 1.05 (hub rows of 10^5 reads, the
    three-level sums) to 3, some positions outside the row range; source
    rows of random width and storage.  Occurrence lists bit-exact, row sums
    against the oracle's fp64 sums, and a second call bitwise equal."""
    r = np.random.default_rng(7000 + seed)
    n = int(r.choice([0, int(r.integers(1, 5000)), int(r.integers(5000, 400_001))], p=[0.05, 0.35, 0.6]))
    rows = int(r.choice([1, int(r.integers(2, 1000)), int(r.integers(1000, 300_001))], p=[0.1, 0.45, 0.45]))
    if r.random() < 0.3:
        idx = r.integers(0, rows, n)
    else:
        idx = (r.zipf(float(r.uniform(1.05, 3.0)), n) - 1) % rows
    idx = idx.astype(np.int32)
    idx[r.random(n) < 0.01] = -1
    D = int(r.integers(1, 200))
    dt = "bf16" if r.random() < 0.5 else "f32"
    _announce(f"index add random seed={seed}: n={n} rows={rows} D={D} {dt}")
    off, occ = _occ_gpu(idx, rows)
    w_off, w_occ = oracle.occurrence_csr(idx, rows)
    assert np.array_equal(off.cpu().numpy(), w_off)
    assert np.array_equal(occ.cpu().numpy()[:int(w_off[-1])], w_occ)
    if n == 0:
        return
    src = _randn((n, D), dt, "cuda", 7100 + seed)
    got = _index_add_gpu(off, occ, n, rows, src)
    want = oracle.index_add_rows(idx, rows, _host(src))
    assert_close(got, want, "f32", f"index add random seed={seed}")
    assert torch.equal(got, _index_add_gpu(off, occ, n, rows, src)), "row sums must be reproducible"


def _indexed_block(b, i, seed):
    """Operands of block i with K read through the de-duplication inverse of
    the block's source node ids and V through that of its edge ids."""
    blk = b.blocks[i]
    _, kidx = np.unique(blk.src_ids, return_inverse=True)
    _, vidx = np.unique(blk.edge_ids, return_inverse=True)
    Uk, Uv = int(kidx.max()) + 1, int(vidx.max()) + 1
    base = 7000 + 16 * seed
    ops = dict(Q=_randn((blk.num_dst, b.H, b.dh), b.dtype, "cuda", base),
               K=_randn((Uk, b.H, b.dh), b.dtype, "cuda", base + 1),
               V=_randn((Uv, b.H, b.dh), b.dtype, "cuda", base + 2),
               dO=_randn((blk.num_dst, b.H, b.dh), b.dtype, "cuda", base + 3))
    return blk, kidx.astype(np.int32), vidx.astype(np.int32), Uk, Uv, ops


BLOCKS = [(0, 0), (1, 0), (2, 0), (2, 1), (3, 0), (3, 1), (4, 0), (4, 1)]


def _cpu(t):
    return t.detach().cpu()


def _rows_full(occ_off, occ, idx, U, E, per_edge, H, dh, what):
    """Occurrence lists bit-exact, then every row's ordered fp64 sum of the
    per-edge gradients against the oracle's."""
    w_off, w_occ = oracle.occurrence_csr(idx, U)
    assert np.array_equal(occ_off.cpu().numpy(), w_off), f"{what} occ_off"
    assert np.array_equal(occ.cpu().numpy()[:E], w_occ), f"{what} occ"
    got = _index_add_gpu(occ_off, occ, E, U, per_edge.reshape(E, H * dh)).cpu()
    want = oracle.index_add_rows(idx, U, _host(per_edge.reshape(E, H * dh)))
    assert_close(got, want, "f32", f"{what} rows")


@pytest.mark.parametrize("cfg,i", BLOCKS)
def test_indexed_attention_workloads(cfg, i):
    """Every segment of the block (forward and per-edge backward) and every
    row gradient against the oracle on the gathered rows."""
    b = make_batch(cfg)
    _announce(f"indexed attention cfg={cfg} block={i}")
    blk, kidx, vidx, Uk, Uv, o = _indexed_block(b, i, cfg)
    off = oracle.csr_offsets(blk.counts)
    N, E, H, dh, dt = blk.num_dst, blk.num_edges, b.H, b.dh, b.dtype
    scale = float(np.float32(1 / np.sqrt(dh)))
    d_off, d_k, d_v = to_dev(off), to_dev(kidx), to_dev(vidx)
    g = fast.tcsr(d_off, E)
    tt = tdtype(dt)
    out = torch.empty((N, H, dh), dtype=tt, device="cuda")
    lse = torch.empty((N, H), device="cuda")
    fast.fast_edge_attention_fwd_indexed(g, H, dh, DT[dt], o["Q"], o["K"], d_k, Uk, o["V"], d_v, Uv,
                                         scale, SLOPE, out, lse)
    dQ = torch.empty((N, H, dh), dtype=tt, device="cuda")
    dKe = torch.empty((E, H, dh), dtype=tt, device="cuda")
    dVe = torch.empty((E, H, dh), dtype=tt, device="cuda")
    fast.fast_edge_attention_bwd_indexed(g, H, dh, DT[dt], o["Q"], o["K"], d_k, Uk, o["V"], d_v,
                                         Uv, scale, SLOPE, lse, o["dO"], dQ, dKe, dVe)
    torch.cuda.synchronize()
    what = f"cfg{cfg}/L{i + 1} indexed"
    ins = dict(Q=_cpu(o["Q"]), dO=_cpu(o["dO"]),
               K=_cpu(o["K"][d_k.long()]), V=_cpu(o["V"][d_v.long()]))   # the rows each edge reads
    check_attention_block_full(off, ins, [_cpu(t) for t in (out, lse, dQ, dKe, dVe)], None, None,
                               scale, SLOPE, dt, what)
    del ins
    # row gradients: occurrence lists bit-exact, then the ordered fp64 sums
    # of the per-edge gradients, every row
    for name, idx, U, per_edge in (("K", kidx, Uk, dKe), ("V", vidx, Uv, dVe)):
        occ_off, occ = _occ_gpu(idx, U)
        _rows_full(occ_off, occ, idx, U, E, per_edge, H, dh, f"{what} d{name}")
    del o, out, dQ, dKe, dVe
    torch.cuda.empty_cache()


@pytest.mark.parametrize("seed", range(16))
def test_indexed_attention_random(seed):
    """Seeded random shapes (H 1-8, dh 1-96, fp32 or bf16, slopes 0.2 / 0 /
    -0.3 / 1) and random indices into fewer compact K and V rows than edges
    (hub rows included): the indexed forward and per-edge backward against
    the oracle on the rows each edge reads, the coefficient form's dQ equal
    to the per-edge backward's, and the row gradients against the oracle's
    sums."""
    r = np.random.default_rng(9800 + seed)
    H = int(r.choice([1, 2, 3, 4, 8]))
    dh = int(r.integers(1, 97))
    dt = "bf16" if r.random() < 0.4 else "f32"
    slope = float(r.choice([0.2, 0.0, -0.3, 1.0]))
    N = int(r.integers(10, 80))
    counts = r.integers(0, 40, N)
    counts[r.random(N) < 0.05] = r.integers(100, 300)
    off = np.concatenate([[0], np.cumsum(counts)]).astype(np.int32)
    E = int(off[-1])
    Uk, Uv = max(1, int(r.integers(1, E + 2) // 2)), max(1, int(r.integers(1, E + 2)))
    kidx = ((r.zipf(1.5, E) - 1) % Uk).astype(np.int32)
    vidx = r.integers(0, Uv, E).astype(np.int32)
    _announce(f"indexed attention random seed={seed}: H={H} dh={dh} {dt} slope={slope} "
              f"N={N} E={E} Uk={Uk} Uv={Uv}")
    base = 9900 + 8 * seed
    o = dict(Q=_randn((N, H, dh), dt, "cuda", base), K=_randn((Uk, H, dh), dt, "cuda", base + 1),
             V=_randn((Uv, H, dh), dt, "cuda", base + 2), dO=_randn((N, H, dh), dt, "cuda", base + 3))
    scale = float(np.float32(1 / np.sqrt(dh)))
    d_off, d_k, d_v = to_dev(off), to_dev(kidx), to_dev(vidx)
    g = fast.tcsr(d_off, E)
    tt = tdtype(dt)
    out = torch.empty((N, H, dh), dtype=tt, device="cuda")
    lse = torch.empty((N, H), device="cuda")
    fast.fast_edge_attention_fwd_indexed(g, H, dh, DT[dt], o["Q"], o["K"], d_k, Uk, o["V"], d_v, Uv,
                                         scale, slope, out, lse)
    dQ = torch.empty((N, H, dh), dtype=tt, device="cuda")
    dKe = torch.empty((max(E, 1), H, dh), dtype=tt, device="cuda")
    dVe = torch.empty((max(E, 1), H, dh), dtype=tt, device="cuda")
    fast.fast_edge_attention_bwd_indexed(g, H, dh, DT[dt], o["Q"], o["K"], d_k, Uk, o["V"], d_v,
                                         Uv, scale, slope, lse, o["dO"], dQ, dKe, dVe)
    dQc = torch.empty((N, H, dh), dtype=tt, device="cuda")
    ge = torch.empty((max(E, 1), H), device="cuda")
    ae = torch.empty((max(E, 1), H), device="cuda")
    fast.fast_edge_attention_bwd_indexed_coef(g, H, dh, DT[dt], o["Q"], o["K"], d_k, Uk, o["V"],
                                              d_v, Uv, scale, slope, lse, o["dO"], dQc, ge, ae)
    torch.cuda.synchronize()
    what = f"indexed random seed={seed}"
    ins = dict(Q=_cpu(o["Q"]), dO=_cpu(o["dO"]),
               K=_cpu(o["K"][d_k.long()]), V=_cpu(o["V"][d_v.long()]))
    check_attention_block_full(off, ins, [_cpu(t) for t in (out, lse, dQ, dKe[:E], dVe[:E])], None,
                               None, scale, slope, dt, what)
    assert torch.equal(dQ, dQc), "coefficient-form dQ differs from the per-edge backward's"
    for name, idx, U, per_edge in (("K", kidx, Uk, dKe[:E]), ("V", vidx, Uv, dVe[:E])):
        occ_off, occ = _occ_gpu(idx, U)
        _rows_full(occ_off, occ, idx, U, E, per_edge, H, dh, f"{what} d{name}")


def test_identity_index_equals_plain_operator():
    _announce("indexed attention with identity index vs plain")
    b = make_batch(1)
    blk = b.blocks[0]
    N, E, H, dh = blk.num_dst, blk.num_edges, b.H, b.dh
    off = to_dev(oracle.csr_offsets(blk.counts))
    g = fast.tcsr(off, E)
    Q, K, V, dO = (_randn(s, "f32", "cuda", 50 + j) for j, s in
                   enumerate([(N, H, dh), (E, H, dh), (E, H, dh), (N, H, dh)]))
    ident = torch.arange(E, dtype=torch.int32, device="cuda")
    scale = float(np.float32(1 / np.sqrt(dh)))
    outs = []
    for indexed in (False, True):
        out = torch.empty((N, H, dh), device="cuda")
        lse = torch.empty((N, H), device="cuda")
        dQ, dK, dV = (torch.empty_like(x) for x in (Q, K, V))
        if indexed:
            fast.fast_edge_attention_fwd_indexed(g, H, dh, fast.F32, Q, K, ident, E, V, None, E, scale,
                                                 SLOPE, out, lse)
            fast.fast_edge_attention_bwd_indexed(g, H, dh, fast.F32, Q, K, ident, E, V, None, E, scale,
                                                 SLOPE, lse, dO, dQ, dK, dV)
        else:
            fast.fast_edge_attention_fwd(g, H, dh, fast.F32, Q, K, V, scale, SLOPE, out, lse)
            fast.fast_edge_attention_bwd(g, H, dh, fast.F32, Q, K, V, scale, SLOPE, lse, dO, dQ, dK, dV)
        torch.cuda.synchronize()
        outs.append((out, lse, dQ, dK, dV))
    for a, c in zip(*outs):
        assert torch.equal(a, c)


def test_index_add_rows_malformed_lists_stay_in_bounds():
    """Occurrence offsets that decrease or leave [0, n] and positions outside
    [0, n) give unspecified sums, but every access stays in range: the call
    succeeds, the sums of the (finite) source rows are finite, and a second
    call gives bitwise the same rows."""
    _announce("index add with malformed occurrence lists")
    r = np.random.default_rng(11)
    n, rows, D = 10_000, 500, 8
    off = torch.as_tensor(r.integers(-5, n + 6, rows + 1).astype(np.int32), device="cuda")
    occ = torch.as_tensor(r.integers(-3, n + 4, n).astype(np.int32), device="cuda")
    src = _randn((n, D), "f32", "cuda", 12)
    got = _index_add_gpu(off, occ, n, rows, src)
    assert torch.isfinite(got).all()
    assert torch.equal(got, _index_add_gpu(off, occ, n, rows, src))


# ------------------------------------------------------------------ coefficient form
def _scaled_rows_gpu(off_occ, occ, n, num_rows, dst_off, N, H, dh, scal, src):
    dst = torch.full((num_rows, H, dh), float("nan"), device="cuda")
    wsb = fast.fast_index_add_scaled_rows_workspace(n, num_rows, H, dh)
    ws = torch.empty(wsb, dtype=torch.uint8, device="cuda")
    dt = fast.BF16 if src.dtype == torch.bfloat16 else fast.F32
    fast.fast_index_add_scaled_rows(off_occ, occ, n, num_rows, dst_off, N, H, dh, dt, scal, src,
                                    dst, ws, wsb)
    torch.cuda.synchronize()
    return dst


@pytest.mark.parametrize("H,dh,dt,rows", [(2, 50, "f32", 300), (4, 32, "bf16", 5000), (1, 7, "f32", 40),
                                          (3, 4, "bf16", 1000), (2, 1, "f32", 100)])
def test_index_add_scaled_rows_vs_oracle(H, dh, dt, rows):
    _announce(f"scaled row sums H={H} dh={dh} {dt} rows={rows}")
    r = np.random.default_rng(H * 100 + dh + rows)
    counts = r.integers(0, 12, 20_000).astype(np.int32)
    counts[::53] = 0                                        # empty segments
    off = oracle.csr_offsets(counts)
    N, E = counts.size, int(off[-1])
    idx = ((r.zipf(1.3, E) - 1) % rows).astype(np.int32)   # hub rows read by thousands of edges
    idx[::97] = -1
    scal = torch.as_tensor(r.standard_normal((E, H)).astype(np.float32), device="cuda")
    src = _randn((N, H, dh), dt, "cuda", H + dh)
    occ_off, occ = _occ_gpu(idx, rows + 2)                  # two rows nobody reads
    got = _scaled_rows_gpu(occ_off, occ, E, rows + 2, to_dev(off), N, H, dh, scal, src)
    want = oracle.index_add_scaled_rows(idx, off, rows + 2, scal.cpu().numpy(), _host(src))
    assert_close(got, want, "f32", f"scaled rows H={H} dh={dh}")
    again = _scaled_rows_gpu(occ_off, occ, E, rows + 2, to_dev(off), N, H, dh, scal, src)
    assert torch.equal(got, again), "scaled row sums must be bitwise reproducible"
    assert torch.all(got[rows:] == 0)


@pytest.mark.parametrize("cfg,i", BLOCKS)
def test_indexed_coefficients_and_row_gradients(cfg, i):
    """Coefficient form: every segment's dQ, and the dK, dV each edge's
    coefficients form, against the oracle; then every row gradient from the
    GPU's coefficients against the oracle's fp64 sums of the same ones."""
    b = make_batch(cfg)
    _announce(f"coefficient-form backward cfg={cfg} block={i}")
    blk, kidx, vidx, Uk, Uv, o = _indexed_block(b, i, cfg)
    off = oracle.csr_offsets(blk.counts)
    N, E, H, dh, dt = blk.num_dst, blk.num_edges, b.H, b.dh, b.dtype
    scale = float(np.float32(1 / np.sqrt(dh)))
    d_off, d_k, d_v = to_dev(off), to_dev(kidx), to_dev(vidx)
    g = fast.tcsr(d_off, E)
    dQ = torch.empty((N, H, dh), dtype=tdtype(dt), device="cuda")
    ge = torch.empty((E, H), device="cuda")
    ae = torch.empty((E, H), device="cuda")
    fast.fast_edge_attention_bwd_indexed_coef(g, H, dh, DT[dt], o["Q"], o["K"], d_k, Uk, o["V"],
                                              d_v, Uv, scale, SLOPE, None, o["dO"], dQ, ge, ae)
    torch.cuda.synchronize()
    what = f"cfg{cfg}/L{i + 1} coefficients"
    Qh, dOh = _cpu(o["Q"]), _cpu(o["dO"])
    Kh, Vh = _cpu(o["K"][d_k.long()]), _cpu(o["V"][d_v.long()])
    dQh, g64, a64 = _cpu(dQ), ge.double().cpu().numpy(), ae.double().cpu().numpy()
    off64 = off.astype(np.int64)

    def one(a, c):
        ea, ec = int(off64[a]), int(off64[c])
        sub = (off64[a:c + 1] - ea).astype(np.int32)
        Q64, dO64 = Qh[a:c].double().numpy(), dOh[a:c].double().numpy()
        K64, V64 = Kh[ea:ec].double().numpy(), Vh[ea:ec].double().numpy()
        r_dQ, r_dK, r_dV, alts = bwd_reference_with_kinks(sub, Q64, K64, V64, dO64, scale, SLOPE)
        lseg = np.repeat(np.arange(c - a), np.diff(sub))
        dK_formed = torch.from_numpy(g64[ea:ec, :, None] * Q64[lseg])
        dV_formed = torch.from_numpy(a64[ea:ec, :, None] * dO64[lseg])
        tag = f"{what} segments [{a}, {c})"
        assert_close(dV_formed, r_dV, dt, tag + " alpha dO")
        assert_bwd_close(dQh[a:c], dK_formed, sub, r_dQ, r_dK, alts, dt, tag)
        return c - a

    assert sum(over_ranges(one, segment_ranges(off64, 64))) == N
    # row gradients from the GPU's coefficients, every row
    for name, idx, U, scal, src in (("K", kidx, Uk, ge, o["Q"]), ("V", vidx, Uv, ae, o["dO"])):
        occ_off, occ = _occ_gpu(idx, U)
        rows_grad = _scaled_rows_gpu(occ_off, occ, E, U, d_off, N, H, dh, scal, src).cpu()
        want = oracle.index_add_scaled_rows(idx, off, U, scal.cpu().numpy(), _host(src))
        assert_close(rows_grad, want, "f32", f"{what} d{name} rows")
    del o, dQ, ge, ae
    torch.cuda.empty_cache()
