"""Pins of the fp64 CPU oracle against facts that do not come from the oracle.

Each check is independent of the oracle's own loops: library routines that
compute the same quantity (np.cumsum, np.unique, numpy fancy indexing,
torch's scaled-dot-product attention and its autograd, scipy's softmax and
logsumexp), dense padded textbook attention, closed forms of the cosine,
softmax invariants, the softmax Jacobian written as a matrix, and central
finite differences.  Together they fail on a dropped term, a wrong sign, a
wrong index or a transposed operand anywhere in the oracle (see
test_oracle_mutations.py, which plants such mistakes and checks that a pin
here catches each one).
"""
import math

import numpy as np
import pytest
import scipy.special
import torch

import oracle
from synth import make_batch, omega_phi, tiny_graph

SLOPE = 0.2


def _csr(counts):
    counts = np.asarray(counts, dtype=np.int32)
    return np.concatenate([[0], np.cumsum(counts)]).astype(np.int32)


def _rand_qkv(N, E, H, dh, seed):
    r = np.random.default_rng(seed)
    return (r.standard_normal((N, H, dh)), r.standard_normal((E, H, dh)),
            r.standard_normal((E, H, dh)), r.standard_normal((N, H, dh)))


def _dense(off, X):
    """Pad per-edge rows [E,H,dh] into [N,Dmax,H,dh] plus a validity mask."""
    N = off.shape[0] - 1
    deg = np.diff(off)
    Dm = max(int(deg.max()) if N else 0, 1)
    out = np.zeros((N, Dm) + X.shape[1:])
    mask = np.zeros((N, Dm), dtype=bool)
    for v in range(N):
        out[v, :deg[v]] = X[off[v]:off[v + 1]]
        mask[v, :deg[v]] = True
    return out, mask


def _dense_attention(off, Q, K, V, scale, slope):
    """Textbook masked attention on padded neighbour tiles (numpy + scipy)."""
    Kd, mask = _dense(off, K)
    Vd, _ = _dense(off, V)
    S = scale * np.einsum("nhd,nkhd->nhk", Q, Kd)
    S = np.where(S > 0, S, slope * S)
    S = np.where(mask[:, None, :], S, -np.inf)
    A = scipy.special.softmax(S, axis=2)
    out = np.einsum("nhk,nkhd->nhd", A, Vd)
    lse = scipy.special.logsumexp(S, axis=2)
    return out, A, lse, mask


# ---------------------------------------------------------------- offsets (a1)
@pytest.mark.parametrize("n", [0, 1, 7, 1000])
def test_offsets_vs_cumsum(n):
    r = np.random.default_rng(n)
    counts = r.integers(0, 25, n).astype(np.int32)
    off = oracle.csr_offsets(counts)
    ref = np.concatenate([[0], np.cumsum(counts)])
    assert off.dtype == np.int32 and np.array_equal(off, ref)
    assert off[-1] == counts.sum() and np.all(np.diff(off) >= 0)


# ---------------------------------------------------------------- dedup (a2)
@pytest.mark.parametrize("case", ["random", "empty", "single", "allsame", "sorted", "zipf"])
def test_dedup_vs_numpy_unique(case):
    r = np.random.default_rng(3)
    ids = {
        "random": r.integers(0, 500, 3000),
        "empty": np.zeros(0, dtype=np.int64),
        "single": np.array([42]),
        "allsame": np.full(1000, 7),
        "sorted": np.arange(0, 2000, 3),
        "zipf": make_batch(2).node_ids,
    }[case].astype(np.int64)
    uni, inv = oracle.dedup(ids)
    ref_u, ref_inv = np.unique(ids, return_inverse=True)
    assert np.array_equal(uni, ref_u)
    assert np.array_equal(inv, ref_inv.reshape(-1))
    assert inv.dtype == np.int32
    if ids.size:
        assert np.array_equal(uni[inv], ids)
        assert np.all(np.diff(uni) > 0)


def test_repetition_rate_definition():
    # Sec. 3.1: R = 1 - N_u / N_i; 12 ids with 7 distinct transfer 7 rows, not 12.
    ids = np.array([5, 9, 5, 2, 9, 9, 11, 2, 40, 41, 5, 3], dtype=np.int64)
    uni, _ = oracle.dedup(ids)
    assert uni.size == 7
    assert math.isclose(1 - uni.size / ids.size, 5 / 12)


# ---------------------------------------------------------------- gather (a3)
@pytest.mark.parametrize("dtype", [np.float32, np.uint16])
def test_gather_identity_slots(dtype):
    r = np.random.default_rng(5)
    table = r.standard_normal((300, 172)).astype(np.float32)
    if dtype == np.uint16:
        table = (table.view(np.uint32) >> 16).astype(np.uint16)   # a bf16 bit table
    ids = r.integers(0, 300, 2000).astype(np.int64)
    uni, inv = oracle.dedup(ids)
    rows, hit, miss = oracle.gather(uni, table)
    assert hit.all() and miss.size == 0
    assert rows.tobytes() == table[uni].tobytes()
    # reconstruction through the inverse index returns every original row
    assert rows[inv].tobytes() == table[ids].tobytes()


def test_gather_slot_map_and_miss_list():
    r = np.random.default_rng(6)
    bound, C = 5000, 700
    cache = r.standard_normal((C, 16)).astype(np.float32)
    slot_map = np.full(bound, -1, dtype=np.int32)
    cached = r.choice(bound, C, replace=False)
    slot_map[cached] = np.arange(C, dtype=np.int32)
    ids = r.integers(0, bound, 4000).astype(np.int64)
    uni, _ = oracle.dedup(ids)
    rows, hit, miss = oracle.gather(uni, cache, slot_map)
    ref_miss = np.flatnonzero(slot_map[uni] < 0)
    assert np.array_equal(miss, ref_miss)
    assert np.array_equal(hit, slot_map[uni] >= 0)
    assert rows[hit].tobytes() == cache[slot_map[uni[hit]]].tobytes()


# ---------------------------------------------------------------- time encoding (a4)
def test_time_encode_zero_dt_and_segment_mapping():
    blk = tiny_graph([3, 0, 5, 1, 4])
    off = _csr(blk.counts)
    t_e = blk.edge_t.copy()
    # edges 1 and 6 get their own destination's time: dt = 0 -> cos(phi) = 1 exactly
    seg = np.repeat(np.arange(blk.num_dst), blk.counts)
    for e in (1, 6):
        t_e[e] = blk.dst_t[seg[e]]
    om, ph = omega_phi(16)
    te = oracle.time_encode(off, blk.dst_t, t_e, om, ph)
    assert np.all(te[[1, 6]] == 1.0)
    others = np.setdiff1d(np.arange(blk.num_edges), [1, 6])
    assert np.all(te[others, 0] != 1.0)


def test_time_encode_closed_forms():
    off = np.array([0, 3], dtype=np.int32)
    t_dst = np.array([1.0], dtype=np.float32)
    t_e = np.array([0.0, 0.0, 1.0], dtype=np.float32)        # dt = 1, 1, 0
    pi32, half32 = np.float32(np.pi), np.float32(np.pi / 2)
    om = np.array([pi32, half32, 0.0], dtype=np.float32)
    ph = np.array([0.0, 0.0, half32], dtype=np.float32)
    te = oracle.time_encode(off, t_dst, t_e, om, ph)
    # cos(pi + d) = -cos(d),  cos(pi/2 + d) = -sin(d), d = fl32(x) - x (known exactly)
    d_pi = float(pi32) - math.pi
    d_half = float(half32) - math.pi / 2
    assert abs(te[0, 0] - (-math.cos(d_pi))) < 1e-15
    assert abs(te[0, 1] - (-math.sin(d_half))) < 1e-15
    assert abs(te[0, 1] + 4.371139e-8) < 1e-13
    assert np.all(np.abs(te[:, 2] - (-math.sin(d_half))) < 1e-15)   # omega = 0 -> cos(phi)
    assert te[2, 0] == 1.0 and te[2, 1] == 1.0                      # dt = 0, phi = 0


def test_time_encode_double_angle_columns():
    # omega_j = 2^j * omega_0 makes every argument exactly twice the previous
    # one, so cos(2x) = 2 cos(x)^2 - 1 links column j+1 to column j.
    blk = tiny_graph([4, 2, 6], seed=11)
    off = _csr(blk.counts)
    om = (np.float32(1.7e-3) * (2.0 ** np.arange(10))).astype(np.float32)
    ph = np.zeros(10, dtype=np.float32)
    te = oracle.time_encode(off, blk.dst_t, blk.edge_t, om, ph)
    np.testing.assert_allclose(te[:, 1:], 2 * te[:, :-1] ** 2 - 1, atol=1e-9)
    assert np.abs(te).max() <= 1.0


def test_time_encode_fp32_difference():
    # dt is one fp32 subtraction: 2^25 - 1 rounds to 2^25 (ties to even), so
    # t_e = 1 and t_e = 0 give the same row, while an fp64 dt would differ.
    off = np.array([0, 2], dtype=np.int32)
    t_dst = np.array([2.0 ** 25], dtype=np.float32)
    t_e = np.array([1.0, 0.0], dtype=np.float32)
    om, ph = np.array([1.0, 0.25], dtype=np.float32), np.zeros(2, dtype=np.float32)
    te = oracle.time_encode(off, t_dst, t_e, om, ph)
    assert np.array_equal(te[0], te[1])
    assert abs(math.cos(2.0 ** 25 - 1) - math.cos(2.0 ** 25)) > 1e-2


# ---------------------------------------------------------------- indexed operands
def test_occurrence_csr_vs_numpy():
    r = np.random.default_rng(2)
    U = 700
    idx = (r.zipf(1.4, 20000) - 1).astype(np.int32)
    idx[::37] = -3                                   # left out
    idx[5::41] = U + 9
    off, occ = oracle.occurrence_csr(idx, U)
    valid = (idx >= 0) & (idx < U)
    assert np.array_equal(np.diff(off), np.bincount(idx[valid], minlength=U))
    pos = np.flatnonzero(valid)
    assert np.array_equal(occ, pos[np.argsort(idx[valid], kind="stable")])


def test_index_add_rows_vs_numpy():
    r = np.random.default_rng(3)
    idx = r.integers(-1, 50, 3000).astype(np.int32)
    src = r.standard_normal((3000, 4, 5))
    got = oracle.index_add_rows(idx, 48, src)
    want = np.zeros((48, 4, 5))
    ok = (idx >= 0) & (idx < 48)
    np.add.at(want, idx[ok], src[ok])
    np.testing.assert_allclose(got, want, rtol=1e-12, atol=1e-12)


def test_bwd_scalars_are_the_per_edge_gradient_coefficients():
    # per-edge coefficients against the pinned backward: g[e,h] Q[v,h,:] is
    # dK[e,h,:] and alpha[e,h] dO[v,h,:] is dV[e,h,:] (v the segment of e);
    # alpha sums to 1 over a non-empty segment; an empty segment has no edges
    r = np.random.default_rng(12)
    counts = [4, 0, 1, 6, 3, 0, 2]
    off = _csr(counts)
    N, E, H, dh = len(counts), int(off[-1]), 3, 5
    Q, dO = r.standard_normal((N, H, dh)), r.standard_normal((N, H, dh))
    K, V = r.standard_normal((E, H, dh)), r.standard_normal((E, H, dh))
    for slope in (SLOPE, 1.0, 0.0):
        dQ, g, al = oracle.edge_attention_bwd_scalars(off, Q, K, V, dO, 0.7, slope)
        rdQ, rdK, rdV = oracle.edge_attention_bwd(off, Q, K, V, dO, 0.7, slope)
        seg = np.repeat(np.arange(N), counts)
        np.testing.assert_allclose(g[:, :, None] * Q[seg], rdK, rtol=1e-12, atol=1e-14)
        np.testing.assert_allclose(al[:, :, None] * dO[seg], rdV, rtol=1e-12, atol=1e-14)
        np.testing.assert_allclose(dQ, rdQ, rtol=1e-12, atol=1e-14)
        sums = np.zeros((N, H))
        np.add.at(sums, seg, al)
        np.testing.assert_allclose(sums[np.array(counts) > 0], 1.0, rtol=1e-12)


def test_index_add_scaled_rows_vs_numpy():
    # the scaled transposed gather is the plain one applied to the per-edge
    # rows scal[e,h] * src[seg e, h, :]; indices outside the rows are left out
    r = np.random.default_rng(13)
    counts = r.integers(0, 6, 300)
    off = _csr(counts)
    N, E, H, dh, U = counts.size, int(off[-1]), 2, 3, 40
    idx = r.integers(-2, U + 2, E).astype(np.int32)
    scal, src = r.standard_normal((E, H)), r.standard_normal((N, H, dh))
    seg = np.repeat(np.arange(N), counts)
    want = np.zeros((U, H, dh))
    ok = (idx >= 0) & (idx < U)
    np.add.at(want, idx[ok], scal[ok][:, :, None] * src[seg[ok]])
    np.testing.assert_allclose(oracle.index_add_scaled_rows(idx, off, U, scal, src), want,
                               rtol=1e-12, atol=1e-12)


def test_indexed_attention_gradients_by_finite_differences():
    # compact K and V rows read by several edges each: the gradient of
    # L = sum(dOut * out) with respect to a compact row is the derivative of
    # the forward taken through every edge that reads it
    r = np.random.default_rng(8)
    counts = [3, 1, 4, 2, 5]
    off = _csr(counts)
    N, E, H, dh, Uk, Uv = len(counts), int(off[-1]), 2, 3, 6, 4
    Q = r.standard_normal((N, H, dh))
    K = r.standard_normal((Uk, H, dh))
    V = r.standard_normal((Uv, H, dh))
    dO = r.standard_normal((N, H, dh))
    kidx = r.integers(0, Uk, E).astype(np.int32)
    vidx = r.integers(0, Uv, E).astype(np.int32)
    kidx[:3] = 2                                     # row 2 read three times
    scale = 1 / math.sqrt(dh)
    _, _, _, dKr, dVr = oracle.edge_attention_bwd_indexed(off, Q, K, kidx, V, vidx, dO, scale, SLOPE)

    def loss(Kx, Vx):
        out = oracle.edge_attention_fwd_indexed(off, Q, Kx, kidx, Vx, vidx, scale, SLOPE)[0]
        return float(np.sum(dO * out))

    hstep = 1e-6
    for (arr, grad, which) in ((K, dKr, 0), (V, dVr, 1)):
        for u in range(arr.shape[0]):
            for h in range(H):
                for i in range(dh):
                    lo, hi = arr.copy(), arr.copy()
                    lo[u, h, i] -= hstep
                    hi[u, h, i] += hstep
                    fd = ((loss(hi, V) - loss(lo, V)) if which == 0 else
                          (loss(K, hi) - loss(K, lo))) / (2 * hstep)
                    assert abs(grad[u, h, i] - fd) <= 1e-6 * (1 + abs(fd)), (which, u, h, i)
    # the same row gradients from the per-edge coefficients: dK row u is the
    # sum of g[e] Q[seg e] over the edges reading u, dV row u that of
    # alpha[e] dO[seg e]; compared with the finite differences above through
    # the gradients they already matched
    _, g, al = oracle.edge_attention_bwd_scalars(off, Q, K[kidx], V[vidx], dO, scale, SLOPE)
    np.testing.assert_allclose(oracle.index_add_scaled_rows(kidx, off, Uk, g, Q), dKr,
                               rtol=1e-12, atol=1e-12)
    np.testing.assert_allclose(oracle.index_add_scaled_rows(vidx, off, Uv, al, dO), dVr,
                               rtol=1e-12, atol=1e-12)
    # identity index: the plain operator
    ident = np.arange(E, dtype=np.int32)
    Ke, Ve = K[kidx], V[vidx]
    a = oracle.edge_attention_fwd_indexed(off, Q, Ke, ident, Ve, None, scale, SLOPE)[0]
    b = oracle.edge_attention_fwd(off, Q, Ke, Ve, scale, SLOPE)[0]
    assert np.array_equal(a, b)


# ---------------------------------------------------------------- most-recent-k sampling
def test_sample_recent_hand_example():
    # node 0 has events at t = 1, 2, 2, 5, 7; node 1 none; node 2 one at t = 3
    indptr = np.array([0, 5, 5, 6], np.int64)
    nbr = np.array([10, 11, 12, 13, 14, 20], np.int64)
    ts = np.array([1, 2, 2, 5, 7, 3], np.float32)
    eid = np.array([100, 101, 102, 103, 104, 200], np.int64)
    roots = np.array([0, 0, 0, 1, 2, 7, -1], np.int64)
    rt = np.array([5, 100, 1, 9, 3.5, 1, 1], np.float32)
    off, src, et, ei = oracle.sample_recent(indptr, nbr, ts, eid, roots, rt, 2)
    # t = 5: earlier events at 1, 2, 2 -> the last two (the two at t = 2);
    # t = 100: the two latest; t = 1: none (strictly earlier only)
    assert off.tolist() == [0, 2, 4, 4, 4, 5, 5, 5]
    assert src.tolist() == [11, 12, 13, 14, 20]
    assert et.tolist() == [2, 2, 5, 7, 3]
    assert ei.tolist() == [101, 102, 103, 104, 200]


@pytest.mark.parametrize("k", [1, 3, 10])
def test_sample_recent_vs_numpy(k):
    from synth import make_temporal_graph, sampler_roots
    g = make_temporal_graph(3000, 20000, seed=k)
    roots, rt = sampler_roots(g, 300, seed=k)
    rt[::7] = g.ev_t[::97][:rt[::7].size]          # some query times equal to event times
    off, src, et, ei = oracle.sample_recent(g.indptr, g.nbr, g.ts, g.eid, roots, rt, k)
    for i, (v, t) in enumerate(zip(roots, rt)):
        lo, hi = g.indptr[v], g.indptr[v + 1]
        pos = lo + np.flatnonzero(g.ts[lo:hi] < t)[-k:] if k else []
        sl = slice(off[i], off[i + 1])
        assert np.array_equal(src[sl], g.nbr[pos]) and np.array_equal(ei[sl], g.eid[pos])
        assert np.array_equal(et[sl], g.ts[pos])
        # the most recent: every earlier entry left out is no later than those taken
        earlier = g.ts[lo:hi][g.ts[lo:hi] < t]
        assert off[i + 1] - off[i] == min(k, earlier.size)
        if earlier.size > k:
            assert np.sort(earlier)[-k - 1] <= et[sl].min()
        assert np.all(et[sl] < t)


# ---------------------------------------------------------------- greedy cache selection (Alg. 1)
def test_access_count_hand_example():
    # batch 0 touches 1, 2 (twice), 5; batch 1 touches 2, 9, 1; batch 2 touches 7
    # and an id outside the universe.  A repeat inside a batch counts once.
    f = oracle.access_count([[1, 2, 2, 5], [2, 9, 1], [7, 12]], 10)
    assert f.tolist() == [0, 2, 2, 0, 0, 1, 0, 1, 0, 1]
    # counters accumulate over calls
    f2 = oracle.access_count([[0, 0, 9]], 10, freq=f)
    assert f2.tolist() == [1, 2, 2, 0, 0, 1, 0, 1, 0, 2]


def test_access_count_vs_numpy():
    r = np.random.default_rng(4)
    bound = 5000
    batches = [r.zipf(1.3, size=int(r.integers(0, 3000))) % bound for _ in range(40)]
    want = np.zeros(bound, dtype=np.int64)
    for b in batches:
        want += np.bincount(np.unique(b), minlength=bound)
    assert np.array_equal(oracle.access_count(batches, bound), want)


def test_greedy_hot_set_hand_example():
    # node counts [3, 1, 2], edge counts [2, 2, 0, 5], budget 4 of 7 ids:
    # e3 (5) beats v0 (3); v0 (3) beats e0 (2); at the tie 2 = 2 the edge
    # wins, so e0 then e1 (ascending id) fill the budget before v2.
    hv, he = oracle.greedy_hot_set([3, 1, 2], [2, 2, 0, 5], 4 / 7)
    assert hv.tolist() == [0] and he.tolist() == [3, 0, 1]
    # budget 5: the edges with count 2 are used up, so v2 (2) beats e2 (0)
    hv, he = oracle.greedy_hot_set([3, 1, 2], [2, 2, 0, 5], 5 / 7)
    assert hv.tolist() == [0, 2] and he.tolist() == [3, 0, 1]
    # budget 1.0: everything, nodes list exhausted first
    hv, he = oracle.greedy_hot_set([3, 1, 2], [2, 2, 0, 5], 1.0)
    assert sorted(hv.tolist()) == [0, 1, 2] and sorted(he.tolist()) == [0, 1, 2, 3]
    # empty budget and empty lists
    assert [x.size for x in oracle.greedy_hot_set([3, 1], [2], 0.0)] == [0, 0]
    hv, he = oracle.greedy_hot_set(np.zeros(0), [4, 1], 1.0)
    assert hv.size == 0 and he.tolist() == [0, 1]


@pytest.mark.parametrize("alpha", [0.0, 0.013, 0.1, 0.37, 0.5, 1.0])
def test_greedy_hot_set_properties(alpha):
    # Properties that pin the selection without re-running it: the budget
    # ceil(alpha * (|V|+|E|)); maximal total frequency (the sum of the
    # budget's largest counts over both lists); every selected count >= every
    # unselected count; at the threshold count edges before nodes and, within
    # a kind, the smallest ids; each list in descending count, ascending id.
    r = np.random.default_rng(int(alpha * 1000) + 1)
    fv = r.integers(0, 6, 3000).astype(np.int32)
    fe = np.minimum(r.zipf(1.6, 7000), 6).astype(np.int32) - 1
    nv, ne = fv.size, fe.size
    hv, he = oracle.greedy_hot_set(fv, fe, alpha)
    B = math.ceil(alpha * (nv + ne))
    assert hv.size + he.size == B
    allf = np.sort(np.concatenate([fv, fe]))[::-1]
    assert fv[hv].sum() + fe[he].sum() == allf[:B].sum()
    if B == 0:
        return
    T = min(fv[hv].min() if hv.size else 99, fe[he].min() if he.size else 99)
    sel_v = np.zeros(nv, bool); sel_v[hv] = True
    sel_e = np.zeros(ne, bool); sel_e[he] = True
    assert np.all(fv[~sel_v] <= T) and np.all(fe[~sel_e] <= T)
    assert np.all(sel_v[fv > T]) and np.all(sel_e[fe > T])
    tie_v, tie_e = np.flatnonzero(fv == T), np.flatnonzero(fe == T)
    if sel_v[tie_v].any():
        assert sel_e[tie_e].all()
    for ties, sel in ((tie_v, sel_v), (tie_e, sel_e)):
        k = int(sel[ties].sum())
        assert np.array_equal(np.flatnonzero(sel & np.isin(np.arange(sel.size), ties)), ties[:k])
    for hot, f in ((hv, fv), (he, fe)):
        order = np.lexsort((hot, -f[hot]))
        assert np.array_equal(order, np.arange(hot.size))


# ---------------------------------------------------------------- time-encoding backward
def _dyadic_time_block(seed):
    """A block whose fp32 time arguments are exact: dt = k/8 (k <= 32),
    omega_j = m/256 in [0.25, 2], phi_j = n/64 in [-1, 1].  omega*dt + phi
    then needs at most 18 significant bits, so it stays exact in fp32 even
    after a perturbation of omega or phi by a multiple of 2^-12."""
    r = np.random.default_rng(seed)
    counts = np.array([3, 0, 5, 1, 4, 2], dtype=np.int32)
    off = _csr(counts)
    N, E, d_t = counts.size, int(off[-1]), 9
    t_dst = (4.0 + r.integers(0, 5, N)).astype(np.float32)
    seg = np.repeat(np.arange(N), counts)
    t_e = (t_dst[seg] - r.integers(0, 33, E) / 8.0).astype(np.float32)
    om = (r.integers(64, 513, d_t) / 256.0).astype(np.float32)
    ph = (r.integers(-64, 65, d_t) / 64.0).astype(np.float32)
    dte = r.standard_normal((E, d_t))
    return off, t_dst, t_e, om, ph, dte


def _te_loss(off, t_dst, t_e, om, ph, dte):
    return float(np.sum(dte * oracle.time_encode(off, t_dst, t_e, om, ph)))


def test_time_encode_bwd_finite_differences():
    # central differences of L = sum(dte * te) through the forward oracle,
    # Richardson-extrapolated from steps 2^-11 and 2^-12 (error O(h^4))
    off, t_dst, t_e, om, ph, dte = _dyadic_time_block(5)
    domega, dphi = oracle.time_encode_bwd(off, t_dst, t_e, om, ph, dte)

    def central(which, j, h):
        lo, hi = [a.copy() for a in (om, ph)], [a.copy() for a in (om, ph)]
        lo[which][j] -= np.float32(h)
        hi[which][j] += np.float32(h)
        return (_te_loss(off, t_dst, t_e, *hi, dte) - _te_loss(off, t_dst, t_e, *lo, dte)) / (2 * h)

    for j in range(om.size):
        for which, got in ((0, domega[j]), (1, dphi[j])):
            d1, d2 = central(which, j, 2.0 ** -11), central(which, j, 2.0 ** -12)
            fd = (4 * d2 - d1) / 3
            assert abs(got - fd) <= 1e-8 * (1 + abs(fd)), (which, j, got, fd)


def test_time_encode_bwd_pythagorean_with_the_forward():
    # one edge per destination and dte = 1: dphi_j = -sin(a_j) and the
    # forward gives cos(a_j) at the same fp32 argument, so dphi^2 + te^2 = 1;
    # domega_j = dphi_j * dt.  Large dt makes a_j ~ 1e4 rad, where an
    # argument not rounded to fp32 as in the forward breaks the identity.
    om, ph = omega_phi(12)
    ph = np.linspace(-1, 1, 12).astype(np.float32)
    for dt in (0.0, 0.75, 3.1e3, 9.87654e3):
        off = np.array([0, 1], dtype=np.int32)
        t_dst = np.array([1e4], dtype=np.float32)
        t_e = np.array([np.float32(1e4) - np.float32(dt)], dtype=np.float32)
        dt32 = float(t_dst[0] - t_e[0])
        te = oracle.time_encode(off, t_dst, t_e, om, ph)[0]
        domega, dphi = oracle.time_encode_bwd(off, t_dst, t_e, om, ph, np.ones((1, 12)))
        np.testing.assert_allclose(dphi ** 2 + te ** 2, 1.0, atol=1e-14)
        np.testing.assert_array_equal(domega, dphi * dt32)


def test_time_encode_bwd_sums_over_edges():
    # the gradient of a block is the sum of the gradients of its edges taken
    # one at a time (each edge as a one-edge block of its own destination)
    off, t_dst, t_e, om, ph, dte = _dyadic_time_block(9)
    domega, dphi = oracle.time_encode_bwd(off, t_dst, t_e, om, ph, dte)
    seg = np.repeat(np.arange(off.size - 1), np.diff(off))
    acc_w, acc_p = np.zeros(om.size), np.zeros(om.size)
    for e in range(t_e.size):
        w, p = oracle.time_encode_bwd(np.array([0, 1], np.int32), t_dst[seg[e]:seg[e] + 1],
                                      t_e[e:e + 1], om, ph, dte[e:e + 1])
        acc_w += w
        acc_p += p
    np.testing.assert_allclose(domega, acc_w, rtol=1e-12, atol=1e-12)
    np.testing.assert_allclose(dphi, acc_p, rtol=1e-12, atol=1e-12)


# ---------------------------------------------------------------- attention forward (a5-a7)
def test_fwd_vs_torch_sdpa():
    # slope = 1 removes the LeakyReLU: the operator is masked scaled-dot-product attention
    counts = [1, 4, 7, 2, 10, 3]
    off = _csr(counts)
    N, E, H, dh = len(counts), off[-1], 3, 5
    Q, K, V, _ = _rand_qkv(N, E, H, dh, 1)
    scale = 0.37
    out, lse, alpha, _ = oracle.edge_attention_fwd(off, Q, K, V, scale, 1.0)
    Kd, mask = _dense(off, K)
    Vd, _ = _dense(off, V)
    q = torch.tensor(Q)[:, :, None, :]                    # [N,H,1,dh]
    k = torch.tensor(Kd).permute(0, 2, 1, 3)              # [N,H,Dm,dh]
    v = torch.tensor(Vd).permute(0, 2, 1, 3)
    m = torch.tensor(mask)[:, None, None, :]
    ref = torch.nn.functional.scaled_dot_product_attention(q, k, v, attn_mask=m, scale=scale)
    np.testing.assert_allclose(out, ref[:, :, 0, :].numpy(), rtol=1e-12, atol=1e-12)


@pytest.mark.parametrize("slope", [0.2, 1.0, 0.0, -0.3])
def test_fwd_vs_dense_masked_attention(slope):
    counts = [5, 0, 1, 3, 8, 2, 0, 6]
    off = _csr(counts)
    N, E, H, dh = len(counts), off[-1], 2, 6
    Q, K, V, _ = _rand_qkv(N, E, H, dh, 2)
    out, lse, alpha, pre = oracle.edge_attention_fwd(off, Q, K, V, 0.5, slope)
    ref_out, A, ref_lse, mask = _dense_attention(off, Q, K, V, 0.5, slope)
    nz = np.diff(off) > 0
    np.testing.assert_allclose(out[nz], ref_out[nz], rtol=1e-12, atol=1e-12)
    np.testing.assert_allclose(lse[nz], ref_lse[nz], rtol=1e-12, atol=1e-12)
    # alpha per edge equals the dense weights at the edge's slot
    for v in np.flatnonzero(nz):
        np.testing.assert_allclose(alpha[off[v]:off[v + 1]].T, A[v][:, :counts[v]], rtol=1e-12)
    # empty segments: zero output, lse = -inf
    assert np.all(out[~nz] == 0.0) and np.all(np.isneginf(lse[~nz]))


def test_softmax_invariants():
    counts = [1, 2, 9, 1, 5, 13]
    off = _csr(counts)
    N, E, H, dh = len(counts), off[-1], 4, 3
    Q, K, V, _ = _rand_qkv(N, E, H, dh, 4)
    out, lse, alpha, _ = oracle.edge_attention_fwd(off, Q, K, V, 0.8, SLOPE)
    seg = np.repeat(np.arange(N), counts)
    sums = np.zeros((N, H))
    np.add.at(sums, seg, alpha)
    np.testing.assert_allclose(sums, 1.0, atol=1e-14)
    # a single-neighbour segment returns its value row exactly
    for v in (0, 3):
        assert np.all(alpha[off[v]] == 1.0)
        assert np.array_equal(out[v], V[off[v]])
    # Q = 0: uniform weights and the mean of V
    out0, _, alpha0, _ = oracle.edge_attention_fwd(off, np.zeros_like(Q), K, V, 0.8, SLOPE)
    np.testing.assert_allclose(alpha0, (1.0 / np.asarray(counts))[seg][:, None] * np.ones(H), rtol=1e-15)
    for v in range(N):
        np.testing.assert_allclose(out0[v], V[off[v]:off[v + 1]].mean(axis=0), rtol=1e-13, atol=1e-15)


def test_permutation_invariance_within_segment():
    counts = [6, 3, 8]
    off = _csr(counts)
    N, E, H, dh = 3, off[-1], 2, 5
    Q, K, V, dO = _rand_qkv(N, E, H, dh, 5)
    r = np.random.default_rng(9)
    perm = np.concatenate([off[v] + r.permutation(counts[v]) for v in range(N)])
    out, lse, alpha, _ = oracle.edge_attention_fwd(off, Q, K, V, 0.6, SLOPE)
    out_p, lse_p, alpha_p, _ = oracle.edge_attention_fwd(off, Q, K[perm], V[perm], 0.6, SLOPE)
    np.testing.assert_allclose(out_p, out, rtol=1e-13, atol=1e-14)
    np.testing.assert_allclose(alpha_p, alpha[perm], rtol=1e-13)
    dQ, dK, dV = oracle.edge_attention_bwd(off, Q, K, V, dO, 0.6, SLOPE)
    dQp, dKp, dVp = oracle.edge_attention_bwd(off, Q, K[perm], V[perm], dO, 0.6, SLOPE)
    np.testing.assert_allclose(dQp, dQ, rtol=1e-12, atol=1e-13)
    np.testing.assert_allclose(dKp, dK[perm], rtol=1e-12, atol=1e-13)
    np.testing.assert_allclose(dVp, dV[perm], rtol=1e-12, atol=1e-13)


def test_huge_logits_stay_finite():
    # the max subtraction (safe softmax, Sec. 4.3) keeps exp() in range
    counts = [4, 7]
    off = _csr(counts)
    Q, K, V, _ = _rand_qkv(2, 11, 2, 8, 6)
    out, lse, alpha, _ = oracle.edge_attention_fwd(off, Q, K, V, 1.0e4, SLOPE)
    assert np.isfinite(out).all() and np.isfinite(lse).all() and np.isfinite(alpha).all()
    ref_out, _, _, _ = _dense_attention(off, Q, K, V, 1.0e4, SLOPE)
    np.testing.assert_allclose(out, ref_out, rtol=1e-10, atol=1e-10)


# ---------------------------------------------------------------- backward (a8, a9)
def test_bwd_vs_torch_autograd_sdpa():
    counts = [2, 5, 1, 9, 4]
    off = _csr(counts)
    N, E, H, dh = len(counts), off[-1], 2, 7
    Q, K, V, dO = _rand_qkv(N, E, H, dh, 7)
    scale = 0.45
    dQ, dK, dV = oracle.edge_attention_bwd(off, Q, K, V, dO, scale, 1.0)
    Kd, mask = _dense(off, K)
    Vd, _ = _dense(off, V)
    q = torch.tensor(Q)[:, :, None, :].requires_grad_()
    k = torch.tensor(Kd).permute(0, 2, 1, 3).contiguous().requires_grad_()
    v = torch.tensor(Vd).permute(0, 2, 1, 3).contiguous().requires_grad_()
    m = torch.tensor(mask)[:, None, None, :]
    o = torch.nn.functional.scaled_dot_product_attention(q, k, v, attn_mask=m, scale=scale)
    (o * torch.tensor(dO)[:, :, None, :]).sum().backward()
    np.testing.assert_allclose(dQ, q.grad[:, :, 0, :].numpy(), rtol=1e-11, atol=1e-12)
    gk = k.grad.permute(0, 2, 1, 3).numpy()
    gv = v.grad.permute(0, 2, 1, 3).numpy()
    np.testing.assert_allclose(dK, gk[mask], rtol=1e-11, atol=1e-12)
    np.testing.assert_allclose(dV, gv[mask], rtol=1e-11, atol=1e-12)


def _loss(off, Q, K, V, dO, scale, slope):
    out, _, _, _ = oracle.edge_attention_fwd(off, Q, K, V, scale, slope)
    return float((out * dO).sum())


@pytest.mark.parametrize("slope", [SLOPE, 0.0, -0.3])
def test_bwd_finite_differences_leaky(slope):
    counts = [3, 1, 6, 0, 4]
    off = _csr(counts)
    N, E, H, dh = len(counts), off[-1], 2, 4
    Q, K, V, dO = _rand_qkv(N, E, H, dh, 8)
    scale = 0.9
    _, _, _, pre = oracle.edge_attention_fwd(off, Q, K, V, scale, slope)
    assert np.abs(pre).min() > 1e-3        # away from the LeakyReLU kink
    assert (pre > 0).any() and (pre < 0).any()
    dQ, dK, dV = oracle.edge_attention_bwd(off, Q, K, V, dO, scale, slope)
    h = 1e-6
    for name, X, G in (("Q", Q, dQ), ("K", K, dK), ("V", V, dV)):
        fd = np.zeros_like(X)
        for idx in np.ndindex(X.shape):
            Xp, Xm = X.copy(), X.copy()
            Xp[idx] += h
            Xm[idx] -= h
            args = {"Q": Q, "K": K, "V": V}
            args[name] = Xp
            lp = _loss(off, args["Q"], args["K"], args["V"], dO, scale, slope)
            args[name] = Xm
            lm = _loss(off, args["Q"], args["K"], args["V"], dO, scale, slope)
            fd[idx] = (lp - lm) / (2 * h)
        np.testing.assert_allclose(G, fd, rtol=1e-6, atol=1e-7, err_msg=name)
    assert np.all(dQ[3] == 0.0)             # empty segment


def test_softmax_bwd_vs_jacobian_matrix():
    counts = [5, 2, 7]
    off = _csr(counts)
    N, E, H, dh = 3, off[-1], 2, 3
    Q, K, _, _ = _rand_qkv(N, E, H, dh, 10)
    r = np.random.default_rng(11)
    dalpha = r.standard_normal((E, H))
    scale = 0.7
    alpha, _, pre = oracle.edge_softmax_fwd(off, Q, K, scale, SLOPE)
    dQ, dK = oracle.edge_softmax_bwd(off, Q, K, scale, SLOPE, alpha, dalpha)
    for v in range(N):
        sl = slice(off[v], off[v + 1])
        for h in range(H):
            a = alpha[sl, h]
            J = np.diag(a) - np.outer(a, a)          # d alpha / d s
            ds = J.T @ dalpha[sl, h]
            dpre = ds * np.where(pre[sl, h] > 0, 1.0, SLOPE)
            g = dpre * scale
            np.testing.assert_allclose(dQ[v, h], g @ K[sl, h, :], rtol=1e-12, atol=1e-13)
            np.testing.assert_allclose(dK[sl, h, :], np.outer(g, Q[v, h]), rtol=1e-12, atol=1e-13)


def test_aggregate_bwd_is_the_transpose():
    # aggregation is bilinear in (alpha, V): its backward is the exact adjoint
    counts = [4, 0, 2, 5]
    off = _csr(counts)
    N, E, H, dh = 4, off[-1], 3, 5
    r = np.random.default_rng(12)
    alpha = r.random((E, H))
    V = r.standard_normal((E, H, dh))
    dO = r.standard_normal((N, H, dh))
    da, dV = oracle.aggregate_bwd(off, alpha, V, dO)
    a2 = r.random((E, H))
    V2 = r.standard_normal((E, H, dh))
    # <dO, agg(a2, V)> = <da, a2> and <dO, agg(alpha, V2)> = <dV, V2>
    np.testing.assert_allclose((dO * oracle.aggregate_fwd(off, a2, V)).sum(), (da * a2).sum(), rtol=1e-12)
    np.testing.assert_allclose((dO * oracle.aggregate_fwd(off, alpha, V2)).sum(), (dV * V2).sum(), rtol=1e-12)


def test_branch_override():
    counts = [3, 4]
    off = _csr(counts)
    Q, K, V, dO = _rand_qkv(2, 7, 2, 4, 13)
    alpha, _, pre = oracle.edge_softmax_fwd(off, Q, K, 0.5, SLOPE)
    assert (pre > 0).any() and (pre < 0).any()
    da = np.random.default_rng(1).standard_normal(alpha.shape)
    ones = np.ones(alpha.shape, np.int8)
    twos = np.full(alpha.shape, 2, np.int8)
    dQ1, dK1 = oracle.edge_softmax_bwd(off, Q, K, 0.5, SLOPE, alpha, da, ones)
    dQr, dKr = oracle.edge_softmax_bwd(off, Q, K, 0.5, 1.0, alpha, da)
    np.testing.assert_allclose(dQ1, dQr, rtol=1e-14, atol=1e-15)
    dQ2, _ = oracle.edge_softmax_bwd(off, Q, K, 0.5, SLOPE, alpha, da, twos)
    dQs, _ = oracle.edge_softmax_bwd(off, Q, K, 0.5 * SLOPE, 1.0, alpha, da)
    # r = slope everywhere equals (scale*slope) with r = 1, since g = ds*r*scale
    np.testing.assert_allclose(dQ2, dQs, rtol=1e-13, atol=1e-15)


# ---------------------------------------------------------------- subgraph contract check
def test_check_tcsr_hand_counted_case():
    # off = [0, 3, 2, 5] with E = 4: segment 1 runs backwards, off[N] != E.
    # src ids -1 and 10 fall outside [0, 10).  dt < 0 where an edge is later
    # than its destination: segment 0 holds edges 0..2 (edge 1: 6 > 5),
    # segment 1 is skipped, segment 2 is [2, 5) cut to [2, 4) (edge 3: 2 > 1).
    off = np.array([0, 3, 2, 5], np.int32)
    v = oracle.check_tcsr(off, 4, src_ids=[-1, 0, 9, 10], src_bound=10,
                          edge_t=[4.0, 6.0, 0.0, 2.0], dst_t=[5.0, 5.0, 1.0])
    assert v.tolist() == [1, 1, 2, 0, 2]
    # every optional array absent: only the offset counters remain
    assert oracle.check_tcsr(off, 4).tolist() == [1, 1, 0, 0, 0]
    # N = 0: the single offset is both first and last
    assert oracle.check_tcsr(np.array([0], np.int32), 0).tolist() == [0, 0, 0, 0, 0]
    assert oracle.check_tcsr(np.array([3], np.int32), 0).tolist() == [0, 2, 0, 0, 0]


@pytest.mark.parametrize("cfg", [0, 1, 2])
def test_check_tcsr_generated_batches_are_clean(cfg):
    b = make_batch(cfg)
    for blk in b.blocks:
        off = oracle.csr_offsets(blk.counts)
        v = oracle.check_tcsr(off, blk.num_edges, blk.src_ids, b.node_bound, blk.edge_ids,
                              b.edge_bound, blk.edge_t, blk.dst_t)
        assert v.tolist() == [0, 0, 0, 0, 0]


def test_check_tcsr_each_planted_fault_hits_its_counter():
    b = make_batch(0)
    blk = b.blocks[0]
    off = oracle.csr_offsets(blk.counts)
    E, N = blk.num_edges, blk.num_dst
    base = dict(src_ids=blk.src_ids.copy(), src_bound=b.node_bound,
                edge_ids=blk.edge_ids.copy(), edge_bound=b.edge_bound,
                edge_t=blk.edge_t.copy(), dst_t=blk.dst_t.copy())
    v = [k for k in range(N) if blk.counts[k] > 0][3]
    e = int(off[v])
    cases = []
    a = dict(base); a["src_ids"] = a["src_ids"].copy(); a["src_ids"][e] = b.node_bound
    cases.append((off, a, 2))
    a = dict(base); a["edge_ids"] = a["edge_ids"].copy(); a["edge_ids"][e] = -1
    cases.append((off, a, 3))
    a = dict(base); a["edge_t"] = a["edge_t"].copy(); a["edge_t"][e] = a["dst_t"][v] + 1.0
    cases.append((off, a, 4))
    o = off.copy(); o[-1] += 1
    cases.append((o, base, 1))
    for o, a, k in cases:
        got = oracle.check_tcsr(o, E, **a)
        want = [0] * 5
        want[k] = 1
        assert got.tolist() == want, (k, got)
    # swapping two adjacent interior offsets with a gap breaks monotonicity once
    o = off.copy()
    i = next(i for i in range(1, N) if o[i + 1] > o[i])
    o[i], o[i + 1] = o[i + 1], o[i]
    assert oracle.check_tcsr(o, E)[0] == 1


# ---------------------------------------------------------------- regression fixture
def test_oracle_matches_stored_regression_fixture():
    import json, os
    from tests.golden import make_golden as mg
    with open(os.path.join(os.path.dirname(mg.__file__), "tiny_oracle.json")) as f:
        stored = json.load(f)
    got = mg.outputs(mg.inputs())
    for k, v in stored.items():
        a, b = np.asarray(got[k], dtype=np.float64), np.asarray(v, dtype=np.float64)
        assert a.shape == b.shape, k
        np.testing.assert_allclose(a, b, rtol=1e-12, atol=1e-14, err_msg=k)
