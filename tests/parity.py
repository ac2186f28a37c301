"""Shared helpers of the GPU parity tests: tolerance rule, device upload,
sub-problems of sampled segments, and the LeakyReLU-kink rule.

Tolerance (elementwise, against the fp64 oracle r):
    fp32 storage:  |x - r| <= 1e-5 + 1e-5 |r|
    bf16 storage:  |x - r| <= 2e-2 + 2e-2 |r|
Integer and byte outputs are compared bit-exactly.
"""
from __future__ import annotations

import os
from concurrent.futures import ThreadPoolExecutor

import numpy as np
import torch

import oracle

TOL = {"f32": (1e-5, 1e-5), "bf16": (2e-2, 2e-2)}
SLOPE = 0.2
EPS32 = float(np.finfo(np.float32).eps)


def tdtype(dt: str):
    return torch.float32 if dt == "f32" else torch.bfloat16


def assert_close(x, ref, dt: str, what: str, mask=None):
    """x: device or host tensor/array; ref: float64 numpy array."""
    if isinstance(x, torch.Tensor):
        x = x.detach().float().cpu().numpy()
    x = np.asarray(x, dtype=np.float64)
    ref = np.asarray(ref, dtype=np.float64)
    assert x.shape == ref.shape, (what, x.shape, ref.shape)
    atol, rtol = TOL[dt]
    bad = ~(np.abs(x - ref) <= atol + rtol * np.abs(ref))
    if mask is not None:
        bad &= mask
    if bad.any():
        idx = np.argwhere(bad)[:5]
        detail = ", ".join(f"{tuple(i)}: got {x[tuple(i)]!r} want {ref[tuple(i)]!r}" for i in idx)
        raise AssertionError(f"{what}: {int(bad.sum())} of {bad.size} elements out of tolerance; {detail}")


def to_dev(a, dtype=None):
    t = torch.from_numpy(np.ascontiguousarray(a)) if isinstance(a, np.ndarray) else a
    if dtype is not None:
        t = t.to(dtype)
    return t.cuda()


def sample_segments(N: int, k: int, seed: int = 0, include=()):
    r = np.random.default_rng(seed)
    s = np.unique(np.concatenate([r.choice(N, size=min(k, N), replace=False),
                                  np.asarray(include, dtype=np.int64)])).astype(np.int64)
    return s


def sub_csr(off: np.ndarray, segs: np.ndarray):
    """Sub-problem of the given segments: (sub offsets, edge index of the sub-edges)."""
    counts = (off[segs + 1] - off[segs]).astype(np.int32)
    sub_off = oracle.csr_offsets(counts)
    eidx = np.concatenate([np.arange(off[s], off[s + 1]) for s in segs]) if len(segs) else \
        np.zeros(0, dtype=np.int64)
    return sub_off, eidx.astype(np.int64)


def kink_band(Q64, K64, sub_off, scale):
    """(e,h) pairs whose fp64 logit lies within the fp32 rounding bound of the
    dot product, where fp32 and fp64 may take different LeakyReLU branches."""
    N, H, dh = Q64.shape
    seg = np.repeat(np.arange(N), np.diff(sub_off))
    absdot = np.einsum("ehd,ehd->eh", np.abs(Q64[seg]), np.abs(K64))
    pre = scale * np.einsum("ehd,ehd->eh", Q64[seg], K64)
    bound = 2.0 * dh * EPS32 * abs(scale) * absdot + 1e-30
    return np.abs(pre) <= bound, seg


def bwd_reference_with_kinks(sub_off, Q64, K64, V64, dO64, scale, slope):
    """Oracle backward plus, for segments holding an ambiguous (e,h) pair,
    the alternatives with that pair's LeakyReLU branch flipped.  Returns
    (dQ, dK, dV, alternatives) where alternatives maps a segment to a list of
    (dQ_row, dK_rows) candidates."""
    dQ, dK, dV = oracle.edge_attention_bwd(sub_off, Q64, K64, V64, dO64, scale, slope)
    band, seg = kink_band(Q64, K64, sub_off, scale)
    alts = {}
    for e, h in zip(*np.nonzero(band)):
        v = int(seg[e])
        s0, s1 = int(sub_off[v]), int(sub_off[v + 1])
        lo = slice(s0, s1)
        for b in (1, 2):
            branch = np.zeros((s1 - s0, Q64.shape[1]), dtype=np.int8)
            branch[e - s0, h] = b
            one_off = np.array([0, s1 - s0], dtype=np.int32)
            q = Q64[v:v + 1]
            dq, dk, _ = oracle.edge_attention_bwd(one_off, q, K64[lo], V64[lo], dO64[v:v + 1], scale,
                                                  slope, branch=branch)
            alts.setdefault(v, []).append((dq[0], dk))
    return dQ, dK, dV, alts


def assert_bwd_close(dQ_gpu, dK_gpu, sub_off, dQ, dK, alts, dt, what):
    """Compare dQ/dK; segments with an ambiguous logit accept any candidate."""
    dQ_gpu = dQ_gpu.detach().float().cpu().numpy().astype(np.float64)
    dK_gpu = dK_gpu.detach().float().cpu().numpy().astype(np.float64)
    N = dQ.shape[0]
    mask_q = np.ones(dQ.shape, dtype=bool)
    mask_k = np.ones(dK.shape, dtype=bool)
    for v in alts:
        mask_q[v] = False
        mask_k[sub_off[v]:sub_off[v + 1]] = False
    assert_close(dQ_gpu, dQ, dt, what + " dQ", mask=mask_q)
    assert_close(dK_gpu, dK, dt, what + " dK", mask=mask_k)
    atol, rtol = TOL[dt]
    for v, cands in alts.items():
        sl = slice(sub_off[v], sub_off[v + 1])
        gq, gk = dQ_gpu[v], dK_gpu[sl]
        options = [(dQ[v], dK[sl])] + cands
        ok = any(np.all(np.abs(gq - q) <= atol + rtol * np.abs(q)) and
                 np.all(np.abs(gk - k) <= atol + rtol * np.abs(k)) for q, k in options)
        assert ok, f"{what}: segment {v} with an ambiguous logit matches no branch choice"
    return N


# ------------------------------------------------------------------ whole blocks on all host threads
def host_threads(limit: int = 16) -> int:
    """Threads for the oracle: the CPUs this process may use, at most `limit`."""
    try:
        n = len(os.sched_getaffinity(0))
    except AttributeError:
        n = os.cpu_count() or 1
    return max(1, min(limit, n))


def segment_ranges(off: np.ndarray, parts: int):
    """Cuts the segments of a block into at most `parts` contiguous ranges
    [a, c) of about equal edge counts (a destination's edges stay together)."""
    off = np.asarray(off, dtype=np.int64)
    N, E = off.shape[0] - 1, int(off[-1])
    if N == 0:
        return []
    cuts = np.searchsorted(off, np.linspace(0, E, parts + 1), side="left").astype(np.int64)
    cuts = np.clip(cuts, 0, N)
    cuts[0], cuts[-1] = 0, N
    cuts = np.maximum.accumulate(cuts)
    return [(int(a), int(c)) for a, c in zip(cuts[:-1], cuts[1:]) if c > a]


def over_ranges(fn, ranges, threads=None):
    """fn(a, c) on every range, on the host threads; the oracle's C routines
    run outside the interpreter lock.  Re-raises the first failure."""
    with ThreadPoolExecutor(threads or host_threads()) as ex:
        return list(ex.map(lambda r: fn(*r), ranges))


def _f64(t):
    if isinstance(t, torch.Tensor):
        return t.double().numpy()
    return np.asarray(t, dtype=np.float64)


def check_attention_block_full(off, ins, fused, fused_nolse, unfused, scale, slope, dt, what,
                               parts=None):
    """Every segment of a layer block against the oracle.  ins: host tensors
    Q, K, V, dO in the storage dtype.  fused / fused_nolse: host (out, lse,
    dQ, dK, dV) of the fused pair with and without the saved lse (out and
    lse of the second are not compared; None skips it); unfused: host (alpha, lse, out,
    dalpha, dV, dQ, dK) of the operator chain, or None.  The block is cut
    into contiguous segment ranges, each checked on its own host thread
    against the oracle run on that range alone."""
    off = np.asarray(off, dtype=np.int64)
    T = host_threads()
    ranges = segment_ranges(off, parts or 4 * T)

    def one(a, c):
        ea, ec = int(off[a]), int(off[c])
        sub = (off[a:c + 1] - ea).astype(np.int32)
        Q, dO = _f64(ins["Q"][a:c]), _f64(ins["dO"][a:c])
        K, V = _f64(ins["K"][ea:ec]), _f64(ins["V"][ea:ec])
        tag = f"{what} segments [{a}, {c})"
        out, lse, alpha, _ = oracle.edge_attention_fwd(sub, Q, K, V, scale, slope)
        dQ, dK, dV, alts = bwd_reference_with_kinks(sub, Q, K, V, dO, scale, slope)
        nz = np.diff(sub) > 0
        g_out, g_lse = fused[0][a:c], _f64(fused[1][a:c])
        assert_close(g_out, out, dt, tag + " fused out")
        assert_close(g_lse[nz], lse[nz], "f32", tag + " fused lse")
        assert np.all(np.isneginf(g_lse[~nz])), tag + ": empty segment lse must be -inf"
        for name, r in (("lse", fused), ("nolse", fused_nolse)):
            if r is None:
                continue
            assert_close(r[4][ea:ec], dV, dt, f"{tag} fused[{name}] dV")
            assert_bwd_close(r[2][a:c], r[3][ea:ec], sub, dQ, dK, alts, dt, f"{tag} fused[{name}]")
        if unfused is not None:
            dalpha, _ = oracle.aggregate_bwd(sub, alpha, V, dO)
            u_alpha, u_lse, u_out, u_dalpha, u_dV, u_dQ, u_dK = unfused
            assert_close(u_alpha[ea:ec], alpha, "f32", tag + " ESM alpha")
            assert_close(_f64(u_lse[a:c])[nz], lse[nz], "f32", tag + " ESM lse")
            assert_close(u_out[a:c], out, dt, tag + " AGG out")
            assert_close(u_dalpha[ea:ec], dalpha, "f32", tag + " AGG dalpha")
            assert_close(u_dV[ea:ec], dV, dt, tag + " AGG dV")
            assert_bwd_close(u_dQ[a:c], u_dK[ea:ec], sub, dQ, dK, alts, dt, tag + " ESM-bwd")
        return c - a

    done = over_ranges(one, ranges, T)
    assert sum(done) == off.shape[0] - 1
    return len(ranges)


def check_time_encode_full(off, dst_t, edge_t, omega, phi, te, dt, what, parts=None):
    """Every row of a block's time encoding (te: host tensor [E, d_t]) against
    the oracle, over contiguous segment ranges on the host threads."""
    off = np.asarray(off, dtype=np.int64)
    T = host_threads()
    ranges = segment_ranges(off, parts or 4 * T)

    def one(a, c):
        ea, ec = int(off[a]), int(off[c])
        sub = (off[a:c + 1] - ea).astype(np.int32)
        ref = oracle.time_encode(sub, dst_t[a:c], edge_t[ea:ec], omega, phi)
        assert_close(te[ea:ec], ref, dt, f"{what} segments [{a}, {c})")
        return ec - ea

    assert sum(over_ranges(one, ranges, T)) == int(off[-1])


def oracle_sample_chunks(g, roots, rt, k, chunk):
    """The oracle over consecutive chunks of roots on all host threads (each
    root's result depends on that root alone), concatenated into one block."""
    cuts = list(range(0, roots.size, chunk)) + [roots.size]
    parts = over_ranges(lambda a, c: oracle.sample_recent(g.indptr, g.nbr, g.ts, g.eid, roots[a:c],
                                                          rt[a:c], k),
                        [(a, c) for a, c in zip(cuts[:-1], cuts[1:]) if c > a])
    if not parts:
        return np.zeros(1, np.int32), np.zeros(0, np.int64), np.zeros(0, np.float32), np.zeros(0, np.int64)
    base = np.cumsum([0] + [int(p[0][-1]) for p in parts[:-1]])
    off = np.concatenate([[0]] + [p[0][1:].astype(np.int64) + b for p, b in zip(parts, base)])
    return (off.astype(np.int32), np.concatenate([p[1] for p in parts]),
            np.concatenate([p[2] for p in parts]), np.concatenate([p[3] for p in parts]))
