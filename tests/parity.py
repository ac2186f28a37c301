"""Shared helpers of the GPU parity tests: tolerance rule, device upload,
sub-problems of sampled segments, and the LeakyReLU-kink rule.

Tolerance (elementwise, against the fp64 oracle r):
    fp32 storage:  |x - r| <= 1e-5 + 1e-5 |r|
    bf16 storage:  |x - r| <= 2e-2 + 2e-2 |r|
Integer and byte outputs are compared bit-exactly.
"""
from __future__ import annotations

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
