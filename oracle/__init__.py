"""NumPy front end of the fp64 CPU oracle (oracle.c).

TEST INFRASTRUCTURE ONLY: imported by the tests, the smoke check and the
benchmark's CPU-baseline leg.  Nothing in the HIP path imports it.

Every function takes host numpy arrays, widens floating operands exactly to
float64, and returns freshly allocated float64 (or integer) results.  The
composite attention functions are the plain compositions of the operator
definitions (edge softmax followed by aggregation; aggregation backward
followed by edge-softmax backward), Sec. 4.3.
"""
from __future__ import annotations

import ctypes as C
import os

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
# FAST_ORACLE_LIB names another build of oracle.c to load (the sanitizer
# test's instrumented build); default: liboracle.so beside this file.
_LIB_PATH = os.environ.get("FAST_ORACLE_LIB") or os.path.join(_HERE, "liboracle.so")
_lib = None

_p = C.c_void_p
_i64 = C.c_int64
_i32 = C.c_int
_f64 = C.c_double

_SIGS = {
    "oracle_csr_offsets": (None, [_p, _i64, _p]),
    "oracle_check_tcsr": (None, [_p, _i64, _i64, _p, _i64, _p, _i64, _p, _p, _p]),
    "oracle_dedup": (_i64, [_p, _i64, _p, _p]),
    "oracle_gather": (_i64, [_p, _i64, _p, _i64, _i64, _p, _p, _p]),
    "oracle_time_encode": (None, [_p, _i64, _p, _p, _p, _p, _i32, _p]),
    "oracle_occurrence_csr": (None, [_p, _i64, _i64, _p, _p]),
    "oracle_index_add_rows": (None, [_p, _i64, _i64, _i64, _p, _p]),
    "oracle_index_add_scaled_rows": (None, [_p, _p, _i64, _i64, _i64, _i64, _p, _p, _p]),
    "oracle_sample_recent": (None, [_p, _i64, _p, _p, _p, _p, _p, _i64, _i32, _p, _p, _p, _p]),
    "oracle_access_count": (None, [_p, _p, _i64, _i64, _p]),
    "oracle_greedy_hot_set": (None, [_p, _i64, _p, _i64, _f64, _p, _p, _p, _p]),
    "oracle_time_encode_bwd": (None, [_p, _i64, _p, _p, _p, _p, _i32, _p, _p, _p]),
    "oracle_edge_softmax_fwd": (None, [_p, _i64, _i32, _i32, _p, _p, _f64, _f64, _p, _p, _p]),
    "oracle_aggregate_fwd": (None, [_p, _i64, _i32, _i32, _p, _p, _p]),
    "oracle_aggregate_bwd": (None, [_p, _i64, _i32, _i32, _p, _p, _p, _p, _p]),
    "oracle_edge_softmax_bwd": (None, [_p, _i64, _i32, _i32, _p, _p, _f64, _f64, _p, _p, _p, _p, _p]),
}


def lib():
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB_PATH):
            from . import build as _b
            _b.build()
        L = C.CDLL(_LIB_PATH)
        for name, (res, args) in _SIGS.items():
            f = getattr(L, name)
            f.restype = res
            f.argtypes = args
        _lib = L
    return _lib


def _ptr(a):
    return None if a is None else a.ctypes.data


def _c(a, dtype):
    return np.ascontiguousarray(a, dtype=dtype)


def _f64(a):
    """Exact widening of an fp32/bf16 (torch or numpy) operand to float64."""
    try:
        import torch
        if isinstance(a, torch.Tensor):
            return a.detach().to("cpu", torch.float64).contiguous().numpy()
    except ImportError:  # pragma: no cover
        pass
    return np.ascontiguousarray(a, dtype=np.float64)


# ------------------------------------------------------------------ integer ops
def csr_offsets(counts):
    counts = _c(counts, np.int32)
    off = np.empty(counts.shape[0] + 1, dtype=np.int32)
    lib().oracle_csr_offsets(_ptr(counts), counts.shape[0], _ptr(off))
    return off


def check_tcsr(off, E, src_ids=None, src_bound=0, edge_ids=None, edge_bound=0,
               edge_t=None, dst_t=None):
    off = _c(off, np.int32)
    c = lambda a, t: None if a is None else _c(a, t)
    src_ids, edge_ids = c(src_ids, np.int64), c(edge_ids, np.int64)
    edge_t, dst_t = c(edge_t, np.float32), c(dst_t, np.float32)
    v = np.zeros(5, dtype=np.int64)
    lib().oracle_check_tcsr(_ptr(off), off.shape[0] - 1, E, _ptr(src_ids), src_bound,
                            _ptr(edge_ids), edge_bound, _ptr(edge_t), _ptr(dst_t), _ptr(v))
    return v


def dedup(ids):
    ids = _c(ids, np.int64)
    n = ids.shape[0]
    uni = np.empty(max(n, 1), dtype=np.int64)
    inv = np.empty(max(n, 1), dtype=np.int32)
    u = lib().oracle_dedup(_ptr(ids), n, _ptr(uni), _ptr(inv))
    return uni[:u].copy(), inv[:n].copy()


def gather(uni, table, slot_map=None):
    """Returns (rows [u, row] same dtype as table, hit mask [u], miss int32 [m])."""
    uni = _c(uni, np.int64)
    table = np.ascontiguousarray(table)
    u = uni.shape[0]
    row_shape = table.shape[1:]
    row_bytes = table.dtype.itemsize * int(np.prod(row_shape, dtype=np.int64))
    rows = np.zeros((u,) + row_shape, dtype=table.dtype)
    miss = np.empty(max(u, 1), dtype=np.int32)
    sm = None if slot_map is None else _c(slot_map, np.int32)
    nm = lib().oracle_gather(_ptr(uni), u, _ptr(table), table.shape[0], row_bytes,
                             _ptr(sm), _ptr(rows), _ptr(miss))
    miss = miss[:nm].copy()
    hit = np.ones(u, dtype=bool)
    hit[miss] = False
    return rows, hit, miss


# ------------------------------------------------------------------ indexed operands
def occurrence_csr(index, num_rows):
    """(occ_off int32 [num_rows+1], occ int32 [valid positions]) of an index."""
    index = _c(index, np.int32)
    n = index.shape[0]
    off = np.empty(num_rows + 1, dtype=np.int32)
    occ = np.empty(2 * n + 1, dtype=np.int32)     # slack: a planted mistake may overrun n
    lib().oracle_occurrence_csr(_ptr(index), n, num_rows, _ptr(off), _ptr(occ))
    return off, occ[:int(off[-1])].copy()


def index_add_rows(index, num_rows, src):
    """dst [num_rows, ...] float64 = sum of the rows of src at the positions of each index value."""
    index = _c(index, np.int32)
    src = _f64(src)
    row_shape = src.shape[1:]
    D = int(np.prod(row_shape, dtype=np.int64))
    dst = np.zeros((num_rows,) + row_shape, dtype=np.float64)
    lib().oracle_index_add_rows(_ptr(index), index.shape[0], num_rows, D,
                                _ptr(np.ascontiguousarray(src.reshape(index.shape[0], D))), _ptr(dst))
    return dst


def index_add_scaled_rows(index, off, num_rows, scal, src):
    """dst [num_rows, H, dh] float64: for every edge e (segment v by off) with
    index[e] == u, add scal[e, h] * src[v, h, :] to row u."""
    index, off = _c(index, np.int32), _c(off, np.int32)
    scal, src = _f64(scal), _f64(src)
    N, H, dh = src.shape
    assert scal.shape == (index.shape[0], H) and off.shape[0] == N + 1
    dst = np.zeros((num_rows, H, dh), dtype=np.float64)
    lib().oracle_index_add_scaled_rows(_ptr(index), _ptr(off), N, num_rows, H, dh, _ptr(scal),
                                       _ptr(src), _ptr(dst))
    return dst


def edge_attention_bwd_scalars(off, Q, K, V, dO, scale, slope):
    """(dQ, g [E,H], alpha [E,H]): the backward written with its per-edge
    coefficients, dK[e,h,:] = g[e,h] * Q[v,h,:] and dV[e,h,:] = alpha[e,h] *
    dO[v,h,:] for edge e of segment v.  From the softmax and aggregation
    definitions (Sec. 4.3): dalpha = <dO[v,h], V[e,h]>, D = sum over the
    segment of alpha * dalpha, g = alpha (dalpha - D) LReLU'(pre) scale."""
    off = _c(off, np.int32)
    alpha, _, pre = edge_softmax_fwd(off, Q, K, scale, slope)
    dalpha, _ = aggregate_bwd(off, alpha, V, dO)
    seg = np.repeat(np.arange(off.shape[0] - 1), np.diff(off))
    D = np.zeros((off.shape[0] - 1, alpha.shape[1]))
    np.add.at(D, seg, alpha * dalpha)
    g = alpha * (dalpha - D[seg]) * np.where(pre > 0, 1.0, slope) * scale
    dQ, _ = edge_softmax_bwd(off, Q, K, scale, slope, alpha, dalpha)
    return dQ, g, alpha


def edge_attention_fwd_indexed(off, Q, K, k_index, V, v_index, scale, slope):
    """Fused forward whose edge e reads row k_index[e] of K and v_index[e] of V
    (None = row e): the plain operator on the gathered rows."""
    K, V = _f64(K), _f64(V)
    Ke = K if k_index is None else K[np.asarray(k_index, np.int64)]
    Ve = V if v_index is None else V[np.asarray(v_index, np.int64)]
    return edge_attention_fwd(off, Q, Ke, Ve, scale, slope)


def edge_attention_bwd_indexed(off, Q, K, k_index, V, v_index, dO, scale, slope):
    """(dQ, dK_edge, dV_edge, dK_rows, dV_rows): the per-edge gradients of the
    gathered operator, and their sums over the edges that read each row."""
    K, V = _f64(K), _f64(V)
    Ke = K if k_index is None else K[np.asarray(k_index, np.int64)]
    Ve = V if v_index is None else V[np.asarray(v_index, np.int64)]
    dQ, dKe, dVe = edge_attention_bwd(off, Q, Ke, Ve, dO, scale, slope)
    dKr = dKe if k_index is None else index_add_rows(k_index, K.shape[0], dKe)
    dVr = dVe if v_index is None else index_add_rows(v_index, V.shape[0], dVe)
    return dQ, dKe, dVe, dKr, dVr


# ------------------------------------------------------------------ temporal sampling
def sample_recent(indptr, nbr, ts, eid, roots, root_t, k):
    """Most-recent-k sampling: (off int32 [R+1], src int64, edge_t float32, edge_id int64)."""
    indptr, nbr, eid = _c(indptr, np.int64), _c(nbr, np.int64), _c(eid, np.int64)
    ts, roots, root_t = _c(ts, np.float32), _c(roots, np.int64), _c(root_t, np.float32)
    R = roots.shape[0]
    valid = roots[(roots >= 0) & (roots < indptr.shape[0] - 1)]
    # room for every entry of every root, more than R * k when degrees are large
    cap = max(R * k, int((indptr[valid + 1] - indptr[valid]).sum()), 1)
    off = np.empty(R + 1, dtype=np.int32)
    src = np.empty(cap, dtype=np.int64)
    et = np.empty(cap, dtype=np.float32)
    ei = np.empty(cap, dtype=np.int64)
    lib().oracle_sample_recent(_ptr(indptr), indptr.shape[0] - 1, _ptr(nbr), _ptr(ts), _ptr(eid),
                               _ptr(roots), _ptr(root_t), R, k, _ptr(off), _ptr(src), _ptr(et),
                               _ptr(ei))
    E = int(off[-1])
    return off, src[:E].copy(), et[:E].copy(), ei[:E].copy()


# ------------------------------------------------------------------ greedy cache selection
def access_count(batches, id_bound, freq=None):
    """Alg. 1 counting over a list of id arrays (one per pre-sampled batch):
    freq[x] = number of batches containing x (added to `freq` if given)."""
    sizes = [len(b) for b in batches]
    ids = _c(np.concatenate([np.asarray(b, dtype=np.int64) for b in batches])
             if batches else np.zeros(0), np.int64)
    off = np.concatenate([[0], np.cumsum(sizes)]).astype(np.int64)
    out = np.zeros(id_bound, dtype=np.int32) if freq is None else _c(freq, np.int32).copy()
    lib().oracle_access_count(_ptr(ids), _ptr(off), len(batches), id_bound, _ptr(out))
    return out


def greedy_hot_set(fv, fe, alpha):
    """Alg. 1 selection: (hot node ids, hot edge ids), each in selection order."""
    fv, fe = _c(fv, np.int32), _c(fe, np.int32)
    nv, ne = fv.shape[0], fe.shape[0]
    hv = np.empty(max(nv, 1), dtype=np.int64)
    he = np.empty(max(ne, 1), dtype=np.int64)
    cv, ce = C.c_int64(0), C.c_int64(0)
    lib().oracle_greedy_hot_set(_ptr(fv), nv, _ptr(fe), ne, float(alpha), _ptr(hv),
                                C.byref(cv), _ptr(he), C.byref(ce))
    return hv[:cv.value].copy(), he[:ce.value].copy()


# ------------------------------------------------------------------ time encoding
def time_encode(off, t_dst, t_e, omega, phi):
    off = _c(off, np.int32)
    t_dst, t_e = _c(t_dst, np.float32), _c(t_e, np.float32)
    omega, phi = _c(omega, np.float32), _c(phi, np.float32)
    N, E, d_t = off.shape[0] - 1, t_e.shape[0], omega.shape[0]
    te = np.zeros((E, d_t), dtype=np.float64)
    lib().oracle_time_encode(_ptr(off), N, _ptr(t_dst), _ptr(t_e), _ptr(omega),
                             _ptr(phi), d_t, _ptr(te))
    return te


def time_encode_bwd(off, t_dst, t_e, omega, phi, dte):
    """Returns (domega [d_t], dphi [d_t]) in float64 for the upstream gradient dte [E, d_t]."""
    off = _c(off, np.int32)
    t_dst, t_e = _c(t_dst, np.float32), _c(t_e, np.float32)
    omega, phi = _c(omega, np.float32), _c(phi, np.float32)
    dte = _f64(dte)
    N, d_t = off.shape[0] - 1, omega.shape[0]
    assert dte.shape == (t_e.shape[0], d_t)
    domega = np.zeros(d_t, dtype=np.float64)
    dphi = np.zeros(d_t, dtype=np.float64)
    lib().oracle_time_encode_bwd(_ptr(off), N, _ptr(t_dst), _ptr(t_e), _ptr(omega), _ptr(phi),
                                 d_t, _ptr(dte), _ptr(domega), _ptr(dphi))
    return domega, dphi


# ------------------------------------------------------------------ attention
def edge_softmax_fwd(off, Q, K, scale, slope):
    """Returns (alpha [E,H], lse [N,H], pre [E,H])."""
    off = _c(off, np.int32)
    Q, K = _f64(Q), _f64(K)
    N, H, dh = Q.shape
    E = K.shape[0]
    alpha = np.zeros((E, H))
    lse = np.zeros((N, H))
    pre = np.zeros((E, H))
    lib().oracle_edge_softmax_fwd(_ptr(off), N, H, dh, _ptr(Q), _ptr(K), scale, slope,
                                  _ptr(pre), _ptr(alpha), _ptr(lse))
    return alpha, lse, pre


def aggregate_fwd(off, alpha, V):
    off = _c(off, np.int32)
    alpha, V = _f64(alpha), _f64(V)
    E, H, dh = V.shape
    N = off.shape[0] - 1
    out = np.zeros((N, H, dh))
    lib().oracle_aggregate_fwd(_ptr(off), N, H, dh, _ptr(alpha), _ptr(V), _ptr(out))
    return out


def aggregate_bwd(off, alpha, V, dout):
    off = _c(off, np.int32)
    alpha, V, dout = _f64(alpha), _f64(V), _f64(dout)
    E, H, dh = V.shape
    N = off.shape[0] - 1
    dalpha = np.zeros((E, H))
    dV = np.zeros((E, H, dh))
    lib().oracle_aggregate_bwd(_ptr(off), N, H, dh, _ptr(alpha), _ptr(V), _ptr(dout),
                               _ptr(dalpha), _ptr(dV))
    return dalpha, dV


def edge_softmax_bwd(off, Q, K, scale, slope, alpha, dalpha, branch=None):
    off = _c(off, np.int32)
    Q, K, alpha, dalpha = _f64(Q), _f64(K), _f64(alpha), _f64(dalpha)
    N, H, dh = Q.shape
    E = K.shape[0]
    dQ = np.zeros((N, H, dh))
    dK = np.zeros((E, H, dh))
    br = None if branch is None else _c(branch, np.int8)
    lib().oracle_edge_softmax_bwd(_ptr(off), N, H, dh, _ptr(Q), _ptr(K), scale, slope,
                                  _ptr(alpha), _ptr(dalpha), _ptr(br), _ptr(dQ), _ptr(dK))
    return dQ, dK


def edge_attention_fwd(off, Q, K, V, scale, slope):
    """Fused operator = edge softmax then aggregation.  Returns (out, lse, alpha, pre)."""
    alpha, lse, pre = edge_softmax_fwd(off, Q, K, scale, slope)
    out = aggregate_fwd(off, alpha, V)
    return out, lse, alpha, pre


def edge_attention_bwd(off, Q, K, V, dout, scale, slope, branch=None):
    """Backward of the fused operator = aggregation backward then edge-softmax
    backward.  Returns (dQ, dK, dV)."""
    alpha, _, _ = edge_softmax_fwd(off, Q, K, scale, slope)
    dalpha, dV = aggregate_bwd(off, alpha, V, dout)
    dQ, dK = edge_softmax_bwd(off, Q, K, scale, slope, alpha, dalpha, branch)
    return dQ, dK, dV
