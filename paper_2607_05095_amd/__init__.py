"""Thin Python binding of libfast.so, the gfx950 temporal-subgraph operators.

Every function has the name and argument order of the C entry point in
include/fast.h.  Arguments are torch tensors resident on the GPU (or None
for optional pointers); the binding only marshals pointers, sizes and the
current HIP stream, and raises FastError for a non-OK status.  All
computation happens in the HIP kernels; there is no fallback path: if the
library is missing the first call raises.
"""
from __future__ import annotations

import ctypes as C
import os

__all__ = [
    "FastError", "lib", "TCSR", "tcsr", "TemporalGraphDesc", "temporal_graph", "F32", "BF16",
    "dtype_of", "fast_sample_recent_workspace", "fast_sample_recent",
    "fast_version", "fast_last_error",
    "fast_csr_offsets_workspace", "fast_csr_offsets", "fast_check_tcsr",
    "fast_csr_offsets_batched_workspace", "fast_csr_offsets_batched", "fast_time_encode_batched",
    "fast_dedup_gather_workspace", "fast_dedup_gather", "fast_dedup_gather_noalloc",
    "NOALLOC_SCRATCH_BYTES",
    "fast_access_count_workspace", "fast_access_count",
    "fast_greedy_hot_set_workspace", "fast_greedy_hot_set", "fast_hot_set_budget",
    "fast_time_encode", "fast_time_encode_bwd_workspace", "fast_time_encode_bwd",
    "fast_edge_softmax_fwd", "fast_edge_softmax_bwd",
    "fast_temporal_aggregate_fwd", "fast_temporal_aggregate_bwd",
    "fast_edge_attention_fwd", "fast_edge_attention_bwd",
    "fast_edge_attention_fwd_packed", "fast_edge_attention_bwd_packed",
    "fast_edge_attention_fwd_indexed", "fast_edge_attention_bwd_indexed",
    "fast_occurrence_csr_workspace", "fast_occurrence_csr",
    "fast_index_add_rows_workspace", "fast_index_add_rows",
    "fast_edge_attention_bwd_indexed_coef",
    "fast_index_add_scaled_rows_workspace", "fast_index_add_scaled_rows",
]

_HERE = os.path.dirname(os.path.abspath(__file__))
# the in-tree build; FAST_LIB names another build of the same sources (the
# sanitizer build of the host code)
LIB_PATH = os.environ.get("FAST_LIB") or os.path.join(_HERE, "libfast.so")

F32, BF16 = 0, 1
NOALLOC_SCRATCH_BYTES = 128 << 20   # FAST_NOALLOC_SCRATCH_BYTES of include/fast.h
_STATUS = {0: "FAST_OK", 1: "FAST_ERR_INVALID_ARG", 2: "FAST_ERR_UNSUPPORTED",
           3: "FAST_ERR_WORKSPACE", 4: "FAST_ERR_HIP"}


class FastError(RuntimeError):
    def __init__(self, status: int, msg: str):
        super().__init__(f"{_STATUS.get(status, status)}: {msg}")
        self.status = status


class TCSR(C.Structure):
    """fast_tcsr_t: a sampled temporal subgraph of one layer block (device pointers)."""
    _fields_ = [
        ("num_dst", C.c_int64),
        ("num_edges", C.c_int64),
        ("dst_offsets", C.c_void_p),
        ("src_ids", C.c_void_p),
        ("edge_t", C.c_void_p),
        ("edge_ids", C.c_void_p),
        ("dst_t", C.c_void_p),
    ]


class TemporalGraphDesc(C.Structure):
    """fast_temporal_graph_t: a T-CSR temporal graph (device pointers)."""
    _fields_ = [
        ("num_nodes", C.c_int64),
        ("num_entries", C.c_int64),
        ("indptr", C.c_void_p),
        ("nbr", C.c_void_p),
        ("ts", C.c_void_p),
        ("eid", C.c_void_p),
    ]


_p, _i64, _i32, _f32, _sz = C.c_void_p, C.c_int64, C.c_int, C.c_float, C.c_size_t
_G = C.POINTER(TCSR)
_TG = C.POINTER(TemporalGraphDesc)
_SIGS = {
    "fast_last_error": (C.c_char_p, []),
    "fast_version": (C.c_char_p, []),
    "fast_csr_offsets_workspace": (_sz, [_i64]),
    "fast_csr_offsets": (_i32, [_p, _i64, _p, _p, _sz, _p]),
    "fast_csr_offsets_batched_workspace": (_sz, [_i32, _p]),
    "fast_csr_offsets_batched": (_i32, [_i32, _p, _p, _p, _p, _sz, _p]),
    "fast_time_encode_batched": (_i32, [_i32, _p, _p, _p, _i32, _p, _i32, _p]),
    "fast_check_tcsr": (_i32, [_G, _i64, _i64, _p, _p]),
    "fast_dedup_gather_workspace": (_sz, [_i64, _i64]),
    "fast_dedup_gather": (_i32, [_p, _i64, _i64, _p, _i64, _i32, _i32, _p, _p, _p, _p,
                                 _p, _p, _p, _p, _sz, _p]),
    "fast_dedup_gather_noalloc": (_i32, [_p, _i64, _i64, _p, _i64, _i32, _i32, _p, _p, _p, _p,
                                         _p, _p, _p, _p]),
    "fast_sample_recent_workspace": (_sz, [_i64]),
    "fast_sample_recent": (_i32, [_TG, _p, _p, _i64, _i32, _p, _p, _p, _p, _p, _sz, _p]),
    "fast_access_count_workspace": (_sz, [_i64]),
    "fast_access_count": (_i32, [_p, _p, _i64, _i64, _p, _p, _sz, _p]),
    "fast_greedy_hot_set_workspace": (_sz, [_i64, _i64, _i32]),
    "fast_hot_set_budget": (_i32, [C.c_double, _i64, _i64, _p]),
    "fast_greedy_hot_set": (_i32, [_p, _i64, _p, _i64, _i32, _i64, _p, _p, _p, _p, _p, _p, _p,
                                   _sz, _p]),
    "fast_time_encode": (_i32, [_G, _p, _p, _i32, _p, _i32, _p]),
    "fast_time_encode_bwd_workspace": (_sz, [_i64, _i32]),
    "fast_time_encode_bwd": (_i32, [_G, _p, _p, _i32, _p, _i32, _p, _p, _p, _sz, _p]),
    "fast_edge_softmax_fwd": (_i32, [_G, _i32, _i32, _i32, _p, _p, _f32, _f32, _p, _p, _p]),
    "fast_edge_softmax_bwd": (_i32, [_G, _i32, _i32, _i32, _p, _p, _f32, _f32, _p, _p, _p, _p, _p]),
    "fast_temporal_aggregate_fwd": (_i32, [_G, _i32, _i32, _i32, _p, _p, _p, _p]),
    "fast_temporal_aggregate_bwd": (_i32, [_G, _i32, _i32, _i32, _p, _p, _p, _p, _p, _p]),
    "fast_edge_attention_fwd": (_i32, [_G, _i32, _i32, _i32, _p, _p, _p, _f32, _f32, _p, _p, _p]),
    "fast_edge_attention_bwd": (_i32, [_G, _i32, _i32, _i32, _p, _p, _p, _f32, _f32, _p, _p,
                                       _p, _p, _p, _p]),
    "fast_edge_attention_fwd_packed": (_i32, [_G, _i32, _i32, _i32, _p, _p, _f32, _f32, _p, _p, _p]),
    "fast_edge_attention_bwd_packed": (_i32, [_G, _i32, _i32, _i32, _p, _p, _f32, _f32, _p, _p, _p,
                                              _p, _p]),
    "fast_edge_attention_fwd_indexed": (_i32, [_G, _i32, _i32, _i32, _p, _p, _p, _i64, _p, _p,
                                               _i64, _f32, _f32, _p, _p, _p]),
    "fast_edge_attention_bwd_indexed": (_i32, [_G, _i32, _i32, _i32, _p, _p, _p, _i64, _p, _p,
                                               _i64, _f32, _f32, _p, _p, _p, _p, _p, _p]),
    "fast_occurrence_csr_workspace": (_sz, [_i64, _i64]),
    "fast_occurrence_csr": (_i32, [_p, _i64, _i64, _p, _p, _p, _sz, _p]),
    "fast_index_add_rows_workspace": (_sz, [_i64, _i64, _i32]),
    "fast_index_add_rows": (_i32, [_p, _p, _i64, _i64, _i32, _i32, _p, _p, _p, _sz, _p]),
    "fast_edge_attention_bwd_indexed_coef": (_i32, [_G, _i32, _i32, _i32, _p, _p, _p, _i64, _p, _p,
                                                    _i64, _f32, _f32, _p, _p, _p, _p, _p, _p]),
    "fast_index_add_scaled_rows_workspace": (_sz, [_i64, _i64, _i32, _i32]),
    "fast_index_add_scaled_rows": (_i32, [_p, _p, _i64, _i64, _p, _i64, _i32, _i32, _i32, _p, _p,
                                          _p, _p, _sz, _p]),
}

_lib = None


def lib():
    """Load libfast.so (built in-tree by build.py); raises if it is absent."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise FastError(-1, f"{LIB_PATH} is not built; run python -m paper_2607_05095_amd.build")
        L = C.CDLL(LIB_PATH)
        for name, (res, args) in _SIGS.items():
            f = getattr(L, name)
            f.restype = res
            f.argtypes = args
        _lib = L
    return _lib


def _ptr(t):
    if t is None:
        return None
    if isinstance(t, int):
        return t
    return t.data_ptr()


def _stream(stream):
    if stream is not None:
        return stream if isinstance(stream, int) else stream.cuda_stream
    import torch
    return torch.cuda.current_stream().cuda_stream


def _check(st: int):
    if st != 0:
        raise FastError(st, fast_last_error())


def dtype_of(t) -> int:
    import torch
    if t.dtype == torch.float32:
        return F32
    if t.dtype == torch.bfloat16:
        return BF16
    raise FastError(2, f"unsupported tensor dtype {t.dtype}")


def tcsr(dst_offsets, num_edges: int, src_ids=None, edge_t=None, edge_ids=None, dst_t=None) -> TCSR:
    """Builds a fast_tcsr_t over device tensors.  The struct keeps a reference
    to each tensor, so a temporary passed here (`x.cuda()`) is not returned to
    torch's caching allocator, and reused, while the struct is alive."""
    g = TCSR(dst_offsets.shape[0] - 1, int(num_edges), _ptr(dst_offsets), _ptr(src_ids),
             _ptr(edge_t), _ptr(edge_ids), _ptr(dst_t))
    g._keep = tuple(t for t in (dst_offsets, src_ids, edge_t, edge_ids, dst_t)
                    if t is not None and not isinstance(t, int))
    return g


def temporal_graph(indptr, nbr, ts, eid) -> TemporalGraphDesc:
    """Builds a fast_temporal_graph_t over device tensors; the struct keeps a
    reference to each tensor while it is alive."""
    g = TemporalGraphDesc(indptr.shape[0] - 1, int(nbr.shape[0]), _ptr(indptr), _ptr(nbr),
                          _ptr(ts), _ptr(eid))
    g._keep = (indptr, nbr, ts, eid)
    return g


# ------------------------------------------------------------------ entry points
def fast_last_error() -> str:
    return lib().fast_last_error().decode()


def fast_version() -> str:
    return lib().fast_version().decode()


def fast_csr_offsets_workspace(n: int) -> int:
    return lib().fast_csr_offsets_workspace(n)


def fast_csr_offsets(counts, n, offsets, ws, ws_bytes, stream=None):
    _check(lib().fast_csr_offsets(_ptr(counts), n, _ptr(offsets), _ptr(ws), ws_bytes,
                                  _stream(stream)))


def _host_ptrs(xs):
    """A host array of device pointers (None for a NULL entry)."""
    return (C.c_void_p * max(len(xs), 1))(*[_ptr(x) for x in xs])


def _host_i64(xs):
    return (C.c_int64 * max(len(xs), 1))(*[int(x) for x in xs])


def fast_csr_offsets_batched_workspace(n) -> int:
    return lib().fast_csr_offsets_batched_workspace(len(n), _host_i64(n))


def fast_csr_offsets_batched(counts, n, offsets, ws, ws_bytes, stream=None):
    """counts, n, offsets: sequences of equal length (one entry per block)."""
    if not (len(counts) == len(n) == len(offsets)):
        raise ValueError("counts, n and offsets must have one entry per block")
    _check(lib().fast_csr_offsets_batched(len(n), _host_ptrs(counts), _host_i64(n),
                                          _host_ptrs(offsets), _ptr(ws), ws_bytes,
                                          _stream(stream)))


def fast_time_encode_batched(graphs, omega, phi, d_t, te, te_dtype, stream=None):
    """graphs: TCSR descriptors, te: outputs, one per block."""
    if len(graphs) != len(te):
        raise ValueError("graphs and te must have one entry per block")
    gs = (C.POINTER(TCSR) * max(len(graphs), 1))(*[C.pointer(g) for g in graphs])
    _check(lib().fast_time_encode_batched(len(graphs), gs, _ptr(omega), _ptr(phi), d_t,
                                          _host_ptrs(te), te_dtype, _stream(stream)))


def fast_check_tcsr(g: TCSR, src_bound, edge_bound, violations, stream=None):
    _check(lib().fast_check_tcsr(C.byref(g), src_bound, edge_bound, _ptr(violations),
                                 _stream(stream)))


def fast_dedup_gather_workspace(n: int, id_bound: int) -> int:
    return lib().fast_dedup_gather_workspace(n, id_bound)


def fast_dedup_gather(ids, n, id_bound, table, table_rows, D, dtype, slot_map, uni, inv,
                      num_unique, rows, miss, num_miss, ws, ws_bytes, stream=None):
    _check(lib().fast_dedup_gather(_ptr(ids), n, id_bound, _ptr(table), table_rows, D, dtype,
                                   _ptr(slot_map), _ptr(uni), _ptr(inv), _ptr(num_unique),
                                   _ptr(rows), _ptr(miss), _ptr(num_miss), _ptr(ws), ws_bytes,
                                   _stream(stream)))


def fast_dedup_gather_noalloc(ids, n, id_bound, table, table_rows, D, dtype, slot_map, uni, inv,
                              num_unique, rows, miss, num_miss, stream=None):
    _check(lib().fast_dedup_gather_noalloc(_ptr(ids), n, id_bound, _ptr(table), table_rows, D,
                                           dtype, _ptr(slot_map), _ptr(uni), _ptr(inv),
                                           _ptr(num_unique), _ptr(rows), _ptr(miss),
                                           _ptr(num_miss), _stream(stream)))


def fast_sample_recent_workspace(num_roots: int) -> int:
    return lib().fast_sample_recent_workspace(num_roots)


def fast_sample_recent(g: TemporalGraphDesc, roots, root_t, num_roots, k, dst_offsets, src_ids,
                       edge_t, edge_ids, ws, ws_bytes, stream=None):
    _check(lib().fast_sample_recent(C.byref(g), _ptr(roots), _ptr(root_t), num_roots, k,
                                    _ptr(dst_offsets), _ptr(src_ids), _ptr(edge_t),
                                    _ptr(edge_ids), _ptr(ws), ws_bytes, _stream(stream)))


def fast_access_count_workspace(id_bound: int) -> int:
    return lib().fast_access_count_workspace(id_bound)


def fast_access_count(ids, batch_offsets, num_batches, id_bound, freq, ws, ws_bytes, stream=None):
    """batch_offsets: a host sequence of num_batches + 1 int64 offsets into ids."""
    offs = (C.c_int64 * (num_batches + 1))(*[int(x) for x in batch_offsets])
    _check(lib().fast_access_count(_ptr(ids), C.cast(offs, C.c_void_p), num_batches, id_bound,
                                   _ptr(freq), _ptr(ws), ws_bytes, _stream(stream)))


def fast_greedy_hot_set_workspace(num_nodes: int, num_edges: int, max_freq: int) -> int:
    return lib().fast_greedy_hot_set_workspace(num_nodes, num_edges, max_freq)


def fast_greedy_hot_set(freq_v, num_nodes, freq_e, num_edges, max_freq, budget, hot_v, num_hot_v,
                        slot_v, hot_e, num_hot_e, slot_e, ws, ws_bytes, stream=None):
    _check(lib().fast_greedy_hot_set(_ptr(freq_v), num_nodes, _ptr(freq_e), num_edges, max_freq,
                                     budget, _ptr(hot_v), _ptr(num_hot_v), _ptr(slot_v),
                                     _ptr(hot_e), _ptr(num_hot_e), _ptr(slot_e), _ptr(ws),
                                     ws_bytes, _stream(stream)))


def fast_hot_set_budget(alpha: float, num_nodes: int, num_edges: int) -> int:
    """Returns the budget the library computes (a host call)."""
    out = C.c_int64(0)
    _check(lib().fast_hot_set_budget(float(alpha), num_nodes, num_edges, C.byref(out)))
    return out.value


def fast_time_encode(g: TCSR, omega, phi, d_t, te, te_dtype, stream=None):
    _check(lib().fast_time_encode(C.byref(g), _ptr(omega), _ptr(phi), d_t, _ptr(te), te_dtype,
                                  _stream(stream)))


def fast_time_encode_bwd_workspace(num_dst: int, d_t: int) -> int:
    return lib().fast_time_encode_bwd_workspace(num_dst, d_t)


def fast_time_encode_bwd(g: TCSR, omega, phi, d_t, dte, dte_dtype, domega, dphi, ws, ws_bytes,
                         stream=None):
    _check(lib().fast_time_encode_bwd(C.byref(g), _ptr(omega), _ptr(phi), d_t, _ptr(dte),
                                      dte_dtype, _ptr(domega), _ptr(dphi), _ptr(ws), ws_bytes,
                                      _stream(stream)))


def fast_edge_softmax_fwd(g: TCSR, H, dh, dtype, Q, K, scale, neg_slope, alpha, lse, stream=None):
    _check(lib().fast_edge_softmax_fwd(C.byref(g), H, dh, dtype, _ptr(Q), _ptr(K), scale,
                                       neg_slope, _ptr(alpha), _ptr(lse), _stream(stream)))


def fast_edge_softmax_bwd(g: TCSR, H, dh, dtype, Q, K, scale, neg_slope, alpha, dalpha, dQ, dK,
                          stream=None):
    _check(lib().fast_edge_softmax_bwd(C.byref(g), H, dh, dtype, _ptr(Q), _ptr(K), scale,
                                       neg_slope, _ptr(alpha), _ptr(dalpha), _ptr(dQ), _ptr(dK),
                                       _stream(stream)))


def fast_temporal_aggregate_fwd(g: TCSR, H, dh, dtype, alpha, V, out, stream=None):
    _check(lib().fast_temporal_aggregate_fwd(C.byref(g), H, dh, dtype, _ptr(alpha), _ptr(V),
                                             _ptr(out), _stream(stream)))


def fast_temporal_aggregate_bwd(g: TCSR, H, dh, dtype, alpha, V, dout, dalpha, dV, stream=None):
    _check(lib().fast_temporal_aggregate_bwd(C.byref(g), H, dh, dtype, _ptr(alpha), _ptr(V),
                                             _ptr(dout), _ptr(dalpha), _ptr(dV), _stream(stream)))


def fast_edge_attention_fwd(g: TCSR, H, dh, dtype, Q, K, V, scale, neg_slope, out, lse,
                            stream=None):
    _check(lib().fast_edge_attention_fwd(C.byref(g), H, dh, dtype, _ptr(Q), _ptr(K), _ptr(V),
                                         scale, neg_slope, _ptr(out), _ptr(lse), _stream(stream)))


def fast_edge_attention_bwd(g: TCSR, H, dh, dtype, Q, K, V, scale, neg_slope, lse, dout, dQ, dK,
                            dV, stream=None):
    _check(lib().fast_edge_attention_bwd(C.byref(g), H, dh, dtype, _ptr(Q), _ptr(K), _ptr(V),
                                         scale, neg_slope, _ptr(lse), _ptr(dout), _ptr(dQ),
                                         _ptr(dK), _ptr(dV), _stream(stream)))


def fast_edge_attention_fwd_packed(g: TCSR, H, dh, dtype, Q, KV, scale, neg_slope, out, lse,
                                   stream=None):
    _check(lib().fast_edge_attention_fwd_packed(C.byref(g), H, dh, dtype, _ptr(Q), _ptr(KV),
                                                scale, neg_slope, _ptr(out), _ptr(lse),
                                                _stream(stream)))


def fast_edge_attention_bwd_packed(g: TCSR, H, dh, dtype, Q, KV, scale, neg_slope, lse, dout, dQ,
                                   dKV, stream=None):
    _check(lib().fast_edge_attention_bwd_packed(C.byref(g), H, dh, dtype, _ptr(Q), _ptr(KV),
                                                scale, neg_slope, _ptr(lse), _ptr(dout),
                                                _ptr(dQ), _ptr(dKV), _stream(stream)))


def fast_edge_attention_fwd_indexed(g: TCSR, H, dh, dtype, Q, K, k_index, k_rows, V, v_index,
                                    v_rows, scale, neg_slope, out, lse, stream=None):
    _check(lib().fast_edge_attention_fwd_indexed(C.byref(g), H, dh, dtype, _ptr(Q), _ptr(K),
                                                 _ptr(k_index), k_rows, _ptr(V), _ptr(v_index),
                                                 v_rows, scale, neg_slope, _ptr(out), _ptr(lse),
                                                 _stream(stream)))


def fast_edge_attention_bwd_indexed(g: TCSR, H, dh, dtype, Q, K, k_index, k_rows, V, v_index,
                                    v_rows, scale, neg_slope, lse, dout, dQ, dK_edge, dV_edge,
                                    stream=None):
    _check(lib().fast_edge_attention_bwd_indexed(C.byref(g), H, dh, dtype, _ptr(Q), _ptr(K),
                                                 _ptr(k_index), k_rows, _ptr(V), _ptr(v_index),
                                                 v_rows, scale, neg_slope, _ptr(lse), _ptr(dout),
                                                 _ptr(dQ), _ptr(dK_edge), _ptr(dV_edge),
                                                 _stream(stream)))


def fast_occurrence_csr_workspace(n: int, num_rows: int) -> int:
    return lib().fast_occurrence_csr_workspace(n, num_rows)


def fast_occurrence_csr(index, n, num_rows, occ_off, occ, ws, ws_bytes, stream=None):
    _check(lib().fast_occurrence_csr(_ptr(index), n, num_rows, _ptr(occ_off), _ptr(occ), _ptr(ws),
                                     ws_bytes, _stream(stream)))


def fast_index_add_rows_workspace(n: int, num_rows: int, D: int) -> int:
    return lib().fast_index_add_rows_workspace(n, num_rows, D)


def fast_index_add_rows(occ_off, occ, n, num_rows, D, src_dtype, src, dst, ws, ws_bytes,
                        stream=None):
    _check(lib().fast_index_add_rows(_ptr(occ_off), _ptr(occ), n, num_rows, D, src_dtype, _ptr(src),
                                     _ptr(dst), _ptr(ws), ws_bytes, _stream(stream)))


def fast_edge_attention_bwd_indexed_coef(g: TCSR, H, dh, dtype, Q, K, k_index, k_rows, V, v_index,
                                         v_rows, scale, neg_slope, lse, dout, dQ, g_edge,
                                         alpha_edge, stream=None):
    _check(lib().fast_edge_attention_bwd_indexed_coef(C.byref(g), H, dh, dtype, _ptr(Q), _ptr(K),
                                                      _ptr(k_index), k_rows, _ptr(V),
                                                      _ptr(v_index), v_rows, scale, neg_slope,
                                                      _ptr(lse), _ptr(dout), _ptr(dQ),
                                                      _ptr(g_edge), _ptr(alpha_edge),
                                                      _stream(stream)))


def fast_index_add_scaled_rows_workspace(n: int, num_rows: int, H: int, dh: int) -> int:
    return lib().fast_index_add_scaled_rows_workspace(n, num_rows, H, dh)


def fast_index_add_scaled_rows(occ_off, occ, n, num_rows, dst_offsets, num_dst, H, dh, src_dtype,
                               scal, src, dst, ws, ws_bytes, stream=None):
    _check(lib().fast_index_add_scaled_rows(_ptr(occ_off), _ptr(occ), n, num_rows,
                                            _ptr(dst_offsets), num_dst, H, dh, src_dtype,
                                            _ptr(scal), _ptr(src), _ptr(dst), _ptr(ws), ws_bytes,
                                            _stream(stream)))
