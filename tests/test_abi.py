"""The C ABI without a GPU: libfast.so loads, exports every function that
include/fast.h declares, and rejects bad arguments on the host (before any
launch) with the documented status codes and a message."""
import ctypes
import os
import re
import subprocess

import pytest

import paper_2607_05095_amd as fast

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "fast.h")

OK, INVALID, UNSUPPORTED, WORKSPACE = 0, 1, 2, 3
FAKE = 0x10000  # a 256-byte aligned stand-in address; never dereferenced on these paths


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(fast_[a-z0-9_]+)\s*\(", text)))


def test_header_declares_the_operator_set():
    names = declared_functions()
    for n in ["fast_csr_offsets", "fast_check_tcsr", "fast_dedup_gather", "fast_time_encode",
              "fast_edge_softmax_fwd", "fast_edge_softmax_bwd",
              "fast_temporal_aggregate_fwd", "fast_temporal_aggregate_bwd",
              "fast_edge_attention_fwd", "fast_edge_attention_bwd", "fast_last_error"]:
        assert n in names


def test_library_exports_every_declared_symbol():
    L = fast.lib()
    missing = [n for n in declared_functions() if not hasattr(L, n)]
    assert not missing, missing
    out = subprocess.run(["nm", "-D", "--defined-only", fast.LIB_PATH], capture_output=True,
                         text=True, check=True).stdout
    exported = set(re.findall(r"\bT (fast_[a-z0-9_]+)\b", out))
    assert set(declared_functions()) <= exported


def test_library_is_built_for_gfx950_only(tmp_path):
    # the device targets bundled in the library's fat binary (its target list only)
    out = subprocess.run(["/opt/rocm/bin/roc-obj-ls", fast.LIB_PATH], capture_output=True, text=True)
    listing = out.stdout if out.returncode == 0 and "gfx" in out.stdout else None
    if listing is None:
        fb = tmp_path / "fatbin"
        dump = subprocess.run(["objcopy", f"--dump-section=.hip_fatbin={fb}", fast.LIB_PATH,
                               str(tmp_path / "lib.copy")], capture_output=True, text=True)
        bundler = "/opt/rocm/llvm/bin/clang-offload-bundler"
        if dump.returncode != 0 or not os.path.exists(bundler):
            pytest.skip("no tool to list the bundled targets")
        listing = subprocess.run([bundler, "--list", "--type=o", f"--input={fb}"], capture_output=True,
                                 text=True, check=True).stdout
    archs = set(re.findall(r"gfx\d+\w*", listing))
    assert archs == {"gfx950"}, archs


def test_version():
    assert "gfx950" in fast.fast_version()


def _g(N=4, E=40, off=FAKE):
    return fast.TCSR(N, E, off, None, FAKE, None, FAKE)


def _attn_fwd(g, H=2, dh=50, dt=0, Q=FAKE, K=FAKE, V=FAKE, out=FAKE, lse=None):
    gp = ctypes.byref(g) if g is not None else None
    return fast.lib().fast_edge_attention_fwd(gp, H, dh, dt, Q, K, V, 1.0, 0.2, out, lse, None)


@pytest.mark.parametrize("kw,status", [
    (dict(g=None), INVALID),
    (dict(g="negN"), INVALID),
    (dict(H=0), INVALID),
    (dict(dh=0), INVALID),
    (dict(dt=7), INVALID),
    (dict(Q=None), INVALID),
    (dict(K=None), INVALID),
    (dict(out=None), INVALID),
    (dict(H=64, dh=128), UNSUPPORTED),        # H*dh > 4096
    (dict(Q=FAKE + 2), UNSUPPORTED),          # fp32 row not 4-byte aligned
    (dict(g="hugeE"), UNSUPPORTED),
    (dict(g="edges_no_dst"), INVALID),
    (dict(g="nullofs"), INVALID),
])
def test_attention_fwd_validation(kw, status):
    g = kw.pop("g", "ok")
    graph = {"ok": _g(), "negN": _g(N=-1), "hugeE": _g(E=1 << 31),
             "edges_no_dst": _g(N=0, E=5), "nullofs": _g(off=None), None: None}[g]
    st = _attn_fwd(graph, **kw)
    assert st == status
    assert fast.fast_last_error() != ""


def test_empty_graph_is_a_no_op_without_launch():
    # N = 0 returns before any HIP call, so it succeeds even with no GPU
    assert _attn_fwd(_g(N=0, E=0), Q=None, K=None, V=None, out=None) == OK
    assert fast.fast_last_error() == ""
    L = fast.lib()
    g = _g(N=0, E=0)
    assert L.fast_time_encode(ctypes.byref(g), FAKE, FAKE, 100, FAKE, 0, None) == OK


def test_other_entry_points_validate():
    L = fast.lib()
    g = _g()
    gp = ctypes.byref(g)
    assert L.fast_edge_attention_bwd(gp, 2, 50, 0, FAKE, FAKE, FAKE, 1.0, 0.2, None, FAKE,
                                     FAKE, None, FAKE, None) == INVALID   # dK NULL
    assert L.fast_edge_softmax_fwd(gp, 2, 50, 0, FAKE, FAKE, 1.0, 0.2, None, None, None) == INVALID
    assert L.fast_edge_softmax_bwd(gp, 2, 50, 0, FAKE, FAKE, 1.0, 0.2, FAKE, None, FAKE, FAKE,
                                   None) == INVALID
    assert L.fast_temporal_aggregate_fwd(gp, 2, 50, 0, None, FAKE, FAKE, None) == INVALID
    assert L.fast_temporal_aggregate_bwd(gp, 2, 50, 0, FAKE, FAKE, FAKE, None, FAKE, None) == INVALID
    assert L.fast_time_encode(gp, FAKE, FAKE, 0, FAKE, 0, None) == INVALID       # d_t = 0
    assert L.fast_time_encode(gp, None, FAKE, 100, FAKE, 0, None) == INVALID     # omega NULL
    assert L.fast_time_encode(gp, FAKE, FAKE, 100, FAKE, 5, None) == INVALID     # dtype
    assert L.fast_csr_offsets(FAKE, -1, FAKE, FAKE, 1 << 20, None) == INVALID
    assert L.fast_csr_offsets(FAKE, 10, FAKE, FAKE, 4, None) == WORKSPACE
    assert L.fast_csr_offsets(FAKE, 10, None, FAKE, 1 << 20, None) == INVALID
    assert L.fast_check_tcsr(None, 0, 0, FAKE, None) == INVALID
    assert L.fast_check_tcsr(gp, 0, 0, None, None) == INVALID              # violations NULL
    assert L.fast_check_tcsr(ctypes.byref(_g(off=None)), 0, 0, FAKE, None) == INVALID
    assert L.fast_check_tcsr(ctypes.byref(_g(N=-1)), 0, 0, FAKE, None) == INVALID
    assert L.fast_check_tcsr(ctypes.byref(_g(E=1 << 31)), 0, 0, FAKE, None) == UNSUPPORTED
    gs = fast.TCSR(4, 40, FAKE, FAKE, None, FAKE, None)
    assert L.fast_check_tcsr(ctypes.byref(gs), -1, 10, FAKE, None) == INVALID  # src_bound
    assert L.fast_check_tcsr(ctypes.byref(gs), 10, -1, FAKE, None) == INVALID  # edge_bound


def test_packed_attention_validation():
    """The packed K|V entry points check their arguments on the host, like
    the separate-array ones, before anything is enqueued."""
    L = fast.lib()
    gp = ctypes.byref(_g())
    fwd = lambda H=2, dh=50, dt=0, Q=FAKE, KV=FAKE, out=FAKE, g=gp: L.fast_edge_attention_fwd_packed(
        g, H, dh, dt, Q, KV, 1.0, 0.2, out, None, None)
    bwd = lambda dt=0, KV=FAKE, dKV=FAKE, dQ=FAKE: L.fast_edge_attention_bwd_packed(
        gp, 2, 50, dt, FAKE, KV, 1.0, 0.2, None, FAKE, dQ, dKV, None)
    assert fwd(KV=None) == INVALID            # edges but no K|V rows
    assert fwd(Q=None) == INVALID
    assert fwd(out=None) == INVALID
    assert fwd(H=0) == INVALID and fwd(dh=0) == INVALID
    assert fwd(dt=5) == INVALID
    assert fwd(H=64, dh=128) == UNSUPPORTED   # H*dh > 4096
    assert fwd(KV=FAKE + 2) == UNSUPPORTED    # fp32 rows not 4-byte aligned
    assert fwd(g=None) == INVALID
    assert bwd(dKV=None) == INVALID and bwd(KV=None) == INVALID and bwd(dQ=None) == INVALID
    assert bwd(dt=3) == INVALID
    # nothing to do: returns before any HIP call
    g0 = _g(N=0, E=0)
    assert L.fast_edge_attention_fwd_packed(ctypes.byref(g0), 2, 50, 0, None, None, 1.0, 0.2,
                                            None, None, None) == OK
    assert L.fast_edge_attention_bwd_packed(ctypes.byref(g0), 2, 50, 0, None, None, 1.0, 0.2,
                                            None, None, None, None, None) == OK


def test_batched_offsets_and_time_encode_validation():
    """The batched entry points check every block on the host first; an empty
    batch and blocks without work return before any HIP call."""
    L = fast.lib()
    arr = lambda *v: (ctypes.c_void_p * len(v))(*v)
    i64 = lambda *v: (ctypes.c_int64 * len(v))(*v)
    ws = L.fast_csr_offsets_batched_workspace(2, i64(100, 5000))
    assert ws >= max(L.fast_csr_offsets_workspace(100), L.fast_csr_offsets_workspace(5000))
    assert L.fast_csr_offsets_batched_workspace(2, i64(100, -1)) == 0
    assert L.fast_csr_offsets_batched_workspace(1, None) == 0
    assert L.fast_csr_offsets_batched_workspace(0, None) > 0
    off = lambda nb, c, n, o, w=ws, wsp=FAKE: L.fast_csr_offsets_batched(nb, c, n, o, wsp, w, None)
    assert off(0, None, None, None) == OK
    assert off(-1, None, None, None) == INVALID
    assert off(2, None, i64(100, 5000), arr(FAKE, FAKE)) == INVALID          # NULL host array
    assert off(2, arr(FAKE, FAKE), i64(100, -3), arr(FAKE, FAKE)) == INVALID
    assert off(2, arr(FAKE, FAKE), i64(100, 5000), arr(FAKE, None)) == INVALID
    assert off(2, arr(FAKE, None), i64(100, 5000), arr(FAKE, FAKE)) == INVALID
    assert off(2, arr(FAKE, FAKE), i64(100, 1 << 31), arr(FAKE, FAKE)) == UNSUPPORTED
    assert off(2, arr(FAKE, FAKE), i64(100, 5000), arr(FAKE, FAKE), w=ws - 1) == WORKSPACE
    assert off(2, arr(FAKE, FAKE), i64(100, 5000), arr(FAKE, FAKE), wsp=None) == WORKSPACE

    gp = lambda g: ctypes.pointer(g)
    garr = lambda *gs: (ctypes.POINTER(fast.TCSR) * len(gs))(*[gp(g) for g in gs])
    te = lambda nb, gs, outs, d_t=100, dt=0, om=FAKE: L.fast_time_encode_batched(
        nb, gs, om, FAKE, d_t, outs, dt, None)
    gE = fast.TCSR(4, 40, FAKE, None, FAKE, None, FAKE)
    g0 = fast.TCSR(0, 0, None, None, None, None, None)
    assert te(0, None, None) == OK
    assert te(-2, None, None) == INVALID
    assert te(1, None, arr(FAKE)) == INVALID
    assert te(2, garr(gE, gE), None) == INVALID
    assert te(2, garr(g0, g0), arr(None, None)) == OK                   # no edges anywhere
    assert te(2, garr(gE, gE), arr(FAKE, FAKE), dt=4) == INVALID
    assert te(2, garr(gE, gE), arr(FAKE, FAKE), d_t=0) == INVALID
    assert te(2, garr(gE, gE), arr(FAKE, FAKE), om=None) == INVALID
    assert te(2, garr(gE, fast.TCSR(0, 5, FAKE, None, FAKE, None, FAKE)), arr(FAKE, FAKE)) == INVALID
    assert te(1, garr(gE), arr(FAKE + 1)) == UNSUPPORTED                   # fp32 rows, odd address


def test_dedup_validation_and_workspace_query():
    L = fast.lib()
    ws = L.fast_dedup_gather_workspace(1000, 1 << 20)
    assert ws >= (1 << 20) // 8 * 2          # bitmap + word ranks
    assert L.fast_dedup_gather_workspace(1000, 1 << 36) == 0
    args = lambda **k: [k.get("ids", FAKE), k.get("n", 1000), k.get("bound", 1 << 20),
                        k.get("table", FAKE), k.get("rows_n", 1 << 20), 100, k.get("dt", 0),
                        k.get("slot", None), FAKE, FAKE, k.get("nu", FAKE), k.get("rows", FAKE),
                        None, None, k.get("wsp", FAKE), k.get("ws", ws), None]
    assert L.fast_dedup_gather(*args(ws=ws - 1)) == WORKSPACE
    assert L.fast_dedup_gather(*args(wsp=FAKE + 16)) == UNSUPPORTED   # misaligned workspace
    assert L.fast_dedup_gather(*args(n=-1)) == INVALID
    assert L.fast_dedup_gather(*args(nu=None)) == INVALID
    assert L.fast_dedup_gather(*args(ids=None)) == INVALID
    assert L.fast_dedup_gather(*args(dt=3)) == INVALID
    assert L.fast_dedup_gather(*args(bound=1 << 36)) == UNSUPPORTED
    assert L.fast_dedup_gather(*args(rows_n=10)) == INVALID      # no slot map, bound > rows
    assert L.fast_dedup_gather(*args(table=None)) == INVALID     # rows wanted, no table


def test_tcsr_keeps_its_tensors_alive():
    # Regression: the struct holds raw device addresses, so a temporary tensor
    # passed to tcsr() must not be freed (and its memory reused by torch's
    # caching allocator) while the struct is in use.
    import gc
    import weakref

    import torch
    t = torch.arange(3, dtype=torch.float32)
    ref = weakref.ref(t)
    g = fast.tcsr(torch.zeros(5, dtype=torch.int32), 3, edge_t=t)
    del t
    gc.collect()
    assert ref() is not None and g.edge_t == ref().data_ptr()
    assert g.num_dst == 4 and g.num_edges == 3 and g.src_ids is None
    del g
    gc.collect()
    assert ref() is None


def test_time_encode_bwd_validation_and_workspace_query():
    L = fast.lib()
    g = _g(N=64, E=640)
    gp = ctypes.byref(g)
    ws = L.fast_time_encode_bwd_workspace(64, 100)
    assert ws >= 2 * 100 * 2 * 8                      # two groups of 32 segments
    assert L.fast_time_encode_bwd_workspace(-1, 100) == 0
    assert L.fast_time_encode_bwd_workspace(64, 0) == 0
    # one partial per workgroup, at most 2048 workgroups whatever N is
    assert L.fast_time_encode_bwd_workspace(10 ** 9, 128) == L.fast_time_encode_bwd_workspace(
        2048 * 32, 128)

    def call(**k):
        return L.fast_time_encode_bwd(
            k.get("g", gp), k.get("om", FAKE), k.get("ph", FAKE), k.get("d_t", 100),
            k.get("dte", FAKE), k.get("dt", 0), k.get("dw", FAKE), k.get("dp", FAKE),
            k.get("ws", FAKE), k.get("wsb", ws), None)

    assert call(g=None) == INVALID
    assert call(d_t=0) == INVALID
    assert call(dt=5) == INVALID
    assert call(dw=None) == INVALID
    assert call(dp=None) == INVALID
    assert call(om=None) == INVALID
    assert call(dte=None) == INVALID
    assert call(wsb=ws - 1) == WORKSPACE
    assert call(ws=None) == WORKSPACE
    assert call(dw=FAKE + 2) == UNSUPPORTED                      # misaligned output
    assert call(d_t=257, wsb=1 << 20) == UNSUPPORTED             # 257 chunks of one column
    assert call(g=ctypes.byref(_g(N=0, E=5))) == INVALID
    assert call(g=ctypes.byref(_g(N=-1))) == INVALID
    assert call(g=ctypes.byref(_g(E=1 << 31))) == UNSUPPORTED
    assert fast.fast_last_error() != ""


def test_hot_set_validation_and_workspace_queries():
    L = fast.lib()
    assert L.fast_access_count_workspace(1000) >= 4000
    assert L.fast_access_count_workspace(-1) == 0
    assert L.fast_access_count_workspace(1 << 32) == 0
    offs = (ctypes.c_int64 * 3)(0, 10, 25)
    bad = (ctypes.c_int64 * 3)(0, 10, 5)
    p = lambda a: ctypes.cast(a, ctypes.c_void_p)
    wsb = L.fast_access_count_workspace(1000)
    # host-side checks (no launch happens for any of these)
    assert L.fast_access_count(FAKE, p(offs), -1, 1000, FAKE, FAKE, wsb, None) == INVALID
    assert L.fast_access_count(FAKE, p(bad), 2, 1000, FAKE, FAKE, wsb, None) == INVALID
    assert L.fast_access_count(FAKE, None, 2, 1000, FAKE, FAKE, wsb, None) == INVALID
    assert L.fast_access_count(None, p(offs), 2, 1000, FAKE, FAKE, wsb, None) == INVALID
    assert L.fast_access_count(FAKE, p(offs), 2, 1000, None, FAKE, wsb, None) == INVALID
    assert L.fast_access_count(FAKE, p(offs), 2, 1000, FAKE, FAKE, wsb - 1, None) == WORKSPACE
    assert L.fast_access_count(FAKE, p(offs), 2, 1 << 32, FAKE, FAKE, wsb, None) == UNSUPPORTED
    assert L.fast_access_count(None, None, 0, 1000, None, None, 0, None) == OK     # nothing to count

    ws = L.fast_greedy_hot_set_workspace(1000, 5000, 64)
    assert ws > 2 * 65 * 4
    assert L.fast_greedy_hot_set_workspace(1000, 5000, -1) == 0
    assert L.fast_greedy_hot_set_workspace(1000, 5000, (1 << 24) + 1) == 0

    def sel(**k):
        return L.fast_greedy_hot_set(
            k.get("fv", FAKE), k.get("nv", 1000), k.get("fe", FAKE), k.get("ne", 5000),
            k.get("mf", 64), k.get("budget", 100), FAKE, k.get("nhv", FAKE), None, FAKE,
            k.get("nhe", FAKE), None, k.get("ws", FAKE), k.get("wsb", ws), None)

    assert sel(nv=-1) == INVALID
    assert sel(budget=-1) == INVALID
    assert sel(mf=-1) == UNSUPPORTED
    assert sel(nv=1 << 31) == UNSUPPORTED
    assert sel(nhv=None) == INVALID
    assert sel(fv=None) == INVALID
    assert sel(fe=None) == INVALID
    assert sel(wsb=ws - 1) == WORKSPACE
    assert sel(ws=FAKE + 8) == UNSUPPORTED                      # workspace alignment


def test_hot_set_budget():
    """Alg. 1's budget (Sec. 4.2): the library's count of ids equals the
    number of ids the oracle's selection loop `while i + j < alpha(|V|+|E|)`
    takes, with the product in fp64."""
    import numpy as np
    import oracle
    b = fast.fast_hot_set_budget
    assert b(0.1, 5, 5) == 1            # fl64(0.1 * 10) == 1.0 although 0.1 > 1/10 exactly
    assert b(0.15, 5, 5) == 2
    assert b(0.0, 5, 5) == 0
    assert b(-0.5, 5, 5) == 0
    assert b(1.0, 5, 5) == 10
    assert b(1.5, 5, 5) == 10           # capped at |V| + |E|
    assert b(float("inf"), 3, 4) == 7
    assert b(0.5, 0, 0) == 0
    assert b(1e-300, 1, 0) == 1         # any positive product takes one id
    rng = np.random.default_rng(7)
    for nv, ne in ((5, 5), (7, 3), (40, 25), (1, 0), (0, 6)):
        fv = rng.integers(0, 4, nv).astype(np.int32)
        fe = rng.integers(0, 4, ne).astype(np.int32)
        for alpha in (0.0, 0.1, 0.15, 0.3, 1 / 3, 0.7, 1.0, 1.5):
            hv, he = oracle.greedy_hot_set(fv, fe, alpha)
            assert b(alpha, nv, ne) == hv.size + he.size, (nv, ne, alpha)
    L = fast.lib()
    out = ctypes.c_int64(0)
    assert L.fast_hot_set_budget(0.5, -1, 5, ctypes.byref(out)) == INVALID
    assert L.fast_hot_set_budget(0.5, 5, -1, ctypes.byref(out)) == INVALID
    assert L.fast_hot_set_budget(float("nan"), 5, 5, ctypes.byref(out)) == INVALID
    assert L.fast_hot_set_budget(0.5, 5, 5, None) == INVALID


def test_sample_recent_validation():
    L = fast.lib()
    tg = fast.TemporalGraphDesc(100, 1000, FAKE, FAKE, FAKE, FAKE)
    gp = ctypes.byref(tg)
    ws = L.fast_sample_recent_workspace(50)
    assert ws > 50 * 12
    assert L.fast_sample_recent_workspace(-1) == 0

    def call(**k):
        return L.fast_sample_recent(k.get("g", gp), k.get("roots", FAKE), k.get("rt", FAKE),
                                    k.get("R", 50), k.get("k", 10), k.get("off", FAKE),
                                    k.get("src", FAKE), FAKE, FAKE, k.get("ws", FAKE),
                                    k.get("wsb", ws), None)
    assert call(g=None) == INVALID
    assert call(k=-1) == INVALID
    assert call(R=-1) == INVALID
    assert call(R=1 << 28, k=16) == UNSUPPORTED
    # k = 0 keeps the product small, but the per-root workspace would not fit
    assert call(R=1 << 31, k=0, wsb=1 << 20) == UNSUPPORTED
    assert call(off=None) == INVALID
    assert call(roots=None) == INVALID
    assert call(src=None) == INVALID
    assert call(wsb=ws - 1) == WORKSPACE
    assert call(ws=FAKE + 64) == UNSUPPORTED
    bad = fast.TemporalGraphDesc(100, 1000, None, FAKE, FAKE, FAKE)
    assert call(g=ctypes.byref(bad)) == INVALID
    bad = fast.TemporalGraphDesc(100, 1000, FAKE, FAKE, None, FAKE)
    assert call(g=ctypes.byref(bad)) == INVALID


def test_indexed_operands_validation():
    L = fast.lib()
    gp = ctypes.byref(_g())
    # an index with no rows behind it; NULL operands; dtype
    assert L.fast_edge_attention_fwd_indexed(gp, 2, 50, 0, FAKE, FAKE, FAKE, 0, FAKE, None, 0,
                                             1.0, 0.2, FAKE, None, None) == INVALID
    assert L.fast_edge_attention_fwd_indexed(gp, 2, 50, 0, FAKE, None, FAKE, 5, FAKE, None, 0,
                                             1.0, 0.2, FAKE, None, None) == INVALID
    assert L.fast_edge_attention_bwd_indexed(gp, 2, 50, 0, FAKE, FAKE, FAKE, 5, FAKE, FAKE, 5,
                                             1.0, 0.2, None, FAKE, FAKE, None, FAKE, None) == INVALID
    assert L.fast_edge_attention_bwd_indexed(gp, 2, 50, 9, FAKE, FAKE, FAKE, 5, FAKE, FAKE, 5,
                                             1.0, 0.2, None, FAKE, FAKE, FAKE, FAKE, None) == INVALID
    ws = L.fast_occurrence_csr_workspace(1000, 50)
    assert ws >= 4 * 1000 * 4 and L.fast_occurrence_csr_workspace(-1, 5) == 0
    assert L.fast_occurrence_csr(FAKE, 1000, 50, FAKE, FAKE, FAKE, ws - 1, None) == WORKSPACE
    assert L.fast_occurrence_csr(None, 1000, 50, FAKE, FAKE, FAKE, ws, None) == INVALID
    assert L.fast_occurrence_csr(FAKE, 1000, 50, None, FAKE, FAKE, ws, None) == INVALID
    assert L.fast_occurrence_csr(FAKE, -1, 50, FAKE, FAKE, FAKE, ws, None) == INVALID
    assert L.fast_occurrence_csr(FAKE, 1000, 50, FAKE, FAKE, FAKE + 8, ws, None) == UNSUPPORTED
    wa = L.fast_index_add_rows_workspace(1000, 50, 100)
    assert wa > 0 and L.fast_index_add_rows_workspace(1000, 50, 0) == 0
    assert L.fast_index_add_rows(FAKE, FAKE, 1000, 50, 100, 0, FAKE, FAKE, FAKE, wa - 1, None) == WORKSPACE
    assert L.fast_index_add_rows(FAKE, FAKE, 1000, 50, 100, 3, FAKE, FAKE, FAKE, wa, None) == INVALID
    assert L.fast_index_add_rows(None, FAKE, 1000, 50, 100, 0, FAKE, FAKE, FAKE, wa, None) == INVALID
    assert L.fast_index_add_rows(FAKE, FAKE, 1000, 50, 100, 0, None, FAKE, FAKE, wa, None) == INVALID
    assert L.fast_index_add_rows(FAKE, FAKE, 1000, 50, 100, 0, FAKE + 2, FAKE, FAKE, wa, None) == UNSUPPORTED
    assert L.fast_index_add_rows(FAKE, FAKE, 1000, 0, 100, 0, FAKE, None, None, 0, None) == OK


def test_coefficient_form_validation():
    L = fast.lib()
    gp = ctypes.byref(_g())
    coef = lambda **k: L.fast_edge_attention_bwd_indexed_coef(
        gp, 2, 50, 0, FAKE, FAKE, FAKE, 5, FAKE, FAKE, 5, 1.0, 0.2, None, FAKE, FAKE,
        k.get("g", FAKE), k.get("al", FAKE), None)
    assert coef(g=None) == INVALID
    assert coef(al=None) == INVALID
    assert coef(g=FAKE + 2) == UNSUPPORTED
    assert L.fast_edge_attention_bwd_indexed_coef(gp, 2, 50, 0, FAKE, FAKE, FAKE, 0, FAKE, None, 0,
                                                  1.0, 0.2, None, FAKE, FAKE, FAKE, FAKE,
                                                  None) == INVALID      # index without rows
    ws = L.fast_index_add_scaled_rows_workspace(1000, 50, 2, 50)
    assert ws >= 1000 * 4 + L.fast_index_add_rows_workspace(1000, 50, 100)
    assert L.fast_index_add_scaled_rows_workspace(1000, 50, 0, 50) == 0
    assert L.fast_index_add_scaled_rows_workspace(-1, 50, 2, 50) == 0
    call = lambda **k: L.fast_index_add_scaled_rows(
        k.get("off", FAKE), FAKE, k.get("n", 1000), k.get("rows", 50), k.get("doff", FAKE),
        k.get("N", 100), k.get("H", 2), 50, k.get("dt", 0), k.get("scal", FAKE), k.get("src", FAKE),
        k.get("dst", FAKE), FAKE, k.get("ws", ws), None)
    assert call(ws=ws - 1) == WORKSPACE
    assert call(H=0) == INVALID
    assert call(dt=3) == INVALID
    assert call(N=-1) == INVALID
    assert call(N=0) == INVALID                  # edges but no destination
    assert call(N=1 << 31) == UNSUPPORTED
    assert call(off=None) == INVALID
    assert call(doff=None) == INVALID
    assert call(scal=None) == INVALID
    assert call(src=FAKE + 2) == UNSUPPORTED
    assert call(scal=FAKE + 2) == UNSUPPORTED
    assert call(rows=0, dst=None, ws=0) == OK    # nothing to write


@pytest.mark.parametrize("flag", ["-DFAST_ATT_BLOCK_BWD=1024", "-DFAST_ATT_BLOCK=1024",
                                  "-DFAST_ATT_BLOCK_BWD=96"])
def test_attention_workgroup_outside_launch_bound_does_not_build(tmp_path, flag):
    """Every attention kernel is compiled for at most 512 threads per
    workgroup; a build whose workgroup size knob exceeds that (or is not a
    whole number of waves) must fail to compile rather than launch a
    workgroup the runtime refuses."""
    hipcc = "/opt/rocm/bin/hipcc"
    if not os.path.exists(hipcc):
        pytest.skip("hipcc not available")
    src = tmp_path / "probe.hip"
    src.write_text('#include "attention.h"\n')
    csrc = os.path.join(ROOT, "paper_2607_05095_amd", "csrc")
    cmd = [hipcc, "--offload-arch=gfx950", "-std=c++17", "-fsyntax-only", "-I",
           os.path.join(ROOT, "include"), "-I", csrc, str(src)]
    good = subprocess.run(cmd, capture_output=True, text=True)
    assert good.returncode == 0, good.stderr
    bad = subprocess.run(cmd + [flag], capture_output=True, text=True)
    assert bad.returncode != 0
    assert "static assertion failed" in bad.stderr
