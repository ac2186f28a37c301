"""Benchmark of the FAST temporal-subgraph hot path on one MI355X.

One step = one pass of the whole hot path over one synthetic batch, with
every input already resident in HBM:
  1. CSR offsets of both layer blocks              (fast_csr_offsets)
  2. within-batch dedup + row gather, node ids     (fast_dedup_gather)
  3. within-batch dedup + cache gather, edge ids   (fast_dedup_gather, slot map)
  4. time encoding of both blocks                  (fast_time_encode)
  5. fused edge softmax + aggregation: forward of layer 1 and layer 2, then
     backward of layer 2 and layer 1               (fast_edge_attention_fwd/bwd)
value = sampled edges per step / step time.  The roofline entry covers the
dominant kernel, the fused backward of the layer-1 block, timed with HIP
events on the stream it runs on.

    python bench.py [--steps K] [--warmup W] [--workload bigdedup|large] [--also W2,...]
                    [--no-pipelined]

`value` times the steps serially on one stream (prep, then attention).  The
line also reports the same steps software-pipelined (unless --no-pipelined):
prep of batch i+1 on a second stream overlaps attention of batch i.  By
default the 1e7-node fp32 workload (bigdedup) is the headline and the bf16
workload with fan-out 20 (large) is measured after it in the same run, under
the key "large", with its own roofline entry and oracle baseline.
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0
VALU_PEAK_LANE_OPS = 256 * 64 * 2.4e9   # 256 CUs x 64 lanes x 2.4 GHz, one instruction per clock
# The paper publishes relative operator gains only (Sec. 6.3, Fig. 9 and
# Table 5), measured on other hardware: context for the line, not a target.
PAPER_CONTEXT = {
    "hardware": "1x NVIDIA A100 40 GB (Sec. 6.1)",
    "edge_softmax_speedup_over_tgl": "up to 4.2x (4.17x LASTFM, 3.46x BITCOIN)",
    "aggregate_speedup": "up to 2.3x over TGL (2.28x BITCOIN), 1.38x over FastGL",
    "absolute_operator_rates": None,
    "source": "Sec. 6.3 (operator ablation, Fig. 9, Table 5)",
}
SLOPE = 0.2
WORKLOADS = {"bigdedup": 4, "large": 3}
METRIC = "sampled edges/sec, fused edge-softmax+aggregation fwd+bwd; % HBM roofline"
TRAFFIC_FILE = os.path.join(ROOT, "profiles", "traffic_attn_bwd_{workload}.json")
KERNEL_SOURCES = ["paper_2607_05095_amd/csrc/attention.h", "paper_2607_05095_amd/csrc/attention_rowmajor.h",
                  "paper_2607_05095_amd/csrc/attention_fused.hip", "paper_2607_05095_amd/csrc/common.h"]


def log(msg):
    print(f"[bench] {msg}", file=sys.stderr, flush=True)


TIME_ENCODE_SOURCES = ["paper_2607_05095_amd/csrc/time_encode.hip", "paper_2607_05095_amd/csrc/common.h"]


def source_hash(paths):
    h = hashlib.sha256()
    for p in paths:
        with open(os.path.join(ROOT, p), "rb") as f:
            h.update(f.read())
    return h.hexdigest()[:16]


def kernel_source_hash():
    return source_hash(KERNEL_SOURCES)


def describe(b):
    n1, e1 = b.blocks[0].num_dst, b.blocks[0].num_edges
    return {
        "workload": f"{b.name}: {b.blocks[1].num_dst} roots, 2 layers fan-out "
                    f"{b.blocks[0].counts.max()}x{b.blocks[0].counts.max()}, "
                    f"{b.sampled_edges} sampled edges per step",
        "layer_blocks": [[blk.num_dst, blk.num_edges] for blk in b.blocks],
        "heads": b.H, "head_dim": b.dh, "time_dim": b.d_t, "storage": b.dtype,
        "node_ids": int(b.node_ids.size), "node_id_bound": b.node_bound, "node_dim": b.node_D,
        "edge_ids": int(b.edge_ids.size), "edge_id_bound": b.edge_bound, "edge_dim": b.edge_D,
        "edge_cache_rows": b.edge_cache_rows,
    }


class Step:
    """Device buffers of a batch and the launch sequences of one step.

    The step is split in two parts: prep (CSR offsets, dedup + gather of node
    and edge rows, time encoding) and attention (fused forward of both layer
    blocks, then fused backward).  Prep outputs live in `slots` buffer sets,
    so that prep of the next batch can run while attention of the current
    batch still reads its own offsets (software pipelining on two streams)."""

    def __init__(self, b, torch, fast, slots=2, kv="packed"):
        from synth import make_block_operands, make_slot_map, make_table, omega_phi
        self.b, self.torch, self.fast, self.slots = b, torch, fast, slots
        # "packed": each edge's K and V rows side by side in one [E, 2, H, dh]
        # array (and dK, dV likewise), the layout a fused K|V projection
        # writes; "separate": four [E, H, dh] arrays
        self.kv = kv
        dev = "cuda"
        tdt = torch.float32 if b.dtype == "f32" else torch.bfloat16
        self.DT = fast.F32 if b.dtype == "f32" else fast.BF16
        self.blocks = []
        for i, blk in enumerate(b.blocks):
            N, E = blk.num_dst, blk.num_edges
            d = dict(N=N, E=E)
            d["counts"] = torch.from_numpy(blk.counts).to(dev)
            d["dst_t"] = torch.from_numpy(blk.dst_t).to(dev)
            d["edge_t"] = torch.from_numpy(blk.edge_t).to(dev)
            d.update(make_block_operands(b, i, device=dev))
            d["out"] = torch.empty((N, b.H, b.dh), dtype=tdt, device=dev)
            d["lse"] = torch.empty((N, b.H), dtype=torch.float32, device=dev)
            d["dQ"] = torch.empty((N, b.H, b.dh), dtype=tdt, device=dev)
            if kv == "packed":
                # the same K and V values, moved into one packed array; K, V,
                # dK and dV stay addressable as [E, H, dh] views
                d["KV"] = torch.empty((E, 2, b.H, b.dh), dtype=tdt, device=dev)
                d["KV"][:, 0] = d.pop("K")
                d["KV"][:, 1] = d.pop("V")
                d["K"], d["V"] = d["KV"][:, 0], d["KV"][:, 1]
                d["dKV"] = torch.empty((E, 2, b.H, b.dh), dtype=tdt, device=dev)
                d["dK"], d["dV"] = d["dKV"][:, 0], d["dKV"][:, 1]
            else:
                d["dK"] = torch.empty((E, b.H, b.dh), dtype=tdt, device=dev)
                d["dV"] = torch.empty((E, b.H, b.dh), dtype=tdt, device=dev)
            d["off"], d["te"], d["g"] = [], [], []
            for _ in range(slots):
                off = torch.empty(N + 1, dtype=torch.int32, device=dev)
                d["off"].append(off)
                d["te"].append(torch.empty((E, b.d_t), dtype=tdt, device=dev))
                d["g"].append(fast.tcsr(off, E, edge_t=d["edge_t"], dst_t=d["dst_t"]))
            self.blocks.append(d)
        # the offsets of all layer blocks: one batched scan per slot
        self.off_n = [d["N"] for d in self.blocks]
        self.ws_off_bytes = fast.fast_csr_offsets_batched_workspace(self.off_n)
        self.ws_off = [torch.empty(self.ws_off_bytes, dtype=torch.uint8, device=dev)
                       for _ in range(slots)]
        om, ph = omega_phi(b.d_t)
        self.omega = torch.from_numpy(om).to(dev)
        self.phi = torch.from_numpy(ph).to(dev)
        self.scale = float(np.float32(1.0 / np.sqrt(b.dh)))
        # node ids: table indexed by id
        log(f"node table {b.node_bound} x {b.node_D} {b.dtype}")
        node_table = make_table(b.node_bound, b.node_D, b.dtype, dev, b.seed, 3)
        # edge ids: a cache with a slot map, or a table indexed by id
        if b.edge_cache_rows:
            log(f"edge cache {b.edge_cache_rows} x {b.edge_D}, slot map over {b.edge_bound}")
            edge_table = make_table(b.edge_cache_rows, b.edge_D, b.dtype, dev, b.seed, 4)
            slot_map = make_slot_map(b, device=dev)
        else:
            edge_table = make_table(b.edge_bound, b.edge_D, b.dtype, dev, b.seed, 4)
            slot_map = None
        self.node = [self._dedup_bufs(b.node_ids, b.node_bound, node_table, None) for _ in range(slots)]
        self.edge = [self._dedup_bufs(b.edge_ids, b.edge_bound, edge_table, slot_map) for _ in range(slots)]

    def _dedup_bufs(self, ids_np, bound, table, slot):
        torch, fast = self.torch, self.fast
        n = ids_np.shape[0]
        d = dict(n=n, bound=bound, table=table, slot=slot)
        d["ids"] = torch.from_numpy(ids_np).cuda()
        d["uni"] = torch.empty(n, dtype=torch.int64, device="cuda")
        d["inv"] = torch.empty(n, dtype=torch.int32, device="cuda")
        d["nu"] = torch.empty(1, dtype=torch.int64, device="cuda")
        d["rows"] = torch.empty((n, table.shape[1]), dtype=table.dtype, device="cuda")
        d["miss"] = torch.empty(n, dtype=torch.int32, device="cuda")
        d["nm"] = torch.empty(1, dtype=torch.int64, device="cuda")
        d["wsb"] = fast.fast_dedup_gather_workspace(n, bound)
        d["ws"] = torch.empty(d["wsb"], dtype=torch.uint8, device="cuda")
        return d

    def _dedup(self, d):
        f = self.fast
        f.fast_dedup_gather(d["ids"], d["n"], d["bound"], d["table"], d["table"].shape[0],
                            d["table"].shape[1], self.DT, d["slot"], d["uni"], d["inv"], d["nu"],
                            d["rows"], d["miss"], d["nm"], d["ws"], d["wsb"])

    @staticmethod
    def _marker(torch, rec, names):
        st = torch.cuda.current_stream()

        def mark(name, fn):
            if rec is None or (names is not None and name not in names):
                fn()
                return
            s, e = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            s.record(st)
            fn()
            e.record(st)
            rec.setdefault(name, []).append((s, e))
        return mark

    def prep(self, slot, rec=None, names=None):
        """Offsets, time encoding, dedup + gather (nodes, edges) into `slot`;
        the offsets and the time encoding of all layer blocks in one batched
        call each.  The three are independent; the time encoding goes first so
        that the write-back of its output overlaps the dedups rather than the
        attention."""
        f, b = self.fast, self.b
        mark = self._marker(self.torch, rec, names)
        mark("offsets", lambda: f.fast_csr_offsets_batched(
            [d["counts"] for d in self.blocks], self.off_n, [d["off"][slot] for d in self.blocks],
            self.ws_off[slot], self.ws_off_bytes))
        mark("time_encode", lambda: f.fast_time_encode_batched(
            [d["g"][slot] for d in self.blocks], self.omega, self.phi, b.d_t,
            [d["te"][slot] for d in self.blocks], self.DT))
        mark("dedup_gather_nodes", lambda: self._dedup(self.node[slot]))
        mark("dedup_gather_edges", lambda: self._dedup(self.edge[slot]))

    def attn(self, slot, rec=None, names=None):
        """Fused forward of layer 1 then layer 2, fused backward of layer 2 then
        layer 1, on the offsets of `slot`."""
        f, b = self.fast, self.b
        mark = self._marker(self.torch, rec, names)
        packed = self.kv == "packed"
        for i, d in enumerate(self.blocks):
            if packed:
                fn = lambda d=d: f.fast_edge_attention_fwd_packed(
                    d["g"][slot], b.H, b.dh, self.DT, d["Q"], d["KV"], self.scale, SLOPE,
                    d["out"], d["lse"])
            else:
                fn = lambda d=d: f.fast_edge_attention_fwd(
                    d["g"][slot], b.H, b.dh, self.DT, d["Q"], d["K"], d["V"], self.scale, SLOPE,
                    d["out"], d["lse"])
            mark(f"attn_fwd_L{i + 1}", fn)
        for i in reversed(range(len(self.blocks))):
            d = self.blocks[i]
            if packed:
                fn = lambda d=d: f.fast_edge_attention_bwd_packed(
                    d["g"][slot], b.H, b.dh, self.DT, d["Q"], d["KV"], self.scale, SLOPE,
                    d["lse"], d["dO"], d["dQ"], d["dKV"])
            else:
                fn = lambda d=d: f.fast_edge_attention_bwd(
                    d["g"][slot], b.H, b.dh, self.DT, d["Q"], d["K"], d["V"], self.scale, SLOPE,
                    d["lse"], d["dO"], d["dQ"], d["dK"], d["dV"])
            mark(f"attn_bwd_L{i + 1}", fn)

    def run_serial(self, rec=None, names=None):
        self.prep(0, rec, names)
        self.attn(0, rec, names)

    def run_pipelined(self, K, side, rec=None, names=None):
        """K steps; prep of batch i+1 runs on stream `side` while attention of
        batch i runs on the current stream.  Dependencies: attention(i) waits
        for prep(i); prep(i+2) reuses slot i % 2 only after attention(i)."""
        torch = self.torch
        main = torch.cuda.current_stream()
        ready = [torch.cuda.Event() for _ in range(self.slots)]
        free = [None] * self.slots
        side.wait_stream(main)

        def enqueue_prep(i):
            s = i % self.slots
            with torch.cuda.stream(side):
                if free[s] is not None:
                    side.wait_event(free[s])
                self.prep(s)
                ready[s].record(side)

        enqueue_prep(0)
        for i in range(K):
            if i + 1 < K:
                enqueue_prep(i + 1)
            s = i % self.slots
            main.wait_event(ready[s])
            self.attn(s, rec, names)
            ev = torch.cuda.Event()
            ev.record(main)
            free[s] = ev
        main.wait_stream(side)


def attn_bwd_bytes(N, E, F, esz, H):
    """Algorithmic bytes of one fused backward launch: read Q, dOut (N rows),
    K, V (E rows), lse, offsets; write dQ (N rows), dK, dV (E rows)."""
    return (4 * E + 3 * N) * F * esz + 4 * N * H + 4 * (N + 1)


def attn_fwd_bytes(N, E, F, esz, H):
    """Read Q (N rows), K, V (E rows), offsets; write out (N rows) and lse."""
    return (2 * E + 2 * N) * F * esz + 4 * N * H + 4 * (N + 1)


def _oracle_time(fn, min_seconds=0.5, max_runs=5):
    """Mean wall time (s) of fn() on the host over up to max_runs calls."""
    times = []
    while len(times) < max_runs and sum(times) < min_seconds:
        t0 = time.perf_counter()
        fn()
        times.append(time.perf_counter() - t0)
    return float(np.mean(times))


def _oracle_entry(seconds, units, unit, sample):
    return {"ms": round(seconds * 1e3, 3), "rate": round(units / seconds, 1), "unit": unit,
            "sample": sample, "cores": 1, "kind": "oracle"}


def time_encode_bwd_bytes(N, E, d_t, esz):
    """Read dte [E, d_t], edge times, destination times and offsets, omega and
    phi; write domega and dphi."""
    return E * (4 + d_t * esz) + 8 * N + 4 + 16 * d_t


def widened_ops(b, step, torch, fast, reps=10, with_oracle=False):
    """Operators beyond the timed step, each timed alone with HIP events on
    its launch stream (mean of `reps` launches after one warm-up): the
    time-encoding backward of each layer block, on a seeded upstream
    gradient, the cache selection of Alg. 1, two hops of most-recent-k
    temporal sampling, and the layer-1 attention with indexed operands."""
    from synth import _randn
    esz = 4 if b.dtype == "f32" else 2
    res = {}
    for i, d in enumerate(step.blocks):
        N, E = d["N"], d["E"]
        dte = _randn((E, b.d_t), b.dtype, "cuda", 4242 + i)
        dw = torch.empty(b.d_t, device="cuda")
        dp = torch.empty(b.d_t, device="cuda")
        wsb = fast.fast_time_encode_bwd_workspace(N, b.d_t)
        ws = torch.empty(wsb, dtype=torch.uint8, device="cuda")
        g = d["g"][0]

        def call():
            fast.fast_time_encode_bwd(g, step.omega, step.phi, b.d_t, dte, step.DT, dw, dp, ws, wsb)
        call()
        st = torch.cuda.current_stream()
        s, e = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        torch.cuda.synchronize()
        s.record(st)
        for _ in range(reps):
            call()
        e.record(st)
        torch.cuda.synchronize()
        ms = s.elapsed_time(e) / reps
        nbytes = time_encode_bwd_bytes(N, E, b.d_t, esz)
        res[f"time_encode_bwd_L{i + 1}"] = {
            "ms": round(ms, 4), "algorithmic_bytes": nbytes, "bound": "alu (fp64 sine per element)",
            "achieved_gbs": round(nbytes / (ms * 1e-3) / 1e9, 1),
            "hbm_frac": round(nbytes / (ms * 1e-3) / 1e9 / HBM_PEAK_GBS, 4),
            "edges_per_s": round(E / (ms * 1e-3), 1),
        }
        if with_oracle and i == 0:
            import oracle
            from synth import omega_phi
            blk = b.blocks[0]
            ns = max(1, blk.num_dst // 10)
            off = oracle.csr_offsets(blk.counts[:ns])
            es = int(off[-1])
            g64 = dte[:es].double().cpu().numpy()
            om, ph = omega_phi(b.d_t)
            sec = _oracle_time(lambda: oracle.time_encode_bwd(off, blk.dst_t[:ns], blk.edge_t[:es],
                                                              om, ph, g64))
            res["time_encode_bwd_L1"]["oracle"] = _oracle_entry(
                sec, es, "edges/s", f"first 10% of the layer-1 segments ({es} edges)")
        del dte, ws
    res.update(hot_set_ops(b, torch, fast, with_oracle=with_oracle))
    res.update(sampler_ops(b, torch, fast, with_oracle=with_oracle))
    res.update(indexed_ops(b, step, torch, fast, with_oracle=with_oracle))
    return res


def indexed_ops(b, step, torch, fast, reps=5, with_oracle=False):
    """The layer-1 fused attention with indexed operands: K read through the
    de-duplication inverse of the block's source node ids, V through that of
    its edge ids (compact rows), then the row gradients of both (occurrence
    lists + ordered row sums)."""
    from synth import _randn
    blk, d = b.blocks[0], step.blocks[0]
    N, E, H, dh = blk.num_dst, blk.num_edges, b.H, b.dh
    F, esz = H * dh, (4 if b.dtype == "f32" else 2)
    _, kidx = np.unique(blk.src_ids, return_inverse=True)
    _, vidx = np.unique(blk.edge_ids, return_inverse=True)
    Uk, Uv = int(kidx.max()) + 1, int(vidx.max()) + 1
    tdt = torch.float32 if b.dtype == "f32" else torch.bfloat16
    K = _randn((Uk, H, dh), b.dtype, "cuda", 9001)
    V = _randn((Uv, H, dh), b.dtype, "cuda", 9002)
    ki = torch.from_numpy(kidx.astype(np.int32)).cuda()
    vi = torch.from_numpy(vidx.astype(np.int32)).cuda()
    g = d["g"][0]
    out = torch.empty((N, H, dh), dtype=tdt, device="cuda")
    lse = torch.empty((N, H), device="cuda")
    dQ = torch.empty((N, H, dh), dtype=tdt, device="cuda")
    dKe = torch.empty((E, H, dh), dtype=tdt, device="cuda")
    dVe = torch.empty((E, H, dh), dtype=tdt, device="cuda")
    bufs = {}
    for name, idx, U in (("K", ki, Uk), ("V", vi, Uv)):
        wo = fast.fast_occurrence_csr_workspace(E, U)
        wa = fast.fast_index_add_rows_workspace(E, U, F)
        bufs[name] = dict(idx=idx, U=U, off=torch.empty(U + 1, dtype=torch.int32, device="cuda"),
                          occ=torch.empty(E, dtype=torch.int32, device="cuda"),
                          wso=torch.empty(wo, dtype=torch.uint8, device="cuda"), wo=wo,
                          wsa=torch.empty(wa, dtype=torch.uint8, device="cuda"), wa=wa,
                          dst=torch.empty((U, F), device="cuda"))

    def fwd():
        fast.fast_edge_attention_fwd_indexed(g, H, dh, step.DT, d["Q"], K, ki, Uk, V, vi, Uv, step.scale,
                                             SLOPE, out, lse)

    def bwd():
        fast.fast_edge_attention_bwd_indexed(g, H, dh, step.DT, d["Q"], K, ki, Uk, V, vi, Uv, step.scale,
                                             SLOPE, lse, d["dO"], dQ, dKe, dVe)

    def occ():
        for x in bufs.values():
            fast.fast_occurrence_csr(x["idx"], E, x["U"], x["off"], x["occ"], x["wso"], x["wo"])

    def add():
        for x, src in ((bufs["K"], dKe), (bufs["V"], dVe)):
            fast.fast_index_add_rows(x["off"], x["occ"], E, x["U"], F, step.DT, src, x["dst"],
                                     x["wsa"], x["wa"])

    # coefficient form: per-edge g and alpha, then row gradients from the
    # segment rows of Q and dOut
    ge = torch.empty((E, H), device="cuda")
    ae = torch.empty((E, H), device="cuda")
    for name, x in bufs.items():
        x["ws_s"] = fast.fast_index_add_scaled_rows_workspace(E, x["U"], H, dh)
        x["wss"] = torch.empty(x["ws_s"], dtype=torch.uint8, device="cuda")
        x["dst_s"] = torch.empty((x["U"], H, dh), device="cuda")

    def bwd_coef():
        fast.fast_edge_attention_bwd_indexed_coef(g, H, dh, step.DT, d["Q"], K, ki, Uk, V, vi, Uv,
                                                  step.scale, SLOPE, lse, d["dO"], dQ, ge, ae)

    def add_scaled():
        for x, scal, src in ((bufs["K"], ge, d["Q"]), (bufs["V"], ae, d["dO"])):
            fast.fast_index_add_scaled_rows(x["off"], x["occ"], E, x["U"], d["off"][0], N, H, dh,
                                            step.DT, scal, src, x["dst_s"], x["wss"], x["ws_s"])
    for f in (fwd, bwd, occ, add, bwd_coef, add_scaled):
        f()
    t = {k: _events_ms(torch, f, reps) for k, f in (("fwd", fwd), ("bwd", bwd), ("occurrence_lists", occ),
                                                   ("row_sums", add))}
    t_coef = {k: _events_ms(torch, f, reps) for k, f in (("bwd_coef", bwd_coef),
                                                         ("scaled_row_sums", add_scaled))}
    # compulsory bytes: each compact row once; per-edge bytes: as the plain operator
    fwd_rows = (2 * N) * F * esz + (Uk + Uv) * F * esz + 8 * E + 4 * N * H + 4 * (N + 1)
    orc = None
    if with_oracle:
        import oracle
        ns = max(1, N // 50)
        off = oracle.csr_offsets(blk.counts[:ns])
        es = int(off[-1])
        Qh, dOh = d["Q"][:ns].cpu(), d["dO"][:ns].cpu()
        Kh, Vh = K.cpu(), V.cpu()
        kh, vh = kidx[:es].astype(np.int32), vidx[:es].astype(np.int32)

        def run():
            oracle.edge_attention_fwd_indexed(off, Qh, Kh, kh, Vh, vh, step.scale, SLOPE)
            oracle.edge_attention_bwd_indexed(off, Qh, Kh, kh, Vh, vh, dOh, step.scale, SLOPE)
        sec = _oracle_time(run)
        orc = _oracle_entry(sec, es, "edges/s",
                            f"first 2% of the layer-1 segments ({es} edges): forward, backward and row sums")
    out_entry = {
        "ms": {k: round(v, 4) for k, v in t.items()},
        "compact_rows": {"K": Uk, "V": Uv, "edges": E},
        "fwd_compulsory_bytes": fwd_rows,
        "fwd_gbs_compulsory": round(fwd_rows / (t["fwd"] * 1e-3) / 1e9, 1),
        "fwd_gbs_per_edge_rows": round(attn_fwd_bytes(N, E, F, esz, H) / (t["fwd"] * 1e-3) / 1e9, 1),
        "note": "K and V read through indices into de-duplicated rows; backward writes per-edge "
                "gradients, then occurrence lists and ordered row sums give the row gradients",
        "edges_per_s": round(E / (sum(t.values()) * 1e-3), 1),
        "coefficient_form_ms": {k: round(v, 4) for k, v in t_coef.items()},
        "coefficient_form_note": "backward writes per-edge g and alpha (8H bytes per edge) instead of "
                                 "dK/dV rows; row gradients sum g*Q[seg] and alpha*dOut[seg] over the "
                                 "same occurrence lists",
        "coefficient_form_edges_per_s": round(
            E / ((t["fwd"] + t["occurrence_lists"] + sum(t_coef.values())) * 1e-3), 1),
    }
    if orc is not None:
        out_entry["oracle"] = orc
    return {"attention_indexed_L1": out_entry}


def sampler_ops(b, torch, fast, num_events=20_000_000, reps=5, with_oracle=False):
    """Two hops of most-recent-k sampling for one batch of this workload's
    shape (roots / 3 events, fan-out k) on an event-stream temporal graph
    over the workload's node universe (each event stored under both ends)."""
    from synth import make_temporal_graph, sampler_roots
    k = int(b.blocks[-1].counts.max())
    g = make_temporal_graph(b.node_bound, num_events, seed=b.seed)
    roots, rt = sampler_roots(g, b.blocks[-1].num_dst // 3, seed=b.seed)
    dg = fast.temporal_graph(*(torch.from_numpy(x).cuda() for x in (g.indptr, g.nbr, g.ts, g.eid)))
    res, q_roots, q_t = {}, torch.from_numpy(roots).cuda(), torch.from_numpy(rt).cuda()
    for hop in (1, 2):
        R = int(q_roots.numel())
        off = torch.empty(R + 1, dtype=torch.int32, device="cuda")
        src = torch.empty(max(R * k, 1), dtype=torch.int64, device="cuda")
        et = torch.empty(max(R * k, 1), dtype=torch.float32, device="cuda")
        ei = torch.empty(max(R * k, 1), dtype=torch.int64, device="cuda")
        wsb = fast.fast_sample_recent_workspace(R)
        ws = torch.empty(wsb, dtype=torch.uint8, device="cuda")

        def call():
            fast.fast_sample_recent(dg, q_roots, q_t, R, k, off, src, et, ei, ws, wsb)
        call()
        ms = _events_ms(torch, call, reps)
        E = int(off[-1].item())
        res[f"sample_recent_hop{hop}"] = {
            "ms": round(ms, 4), "roots": R, "k": k, "sampled_edges": E,
            "graph": f"{g.num_nodes} nodes, {num_events} events ({int(g.indptr[-1])} entries)",
            "bound": "latency (binary search per root over its time-sorted entries)",
            "sampled_edges_per_s": round(E / (ms * 1e-3), 1),
        }
        q_roots, q_t = src[:E].clone(), et[:E].clone()
        if with_oracle and hop == 1:
            import oracle
            nr = max(1, roots.size // 10)
            holder = {}
            sec = _oracle_time(lambda: holder.update(
                r=oracle.sample_recent(g.indptr, g.nbr, g.ts, g.eid, roots[:nr], rt[:nr], k)))
            ne = int(holder["r"][0][-1])
            res["sample_recent_hop1"]["oracle"] = _oracle_entry(
                sec, ne, "sampled edges/s", f"first 10% of the hop-1 roots ({nr} roots, {ne} edges)")
    return res


def _events_ms(torch, fn, reps):
    st = torch.cuda.current_stream()
    s, e = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    s.record(st)
    for _ in range(reps):
        fn()
    e.record(st)
    torch.cuda.synchronize()
    return s.elapsed_time(e) / reps


def hot_set_ops(b, torch, fast, num_batches=8, alpha=0.01, reps=3, with_oracle=False):
    """SlimCache's pre-training cache selection (Alg. 1) over `num_batches`
    pre-sampled batches of this workload's graph: access counting of node and
    edge ids, then the greedy selection of alpha * (|V| + |E|) ids with both
    slot maps."""
    from synth import presampled_ids
    nodes, edges, nb, eb = presampled_ids(b.cfg, num_batches)
    res = {}
    freqs = []
    for kind, batches, bound in (("nodes", nodes, nb), ("edges", edges, eb)):
        ids = torch.from_numpy(np.concatenate(batches)).cuda()
        offs = np.concatenate([[0], np.cumsum([x.size for x in batches])]).astype(np.int64)
        f = torch.zeros(bound, dtype=torch.int32, device="cuda")
        wsb = fast.fast_access_count_workspace(bound)
        ws = torch.empty(wsb, dtype=torch.uint8, device="cuda")

        def count():
            fast.fast_access_count(ids, offs, num_batches, bound, f, ws, wsb)
        count()
        ms = _events_ms(torch, count, reps)
        f.zero_()
        count()
        freqs.append(f)
        n = int(ids.numel())
        res[f"access_count_{kind}"] = {
            "ms": round(ms, 4), "ids": n, "id_bound": bound, "batches": num_batches,
            "bound": "random 4-byte atomics (one mask OR per id, one add per distinct id and batch)",
            "ids_per_s": round(n / (ms * 1e-3), 1),
        }
        if with_oracle:
            import oracle
            sec = _oracle_time(lambda: oracle.access_count(batches[:1], bound))
            res[f"access_count_{kind}"]["oracle"] = _oracle_entry(
                sec, batches[0].size, "ids/s", f"one pre-sampled batch ({batches[0].size} ids)")
        del ids, ws
    fv, fe = freqs
    B = fast.fast_hot_set_budget(alpha, nb, eb)
    hv = torch.empty(max(min(B, nb), 1), dtype=torch.int64, device="cuda")
    he = torch.empty(max(min(B, eb), 1), dtype=torch.int64, device="cuda")
    nhv = torch.empty(1, dtype=torch.int64, device="cuda")
    nhe = torch.empty(1, dtype=torch.int64, device="cuda")
    sv = torch.empty(nb, dtype=torch.int32, device="cuda")
    se = torch.empty(eb, dtype=torch.int32, device="cuda")
    wsb = fast.fast_greedy_hot_set_workspace(nb, eb, num_batches)
    ws = torch.empty(wsb, dtype=torch.uint8, device="cuda")

    def select():
        fast.fast_greedy_hot_set(fv, nb, fe, eb, num_batches, B, hv, nhv, sv, he, nhe, se, ws, wsb)
    select()
    ms = _events_ms(torch, select, reps)
    nbytes = greedy_hot_set_bytes(nb, eb, B)
    res["greedy_hot_set"] = {
        "ms": round(ms, 4), "budget": B, "hot_nodes": int(nhv.item()), "hot_edges": int(nhe.item()),
        "algorithmic_bytes": nbytes, "bound": "hbm",
        "achieved_gbs": round(nbytes / (ms * 1e-3) / 1e9, 1),
        "hbm_frac": round(nbytes / (ms * 1e-3) / 1e9 / HBM_PEAK_GBS, 4),
        "ids_per_s": round((nb + eb) / (ms * 1e-3), 1),
    }
    if with_oracle:
        import oracle
        sv_n, se_n = max(1, nb // 100), max(1, eb // 100)
        fv_h, fe_h = fv[:sv_n].cpu().numpy(), fe[:se_n].cpu().numpy()
        sec = _oracle_time(lambda: oracle.greedy_hot_set(fv_h, fe_h, alpha))
        res["greedy_hot_set"]["oracle"] = _oracle_entry(
            sec, sv_n + se_n, "ids/s", f"first 1% of each universe ({sv_n} nodes, {se_n} edges)")
    return res


def offsets_bytes(N):
    """Counts read, offsets written."""
    return 4 * N + 4 * (N + 1)


def dedup_gather_bytes(n, u, hits, row_bytes, slot_map):
    """Per id 8 + 4 (id read, inverse written); per distinct id 8 (uni) and,
    through a slot map, 4 (its slot); per cached row 2 x row_bytes (read and
    written); per miss 4 (its miss-list entry)."""
    return 12 * n + u * (8 + (4 if slot_map else 0)) + hits * 2 * row_bytes + (u - hits) * 4


def step_roofline(b, breakdown, ms, nodes, edges):
    """Algorithmic bytes of every operator of the step (inputs read once,
    outputs written once; `nodes`/`edges` = (ids, distinct, cached) of the
    two dedup + gathers) against the per-operator times and the whole serial
    step."""
    esz = 4 if b.dtype == "f32" else 2
    F = b.H * b.dh
    ops = {"offsets": sum(offsets_bytes(x.num_dst) for x in b.blocks),
           "time_encode": sum(x.num_edges * (4 + b.d_t * esz) + 8 * x.num_dst for x in b.blocks),
           "dedup_gather_nodes": dedup_gather_bytes(*nodes, b.node_D * esz, False),
           "dedup_gather_edges": dedup_gather_bytes(*edges, b.edge_D * esz, bool(b.edge_cache_rows))}
    for i, x in enumerate(b.blocks):
        ops[f"attn_fwd_L{i + 1}"] = attn_fwd_bytes(x.num_dst, x.num_edges, F, esz, b.H)
        ops[f"attn_bwd_L{i + 1}"] = attn_bwd_bytes(x.num_dst, x.num_edges, F, esz, b.H)
    frac = lambda nb, t: round(nb / (t * 1e-3) / 1e9 / HBM_PEAK_GBS, 4) if t and t > 0 else None
    total = sum(ops.values())
    return {"algorithmic_bytes": total, "hbm_frac": frac(total, ms),
            "operators": {k: {"ms": round(breakdown.get(k, 0.0), 4), "bytes": v,
                              "hbm_frac": frac(v, breakdown.get(k))} for k, v in ops.items()},
            "note": "each operator's inputs read once and outputs written once, summed over the "
                    "step, against the serial step time (operators: their breakdown times)"}


def greedy_hot_set_bytes(nv, ne, B):
    """Read every count once, write every slot-map entry, write the hot ids."""
    return 4 * (nv + ne) + 4 * (nv + ne) + 8 * B


def time_encode_summary(b, breakdown, counters=None):
    """Time encoding of all layer blocks (one batched launch) in the serial
    step: algorithmic bytes E (4 + d_t b) + 8 N per block against the measured
    time; with a counter record of that launch taken on the current
    time-encoding source, also its VALU utilisation (VALU wave instructions x
    64 lanes over the time, against 256 CUs x 64 lanes x 2.4 GHz)."""
    b_out = 4 if b.dtype == "f32" else 2
    ms = breakdown.get("time_encode", 0.0)
    nbytes = sum(x.num_edges * (4 + b.d_t * b_out) + 8 * x.num_dst for x in b.blocks)
    res = {"ms": round(ms, 4), "algorithmic_bytes": nbytes,
           "hbm_frac": round(nbytes / (ms * 1e-3) / 1e9 / HBM_PEAK_GBS, 4) if ms > 0 else None,
           "cosines_per_s": sum(x.num_edges for x in b.blocks) * b.d_t / (ms * 1e-3) if ms > 0 else None}
    v = (counters or {}).get("time_encode_valu")
    if v and v.get("source_sha") == source_hash(TIME_ENCODE_SOURCES) and ms > 0:
        lane = v["valu_wave_insts_per_launch"] * 64 / (ms * 1e-3)
        res["valu"] = {"lane_insts_per_s": lane, "frac": round(lane / VALU_PEAK_LANE_OPS, 4),
                       "source": v.get("source")}
    return res


def host_cpu_model():
    """Model name of the host CPU (first entry of /proc/cpuinfo), or None."""
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return None


def attention_sequence_ms(step, torch, reps=50, warm=5):
    """Median over `reps` runs of the fused attention of one step as a unit:
    HIP events on the launch stream around the four launches (layer-1 and
    layer-2 forward, layer-2 and layer-1 backward), after `warm` warm-ups."""
    st = torch.cuda.current_stream()
    for _ in range(warm):
        step.attn(0)
    times = []
    for _ in range(reps):
        s, e = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        s.record(st)
        step.attn(0)
        e.record(st)
        e.synchronize()
        times.append(s.elapsed_time(e))
    return float(np.median(times))


def cpu_baseline(b, step, torch, frac, min_seconds=10.0):
    """The fp64 oracle, single-threaded, on a bounded sample of the same batch:
    the first `frac` of the segments of each layer block and the matching
    share of node and edge ids, through the same sequence of operators,
    repeated until about `min_seconds` of CPU time (at most 5 passes); the
    median pass time gives the rate."""
    import oracle
    from synth import omega_phi
    om, ph = omega_phi(b.d_t)
    sample_edges = 0
    # inputs for the sample (host copies, outside the timed region)
    blocks = []
    for i, blk in enumerate(b.blocks):
        ns = max(1, int(blk.num_dst * frac))
        counts = blk.counts[:ns]
        es = int(counts.sum())
        d = step.blocks[i]
        blocks.append(dict(counts=counts, dst_t=blk.dst_t[:ns], edge_t=blk.edge_t[:es],
                           Q=d["Q"][:ns].cpu(), K=d["K"][:es].cpu(), V=d["V"][:es].cpu(),
                           dO=d["dO"][:ns].cpu()))
        sample_edges += es
    nn, ne = int(b.node_ids.size * frac), int(b.edge_ids.size * frac)
    node_ids, edge_ids = b.node_ids[:nn], b.edge_ids[:ne]
    bits = torch.int16 if b.dtype == "bf16" else torch.int32
    node_table = step.node[0]["table"].view(bits).cpu().numpy()
    edge_table = step.edge[0]["table"].view(bits).cpu().numpy()
    slot = None if step.edge[0]["slot"] is None else step.edge[0]["slot"].cpu().numpy()
    scale = step.scale

    def one_pass():
        offs = [oracle.csr_offsets(x["counts"]) for x in blocks]
        uni, _ = oracle.dedup(node_ids)
        oracle.gather(uni, node_table)
        uni, _ = oracle.dedup(edge_ids)
        oracle.gather(uni, edge_table, slot)
        for x, off in zip(blocks, offs):
            oracle.time_encode(off, x["dst_t"], x["edge_t"], om, ph)
        for x, off in zip(blocks, offs):
            oracle.edge_attention_fwd(off, x["Q"], x["K"], x["V"], scale, SLOPE)
        for x, off in reversed(list(zip(blocks, offs))):
            oracle.edge_attention_bwd(off, x["Q"], x["K"], x["V"], x["dO"], scale, SLOPE)

    times = []
    while len(times) < 5 and sum(times) < min_seconds:
        t0 = time.perf_counter()
        one_pass()
        times.append(time.perf_counter() - t0)
    dt = float(np.median(times))
    res = {
        "value": sample_edges / dt, "unit": "sampled edges/s", "cores": 1, "kind": "oracle",
        "host_threads": os.cpu_count(), "cpu_model": host_cpu_model(),
        "sample": f"{frac:.0%} of the segments of each layer block ({sample_edges} sampled edges) "
                  f"and of the node/edge ids, through offsets, dedup+gather, time encoding and "
                  f"fused attention fwd+bwd in fp64, single-threaded; median of {len(times)} "
                  f"passes, {sum(times):.1f} s in total",
        "seconds_per_pass": round(dt, 3),
    }
    res["all_cores"] = cpu_baseline_threads(blocks, node_ids, edge_ids, node_table, edge_table,
                                            slot, om, ph, scale, sample_edges)
    return res


def segment_shares(blocks, T):
    """Cut every layer block into T contiguous destination ranges (equal
    segment counts): shares[t] holds, per block, range t's counts, times and
    Q/K/V/dOut rows (a destination's edges are contiguous in CSR order)."""
    shares = [[] for _ in range(T)]
    for x in blocks:
        counts = np.asarray(x["counts"])
        ns = counts.shape[0]
        ends = np.concatenate([[0], np.cumsum(counts)])
        cuts = np.linspace(0, ns, T + 1).astype(np.int64)
        for t in range(T):
            a, c = int(cuts[t]), int(cuts[t + 1])
            ea, ec = int(ends[a]), int(ends[c])
            shares[t].append(dict(counts=counts[a:c], dst_t=x["dst_t"][a:c], edge_t=x["edge_t"][ea:ec],
                                  Q=x["Q"][a:c], K=x["K"][ea:ec], V=x["V"][ea:ec], dO=x["dO"][a:c]))
    return shares


def cpu_baseline_threads(blocks, node_ids, edge_ids, node_table, edge_table, slot, om, ph,
                         scale, sample_edges, max_threads=16, passes=3):
    """The same oracle pass on all the host threads this process may use (at
    most `max_threads`): the per-destination operators (offsets, time encoding,
    fused attention fwd+bwd) of each layer block run over T disjoint
    contiguous segment ranges, one range per thread, beside the two
    dedup+gathers, which need the whole id list.  The oracle is unchanged:
    its C routines run outside the interpreter lock, and every segment's
    result depends on that segment's rows alone."""
    from concurrent.futures import ThreadPoolExecutor

    import oracle
    try:
        T = min(max_threads, len(os.sched_getaffinity(0)))
    except AttributeError:
        T = min(max_threads, os.cpu_count() or 1)
    oracle.lib()
    shares = segment_shares(blocks, T)

    def segments(share):
        offs = [oracle.csr_offsets(x["counts"]) for x in share]
        for x, off in zip(share, offs):
            oracle.time_encode(off, x["dst_t"], x["edge_t"], om, ph)
        for x, off in zip(share, offs):
            oracle.edge_attention_fwd(off, x["Q"], x["K"], x["V"], scale, SLOPE)
        for x, off in reversed(list(zip(share, offs))):
            oracle.edge_attention_bwd(off, x["Q"], x["K"], x["V"], x["dO"], scale, SLOPE)

    def rows(ids, table, sm):
        uni, _ = oracle.dedup(ids)
        oracle.gather(uni, table, sm)

    walls = []
    with ThreadPoolExecutor(max_workers=T) as pool:
        for _ in range(passes):
            t0 = time.perf_counter()
            futs = [pool.submit(rows, node_ids, node_table, None),
                    pool.submit(rows, edge_ids, edge_table, slot)]
            futs += [pool.submit(segments, sh) for sh in shares]
            for f in futs:
                f.result()
            walls.append(time.perf_counter() - t0)
    wall = float(np.median(walls))
    return {"value": sample_edges / wall, "unit": "sampled edges/s", "cores": T,
            "seconds_per_pass": round(wall, 3),
            "how": f"median of {passes} passes of the same sample: {T} threads over disjoint "
                   f"segment ranges plus the two dedup+gathers, unchanged oracle routines"}


CEILING_EXE = os.path.join(ROOT, "paper_2607_05095_amd", "probe", "stream_ceiling")


def stream_ceilings():
    """The GPU's streaming ceilings (read, write, copy, two-in-two-out) from
    the probe built beside the library, run as a child process before this
    process touches the GPU; None when the probe is not built."""
    import subprocess
    if not os.path.exists(CEILING_EXE):
        return None
    try:
        r = subprocess.run([CEILING_EXE], capture_output=True, text=True, timeout=180)
    except subprocess.TimeoutExpired:
        return {"error": "probe timed out"}
    if r.returncode != 0:
        return {"error": (r.stdout + r.stderr)[-300:]}
    return json.loads(r.stdout.strip().splitlines()[-1])


def ceiling_fracs(achieved_gbs, ceilings):
    """The dominant kernel's bandwidth as a fraction of each measured ceiling
    (plain and streaming loads/stores alike)."""
    if not ceilings or "copy" not in ceilings:
        return None
    return {k: round(achieved_gbs / (ceilings[k]["TB_per_s"] * 1e3), 4)
            for k in ("copy", "copy_nt", "mix22", "read", "read_nt", "write", "write_nt")
            if k in ceilings}


def read_counters(workload):
    """rocprofv3 counter record of the dominant kernel on this workload (HBM
    bytes per launch, L2 hit rate, occupancy), from the committed summary, or
    an empty dict when there is none for this workload or the kernel source
    changed since the counters were taken."""
    try:
        with open(TRAFFIC_FILE.format(workload=workload)) as f:
            t = json.load(f)
    except (OSError, ValueError):
        return {}
    if t.get("kernel_source_sha") != kernel_source_hash() or t.get("workload") != workload:
        return {}
    return t


def read_traffic(workload):
    """HBM bytes per launch of the dominant kernel, or None (see read_counters)."""
    return read_counters(workload).get("bytes_per_launch")


def measure(name, args, torch, fast, headline, ceilings=None):
    """Builds workload `name`, times K serial steps and the fused attention
    sequence, and returns its result dict.  The headline workload also gets
    the pipelined and graph timings and the widened operators."""
    from synth import make_batch
    b = make_batch(WORKLOADS[name])
    log(f"workload {b.name}: blocks {[(x.num_dst, x.num_edges) for x in b.blocks]}")
    step = Step(b, torch, fast, kv=args.kv)
    side = torch.cuda.Stream()
    torch.cuda.synchronize()
    for _ in range(args.warmup):
        step.run_serial()
    if headline and args.pipelined:
        step.run_pipelined(max(args.warmup, 1), side)
    torch.cuda.synchronize()
    log("warmup done")

    def timed(fn):
        s, e = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        torch.cuda.synchronize()
        s.record()
        fn()
        e.record()
        torch.cuda.synchronize()
        return s.elapsed_time(e) / args.steps

    # timed region: K whole steps, serial schedule; HIP events only around the
    # dominant kernel, on the stream it is launched on
    rec = {}
    dominant = ["attn_bwd_L1"]

    def serial_steps():
        for _ in range(args.steps):
            step.run_serial(rec, dominant)
    ms = timed(serial_steps)
    bwd_ms = float(np.mean([s.elapsed_time(e) for s, e in rec["attn_bwd_L1"]]))
    log(f"{name}: {ms:.3f} ms/step (serial)")
    # optionally, the same K steps software-pipelined over two streams
    ms_pipe = None
    if headline and args.pipelined:
        ms_pipe = timed(lambda: step.run_pipelined(args.steps, side))
        log(f"{ms_pipe:.3f} ms/step (pipelined)")

    # optionally, the serial step captured once as a HIP graph, replayed K times
    ms_graph = None
    if headline and args.graph:
        graph = torch.cuda.CUDAGraph()
        with torch.cuda.graph(graph):
            step.run_serial()
        graph.replay()
        torch.cuda.synchronize()
        ms_graph = timed(lambda: [graph.replay() for _ in range(args.steps)])
        log(f"{ms_graph:.3f} ms/step (graph replay)")

    # per-operator breakdown: separate serial steps, every operator timed
    rec_all = {}
    for _ in range(3):
        step.run_serial(rec_all)
    torch.cuda.synchronize()
    breakdown = {k: float(np.mean([s.elapsed_time(e) for s, e in v])) for k, v in rec_all.items()}
    dd = {}
    for kind, d in (("nodes", step.node[0]), ("edges", step.edge[0])):
        u, nm = int(d["nu"].item()), int(d["nm"].item())
        dd[kind] = (d["n"], u, u - nm)

    widened = None
    if headline:
        widened = widened_ops(b, step, torch, fast, with_oracle=not args.no_cpu_baseline)
        log(f"widened ops: {widened}")

    esz = 4 if b.dtype == "f32" else 2
    F = b.H * b.dh
    L1 = b.blocks[0]
    bwd_bytes = attn_bwd_bytes(L1.num_dst, L1.num_edges, F, esz, b.H)
    achieved = bwd_bytes / (bwd_ms * 1e-3) / 1e9
    fused_ms = attention_sequence_ms(step, torch)
    fused_bytes = sum(attn_fwd_bytes(x.num_dst, x.num_edges, F, esz, b.H) +
                      attn_bwd_bytes(x.num_dst, x.num_edges, F, esz, b.H) for x in b.blocks)
    fused_bytes_no_lse = sum((6 * x.num_edges + 5 * x.num_dst) * F * esz for x in b.blocks)
    counters = read_counters(name)
    roofline = {
        "kernel": "k_attn_bwd (fused ESM+AGG backward, layer-1 block)",
        "bound": "hbm", "achieved": round(achieved, 1), "peak": HBM_PEAK_GBS, "unit": "GB/s",
        "frac": round(achieved / HBM_PEAK_GBS, 4), "traffic": counters.get("bytes_per_launch"),
        "algorithmic_bytes_per_launch": bwd_bytes, "avg_launch_ms": round(bwd_ms, 4),
        "l2_hit_rate": counters.get("l2_hit_rate"),
        "occupancy_pct": counters.get("occupancy_pct"),
        "frac_of_measured_ceiling": ceiling_fracs(achieved, ceilings),
    }
    result = {
        "value": b.sampled_edges / (ms * 1e-3),
        "unit": "sampled edges/s",
        "ms_per_step": round(ms, 4),
        "dtype": b.dtype,
        "config": dict(describe(b), kv_layout=args.kv),
        "roofline": roofline,
        "fused_attention": {
            "edges_per_s": b.sampled_edges / (fused_ms * 1e-3), "ms": round(fused_ms, 4),
            "timing": "HIP events around the four launches (L1 fwd, L2 fwd, L2 bwd, L1 bwd), "
                      "5 warm-ups, median of 50",
            "algorithmic_bytes": fused_bytes,
            "hbm_frac": round(fused_bytes / (fused_ms * 1e-3) / 1e9 / HBM_PEAK_GBS, 4),
            "algorithmic_bytes_without_lse": fused_bytes_no_lse,
            "hbm_frac_without_lse": round(fused_bytes_no_lse / (fused_ms * 1e-3) / 1e9 / HBM_PEAK_GBS, 4),
        },
        "time_encode": time_encode_summary(b, breakdown, counters),
        "breakdown_ms": {k: round(v, 4) for k, v in breakdown.items()},
        "step_roofline": step_roofline(b, breakdown, ms, dd["nodes"], dd["edges"]),
    }
    if widened is not None:
        result["widened_ops"] = widened
    if ms_pipe is not None:
        result["pipelined"] = {
            "ms_per_step": round(ms_pipe, 4),
            "value": b.sampled_edges / (ms_pipe * 1e-3),
            "hbm_frac": round(result["step_roofline"]["algorithmic_bytes"] / (ms_pipe * 1e-3) / 1e9
                              / HBM_PEAK_GBS, 4),
            "schedule": "prep of batch i+1 on a second stream overlaps attention of batch i; "
                        "attention(i) waits for prep(i); double-buffered prep outputs",
        }
    if ms_graph is not None:
        result["graph"] = {
            "ms_per_step": round(ms_graph, 4),
            "value": b.sampled_edges / (ms_graph * 1e-3),
            "schedule": "the serial step captured once as a HIP graph, replayed K times",
        }
    if not args.no_cpu_baseline:
        log(f"{name}: cpu baseline (oracle) ...")
        cb = cpu_baseline(b, step, torch, args.cpu_frac)
        cb["gpu_over_cpu"] = round(result["value"] / cb["value"], 1)
        cb["all_cores"]["gpu_over_cpu"] = round(result["value"] / cb["all_cores"]["value"], 1)
        result["cpu_baseline"] = cb
    del step
    return result


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--warmup", type=int, default=10)
    ap.add_argument("--workload", choices=sorted(WORKLOADS), default="bigdedup",
                    help="the headline workload of the line")
    ap.add_argument("--also", default=None,
                    help="comma-separated workloads measured after the headline one, each under "
                         "its own key (default: large when the headline is bigdedup; 'none' "
                         "measures the headline only)")
    ap.add_argument("--cpu-frac", type=float, default=1.0)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-pipelined", dest="pipelined", action="store_false",
                    help="skip the second timing of the steps software-pipelined over two streams")
    ap.add_argument("--graph", action="store_true",
                    help="also time the serial step captured once as a HIP graph and replayed")
    ap.add_argument("--copy-calibration", action="store_true",
                    help="only run a plain 1 GiB device copy (counter calibration)")
    ap.add_argument("--kv", choices=["packed", "separate"], default="packed",
                    help="layout of the attention's per-edge K and V rows (and their gradients): "
                         "one packed [E, 2, H, dh] array, or separate [E, H, dh] arrays")
    ap.add_argument("--no-ceilings", action="store_true",
                    help="skip the streaming-ceiling probe (it runs as a child process before this "
                         "process touches the GPU; profilers that initialise the GPU first need this)")
    args = ap.parse_args()
    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        print(json.dumps({"error": "bench.py runs on one GPU only; the multi-GPU sharding "
                                   "design is described but not built", "n_gpus": args.gpus}))
        sys.exit(2)
    if args.also is None:
        also = ["large"] if args.workload == "bigdedup" else []
    else:
        also = [w for w in args.also.split(",") if w and w != "none"]
    for w in also:
        if w not in WORKLOADS or w == args.workload:
            ap.error(f"--also: unknown or repeated workload {w!r}")

    # streaming ceilings of this GPU, before this process initialises it
    ceilings = None if (args.copy_calibration or args.no_ceilings) else stream_ceilings()

    import torch
    import paper_2607_05095_amd as fast

    if args.copy_calibration:
        x = torch.empty(1 << 28, dtype=torch.float32, device="cuda").fill_(1.0)
        y = torch.empty_like(x)
        for _ in range(5):
            y.copy_(x)
        torch.cuda.synchronize()
        print(json.dumps({"copy_bytes_each_way": x.numel() * 4, "copies": 5}))
        return

    head = measure(args.workload, args, torch, fast, headline=True, ceilings=ceilings)
    result = {
        "metric": METRIC,
        "value": head.pop("value"),
        "unit": head.pop("unit"),
        "n_gpus": 1, "steps": args.steps, "warmup": args.warmup,
        "ms_per_step": head.pop("ms_per_step"),
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
        "dtype": head.pop("dtype"), "data": "synthetic",
        "config": head.pop("config"),
    }
    cb = head.pop("cpu_baseline", None)
    result.update(head)
    result.update({
        "schedule": "serial: prep (offsets, time encoding, dedup+gather) then attention of each "
                    "batch on one stream",
        "widened_note": "operators beyond the timed step, timed alone outside the timed region; "
                        "with the CPU baseline, each also gives the oracle's rate on a bounded sample",
        "breakdown_note": "operators timed one by one in 3 extra serial steps outside the timed region",
        "kernel_source_sha": kernel_source_hash(),
        "paper_context": PAPER_CONTEXT,
    })
    if cb is not None:
        result["cpu_baseline"] = cb
    result["stream_ceilings"] = ceilings
    result["stream_ceilings_note"] = (
        "plain read / write / copy / two-in-two-out kernels over 2 GiB buffers on this GPU, one "
        "16-byte element per thread, and read / write / copy with streaming (non-temporal) loads "
        "and stores (_nt) (paper_2607_05095_amd/probe/stream_ceiling.hip), median of "
        "15 launches; roofline.frac_of_measured_ceiling divides the dominant kernel's bandwidth by them")
    for w in also:
        torch.cuda.synchronize()
        torch.cuda.empty_cache()
        r = measure(w, args, torch, fast, headline=False, ceilings=ceilings)
        r["note"] = ("measured in the same run after the headline workload's buffers were freed: "
                     "K serial steps, the fused attention sequence, the dominant kernel's roofline "
                     "and the oracle on the same batch")
        result[w] = r
    print(json.dumps(result), flush=True)


if __name__ == "__main__":
    main()
