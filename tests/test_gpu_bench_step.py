"""The benchmark's timed step computes the hot path correctly: one serial step
of bench.Step on small workloads against the oracle (offsets, dedup + gather
of node and edge rows, time encoding, fused attention forward and backward
of both layer blocks), and the two-stream pipelined schedule leaves bitwise
the same results as the serial one (every kernel is deterministic)."""
import os
import sys

import numpy as np
import pytest
import torch

import oracle
import paper_2607_05095_amd as fast
from synth import make_batch, omega_phi
from tests.parity import (SLOPE, assert_bwd_close, assert_close, bwd_reference_with_kinks,
                          check_attention_block_full, check_time_encode_full)

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)
import bench  # noqa: E402

pytestmark = pytest.mark.gpu


def _host(t):
    return t.detach().float().cpu().double().numpy()


def _snapshot(step, slot):
    snap = []
    for d in step.blocks:
        snap += [d["off"][slot], d["te"][slot], d["out"], d["lse"], d["dQ"], d["dK"], d["dV"]]
    for x in (step.node[slot], step.edge[slot]):
        u = int(x["nu"].item())                 # only the first u entries are written
        snap += [x["uni"][:u], x["inv"], x["nu"], x["rows"][:u], x["nm"]]
    return [t.clone() for t in snap]


@pytest.mark.parametrize("cfg", [0, 2])
def test_bench_step_matches_the_oracle(cfg):
    print(f"[parity] bench step cfg={cfg}", flush=True)
    b = make_batch(cfg)
    step = bench.Step(b, torch, fast)
    step.run_serial()
    torch.cuda.synchronize()
    om, ph = omega_phi(b.d_t)
    for i, (blk, d) in enumerate(zip(b.blocks, step.blocks)):
        what = f"cfg{cfg}/L{i + 1}"
        off = oracle.csr_offsets(blk.counts)
        assert np.array_equal(d["off"][0].cpu().numpy(), off), what + " offsets"
        te = oracle.time_encode(off, blk.dst_t, blk.edge_t, om, ph)
        assert_close(d["te"][0], te, b.dtype, what + " time encoding")
        Q, K, V, dO = (_host(d[k]) for k in ("Q", "K", "V", "dO"))
        out, lse, _, _ = oracle.edge_attention_fwd(off, Q, K, V, step.scale, SLOPE)
        assert_close(d["out"], out, b.dtype, what + " out")
        nz = np.diff(off) > 0
        assert_close(_host(d["lse"])[nz], lse[nz], "f32", what + " lse")
        dQ, dK, dV, alts = bwd_reference_with_kinks(off, Q, K, V, dO, step.scale, SLOPE)
        assert_close(d["dV"], dV, b.dtype, what + " dV")
        assert_bwd_close(d["dQ"], d["dK"], off, dQ, dK, alts, b.dtype, what)
    for name, ids, x in (("nodes", b.node_ids, step.node[0]), ("edges", b.edge_ids, step.edge[0])):
        uni, inv = oracle.dedup(ids)
        u = int(x["nu"].item())
        assert u == uni.size and np.array_equal(x["uni"][:u].cpu().numpy(), uni), name
        assert np.array_equal(x["inv"].cpu().numpy(), inv), name
        table = x["table"].cpu().numpy() if b.dtype == "f32" else x["table"].view(torch.int16).cpu().numpy()
        slot = None if x["slot"] is None else x["slot"].cpu().numpy()
        rows, hit, miss = oracle.gather(uni, table, slot)
        got = x["rows"][:u].cpu().numpy() if b.dtype == "f32" else x["rows"][:u].view(torch.int16).cpu().numpy()
        assert np.array_equal(got[hit], rows[hit]), name + " rows"
        assert int(x["nm"].item()) == miss.size, name + " misses"


@pytest.mark.parametrize("workload", ["bigdedup", "large"])
def test_bench_step_full_size_matches_the_oracle(workload):
    """The step the benchmark times, at its full size: one serial step of
    bench.Step, then every output of it against the oracle -- offsets and
    dedup + gather bit-exact, the time encoding row by row and the fused
    attention segment by segment over ranges on all host threads."""
    b = make_batch(bench.WORKLOADS[workload])
    print(f"[parity] bench step {workload} (full size)", flush=True)
    step = bench.Step(b, torch, fast)
    step.run_serial()
    torch.cuda.synchronize()
    om, ph = omega_phi(b.d_t)
    for i, (blk, d) in enumerate(zip(b.blocks, step.blocks)):
        what = f"{workload}/L{i + 1}"
        print(f"[parity]   {what}: N={blk.num_dst} E={blk.num_edges}", flush=True)
        off = oracle.csr_offsets(blk.counts)
        assert np.array_equal(d["off"][0].cpu().numpy(), off), what + " offsets"
        check_time_encode_full(off, blk.dst_t, blk.edge_t, om, ph, d["te"][0].cpu(), b.dtype,
                               what + " time encoding")
        ins = {k: d[k].cpu() for k in ("Q", "K", "V", "dO")}
        outs = [d[k].cpu() for k in ("out", "lse", "dQ", "dK", "dV")]
        check_attention_block_full(off, ins, outs, None, None, step.scale, SLOPE, b.dtype,
                                   what + " attention")
        del ins, outs
    for name, ids, x in (("nodes", b.node_ids, step.node[0]), ("edges", b.edge_ids, step.edge[0])):
        print(f"[parity]   {workload} dedup + gather of {name}: n={ids.size}", flush=True)
        uni, inv = oracle.dedup(ids)
        u = int(x["nu"].item())
        assert u == uni.size and np.array_equal(x["uni"][:u].cpu().numpy(), uni), name
        assert np.array_equal(x["inv"].cpu().numpy(), inv), name
        bits = torch.int32 if b.dtype == "f32" else torch.int16
        slot = None if x["slot"] is None else x["slot"].cpu().numpy()
        rows, hit, miss = oracle.gather(uni, x["table"].view(bits).cpu().numpy(), slot)
        got = x["rows"][:u].view(bits).cpu().numpy()
        assert np.array_equal(got[hit], rows[hit]), name + " rows"
        m = int(x["nm"].item())
        assert m == miss.size and np.array_equal(x["miss"][:m].cpu().numpy(), miss), name + " misses"
    del step
    torch.cuda.empty_cache()


def test_pipelined_schedule_leaves_the_serial_results():
    print("[parity] bench pipelined vs serial", flush=True)
    b = make_batch(2)
    step = bench.Step(b, torch, fast)
    step.run_serial()
    torch.cuda.synchronize()
    serial = _snapshot(step, 0)
    for x in step.blocks:                      # poison the shared outputs
        for k in ("out", "dQ", "dK", "dV"):
            x[k].fill_(float("nan"))
    side = torch.cuda.Stream()
    step.run_pipelined(3, side)                 # batches 0, 1, 2 use slots 0, 1, 0
    torch.cuda.synchronize()
    piped = _snapshot(step, 0)
    for a, c in zip(serial, piped):
        assert torch.equal(a, c)
    piped1 = _snapshot(step, 1)
    for a, c in zip(serial, piped1):
        assert torch.equal(a, c)


@pytest.mark.parametrize("cfg", [0, 2])
def test_graph_replays_match_the_eager_step(cfg):
    """One step captured as a HIP graph (every call takes caller buffers and
    enqueues only kernels: no allocation, synchronisation or memset) gives
    bitwise the eager step's results on every replay, with eager work and
    synchronisations between the replays."""
    print(f"[parity] bench step as a graph cfg={cfg}", flush=True)
    b = make_batch(cfg)
    step = bench.Step(b, torch, fast)
    step.run_serial()
    torch.cuda.synchronize()
    eager = _snapshot(step, 0)
    graph = torch.cuda.CUDAGraph()
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        step.run_serial()                       # warm-up on the capture stream
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    with torch.cuda.graph(graph):
        step.run_serial()
    for rep in range(3):
        for x in step.blocks:                   # poison, eagerly, between replays
            for k in ("out", "dQ", "dK", "dV"):
                x[k].fill_(float("nan"))
            x["te"][0].fill_(float("nan"))
        for x in (step.node[0], step.edge[0]):
            x["rows"].fill_(float("nan"))
            x["uni"].fill_(-7)
        torch.cuda.synchronize()
        graph.replay()
        torch.cuda.synchronize()
        for a, c in zip(eager, _snapshot(step, 0)):
            assert torch.equal(a, c), f"replay {rep}"
