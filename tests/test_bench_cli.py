"""bench.py's contract on the CPU: a multi-GPU request exits with a message."""
import json
import os
import subprocess
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def test_multi_gpu_request_is_refused():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"],
                       capture_output=True, text=True, timeout=120)
    assert r.returncode == 2
    msg = json.loads(r.stdout.strip().splitlines()[-1])
    assert "one GPU" in msg["error"]


def test_byte_models_match_the_design_figures():
    sys.path.insert(0, ROOT)
    import bench
    # fused backward of the bigdedup layer-1 block (N=264,000, E=2,640,000, F=100, fp32, H=2)
    assert bench.attn_bwd_bytes(264_000, 2_640_000, 100, 4, 2) == 4_543_968_004
    # (6E + 5N) F b for fwd+bwd of both blocks, plus lse and offsets
    fb = sum(bench.attn_fwd_bytes(n, e, 100, 4, 2) + bench.attn_bwd_bytes(n, e, 100, 4, 2)
             for n, e in ((264_000, 2_640_000), (24_000, 240_000)))
    assert abs(fb - 7_488_000_000) / 7_488_000_000 < 0.001


def test_step_byte_models():
    """The prep operators' byte models on the 1e7-node batch: node ids read
    their 400-byte rows straight from the table, edge ids through the cache's
    slot map (291,717 of 541,340 distinct ids cached)."""
    sys.path.insert(0, ROOT)
    import bench
    assert bench.offsets_bytes(264_000) == 2_112_004
    assert bench.dedup_gather_bytes(2_664_000, 413_064, 413_064, 400, False) == \
        12 * 2_664_000 + 413_064 * (8 + 800)
    assert bench.dedup_gather_bytes(2_640_000, 541_340, 291_717, 688, True) == \
        12 * 2_640_000 + 541_340 * 12 + 291_717 * 1376 + (541_340 - 291_717) * 4
    from synth import make_batch
    b = make_batch(0)
    n_ids, e_ids = int(b.node_ids.size), int(b.edge_ids.size)
    rec = bench.step_roofline(b, {"attn_bwd_L1": 0.5}, 2.0, (n_ids, 10, 10), (e_ids, 20, 15))
    ops = rec["operators"]
    assert rec["algorithmic_bytes"] == sum(o["bytes"] for o in ops.values())
    assert set(ops) == {"offsets", "time_encode", "dedup_gather_nodes", "dedup_gather_edges"} | \
        {f"attn_{d}_L{i + 1}" for d in ("fwd", "bwd") for i in range(len(b.blocks))}
    F, esz = b.H * b.dh, 4 if b.dtype == "f32" else 2
    L1 = b.blocks[0]
    assert ops["attn_bwd_L1"]["bytes"] == bench.attn_bwd_bytes(L1.num_dst, L1.num_edges, F, esz, b.H)
    assert abs(ops["attn_bwd_L1"]["hbm_frac"] - ops["attn_bwd_L1"]["bytes"] / 0.5e-3 / 8e12) < 1e-4
    assert ops["offsets"]["hbm_frac"] is None                      # no time recorded
    assert abs(rec["hbm_frac"] - rec["algorithmic_bytes"] / 2e-3 / 8e12) < 1e-4


def test_counter_records_are_whole_and_checked_against_the_source(tmp_path, monkeypatch):
    sys.path.insert(0, ROOT)
    import bench
    for w in ("bigdedup", "large"):
        with open(bench.TRAFFIC_FILE.format(workload=w)) as f:
            rec = json.load(f)
        assert rec["workload"] == w
        assert 0 < rec["l2_hit_rate"] < 1 and 0 < rec["occupancy_pct"] <= 100
        assert rec["bytes_per_launch"] > 0 and os.path.exists(os.path.join(ROOT, rec["source"]))
        te = rec["time_encode_valu"]
        assert te["valu_wave_insts_per_launch"] > 0
        assert "k_time_encode<" in te["kernel"] or "k_time_encode_batch<" in te["kernel"]
        # a record taken on other kernel sources is not reported
        stale = dict(rec, kernel_source_sha="0" * 16)
        (tmp_path / f"t_{w}.json").write_text(json.dumps(stale))
    monkeypatch.setattr(bench, "TRAFFIC_FILE", str(tmp_path / "t_{workload}.json"))
    assert bench.read_counters("bigdedup") == {} and bench.read_traffic("large") is None


def test_segment_shares_recompose_the_whole_block():
    """The all-cores CPU baseline runs the oracle over contiguous segment
    ranges; the ranges' results, concatenated, are the whole block's."""
    import numpy as np

    import bench
    import oracle
    from synth import make_batch
    b = make_batch(2)
    blk = b.blocks[0]
    N, E = blk.num_dst, int(blk.counts.sum())
    r = np.random.default_rng(5)
    x = dict(counts=blk.counts, dst_t=blk.dst_t, edge_t=blk.edge_t,
             Q=r.standard_normal((N, 2, 8)), K=r.standard_normal((E, 2, 8)),
             V=r.standard_normal((E, 2, 8)), dO=r.standard_normal((N, 2, 8)))
    shares = bench.segment_shares([x], 5)
    assert sum(int(sh[0]["counts"].sum()) for sh in shares) == E
    off = oracle.csr_offsets(blk.counts)
    out, lse, _, _ = oracle.edge_attention_fwd(off, x["Q"], x["K"], x["V"], 0.3, 0.2)
    dQ, dK, dV = oracle.edge_attention_bwd(off, x["Q"], x["K"], x["V"], x["dO"], 0.3, 0.2)
    parts = []
    for sh in shares:
        y = sh[0]
        o = oracle.csr_offsets(y["counts"])
        parts.append(oracle.edge_attention_fwd(o, y["Q"], y["K"], y["V"], 0.3, 0.2)[0:1]
                     + oracle.edge_attention_bwd(o, y["Q"], y["K"], y["V"], y["dO"], 0.3, 0.2))
    for k, ref in enumerate((out, dQ, dK, dV)):
        assert np.array_equal(np.concatenate([p[k] for p in parts]), ref)


def test_time_encode_valu_only_from_counters_of_the_current_source():
    sys.path.insert(0, ROOT)
    import bench
    from synth import make_batch
    b = make_batch(4)
    bd = {"time_encode": 0.2}
    rec = {"time_encode_valu": {"valu_wave_insts_per_launch": 5.6e7, "source": "x",
                                "source_sha": bench.source_hash(bench.TIME_ENCODE_SOURCES)}}
    v = bench.time_encode_summary(b, bd, rec)["valu"]
    assert abs(v["lane_insts_per_s"] - 5.6e7 * 64 / 2e-4) < 1 and 0 < v["frac"] < 1
    rec["time_encode_valu"]["source_sha"] = "0" * 16
    assert "valu" not in bench.time_encode_summary(b, bd, rec)


def test_ceiling_fractions_cover_plain_and_streaming_probes():
    """The dominant kernel's bandwidth is set against every ceiling the probe
    reports, the streaming (non-temporal) ones included, and an older probe
    output without them still gives the plain fractions."""
    import bench
    tb = {"read": 6.7, "write": 6.7, "copy": 6.1, "mix22": 5.7, "read_nt": 7.0, "write_nt": 6.6,
          "copy_nt": 6.4}
    full = {k: {"TB_per_s": v} for k, v in tb.items()}
    fr = bench.ceiling_fracs(5720.0, full)
    assert set(fr) == set(tb)
    assert fr["copy_nt"] == round(5720.0 / 6400.0, 4) and fr["copy"] == round(5720.0 / 6100.0, 4)
    plain = {k: v for k, v in full.items() if not k.endswith("_nt")}
    assert set(bench.ceiling_fracs(5720.0, plain)) == {"read", "write", "copy", "mix22"}
    assert bench.ceiling_fracs(5720.0, None) is None
    assert bench.ceiling_fracs(5720.0, {"error": "probe timed out"}) is None
