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


def test_counter_records_are_whole_and_checked_against_the_source(tmp_path, monkeypatch):
    sys.path.insert(0, ROOT)
    import bench
    for w in ("bigdedup", "large"):
        with open(bench.TRAFFIC_FILE.format(workload=w)) as f:
            rec = json.load(f)
        assert rec["workload"] == w
        assert 0 < rec["l2_hit_rate"] < 1 and 0 < rec["occupancy_pct"] <= 100
        assert rec["bytes_per_launch"] > 0 and os.path.exists(os.path.join(ROOT, rec["source"]))
        # a record taken on other kernel sources is not reported
        stale = dict(rec, kernel_source_sha="0" * 16)
        (tmp_path / f"t_{w}.json").write_text(json.dumps(stale))
    monkeypatch.setattr(bench, "TRAFFIC_FILE", str(tmp_path / "t_{workload}.json"))
    assert bench.read_counters("bigdedup") == {} and bench.read_traffic("large") is None
