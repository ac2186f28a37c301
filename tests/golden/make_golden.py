"""Writes tiny_oracle.json: oracle outputs on a small hand-sized graph.

Calls only the oracle (and the seeded generators for the inputs).  Run from
the repository root: python tests/golden/make_golden.py
"""
import json
import os
import sys

import numpy as np

ROOT = os.path.dirname(os.path.dirname(os.path.dirname(os.path.abspath(__file__))))
sys.path.insert(0, ROOT)

import oracle  # noqa: E402

HERE = os.path.dirname(os.path.abspath(__file__))


def inputs():
    r = np.random.default_rng(20260)
    counts = np.array([3, 0, 1, 4, 2], dtype=np.int32)
    E, N, H, dh = int(counts.sum()), counts.size, 2, 3
    return dict(
        counts=counts,
        Q=np.round(r.standard_normal((N, H, dh)), 3),
        K=np.round(r.standard_normal((E, H, dh)), 3),
        V=np.round(r.standard_normal((E, H, dh)), 3),
        dO=np.round(r.standard_normal((N, H, dh)), 3),
        dst_t=np.array([10.0, 20.0, 30.0, 40.0, 50.0], dtype=np.float32),
        edge_t=np.array([1.0, 2.5, 9.0, 29.0, 0.5, 12.0, 39.0, 40.0, 7.0, 49.5], dtype=np.float32),
        omega=np.array([1.0, 0.1, 0.01, 0.001], dtype=np.float32),
        phi=np.zeros(4, dtype=np.float32),
        ids=np.array([7, 3, 7, 11, 3, 3, 0, 42, 11, 7], dtype=np.int64),
        scale=0.5, slope=0.2,
    )


def outputs(x):
    off = oracle.csr_offsets(x["counts"])
    out, lse, alpha, _ = oracle.edge_attention_fwd(off, x["Q"], x["K"], x["V"], x["scale"], x["slope"])
    dQ, dK, dV = oracle.edge_attention_bwd(off, x["Q"], x["K"], x["V"], x["dO"], x["scale"], x["slope"])
    te = oracle.time_encode(off, x["dst_t"], x["edge_t"], x["omega"], x["phi"])
    uni, inv = oracle.dedup(x["ids"])
    return dict(off=off, out=out, lse=lse, alpha=alpha, dQ=dQ, dK=dK, dV=dV, te=te, uni=uni, inv=inv)


if __name__ == "__main__":
    o = outputs(inputs())
    with open(os.path.join(HERE, "tiny_oracle.json"), "w") as f:
        json.dump({k: np.asarray(v).tolist() for k, v in o.items()}, f, indent=1)
    print("wrote tiny_oracle.json")
