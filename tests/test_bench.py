"""bench.py's contract on the host: one GPU only, and the algorithmic bytes and flops
it divides by (closed forms of the layer's data movement and contractions)."""
import os
import subprocess
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)


def test_more_than_one_gpu_is_refused():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"], capture_output=True,
                       text=True, timeout=120)
    assert r.returncode == 2
    assert "one GPU" in r.stderr


def test_algorithmic_counts_closed_forms():
    import bench
    from workloads import get_workload
    wl = get_workload("wide")
    counts = [wl.T * wl.k // wl.N] * wl.N          # every expert 512 rows
    a = bench.algorithmic(wl, counts)
    P, D, H, e = wl.T * wl.k, wl.D, wl.H, 2
    assert a["ffn_fwd"]["flops"] == 4 * P * D * H
    assert a["ffn_bwd"]["flops"] == 8 * P * D * H
    assert a["gate_topk"]["bytes"] == wl.T * D * e + wl.dM * D * e + wl.T * wl.k * 12
    # dispatch reads x once and writes every pair's row once
    assert a["dispatch"]["bytes"] == wl.T * D * e + P * D * e + wl.T * wl.k * 12
    # recompute adds one up-projection pass: 2 P D H flops
    r = bench.algorithmic(wl, counts, recompute=True)
    assert r["ffn_bwd"]["flops"] - a["ffn_bwd"]["flops"] == 2 * P * D * H
    # experts without rows carry no weight traffic
    half = [c if i % 2 == 0 else 0 for i, c in enumerate(counts)]
    h = bench.algorithmic(wl, half)
    wbytes = wl.N * (2 * D * H + H + D) * e
    assert a["ffn_fwd"]["bytes"] - h["ffn_fwd"]["bytes"] == wbytes // 2 + (P // 2) * (D * e + 3 * H * e + D * e)


def test_block_workload_flops():
    import bench
    from workloads import get_workload
    wl = get_workload("ffblock")
    counts = [wl.T * wl.k // wl.N] * wl.N
    b = bench.algorithmic_block(wl, counts)
    P, D, F = wl.T * wl.k, wl.D, wl.H
    # three linear layers D->F, F->F, F->D: 2 P (D F + F F + F D) flops forward
    assert b["ffn_fwd"]["flops"] == 2 * P * (2 * D * F + F * F)
    assert b["ffn_bwd"]["flops"] == 2 * b["ffn_fwd"]["flops"]
