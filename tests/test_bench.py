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


def test_kernel_rooflines_closed_forms():
    import bench
    from workloads import get_workload
    wl = get_workload("wide")
    counts = [wl.T * wl.k // wl.N] * wl.N
    P, D, H, e = wl.T * wl.k, wl.D, wl.H, 2
    dw = bench.kernel_algorithmic("grouped_gemm2<GM=1,AT=1,BT=1,EPI=0,256x256,ST=2,BK=64>", wl, counts)
    assert dw[0] == "expert weight-gradient GEMM" and dw[1] == 2 * P * D * H
    # reads both row operands once and writes every expert's gradient once
    assert dw[2] == P * (D + H) * e + wl.N * D * H * e
    up = bench.kernel_algorithmic("grouped_gemm2<GM=0,AT=0,BT=0,EPI=2,256x256,ST=2,BK=64>", wl, counts)
    assert up[1] == 2 * P * D * H and up[2] == wl.N * (D * H + H) * e + P * (D + 2 * H) * e
    # the per-launch flops of the five GEMM kinds of one step add up to the call totals
    names = ["grouped_gemm2<GM=0,AT=0,BT=0,EPI=2", "grouped_gemm2<GM=0,AT=0,BT=0,EPI=1",
             "grouped_gemm2<GM=0,AT=0,BT=1,EPI=3", "grouped_gemm2<GM=0,AT=0,BT=1,EPI=0"]
    fl = sum(bench.kernel_algorithmic(n, wl, counts)[1] for n in names) + 2 * dw[1]
    a = bench.algorithmic(wl, counts)
    assert fl == a["ffn_fwd"]["flops"] + a["ffn_bwd"]["flops"]
    r = bench.roofline_of(dw[1], dw[2], 0.02, bench.PEAK_BF16_TFLOPS)
    assert r["bound"] == "mfma" and abs(r["achieved"] - dw[1] / 0.02 / 1e12) < 0.1


def test_block_kernel_rooflines_closed_forms():
    """The LayerNorm block layer's per-launch figures: each GEMM kind is launched once per
    linear layer, so three launches of the three kinds add up to the call totals, and the
    LayerNorm row kernels move each [rows, F] tensor once."""
    import bench
    from workloads import get_workload
    wl = get_workload("ffblock")
    counts = [wl.T * wl.k // wl.N] * wl.N
    P, D, F, e = wl.T * wl.k, wl.D, wl.H, 2
    b = bench.algorithmic_block(wl, counts)
    fwd = bench.kernel_algorithmic("grouped_gemm2<GM=0,AT=0,BT=0,EPI=1,288x256,ST=2,BK=64,XB>", wl, counts)
    dgr = bench.kernel_algorithmic("grouped_gemm2<GM=0,AT=0,BT=1,EPI=0,288x256,ST=2,BK=64,XB>", wl, counts)
    wgr = bench.kernel_algorithmic("grouped_gemm2<GM=1,AT=1,BT=1,EPI=0,256x256,ST=2,BK=64>", wl, counts)
    assert 3 * fwd[1] == b["ffn_fwd"]["flops"]
    assert 3 * (dgr[1] + wgr[1]) == b["ffn_bwd"]["flops"]
    # weight gradients: both row operands once, every expert's gradient written once
    assert 3 * wgr[2] == P * (2 * D + 2 * F + 2 * F) * e + wl.N * (2 * D * F + F * F) * e
    ln = bench.kernel_algorithmic("(ln_act_fwd_kernel<E, 8, ACT>)", wl, counts)
    assert ln[1] == 0 and ln[2] == 2 * P * F * e + 8 * P + 2 * wl.N * F * e
    r = bench.roofline_of(ln[1], ln[2], 1e-3, bench.PEAK_BF16_TFLOPS)
    assert r["bound"] == "hbm"
