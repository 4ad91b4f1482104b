#!/usr/bin/env python3
"""Benchmark of one DMoE layer, forward + backward, on one MI355X.

    python bench.py [--gpus 1] [--steps K] [--warmup W] [--workload wide] [--no-extra]

A step is one pass of the whole layer over one batch of synthetic input:
gate + TopK + weights, dispatch, expert FFN forward, combine, and the backward of
all of them (combine, gate, expert FFN, dispatch).  Inputs and weights are
resident in HBM before the timed region.  Prints one JSON line.

Inside the timed region every kernel the library enqueues is timed with HIP events
on its stream (the library's launch trace), so the line reports each kernel's
per-launch duration and roofline fraction and names the kernel that takes the most
time per step.  After the timed region a cold pass flushes the memory-side cache
before each step and times the gate and the dispatch again.  The other workloads
(1024- and 4096-expert layers, the LayerNorm block experts, the tiny fp32 layer)
are then timed for a few steps each and reported under "workloads".
"""
import argparse
import gc
import json
import os
import re
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

METRIC = "DMoE layer fwd+bwd tokens/sec on 1 MI355X; expert-GEMM MFMA util %; gate HBM GB/s"
PEAK_BF16_TFLOPS = 2516.6      # MI355X dense bf16 MFMA
PEAK_F32_TFLOPS = 157.3
PEAK_HBM_GBS = 8000.0
CALLS = ("gate_topk", "dispatch", "ffn_fwd", "combine", "combine_bwd", "gate_topk_bwd", "ffn_bwd",
         "dispatch_bwd")
FWD_CALLS = ("gate_topk", "dispatch", "ffn_fwd", "combine")
EXTRA_WORKLOADS = ("tfm_fwd", "tfm_fail_skew", "grid3d", "ffblock", "tiny_f32")
COLD_WORKLOADS = ("wide", "grid3d")
FLUSH_BYTES = 1 << 30          # memory-side cache flush: 1 GiB written, then 1 GiB read

# The paper's own throughput figure, reported beside the result as context only: it is
# system-level training over the internet, not a single-GPU layer measurement.
PAPER_CONTEXT = {
    "value": "300.8 +- 15.9 samples/s",
    "what": ("Learning@home training throughput, 224 feed-forward blocks 1024-4096-4096-1024 with "
             "LayerNorm and ReLU, batch 2048, 64 trainers (Sec. 4.1, Table 2)"),
    "hardware": "3 cloud Tesla K80 instances in three regions, network latency 92.49 +- 32.42 ms",
    "model_parallel_same_setup": "7.23 +- 0.06 samples/s",
    "note": "context, not the target: a different machine, precision and measurement",
}


def algorithmic(wl, counts, recompute=False, sgd=False):
    """Algorithmic bytes and flops per call (what the method must move/compute)."""
    e = 2 if wl.dtype == "bf16" else 4
    T, D, H, dM, k = wl.T, wl.D, wl.H, wl.dM, wl.k
    rows = int(sum(counts))
    touched = int(sum(1 for c in counts if c > 0))
    wbytes = touched * (2 * D * H + H + D) * e
    out = {}
    out["gate_topk"] = dict(bytes=T * D * e + dM * D * e + T * k * 12, flops=2 * T * D * dM)
    out["dispatch"] = dict(bytes=T * D * e + rows * D * e + T * k * 12, flops=0)
    out["ffn_fwd"] = dict(bytes=wbytes + rows * (D * e + 3 * H * e + D * e), flops=4 * rows * D * H)
    out["combine"] = dict(bytes=rows * D * e + T * D * e, flops=2 * rows * D)
    out["combine_bwd"] = dict(bytes=T * D * e + 2 * rows * D * e, flops=4 * rows * D)
    out["gate_topk_bwd"] = dict(bytes=T * D * e + dM * D * e, flops=2 * T * D * dM)
    # dh: read dy_perm, W2, h; write dh.  dW2: read dy_perm, a; write dW2.
    # dx_perm: read dh, W1; write dx_perm.  dW1: read dh, x_perm; write dW1.
    out["ffn_bwd"] = dict(bytes=2 * wbytes + rows * (D * e + 2 * H * e) + rows * (D * e + H * e)
                          + rows * (H * e + D * e) + rows * (H * e + D * e), flops=8 * rows * D * H)
    if sgd:         # weight tiles read and written instead of dW written
        out["ffn_bwd"]["bytes"] += wbytes // 2
    if recompute:   # up-projection again: read x_perm and W1, write h and a
        out["ffn_bwd"]["bytes"] += wbytes // 2 + rows * (D * e + 2 * H * e)
        out["ffn_bwd"]["flops"] += 2 * rows * D * H
    out["dispatch_bwd"] = dict(bytes=rows * D * e + T * D * e + T * k * dM * 0, flops=0)
    return out


def algorithmic_block(wl, counts):
    """Algorithmic bytes and flops of the block-expert calls (Linear, LayerNorm+act,
    Linear, LayerNorm+act, Linear per expert): each weight read once per pass (twice in
    the backward: data and weight gradients) and each gradient written once; every
    row tensor read or written once per step that uses it."""
    e = 2 if wl.dtype == "bf16" else 4
    D, F = wl.D, wl.H
    rows = int(sum(counts))
    touched = int(sum(1 for c in counts if c > 0))
    wbytes = touched * (2 * D * F + F * F + 6 * F + D) * e
    flops = 2 * rows * F * (2 * D + F)
    # fwd rows: GEMM1 x->h1, LN1 h1->a1 (+stats), GEMM2 a1->h2, LN2 h2->a2, GEMM3 a2->y
    fwd_rows = rows * ((2 * D + 8 * F) * e + 16)
    # bwd rows: dW3 (dy, a2), da2 (dy -> g2), db3 (dy), LN2 bwd (g2, h2 twice; g2 out),
    # db2, dW2 (g2, a1), da1 (g2 -> g1), LN1 bwd, db1, dW1 (g1, x), dx (g1 -> dx)
    bwd_rows = rows * ((5 * D + 21 * F) * e + 32)
    return {"ffn_fwd": dict(bytes=wbytes + fwd_rows, flops=flops),
            "ffn_bwd": dict(bytes=3 * wbytes + bwd_rows, flops=2 * flops)}


_GEMM2 = re.compile(r"grouped_gemm2<GM=(\d),AT=(\d),BT=(\d),EPI=(\d)")


def kernel_algorithmic(name, wl, counts, sgd=False):
    """(role, flops, bytes) of one launch of kernel `name`, or None for kernels without a
    per-launch closed form here.  A grouped GEMM launch multiplies every alive pair's row
    once (2 rows n_in n_out flops) and reads each touched expert's weight matrix once;
    the per-row operands and outputs are read or written once.  The LayerNorm block
    launches each GEMM kind once per linear layer (D->F, F->F, F->D): its figures are
    the mean over the three, matching the mean launch time they are divided by."""
    e = 2 if wl.dtype == "bf16" else 4
    T, D, H, k, dM = wl.T, wl.D, wl.H, wl.k, wl.dM
    rows = int(sum(counts))
    touched = int(sum(1 for c in counts if c > 0))
    if wl.expert == "ffblock":
        return _block_kernel_algorithmic(name, wl, rows, touched, e)
    w = touched * D * H * e
    f = 2 * rows * D * H
    m = _GEMM2.match(name)
    if m:
        gm, bt, epi = int(m.group(1)), int(m.group(3)), int(m.group(4))
        if gm == 1:       # weight gradient: read the rows of both operands, write dW (SGD: read W too)
            return "expert weight-gradient GEMM", f, rows * (D + H) * e + (2 * w if epi == 5 else w)
        if epi == 2:      # up-projection with bias and activation: read x_perm, W1, b1; write h and a
            return "expert up-projection GEMM", f, w + touched * H * e + rows * (D + 2 * H) * e
        if epi == 1:      # down-projection with bias: read a, W2, b2; write y_perm
            return "expert down-projection GEMM", f, w + touched * D * e + rows * (H + D) * e
        if epi == 3:      # dh = (dy W2) act'(h): read dy_perm, W2, h; write dh
            return "expert dh GEMM", f, w + rows * (D + 2 * H) * e
        if epi == 0 and bt == 1:   # dx_perm = dh W1: read dh, W1; write dx_perm
            return "expert dx GEMM", f, w + rows * (H + D) * e
        return None
    return _routing_kernel_algorithmic(name, wl, rows, e)


def _routing_kernel_algorithmic(name, wl, rows, e):
    T, D, k, dM = wl.T, wl.D, wl.k, wl.dM
    if name.startswith("gate_topk_mfma"):
        return "gate scores + TopK (MFMA)", 2 * T * D * dM, T * D * e + dM * D * e + T * k * 12
    if name.startswith("gather_rows"):
        return "dispatch row gather", 0, T * D * e + rows * D * e
    if name.startswith("combine_kernel"):
        return "combine", 2 * rows * D, rows * D * e + T * D * e + T * k * 8
    if name.startswith("combine_bwd_kernel"):
        return "combine backward", 4 * rows * D, T * D * e + 2 * rows * D * e + T * k * 8
    if name.startswith("dispatch_bwd_kernel"):
        return "dispatch backward", 0, rows * D * e + T * D * e + T * k * 8
    return None


def _block_kernel_algorithmic(name, wl, rows, touched, e):
    """Per-launch figures of the LayerNorm block layer's kernels (Linear D->F, LayerNorm +
    act, Linear F->F, LayerNorm + act, Linear F->D): GEMMs as the mean over the three
    linear layers; the LayerNorm row kernels read and write each [rows, F] tensor once,
    plus 8 bytes of fp32 statistics per row and the touched experts' scale and shift."""
    D, F = wl.D, wl.H
    layers = ((D, F), (F, F), (F, D))
    m = _GEMM2.match(name)
    if m:
        gm, bt, epi = int(m.group(1)), int(m.group(3)), int(m.group(4))
        fl = sum(2 * rows * a * b for a, b in layers) // 3
        wts = sum(touched * a * b * e for a, b in layers) // 3
        if gm == 1:       # weight gradients: both row operands in, every touched dW out
            return ("block weight-gradient GEMM (mean of 3 layers)", fl,
                    sum(rows * (a + b) * e for a, b in layers) // 3 + wts)
        if epi == 1:      # forward with bias: rows in, weights and bias in, rows out
            return ("block forward GEMM (mean of 3 layers)", fl,
                    wts + sum(touched * b * e + rows * (a + b) * e for a, b in layers) // 3)
        if epi == 0 and bt == 1:   # data gradients
            return "block data-gradient GEMM (mean of 3 layers)", fl, wts + sum(rows * (a + b) * e for a, b in layers) // 3
        return None
    lnp = 2 * touched * F * e + 8 * rows
    if name.startswith("(ln_act_fwd_kernel"):
        return "LayerNorm + act forward", 0, 2 * rows * F * e + lnp
    if name.startswith("(ln_act_bwd_rows_kernel"):
        return "LayerNorm + act backward (rows)", 0, 3 * rows * F * e + lnp
    if name.startswith("(ln_act_bwd_params_kernel"):
        return "LayerNorm + act backward (scale, shift)", 0, 2 * rows * F * e + lnp + 2 * touched * F * e
    return _routing_kernel_algorithmic(name, wl, rows, e)


def roofline_of(flops, nbytes, seconds, peak_tf):
    ridge = peak_tf * 1e12 / (PEAK_HBM_GBS * 1e9)
    if flops and flops / max(nbytes, 1) >= ridge:
        ach = flops / seconds / 1e12
        return {"bound": "mfma", "achieved": round(ach, 1), "peak": peak_tf, "unit": "TFLOP/s",
                "frac": round(ach / peak_tf, 4)}
    ach = nbytes / seconds / 1e9
    return {"bound": "hbm", "achieved": round(ach, 1), "peak": PEAK_HBM_GBS, "unit": "GB/s",
            "frac": round(ach / PEAK_HBM_GBS, 4)}


def blas_threads():
    try:
        from threadpoolctl import threadpool_info
        return max([p.get("num_threads", 1) for p in threadpool_info() if p.get("user_api") == "blas"] or [1])
    except Exception:
        return os.cpu_count() or 1


def cpu_baseline(wl, inp, counts, budget_s=12.0, max_experts=16):
    """The oracle, as it stands, on a bounded sample of the same workload: routing
    (gate, TopK, weights), dispatch and (with a backward) the gate backward for every
    token, then the expert blocks (forward, and backward when the workload has one) for
    a few experts, extrapolated linearly in pairs to the whole batch."""
    import numpy as np
    import oracle as O
    threads = blas_threads()
    x = O.to64(inp["x"])
    Wg, bg = O.to64(inp["Wg"]), O.to64(inp["bg"])
    alive = inp["alive"].cpu().numpy()
    dy = O.to64(inp["dy"])
    N = wl.N

    t0 = time.perf_counter()
    r = O.routing(x, Wg, bg, alive, wl.d, wl.M, wl.k)
    c, off, row_token, pos = O.dispatch(r["idx"], alive, N)
    if wl.backward:
        O.gate_backward(r["w"], np.zeros_like(r["w"]), r["idx"], alive, x, Wg, wl.d, wl.M)
    t_route = time.perf_counter() - t0

    live = [int(e) for e in np.nonzero(c)[0]]
    rng = np.random.default_rng(0)
    rng.shuffle(live)
    t_exp, pairs, used = 0.0, 0, 0
    for e in live:
        rows = row_token[off[e]:off[e + 1]]
        if wl.expert == "ffblock":
            prm = {n: O.to64(v[e]) for n, v in inp["params"].items()}                # not timed
            t1 = time.perf_counter()
            X = x[rows]
            fw = O.ffblock_forward_stored(X, prm, wl.act)
            if wl.backward:
                O.ffblock_backward(X, fw, dy[rows], prm, wl.act)
        else:
            W1, b1, W2, b2 = (O.to64(inp[n][e]) for n in ("W1", "b1", "W2", "b2"))   # not timed
            t1 = time.perf_counter()
            X = x[rows]
            h, a, y = O.expert_forward(X, W1, b1, W2, b2, wl.act)
            if wl.backward:
                O.expert_backward(X, h, a, dy[rows], W1, W2, wl.act)
        t_exp += time.perf_counter() - t1
        pairs += len(rows)
        used += 1
        if t_exp + t_route > budget_s or used >= max_experts:
            break
    total_pairs = int(off[-1])
    est = t_route + t_exp * total_pairs / max(pairs, 1)
    passes = "fwd+bwd" if wl.backward else "fwd"
    return {"value": round(wl.T / est, 2), "unit": "tokens/s", "cores": int(threads), "kind": "oracle",
            "sample": (f"fp64 NumPy oracle ({passes}) on {threads} BLAS thread(s): routing, dispatch"
                       f"{' and gate backward' if wl.backward else ''} for all {wl.T} tokens ({t_route:.2f} s) "
                       f"+ expert {passes} for {used} experts ({pairs} of {total_pairs} pairs, {t_exp:.2f} s), "
                       f"extrapolated linearly in pairs"),
            "seconds_measured": round(t_route + t_exp, 3)}


def cpu_baselines(wl, inp, counts, budget_s=12.0, one_budget_s=8.0):
    """The oracle on the host's BLAS threads, then on one thread (smaller sample)."""
    out = cpu_baseline(wl, inp, counts, budget_s=budget_s)
    try:
        from threadpoolctl import threadpool_limits
        with threadpool_limits(limits=1, user_api="blas"):
            one = cpu_baseline(wl, inp, counts, budget_s=one_budget_s, max_experts=4)
        out["one_thread"] = {k: one[k] for k in ("value", "unit", "cores", "sample", "seconds_measured")}
    except Exception as ex:  # threadpoolctl missing: report the main figure only
        out["one_thread"] = {"error": str(ex)}
    return out


TRAFFIC_FILE = os.path.join(ROOT, "profiles", "traffic_wide.json")
KERNEL_SOURCES = ("gemm.hpp", "gemm2.hpp", "grouped.hpp", "ffn.hip", "common.hpp")


def kernel_source_hash():
    """Hash of the GEMM sources: counter readings are valid only for the exact kernels
    they were taken on."""
    import hashlib
    h = hashlib.sha256()
    for f in KERNEL_SOURCES:
        with open(os.path.join(ROOT, "paper_2002_04013_amd", "csrc", f), "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()[:16]


def measured_traffic(workload, kernel):
    """HBM bytes per launch of `kernel` (FETCH_SIZE + WRITE_SIZE from two rocprofv3
    counter runs, scaled by the copy-kernel calibration) from the committed counter
    summary, or None if there is none for this workload, kernel and kernel source."""
    try:
        with open(TRAFFIC_FILE) as f:
            t = json.load(f)
    except (OSError, ValueError):
        return None
    if t.get("workload") != workload or t.get("kernel_source_hash") != kernel_source_hash():
        return None
    k = t.get("kernels", {}).get(kernel)
    return None if k is None else k.get("bytes_per_launch")


def copy_calibration(nbytes=4 << 30, reps=5):
    """A plain device-to-device copy of known size, for scaling the FETCH_SIZE and
    WRITE_SIZE counters: each dispatch reads and writes exactly nbytes."""
    import torch
    src = torch.empty(nbytes // 2, dtype=torch.bfloat16, device="cuda")
    src.fill_(1.0)
    dst = torch.empty_like(src)
    torch.cuda.synchronize()
    for _ in range(reps):
        dst.copy_(src)
    torch.cuda.synchronize()
    print(json.dumps({"copy_bytes_read": nbytes, "copy_bytes_written": nbytes, "reps": reps}), flush=True)


def vendor_gemm(reps=5):
    """The vendor library (torch.bmm, hipBLASLt) on the wide workload's expert GEMM shapes,
    256 experts of exactly 512 rows, bf16, contiguous operands, no epilogue: a reference
    point for the grouped kernels, not part of the layer."""
    import torch
    E = 256
    shapes = [("up", 512, 4096, 16384), ("down", 512, 16384, 4096),
              ("dW1 = dh^T x", 16384, 512, 4096), ("dW2 = dy^T a", 4096, 512, 16384)]
    out = []
    for name, M, K, N in shapes:
        A = torch.randn(E, M, K, device="cuda", dtype=torch.bfloat16)
        B = torch.randn(E, K, N, device="cuda", dtype=torch.bfloat16) * 0.01
        C = torch.empty(E, M, N, device="cuda", dtype=torch.bfloat16)
        for _ in range(2):
            torch.bmm(A, B, out=C)
        torch.cuda.synchronize()
        ev = [torch.cuda.Event(enable_timing=True) for _ in range(2)]
        ev[0].record()
        for _ in range(reps):
            torch.bmm(A, B, out=C)
        ev[1].record()
        torch.cuda.synchronize()
        ms = ev[0].elapsed_time(ev[1]) / reps
        tf = 2.0 * E * M * K * N / (ms * 1e-3) / 1e12
        out.append({"gemm": name, "batch": E, "M": M, "K": K, "N": N, "ms": round(ms, 3),
                    "tflops": round(tf, 1), "frac": round(tf / PEAK_BF16_TFLOPS, 4)})
        log(f"vendor {name}: {ms:.3f} ms, {tf:.1f} TFLOP/s")
        del A, B, C
        torch.cuda.empty_cache()
    print(json.dumps({"vendor_gemm": out, "library": "torch.bmm (hipBLASLt)"}), flush=True)


def log(msg):
    print(f"[bench] {msg}", file=sys.stderr, flush=True)


def run_workload(name, steps, warmup, recompute=False, sgd=False, alive_topk=False, cold_steps=0,
                 cpu=False, cpu_budget=(12.0, 8.0)):
    """Build one workload's inputs and layer, time `steps` steps after `warmup`, trace
    every kernel in the timed region, time a few more steps with call-boundary events
    only, optionally time `cold_steps` more steps each after a cache flush, and return
    the measurements."""
    import torch
    from paper_2002_04013_amd import DMoEBlockLayer, DMoELayer, abi
    from workloads import (get_workload, make_alive, make_block_experts, make_dy, make_experts, make_gate,
                           make_x)

    wl = get_workload(name)
    block = wl.expert == "ffblock"
    dev = torch.device("cuda:0")
    t_gen = time.perf_counter()
    Wg, bg = make_gate(wl, dev)
    inp = dict(x=make_x(wl, dev), dy=make_dy(wl, dev), Wg=Wg, bg=bg, alive=make_alive(wl, dev))
    dWg, dbg = torch.empty_like(Wg), torch.empty_like(bg)
    flags = abi.DMOE_FLAG_ALIVE_TOPK if alive_topk else 0
    if block:
        prm = make_block_experts(wl, dev)
        inp["params"] = prm
        grads = {n: torch.empty_like(v) for n, v in prm.items()}
        L = DMoEBlockLayer(wl.T, wl.D, wl.H, wl.d, wl.M, wl.k, wl.dtype, wl.act, device=dev, flags=flags)
    else:
        W1, b1, W2, b2 = make_experts(wl, dev)
        inp.update(W1=W1, b1=b1, W2=W2, b2=b2)
        dW1, db1 = torch.empty_like(W1), torch.empty_like(b1)
        dW2, db2 = torch.empty_like(W2), torch.empty_like(b2)
        L = DMoELayer(wl.T, wl.D, wl.H, wl.d, wl.M, wl.k, wl.dtype, wl.act, device=dev, dh_aliases_h=False,
                      flags=flags)
    torch.cuda.synchronize()
    log(f"{wl.name}: inputs ready in {time.perf_counter() - t_gen:.1f} s")

    x, alive = inp["x"], inp["alive"]
    Dm = L.dims
    stream = torch.cuda.current_stream()
    calls = [
        ("gate_topk", lambda: abi.dmoe_gate_topk(Dm, x, Wg, bg, alive, L.idx, L.w, None, None, L.ws)),
        ("dispatch", lambda: abi.dmoe_dispatch(Dm, x, L.idx, alive, L.counts, L.offsets, L.row_token,
                                               L.pos, L.x_perm, L.ws)),
        ("ffn_fwd", (lambda: abi.dmoe_expert_ffblock_fwd(Dm, L.offsets, L.x_perm, prm, L.acts, L.y_perm,
                                                         L.ws)) if block else
         (lambda: abi.dmoe_expert_ffn_fwd(Dm, L.offsets, L.x_perm, W1, b1, W2, b2, L.h, L.a,
                                          L.y_perm, L.ws))),
        ("combine", lambda: abi.dmoe_combine(Dm, L.y_perm, L.pos, L.w, L.y)),
        ("combine_bwd", lambda: abi.dmoe_combine_bwd(Dm, inp["dy"], L.y_perm, L.pos, L.w, L.dy_perm, L.dw)),
        ("gate_topk_bwd", lambda: abi.dmoe_gate_topk_bwd(Dm, x, L.idx, L.w, L.dw, alive, L.dg, dWg, dbg,
                                                         L.ws)),
        ("ffn_bwd", (lambda: abi.dmoe_expert_ffblock_bwd(Dm, L.offsets, L.x_perm, prm, L.acts, L.dy_perm,
                                                         L.g1, L.g2, L.dx_perm, grads, L.ws)) if block else
         (lambda: abi.dmoe_expert_ffn_bwd_sgd(Dm, L.offsets, L.counts, L.x_perm, L.h, L.a, L.dy_perm, W1, b1,
                                              W2, b2, 1e-4, L.dh, L.dx_perm, L.ws)) if sgd else
         (lambda: abi.dmoe_expert_ffn_bwd_recompute(Dm, L.offsets, L.counts, L.x_perm, W1, b1, W2,
                                                    L.dy_perm, L.h, L.a, L.dx_perm, dW1, db1, dW2, db2,
                                                    L.ws)) if recompute else
         (lambda: abi.dmoe_expert_ffn_bwd(Dm, L.offsets, L.counts, L.x_perm, L.h, L.a, L.dy_perm, W1, W2,
                                          L.dh, L.dx_perm, dW1, db1, dW2, db2, L.ws))),
        ("dispatch_bwd", lambda: abi.dmoe_dispatch_bwd(Dm, L.dx_perm, L.pos, L.idx, L.dg, Wg, L.dx)),
    ]
    calls = [(n, f) for n, f in calls if wl.backward or n in FWD_CALLS]
    timed = [n for n, _ in calls]

    def step(ev=None):
        for n, fn in calls:
            if ev is not None:
                ev[n][0].record(stream)
            fn()
            if ev is not None:
                ev[n][1].record(stream)

    def new_events(k):
        return [{n: (torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for n in timed}
                for _ in range(k)]

    for _ in range(warmup):
        step()
    torch.cuda.synchronize()
    counts = L.counts.cpu().tolist()

    evs = new_events(steps)
    trace = abi.Trace(capacity=steps * 64, stream=stream)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    with trace:
        for i in range(steps):
            step(evs[i])
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    ms = {n: sum(e[n][0].elapsed_time(e[n][1]) for e in evs) / steps for n in timed}
    per_step = sorted(e[timed[0]][0].elapsed_time(e[timed[-1]][1]) for e in evs)
    kern = trace.kernels()
    log(f"{wl.name}: {steps} steps in {wall:.3f} s; per call ms: " +
        ", ".join(f"{n} {v:.3f}" for n, v in ms.items()))

    alg = algorithmic(wl, counts, recompute, sgd)
    if block:
        alg.update(algorithmic_block(wl, counts))
    peak_tf = PEAK_BF16_TFLOPS if wl.dtype == "bf16" else PEAK_F32_TFLOPS

    # per-kernel table from the trace
    agg = {}
    for kname, t in kern:
        a = agg.setdefault(kname, [0, 0.0])
        a[0] += 1
        a[1] += t
    kernels = []
    for kname, (n, t) in sorted(agg.items(), key=lambda kv: -kv[1][1]):
        row = {"name": kname, "launches_per_step": round(n / steps, 3), "ms_per_step": round(t / steps, 4),
               "ms_per_launch": round(t / n, 4)}
        ka = kernel_algorithmic(kname, wl, counts, sgd)
        if ka is not None:
            role, fl, nb = ka
            row.update(role=role, flops_per_launch=fl, bytes_per_launch=nb)
            row.update(roofline_of(fl, nb, t / n * 1e-3, peak_tf))
        kernels.append(row)

    def call_roof(n):
        a = alg[n]
        return roofline_of(a["flops"], a["bytes"], ms[n] * 1e-3, peak_tf)

    out = {"wl": wl, "counts": counts, "wall": wall, "ms": ms, "per_step": per_step, "kernels": kernels,
           "call_roofline": {n: call_roof(n) for n in timed}, "alg": alg, "peak_tf": peak_tf,
           "traced": trace.count, "inp_host": None}

    # The calls once more with call-boundary events only: the trace's event after every
    # kernel adds a few microseconds at each kernel boundary, a visible share of the
    # short calls (gate, dispatch, combine), so their fractions come from these steps.
    n_u = min(steps, 5)
    uev = new_events(n_u)
    for i in range(n_u):
        step(uev[i])
    torch.cuda.synchronize()
    ms_u = {n: sum(e[n][0].elapsed_time(e[n][1]) for e in uev) / n_u for n in timed}
    out["ms_untraced"] = ms_u
    out["per_step_untraced"] = sorted(e[timed[0]][0].elapsed_time(e[timed[-1]][1]) for e in uev)
    out["call_roofline_untraced"] = {n: roofline_of(alg[n]["flops"], alg[n]["bytes"], ms_u[n] * 1e-3, peak_tf)
                                     for n in timed}

    # The same step recorded once into a HIP graph and replayed: the entry points
    # allocate nothing and never synchronise, so a caller can run a whole step as one
    # graph launch.  The replays are timed between two events; the kernels are the same,
    # only the launch overhead between them changes (what matters for short steps).
    try:
        graph = torch.cuda.CUDAGraph()
        with torch.cuda.graph(graph):
            step()
        torch.cuda.synchronize()
        graph.replay()
        torch.cuda.synchronize()
        n_g = min(steps, 5) if wl.T * wl.D >= (1 << 24) else steps
        g0, g1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        g0.record(stream)
        for _ in range(n_g):
            graph.replay()
        g1.record(stream)
        torch.cuda.synchronize()
        out["graph_ms_per_step"] = g0.elapsed_time(g1) / n_g
        del graph
    except RuntimeError as ex:              # reported, not fatal: the eager figures stand
        out["graph_ms_per_step"] = None
        out["graph_error"] = str(ex)[:200]

    if cold_steps:
        # Cold memory-side cache: before each step, outside any timed interval, write
        # FLUSH_BYTES to one scratch buffer and read FLUSH_BYTES from another, so the
        # step's first reads (the gate's x) come from HBM and no dirty lines of the
        # previous step are left to write back.
        # The calls are timed untraced (call-boundary events only); the main kernels'
        # durations come from as many traced cold steps after them.
        fw = torch.empty(FLUSH_BYTES // 2, dtype=torch.int16, device=dev)
        fr = torch.ones(FLUSH_BYTES // 4, dtype=torch.float32, device=dev)
        cev = new_events(cold_steps)
        ctrs = [abi.Trace(capacity=64, stream=stream) for _ in range(cold_steps)]
        sink = torch.zeros((), dtype=torch.float32, device=dev)
        for i in range(cold_steps):
            fw.fill_(i)
            sink += fr.sum()
            step(cev[i])
        for i in range(cold_steps):
            fw.fill_(i + cold_steps)
            sink += fr.sum()
            with ctrs[i]:
                step()
        torch.cuda.synchronize()
        cms = {n: sum(e[n][0].elapsed_time(e[n][1]) for e in cev) / cold_steps for n in ("gate_topk", "dispatch")}
        ck = {}
        for ctr in ctrs:
            for kname, t in ctr.kernels():
                if kname.startswith("gate_topk_mfma") or kname.startswith("gather_rows"):
                    ck.setdefault(kname, []).append(t)
        cold = {}
        for n in ("gate_topk", "dispatch"):
            warm_r = out["call_roofline_untraced"][n]
            cold_r = roofline_of(alg[n]["flops"], alg[n]["bytes"], cms[n] * 1e-3, peak_tf)
            cold[n] = {"warm_ms": round(ms_u[n], 4), "cold_ms": round(cms[n], 4),
                       "warm_frac": warm_r["frac"], "cold_frac": cold_r["frac"], "bound": cold_r["bound"],
                       "cold_achieved": cold_r["achieved"], "unit": cold_r["unit"]}
        for kname, ts in ck.items():
            ka = kernel_algorithmic(kname, wl, counts)
            t = sum(ts) / len(ts)
            r = roofline_of(ka[1], ka[2], t * 1e-3, peak_tf) if ka else {}
            cold[kname] = {"cold_ms_per_launch": round(t, 4), **{k: r[k] for k in ("achieved", "unit", "frac")
                                                                 if k in r}}
        out["cold"] = cold
        out["cold_protocol"] = (f"before each of {cold_steps} steps, outside the timed calls: write "
                                f"{FLUSH_BYTES >> 20} MiB, then read another {FLUSH_BYTES >> 20} MiB; "
                                f"calls timed with call-boundary events only, kernels in {cold_steps} more "
                                f"such steps with the per-kernel trace")
        del fw, fr

    if sgd and not block:
        # What the fused update replaces: the gradient-returning backward, then a separate
        # SGD step over the same parameters (torch's in-place add, for comparison only).
        n_c = min(steps, 5)
        ce = [[torch.cuda.Event(enable_timing=True) for _ in range(3)] for _ in range(n_c)]
        for i in range(n_c):
            ce[i][0].record(stream)
            abi.dmoe_expert_ffn_bwd(Dm, L.offsets, L.counts, L.x_perm, L.h, L.a, L.dy_perm, W1, W2, L.dh,
                                    L.dx_perm, dW1, db1, dW2, db2, L.ws)
            ce[i][1].record(stream)
            for prm_t, grad_t in ((W1, dW1), (b1, db1), (W2, dW2), (b2, db2)):
                prm_t.add_(grad_t, alpha=-1e-4)
            ce[i][2].record(stream)
        torch.cuda.synchronize()
        t_b = sum(c[0].elapsed_time(c[1]) for c in ce) / n_c
        t_u = sum(c[1].elapsed_time(c[2]) for c in ce) / n_c
        out["sgd_comparison"] = {
            "fused_sgd_backward_ms": round(ms["ffn_bwd"], 3),
            "gradient_backward_ms": round(t_b, 3), "separate_update_ms": round(t_u, 3),
            "gradient_backward_plus_update_ms": round(t_b + t_u, 3),
            "note": "separate update: torch in-place add of -lr * gradient to W1, b1, W2, b2 (comparison only)"}

    if cpu:
        host = {n: v for n, v in inp.items()}
        for n in ("x", "dy", "Wg", "bg", "alive"):
            host[n] = inp[n].cpu()
        out["cpu_baseline"] = cpu_baselines(wl, host, counts, *cpu_budget)
    del inp, L, calls, step
    return out


def workload_config(wl, recompute=False, sgd=False, alive_topk=False):
    block = wl.expert == "ffblock"
    return {"workload": wl.name, "tokens": wl.T, "d_model": wl.D, "expert_hidden": wl.H,
            "grid": f"{'x'.join([str(wl.M)] * wl.d)}", "experts": wl.N, "k": wl.k,
            "act": wl.act, "p_alive": wl.p_alive, "pass": "fwd+bwd" if wl.backward else "fwd",
            "activations": "recomputed in backward" if recompute else "stored",
            "expert_update": "fused SGD in the backward" if sgd else "gradients returned",
            "topk": "among alive experts" if alive_topk else "all experts, dead ones weighted 0",
            "expert": ("Linear-LayerNorm-act-Linear-LayerNorm-act-Linear" if block else "Linear-act-Linear")}


def summary(r, steps):
    """The measurements of an extra workload, for the "workloads" key."""
    wl = r["wl"]
    rows = int(sum(r["counts"]))
    out = {"config": workload_config(wl), "dtype": wl.dtype, "steps": steps,
           "ms_per_step": round(r["wall"] * 1e3 / steps, 3),
           "tokens_per_s": round(wl.T * steps / r["wall"], 1),
           "step_device_ms_median": round(r["per_step"][len(r["per_step"]) // 2], 4),
           "graph_replay_ms_per_step": (round(r["graph_ms_per_step"], 4) if r["graph_ms_per_step"] else
                                        r.get("graph_error")),
           "graph_replay_tokens_per_s": (round(wl.T / (r["graph_ms_per_step"] * 1e-3), 1)
                                         if r["graph_ms_per_step"] else None),
           "calls_ms": {n: round(v, 4) for n, v in r["ms"].items()},
           "calls_ms_untraced": {n: round(v, 4) for n, v in r["ms_untraced"].items()},
           "calls_roofline": {n: {k: v[k] for k in ("bound", "achieved", "unit", "frac")}
                              for n, v in r["call_roofline_untraced"].items()},
           "rows_used": rows, "max_rows_per_expert": int(max(r["counts"])),
           "experts_without_rows": int(sum(1 for c in r["counts"] if c == 0)),
           "top_kernels": r["kernels"][:6]}
    if wl.name == "tiny_f32":
        out["step_device_us_median"] = round(r["per_step"][len(r["per_step"]) // 2] * 1e3, 1)
        pu = r["per_step_untraced"]
        out["step_device_us_median_untraced"] = round(pu[len(pu) // 2] * 1e3, 1)
    if "cold" in r:
        out["cold"] = r["cold"]
        out["cold_protocol"] = r["cold_protocol"]
    if "cpu_baseline" in r:
        out["cpu_baseline"] = r["cpu_baseline"]
    return out


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--workload", default="wide")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-extra", action="store_true", help="time only --workload (no other workloads)")
    ap.add_argument("--cold-steps", type=int, default=5)
    ap.add_argument("--recompute", action="store_true",
                    help="backward regenerates h and a (dmoe_expert_ffn_bwd_recompute)")
    ap.add_argument("--alive-topk", action="store_true",
                    help="TopK among the alive experts only (DMOE_FLAG_ALIVE_TOPK)")
    ap.add_argument("--sgd", action="store_true",
                    help="backward updates the expert parameters in place (dmoe_expert_ffn_bwd_sgd, lr 1e-4)")
    ap.add_argument("--copy-calibration", action="store_true",
                    help="only run a plain 4 GiB device copy (counter calibration)")
    ap.add_argument("--vendor-gemm", action="store_true",
                    help="only time the vendor library's batched GEMM on the wide expert shapes (reference)")
    args = ap.parse_args()
    if args.copy_calibration:
        copy_calibration()
        return
    if args.vendor_gemm:
        vendor_gemm()
        return
    ws_env = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or ws_env != 1:
        print("bench.py: the DMoE layer path here runs on one GPU only; "
              "multi-GPU (--gpus > 1) is not supported", file=sys.stderr)
        sys.exit(2)

    import torch
    from workloads import get_workload

    wl = get_workload(args.workload)
    if wl.expert == "ffblock" and (args.recompute or args.sgd):
        print("bench.py: --recompute and --sgd apply to the Linear-act-Linear experts only", file=sys.stderr)
        sys.exit(2)
    torch.cuda.set_device(0)
    modes = dict(recompute=args.recompute, sgd=args.sgd, alive_topk=args.alive_topk)
    r = run_workload(args.workload, args.steps, args.warmup,
                     cold_steps=args.cold_steps if args.workload in COLD_WORKLOADS else 0,
                     cpu=not args.no_cpu_baseline, **modes)
    ms, kernels, peak_tf = r["ms"], r["kernels"], r["peak_tf"]

    # the roofline object: the kernel that takes the most device time per step
    dom = kernels[0]
    if "frac" in dom:
        roofline = {k: dom[k] for k in ("bound", "achieved", "peak", "unit", "frac")}
    else:
        roofline = {"bound": None, "achieved": None, "peak": None, "unit": None, "frac": None}
    roofline.update(kernel=dom["name"], role=dom.get("role"), launches_per_step=dom["launches_per_step"],
                    ms_per_launch=dom["ms_per_launch"], flops_per_launch=dom.get("flops_per_launch"),
                    bytes_per_launch=dom.get("bytes_per_launch"),
                    traffic=measured_traffic(wl.name, dom["name"]),
                    timing="HIP events on the launch stream around every kernel of the timed steps")
    result = {
        "metric": METRIC,
        "value": round(wl.T * args.steps / r["wall"], 1),
        "unit": "tokens/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(r["wall"] * 1e3 / args.steps, 3),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": wl.dtype,
        "data": "synthetic (seeded N(0,1) inputs, N(0,1/fan_in) weights, random init)",
        "config": workload_config(wl, **modes),
        "roofline": roofline,
        "kernels": kernels,
        "roofline_ffn_fwd": r["call_roofline"]["ffn_fwd"],
        "roofline_ffn_bwd": r["call_roofline"].get("ffn_bwd"),
        "gate_topk": r["call_roofline_untraced"]["gate_topk"],
        "dispatch": r["call_roofline_untraced"]["dispatch"],
        "calls_ms": {n: round(v, 4) for n, v in ms.items()},
        "calls_ms_untraced": {n: round(v, 4) for n, v in r["ms_untraced"].items()},
        "calls_timing": ("calls_ms: the timed steps, with an event after every kernel; calls_ms_untraced, "
                         "gate_topk and dispatch: 5 more steps with events at call boundaries only"),
        "step_ms": {"median": round(r["per_step"][len(r["per_step"]) // 2], 3), "min": round(r["per_step"][0], 3),
                    "max": round(r["per_step"][-1], 3)},
        "graph_replay_ms_per_step": (round(r["graph_ms_per_step"], 3) if r["graph_ms_per_step"] else
                                     r.get("graph_error")),
        "paper_context": PAPER_CONTEXT,
    }
    if "cold" in r:
        result["gate_dispatch_cold"] = r["cold"]
        result["cold_protocol"] = r["cold_protocol"]
    if "cpu_baseline" in r:
        result["cpu_baseline"] = r["cpu_baseline"]
    if "sgd_comparison" in r:
        result["sgd_comparison"] = r["sgd_comparison"]
    del r
    gc.collect()
    torch.cuda.empty_cache()

    if not args.no_extra and not any(modes.values()):
        extra = {}
        for name in EXTRA_WORKLOADS:
            if name == args.workload:
                continue
            st = 20 if name == "tiny_f32" else 5
            rr = run_workload(name, st, 2, cold_steps=3 if name in COLD_WORKLOADS else 0,
                              cpu=not args.no_cpu_baseline, cpu_budget=(3.0, 3.0))
            extra[name] = summary(rr, st)
            del rr
            gc.collect()
            torch.cuda.empty_cache()
        result["workloads"] = extra
    print(json.dumps(result), flush=True)


if __name__ == "__main__":
    main()
