#!/usr/bin/env python3
"""Benchmark of one DMoE layer, forward + backward, on one MI355X.

    python bench.py [--gpus 1] [--steps K] [--warmup W] [--workload wide]

A step is one pass of the whole layer over one batch of synthetic input:
gate + TopK + weights, dispatch, expert FFN forward, combine, and the backward of
all of them (combine, gate, expert FFN, dispatch).  Inputs and weights are
resident in HBM before the timed region.  Prints one JSON line.
"""
import argparse
import json
import os
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


def cpu_baseline(wl, inp, counts, budget_s=12.0):
    """The oracle, as it stands, on a bounded sample of the same workload: routing
    (gate, TopK, weights), dispatch and the gate backward for every token, then the
    expert blocks forward+backward for a few experts, extrapolated linearly in pairs
    to the whole batch."""
    import numpy as np
    import oracle as O
    try:
        from threadpoolctl import threadpool_info
        threads = max([p.get("num_threads", 1) for p in threadpool_info() if p.get("user_api") == "blas"]
                      or [1])
    except Exception:
        threads = os.cpu_count() or 1
    x = O.to64(inp["x"])
    Wg, bg = O.to64(inp["Wg"]), O.to64(inp["bg"])
    alive = inp["alive"].cpu().numpy()
    dy = O.to64(inp["dy"])
    N = wl.N

    t0 = time.perf_counter()
    r = O.routing(x, Wg, bg, alive, wl.d, wl.M, wl.k)
    c, off, row_token, pos = O.dispatch(r["idx"], alive, N)
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
            O.ffblock_backward(X, fw, dy[rows], prm, wl.act)
        else:
            W1, b1, W2, b2 = (O.to64(inp[n][e]) for n in ("W1", "b1", "W2", "b2"))   # not timed
            t1 = time.perf_counter()
            X = x[rows]
            h, a, y = O.expert_forward(X, W1, b1, W2, b2, wl.act)
            O.expert_backward(X, h, a, dy[rows], W1, W2, wl.act)
        t_exp += time.perf_counter() - t1
        pairs += len(rows)
        used += 1
        if t_exp + t_route > budget_s or used >= 16:
            break
    total_pairs = int(off[-1])
    est = t_route + t_exp * total_pairs / max(pairs, 1)
    return {"value": round(wl.T / est, 2), "unit": "tokens/s", "cores": int(threads), "kind": "oracle",
            "sample": (f"fp64 NumPy oracle: routing, dispatch and gate backward for all {wl.T} tokens "
                       f"({t_route:.2f} s) + expert fwd+bwd for {used} experts ({pairs} of "
                       f"{total_pairs} pairs, {t_exp:.2f} s), extrapolated linearly in pairs"),
            "seconds_measured": round(t_route + t_exp, 3)}


TRAFFIC_FILE = os.path.join(ROOT, "profiles", "traffic_wide.json")
KERNEL_SOURCES = ("gemm.hpp", "gemm2.hpp", "grouped.hpp", "ffn.hip", "common.hpp")


def kernel_source_hash():
    """Hash of the sources of the dominant kernel: counter readings are valid only
    for the exact kernel they were taken on."""
    import hashlib
    h = hashlib.sha256()
    for f in KERNEL_SOURCES:
        with open(os.path.join(ROOT, "paper_2002_04013_amd", "csrc", f), "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()[:16]


def measured_traffic(workload):
    """HBM bytes per dmoe_expert_ffn_fwd call from the committed rocprofv3 counter
    summary (FETCH_SIZE + WRITE_SIZE of its GEMM launches, scaled by the copy-kernel
    calibration), or None if there is none for this workload and kernel source."""
    try:
        with open(TRAFFIC_FILE) as f:
            t = json.load(f)
    except (OSError, ValueError):
        return None
    if t.get("workload") != workload or t.get("kernel_source_hash") != kernel_source_hash():
        return None
    return t.get("ffn_fwd_bytes")


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


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=10)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--workload", default="wide")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--recompute", action="store_true",
                    help="backward regenerates h and a (dmoe_expert_ffn_bwd_recompute)")
    ap.add_argument("--alive-topk", action="store_true",
                    help="TopK among the alive experts only (DMOE_FLAG_ALIVE_TOPK)")
    ap.add_argument("--sgd", action="store_true",
                    help="backward updates the expert parameters in place (dmoe_expert_ffn_bwd_sgd, lr 1e-4)")
    ap.add_argument("--copy-calibration", action="store_true",
                    help="only run a plain 4 GiB device copy (counter calibration)")
    args = ap.parse_args()
    if args.copy_calibration:
        copy_calibration()
        return
    ws_env = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or ws_env != 1:
        print("bench.py: this build runs the DMoE layer on one GPU only; "
              "multi-GPU (--gpus > 1) is not supported", file=sys.stderr)
        sys.exit(2)

    import torch
    from paper_2002_04013_amd import DMoEBlockLayer, DMoELayer
    from workloads import (get_workload, make_alive, make_block_experts, make_dy, make_experts, make_gate,
                           make_x)

    wl = get_workload(args.workload)
    block = wl.expert == "ffblock"
    if block and (args.recompute or args.sgd):
        print("bench.py: --recompute and --sgd apply to the Linear-act-Linear experts only", file=sys.stderr)
        sys.exit(2)
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    t_gen = time.perf_counter()
    Wg, bg = make_gate(wl, dev)
    inp = dict(x=make_x(wl, dev), dy=make_dy(wl, dev), Wg=Wg, bg=bg, alive=make_alive(wl, dev))
    dWg, dbg = torch.empty_like(Wg), torch.empty_like(bg)
    from paper_2002_04013_amd.abi import DMOE_FLAG_ALIVE_TOPK
    flags = DMOE_FLAG_ALIVE_TOPK if args.alive_topk else 0
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
    print(f"[bench] {wl.name}: inputs ready in {time.perf_counter() - t_gen:.1f} s", file=sys.stderr,
          flush=True)

    x, alive = inp["x"], inp["alive"]
    from paper_2002_04013_amd import abi
    Dm = L.dims
    stream = torch.cuda.current_stream()

    def step(ev=None):
        calls = [
            ("gate_topk", lambda: abi.dmoe_gate_topk(Dm, x, Wg, bg, alive, L.idx, L.w, None, None, L.ws)),
            ("dispatch", lambda: abi.dmoe_dispatch(Dm, x, L.idx, alive, L.counts, L.offsets, L.row_token,
                                                   L.pos, L.x_perm, L.ws)),
            ("ffn_fwd", (lambda: abi.dmoe_expert_ffblock_fwd(Dm, L.offsets, L.x_perm, prm, L.acts, L.y_perm,
                                                             L.ws)) if block else
             (lambda: abi.dmoe_expert_ffn_fwd(Dm, L.offsets, L.x_perm, W1, b1, W2, b2, L.h, L.a,
                                              L.y_perm, L.ws))),
            ("combine", lambda: abi.dmoe_combine(Dm, L.y_perm, L.pos, L.w, L.y)),
            ("combine_bwd", lambda: abi.dmoe_combine_bwd(Dm, inp["dy"], L.y_perm, L.pos, L.w, L.dy_perm,
                                                         L.dw)),
            ("gate_topk_bwd", lambda: abi.dmoe_gate_topk_bwd(Dm, x, L.idx, L.w, L.dw, alive, L.dg, dWg, dbg,
                                                             L.ws)),
            ("ffn_bwd", (lambda: abi.dmoe_expert_ffblock_bwd(Dm, L.offsets, L.x_perm, prm, L.acts, L.dy_perm,
                                                             L.g1, L.g2, L.dx_perm, grads, L.ws)) if block else
             (lambda: abi.dmoe_expert_ffn_bwd_sgd(Dm, L.offsets, L.counts, L.x_perm, L.h, L.a,
                                                             L.dy_perm, W1, b1, W2, b2, 1e-4, L.dh, L.dx_perm,
                                                             L.ws)) if args.sgd else
             (lambda: abi.dmoe_expert_ffn_bwd_recompute(Dm, L.offsets, L.counts, L.x_perm, W1, b1, W2,
                                                        L.dy_perm, L.h, L.a, L.dx_perm, dW1, db1,
                                                        dW2, db2, L.ws)) if args.recompute else
             (lambda: abi.dmoe_expert_ffn_bwd(Dm, L.offsets, L.counts, L.x_perm, L.h, L.a,
                                              L.dy_perm, W1, W2, L.dh, L.dx_perm, dW1, db1, dW2,
                                              db2, L.ws))),
            ("dispatch_bwd", lambda: abi.dmoe_dispatch_bwd(Dm, L.dx_perm, L.pos, L.idx, L.dg, Wg, L.dx)),
        ]
        for name, fn in calls:
            if not wl.backward and name not in FWD_CALLS:
                continue
            if ev is not None:
                ev[name][0].record(stream)
            fn()
            if ev is not None:
                ev[name][1].record(stream)

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    counts = L.counts.cpu().tolist()

    timed = [n for n in CALLS if wl.backward or n in FWD_CALLS]
    evs = [{n: (torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for n in timed}
           for _ in range(args.steps)]
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for i in range(args.steps):
        step(evs[i])
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    ms = {n: sum(e[n][0].elapsed_time(e[n][1]) for e in evs) / args.steps for n in timed}
    # per-step device time (first call's start to last call's end event of each step)
    per_step = sorted(e[timed[0]][0].elapsed_time(e[timed[-1]][1]) for e in evs)
    print(f"[bench] {args.steps} steps in {wall:.3f} s; per call ms: " +
          ", ".join(f"{n} {v:.3f}" for n, v in ms.items()), file=sys.stderr, flush=True)

    alg = algorithmic(wl, counts, args.recompute, args.sgd)
    if block:
        alg.update(algorithmic_block(wl, counts))
    peak_tf = PEAK_BF16_TFLOPS if wl.dtype == "bf16" else PEAK_F32_TFLOPS
    ridge = peak_tf * 1e12 / (PEAK_HBM_GBS * 1e9)

    def roof(name):
        a = alg[name]
        t = ms[name] * 1e-3
        ai = a["flops"] / max(a["bytes"], 1)
        if a["flops"] and ai >= ridge:
            ach = a["flops"] / t / 1e12
            return {"bound": "mfma", "achieved": round(ach, 1), "peak": peak_tf, "unit": "TFLOP/s",
                    "frac": round(ach / peak_tf, 4)}
        ach = a["bytes"] / t / 1e9
        return {"bound": "hbm", "achieved": round(ach, 1), "peak": PEAK_HBM_GBS, "unit": "GB/s",
                "frac": round(ach / PEAK_HBM_GBS, 4)}

    kern = ("grouped_gemm2 x3 + ln_act_fwd_kernel x2 (dmoe_expert_ffblock_fwd)" if block else
            "grouped_gemm2 (dmoe_expert_ffn_fwd: up- and down-projection launches + 1-block tile plan)")
    roofline = dict(roof("ffn_fwd"), kernel=kern, traffic=measured_traffic(wl.name),
                    per_launch={"flops": alg["ffn_fwd"]["flops"], "bytes": alg["ffn_fwd"]["bytes"],
                                "ms": round(ms["ffn_fwd"], 4)})
    result = {
        "metric": METRIC,
        "value": round(wl.T * args.steps / wall, 1),
        "unit": "tokens/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(wall * 1e3 / args.steps, 3),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": wl.dtype,
        "data": "synthetic (seeded N(0,1) inputs, N(0,1/fan_in) weights, random init)",
        "config": {"workload": wl.name, "tokens": wl.T, "d_model": wl.D, "expert_hidden": wl.H,
                   "grid": f"{'x'.join([str(wl.M)] * wl.d)}", "experts": wl.N, "k": wl.k,
                   "act": wl.act, "p_alive": wl.p_alive, "pass": "fwd+bwd" if wl.backward else "fwd",
                   "activations": "recomputed in backward" if args.recompute else "stored",
                   "expert_update": "fused SGD in the backward" if args.sgd else "gradients returned",
                   "topk": "among alive experts" if args.alive_topk else "all experts, dead ones weighted 0",
                   "expert": ("Linear-LayerNorm-act-Linear-LayerNorm-act-Linear" if block else
                              "Linear-act-Linear")},
        "roofline": roofline,
        "roofline_ffn_bwd": roof("ffn_bwd") if wl.backward else None,
        "gate_topk": roof("gate_topk"),
        "dispatch": roof("dispatch"),
        "calls_ms": {n: round(v, 4) for n, v in ms.items()},
        "step_ms": {"median": round(per_step[len(per_step) // 2], 3), "min": round(per_step[0], 3),
                    "max": round(per_step[-1], 3)},
    }
    if not args.no_cpu_baseline:
        host = {n: v for n, v in inp.items()}
        for n in ("x", "dy", "Wg", "bg", "alive"):
            host[n] = inp[n].cpu()
        result["cpu_baseline"] = cpu_baseline(wl, host, counts)
    print(json.dumps(result), flush=True)


if __name__ == "__main__":
    main()
