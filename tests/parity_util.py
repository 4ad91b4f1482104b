"""Helpers of the GPU parity tests: run the HIP path through the C ABI and the
oracle on the same seeded inputs, and compare them."""
import sys

import numpy as np
import torch

import oracle as O
from workloads import make_inputs

RTOL = {"bf16": 2e-2, "f32": 1e-5}


def say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


def assert_close(gpu, ref, rtol, name):
    """|gpu - ref| <= rtol * (|ref| + rms(ref)), elementwise."""
    g = O.to64(gpu)
    r = np.asarray(ref, np.float64)
    assert g.shape == r.shape, (name, g.shape, r.shape)
    if r.size == 0:
        return
    assert np.isfinite(g).all(), f"{name}: non-finite values"
    rms = float(np.sqrt(np.mean(r * r)))
    err = np.abs(g - r)
    lim = rtol * (np.abs(r) + rms) + 1e-30
    bad = err > lim
    if bad.any():
        i = np.unravel_index(np.argmax(err / lim), err.shape)
        raise AssertionError(f"{name}: {int(bad.sum())}/{bad.size} out of tolerance; worst at {i}: "
                             f"gpu {g[i]!r} ref {r[i]!r} (rtol {rtol}, rms {rms:.3g})")


def gpu_run(wl, inp, backward=True, dh_aliases_h=False, flags=0, recompute=False, clobber_h=False):
    """Forward (and backward) through the C ABI on cuda:0; returns CPU copies.
    recompute: backward through dmoe_expert_ffn_bwd_recompute; clobber_h: overwrite
    h and a between the passes (they must not be needed then)."""
    from paper_2002_04013_amd import DMoELayer
    dev = torch.device("cuda")
    t = {n: v.to(dev) for n, v in inp.items()}
    L = DMoELayer(wl.T, wl.D, wl.H, wl.d, wl.M, wl.k, wl.dtype, wl.act, dh_aliases_h=dh_aliases_h,
                  flags=flags, recompute=recompute)
    out = {}
    L.forward(t["x"], t["Wg"], t["bg"], t["alive"], t["W1"], t["b1"], t["W2"], t["b2"])
    if clobber_h:
        fwd_h, fwd_a = L.h.clone(), L.a.clone()
        L.h.fill_(-3.0)
        L.a.fill_(5.0)
    if backward:
        dt = L.dt
        sentinel = 7.0
        dW1 = torch.full_like(t["W1"], sentinel)
        db1 = torch.full_like(t["b1"], sentinel)
        dW2 = torch.full_like(t["W2"], sentinel)
        db2 = torch.full_like(t["b2"], sentinel)
        dWg = torch.empty_like(t["Wg"])
        dbg = torch.empty_like(t["bg"])
        L.backward(t["dy"], t["x"], t["Wg"], t["alive"], t["W1"], t["W2"], dW1, db1, dW2, db2, dWg, dbg,
                   b1=t["b1"])
        out.update(dW1=dW1, db1=db1, dW2=dW2, db2=db2, dWg=dWg, dbg=dbg, dx=L.dx, dw=L.dw, dg=L.dg,
                   dy_perm=L.dy_perm, dx_perm=L.dx_perm, dh=L.h if recompute else L.dh)
    torch.cuda.synchronize()
    out.update(idx=L.idx, w=L.w, g=L.g, scores=L.scores, counts=L.counts, offsets=L.offsets,
               row_token=L.row_token, pos=L.pos, x_perm=L.x_perm, h=L.h, a=L.a, y_perm=L.y_perm, y=L.y)
    if clobber_h:
        out.update(h=fwd_h, a=fwd_a)
    return {k: v.detach().cpu() for k, v in out.items()}


def oracle_run(wl, inp, backward=True, alive_topk=False):
    f = {n: O.to64(v) for n, v in inp.items() if n != "alive"}
    alive = inp["alive"].cpu().numpy()
    ex = (f["W1"], f["b1"], f["W2"], f["b2"])
    # a bf16 layer keeps h, a, expert outputs and their row gradients in bf16
    store = O.round_bf16 if wl.dtype == "bf16" else None
    fwd = O.layer_forward(f["x"], f["Wg"], f["bg"], ex, alive, wl.d, wl.M, wl.k, wl.act, store=store,
                          alive_topk=alive_topk)
    bwd = O.layer_backward(fwd, f["dy"], f["x"], f["Wg"], ex, alive, wl.d, wl.M, wl.k, wl.act,
                           store=store) if backward else None
    return fwd, bwd


def score_error_bound(x64, Wg64, dtype):
    """Per-score bound on |GPU score - exact score| before the final fp32 rounding.
    fp32 layers accumulate exactly (fp64); bf16 layers sum exact bf16 products in
    fp32 chunks of 32 (MFMA) and add the chunks in fp64: the error is at most
    (gamma_32 + (D/32 + 8) 2^-52) sum_k |x_k w_k|, gamma_n = n u/(1 - n u), u = 2^-23."""
    if dtype != "bf16":
        return np.zeros((x64.shape[0], Wg64.shape[0]))
    D = x64.shape[1]
    u = 2.0 ** -23
    g32 = 32 * u / (1 - 32 * u) + (D // 32 + 8) * 2.0 ** -52
    A = np.abs(x64) @ np.abs(Wg64).T
    return g32 * A * 1.001


def check_gate(wl, gpu_scores, gpu_w, gpu_g, S, w_ref, g_ref, x64, Wg64):
    """Scores within the arithmetic's bound of exact (plus one fp32 rounding); weights
    and totals within the bound that score error implies (softmax: |dw| <= 2 w max|dg|)."""
    delta = score_error_bound(x64, Wg64, wl.dtype)
    sc = O.to64(gpu_scores)
    assert np.all(np.abs(sc - S) <= delta + np.abs(S) * 2.0 ** -23 + 1e-30), "scores"
    dg = wl.d * (delta.max(axis=1) + np.abs(S).max(axis=1) * 2.0 ** -23)     # per token
    tol = 1e-6 + 2.0 * dg[:, None]
    assert np.all(np.abs(O.to64(gpu_w) - w_ref) <= tol * (np.abs(w_ref) + 1e-6) + 1e-6), "w"
    if gpu_g is not None:
        assert np.all(np.abs(O.to64(gpu_g) - g_ref) <= dg[:, None] + 1e-6 * (1 + np.abs(g_ref))), "g"


def compare(wl, inp, gpu, fwd, bwd):
    """Full comparison of one run: integers bit-exact, floats to the tolerance."""
    rtol = RTOL[wl.dtype]
    T, k, N = wl.T, wl.k, wl.N
    check_gate(wl, gpu["scores"], gpu["w"], gpu["g"], fwd["S"], fwd["w"], fwd["g"], O.to64(inp["x"]),
               O.to64(inp["Wg"]))
    # TopK: bit-exact set and order
    np.testing.assert_array_equal(gpu["idx"].numpy(), fwd["idx"], "idx")
    # dispatch: exact
    np.testing.assert_array_equal(gpu["counts"].numpy(), fwd["counts"], "counts")
    np.testing.assert_array_equal(gpu["offsets"].numpy(), fwd["offsets"], "offsets")
    rows = int(fwd["offsets"][-1])
    np.testing.assert_array_equal(gpu["row_token"].numpy()[:rows], fwd["row_token"], "row_token")
    np.testing.assert_array_equal(gpu["pos"].numpy(), fwd["pos"], "pos")
    xp = gpu["x_perm"][:rows]
    assert torch.equal(xp, inp["x"][torch.from_numpy(fwd["row_token"]).long()]), "x_perm"
    if rows:
        assert_close(gpu["h"][:rows], fwd["h"], rtol, "h")
        assert_close(gpu["a"][:rows], fwd["a"], rtol, "a")
        assert_close(gpu["y_perm"][:rows], fwd["y_perm"], rtol, "y_perm")
    assert_close(gpu["y"], fwd["y"], rtol, "y")
    if bwd is None:
        return
    assert_close(gpu["dw"], bwd["dw"], rtol, "dw")
    assert_close(gpu["dg"], bwd["dg"], rtol, "dg")
    if rows:
        assert_close(gpu["dy_perm"][:rows], bwd["dy_perm"], rtol, "dy_perm")
        assert_close(gpu["dx_perm"][:rows], bwd["dx_perm"], rtol, "dx_perm")
    assert_close(gpu["dx"], bwd["dx"], rtol, "dx")
    assert_close(gpu["dWg"], bwd["dWg"], rtol, "dWg")
    assert_close(gpu["dbg"], bwd["dbg"], rtol, "dbg")
    counts = fwd["counts"]
    for e in range(N):
        if counts[e] > 0:
            dW1, db1, dW2, db2 = bwd["expert_grads"][e]
            assert_close(gpu["dW1"][e], dW1, rtol, f"dW1[{e}]")
            assert_close(gpu["db1"][e], db1, rtol, f"db1[{e}]")
            assert_close(gpu["dW2"][e], dW2, rtol, f"dW2[{e}]")
            assert_close(gpu["db2"][e], db2, rtol, f"db2[{e}]")
        else:   # untouched experts keep the caller's contents
            for n in ("dW1", "db1", "dW2", "db2"):
                assert bool((gpu[n][e].float() == 7.0).all()), f"{n}[{e}] was written"
