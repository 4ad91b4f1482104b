"""GPU parity at the full workload sizes, in the launch configuration bench.py times
(the four large Linear-act-Linear workloads, and the LayerNorm block workload in
test_fullsize_ffblock).

Inputs are drawn on the GPU (the weights of the large workloads do not fit the
host) and the oracle reads back what it needs.  Checked against the oracle:
  * every token: gate scores (within one fp32 ulp of exact), TopK indices and
    order (bit-exact), Eq. 1 weights, and the whole dispatch (bit-exact);
  * sampled experts (the busiest and, at the 1024- and 4096-expert workloads, 16
    more spread over the row counts; 4 more at the wide workload, whose experts take
    1 GB each in fp64): h, a and y of all their rows, and in the backward pass
    dy_perm and dx_perm rows and dW1, db1, dW2, db2;
  * sampled tokens: y, dw, dg and dx, computed by the oracle through the token's
    own experts end to end;
  * every token, stage by stage from the GPU's own inputs to the stage, in fp64 on
    the host (Eq. 1 and its derivative): the combine (y from y_perm, w, pos), the
    combine backward (dy_perm and dw from dy, y_perm, w, pos), the softmax gradient
    (dg from w, dw), the dispatch backward (dx from dx_perm, pos and the gate's share
    dg Wg) and the gate layers' gradients (dWg = ds^T x and dbg = sum_t ds, ds built
    from dg and idx).  The bounds are those of the arithmetic: fp32 sums in a fixed
    order and one rounding to the stored dtype.
"""
import gc

import numpy as np
import pytest
import torch

import oracle as O
from parity_util import RTOL, assert_close, check_gate, say
from workloads import get_workload, make_alive, make_dy, make_experts, make_gate, make_x

pytestmark = [pytest.mark.gpu, pytest.mark.slow]

BIG = ["tfm_fwd", "tfm_fail_skew", "grid3d", "wide"]


def _free():
    gc.collect()
    torch.cuda.empty_cache()


U32, U_BF16 = 2.0 ** -24, 2.0 ** -8      # fp32 unit roundoff; bf16 half-ulp relative bound


def _within(gpu, ref, bound, name):
    g = O.to64(gpu)
    assert g.shape == ref.shape, (name, g.shape, ref.shape)
    assert np.isfinite(g).all(), f"{name}: non-finite values"
    bad = np.abs(g - ref) > bound
    if bad.any():
        i = np.unravel_index(np.argmax(np.abs(g - ref) - bound), g.shape)
        raise AssertionError(f"{name}: {int(bad.sum())}/{bad.size} beyond the bound; worst at {i}: "
                             f"gpu {g[i]!r} ref {ref[i]!r} bound {bound[i]!r}")


def stage_checks(wl, L, x, dy, Wg, alive_h, dWg=None, dbg=None, chunk=1024):
    """Every token, each stage from the GPU's own inputs to it (fp64 on the host).
    fp32 accumulation of n terms in a fixed order is within n u sum|terms| of the
    exact sum (u = 2^-24, each product rounded once more), and a bf16 output adds
    one rounding of at most 2^-8 of its value."""
    T, k, D, d, M = wl.T, wl.k, wl.D, wl.d, wl.M
    bf = wl.dtype == "bf16"
    r_out = U_BF16 if bf else U32
    idx_h = L.idx.cpu().numpy()
    pos_h = L.pos.cpu().numpy()
    w_h = L.w.cpu().numpy().astype(np.float64)
    valid = pos_h >= 0
    # grid digits of every chosen expert (u_0 most significant)
    digits = np.stack([(idx_h // M ** (d - 1 - i)) % M for i in range(d)], axis=-1)     # [T, k, d]
    if wl.backward:
        dw_h = L.dw.cpu().numpy().astype(np.float64)
        dg_h = L.dg.cpu().numpy().astype(np.float64)
        # softmax gradient over the alive chosen experts: dg = w (dw - sum_l w_l dw_l)
        wd = np.where(valid, w_h * dw_h, 0.0)
        s = wd.sum(axis=1, keepdims=True)
        dg_ref = np.where(valid, w_h * (dw_h - s), 0.0)
        mag = np.where(valid, np.abs(w_h) * (np.abs(dw_h) + np.abs(wd).sum(axis=1, keepdims=True)), 0.0)
        _within(L.dg, dg_ref, (k + 3) * 2 * U32 * mag + 1e-30, "dg (every token)")
        Wg64 = O.to64(Wg)
    for t0 in range(0, T, chunk):
        t1 = min(T, t0 + chunk)
        p = L.pos[t0:t1].long()
        pc = p.clamp(min=0)
        v = valid[t0:t1]
        wv = np.where(v, w_h[t0:t1], 0.0)
        yp = O.to64(L.y_perm[pc.reshape(-1)]).reshape(t1 - t0, k, D)                    # rows of the pairs
        terms = wv[:, :, None] * yp
        y_ref = terms.sum(axis=1)
        bound = r_out * np.abs(y_ref) + (k + 2) * 2 * U32 * np.abs(terms).sum(axis=1) + 1e-30
        _within(L.y[t0:t1], y_ref, bound, f"y (combine, tokens {t0}..{t1})")
        if not wl.backward:
            continue
        dy64 = O.to64(dy[t0:t1])
        # combine backward: dy_perm rows = w dy (one fp32 product, one rounding), dw = <dy, y_perm row>
        dyp_ref = wv[:, :, None] * dy64[:, None, :]
        dyp = O.to64(L.dy_perm[pc.reshape(-1)]).reshape(t1 - t0, k, D)
        dyp = np.where(v[:, :, None], dyp, 0.0)
        _within(dyp, dyp_ref, (r_out + 2 * U32) * np.abs(dyp_ref) + 1e-30, f"dy_perm (tokens {t0}..{t1})")
        prod = dy64[:, None, :] * yp
        dw_ref = np.where(v, prod.sum(axis=2), 0.0)
        gD = D * U32 / (1 - D * U32)
        _within(L.dw[t0:t1], dw_ref, 2 * gD * np.abs(prod).sum(axis=2) + 1e-30, f"dw (tokens {t0}..{t1})")
        # dispatch backward: dx = sum over alive pairs of dx_perm rows + sum_j dg_j sum_i Wg[i M + u_i]
        dxp = O.to64(L.dx_perm[pc.reshape(-1)]).reshape(t1 - t0, k, D)
        dxp = np.where(v[:, :, None], dxp, 0.0)
        gate_rows = Wg64[(np.arange(d) * M)[None, None, :] + digits[t0:t1]]                # [t, k, d, D]
        gterm = dg_h[t0:t1, :, None, None] * gate_rows
        dx_ref = dxp.sum(axis=1) + gterm.sum(axis=(1, 2))
        mag = np.abs(dxp).sum(axis=1) + np.abs(gterm).sum(axis=(1, 2))
        _within(L.dx[t0:t1], dx_ref, r_out * np.abs(dx_ref) + (k + k * d + 2) * 2 * U32 * mag + 1e-30,
                f"dx (dispatch backward, tokens {t0}..{t1})")
    if wl.backward and dWg is not None:
        # gate layers: ds[t, i M + u_i(idx[t, j])] += dg[t, j]; dWg = ds^T x, dbg = sum_t ds
        ds = np.zeros((T, d * M))
        for j in range(k):
            for i in range(d):
                np.add.at(ds, (np.arange(T), i * M + digits[:, j, i]), dg_h[:, j])
        x64 = O.to64(x)
        rtol = RTOL[wl.dtype]
        assert_close(dWg, ds.T @ x64, rtol, "dWg (every token)")
        if dbg is not None:
            assert_close(dbg, ds.sum(axis=0), rtol, "dbg (every token)")


@pytest.mark.parametrize("name", BIG)
def test_fullsize_parity(name):
    from paper_2002_04013_amd import DMoELayer
    wl = get_workload(name)
    say(f"[fullsize] {name}: T={wl.T} D={wl.D} H={wl.H} grid {wl.M}^{wl.d} k={wl.k} "
        f"p_alive={wl.p_alive} backward={wl.backward}")
    dev = torch.device("cuda")
    store = O.round_bf16
    rtol = RTOL[wl.dtype]
    Wg, bg = make_gate(wl, dev)
    x, dy, alive = make_x(wl, dev), make_dy(wl, dev), make_alive(wl, dev)
    W1, b1, W2, b2 = make_experts(wl, dev)
    L = DMoELayer(wl.T, wl.D, wl.H, wl.d, wl.M, wl.k, wl.dtype, wl.act, device=dev)
    L.forward(x, Wg, bg, alive, W1, b1, W2, b2)
    if wl.backward:
        dW1, db1 = torch.full_like(W1, 7.0), torch.full_like(b1, 7.0)
        dW2, db2 = torch.full_like(W2, 7.0), torch.full_like(b2, 7.0)
        dWg, dbg = torch.empty_like(Wg), torch.empty_like(bg)
        L.backward(dy, x, Wg, alive, W1, W2, dW1, db1, dW2, db2, dWg, dbg)
    torch.cuda.synchronize()
    say(f"[fullsize] {name}: GPU pass done")

    # ---------------------------------------------------------------- routing, every token
    x64, Wg64, bg64 = O.to64(x), O.to64(Wg), O.to64(bg)
    dy64 = O.to64(dy) if wl.backward else None
    alive_h = alive.cpu().numpy()
    S = O.gate_scores(x64, Wg64, bg64)
    S32 = O.decision_scores(S)
    if wl.N <= 1024:
        idx, _ = O.topk_bruteforce(S32, wl.d, wl.M, wl.k)
    else:   # pinned equal to brute force; ranks only the product of per-dimension lists
        idx, _ = O.topk_product_key(S32, wl.d, wl.M, wl.k)
    g = O.chosen_totals(S, idx, wl.d, wl.M)
    w = O.mixture_weights(g, idx, alive_h)
    check_gate(wl, L.scores, L.w, None, S, w, g, x64, Wg64)
    np.testing.assert_array_equal(L.idx.cpu().numpy(), idx, "idx")
    # the exact-accumulation path gives the same routing, bit for bit
    from paper_2002_04013_amd import abi
    idx2 = torch.empty_like(L.idx)
    w2 = torch.empty_like(L.w)
    abi.dmoe_gate_topk(abi.make_dims(wl.T, wl.D, wl.H, wl.d, wl.M, wl.k, wl.dtype, wl.act,
                                     abi.DMOE_FLAG_GATE_EXACT), x, Wg, bg, alive, idx2, w2, None, None, L.ws)
    assert torch.equal(idx2, L.idx), "exact-path routing differs"
    counts, offsets, row_token, pos = O.dispatch(idx, alive_h, wl.N)
    np.testing.assert_array_equal(L.counts.cpu().numpy(), counts, "counts")
    np.testing.assert_array_equal(L.offsets.cpu().numpy(), offsets, "offsets")
    rows_used = int(offsets[-1])
    np.testing.assert_array_equal(L.row_token[:rows_used].cpu().numpy(), row_token, "row_token")
    np.testing.assert_array_equal(L.pos.cpu().numpy(), pos, "pos")
    live = np.nonzero(counts)[0]
    say(f"[fullsize] {name}: routing + dispatch exact; {rows_used} rows, {len(live)} experts used, "
        f"max rows/expert {counts.max()}, dead-token count "
        f"{int((~alive_h[idx].astype(bool)).all(axis=1).sum())}")

    # pair of each row
    row_pair = np.empty(rows_used, np.int64)
    ok = pos >= 0
    row_pair[pos[ok]] = np.nonzero(ok.reshape(-1))[0]

    cache = {}

    def expert(e):
        if e not in cache:
            cache[e] = tuple(O.to64(t[e]) for t in (W1, b1, W2, b2))
        return cache[e]

    # ---------------------------------------------------------------- sampled experts
    rng = np.random.default_rng(0)
    by_count = live[np.argsort(-counts[live], kind="stable")]
    more = 4 if wl.D * wl.H > (1 << 24) else 16        # the wide experts take 1 GB each in fp64
    spread = by_count[np.linspace(1, len(by_count) - 1, more).astype(int)]
    sample_e = sorted({int(by_count[0])} | {int(e) for e in spread})
    for e in sample_e:
        lo, hi = int(offsets[e]), int(offsets[e + 1])
        E1, c1, E2, c2 = expert(e)
        X = x64[row_token[lo:hi]]
        h, a, y = O.expert_forward_stored(X, E1, c1, E2, c2, wl.act, store)
        assert_close(L.h[lo:hi], h, rtol, f"h[e={e}]")
        assert_close(L.a[lo:hi], a, rtol, f"a[e={e}]")
        assert_close(L.y_perm[lo:hi], y, rtol, f"y_perm[e={e}]")
        if wl.backward:
            pr = row_pair[lo:hi]
            wr = w.reshape(-1)[pr]
            dY = store(wr[:, None] * dy64[pr // wl.k])
            dX, gW1, gb1, gW2, gb2 = O.expert_backward(X, h, a, dY, E1, E2, wl.act, store)
            assert_close(L.dy_perm[lo:hi], dY, rtol, f"dy_perm[e={e}]")
            assert_close(L.dx_perm[lo:hi], dX, rtol, f"dx_perm[e={e}]")
            assert_close(dW1[e], gW1, rtol, f"dW1[{e}]")
            assert_close(db1[e], gb1, rtol, f"db1[{e}]")
            assert_close(dW2[e], gW2, rtol, f"dW2[{e}]")
            assert_close(db2[e], gb2, rtol, f"db2[{e}]")
        say(f"[fullsize] {name}: expert {e} ({hi - lo} rows) ok")
        cache.pop(e, None)
    if wl.backward:
        dead = np.nonzero(counts == 0)[0]
        for e in dead[:3]:
            assert bool((dW1[int(e)][:4].float() == 7.0).all()), f"dW1[{e}] written"

    # ---------------------------------------------------------------- sampled tokens
    toks = sorted(set(int(t) for t in rng.choice(wl.T, size=3, replace=False)) |
                  {int(row_token[int(offsets[sample_e[0]])])})
    y_ref, dw_ref, dg_ref, dx_ref = [], [], [], []
    for t in toks:
        yt = np.zeros(wl.D)
        dwt = np.zeros(wl.k)
        saved = []
        for j in range(wl.k):
            e = int(idx[t, j])
            if not alive_h[e]:
                saved.append(None)
                continue
            E1, c1, E2, c2 = expert(e)
            h, a, y = O.expert_forward_stored(x64[t:t + 1], E1, c1, E2, c2, wl.act, store)
            yt += w[t, j] * y[0]
            if wl.backward:
                dwt[j] = float(dy64[t] @ y[0])
            saved.append((h, a, E1, E2))
        y_ref.append(yt)
        if wl.backward:
            dgt, _, dx_gate, _, _ = O.gate_backward(w[t:t + 1], dwt[None, :], idx[t:t + 1], alive_h,
                                                   x64[t:t + 1], Wg64, wl.d, wl.M)
            dxt = dx_gate[0].copy()
            for j in range(wl.k):
                if saved[j] is None:
                    continue
                h, a, E1, E2 = saved[j]
                dY = store(w[t, j] * dy64[t:t + 1])
                dxt += O.expert_backward(x64[t:t + 1], h, a, dY, E1, E2, wl.act, store)[0][0]
            dw_ref.append(dwt)
            dg_ref.append(dgt[0])
            dx_ref.append(dxt)
    tsel = torch.tensor(toks, device=dev)
    assert_close(L.y[tsel], np.array(y_ref), rtol, "y (sampled tokens)")
    if wl.backward:
        assert_close(L.dw[tsel], np.array(dw_ref), rtol, "dw (sampled tokens)")
        assert_close(L.dg[tsel], np.array(dg_ref), rtol, "dg (sampled tokens)")
        assert_close(L.dx[tsel], np.array(dx_ref), rtol, "dx (sampled tokens)")
    say(f"[fullsize] {name}: sampled tokens {toks} ok")
    cache.clear()
    stage_checks(wl, L, x, dy, Wg, alive_h, dWg if wl.backward else None, dbg if wl.backward else None)
    say(f"[fullsize] {name}: every-token stage checks ok")
    del L, W1, b1, W2, b2, x, dy
    if wl.backward:
        del dW1, db1, dW2, db2, dWg, dbg
    _free()


def test_fullsize_ffblock():
    """The LayerNorm feed-forward block workload at full size (131072 tokens, d_model
    1024, blocks 1024 -> 4096 -> 4096 -> 1024, 16x16 grid, top-4), in the launch
    configuration bench.py times.  The LayerNorm scale and shift use the "split"
    initialisation (scale 1/2, shift +-3 per feature) so that no ReLU decision lies
    near its kink (asserted) and the backward compares element by element; the
    kernels and launch shapes do not depend on these values.  Checked: routing and
    dispatch of every token; every kept tensor, row gradient and parameter gradient
    of two sampled experts (the busiest and a median one); y, dw, dg and dx of sampled
    tokens through single-row evaluations of their experts; and every token's combine,
    combine backward, softmax gradient, dispatch backward and gate-layer gradients
    from the GPU's own inputs to each stage (stage_checks)."""
    import dataclasses
    from paper_2002_04013_amd import DMoEBlockLayer
    from workloads import BLOCK_PARAMS, make_block_experts
    wl = dataclasses.replace(get_workload("ffblock"), ln_init="split")
    say(f"[fullsize] ffblock: T={wl.T} D={wl.D} F={wl.H} grid {wl.M}^{wl.d} k={wl.k} ln_init={wl.ln_init}")
    dev = torch.device("cuda")
    store = O.round_bf16
    rtol = RTOL[wl.dtype]
    Wg, bg = make_gate(wl, dev)
    x, dy, alive = make_x(wl, dev), make_dy(wl, dev), make_alive(wl, dev)
    prm = make_block_experts(wl, dev)
    L = DMoEBlockLayer(wl.T, wl.D, wl.H, wl.d, wl.M, wl.k, wl.dtype, wl.act, device=dev)
    L.forward(x, Wg, bg, alive, prm)
    grads = {n: torch.full_like(v, 7.0) for n, v in prm.items()}
    dWg, dbg = torch.empty_like(Wg), torch.empty_like(bg)
    L.backward(dy, x, Wg, alive, prm, grads, dWg, dbg)
    torch.cuda.synchronize()
    say("[fullsize] ffblock: GPU pass done")

    x64, Wg64, bg64, dy64 = O.to64(x), O.to64(Wg), O.to64(bg), O.to64(dy)
    alive_h = alive.cpu().numpy()
    S = O.gate_scores(x64, Wg64, bg64)
    idx, _ = O.topk_bruteforce(O.decision_scores(S), wl.d, wl.M, wl.k)
    g = O.chosen_totals(S, idx, wl.d, wl.M)
    w = O.mixture_weights(g, idx, alive_h)
    check_gate(wl, L.scores, L.w, None, S, w, g, x64, Wg64)
    np.testing.assert_array_equal(L.idx.cpu().numpy(), idx, "idx")
    counts, offsets, row_token, pos = O.dispatch(idx, alive_h, wl.N)
    np.testing.assert_array_equal(L.counts.cpu().numpy(), counts, "counts")
    np.testing.assert_array_equal(L.offsets.cpu().numpy(), offsets, "offsets")
    rows_used = int(offsets[-1])
    np.testing.assert_array_equal(L.row_token[:rows_used].cpu().numpy(), row_token, "row_token")
    np.testing.assert_array_equal(L.pos.cpu().numpy(), pos, "pos")
    live = np.nonzero(counts)[0]
    say(f"[fullsize] ffblock: routing + dispatch exact; {rows_used} rows, max rows/expert {counts.max()}")

    row_pair = np.empty(rows_used, np.int64)
    ok = pos >= 0
    row_pair[pos[ok]] = np.nonzero(ok.reshape(-1))[0]
    cache = {}

    def expert(e):
        if e not in cache:
            cache[e] = {n: O.to64(prm[n][e]) for n in BLOCK_PARAMS}
        return cache[e]

    by_count = live[np.argsort(-counts[live], kind="stable")]
    sample_e = sorted({int(by_count[0]), int(by_count[len(by_count) // 2])})
    for e in sample_e:
        lo, hi = int(offsets[e]), int(offsets[e + 1])
        p = expert(e)
        X = x64[row_token[lo:hi]]
        fw = O.ffblock_forward_stored(X, p, wl.act, store)
        for hn, gn, bn in (("h1", "g1", "be1"), ("h2", "g2", "be2")):
            z = O.layernorm_act_forward(fw[hn], p[gn], p[bn], wl.act)["z"]
            assert np.abs(z).min() > 1e-2, (e, hn, np.abs(z).min())
        for n in ("h1", "a1", "h2", "a2"):
            assert_close(L.acts[n][lo:hi], fw[n], rtol, f"{n}[e={e}]")
        assert_close(L.y_perm[lo:hi], fw["y"], rtol, f"y_perm[e={e}]")
        pr = row_pair[lo:hi]
        dY = store(w.reshape(-1)[pr][:, None] * dy64[pr // wl.k])
        bw = O.ffblock_backward(X, fw, dY, p, wl.act, store)
        assert_close(L.dy_perm[lo:hi], dY, rtol, f"dy_perm[e={e}]")
        assert_close(L.g2[lo:hi], bw["dh2"], rtol, f"dh2[e={e}]")
        assert_close(L.g1[lo:hi], bw["dh1"], rtol, f"dh1[e={e}]")
        assert_close(L.dx_perm[lo:hi], bw["dX"], rtol, f"dx_perm[e={e}]")
        for n in BLOCK_PARAMS:
            assert_close(grads[n][e], bw["grads"][n], rtol, f"d{n}[{e}]")
        say(f"[fullsize] ffblock: expert {e} ({hi - lo} rows) ok")
    for e in np.nonzero(counts == 0)[0][:3]:
        assert bool((grads["W1"][int(e)][:4].float() == 7.0).all()), f"dW1[{e}] written"

    rng = np.random.default_rng(1)
    toks = sorted(int(t) for t in rng.choice(wl.T, size=4, replace=False))
    y_ref, dw_ref, dg_ref, dx_ref = [], [], [], []
    for t in toks:
        yt, dwt, outs = np.zeros(wl.D), np.zeros(wl.k), []
        for j in range(wl.k):
            e = int(idx[t, j])
            if not alive_h[e]:
                outs.append(None)
                continue
            fw = O.ffblock_forward_stored(x64[t:t + 1], expert(e), wl.act, store)
            yt += w[t, j] * fw["y"][0]
            dwt[j] = float(dy64[t] @ fw["y"][0])
            outs.append(fw)
        dgt, _, dx_gate, _, _ = O.gate_backward(w[t:t + 1], dwt[None, :], idx[t:t + 1], alive_h, x64[t:t + 1],
                                               Wg64, wl.d, wl.M)
        dxt = dx_gate[0].copy()
        for j, fw in enumerate(outs):
            if fw is not None:
                dY = store(w[t, j] * dy64[t:t + 1])
                dxt += O.ffblock_backward(x64[t:t + 1], fw, dY, expert(int(idx[t, j])), wl.act, store)["dX"][0]
        y_ref.append(yt)
        dw_ref.append(dwt)
        dg_ref.append(dgt[0])
        dx_ref.append(dxt)
    tsel = torch.tensor(toks, device=dev)
    assert_close(L.y[tsel], np.array(y_ref), rtol, "y (sampled tokens)")
    assert_close(L.dw[tsel], np.array(dw_ref), rtol, "dw (sampled tokens)")
    assert_close(L.dg[tsel], np.array(dg_ref), rtol, "dg (sampled tokens)")
    assert_close(L.dx[tsel], np.array(dx_ref), rtol, "dx (sampled tokens)")
    say(f"[fullsize] ffblock: sampled tokens {toks} ok")
    cache.clear()
    stage_checks(wl, L, x, dy, Wg, alive_h, dWg, dbg)
    say("[fullsize] ffblock: every-token stage checks ok")
    del L, prm, grads, x, dy
    _free()
