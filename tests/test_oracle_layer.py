"""Pins of the oracle's weights, experts, dispatch and backward (CPU only).

Independent references: hand-worked fixtures, scipy/torch library routines,
torch.autograd on a dense fp64 reformulation of the layer (written here with
torch ops only), central finite differences and invariants of Eq. 1.
"""
import math
import zlib

import numpy as np
import pytest
import torch
from scipy.special import softmax

import oracle as O
from conftest import read_golden


# ------------------------------------------------------------------ weights

def test_weights_golden_dyadic():
    rows = read_golden("weights_dyadic.txt")
    g = None
    alive = None
    checked = 0
    for key, vals in rows:
        if key == "g":
            g = np.array([[{"ln4": math.log(4), "ln2": math.log(2)}.get(v, None) or float(v)
                           for v in vals]])
        elif key == "alive":
            alive = np.array([int(v) for v in vals], np.uint8)
        elif key == "w":
            idx = np.arange(4)[None, :]
            w = O.mixture_weights(g, idx, alive)
            np.testing.assert_allclose(w[0], [float(v) for v in vals], rtol=1e-15, atol=1e-16)
            checked += 1
    assert checked == 4


def test_weights_dense_softmax_k_equals_N():
    rng = np.random.default_rng(0)
    S32 = rng.standard_normal((20, 7)).astype(np.float32)
    idx, g = O.topk_bruteforce(S32, 1, 7, 7)
    w = O.mixture_weights(g, idx, None)
    dense = softmax(S32.astype(np.float64), axis=1)
    np.testing.assert_allclose(w, np.take_along_axis(dense, idx, 1), rtol=1e-14, atol=1e-16)


def test_weights_invariants():
    rng = np.random.default_rng(1)
    T, k, N = 200, 4, 16
    g = -np.sort(-rng.standard_normal((T, k)) * 3, axis=1)     # non-increasing like TopK output
    idx = np.stack([rng.permutation(N)[:k] for _ in range(T)])
    alive = (rng.random(N) < 0.6).astype(np.uint8)
    w = O.mixture_weights(g, idx, alive)
    live = alive[idx].astype(bool)
    any_live = live.any(axis=1)
    np.testing.assert_allclose(w[any_live].sum(axis=1), 1.0, rtol=0, atol=4 * k * 2.0 ** -52)
    assert (w[~live] == 0).all()
    assert (w[~any_live] == 0).all()
    for t in range(T):   # non-increasing over alive slots
        ws = w[t][live[t]]
        assert (np.diff(ws) <= 1e-15).all()
    # translation invariance of Eq. 1
    np.testing.assert_allclose(O.mixture_weights(g + 123.0, idx, alive), w, rtol=1e-12, atol=1e-15)


# ------------------------------------------------------------------ activations, experts

def test_gelu_matches_torch():
    h = np.linspace(-8, 8, 4001)
    ref = torch.nn.functional.gelu(torch.from_numpy(h), approximate="none").numpy()
    np.testing.assert_allclose(O.act(h, "gelu"), ref, rtol=1e-14, atol=1e-15)
    np.testing.assert_array_equal(O.act(h, "relu"), torch.relu(torch.from_numpy(h)).numpy())


def test_act_grad_matches_autograd_and_fd():
    h = torch.linspace(-6, 6, 1201, dtype=torch.float64, requires_grad=True)
    torch.nn.functional.gelu(h, approximate="none").sum().backward()
    np.testing.assert_allclose(O.act_grad(h.detach().numpy(), "gelu"), h.grad.numpy(),
                               rtol=1e-13, atol=1e-14)
    x = np.linspace(-5, 5, 101)
    eps = 1e-6
    fd = (O.act(x + eps, "gelu") - O.act(x - eps, "gelu")) / (2 * eps)
    np.testing.assert_allclose(O.act_grad(x, "gelu"), fd, rtol=1e-7, atol=1e-8)
    assert O.act_grad(np.array([0.0]), "relu")[0] == 0.0
    assert O.act_grad(np.array([1e-30]), "relu")[0] == 1.0


def test_expert_forward_backward_vs_torch():
    rng = np.random.default_rng(2)
    X = rng.standard_normal((9, 16))
    W1, b1 = rng.standard_normal((32, 16)), rng.standard_normal(32)
    W2, b2 = rng.standard_normal((16, 32)), rng.standard_normal(16)
    dY = rng.standard_normal((9, 16))
    for kind in ("relu", "gelu"):
        h, a, y = O.expert_forward(X, W1, b1, W2, b2, kind)
        tX, tW1, tb1, tW2, tb2 = (torch.tensor(v, requires_grad=True) for v in (X, W1, b1, W2, b2))
        F = torch.nn.functional
        act = F.relu if kind == "relu" else (lambda z: F.gelu(z, approximate="none"))
        ty = F.linear(act(F.linear(tX, tW1, tb1)), tW2, tb2)
        np.testing.assert_allclose(y, ty.detach().numpy(), rtol=1e-12, atol=1e-12)
        (ty * torch.from_numpy(dY)).sum().backward()
        dX, dW1, db1, dW2, db2 = O.expert_backward(X, h, a, dY, W1, W2, kind)
        for mine, ref in ((dX, tX), (dW1, tW1), (db1, tb1), (dW2, tW2), (db2, tb2)):
            np.testing.assert_allclose(mine, ref.grad.numpy(), rtol=1e-11, atol=1e-11)


# ------------------------------------------------------------------ dispatch

def _dispatch_loops(idx, alive, N):
    T, k = idx.shape
    rows = []
    for e in range(N):
        if not alive[e]:
            continue
        for t in range(T):
            for j in range(k):
                if idx[t, j] == e:
                    rows.append((e, t, j))
    counts = [sum(1 for r in rows if r[0] == e) for e in range(N)]
    pos = -np.ones((T, k), np.int64)
    for n, (e, t, j) in enumerate(rows):
        pos[t, j] = n
    return np.array(counts), np.array([r[1] for r in rows], np.int64), pos


def test_dispatch_vs_loops():
    rng = np.random.default_rng(3)
    for T, k, N, p in [(30, 2, 8, 1.0), (50, 4, 16, 0.7), (7, 3, 5, 0.0), (1, 1, 1, 1.0)]:
        idx = np.stack([rng.permutation(N)[:k] for _ in range(T)])
        alive = (rng.random(N) < p).astype(np.uint8)
        counts, offsets, row_token, pos = O.dispatch(idx, alive, N)
        c2, rt2, pos2 = _dispatch_loops(idx, alive, N)
        np.testing.assert_array_equal(counts, c2)
        np.testing.assert_array_equal(row_token, rt2)
        np.testing.assert_array_equal(pos, pos2)
        assert offsets[0] == 0 and (np.diff(offsets) == counts).all()


def test_undispatch_of_dispatch_is_k_fold_sum():
    rng = np.random.default_rng(4)
    T, k, N, D = 40, 3, 10, 5
    idx = np.stack([rng.permutation(N)[:k] for _ in range(T)])
    alive = np.ones(N, np.uint8)
    x = rng.standard_normal((T, D))
    counts, offsets, row_token, pos = O.dispatch(idx, alive, N)
    xp = x[row_token]
    back = np.zeros_like(x)
    for j in range(k):
        back += xp[pos[:, j]]
    np.testing.assert_allclose(back, k * x, rtol=1e-15)


# ------------------------------------------------------------------ whole layer

def _problem(T=48, D=16, H=24, d=2, M=3, k=3, p=0.8, seed=0, identical=False):
    rng = np.random.default_rng(seed)
    N = M ** d
    x = rng.standard_normal((T, D))
    Wg = rng.standard_normal((d * M, D)) / math.sqrt(D)
    bg = rng.standard_normal(d * M) / math.sqrt(D)
    W1 = rng.standard_normal((N, H, D)) / math.sqrt(D)
    b1 = rng.standard_normal((N, H)) / math.sqrt(D)
    W2 = rng.standard_normal((N, D, H)) / math.sqrt(H)
    b2 = rng.standard_normal((N, D)) / math.sqrt(H)
    if identical:
        W1[:], b1[:], W2[:], b2[:] = W1[0], b1[0], W2[0], b2[0]
    alive = (rng.random(N) < p).astype(np.uint8)
    dy = rng.standard_normal((T, D))
    return dict(x=x, Wg=Wg, bg=bg, W1=W1, b1=b1, W2=W2, b2=b2, alive=alive, dy=dy,
                d=d, M=M, k=k)


def _run(P, kind):
    ex = (P["W1"], P["b1"], P["W2"], P["b2"])
    fwd = O.layer_forward(P["x"], P["Wg"], P["bg"], ex, P["alive"], P["d"], P["M"], P["k"], kind)
    bwd = O.layer_backward(fwd, P["dy"], P["x"], P["Wg"], ex, P["alive"], P["d"], P["M"],
                           P["k"], kind)
    return fwd, bwd


def _torch_dense_layer(P, kind):
    """Dense fp64 reformulation with torch ops only: every expert on every token,
    TopK by torch.topk over all cell totals, Eq. 1 weights by a masked softmax."""
    F = torch.nn.functional
    t = {n: torch.tensor(P[n], requires_grad=True) for n in ("x", "Wg", "bg", "W1", "b1", "W2", "b2")}
    d, M, k = P["d"], P["M"], P["k"]
    S = F.linear(t["x"], t["Wg"], t["bg"])
    S32 = S.detach().float().double()          # decisions on fp32 scores
    T = S.shape[0]
    tot_dec = torch.zeros(T, 1, dtype=torch.float64)
    tot = torch.zeros(T, 1, dtype=torch.float64)
    for i in range(d):
        tot_dec = (tot_dec[:, :, None] + S32[:, None, i * M:(i + 1) * M]).reshape(T, -1)
        tot = (tot[:, :, None] + S[:, None, i * M:(i + 1) * M]).reshape(T, -1)
    _, idx = torch.topk(tot_dec, k, dim=1)
    g = torch.gather(tot, 1, idx)
    live = torch.from_numpy(P["alive"].astype(bool))[idx]
    logits = g.masked_fill(~live, float("-inf"))
    w = torch.softmax(logits, dim=1)
    w = torch.where(live, w, torch.zeros_like(w))
    w = torch.nan_to_num(w, nan=0.0)
    act = F.relu if kind == "relu" else (lambda z: F.gelu(z, approximate="none"))
    h = torch.einsum("td,nhd->tnh", t["x"], t["W1"]) + t["b1"][None]
    yall = torch.einsum("tnh,ndh->tnd", act(h), t["W2"]) + t["b2"][None]       # [T, N, D]
    ysel = torch.gather(yall, 1, idx[:, :, None].expand(-1, -1, yall.shape[2]))
    y = (w[:, :, None] * ysel).sum(1)
    (y * torch.from_numpy(P["dy"])).sum().backward()
    return idx.numpy(), w.detach().numpy(), y.detach().numpy(), {n: v.grad.numpy() for n, v in t.items()}


@pytest.mark.parametrize("kind", ["relu", "gelu"])
@pytest.mark.parametrize("shape", [dict(d=2, M=3, k=3, p=0.8), dict(d=3, M=2, k=4, p=0.6),
                                   dict(d=1, M=6, k=6, p=1.0), dict(d=2, M=4, k=2, p=0.3)])
def test_layer_vs_torch_autograd(kind, shape):
    P = _problem(seed=zlib.crc32(repr((kind, sorted(shape.items()))).encode()) % 1000, **shape)
    fwd, bwd = _run(P, kind)
    idx, w, y, grads = _torch_dense_layer(P, kind)
    np.testing.assert_array_equal(fwd["idx"], idx)
    np.testing.assert_allclose(fwd["w"], w, rtol=1e-12, atol=1e-14)
    np.testing.assert_allclose(fwd["y"], y, rtol=1e-11, atol=1e-12)
    np.testing.assert_allclose(bwd["dx"], grads["x"], rtol=1e-10, atol=1e-11)
    np.testing.assert_allclose(bwd["dWg"], grads["Wg"], rtol=1e-10, atol=1e-11)
    np.testing.assert_allclose(bwd["dbg"], grads["bg"], rtol=1e-10, atol=1e-11)
    N = P["M"] ** P["d"]
    for e in range(N):
        if e in bwd["expert_grads"]:
            dW1, db1, dW2, db2 = bwd["expert_grads"][e]
        else:
            dW1 = db1 = dW2 = db2 = 0.0
        np.testing.assert_allclose(dW1, grads["W1"][e], rtol=1e-10, atol=1e-11)
        np.testing.assert_allclose(db1, grads["b1"][e], rtol=1e-10, atol=1e-11)
        np.testing.assert_allclose(dW2, grads["W2"][e], rtol=1e-10, atol=1e-11)
        np.testing.assert_allclose(db2, grads["b2"][e], rtol=1e-10, atol=1e-11)


def test_layer_finite_differences():
    P = _problem(T=12, D=8, H=10, d=2, M=3, k=2, p=1.0, seed=11)
    kind = "gelu"
    fwd, bwd = _run(P, kind)
    ex = lambda Q: (Q["W1"], Q["b1"], Q["W2"], Q["b2"])

    def loss(Q):
        f = O.layer_forward(Q["x"], Q["Wg"], Q["bg"], ex(Q), Q["alive"], 2, 3, 2, kind)
        assert (f["idx"] == fwd["idx"]).all()      # steps stay inside one routing cell
        return float((f["y"] * Q["dy"]).sum())

    eps = 1e-6
    rng = np.random.default_rng(0)
    checks = [("x", bwd["dx"]), ("Wg", bwd["dWg"])]
    e0 = int(fwd["idx"][0, 0])
    for name, grad in checks + [("W1", None), ("b2", None)]:
        for _ in range(4):
            Q = {n: (v.copy() if isinstance(v, np.ndarray) else v) for n, v in P.items()}
            if name in ("W1", "b2"):
                arr = Q[name][e0]
                i = tuple(rng.integers(0, s) for s in arr.shape)
                g_idx = {"W1": 0, "b2": 3}[name]
                an = bwd["expert_grads"][e0][g_idx][i]
            else:
                arr = Q[name]
                i = tuple(rng.integers(0, s) for s in arr.shape)
                an = grad[i]
            base = arr[i]
            arr[i] = base + eps
            lp = loss(Q)
            arr[i] = base - eps
            lm = loss(Q)
            arr[i] = base
            fd = (lp - lm) / (2 * eps)
            assert abs(fd - an) <= 1e-6 * (1 + abs(an)), (name, i, fd, an)


def test_identical_experts_reproduce_single_expert():
    P = _problem(T=64, D=12, H=20, d=2, M=4, k=3, p=0.7, seed=5, identical=True)
    fwd, bwd = _run(P, "gelu")
    _, _, y1 = O.expert_forward(P["x"], P["W1"][0], P["b1"][0], P["W2"][0], P["b2"][0], "gelu")
    any_live = P["alive"][fwd["idx"]].astype(bool).any(axis=1)
    np.testing.assert_allclose(fwd["y"][any_live], y1[any_live], rtol=1e-12, atol=1e-12)
    assert (fwd["y"][~any_live] == 0).all()
    # the output does not depend on the gate: its gradients vanish
    np.testing.assert_allclose(bwd["dg"], 0, atol=1e-12)
    np.testing.assert_allclose(bwd["dWg"], 0, atol=1e-11)
    np.testing.assert_allclose(bwd["dbg"], 0, atol=1e-11)


def test_token_permutation_equivariance():
    P = _problem(T=40, d=2, M=3, k=3, p=0.8, seed=9)
    fwd, bwd = _run(P, "relu")
    perm = np.random.default_rng(1).permutation(40)
    Q = dict(P, x=P["x"][perm], dy=P["dy"][perm])
    fwd2, bwd2 = _run(Q, "relu")
    np.testing.assert_array_equal(fwd2["idx"], fwd["idx"][perm])
    np.testing.assert_allclose(fwd2["y"], fwd["y"][perm], rtol=1e-13, atol=1e-13)
    np.testing.assert_allclose(bwd2["dx"], bwd["dx"][perm], rtol=1e-12, atol=1e-12)
    np.testing.assert_allclose(bwd2["dWg"], bwd["dWg"], rtol=1e-11, atol=1e-12)


def test_all_dead_tokens_are_zero():
    P = _problem(T=30, d=2, M=3, k=2, p=0.0, seed=3)
    fwd, bwd = _run(P, "gelu")
    assert (fwd["y"] == 0).all() and (fwd["w"] == 0).all()
    assert (bwd["dx"] == 0).all() and (bwd["dWg"] == 0).all()
    assert fwd["offsets"][-1] == 0


# ------------------------------------------------------------------ bf16 storage rounding

def test_round_bf16_matches_torch_and_ties_to_even():
    g = torch.Generator().manual_seed(0)
    v = torch.randn(100000, generator=g) * torch.exp(torch.randn(100000, generator=g) * 5)
    ref = v.to(torch.bfloat16).double().numpy()
    np.testing.assert_array_equal(O.round_bf16(v.double().numpy()), ref)
    # exact halfway cases: 1 + 2^-8 lies between 1 and 1 + 2^-7 -> even (1.0);
    # 1 + 3*2^-8 lies between 1 + 2^-7 and 1 + 2^-6 -> even (1 + 2^-6)
    np.testing.assert_array_equal(O.round_bf16(np.array([1 + 2.0 ** -8, 1 + 3 * 2.0 ** -8, -(1 + 2.0 ** -8)])),
                                  [1.0, 1 + 2.0 ** -6, -1.0])
    assert O.round_bf16(np.array([0.0]))[0] == 0.0


def test_storage_rounding_only_perturbs_at_bf16_level():
    P = _problem(T=64, D=16, H=24, d=2, M=3, k=3, p=0.8, seed=21)
    ex = (P["W1"], P["b1"], P["W2"], P["b2"])
    args = (P["x"], P["Wg"], P["bg"], ex, P["alive"], 2, 3, 3, "gelu")
    f0 = O.layer_forward(*args)
    f1 = O.layer_forward(*args, store=O.round_bf16)
    np.testing.assert_array_equal(f0["idx"], f1["idx"])
    np.testing.assert_array_equal(f1["h"], O.round_bf16(f0["h"]))
    np.testing.assert_array_equal(f1["a"], O.round_bf16(f0["a"]))
    rms = np.sqrt(np.mean(f0["y"] ** 2))
    assert np.max(np.abs(f1["y"] - f0["y"])) < 2 ** -6 * rms
    b0 = O.layer_backward(f0, P["dy"], P["x"], P["Wg"], ex, P["alive"], 2, 3, 3, "gelu")
    b1 = O.layer_backward(f1, P["dy"], P["x"], P["Wg"], ex, P["alive"], 2, 3, 3, "gelu",
                          store=O.round_bf16)
    for n in ("dx", "dWg"):
        rms = np.sqrt(np.mean(b0[n] ** 2))
        assert np.max(np.abs(b1[n] - b0[n])) < 2 ** -5 * rms, n


def test_sgd_step_pins():
    """W - lr dW with one rounding to the storage dtype."""
    W = np.array([1.0, -2.0, 0.5, 3.0])
    g = np.array([2.0, -4.0, 0.25, 0.0])
    np.testing.assert_array_equal(O.sgd_step(W, g, 0.5), [0.0, 0.0, 0.375, 3.0])
    np.testing.assert_array_equal(O.sgd_step(W, g, 0.0), W)
    # just below 1 the bf16 values (8 significant bits) are 2^-8 apart: 1 - 2^-8 and 1.
    # 1 - 2^-9 is the halfway case and rounds to the even significand, 1.0;
    # 1 - 3 * 2^-10 is nearer to 1 - 2^-8
    assert O.sgd_step(np.array([1.0]), np.array([2.0 ** -9]), 1.0, O.round_bf16)[0] == 1.0
    assert O.sgd_step(np.array([1.0]), np.array([3 * 2.0 ** -10]), 1.0, O.round_bf16)[0] == 1.0 - 2.0 ** -8
    # fp32 rounding: 1 + 2^-25 is below half an ulp of 1 (2^-24)
    assert O.sgd_step(np.array([1.0]), np.array([-(2.0 ** -25)]), 1.0, O.round_f32)[0] == 1.0
    assert O.sgd_step(np.array([1.0]), np.array([-(2.0 ** -23)]), 1.0, O.round_f32)[0] == 1.0 + 2.0 ** -23
