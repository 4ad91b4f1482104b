"""Pins of the oracle's feed-forward block expert (Sec. 4.1: linear layers with layer
normalisation and an activation between them), CPU only.

Independent references: torch's layer_norm and nn modules in fp64 with autograd,
the defining invariants of layer normalisation (zero mean and unit variance of the
normalised row; its input gradient orthogonal to the constant row and to the
normalised row; invariance under positive scaling of the input), and central
finite differences through the whole DMoE layer.
"""
import math

import numpy as np
import pytest
import torch

import oracle as O

Fn = torch.nn.functional


def _torch_act(kind):
    return Fn.relu if kind == "relu" else (lambda z: Fn.gelu(z, approximate="none"))


def _params(rng, D, F, ln="standard"):
    """One block's parameters: N(0, 1/fan_in) weights and biases; layer-norm scale and
    shift either at their usual initial values (1, 0) or drawn."""
    p = dict(W1=rng.standard_normal((F, D)) / math.sqrt(D), b1=rng.standard_normal(F) / math.sqrt(D),
             W2=rng.standard_normal((F, F)) / math.sqrt(F), b2=rng.standard_normal(F) / math.sqrt(F),
             W3=rng.standard_normal((D, F)) / math.sqrt(F), b3=rng.standard_normal(D) / math.sqrt(F))
    if ln == "standard":
        p.update(g1=np.ones(F), be1=np.zeros(F), g2=np.ones(F), be2=np.zeros(F))
    else:
        p.update(g1=1 + 0.3 * rng.standard_normal(F), be1=0.2 * rng.standard_normal(F),
                 g2=1 + 0.3 * rng.standard_normal(F), be2=0.2 * rng.standard_normal(F))
    return p


@pytest.mark.parametrize("kind", ["relu", "gelu"])
def test_layernorm_act_forward_vs_torch(kind):
    rng = np.random.default_rng(1)
    h = rng.standard_normal((37, 48)) * 3 + 1.5
    g, b = 1 + 0.5 * rng.standard_normal(48), rng.standard_normal(48)
    f = O.layernorm_act_forward(h, g, b, kind)
    ref = Fn.layer_norm(torch.tensor(h), (48,), torch.tensor(g), torch.tensor(b), eps=O.LN_EPS)
    np.testing.assert_allclose(f["z"], ref.numpy(), rtol=1e-13, atol=1e-13)
    np.testing.assert_allclose(f["a"], _torch_act(kind)(ref).numpy(), rtol=1e-13, atol=1e-13)
    np.testing.assert_allclose(f["mean"], h.mean(axis=1), rtol=1e-14)
    np.testing.assert_allclose(f["rstd"], 1 / np.sqrt(h.var(axis=1) + O.LN_EPS), rtol=1e-13)


@pytest.mark.parametrize("kind", ["relu", "gelu"])
def test_layernorm_act_backward_vs_autograd(kind):
    rng = np.random.default_rng(2)
    h = rng.standard_normal((29, 40)) * 2 - 0.7
    g, b = 1 + 0.5 * rng.standard_normal(40), 0.3 * rng.standard_normal(40)
    da = rng.standard_normal((29, 40))
    dh, dg, db = O.layernorm_act_backward(da, h, g, b, kind)
    th, tg, tb = (torch.tensor(v, requires_grad=True) for v in (h, g, b))
    out = _torch_act(kind)(Fn.layer_norm(th, (40,), tg, tb, eps=O.LN_EPS))
    (out * torch.tensor(da)).sum().backward()
    np.testing.assert_allclose(dh, th.grad.numpy(), rtol=1e-11, atol=1e-12)
    np.testing.assert_allclose(dg, tg.grad.numpy(), rtol=1e-11, atol=1e-12)
    np.testing.assert_allclose(db, tb.grad.numpy(), rtol=1e-11, atol=1e-12)


def test_layernorm_invariants():
    rng = np.random.default_rng(3)
    h = rng.standard_normal((50, 64)) * 5 + 2
    ones, zeros = np.ones(64), np.zeros(64)
    f = O.layernorm_act_forward(h, ones, zeros, "gelu")
    var = h.var(axis=1)
    np.testing.assert_allclose(f["n"].mean(axis=1), 0, atol=1e-14)
    np.testing.assert_allclose((f["n"] ** 2).mean(axis=1), var / (var + O.LN_EPS), rtol=1e-13)
    # the input gradient is orthogonal to the constant row and to the normalised row
    # (exactly so without eps; with eps the second holds up to eps / (var + eps))
    da = rng.standard_normal(h.shape)
    g, b = 1 + rng.standard_normal(64), rng.standard_normal(64)
    dh, _, _ = O.layernorm_act_backward(da, h, g, b, "gelu", eps=0.0)
    n = O.layernorm_act_forward(h, g, b, "gelu", eps=0.0)["n"]
    scale = np.abs(dh).sum(axis=1)
    np.testing.assert_allclose(dh.sum(axis=1) / scale, 0, atol=1e-14)
    np.testing.assert_allclose((dh * n).sum(axis=1) / scale, 0, atol=1e-13)
    # positive scaling of the input leaves the output unchanged and scales dh by 1/c
    c = 7.25
    f1 = O.layernorm_act_forward(h, g, b, "relu", eps=0.0)
    f2 = O.layernorm_act_forward(c * h, g, b, "relu", eps=0.0)
    np.testing.assert_allclose(f2["a"], f1["a"], rtol=1e-13, atol=1e-13)
    d1, _, _ = O.layernorm_act_backward(da, h, g, b, "relu", eps=0.0)
    d2, _, _ = O.layernorm_act_backward(da, c * h, g, b, "relu", eps=0.0)
    np.testing.assert_allclose(d2 * c, d1, rtol=1e-12, atol=1e-13)


@pytest.mark.parametrize("kind", ["relu", "gelu"])
@pytest.mark.parametrize("ln", ["standard", "drawn"])
def test_block_vs_torch_modules(kind, ln):
    """The block as torch nn modules (Linear, LayerNorm, activation) in fp64."""
    rng = np.random.default_rng(4)
    D, F, R = 12, 20, 17
    p = _params(rng, D, F, ln)
    X = rng.standard_normal((R, D))
    dY = rng.standard_normal((R, D))
    fw = O.ffblock_forward_stored(X, p, kind)
    bw = O.ffblock_backward(X, fw, dY, p, kind)
    torch.manual_seed(0)
    l1, l2, l3 = (torch.nn.Linear(D, F).double(), torch.nn.Linear(F, F).double(),
                  torch.nn.Linear(F, D).double())
    n1, n2 = torch.nn.LayerNorm(F, eps=O.LN_EPS).double(), torch.nn.LayerNorm(F, eps=O.LN_EPS).double()
    with torch.no_grad():
        for mod, w, b in ((l1, "W1", "b1"), (l2, "W2", "b2"), (l3, "W3", "b3"),
                          (n1, "g1", "be1"), (n2, "g2", "be2")):
            mod.weight.copy_(torch.tensor(p[w]))
            mod.bias.copy_(torch.tensor(p[b]))
    actf = torch.nn.ReLU() if kind == "relu" else torch.nn.GELU()
    block = torch.nn.Sequential(l1, n1, actf, l2, n2, actf, l3)
    tX = torch.tensor(X, requires_grad=True)
    out = block(tX)
    (out * torch.tensor(dY)).sum().backward()
    np.testing.assert_allclose(fw["y"], out.detach().numpy(), rtol=1e-12, atol=1e-12)
    np.testing.assert_allclose(bw["dX"], tX.grad.numpy(), rtol=1e-10, atol=1e-11)
    for mod, w, b in ((l1, "W1", "b1"), (l2, "W2", "b2"), (l3, "W3", "b3"),
                      (n1, "g1", "be1"), (n2, "g2", "be2")):
        np.testing.assert_allclose(bw["grads"][w], mod.weight.grad.numpy(), rtol=1e-10, atol=1e-11)
        np.testing.assert_allclose(bw["grads"][b], mod.bias.grad.numpy(), rtol=1e-10, atol=1e-11)


def _layer_problem(seed=5, T=14, D=6, F=10, d=2, M=2, k=2, p_alive=1.0, ln="drawn"):
    rng = np.random.default_rng(seed)
    N = M ** d
    P = dict(x=rng.standard_normal((T, D)), Wg=rng.standard_normal((d * M, D)) / math.sqrt(D),
             bg=rng.standard_normal(d * M) / math.sqrt(D), dy=rng.standard_normal((T, D)),
             alive=(rng.random(N) < p_alive).astype(np.uint8), d=d, M=M, k=k)
    P["experts"] = [_params(rng, D, F, ln) for _ in range(N)]
    return P


def _layer(P, kind, x=None, experts=None):
    ex = experts or P["experts"]
    f = O.layer_forward(P["x"] if x is None else x, P["Wg"], P["bg"], lambda e: ex[e], P["alive"], P["d"],
                        P["M"], P["k"], kind, expert="ffblock")
    return f


def test_layer_ffblock_finite_differences():
    P = _layer_problem()
    kind = "gelu"
    fwd = _layer(P, kind)
    bwd = O.layer_backward(fwd, P["dy"], P["x"], P["Wg"], lambda e: P["experts"][e], P["alive"], P["d"],
                           P["M"], P["k"], kind, expert="ffblock")

    def loss(x=None, experts=None):
        f = _layer(P, kind, x, experts)
        assert (f["idx"] == fwd["idx"]).all()      # steps stay inside one routing cell
        return float((f["y"] * P["dy"]).sum())

    eps = 1e-6
    rng = np.random.default_rng(0)
    for _ in range(6):
        i = tuple(rng.integers(0, s) for s in P["x"].shape)
        x = P["x"].copy()
        x[i] += eps
        lp = loss(x=x)
        x[i] -= 2 * eps
        lm = loss(x=x)
        fd = (lp - lm) / (2 * eps)
        assert abs(fd - bwd["dx"][i]) <= 1e-6 * (1 + abs(fd)), (i, fd, bwd["dx"][i])
    e0 = int(fwd["idx"][0, 0])
    for name in ("W1", "g1", "be1", "W2", "b2", "g2", "W3", "b3"):
        arr0 = P["experts"][e0][name]
        i = tuple(rng.integers(0, s) for s in arr0.shape)
        vals = []
        for sgn in (1, -1):
            ex = [dict(q) for q in P["experts"]]
            ex[e0] = {n: v.copy() for n, v in ex[e0].items()}
            ex[e0][name][i] += sgn * eps
            vals.append(loss(experts=ex))
        fd = (vals[0] - vals[1]) / (2 * eps)
        an = bwd["expert_grads"][e0][name][i]
        assert abs(fd - an) <= 1e-6 * (1 + abs(fd)), (name, i, fd, an)


def test_layer_ffblock_identical_experts():
    """All experts equal: y = f(x) for every token with an alive chosen expert."""
    P = _layer_problem(seed=6, T=20, p_alive=0.75)
    for e in range(1, len(P["experts"])):
        P["experts"][e] = P["experts"][0]
    f = _layer(P, "relu")
    single = O.ffblock_forward_stored(P["x"], P["experts"][0], "relu")["y"]
    live = P["alive"][f["idx"]].astype(bool).any(axis=1)
    np.testing.assert_allclose(f["y"][live], single[live], rtol=1e-12, atol=1e-13)
    assert (f["y"][~live] == 0).all()


def test_block_storage_rounding_stays_at_bf16_level():
    """The bf16 storage model only perturbs at the bf16 rounding level."""
    rng = np.random.default_rng(7)
    D, F, R = 16, 32, 24
    p = _params(rng, D, F, "drawn")
    X = O.round_bf16(rng.standard_normal((R, D)))
    dY = O.round_bf16(rng.standard_normal((R, D)))
    exact = O.ffblock_forward_stored(X, p, "gelu")
    st = O.ffblock_forward_stored(X, p, "gelu", store=O.round_bf16)
    for n in ("h1", "a1", "h2", "a2", "y"):
        assert np.array_equal(O.round_bf16(st[n]), st[n]), n
        rel = np.abs(st[n] - exact[n]).max() / np.abs(exact[n]).max()
        assert rel < 2.0 ** -6, (n, rel)
    bx = O.ffblock_backward(X, exact, dY, p, "gelu")
    bs = O.ffblock_backward(X, st, dY, p, "gelu", store=O.round_bf16)
    rel = np.abs(bs["dX"] - bx["dX"]).max() / np.abs(bx["dX"]).max()
    assert rel < 2.0 ** -5, rel
