"""The feed-forward block expert of Sec. 4.1 -- TEST INFRASTRUCTURE ONLY.

Sec. 4.1 describes its experts as feed-forward blocks of hidden sizes
1024 -> 4096 -> 4096 -> 1024 with layer normalisation and ReLU between the
layers.  Read here as

    h1 = x W1^T + b1,  a1 = act(LN(h1; g1, be1)),
    h2 = a1 W2^T + b2, a2 = act(LN(h2; g2, be2)),
    y  = a2 W3^T + b3,

with LN(h; g, b) = g * (h - mean(h)) / sqrt(var(h) + eps) + b over the features
of one row (the biased variance layer normalisation defines) and eps = 1e-5.
Plain fp64 NumPy; nothing here is shared with the HIP path.
"""
import numpy as np

from .dmoe import act, act_grad, _identity

LN_EPS = 1e-5

PARAM_NAMES = ("W1", "b1", "g1", "be1", "W2", "b2", "g2", "be2", "W3", "b3")


def layernorm_act_forward(h, gamma, beta, kind, eps=LN_EPS):
    """Layer normalisation of each row followed by the activation:
    mean = sum_f h_f / F, var = sum_f (h_f - mean)^2 / F, rstd = 1 / sqrt(var + eps),
    n = (h - mean) rstd, z = gamma n + beta, a = act(z).
    Returns dict(mean, rstd, n, z, a) (mean and rstd per row)."""
    h = np.asarray(h, np.float64)
    F = h.shape[-1]
    mean = h.sum(axis=-1) / F
    c = h - mean[..., None]
    var = (c * c).sum(axis=-1) / F
    rstd = 1.0 / np.sqrt(var + eps)
    n = c * rstd[..., None]
    z = np.asarray(gamma, np.float64) * n + np.asarray(beta, np.float64)
    return dict(mean=mean, rstd=rstd, n=n, z=z, a=act(z, kind))


def layernorm_act_backward(da, h, gamma, beta, kind, eps=LN_EPS):
    """Backward of layernorm_act_forward over a batch of rows, given the output
    gradient da: dz = da act'(z), dgamma = sum over rows of dz n, dbeta = sum over
    rows of dz, and with dn = dz gamma the input gradient
        dh = rstd (dn - mean_f(dn) - n mean_f(dn n))
    (n depends on h directly and through mean and rstd).  Returns (dh, dgamma, dbeta)."""
    f = layernorm_act_forward(h, gamma, beta, kind, eps)
    n, z, rstd = f["n"], f["z"], f["rstd"]
    da = np.asarray(da, np.float64)
    F = n.shape[-1]
    dz = da * act_grad(z, kind)
    dgamma = (dz * n).sum(axis=0)
    dbeta = dz.sum(axis=0)
    dn = dz * np.asarray(gamma, np.float64)
    m1 = dn.sum(axis=-1, keepdims=True) / F
    m2 = (dn * n).sum(axis=-1, keepdims=True) / F
    dh = rstd[:, None] * (dn - m1 - n * m2)
    return dh, dgamma, dbeta


def ffblock_forward_stored(X, p, kind, store=None):
    """The block on a batch of rows X, as a layer with storage dtype `store` keeps it:
    each linear layer's output (h1, h2, y) and each activation (a1, a2) is rounded
    to the storage dtype, and the next step reads the rounded value; the layer
    normalisation statistics are those of the rounded h.  p maps PARAM_NAMES to one
    expert's fp64 parameters.  Returns dict(h1, a1, mean1, rstd1, h2, a2, mean2,
    rstd2, y)."""
    store = store or _identity
    X = np.asarray(X, np.float64)
    h1 = store(X @ p["W1"].T + p["b1"][None, :])
    l1 = layernorm_act_forward(h1, p["g1"], p["be1"], kind)
    a1 = store(l1["a"])
    h2 = store(a1 @ p["W2"].T + p["b2"][None, :])
    l2 = layernorm_act_forward(h2, p["g2"], p["be2"], kind)
    a2 = store(l2["a"])
    y = store(a2 @ p["W3"].T + p["b3"][None, :])
    return dict(h1=h1, a1=a1, mean1=l1["mean"], rstd1=l1["rstd"],
                h2=h2, a2=a2, mean2=l2["mean"], rstd2=l2["rstd"], y=y)


def ffblock_backward(X, fw, dY, p, kind, store=None):
    """Gradients of the block for a batch, from the stored forward tensors fw:
        dW3 = dY^T a2, db3 = sum dY, da2 = dY W3,
        (dh2, dg2, dbe2) = LN-act backward of da2 at h2,
        dW2 = dh2^T a1, db2 = sum dh2, da1 = dh2 W2,
        (dh1, dg1, dbe1) = LN-act backward of da1 at h1,
        dW1 = dh1^T X, db1 = sum dh1, dX = dh1 W1.
    store rounds the row gradients a layer keeps in its storage dtype (da2, dh2,
    da1, dh1, dX).  Returns dict(dX, dh2, dh1, grads) with grads keyed by
    PARAM_NAMES."""
    store = store or _identity
    X = np.asarray(X, np.float64)
    dY = np.asarray(dY, np.float64)
    g = {}
    g["W3"] = dY.T @ fw["a2"]
    g["b3"] = dY.sum(axis=0)
    da2 = store(dY @ p["W3"])
    dh2, g["g2"], g["be2"] = layernorm_act_backward(da2, fw["h2"], p["g2"], p["be2"], kind)
    dh2 = store(dh2)
    g["W2"] = dh2.T @ fw["a1"]
    g["b2"] = dh2.sum(axis=0)
    da1 = store(dh2 @ p["W2"])
    dh1, g["g1"], g["be1"] = layernorm_act_backward(da1, fw["h1"], p["g1"], p["be1"], kind)
    dh1 = store(dh1)
    g["W1"] = dh1.T @ X
    g["b1"] = dh1.sum(axis=0)
    dX = store(dh1 @ p["W1"])
    return dict(dX=dX, dh2=dh2, dh1=dh1, grads=g)
