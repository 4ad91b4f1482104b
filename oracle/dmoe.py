"""fp64 NumPy oracle of one DMoE layer, forward and backward (test infrastructure only).

Conventions (the readings are listed with their reasons in the design notes):
  * Gate layer i owns columns [i*M, (i+1)*M) of the score matrix S [T, d*M].
  * Expert uid (u_0, ..., u_{d-1}) has flat index sum_i u_i * M**(d-1-i): u_0 is
    the most significant digit, so flat order is the order of uid prefixes
    (App. C keys experts by uid prefix, leftmost dimension first).
  * Selection compares the fp32 rounding of the exact scores; a cell's total
    g(x, f) adds the d fp32 scores in fp64 in dimension order.  Ties in g are
    broken by the lower flat index, ties inside one dimension by the lower index.
  * Expert weights use the nn.Linear layout [out, in].
"""
import itertools

import numpy as np
from scipy.special import erf

SQRT2 = np.sqrt(2.0)
SQRT2PI = np.sqrt(2.0 * np.pi)


def to64(a):
    """fp64 NumPy copy of a NumPy array or a torch tensor (bf16 widens exactly)."""
    if hasattr(a, "detach"):
        a = a.detach().to("cpu")
        if a.dtype.is_floating_point:
            a = a.double()
        a = a.numpy()
    return np.asarray(a, dtype=np.float64)


def round_bf16(a):
    """Round to the nearest value with 8 significant bits (bf16), ties to even.
    This is the storage rounding of a layer whose activations are kept in bf16
    (normal range; bf16 shares fp32's exponent range)."""
    a = np.asarray(a, np.float64)
    m, e = np.frexp(a)                      # a = m 2^e, 0.5 <= |m| < 1
    return np.ldexp(np.rint(m * 256.0) / 256.0, e)


def _identity(a):
    return a


# ---------------------------------------------------------------- gating (Sec. 3.2)

def gate_scores(x, Wg, bg=None):
    """S = [g_0(x) | ... | g_{d-1}(x)]: the d linear layers of the structured gate
    (Sec. 3.2; App. C), each mapping d_model to M scores.  Exact products in fp64."""
    S = np.asarray(x, np.float64) @ np.asarray(Wg, np.float64).T
    if bg is not None:
        S = S + np.asarray(bg, np.float64)[None, :]
    return S


def decision_scores(S):
    """The per-dimension scores that selection compares: fp32 rounding of S."""
    return np.asarray(S, np.float64).astype(np.float32)


def flat_index(u, M):
    """uid tuple(s) (..., d) -> flat expert index, u_0 most significant."""
    u = np.asarray(u, np.int64)
    f = np.zeros(u.shape[:-1], np.int64)
    for i in range(u.shape[-1]):
        f = f * M + u[..., i]
    return f


def uid_of(flat, d, M):
    """flat expert index -> uid (..., d)."""
    flat = np.asarray(flat, np.int64)
    u = np.empty(flat.shape + (d,), np.int64)
    rem = flat.copy()
    for i in range(d - 1, -1, -1):
        u[..., i] = rem % M
        rem //= M
    return u


def cell_totals(S32, d, M):
    """g(x, f) = sum_i g_i(x)[u_i] for every cell f of the grid (Sec. 3.2), as a
    [T, M**d] array whose column is the flat index.  fp64 sum in dim order."""
    S32 = np.asarray(S32)
    T = S32.shape[0]
    g = np.zeros((T, 1), np.float64)
    for i in range(d):
        s = S32[:, i * M:(i + 1) * M].astype(np.float64)
        g = (g[:, :, None] + s[:, None, :]).reshape(T, -1)
    return g


def _rank_desc(values, ids):
    """Order of positions by (value desc, id asc)."""
    return np.lexsort((np.asarray(ids), -np.asarray(values, np.float64)))


def topk_bruteforce(S32, d, M, k):
    """TopK of Eq. 1 by its definition: rank every grid cell by its total g (ties:
    lower flat index first) and keep the first k.  Returns idx [T,k], g [T,k]."""
    g = cell_totals(S32, d, M)
    T, N = g.shape
    if not 1 <= k <= N:
        raise ValueError("k must be in [1, M**d]")
    flat = np.broadcast_to(np.arange(N), (T, N))
    order = np.lexsort((flat, -g), axis=-1)[:, :k]
    return order.astype(np.int64), np.take_along_axis(g, order, axis=1)


def topk_beam(S32, d, M, k, active=None):
    """The dimension-by-dimension search of Algorithm 1 (App. C), for all tokens at
    once.  A beam of at most k uid prefixes (as flat codes of their leading digits)
    starts as the k best indices of grid dimension 0 by their score g_0; dimension i
    then extends every kept prefix by each index j whose longer prefix leads to an
    expert that exists, the candidate's score being the prefix score plus g_i(x)[j]
    (fp64, in dimension order), and keeps the k best candidates, ties to the
    lexicographically smaller prefix.  active: bool [M**d] marking the experts that
    exist, or None for the fully populated grid.  Raises if some token's beam ends
    with fewer than k prefixes."""
    S32 = np.asarray(S32)
    T = S32.shape[0]
    exists = np.ones(M ** d, bool) if active is None else np.asarray(active, bool).reshape(-1)
    codes = np.broadcast_to(np.arange(M), (T, M))
    score = S32[:, :M].astype(np.float64)
    keep = np.lexsort((codes, -score), axis=-1)[:, :k]
    codes, score = np.take_along_axis(codes, keep, 1), np.take_along_axis(score, keep, 1)
    live = np.ones(codes.shape, bool)
    for i in range(1, d):
        # a prefix of i+1 digits leads to an expert if any cell below it exists
        reach = exists.reshape(M ** (i + 1), -1).any(axis=1)
        cand = (codes[:, :, None] * M + np.arange(M)).reshape(T, -1)
        csc = (score[:, :, None] + S32[:, None, i * M:(i + 1) * M].astype(np.float64)).reshape(T, -1)
        ok = (live[:, :, None] & reach[(codes[:, :, None] * M + np.arange(M))]).reshape(T, -1)
        # usable candidates first, then score descending, then the smaller prefix
        keep = np.lexsort((cand, -np.where(ok, csc, 0.0), ~ok), axis=-1)[:, :k]
        codes, score = np.take_along_axis(cand, keep, 1), np.take_along_axis(csc, keep, 1)
        live = np.take_along_axis(ok, keep, 1)
    if not live.all() or codes.shape[1] < k:
        raise ValueError("fewer than k experts reachable by the beam")
    return codes.astype(np.int64), score


def topk_alive_bruteforce(S32, d, M, k, alive):
    """TopK among the experts that respond (the partially populated grid of App. C,
    whose Algorithm 1 only extends prefixes with active suffixes): every cell of the
    grid ranked by (alive first, total desc, flat asc) and the k first kept, so the
    k best alive experts are chosen; when fewer than k are alive, the best dead
    cells fill the remaining places (they get weight 0 in Eq. 1)."""
    g = cell_totals(S32, d, M)                       # [T, N]
    T, N = g.shape
    if k > N:
        raise ValueError("k > number of experts")
    live = np.asarray(alive, bool).reshape(-1)
    ids = np.arange(N)
    idx = np.empty((T, k), np.int64)
    gg = np.empty((T, k), np.float64)
    for t in range(T):
        order = np.lexsort((ids, -g[t], ~live))[:k]     # last key sorts first: alive, total, flat
        idx[t] = order
        gg[t] = g[t, order]
    return idx, gg


def topk_product_key(S32, d, M, k):
    """Centralised top-k search App. C refers to (product-key layers): the k best
    cells of an additive score lie in the Cartesian product of the per-dimension
    top-min(k, M) index lists, so only that product is ranked."""
    S32 = np.asarray(S32)
    T = S32.shape[0]
    L = min(k, M)
    out_idx = np.empty((T, k), np.int64)
    out_g = np.empty((T, k), np.float64)
    for t in range(T):
        lists = []
        for i in range(d):
            s = S32[t, i * M:(i + 1) * M]
            lists.append(_rank_desc(s, np.arange(M))[:L])
        cells = np.array(list(itertools.product(*lists)), np.int64)     # (L**d, d)
        tot = np.zeros(len(cells), np.float64)
        for i in range(d):
            tot = tot + S32[t, i * M + cells[:, i]].astype(np.float64)
        flat = flat_index(cells, M)
        order = _rank_desc(tot, flat)[:k]
        if len(order) < k:
            raise ValueError("k exceeds the product of the per-dimension lists")
        out_idx[t] = flat[order]
        out_g[t] = tot[order]
    return out_idx, out_g


# ------------------------------------------------------------ weights (Eq. 1)

def mixture_weights(g, idx, alive=None):
    """Eq. 1 weights exp(g_j) / sum_l exp(g_l) over the chosen experts, with
    experts that do not respond excluded and the remaining weights renormalised
    to sum to 1 (Sec. 3.1 fault tolerance; Sec. 3.2).  A token whose chosen
    experts are all dead gets all-zero weights.  Shifted by the alive maximum."""
    g = np.asarray(g, np.float64)
    if alive is None:
        live = np.ones(g.shape, bool)
    else:
        live = np.asarray(alive)[np.asarray(idx)].astype(bool)
    gm = np.where(live, g, -np.inf)
    m = gm.max(axis=1, keepdims=True)
    m = np.where(np.isfinite(m), m, 0.0)
    e = np.where(live, np.exp(g - m), 0.0)
    s = e.sum(axis=1, keepdims=True)
    return np.where(s > 0, e / np.where(s > 0, s, 1.0), 0.0)


# ------------------------------------------------------------ experts

def act(h, kind):
    """ReLU, or GELU in its erf form 0.5 h (1 + erf(h / sqrt 2)) (Sec. 4.1 cites GELU)."""
    h = np.asarray(h, np.float64)
    if kind == "relu":
        return np.maximum(h, 0.0)
    if kind == "gelu":
        return 0.5 * h * (1.0 + erf(h / SQRT2))
    raise ValueError(kind)


def act_grad(h, kind):
    """Derivative of act: ReLU' = [h > 0] (0 at h = 0); GELU' = Phi(h) + h phi(h)."""
    h = np.asarray(h, np.float64)
    if kind == "relu":
        return (h > 0).astype(np.float64)
    if kind == "gelu":
        return 0.5 * (1.0 + erf(h / SQRT2)) + h * np.exp(-0.5 * h * h) / SQRT2PI
    raise ValueError(kind)


def expert_forward(X, W1, b1, W2, b2, kind):
    """Expert f(x) = W2 act(W1 x + b1) + b2 on a batch of rows (the feed-forward
    experts of Sec. 4.1).  Returns (h, a, y)."""
    h = X @ W1.T + b1[None, :]
    a = act(h, kind)
    y = a @ W2.T + b2[None, :]
    return h, a, y


def expert_forward_stored(X, W1, b1, W2, b2, kind, store=None):
    """expert_forward as a layer with storage dtype `store` keeps it: the activation
    is computed from the exact pre-activation, then h and a are rounded, and the
    output is computed from the rounded a and rounded in turn."""
    store = store or _identity
    h = X @ W1.T + b1[None, :]
    a = store(act(h, kind))
    return store(h), a, store(a @ W2.T + b2[None, :])


def expert_backward(X, h, a, dY, W1, W2, kind, store=None):
    """Gradients of the expert block for a batch: (dX, dW1, db1, dW2, db2).
    store (optional) rounds the tensors a layer keeps in its storage dtype:
    here the pre-activation gradient dH and the input gradient dX."""
    store = store or _identity
    dA = dY @ W2
    dH = store(dA * act_grad(h, kind))
    return store(dH @ W1), dH.T @ X, dH.sum(axis=0), dY.T @ a, dY.sum(axis=0)


# ------------------------------------------------------------ dispatch (Sec. 3.3)

def round_f32(a):
    """fp32 rounding (round to nearest even) of fp64 values, returned in fp64."""
    return np.asarray(a, np.float64).astype(np.float32).astype(np.float64)


def sgd_step(param, grad, lr, store=None):
    """Gradient-descent update of an expert's parameters, as the Runtime's Backward
    applies it (Sec. 3.3): param - lr * grad, rounded once to the storage dtype by
    `store` (round_bf16, round_f32, or None for exact)."""
    store = store or _identity
    return store(np.asarray(param, np.float64) - lr * np.asarray(grad, np.float64))


def dispatch(idx, alive, N):
    """Group the alive (token, slot) pairs by expert, the way the Runtime collects
    the requests for each of its experts into one batch (Sec. 3.3).  Within an
    expert, rows follow token order.  Returns counts [N], offsets [N+1],
    row_token [rows], pos [T,k] (row of each pair, -1 if its expert is dead)."""
    idx = np.asarray(idx, np.int64)
    T, k = idx.shape
    live = np.ones(N, bool) if alive is None else np.asarray(alive).astype(bool)
    pair_e = idx.reshape(-1)
    pair_ok = live[pair_e]
    pairs = np.nonzero(pair_ok)[0]                     # pair ids, ascending
    order = pairs[np.argsort(pair_e[pairs], kind="stable")]
    counts = np.bincount(pair_e[pairs], minlength=N).astype(np.int64)
    offsets = np.concatenate([[0], np.cumsum(counts)]).astype(np.int64)
    row_token = (order // k).astype(np.int64)
    pos = np.full(T * k, -1, np.int64)
    pos[order] = np.arange(len(order))
    return counts, offsets, row_token, pos.reshape(T, k)


# ------------------------------------------------------------ the layer

def chosen_totals(S, idx, d, M):
    """g(x, f) = sum_i g_i(x)[u_i] (Sec. 3.2) of the chosen experts, from the exact
    fp64 scores S (the weights of Eq. 1 use these, not the fp32 decision copy)."""
    u = uid_of(idx, d, M)
    T = S.shape[0]
    g = np.zeros(idx.shape, np.float64)
    for i in range(d):
        g = g + S[np.arange(T)[:, None], i * M + u[:, :, i]]
    return g


def routing(x, Wg, bg, alive, d, M, k, alive_topk=False):
    """Gate, TopK and Eq. 1 weights for a batch of tokens.  TopK compares the fp32
    decision scores; the weights use the exact totals of the chosen experts.
    alive_topk: TopK among the alive experts (topk_alive_bruteforce)."""
    S = gate_scores(x, Wg, bg)
    S32 = decision_scores(S)
    if alive_topk:
        idx, g32 = topk_alive_bruteforce(S32, d, M, k, np.ones(M ** d) if alive is None else alive)
    else:
        idx, g32 = topk_bruteforce(S32, d, M, k)
    g = chosen_totals(S, idx, d, M)
    w = mixture_weights(g, idx, alive)
    return dict(S=S, S32=S32, idx=idx, g32=g32, g=g, w=w)


def _expert_getter(experts):
    if callable(experts):
        return experts
    W1, b1, W2, b2 = experts
    return lambda e: (W1[e], b1[e], W2[e], b2[e])


def layer_forward(x, Wg, bg, experts, alive, d, M, k, kind, only_experts=None, store=None, alive_topk=False,
                  expert="ffn"):
    """DMoE(x) of Eq. 1: sum over the alive chosen experts of f(x) times its
    renormalised weight.  experts is (W1, b1, W2, b2) stacked over experts or a
    callable e -> (W1_e, b1_e, W2_e, b2_e), all fp64.  only_experts restricts the
    expert evaluation to a subset (rows of other experts stay NaN, and so does y
    for tokens that use them).  Returns a dict with the routing, the dispatch,
    the per-row h, a, y_perm (expert-grouped order) and the layer output y.
    store (optional) rounds the tensors a bf16 layer keeps in bf16 (h, a and the
    expert outputs); all arithmetic stays exact.
    expert="ffblock": the experts are the LayerNorm feed-forward blocks of Sec. 4.1
    (oracle.ffblock); experts(e) then returns a dict of that expert's parameters and
    the per-row tensors are h1, a1, mean1, rstd1, h2, a2, mean2, rstd2 instead of h, a."""
    store = store or _identity
    x = np.asarray(x, np.float64)
    T, D = x.shape
    N = M ** d
    r = routing(x, Wg, bg, alive, d, M, k, alive_topk)
    counts, offsets, row_token, pos = dispatch(r["idx"], alive, N)
    get = _expert_getter(experts) if expert == "ffn" else None
    rows = int(offsets[-1])
    h = a = None
    y_perm = np.full((rows, D), np.nan)
    hs, as_ = {}, {}
    todo = np.nonzero(counts)[0] if only_experts is None else \
        [e for e in only_experts if counts[e] > 0]
    if expert == "ffblock":
        from .ffblock import ffblock_forward_stored
        per_row = {}
        for e in todo:
            lo, hi = offsets[e], offsets[e + 1]
            fw = ffblock_forward_stored(x[row_token[lo:hi]], experts(e), kind, store)
            y_perm[lo:hi] = fw.pop("y")
            for name, v in fw.items():
                if name not in per_row:
                    per_row[name] = np.full((rows,) + v.shape[1:], np.nan)
                per_row[name][lo:hi] = v
        todo = []
    elif expert != "ffn":
        raise ValueError(expert)
    else:
        per_row = {}
    for e in todo:
        lo, hi = offsets[e], offsets[e + 1]
        W1, b1, W2, b2 = get(e)
        he, ae, ye = expert_forward_stored(x[row_token[lo:hi]], W1, b1, W2, b2, kind, store)
        hs[e], as_[e] = he, ae
        y_perm[lo:hi] = ye
    if hs:
        H = next(iter(hs.values())).shape[1]
        h = np.full((rows, H), np.nan)
        a = np.full((rows, H), np.nan)
        for e in hs:
            h[offsets[e]:offsets[e + 1]] = hs[e]
            a[offsets[e]:offsets[e + 1]] = as_[e]
    y = np.zeros((T, D))
    for j in range(k):
        p = pos[:, j]
        ok = p >= 0
        y[ok] += r["w"][ok, j][:, None] * y_perm[p[ok]]
    return dict(r, counts=counts, offsets=offsets, row_token=row_token, pos=pos,
                h=h, a=a, y_perm=y_perm, y=y, **per_row)


def gate_backward(w, dw, idx, alive, x, Wg, d, M):
    """Backward of the Eq. 1 weights and the gate.  TopK is piecewise constant, so
    the gradient reaches the gate only through the softmax over the chosen alive
    experts: dg_j = w_j (dw_j - sum_l w_l dw_l).  Each chosen expert passes dg_j to
    the score of its index in every grid dimension; the gate layers then give
    dx = ds Wg, dWg = ds^T x, dbg = sum_t ds.  Returns (dg, ds, dx_gate, dWg, dbg)."""
    w = np.asarray(w, np.float64)
    dw = np.asarray(dw, np.float64)
    T, k = w.shape
    live = np.ones(w.shape, bool) if alive is None else \
        np.asarray(alive)[np.asarray(idx)].astype(bool)
    dg = np.where(live, w * (dw - (w * dw).sum(axis=1, keepdims=True)), 0.0)
    u = uid_of(idx, d, M)                              # [T, k, d]
    ds = np.zeros((T, d * M))
    for j in range(k):
        for i in range(d):
            np.add.at(ds, (np.arange(T), i * M + u[:, j, i]), dg[:, j])
    x = np.asarray(x, np.float64)
    return dg, ds, ds @ np.asarray(Wg, np.float64), ds.T @ x, ds.sum(axis=0)


def layer_backward(fwd, dy, x, Wg, experts, alive, d, M, k, kind, only_experts=None, store=None,
                   expert="ffn"):
    """Gradients of <DMoE(x), dy> with respect to x, the gate and the experts.

    dw_tj = <dy_t, f_j(x_t)> for alive chosen experts; the expert f_j receives
    w_tj dy_t as its output gradient; dx gathers every expert's input gradient
    plus the gate's.  Expert gradients are returned only for experts that got
    rows (an expert with no rows has zero gradient).  store (optional) rounds the
    tensors a bf16 layer keeps in bf16 (output gradients per row, dH, dX per row).
    expert="ffblock": the LayerNorm blocks of Sec. 4.1; expert_grads[e] is then a dict
    keyed by the parameter names, and the row gradients dh2, dh1 are returned too."""
    store = store or _identity
    x = np.asarray(x, np.float64)
    dy = np.asarray(dy, np.float64)
    T, D = x.shape
    w, pos, idx = fwd["w"], fwd["pos"], fwd["idx"]
    offsets, row_token, counts = fwd["offsets"], fwd["row_token"], fwd["counts"]
    y_perm = fwd["y_perm"]
    dw = np.zeros((T, k))
    dy_perm = np.zeros_like(y_perm)
    for j in range(k):
        p = pos[:, j]
        ok = p >= 0
        dw[ok, j] = np.einsum("td,td->t", dy[ok], y_perm[p[ok]])
        dy_perm[p[ok]] = store(w[ok, j][:, None] * dy[ok])
    dg, ds, dx_gate, dWg, dbg = gate_backward(w, dw, idx, alive, x, Wg, d, M)
    dx_perm = np.full((y_perm.shape[0], D), np.nan)
    grads = {}
    todo = np.nonzero(counts)[0] if only_experts is None else \
        [e for e in only_experts if counts[e] > 0]
    extra = {}
    if expert == "ffblock":
        from .ffblock import ffblock_backward
        names = ("h1", "a1", "h2", "a2")
        for e in todo:
            lo, hi = offsets[e], offsets[e + 1]
            fw = {n: fwd[n][lo:hi] for n in names}
            bw = ffblock_backward(x[row_token[lo:hi]], fw, dy_perm[lo:hi], experts(e), kind, store)
            dx_perm[lo:hi] = bw["dX"]
            for n in ("dh2", "dh1"):
                if n not in extra:
                    extra[n] = np.full((y_perm.shape[0],) + bw[n].shape[1:], np.nan)
                extra[n][lo:hi] = bw[n]
            grads[e] = bw["grads"]
        todo = []
    elif expert != "ffn":
        raise ValueError(expert)
    get = _expert_getter(experts) if expert == "ffn" else None
    for e in todo:
        lo, hi = offsets[e], offsets[e + 1]
        W1, b1, W2, b2 = get(e)
        dX, dW1, db1, dW2, db2 = expert_backward(
            x[row_token[lo:hi]], fwd["h"][lo:hi], fwd["a"][lo:hi], dy_perm[lo:hi], W1, W2, kind,
            store)
        dx_perm[lo:hi] = dX
        grads[e] = (dW1, db1, dW2, db2)
    dx = dx_gate.copy()
    for j in range(k):
        p = pos[:, j]
        ok = p >= 0
        dx[ok] += dx_perm[p[ok]]
    return dict(dw=dw, dg=dg, ds=ds, dy_perm=dy_perm, dx_perm=dx_perm, dx=dx,
                dWg=dWg, dbg=dbg, expert_grads=grads, **extra)
