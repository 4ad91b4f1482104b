"""Pins of the oracle's gate and TopK (CPU only).

Each check comes from outside the oracle's own code: hand-worked fixtures,
a library stable sort, three different search algorithms that must agree, and
invariants of the definition (scale invariance, constructed ties, the
product-key property).
"""
import itertools
import math

import numpy as np
import pytest
import torch

import oracle as O
from conftest import read_golden


def _f32(a):
    return np.asarray(a, dtype=np.float32)


# ------------------------------------------------------------------ golden cases

def test_golden_grid3x3():
    rows = read_golden("topk_grid3x3.txt")
    d = int(dict(rows)["d"][0])
    M = int(dict(rows)["M"][0])
    S32 = _f32([[float(v) for v in dict(rows)["scores"]]])
    cases, cur = [], None
    for key, vals in rows:
        if key == "k":
            cur = {"k": int(vals[0])}
            cases.append(cur)
        elif key in ("idx", "g") and cur is not None:
            cur[key] = [float(v) for v in vals]
    assert len(cases) == 3
    for c in cases:
        for fn in (O.topk_bruteforce, O.topk_beam, O.topk_product_key):
            idx, g = fn(S32, d, M, c["k"])
            assert idx[0].tolist() == [int(v) for v in c["idx"]], fn.__name__
            assert g[0].tolist() == c["g"], fn.__name__


def test_golden_appC_six_experts():
    kv = dict(read_golden("beam_appC_six_experts.txt"))
    d, M, k = int(kv["d"][0]), int(kv["M"][0]), int(kv["k"][0])
    S32 = _f32([[float(v) for v in kv["scores"]]])
    table = {}
    for item in kv["active"]:
        p, suf = item.split(":")
        table[(int(p),)] = [int(s) for s in suf.split(",")]
    active = np.zeros(M ** d, bool)
    for (p,), sufs in table.items():
        active[[p * M + s for s in sufs]] = True
    idx, g = O.topk_beam(S32, d, M, k, active=active)
    assert idx[0].tolist() == [int(v) for v in kv["beam_idx"]]
    assert g[0].tolist() == [float(v) for v in kv["beam_g"]]
    # exact best among the six active experts, by brute force over the table
    tot = O.cell_totals(S32, d, M)[0]
    live = [p[0] * M + s for p, sufs in table.items() for s in sufs]
    best = sorted(live, key=lambda f: (-tot[f], f))[:k]
    assert best == [int(v) for v in kv["exact_active_idx"]]
    assert [tot[f] for f in best] == [float(v) for v in kv["exact_active_g"]]
    # fully populated grid: Algorithm 1 equals brute force equals the fixture
    for fn in (O.topk_bruteforce, O.topk_beam, O.topk_product_key):
        idx, g = fn(S32, d, M, k)
        assert idx[0].tolist() == [int(v) for v in kv["full_idx"]]
        assert g[0].tolist() == [float(v) for v in kv["full_g"]]


# ------------------------------------------------------------------ agreement of three searches

GRIDS = [(1, 1), (1, 5), (1, 8), (2, 1), (2, 3), (2, 4), (2, 6), (3, 2), (3, 3), (3, 4), (4, 2), (4, 3)]


@pytest.mark.parametrize("d,M", GRIDS)
@pytest.mark.parametrize("kind", ["normal", "ties"])
def test_three_searches_agree(d, M, kind):
    rng = np.random.default_rng(1000 * d + M + (7 if kind == "ties" else 0))
    N = M ** d
    T = 40
    if kind == "normal":
        S32 = _f32(rng.standard_normal((T, d * M)))
    else:  # small integer scores: many exact ties in the totals
        S32 = _f32(rng.integers(-2, 3, size=(T, d * M)))
    for k in sorted({min(1, N), min(2, N), min(3, N), min(4, N), min(8, N), N}):
        bi, bg = O.topk_bruteforce(S32, d, M, k)
        ai, ag = O.topk_beam(S32, d, M, k)
        pi, pg = O.topk_product_key(S32, d, M, k)
        np.testing.assert_array_equal(bi, ai)
        np.testing.assert_array_equal(bi, pi)
        np.testing.assert_array_equal(bg, ag)
        np.testing.assert_array_equal(bg, pg)


def test_python_sorted_definition_tiny():
    """Brute force with Python's own sort and itertools on tiny grids."""
    rng = np.random.default_rng(5)
    for d, M, k in [(2, 3, 4), (3, 2, 5), (2, 4, 16), (1, 6, 3)]:
        S32 = _f32(rng.integers(-3, 4, size=(12, d * M)) * 0.5)
        idx, g = O.topk_bruteforce(S32, d, M, k)
        for t in range(S32.shape[0]):
            cells = []
            for u in itertools.product(range(M), repeat=d):
                tot = 0.0
                for i in range(d):
                    tot = tot + float(S32[t, i * M + u[i]])
                flat = 0
                for i in range(d):
                    flat = flat * M + u[i]
                cells.append((-tot, flat, tot))
            cells.sort()
            assert idx[t].tolist() == [c[1] for c in cells[:k]]
            assert g[t].tolist() == [c[2] for c in cells[:k]]


def test_d1_is_stable_argsort():
    rng = np.random.default_rng(2)
    S32 = _f32(rng.integers(-4, 5, size=(50, 9)))
    for k in (1, 3, 9):
        idx, g = O.topk_bruteforce(S32, 1, 9, k)
        ref = np.argsort(-S32.astype(np.float64), axis=1, kind="stable")[:, :k]
        np.testing.assert_array_equal(idx, ref)


def test_d1_matches_torch_topk_without_ties():
    rng = np.random.default_rng(3)
    S32 = _f32(rng.standard_normal((64, 32)))
    idx, g = O.topk_bruteforce(S32, 1, 32, 5)
    v, i = torch.topk(torch.from_numpy(S32.astype(np.float64)), 5, dim=1)
    np.testing.assert_array_equal(idx, i.numpy())
    np.testing.assert_array_equal(g, v.numpy())


def test_scale_invariance():
    rng = np.random.default_rng(4)
    S32 = _f32(rng.standard_normal((30, 3 * 5)))
    for c in (0.25, 4.0, 1024.0):      # powers of two: scaling is exact
        a, _ = O.topk_bruteforce(S32, 3, 5, 6)
        b, _ = O.topk_bruteforce(_f32(S32 * c), 3, 5, 6)
        np.testing.assert_array_equal(a, b)


def test_constructed_ties_pick_lowest_flat():
    S32 = np.zeros((3, 2 * 4), np.float32)
    for fn in (O.topk_bruteforce, O.topk_beam, O.topk_product_key):
        idx, g = fn(S32, 2, 4, 5)
        assert (idx == np.arange(5)).all()
        assert (g == 0).all()


def test_product_key_property():
    """The exact top-k cells lie inside the product of per-dimension top-k lists."""
    rng = np.random.default_rng(6)
    for d, M, k in [(2, 8, 4), (3, 5, 4), (2, 16, 7), (4, 3, 6)]:
        S32 = _f32(rng.standard_normal((60, d * M)))
        idx, _ = O.topk_bruteforce(S32, d, M, k)
        u = O.uid_of(idx, d, M)
        L = min(k, M)
        for i in range(d):
            s = S32[:, i * M:(i + 1) * M].astype(np.float64)
            rank = np.argsort(np.argsort(-s, axis=1, kind="stable"), axis=1)   # 0-based rank
            r = np.take_along_axis(rank, u[:, :, i], axis=1)
            assert (r < L).all()


def test_product_rank_bound():
    """Tighter: a chosen cell has prod_i (rank_i + 1) <= k (it is dominated by
    prod_i (rank_i + 1) - 1 cells)."""
    rng = np.random.default_rng(7)
    for d, M, k in [(2, 32, 4), (3, 16, 4), (2, 16, 4), (2, 4, 2)]:
        S32 = _f32(rng.standard_normal((200, d * M)))
        idx, _ = O.topk_bruteforce(S32, d, M, k)
        u = O.uid_of(idx, d, M)
        prod = np.ones(idx.shape, np.int64)
        for i in range(d):
            s = S32[:, i * M:(i + 1) * M].astype(np.float64)
            rank = np.argsort(np.argsort(-s, axis=1, kind="stable"), axis=1)
            prod *= np.take_along_axis(rank, u[:, :, i], axis=1) + 1
        assert (prod <= k).all()


def test_flat_index_roundtrip_and_prefix_order():
    d, M = 3, 5
    f = np.arange(M ** d)
    u = O.uid_of(f, d, M)
    np.testing.assert_array_equal(O.flat_index(u, M), f)
    # flat order is lexicographic uid order (prefix keys of App. C)
    tuples = [tuple(r) for r in u.tolist()]
    assert tuples == sorted(tuples)


def test_gate_scores_match_torch_linear():
    rng = np.random.default_rng(8)
    x = rng.standard_normal((17, 24))
    W = rng.standard_normal((10, 24))
    b = rng.standard_normal(10)
    ref = torch.nn.functional.linear(torch.from_numpy(x), torch.from_numpy(W), torch.from_numpy(b))
    np.testing.assert_allclose(O.gate_scores(x, W, b), ref.numpy(), rtol=1e-13, atol=1e-13)


def test_bf16_products_exact_in_fp64():
    """bf16 inputs make every product exact in fp64: the gate scores of short rows
    equal the exact rational sum (fractions)."""
    from fractions import Fraction
    g = torch.Generator().manual_seed(0)
    x = torch.randn(4, 16, generator=g).to(torch.bfloat16).double().numpy()
    W = torch.randn(6, 16, generator=g).to(torch.bfloat16).double().numpy()
    S = O.gate_scores(x, W, None)
    for t in range(4):
        for c in range(6):
            exact = sum(Fraction(float(x[t, j])) * Fraction(float(W[c, j])) for j in range(16))
            assert abs(Fraction(float(S[t, c])) - exact) <= abs(exact) * Fraction(1, 2 ** 50)


# ------------------------------------------------------------------ TopK among alive experts

def test_alive_topk_golden_six_experts():
    """The App. C example: six active experts; the exact best among them is the
    fixture's exact_active (which Algorithm 1's beam need not find)."""
    kv = dict(read_golden("beam_appC_six_experts.txt"))
    d, M, k = int(kv["d"][0]), int(kv["M"][0]), int(kv["k"][0])
    S32 = _f32([[float(v) for v in kv["scores"]]])
    alive = np.zeros(M ** d)
    for item in kv["active"]:
        p, suf = item.split(":")
        for s_ in suf.split(","):
            alive[int(p) * M + int(s_)] = 1
    idx, g = O.topk_alive_bruteforce(S32, d, M, k, alive)
    assert idx[0].tolist() == [int(v) for v in kv["exact_active_idx"]]
    assert g[0].tolist() == [float(v) for v in kv["exact_active_g"]]


@pytest.mark.parametrize("d,M", [(1, 6), (2, 4), (3, 3)])
def test_alive_topk_reductions(d, M):
    """All alive (or all dead): the plain TopK.  Alive experts always come first, in
    the plain order; with fewer than k alive, the best dead ones follow, in order."""
    rng = np.random.default_rng(7 * d + M)
    N, T = M ** d, 30
    S32 = _f32(rng.standard_normal((T, d * M)))
    for k in sorted({1, 2, min(4, N), N}):
        ref, rg = O.topk_bruteforce(S32, d, M, k)
        for alive in (np.ones(N), np.zeros(N)):
            idx, g = O.topk_alive_bruteforce(S32, d, M, k, alive)
            np.testing.assert_array_equal(idx, ref)
            np.testing.assert_array_equal(g, rg)
        alive = (rng.random(N) < 0.5).astype(float)
        alive[0] = 1.0
        idx, _ = O.topk_alive_bruteforce(S32, d, M, k, alive)
        full, _ = O.topk_bruteforce(S32, d, M, N)
        for t in range(T):
            order_live = [f for f in full[t] if alive[f]]
            order_dead = [f for f in full[t] if not alive[f]]
            assert idx[t].tolist() == (order_live + order_dead)[:k]
