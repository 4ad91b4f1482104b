"""GPU parity: the HIP path (through the C ABI) against the oracle, element by
element, on seeded inputs small enough for the oracle to finish in seconds while
still spanning several GEMM tiles and ragged tails."""
import numpy as np
import pytest
import torch

from parity_util import RTOL, assert_close, compare, gpu_run, oracle_run, say
from workloads import Workload, make_inputs, small_workload

pytestmark = pytest.mark.gpu

CASES = {
    # the tiny fp32 workload exactly as named (64 tokens, 4x4 grid, top-2, ReLU)
    "tiny_f32": small_workload("tiny_f32"),
    # bf16, skinny experts (few rows each): 32-row GEMM tiles, ragged rows, dead experts
    "bf16_skinny": Workload("bf16_skinny", 10, T=512, D=256, H=512, d=2, M=8, k=4, dtype="bf16",
                            act="gelu", p_alive=0.8),
    # bf16, fat experts (hundreds of rows each): the 256x256-tile GEMM configuration
    "bf16_fat": Workload("bf16_fat", 11, T=2048, D=128, H=256, d=2, M=4, k=2, dtype="bf16",
                         act="gelu", p_alive=0.9),
    # fat experts of ~540 rows (one grid dimension, top-1): m-tiles of up to 288 rows
    # split each expert evenly (the ninth, shared 32-row block live), expert hidden size
    # off the 256-column tile grid
    "bf16_fat_xb": Workload("bf16_fat_xb", 31, T=4300, D=128, H=192, d=1, M=8, k=1, dtype="bf16",
                            act="gelu"),
    # 3-D grid, token count off the tile grid, ReLU
    "bf16_grid3d": Workload("bf16_grid3d", 12, T=333, D=128, H=192, d=3, M=3, k=4, dtype="bf16",
                            act="relu", p_alive=0.85),
    # d = 1 with k = N: a dense softmax mixture
    "f32_dense": Workload("f32_dense", 13, T=100, D=64, H=128, d=1, M=8, k=8, dtype="f32",
                          act="gelu"),
    # skewed gate as in the failure+skew workload, at a small size
    "bf16_skew": Workload("bf16_skew", 14, T=1024, D=256, H=256, d=2, M=16, k=4, dtype="bf16",
                          act="gelu", p_alive=0.9, gate_scale=4.0, skew_rows=4),
    # the same skew at twice the tokens: 11 experts hold more than 128 rows (up to 301),
    # so the few-rows weight-gradient GEMM (32-deep k-steps, 4 stages) wraps its ring
    "bf16_skew_deep": Workload("bf16_skew_deep", 30, T=2048, D=128, H=256, d=2, M=16, k=4, dtype="bf16",
                               act="gelu", p_alive=0.9, gate_scale=4.0, skew_rows=4),
    # 4-D grid, fp32
    "f32_grid4d": Workload("f32_grid4d", 15, T=200, D=64, H=64, d=4, M=3, k=5, dtype="f32",
                           act="gelu", p_alive=0.7),
    # bf16 gate with 96 columns: three 32-column MFMA blocks per token group
    "bf16_gate96": Workload("bf16_gate96", 16, T=300, D=192, H=128, d=2, M=48, k=3, dtype="bf16",
                            act="gelu", p_alive=0.9),
    # bf16 gate with 128 columns: the exact fp64 gate path
    "bf16_gate128": Workload("bf16_gate128", 17, T=200, D=128, H=128, d=2, M=64, k=8, dtype="bf16",
                             act="relu", p_alive=0.95),
    # near the largest grid: 25x25x25 = 15625 experts (most without rows), k = 8 (the
    # largest), 75 gate columns (three MFMA column blocks), 10% dead
    "bf16_maxgrid": Workload("bf16_maxgrid", 18, T=700, D=64, H=64, d=3, M=25, k=8, dtype="bf16",
                             act="gelu", p_alive=0.9),
    # d_model >= 2048: the MFMA gate's two-wave blocks; 33 groups of 64 (one wave takes
    # one group more), token count off the 32-token blocks
    "bf16_wide_gate": Workload("bf16_wide_gate", 19, T=150, D=2112, H=64, d=2, M=16, k=4, dtype="bf16",
                               act="gelu", p_alive=0.9),
    # degenerate grids of one expert (M = 1): every token's TopK is that expert with
    # weight 1; one gate column (bf16, MFMA gate, 700 rows on the fat tiles) or two
    # (fp32, d = 2)
    "bf16_one_expert": Workload("bf16_one_expert", 32, T=700, D=128, H=128, d=1, M=1, k=1, dtype="bf16",
                                act="gelu"),
    "f32_one_expert_2d": Workload("f32_one_expert_2d", 33, T=50, D=64, H=64, d=2, M=1, k=1, dtype="f32",
                                  act="relu"),
}


@pytest.mark.parametrize("name", list(CASES))
def test_layer_parity(name):
    wl = CASES[name]
    say(f"[parity] {name}: T={wl.T} D={wl.D} H={wl.H} d={wl.d} M={wl.M} k={wl.k} {wl.dtype}")
    inp = make_inputs(wl, "cpu")
    gpu = gpu_run(wl, inp, backward=wl.backward)
    fwd, bwd = oracle_run(wl, inp, backward=wl.backward)
    compare(wl, inp, gpu, fwd, bwd)


def test_dh_may_alias_h():
    wl = CASES["bf16_skinny"]
    say("[parity] dh aliasing h")
    inp = make_inputs(wl, "cpu")
    a = gpu_run(wl, inp, dh_aliases_h=False)
    b = gpu_run(wl, inp, dh_aliases_h=True)
    for n in ("dx", "dW1", "dW2", "db1", "db2", "dWg"):
        assert torch.equal(a[n], b[n]), n


def test_all_experts_dead():
    wl = Workload("dead", 20, T=96, D=64, H=128, d=2, M=4, k=3, dtype="bf16", act="gelu", p_alive=0.0)
    say("[parity] all experts dead")
    inp = make_inputs(wl, "cpu")
    gpu = gpu_run(wl, inp)
    fwd, bwd = oracle_run(wl, inp)
    compare(wl, inp, gpu, fwd, bwd)
    assert int(gpu["offsets"][-1]) == 0
    assert (gpu["y"].float() == 0).all() and (gpu["w"] == 0).all()
    assert (gpu["dx"].float() == 0).all() and (gpu["dWg"].float() == 0).all()


def test_single_alive_expert():
    wl = Workload("one_alive", 21, T=128, D=64, H=64, d=2, M=4, k=4, dtype="f32", act="relu")
    say("[parity] single alive expert")
    inp = make_inputs(wl, "cpu")
    alive = torch.zeros(wl.N, dtype=torch.uint8)
    alive[5] = 1
    inp["alive"] = alive
    gpu = gpu_run(wl, inp)
    fwd, bwd = oracle_run(wl, inp)
    compare(wl, inp, gpu, fwd, bwd)
    w = gpu["w"].numpy()
    chosen = gpu["idx"].numpy() == 5
    np.testing.assert_array_equal(w[chosen], 1.0)
    assert (w[~chosen] == 0).all()


def test_empty_batch():
    from paper_2002_04013_amd import DMoELayer
    say("[parity] T = 0")
    wl = Workload("empty", 22, T=0, D=64, H=64, d=2, M=4, k=2, dtype="bf16", act="gelu")
    inp = make_inputs(wl, "cpu")
    t = {n: v.cuda() for n, v in inp.items()}
    L = DMoELayer(0, 64, 64, 2, 4, 2, "bf16", "gelu")
    L.forward(t["x"], t["Wg"], t["bg"], t["alive"], t["W1"], t["b1"], t["W2"], t["b2"])
    dWg = torch.full_like(t["Wg"], 3.0)
    dbg = torch.full_like(t["bg"], 3.0)
    dW1 = torch.full_like(t["W1"], 7.0)
    L.backward(t["dy"], t["x"], t["Wg"], t["alive"], t["W1"], t["W2"], dW1, t["b1"].clone(),
               t["W2"].clone(), t["b2"].clone(), dWg, dbg)
    torch.cuda.synchronize()
    assert (L.counts.cpu() == 0).all() and (L.offsets.cpu() == 0).all()
    assert (dWg.float().cpu() == 0).all() and (dbg.float().cpu() == 0).all()
    assert (dW1.float().cpu() == 7.0).all()


def test_identical_experts_invariant():
    """Every expert equal: y = f(x) for tokens with an alive expert; gate grads 0."""
    wl = Workload("same", 23, T=256, D=128, H=128, d=2, M=4, k=3, dtype="f32", act="gelu", p_alive=0.75)
    say("[parity] identical experts")
    inp = make_inputs(wl, "cpu", identical_experts=True)
    gpu = gpu_run(wl, inp)
    import oracle as O
    f = {n: O.to64(v) for n, v in inp.items()}
    _, _, y1 = O.expert_forward(f["x"], f["W1"][0], f["b1"][0], f["W2"][0], f["b2"][0], "gelu")
    live = inp["alive"].numpy()[gpu["idx"].numpy()].astype(bool).any(axis=1)
    assert_close(gpu["y"].numpy()[live], y1[live], 1e-5, "y vs single expert")
    assert (gpu["y"].numpy()[~live] == 0).all()
    np.testing.assert_allclose(gpu["dg"].numpy(), 0, atol=1e-5)


def test_deterministic():
    wl = CASES["bf16_skew"]
    say("[parity] determinism")
    inp = make_inputs(wl, "cpu")
    a = gpu_run(wl, inp)
    b = gpu_run(wl, inp)
    for n in a:
        assert torch.equal(a[n], b[n]) or n in ("row_token", "x_perm", "h", "a", "y_perm", "dy_perm",
                                                 "dx_perm", "dh"), n
    rows = int(a["offsets"][-1])
    for n in ("row_token", "x_perm", "h", "a", "y_perm", "dy_perm", "dx_perm", "dh"):
        assert torch.equal(a[n][:rows], b[n][:rows]), n


def test_token_permutation_equivariance():
    wl = CASES["bf16_skinny"]
    say("[parity] token permutation")
    inp = make_inputs(wl, "cpu")
    perm = torch.randperm(wl.T, generator=torch.Generator().manual_seed(3))
    inp2 = dict(inp, x=inp["x"][perm], dy=inp["dy"][perm])
    a = gpu_run(wl, inp)
    b = gpu_run(wl, inp2)
    assert torch.equal(b["idx"], a["idx"][perm])
    assert torch.equal(b["y"], a["y"][perm])
    assert torch.equal(b["dx"], a["dx"][perm])


def test_gate_exact_flag_same_routing():
    """DMOE_FLAG_GATE_EXACT computes every token's scores with exact fp64 accumulation
    (the fallback path of the certified MFMA gate): same TopK, bit for bit."""
    from paper_2002_04013_amd.abi import DMOE_FLAG_GATE_EXACT
    wl = CASES["bf16_skew"]
    say("[parity] exact-gate flag")
    inp = make_inputs(wl, "cpu")
    a = gpu_run(wl, inp, backward=False)
    b = gpu_run(wl, inp, backward=False, flags=DMOE_FLAG_GATE_EXACT)
    assert torch.equal(a["idx"], b["idx"])
    fwd, _ = oracle_run(wl, inp, backward=False)
    np.testing.assert_array_equal(b["idx"].numpy(), fwd["idx"])
    S = fwd["S"]   # exact path: one fp32 rounding of the fp64-accumulated score
    assert np.all(np.abs(b["scores"].double().numpy() - S) <= np.abs(S) * 2.0 ** -23 + 1e-30)


def test_gate_exact_ties_fall_back():
    """Duplicated gate rows make exactly tied scores and totals: no certificate is
    possible, every affected token takes the exact path and ties go to the lower
    flat index, as in the oracle."""
    wl = Workload("ties", 24, T=512, D=128, H=128, d=2, M=8, k=4, dtype="bf16", act="gelu", p_alive=0.9)
    say("[parity] exact ties in the gate")
    inp = make_inputs(wl, "cpu")
    Wg, bg = inp["Wg"].clone(), inp["bg"].clone()
    for i in range(wl.d):          # rows u and u+1 equal in every dimension, for even u
        for u in range(0, wl.M, 2):
            Wg[i * wl.M + u + 1] = Wg[i * wl.M + u]
            bg[i * wl.M + u + 1] = bg[i * wl.M + u]
    inp["Wg"], inp["bg"] = Wg, bg
    gpu = gpu_run(wl, inp)
    fwd, bwd = oracle_run(wl, inp)
    compare(wl, inp, gpu, fwd, bwd)


@pytest.mark.parametrize("name", ["bf16_skinny", "bf16_fat", "f32_grid4d"])
def test_recompute_backward(name):
    """dmoe_expert_ffn_bwd_recompute: h and a regenerated from x_perm, W1, b1 (the
    forward's copies are overwritten before the backward): gradients bit-identical to
    the backward given the stored activations, and equal to the oracle's."""
    wl = CASES[name]
    say(f"[parity] recompute backward {name}")
    inp = make_inputs(wl, "cpu")
    a = gpu_run(wl, inp)
    b = gpu_run(wl, inp, recompute=True, clobber_h=True)
    rows = int(a["offsets"][-1])
    for n in ("dW1", "db1", "dW2", "db2", "dWg", "dbg", "dx", "dw", "dg"):
        assert torch.equal(a[n], b[n]), n
    for n in ("dx_perm", "dy_perm", "dh"):
        assert torch.equal(a[n][:rows], b[n][:rows]), n
    fwd, bwd = oracle_run(wl, inp)
    compare(wl, inp, b, fwd, bwd)


def _ulp(ref, dtype):
    """One unit in the last place of |ref| in the storage dtype (bf16: 8 significant
    bits, fp32: 24), for ref != 0; the smallest normal's for ref == 0."""
    bits = 8 if dtype == "bf16" else 24
    e = np.floor(np.log2(np.maximum(np.abs(ref), 2.0 ** -126)))
    return 2.0 ** (e - bits + 1)


@pytest.mark.parametrize("name", ["bf16_skinny", "bf16_skew_deep", "bf16_fat", "f32_grid4d"])
def test_sgd_backward(name):
    """dmoe_expert_ffn_bwd_sgd: dh and dx_perm bit-identical to the plain backward
    (computed from the parameters on entry); each parameter becomes
    store(W - lr dW) of the oracle's dW within one unit of the storage dtype's last
    place plus the dW tolerance; experts without rows keep their parameters bit for
    bit.  lr is scaled so the update is about a quarter of the weights' magnitude."""
    import oracle as O
    from paper_2002_04013_amd import DMoELayer, abi
    wl = CASES[name]
    say(f"[parity] sgd backward {name}")
    inp = make_inputs(wl, "cpu")
    ref = gpu_run(wl, inp)
    fwd, bwd = oracle_run(wl, inp)
    rms = lambda v: float(np.sqrt(np.mean(np.square(v)))) if v.size else 1.0
    # dense oracle gradients (zero for experts without rows)
    grads = {}
    for q, n in enumerate(("dW1", "db1", "dW2", "db2")):
        g = np.zeros(inp[n[1:]].shape)
        for e, gr in bwd["expert_grads"].items():
            g[e] = gr[q]
        grads[n] = g
    lr = 0.25 * rms(O.to64(inp["W1"])) / max(rms(grads["dW1"][ref["counts"].numpy() > 0]), 1e-30)
    dev = torch.device("cuda")
    t = {n: v.to(dev) for n, v in inp.items()}
    L = DMoELayer(wl.T, wl.D, wl.H, wl.d, wl.M, wl.k, wl.dtype, wl.act)
    L.forward(t["x"], t["Wg"], t["bg"], t["alive"], t["W1"], t["b1"], t["W2"], t["b2"])
    abi.dmoe_combine_bwd(L.dims, t["dy"], L.y_perm, L.pos, L.w, L.dy_perm, L.dw)
    P = {n: t[n].clone() for n in ("W1", "b1", "W2", "b2")}
    abi.dmoe_expert_ffn_bwd_sgd(L.dims, L.offsets, L.counts, L.x_perm, L.h, L.a, L.dy_perm, P["W1"], P["b1"],
                                P["W2"], P["b2"], lr, L.dh, L.dx_perm, L.ws)
    torch.cuda.synchronize()
    rows = int(ref["offsets"][-1])
    assert torch.equal(L.dh[:rows].cpu(), ref["dh"][:rows]), "dh"
    assert torch.equal(L.dx_perm[:rows].cpu(), ref["dx_perm"][:rows]), "dx_perm"
    store = O.round_bf16 if wl.dtype == "bf16" else O.round_f32
    counts = ref["counts"].numpy()
    rtol = RTOL[wl.dtype]
    for n, g in (("W1", "dW1"), ("b1", "db1"), ("W2", "dW2"), ("b2", "db2")):
        old = O.to64(inp[n])
        want = O.sgd_step(old, grads[g], lr, store)
        got = O.to64(P[n].cpu())
        live = counts > 0
        dg = grads[g][live]
        tol = _ulp(want[live], wl.dtype) + lr * rtol * (np.abs(dg) + rms(dg))
        assert np.all(np.abs(got[live] - want[live]) <= tol), n
        np.testing.assert_array_equal(got[~live], old[~live], n + " (experts without rows)")
        if n in ("W1", "W2"):   # the update is visible, not absorbed by the rounding
            assert np.median(np.abs(got[live] - old[live])) > 2 * np.median(_ulp(old[live], wl.dtype)), n


@pytest.mark.parametrize("name", ["bf16_skew", "bf16_grid3d", "f32_grid4d", "few_alive", "bf16_maxgrid",
                                  "alive_many"])
def test_alive_topk(name):
    """DMOE_FLAG_ALIVE_TOPK: TopK among the alive experts (dead ones only to fill up
    when fewer than k respond), the whole layer forward and backward against the
    oracle's topk_alive_bruteforce routing; the chosen set differs from the plain
    TopK's on these partially alive grids."""
    from paper_2002_04013_amd.abi import DMOE_FLAG_ALIVE_TOPK
    # alive_many: more 8-token passes than blocks (every block loops), half the grid alive
    wl = CASES.get(name) or {
        "few_alive": Workload("few_alive", 30, T=160, D=64, H=64, d=2, M=8, k=4, dtype="bf16", act="gelu",
                              p_alive=0.05),
        "alive_many": Workload("alive_many", 31, T=8300, D=64, H=64, d=2, M=8, k=4, dtype="bf16", act="relu",
                               p_alive=0.5),
    }[name]
    say(f"[parity] alive TopK {name}")
    inp = make_inputs(wl, "cpu")
    if name == "few_alive":
        alive = torch.zeros(wl.N, dtype=torch.uint8)
        alive[[3, 17, 40]] = 1                     # three alive experts, k = 4
        inp["alive"] = alive
    gpu = gpu_run(wl, inp, flags=DMOE_FLAG_ALIVE_TOPK)
    fwd, bwd = oracle_run(wl, inp, alive_topk=True)
    compare(wl, inp, gpu, fwd, bwd)
    plain, _ = oracle_run(wl, inp, backward=False)
    assert not np.array_equal(plain["idx"], fwd["idx"])
    live = inp["alive"].numpy().astype(bool)
    chosen_live = live[gpu["idx"].numpy()].sum(axis=1)
    assert (chosen_live == min(wl.k, int(live.sum()))).all()


@pytest.mark.parametrize("flags", [0, 2])
def test_non_finite_inputs_keep_indices_valid(flags):
    """Tokens whose x holds NaN or infinities get an unspecified choice, but every
    index stays a valid expert id and the dispatch stays consistent; the other tokens
    are routed as usual."""
    wl = CASES["bf16_skinny"]
    say(f"[parity] non-finite inputs, flags={flags}")
    inp = make_inputs(wl, "cpu")
    x = inp["x"].clone()
    x[3, 5] = float("nan")
    x[10, :] = float("inf")
    x[11, 0] = -float("inf")
    inp["x"] = x
    gpu = gpu_run(wl, inp, backward=False, flags=flags)
    idx = gpu["idx"].numpy()
    assert idx.min() >= 0 and idx.max() < wl.N
    counts = gpu["counts"].numpy()
    offsets = gpu["offsets"].numpy()
    assert offsets[0] == 0 and np.all(np.diff(offsets) == counts)
    clean = inp.copy()
    clean["x"] = make_inputs(wl, "cpu")["x"]
    ref = gpu_run(wl, clean, backward=False, flags=flags)
    keep = np.ones(wl.T, bool)
    keep[[3, 10, 11]] = False
    np.testing.assert_array_equal(idx[keep], ref["idx"].numpy()[keep])
