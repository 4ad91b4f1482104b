"""GPU parity of the feed-forward block experts with layer normalisation (Sec. 4.1)
against the oracle, through the C ABI.

The activation's derivative after layer normalisation is a decision (ReLU: z > 0).
Where an exact z lies within the GPU's rounding error of the kink, either branch is a
correct result of the GPU's arithmetic, so the inputs are built to leave no such
element: the LayerNorm step tests zero da where the exact |z| is below a margin, and
the bf16 ReLU layer cases use LayerNorm shifts of +-3 with scale 1/2 (ln_init "split",
|z| >= 1/2 wherever |n| < 5; the test asserts the margin).  fp32 cases use the usual
LayerNorm initialisation (scale 1, shift 0), where the ambiguity window is ~1e-7;
GELU cases have no decision at all.
"""
import zlib

import numpy as np
import pytest
import torch

import oracle as O
from parity_util import RTOL, assert_close, check_gate, say
from workloads import Workload, BLOCK_PARAMS, make_block_inputs

pytestmark = pytest.mark.gpu

CASES = {
    "f32_relu": Workload("ffb_f32_relu", 40, T=96, D=64, H=128, d=2, M=3, k=2, dtype="f32", act="relu",
                         p_alive=0.8, expert="ffblock"),
    "f32_gelu_split": Workload("ffb_f32_gelu", 41, T=80, D=64, H=192, d=1, M=5, k=3, dtype="f32", act="gelu",
                               expert="ffblock", ln_init="split"),
    "bf16_relu_split": Workload("ffb_bf16_relu", 42, T=300, D=128, H=256, d=2, M=4, k=2, dtype="bf16",
                                act="relu", p_alive=0.9, expert="ffblock", ln_init="split"),
    "bf16_gelu": Workload("ffb_bf16_gelu", 43, T=257, D=64, H=320, d=3, M=2, k=3, dtype="bf16", act="gelu",
                          expert="ffblock"),
    # P >= 96 N: the 256x256-tile GEMM configuration of the full-size workload
    "bf16_fat_split": Workload("ffb_bf16_fat", 44, T=1600, D=128, H=256, d=2, M=3, k=2, dtype="bf16",
                               act="relu", expert="ffblock", ln_init="split"),
}


def _offsets_from_counts(counts):
    return np.concatenate([[0], np.cumsum(counts)]).astype(np.int32)


@pytest.mark.parametrize("dtype,kind,F", [("f32", "relu", 128), ("f32", "gelu", 320), ("bf16", "relu", 256),
                                          ("bf16", "gelu", 4096), ("bf16", "relu", 64)])
def test_ln_act_step(dtype, kind, F):
    """dmoe_ln_act_fwd / _bwd on the same seeded rows as the oracle: stats, a, dh
    (separate buffer and in place over da), dgamma and dbeta of every expert with rows."""
    from paper_2002_04013_amd import abi
    say(f"[ffblock] LN step {dtype} {kind} F={F}")
    g = torch.Generator().manual_seed(zlib.crc32(f"{dtype}/{kind}/{F}".encode()))
    N, T, k = 9, 160, 2
    counts = np.array([37, 0, 41, 3, 0, 96, 1, 22, 100])
    P = int(counts.sum())
    assert P <= T * k
    off = _offsets_from_counts(counts)
    dt = torch.float32 if dtype == "f32" else torch.bfloat16
    h = (torch.randn(T * k, F, generator=g) * 2 + 0.5).to(dt)
    gam = (1 + 0.5 * torch.randn(N, F, generator=g)).to(dt)
    bet = (0.5 * torch.randn(N, F, generator=g)).to(dt)
    da = torch.randn(T * k, F, generator=g).to(dt)
    # no decision near the kink: da = 0 where the exact |z| < 1e-3
    e_of = np.repeat(np.arange(N), counts)
    h64, g64, b64 = O.to64(h), O.to64(gam), O.to64(bet)
    z = np.zeros((T * k, F))
    fw = O.layernorm_act_forward(h64[:P], g64[e_of], b64[e_of], kind)
    z[:P] = fw["z"]
    near = np.zeros((T * k, F), bool)
    near[:P] = np.abs(z[:P]) < 1e-3
    da = torch.where(torch.from_numpy(near), torch.zeros_like(da), da)
    dims = abi.make_dims(T, 64, F, 2, 3, k, dtype, kind)
    dev = torch.device("cuda")
    t = dict(h=h, gam=gam, bet=bet, da=da, off=torch.from_numpy(off))
    t = {n: v.to(dev) for n, v in t.items()}
    a = torch.full((T * k, F), 9.0, dtype=dt, device=dev)
    st = torch.zeros(T * k, 2, dtype=torch.float32, device=dev)
    abi.dmoe_ln_act_fwd(dims, t["off"], t["h"], t["gam"], t["bet"], a, st)
    dh = torch.empty_like(a)
    dg = torch.full((N, F), 7.0, dtype=dt, device=dev)
    db = torch.full((N, F), 7.0, dtype=dt, device=dev)
    abi.dmoe_ln_act_bwd(dims, t["off"], t["h"], st, t["gam"], t["bet"], t["da"], dh, dg, db)
    dh2 = t["da"].clone()
    dg2, db2 = torch.full_like(dg, 7.0), torch.full_like(db, 7.0)
    abi.dmoe_ln_act_bwd(dims, t["off"], t["h"], st, t["gam"], t["bet"], dh2, dh2, dg2, db2)
    torch.cuda.synchronize()
    rtol = RTOL[dtype]
    stc = st.cpu().numpy().astype(np.float64)
    np.testing.assert_allclose(stc[:P, 0], fw["mean"], rtol=1e-5, atol=1e-6 * np.abs(fw["mean"]).max())
    np.testing.assert_allclose(stc[:P, 1], fw["rstd"], rtol=1e-5)
    store = O.round_bf16 if dtype == "bf16" else (lambda v: v)
    assert_close(a[:P].cpu(), store(fw["a"]), rtol, "a")
    assert bool((a[P:] == 9.0).all()), "rows past offsets[N] were written"
    for e in range(N):
        lo, hi = off[e], off[e + 1]
        if hi == lo:
            assert bool((dg[e] == 7.0).all() and (db[e] == 7.0).all()), f"expert {e} without rows was written"
            continue
        ref_dh, ref_dg, ref_db = O.layernorm_act_backward(O.to64(da[lo:hi]), h64[lo:hi], g64[e], b64[e], kind)
        assert_close(dh[lo:hi].cpu(), ref_dh, rtol, f"dh[{e}]")
        assert_close(dg[e].cpu(), ref_dg, rtol, f"dgamma[{e}]")
        assert_close(db[e].cpu(), ref_db, rtol, f"dbeta[{e}]")
    assert torch.equal(dh2[:P], dh[:P]), "in-place dh differs"
    assert torch.equal(dg2, dg) and torch.equal(db2, db)


def _gpu_block(wl, inp):
    from paper_2002_04013_amd import DMoEBlockLayer
    dev = torch.device("cuda")
    t = {n: v.to(dev) for n, v in inp.items() if n != "params"}
    prm = {n: v.to(dev) for n, v in inp["params"].items()}
    L = DMoEBlockLayer(wl.T, wl.D, wl.H, wl.d, wl.M, wl.k, wl.dtype, wl.act, device=dev)
    L.forward(t["x"], t["Wg"], t["bg"], t["alive"], prm)
    grads = {n: torch.full_like(v, 7.0) for n, v in prm.items()}
    dWg, dbg = torch.empty_like(t["Wg"]), torch.empty_like(t["bg"])
    L.backward(t["dy"], t["x"], t["Wg"], t["alive"], prm, grads, dWg, dbg)
    torch.cuda.synchronize()
    out = dict(idx=L.idx, w=L.w, g=L.g, scores=L.scores, counts=L.counts, offsets=L.offsets, y=L.y,
               y_perm=L.y_perm, dy_perm=L.dy_perm, dw=L.dw, dg=L.dg, g1=L.g1, g2=L.g2, dx_perm=L.dx_perm,
               dx=L.dx, dWg=dWg, dbg=dbg, **L.acts)
    out = {n: v.cpu() for n, v in out.items()}
    out["grads"] = {n: v.cpu() for n, v in grads.items()}
    return out


def _oracle_block(wl, inp):
    f = lambda v: O.to64(v)
    x, Wg, bg, dy = f(inp["x"]), f(inp["Wg"]), f(inp["bg"]), f(inp["dy"])
    alive = inp["alive"].numpy()
    prm = {n: f(v) for n, v in inp["params"].items()}
    experts = lambda e: {n: prm[n][e] for n in BLOCK_PARAMS}
    store = O.round_bf16 if wl.dtype == "bf16" else None
    fwd = O.layer_forward(x, Wg, bg, experts, alive, wl.d, wl.M, wl.k, wl.act, store=store, expert="ffblock")
    bwd = O.layer_backward(fwd, dy, x, Wg, experts, alive, wl.d, wl.M, wl.k, wl.act, store=store,
                           expert="ffblock")
    return fwd, bwd, prm


@pytest.mark.parametrize("name", list(CASES))
def test_ffblock_layer_parity(name):
    wl = CASES[name]
    say(f"[ffblock] layer parity {name}: T={wl.T} D={wl.D} F={wl.H} grid {wl.M}^{wl.d} k={wl.k} "
        f"{wl.dtype} {wl.act} ln={wl.ln_init}")
    inp = make_block_inputs(wl, "cpu")
    gpu = _gpu_block(wl, inp)
    fwd, bwd, prm = _oracle_block(wl, inp)
    rtol = RTOL[wl.dtype]
    check_gate(wl, gpu["scores"], gpu["w"], gpu["g"], fwd["S"], fwd["w"], fwd["g"], O.to64(inp["x"]),
               O.to64(inp["Wg"]))
    np.testing.assert_array_equal(gpu["idx"].numpy(), fwd["idx"], "idx")
    np.testing.assert_array_equal(gpu["counts"].numpy(), fwd["counts"], "counts")
    np.testing.assert_array_equal(gpu["offsets"].numpy(), fwd["offsets"], "offsets")
    rows = int(fwd["offsets"][-1])
    if wl.act == "relu" and wl.dtype == "bf16":
        # the inputs leave every activation decision at least 1e-2 from the kink
        for i, (hn, gn, bn) in enumerate((("h1", "g1", "be1"), ("h2", "g2", "be2"))):
            e_of = np.repeat(np.arange(wl.N), fwd["counts"])
            z = O.layernorm_act_forward(fwd[hn], prm[gn][e_of], prm[bn][e_of], wl.act)["z"]
            assert np.abs(z).min() > 1e-2, (hn, np.abs(z).min())
    if rows:
        for n in ("h1", "a1", "h2", "a2"):
            assert_close(gpu[n][:rows], fwd[n], rtol, n)
        # statistics of the stored h: each stored value is within one storage ulp of the
        # oracle's (2^-8 relative for bf16), so the mean moves by at most that much of
        # mean|h| and rstd by that relative amount (fp32: accumulation error only)
        u = 2.0 ** -7 if wl.dtype == "bf16" else 1e-5
        for n, (hn, mn, rn) in (("st1", ("h1", "mean1", "rstd1")), ("st2", ("h2", "mean2", "rstd2"))):
            st = gpu[n][:rows].numpy().astype(np.float64)
            np.testing.assert_allclose(st[:, 1], fwd[rn], rtol=u, err_msg=n)
            assert np.all(np.abs(st[:, 0] - fwd[mn]) <= u * np.abs(fwd[hn]).mean(axis=1) + 1e-30), n
        assert_close(gpu["y_perm"][:rows], fwd["y_perm"], rtol, "y_perm")
        assert_close(gpu["dy_perm"][:rows], bwd["dy_perm"], rtol, "dy_perm")
        assert_close(gpu["g2"][:rows], bwd["dh2"], rtol, "dh2")
        assert_close(gpu["g1"][:rows], bwd["dh1"], rtol, "dh1")
        assert_close(gpu["dx_perm"][:rows], bwd["dx_perm"], rtol, "dx_perm")
    assert_close(gpu["y"], fwd["y"], rtol, "y")
    assert_close(gpu["dw"], bwd["dw"], rtol, "dw")
    assert_close(gpu["dg"], bwd["dg"], rtol, "dg")
    assert_close(gpu["dx"], bwd["dx"], rtol, "dx")
    assert_close(gpu["dWg"], bwd["dWg"], rtol, "dWg")
    assert_close(gpu["dbg"], bwd["dbg"], rtol, "dbg")
    counts = fwd["counts"]
    for e in range(wl.N):
        for n in BLOCK_PARAMS:
            if counts[e] > 0:
                assert_close(gpu["grads"][n][e], bwd["expert_grads"][e][n], rtol, f"d{n}[{e}]")
            else:
                assert bool((gpu["grads"][n][e].float() == 7.0).all()), f"d{n}[{e}] was written"


def test_ffblock_deterministic():
    wl = CASES["bf16_gelu"]
    inp = make_block_inputs(wl, "cpu")
    a, b = _gpu_block(wl, inp), _gpu_block(wl, inp)
    for n in ("y", "dx", "dWg", "g1", "g2"):
        assert torch.equal(a[n], b[n]), n
    for n in BLOCK_PARAMS:
        assert torch.equal(a["grads"][n], b["grads"][n]), n
