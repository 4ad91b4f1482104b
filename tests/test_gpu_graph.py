"""The layer's calls recorded into a HIP graph and replayed.

The entry points allocate nothing, never synchronise and clear device memory with
kernels (no memset nodes), so a whole forward+backward step can be captured once
and replayed.  Each replay runs after eager work that overwrites the layer's
outputs, the workspace and the caller's gradient buffers, with synchronisations in
between, and must reproduce the eager step bit for bit (the path has no
floating-point atomics).  The junk written into the workspace before each replay
also checks that no entry point reads workspace memory it has not written itself.
"""
import pytest
import torch

from parity_util import say
from workloads import Workload, make_inputs, small_workload

pytestmark = pytest.mark.gpu

CASES = {
    "tiny_f32": small_workload("tiny_f32"),
    # few rows per expert: 32-row GEMM tiles, 32-deep weight-gradient k-steps
    "bf16_skinny": Workload("bf16_skinny", 40, T=512, D=256, H=512, d=2, M=8, k=4, dtype="bf16",
                            act="gelu", p_alive=0.8),
    # hundreds of rows per expert: 256x256 tiles
    "bf16_fat": Workload("bf16_fat", 41, T=2048, D=128, H=256, d=2, M=4, k=2, dtype="bf16",
                         act="relu", p_alive=0.9),
}

REPLAYS = 3


@pytest.mark.parametrize("name", list(CASES))
def test_graph_replay_matches_eager(name):
    from paper_2002_04013_amd import DMoELayer
    wl = CASES[name]
    say(f"[graph] {name}: T={wl.T} D={wl.D} H={wl.H} d={wl.d} M={wl.M} k={wl.k} {wl.dtype}")
    dev = torch.device("cuda")
    t = {n: v.to(dev) for n, v in make_inputs(wl, "cpu").items()}
    L = DMoELayer(wl.T, wl.D, wl.H, wl.d, wl.M, wl.k, wl.dtype, wl.act, device=dev)
    grads = {n: torch.empty_like(t[p]) for n, p in
             (("dW1", "W1"), ("db1", "b1"), ("dW2", "W2"), ("db2", "b2"), ("dWg", "Wg"), ("dbg", "bg"))}

    def reset_grads():
        # experts without rows keep the caller's gradients: start every step from 7
        for n in ("dW1", "db1", "dW2", "db2"):
            grads[n].fill_(7.0)

    def step():
        L.forward(t["x"], t["Wg"], t["bg"], t["alive"], t["W1"], t["b1"], t["W2"], t["b2"])
        L.backward(t["dy"], t["x"], t["Wg"], t["alive"], t["W1"], t["W2"], grads["dW1"], grads["db1"],
                   grads["dW2"], grads["db2"], grads["dWg"], grads["dbg"])

    def results():
        out = {n: getattr(L, n) for n in ("idx", "w", "g", "counts", "offsets", "y", "dw", "dg", "dx")}
        out.update(grads)
        return {n: v.clone() for n, v in out.items()}

    reset_grads()
    step()
    torch.cuda.synchronize()
    eager = results()
    say(f"[graph] {name}: eager step done")

    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        step()
    torch.cuda.synchronize()
    say(f"[graph] {name}: captured")

    for r in range(REPLAYS):
        # eager work between replays: clobber outputs and the workspace
        for n in ("y", "dx", "w", "dw", "dg"):
            getattr(L, n).fill_(float("nan"))
        L.idx.fill_(-5)
        L.ws.fill_(0xA5 if r % 2 == 0 else 0x3C)
        for v in grads.values():
            v.fill_(-1.0)
        reset_grads()
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        got = results()
        for n, v in eager.items():
            assert torch.equal(got[n], v), f"replay {r}: {n} differs from the eager step"
        say(f"[graph] {name}: replay {r} matches")


BLOCK_CASES = {
    # LayerNorm block experts, few rows per expert (32-row tiles) and many (256x256 tiles)
    "block_bf16_skinny": Workload("graph_block_skinny", 42, T=300, D=128, H=256, d=2, M=4, k=2, dtype="bf16",
                                  act="relu", p_alive=0.9, expert="ffblock"),
    "block_bf16_fat": Workload("graph_block_fat", 43, T=1600, D=128, H=256, d=2, M=3, k=2, dtype="bf16",
                               act="gelu", expert="ffblock"),
}


@pytest.mark.parametrize("name", list(BLOCK_CASES))
def test_block_graph_replay_matches_eager(name):
    """The same for the layer with LayerNorm block experts (gate, dispatch, the block's
    grouped GEMMs and LayerNorm row kernels, combine, and their backward)."""
    from paper_2002_04013_amd import DMoEBlockLayer
    from workloads import make_block_inputs
    wl = BLOCK_CASES[name]
    say(f"[graph] {name}: T={wl.T} D={wl.D} F={wl.H} d={wl.d} M={wl.M} k={wl.k} {wl.dtype} {wl.act}")
    dev = torch.device("cuda")
    inp = make_block_inputs(wl, "cpu")
    t = {n: v.to(dev) for n, v in inp.items() if n != "params"}
    prm = {n: v.to(dev) for n, v in inp["params"].items()}
    L = DMoEBlockLayer(wl.T, wl.D, wl.H, wl.d, wl.M, wl.k, wl.dtype, wl.act, device=dev)
    grads = {n: torch.empty_like(v) for n, v in prm.items()}
    dWg, dbg = torch.empty_like(t["Wg"]), torch.empty_like(t["bg"])

    def step():
        L.forward(t["x"], t["Wg"], t["bg"], t["alive"], prm)
        L.backward(t["dy"], t["x"], t["Wg"], t["alive"], prm, grads, dWg, dbg)

    def results():
        out = {n: getattr(L, n) for n in ("idx", "w", "counts", "offsets", "y", "dw", "dg", "dx")}
        out.update({"g_" + n: v for n, v in grads.items()}, dWg=dWg, dbg=dbg)
        return {n: v.clone() for n, v in out.items()}

    def reset_grads():
        for v in grads.values():
            v.fill_(7.0)

    reset_grads()
    step()
    torch.cuda.synchronize()
    eager = results()
    say(f"[graph] {name}: eager step done")
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        step()
    torch.cuda.synchronize()
    for r in range(REPLAYS):
        for n in ("y", "dx", "w", "dw", "dg"):
            getattr(L, n).fill_(float("nan"))
        for v in L.acts.values():
            v.fill_(float("nan"))
        L.idx.fill_(-5)
        L.ws.fill_(0x5A if r % 2 == 0 else 0xC3)
        dWg.fill_(-1.0)
        dbg.fill_(-1.0)
        reset_grads()
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        got = results()
        for n, v in eager.items():
            assert torch.equal(got[n], v), f"replay {r}: {n} differs from the eager step"
        say(f"[graph] {name}: replay {r} matches")
