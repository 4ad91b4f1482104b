"""dmoe_expert_ffn_fwd_noalloc (the expert forward with its tile plan in the library's
static device scratch) against dmoe_expert_ffn_fwd with a caller workspace: the same
outputs bit for bit, over consecutive calls whose sizes shrink (a later call must not
read what an earlier, larger one left in the shared scratch)."""
import pytest
import torch

from paper_2002_04013_amd import abi

pytestmark = pytest.mark.gpu


def _case(T, D, H, M, d, k, dtype, seed):
    dev = torch.device("cuda:0")
    g = torch.Generator(device="cpu").manual_seed(seed)
    N, P = M ** d, T * k
    dt = torch.bfloat16 if dtype == "bf16" else torch.float32
    # rows per expert: a seeded random partition of the P pairs, some experts empty
    cut = torch.sort(torch.randint(0, P + 1, (N - 1,), generator=g)).values
    offsets = torch.cat([torch.zeros(1, dtype=torch.int64), cut, torch.full((1,), P)]).to(torch.int32)
    rn = lambda *s, sc=1.0: (torch.randn(*s, generator=g) * sc).to(dt).to(dev)
    x_perm = rn(P, D)
    W1, b1 = rn(N, H, D, sc=D ** -0.5), rn(N, H, sc=D ** -0.5)
    W2, b2 = rn(N, D, H, sc=H ** -0.5), rn(N, D, sc=H ** -0.5)
    dims = abi.make_dims(T, D, H, d, M, k, dtype, "gelu")
    return dims, offsets.to(dev), x_perm, (W1, b1, W2, b2), P


def _outs(P, D, H, dt):
    e = lambda *s: torch.full(s, float("nan"), dtype=dt, device="cuda:0")
    return e(P, H), e(P, H), e(P, D)


def test_noalloc_matches_workspace_form():
    torch.cuda.set_device(0)
    # sizes shrink from call to call: fat tiles (many rows per expert), then few rows per
    # expert with fewer experts, then a tiny fp32 layer
    cases = [(4096, 256, 512, 4, 2, 2, "bf16", 1), (1500, 128, 256, 8, 2, 2, "bf16", 2),
             (100, 64, 128, 3, 2, 2, "f32", 3)]
    for T, D, H, M, d, k, dtype, seed in cases:
        dims, offsets, x_perm, (W1, b1, W2, b2), P = _case(T, D, H, M, d, k, dtype, seed)
        dt = x_perm.dtype
        ws = torch.empty(abi.workspace_bytes(dims), dtype=torch.uint8, device="cuda:0")
        h0, a0, y0 = _outs(P, D, H, dt)
        abi.dmoe_expert_ffn_fwd(dims, offsets, x_perm, W1, b1, W2, b2, h0, a0, y0, ws)
        h1, a1, y1 = _outs(P, D, H, dt)
        abi.dmoe_expert_ffn_fwd_noalloc(dims, offsets, x_perm, W1, b1, W2, b2, h1, a1, y1)
        torch.cuda.synchronize()
        for name, ref, got in (("h", h0, h1), ("a", a0, a1), ("y_perm", y0, y1)):
            assert not torch.isnan(ref.float()).any(), f"{name}: reference left rows unwritten"
            assert torch.equal(ref, got), f"{name} differs (T={T}, N={M ** d}, {dtype})"


def test_noalloc_rejects_bad_arguments():
    dims = abi.make_dims(64, 64, 64, 2, 4, 2, "bf16", "gelu")
    z = torch.zeros(1, dtype=torch.bfloat16, device="cuda:0")
    with pytest.raises(abi.DmoeError):
        abi.dmoe_expert_ffn_fwd_noalloc(dims, None, z, z, z, z, z, z, z, z)
