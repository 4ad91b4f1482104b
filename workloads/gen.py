"""Seeded generators for the DMoE workloads (torch RNG, per tensor and per expert).

Each tensor gets its own generator, seeded from (workload seed, workload id,
tensor id, expert), so any single expert can be drawn again on its own.  The
draw depends on the device type of the generator (torch's CPU and GPU streams
differ), so a test that compares two sides draws once and hands both sides the
same tensors.
"""
import torch

from .configs import Workload

_MASK64 = (1 << 64) - 1

# tensor ids
_X, _WG, _BG, _W1, _B1, _W2, _B2, _ALIVE, _DY, _SKEW, _W3, _B3, _LN = range(13)


def _mix(z: int) -> int:
    # SplitMix64 finaliser (Steele, Lea, Flood 2014) used as a seed hash.
    z = (z + 0x9E3779B97F4A7C15) & _MASK64
    z = ((z ^ (z >> 30)) * 0xBF58476D1CE4E5B9) & _MASK64
    z = ((z ^ (z >> 27)) * 0x94D049BB133111EB) & _MASK64
    return z ^ (z >> 31)


def tensor_seed(seed: int, cfg_id: int, tensor_id: int, index: int = 0) -> int:
    z = _mix(seed)
    for v in (cfg_id, tensor_id, index):
        z = _mix(z ^ (v & _MASK64))
    return z & ((1 << 63) - 1)


def _gen(device, seed):
    g = torch.Generator(device=device)
    g.manual_seed(seed)
    return g


def storage_dtype(wl: Workload):
    return torch.float32 if wl.dtype == "f32" else torch.bfloat16


def _randn(shape, scale, wl, tid, index, device):
    g = _gen(device, tensor_seed(wl.seed, wl.cfg_id, tid, index))
    v = torch.randn(shape, generator=g, device=device, dtype=torch.float32)
    if scale != 1.0:
        v.mul_(scale)           # scale is a power of two: exact
    return v.to(storage_dtype(wl))


def make_x(wl: Workload, device="cpu"):
    return _randn((wl.T, wl.D), 1.0, wl, _X, 0, device)


def make_dy(wl: Workload, device="cpu"):
    return _randn((wl.T, wl.D), 1.0, wl, _DY, 0, device)


def make_gate(wl: Workload, device="cpu"):
    """Gate weight [d*M, D] and bias [d*M]; block i of rows is the linear layer g_i."""
    s = wl.D ** -0.5
    g = torch.randn((wl.dM, wl.D), generator=_gen(device, tensor_seed(wl.seed, wl.cfg_id, _WG)),
                    device=device, dtype=torch.float32) * s
    b = torch.randn((wl.dM,), generator=_gen(device, tensor_seed(wl.seed, wl.cfg_id, _BG)),
                    device=device, dtype=torch.float32) * s
    if wl.gate_scale != 1.0 or wl.skew_rows:
        scale = torch.full((wl.dM,), float(wl.gate_scale), dtype=torch.float32)
        if wl.skew_rows:
            gs = _gen("cpu", tensor_seed(wl.seed, wl.cfg_id, _SKEW))
            for i in range(wl.d):
                hot = torch.randperm(wl.M, generator=gs)[: wl.skew_rows]
                scale[i * wl.M + hot] *= 4.0
        scale = scale.to(device)
        g = g * scale[:, None]
        b = b * scale
    return g.to(storage_dtype(wl)), b.to(storage_dtype(wl))


def make_alive(wl: Workload, device="cpu"):
    """uint8 [N]: 1 if the expert responds.  Drawn on the CPU for every device."""
    if wl.p_alive >= 1.0:
        a = torch.ones(wl.N, dtype=torch.uint8)
    else:
        g = _gen("cpu", tensor_seed(wl.seed, wl.cfg_id, _ALIVE))
        a = (torch.rand(wl.N, generator=g) < wl.p_alive).to(torch.uint8)
    return a.to(device)


def make_expert(wl: Workload, e: int, device="cpu"):
    """(W1 [H,D], b1 [H], W2 [D,H], b2 [D]) of expert e (nn.Linear layout [out, in])."""
    s1, s2 = wl.D ** -0.5, wl.H ** -0.5
    return (_randn((wl.H, wl.D), s1, wl, _W1, e, device),
            _randn((wl.H,), s1, wl, _B1, e, device),
            _randn((wl.D, wl.H), s2, wl, _W2, e, device),
            _randn((wl.D,), s2, wl, _B2, e, device))


def make_experts(wl: Workload, device="cpu", identical=False):
    """All experts stacked: W1 [N,H,D], b1 [N,H], W2 [N,D,H], b2 [N,D].

    Drawn expert by expert into preallocated storage, so the fp32 staging is
    one expert at a time.  identical=True gives every expert expert 0's weights.
    """
    dt = storage_dtype(wl)
    N, D, H = wl.N, wl.D, wl.H
    W1 = torch.empty((N, H, D), dtype=dt, device=device)
    b1 = torch.empty((N, H), dtype=dt, device=device)
    W2 = torch.empty((N, D, H), dtype=dt, device=device)
    b2 = torch.empty((N, D), dtype=dt, device=device)
    for e in range(N):
        w1, c1, w2, c2 = make_expert(wl, 0 if identical else e, device)
        W1[e].copy_(w1)
        b1[e].copy_(c1)
        W2[e].copy_(w2)
        b2[e].copy_(c2)
    return W1, b1, W2, b2


def make_inputs(wl: Workload, device="cpu", identical_experts=False):
    Wg, bg = make_gate(wl, device)
    W1, b1, W2, b2 = make_experts(wl, device, identical=identical_experts)
    return dict(x=make_x(wl, device), Wg=Wg, bg=bg, alive=make_alive(wl, device),
                W1=W1, b1=b1, W2=W2, b2=b2, dy=make_dy(wl, device))


# ---------------------------------------------------------------- block experts

BLOCK_PARAMS = ("W1", "b1", "g1", "be1", "W2", "b2", "g2", "be2", "W3", "b3")


def make_block_expert(wl: Workload, e: int, device="cpu"):
    """Parameters of feed-forward block expert e (hidden width F = wl.H), nn.Linear and
    nn.LayerNorm layouts: W1 [F,D], b1 [F] ~ N(0, 1/D); W2 [F,F], b2 [F] ~ N(0, 1/F);
    W3 [D,F], b3 [D] ~ N(0, 1/F); LayerNorm scale g and shift be [F] at 1 and 0
    (ln_init "standard"), or scale 1/2 and shift +3 or -3 by a seeded sign per feature
    ("split": every normalised value lands at least 1/2 away from the activation's kink
    for |n| < 5)."""
    D, F = wl.D, wl.H
    s1, s2 = D ** -0.5, F ** -0.5
    dt = storage_dtype(wl)
    p = dict(W1=_randn((F, D), s1, wl, _W1, e, device), b1=_randn((F,), s1, wl, _B1, e, device),
             W2=_randn((F, F), s2, wl, _W2, e, device), b2=_randn((F,), s2, wl, _B2, e, device),
             W3=_randn((D, F), s2, wl, _W3, e, device), b3=_randn((D,), s2, wl, _B3, e, device))
    for i, (gn, bn) in enumerate((("g1", "be1"), ("g2", "be2"))):
        if wl.ln_init == "standard":
            p[gn] = torch.ones(F, dtype=dt, device=device)
            p[bn] = torch.zeros(F, dtype=dt, device=device)
        elif wl.ln_init == "split":
            g = _gen("cpu", tensor_seed(wl.seed, wl.cfg_id, _LN, 2 * e + i))
            sign = torch.randint(0, 2, (F,), generator=g).to(torch.float32) * 2 - 1
            p[gn] = torch.full((F,), 0.5, dtype=dt, device=device)
            p[bn] = (3.0 * sign).to(dt).to(device)
        else:
            raise ValueError(wl.ln_init)
    return p


def make_block_experts(wl: Workload, device="cpu"):
    """Every block expert's parameters stacked over experts (dict keyed by BLOCK_PARAMS)."""
    one = make_block_expert(wl, 0, device)
    out = {n: torch.empty((wl.N,) + tuple(v.shape), dtype=v.dtype, device=device) for n, v in one.items()}
    for e in range(wl.N):
        p = one if e == 0 else make_block_expert(wl, e, device)
        for n in BLOCK_PARAMS:
            out[n][e].copy_(p[n])
    return out


def make_block_inputs(wl: Workload, device="cpu"):
    Wg, bg = make_gate(wl, device)
    return dict(x=make_x(wl, device), Wg=Wg, bg=bg, alive=make_alive(wl, device), dy=make_dy(wl, device),
                params=make_block_experts(wl, device))
