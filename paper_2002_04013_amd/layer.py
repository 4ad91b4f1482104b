"""One DMoE layer on one GPU: buffers (torch.empty on the device) and the order of
the C-ABI calls for the forward and the backward pass.

Forward:  gate_topk -> dispatch -> expert_ffn_fwd -> combine   (DMoELayer)
Backward: combine_bwd -> gate_topk_bwd -> expert_ffn_bwd -> dispatch_bwd
With recompute=True the backward regenerates h and a (expert_ffn_bwd_recompute), so
they need not be kept from the forward: h and a are then scratch shared by both passes.
"""
import torch

from . import abi


class DMoELayer:
    """Device buffers for one layer shape; parameters are passed per call."""

    def __init__(self, T, D, H, d, M, k, dtype="bf16", act="gelu", device="cuda",
                 dh_aliases_h=False, flags=0, recompute=False):
        self.dims = abi.make_dims(T, D, H, d, M, k, dtype, act, flags)
        self.T, self.D, self.H, self.d, self.M, self.k = T, D, H, d, M, k
        self.recompute = recompute
        self.N = M ** d
        self.P = T * k
        self.dt = torch.bfloat16 if dtype == "bf16" else torch.float32
        dev = torch.device(device)
        e = lambda *s, dt=None: torch.empty(s, dtype=dt or self.dt, device=dev)
        i32 = torch.int32
        nws = abi.workspace_bytes(self.dims)
        if nws == 0:
            raise abi.DmoeError("unsupported layer shape")
        self.ws = torch.empty(nws, dtype=torch.uint8, device=dev)
        P, N = self.P, self.N
        self.idx = e(T, k, dt=i32)
        self.w = e(T, k, dt=torch.float32)
        self.g = e(T, k, dt=torch.float32)
        self.scores = e(T, d * M, dt=torch.float32)
        self.counts = e(N, dt=i32)
        self.offsets = e(N + 1, dt=i32)
        self.row_token = e(max(P, 1), dt=i32)
        self.pos = e(T, k, dt=i32)
        self.x_perm = e(max(P, 1), D)
        self.h = e(max(P, 1), H)
        self.a = e(max(P, 1), H)
        self.y_perm = e(max(P, 1), D)
        self.y = e(T, D)
        # backward
        self.dy_perm = e(max(P, 1), D)
        self.dw = e(T, k, dt=torch.float32)
        self.dg = e(T, k, dt=torch.float32)
        self.dh = self.h if dh_aliases_h else e(max(P, 1), H)
        self.dx_perm = e(max(P, 1), D)
        self.dx = e(T, D)

    def forward(self, x, Wg, bg, alive, W1, b1, W2, b2, scores=True):
        D = self.dims
        abi.dmoe_gate_topk(D, x, Wg, bg, alive, self.idx, self.w, self.g,
                           self.scores if scores else None, self.ws)
        abi.dmoe_dispatch(D, x, self.idx, alive, self.counts, self.offsets, self.row_token,
                          self.pos, self.x_perm, self.ws)
        abi.dmoe_expert_ffn_fwd(D, self.offsets, self.x_perm, W1, b1, W2, b2, self.h, self.a,
                                self.y_perm, self.ws)
        abi.dmoe_combine(D, self.y_perm, self.pos, self.w, self.y)
        return self.y

    def backward(self, dy, x, Wg, alive, W1, W2, dW1, db1, dW2, db2, dWg, dbg, b1=None):
        """b1 is needed only with recompute=True (the up-projection is run again)."""
        D = self.dims
        abi.dmoe_combine_bwd(D, dy, self.y_perm, self.pos, self.w, self.dy_perm, self.dw)
        abi.dmoe_gate_topk_bwd(D, x, self.idx, self.w, self.dw, alive, self.dg, dWg, dbg, self.ws)
        if self.recompute:
            if b1 is None:
                raise abi.DmoeError("recompute=True needs b1 in backward")
            abi.dmoe_expert_ffn_bwd_recompute(D, self.offsets, self.counts, self.x_perm, W1, b1, W2,
                                              self.dy_perm, self.h, self.a, self.dx_perm, dW1, db1, dW2,
                                              db2, self.ws)
        else:
            abi.dmoe_expert_ffn_bwd(D, self.offsets, self.counts, self.x_perm, self.h, self.a,
                                    self.dy_perm, W1, W2, self.dh, self.dx_perm, dW1, db1, dW2, db2,
                                    self.ws)
        abi.dmoe_dispatch_bwd(D, self.dx_perm, self.pos, self.idx, self.dg, Wg, self.dx)
        return self.dx


class DMoEBlockLayer:
    """A DMoE layer whose experts are the feed-forward blocks with layer normalisation
    (dmoe_expert_ffblock_*): H is the block's hidden width F.  Parameters are dicts of
    device tensors keyed by abi.FFBLOCK_PARAMS; the per-row tensors the forward keeps
    are in self.acts, the backward's row gradients in g1 (dh1) and g2 (dh2).

    Forward:  gate_topk -> dispatch -> expert_ffblock_fwd -> combine
    Backward: combine_bwd -> gate_topk_bwd -> expert_ffblock_bwd -> dispatch_bwd
    """

    def __init__(self, T, D, H, d, M, k, dtype="bf16", act="relu", device="cuda", flags=0):
        self.dims = abi.make_dims(T, D, H, d, M, k, dtype, act, flags)
        self.T, self.D, self.H, self.d, self.M, self.k = T, D, H, d, M, k
        self.N = M ** d
        self.P = T * k
        self.dt = torch.bfloat16 if dtype == "bf16" else torch.float32
        dev = torch.device(device)
        e = lambda *s, dt=None: torch.empty(s, dtype=dt or self.dt, device=dev)
        i32, f32 = torch.int32, torch.float32
        nws = abi.workspace_bytes(self.dims)
        if nws == 0:
            raise abi.DmoeError("unsupported layer shape")
        self.ws = torch.empty(nws, dtype=torch.uint8, device=dev)
        P, N, R = self.P, self.N, max(self.P, 1)
        self.idx = e(T, k, dt=i32)
        self.w = e(T, k, dt=f32)
        self.g = e(T, k, dt=f32)
        self.scores = e(T, d * M, dt=f32)
        self.counts = e(N, dt=i32)
        self.offsets = e(N + 1, dt=i32)
        self.row_token = e(R, dt=i32)
        self.pos = e(T, k, dt=i32)
        self.x_perm = e(R, D)
        self.acts = dict(h1=e(R, H), a1=e(R, H), st1=e(R, 2, dt=f32), h2=e(R, H), a2=e(R, H), st2=e(R, 2, dt=f32))
        self.y_perm = e(R, D)
        self.y = e(T, D)
        self.dy_perm = e(R, D)
        self.dw = e(T, k, dt=f32)
        self.dg = e(T, k, dt=f32)
        self.g1 = e(R, H)
        self.g2 = e(R, H)
        self.dx_perm = e(R, D)
        self.dx = e(T, D)

    def forward(self, x, Wg, bg, alive, params, scores=True):
        D = self.dims
        abi.dmoe_gate_topk(D, x, Wg, bg, alive, self.idx, self.w, self.g,
                           self.scores if scores else None, self.ws)
        abi.dmoe_dispatch(D, x, self.idx, alive, self.counts, self.offsets, self.row_token,
                          self.pos, self.x_perm, self.ws)
        abi.dmoe_expert_ffblock_fwd(D, self.offsets, self.x_perm, params, self.acts, self.y_perm, self.ws)
        abi.dmoe_combine(D, self.y_perm, self.pos, self.w, self.y)
        return self.y

    def backward(self, dy, x, Wg, alive, params, grads, dWg, dbg):
        D = self.dims
        abi.dmoe_combine_bwd(D, dy, self.y_perm, self.pos, self.w, self.dy_perm, self.dw)
        abi.dmoe_gate_topk_bwd(D, x, self.idx, self.w, self.dw, alive, self.dg, dWg, dbg, self.ws)
        abi.dmoe_expert_ffblock_bwd(D, self.offsets, self.x_perm, params, self.acts, self.dy_perm, self.g1,
                                    self.g2, self.dx_perm, grads, self.ws)
        abi.dmoe_dispatch_bwd(D, self.dx_perm, self.pos, self.idx, self.dg, Wg, self.dx)
        return self.dx
