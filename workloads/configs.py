"""The DMoE workloads, named by what they are.

Shapes follow the paper's Transformer-style experts (d_model 1024, FFN 4096,
GELU; top-4 routing; a 10% expert failure rate), a wide layer that replaces
a Transformer FFN (d_model 4096, FFN 16384), and the paper's feed-forward block
experts with layer normalisation (1024 -> 4096 -> 4096 -> 1024, ReLU).
"""
from dataclasses import dataclass, replace


@dataclass(frozen=True)
class Workload:
    name: str
    cfg_id: int          # seeds the generators; distinct per workload
    T: int               # tokens
    D: int               # d_model
    H: int               # expert hidden size
    d: int               # grid dimensions
    M: int               # indices per grid dimension
    k: int               # experts per token
    dtype: str           # "f32" or "bf16" (storage of x, weights, activations)
    act: str             # "relu" or "gelu" (erf form)
    p_alive: float = 1.0 # Bernoulli probability that an expert responds
    gate_scale: float = 1.0
    skew_rows: int = 0   # per grid dim, this many indices get a further x4 gate scale
    backward: bool = True
    seed: int = 0
    expert: str = "ffn"  # "ffn": Linear-act-Linear; "ffblock": the LayerNorm block of Sec. 4.1
    ln_init: str = "standard"  # ffblock: LayerNorm scale 1, shift 0; "split": scale 1/2, shift +-3

    @property
    def N(self) -> int:
        return self.M ** self.d

    @property
    def dM(self) -> int:
        return self.d * self.M

    @property
    def P(self) -> int:
        return self.T * self.k


WORKLOADS = {
    # 64 tokens, d_model 64, 4x4 grid, top-2, ReLU experts, fp32.
    "tiny_f32": Workload("tiny_f32", 0, T=64, D=64, H=256, d=2, M=4, k=2,
                         dtype="f32", act="relu"),
    # Transformer-scale forward: 4096 tokens, 32x32 grid, top-4, 1024->4096->1024 GELU.
    "tfm_fwd": Workload("tfm_fwd", 1, T=4096, D=1024, H=4096, d=2, M=32, k=4,
                        dtype="bf16", act="gelu", backward=False),
    # Same shapes, fwd+bwd, 10% of experts dead and a concentrated (skewed) gate.
    "tfm_fail_skew": Workload("tfm_fail_skew", 2, T=4096, D=1024, H=4096, d=2, M=32,
                              k=4, dtype="bf16", act="gelu", p_alive=0.9,
                              gate_scale=4.0, skew_rows=4),
    # 3-D grid 16x16x16, 16384 tokens, 5% of experts dead.
    "grid3d": Workload("grid3d", 3, T=16384, D=1024, H=4096, d=3, M=16, k=4,
                       dtype="bf16", act="gelu", p_alive=0.95),
    # Wide layer: 32768 tokens (16 x 2048), d_model 4096, 16x16 grid, 4096->16384->4096.
    "wide": Workload("wide", 4, T=32768, D=4096, H=16384, d=2, M=16, k=4,
                     dtype="bf16", act="gelu"),
    # The paper's own expert (Sec. 4.1): feed-forward blocks 1024->4096->4096->1024 with
    # LayerNorm and ReLU between the layers, batches of 2048 rows per block: 131072
    # tokens, 16x16 grid (256 blocks), top-4 -> 2048 rows per expert on average.
    "ffblock": Workload("ffblock", 5, T=131072, D=1024, H=4096, d=2, M=16, k=4,
                        dtype="bf16", act="relu", expert="ffblock"),
}


def get_workload(name: str) -> Workload:
    return WORKLOADS[name]


def small_workload(base: str, **kw) -> Workload:
    """A reduced copy of a named workload (for parity cases the oracle finishes fast)."""
    return replace(WORKLOADS[base], **kw)
