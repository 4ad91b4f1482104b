"""DMoE layer (Learning@home, arXiv 2002.04013) on one MI355X: HIP kernels behind
a C ABI (include/dmoe.h, libdmoe.so) and a thin Python binding."""
from . import abi
from .abi import (DmoeError, Dims, make_dims, workspace_bytes, dmoe_gate_topk, dmoe_dispatch,
                  dmoe_expert_ffn_fwd, dmoe_combine, dmoe_combine_bwd, dmoe_gate_topk_bwd,
                  dmoe_expert_ffn_bwd, dmoe_dispatch_bwd, dmoe_expert_ffn_bwd_recompute,
                  dmoe_expert_ffn_bwd_sgd, dmoe_expert_ffblock_fwd, dmoe_expert_ffblock_bwd, dmoe_ln_act_fwd,
                  dmoe_ln_act_bwd)
from .layer import DMoELayer, DMoEBlockLayer

__all__ = ["abi", "DmoeError", "Dims", "make_dims", "workspace_bytes", "dmoe_gate_topk",
           "dmoe_dispatch", "dmoe_expert_ffn_fwd", "dmoe_combine", "dmoe_combine_bwd",
           "dmoe_gate_topk_bwd", "dmoe_expert_ffn_bwd", "dmoe_dispatch_bwd", "dmoe_expert_ffn_bwd_recompute",
           "dmoe_expert_ffn_bwd_sgd", "dmoe_expert_ffblock_fwd", "dmoe_expert_ffblock_bwd", "dmoe_ln_act_fwd",
           "dmoe_ln_act_bwd", "DMoELayer", "DMoEBlockLayer"]
