"""CPU oracle for the DMoE layer -- TEST INFRASTRUCTURE ONLY.

Plain, slow, fp64 NumPy statement of what one Decentralized Mixture-of-Experts
layer computes (Ryabinin & Gusev, "Towards Crowdsourced Training of Large
Neural Networks using Decentralized Mixture-of-Experts", arXiv 2002.04013):

  * the grid-factored gate, d linear layers g_i whose scores add up over the
    expert grid (Sec. 3.2, restated in App. C);
  * TopK over the grid, by brute force over every cell, by the beam search of
    App. C (Algorithm 1) and by the product-key shortcut App. C points to, and
    TopK among the alive experts only (brute force);
  * the Eq. 1 softmax weights over the chosen experts, with non-responding
    experts excluded and the rest renormalised (Sec. 3.1, Sec. 3.2);
  * grouping of (token, expert) pairs per expert (the Runtime batching of
    Sec. 3.3), the expert feed-forward blocks and the weighted sum of Eq. 1;
  * the backward pass of all of the above, and the gradient-descent update of an
    expert's parameters that the Runtime's Backward applies (Sec. 3.3);
  * the feed-forward block expert of Sec. 4.1 with layer normalisation between its
    linear layers (oracle.ffblock).

Only tests/, __graft_entry__.smoke() and bench.py's CPU-baseline leg may import
this package.  The product path never calls it, and it imports nothing from
the HIP path.  Every function is pinned by tests marked "not gpu" against
brute force, library routines, closed forms, autograd or hand-worked cases.
"""
from .dmoe import (
    to64, gate_scores, decision_scores, flat_index, uid_of, cell_totals,
    topk_bruteforce, topk_beam, topk_product_key, topk_alive_bruteforce, mixture_weights, act, act_grad,
    dispatch, expert_forward, expert_backward, gate_backward, layer_forward,
    layer_backward, routing, chosen_totals, round_bf16, expert_forward_stored, round_f32, sgd_step,
)
from .ffblock import (
    LN_EPS, PARAM_NAMES, layernorm_act_forward, layernorm_act_backward, ffblock_forward_stored,
    ffblock_backward,
)

__all__ = [
    "to64", "gate_scores", "decision_scores", "flat_index", "uid_of", "cell_totals",
    "topk_bruteforce", "topk_beam", "topk_product_key", "mixture_weights", "act",
    "act_grad", "dispatch", "expert_forward", "expert_backward", "gate_backward",
    "layer_forward", "layer_backward", "routing", "chosen_totals", "round_bf16", "expert_forward_stored",
    "round_f32", "sgd_step", "topk_alive_bruteforce", "LN_EPS", "PARAM_NAMES", "layernorm_act_forward",
    "layernorm_act_backward", "ffblock_forward_stored", "ffblock_backward",
]
