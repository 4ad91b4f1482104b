"""Seeded synthetic inputs for the DMoE layer, shared by the HIP path and the oracle.

This package holds no arithmetic of the method: it only names the workloads
(shapes, dtypes, activation, failure rate) and draws their random tensors.
The random draws are torch generators seeded per tensor and per expert, so one
expert's weights can be regenerated on their own.

Recipe (every workload, seed 0 unless a test says otherwise):
  x ~ N(0,1), dy ~ N(0,1)                         shape [T, D]
  gate weight Wg ~ N(0, 1/D), bias bg ~ N(0, 1/D)  shapes [d*M, D], [d*M]
  W1_e ~ N(0, 1/D), b1_e ~ N(0, 1/D)              shapes [H, D], [H]
  W2_e ~ N(0, 1/H), b2_e ~ N(0, 1/H)              shapes [D, H], [D]
  alive_e ~ Bernoulli(p_alive)                     shape [N], uint8
Block experts (LayerNorm feed-forward blocks, hidden width F = H):
  W1 ~ N(0, 1/D), W2, W3 and b2, b3 ~ N(0, 1/F); LayerNorm scale 1 and shift 0,
  or scale 1/2 and shift +-3 per feature (ln_init "split")
Draws are fp32 and are rounded to the layer dtype (bf16 round-to-nearest-even).
Every fan-in here is a power of four, so 1/sqrt(fan_in) is an exact power of two.
"""
from .configs import WORKLOADS, Workload, get_workload, small_workload
from .gen import (make_gate, make_alive, make_x, make_dy, make_expert,
                  make_experts, make_inputs, tensor_seed, BLOCK_PARAMS, make_block_expert,
                  make_block_experts, make_block_inputs)

__all__ = ["WORKLOADS", "Workload", "get_workload", "small_workload", "make_gate",
           "make_alive", "make_x", "make_dy", "make_expert", "make_experts",
           "make_inputs", "tensor_seed", "BLOCK_PARAMS", "make_block_expert", "make_block_experts",
           "make_block_inputs"]
