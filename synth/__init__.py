"""Seeded synthetic workloads (shapes, weights, inputs) for the drafting path.

Shared by the oracle and the GPU path; holds no drafting arithmetic.
"""
from .configs import (DraftConfig, CONFIGS, TINY_F32, L3_8B_BS1, L3_8B_BS16, L3_8B_TREE,
                      L3_70B_BS32, L3_8B_BS1_CATCHUP, L3_8B_BS16_CATCHUP, L3_8B_BS1_T1, L2_7B_BS1, L2_7B_BS1_M1,
                      L2_7B_BS1_M2, SMALL_BF16_CHAIN,
                      SMALL_BF16_TREE, SMALL_F32_CHAIN, scoring_target)
from .gen import (ParamSet, Weights, Inputs, make_weights, make_param_set, make_inputs,
                  ctx_lengths, new_counts, make_verify_chain,
                  make_verify_tree_targets, host_weights, host_inputs, to_host, derive_seed, torch_dtype)
