"""CPU oracle of the PRISM drafting hot path.

TEST INFRASTRUCTURE: only the test suite, the smoke check and the benchmark's
CPU-baseline leg may import, call, link or execute anything in this package.
The GPU library and its Python binding never do, and the two share no code;
only the seeded input generator (package `synth`) serves both.

Parity status of each function (what pins it) is listed in the test module
tests/test_oracle_pins.py; no function here is "parity unpinned".
"""
from .draft import (Oracle, brute_chain, round_bf16, rmsnorm, silu, rope, rope_cos_sin,
                    softmax_attend, logsumexp, topk_ids, sample_inverse_cdf)
from ._native import linear, widen, build as build_native
from .verify import (verify_chain_greedy, verify_chain_sample, verify_tree_greedy, softmax_t,
                     draw_from)
