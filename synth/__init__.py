"""Seeded synthetic workloads for the WaS decode step: shapes and random inputs.

This module holds no arithmetic of the method. It only states workload shapes
and draws seeded random tensors, which the oracle (tests) and the HIP library
(tests, bench, smoke) then both consume.

Shapes follow the models the paper evaluates (SiDP, §5.1 "Baseline and
models": Qwen3-32B, Qwen2.5-72B, Llama-3.1-70B) and the context-length mix of
its workloads (§5.1 "Workload": average S = 1K / 2K / 4K). There are no
trained weights or datasets here: weights are N(0, 0.02), KV and hidden states
N(0, 1), context lengths uniform integers in a range, block tables a seeded
permutation of the physical KV blocks.
"""

from .configs import CONFIGS, get_config, qkv_out, layer_param_count  # noqa: F401
from .gen import (  # noqa: F401
    context_lengths,
    hidden_input,
    layer_weights,
    kv_prefill,
    seed_for,
)
