"""Plain, slow CPU oracle for the Weight-as-a-Service decode step.

TEST INFRASTRUCTURE ONLY. Only tests/, __graft_entry__.smoke() and the
cpu_baseline leg of bench.py may import this package. The HIP library and its
Python binding never import, call or link anything here, and nothing here
imports them: the two sides share no code. Inputs reach both from the seeded
generators in synth/.

What it computes (SiDP, arXiv 2605.28095):
  * §2.1: a decoder-only transformer is a stack of L identical blocks, each
    made of self-attention with query/key/value/output projections and a
    two-layer FFN with a non-linearity in between.
  * §2.2: a decode iteration produces one new token per scheduled sequence;
    the engine keeps each request's KV state (here: a paged KV cache).
  * §4.1, §4.2: Weight-as-a-Service only changes where a layer's weights live
    and how they are fetched (a pool plus a small cache of slots); the model's
    numerics are unchanged. So the oracle of the decode step is the plain
    layer definition, whatever the weight placement; decode.py holds it.
  * §4.2 "Asynchronous buffer management": pre-allocated cache slots, fills
    issued ahead on a side stream, completion notifications before compute,
    and a slot freed once compute on it is done; schedule.py holds the order
    of those operations.
  * kvalloc.py holds the paged-KV block allocation (a seeded permutation of the
    physical blocks) and the token -> slot mapping.
  * §4.3 "Consistent mode switching": orchestrator.py holds the group-wide
    choice between WaS and CaS from the engines' active sequences, B_th and
    hysteresis.

The per-op equations (RMSNorm, rotate-half RoPE, grouped-query attention,
SwiGLU, per-head QK RMSNorm, QKV bias) are not printed in the paper; they are
the public definitions of the model families it evaluates (§5.1: Qwen3-32B,
Qwen2.5-72B, Llama-3.1-70B). The tests pin them against library routines
(torch.nn.functional, transformers' decoder layers) and closed forms.

Arithmetic is float64. With round_bf16=True the oracle rounds to bfloat16
exactly where a bf16 model stores a tensor (normed activations, projection
outputs, rotated q/k and the cached v, attention output, SwiGLU output); the
residual stream is never rounded. With round_bf16=False nothing but the inputs
is bf16.
"""

from .decode import (  # noqa: F401
    bf16_bits_to_f64,
    round_to_bf16,
    f64_to_bf16_bits,
    rms_norm,
    rope_rotate_half,
    silu,
    linear,
    swiglu,
    ffn,
    cas_ffn,
    paged_gqa_attention,
    decode_layer,
    decode_stack,
)
from .kvalloc import splitmix64_stream, fisher_yates, allocate_block_tables, slot_of  # noqa: F401
from .schedule import was_schedule, owned, streamed_layer, peak_shift_order  # noqa: F401
