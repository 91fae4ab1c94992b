"""Seeded random inputs. Every tensor draws from its own torch generator,
seeded from (seed, layer, tensor id), so any one layer or tensor can be
regenerated alone, on the device that will consume it.

Values are plain random draws; nothing here computes a step of the method.
"""

import numpy as np
import torch

from .configs import WEIGHT_STD, qkv_out

_TENSOR_IDS = {
    "w_q": 1, "w_k": 2, "w_v": 3, "w_o": 4, "w_gate": 5, "w_up": 6, "w_down": 7,
    "b_q": 8, "b_k": 9, "b_v": 10, "g_attn": 11, "g_mlp": 12, "g_q": 13, "g_k": 14,
    "hidden": 20, "kv_k": 21, "kv_v": 22,
}


def seed_for(seed, layer, tensor):
    """A stable 63-bit seed for one tensor."""
    tid = _TENSOR_IDS[tensor] if isinstance(tensor, str) else int(tensor)
    h = (int(seed) * 1_000_003 + int(layer) * 10_007 + tid * 101 + 12_345) & ((1 << 63) - 1)
    return h


def _gen(device, seed):
    g = torch.Generator(device=device)
    g.manual_seed(seed)
    return g


def _randn(shape, device, seed, std=1.0, dtype=torch.bfloat16):
    g = _gen(device, seed)
    t = torch.randn(shape, generator=g, device=device, dtype=torch.float32)
    if std != 1.0:
        t.mul_(std)
    return t.to(dtype)


def context_lengths(cfg, seed=0, batch=None):
    """Per-sequence cached-token counts, uniform integers in [ctx_lo, ctx_hi]."""
    b = cfg["batch"] if batch is None else batch
    rng = np.random.default_rng([int(seed), 7_777])
    return rng.integers(cfg["ctx_lo"], cfg["ctx_hi"] + 1, size=b, dtype=np.int64).astype(np.int32)


def hidden_input(cfg, seed=0, device="cpu", batch=None):
    """Residual-stream input x, float32 [B, H], N(0, 1)."""
    b = cfg["batch"] if batch is None else batch
    return _randn((b, cfg["hidden"]), device, seed_for(seed, 0, "hidden"), dtype=torch.float32)


def layer_weights(cfg, layer, seed=0, device="cpu", gains="one"):
    """One layer's bf16 weights in nn.Linear layout [out, in].

    gains: "one" -> every norm gain 1.0; "random" -> 1 + N(0, 0.1), so that a
    parity test also exercises gain indexing.
    """
    H, D, F = cfg["hidden"], cfg["head_dim"], cfg["ffn_dim"]
    Hq, Hkv = cfg["num_q_heads"], cfg["num_kv_heads"]
    s = lambda name: seed_for(seed, layer, name)  # noqa: E731
    w = {
        "w_q": _randn((Hq * D, H), device, s("w_q"), WEIGHT_STD),
        "w_k": _randn((Hkv * D, H), device, s("w_k"), WEIGHT_STD),
        "w_v": _randn((Hkv * D, H), device, s("w_v"), WEIGHT_STD),
        "w_o": _randn((H, Hq * D), device, s("w_o"), WEIGHT_STD),
        "w_gate": _randn((F, H), device, s("w_gate"), WEIGHT_STD),
        "w_up": _randn((F, H), device, s("w_up"), WEIGHT_STD),
        "w_down": _randn((H, F), device, s("w_down"), WEIGHT_STD),
    }
    if cfg["qkv_bias"]:
        w["b_q"] = _randn((Hq * D,), device, s("b_q"), WEIGHT_STD)
        w["b_k"] = _randn((Hkv * D,), device, s("b_k"), WEIGHT_STD)
        w["b_v"] = _randn((Hkv * D,), device, s("b_v"), WEIGHT_STD)

    def gain(n, name):
        if gains == "one":
            return torch.ones((n,), device=device, dtype=torch.bfloat16)
        return (1.0 + _randn((n,), device, s(name), 0.1, torch.float32)).to(torch.bfloat16)

    w["g_attn"] = gain(H, "g_attn")
    w["g_mlp"] = gain(H, "g_mlp")
    if cfg["qk_norm"]:
        w["g_q"] = gain(D, "g_q")
        w["g_k"] = gain(D, "g_k")
    assert w["w_q"].shape[0] + 2 * w["w_k"].shape[0] == qkv_out(cfg)
    return w


def kv_prefill(cfg, num_phys_blocks, region=0, seed=0, device="cpu"):
    """Cached keys and values of one KV region, bf16, N(0, 1), in the
    token-major block layout [num_phys_blocks, Hkv, block_size, D] for both."""
    shape = (num_phys_blocks, cfg["num_kv_heads"], cfg["block_size"], cfg["head_dim"])
    k = _randn(shape, device, seed_for(seed, 10_000 + region, "kv_k"))
    v = _randn(shape, device, seed_for(seed, 10_000 + region, "kv_v"))
    return k, v
