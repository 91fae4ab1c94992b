"""Workload table: model shapes, batch, context-length ranges.

Each entry names a workload by what it is. Model shapes are the public
architectures of the models evaluated in the paper (§5.1); the context
ranges stand in for its three workload lengths (§5.1 "Workload").

Per-layer knobs that the paper does not state (norm epsilon, RoPE base,
gains) take the values of the public model families:
  * Llama-3.1-style: RMSNorm eps 1e-5, RoPE base 500000 (tiny case: 10000).
  * Qwen-style: RMSNorm eps 1e-6, RoPE base 1e6; Qwen2.5 has a QKV bias,
    Qwen3 has a per-head RMSNorm on q and k (eps 1e-6).
RoPE is applied without frequency scaling.
"""

CONFIGS = {
    # Tiny single decoder layer: fits the oracle in milliseconds.
    "tiny_layer": dict(
        num_layers=1, hidden=256, num_q_heads=4, num_kv_heads=2, head_dim=64,
        ffn_dim=688, qkv_bias=0, qk_norm=0, rms_eps=1e-5, qk_norm_eps=1e-6,
        rope_theta=10000.0, block_size=16,
        batch=8, ctx_lo=16, ctx_hi=64, num_phys_blocks=64, kv_regions=1,
    ),
    # Qwen3-32B-shaped single layer, average context ~1K.
    "qwen3_32b_layer": dict(
        num_layers=1, hidden=5120, num_q_heads=64, num_kv_heads=8, head_dim=128,
        ffn_dim=25600, qkv_bias=0, qk_norm=1, rms_eps=1e-6, qk_norm_eps=1e-6,
        rope_theta=1e6, block_size=16,
        batch=256, ctx_lo=512, ctx_hi=2048, num_phys_blocks=None, kv_regions=1,
    ),
    # Llama-3.1-70B-shaped single layer, average context ~2.5K.
    "llama70b_layer": dict(
        num_layers=1, hidden=8192, num_q_heads=64, num_kv_heads=8, head_dim=128,
        ffn_dim=28672, qkv_bias=0, qk_norm=0, rms_eps=1e-5, qk_norm_eps=1e-6,
        rope_theta=500000.0, block_size=16,
        batch=256, ctx_lo=1024, ctx_hi=4096, num_phys_blocks=None, kv_regions=1,
    ),
    # Qwen2.5-72B-shaped stack of 8 layers streamed through a 2-slot cache.
    "qwen25_72b_stack8": dict(
        num_layers=8, hidden=8192, num_q_heads=64, num_kv_heads=8, head_dim=128,
        ffn_dim=29568, qkv_bias=1, qk_norm=0, rms_eps=1e-6, qk_norm_eps=1e-6,
        rope_theta=1e6, block_size=16,
        batch=256, ctx_lo=512, ctx_hi=4096, num_phys_blocks=None, kv_regions=8,
    ),
    # Llama-3.1-70B-shaped full 80-layer stack streamed through a 2-slot
    # cache; the KV cache fills the HBM left after the weight pool, so
    # layers share KV regions (layer l uses region l mod R).
    "llama70b_stack80": dict(
        num_layers=80, hidden=8192, num_q_heads=64, num_kv_heads=8, head_dim=128,
        ffn_dim=28672, qkv_bias=0, qk_norm=0, rms_eps=1e-5, qk_norm_eps=1e-6,
        rope_theta=500000.0, block_size=16,
        batch=256, ctx_lo=1024, ctx_hi=8192, num_phys_blocks=None, kv_regions=None,
    ),
}

WEIGHT_STD = 0.02


def get_config(name, **overrides):
    if name not in CONFIGS:
        raise KeyError(f"unknown workload {name!r}; known: {sorted(CONFIGS)}")
    cfg = dict(CONFIGS[name])
    cfg["name"] = name
    cfg.update(overrides)
    return cfg


def qkv_out(cfg):
    """Rows of the fused QKV weight: (Hq + 2 Hkv) * D."""
    return (cfg["num_q_heads"] + 2 * cfg["num_kv_heads"]) * cfg["head_dim"]


def layer_param_count(cfg):
    """Projection parameters of one layer (QKV, O, gate, up, down)."""
    H, D, F = cfg["hidden"], cfg["head_dim"], cfg["ffn_dim"]
    return H * qkv_out(cfg) + cfg["num_q_heads"] * D * H + 3 * H * F
