"""The decode step of a dense decoder layer stack, written out plainly in
float64 numpy. Test infrastructure only (see the package docstring).

Readings of points the paper leaves open:
  * RMSNorm: y = x / sqrt(mean(x^2) + eps) * g, eps inside the root, mean over
    the hidden dimension, the gain applied before any rounding.
  * RoPE: rotate-half pairing (i, i + D/2), theta_i = base^(-2i/D), applied at
    position p = number of tokens already cached; no frequency scaling.
  * A sequence with ctx cached tokens writes its new k, v at position ctx and
    then attends over ctx + 1 keys (the cached ones and its own).
  * Grouped-query attention: query head h reads KV head h // (Hq / Hkv);
    scale 1/sqrt(D); softmax with max subtraction; no masking extras.
  * Per-head QK RMSNorm (Qwen3 family): after the projection and bias, before
    RoPE, over the head dimension; the normed, rotated k is what is cached.
  * SwiGLU: a = silu(h W_gate^T) * (h W_up^T), silu(z) = z / (1 + e^-z).
  * Keys are cached after RoPE and never rotated again.
"""

import numpy as np


# --------------------------------------------------------------------------
# bfloat16 storage
# --------------------------------------------------------------------------

def bf16_bits_to_f64(bits):
    """bfloat16 bit patterns (uint16) -> float64, exactly."""
    b = np.ascontiguousarray(np.asarray(bits, dtype=np.uint16))
    with np.errstate(invalid="ignore"):
        return (b.astype(np.uint32) << np.uint32(16)).view(np.float32).astype(np.float64)


def f64_to_bf16_bits(x):
    """float64 -> bfloat16 bit patterns, round to nearest even (through float32)."""
    f = np.ascontiguousarray(np.asarray(x, dtype=np.float64).astype(np.float32))
    u = f.view(np.uint32)
    with np.errstate(over="ignore"):
        r = (u + np.uint32(0x7FFF) + ((u >> np.uint32(16)) & np.uint32(1))) >> np.uint32(16)
    r = np.where(np.isnan(f), np.uint32(0x7FC0), r)
    return r.astype(np.uint16)


def round_to_bf16(x):
    """float64 -> the nearest bfloat16 value, as float64."""
    return bf16_bits_to_f64(f64_to_bf16_bits(x))


# --------------------------------------------------------------------------
# Per-op definitions
# --------------------------------------------------------------------------

def rms_norm(x, g, eps):
    """RMSNorm over the last axis: x / sqrt(mean(x^2) + eps) * g."""
    x = np.asarray(x, dtype=np.float64)
    ms = np.mean(x * x, axis=-1, keepdims=True)
    return x / np.sqrt(ms + eps) * g


def rope_rotate_half(x, pos, theta):
    """Rotary position embedding, rotate-half convention.

    x: (..., D) with the position axis given by `pos` broadcastable to x[..., 0].
    For i < D/2 the pair (x_i, x_{i+D/2}) is rotated by the angle pos * theta_i,
    theta_i = theta^(-2i/D), angles in float64.
    """
    x = np.asarray(x, dtype=np.float64)
    D = x.shape[-1]
    half = D // 2
    i = np.arange(half, dtype=np.float64)
    inv_freq = theta ** (-2.0 * i / D)
    ang = np.asarray(pos, dtype=np.float64)[..., None] * inv_freq
    c, s = np.cos(ang), np.sin(ang)
    a, b = x[..., :half], x[..., half:]
    return np.concatenate([a * c - b * s, b * c + a * s], axis=-1)


def silu(z):
    """SiLU: z / (1 + exp(-z))."""
    z = np.asarray(z, dtype=np.float64)
    with np.errstate(over="ignore"):
        return z / (1.0 + np.exp(-z))


def linear(x, w, b=None):
    """Dense projection in nn.Linear layout: x W^T (+ b)."""
    y = np.asarray(x, dtype=np.float64) @ np.asarray(w, dtype=np.float64).T
    return y if b is None else y + b


def swiglu(h, w_gate, w_up):
    """SwiGLU FFN input: silu(h W_gate^T) * (h W_up^T)."""
    return silu(linear(h, w_gate)) * linear(h, w_up)


def ffn(h, w_gate, w_up, w_down, round_bf16=False):
    """The FFN of a decoder layer on already normed rows h: down(SwiGLU(h)),
    with the SwiGLU output rounded to bf16 where a bf16 model stores it."""
    a = swiglu(h, w_gate, w_up)
    if round_bf16:
        a = round_to_bf16(a)
    return linear(a, w_down)


def cas_ffn(inputs, w_gate, w_up, w_down, round_bf16=False):
    """Compute-as-a-Service at a layer's owner (§4.3): the rows of all replicas
    that are not running a dummy iteration are stacked into one batch, the
    FFN runs once over it, and the output is cut back at the same row
    boundaries. inputs: per replica an (rows, H) array, or None for a dummy
    replica. Returns the per-replica outputs (None for dummies)."""
    live = [x for x in inputs if x is not None and len(x) > 0]
    if not live:
        return [None for _ in inputs]
    y = ffn(np.concatenate(live, axis=0), w_gate, w_up, w_down, round_bf16)
    out, o = [], 0
    for x in inputs:
        if x is None or len(x) == 0:
            out.append(None)
            continue
        out.append(y[o:o + len(x)])
        o += len(x)
    return out


def paged_gqa_attention(q, k_cache, v_cache, block_table, seq_len, block_size):
    """Decode attention of one sequence over its paged KV.

    q: (Hq, D) float64. k_cache, v_cache: (num_blocks, Hkv, block_size, D).
    block_table: logical block j -> physical block. Token t lives in physical
    block block_table[t // block_size] at offset t % block_size.
    Returns (Hq, D): for each head, softmax(q K^T / sqrt(D)) V over tokens
    0..seq_len-1 of its KV head.
    """
    Hq, D = q.shape
    Hkv = k_cache.shape[1]
    group = Hq // Hkv
    t = np.arange(seq_len)
    blocks = np.asarray(block_table)[t // block_size]
    if np.any(blocks < 0):
        raise ValueError("a token of the sequence lies in an unallocated block")
    offs = t % block_size
    K = k_cache[blocks, :, offs, :]  # (seq, Hkv, D)
    V = v_cache[blocks, :, offs, :]
    out = np.empty((Hq, D), dtype=np.float64)
    for h in range(Hq):
        g = h // group
        s = K[:, g, :] @ q[h] / np.sqrt(D)
        s = s - np.max(s)
        p = np.exp(s)
        p = p / np.sum(p)
        out[h] = p @ V[:, g, :]
    return out


# --------------------------------------------------------------------------
# One decoder layer, one decode iteration
# --------------------------------------------------------------------------

def _w(lw, name):
    """Weight as float64 (accepts bf16 bit patterns or float arrays)."""
    a = lw[name]
    if a.dtype == np.uint16:
        return bf16_bits_to_f64(a)
    return np.asarray(a, dtype=np.float64)


def decode_layer(x, lw, cfg, k_cache, v_cache, positions, block_tables, round_bf16=True):
    """One layer of one decode iteration for a batch of sequences.

    x: (B, H) float64 residual stream (one new token per sequence).
    lw: the layer's weights, nn.Linear layout [out, in] (bf16 bits or floats).
    cfg: mapping with hidden, num_q_heads, num_kv_heads, head_dim, ffn_dim,
         qkv_bias, qk_norm, rms_eps, qk_norm_eps, rope_theta, block_size.
    k_cache, v_cache: this layer's KV region, (num_blocks, Hkv, bs, D) float64;
         the new token's k and v are written into them (in place).
    positions: (B,) cached-token counts; the new token sits at that position.
    block_tables: (B, max_blocks) logical -> physical blocks (-1 = unused).
    Returns the layer's output residual stream (B, H).
    """
    rb = round_to_bf16 if round_bf16 else (lambda t: t)
    x = np.asarray(x, dtype=np.float64)
    B = x.shape[0]
    Hq, Hkv, D = cfg["num_q_heads"], cfg["num_kv_heads"], cfg["head_dim"]
    bs = cfg["block_size"]

    # Self-attention sub-block.
    h = rb(rms_norm(x, _w(lw, "g_attn"), cfg["rms_eps"]))
    bias = cfg["qkv_bias"]
    q = linear(h, _w(lw, "w_q"), _w(lw, "b_q") if bias else None)
    k = linear(h, _w(lw, "w_k"), _w(lw, "b_k") if bias else None)
    v = linear(h, _w(lw, "w_v"), _w(lw, "b_v") if bias else None)
    q, k, v = rb(q), rb(k), rb(v)
    q = q.reshape(B, Hq, D)
    k = k.reshape(B, Hkv, D)
    v = v.reshape(B, Hkv, D)
    if cfg["qk_norm"]:
        q = rms_norm(q, _w(lw, "g_q"), cfg["qk_norm_eps"])
        k = rms_norm(k, _w(lw, "g_k"), cfg["qk_norm_eps"])
    pos = np.asarray(positions, dtype=np.int64)
    q = rb(rope_rotate_half(q, pos[:, None], cfg["rope_theta"]))
    k = rb(rope_rotate_half(k, pos[:, None], cfg["rope_theta"]))

    # Append the new token's key and value to each sequence's paged cache.
    for b in range(B):
        p = int(pos[b])
        blk = int(block_tables[b][p // bs])
        if blk < 0:
            raise ValueError(f"sequence {b}: no block allocated for position {p}")
        k_cache[blk, :, p % bs, :] = k[b]
        v_cache[blk, :, p % bs, :] = v[b]

    o = np.empty((B, Hq, D), dtype=np.float64)
    for b in range(B):
        o[b] = paged_gqa_attention(q[b], k_cache, v_cache, block_tables[b], int(pos[b]) + 1, bs)
    o = rb(o.reshape(B, Hq * D))
    x1 = x + linear(o, _w(lw, "w_o"))

    # FFN sub-block.
    h2 = rb(rms_norm(x1, _w(lw, "g_mlp"), cfg["rms_eps"]))
    a = rb(swiglu(h2, _w(lw, "w_gate"), _w(lw, "w_up")))
    return x1 + linear(a, _w(lw, "w_down"))


def decode_stack(x, layers, cfg, k_regions, v_regions, positions, block_tables, round_bf16=True):
    """L layers of one decode iteration. Layer l reads and writes KV region
    l mod R, R = len(k_regions). layers: sequence of per-layer weight mappings,
    or a callable layer_index -> mapping (so weights can be produced one
    layer at a time)."""
    L = cfg["num_layers"]
    R = len(k_regions)
    get = layers if callable(layers) else (lambda l: layers[l])
    for l in range(L):
        x = decode_layer(x, get(l), cfg, k_regions[l % R], v_regions[l % R],
                         positions, block_tables, round_bf16)
    return x
