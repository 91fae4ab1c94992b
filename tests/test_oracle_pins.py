"""Pins of the oracle against things other than itself: published test
vectors, library routines, closed forms, invariants and brute force. CPU only.

A plausible mistake anywhere in the oracle (a dropped term, a wrong sign or
index, a transposed operand) should fail at least one of these.
"""

import math
import os

import numpy as np
import pytest
import torch
import torch.nn.functional as F

import oracle
from oracle import decode as od
from oracle import kvalloc as ka
from oracle.schedule import was_schedule, streamed_layer
import synth

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


# ---------------------------------------------------------------- bf16 storage

def test_bf16_roundtrip_and_rne():
    # Every bf16 pattern survives bits -> f64 -> bits (finite and inf).
    bits = np.arange(0, 1 << 16, dtype=np.uint32).astype(np.uint16)
    vals = od.bf16_bits_to_f64(bits)
    finite = ~np.isnan(vals)
    assert np.array_equal(od.f64_to_bf16_bits(vals[finite]), bits[finite])
    # torch's own float32 -> bfloat16 conversion (round to nearest even) as the reference.
    x = np.random.default_rng(0).standard_normal(100_000).astype(np.float32) * 37.0
    x = np.concatenate([x, np.float32([1.0 + 2 ** -8, 1.0 + 3 * 2 ** -8, -1.0 - 2 ** -8, 65504.0, 3.0e38])])
    ref = torch.from_numpy(x).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    assert np.array_equal(od.f64_to_bf16_bits(x.astype(np.float64)), ref)


# ---------------------------------------------------------------- per-op pins

def test_rms_norm_matches_torch_library():
    rng = np.random.default_rng(1)
    x = rng.standard_normal((5, 96)) * 3.0
    g = 1.0 + 0.1 * rng.standard_normal(96)
    ref = F.rms_norm(torch.from_numpy(x), (96,), torch.from_numpy(g), eps=1e-5).numpy()
    np.testing.assert_allclose(od.rms_norm(x, g, 1e-5), ref, rtol=1e-13, atol=1e-13)


def test_rms_norm_closed_form_constant_vector():
    c, eps = 0.37, 1e-6
    y = od.rms_norm(np.full((1, 64), c), np.full(64, 2.0), eps)
    np.testing.assert_allclose(y, 2.0 * c / math.sqrt(c * c + eps), rtol=1e-15)


def test_silu_matches_torch_library():
    z = np.linspace(-30, 30, 2001)
    np.testing.assert_allclose(od.silu(z), F.silu(torch.from_numpy(z)).numpy(), rtol=1e-14, atol=1e-300)


def _rope_complex(x, pos, theta):
    """RoPE as complex multiplication: (x_i + i x_{i+D/2}) * exp(i pos theta_i)."""
    D = x.shape[-1]
    half = D // 2
    z = x[..., :half] + 1j * x[..., half:]
    freqs = theta ** (-np.arange(0, D, 2) / D)
    z = z * np.exp(1j * pos * freqs)
    return np.concatenate([z.real, z.imag], axis=-1)


def test_rope_matches_complex_rotation():
    rng = np.random.default_rng(2)
    x = rng.standard_normal((3, 128))
    for pos in (0, 1, 17, 4095, 8192):
        np.testing.assert_allclose(od.rope_rotate_half(x, np.full(3, pos), 500000.0),
                                   _rope_complex(x, pos, 500000.0), rtol=1e-12, atol=1e-12)


def test_rope_identity_norm_and_relative_position():
    rng = np.random.default_rng(3)
    q, k = rng.standard_normal(64), rng.standard_normal(64)
    np.testing.assert_array_equal(od.rope_rotate_half(q[None], np.array([0]), 1e4)[0], q)
    r = od.rope_rotate_half(q[None], np.array([123]), 1e4)[0]
    # pairwise norms preserved
    np.testing.assert_allclose(r[:32] ** 2 + r[32:] ** 2, q[:32] ** 2 + q[32:] ** 2, rtol=1e-12)
    # q_m . k_n depends only on m - n
    dots = [od.rope_rotate_half(q[None], np.array([m]), 1e4)[0] @ od.rope_rotate_half(k[None], np.array([m - 5]), 1e4)[0]
            for m in (5, 40, 300)]
    np.testing.assert_allclose(dots, dots[0], rtol=1e-11)


def _paged_case(rng, Hq=8, Hkv=2, D=32, bs=16, nblk=12, seq=37):
    k_cache = rng.standard_normal((nblk, Hkv, bs, D))
    v_cache = rng.standard_normal((nblk, Hkv, bs, D))
    table = rng.permutation(nblk)[: -(-seq // bs)]
    q = rng.standard_normal((Hq, D))
    return q, k_cache, v_cache, table


def _gather(cache, table, seq, bs):
    t = np.arange(seq)
    return cache[np.asarray(table)[t // bs], :, t % bs, :]  # (seq, Hkv, D)


def test_attention_matches_torch_sdpa():
    rng = np.random.default_rng(4)
    for seq in (1, 15, 16, 17, 37):
        q, kc, vc, tab = _paged_case(rng, seq=seq)
        out = od.paged_gqa_attention(q, kc, vc, tab, seq, 16)
        K = torch.from_numpy(_gather(kc, tab, seq, 16)).permute(1, 0, 2)  # (Hkv, seq, D)
        V = torch.from_numpy(_gather(vc, tab, seq, 16)).permute(1, 0, 2)
        ref = F.scaled_dot_product_attention(torch.from_numpy(q)[:, None, :], K.repeat_interleave(4, 0),
                                             V.repeat_interleave(4, 0))[:, 0, :].numpy()
        np.testing.assert_allclose(out, ref, rtol=1e-12, atol=1e-12)


def test_attention_closed_forms():
    rng = np.random.default_rng(5)
    q, kc, vc, tab = _paged_case(rng, seq=1)
    out = od.paged_gqa_attention(q, kc, vc, tab, 1, 16)
    # one cached token: every head returns that token's V row of its group
    for h in range(8):
        np.testing.assert_array_equal(out[h], vc[tab[0], h // 4, 0, :])
    # all-equal keys: the mean of V
    q, kc, vc, tab = _paged_case(rng, seq=29)
    kc[:] = rng.standard_normal(32)
    out = od.paged_gqa_attention(q, kc, vc, tab, 29, 16)
    Vg = _gather(vc, tab, 29, 16)
    for h in range(8):
        np.testing.assert_allclose(out[h], Vg[:, h // 4, :].mean(axis=0), rtol=1e-12, atol=1e-14)


def test_attention_softmax_rows_sum_to_one():
    # V = 1 everywhere -> output is the row sum of the softmax, i.e. 1
    rng = np.random.default_rng(6)
    q, kc, vc, tab = _paged_case(rng, seq=40)
    q *= 10.0
    out = od.paged_gqa_attention(q, kc, np.ones_like(vc), tab, 40, 16)
    np.testing.assert_allclose(out, 1.0, rtol=1e-12)


def test_attention_physical_block_permutation_invariance():
    rng = np.random.default_rng(7)
    q, kc, vc, tab = _paged_case(rng, seq=45, nblk=10)
    out1 = od.paged_gqa_attention(q, kc, vc, tab, 45, 16)
    perm = rng.permutation(10)  # move every physical block elsewhere
    kc2, vc2 = np.empty_like(kc), np.empty_like(vc)
    kc2[perm], vc2[perm] = kc, vc
    out2 = od.paged_gqa_attention(q, kc2, vc2, perm[tab], 45, 16)
    np.testing.assert_array_equal(out1, out2)


# ---------------------------------------------------------------- block tables

def _golden_splitmix():
    rows = {}
    with open(os.path.join(GOLDEN, "splitmix64_vectors.txt")) as f:
        for line in f:
            line = line.strip()
            if not line or line.startswith("#"):
                continue
            seed, vals = line.split(":")
            rows[int(seed)] = [int(v) for v in vals.split()]
    return rows


def test_splitmix64_published_vectors():
    for seed, vals in _golden_splitmix().items():
        assert ka.splitmix64_stream(seed, len(vals)) == vals


def test_fisher_yates_is_uniform_permutation():
    # Durstenfeld's rule j = r mod (i+1) reaches every permutation; the
    # off-by-one j = r mod i (Sattolo) would only reach the 2 cyclic ones of 3.
    seen = {}
    for seed in range(3000):
        p = tuple(ka.fisher_yates(3, seed))
        seen[p] = seen.get(p, 0) + 1
    assert len(seen) == 6
    counts = np.array(list(seen.values()))
    chi2 = ((counts - 500.0) ** 2 / 500.0).sum()
    assert chi2 < 20.5  # 5 dof, p ~ 0.001
    for n in (1, 2, 64, 1000):
        assert sorted(ka.fisher_yates(n, 11)) == list(range(n))


def test_block_tables_properties():
    ctx = [16, 17, 0, 63, 64, 31]
    tabs = ka.allocate_block_tables(ctx, 1, 64, 6, seed=3)
    used = []
    for c, row in zip(ctx, tabs):
        need = -(-(c + 1) // 16)
        assert all(b >= 0 for b in row[:need]) and all(b == -1 for b in row[need:])
        used += row[:need]
    assert len(used) == len(set(used)) and all(0 <= b < 64 for b in used)
    # the blocks are handed out in permutation order
    assert used == ka.fisher_yates(64, 3)[:len(used)]
    # exhaustion and table-width overflow are refused
    assert ka.allocate_block_tables([500], 1, 16, 64, seed=0) is None
    assert ka.allocate_block_tables([100], 1, 64, 4, seed=0) is None


def test_slot_mapping_brute_force():
    # Enumerate every token of every sequence; slots must be distinct and
    # land in the block the table names, at the token's offset.
    ctx = [5, 33, 48]
    tabs = ka.allocate_block_tables(ctx, 1, 20, 4, seed=9)
    slots = set()
    for c, row in zip(ctx, tabs):
        for p in range(c + 1):
            s = ka.slot_of(row, p)
            assert s // 16 == row[p // 16] and s % 16 == p % 16
            slots.add(s)
    assert len(slots) == sum(c + 1 for c in ctx)


def test_ffn_matches_transformers_mlp():
    """The oracle's FFN against transformers' LlamaMLP (SiLU-gated) in float64."""
    from transformers import LlamaConfig
    from transformers.models.llama.modeling_llama import LlamaMLP
    H, F = 48, 80
    g = torch.Generator().manual_seed(5)
    hc = LlamaConfig(hidden_size=H, intermediate_size=F, hidden_act="silu", num_attention_heads=4,
                     num_key_value_heads=4)
    mlp = LlamaMLP(hc).to(torch.float64)
    with torch.no_grad():
        for lin in (mlp.gate_proj, mlp.up_proj, mlp.down_proj):
            lin.weight.copy_(torch.randn(lin.weight.shape, generator=g, dtype=torch.float64) * 0.1)
        x = torch.randn(7, H, generator=g, dtype=torch.float64)
        want = mlp(x).numpy()
    got = oracle.ffn(x.numpy(), mlp.gate_proj.weight.detach().numpy(), mlp.up_proj.weight.detach().numpy(),
                     mlp.down_proj.weight.detach().numpy())
    np.testing.assert_allclose(got, want, rtol=1e-12, atol=1e-12)


def test_ffn_bf16_rounding_point():
    """In bf16 mode the SwiGLU output is rounded before the down projection: the
    result differs from the exact one, by at most the round-to-nearest bound
    (half a bf16 ulp, 2^-9 relative, on every term), and the decode layer's FFN
    (attention projections zeroed) is exactly this FFN of its normed input."""
    cfg = synth.get_config("tiny_layer")
    w, lw, ctx, tabs, kc, vc, x = _tiny_inputs(cfg)
    wg, wu, wd = (od.bf16_bits_to_f64(lw[k]) for k in ("w_gate", "w_up", "w_down"))
    h = od.round_to_bf16(od.rms_norm(x, od.bf16_bits_to_f64(lw["g_mlp"]), cfg["rms_eps"]))
    yr = oracle.ffn(h, wg, wu, wd, round_bf16=True)
    ye = oracle.ffn(h, wg, wu, wd, round_bf16=False)
    a = od.swiglu(h, wg, wu)
    bound = 2.0 ** -9 * (np.abs(a) @ np.abs(wd).T)
    assert np.any(yr != ye)
    assert np.all(np.abs(yr - ye) <= bound * (1 + 1e-12))
    lz = dict(lw)
    lz["w_o"] = np.zeros_like(lw["w_o"])
    x2 = od.decode_layer(x, lz, cfg, kc.copy(), vc.copy(), ctx, tabs, round_bf16=True)
    np.testing.assert_allclose(x2 - x, yr, rtol=1e-12, atol=1e-12)


def test_cas_ffn_is_per_replica_ffn():
    """CaS fuses the replicas' rows into one FFN call and cuts the output back:
    every live replica gets exactly its own rows' FFN, in order, and dummy
    replicas get nothing (§4.3, numerically equivalent to computing locally)."""
    rng = np.random.default_rng(2)
    H, F = 16, 24
    wg, wu, wd = rng.normal(size=(F, H)), rng.normal(size=(F, H)), rng.normal(size=(H, F))
    xs = [rng.normal(size=(3, H)), None, rng.normal(size=(1, H)), np.zeros((0, H)), rng.normal(size=(5, H))]
    ys = oracle.cas_ffn(xs, wg, wu, wd)
    assert ys[1] is None and ys[3] is None
    for x, y in zip(xs, ys):
        if y is not None:
            assert y.shape == x.shape
            np.testing.assert_allclose(y, oracle.ffn(x, wg, wu, wd), rtol=1e-13, atol=1e-12)
    assert oracle.cas_ffn([None, None], wg, wu, wd) == [None, None]


# ---------------------------------------------------------------- schedule

def test_was_schedule_ordering():
    """Properties the paper's buffer management requires, checked on the
    issue order: every layer is fully read into its slot before compute on it
    starts, a slot is refilled only after its previous layer released it, at
    most two layers occupy the cache, and the lookahead is one layer."""
    L, steps = 5, 3
    ops = was_schedule(L, steps)
    total = L * steps
    pos = {op: i for i, op in enumerate(ops)}
    assert len(pos) == len(ops)  # no duplicates
    for g in range(total):
        s = g % 2
        # compute on layer g: wait for its fill, then both halves, then release
        seq = [pos[(k, g, s)] for k in ("wait_fill", "attn", "mid", "proj", "done")]
        assert seq == sorted(seq)
        # both tiles of layer g were issued before the wait on them
        assert pos[("fill_a", g, s)] < pos[("fill_b", g, s)] < pos[("wait_fill", g, s)]
        if g >= 1:
            # tile A of layer g + 1 waits for layer g - 1 (same slot) to be released
            assert pos[("done", g - 1, (g + 1) % 2)] < pos[("wait_done", g - 1, (g + 1) % 2)]
            assert pos[("wait_done", g - 1, (g + 1) % 2)] < pos[("fill_a", g + 1, (g + 1) % 2)]
        # tile B of layer g + 1 follows layer g's attention half
        assert pos[("mid", g, s)] < pos[("wait_mid", g, s)] < pos[("fill_b", g + 1, (g + 1) % 2)]
        # lookahead of one layer: layer g + 2 is not read before layer g is released
        if ("fill_a", g + 2, s) in pos:
            assert pos[("done", g, s)] < pos[("fill_a", g + 2, s)]
    # fills are issued for every layer, plus one ahead into the next iteration
    assert [g for (k, g, s) in ops if k == "fill_a"] == list(range(total + 1))
    assert was_schedule(L, 0) == []


def test_was_schedule_with_owned_layers():
    """With d pooling ranks, rank r computes the layers it owns (l mod d = r)
    straight from its pool and streams the rest through the ring: owned
    layers get no read and no slot, every other layer keeps the properties
    above, and layer order is kept."""
    L, steps, d, r = 7, 3, 3, 1
    ops = was_schedule(L, steps, d, r)
    assert was_schedule(L, steps) == was_schedule(L, steps, 0, 0)
    streamed = [l for l in range(L) if l % d != r]
    local = [n for (k, n, s) in ops if k == "local"]
    assert local == [t * L + l for t in range(steps) for l in range(L) if l % d == r]
    ring_only = [op for op in ops if op[0] != "local"]
    assert ring_only == was_schedule(len(streamed), steps)  # the ring sees the non-owned layers only
    # compute happens in layer order: each step's layers appear as l = 0 .. L-1
    order = []
    for k, n, s in ops:
        if k == "local":
            order.append(n % L)
        elif k == "attn":
            order.append(streamed_layer(n, L, d, r))
    assert order == [l for _ in range(steps) for l in range(L)]
    # owning every layer (d = 1) leaves no ring at all; owning none is the plain ring
    assert all(k == "local" for (k, n, s) in was_schedule(4, 2, 1, 0))
    assert was_schedule(4, 2, 5, 4) == was_schedule(4, 2)  # rank 4 of 5 owns none of 4 layers


# ---------------------------------------------------------------- whole layer

def _tiny_inputs(cfg, seed=0, gains="random"):
    w = synth.layer_weights(cfg, 0, seed=seed, gains=gains)
    lw = {k: v.view(torch.int16).numpy().view(np.uint16) for k, v in w.items()}
    ctx = synth.context_lengths(cfg, seed)
    tabs = np.array(ka.allocate_block_tables(ctx, 1, cfg["num_phys_blocks"], 5, seed))
    kb, vb = synth.kv_prefill(cfg, cfg["num_phys_blocks"], 0, seed)
    kc = od.bf16_bits_to_f64(kb.view(torch.int16).numpy().view(np.uint16))
    vc = od.bf16_bits_to_f64(vb.view(torch.int16).numpy().view(np.uint16))
    x = synth.hidden_input(cfg, seed).double().numpy()
    return w, lw, ctx, tabs, kc, vc, x


def _hf_layer(family, cfg, w):
    if family == "llama":
        from transformers import LlamaConfig as C
        from transformers.models.llama.modeling_llama import LlamaDecoderLayer as Layer, LlamaRotaryEmbedding as Rot
    elif family == "qwen2":
        from transformers import Qwen2Config as C
        from transformers.models.qwen2.modeling_qwen2 import Qwen2DecoderLayer as Layer, Qwen2RotaryEmbedding as Rot
    else:
        from transformers import Qwen3Config as C
        from transformers.models.qwen3.modeling_qwen3 import Qwen3DecoderLayer as Layer, Qwen3RotaryEmbedding as Rot
    hc = C(hidden_size=cfg["hidden"], intermediate_size=cfg["ffn_dim"], num_attention_heads=cfg["num_q_heads"],
           num_key_value_heads=cfg["num_kv_heads"], head_dim=cfg["head_dim"], rms_norm_eps=cfg["rms_eps"],
           rope_theta=cfg["rope_theta"], max_position_embeddings=8192, attn_implementation="eager",
           num_hidden_layers=1)
    layer = Layer(hc, layer_idx=0).to(torch.float64).eval()
    sd = lambda t: t.to(torch.float64)  # noqa: E731
    with torch.no_grad():
        a = layer.self_attn
        a.q_proj.weight.copy_(sd(w["w_q"]))
        a.k_proj.weight.copy_(sd(w["w_k"]))
        a.v_proj.weight.copy_(sd(w["w_v"]))
        a.o_proj.weight.copy_(sd(w["w_o"]))
        if family == "qwen2":
            a.q_proj.bias.copy_(sd(w["b_q"]))
            a.k_proj.bias.copy_(sd(w["b_k"]))
            a.v_proj.bias.copy_(sd(w["b_v"]))
        if family == "qwen3":
            a.q_norm.weight.copy_(sd(w["g_q"]))
            a.k_norm.weight.copy_(sd(w["g_k"]))
        layer.mlp.gate_proj.weight.copy_(sd(w["w_gate"]))
        layer.mlp.up_proj.weight.copy_(sd(w["w_up"]))
        layer.mlp.down_proj.weight.copy_(sd(w["w_down"]))
        layer.input_layernorm.weight.copy_(sd(w["g_attn"]))
        layer.post_attention_layernorm.weight.copy_(sd(w["g_mlp"]))
    return layer, Rot(hc).to(torch.float64)


@pytest.mark.parametrize("family", ["llama", "qwen2", "qwen3"])
def test_decode_layer_matches_transformers(family):
    """The whole layer against the public model-family implementation
    (transformers, float64, eager attention) driven through one decode step
    with a cache prefilled from the paged blocks."""
    from transformers import DynamicCache
    cfg = synth.get_config("tiny_layer", qkv_bias=int(family == "qwen2"), qk_norm=int(family == "qwen3"),
                           rms_eps=1e-5 if family == "llama" else 1e-6)
    w, lw, ctx, tabs, kc, vc, x = _tiny_inputs(cfg)
    kc0, vc0 = kc.copy(), vc.copy()
    out = od.decode_layer(x, lw, cfg, kc, vc, ctx, tabs, round_bf16=False)
    layer, rot = _hf_layer(family, cfg, w)
    for b in range(cfg["batch"]):
        c = int(ctx[b])
        K = torch.from_numpy(_gather(kc0, tabs[b], c, 16)).permute(1, 0, 2)[None]  # (1, Hkv, c, D)
        V = torch.from_numpy(_gather(vc0, tabs[b], c, 16)).permute(1, 0, 2)[None]
        cache = DynamicCache()
        cache.update(K.clone(), V.clone(), 0)
        hs = torch.from_numpy(x[b])[None, None]
        pid = torch.tensor([[c]])
        with torch.no_grad():
            y = layer(hs, attention_mask=None, position_ids=pid, past_key_values=cache, use_cache=True,
                      position_embeddings=rot(hs, pid))
        y = y[0] if isinstance(y, tuple) else y
        np.testing.assert_allclose(out[b], y[0, 0].numpy(), rtol=2e-5, atol=2e-5)
        # the cache row written for the new token equals what transformers appended
        k_new = kc[tabs[b][c // 16], :, c % 16, :]
        np.testing.assert_allclose(k_new, cache.layers[0].keys[0, :, c, :].numpy(), rtol=2e-5, atol=2e-5)


def test_decode_layer_zero_projections_keep_residual_and_write_kv():
    cfg = synth.get_config("tiny_layer")
    w, lw, ctx, tabs, kc, vc, x = _tiny_inputs(cfg)
    lw["w_o"] = np.zeros_like(lw["w_o"])
    lw["w_down"] = np.zeros_like(lw["w_down"])
    kc0 = kc.copy()
    cfg2 = dict(cfg, num_layers=3)
    out = od.decode_stack(x, [lw] * 3, cfg2, [kc], [vc], ctx, tabs)
    np.testing.assert_array_equal(out, x)
    changed = np.argwhere(np.any(kc != kc0, axis=(1, 3)))
    expect = {(int(tabs[b][c // 16]), int(c % 16)) for b, c in enumerate(ctx)}
    got = {(int(r[0]), int(r[2])) for r in np.argwhere(np.any(kc != kc0, axis=-1))}
    assert got == expect and len(changed) > 0


def test_decode_layer_rows_independent():
    cfg = synth.get_config("tiny_layer")
    w, lw, ctx, tabs, kc, vc, x = _tiny_inputs(cfg)
    full = od.decode_layer(x, lw, cfg, kc.copy(), vc.copy(), ctx, tabs)
    for b in (0, 5):
        one = od.decode_layer(x[b:b + 1], lw, cfg, kc.copy(), vc.copy(), ctx[b:b + 1], tabs[b:b + 1])
        np.testing.assert_array_equal(one[0], full[b])


def _bf(t):
    """torch float64 -> nearest bfloat16 (round to nearest even through float32,
    torch's own conversion), back as float64."""
    return t.to(torch.float32).to(torch.bfloat16).to(torch.float64)


def _attention_block_by_torch(x, lw, cfg, kc, vc, pos, tabs):
    """The attention sub-block of one decode step with bf16 storage at the
    model's storage points (normed input, projection outputs, rotated q and k,
    cached v, attention output), built from torch library routines in float64
    (rms_norm, matmul, complex-multiplication RoPE, scaled_dot_product_attention)
    and torch's bf16 conversion. Returns the new tokens' cached k and v
    (B, Hkv, D) and the attention output o (B, Hq * D)."""
    H, Hq, Hkv, D, bs = cfg["hidden"], cfg["num_q_heads"], cfg["num_kv_heads"], cfg["head_dim"], cfg["block_size"]
    w = {n: torch.from_numpy(od.bf16_bits_to_f64(a)) for n, a in lw.items()}
    xt = torch.from_numpy(x)
    B = xt.shape[0]
    h = _bf(F.rms_norm(xt, (H,), weight=w["g_attn"], eps=cfg["rms_eps"]))
    q = _bf(h @ w["w_q"].T).reshape(B, Hq, D)
    k = _bf(h @ w["w_k"].T).reshape(B, Hkv, D)
    v = _bf(h @ w["w_v"].T).reshape(B, Hkv, D)
    p = np.asarray(pos)[:, None, None]
    q = _bf(torch.from_numpy(_rope_complex(q.numpy(), p, cfg["rope_theta"])))
    k = _bf(torch.from_numpy(_rope_complex(k.numpy(), p, cfg["rope_theta"])))
    o = torch.empty(B, Hq, D, dtype=torch.float64)
    for b in range(B):
        c = int(pos[b])
        K = torch.cat([torch.from_numpy(_gather(kc, tabs[b], c, bs)), k[b][None]], 0).permute(1, 0, 2)  # (Hkv, c+1, D)
        V = torch.cat([torch.from_numpy(_gather(vc, tabs[b], c, bs)), v[b][None]], 0).permute(1, 0, 2)
        rep = Hq // Hkv
        o[b] = F.scaled_dot_product_attention(q[b][:, None], K.repeat_interleave(rep, 0).contiguous(),
                                              V.repeat_interleave(rep, 0).contiguous())[:, 0]
    return k.numpy(), v.numpy(), _bf(o.reshape(B, Hq * D)).numpy()


def _is_bf16(a):
    return np.array_equal(od.round_to_bf16(a), a)


def _pass_through_attention(lw, cfg):
    """W_o = identity (the attention output lands unchanged on the residual),
    W_down = 0 (the FFN adds nothing): x2 - x is the stored attention output."""
    lz = dict(lw)
    one = np.uint16(0x3F80)  # bf16 1.0
    lz["w_o"] = (np.eye(cfg["hidden"], cfg["num_q_heads"] * cfg["head_dim"]) * one).astype(np.uint16)
    lz["w_down"] = np.zeros_like(lw["w_down"])
    return lz


def test_attention_storage_points_exact_case():
    """Every token attends only to itself (empty contexts), so o equals the new v
    exactly; each v element sums two normed inputs with weight 1.0, so the
    float64 arithmetic is exact and the only roundings are the storage points.
    Rounding the normed input h first, then the sum, differs from rounding the
    sum once: the pin fails if h is not stored in bf16. The cached v must be
    bf16 (fails if the projection output is not rounded)."""
    cfg = synth.get_config("tiny_layer")
    w, lw, ctx, tabs, kc, vc, x = _tiny_inputs(cfg)
    H, KD = cfg["hidden"], cfg["num_kv_heads"] * cfg["head_dim"]
    wv = np.zeros((KD, H), np.uint16)
    j = np.arange(KD)
    wv[j, 2 * j] = wv[j, 2 * j + 1] = 0x3F80
    lz = _pass_through_attention(dict(lw, w_v=wv), cfg)
    pos = np.zeros(cfg["batch"], np.int64)
    tabs0 = np.array(ka.allocate_block_tables(pos, 1, cfg["num_phys_blocks"], 5, 0))
    kc1, vc1 = kc.copy(), vc.copy()
    out = od.decode_layer(x, lz, cfg, kc1, vc1, pos, tabs0, round_bf16=True)
    k_t, v_t, o_t = _attention_block_by_torch(x, lz, cfg, kc, vc, pos, tabs0)
    np.testing.assert_array_equal(out - x, o_t)
    for b in range(cfg["batch"]):
        blk = tabs0[b][0]
        np.testing.assert_array_equal(vc1[blk, :, 0, :], v_t[b])
        np.testing.assert_array_equal(kc1[blk, :, 0, :], k_t[b])
    # the case does tell the two orders of rounding apart
    h = F.rms_norm(torch.from_numpy(x), (H,), weight=torch.from_numpy(od.bf16_bits_to_f64(lw["g_attn"])),
                   eps=cfg["rms_eps"])
    once = _bf(h @ torch.from_numpy(od.bf16_bits_to_f64(wv)).T).numpy()
    assert np.mean(once != v_t.reshape(cfg["batch"], KD)) > 0.05


def test_attention_storage_points_cached_contexts():
    """Random weights, contexts 16..64: the new key and value written to the
    cache are bf16 numbers (fails if the rotated k or the projected v is left
    unrounded) and match the torch evaluation; the attention output matches it
    too (fails if the rotated q or the normed input is left unrounded: the
    scores move, and the output rounds differently in many places). Float64
    summation order may flip a rounding at a boundary, so a handful of
    elements may differ by one bf16 step; a missing storage rounding moves
    far more."""
    cfg = synth.get_config("tiny_layer")
    w, lw, ctx, tabs, kc, vc, x = _tiny_inputs(cfg)
    lz = _pass_through_attention(lw, cfg)
    kc1, vc1 = kc.copy(), vc.copy()
    out = od.decode_layer(x, lz, cfg, kc1, vc1, ctx, tabs, round_bf16=True)
    k_t, v_t, o_t = _attention_block_by_torch(x, lz, cfg, kc, vc, ctx, tabs)
    bs = cfg["block_size"]
    kn = np.stack([kc1[tabs[b][c // bs], :, c % bs, :] for b, c in enumerate(ctx)])
    vn = np.stack([vc1[tabs[b][c // bs], :, c % bs, :] for b, c in enumerate(ctx)])
    got_o = out - x

    def close(got, want, what):
        assert _is_bf16(got), f"{what}: not bf16 numbers"
        d = got != want
        assert d.mean() <= 0.01, f"{what}: {d.mean():.2%} of elements differ"
        np.testing.assert_allclose(got, want, rtol=2.0 ** -7, atol=0)

    close(kn, k_t, "cached k")
    close(vn, v_t, "cached v")
    close(got_o, o_t, "attention output")


def test_bf16_mode_close_to_exact_mode():
    cfg = synth.get_config("tiny_layer")
    w, lw, ctx, tabs, kc, vc, x = _tiny_inputs(cfg)
    a = od.decode_layer(x, lw, cfg, kc.copy(), vc.copy(), ctx, tabs, round_bf16=True)
    b = od.decode_layer(x, lw, cfg, kc.copy(), vc.copy(), ctx, tabs, round_bf16=False)
    rel = np.max(np.abs(a - b), axis=1) / np.max(np.abs(b), axis=1)
    assert rel.max() < 5e-3
    assert np.any(a != b)


# ---------------------------------------------------------------- mode switching (§4.3)

def test_mode_schedule_switches_after_a_persistent_drop():
    from oracle.orchestrator import WAS, CAS, mode_schedule
    b_th, h, W = 64, 0.5, 4
    # above the threshold throughout: never leaves WaS
    assert mode_schedule([[200, 100]] * 20, b_th, h, W) == [WAS] * 20
    # the effective batch drops below B_th from iteration 5 on: the first CaS iteration is 5 + W
    trace = [[100, 100]] * 5 + [[40, 40]] * 15
    modes = mode_schedule(trace, b_th, h, W)
    assert modes.index(CAS) == 5 + W and all(m == CAS for m in modes[5 + W:])
    # dips shorter than the window never switch
    trace = ([[100, 100]] * 3 + [[10, 10]] * (W - 1)) * 5
    assert mode_schedule(trace, b_th, h, W) == [WAS] * len(trace)
    # the effective batch is the mean over all engines, idle ones (0 active) included
    trace = [[100, 100, 0, 0]] * 10  # mean 50 < 64 although two engines run 100 rows
    assert mode_schedule(trace, b_th, h, W)[W] == CAS


def test_mode_schedule_hysteresis():
    from oracle.orchestrator import WAS, CAS, mode_schedule
    b_th, h, W = 64, 0.5, 3
    down = [[10, 10]] * W           # into CaS
    band = [[80, 80]] * 10          # above B_th but below B_th * 1.5 = 96: stays in CaS
    up = [[100, 100]] * (W + 2)     # at least 96: back to WaS after W iterations
    modes = mode_schedule(down + band + up, b_th, h, W)
    assert modes[W:W + 10] == [CAS] * 10
    k = W + 10  # first iteration at or above B_th * (1 + h); WaS from k + W on
    assert modes[k:k + W] == [CAS] * W and modes[k + W:] == [WAS] * 2
    # exactly at the upper edge counts as "at least"
    assert mode_schedule(down + [[96, 96]] * (W + 1), b_th, h, W)[2 * W] == WAS


def test_mode_schedule_invariants_on_random_traces():
    """On random tails: every switch is preceded by exactly the window of
    qualifying iterations in the old mode, and successive switches are at
    least a window apart (no flapping)."""
    from oracle.orchestrator import WAS, CAS, effective_batch, mode_schedule
    rng = np.random.default_rng(5)
    for _ in range(200):
        n, T, W = int(rng.integers(1, 9)), int(rng.integers(5, 80)), int(rng.integers(1, 6))
        b_th, h = float(rng.integers(8, 128)), float(rng.uniform(0, 1))
        trace = [list(map(int, rng.integers(0, 256, n))) for _ in range(T)]
        modes = mode_schedule(trace, b_th, h, W)
        assert modes[0] == WAS
        last = None
        for t in range(1, T):
            if modes[t] != modes[t - 1]:
                window = [effective_batch(trace[s]) for s in range(t - W, t)]
                assert t - W >= 0 and all(m == modes[t - 1] for m in modes[t - W:t])
                if modes[t] == CAS:
                    assert all(b < b_th for b in window)
                else:
                    assert all(b >= b_th * (1 + h) for b in window)
                assert last is None or t - last >= W
                last = t


# ------------------------------------------------------------------ peak shifting (§4.2)

def test_peak_shift_follows_the_text_on_one_cycle():
    # d = 4, cycle starting at layer 0: rank 2 starts at layer 2 (its own, skipped) and
    # wraps within the cycle: 3, 0, 1; rank 0 pulls 1, 2, 3; rank 3 pulls 0, 1, 2
    assert [l for l, _ in oracle.peak_shift_order(4, 4, 2)] == [3, 0, 1]
    assert [l for l, _ in oracle.peak_shift_order(4, 4, 0)] == [1, 2, 3]
    assert [l for l, _ in oracle.peak_shift_order(4, 4, 3)] == [0, 1, 2]
    assert oracle.peak_shift_order(7, 1, 0) == []  # one rank owns everything


def test_peak_shift_covers_every_remote_layer_once():
    # property (i): within each cycle a rank gets every layer it does not own after at
    # most d - 1 pulls, never its own, and never one from outside the cycle
    for d in range(2, 9):
        for L in (d, 2 * d, 3 * d + 1, 5 * d - 1, 80):
            for r in range(d):
                order = oracle.peak_shift_order(L, d, r)
                layers = [l for l, _ in order]
                assert sorted(layers) == [l for l in range(L) if l % d != r], (d, L, r)
                assert all(owner == l % d and owner != r for l, owner in order)
                for c in range(0, L, d):
                    in_cycle = [i for i, l in enumerate(layers) if c <= l < c + d]
                    assert len(in_cycle) <= d - 1
                    assert in_cycle == list(range(in_cycle[0], in_cycle[0] + len(in_cycle))) if in_cycle else True


def test_peak_shift_spreads_each_step_over_distinct_owners():
    # property (ii): at the k-th pull of a full cycle, the d ranks read d - 1 ... d
    # different owners (the text says ranks "tend to" differ; this scheme makes it exact)
    for d in range(2, 9):
        L = 3 * d
        orders = [oracle.peak_shift_order(L, d, r) for r in range(d)]
        for cyc in range(L // d):
            for k in range(d - 1):
                owners = [orders[r][cyc * (d - 1) + k][1] for r in range(d)]
                assert len(set(owners)) == d, (d, cyc, k, owners)
                layers = [orders[r][cyc * (d - 1) + k][0] for r in range(d)]
                assert all(cyc * d <= l < (cyc + 1) * d for l in layers)
