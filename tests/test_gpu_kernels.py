"""Per-kernel parity of the HIP library against the oracle, through the C ABI.

Tolerances follow from the arithmetic: the kernels evaluate in fp32 and the
oracle in float64, so a bf16 output can differ by one bf16 spacing where the
exact value sits near a rounding boundary (assert_bf16_within_ulp, 1 ulp).
Attention feeds its softmax probabilities to the bf16 MFMA as a high plus a
low bf16 part (about 16 significant bits), so |o - o*| <= 2^-16 sum_j P_j |v_j|
plus fp32 rounding; the test allows 2^-12 sum_j P_j |v_j| (sum_j P_j |v_j| is
the oracle's attention applied to |V|) plus one bf16 ulp of the output.
"""

import numpy as np
import pytest
import torch

import oracle
import synth
from gpu_helpers import assert_bf16_within_ulp, bits, dot_abs_tol, f64

pytestmark = pytest.mark.gpu


def _dev():
    return torch.device("cuda")


@pytest.fixture(scope="module")
def tiny_handle(lib):
    """A handle for single-kernel calls; 70B layer shapes, so its split-K
    scratch covers every projection size used below."""
    cfg = synth.get_config("llama70b_layer")
    h = lib.sidp_create(lib.make_config(cfg, 512, 9000))
    yield h
    lib.sidp_destroy(h)


# ------------------------------------------------------------------ RMSNorm

@pytest.mark.parametrize("rows,n", [(1, 256), (8, 256), (37, 5120), (256, 8192), (3, 12)])
def test_rmsnorm_parity(lib, rows, n):
    g = torch.Generator().manual_seed(rows * 7 + n)
    x = torch.randn(rows, n, generator=g) * 3.0
    gain = (1 + 0.1 * torch.randn(n, generator=g)).to(torch.bfloat16)
    out = torch.empty(rows, n, dtype=torch.bfloat16, device=_dev())
    lib.sidp_rmsnorm(x.to(_dev()), gain.to(_dev()), 1e-5, out, rows, n)
    torch.cuda.synchronize()
    want = oracle.rms_norm(x.double().numpy(), oracle.bf16_bits_to_f64(bits(gain)), 1e-5)
    assert_bf16_within_ulp(bits(out), want, what="rmsnorm")


# ------------------------------------------------------------------ projections

LINEAR_CASES = [
    # m, k, n, epilogue, bias
    (1, 256, 512, 0, False),
    (8, 256, 512, 0, True),
    (31, 688, 256, 1, False),      # K tail (688 = 10*64 + 48)
    (8, 256, 688, 2, False),       # SwiGLU with an N tail
    (64, 5120, 1024, 0, False),
    (100, 1024, 8192, 1, False),   # split-K path
    (256, 8192, 1024, 0, True),
    (256, 1024, 512, 2, False),
    (300, 512, 640, 1, False),     # two row blocks, ragged
    (512, 1024, 512, 2, False),
    (17, 4096, 2048, 1, False),
    (128, 3072, 1024, 1, False),   # three k-tiles per split: whole rounds of the three-deep ring only
    (100, 256, 45056, 0, True),    # enough column tiles for one split
    (200, 512, 28672, 2, False),   # SwiGLU without a split past 64 rows: the gate/up launch of a decode step
    # 256-row workgroups with LDS-staged weights (k_gemm alone would run one unsplit round on 160 of
    # 256 CUs): split partials reduced with the bias, with SwiGLU, and in place on the residual with
    # ragged rows and columns (groups past N idle)
    (512, 512, 10240, 0, True),
    (512, 512, 5120, 2, False),
    (400, 512, 9000, 1, False),
]


@pytest.mark.parametrize("m,k,n,epi,use_bias", LINEAR_CASES)
def test_linear_parity(lib, tiny_handle, m, k, n, epi, use_bias):
    g = torch.Generator().manual_seed(m * 131 + k * 7 + n + epi)
    x = torch.randn(m, k, generator=g).to(torch.bfloat16)
    dev = _dev()
    if epi == lib.SIDP_EPI_SWIGLU:
        wg = (0.02 * torch.randn(n, k, generator=g)).to(torch.bfloat16)
        wu = (0.02 * torch.randn(n, k, generator=g)).to(torch.bfloat16)
        packed = torch.empty(lib.sidp_packed_bytes(2 * ((n + 31) // 32 * 32), k), dtype=torch.uint8, device=dev)
        lib.sidp_pack_gate_up(wg.to(dev), wu.to(dev), n, k, packed)
    else:
        w = (0.02 * torch.randn(n, k, generator=g)).to(torch.bfloat16)
        packed = torch.empty(lib.sidp_packed_bytes(n, k), dtype=torch.uint8, device=dev)
        lib.sidp_pack_linear(w.to(dev), n, k, packed)
    bias = (0.02 * torch.randn(n, generator=g)).to(torch.bfloat16) if use_bias else None
    resid = torch.randn(m, n, generator=g) if epi == lib.SIDP_EPI_RESID else None
    if epi == lib.SIDP_EPI_RESID:
        out = resid.to(dev).clone()  # in place, as the decode step uses it
        lib.sidp_linear(tiny_handle, x.to(dev), m, k, packed, n, epi, None, out, out)
    else:
        out = torch.empty(m, n, dtype=torch.bfloat16, device=dev)
        lib.sidp_linear(tiny_handle, x.to(dev), m, k, packed, n, epi, bias.to(dev) if use_bias else None, None, out)
    torch.cuda.synchronize()
    xf = f64(x)
    if epi == lib.SIDP_EPI_SWIGLU:
        gf, uf = f64(wg), f64(wu)
        want = oracle.swiglu(xf, gf, uf)
        # silu'(z) <= 1.1: the gate's sum error passes through scaled by |up|
        tol = 1.1 * dot_abs_tol(xf, gf) * np.abs(oracle.linear(xf, uf)) + \
            np.abs(oracle.silu(oracle.linear(xf, gf))) * dot_abs_tol(xf, uf)
        assert_bf16_within_ulp(bits(out), want, what="swiglu", abs_tol=tol)
    else:
        want = oracle.linear(xf, f64(w), f64(bias) if use_bias else None)
        if epi == lib.SIDP_EPI_BF16:
            assert_bf16_within_ulp(bits(out), want, what="linear", abs_tol=dot_abs_tol(xf, f64(w)))
        else:
            want = resid.double().numpy() + want
            got = out.double().cpu().numpy()
            # fp32 accumulation over k terms: |err| << 1e-4 of the row scale
            scale = np.max(np.abs(want), axis=1, keepdims=True)
            assert np.all(np.abs(got - want) <= 2e-5 * scale), np.max(np.abs(got - want) / scale)


def test_linear_rejects_bad_arguments(lib, tiny_handle):
    dev = _dev()
    x = torch.zeros(4, 256, dtype=torch.bfloat16, device=dev)
    p = torch.zeros(lib.sidp_packed_bytes(64, 256), dtype=torch.uint8, device=dev)
    out = torch.zeros(4, 64, dtype=torch.float32, device=dev)
    E = lib.SIDP_EINVAL
    assert lib.raw_call("sidp_linear", tiny_handle, x.data_ptr(), 4, 256, p.data_ptr(), 64, 1, None, None,
                        out.data_ptr(), None) == E  # residual missing
    assert lib.raw_call("sidp_linear", tiny_handle, x.data_ptr(), 4, 250, p.data_ptr(), 64, 0, None, None,
                        out.data_ptr(), None) == E  # k not a multiple of 8
    assert lib.raw_call("sidp_linear", tiny_handle, x.data_ptr(), 513, 256, p.data_ptr(), 64, 0, None, None,
                        out.data_ptr(), None) == E  # m beyond max_batch
    # packed weights past the kernels' 32-bit buffer offsets (2^21 x 2^12 bf16 = 16 GiB): refused
    # on the host before any launch (the buffers are never touched)
    assert lib.raw_call("sidp_linear", tiny_handle, x.data_ptr(), 4, 1 << 12, p.data_ptr(), 1 << 21, 0, None, None,
                        out.data_ptr(), None) == E


# ------------------------------------------------------------------ RoPE + KV append

@pytest.mark.parametrize("name,qk_norm", [("tiny_layer", 0), ("tiny_layer", 1), ("qwen3_32b_layer", 1),
                                          ("llama70b_layer", 0)])
def test_rope_append_parity(lib, name, qk_norm):
    cfg = synth.get_config(name, qk_norm=qk_norm)
    Hq, Hkv, D = cfg["num_q_heads"], cfg["num_kv_heads"], cfg["head_dim"]
    B = 9
    ctx = np.array([0, 1, 15, 16, 17, 31, 32, 100, 1000], np.int32)
    tables = lib.sidp_kv_alloc(ctx, 1, 16, 200, 5, 64)
    nblk, R, region = 200, 2, 1
    dev = _dev()
    cfgm = dict(cfg, num_layers=1)
    h = lib.sidp_create(lib.make_config(cfgm, B, 2048))
    try:
        kc = torch.full((R, nblk, Hkv, D // 8, 16, 8), float("nan"), dtype=torch.bfloat16, device=dev)
        vc = torch.full((R, nblk, Hkv, D, 16), float("nan"), dtype=torch.bfloat16, device=dev)
        lib.sidp_kv_attach(h, kc, vc, nblk, R)
        g = torch.Generator().manual_seed(11)
        qkv = torch.randn(B, (Hq + 2 * Hkv) * D, generator=g).to(torch.bfloat16)
        gq = (1 + 0.1 * torch.randn(D, generator=g)).to(torch.bfloat16)
        gk = (1 + 0.1 * torch.randn(D, generator=g)).to(torch.bfloat16)
        q_out = torch.empty(B, Hq, D, dtype=torch.bfloat16, device=dev)
        bt = torch.tensor(tables, dtype=torch.int32, device=dev)
        pos = torch.tensor(ctx, dtype=torch.int32, device=dev)
        kc0, vc0 = bits(lib.k_blocks_from_lib(kc)), bits(vc)
        lib.sidp_rope_append(h, qkv.to(dev), pos, bt, 64, B, gq.to(dev), gk.to(dev), region, q_out)
        lib.sidp_sync(h)
        qf = f64(qkv)
        q = qf[:, :Hq * D].reshape(B, Hq, D)
        k = qf[:, Hq * D:(Hq + Hkv) * D].reshape(B, Hkv, D)
        vb = bits(qkv)[:, (Hq + Hkv) * D:].reshape(B, Hkv, D)
        if qk_norm:
            q = oracle.rms_norm(q, f64(gq), cfg["qk_norm_eps"])
            k = oracle.rms_norm(k, f64(gk), cfg["qk_norm_eps"])
        q = oracle.rope_rotate_half(q, ctx[:, None], cfg["rope_theta"])
        k = oracle.rope_rotate_half(k, ctx[:, None], cfg["rope_theta"])
        assert_bf16_within_ulp(bits(q_out), q, what="rotated q")
        kc1, vc1 = bits(lib.k_blocks_from_lib(kc)), bits(vc)
        expect_k, expect_v = kc0.copy(), vc0.copy()
        for b in range(B):
            p = int(ctx[b])
            blk = tables[b][p // 16]
            assert_bf16_within_ulp(kc1[region, blk, :, p % 16, :], k[b], what=f"cached k row {b}")
            expect_k[region, blk, :, p % 16, :] = kc1[region, blk, :, p % 16, :]
            expect_v[region, blk, :, :, p % 16] = vb[b]
        # values are stored exactly; nothing else in either cache changed
        assert np.array_equal(vc1, expect_v)
        assert np.array_equal(kc1, expect_k)
    finally:
        lib.sidp_destroy(h)


# ------------------------------------------------------------------ attention

def _attn_setup(lib, cfg, seqs, nblk_extra=7, seed=3, equal_keys=False, q_scale=1.0):
    Hq, Hkv, D = cfg["num_q_heads"], cfg["num_kv_heads"], cfg["head_dim"]
    B = len(seqs)
    ctx = np.asarray(seqs, np.int32) - 1
    need = [-(-s // 16) for s in seqs]
    nblk = sum(need) + nblk_extra
    tables = lib.sidp_kv_alloc(ctx, 1, 16, nblk, seed, max(need))
    g = torch.Generator().manual_seed(seed)
    k = torch.randn(nblk, Hkv, 16, D, generator=g).to(torch.bfloat16)
    v = torch.randn(nblk, Hkv, 16, D, generator=g).to(torch.bfloat16)
    if equal_keys:
        k[:] = torch.randn(D, generator=g).to(torch.bfloat16)
    q = (q_scale * torch.randn(B, Hq, D, generator=g)).to(torch.bfloat16)
    # slots past each sequence's end hold NaN: the kernel must never use them
    for b, s in enumerate(seqs):
        for t in range(s, need[b] * 16):
            blk = tables[b][t // 16]
            k[blk, :, t % 16, :] = float("nan")
            v[blk, :, t % 16, :] = float("nan")
    return ctx, tables, nblk, k, v, q, max(need)


def _attn_run(lib, cfg, ctx, tables, nblk, k, v, q, maxb, regions=1, region=0):
    dev = _dev()
    B = len(ctx)
    Hq, Hkv, D = cfg["num_q_heads"], cfg["num_kv_heads"], cfg["head_dim"]
    h = lib.sidp_create(lib.make_config(dict(cfg, num_layers=1), B, maxb * 16 + 16))
    try:
        kc = torch.zeros(regions, nblk, Hkv, D // 8, 16, 8, dtype=torch.bfloat16, device=dev)
        vc = torch.zeros(regions, nblk, Hkv, D, 16, dtype=torch.bfloat16, device=dev)
        kc[region] = lib.k_blocks_to_lib(k.to(dev))
        vc[region] = v.to(dev).transpose(-1, -2)
        lib.sidp_kv_attach(h, kc, vc, nblk, regions)
        out = torch.empty(B, Hq, D, dtype=torch.bfloat16, device=dev)
        bt = torch.tensor(tables, dtype=torch.int32, device=dev)
        lib.sidp_attention(h, q.to(dev), region, torch.tensor(ctx, dtype=torch.int32, device=dev), bt, maxb, B, out)
        lib.sidp_sync(h)
        return bits(out)
    finally:
        lib.sidp_destroy(h)


def _attn_oracle(cfg, ctx, tables, k, v, q, absv=False):
    kf, vf, qf = f64(k), f64(v), f64(q)
    if absv:
        vf = np.abs(vf)
    return np.stack([oracle.paged_gqa_attention(qf[b], kf, vf, tables[b], int(ctx[b]) + 1, 16)
                     for b in range(len(ctx))])


ATTN_SEQS = [1, 2, 15, 16, 17, 31, 32, 33, 100, 511, 512, 513, 1024, 1500, 2047, 2048, 2049, 4096, 4097]


@pytest.mark.parametrize("name,q_scale", [("tiny_layer", 1.0), ("llama70b_layer", 1.0), ("llama70b_layer", 4.0)])
def test_attention_parity(lib, name, q_scale):
    cfg = synth.get_config(name)
    ctx, tables, nblk, k, v, q, maxb = _attn_setup(lib, cfg, ATTN_SEQS, q_scale=q_scale)
    got = _attn_run(lib, cfg, ctx, tables, nblk, k, v, q, maxb, regions=2, region=1)
    want = _attn_oracle(cfg, ctx, tables, k, v, q)
    pv = _attn_oracle(cfg, ctx, tables, k, v, q, absv=True)  # sum_j P_j |v_j|
    assert_bf16_within_ulp(got, want, what="attention", abs_tol=2.0 ** -12 * pv)


def _many_short_seqs(n=2048, seed=11):
    return np.random.default_rng(seed).integers(1, 301, n).tolist()


@pytest.mark.parametrize("hq,hkv,d,seqs", [
    (16, 1, 128, ATTN_SEQS),   # the largest query group: 16 heads fill the MFMA columns and the (m, l) line
    (8, 2, 64, ATTN_SEQS),     # head dim 64 over several partitions
    (16, 1, 128, "many"),      # 2048 sequences x 1 KV head: whole-sequence items, no combine
])
def test_attention_parity_group_shapes(lib, hq, hkv, d, seqs):
    cfg = synth.get_config("tiny_layer", num_q_heads=hq, num_kv_heads=hkv, head_dim=d)
    seqs = _many_short_seqs() if seqs == "many" else seqs
    ctx, tables, nblk, k, v, q, maxb = _attn_setup(lib, cfg, seqs)
    got = _attn_run(lib, cfg, ctx, tables, nblk, k, v, q, maxb)
    want = _attn_oracle(cfg, ctx, tables, k, v, q)
    pv = _attn_oracle(cfg, ctx, tables, k, v, q, absv=True)
    assert_bf16_within_ulp(got, want, what=f"attention {hq}/{hkv} x {d}", abs_tol=2.0 ** -12 * pv)


def test_attention_longest_context(lib):
    """A sequence at the longest context a handle accepts (2^20 positions:
    512 partitions merged by the combine kernel), ragged in its last block,
    beside a short and a two-partition one."""
    cfg = synth.get_config("tiny_layer")
    seqs = [(1 << 20) - 21, 5, 2049]
    ctx, tables, nblk, k, v, q, maxb = _attn_setup(lib, cfg, seqs, nblk_extra=3)
    assert maxb * 16 + 16 == 1 << 20  # the handle's max_seq_len at its limit
    got = _attn_run(lib, cfg, ctx, tables, nblk, k, v, q, maxb)
    want = _attn_oracle(cfg, ctx, tables, k, v, q)
    pv = _attn_oracle(cfg, ctx, tables, k, v, q, absv=True)
    assert_bf16_within_ulp(got, want, what="attention, longest context", abs_tol=2.0 ** -12 * pv)


def test_attention_closed_forms_on_gpu(lib):
    cfg = synth.get_config("llama70b_layer")
    # one cached token: the output is exactly that token's V row
    ctx, tables, nblk, k, v, q, maxb = _attn_setup(lib, cfg, [1, 1, 1])
    got = _attn_run(lib, cfg, ctx, tables, nblk, k, v, q, maxb)
    for b in range(3):
        for hq in range(cfg["num_q_heads"]):
            assert np.array_equal(got[b, hq], bits(v)[tables[b][0], hq // 8, 0, :])
    # all-equal keys: the mean of V over the sequence
    ctx, tables, nblk, k, v, q, maxb = _attn_setup(lib, cfg, [40, 700], equal_keys=True)
    got = _attn_run(lib, cfg, ctx, tables, nblk, k, v, q, maxb)
    vf = f64(v)
    for b, s in enumerate([40, 700]):
        t = np.arange(s)
        V = vf[np.asarray(tables[b])[t // 16], :, t % 16, :]  # (s, Hkv, D)
        mean = V.mean(axis=0)
        want = np.repeat(mean, 8, axis=0)
        assert_bf16_within_ulp(got[b], want, what="equal-keys mean")


def test_attention_block_permutation_invariance_bitexact(lib):
    cfg = synth.get_config("llama70b_layer")
    seqs = [17, 513, 1030]
    ctx, tables, nblk, k, v, q, maxb = _attn_setup(lib, cfg, seqs)
    out1 = _attn_run(lib, cfg, ctx, tables, nblk, k, v, q, maxb)
    perm = torch.randperm(nblk, generator=torch.Generator().manual_seed(99))
    k2, v2 = torch.empty_like(k), torch.empty_like(v)
    k2[perm], v2[perm] = k, v
    tables2 = [[int(perm[b]) if b >= 0 else -1 for b in row] for row in tables]
    out2 = _attn_run(lib, cfg, ctx, tables2, nblk, k2, v2, q, maxb)
    assert np.array_equal(out1, out2)


def test_attention_bad_block_index_is_reported(lib):
    """A block index past the cache inside a sequence's attended range: the
    kernel reads block 0 instead (never out of bounds) and latches the error,
    which sync reports; a good call afterwards is clean."""
    cfg = synth.get_config("llama70b_layer")
    dev = _dev()
    seqs = [40, 700]
    ctx, tables, nblk, k, v, q, maxb = _attn_setup(lib, cfg, seqs)
    B, Hq, Hkv, D = len(seqs), cfg["num_q_heads"], cfg["num_kv_heads"], cfg["head_dim"]
    h = lib.sidp_create(lib.make_config(dict(cfg, num_layers=1), B, maxb * 16 + 16))
    try:
        kc = torch.zeros(1, nblk, Hkv, D // 8, 16, 8, dtype=torch.bfloat16, device=dev)
        vc = torch.zeros(1, nblk, Hkv, D, 16, dtype=torch.bfloat16, device=dev)
        kc[0] = lib.k_blocks_to_lib(k.to(dev))
        vc[0] = v.to(dev).transpose(-1, -2)
        lib.sidp_kv_attach(h, kc, vc, nblk, 1)
        out = torch.empty(B, Hq, D, dtype=torch.bfloat16, device=dev)
        pos = torch.tensor(ctx, dtype=torch.int32, device=dev)
        bad = [list(r) for r in tables]
        bad[1][3] = nblk + 5
        lib.sidp_attention(h, q.to(dev), 0, pos, torch.tensor(bad, dtype=torch.int32, device=dev), maxb, B, out)
        with pytest.raises(lib.SidpError) as e:
            lib.sidp_sync(h)
        assert e.value.code == lib.SIDP_EINVAL
        lib.sidp_attention(h, q.to(dev), 0, pos, torch.tensor(tables, dtype=torch.int32, device=dev), maxb, B, out)
        lib.sidp_sync(h)
    finally:
        lib.sidp_destroy(h)


# ------------------------------------------------------------------ slot mapping, copy

def test_slot_mapping_bitexact_and_error(lib, tiny_handle):
    dev = _dev()
    ctx = np.array([0, 15, 16, 63, 64, 200], np.int32)
    tables = lib.sidp_kv_alloc(ctx, 1, 16, 64, 2, 16)
    bt = torch.tensor(tables, dtype=torch.int32, device=dev)
    slots = torch.empty(len(ctx), dtype=torch.int32, device=dev)
    lib.sidp_slot_mapping(tiny_handle, torch.tensor(ctx, dtype=torch.int32, device=dev), bt, 16, len(ctx), slots)
    lib.sidp_sync(tiny_handle)
    want = [oracle.slot_of(tables[b], int(ctx[b])) for b in range(len(ctx))]
    assert slots.cpu().tolist() == want
    # a position whose block is unallocated (-1 in the table) maps to -1 and is reported
    bad = torch.tensor([0, 15 * 16], dtype=torch.int32, device=dev)
    lib.sidp_slot_mapping(tiny_handle, bad, bt, 16, 2, slots)
    with pytest.raises(lib.SidpError) as e:
        lib.sidp_sync(tiny_handle)
    assert e.value.code == lib.SIDP_EINVAL
    assert slots[:2].cpu().tolist() == [tables[0][0] * 16, -1]


@pytest.mark.parametrize("nbytes,grid", [(16, 0), (4096 + 5, 3), (1 << 20, 64), ((64 << 20) + 48, 0)])
def test_copy_bitexact(lib, nbytes, grid):
    dev = _dev()
    src = torch.randint(0, 256, (nbytes,), dtype=torch.uint8, device=dev)
    dst = torch.zeros(nbytes + 64, dtype=torch.uint8, device=dev)
    lib.sidp_copy(src, dst, nbytes, grid)
    torch.cuda.synchronize()
    assert torch.equal(dst[:nbytes], src)
    assert int(dst[nbytes:].sum()) == 0
