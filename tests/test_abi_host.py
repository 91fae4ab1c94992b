"""The C-ABI library on the CPU: it loads, exports every symbol the header
declares, and its host-only logic (block-table allocation, slot-ring plan,
argument validation) matches the oracle bit for bit. No GPU work is issued."""

import ctypes
import os
import re

import numpy as np
import pytest

import oracle
import synth

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _header_symbols():
    text = open(os.path.join(ROOT, "include", "sidp.h")).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(sidp_[a-z0-9_]+)\s*\(", text)))


def test_library_exports_every_declared_symbol():
    import paper_2605_28095_amd as sidp
    syms = _header_symbols()
    assert len(syms) >= 20
    lib = ctypes.CDLL(sidp.LIB_PATH)
    missing = [s for s in syms if not hasattr(lib, s)]
    assert not missing, missing
    assert sorted(sidp.EXPORTED) == syms


def test_strerror_names_every_code():
    import paper_2605_28095_amd as sidp
    for code in (0, -1, -2, -3, -4, -5):
        assert sidp.strerror(code) and sidp.strerror(code) != "unknown status"
    assert sidp.strerror(7) == "unknown status"


@pytest.mark.parametrize("name", ["tiny_layer", "qwen3_32b_layer", "llama70b_stack80"])
def test_kv_alloc_bit_exact_vs_oracle(name):
    import paper_2605_28095_amd as sidp
    cfg = synth.get_config(name)
    ctx = synth.context_lengths(cfg, seed=0)
    reserve = 1
    need = int(sum(-(-(int(c) + reserve) // 16) for c in ctx))
    nblk = cfg["num_phys_blocks"] or need + 37
    maxb = int(max(-(-(int(c) + reserve) // 16) for c in ctx)) + 2
    for seed in (0, 1, 12345):
        got = sidp.sidp_kv_alloc(ctx, reserve, 16, nblk, seed, maxb)
        want = oracle.allocate_block_tables(ctx, reserve, nblk, maxb, seed)
        assert got == want


def test_kv_alloc_errors():
    import paper_2605_28095_amd as sidp
    with pytest.raises(sidp.SidpError) as e:
        sidp.sidp_kv_alloc([100, 100], 1, 16, 10, 0, 16)
    assert e.value.code == sidp.SIDP_ENOBLOCKS
    with pytest.raises(sidp.SidpError) as e:
        sidp.sidp_kv_alloc([100], 1, 16, 100, 0, 4)  # table too narrow
    assert e.value.code == sidp.SIDP_ENOBLOCKS
    with pytest.raises(sidp.SidpError) as e:
        sidp.sidp_kv_alloc([-3], 1, 16, 100, 0, 4)
    assert e.value.code == sidp.SIDP_EINVAL
    assert sidp.sidp_kv_alloc([], 1, 16, 0, 0, 1) == []


@pytest.mark.parametrize("L,steps,ranks,rank", [(1, 1, 0, 0), (3, 2, 0, 0), (80, 3, 0, 0), (8, 0, 0, 0),
                                               (7, 3, 3, 1), (80, 2, 8, 0), (4, 2, 1, 0), (5, 2, 2, 1), (3, 1, 9, 8)])
def test_plan_matches_oracle_schedule(L, steps, ranks, rank):
    import paper_2605_28095_amd as sidp
    assert sidp.sidp_plan(L, steps, ranks, rank) == oracle.was_schedule(L, steps, ranks, rank)


def test_plan_and_pooling_reject_bad_ranks():
    import paper_2605_28095_amd as sidp
    for ranks, rank in [(-1, 0), (2, 2), (3, -1)]:
        assert sidp.raw_call("sidp_plan", 4, 1, ranks, rank, None, None) == sidp.SIDP_EINVAL
    assert sidp.raw_call("sidp_set_pooling", None, 0, 0, 0) == sidp.SIDP_EINVAL


def test_config_validation_on_host():
    import paper_2605_28095_amd as sidp
    cfg = synth.get_config("llama70b_layer")
    good = sidp.make_config(cfg, 256, 8192)
    lb = sidp.sidp_layer_bytes(good)
    assert sidp.sidp_pool_bytes(good) == cfg["num_layers"] * lb
    assert sidp.sidp_slot_bytes(good) == 2 * lb
    # packed projections plus small vectors, all 256-byte aligned
    assert lb % 256 == 0
    assert 2 * synth.layer_param_count(cfg) <= lb < 2 * synth.layer_param_count(cfg) + 64 * 1024
    for field, bad in [("head_dim", 96), ("num_kv_heads", 7), ("block_size", 32), ("hidden", 100),
                       ("ffn_dim", 20), ("max_batch", 0), ("hidden", 1 << 18), ("ffn_dim", 1 << 21)]:
        c = sidp.make_config(cfg, 256, 8192)
        setattr(c, field, bad)
        assert sidp.sidp_layer_bytes(c) == 0, field
        assert sidp.sidp_pool_bytes(c) == 0 and sidp.sidp_slot_bytes(c) == 0, field
    c = sidp.make_config(cfg, 256, 8192)
    c.num_q_heads = 64
    c.num_kv_heads = 2  # group of 32 query heads per KV head is not supported
    assert sidp.sidp_layer_bytes(c) == 0
    # each field in range, but the packed gate/up (2 * 2^20 x 2^15 bf16 = 128 GiB) would overflow
    # the projections' 32-bit buffer offsets
    c = sidp.make_config(cfg, 256, 8192)
    c.hidden, c.ffn_dim = 1 << 15, 1 << 20
    assert sidp.sidp_layer_bytes(c) == 0
    assert sidp.sidp_kv_region_bytes(good, 10) == 10 * 8 * 16 * 128 * 2
    assert sidp.sidp_packed_bytes(688, 256) == 704 * 256 * 2


def test_null_handle_calls_are_rejected():
    import paper_2605_28095_amd as sidp
    assert sidp.raw_call("sidp_sync", None) == sidp.SIDP_EINVAL
    assert sidp.raw_call("sidp_destroy", None) == sidp.SIDP_EINVAL
    assert sidp.raw_call("sidp_decode_step", None, None, None, None, 1, 1, 0, None, None) == sidp.SIDP_EINVAL
    assert sidp.raw_call("sidp_plan", 0, 1, 0, 0, None, None) == sidp.SIDP_EINVAL
    assert sidp.raw_call("sidp_set_fill_tiles", None, 25, 0, 0, 1) == sidp.SIDP_EINVAL
    assert sidp.raw_call("sidp_debug_inject_hip_error", None, 1) == sidp.SIDP_EINVAL
    assert sidp.raw_call("sidp_pool_init", None, None, 0, None, 0, None, 0, None) == sidp.SIDP_EINVAL


def test_key_block_layout_helpers():
    """Key blocks in the library's layout: element (token t, dim d) of a
    (block, kv head) piece sits at ((d // 8) * block_size + t) * 8 + d % 8, so
    the 16 tokens x 32 dims of one QK fragment are one contiguous 1 KB run."""
    import torch
    import paper_2605_28095_amd as sidp
    nblk, hkv, bs, d = 3, 2, 16, 128
    k = torch.arange(nblk * hkv * bs * d, dtype=torch.int64).reshape(nblk, hkv, bs, d)
    kl = sidp.k_blocks_to_lib(k).contiguous()
    assert kl.shape == (nblk, hkv, d // 8, bs, 8)
    flat = kl.reshape(nblk, hkv, -1)
    for t, dd in [(0, 0), (15, 127), (7, 45), (9, 8), (3, 100)]:
        assert flat[2, 1, ((dd // 8) * bs + t) * 8 + dd % 8] == k[2, 1, t, dd]
    # fragment kk of lane (token t, group g) covers dims 32 kk + 8 g .. + 7: 16-byte piece 64 kk + 16 g + t
    pieces = flat[1, 0].reshape(-1, 8)
    for kk in range(d // 32):
        run = pieces[64 * kk:64 * kk + 64]
        for lane in (0, 17, 63):
            g, t = lane // 16, lane % 16
            assert torch.equal(run[lane], k[1, 0, t, 32 * kk + 8 * g:32 * kk + 8 * g + 8])
    assert torch.equal(sidp.k_blocks_from_lib(kl), k)


def test_mode_update_matches_oracle():
    """The library's WaS/CaS choice equals the oracle's on random job tails
    (thresholds drawn as float32 values, which both sides then use exactly)."""
    import paper_2605_28095_amd as sidp
    from oracle.orchestrator import mode_schedule
    rng = np.random.default_rng(11)
    for _ in range(300):
        n, T, W = int(rng.integers(1, 9)), int(rng.integers(1, 120)), int(rng.integers(1, 7))
        b_th = float(np.float32(rng.uniform(1, 200)))
        h = float(np.float32(rng.choice([0.0, 0.25, 0.5, float(rng.uniform(0, 1))])))
        # a shrinking tail with noise, sometimes recovering
        base = np.maximum(0, 256 - np.cumsum(rng.integers(0, 12, T)))
        trace = [list(map(int, np.clip(base[t] + rng.integers(-20, 21, n), 0, None))) for t in range(T)]
        if rng.random() < 0.3:
            trace = trace[::-1]
        assert sidp.mode_schedule(b_th, h, W, trace) == mode_schedule(trace, b_th, h, W)


def test_mode_update_rejects_bad_arguments():
    import paper_2605_28095_amd as sidp
    st = sidp.sidp_mode_state(0, 0)
    for pol, active in [(sidp.sidp_mode_policy(0.0, 0.5, 3), [4]), (sidp.sidp_mode_policy(8.0, -0.1, 3), [4]),
                        (sidp.sidp_mode_policy(8.0, 0.5, 0), [4]), (sidp.sidp_mode_policy(8.0, 0.5, 3), [4, -1])]:
        with pytest.raises(sidp.SidpError) as e:
            sidp.sidp_mode_update(pol, st, active)
        assert e.value.code == sidp.SIDP_EINVAL
        assert (st.mode, st.run) == (0, 0)  # unchanged
    with pytest.raises(sidp.SidpError):
        sidp.sidp_mode_update(sidp.sidp_mode_policy(8.0, 0.5, 3), st, [])


def test_peak_shift_plan_matches_oracle():
    import paper_2605_28095_amd as lib
    for d in range(1, 9):
        for L in (1, d, 2 * d + 1, 80):
            for r in range(d):
                assert lib.sidp_peak_shift_plan(L, d, r) == oracle.peak_shift_order(L, d, r), (L, d, r)


def test_peak_shift_plan_rejects_bad_arguments():
    import paper_2605_28095_amd as lib
    n = ctypes.c_int32(100)
    buf = (ctypes.c_int32 * 200)()
    f = lib._lib.sidp_peak_shift_plan
    E = lib.SIDP_EINVAL
    assert f(0, 4, 0, buf, ctypes.byref(n)) == E
    assert f(8, 0, 0, buf, ctypes.byref(n)) == E
    assert f(8, 4, 4, buf, ctypes.byref(n)) == E
    assert f(8, 4, -1, buf, ctypes.byref(n)) == E
    assert f(8, 4, 0, buf, None) == E
    small = ctypes.c_int32(5)  # rank 0 of 4 over 8 layers pulls 6
    assert f(8, 4, 0, buf, ctypes.byref(small)) == E
    assert f(8, 4, 0, None, ctypes.byref(n)) == E
    one = ctypes.c_int32(0)
    assert f(5, 1, 0, None, ctypes.byref(one)) == lib.SIDP_OK and one.value == 0  # nothing to pull


# The launches the projections get on a 256-CU MI355X, pinned: the 70B shapes at
# the benchmark's batch (B=256) and at B=512, where QKV moves to the
# LDS-staged-weight kernel because the register-fed one would run one unsplit
# round of 160 workgroups. Each tuple: (m, n, k, epilogue) -> (kernel, waves,
# rows per workgroup, splits, workgroups).
LINEAR_PLANS = [
    ((256, 10240, 8192, 0), (0, 4, 128, 3, 240)),   # QKV
    ((256, 8192, 8192, 1), (0, 4, 128, 4, 256)),    # O
    ((256, 28672, 8192, 2), (0, 7, 128, 1, 256)),   # gate/up + SwiGLU, 7-wave workgroups
    ((256, 8192, 28672, 1), (0, 4, 128, 4, 256)),   # down
    ((512, 10240, 8192, 0), (1, 8, 256, 3, 240)),   # QKV at 512 rows: LDS-staged weights
    ((512, 8192, 8192, 1), (0, 4, 128, 2, 256)),
    ((512, 28672, 8192, 2), (0, 7, 128, 1, 512)),
    ((384, 10240, 8192, 0), (0, 4, 128, 2, 240)),   # 120 workgroups x 2 splits: no LDS-staged kernel
    ((16, 10240, 8192, 0), (0, 4, 32, 6, 240)),
    ((64, 28672, 8192, 2), (0, 4, 64, 1, 224)),
]


@pytest.mark.parametrize("shape,want", LINEAR_PLANS)
def test_linear_plan_at_model_shapes(shape, want):
    import paper_2605_28095_amd as sidp
    m, n, k, epi = shape
    p = sidp.sidp_linear_plan(m, n, k, epi, 256)
    assert (p["kernel"], p["waves"], p["rows"], p["splits"], p["workgroups"]) == want
    ncols = 2 * ((n + 31) // 32 * 32) if epi == 2 else n
    assert p["ws_bytes"] == (p["splits"] * m * ((ncols + 63) // 64 * 64) * 4 if p["splits"] > 1 else 0)


def test_noalloc_scratch_holds_every_split_on_256_cus():
    """The scratch of sidp_linear_noalloc is as large as the header says and
    holds the split-K partials of every projection plan on a 256-CU MI355X up
    to its 4096-row limit, both kernels included."""
    import paper_2605_28095_amd as sidp
    hdr = open(os.path.join(os.path.dirname(__file__), "..", "include", "sidp.h")).read()
    m = re.search(r"#define SIDP_NOALLOC_SCRATCH_BYTES \((\d+)u << (\d+)\)", hdr)
    assert m and int(m.group(1)) << int(m.group(2)) == sidp.SIDP_NOALLOC_SCRATCH_BYTES
    most, kernels = 0, set()
    for rows in [1, 40, 128, 129, 200, 256, 257, 384, 400, 512, 640, 768, 1024, 2048, 4096]:
        for n in [64, 520, 1000, 1280, 4096, 8192, 10240, 14336, 28672, 32768]:
            for k in [256, 1024, 8192, 28672]:
                for epi in (0, 2):
                    p = sidp.sidp_linear_plan(rows, n, k, epi, 256)
                    assert p["ws_bytes"] <= sidp.SIDP_NOALLOC_SCRATCH_BYTES, (rows, n, k, epi, p)
                    most = max(most, p["ws_bytes"])
                    kernels.add(p["kernel"])
    assert kernels == {0, 1} and most > 32 << 20


def test_linear_plan_rejects_bad_arguments():
    import paper_2605_28095_amd as sidp
    E = sidp.SIDP_EINVAL
    out = [ctypes.c_int32() for _ in range(5)]
    ws = ctypes.c_uint64()
    refs = [ctypes.byref(o) for o in out] + [ctypes.byref(ws)]
    ok = (256, 8192, 8192, 1, 256)
    assert sidp.raw_call("sidp_linear_plan", *ok, *refs) == 0
    for bad in [(0, 8192, 8192, 1, 256), (256, 0, 8192, 1, 256), (256, 8192, 250, 1, 256),
                (256, 8192, 8192, 3, 256), (256, 8192, 8192, 1, 0), (4, 1 << 21, 1 << 12, 0, 256)]:
        assert sidp.raw_call("sidp_linear_plan", *bad, *refs) == E, bad
    assert sidp.raw_call("sidp_linear_plan", *ok, *refs[:-1], None) == E
