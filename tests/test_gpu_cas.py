"""Compute-as-a-Service at a layer's owner (§4.3) on the GPU, through the C
ABI: the replicas' FFN inputs are concatenated into the owner's staging
buffer, the FFN runs once over all rows, and the output is cut back per
replica. Checked against the oracle's CaS (the per-replica FFN), bit for bit
against per-replica calls where the fused call keeps the same split-K
partition, and dummy replicas must stay untouched."""

import numpy as np
import pytest
import torch

import oracle
import synth
from gpu_helpers import Stack, f64, row_rel_err

pytestmark = pytest.mark.gpu

# per-row inf-norm relative error: fp32 accumulation against float64, with the
# SwiGLU output rounded to bf16 on both sides
CAS_TOL = 2e-3


def _layer_f64(st, layer):
    w = st.layer_weights(layer)
    if isinstance(next(iter(w.values())), np.ndarray) and next(iter(w.values())).dtype == np.uint16:
        return {k: oracle.bf16_bits_to_f64(v) for k, v in w.items()}
    return w


def _inputs(H, rows, seed):
    g = torch.Generator(device="cuda").manual_seed(seed)
    return [(0.5 * torch.randn(r, H, device="cuda", generator=g)).to(torch.bfloat16) if r else None for r in rows]


def _run(lib, st, layer, xs, rows, sentinel=7.0):
    H = st.cfg["hidden"]
    ys = [torch.full((max(r, 1), H), sentinel, device="cuda", dtype=torch.float32) for r in rows]
    lib.sidp_cas_ffn(st.dec.h, layer, xs, rows, ys)
    st.dec.sync()
    return ys


def test_cas_ffn_small_vs_oracle_and_per_replica_bitexact(lib):
    cfg = synth.get_config("tiny_layer", num_layers=2)  # H 256, F 688: ragged FFN tail
    st = Stack(cfg, gains="random")
    try:
        H = cfg["hidden"]
        rows = [2, 0, 3, 1, 0, 2]  # 8 rows: the handle's max_batch
        xs = _inputs(H, rows, seed=11)
        ys = _run(lib, st, 1, xs, rows)
        w = _layer_f64(st, 1)
        want = oracle.cas_ffn([f64(x) if x is not None else None for x in xs], w["w_gate"], w["w_up"],
                              w["w_down"], round_bf16=True)
        for r, n in enumerate(rows):
            if n == 0:
                assert torch.all(ys[r] == 7.0), f"dummy replica {r} was written"
                assert want[r] is None
                continue
            got = ys[r].double().cpu().numpy()
            e = row_rel_err(got, want[r])
            assert e.max() <= CAS_TOL, (r, e)
        # one replica at a time: the same rows give the same bits (fused total
        # and single replicas use the same split-K partition at <= 128 rows)
        for r, n in enumerate(rows):
            if n == 0:
                continue
            solo = _run(lib, st, 1, [xs[r]], [n])[0]
            assert torch.equal(solo, ys[r]), f"replica {r}: fused rows differ from a per-replica call"
        # all dummies: nothing runs, nothing is written
        ys0 = _run(lib, st, 0, [None, None], [0, 0])
        assert all(torch.all(y == 7.0) for y in ys0)
    finally:
        st.close()


def test_cas_ffn_full_size_sampled_rows(lib):
    """The 70B layer's FFN over 256 fused rows from three replicas (one dummy),
    checked on sampled rows of every live replica."""
    cfg = synth.get_config("llama70b_layer")
    st = Stack(cfg, keep_weights=False)
    try:
        H = cfg["hidden"]
        rows = [100, 0, 156]
        xs = _inputs(H, rows, seed=12)
        ys = _run(lib, st, 0, xs, rows)
        assert torch.all(ys[1] == 7.0)
        w = st.layer_weights(0)
        for r, picks in [(0, [0, 99]), (2, [0, 77, 155])]:
            x = f64(xs[r])[picks]
            want = oracle.ffn(x, w["w_gate"], w["w_up"], w["w_down"], round_bf16=True)
            got = ys[r].double().cpu().numpy()[picks]
            e = row_rel_err(got, want)
            assert e.max() <= CAS_TOL, (r, e)
    finally:
        st.close()


def test_cas_ffn_rejects_bad_arguments(lib):
    cfg = synth.get_config("tiny_layer", num_layers=1)
    st = Stack(cfg, gains="one")
    try:
        H = cfg["hidden"]
        x = torch.zeros(4, H, device="cuda", dtype=torch.bfloat16)
        y = torch.zeros(4, H, device="cuda", dtype=torch.float32)
        for args in [(1, [x], [4], [y]),                      # no such layer
                     (0, [x], [-1], [y]),                     # negative rows
                     (0, [x] * 17, [1] * 17, [y] * 17),       # too many replicas
                     (0, [x, x], [st.batch, 1], [y, y])]:     # more rows than max_batch
            with pytest.raises(lib.SidpError) as e:
                lib.sidp_cas_ffn(st.dec.h, *args)
            assert e.value.code == lib.SIDP_EINVAL
        flat = torch.zeros(4 * H + 8, device="cuda", dtype=torch.bfloat16)
        xm = flat[4:4 + 4 * H].view(4, H)  # 8 bytes past a 16-byte boundary
        with pytest.raises(lib.SidpError) as e:
            lib.sidp_cas_ffn(st.dec.h, 0, [xm], [4], [y])
        assert e.value.code == lib.SIDP_EINVAL
    finally:
        st.close()
