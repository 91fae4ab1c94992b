"""The allocation-free projection (sidp_linear_noalloc) against sidp_linear:
the same kernels and split of K, so the same bits, through the C ABI; two
calls in a row (the second smaller) so the shared scratch keeps the first
call's partials when the second starts; and its argument checks."""

import numpy as np
import pytest
import torch

pytestmark = pytest.mark.gpu


def _case(lib, h, m, n, k, epi, seed):
    dev = torch.device("cuda")
    g = torch.Generator(device=dev).manual_seed(seed)
    x = torch.randn(m, k, device=dev, generator=g).bfloat16()
    if epi == lib.SIDP_EPI_SWIGLU:
        wg = (0.05 * torch.randn(n, k, device=dev, generator=g)).bfloat16()
        wu = (0.05 * torch.randn(n, k, device=dev, generator=g)).bfloat16()
        pk = torch.empty(lib.sidp_packed_bytes(2 * (-(-n // 32) * 32), k), dtype=torch.uint8, device=dev)
        lib.sidp_pack_gate_up(wg, wu, n, k, pk)
    else:
        w = (0.05 * torch.randn(n, k, device=dev, generator=g)).bfloat16()
        pk = torch.empty(lib.sidp_packed_bytes(n, k), dtype=torch.uint8, device=dev)
        lib.sidp_pack_linear(w, n, k, pk)
    bias = (0.1 * torch.randn(n, device=dev, generator=g)).bfloat16() if epi == lib.SIDP_EPI_BF16 else None
    resid = torch.randn(m, n, device=dev, generator=g) if epi == lib.SIDP_EPI_RESID else None
    dt = torch.float32 if epi == lib.SIDP_EPI_RESID else torch.bfloat16
    ref = torch.empty(m, n, device=dev, dtype=dt)
    got = torch.full((m, n), float("nan"), device=dev, dtype=dt)
    lib.sidp_linear(h, x, m, k, pk, n, epi, bias, resid, ref)
    torch.cuda.synchronize()
    return x, pk, bias, resid, ref, got


def test_noalloc_projection_matches_handle_projection_twice(lib):
    import synth
    cfg = synth.get_config("llama70b_layer")
    h = lib.sidp_create(lib.make_config(cfg, 512, 64))
    try:
        s = torch.cuda.current_stream().cuda_stream
        # first call: QKV with bias at 512 rows (the LDS-staged kernel, 3 splits,
        # 60 MiB of partials); then the O projection at 256 rows (4 splits, 32 MiB)
        # and smaller ragged ones, each starting on what the one before left
        cases = [(512, 10240, 8192, lib.SIDP_EPI_BF16, 4), (256, 8192, 8192, lib.SIDP_EPI_RESID, 1),
                 (40, 1000, 520, lib.SIDP_EPI_BF16, 2), (96, 688, 256, lib.SIDP_EPI_SWIGLU, 3)]
        for m, n, k, epi, seed in cases:
            print(f"noalloc case m={m} n={n} k={k} epilogue={epi}", flush=True)
            x, pk, bias, resid, ref, got = _case(lib, h, m, n, k, epi, seed)
            rc = lib.raw_call("sidp_linear_noalloc", x.data_ptr(), m, k, pk.data_ptr(), n, epi,
                              bias.data_ptr() if bias is not None else None,
                              resid.data_ptr() if resid is not None else None, got.data_ptr(), s)
            assert rc == lib.SIDP_OK
            torch.cuda.synchronize()
            a = ref.view(torch.int32 if ref.dtype == torch.float32 else torch.int16).cpu().numpy()
            b = got.view(torch.int32 if got.dtype == torch.float32 else torch.int16).cpu().numpy()
            assert np.array_equal(a, b), (m, n, k, epi)
    finally:
        lib.sidp_destroy(h)


def test_noalloc_projection_rejects_bad_arguments(lib):
    E = lib.SIDP_EINVAL
    dev = torch.device("cuda")
    x = torch.zeros(8, 64, device=dev, dtype=torch.bfloat16)
    pk = torch.zeros(lib.sidp_packed_bytes(64, 64), dtype=torch.uint8, device=dev)
    out = torch.zeros(8, 64, device=dev, dtype=torch.bfloat16)
    p = (x.data_ptr(), pk.data_ptr(), out.data_ptr())
    call = lambda m, k, n, epi, bias=None, resid=None: lib.raw_call(  # noqa: E731
        "sidp_linear_noalloc", p[0], m, k, p[1], n, epi, bias, resid, p[2], None)
    assert call(0, 64, 64, 0) == E          # no rows
    assert call(4097, 64, 64, 0) == E       # past 4096 rows
    assert call(8, 60, 64, 0) == E          # k not a multiple of 8
    assert call(8, 64, 64, 1) == E          # residual epilogue without a residual
    assert call(8, 64, 64, 2, bias=x.data_ptr()) == E  # bias only with the bf16 epilogue
    assert call(8, 64, 64, 3) == E          # no such epilogue
    assert lib.raw_call("sidp_linear_noalloc", None, 8, 64, p[1], 64, 0, None, None, p[2], None) == E
