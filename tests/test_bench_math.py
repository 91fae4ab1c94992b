"""The byte and flop counts bench.py divides by to report roofline fractions,
checked against figures derived by hand from the shapes and against what the
hardware counters measured for the same launches (CPU only)."""

import numpy as np

import bench
import synth


def _attended(cfg, seed=0):
    # each sequence attends over its cached context plus the new token
    return int(np.sum(synth.context_lengths(cfg, seed, cfg["batch"]).astype(np.int64) + 1))


def test_staged_bytes_ffn_only_is_the_ffn_tail():
    cfg = synth.get_config("llama70b_stack80")
    H, F = 8192, 28672
    # FFN norm gain (16 KB) + gate/up packed (2F rows x H) + down packed (H rows x F), bf16
    want = H * 2 + 2 * F * H * 2 + H * F * 2
    assert want == 1_409_302_528
    assert bench.staged_bytes(cfg, 1_711_308_800, "ffn") == want
    assert bench.staged_bytes(cfg, 1_711_308_800, "layer") == 1_711_308_800


def test_algorithmic_work_70b_b256():
    cfg = synth.get_config("llama70b_stack80")
    B, S = 256, _attended(cfg)
    w = bench.algorithmic_work(cfg, B, S, 1_711_308_800)
    # attention: K and V of every attended token (2 x 8 heads x 128 x 2 B), q in and o out
    assert w["attention"][0] == S * 4096 + 2 * B * 8192 * 2
    assert w["attention"][0] == 4_664_586_240  # the bench workload's figure (contexts from seed 0)
    # QK^T and P.V: 2 flops per multiply-add, 64 query heads x 128 dims per attended token, twice
    assert w["attention"][1] == 4 * 64 * 128 * S
    # gate/up: the 57344 x 8192 packed weights, the normed input, the SwiGLU output
    assert w["gate_up"] == (2 * 28672 * 8192 * 2 + B * 8192 * 2 + B * 28672 * 2, 2 * B * 57344 * 8192)
    assert w["gate_up"][0] == 958_398_464
    # hardware counters (SQ_INSTS_VALU_MFMA_MOPS_BF16 x 512 per dispatch) on this exact launch:
    # gate/up 469,762,048 MOPs, down 234,881,024, QKV 83,886,080, O 67,108,864
    assert w["gate_up"][1] == 469_762_048 * 512
    assert w["down"][1] == 234_881_024 * 512
    assert w["qkv"][1] == 83_886_080 * 512
    assert w["o_proj"][1] == 67_108_864 * 512
    # a layer's fill reads and writes the staged bytes once over two launches
    assert w["fill"][0] == 1_711_308_800


def test_attended_tokens_follow_the_context_recipe():
    cfg = synth.get_config("llama70b_stack80")
    ctx = synth.context_lengths(cfg, 0, 256)
    assert ctx.min() >= 1024 and ctx.max() <= 8192
    assert abs(ctx.mean() - (1024 + 8192) / 2) < 200  # uniform over [1024, 8192]


def test_tail_trace_is_a_draining_continuous_batch():
    a = bench.tail_trace(engines=3, batch=16, requests=200, max_len=64, seed=1)
    T, E = a.shape
    assert E == 3 and a[0].tolist() == [16] * 3
    assert (np.diff(a, axis=0) <= 0).all() and (a >= 0).all()  # nobody joins once the queue is dry
    assert a[-1].max() >= 1  # the last iteration still has work
    # every engine's total work (lane-iterations) is the sum of its requests' lengths
    rng = np.random.default_rng([1, 4242])
    for e in range(E):
        assert a[:, e].sum() == rng.integers(1, 65, 200).sum()
    # greedy assignment: an engine stays full until its queue is empty, so its batch
    # decays over at most one maximum request length
    for e in range(E):
        full_until = int(np.argmax(a[:, e] < 16))
        drained = int(np.argmax(a[:, e] == 0)) if (a[:, e] == 0).any() else T
        assert drained - full_until <= 64


def test_tail_leg_mode_choice_matches_the_oracle():
    from oracle import orchestrator
    bt, W, h = 6.0, 8, 0.5
    a = bench.tail_trace(engines=3, batch=16, requests=200, max_len=64, seed=1)
    want = orchestrator.mode_schedule(a.tolist(), bt, h, W)
    r = bench.tail_leg({"x": bt}, engines=3, batch=16, requests=200, max_len=64, window=W, hysteresis=h, seed=1)
    got = r["by_b_th"]["x"]
    assert r["iterations"] == len(want)
    assert got["was_fraction"] == round(want.count(orchestrator.WAS) / len(want), 4)
    assert got["first_cas_iteration"] == want.index(orchestrator.CAS)
    assert got["switches"] == sum(1 for p, q in zip(want, want[1:]) if p != q) == 1


def test_traffic_record_is_used_only_while_the_kernel_sources_match(tmp_path, monkeypatch):
    """bench.py reports the counted HBM traffic of the roofline kernel from a
    counter summary under profiles/ only while the kernel's sources hash to
    the value recorded with the counters; after any change to them it reports
    none. Checked on a copy of the attention kernel's sources with a record
    written for them."""
    import hashlib
    import json
    import os
    import shutil
    sources = ["paper_2605_28095_amd/csrc/k_attn.hip", "paper_2605_28095_amd/csrc/common.h"]
    root = tmp_path / "repo"
    (root / "profiles").mkdir(parents=True)
    h = hashlib.sha256()
    for src in sources:
        (root / src).parent.mkdir(parents=True, exist_ok=True)
        shutil.copy(os.path.join(bench.ROOT, src), root / src)
        h.update((root / src).read_bytes())
    rec = {"kernel": "attention", "source_sha256": h.hexdigest(), "sources": sources,
           "traffic_bytes_per_launch": 4716188566}
    (root / "profiles" / "attention_x_traffic.md").write_text("# counters\n\n```json\n" + json.dumps(rec) + "\n```\n")
    monkeypatch.setattr(bench, "ROOT", str(root))
    assert bench.measured_traffic("attention") == 4716188566
    assert bench.measured_traffic("gate_up") is None
    with open(root / sources[0], "a") as f:
        f.write("\n")
    assert bench.measured_traffic("attention") is None
