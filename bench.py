#!/usr/bin/env python3
"""Decode-step benchmark of the Weight-as-a-Service path on one MI355X.

Default workload: an 80-layer Llama-3.1-70B-shaped stack (hidden 8192, 64/8
heads, head_dim 128, FFN 28672, bf16) at batch 256, context lengths uniform in
[1024, 8192], 16-token paged KV. All 80 layers' weights (137 GB) sit in a pool
region of HBM and stream through a 2-slot weight cache on a copy stream while
the previous layer computes. The KV cache fills the HBM left over; layers share
KV regions (layer l uses region l mod R) when there are fewer regions than
layers. Inputs are seeded synthetic tensors already resident in HBM.

Prints one JSON line: decode tokens/s (batch / step time), the roofline of the
dominant kernel (live HIP-event timing inside the timed region), and the
oracle's throughput on the host over a bounded sample.
"""

import argparse
import json
import os
import statistics
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

METRIC = "decode tok/s at B=256 (70B-shape stack); MFMA util %; HBM GB/s"
HBM_PEAK_GBS = 8000.0       # MI355X HBM3E, published
MFMA_BF16_PEAK_TFS = 2500.0  # MI355X dense bf16 MFMA, published

DESCR = {
    "llama70b_stack80": "Llama-3.1-70B-shaped 80-layer stack, weights streamed through a 2-slot HBM cache",
    "qwen25_72b_stack8": "Qwen2.5-72B-shaped 8-layer stack, weights streamed through a 2-slot HBM cache",
    "llama70b_layer": "Llama-3.1-70B-shaped single layer",
    "qwen3_32b_layer": "Qwen3-32B-shaped single layer",
    "tiny_layer": "tiny single layer",
}
# Depth of the model a workload is shaped like: shallower stacks also report
# the per-layer time and the tok/s projected to the model's depth.
MODEL_LAYERS = {"llama70b_stack80": 80, "qwen25_72b_stack8": 80, "llama70b_layer": 80, "qwen3_32b_layer": 64}


def log(msg):
    print(f"[bench] {msg}", file=sys.stderr, flush=True)


def staged_bytes(cfg, layer_bytes, pooling):
    """Bytes of a layer blob a slot fill copies: the whole blob, or its FFN part
    (FFN norm gain, packed gate/up and down projections, 256-byte aligned)."""
    if pooling == "layer":
        return layer_bytes
    H, F = cfg["hidden"], cfg["ffn_dim"]
    r = lambda a, b: -(-a // b) * b  # noqa: E731
    return r(H * 2, 256) + r(r(2 * r(F, 32), 64) * r(H, 64) * 2, 256) + r(r(H, 64) * r(F, 64) * 2, 256)


def algorithmic_work(cfg, B, seq_total, fill_bytes):
    """Bytes and flops each kernel class must move / perform for one launch at
    batch B (seq_total = sum over sequences of attended tokens); a layer's fill
    is two launches that together read and write fill_bytes."""
    H, D, F = cfg["hidden"], cfg["head_dim"], cfg["ffn_dim"]
    Hq, Hkv = cfg["num_q_heads"], cfg["num_kv_heads"]
    QD, KD = Hq * D, Hkv * D
    NQKV = QD + 2 * KD
    kv_tok = 2 * KD * 2  # K and V bytes per token
    w = {
        "norm_attn": (B * H * 4 + H * 2 + B * H * 2, 0),
        "qkv": (NQKV * H * 2 + B * H * 2 + B * NQKV * 2, 2 * B * NQKV * H),
        "rope_append": (B * NQKV * 2 + B * QD * 2 + B * kv_tok, 0),
        "attention": (seq_total * kv_tok + 2 * B * QD * 2, 4 * Hq * D * seq_total),
        # the O projection's reduction also writes the FFN norm's bf16 output
        "o_proj": (H * QD * 2 + B * QD * 2 + 2 * B * H * 4 + H * 2 + B * H * 2, 2 * B * H * QD),
        "norm_mlp": (B * H * 4 + H * 2 + B * H * 2, 0),
        "gate_up": (2 * F * H * 2 + B * H * 2 + B * F * 2, 2 * B * 2 * F * H),
        # and the down projection's reduction writes the next layer's attention-norm output
        "down": (H * F * 2 + B * F * 2 + 2 * B * H * 4 + H * 2 + B * H * 2, 2 * B * H * F),
        "fill": (fill_bytes, 0),  # read + write 2 x fill_bytes per streamed layer, over its fill launches
        "wait_fill": (0, 0),
    }
    return w


def measured_traffic(kernel):
    """HBM bytes per launch of `kernel` from the committed counter summary,
    or None if there is none or the kernel's sources changed since."""
    import glob
    import hashlib
    for path in glob.glob(os.path.join(ROOT, "profiles", "*_traffic.md")):
        text = open(path).read()
        start = text.rfind("```json")
        if start < 0:
            continue
        try:
            rec = json.loads(text[start + 7:text.index("```", start + 7)])
        except ValueError:
            continue
        if rec.get("kernel") != kernel:
            continue
        h = hashlib.sha256()
        try:
            for src in rec["sources"]:
                h.update(open(os.path.join(ROOT, src), "rb").read())
        except OSError:
            return None
        return rec["traffic_bytes_per_launch"] if h.hexdigest() == rec["source_sha256"] else None
    return None


def cpu_baseline_one_core(cfg, weights_for_layer, kv_rows, x_rows, pos_rows, tabs_rows):
    """The oracle on one layer of the same sample, with the calling thread
    pinned to one host core and BLAS limited to one thread; returns tokens/s
    extrapolated to the full stack, the core, and the seconds it took."""
    import numpy as np
    from threadpoolctl import threadpool_limits

    import oracle
    prev = os.sched_getaffinity(0)
    core = min(prev)
    k_np, v_np = kv_rows
    with threadpool_limits(limits=1):
        os.sched_setaffinity(0, {core})
        try:
            t0 = time.perf_counter()
            x = oracle.decode_layer(x_rows.copy(), weights_for_layer(0), cfg, k_np.copy(), v_np.copy(), pos_rows,
                                    tabs_rows, True)
            dt = time.perf_counter() - t0
        finally:
            os.sched_setaffinity(0, prev)
    assert np.all(np.isfinite(x))
    return x.shape[0] / (dt * cfg["num_layers"]), core, dt


def cpu_baseline(cfg, weights_for_layer, kv_rows, x_rows, pos_rows, tabs_rows, n_layers_sample):
    """Times the oracle (as it stands) on a bounded sample: n_layers_sample
    layers for the sampled rows; returns tokens/s extrapolated to the full
    stack and the BLAS thread count it ran with."""
    import numpy as np

    import oracle
    try:
        from threadpoolctl import threadpool_info
        threads = max([i.get("num_threads", 1) for i in threadpool_info() if i.get("user_api") == "blas"] or [1])
    except Exception:
        threads = os.cpu_count() or 1
    k_np, v_np = kv_rows
    x = x_rows.copy()
    t0 = time.perf_counter()
    for l in range(n_layers_sample):
        x = oracle.decode_layer(x, weights_for_layer(l), cfg, k_np.copy(), v_np.copy(), pos_rows, tabs_rows, True)
    dt = time.perf_counter() - t0
    rows = x.shape[0]
    per_layer = dt / n_layers_sample
    assert np.all(np.isfinite(x))
    return rows / (per_layer * cfg["num_layers"]), threads, dt


def cas_leg(dec, cfg, replicas, rows, stream, reps=20):
    """Owner-side Compute-as-a-Service on layer 0: the FFN over `replicas`
    replicas' rows fused into one call, against one call per replica."""
    import torch
    import paper_2605_28095_amd as sidp
    H = cfg["hidden"]
    dev = torch.device("cuda")
    g = torch.Generator(device=dev).manual_seed(7)
    xs = [(0.5 * torch.randn(rows, H, device=dev, generator=g)).to(torch.bfloat16) for _ in range(replicas)]
    ys = [torch.empty(rows, H, device=dev, dtype=torch.float32) for _ in range(replicas)]

    def timed(fn):
        for _ in range(3):
            fn()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        torch.cuda.synchronize()
        e0.record(stream)
        for _ in range(reps):
            fn()
        e1.record(stream)
        torch.cuda.synchronize()
        return e0.elapsed_time(e1) / reps

    fused = timed(lambda: sidp.sidp_cas_ffn(dec.h, 0, xs, [rows] * replicas, ys, stream))
    separate = timed(lambda: [sidp.sidp_cas_ffn(dec.h, 0, [x], [rows], [y], stream) for x, y in zip(xs, ys)])
    dec.sync()
    log(f"CaS FFN, {replicas} x {rows} rows: fused {fused:.3f} ms, one call per replica {separate:.3f} ms")
    return {"replicas": replicas, "rows_per_replica": rows, "layer": 0, "fused_ms": round(fused, 4),
            "per_replica_ms": round(separate, 4), "fusion_speedup": round(separate / fused, 3)}


# MI355X xGMI: 7 links of about 153 GB/s per direction; a rank pulling from its
# d - 1 = 7 owners at once (peak-shifted) sees at most all of them.
XGMI_LINK_GBS = 153.0
XGMI_LINKS = 7


def bth_leg(dec, hidden, pos, bt, stage_bytes, L, batches, stream, reps=3):
    """§4.3 profile: per-layer forward time T(B) from resident steps on the
    first B rows, against the time to fetch one layer's staged weights (the
    emulated same-HBM copy, measured; one and seven xGMI links, modeled).
    B_th is the smallest profiled B with T(B) >= the fetch time."""
    import torch
    import paper_2605_28095_amd as sidp
    layer_ms = []
    for b in batches:
        h = hidden[:b].clone()
        for _ in range(2):
            dec.step(h, pos[:b], bt[:b], sidp.SIDP_RESIDENT, compute=stream)
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        torch.cuda.synchronize()
        e0.record(stream)
        for _ in range(reps):
            dec.step(h, pos[:b], bt[:b], sidp.SIDP_RESIDENT, compute=stream)
        e1.record(stream)
        torch.cuda.synchronize()
        layer_ms.append(e0.elapsed_time(e1) / reps / L)
    # the emulated fetch alone: one layer's staged bytes, pool -> slot, whole chip
    src = torch.empty(stage_bytes, dtype=torch.uint8, device=hidden.device)
    dst = torch.empty_like(src)
    for _ in range(2):
        sidp.sidp_copy(src, dst, stage_bytes, 0, stream)
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    e0.record(stream)
    for _ in range(5):
        sidp.sidp_copy(src, dst, stage_bytes, 0, stream)
    e1.record(stream)
    torch.cuda.synchronize()
    fetch = {"same_hbm_copy": e0.elapsed_time(e1) / 5,
             "xgmi_7_links_modeled": stage_bytes / (XGMI_LINKS * XGMI_LINK_GBS * 1e9) * 1e3,
             "xgmi_1_link_modeled": stage_bytes / (XGMI_LINK_GBS * 1e9) * 1e3}
    del src, dst
    bth = {k: next((b for b, t in zip(batches, layer_ms) if t >= f), None) for k, f in fetch.items()}

    def crossing(f):  # the batch where T(B) reaches f, linear between profiled points
        if layer_ms[0] >= f:
            return float(batches[0])
        for (b0, t0), (b1, t1) in zip(zip(batches, layer_ms), zip(batches[1:], layer_ms[1:])):
            if t0 < f <= t1:
                return b0 + (b1 - b0) * (f - t0) / (t1 - t0)
        return None
    bth_interp = {k: (round(crossing(f), 1) if crossing(f) is not None else None) for k, f in fetch.items()}
    log("B_th profile: " + ", ".join(f"B={b}: {t:.3f} ms/layer" for b, t in zip(batches, layer_ms)))
    log("fetch per layer: " + ", ".join(f"{k} {v:.3f} ms" for k, v in fetch.items()) + f"; B_th {bth}")
    return {"batches": batches, "layer_ms": [round(t, 4) for t in layer_ms],
            "fetch_ms": {k: round(v, 4) for k, v in fetch.items()}, "staged_bytes": stage_bytes, "b_th": bth,
            "b_th_interp": bth_interp,
            "note": "B_th = smallest profiled batch whose resident per-layer time covers the fetch; null: none"}


def tail_trace(engines, batch, requests, max_len, seed=0):
    """Active sequences per engine and iteration of a synthetic offline job:
    each of `engines` engines serves `requests` requests with output lengths
    U[1, max_len] through `batch` continuous-batching lanes, each waiting
    request taking the first lane to free up, so the batch stays full until
    the queue runs dry and then decays. Returns an int64 array [T, engines]."""
    import heapq
    import numpy as np
    rng = np.random.default_rng([seed, 4242])
    lane_ends = []
    for _ in range(engines):
        lanes = [0] * batch
        for n in rng.integers(1, max_len + 1, requests).tolist():
            heapq.heapreplace(lanes, lanes[0] + n)
        lane_ends.append(np.sort(np.array(lanes, np.int64)))
    T = int(max(e[-1] for e in lane_ends))
    # active lanes of engine e at iteration t: lanes whose work ends after t
    return np.stack([batch - np.searchsorted(e, np.arange(T), side="right") for e in lane_ends], axis=1)


def tail_leg(b_th, engines=8, batch=256, requests=None, max_len=2048, window=64, hysteresis=0.5, seed=0):
    """§4.3 mode switching over the tail of a synthetic offline job
    (tail_trace; by default 16 requests per lane): the library's mode choice
    (sidp_mode_update) runs on every iteration's per-engine active counts with
    each B_th estimate."""
    import paper_2605_28095_amd as sidp
    requests = requests or 16 * batch
    active = tail_trace(engines, batch, requests, max_len, seed)
    T = active.shape[0]
    out = {"engines": engines, "batch": batch, "requests_per_engine": requests, "max_output_len": max_len,
           "window": window, "hysteresis": hysteresis, "iterations": T, "by_b_th": {}, "skipped": {}}
    for name, bt in b_th.items():
        if bt is None:
            out["skipped"][name] = "no profiled batch hides this fetch: the job would run in CaS throughout"
            continue
        modes = sidp.mode_schedule(float(bt), hysteresis, window, active.tolist())
        switches = int(sum(1 for a, b in zip(modes, modes[1:]) if a != b))
        first_cas = next((t for t, m in enumerate(modes) if m == sidp.SIDP_MODE_CAS), None)
        out["by_b_th"][name] = {
            "b_th": bt, "was_fraction": round(modes.count(sidp.SIDP_MODE_WAS) / T, 4), "switches": switches,
            "first_cas_iteration": first_cas,
            "mean_active_at_switch": (round(float(active[first_cas].mean()), 1) if first_cas is not None else None)}
        log(f"tail ({name}, B_th {bt}): {100 * modes.count(sidp.SIDP_MODE_WAS) / T:.1f}% of {T} iterations in WaS, "
            f"{switches} switch(es), CaS from iteration {first_cas}")
    return out


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=10)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--workload", default="llama70b_stack80")
    ap.add_argument("--batch", type=int, default=256)
    ap.add_argument("--mode", choices=["streamed", "resident"], default="streamed")
    ap.add_argument("--copy", choices=["background", "burst", "memcpy", "sdma"], default="background")
    ap.add_argument("--pooling", choices=["layer", "ffn"], default="layer",
                    help="stage whole layers, or only their FFN part (attention weights read in place)")
    ap.add_argument("--ranks", type=int, default=0, help="pooling ranks d: layers l with l %% d == rank are owned")
    ap.add_argument("--rank", type=int, default=0)
    ap.add_argument("--cas", type=int, default=0,
                    help="also time the owner-side CaS FFN over this many replicas (0: skip)")
    ap.add_argument("--cas-rows", type=int, default=16, help="rows per CaS replica")
    ap.add_argument("--tail", action="store_true",
                    help="also run the WaS/CaS mode choice over a synthetic job tail with the profiled B_th, "
                         "engines of --batch lanes (implies --bth)")
    ap.add_argument("--bth", action="store_true",
                    help="also profile B_th: the smallest batch whose layer time covers one layer's weight fetch")
    ap.add_argument("--fill-split", type=int, default=25, help="percent of a layer's fill in its first tile")
    ap.add_argument("--fill-loads", type=int, nargs=2, default=[0, 0], metavar=("A", "B"),
                    help="16-byte loads in flight per fill lane in the two tiles (0 0: the batch default)")
    ap.add_argument("--whole-fill-wait", action="store_true",
                    help="a layer waits for its whole fill before it starts (default: each kernel waits for its part)")
    ap.add_argument("--seed", type=int, default=0)
    ap.add_argument("--kv-regions", type=int, default=0, help="0: fill the HBM left after the pool")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-resident-compare", action="store_true")
    ap.add_argument("--copy-calibration", type=int, default=0, metavar="BYTES",
                    help="only copy BYTES once through the library's copy kernel and exit: the known-size "
                         "transfer that scales the HBM traffic counters")
    args = ap.parse_args()

    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py measures one GPU's share of the decode step; runs on several GPUs are not "
              "implemented (each GPU would run this same step on its own batch and pull the layers it "
              "does not own over xGMI).", file=sys.stderr)
        sys.exit(2)

    import numpy as np
    import torch

    import paper_2605_28095_amd as sidp
    import synth

    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    if args.copy_calibration > 0:
        n = args.copy_calibration
        src = torch.full((n,), 1, dtype=torch.uint8, device=dev)
        dst = torch.empty(n, dtype=torch.uint8, device=dev)
        torch.cuda.synchronize()
        sidp.sidp_copy(src, dst, n, 1024)
        torch.cuda.synchronize()
        ok = bool(torch.equal(src, dst))
        log(f"copy calibration: {n} bytes, 1024 workgroups, {'ok' if ok else 'MISMATCH'}")
        sys.exit(0 if ok else 1)
    cfg = synth.get_config(args.workload)
    B, L = args.batch, cfg["num_layers"]
    ctx = synth.context_lengths(cfg, args.seed, B)
    reserve = 1
    need = [-(-(int(c) + reserve) // 16) for c in ctx]
    nblk, maxb = int(sum(need)), int(max(need))
    tables = sidp.sidp_kv_alloc(ctx, reserve, 16, nblk, args.seed, maxb)
    max_seq = int(ctx.max()) + reserve + 16

    config = sidp.make_config(cfg, B, max_seq)
    layer_bytes = sidp.sidp_layer_bytes(config)
    region_pair = 2 * sidp.sidp_kv_region_bytes(config, nblk)
    free, total = torch.cuda.mem_get_info(dev)
    margin = 24 << 30
    if args.kv_regions > 0:
        R = args.kv_regions
    else:
        R = int(min(L, (free - (L + 2) * layer_bytes - margin) // region_pair))
    if R < 1:
        raise SystemExit(f"not enough HBM: free {free / 1e9:.1f} GB, pool {L * layer_bytes / 1e9:.1f} GB")
    log(f"{args.workload}: L={L} B={B} pool {L * layer_bytes / 1e9:.1f} GB, slots {2 * layer_bytes / 1e9:.2f} GB, "
        f"KV {R} regions x {region_pair / 1e9:.2f} GB, free {free / 1e9:.1f} of {total / 1e9:.1f} GB")

    t_setup = time.perf_counter()
    dec = sidp.WaSDecoder(cfg, B, max_seq, nblk, R, device=dev, slots=(args.mode == "streamed"))
    sample_rows = list(range(16))
    sample_layers = min(8, L)
    keep_w = {}
    for l in range(L):
        w = synth.layer_weights(cfg, l, seed=args.seed, device=dev)
        dec.load_layer(l, w)
        torch.cuda.synchronize()
        if l < sample_layers and not args.no_cpu_baseline:
            keep_w[l] = {k: v.view(torch.int16).cpu().numpy().view(np.uint16) for k, v in w.items()}
        del w
    log(f"pool loaded in {time.perf_counter() - t_setup:.1f}s")
    k0, v0 = synth.kv_prefill(cfg, nblk, 0, seed=args.seed, device=dev)
    # the oracle's sample: the sampled rows' blocks, straight from the generator
    if not args.no_cpu_baseline:
        import oracle
        sel = np.concatenate([np.asarray(tables[r][:need[r]]) for r in sample_rows])
        idx = torch.as_tensor(sel, dtype=torch.long, device=dev)
        kv_rows = (oracle.bf16_bits_to_f64(k0.index_select(0, idx).view(torch.int16).cpu().numpy().view(np.uint16)),
                   oracle.bf16_bits_to_f64(v0.index_select(0, idx).view(torch.int16).cpu().numpy().view(np.uint16)))
        width = max(need[r] for r in sample_rows)
        tabs_rows, o = [], 0
        for r in sample_rows:
            tabs_rows.append(list(range(o, o + need[r])) + [-1] * (width - need[r]))
            o += need[r]
    dec.set_k_natural(0, k0)
    dec.v_view()[0].copy_(v0.transpose(-1, -2))
    del k0, v0
    for r in range(1, R):  # every region holds the same content; each layer still reads its own region
        dec.k_view()[r].copy_(dec.k_view()[0])
        dec.v_view()[r].copy_(dec.v_view()[0])
    x0 = synth.hidden_input(cfg, args.seed, device=dev, batch=B)
    hidden = x0.clone()
    pos = torch.tensor(ctx, dtype=torch.int32, device=dev)
    bt = torch.tensor(tables, dtype=torch.int32, device=dev)
    torch.cuda.synchronize()
    log(f"setup done in {time.perf_counter() - t_setup:.1f}s")

    compute = torch.cuda.current_stream(dev)
    copy_stream = torch.cuda.Stream(dev) if args.mode == "streamed" else None
    flags = sidp.SIDP_STREAMED if args.mode == "streamed" else sidp.SIDP_RESIDENT
    if args.copy == "memcpy":
        flags |= sidp.SIDP_COPY_MEMCPY
    elif args.copy == "burst":
        flags |= sidp.SIDP_COPY_BURST
    elif args.copy == "sdma":
        flags |= sidp.SIDP_COPY_SDMA

    dec.set_pooling(sidp.SIDP_POOL_FFN if args.pooling == "ffn" else sidp.SIDP_POOL_LAYER, args.ranks, args.rank)
    sidp.sidp_set_fill_tiles(dec.h, args.fill_split, args.fill_loads[0], args.fill_loads[1],
                             0 if args.whole_fill_wait else 1)
    for i in range(args.warmup):
        dec.step(hidden, pos, bt, flags, compute=compute, copy=copy_stream)
    dec.sync()
    sidp.sidp_timing_collect(dec.h)
    log(f"warmup {args.warmup} steps done")

    seq_total = int(ctx.sum()) + B
    streamed_layers = L - sum(1 for l in range(L) if args.ranks > 0 and l % args.ranks == args.rank)
    fill_bytes = staged_bytes(cfg, layer_bytes, args.pooling)
    work = algorithmic_work(cfg, B, seq_total, fill_bytes)

    def kernel_table(timing, steps):
        table = {}
        for name, (ms, n) in timing.items():
            if n == 0:
                continue
            avg = ms / n
            byts, flops = work[name]
            if name == "fill":  # a layer's fill is several launches that together read and write it once
                byts = int(2 * fill_bytes * streamed_layers * steps / n)
            row = {"launches": n, "ms_per_launch": round(avg, 5), "ms_per_step": round(ms / steps, 4)}
            if avg > 0 and byts > 0:
                row.update({
                    "GB_per_s": round(byts / (avg * 1e-3) / 1e9, 1),
                    "TFLOP_per_s": round(flops / (avg * 1e-3) / 1e12, 1) if flops else None,
                    "hbm_frac": round(byts / (avg * 1e-3) / 1e9 / HBM_PEAK_GBS, 4),
                    "mfma_frac": round(flops / (avg * 1e-3) / 1e12 / MFMA_BF16_PEAK_TFS, 4) if flops else None,
                    "bytes_per_launch": byts,
                })
            table[name] = row
        return table

    # per-class breakdown: a few steps with every kernel class bracketed by HIP
    # events (each pair is a packet on the stream, so the timed region below
    # brackets only the class the roofline line reports)
    breakdown_steps = 3
    sidp.sidp_timing_select(dec.h, sidp.KERNEL_CLASSES)
    for i in range(breakdown_steps):
        dec.step(hidden, pos, bt, flags | sidp.SIDP_TIMING, compute=compute, copy=copy_stream)
    dec.sync()
    kernels = kernel_table(sidp.sidp_timing_collect(dec.h), breakdown_steps)
    compute_classes = [k for k in kernels if k not in ("fill", "wait_fill")]
    dom = max(compute_classes, key=lambda k: kernels[k]["ms_per_step"])

    # timed region: exactly K steps, synchronized on both sides; the dominant
    # class is timed live on its stream
    sidp.sidp_timing_select(dec.h, [dom])
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    w0 = time.perf_counter()
    # an event after every step on the compute stream gives the per-step spread
    ev = [torch.cuda.Event(enable_timing=True) for _ in range(args.steps)]
    e0.record(compute)
    for i in range(args.steps):
        dec.step(hidden, pos, bt, flags | sidp.SIDP_TIMING, compute=compute, copy=copy_stream)
        if i + 1 < args.steps:
            ev[i].record(compute)
    e1.record(compute)
    torch.cuda.synchronize()
    dec.sync()
    wall = time.perf_counter() - w0
    ms_total = e0.elapsed_time(e1)
    marks = [e0] + ev[:args.steps - 1] + [e1]
    step_ms = sorted(marks[i].elapsed_time(marks[i + 1]) for i in range(args.steps))
    ms_per_step = ms_total / args.steps
    value = B / (ms_per_step / 1e3)
    dk = kernel_table(sidp.sidp_timing_collect(dec.h), args.steps)[dom]
    sidp.sidp_timing_select(dec.h, sidp.KERNEL_CLASSES)
    log(f"timed {args.steps} steps: {ms_per_step:.2f} ms/step, {value:.1f} tok/s (wall {wall:.2f}s)")

    traffic = measured_traffic(dom) if args.workload == "llama70b_stack80" and B == 256 else None
    roofline = {"kernel": dom, "bound": "hbm", "achieved": dk["GB_per_s"], "peak": HBM_PEAK_GBS, "unit": "GB/s",
                "frac": dk["hbm_frac"], "traffic": traffic,
                "bytes_per_launch": dk["bytes_per_launch"], "ms_per_launch": dk["ms_per_launch"],
                "launches": dk["launches"]}

    resident_ms = None
    if args.mode == "streamed" and not args.no_resident_compare:
        for i in range(2):
            dec.step(hidden, pos, bt, sidp.SIDP_RESIDENT, compute=compute)
        torch.cuda.synchronize()
        r0, r1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        r0.record(compute)
        nres = max(3, args.steps // 2)
        for i in range(nres):
            dec.step(hidden, pos, bt, sidp.SIDP_RESIDENT, compute=compute)
        r1.record(compute)
        torch.cuda.synchronize()
        resident_ms = r0.elapsed_time(r1) / nres
        log(f"resident (no streaming) {resident_ms:.2f} ms/step")
    dec.sync()

    cpu = None
    if not args.no_cpu_baseline:
        val, threads, dt = cpu_baseline(cfg, lambda l: keep_w[l], kv_rows, x0[sample_rows].double().cpu().numpy(),
                                        ctx[sample_rows], np.asarray(tabs_rows), sample_layers)
        val1, core, dt1 = cpu_baseline_one_core(cfg, lambda l: keep_w[l], kv_rows,
                                                x0[sample_rows].double().cpu().numpy(), ctx[sample_rows],
                                                np.asarray(tabs_rows))
        cpu = {"value": round(val, 3), "unit": "tok/s", "cores": threads, "kind": "oracle",
               "sample": f"{sample_layers} of {L} layers for {len(sample_rows)} of {B} sequences (full contexts), "
                         f"float64 with bf16 storage rounding; {dt:.1f}s; tok/s = rows / (s per layer x {L})",
               "host_cpus": os.cpu_count(), "blas_threads": threads,
               "one_core": {"value": round(val1, 4), "unit": "tok/s", "cores": 1, "core": core,
                            "sample": f"layer 0 for the same {len(sample_rows)} sequences, this thread pinned to "
                                      f"host core {core}, one BLAS thread; {dt1:.1f}s"}}
        log(f"oracle baseline: {val:.3f} tok/s over {dt:.1f}s with {threads} BLAS threads "
            f"({os.cpu_count()} host CPUs); one core: {val1:.4f} tok/s over {dt1:.1f}s")

    cas = cas_leg(dec, cfg, args.cas, args.cas_rows, compute) if args.cas > 0 else None
    bth = None
    if args.bth or args.tail:
        batches = [b for b in (1, 2, 4, 8, 16, 32, 64, 128, 256, 512) if b <= B]
        bth = bth_leg(dec, hidden, pos, bt, fill_bytes, L, batches, compute)

    out = {
        "metric": METRIC, "value": round(value, 2), "unit": "tok/s", "n_gpus": 1, "steps": args.steps,
        "warmup": args.warmup, "ms_per_step": round(ms_per_step, 3), "higher_is_better": True, "scaling": "weak",
        "vs_baseline": None, "dtype": "bf16", "data": "synthetic",
        "config": {
            "workload": f"{args.workload}: {DESCR.get(args.workload, args.workload)}",
            "global_batch": B, "layers": L, "seq_len": f"ctx U[{cfg['ctx_lo']},{cfg['ctx_hi']}], mean {ctx.mean():.0f}",
            "parallelism": "single GPU", "mode": args.mode, "copy": args.copy, "kv_regions": R,
            "layer_bytes": layer_bytes, "pooling": args.pooling, "staged_bytes": fill_bytes,
            "owned_layers": sum(1 for l in range(L) if args.ranks > 0 and l % args.ranks == args.rank),
            "fill": {"first_tile_percent": args.fill_split, "loads": args.fill_loads,
                     "waits": "whole fill" if args.whole_fill_wait else "per part"},
        },
        "roofline": roofline,
        "cpu_baseline": cpu,
        "kernels": kernels,
        "kernels_note": (f"per-class HIP-event timing of {breakdown_steps} steps run before the timed region with every "
                         "class bracketed; the timed region brackets only the roofline kernel's class"),
        "step_ms": {"p10": round(float(np.percentile(step_ms, 10)), 3), "median": round(float(np.median(step_ms)), 3),
                    "p90": round(float(np.percentile(step_ms, 90)), 3),
                    "tok_s_at_median": round(B / (float(np.median(step_ms)) / 1e3), 2)},
        "resident_ms_per_step": round(resident_ms, 3) if resident_ms else None,
        "fill_stall_ms_per_step": kernels["wait_fill"]["ms_per_step"] if "wait_fill" in kernels else None,
    }
    depth = MODEL_LAYERS.get(args.workload)
    if depth and depth != L:
        out["projection"] = {"t_layer_ms": round(ms_per_step / L, 4), "model_layers": depth,
                             "projected_tok_s": round(B / (ms_per_step / L * depth / 1e3), 2),
                             "note": "a projection: this stack's per-layer step time times the model's depth"}
    if cas:
        out["cas"] = cas
    if bth:
        out["bth"] = bth
    if args.tail:
        out["tail"] = tail_leg(bth["b_th_interp"], batch=B)
    print(json.dumps(out), flush=True)
    dec.close()


if __name__ == "__main__":
    main()
