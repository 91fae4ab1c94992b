"""Shared set-up for the GPU parity tests: seeded inputs from synth/, laid
out for the library through its binding, and the same inputs handed to the
oracle. Oracle inputs are taken from the generator's tensors, never from
anything the library wrote."""

import numpy as np
import torch

import oracle
import synth


def bits(t):
    """bf16 torch tensor -> numpy uint16 bit patterns (host copy)."""
    return t.detach().contiguous().cpu().view(torch.int16).numpy().view(np.uint16)


def f64(t):
    """bf16 torch tensor -> float64 numpy."""
    return oracle.bf16_bits_to_f64(bits(t))


def bf16_ulp(x):
    """Spacing of bfloat16 numbers at |x| (for |x| >= smallest normal)."""
    ax = np.maximum(np.abs(x), 2.0 ** -126)
    return 2.0 ** (np.floor(np.log2(ax)) - 7)


def assert_bf16_within_ulp(got_bits, want_f64, max_ulp=1, what="", abs_tol=0.0, max_diff_frac=0.02):
    """GPU bf16 output vs the oracle's float64 value rounded to bf16: at most
    max_ulp bf16 spacings apart (fp32 vs fp64 evaluation may round a value
    sitting near a rounding boundary the other way), plus abs_tol for the
    fp32 evaluation error itself where it is not small against the result
    (sums that cancel; see dot_abs_tol)."""
    got = oracle.bf16_bits_to_f64(got_bits)
    want = oracle.round_to_bf16(want_f64)
    assert np.all(np.isfinite(got)), f"{what}: non-finite output"
    diff = np.abs(got - want)
    tol = max_ulp * bf16_ulp(want) * (1 + 1e-12) + abs_tol
    bad = diff > tol
    # A faithful round-to-nearest-even differs from the oracle's rounding only
    # where fp32 and float64 straddle a rounding boundary: rare.
    if (diff > 0).mean() > max_diff_frac:
        raise AssertionError(f"{what}: {(diff > 0).mean():.3%} of elements differ from the oracle's rounding")
    if bad.any():
        i = np.unravel_index(np.argmax(np.where(bad, diff / tol, 0)), diff.shape)
        raise AssertionError(
            f"{what}: {bad.sum()} of {bad.size} elements beyond {max_ulp} ulp; worst at {i}: "
            f"got {got[i]!r} oracle {np.asarray(want_f64)[i]!r} (rounded {want[i]!r}); "
            f"{int((diff > 0).sum())} elements differ at all")


def dot_abs_tol(x, w):
    """Error allowance of fp32-accumulated dot products x W^T: 2^-20 (16 fp32
    ulps) times sum_k |x_k w_k|, the scale every rounding error of the sum is
    relative to. Only matters where the sum cancels to far below that scale."""
    return 2.0 ** -20 * (np.abs(x) @ np.abs(w).T)


def row_rel_err(got, want):
    """Per-row inf-norm relative error max_i |y - y*| / max_i |y*|."""
    got = np.asarray(got, dtype=np.float64)
    want = np.asarray(want, dtype=np.float64)
    return np.max(np.abs(got - want), axis=-1) / np.max(np.abs(want), axis=-1)


def blocks_needed(ctx, reserve, bs=16):
    return [-(-(int(c) + reserve) // bs) for c in ctx]


class Stack:
    """A decoder stack set up on the GPU from seeded inputs.

    The KV content of every region is drawn by synth.kv_prefill in the
    token-major block layout and written into the library's caches in the
    layouts it stores them in (K as [d / 8][token][d % 8] per block, V
    transposed). `kv_natural[r]` keeps the
    generator's tensors for the oracle.
    """

    def __init__(self, cfg, batch=None, seed=0, gains="one", regions=1, ctx=None, reserve=1, slack_blocks=0,
                 device="cuda", gen_device=None, max_seq_len=None, keep_weights=True):
        import paper_2605_28095_amd as sidp
        self.sidp = sidp
        self.cfg = dict(cfg)
        self.batch = batch or cfg["batch"]
        self.seed = seed
        self.gains = gains
        self.device = torch.device(device)
        self.gen_device = gen_device or device
        self.ctx = np.asarray(ctx if ctx is not None else synth.context_lengths(cfg, seed, self.batch), np.int32)
        self.reserve = reserve
        need = blocks_needed(self.ctx, reserve)
        self.nblk = cfg.get("num_phys_blocks") or (sum(need) + slack_blocks)
        self.max_blocks = max(need)
        self.tables = sidp.sidp_kv_alloc(self.ctx, reserve, 16, self.nblk, seed, self.max_blocks)
        self.regions = regions
        self.max_seq_len = max_seq_len or (int(self.ctx.max()) + reserve + 16)
        self.dec = sidp.WaSDecoder(cfg, self.batch, self.max_seq_len, self.nblk, regions, device=device)
        self.weights = []
        for l in range(cfg["num_layers"]):
            w = synth.layer_weights(cfg, l, seed=seed, device=self.gen_device, gains=gains)
            wd = {k: v.to(self.device) for k, v in w.items()}
            self.dec.load_layer(l, wd)
            torch.cuda.synchronize()
            self.weights.append({k: bits(v) for k, v in w.items()} if keep_weights else None)
            del w, wd
        self.kv_natural = []
        for r in range(regions):
            k, v = synth.kv_prefill(cfg, self.nblk, r, seed, device=self.gen_device)
            self.dec.set_k_natural(r, k.to(self.device))
            self.dec.v_view()[r].copy_(v.to(self.device).transpose(-1, -2))
            self.kv_natural.append((k, v))
        self.x0 = synth.hidden_input(cfg, seed, device=self.gen_device, batch=self.batch)
        self.hidden = self.x0.to(self.device).clone()
        self.positions = torch.tensor(self.ctx, dtype=torch.int32, device=self.device)
        self.bt = torch.tensor(self.tables, dtype=torch.int32, device=self.device)
        torch.cuda.synchronize()

    def layer_weights(self, l):
        """Layer l's weights for the oracle: bf16 bit patterns when kept, else
        regenerated and widened to float64 (an exact conversion) on the
        generator's device."""
        if self.weights[l] is not None:
            return self.weights[l]
        w = synth.layer_weights(self.cfg, l, seed=self.seed, device=self.gen_device, gains=self.gains)
        return {k: v.cpu().double().numpy() for k, v in w.items()}

    def reset(self):
        """Restore hidden states and KV caches to the generated inputs."""
        self.hidden.copy_(self.x0.to(self.device))
        for r, (k, v) in enumerate(self.kv_natural):
            self.dec.set_k_natural(r, k.to(self.device))
            self.dec.v_view()[r].copy_(v.to(self.device).transpose(-1, -2))
        torch.cuda.synchronize()

    def oracle_inputs(self, rows):
        """Oracle inputs for a subset of rows: compact per-region caches holding
        only those rows' blocks (in logical order), remapped block tables."""
        rows = list(rows)
        need = blocks_needed(self.ctx[rows], self.reserve)
        sel = np.concatenate([np.asarray(self.tables[r][:n]) for r, n in zip(rows, need)])
        tabs, o = [], 0
        width = max(need)
        for n in need:
            tabs.append(list(range(o, o + n)) + [-1] * (width - n))
            o += n
        idx = torch.as_tensor(sel, dtype=torch.long, device=self.kv_natural[0][0].device)
        kr = [f64(k.index_select(0, idx)) for (k, v) in self.kv_natural]
        vr = [f64(v.index_select(0, idx)) for (k, v) in self.kv_natural]
        x = self.x0[rows].double().cpu().numpy()
        return x, kr, vr, self.ctx[rows], np.asarray(tabs)

    def run_oracle(self, rows, steps=1, round_bf16=True):
        x, kr, vr, pos, tabs = self.oracle_inputs(rows)
        for s in range(steps):
            x = oracle.decode_stack(x, self.layer_weights, self.cfg, kr, vr, pos + s, tabs, round_bf16)
        return x, kr, vr, tabs

    def run_oracle_both(self, rows):
        """One step of the whole stack for `rows` in both oracle evaluations
        (bf16 storage rounding, exact), fetching each layer's weights once."""
        x, kr, vr, pos, tabs = self.oracle_inputs(rows)
        kr2, vr2 = [k.copy() for k in kr], [v.copy() for v in vr]
        xb, xe = x, x.copy()
        R = len(kr)
        for l in range(self.cfg["num_layers"]):
            w = self.layer_weights(l)
            xb = oracle.decode_layer(xb, w, self.cfg, kr[l % R], vr[l % R], pos, tabs, True)
            xe = oracle.decode_layer(xe, w, self.cfg, kr2[l % R], vr2[l % R], pos, tabs, False)
            if (l + 1) % 10 == 0:
                print(f"oracle: {l + 1} of {self.cfg['num_layers']} layers", flush=True)
        return xb, xe

    def close(self):
        self.dec.close()
