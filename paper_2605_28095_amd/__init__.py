"""Python binding of libsidp, the MI355X Weight-as-a-Service decode step.

Argument marshalling only: every step of the decode path runs in the HIP
library (paper_2605_28095_amd/_lib/libsidp.so, built by build.py). Functions
carry the C names; a non-zero status raises SidpError. Pointer arguments
accept an int address or any object with .data_ptr() (a torch tensor);
streams accept an int handle or an object with .cuda_stream.

Importing this module loads the library and fails loudly if it is not built.
"""

import ctypes
import os

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "_lib", "libsidp.so")

SIDP_OK = 0
SIDP_EINVAL = -1
SIDP_ENOBLOCKS = -2
SIDP_ESTATE = -3
SIDP_EHIP = -4
SIDP_ENOMEM = -5

SIDP_RESIDENT = 0x0
SIDP_STREAMED = 0x1
SIDP_COPY_MEMCPY = 0x2
SIDP_COPY_BURST = 0x4
SIDP_COPY_SDMA = 0x8
SIDP_DEBUG_POISON = 0x10
SIDP_DEBUG_DELAY = 0x20
SIDP_TIMING = 0x40

KERNEL_CLASSES = ["norm_attn", "qkv", "rope_append", "attention", "o_proj", "norm_mlp", "gate_up", "down", "fill",
                  "wait_fill"]

SIDP_EPI_BF16 = 0
SIDP_EPI_RESID = 1
SIDP_EPI_SWIGLU = 2

SIDP_NOALLOC_SCRATCH_BYTES = 64 << 20  # sidp_linear_noalloc's per-device scratch

PLAN_OPS = {0: "fill_a", 1: "fill_b", 2: "wait_fill", 3: "attn", 4: "mid", 5: "proj", 6: "done", 7: "wait_done",
            8: "wait_mid", 9: "local"}

SIDP_POOL_LAYER = 0
SIDP_POOL_FFN = 1

EXPORTED = [
    "sidp_strerror", "sidp_last_hip_error", "sidp_create", "sidp_destroy", "sidp_layer_bytes",
    "sidp_pool_bytes", "sidp_slot_bytes",
    "sidp_pool_init", "sidp_pool_load_layer", "sidp_kv_alloc", "sidp_kv_region_bytes", "sidp_kv_attach",
    "sidp_decode_step", "sidp_sync", "sidp_plan", "sidp_peak_shift_plan", "sidp_rmsnorm", "sidp_packed_bytes", "sidp_pack_linear",
    "sidp_pack_gate_up", "sidp_linear", "sidp_slot_mapping", "sidp_rope_append", "sidp_attention", "sidp_copy",
    "sidp_timing_collect", "sidp_set_pooling", "sidp_cas_ffn", "sidp_timing_select", "sidp_mode_update",
    "sidp_set_fill_tiles", "sidp_debug_inject_hip_error", "sidp_linear_noalloc", "sidp_linear_plan",
]

SIDP_CAS_MAX_REPLICAS = 16


class SidpError(RuntimeError):
    def __init__(self, code, where):
        self.code = code
        super().__init__(f"{where}: {code} ({strerror(code)})")


class sidp_config(ctypes.Structure):
    _fields_ = [(n, ctypes.c_int32) for n in (
        "num_layers", "hidden", "num_q_heads", "num_kv_heads", "head_dim", "ffn_dim", "qkv_bias", "qk_norm",
        "block_size", "max_batch", "max_seq_len")] + [
        ("rms_eps", ctypes.c_float), ("qk_norm_eps", ctypes.c_float), ("rope_theta", ctypes.c_float)]


class sidp_mode_policy(ctypes.Structure):
    _fields_ = [("b_th", ctypes.c_float), ("hysteresis", ctypes.c_float), ("window", ctypes.c_int32)]


class sidp_mode_state(ctypes.Structure):
    _fields_ = [("mode", ctypes.c_int32), ("run", ctypes.c_int32)]


SIDP_MODE_WAS = 0
SIDP_MODE_CAS = 1


class sidp_layer_weights(ctypes.Structure):
    _fields_ = [(n, ctypes.c_void_p) for n in (
        "w_q", "w_k", "w_v", "w_o", "w_gate", "w_up", "w_down", "b_q", "b_k", "b_v", "g_attn", "g_mlp",
        "g_q", "g_k")]


def _load():
    if not os.path.exists(LIB_PATH):
        raise ImportError(f"{LIB_PATH} is not built; run python paper_2605_28095_amd/build.py "
                          "(or __graft_entry__.build()) first")
    return ctypes.CDLL(LIB_PATH)


_lib = _load()

_P = ctypes.c_void_p
_I = ctypes.c_int32
_Z = ctypes.c_size_t
_PI = ctypes.POINTER(ctypes.c_int32)
_sigs = {
    "sidp_strerror": (ctypes.c_char_p, [ctypes.c_int]),
    "sidp_last_hip_error": (ctypes.c_int, [_P]),
    "sidp_create": (ctypes.c_int, [ctypes.POINTER(sidp_config), ctypes.POINTER(_P)]),
    "sidp_destroy": (ctypes.c_int, [_P]),
    "sidp_layer_bytes": (_Z, [ctypes.POINTER(sidp_config)]),
    "sidp_pool_bytes": (_Z, [ctypes.POINTER(sidp_config)]),
    "sidp_slot_bytes": (_Z, [ctypes.POINTER(sidp_config)]),
    "sidp_pool_init": (ctypes.c_int, [_P, _P, _Z, _P, _Z, ctypes.POINTER(sidp_layer_weights), _I, _P]),
    "sidp_pool_load_layer": (ctypes.c_int, [_P, _I, ctypes.POINTER(sidp_layer_weights), _P]),
    "sidp_kv_alloc": (ctypes.c_int, [_I, _PI, _I, _I, _I, ctypes.c_uint64, _I, _PI]),
    "sidp_kv_region_bytes": (_Z, [ctypes.POINTER(sidp_config), _I]),
    "sidp_kv_attach": (ctypes.c_int, [_P, _P, _P, _I, _I]),
    "sidp_decode_step": (ctypes.c_int, [_P, _P, _P, _P, _I, _I, _I, _P, _P]),
    "sidp_sync": (ctypes.c_int, [_P]),
    "sidp_plan": (ctypes.c_int, [_I, _I, _I, _I, _PI, _PI]),
    "sidp_peak_shift_plan": (ctypes.c_int, [_I, _I, _I, _PI, _PI]),
    "sidp_set_pooling": (ctypes.c_int, [_P, _I, _I, _I]),
    "sidp_set_fill_tiles": (ctypes.c_int, [_P, _I, _I, _I, _I]),
    "sidp_debug_inject_hip_error": (ctypes.c_int, [_P, _I]),
    "sidp_cas_ffn": (ctypes.c_int, [_P, _I, _I, ctypes.POINTER(_P), _PI, ctypes.POINTER(_P), _P]),
    "sidp_timing_select": (ctypes.c_int, [_P, ctypes.c_uint32]),
    "sidp_rmsnorm": (ctypes.c_int, [_P, _P, ctypes.c_float, _P, _I, _I, _P]),
    "sidp_packed_bytes": (_Z, [_I, _I]),
    "sidp_pack_linear": (ctypes.c_int, [_P, _I, _I, _P, _P]),
    "sidp_pack_gate_up": (ctypes.c_int, [_P, _P, _I, _I, _P, _P]),
    "sidp_linear": (ctypes.c_int, [_P, _P, _I, _I, _P, _I, _I, _P, _P, _P, _P]),
    "sidp_linear_noalloc": (ctypes.c_int, [_P, _I, _I, _P, _I, _I, _P, _P, _P, _P]),
    "sidp_linear_plan": (ctypes.c_int, [_I, _I, _I, _I, _I, _PI, _PI, _PI, _PI, _PI,
                                        ctypes.POINTER(ctypes.c_uint64)]),
    "sidp_slot_mapping": (ctypes.c_int, [_P, _P, _P, _I, _I, _P, _P]),
    "sidp_rope_append": (ctypes.c_int, [_P, _P, _P, _P, _I, _I, _P, _P, _I, _P, _P]),
    "sidp_attention": (ctypes.c_int, [_P, _P, _I, _P, _P, _I, _I, _P, _P]),
    "sidp_copy": (ctypes.c_int, [_P, _P, _Z, _I, _P]),
    "sidp_timing_collect": (ctypes.c_int, [_P, ctypes.POINTER(ctypes.c_double), _PI]),
    "sidp_mode_update": (ctypes.c_int, [ctypes.POINTER(sidp_mode_policy), ctypes.POINTER(sidp_mode_state), _I, _PI,
                                        _PI]),
}
for _name, (_res, _args) in _sigs.items():
    _f = getattr(_lib, _name)
    _f.restype = _res
    _f.argtypes = _args


def _ptr(x):
    """Device (or host) address of a tensor for the C ABI, which takes dense
    row-major buffers: a strided view would be read as if it were dense."""
    if x is None:
        return None
    if isinstance(x, int):
        return x
    if not x.is_contiguous():
        raise ValueError("the C ABI takes contiguous buffers; pass .contiguous()")
    return x.data_ptr()


def _stream(s):
    if s is None:
        return None
    if isinstance(s, int):
        return s
    return s.cuda_stream


def _check(code, where):
    if code != SIDP_OK:
        raise SidpError(code, where)


def strerror(code):
    return _lib.sidp_strerror(code).decode()


sidp_strerror = strerror


def make_config(cfg, max_batch, max_seq_len):
    """sidp_config from a mapping with the model-shape keys."""
    return sidp_config(
        num_layers=cfg["num_layers"], hidden=cfg["hidden"], num_q_heads=cfg["num_q_heads"],
        num_kv_heads=cfg["num_kv_heads"], head_dim=cfg["head_dim"], ffn_dim=cfg["ffn_dim"],
        qkv_bias=int(cfg["qkv_bias"]), qk_norm=int(cfg["qk_norm"]), block_size=cfg["block_size"],
        max_batch=max_batch, max_seq_len=max_seq_len, rms_eps=cfg["rms_eps"],
        qk_norm_eps=cfg["qk_norm_eps"], rope_theta=cfg["rope_theta"])


def sidp_last_hip_error(h):
    return _lib.sidp_last_hip_error(h)


def sidp_create(config):
    h = _P()
    _check(_lib.sidp_create(ctypes.byref(config), ctypes.byref(h)), "sidp_create")
    return h.value


def sidp_destroy(h):
    _check(_lib.sidp_destroy(h), "sidp_destroy")


def sidp_layer_bytes(config):
    return _lib.sidp_layer_bytes(ctypes.byref(config))


def sidp_pool_bytes(config):
    return _lib.sidp_pool_bytes(ctypes.byref(config))


def sidp_slot_bytes(config):
    return _lib.sidp_slot_bytes(ctypes.byref(config))


def _layer_struct(weights):
    return sidp_layer_weights(**{k: _ptr(v) for k, v in weights.items() if k in dict(sidp_layer_weights._fields_)})


def sidp_pool_init(h, pool, pool_bytes, slots, slots_bytes, layers=None, stream=None):
    """Registers the pool and slots; with `layers` (one mapping name -> device
    tensor per layer) also loads every layer into the pool."""
    arr, n = None, 0
    if layers is not None:
        n = len(layers)
        arr = (sidp_layer_weights * max(n, 1))(*[_layer_struct(w) for w in layers])
    _check(_lib.sidp_pool_init(h, _ptr(pool), pool_bytes, _ptr(slots), slots_bytes, arr, n, _stream(stream)),
           "sidp_pool_init")


def sidp_pool_load_layer(h, layer, weights, stream=None):
    """weights: mapping name -> device tensor (names of sidp_layer_weights)."""
    w = _layer_struct(weights)
    _check(_lib.sidp_pool_load_layer(h, layer, ctypes.byref(w), _stream(stream)), "sidp_pool_load_layer")


def sidp_kv_alloc(ctx_lens, reserve_tokens, block_size, num_phys_blocks, seed, max_blocks_per_seq):
    """Host-only block-table allocation; returns a list of rows."""
    n = len(ctx_lens)
    ctx = (ctypes.c_int32 * max(n, 1))(*[int(c) for c in ctx_lens])
    out = (ctypes.c_int32 * max(n * max_blocks_per_seq, 1))()
    _check(_lib.sidp_kv_alloc(n, ctx, reserve_tokens, block_size, num_phys_blocks, ctypes.c_uint64(seed),
                              max_blocks_per_seq, out), "sidp_kv_alloc")
    return [list(out[b * max_blocks_per_seq:(b + 1) * max_blocks_per_seq]) for b in range(n)]


def sidp_kv_region_bytes(config, num_phys_blocks):
    return _lib.sidp_kv_region_bytes(ctypes.byref(config), num_phys_blocks)


def sidp_kv_attach(h, k_cache, v_cache, num_phys_blocks, num_regions):
    _check(_lib.sidp_kv_attach(h, _ptr(k_cache), _ptr(v_cache), num_phys_blocks, num_regions), "sidp_kv_attach")


def sidp_decode_step(h, hidden, positions, block_tables, max_blocks_per_seq, batch, flags, compute, copy=None):
    _check(_lib.sidp_decode_step(h, _ptr(hidden), _ptr(positions), _ptr(block_tables), max_blocks_per_seq, batch,
                                 flags, _stream(compute), _stream(copy)), "sidp_decode_step")


def sidp_sync(h):
    _check(_lib.sidp_sync(h), "sidp_sync")


def sidp_plan(num_layers, steps, ranks=0, rank=0):
    """Ring operations in issue order, as (kind name, g, slot)."""
    cap = 9 * num_layers * steps + 2
    buf = (ctypes.c_int32 * (3 * cap))()
    n = ctypes.c_int32(cap)
    _check(_lib.sidp_plan(num_layers, steps, ranks, rank, buf, ctypes.byref(n)), "sidp_plan")
    return [(PLAN_OPS[buf[3 * i]], buf[3 * i + 1], buf[3 * i + 2]) for i in range(n.value)]


def sidp_linear_plan(m, n, k, epilogue, num_cus=256):
    """The launch a projection gets (host only): kernel (0 registers, 1
    LDS-staged weights), waves and rows per workgroup, split-K count,
    workgroups and bytes of partials."""
    out = [ctypes.c_int32() for _ in range(5)]
    ws = ctypes.c_uint64()
    _check(_lib.sidp_linear_plan(m, n, k, epilogue, num_cus, *[ctypes.byref(o) for o in out], ctypes.byref(ws)),
           "sidp_linear_plan")
    names = ("kernel", "waves", "rows", "splits", "workgroups")
    return dict({nm: o.value for nm, o in zip(names, out)}, ws_bytes=ws.value)


def sidp_peak_shift_plan(num_layers, ranks, rank):
    """Peak-shifted pull order of one rank for one iteration, as (layer, owner)."""
    cap = max(1, num_layers)
    buf = (ctypes.c_int32 * (2 * cap))()
    n = ctypes.c_int32(cap)
    _check(_lib.sidp_peak_shift_plan(num_layers, ranks, rank, buf, ctypes.byref(n)), "sidp_peak_shift_plan")
    return [(buf[2 * i], buf[2 * i + 1]) for i in range(n.value)]


def sidp_mode_update(policy, state, active):
    """Advances `state` (a sidp_mode_state) by one iteration whose engines have
    `active` sequences each; returns the mode of the next iteration."""
    arr = (ctypes.c_int32 * len(active))(*[int(a) for a in active])
    mode = ctypes.c_int32(-1)
    _check(_lib.sidp_mode_update(ctypes.byref(policy), ctypes.byref(state), len(active), arr, ctypes.byref(mode)),
           "sidp_mode_update")
    return mode.value


def mode_schedule(b_th, hysteresis, window, batches):
    """The mode of every iteration of a trace (list of per-engine active
    counts per iteration), the job starting in WaS."""
    pol = sidp_mode_policy(b_th, hysteresis, window)
    st = sidp_mode_state(SIDP_MODE_WAS, 0)
    modes, mode = [], SIDP_MODE_WAS
    for active in batches:
        modes.append(mode)
        mode = sidp_mode_update(pol, st, active)
    return modes


def sidp_set_pooling(h, mode, ranks=0, rank=0):
    _check(_lib.sidp_set_pooling(h, mode, ranks, rank), "sidp_set_pooling")


def sidp_set_fill_tiles(h, first_tile_percent=25, loads_a=0, loads_b=0, part_waits=1):
    _check(_lib.sidp_set_fill_tiles(h, first_tile_percent, loads_a, loads_b, part_waits), "sidp_set_fill_tiles")


def sidp_debug_inject_hip_error(h, hip_error):
    _check(_lib.sidp_debug_inject_hip_error(h, hip_error), "sidp_debug_inject_hip_error")


def sidp_cas_ffn(h, layer, xs, rows, ys, stream=None):
    """Owner-side CaS FFN: xs[r] bf16 [rows[r], H] in, ys[r] fp32 [rows[r], H]
    out; rows[r] == 0 marks a dummy replica (xs[r], ys[r] may be None)."""
    n = len(rows)
    xp = (_P * n)(*[_ptr(x) if x is not None else None for x in xs])
    yp = (_P * n)(*[_ptr(y) if y is not None else None for y in ys])
    rr = (ctypes.c_int32 * n)(*rows)
    _check(_lib.sidp_cas_ffn(h, layer, n, xp, rr, yp, _stream(stream)), "sidp_cas_ffn")


def sidp_rmsnorm(x, gain, eps, out, rows, n, stream=None):
    _check(_lib.sidp_rmsnorm(_ptr(x), _ptr(gain), eps, _ptr(out), rows, n, _stream(stream)), "sidp_rmsnorm")


def sidp_packed_bytes(n, k):
    return _lib.sidp_packed_bytes(n, k)


def sidp_pack_linear(w, n, k, packed, stream=None):
    _check(_lib.sidp_pack_linear(_ptr(w), n, k, _ptr(packed), _stream(stream)), "sidp_pack_linear")


def sidp_pack_gate_up(w_gate, w_up, f, k, packed, stream=None):
    _check(_lib.sidp_pack_gate_up(_ptr(w_gate), _ptr(w_up), f, k, _ptr(packed), _stream(stream)),
           "sidp_pack_gate_up")


def sidp_linear(h, x, m, k, packed, n, epilogue, bias, residual, out, stream=None):
    _check(_lib.sidp_linear(h, _ptr(x), m, k, _ptr(packed), n, epilogue, _ptr(bias), _ptr(residual), _ptr(out),
                            _stream(stream)), "sidp_linear")


def sidp_linear_noalloc(x, m, k, packed, n, epilogue, bias, residual, out, stream=None):
    _check(_lib.sidp_linear_noalloc(_ptr(x), m, k, _ptr(packed), n, epilogue, _ptr(bias), _ptr(residual), _ptr(out),
                                    _stream(stream)), "sidp_linear_noalloc")


def sidp_slot_mapping(h, positions, block_tables, max_blocks_per_seq, batch, slots, stream=None):
    _check(_lib.sidp_slot_mapping(h, _ptr(positions), _ptr(block_tables), max_blocks_per_seq, batch, _ptr(slots),
                                  _stream(stream)), "sidp_slot_mapping")


def sidp_rope_append(h, qkv, positions, block_tables, max_blocks_per_seq, batch, g_q, g_k, region, q_out,
                     stream=None):
    _check(_lib.sidp_rope_append(h, _ptr(qkv), _ptr(positions), _ptr(block_tables), max_blocks_per_seq, batch,
                                 _ptr(g_q), _ptr(g_k), region, _ptr(q_out), _stream(stream)), "sidp_rope_append")


def sidp_attention(h, q, region, positions, block_tables, max_blocks_per_seq, batch, out, stream=None):
    _check(_lib.sidp_attention(h, _ptr(q), region, _ptr(positions), _ptr(block_tables), max_blocks_per_seq, batch,
                               _ptr(out), _stream(stream)), "sidp_attention")


def sidp_copy(src, dst, nbytes, grid=0, stream=None):
    _check(_lib.sidp_copy(_ptr(src), _ptr(dst), nbytes, grid, _stream(stream)), "sidp_copy")


def sidp_timing_select(h, classes):
    """Bracket only the named kernel classes (names from KERNEL_CLASSES) under SIDP_TIMING."""
    mask = 0
    for c in classes:
        mask |= 1 << KERNEL_CLASSES.index(c)
    _check(_lib.sidp_timing_select(h, mask), "sidp_timing_select")


def sidp_timing_collect(h):
    """{kernel class: (total ms, launches)} for the SIDP_TIMING intervals since the last collect."""
    ms = (ctypes.c_double * len(KERNEL_CLASSES))()
    n = (ctypes.c_int32 * len(KERNEL_CLASSES))()
    _check(_lib.sidp_timing_collect(h, ms, n), "sidp_timing_collect")
    return {k: (ms[i], n[i]) for i, k in enumerate(KERNEL_CLASSES)}


def raw_call(name, *args):
    """The C entry point's status code without raising (for error-path tests)."""
    return getattr(_lib, name)(*args)


from .model import WaSDecoder, k_blocks_from_lib, k_blocks_to_lib  # noqa: E402,F401
