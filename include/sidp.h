/*
 * sidp.h - C ABI of the MI355X Weight-as-a-Service decode step.
 *
 * One GPU's share of SiDP's Weight-as-a-Service mode (arXiv 2605.28095):
 * every layer's weights live in a pool, are copied layer by layer into a ring
 * of two pre-allocated cache slots on a side stream, and the batch's decode
 * tokens run through the layer from its slot while the next layer is being
 * fetched (§4.2 "Asynchronous one-sided reading", "Asynchronous buffer
 * management"; §4.4 "Implementation"). On one GPU the owner's pool is a second
 * region of the same HBM.
 *
 * The layer is a dense decoder block (§2.1): RMSNorm, fused QKV projection
 * (optional bias), optional per-head QK RMSNorm, rotary embedding, append of
 * the new token's key/value to a paged KV cache, grouped-query attention
 * decode, output projection with residual, RMSNorm, gate/up projection with
 * SwiGLU, down projection with residual. One new token per sequence per call
 * (§2.2).
 *
 * Conventions for every entry point:
 *  - Return value: SIDP_OK (0) or a negative SIDP_E* code; no exceptions or
 *    aborts cross the ABI. sidp_strerror() names a code.
 *  - "device" pointers are HIP device memory of the current device; "host"
 *    pointers are ordinary host memory. The caller owns every buffer it
 *    passes; the library never frees caller memory and keeps pointers given
 *    to sidp_pool_init / sidp_kv_attach until sidp_destroy.
 *  - Streams are hipStream_t values passed as void* (NULL = null stream).
 *    Work is enqueued asynchronously; device-side input errors (a position
 *    outside its block table, a block index out of range) are latched in the
 *    handle and reported by sidp_sync.
 *  - bf16 is IEEE bfloat16 stored as 16-bit words; rounding from fp32 is
 *    round-to-nearest-even.
 *  - After SIDP_EHIP a handle is poisoned: later calls return SIDP_ESTATE.
 *  - One handle per host thread; calls on one handle are not thread-safe.
 */
#ifndef SIDP_H
#define SIDP_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* ---- status codes ---- */
#define SIDP_OK          0
#define SIDP_EINVAL     (-1) /* bad argument, unsupported shape, or bad device-side input */
#define SIDP_ENOBLOCKS  (-2) /* paged-KV blocks or block-table width exhausted */
#define SIDP_ESTATE     (-3) /* call out of order, or handle poisoned */
#define SIDP_EHIP       (-4) /* a HIP runtime call failed (sidp_last_hip_error) */
#define SIDP_ENOMEM     (-5) /* library-owned device memory could not be allocated */

/* ---- sidp_decode_step flags ---- */
#define SIDP_RESIDENT      0x0  /* each layer computes straight from its pool blob */
#define SIDP_STREAMED      0x1  /* layers stream through the 2-slot cache ring */
#define SIDP_COPY_MEMCPY   0x2  /* slot fills by hipMemcpyAsync                                  */
#define SIDP_COPY_BURST    0x4  /* slot fills by a full-grid copy kernel                         */
#define SIDP_COPY_SDMA     0x8  /* slot fills by hipMemcpyAsync of kind DeviceToDeviceNoCU: the  */
                                /* DMA engines, no compute units                                 */
                                /* default: a background fill kernel sized to run beside compute */
#define SIDP_DEBUG_POISON  0x10 /* before each fill, write NaN bytes over the slot */
#define SIDP_DEBUG_DELAY   0x20 /* before each fill launch, spin ~200 us on the copy stream */
#define SIDP_TIMING        0x40 /* bracket each kernel class with HIP events (sidp_timing_collect) */

/* ---- kernel classes timed under SIDP_TIMING ---- */
#define SIDP_K_NORM_ATTN  0 /* RMSNorm before attention (first layer of a step) */
#define SIDP_K_QKV        1 /* QKV projection (+bias), split-K partials       */
#define SIDP_K_ROPE       2 /* QKV reduce + QK-norm + RoPE + KV append         */
#define SIDP_K_ATTN       3 /* paged attention (+ partition combine)           */
#define SIDP_K_O          4 /* O projection + residual + RMSNorm before the FFN */
#define SIDP_K_NORM_MLP   5 /* RMSNorm before the FFN when not fused (unused)  */
#define SIDP_K_GATE_UP    6 /* gate/up projection + SwiGLU                     */
#define SIDP_K_DOWN       7 /* down projection + residual (+ next layer's attention RMSNorm) */
#define SIDP_K_FILL       8 /* slot fill (copy stream)                */
#define SIDP_K_WAIT_FILL  9 /* compute stream blocked on a slot fill  */
#define SIDP_NUM_KCLASSES 10

/* ---- sidp_linear epilogues ---- */
#define SIDP_EPI_BF16    0 /* out bf16 [m, n] = x W^T (+ bias)                      */
#define SIDP_EPI_RESID   1 /* out fp32 [m, n] = residual + x W^T (may alias residual) */
#define SIDP_EPI_SWIGLU  2 /* out bf16 [m, f] = silu(x Wg^T) * (x Wu^T), W from sidp_pack_gate_up */

typedef struct sidp_handle sidp_handle;

/* Model shape and limits. All counts > 0 unless stated. */
typedef struct sidp_config {
  int32_t num_layers;    /* L, layers in the stack                                  */
  int32_t hidden;        /* H, multiple of 64                                        */
  int32_t num_q_heads;   /* Hq                                                       */
  int32_t num_kv_heads;  /* Hkv; Hq % Hkv == 0 and Hq / Hkv <= 16                   */
  int32_t head_dim;      /* D: 64 or 128                                             */
  int32_t ffn_dim;       /* F, multiple of 16                                        */
  int32_t qkv_bias;      /* 1: QKV projection has a bias (Qwen2.5 family)            */
  int32_t qk_norm;       /* 1: per-head RMSNorm on q and k before RoPE (Qwen3 family) */
  int32_t block_size;    /* paged-KV tokens per block; must be 16                    */
  int32_t max_batch;     /* largest batch any call will use (sizes scratch)          */
  int32_t max_seq_len;   /* largest position + 1 any call will use (RoPE table)      */
  float rms_eps;         /* RMSNorm epsilon (inside the square root)                 */
  float qk_norm_eps;     /* epsilon of the per-head QK RMSNorm                       */
  float rope_theta;      /* RoPE base; rotate-half pairing (i, i + D/2)              */
} sidp_config;

/* One layer's weights, device pointers to bf16 arrays in nn.Linear layout
 * [out_features, in_features], row-major. Bias and QK-norm pointers are read
 * only when the config enables them (else may be NULL). */
typedef struct sidp_layer_weights {
  const void *w_q;    /* [Hq*D, H]  */
  const void *w_k;    /* [Hkv*D, H] */
  const void *w_v;    /* [Hkv*D, H] */
  const void *w_o;    /* [H, Hq*D]  */
  const void *w_gate; /* [F, H]     */
  const void *w_up;   /* [F, H]     */
  const void *w_down; /* [H, F]     */
  const void *b_q, *b_k, *b_v; /* [Hq*D], [Hkv*D], [Hkv*D] */
  const void *g_attn; /* [H] RMSNorm gain before attention */
  const void *g_mlp;  /* [H] RMSNorm gain before the FFN   */
  const void *g_q, *g_k; /* [D] per-head QK RMSNorm gains  */
} sidp_layer_weights;

/* ---- errors ---- */
const char *sidp_strerror(int code);
/* The hipError_t value behind the last SIDP_EHIP on this handle (0 if none). */
int sidp_last_hip_error(const sidp_handle *h);

/* ---- handle ----
 * sidp_create validates the config (SIDP_EINVAL), binds the handle to the
 * current HIP device, and allocates the library's own device memory:
 * activations for max_batch rows, split-K and attention partials, the RoPE
 * cos/sin table (max_seq_len x D/2, computed on the host in double precision
 * and stored as fp32), the device error word and the fill/consume events of
 * the slot ring. The slot ring is the paper's pre-allocated cache slots with
 * completion notifications (§4.2 "Asynchronous buffer management", §4.4). */
int sidp_create(const sidp_config *cfg, sidp_handle **out);
/* Waits for the handle's outstanding work, frees what sidp_create allocated. */
int sidp_destroy(sidp_handle *h);

/* ---- weight pool and cache slots (§4.1 initialisation; §4.2; §4.4 slots) ----
 * Bytes of one packed layer blob: the pool stride and the size of one slot.
 * Returns 0 for an invalid config. */
size_t sidp_layer_bytes(const sidp_config *cfg);
/* Bytes the pool needs (num_layers blobs, §4.1) and the two cache slots
 * need (§4.2), i.e. num_layers and 2 times sidp_layer_bytes; 0 for an
 * invalid config. Host only. */
size_t sidp_pool_bytes(const sidp_config *cfg);
size_t sidp_slot_bytes(const sidp_config *cfg);
/* Registers caller-owned device memory: `pool` holds num_layers blobs
 * (pool_bytes >= L * sidp_layer_bytes), `slots` holds 2 slots
 * (slots_bytes >= 2 * sidp_layer_bytes; may be NULL/0 if only
 * SIDP_RESIDENT steps will run). Both must be 256-byte aligned.
 * With `layers` (host array of n_layers = num_layers entries, device
 * pointers as in sidp_pool_load_layer) it also puts every layer's weights
 * into the pool: the owner registering its layers (§4.1), equivalent to one
 * sidp_pool_load_layer call per layer on `stream`; with layers NULL,
 * n_layers must be 0 and layers are loaded later, one call each.
 * SIDP_EINVAL for bad memory, n_layers not matching, or a layer's missing
 * pointer (layers before it are loaded). Restarts the slot ring; call it
 * when no decode step is in flight on the handle (after sidp_sync). */
int sidp_pool_init(sidp_handle *h, void *pool, size_t pool_bytes, void *slots, size_t slots_bytes,
                   const sidp_layer_weights *layers, int32_t n_layers, void *stream);
/* Packs one layer's weights (device pointers, layout above) into its pool
 * blob: norm gains, QKV bias, then the QKV, O, interleaved gate/up and down
 * matrices re-laid into the GEMM's fragment order. Asynchronous on `stream`;
 * the sources may be freed once the stream has passed this call. Restarts
 * the slot ring (the slots may hold the layer's old blob): call it only when
 * no decode step is in flight on the handle, i.e. after sidp_sync. */
int sidp_pool_load_layer(sidp_handle *h, int32_t layer, const sidp_layer_weights *w, void *stream);

/* ---- paged KV cache (per-request KV state, §2.2) ----
 * Host-only (no GPU work): builds block tables. Physical blocks
 * [0, num_phys_blocks) are handed out in the order of a Fisher-Yates
 * (Durstenfeld) shuffle driven by splitmix64(seed); sequence b takes the next
 * ceil((ctx_lens[b] + reserve_tokens) / block_size) of them as its logical
 * blocks 0, 1, .... block_tables (host, [batch, max_blocks_per_seq], int32)
 * receives them, padded with -1. Returns SIDP_ENOBLOCKS if the blocks or the
 * table width do not suffice, SIDP_EINVAL for bad sizes. */
int sidp_kv_alloc(int32_t batch, const int32_t *ctx_lens, int32_t reserve_tokens, int32_t block_size,
                  int32_t num_phys_blocks, uint64_t seed, int32_t max_blocks_per_seq, int32_t *block_tables);
/* Bytes of one KV region of the K cache (the V cache has the same size):
 * num_phys_blocks * Hkv * block_size * D * 2. */
size_t sidp_kv_region_bytes(const sidp_config *cfg, int32_t num_phys_blocks);
/* Registers caller-owned KV caches of num_regions regions each. Layer l reads
 * and writes region l % num_regions. Layouts (bf16):
 *   K: [region][block][kv_head][d / 8][token in block][d % 8]
 *   V: [region][block][kv_head][d][token in block]   (transposed per block)
 * Both keep a (block, kv_head) pair's tokens in one contiguous
 * block_size * D * 2-byte piece; the orders inside it are the ones the
 * attention kernel's matrix fragments read as whole contiguous runs.
 * Cached keys are stored after RoPE (and after QK-norm when enabled). */
int sidp_kv_attach(sidp_handle *h, void *k_cache, void *v_cache, int32_t num_phys_blocks, int32_t num_regions);

/* ---- the decode step (§2.2 iteration; §4.2 WaS) ----
 * Runs one decode iteration of all L layers for `batch` sequences.
 *  hidden       device fp32 [batch, H], the residual stream: input token
 *               states, overwritten with the last layer's output.
 *  positions    device int32 [batch]: tokens already cached per sequence; the
 *               new token's k, v are written at that position and attention
 *               covers positions[b] + 1 keys. The caller advances positions.
 *  block_tables device int32 [batch, max_blocks_per_seq] (from sidp_kv_alloc).
 *  flags        SIDP_RESIDENT or SIDP_STREAMED, optionally | one SIDP_COPY_* engine
 *               and the SIDP_DEBUG_* bits.
 *  compute      stream for the layer kernels.
 *  copy         stream for slot fills (STREAMED only; must differ from compute).
 * STREAMED keeps a ring of 2 slots: layer g (counted across calls) computes
 * from slot g % 2, each of its kernels after the part of the fill it reads
 * has landed (see sidp_plan); the fill of layer g + 2 waits
 * for layer g's compute to release the slot. The copy stream thus runs two
 * layers ahead, into the next call's first layers too. RESIDENT and STREAMED
 * give bit-identical results (the paper's modes change only where weights
 * live, §4.1). Returns without waiting for the GPU.
 * Calls that use the handle's own buffers (decode steps, sidp_cas_ffn,
 * sidp_linear, sidp_attention) are ordered as if on one stream: a call on a
 * compute stream other than the previous call's first waits (on the device)
 * for the previous call's work to finish. */
int sidp_decode_step(sidp_handle *h, float *hidden, const int32_t *positions, const int32_t *block_tables,
                     int32_t max_blocks_per_seq, int32_t batch, int32_t flags, void *compute, void *copy);
/* Waits for all work the handle enqueued on both streams; returns
 * SIDP_EINVAL if a kernel latched a device-side input error since the last
 * sync (and clears it), SIDP_EHIP on an asynchronous HIP error. */
int sidp_sync(sidp_handle *h);

/* ---- timing ----
 * Waits for every event pair recorded under SIDP_TIMING since the last
 * collect and returns, per kernel class, the summed elapsed milliseconds
 * (ms[SIDP_NUM_KCLASSES], host) and the number of timed launches
 * (launches[SIDP_NUM_KCLASSES], host); then recycles the events. Each pair
 * brackets one layer's launches of that class on the stream they run on:
 * the attention's pair takes its times from the attention kernels' own
 * dispatches, the other classes' are event records around their launches. */
int sidp_timing_collect(sidp_handle *h, double *ms, int32_t *launches);
/* Which kernel classes SIDP_TIMING brackets: bit i selects class i
 * (SIDP_K_*); all by default. An event record is a packet on the stream
 * that delays the next kernel by a few microseconds, so a caller timing one
 * class leaves the others unbracketed (timing the attention alone adds one
 * such packet per layer, before the attention). SIDP_EINVAL for bits past
 * SIDP_NUM_KCLASSES. */
int sidp_timing_select(sidp_handle *h, uint32_t class_mask);

/* ---- pooling ----
 * What the weight cache stages, and which layers this rank owns (§4.1: each
 * rank keeps the FFN weights of the layers it owns in its pool and reads the
 * others from their owners; attention weights stay with every replica).
 *   mode  SIDP_POOL_LAYER: a streamed layer's whole blob is staged (default);
 *         SIDP_POOL_FFN: only its FFN part (norm gain, gate/up, down) is
 *         staged, its attention part is read from the pool in place.
 *   ranks, rank: with ranks > 0, layer l with l % ranks == rank is owned and
 *         computed straight from the pool in streamed steps (no slot, no
 *         copy); ranks = 0 owns no layer (default). 0 <= rank < ranks.
 * On one GPU the pool stands in for both this rank's pool and the owners' pools
 * of the layers it streams. Restarts the slot ring; call it only when no step
 * is in flight on the handle (after sidp_sync). SIDP_EINVAL on bad arguments. */
#define SIDP_POOL_LAYER 0
#define SIDP_POOL_FFN   1
int sidp_set_pooling(sidp_handle *h, int32_t mode, int32_t ranks, int32_t rank);

/* ---- fill tiles (§4.2 "Asynchronous one-sided reading": a layer is fetched
 * in tensor tiles, each with its own completion notification) ----
 * A streamed layer's fill is two tiles on the copy stream: the first
 * `first_tile_percent` percent of the staged bytes as soon as the slot is
 * released, the rest once the previous layer's attention half has been
 * issued, so that it runs beside that layer's projections. loads_a and
 * loads_b are the 16-byte loads each lane of the fill kernel keeps in flight
 * in the two tiles (2, 4 or 8; 0 = the default for the step's batch: 8 and 8
 * below 160 rows; 8 and 4 below 384 rows with part waits; else 4 and 2).
 * part_waits = 1: each kernel that reads
 * the slot waits only for the fill launch holding its weights (see
 * sidp_plan), so the compute stream does not stall on the rest of the fill;
 * 0: a layer waits for its whole fill before its first kernel. Defaults:
 * 25, 0, 0, 1. Takes effect from the next decode step. SIDP_EINVAL for a
 * percent outside [0, 100], another load count, or part_waits not 0 or 1. */
int sidp_set_fill_tiles(sidp_handle *h, int32_t first_tile_percent, int32_t loads_a, int32_t loads_b,
                        int32_t part_waits);

/* ---- Compute-as-a-Service, owner side ----
 * §4.3: in the small-batch tail, non-owner replicas send their FFN inputs to
 * the layer's owner, which concatenates them with its own rows in a staging
 * buffer, runs the FFN once over all of them, splits the output along the same
 * row boundaries and returns each slice; replicas running dummy iterations
 * send nothing and get no compute. This handle is the owner: it computes
 * layer `layer`'s FFN from its pool (the layer must be loaded).
 *   x_in[r]  device, bf16 [rows[r], hidden] row-major, 16-byte aligned:
 *            replica r's FFN input (the RMSNorm output before the FFN).
 *   rows[r]  host; 0 marks a dummy replica: x_in[r], y_out[r] are not touched.
 *   y_out[r] device, fp32 [rows[r], hidden], 16-byte aligned: receives
 *            down(silu(x Wg^T) * (x Wu^T)), the FFN output without the
 *            residual, which the replica adds to its residual stream (as
 *            the streamed step's down projection does).
 * Rows are processed in replica order; sum of rows <= max_batch and
 * n_replicas <= SIDP_CAS_MAX_REPLICAS, else SIDP_EINVAL. On one GPU the
 * transfers into the staging buffer and back are device copies. The math is
 * the decode step's FFN; the fused projections split K by the total row
 * count, so a row's output can differ from a per-replica run in fp32
 * summation order only. Uses the handle's activation buffers: do not overlap
 * with a decode step on the same handle. */
#define SIDP_CAS_MAX_REPLICAS 16
int sidp_cas_ffn(sidp_handle *h, int32_t layer, int32_t n_replicas, const void *const *x_in, const int32_t *rows,
                 void *const *y_out, void *stream);

/* ---- the slot-ring plan (host only) ----
 * The order in which sidp_decode_step issues its operations on the two
 * streams, for `steps` streamed calls of num_layers layers with 2 slots, on
 * rank `rank` of `ranks` pooling ranks (ranks = 0: no owned layers; see
 * sidp_set_pooling). Streamed layers are counted across calls by g (g-th
 * non-owned layer instance): layer g computes from slot g % 2 while layer
 * g + 1 is copied into the other slot as two tiles (§4.2 "tensor tiles", each
 * with its notification): tile A once layer g - 1 has released the slot, tile
 * B once layer g's attention half has been issued, so that it runs beside
 * layer g's projections. Each kernel that reads the slot waits only for the
 * tile holding the last byte it reads (unless sidp_set_fill_tiles asks for
 * whole-fill waits): the attention half for the bytes below W_o (op 2), the
 * O projection and its fused norm for those below the gate/up weights, the
 * FFN for the whole fill (both inside op 5). Each op is 3 int32
 * {kind, g, slot}; kinds:
 *   0 copy tile A of layer g          1 copy tile B of layer g, then mark filled
 *   2 compute waits for the attention half's part of the fill
 *   3 attention half of layer g
 *   4 mark attention half issued      5 projection half of layer g
 *   6 mark slot released              7 copy stream waits for the release
 *   8 copy stream waits for the attention half
 *   9 an owned layer computed from the pool; g = call * num_layers + layer, slot -1.
 * ops (host, 3 * *n_ops int32) receives up to *n_ops ops; on return *n_ops is
 * the number written. SIDP_EINVAL if the capacity is too small or the
 * arguments are bad. */
int sidp_plan(int32_t num_layers, int32_t steps, int32_t ranks, int32_t rank, int32_t *ops, int32_t *n_ops);

/* ---- Peak-shifted pull order (host only; §4.2 "Peak shifting") ----
 * With d = `ranks` ranks pooling their weights (layer l owned by rank l mod d,
 * §4.1), the order in which rank `rank` pulls the layers it does not own
 * during one decode iteration: layers form cycles of d consecutive indices,
 * and in the cycle starting at layer c the rank walks c + rank, c + rank + 1,
 * ... with wrap-around inside the cycle, skipping its own layer. So the k-th
 * pulls of the d ranks in a full cycle all read different owners. Writes
 * (layer, owner) pairs to `pairs` (host int32 [2 * *n], caller-owned; *n is
 * the capacity in pairs on entry, the count on return, num_layers - ceil
 * (num_layers / d) at most). This is the order a multi-GPU reader would issue
 * its one-sided pulls in; on one GPU nothing is pulled. SIDP_EINVAL for
 * num_layers < 1, ranks < 1, rank outside [0, ranks), a null n, a too-small
 * capacity or a null pairs with a non-empty order. */
int sidp_peak_shift_plan(int32_t num_layers, int32_t ranks, int32_t rank, int32_t *pairs, int32_t *n);

/* ---- WaS / CaS mode choice (host only; §4.3 "Consistent mode switching") ----
 * The job orchestrator picks one mode for every engine of the group, so all
 * ranks agree on each layer's communication pattern. WaS stays while the
 * effective batch (mean active sequences over the group's engines, idle ones
 * counted as 0) is at least b_th, the smallest batch whose forward time hides
 * a layer's weight fetch (from offline profiling, e.g. bench.py --bth); after
 * `window` consecutive iterations below b_th the group switches to CaS, and
 * back to WaS only after `window` consecutive iterations at or above
 * b_th * (1 + hysteresis). A decision applies from the next iteration.
 * sidp_mode_update takes iteration t's per-engine active counts
 * (`active`, host int32 [n_engines], each >= 0), advances `state` (caller
 * owned; all zeros = WaS, the job's start) and writes the mode iteration t + 1
 * runs in to *mode. SIDP_EINVAL for null pointers, n_engines < 1, a negative
 * count, b_th <= 0 or NaN, hysteresis < 0, window < 1 or a state whose mode is
 * neither value; the state is then unchanged. */
#define SIDP_MODE_WAS 0
#define SIDP_MODE_CAS 1
typedef struct {
  float b_th;
  float hysteresis;
  int32_t window;
} sidp_mode_policy;
typedef struct {
  int32_t mode; /* SIDP_MODE_WAS or SIDP_MODE_CAS */
  int32_t run;  /* consecutive iterations the switching condition has held */
} sidp_mode_state;
int sidp_mode_update(const sidp_mode_policy *policy, sidp_mode_state *state, int32_t n_engines, const int32_t *active,
                     int32_t *mode);

/* ---- failure injection (tests of the error contract) ----
 * Makes the next HIP runtime call that the handle checks fail with
 * `hip_error` (a non-zero hipError_t value) before reaching the runtime, as
 * if the runtime had returned it: that call returns SIDP_EHIP,
 * sidp_last_hip_error reports hip_error, and the handle is poisoned (later
 * calls return SIDP_ESTATE; sidp_destroy still frees it). No GPU work is
 * faulted. SIDP_EINVAL for hip_error 0. */
int sidp_debug_inject_hip_error(sidp_handle *h, int32_t hip_error);

/* ---- single kernels, for parity checks and reuse ----
 * All enqueue on `stream` and return immediately. */

/* RMSNorm (K1/K6): out[r] = bf16(x[r] / sqrt(mean(x[r]^2) + eps) * gain).
 * x device fp32 [rows, n]; gain device bf16 [n]; out device bf16 [rows, n];
 * n multiple of 4. */
int sidp_rmsnorm(const float *x, const void *gain, float eps, void *out, int32_t rows, int32_t n, void *stream);

/* The launch sidp_linear, sidp_linear_noalloc and the decode step make for
 * the projection out[m, n] = x[m, k] W[n, k]^T with `epilogue` on a GPU with
 * `num_cus` compute units (host only, no device call). kernel: 0 = weights
 * streamed into registers by each 128-row block, 1 = 256-row workgroups whose
 * weight tiles are staged once in LDS (taken where kernel 0 would run one
 * unsplit round on under three quarters of the CUs). waves: per workgroup (4,
 * 7 or 8). rows_per_workgroup: 32, 64, 128 or 256. splits: the split-K count
 * (fp32 partials reduced in split order). workgroups: the grid launched.
 * ws_bytes: bytes of partials (0 without a split). All outputs host,
 * caller-owned. SIDP_EINVAL for a null output, m < 1, n < 1, k < 8 or not a
 * multiple of 8, n or k above 2^24, num_cus < 1, an unknown epilogue, or
 * sizes past the kernels' 32-bit buffer offsets. */
int sidp_linear_plan(int32_t m, int32_t n, int32_t k, int32_t epilogue, int32_t num_cus, int32_t *kernel,
                     int32_t *waves, int32_t *rows_per_workgroup, int32_t *splits, int32_t *workgroups,
                     uint64_t *ws_bytes);

/* Bytes of a matrix [n, k] packed for sidp_linear (n padded to 64, k to 64). */
size_t sidp_packed_bytes(int32_t n, int32_t k);
/* Packs W (device bf16 [n, k], nn.Linear layout) into `packed`
 * (device, sidp_packed_bytes(n, k) bytes, 256-byte aligned). */
int sidp_pack_linear(const void *w, int32_t n, int32_t k, void *packed, void *stream);
/* Packs gate and up (device bf16 [f, k] each) interleaved 32 rows at a time
 * for SIDP_EPI_SWIGLU; `packed` needs sidp_packed_bytes(2 * f32, k) bytes
 * where f32 = f rounded up to 32. */
int sidp_pack_gate_up(const void *w_gate, const void *w_up, int32_t f, int32_t k, void *packed, void *stream);
/* Dense projection on MFMA: x device bf16 [m, k] row-major times packed W^T.
 * m <= max_batch of the handle; n = output columns (for SWIGLU: f).
 * bias: device bf16 [n] or NULL (EPI_BF16 only); residual: device fp32 [m, n]
 * (EPI_RESID only; may equal out). Uses the handle's split-K scratch. */
int sidp_linear(sidp_handle *h, const void *x, int32_t m, int32_t k, const void *packed, int32_t n,
                int32_t epilogue, const void *bias, const float *residual, void *out, void *stream);

/* ---- the projection without allocation ----
 * For callers that cannot allocate device memory (code under HIP graph
 * capture, serving loops that forbid allocation): the projection of
 * sidp_linear without a handle, on the current device. Same arguments,
 * layouts and results as sidp_linear, bit for bit (the same kernels and the
 * same split of K); m <= 4096. Allocates nothing: the split-K partials go to
 * a scratch array of SIDP_NOALLOC_SCRATCH_BYTES that the library's code
 * object holds in each device's memory from module load until the process
 * ends (64 MiB: the most any split needs on a 256-CU MI355X, where the
 * splits x row blocks x column blocks of a launch stay within the CU count
 * and a workgroup's fp32 partial block is at most 256 x 256). SIDP_EINVAL
 * for bad arguments and when this shape's partials would outgrow the scratch
 * (possible only on a device with more CUs); SIDP_EHIP if the runtime fails.
 * Every call on a device shares that device's scratch, and nothing in it must
 * start at zero (each split writes its partials before they are summed);
 * calls that overlap in time on one device (on different streams) race. */
#define SIDP_NOALLOC_SCRATCH_BYTES (64u << 20)
int sidp_linear_noalloc(const void *x, int32_t m, int32_t k, const void *packed, int32_t n, int32_t epilogue,
                        const void *bias, const float *residual, void *out, void *stream);

/* Slot mapping (K9): slots[b] = bt[b][p / bs] * bs + p % bs, p = positions[b];
 * device int32 arrays. An entry out of range yields -1 and latches
 * SIDP_EINVAL for sidp_sync. */
int sidp_slot_mapping(sidp_handle *h, const int32_t *positions, const int32_t *block_tables,
                      int32_t max_blocks_per_seq, int32_t batch, int32_t *slots, void *stream);
/* QK-norm (when configured) + RoPE + KV append for one layer's KV region:
 * qkv device bf16 [batch, (Hq + 2 Hkv) D] (q heads, then k heads, then v
 * heads); q_out device bf16 [batch, Hq, D] receives the rotated queries; the
 * rotated keys and the values are written into region `region` of the attached
 * caches at each sequence's position. g_q/g_k: device bf16 [D] or NULL. */
int sidp_rope_append(sidp_handle *h, const void *qkv, const int32_t *positions, const int32_t *block_tables,
                     int32_t max_blocks_per_seq, int32_t batch, const void *g_q, const void *g_k,
                     int32_t region, void *q_out, void *stream);
/* Paged GQA decode attention (K4) over region `region`: for each sequence b
 * and query head h, softmax(q K^T / sqrt(D)) V over tokens [0, positions[b]]
 * of KV head h / (Hq / Hkv). q device bf16 [batch, Hq, D]; out device bf16
 * [batch, Hq, D]. */
int sidp_attention(sidp_handle *h, const void *q, int32_t region, const int32_t *positions,
                   const int32_t *block_tables, int32_t max_blocks_per_seq, int32_t batch, void *out,
                   void *stream);
/* Device-to-device copy by the library's copy kernel (the slot-fill engine),
 * using `grid` workgroups (0 = default). src, dst 16-byte aligned. */
int sidp_copy(const void *src, void *dst, size_t bytes, int32_t grid, void *stream);

#ifdef __cplusplus
}
#endif
#endif /* SIDP_H */
