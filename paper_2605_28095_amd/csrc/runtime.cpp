// Host runtime of the Weight-as-a-Service decode step: handle and config,
// the layer blob layout of the weight pool, the two-slot cache ring driven by
// HIP events, the paged-KV block allocator, and the per-layer kernel sequence.
//
// Paper: SiDP (arXiv 2605.28095). §4.2 "Asynchronous one-sided reading": the
// non-owner issues non-blocking device-to-device copies of a layer's weights
// into its local cache ahead of use (a lookahead window). §4.2 "Asynchronous
// buffer management": pre-allocated slots; reserve a slot, issue reads,
// attach a notification the compute waits on right before launch; the slot is
// freed once compute signals done. §4.4: copies on separate streams,
// notifications by events, no CPU barrier. Here the order is static (layers
// are visited in order), so the housekeeper thread becomes two
// hipStreamWaitEvent edges per layer and the ring needs no host thread.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <cstdlib>
#include <cstring>
#include <new>
#include <vector>

#include "../../include/sidp.h"
#include "internal.h"

using namespace sidp;

namespace {

constexpr int kSlots = 2;
constexpr size_t kAlign = 256;
constexpr int64_t kDelayTicks = 20000;  // 200 us of the 100 MHz constant clock
constexpr int kFillPartAPercent = 25;  // share of a layer's fill issued before its predecessor's attention
constexpr int kFillSmallBatch = 160;   // below this many rows both fill tiles keep 8 loads per lane in flight
constexpr int kFillLongBatch = 384;    // from this many rows the projections outlast a gentle tile B
constexpr int kBurstGrid = 512;        // workgroups of the whole-chip burst copy (SIDP_COPY_BURST)

size_t align_up(size_t v, size_t a) { return (v + a - 1) / a * a; }
int round_up_i(int a, int b) { return (a + b - 1) / b * b; }

// A layer's blob: the attention part (norm gain, QK-norm gains, QKV bias, QKV
// and O projections), then the FFN part from `ffn_lo` on (FFN norm gain,
// gate/up, down), so that FFN-only pooling stages one contiguous range.
struct BlobLayout {
  size_t g_attn, g_q, g_k, bias, w_qkv, w_o, ffn_lo, g_mlp, w_gu, w_d, total;
};

int qkv_rows(const sidp_config& c) { return (c.num_q_heads + 2 * c.num_kv_heads) * c.head_dim; }

BlobLayout blob_layout(const sidp_config& c) {
  BlobLayout b;
  size_t o = 0;
  const size_t H = (size_t)c.hidden, D = (size_t)c.head_dim;
  b.g_attn = o; o = align_up(o + H * 2, kAlign);
  b.g_q = o;    o = align_up(o + (c.qk_norm ? D * 2 : 0), kAlign);
  b.g_k = o;    o = align_up(o + (c.qk_norm ? D * 2 : 0), kAlign);
  b.bias = o;   o = align_up(o + (c.qkv_bias ? (size_t)qkv_rows(c) * 2 : 0), kAlign);
  b.w_qkv = o;  o = align_up(o + packed_bytes(qkv_rows(c), c.hidden), kAlign);
  b.w_o = o;    o = align_up(o + packed_bytes(c.hidden, c.num_q_heads * c.head_dim), kAlign);
  b.ffn_lo = o;
  b.g_mlp = o;  o = align_up(o + H * 2, kAlign);
  b.w_gu = o;   o = align_up(o + packed_bytes(2 * round_up_i(c.ffn_dim, 32), c.hidden), kAlign);
  b.w_d = o;    o = align_up(o + packed_bytes(c.hidden, c.ffn_dim), kAlign);
  b.total = o;
  return b;
}

bool config_ok(const sidp_config* c) {
  if (!c) return false;
  if (c->num_layers < 1 || c->hidden < 64 || c->hidden % 64 || c->hidden > (1 << 17)) return false;
  if (c->head_dim != 64 && c->head_dim != 128) return false;
  if (c->num_q_heads < 1 || c->num_kv_heads < 1 || c->num_q_heads % c->num_kv_heads) return false;
  if (c->num_q_heads > 1024 || c->num_layers > 4096) return false;
  if (c->num_q_heads / c->num_kv_heads > 16) return false;
  if (c->ffn_dim < 16 || c->ffn_dim % 16 || c->ffn_dim > (1 << 20)) return false;
  if (c->block_size != 16) return false;
  if (c->max_batch < 1 || c->max_batch > 4096) return false;
  if (c->max_seq_len < 1 || c->max_seq_len > (1 << 20)) return false;
  if (!(c->rms_eps > 0.f) || !(c->rope_theta > 1.f)) return false;
  if (c->qk_norm && !(c->qk_norm_eps > 0.f)) return false;
  // every projection within the GEMM's 32-bit buffer offsets at the largest batch
  const int QD = c->num_q_heads * c->head_dim;
  if (!gemm_fits(c->max_batch, qkv_rows(*c), c->hidden) || !gemm_fits(c->max_batch, c->hidden, QD) ||
      !gemm_fits(c->max_batch, 2 * round_up_i(c->ffn_dim, 32), c->hidden) ||
      !gemm_fits(c->max_batch, c->hidden, c->ffn_dim))
    return false;
  return true;
}

// Ring operations, in host issue order (shared with sidp_plan). Layer g
// (counted across calls) computes from slot g % 2 while layer g + 1 is copied
// into the other slot, in two parts: part A as soon as layer g - 1 has
// released that slot, part B once layer g's attention half has been issued,
// so that it runs beside the projections (MFMA-bound, spare HBM bandwidth).
enum {
  OP_FILL_A = 0,     // copy stream: first part of layer g's blob into slot
  OP_FILL_B = 1,     // copy stream: the rest, then mark the slot filled
  OP_WAIT_FILL = 2,  // compute stream waits for the slot's fill
  OP_ATTN = 3,       // compute: attention half of layer g
  OP_MID = 4,        // compute: mark layer g's attention half issued
  OP_PROJ = 5,       // compute: projection half of layer g
  OP_DONE = 6,       // compute: mark the slot released
  OP_WAIT_DONE = 7,  // copy stream waits for layer g to release its slot
  OP_WAIT_MID = 8,   // copy stream waits for layer g's attention half
  OP_LOCAL = 9,      // compute: a layer this rank owns, straight from the pool (g = step * L + layer)
};
struct RingOp {
  int kind;
  int64_t g;
  int slot;
};

void ring_prologue(int64_t g0, std::vector<RingOp>& ops) {
  ops.push_back({OP_FILL_A, g0, (int)(g0 % kSlots)});
  ops.push_back({OP_FILL_B, g0, (int)(g0 % kSlots)});
}
// first: g is the first streamed layer since pool_init (its neighbour slot was never used).
void ring_layer(int64_t g, bool first, std::vector<RingOp>& ops) {
  const int s = (int)(g % kSlots), n = (int)((g + 1) % kSlots);
  if (!first) ops.push_back({OP_WAIT_DONE, g - 1, n});
  ops.push_back({OP_FILL_A, g + 1, n});
  ops.push_back({OP_WAIT_FILL, g, s});
  ops.push_back({OP_ATTN, g, s});
  ops.push_back({OP_MID, g, s});
  ops.push_back({OP_WAIT_MID, g, s});
  ops.push_back({OP_FILL_B, g + 1, n});
  ops.push_back({OP_PROJ, g, s});
  ops.push_back({OP_DONE, g, s});
}

bool layer_owned(int l, int ranks, int rank) { return ranks > 0 && l % ranks == rank; }

// The operations of one decode step over layers 0 .. L-1. Layers this rank
// owns are computed from the pool (OP_LOCAL, g = step * L + l); the others go
// through the ring, whose counter and started flag carry across steps.
void build_step(int L, int ranks, int rank, int64_t step, int64_t* ring_g, bool* ring_started,
                std::vector<RingOp>& ops) {
  bool any_streamed = false;
  for (int l = 0; l < L; l++) any_streamed |= !layer_owned(l, ranks, rank);
  bool first = false;
  if (any_streamed && !*ring_started) {
    ring_prologue(*ring_g, ops);
    *ring_started = true;
    first = true;
  }
  for (int l = 0; l < L; l++) {
    if (layer_owned(l, ranks, rank)) {
      ops.push_back({OP_LOCAL, step * L + l, -1});
      continue;
    }
    ring_layer((*ring_g)++, first, ops);
    first = false;
  }
}

}  // namespace

struct sidp_handle;
static hipError_t take_injected(sidp_handle* h);

struct sidp_handle {
  sidp_config cfg;
  BlobLayout blob;
  int device = 0, num_cus = 256;
  int last_hip = 0;
  bool poisoned = false;
  // pool and slots (caller-owned)
  uint8_t* pool = nullptr;
  size_t pool_bytes = 0;
  uint8_t* slots = nullptr;
  size_t slots_bytes = 0;
  std::vector<char> loaded;
  // KV caches (caller-owned)
  uint16_t* k_cache = nullptr;
  uint16_t* v_cache = nullptr;
  int nblk = 0, regions = 0;
  // library-owned device memory
  uint16_t *h = nullptr, *qkv = nullptr, *q = nullptr, *o = nullptr, *act = nullptr;
  float* ws = nullptr;
  size_t ws_bytes = 0;
  float* attn_part = nullptr;
  int attn_max_parts = 0;
  int32_t* attn_plan = nullptr;  // attention work list, rebuilt once per decode step
  // The attention-norm gains of every layer ([L][H] bf16, 16 KB per layer at
  // H = 8192), kept resident beside the pool so that layer l's down-projection
  // reduction can apply layer l + 1's norm before layer l + 1's slot is read.
  uint16_t* g_attn_all = nullptr;
  float* cas_y = nullptr;  // owner-side FFN output of the concatenated CaS rows [max_batch][H] fp32
  float *rope_cos = nullptr, *rope_sin = nullptr;
  uint32_t* err = nullptr;
  hipEvent_t filled[kSlots] = {}, consumed[kSlots] = {}, mid[kSlots] = {};
  // A slot's fill is two launches on the copy stream, tiles A and B;
  // tile_a[slot] is recorded after tile A, filled[slot] after tile B. Each
  // kernel that reads the slot waits only for the tile holding the last byte
  // it reads, so the rest of the fill may still run beside it.
  hipEvent_t tile_a[kSlots] = {};
  // Recorded on the compute stream after each call that uses the handle's
  // buffers; a later call on another stream waits for it first.
  hipEvent_t work_done = nullptr;
  bool work_recorded = false;
  int inject_hip = 0;  // sidp_debug_inject_hip_error: the next checked HIP call fails with this code
  int fill_pct = 0;       // percent of the staged range in fill part A
  // 16-byte loads in flight per lane of the background fill. Part A starts when
  // the slot is released and mostly overlaps the next layer's QKV projection and
  // KV append (latency-bound, spare bandwidth), so it may press harder; part B
  // runs beside the projections, which lose more than the fill gains when it does.
  // Below kFillSmallBatch rows a layer computes in less time than its fill takes,
  // so both parts press harder there. 0: the per-batch default of issue_fill;
  // else a fixed count.
  int fill_loads_a = 0, fill_loads_b = 0;
  // 1: each kernel that reads a slot waits only for the fill launch holding
  // its weights; 0: the layer waits for its whole fill before it starts
  int part_waits = 1;
  int step_batch = 0;  // rows of the decode step being issued
  // pooling: which part of a layer is staged, and which layers this rank owns
  int pool_mode = SIDP_POOL_LAYER;
  int ranks = 0, rank = 0;          // layer l is owned (never staged) when ranks > 0 and l % ranks == rank
  std::vector<int> streamed_layers;  // the layers that are staged, in order
  // ring state
  bool ring_started = false;
  int64_t ring_g = 0;  // global index of the next streamed layer
  hipStream_t last_compute = nullptr, last_copy = nullptr;
  bool any_copy = false;
  // SIDP_TIMING: event pairs per kernel class launch, recycled by sidp_timing_collect
  struct TimedPair {
    int cls;
    hipEvent_t a, b;
  };
  std::vector<hipEvent_t> event_pool;
  std::vector<TimedPair> timed;
  bool timing = false;
  uint32_t timing_mask = (1u << SIDP_NUM_KCLASSES) - 1;  // classes SIDP_TIMING brackets
};

static hipError_t take_injected(sidp_handle* h) {
  const hipError_t e = (hipError_t)h->inject_hip;
  h->inject_hip = 0;
  return e;
}

#define HIPCHK(h, expr)                                                      \
  do {                                                                       \
    hipError_t e_ = (h)->inject_hip ? take_injected(h) : (hipError_t)(expr); \
    if (e_ != hipSuccess) {                                                  \
      (h)->last_hip = (int)e_;         \
      (h)->poisoned = true;            \
      return SIDP_EHIP;                \
    }                                  \
  } while (0)

extern "C" {

const char* sidp_strerror(int code) {
  switch (code) {
    case SIDP_OK: return "ok";
    case SIDP_EINVAL: return "invalid argument or device-side input error";
    case SIDP_ENOBLOCKS: return "paged-KV blocks or block-table width exhausted";
    case SIDP_ESTATE: return "call out of order or handle poisoned";
    case SIDP_EHIP: return "HIP runtime error";
    case SIDP_ENOMEM: return "device memory allocation failed";
    default: return "unknown status";
  }
}

int sidp_last_hip_error(const sidp_handle* h) { return h ? h->last_hip : 0; }

size_t sidp_layer_bytes(const sidp_config* cfg) {
  if (!config_ok(cfg)) return 0;
  return blob_layout(*cfg).total;
}

size_t sidp_pool_bytes(const sidp_config* cfg) {
  if (!config_ok(cfg)) return 0;
  return (size_t)cfg->num_layers * blob_layout(*cfg).total;
}

size_t sidp_slot_bytes(const sidp_config* cfg) {
  if (!config_ok(cfg)) return 0;
  return (size_t)kSlots * blob_layout(*cfg).total;
}

static void free_device(sidp_handle* h) {
  void* ptrs[] = {h->h, h->qkv, h->q, h->o, h->act, h->ws, h->attn_part, h->attn_plan, h->g_attn_all, h->cas_y, h->rope_cos, h->rope_sin, h->err};
  for (void* p : ptrs)
    if (p) (void)hipFree(p);
  for (int i = 0; i < kSlots; i++) {
    if (h->filled[i]) (void)hipEventDestroy(h->filled[i]);
    if (h->tile_a[i]) (void)hipEventDestroy(h->tile_a[i]);
    if (h->consumed[i]) (void)hipEventDestroy(h->consumed[i]);
    if (h->mid[i]) (void)hipEventDestroy(h->mid[i]);
  }
  if (h->work_done) (void)hipEventDestroy(h->work_done);
  for (auto& t : h->timed) {
    (void)hipEventDestroy(t.a);
    (void)hipEventDestroy(t.b);
  }
  for (hipEvent_t e : h->event_pool) (void)hipEventDestroy(e);
}

int sidp_create(const sidp_config* cfg, sidp_handle** out) {
  if (!out) return SIDP_EINVAL;
  *out = nullptr;
  if (!config_ok(cfg)) return SIDP_EINVAL;
  sidp_handle* h = new (std::nothrow) sidp_handle();
  if (!h) return SIDP_ENOMEM;
  h->cfg = *cfg;
  h->blob = blob_layout(*cfg);
  h->loaded.assign(cfg->num_layers, 0);
  const sidp_config& c = *cfg;
  auto fail = [&](int code) {
    free_device(h);
    delete h;
    return code;
  };
  if (hipGetDevice(&h->device) != hipSuccess) return fail(SIDP_EHIP);
  if (hipDeviceGetAttribute(&h->num_cus, hipDeviceAttributeMultiprocessorCount, h->device) != hipSuccess)
    return fail(SIDP_EHIP);

  const size_t B = (size_t)c.max_batch, H = (size_t)c.hidden, D = (size_t)c.head_dim;
  const size_t QD = (size_t)c.num_q_heads * D;
  size_t ws = 0;
  for (int m = 1; m <= c.max_batch; m++) {
    ws = std::max(ws, gemm_ws_bytes(m, qkv_rows(c), c.hidden, h->num_cus));
    ws = std::max(ws, gemm_ws_bytes(m, c.hidden, (int)QD, h->num_cus));
    ws = std::max(ws, gemm_ws_bytes(m, 2 * round_up_i(c.ffn_dim, 32), c.hidden, h->num_cus));
    ws = std::max(ws, gemm_ws_bytes(m, c.hidden, c.ffn_dim, h->num_cus));
  }
  h->ws_bytes = ws;
  const int max_seq16 = round_up_i(c.max_seq_len, 16);
  h->attn_max_parts = (max_seq16 + attn_part_tokens() - 1) / attn_part_tokens();
  const size_t part_bytes = attn_ws_bytes(c.max_batch, c.num_q_heads, c.num_kv_heads, c.head_dim, max_seq16);
  struct {
    void** p;
    size_t bytes;
  } allocs[] = {
      {(void**)&h->h, B * H * 2},
      {(void**)&h->qkv, B * (size_t)qkv_rows(c) * 2},
      {(void**)&h->q, B * QD * 2},
      {(void**)&h->o, B * QD * 2},
      {(void**)&h->act, B * (size_t)c.ffn_dim * 2},
      {(void**)&h->ws, std::max<size_t>(ws, 256)},
      {(void**)&h->attn_part, std::max<size_t>(part_bytes, 256)},
      {(void**)&h->attn_plan, attn_plan_bytes(c.max_batch, h->attn_max_parts)},
      {(void**)&h->g_attn_all, (size_t)c.num_layers * H * 2},
      {(void**)&h->cas_y, B * H * 4},
      {(void**)&h->rope_cos, (size_t)c.max_seq_len * (D / 2) * 4},
      {(void**)&h->rope_sin, (size_t)c.max_seq_len * (D / 2) * 4},
      {(void**)&h->err, 256},
  };
  for (auto& a : allocs)
    if (hipMalloc(a.p, a.bytes) != hipSuccess) return fail(SIDP_ENOMEM);
  if (hipMemset(h->err, 0, 256) != hipSuccess) return fail(SIDP_EHIP);

  // RoPE table: angle p * theta^(-2i/D) in double, stored as fp32 cos/sin.
  std::vector<float> cs((size_t)c.max_seq_len * (D / 2)), sn(cs.size());
  for (int p = 0; p < c.max_seq_len; p++)
    for (size_t i = 0; i < D / 2; i++) {
      const double ang = (double)p * std::pow((double)c.rope_theta, -2.0 * (double)i / (double)D);
      cs[(size_t)p * (D / 2) + i] = (float)std::cos(ang);
      sn[(size_t)p * (D / 2) + i] = (float)std::sin(ang);
    }
  if (hipMemcpy(h->rope_cos, cs.data(), cs.size() * 4, hipMemcpyHostToDevice) != hipSuccess) return fail(SIDP_EHIP);
  if (hipMemcpy(h->rope_sin, sn.data(), sn.size() * 4, hipMemcpyHostToDevice) != hipSuccess) return fail(SIDP_EHIP);
  for (int i = 0; i < kSlots; i++) {
    if (hipEventCreateWithFlags(&h->filled[i], hipEventDisableTiming) != hipSuccess) return fail(SIDP_EHIP);
    if (hipEventCreateWithFlags(&h->tile_a[i], hipEventDisableTiming) != hipSuccess) return fail(SIDP_EHIP);
    if (hipEventCreateWithFlags(&h->consumed[i], hipEventDisableTiming) != hipSuccess) return fail(SIDP_EHIP);
    if (hipEventCreateWithFlags(&h->mid[i], hipEventDisableTiming) != hipSuccess) return fail(SIDP_EHIP);
  }
  if (hipEventCreateWithFlags(&h->work_done, hipEventDisableTiming) != hipSuccess) return fail(SIDP_EHIP);
  h->fill_pct = kFillPartAPercent;
  for (int l = 0; l < c.num_layers; l++) h->streamed_layers.push_back(l);
  *out = h;
  return SIDP_OK;
}

int sidp_destroy(sidp_handle* h) {
  if (!h) return SIDP_EINVAL;
  (void)hipDeviceSynchronize();
  free_device(h);
  delete h;
  return SIDP_OK;
}

int sidp_pool_init(sidp_handle* h, void* pool, size_t pool_bytes, void* slots, size_t slots_bytes,
                   const sidp_layer_weights* layers, int32_t n_layers, void* stream) {
  if (!h) return SIDP_EINVAL;
  if (h->poisoned) return SIDP_ESTATE;
  if (layers ? n_layers != h->cfg.num_layers : n_layers != 0) return SIDP_EINVAL;
  const size_t lb = h->blob.total;
  if (!pool || pool_bytes < lb * (size_t)h->cfg.num_layers || ((uintptr_t)pool % kAlign)) return SIDP_EINVAL;
  if (slots && (slots_bytes < lb * kSlots || ((uintptr_t)slots % kAlign))) return SIDP_EINVAL;
  h->pool = (uint8_t*)pool;
  h->pool_bytes = pool_bytes;
  h->slots = (uint8_t*)slots;
  h->slots_bytes = slots ? slots_bytes : 0;
  h->loaded.assign(h->cfg.num_layers, 0);
  h->ring_started = false;
  h->ring_g = 0;
  for (int l = 0; layers && l < n_layers; l++) {
    const int e = sidp_pool_load_layer(h, l, &layers[l], stream);
    if (e != SIDP_OK) return e;
  }
  return SIDP_OK;
}

int sidp_pool_load_layer(sidp_handle* h, int32_t layer, const sidp_layer_weights* w, void* stream) {
  if (!h || !w) return SIDP_EINVAL;
  if (h->poisoned || !h->pool) return SIDP_ESTATE;
  const sidp_config& c = h->cfg;
  if (layer < 0 || layer >= c.num_layers) return SIDP_EINVAL;
  if (!w->w_q || !w->w_k || !w->w_v || !w->w_o || !w->w_gate || !w->w_up || !w->w_down || !w->g_attn || !w->g_mlp)
    return SIDP_EINVAL;
  if (c.qkv_bias && (!w->b_q || !w->b_k || !w->b_v)) return SIDP_EINVAL;
  if (c.qk_norm && (!w->g_q || !w->g_k)) return SIDP_EINVAL;
  hipStream_t s = (hipStream_t)stream;
  uint8_t* base = h->pool + (size_t)layer * h->blob.total;
  const size_t H = c.hidden, D = c.head_dim, QD = (size_t)c.num_q_heads * D, KD = (size_t)c.num_kv_heads * D;
  HIPCHK(h, hipMemcpyAsync(base + h->blob.g_attn, w->g_attn, H * 2, hipMemcpyDeviceToDevice, s));
  HIPCHK(h, hipMemcpyAsync(h->g_attn_all + (size_t)layer * H, w->g_attn, H * 2, hipMemcpyDeviceToDevice, s));
  HIPCHK(h, hipMemcpyAsync(base + h->blob.g_mlp, w->g_mlp, H * 2, hipMemcpyDeviceToDevice, s));
  if (c.qk_norm) {
    HIPCHK(h, hipMemcpyAsync(base + h->blob.g_q, w->g_q, D * 2, hipMemcpyDeviceToDevice, s));
    HIPCHK(h, hipMemcpyAsync(base + h->blob.g_k, w->g_k, D * 2, hipMemcpyDeviceToDevice, s));
  }
  if (c.qkv_bias) {
    HIPCHK(h, hipMemcpyAsync(base + h->blob.bias, w->b_q, QD * 2, hipMemcpyDeviceToDevice, s));
    HIPCHK(h, hipMemcpyAsync(base + h->blob.bias + QD * 2, w->b_k, KD * 2, hipMemcpyDeviceToDevice, s));
    HIPCHK(h, hipMemcpyAsync(base + h->blob.bias + (QD + KD) * 2, w->b_v, KD * 2, hipMemcpyDeviceToDevice, s));
  }
  // Fused QKV: the q, k and v row blocks are multiples of 64 rows, so their
  // packed forms concatenate along the column groups.
  uint8_t* wqkv = base + h->blob.w_qkv;
  HIPCHK(h, launch_pack_qkv(w->w_q, w->w_k, w->w_v, (int)QD, (int)KD, (int)H, wqkv, s));
  HIPCHK(h, launch_pack_linear(w->w_o, (int)H, (int)QD, base + h->blob.w_o, s));
  HIPCHK(h, launch_pack_gate_up(w->w_gate, w->w_up, c.ffn_dim, (int)H, base + h->blob.w_gu, s));
  HIPCHK(h, launch_pack_linear(w->w_down, (int)H, c.ffn_dim, base + h->blob.w_d, s));
  h->loaded[layer] = 1;
  // the slots may hold (or be filling) the layer's old blob: restart the ring
  h->ring_started = false;
  h->ring_g = 0;
  return SIDP_OK;
}

// ---------------------------------------------------------------- paged KV

static uint64_t splitmix64_next(uint64_t* state) {
  uint64_t z = (*state += 0x9E3779B97F4A7C15ull);
  z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
  z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
  return z ^ (z >> 31);
}

int sidp_kv_alloc(int32_t batch, const int32_t* ctx_lens, int32_t reserve_tokens, int32_t block_size,
                  int32_t num_phys_blocks, uint64_t seed, int32_t max_blocks_per_seq, int32_t* block_tables) {
  if (batch < 0 || reserve_tokens < 0 || block_size < 1 || num_phys_blocks < 0 || max_blocks_per_seq < 1)
    return SIDP_EINVAL;
  if (batch > 0 && (!ctx_lens || !block_tables)) return SIDP_EINVAL;
  std::vector<int32_t> perm((size_t)num_phys_blocks);
  for (int32_t i = 0; i < num_phys_blocks; i++) perm[i] = i;
  uint64_t st = seed;
  for (int32_t i = num_phys_blocks - 1; i >= 1; i--) {
    const uint64_t j = splitmix64_next(&st) % (uint64_t)(i + 1);
    std::swap(perm[i], perm[j]);
  }
  int64_t next = 0;
  for (int32_t b = 0; b < batch; b++) {
    if (ctx_lens[b] < 0) return SIDP_EINVAL;
    const int64_t need = ((int64_t)ctx_lens[b] + reserve_tokens + block_size - 1) / block_size;
    if (need > max_blocks_per_seq || next + need > num_phys_blocks) return SIDP_ENOBLOCKS;
    int32_t* row = block_tables + (int64_t)b * max_blocks_per_seq;
    for (int64_t j = 0; j < max_blocks_per_seq; j++) row[j] = j < need ? perm[next + j] : -1;
    next += need;
  }
  return SIDP_OK;
}

size_t sidp_kv_region_bytes(const sidp_config* cfg, int32_t num_phys_blocks) {
  if (!config_ok(cfg) || num_phys_blocks < 1) return 0;
  return (size_t)num_phys_blocks * cfg->num_kv_heads * cfg->block_size * cfg->head_dim * 2;
}

int sidp_kv_attach(sidp_handle* h, void* k_cache, void* v_cache, int32_t num_phys_blocks, int32_t num_regions) {
  if (!h || !k_cache || !v_cache || num_phys_blocks < 1 || num_regions < 1) return SIDP_EINVAL;
  if (h->poisoned) return SIDP_ESTATE;
  if (((uintptr_t)k_cache % 16) || ((uintptr_t)v_cache % 16)) return SIDP_EINVAL;
  h->k_cache = (uint16_t*)k_cache;
  h->v_cache = (uint16_t*)v_cache;
  h->nblk = num_phys_blocks;
  h->regions = num_regions;
  return SIDP_OK;
}

// ---------------------------------------------------------------- decode step

static KvView kv_view(const sidp_handle* h) {
  KvView v;
  v.k = h->k_cache;
  v.v = h->v_cache;
  v.nblk = h->nblk;
  v.regions = h->regions;
  v.hkv = h->cfg.num_kv_heads;
  v.d = h->cfg.head_dim;
  v.bs = h->cfg.block_size;
  return v;
}

// Calls that use the handle's buffers (activations, partials, work list) are
// ordered like one stream: a call on a stream other than the previous call's
// first waits for the previous call's work (the event recorded after it).
static hipError_t begin_call(sidp_handle* h, hipStream_t s) {
  if (h->work_recorded && s != h->last_compute) return hipStreamWaitEvent(s, h->work_done, 0);
  return hipSuccess;
}
static hipError_t finish_call(sidp_handle* h, hipStream_t s) {
  h->last_compute = s;
  h->work_recorded = true;
  return hipEventRecord(h->work_done, s);
}

static LinearCall linear_call(const sidp_handle* h, const void* x, int m, int k, const void* packed, int n, int epi,
                              const void* bias, const float* resid, void* out) {
  LinearCall c;
  c.x = x;
  c.m = m;
  c.k = k;
  c.packed = packed;
  c.n = n;
  c.epilogue = epi;
  c.bias = bias;
  c.residual = resid;
  c.out = out;
  c.ws = h->ws;
  c.ws_bytes = h->ws_bytes;
  c.num_cus = h->num_cus;
  return c;
}

// SIDP_TIMING: open a timed interval of kernel class `cls` on stream s.
static bool timed_class(const sidp_handle* h, int cls) { return h->timing && ((h->timing_mask >> cls) & 1u); }

// Takes a (start, stop) event pair for an interval of class `cls` and lists
// it for sidp_timing_collect.
static hipError_t time_pair(sidp_handle* h, int cls, hipEvent_t* start, hipEvent_t* stop) {
  hipEvent_t ev[2];
  for (int i = 0; i < 2; i++) {
    if (!h->event_pool.empty()) {
      ev[i] = h->event_pool.back();
      h->event_pool.pop_back();
    } else {
      hipError_t e = hipEventCreate(&ev[i]);
      if (e != hipSuccess) return e;
    }
  }
  h->timed.push_back({cls, ev[0], ev[1]});
  *start = ev[0];
  *stop = ev[1];
  return hipSuccess;
}

static hipError_t time_begin(sidp_handle* h, int cls, hipStream_t s) {
  if (!timed_class(h, cls)) return hipSuccess;
  hipEvent_t start, stop;
  hipError_t e = time_pair(h, cls, &start, &stop);
  return e != hipSuccess ? e : hipEventRecord(start, s);
}
static hipError_t time_end(sidp_handle* h, int cls, hipStream_t s) {
  if (!timed_class(h, cls)) return hipSuccess;
  return hipEventRecord(h->timed.back().b, s);
}

#define TIMED(h, cls, s, expr)                                      \
  do {                                                              \
    hipError_t te_;                                                 \
    if ((te_ = time_begin((h), (cls), (s))) != hipSuccess) return te_; \
    if ((te_ = (expr)) != hipSuccess) return te_;                   \
    if ((te_ = time_end((h), (cls), (s))) != hipSuccess) return te_; \
  } while (0)

// The attention half of a layer (norm, QKV, QK-norm/RoPE/KV append,
// attention), reading weights from `wb` (a pool blob or a slot).
static hipError_t run_attn_half(sidp_handle* h, const uint8_t* wb, int layer, float* hidden, const int32_t* positions,
                                const int32_t* bt, int max_blocks, int B, hipStream_t s) {
  const sidp_config& c = h->cfg;
  const BlobLayout& L = h->blob;
  const int H = c.hidden, D = c.head_dim;
  // a2: RMSNorm before attention; for layers after the first of a step the
  // previous layer's down-projection reduction has already written it
  if (layer == 0) TIMED(h, SIDP_K_NORM_ATTN, s, launch_rmsnorm(hidden, wb + L.g_attn, c.rms_eps, h->h, B, H, s));
  // a3: QKV projection (+ bias). With split-K its partials are reduced by the
  // RoPE kernel below, which rounds to bf16 exactly where the projection would.
  const uint16_t* qkv_bias = c.qkv_bias ? (const uint16_t*)(wb + L.bias) : nullptr;
  LinearCall qc = linear_call(h, h->h, B, H, wb + L.w_qkv, qkv_rows(c), SIDP_EPI_BF16, qkv_bias, nullptr, h->qkv);
  qc.defer_reduce = true;
  const int qkv_splits = gemm_splits(B, qkv_rows(c), H, h->num_cus);
  TIMED(h, SIDP_K_QKV, s, launch_linear(qc, s));
  // a4/a5: QK-norm, RoPE, KV append at the slot of each sequence's position
  RopeCall r;
  r.qkv = h->qkv;
  r.ws = qkv_splits > 1 ? h->ws : nullptr;
  r.splits = qkv_splits;
  r.ws_np = round_up_i(qkv_rows(c), 64);
  r.bias = qkv_bias;
  r.positions = positions;
  r.block_tables = bt;
  r.max_blocks = max_blocks;
  r.batch = B;
  r.hq = c.num_q_heads;
  r.hkv = c.num_kv_heads;
  r.d = D;
  r.g_q = c.qk_norm ? (const uint16_t*)(wb + L.g_q) : nullptr;
  r.g_k = c.qk_norm ? (const uint16_t*)(wb + L.g_k) : nullptr;
  r.qk_eps = c.qk_norm_eps;
  r.rope_cos = h->rope_cos;
  r.rope_sin = h->rope_sin;
  r.max_seq = c.max_seq_len;
  r.kv = kv_view(h);
  r.region = layer % h->regions;
  r.q_out = h->q;
  r.err = h->err;
  TIMED(h, SIDP_K_ROPE, s, launch_rope_append(r, s));
  // a6: paged GQA attention
  AttnCall a;
  a.q = h->q;
  a.positions = positions;
  a.block_tables = bt;
  a.max_blocks = max_blocks;
  a.batch = B;
  a.hq = c.num_q_heads;
  a.hkv = c.num_kv_heads;
  a.d = D;
  a.kv = kv_view(h);
  a.region = layer % h->regions;
  a.out = h->o;
  a.part = h->attn_part;
  a.max_parts = h->attn_max_parts;
  a.err = h->err;
  a.num_cus = h->num_cus;
  a.plan = h->attn_plan;
  if (!timed_class(h, SIDP_K_ATTN)) return launch_attention(a, s);
  // timed through the attention kernels' own dispatches: no marker packets
  // between the RoPE kernel, the attention and the O projection
  hipEvent_t start, stop;
  const hipError_t e = time_pair(h, SIDP_K_ATTN, &start, &stop);
  return e != hipSuccess ? e : launch_attention(a, s, start, stop);
}

// The compute stream's waits for the tiles of a slot fill (streamed layers
// only): before a kernel that reads the slot, the tile holding the last byte
// it reads.
struct SlotWaits {
  sidp_handle* h;
  int slot;         // -1: weights read in place, no wait
  size_t tile_a_end;  // end of tile A in the blob (tile B ends at the staged range's end)
  int done = -1;    // the last tile already waited for (0: A, 1: B)
};

// Waits (on s) until the bytes of the slot below `need_end` have landed.
static hipError_t wait_slot_bytes(SlotWaits* w, size_t need_end, hipStream_t s) {
  if (!w || w->slot < 0) return hipSuccess;
  const int tile = need_end <= w->tile_a_end ? 0 : 1;
  if (tile <= w->done) return hipSuccess;
  hipError_t e;
  if ((e = time_begin(w->h, SIDP_K_WAIT_FILL, s)) != hipSuccess) return e;
  if ((e = hipStreamWaitEvent(s, tile ? w->h->filled[w->slot] : w->h->tile_a[w->slot], 0)) != hipSuccess) return e;
  w->done = tile;
  return time_end(w->h, SIDP_K_WAIT_FILL, s);
}

// The projection half of a layer (O + residual, norm, gate/up + SwiGLU,
// down + residual).
// `wa` holds the layer's attention part (W_o), `wf` its FFN part; both are
// the same blob unless only the FFN part is staged.
static hipError_t run_proj_half(sidp_handle* h, const uint8_t* wa, const uint8_t* wf, int layer, float* hidden, int B,
                                hipStream_t s, SlotWaits* waits = nullptr) {
  const sidp_config& c = h->cfg;
  const BlobLayout& L = h->blob;
  const int H = c.hidden, QD = c.num_q_heads * c.head_dim;
  hipError_t e;
  // W_o and the FFN norm gain lie below the gate/up weights
  if ((e = wait_slot_bytes(waits, L.w_gu, s)) != hipSuccess) return e;
  // a7 + a8: O projection + residual (in place on the fp32 residual stream),
  // then the RMSNorm before the FFN, fused into the split-K reduction
  LinearCall oc = linear_call(h, h->o, B, QD, wa + L.w_o, H, SIDP_EPI_RESID, nullptr, hidden, hidden);
  oc.norm_gain = wf + L.g_mlp;
  oc.norm_eps = c.rms_eps;
  oc.norm_out = h->h;
  TIMED(h, SIDP_K_O, s, launch_linear(oc, s));
  // a9: gate/up projection + SwiGLU; the FFN's weights (gate/up, then down)
  // take one wait, for the whole fill: a second wait inside the FFN gained
  // nothing measurable and its timing brackets cost about 1 ms per step
  if ((e = wait_slot_bytes(waits, L.total, s)) != hipSuccess) return e;
  TIMED(h, SIDP_K_GATE_UP, s,
        launch_linear(linear_call(h, h->h, B, H, wf + L.w_gu, c.ffn_dim, SIDP_EPI_SWIGLU, nullptr, nullptr, h->act),
                      s));
  // a10: down projection + residual, fused with the next layer's attention
  // norm (a2 of layer + 1) when there is a next layer in this step
  LinearCall dc = linear_call(h, h->act, B, c.ffn_dim, wf + L.w_d, H, SIDP_EPI_RESID, nullptr, hidden, hidden);
  if (layer + 1 < c.num_layers) {
    dc.norm_gain = h->g_attn_all + (size_t)(layer + 1) * H;
    dc.norm_eps = c.rms_eps;
    dc.norm_out = h->h;
  }
  TIMED(h, SIDP_K_DOWN, s, launch_linear(dc, s));
  return hipSuccess;
}

static hipError_t run_layer(sidp_handle* h, const uint8_t* wb, int layer, float* hidden, const int32_t* positions,
                            const int32_t* bt, int max_blocks, int B, hipStream_t s) {
  hipError_t e = run_attn_half(h, wb, layer, hidden, positions, bt, max_blocks, B, s);
  if (e != hipSuccess) return e;
  return run_proj_half(h, wb, wb, layer, hidden, B, s);
}

// The staged byte range [lo, hi) of a layer blob and the end `mid` of fill part A.
static void staged_range(const sidp_handle* h, size_t* lo, size_t* mid, size_t* hi) {
  *lo = h->pool_mode == SIDP_POOL_FFN ? h->blob.ffn_lo : 0;
  *hi = h->blob.total;
  *mid = std::min(*hi, *lo + align_up((*hi - *lo) * (size_t)h->fill_pct / 100, kAlign));
}

// The layer that ring instance g computes.
static int ring_layer_index(const sidp_handle* h, int64_t g) {
  return h->streamed_layers[(size_t)(g % (int64_t)h->streamed_layers.size())];
}

// Part of one slot fill on the copy stream: bytes [lo, hi) of the blob of
// ring instance g's layer, from the pool into slot `slot`.
static hipError_t issue_fill(sidp_handle* h, int64_t g, int slot, size_t lo, size_t hi, int flags, hipStream_t cp) {
  const size_t lb = h->blob.total;
  uint8_t* dst = h->slots + (size_t)slot * lb;
  const uint8_t* src = h->pool + (size_t)ring_layer_index(h, g) * lb;
  const bool part_a = lo == (h->pool_mode == SIDP_POOL_FFN ? h->blob.ffn_lo : 0);
  hipError_t e;
  if (part_a && (flags & SIDP_DEBUG_POISON))  // the whole slot, unstaged parts included
    if ((e = launch_poison(dst, lb, cp)) != hipSuccess) return e;
  if (hi <= lo) return hipSuccess;
  if (flags & SIDP_DEBUG_DELAY)  // every launch lands late: a missing wait on any part reads poison
    if ((e = launch_spin(kDelayTicks, cp)) != hipSuccess) return e;
  if ((e = time_begin(h, SIDP_K_FILL, cp)) != hipSuccess) return e;
  if (flags & SIDP_COPY_MEMCPY) e = hipMemcpyAsync(dst + lo, src + lo, hi - lo, hipMemcpyDeviceToDevice, cp);
  else if (flags & SIDP_COPY_SDMA) e = hipMemcpyAsync(dst + lo, src + lo, hi - lo, hipMemcpyDeviceToDeviceNoCU, cp);
  else if (flags & SIDP_COPY_BURST) e = launch_copy(src + lo, dst + lo, hi - lo, kBurstGrid, cp);
  else {
    // Defaults: below kFillSmallBatch rows a layer computes in less time than
    // its fill takes, so both tiles keep 8 loads per lane in flight (at 16,
    // 64 and 128 rows 1-2% faster than 8 and 4; at 192 rows 5% slower).
    // From there tile A keeps 8 and tile B 4 below kFillLongBatch rows when
    // each kernel waits only for its part (tile B then has to land within the
    // projections, or its tail and the next tile A run into the attention; at
    // 256 rows 8 and 4 ran 1.3% faster than 4 and 4). Otherwise 4 and 2: from
    // kFillLongBatch rows the projections last long enough for a gentler fill
    // (4 and 2 beat 8 and 4 at 384 and 512 rows), and when the layer waits for
    // its whole fill any more slows the projections beside it more than the
    // stall it saves.
    const bool small = h->step_batch < kFillSmallBatch;
    const bool press = small || (h->part_waits && h->step_batch < kFillLongBatch);
    const int la = h->fill_loads_a ? h->fill_loads_a : (press ? 8 : 4);
    const int lb = h->fill_loads_b ? h->fill_loads_b : (small ? 8 : press ? 4 : 2);
    e = launch_fill_bg(src + lo, dst + lo, hi - lo, h->num_cus, part_a ? la : lb, cp);
  }
  if (e != hipSuccess) return e;
  return time_end(h, SIDP_K_FILL, cp);
}

int sidp_decode_step(sidp_handle* h, float* hidden, const int32_t* positions, const int32_t* block_tables,
                     int32_t max_blocks_per_seq, int32_t batch, int32_t flags, void* compute, void* copy) {
  if (!h) return SIDP_EINVAL;
  if (h->poisoned) return SIDP_ESTATE;
  const sidp_config& c = h->cfg;
  if (!hidden || !positions || !block_tables || batch < 1 || batch > c.max_batch || max_blocks_per_seq < 1)
    return SIDP_EINVAL;
  if (!h->pool || !h->k_cache) return SIDP_ESTATE;
  for (int l = 0; l < c.num_layers; l++)
    if (!h->loaded[l]) return SIDP_ESTATE;
  const int parts = (max_blocks_per_seq * c.block_size + attn_part_tokens() - 1) / attn_part_tokens();
  if (parts > h->attn_max_parts) return SIDP_EINVAL;
  const bool streamed = flags & SIDP_STREAMED;
  h->timing = (flags & SIDP_TIMING) != 0;
  h->step_batch = batch;
  hipStream_t cs = (hipStream_t)compute, cp = (hipStream_t)copy;
  if (streamed && (!h->slots || cp == cs)) return SIDP_EINVAL;
  HIPCHK(h, begin_call(h, cs));
  {
    // the attention work list depends on the positions only: one per step
    AttnCall a{};
    a.positions = positions;
    a.batch = batch;
    a.max_blocks = max_blocks_per_seq;
    a.hkv = c.num_kv_heads;
    a.num_cus = h->num_cus;
    a.kv = kv_view(h);
    a.plan = h->attn_plan;
    a.err = h->err;
    HIPCHK(h, launch_attn_plan(a, cs));
  }

  if (!streamed) {
    for (int l = 0; l < c.num_layers; l++)
      HIPCHK(h, run_layer(h, h->pool + (size_t)l * h->blob.total, l, hidden, positions, block_tables,
                          max_blocks_per_seq, batch, cs));
    HIPCHK(h, finish_call(h, cs));
    return SIDP_OK;
  }

  h->last_copy = cp;
  h->any_copy = true;
  std::vector<RingOp> ops;
  build_step(c.num_layers, h->ranks, h->rank, 0, &h->ring_g, &h->ring_started, ops);
  const size_t lb = h->blob.total;
  size_t st_lo, st_mid, st_hi;
  staged_range(h, &st_lo, &st_mid, &st_hi);
  SlotWaits waits{h, -1, 0};
  const bool ffn_only = h->pool_mode == SIDP_POOL_FFN;
  for (const RingOp& op : ops) {
    const uint8_t* slot = op.slot >= 0 ? h->slots + (size_t)op.slot * lb : nullptr;
    const int layer = op.kind == OP_LOCAL ? (int)(op.g % c.num_layers) : ring_layer_index(h, op.g);
    const uint8_t* own = h->pool + (size_t)layer * lb;  // the layer's blob in the pool
    switch (op.kind) {
      case OP_FILL_A:
        HIPCHK(h, issue_fill(h, op.g, op.slot, st_lo, st_mid, flags, cp));
        HIPCHK(h, hipEventRecord(h->tile_a[op.slot], cp));
        break;
      case OP_FILL_B:
        HIPCHK(h, issue_fill(h, op.g, op.slot, st_mid, st_hi, flags, cp));
        HIPCHK(h, hipEventRecord(h->filled[op.slot], cp));
        break;
      case OP_WAIT_FILL:
        // The compute stream waits for the part of the fill the attention half
        // reads (its gains, bias and W_qkv, below W_o; nothing when only the
        // FFN part is staged); the projections wait for theirs in turn. Under
        // SIDP_TIMING each wait is bracketed: the compute stall on the fill.
        waits = SlotWaits{h, op.slot, st_mid};
        if (!h->part_waits) HIPCHK(h, wait_slot_bytes(&waits, h->blob.total, cs));
        else if (!ffn_only) HIPCHK(h, wait_slot_bytes(&waits, h->blob.w_o, cs));
        break;
      case OP_ATTN:
        HIPCHK(h, run_attn_half(h, ffn_only ? own : slot, layer, hidden, positions, block_tables, max_blocks_per_seq,
                                batch, cs));
        break;
      case OP_MID:
        HIPCHK(h, hipEventRecord(h->mid[op.slot], cs));
        break;
      case OP_PROJ:
        HIPCHK(h, run_proj_half(h, ffn_only ? own : slot, slot, layer, hidden, batch, cs, &waits));
        break;
      case OP_DONE:
        HIPCHK(h, hipEventRecord(h->consumed[op.slot], cs));
        break;
      case OP_WAIT_DONE:
        HIPCHK(h, hipStreamWaitEvent(cp, h->consumed[op.slot], 0));
        break;
      case OP_WAIT_MID:
        HIPCHK(h, hipStreamWaitEvent(cp, h->mid[op.slot], 0));
        break;
      case OP_LOCAL:
        HIPCHK(h, run_layer(h, own, layer, hidden, positions, block_tables, max_blocks_per_seq, batch, cs));
        break;
    }
  }
  HIPCHK(h, finish_call(h, cs));
  return SIDP_OK;
}

int sidp_timing_select(sidp_handle* h, uint32_t class_mask) {
  if (!h) return SIDP_EINVAL;
  if (class_mask >> SIDP_NUM_KCLASSES) return SIDP_EINVAL;
  h->timing_mask = class_mask;
  return SIDP_OK;
}

static_assert(SIDP_CAS_MAX_REPLICAS == kMaxReplicas, "replica table size");

int sidp_cas_ffn(sidp_handle* h, int32_t layer, int32_t n_replicas, const void* const* x_in, const int32_t* rows,
                 void* const* y_out, void* stream) {
  if (!h || !x_in || !rows || !y_out || n_replicas < 1 || n_replicas > SIDP_CAS_MAX_REPLICAS) return SIDP_EINVAL;
  if (h->poisoned) return SIDP_ESTATE;
  const sidp_config& c = h->cfg;
  if (layer < 0 || layer >= c.num_layers) return SIDP_EINVAL;
  if (!h->pool || !h->loaded[layer]) return SIDP_ESTATE;
  const int H = c.hidden;
  RowMove in{}, out{};
  int total = 0, n = 0;
  for (int r = 0; r < n_replicas; r++) {
    if (rows[r] < 0) return SIDP_EINVAL;
    if (rows[r] == 0) continue;  // a dummy replica: nothing moved, nothing computed
    if (!x_in[r] || !y_out[r] || ((uintptr_t)x_in[r] % 16) || ((uintptr_t)y_out[r] % 16)) return SIDP_EINVAL;
    if (total + rows[r] > c.max_batch) return SIDP_EINVAL;
    in.rep[n] = const_cast<void*>(x_in[r]);
    out.rep[n] = y_out[r];
    in.row_off[n] = out.row_off[n] = total;
    total += rows[r];
    n++;
  }
  if (total == 0) return SIDP_OK;
  in.row_off[n] = out.row_off[n] = total;
  in.n = out.n = n;
  in.row_bytes = (size_t)H * 2;
  out.row_bytes = (size_t)H * 4;
  in.staging = h->h;
  out.staging = h->cas_y;
  in.gather = 1;
  out.gather = 0;
  hipStream_t s = (hipStream_t)stream;
  const uint8_t* wb = h->pool + (size_t)layer * h->blob.total;
  HIPCHK(h, begin_call(h, s));
  HIPCHK(h, launch_rows_move(in, s));
  HIPCHK(h, launch_linear(linear_call(h, h->h, total, H, wb + h->blob.w_gu, c.ffn_dim, SIDP_EPI_SWIGLU, nullptr,
                                      nullptr, h->act), s));
  HIPCHK(h, launch_linear(linear_call(h, h->act, total, c.ffn_dim, wb + h->blob.w_d, H, SIDP_EPI_RESID, nullptr,
                                      nullptr, h->cas_y), s));
  HIPCHK(h, launch_rows_move(out, s));
  HIPCHK(h, finish_call(h, s));
  return SIDP_OK;
}

int sidp_set_pooling(sidp_handle* h, int32_t mode, int32_t ranks, int32_t rank) {
  if (!h) return SIDP_EINVAL;
  if (h->poisoned) return SIDP_ESTATE;
  if (mode != SIDP_POOL_LAYER && mode != SIDP_POOL_FFN) return SIDP_EINVAL;
  if (ranks < 0 || (ranks > 0 && (rank < 0 || rank >= ranks))) return SIDP_EINVAL;
  h->pool_mode = mode;
  h->ranks = ranks;
  h->rank = ranks > 0 ? rank : 0;
  h->streamed_layers.clear();
  for (int l = 0; l < h->cfg.num_layers; l++)
    if (!layer_owned(l, h->ranks, h->rank)) h->streamed_layers.push_back(l);
  // the slots no longer hold what the ring expects: restart it
  h->ring_started = false;
  h->ring_g = 0;
  return SIDP_OK;
}

int sidp_set_fill_tiles(sidp_handle* h, int32_t first_tile_percent, int32_t loads_a, int32_t loads_b,
                        int32_t part_waits) {
  if (!h) return SIDP_EINVAL;
  if (h->poisoned) return SIDP_ESTATE;
  auto loads_ok = [](int32_t n) { return n == 0 || n == 2 || n == 4 || n == 8; };
  if (first_tile_percent < 0 || first_tile_percent > 100 || !loads_ok(loads_a) || !loads_ok(loads_b) ||
      (part_waits != 0 && part_waits != 1))
    return SIDP_EINVAL;
  h->part_waits = part_waits;
  h->fill_pct = first_tile_percent;
  h->fill_loads_a = loads_a;
  h->fill_loads_b = loads_b;
  return SIDP_OK;
}

int sidp_debug_inject_hip_error(sidp_handle* h, int32_t hip_error) {
  if (!h || hip_error == 0) return SIDP_EINVAL;
  if (h->poisoned) return SIDP_ESTATE;
  h->inject_hip = hip_error;
  return SIDP_OK;
}

int sidp_sync(sidp_handle* h) {
  if (!h) return SIDP_EINVAL;
  if (h->poisoned) return SIDP_ESTATE;
  HIPCHK(h, hipStreamSynchronize(h->last_compute));
  if (h->any_copy) HIPCHK(h, hipStreamSynchronize(h->last_copy));
  HIPCHK(h, hipDeviceSynchronize());
  uint32_t err = 0;
  HIPCHK(h, hipMemcpy(&err, h->err, 4, hipMemcpyDeviceToHost));
  if (err) {
    HIPCHK(h, hipMemset(h->err, 0, 4));
    return SIDP_EINVAL;
  }
  return SIDP_OK;
}

int sidp_timing_collect(sidp_handle* h, double* ms, int32_t* launches) {
  if (!h || !ms || !launches) return SIDP_EINVAL;
  if (h->poisoned) return SIDP_ESTATE;
  for (int i = 0; i < SIDP_NUM_KCLASSES; i++) {
    ms[i] = 0.0;
    launches[i] = 0;
  }
  for (auto& t : h->timed) {
    HIPCHK(h, hipEventSynchronize(t.b));
    float el = 0.f;
    HIPCHK(h, hipEventElapsedTime(&el, t.a, t.b));
    ms[t.cls] += el;
    launches[t.cls]++;
    h->event_pool.push_back(t.a);
    h->event_pool.push_back(t.b);
  }
  h->timed.clear();
  return SIDP_OK;
}

int sidp_peak_shift_plan(int32_t num_layers, int32_t ranks, int32_t rank, int32_t* pairs, int32_t* n) {
  if (num_layers < 1 || ranks < 1 || rank < 0 || rank >= ranks || !n) return SIDP_EINVAL;
  std::vector<int32_t> order;  // layers, in pull order
  for (int64_t c = 0; c < num_layers; c += ranks)
    for (int k = 1; k < ranks; k++) {  // k = 0 is the rank's own layer of the cycle
      const int64_t layer = c + (rank + k) % ranks;
      if (layer < num_layers) order.push_back((int32_t)layer);
    }
  if ((int64_t)order.size() > *n) return SIDP_EINVAL;
  if (!order.empty() && !pairs) return SIDP_EINVAL;
  for (size_t i = 0; i < order.size(); i++) {
    pairs[2 * i] = order[i];
    pairs[2 * i + 1] = order[i] % ranks;
  }
  *n = (int32_t)order.size();
  return SIDP_OK;
}

int sidp_plan(int32_t num_layers, int32_t steps, int32_t ranks, int32_t rank, int32_t* ops_out, int32_t* n_ops) {
  if (num_layers < 1 || steps < 0 || !n_ops) return SIDP_EINVAL;
  if (ranks < 0 || (ranks > 0 && (rank < 0 || rank >= ranks))) return SIDP_EINVAL;
  std::vector<RingOp> ops;
  int64_t ring_g = 0;
  bool started = false;
  for (int t = 0; t < steps; t++) build_step(num_layers, ranks, rank, t, &ring_g, &started, ops);
  if ((int64_t)ops.size() > *n_ops) return SIDP_EINVAL;
  if (!ops.empty() && !ops_out) return SIDP_EINVAL;
  for (size_t i = 0; i < ops.size(); i++) {
    ops_out[3 * i] = ops[i].kind;
    ops_out[3 * i + 1] = (int32_t)ops[i].g;
    ops_out[3 * i + 2] = ops[i].slot;
  }
  *n_ops = (int32_t)ops.size();
  return SIDP_OK;
}

// ---------------------------------------------------------------- mode choice

int sidp_mode_update(const sidp_mode_policy* p, sidp_mode_state* st, int32_t n_engines, const int32_t* active,
                     int32_t* mode) {
  if (!p || !st || !active || !mode || n_engines < 1) return SIDP_EINVAL;
  if (!(p->b_th > 0.f) || !(p->hysteresis >= 0.f) || p->window < 1) return SIDP_EINVAL;
  if (st->mode != SIDP_MODE_WAS && st->mode != SIDP_MODE_CAS) return SIDP_EINVAL;
  double sum = 0.0;
  for (int32_t i = 0; i < n_engines; i++) {
    if (active[i] < 0) return SIDP_EINVAL;
    sum += active[i];
  }
  const double b = sum / n_engines;
  const bool cond = st->mode == SIDP_MODE_WAS ? b < (double)p->b_th : b >= (double)p->b_th * (1.0 + p->hysteresis);
  st->run = cond ? st->run + 1 : 0;
  if (st->run >= p->window) {
    st->mode = st->mode == SIDP_MODE_WAS ? SIDP_MODE_CAS : SIDP_MODE_WAS;
    st->run = 0;
  }
  *mode = st->mode;
  return SIDP_OK;
}

// ---------------------------------------------------------------- single kernels

int sidp_rmsnorm(const float* x, const void* gain, float eps, void* out, int32_t rows, int32_t n, void* stream) {
  if (!x || !gain || !out || rows < 0 || n < 4 || n % 4 || !(eps > 0.f)) return SIDP_EINVAL;
  return launch_rmsnorm(x, gain, eps, out, rows, n, (hipStream_t)stream) == hipSuccess ? SIDP_OK : SIDP_EHIP;
}

size_t sidp_packed_bytes(int32_t n, int32_t k) {
  if (n < 1 || k < 1) return 0;
  return packed_bytes(n, k);
}

int sidp_pack_linear(const void* w, int32_t n, int32_t k, void* packed, void* stream) {
  if (!w || !packed || n < 1 || k < 1 || n > (1 << 24) || k > (1 << 24)) return SIDP_EINVAL;
  return launch_pack_linear(w, n, k, packed, (hipStream_t)stream) == hipSuccess ? SIDP_OK : SIDP_EHIP;
}

int sidp_pack_gate_up(const void* w_gate, const void* w_up, int32_t f, int32_t k, void* packed, void* stream) {
  if (!w_gate || !w_up || !packed || f < 1 || k < 1 || f > (1 << 24) || k > (1 << 24)) return SIDP_EINVAL;
  return launch_pack_gate_up(w_gate, w_up, f, k, packed, (hipStream_t)stream) == hipSuccess ? SIDP_OK : SIDP_EHIP;
}

int sidp_linear(sidp_handle* h, const void* x, int32_t m, int32_t k, const void* packed, int32_t n, int32_t epilogue,
                const void* bias, const float* residual, void* out, void* stream) {
  if (!h || !x || !packed || !out || m < 1 || m > h->cfg.max_batch || k < 8 || k % 8 || n < 1) return SIDP_EINVAL;
  if (k > (1 << 24) || n > (1 << 24)) return SIDP_EINVAL;
  if (h->poisoned) return SIDP_ESTATE;
  if (epilogue < SIDP_EPI_BF16 || epilogue > SIDP_EPI_SWIGLU) return SIDP_EINVAL;
  if (epilogue == SIDP_EPI_RESID && !residual) return SIDP_EINVAL;
  if (epilogue != SIDP_EPI_BF16 && bias) return SIDP_EINVAL;
  const int ncols = epilogue == SIDP_EPI_SWIGLU ? 2 * round_up_i(n, 32) : n;
  if (!gemm_fits(m, ncols, k)) return SIDP_EINVAL;
  if (gemm_ws_bytes(m, ncols, k, h->num_cus) > h->ws_bytes) return SIDP_EINVAL;
  HIPCHK(h, begin_call(h, (hipStream_t)stream));
  HIPCHK(h, launch_linear(linear_call(h, x, m, k, packed, n, epilogue, bias, residual, out), (hipStream_t)stream));
  HIPCHK(h, finish_call(h, (hipStream_t)stream));
  return SIDP_OK;
}

int sidp_linear_plan(int32_t m, int32_t n, int32_t k, int32_t epilogue, int32_t num_cus, int32_t* kernel,
                     int32_t* waves, int32_t* rows_per_workgroup, int32_t* splits, int32_t* workgroups,
                     uint64_t* ws_bytes) {
  if (!kernel || !waves || !rows_per_workgroup || !splits || !workgroups || !ws_bytes) return SIDP_EINVAL;
  if (m < 1 || k < 8 || k % 8 || n < 1 || k > (1 << 24) || n > (1 << 24) || num_cus < 1) return SIDP_EINVAL;
  if (epilogue < SIDP_EPI_BF16 || epilogue > SIDP_EPI_SWIGLU) return SIDP_EINVAL;
  const int ncols = epilogue == SIDP_EPI_SWIGLU ? 2 * round_up_i(n, 32) : n;
  if (!gemm_fits(m, ncols, k)) return SIDP_EINVAL;
  const GemmPlan p = plan_linear(m, n, k, epilogue, num_cus);
  *kernel = p.kernel;
  *waves = p.waves;
  *rows_per_workgroup = p.rows;
  *splits = p.splits;
  *workgroups = p.workgroups;
  *ws_bytes = p.ws_bytes;
  return SIDP_OK;
}

int sidp_slot_mapping(sidp_handle* h, const int32_t* positions, const int32_t* block_tables,
                      int32_t max_blocks_per_seq, int32_t batch, int32_t* slots, void* stream) {
  if (!h || !positions || !block_tables || !slots || batch < 0 || max_blocks_per_seq < 1) return SIDP_EINVAL;
  if (h->poisoned) return SIDP_ESTATE;
  const int nblk = h->nblk > 0 ? h->nblk : 0x7fffffff / h->cfg.block_size;
  HIPCHK(h, launch_slot_mapping(positions, block_tables, max_blocks_per_seq, batch, h->cfg.block_size, nblk, slots,
                                h->err, (hipStream_t)stream));
  h->last_compute = (hipStream_t)stream;
  return SIDP_OK;
}

int sidp_rope_append(sidp_handle* h, const void* qkv, const int32_t* positions, const int32_t* block_tables,
                     int32_t max_blocks_per_seq, int32_t batch, const void* g_q, const void* g_k, int32_t region,
                     void* q_out, void* stream) {
  if (!h || !qkv || !positions || !block_tables || !q_out || batch < 0 || batch > h->cfg.max_batch) return SIDP_EINVAL;
  if (h->poisoned) return SIDP_ESTATE;
  if (!h->k_cache || region < 0 || region >= h->regions || max_blocks_per_seq < 1) return SIDP_EINVAL;
  if (h->cfg.qk_norm && (!g_q || !g_k)) return SIDP_EINVAL;
  RopeCall r;
  r.qkv = (const uint16_t*)qkv;
  r.ws = nullptr;
  r.splits = 1;
  r.ws_np = 0;
  r.bias = nullptr;
  r.positions = positions;
  r.block_tables = block_tables;
  r.max_blocks = max_blocks_per_seq;
  r.batch = batch;
  r.hq = h->cfg.num_q_heads;
  r.hkv = h->cfg.num_kv_heads;
  r.d = h->cfg.head_dim;
  r.g_q = h->cfg.qk_norm ? (const uint16_t*)g_q : nullptr;
  r.g_k = h->cfg.qk_norm ? (const uint16_t*)g_k : nullptr;
  r.qk_eps = h->cfg.qk_norm_eps;
  r.rope_cos = h->rope_cos;
  r.rope_sin = h->rope_sin;
  r.max_seq = h->cfg.max_seq_len;
  r.kv = kv_view(h);
  r.region = region;
  r.q_out = (uint16_t*)q_out;
  r.err = h->err;
  HIPCHK(h, launch_rope_append(r, (hipStream_t)stream));
  h->last_compute = (hipStream_t)stream;
  return SIDP_OK;
}

int sidp_attention(sidp_handle* h, const void* q, int32_t region, const int32_t* positions,
                   const int32_t* block_tables, int32_t max_blocks_per_seq, int32_t batch, void* out, void* stream) {
  if (!h || !q || !positions || !block_tables || !out || batch < 0 || batch > h->cfg.max_batch) return SIDP_EINVAL;
  if (h->poisoned) return SIDP_ESTATE;
  if (!h->k_cache || region < 0 || region >= h->regions || max_blocks_per_seq < 1) return SIDP_EINVAL;
  const int parts = (max_blocks_per_seq * h->cfg.block_size + attn_part_tokens() - 1) / attn_part_tokens();
  if (parts > h->attn_max_parts) return SIDP_EINVAL;
  AttnCall a;
  a.q = (const uint16_t*)q;
  a.positions = positions;
  a.block_tables = block_tables;
  a.max_blocks = max_blocks_per_seq;
  a.batch = batch;
  a.hq = h->cfg.num_q_heads;
  a.hkv = h->cfg.num_kv_heads;
  a.d = h->cfg.head_dim;
  a.kv = kv_view(h);
  a.region = region;
  a.out = (uint16_t*)out;
  a.part = h->attn_part;
  a.max_parts = h->attn_max_parts;
  a.err = h->err;
  a.num_cus = h->num_cus;
  a.plan = h->attn_plan;
  HIPCHK(h, begin_call(h, (hipStream_t)stream));
  HIPCHK(h, launch_attn_plan(a, (hipStream_t)stream));
  HIPCHK(h, launch_attention(a, (hipStream_t)stream));
  HIPCHK(h, finish_call(h, (hipStream_t)stream));
  return SIDP_OK;
}

int sidp_copy(const void* src, void* dst, size_t bytes, int32_t grid, void* stream) {
  if ((!src || !dst) && bytes) return SIDP_EINVAL;
  if (((uintptr_t)src % 16) || ((uintptr_t)dst % 16) || grid < 0) return SIDP_EINVAL;
  return launch_copy(src, dst, bytes, grid, (hipStream_t)stream) == hipSuccess ? SIDP_OK : SIDP_EHIP;
}

}  // extern "C"
