// Kernel launchers shared between the kernel sources and the host runtime.
#pragma once
#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

#include "../../include/sidp.h"

namespace sidp {

struct LinearCall {
  const void* x;
  int m, k;
  const void* packed;
  int n;
  int epilogue;
  const void* bias;
  const float* residual;
  void* out;
  float* ws;
  size_t ws_bytes;
  int num_cus;
  // optional RMSNorm of the result (EPI_RESID in place only): norm_out = bf16(rmsnorm(out) * norm_gain)
  const void* norm_gain = nullptr;
  float norm_eps = 0.f;
  void* norm_out = nullptr;
  // leave split-K partials in ws for the consumer to reduce (it must sum them
  // in split order and apply the epilogue); ignored when there is one split
  bool defer_reduce = false;
};

size_t packed_bytes(int n, int k);
bool gemm_fits(int m, int n_cols_packed, int k);  // within the kernels' 32-bit buffer offsets
int gemm_splits(int M, int n_cols_packed, int K, int num_cus);
size_t gemm_ws_bytes(int M, int n_cols_packed, int K, int num_cus);
// The launch launch_linear makes for an [m, k] x [n, k]^T projection: kernel
// 0 = k_gemm (weights into registers), 1 = k_gemm_lw (256-row workgroups,
// weight tiles staged in LDS); waves and rows per workgroup; split-K count;
// workgroups launched; bytes of fp32 partials (0 without a split).
struct GemmPlan {
  int kernel, waves, rows, splits, workgroups;
  size_t ws_bytes;
};
GemmPlan plan_linear(int m, int n, int k, int epilogue, int num_cus);
hipError_t launch_pack_linear(const void* w, int n, int k, void* packed, hipStream_t s);
// W_q [nq, k], W_k and W_v [nkv, k] packed as the one stacked matrix [nq + 2 nkv, k]
hipError_t launch_pack_qkv(const void* wq, const void* wk, const void* wv, int nq, int nkv, int k, void* packed,
                           hipStream_t s);
hipError_t launch_pack_gate_up(const void* wg, const void* wu, int f, int k, void* packed, hipStream_t s);
hipError_t launch_linear(const LinearCall& c, hipStream_t s);

hipError_t launch_rmsnorm(const float* x, const void* gain, float eps, void* out, int rows, int n, hipStream_t s);
bool reduce_resid_norm_fits(int n);
hipError_t launch_reduce_resid_norm(const float* ws, int splits, int M, int NP, int n, float* x, const void* gain,
                                    float eps, void* h, hipStream_t s);

struct KvView {
  uint16_t* k;            // [regions][nblk][Hkv][D / 8][bs][8]
  uint16_t* v;            // [regions][nblk][Hkv][D][bs]
  int nblk, regions;
  int hkv, d, bs;
};

struct RopeCall {
  const uint16_t* qkv;    // bf16 projection output [B][heads * D], or
  const float* ws;        // its split-K partials [splits][B][ws_np] (reduced here, in split order, + bias)
  int splits, ws_np;
  const uint16_t* bias;   // with ws only
  const int32_t* positions;
  const int32_t* block_tables;
  int max_blocks, batch;
  int hq, hkv, d;
  const uint16_t* g_q;
  const uint16_t* g_k;
  float qk_eps;
  const float* rope_cos;  // [max_seq][D/2]
  const float* rope_sin;
  int max_seq;
  KvView kv;
  int region;
  uint16_t* q_out;
  uint32_t* err;
};
hipError_t launch_rope_append(const RopeCall& c, hipStream_t s);
hipError_t launch_slot_mapping(const int32_t* positions, const int32_t* bt, int max_blocks, int batch, int bs,
                               int nblk, int32_t* slots, uint32_t* err, hipStream_t s);

struct AttnCall {
  const uint16_t* q;  // [B][Hq][D]
  const int32_t* positions;
  const int32_t* block_tables;
  int max_blocks, batch;
  int hq, hkv, d;
  KvView kv;
  int region;
  uint16_t* out;      // [B][Hq][D]
  float* part;        // partials [B][Hkv][max_parts] records of Hq/Hkv*D + 32 floats: o[Hq/Hkv][D], (m, l) per head, pad
  int max_parts;
  uint32_t* err;
  int num_cus;
  int32_t* plan;      // work list written by launch_attn_plan: [0] count, [1 + i] b | part << 16
  int part_tokens;    // partition length, set by launch_attention (attn_part_tokens_for)
};
int attn_part_tokens();  // the partition quantum (and shortest partition)
int attn_part_tokens_for(int batch, int hkv, int max_tokens, int num_cus);
size_t attn_ws_bytes(int max_batch, int hq, int hkv, int d, int max_seq);
size_t attn_plan_bytes(int max_batch, int max_parts);
// Builds the work list from positions; needed once per set of positions (a
// decode step shares it across its layers). Reads positions, batch,
// max_blocks, kv.bs, plan, err.
hipError_t launch_attn_plan(const AttnCall& c, hipStream_t s);
// With `start`/`stop`, the events take the start time of the attention's
// first kernel and the end time of its last from those kernels' own
// dispatches (no marker packets between the kernels of the stream).
hipError_t launch_attention(const AttnCall& c, hipStream_t s, hipEvent_t start = nullptr,
                            hipEvent_t stop = nullptr);

hipError_t launch_copy(const void* src, void* dst, size_t bytes, int grid, hipStream_t s);

// Rows moved between per-replica buffers and one contiguous staging buffer:
// staging row i belongs to replica r with row_off[r] <= i < row_off[r + 1].
constexpr int kMaxReplicas = 16;
struct RowMove {
  void* rep[kMaxReplicas];
  int row_off[kMaxReplicas + 1];
  int n;             // replicas listed
  size_t row_bytes;  // a multiple of 16
  void* staging;
  int gather;        // 1: replicas -> staging; 0: staging -> replicas
};
hipError_t launch_rows_move(const RowMove& m, hipStream_t s);
// loads: 16-byte loads in flight per lane (2, 4 or 8): how hard the fill
// presses on HBM while it shares the chip with the layer kernels
hipError_t launch_fill_bg(const void* src, void* dst, size_t bytes, int num_cus, int loads, hipStream_t s);
hipError_t launch_poison(void* dst, size_t bytes, hipStream_t s);
hipError_t launch_spin(int64_t cycles, hipStream_t s);

}  // namespace sidp
