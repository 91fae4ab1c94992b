// Per-head QK RMSNorm (Qwen3 family), rotary embedding, and the append of the
// new token's key and value to the paged KV cache (K3), plus the slot mapping
// slot = block_table[p / bs] * bs + p % bs (K9). One wave per (sequence,
// head), four heads per workgroup; lane i owns the rotate-half pair
// (i, i + D/2). The projection output is read either as bf16 or, when the QKV
// projection left split-K partials, reduced here: the partials are summed in
// split order, the bias added and the result rounded to bf16, which is the
// same value the projection's own reduction would have stored.
#include "common.h"
#include "internal.h"

namespace sidp {

__global__ void __launch_bounds__(256) k_rope_append(RopeCall c) {
  const int b = blockIdx.x;
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int D = c.d, half = D >> 1;
  const int heads = c.hq + 2 * c.hkv;
  const int h = blockIdx.y * 4 + wave;
  if (h >= heads) return;
  const int pos = c.positions[b];
  const int lb = pos >= 0 ? pos / c.kv.bs : -1;
  const bool ok_pos = pos >= 0 && lb < c.max_blocks && pos < c.max_seq;
  const int blk = ok_pos ? c.block_tables[(int64_t)b * c.max_blocks + lb] : -1;
  const bool ok_blk = blk >= 0 && blk < c.kv.nblk;
  if (threadIdx.x == 0 && blockIdx.y == 0) {
    if (!ok_pos) atomicOr(c.err, SIDP_DEVERR_POSITION);
    else if (!ok_blk) atomicOr(c.err, SIDP_DEVERR_BLOCK);
  }
  const int off = ok_pos ? pos % c.kv.bs : 0;
  const int rpos = ok_pos ? pos : 0;
  const int64_t region_base = (int64_t)c.region * c.kv.nblk;

  const bool is_q = h < c.hq, is_k = !is_q && h < c.hq + c.hkv;
  const bool act = lane < half;
  const int col0 = h * D + lane, col1 = col0 + half;
  uint16_t v0 = 0, v1 = 0;  // the bf16 projection output of this lane's pair
  if (act) {
    if (c.ws) {
      // four splits' partials in flight at a time, summed in split order
      float s0 = 0.f, s1 = 0.f;
      for (int sp0 = 0; sp0 < c.splits; sp0 += 4) {
        float p0[4], p1[4];
#pragma unroll
        for (int j = 0; j < 4; j++)
          if (sp0 + j < c.splits) {
            const float* pr = c.ws + ((int64_t)(sp0 + j) * c.batch + b) * c.ws_np;
            p0[j] = pr[col0];
            p1[j] = pr[col1];
          }
#pragma unroll
        for (int j = 0; j < 4; j++)
          if (sp0 + j < c.splits) {
            s0 += p0[j];
            s1 += p1[j];
          }
      }
      if (c.bias) {
        s0 += bf2f(c.bias[col0]);
        s1 += bf2f(c.bias[col1]);
      }
      v0 = f2bf(s0);
      v1 = f2bf(s1);
    } else {
      const uint16_t* src = c.qkv + (int64_t)b * heads * D;
      v0 = src[col0];
      v1 = src[col1];
    }
  }
  if (!is_q && !is_k) {  // value head: store as is, transposed block layout [d][token]
    if (act && ok_blk) {
      const int vh = h - c.hq - c.hkv;
      uint16_t* vb = c.kv.v + ((region_base + blk) * c.kv.hkv + vh) * (int64_t)D * c.kv.bs;
      vb[(int64_t)lane * c.kv.bs + off] = v0;
      vb[(int64_t)(lane + half) * c.kv.bs + off] = v1;
    }
    return;
  }
  float x0 = bf2f(v0), x1 = bf2f(v1);
  const uint16_t* gn = is_q ? c.g_q : c.g_k;
  if (gn) {
    const float ss = wave_sum(x0 * x0 + x1 * x1);
    const float r = 1.0f / sqrtf(ss / (float)D + c.qk_eps);
    if (act) {
      x0 = x0 * r * bf2f(gn[lane]);
      x1 = x1 * r * bf2f(gn[lane + half]);
    }
  }
  if (!act) return;
  const float cs = c.rope_cos[(int64_t)rpos * half + lane];
  const float sn = c.rope_sin[(int64_t)rpos * half + lane];
  const float y0 = x0 * cs - x1 * sn;
  const float y1 = x1 * cs + x0 * sn;
  if (is_q) {
    uint16_t* qo = c.q_out + ((int64_t)b * c.hq + h) * D;
    qo[lane] = f2bf(y0);
    qo[lane + half] = f2bf(y1);
  } else if (ok_blk) {
    // key blocks are [d / 8][token][d % 8]
    const int kh = h - c.hq;
    uint16_t* kb = c.kv.k + ((region_base + blk) * c.kv.hkv + kh) * (int64_t)D * c.kv.bs;
    const int d0 = lane, d1 = lane + half;
    kb[((d0 >> 3) * c.kv.bs + off) * 8 + (d0 & 7)] = f2bf(y0);
    kb[((d1 >> 3) * c.kv.bs + off) * 8 + (d1 & 7)] = f2bf(y1);
  }
}

hipError_t launch_rope_append(const RopeCall& c, hipStream_t s) {
  if (c.batch <= 0) return hipSuccess;
  const int heads = c.hq + 2 * c.hkv;
  k_rope_append<<<dim3(c.batch, (heads + 3) / 4), 256, 0, s>>>(c);
  return hipGetLastError();
}

__global__ void k_slot_mapping(const int32_t* __restrict__ positions, const int32_t* __restrict__ bt, int max_blocks,
                               int batch, int bs, int nblk, int32_t* __restrict__ slots, uint32_t* err) {
  const int b = blockIdx.x * blockDim.x + threadIdx.x;
  if (b >= batch) return;
  const int p = positions[b];
  int s = -1;
  if (p < 0 || p / bs >= max_blocks) {
    atomicOr(err, SIDP_DEVERR_POSITION);
  } else {
    const int blk = bt[(int64_t)b * max_blocks + p / bs];
    if (blk < 0 || blk >= nblk) atomicOr(err, SIDP_DEVERR_BLOCK);
    else s = blk * bs + p % bs;
  }
  slots[b] = s;
}

hipError_t launch_slot_mapping(const int32_t* positions, const int32_t* bt, int max_blocks, int batch, int bs,
                               int nblk, int32_t* slots, uint32_t* err, hipStream_t s) {
  if (batch <= 0) return hipSuccess;
  k_slot_mapping<<<(batch + 255) / 256, 256, 0, s>>>(positions, bt, max_blocks, batch, bs, nblk, slots, err);
  return hipGetLastError();
}

}  // namespace sidp
