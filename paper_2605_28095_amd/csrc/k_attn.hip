// Paged grouped-query decode attention on gfx950 (K4).
//
// Work item: (sequence b, KV head g, 512-token partition); 4 waves, 128
// tokens each, in chunks of 32 tokens = two 16-token KV blocks. The query
// heads of a KV group (up to 16) ride in the MFMA's 16 columns, so every KV
// byte is read once for all heads of its group:
//   S^T[token][head] = K[token][:] . Q^T[:][head]   (v_mfma_f32_16x16x32_bf16,
//                                                    A = K rows straight from the block)
//   O^T[dim][head]  += V^T[dim][token] . P[token][head]
// V blocks are stored transposed ([d][token]) so V^T fragments are 8-byte
// row pieces; the MFMA's k order of tokens is permuted identically on P and
// V^T so that the softmax probabilities never leave the lanes that computed
// them. Softmax is online (running max, rescale) in base-2 units; partitions
// of one (b, g) are merged in LDS and, when a sequence spans several
// partitions, by a log-sum-exp combine kernel. Fixed reduction order: the
// result does not depend on scheduling.
#include "common.h"
#include "internal.h"

namespace sidp {

constexpr int kPartTokens = 512;
constexpr int kWaveTokens = 128;
constexpr float kLog2e = 1.4426950408889634f;

int attn_part_tokens() { return kPartTokens; }

size_t attn_ws_bytes(int max_batch, int hq, int d, int max_seq) {
  const int parts = (max_seq + kPartTokens - 1) / kPartTokens;
  return (size_t)max_batch * hq * parts * (d + 2) * sizeof(float);
}

template <int D>
__global__ void __launch_bounds__(256) k_attn(AttnCall a) {
  constexpr int KK = D / 32;   // k steps of the QK product
  constexpr int JD = D / 16;   // 16-dim column tiles of the PV product
  __shared__ float s_m[4][16], s_l[4][16];
  __shared__ float s_o[4][16][D + 1];

  const int b = blockIdx.z, g = blockIdx.y, part = blockIdx.x;
  const int seq = a.positions[b] + 1;
  if (seq < 1 || seq > a.max_blocks * a.kv.bs) {  // position outside its block table
    if (part == 0 && g == 0 && threadIdx.x == 0) atomicOr(a.err, SIDP_DEVERR_POSITION);
    return;
  }
  const int nparts = (seq + kPartTokens - 1) / kPartTokens;
  if (part >= nparts) return;
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int group = a.hq / a.hkv;
  const int head = lane & 15, lg = lane >> 4;

  // Q^T as the B operand: lane holds dims lg*8..lg*8+7 (+32 kk) of head `head`.
  bf16x8_t qb[KK];
#pragma unroll
  for (int kk = 0; kk < KK; kk++) {
    u32x4_t v = {0u, 0u, 0u, 0u};
    if (head < group) v = *(const u32x4_t*)(a.q + ((int64_t)b * a.hq + g * group + head) * D + lg * 8 + kk * 32);
    qb[kk] = as_bf16x8(v);
  }

  const int t_begin = part * kPartTokens + wave * kWaveTokens;
  const int t_end = min(t_begin + kWaveTokens, seq);
  const float scale = kLog2e / sqrtf((float)D);
  const int64_t region_blk = (int64_t)a.region * a.kv.nblk;
  const int32_t* bt = a.block_tables + (int64_t)b * a.max_blocks;

  float m_run = -INFINITY, l_run = 0.f;
  f32x4_t o[JD];
#pragma unroll
  for (int j = 0; j < JD; j++) o[j] = f32x4_t{0.f, 0.f, 0.f, 0.f};

  for (int t0 = t_begin; t0 < t_end; t0 += 32) {
    const int lb0 = t0 / 16;
    int blk[2];
    blk[0] = bt[lb0];
    blk[1] = (t0 + 16 < seq) ? bt[lb0 + 1] : blk[0];
#pragma unroll
    for (int j = 0; j < 2; j++) {
      if (blk[j] < 0 || blk[j] >= a.kv.nblk) {
        if (lane == 0) atomicOr(a.err, SIDP_DEVERR_BLOCK);
        blk[j] = 0;
      }
    }
    // K fragments (A operand): token lane&15 of block j, dims lg*8 + 32kk.
    u32x4_t kf[2][KK];
#pragma unroll
    for (int j = 0; j < 2; j++) {
      const uint16_t* kp = a.kv.k + (((region_blk + blk[j]) * a.kv.hkv + g) * 16 + head) * D + lg * 8;
#pragma unroll
      for (int kk = 0; kk < KK; kk++) kf[j][kk] = *(const u32x4_t*)(kp + kk * 32);
    }
    // V^T fragments (A operand of PV): dim 16jd + lane&15, tokens lg*4..lg*4+3 of each block.
    u32x2_t vf[JD][2];
#pragma unroll
    for (int j = 0; j < 2; j++) {
      const uint16_t* vp = a.kv.v + ((region_blk + blk[j]) * a.kv.hkv + g) * (int64_t)D * 16 + lg * 4;
#pragma unroll
      for (int jd = 0; jd < JD; jd++) vf[jd][j] = *(const u32x2_t*)(vp + (jd * 16 + head) * 16);
    }

    f32x4_t s[2];
#pragma unroll
    for (int j = 0; j < 2; j++) {
      s[j] = f32x4_t{0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int kk = 0; kk < KK; kk++)
        s[j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(as_bf16x8(kf[j][kk]), qb[kk], s[j], 0, 0, 0);
    }
    // scale, mask, chunk max per head
    float cmax = -INFINITY;
#pragma unroll
    for (int j = 0; j < 2; j++)
#pragma unroll
      for (int r = 0; r < 4; r++) {
        const int t = t0 + 16 * j + lg * 4 + r;
        float v = s[j][r] * scale;
        v = (t < seq) ? v : -INFINITY;
        s[j][r] = v;
        cmax = fmaxf(cmax, v);
      }
    cmax = fmaxf(cmax, __shfl_xor(cmax, 16, 64));
    cmax = fmaxf(cmax, __shfl_xor(cmax, 32, 64));
    const float m_new = fmaxf(m_run, cmax);
    const float alpha = exp2f(m_run - m_new);
    m_run = m_new;
    // Probabilities enter the bf16 MFMA as a high and a low bf16 part
    // (p = hi + lo to about 16 significant bits), so P.V is as accurate as
    // an fp32 product; attention is HBM-bound and the second MFMA is free.
    float psum = 0.f;
    float p[8];
#pragma unroll
    for (int r = 0; r < 4; r++) {
      p[r] = exp2f(s[0][r] - m_new);      // slots 0..3: block 0 tokens lg*4 + r
      p[4 + r] = exp2f(s[1][r] - m_new);  // slots 4..7: block 1 tokens lg*4 + r
      psum += p[r] + p[4 + r];
    }
    l_run = l_run * alpha + psum;
    uint32_t hi[4], lo[4];
#pragma unroll
    for (int i = 0; i < 4; i++) {
      const uint16_t h0 = f2bf(p[2 * i]), h1 = f2bf(p[2 * i + 1]);
      hi[i] = (uint32_t)h0 | ((uint32_t)h1 << 16);
      lo[i] = pack_bf2(p[2 * i] - bf2f(h0), p[2 * i + 1] - bf2f(h1));
    }
    const bf16x8_t pb = as_bf16x8(u32x4_t{hi[0], hi[1], hi[2], hi[3]});
    const bf16x8_t pl = as_bf16x8(u32x4_t{lo[0], lo[1], lo[2], lo[3]});
    const bool tail = t0 + 32 > seq;
#pragma unroll
    for (int jd = 0; jd < JD; jd++) {
      u32x2_t v0 = vf[jd][0], v1 = vf[jd][1];
      if (tail) {  // invalid tokens may hold anything (NaN); zero them so 0 * V stays 0
        const int tb = t0 + lg * 4;
        if (tb + 0 >= seq) v0.x &= 0xffff0000u;
        if (tb + 1 >= seq) v0.x &= 0x0000ffffu;
        if (tb + 2 >= seq) v0.y &= 0xffff0000u;
        if (tb + 3 >= seq) v0.y &= 0x0000ffffu;
        if (tb + 16 >= seq) v1.x &= 0xffff0000u;
        if (tb + 17 >= seq) v1.x &= 0x0000ffffu;
        if (tb + 18 >= seq) v1.y &= 0xffff0000u;
        if (tb + 19 >= seq) v1.y &= 0x0000ffffu;
      }
      const bf16x8_t va = as_bf16x8(u32x4_t{v0.x, v0.y, v1.x, v1.y});
      o[jd] = o[jd] * alpha;
      o[jd] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(va, pb, o[jd], 0, 0, 0);
      o[jd] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(va, pl, o[jd], 0, 0, 0);
    }
  }
  // l over the four lane groups holding different tokens of the same head
  l_run += __shfl_xor(l_run, 16, 64);
  l_run += __shfl_xor(l_run, 32, 64);

  if (lg == 0) {
    s_m[wave][head] = m_run;
    s_l[wave][head] = l_run;
  }
#pragma unroll
  for (int jd = 0; jd < JD; jd++)
#pragma unroll
    for (int r = 0; r < 4; r++) s_o[wave][head][jd * 16 + lg * 4 + r] = o[jd][r];
  __syncthreads();

  // Merge the four waves: thread -> (head, dim) pairs of this group.
  for (int i = threadIdx.x; i < group * D; i += 256) {
    const int hh = i / D, d = i % D;
    float M = -INFINITY;
#pragma unroll
    for (int w = 0; w < 4; w++) M = fmaxf(M, s_m[w][hh]);
    float L = 0.f, O = 0.f;
#pragma unroll
    for (int w = 0; w < 4; w++) {
      const float f = (s_m[w][hh] == -INFINITY) ? 0.f : exp2f(s_m[w][hh] - M);
      L += s_l[w][hh] * f;
      O += s_o[w][hh][d] * f;
    }
    const int qh = g * group + hh;
    if (nparts == 1) {
      a.out[((int64_t)b * a.hq + qh) * D + d] = f2bf(O / L);
    } else {
      float* p = a.part + (((int64_t)b * a.hq + qh) * a.max_parts + part) * (D + 2);
      p[d] = O;
      if (d == 0) {
        p[D] = M;
        p[D + 1] = L;
      }
    }
  }
}

// Log-sum-exp merge of a sequence's partitions: one workgroup per (head, b).
template <int D>
__global__ void __launch_bounds__(D) k_attn_combine(AttnCall a) {
  const int qh = blockIdx.x, b = blockIdx.y;
  const int seq = a.positions[b] + 1;
  if (seq < 1 || seq > a.max_blocks * a.kv.bs) return;
  const int nparts = (seq + kPartTokens - 1) / kPartTokens;
  if (nparts <= 1) return;
  const float* p = a.part + ((int64_t)b * a.hq + qh) * a.max_parts * (D + 2);
  float M = -INFINITY;
  for (int i = 0; i < nparts; i++) M = fmaxf(M, p[i * (D + 2) + D]);
  float L = 0.f, O = 0.f;
  const int d = threadIdx.x;
  for (int i = 0; i < nparts; i++) {
    const float f = exp2f(p[i * (D + 2) + D] - M);
    L += p[i * (D + 2) + D + 1] * f;
    O += p[i * (D + 2) + d] * f;
  }
  a.out[((int64_t)b * a.hq + qh) * D + d] = f2bf(O / L);
}

hipError_t launch_attention(const AttnCall& c, hipStream_t s) {
  if (c.batch <= 0) return hipSuccess;
  const int parts = (c.max_blocks * c.kv.bs + kPartTokens - 1) / kPartTokens;
  if (parts > c.max_parts) return hipErrorInvalidValue;
  dim3 grid(parts, c.hkv, c.batch);
  if (c.d == 128) {
    k_attn<128><<<grid, 256, 0, s>>>(c);
    if (parts > 1) k_attn_combine<128><<<dim3(c.hq, c.batch), 128, 0, s>>>(c);
  } else if (c.d == 64) {
    k_attn<64><<<grid, 256, 0, s>>>(c);
    if (parts > 1) k_attn_combine<64><<<dim3(c.hq, c.batch), 64, 0, s>>>(c);
  } else {
    return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

}  // namespace sidp
