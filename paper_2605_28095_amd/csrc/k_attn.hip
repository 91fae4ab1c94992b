// Paged grouped-query decode attention on gfx950 (K4).
//
// Work is a list of items (sequence b, partition p, KV head g). The partition
// length is chosen per launch (attn_part_tokens_for): whole sequences when
// the batch alone gives every workgroup several items, else as many
// 2048-token multiples as that takes. A planning kernel, run once per set of
// positions, lists the full partitions first and then each sequence's shorter
// last partition by decreasing length; a persistent grid of 4-wave workgroups
// walks that list in snake order (workgroup w takes items w, 2G - 1 - w,
// 2G + w, ...), which keeps the workgroups' totals within about one short item
// of each other. Within an item each wave owns a quarter of the tokens,
// processed in chunks of 32 tokens = two 16-token KV blocks, with the next
// chunk's K/V loads in flight while the current one computes. The query heads of a KV group (up to
// 16) ride in the MFMA's 16 columns, so every KV byte is read once for all of
// them:
//   S^T[token][head] = K[token][:] . Q^T[:][head]   (v_mfma_f32_16x16x32_bf16)
//   O^T[dim][head]  += V^T[dim][token] . P[token][head]
// V blocks are stored transposed ([d][token]) so V^T fragments are 8-byte row
// pieces; the MFMA's k order of tokens is permuted identically on P and V^T so
// that the softmax probabilities never leave the lanes that computed them. P
// is split into high and low bf16 parts (two MFMAs), keeping the product at
// fp32-like accuracy. Softmax is online in base-2 units; the four waves of an
// item are merged in LDS; a sequence spanning several partitions is merged
// by a log-sum-exp combine kernel. Every reduction has a fixed order.
#include <hip/hip_ext.h>
#include "common.h"
#include "internal.h"

namespace sidp {

constexpr int kPartQuantum = 2048;  // partition lengths are multiples of this
constexpr float kLog2e = 1.4426950408889634f;

int attn_part_tokens() { return kPartQuantum; }

// Partition length of a launch. Whole sequences (no partial records and no
// combine) when batch x Hkv items already give each of the 2 x CUs persistent
// workgroups four of them; otherwise the longest sequence the block tables
// allow is cut into as many pieces as that takes, rounded up to the quantum.
// Partials written for a later merge cost HBM writes beside the KV stream
// that slow it by more than their bytes, so fewer partitions are better as
// long as the workgroups stay balanced.
int attn_part_tokens_for(int batch, int hkv, int max_tokens, int num_cus) {
  const int64_t items = (int64_t)std::max(batch, 1) * std::max(hkv, 1);
  const int64_t want = 4 * 2 * (int64_t)std::max(num_cus, 1);
  const int64_t pieces = items >= want ? 1 : (want + items - 1) / items;
  const int64_t p = (max_tokens + pieces - 1) / pieces;
  return (int)std::max<int64_t>(kPartQuantum, (p + kPartQuantum - 1) / kPartQuantum * kPartQuantum);
}

// One partial record per (sequence, KV head, partition): the group's outputs
// o[group][D], then a 128-byte line with (m, l) of each query head, zero
// padded. Records are whole cache lines (group * D is a multiple of 64), so
// every write of a record covers whole lines: HBM has no write mask, and a
// partly written line costs the memory controller a read-modify-write.
static __host__ __device__ inline int attn_rec_floats(int group, int d) { return group * d + 32; }

size_t attn_ws_bytes(int max_batch, int hq, int hkv, int d, int max_seq) {
  const int parts = (max_seq + kPartQuantum - 1) / kPartQuantum;
  return (size_t)max_batch * hkv * parts * attn_rec_floats(hq / hkv, d) * sizeof(float);
}

size_t attn_plan_bytes(int max_batch, int max_parts) { return (1 + (size_t)max_batch * max_parts) * sizeof(int32_t); }

// The work list. plan[0] = number of (sequence, partition) entries; entry i is
// plan[1 + i] = b | part << 16. Full partitions (ptok tokens) come first, in
// (b, part) order; then the last, shorter partition of every sequence that
// has one, by decreasing length and then increasing b (a bitonic sort in
// LDS). Positions outside a sequence's block table give no entries and set
// the position error bit.
__global__ void __launch_bounds__(256) k_attn_plan(const int32_t* __restrict__ positions, int batch, int np2,
                                                   int max_tokens, int ptok, int32_t* __restrict__ plan,
                                                   uint32_t* __restrict__ err) {
  extern __shared__ int lds_plan[];
  int* s_key = lds_plan;     // [np2] tokens in the last partition (0: none)
  int* s_b = s_key + np2;    // [np2] its sequence
  int* s_full = s_b + np2;   // [batch] full partitions of each sequence
  __shared__ int s_scan[256];
  __shared__ int s_npart;
  const int t = threadIdx.x;
  if (t == 0) s_npart = 0;
  __syncthreads();
  for (int b = t; b < np2; b += 256) {
    int full = 0, rem = 0;
    if (b < batch) {
      const int seq = positions[b] + 1;
      if (seq >= 1 && seq <= max_tokens) {
        full = seq / ptok;
        rem = seq % ptok;
      } else {
        atomicOr(err, SIDP_DEVERR_POSITION);
      }
      s_full[b] = full;
      if (rem > 0) atomicAdd(&s_npart, 1);
    }
    s_key[b] = rem;
    s_b[b] = b;
  }
  __syncthreads();
  // exclusive prefix of the full counts; thread t owns sequences [t * per, t * per + per)
  const int per = (batch + 255) / 256;
  int local = 0;
  for (int i = 0; i < per; i++) {
    const int b = t * per + i;
    if (b < batch) local += s_full[b];
  }
  s_scan[t] = local;
  __syncthreads();
  for (int off = 1; off < 256; off <<= 1) {
    const int v = t >= off ? s_scan[t - off] : 0;
    __syncthreads();
    s_scan[t] += v;
    __syncthreads();
  }
  int run = s_scan[t] - local;
  for (int i = 0; i < per; i++) {
    const int b = t * per + i;
    if (b < batch) {
      for (int p = 0; p < s_full[b]; p++) plan[1 + run + p] = b | (p << 16);
      run += s_full[b];
    }
  }
  const int nfull = s_scan[255];
  // bitonic sort of (length descending, b ascending)
  for (int k = 2; k <= np2; k <<= 1) {
    for (int j = k >> 1; j > 0; j >>= 1) {
      __syncthreads();
      for (int i = t; i < np2; i += 256) {
        const int l = i ^ j;
        if (l > i) {
          const int ki = s_key[i], kl = s_key[l], bi = s_b[i], bl = s_b[l];
          const bool i_first = ki > kl || (ki == kl && bi < bl);
          if (((i & k) == 0) != i_first) {
            s_key[i] = kl;
            s_key[l] = ki;
            s_b[i] = bl;
            s_b[l] = bi;
          }
        }
      }
    }
  }
  __syncthreads();
  for (int i = t; i < s_npart; i += 256) {
    const int b = s_b[i];
    plan[1 + nfull + i] = b | (s_full[b] << 16);
  }
  if (t == 0) plan[0] = nfull + s_npart;
}

template <int D>
struct Chunk {
  u32x4_t k[2][D / 32];  // K fragments: token lane&15, dims (lane>>4)*8 + 32kk
  u32x2_t v[D / 16][2];  // V^T fragments: dim 16jd + lane&15, tokens (lane>>4)*4..+3
};

// Block tables and positions are read through the scalar cache: the reads are
// uniform per wave and nothing writes those arrays during the kernel, and
// scalar loads are counted apart from the vector loads of the KV stream. (A
// vector load of a block index would have to complete before the next
// chunk's addresses exist, and vector loads complete in order, so every such
// read would drain the chunk already in flight.)
typedef const __attribute__((address_space(4))) int32_t cint32_t;

// A chunk's source: one KV head of one sequence, tokens t0 .. t0 + 31.
struct ChunkSrc {
  cint32_t* bt;
  int seq, g, t0;
};

// Loads the 24 fragments of a chunk. Every call issues the same loads, so the
// compiler's wait before a chunk's compute counts exactly the other buffer's
// loads. A block's base address is uniform (scalar registers); each lane adds
// a fixed 32-bit byte offset, k_lane or v_lane, so no 64-bit per-lane address
// is rebuilt per chunk. An out-of-range block index is replaced by block 0
// and flagged.
template <int D>
__device__ __forceinline__ void load_chunk(const AttnCall& a, const ChunkSrc& src, int64_t region_blk,
                                           uint32_t k_lane, uint32_t v_lane, bool& bad, Chunk<D>& c) {
  constexpr int KK = D / 32, JD = D / 16;
  constexpr int64_t kBlockBytes = 16 * D * 2;  // one KV head of one 16-token block, K or V
  int blk[2];
  blk[0] = src.bt[src.t0 >> 4];
  blk[1] = (src.t0 + 16 < src.seq) ? src.bt[(src.t0 >> 4) + 1] : blk[0];
#pragma unroll
  for (int j = 0; j < 2; j++) {
    if (blk[j] < 0 || blk[j] >= a.kv.nblk) {
      bad = true;
      blk[j] = 0;
    }
  }
#pragma unroll
  for (int j = 0; j < 2; j++) {
    const int64_t off = ((region_blk + blk[j]) * a.kv.hkv + src.g) * kBlockBytes;
    const char* kb = (const char*)a.kv.k + off;
    const char* vb = (const char*)a.kv.v + off;
    // non-temporal: each KV byte is read once per layer, and streaming loads
    // that do not allocate in the caches read HBM about 10% faster
#pragma unroll
    for (int kk = 0; kk < KK; kk++) c.k[j][kk] = __builtin_nontemporal_load((const u32x4_t*)(kb + k_lane + kk * 1024));
#pragma unroll
    for (int jd = 0; jd < JD; jd++) c.v[jd][j] = __builtin_nontemporal_load((const u32x2_t*)(vb + v_lane + jd * 512));
  }
}

// Tokens from `te` on (the end of this wave's range) are masked; a chunk that
// starts at or past `te` changes nothing: every score is -inf, so P is 0 and
// alpha is 1 (or 0 while m_run is still -inf, when o and l_run are 0 anyway:
// the exponents are then taken against 0 instead of -inf).
template <int D>
__device__ __forceinline__ void compute_chunk(const Chunk<D>& c, const bf16x8_t (&qb)[D / 32], int t0, int te,
                                              int lane, float scale, float& m_run, float& l_run,
                                              f32x4_t (&o)[D / 16]) {
  constexpr int KK = D / 32, JD = D / 16;
  const int lg = lane >> 4;
  f32x4_t s[2];
#pragma unroll
  for (int j = 0; j < 2; j++) {
    s[j] = f32x4_t{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int kk = 0; kk < KK; kk++)
      s[j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(as_bf16x8(c.k[j][kk]), qb[kk], s[j], 0, 0, 0);
  }
  const bool tail = t0 + 32 > te;
  float cmax = -INFINITY;
#pragma unroll
  for (int j = 0; j < 2; j++)
#pragma unroll
    for (int r = 0; r < 4; r++) {
      float v = s[j][r] * scale;
      if (tail && t0 + 16 * j + lg * 4 + r >= te) v = -INFINITY;
      s[j][r] = v;
      cmax = fmaxf(cmax, v);
    }
  cmax = fmaxf(cmax, __shfl_xor(cmax, 16, 64));
  cmax = fmaxf(cmax, __shfl_xor(cmax, 32, 64));
  const float m_new = fmaxf(m_run, cmax);
  const float m_ref = m_new == -INFINITY ? 0.f : m_new;
  const float alpha = exp2f(m_run - m_ref);
  m_run = m_new;
  float p[8];
  float psum = 0.f;
#pragma unroll
  for (int r = 0; r < 4; r++) {
    p[r] = exp2f(s[0][r] - m_ref);      // slots 0..3: block 0 tokens lg*4 + r
    p[4 + r] = exp2f(s[1][r] - m_ref);  // slots 4..7: block 1 tokens lg*4 + r
    psum += p[r] + p[4 + r];
  }
  l_run = l_run * alpha + psum;
  // P as high + low bf16 parts
  uint32_t hi[4], lo[4];
#pragma unroll
  for (int i = 0; i < 4; i++) {
    hi[i] = pack_bf2(p[2 * i], p[2 * i + 1]);
    lo[i] = pack_bf2(p[2 * i] - bf2f((uint16_t)(hi[i] & 0xffffu)), p[2 * i + 1] - bf2f((uint16_t)(hi[i] >> 16)));
  }
  const bf16x8_t pb = as_bf16x8(u32x4_t{hi[0], hi[1], hi[2], hi[3]});
  const bf16x8_t pl = as_bf16x8(u32x4_t{lo[0], lo[1], lo[2], lo[3]});
#pragma unroll
  for (int jd = 0; jd < JD; jd++) {
    u32x2_t v0 = c.v[jd][0], v1 = c.v[jd][1];
    if (tail) {  // invalid tokens may hold anything (NaN); zero them so 0 * V stays 0
      const int tb = t0 + lg * 4;
      if (tb + 0 >= te) v0.x &= 0xffff0000u;
      if (tb + 1 >= te) v0.x &= 0x0000ffffu;
      if (tb + 2 >= te) v0.y &= 0xffff0000u;
      if (tb + 3 >= te) v0.y &= 0x0000ffffu;
      if (tb + 16 >= te) v1.x &= 0xffff0000u;
      if (tb + 17 >= te) v1.x &= 0x0000ffffu;
      if (tb + 18 >= te) v1.y &= 0xffff0000u;
      if (tb + 19 >= te) v1.y &= 0x0000ffffu;
    }
    const bf16x8_t va = as_bf16x8(u32x4_t{v0.x, v0.y, v1.x, v1.y});
    o[jd] = o[jd] * alpha;
    o[jd] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(va, pb, o[jd], 0, 0, 0);
    o[jd] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(va, pl, o[jd], 0, 0, 0);
  }
}

__device__ __forceinline__ int seq_parts(const AttnCall& a, int b) {
  const int seq = a.positions[b] + 1;
  if (seq < 1 || seq > a.max_blocks * a.kv.bs) return 0;  // position outside its block table
  return (seq + a.part_tokens - 1) / a.part_tokens;
}

// Item i of the work list is (entry i / Hkv of the plan, KV head i % Hkv).
// Two 4-wave workgroups per CU; a wave holds 218 VGPRs (224 allocated), so
// two of them and a slot-fill wave (at most 48) fit in a SIMD's 512.
template <int D>
__global__ void __launch_bounds__(256, 2) k_attn(AttnCall a) {
  constexpr int KK = D / 32, JD = D / 16;
  extern __shared__ __attribute__((aligned(16))) float smem_f[];
  float* s_m = smem_f;                             // [4][16]
  float* s_l = s_m + 64;                           // [4][16]
  float* s_o = s_l + 64;                           // [4][16][D + 1]

  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6), lane = threadIdx.x & 63;
  const int head = lane & 15, lg = lane >> 4;
  const int group = a.hq / a.hkv;

  cint32_t* plan = (cint32_t*)a.plan;
  const int total_items = plan[0] * a.hkv;
  const float scale = kLog2e / sqrtf((float)D);
  const int64_t region_blk = (int64_t)a.region * a.kv.nblk;
  cint32_t* positions = (cint32_t*)a.positions;

  // An item's parameters; all uniform. This wave's tokens are [tb, te).
  struct Item {
    int b, part, nparts, seq, g, tb, te;
    cint32_t* bt;
  };
  auto get_item = [&](int item, Item& it) {
    const int e = plan[1 + item / a.hkv];
    it.g = item % a.hkv;
    it.b = e & 0xffff;
    it.part = e >> 16;
    it.seq = positions[it.b] + 1;
    it.nparts = (it.seq + a.part_tokens - 1) / a.part_tokens;
    it.bt = (cint32_t*)(a.block_tables + (int64_t)it.b * a.max_blocks);
    // the partition's tokens split evenly over the four waves in whole pairs of
    // 32-token chunks (only the last wave's remainder can be an odd count, whose
    // masked extra chunk re-reads HBM: non-temporal loads leave nothing in L2),
    // so a sequence's shorter last partition keeps all four waves loading
    const int len = min(it.seq - it.part * a.part_tokens, a.part_tokens);
    const int share = ((len + 3) / 4 + 63) / 64 * 64;
    it.tb = it.part * a.part_tokens + wave * share;
    it.te = min(it.tb + share, it.seq);
  };
  // the r-th item of this workgroup in snake order over the sorted list
  auto item_of = [&](int r) {
    const int G = gridDim.x;
    return (r & 1) ? (r + 1) * G - 1 - (int)blockIdx.x : r * G + (int)blockIdx.x;
  };
  // Query heads ride in the 16 MFMA columns; lanes past the group load a
  // duplicate of the group's first head (finite values whose columns are never
  // merged or written), so the loaded fragments feed the MFMA unmodified and
  // no wait is needed until the first chunk's compute.
  auto load_q = [&](const Item& it, bf16x8_t (&q)[KK]) {
    const int qh = it.g * group + (head < group ? head : 0);
#pragma unroll
    for (int kk = 0; kk < KK; kk++)
      q[kk] = as_bf16x8(*(const u32x4_t*)(a.q + ((int64_t)it.b * a.hq + qh) * D + lg * 8 + kk * 32));
  };

  // K fragment: token lane & 15, dims (lane >> 4) * 8 + 32 kk; V^T fragment:
  // dim 16 jd + (lane & 15), tokens (lane >> 4) * 4 .. + 3 (byte offsets).
  // K blocks are stored [d / 8][token][d % 8], so the K fragment of MFMA kk is
  // the contiguous 1 KB run of 16-byte pieces 64 kk + lane: whole cache lines
  // per load instruction, which streaming (non-temporal) loads need.
  const uint32_t k_lane = (uint32_t)lane * 16u;
  const uint32_t v_lane = (uint32_t)(head * 16 + lg * 4) * 2u;
  bool bad = false;
  int round = 0;
  int item = item_of(0);
  if (item < total_items) {
    // The chunk stream of a wave runs across its items: the load slot after an
    // item's last chunk fetches the first chunk of the wave's part of the next
    // item (or, if there is none, re-reads the last chunk: an L2 hit that keeps
    // every iteration's loads identical), so that load is in flight while the
    // item's partial results are merged and written.
    Item cur;
    get_item(item, cur);
    bf16x8_t qb[KK];
    load_q(cur, qb);
    // Wait for the first queries here, once: later the merge reuses dead
    // query registers, and a load into them still pending on some path (a
    // wave without tokens in its first item never reads qb) would make that
    // reuse wait for every load in flight.
#pragma unroll
    for (int kk = 0; kk < KK; kk++) asm volatile("" ::"v"(qb[kk]));
    Chunk<D> ca, cb;
    // (a wave without tokens in its first item reads the item's first chunk: masked)
    load_chunk<D>(a, ChunkSrc{cur.bt, cur.seq, cur.g, cur.tb < cur.te ? cur.tb : cur.part * a.part_tokens}, region_blk,
                  k_lane, v_lane, bad, ca);
    for (;;) {
      const int nitem = item_of(round + 1);
      const bool has_next = nitem < total_items;
      Item nx = cur;
      if (has_next) get_item(nitem, nx);
      const bool pf = has_next && nx.tb < nx.te;
      const int n = cur.te > cur.tb ? (cur.te - cur.tb + 31) / 32 : 0;  // this wave's chunks in the item
      // Chunks are taken in pairs, at least one pair per item: an odd count
      // gets a masked extra chunk, a wave without tokens two, so that every
      // path through an item issues its loads in the same order, the prefetch
      // always lands in ca, and no wait the compiler places for a register
      // reuse or copy reaches a load still in flight.
      const int n2 = __builtin_amdgcn_readfirstlane(max(2, (n + 1) & ~1));
      // source of stream slot i of this item (slot n2 is the prefetch; the
      // extra chunk and a missing prefetch re-read the last chunk, or the
      // item's first chunk when this wave has none: L2 hits)
      auto src_of = [&](int i) -> ChunkSrc {
        if (i < n) return ChunkSrc{cur.bt, cur.seq, cur.g, cur.tb + 32 * i};
        if (i == n2 && pf) return ChunkSrc{nx.bt, nx.seq, nx.g, nx.tb};
        return ChunkSrc{cur.bt, cur.seq, cur.g, n > 0 ? cur.tb + 32 * (n - 1) : cur.part * a.part_tokens};
      };

      float m_run = -INFINITY, l_run = 0.f;
      f32x4_t o[JD];
#pragma unroll
      for (int j = 0; j < JD; j++) o[j] = f32x4_t{0.f, 0.f, 0.f, 0.f};
      int ci = 0;
      do {
        load_chunk<D>(a, src_of(ci + 1), region_blk, k_lane, v_lane, bad, cb);
        compute_chunk<D>(ca, qb, cur.tb + 32 * ci, cur.te, lane, scale, m_run, l_run, o);
        load_chunk<D>(a, src_of(ci + 2), region_blk, k_lane, v_lane, bad, ca);
        compute_chunk<D>(cb, qb, cur.tb + 32 * (ci + 1), cur.te, lane, scale, m_run, l_run, o);
        ci += 2;
      } while (ci < n2);
      // qb is dead until the next item's first chunk: load the next item's
      // queries into it (this item's again when it is the last one, so that
      // every path issues the same loads)
      load_q(nx, qb);

      l_run += __shfl_xor(l_run, 16, 64);
      l_run += __shfl_xor(l_run, 32, 64);
      if (lg == 0) {
        s_m[wave * 16 + head] = m_run;
        s_l[wave * 16 + head] = l_run;
      }
#pragma unroll
      for (int jd = 0; jd < JD; jd++)
#pragma unroll
        for (int r = 0; r < 4; r++) s_o[(wave * 16 + head) * (D + 1) + jd * 16 + lg * 4 + r] = o[jd][r];
      __syncthreads();
      // Merge the four waves' results: the output rows of a one-partition
      // sequence, else the item's partial record (each wave writes whole
      // lines of it, the first 32 threads its (m, l) line).
      {
        const int64_t row0 = (int64_t)cur.b * a.hq + cur.g * group;  // the group's first query head
        const int rf = attn_rec_floats(group, D);
        float* rec = a.part + ((int64_t)(cur.b * a.hkv + cur.g) * a.max_parts + cur.part) * rf;
        for (int i = threadIdx.x; i < group * D; i += 256) {
          const int hh = i / D, d = i % D;
          float M = -INFINITY;
#pragma unroll
          for (int w = 0; w < 4; w++) M = fmaxf(M, s_m[w * 16 + hh]);
          float L = 0.f, O = 0.f;
#pragma unroll
          for (int w = 0; w < 4; w++) {
            const float mw = s_m[w * 16 + hh];
            const float f = (mw == -INFINITY) ? 0.f : exp2f(mw - M);
            L += s_l[w * 16 + hh] * f;
            O += s_o[(w * 16 + hh) * (D + 1) + d] * f;
          }
          if (cur.nparts == 1) a.out[(row0 + hh) * D + d] = f2bf(O / L);
          else rec[i] = O;
        }
        if (cur.nparts > 1 && threadIdx.x < 32) {
          const int t = threadIdx.x, hh = t >> 1;
          float v = 0.f;
          if (hh < group) {
            float M = -INFINITY;
#pragma unroll
            for (int w = 0; w < 4; w++) M = fmaxf(M, s_m[w * 16 + hh]);
            float L = 0.f;
#pragma unroll
            for (int w = 0; w < 4; w++) {
              const float mw = s_m[w * 16 + hh];
              L += s_l[w * 16 + hh] * ((mw == -INFINITY) ? 0.f : exp2f(mw - M));
            }
            v = (t & 1) ? L : M;
          }
          rec[group * D + t] = v;
        }
      }
      __syncthreads();  // s_m, s_l and s_o are reused by the next item
      if (!has_next) break;
      cur = nx;
      item = nitem;
      round++;
    }
  }
  if (bad && lane == 0) atomicOr(a.err, SIDP_DEVERR_BLOCK);
}

// Log-sum-exp merge of a sequence's partitions: one workgroup per (KV head,
// sequence) covering the group's query heads, four dims per thread (16-byte
// loads from the partial records). Partitions are summed in index order.
template <int D>
__global__ void __launch_bounds__(256) k_attn_combine(AttnCall a) {
  const int g = blockIdx.x, b = blockIdx.y;
  const int group = a.hq / a.hkv;
  const int nparts = seq_parts(a, b);
  if (nparts <= 1) return;
  const int rf = attn_rec_floats(group, D);
  const float* recs = a.part + ((int64_t)b * a.hkv + g) * a.max_parts * rf;  // partition j at j * rf
  for (int i = threadIdx.x; i < group * (D / 4); i += 256) {
    const int hh = i / (D / 4), d = (i % (D / 4)) * 4;
    const float* ml = recs + group * D + 2 * hh;  // (m, l) of head hh, partition 0
    float M = -INFINITY;
    for (int j = 0; j < nparts; j++) M = fmaxf(M, ml[j * rf]);
    float L = 0.f;
    f32x4_t O = {0.f, 0.f, 0.f, 0.f};
    for (int j = 0; j < nparts; j++) {
      const float f = exp2f(ml[j * rf] - M);
      L += ml[j * rf + 1] * f;
      const f32x4_t v = *(const f32x4_t*)(recs + j * rf + hh * D + d);
      O += v * f;
    }
    uint16_t* o = a.out + ((int64_t)b * a.hq + g * group + hh) * D + d;
    *(uint32_t*)o = pack_bf2(O[0] / L, O[1] / L);
    *(uint32_t*)(o + 2) = pack_bf2(O[2] / L, O[3] / L);
  }
}

hipError_t launch_attn_plan(const AttnCall& c, hipStream_t s) {
  if (c.batch <= 0) return hipSuccess;
  int np2 = 1;
  while (np2 < c.batch) np2 <<= 1;
  const size_t lds = (size_t)(2 * np2 + c.batch) * sizeof(int);
  if (lds > 64 * 1024) return hipErrorInvalidValue;
  const int max_tokens = c.max_blocks * c.kv.bs;
  const int ptok = attn_part_tokens_for(c.batch, c.hkv, max_tokens, c.num_cus);
  k_attn_plan<<<1, 256, lds, s>>>(c.positions, c.batch, np2, max_tokens, ptok, c.plan, c.err);
  return hipGetLastError();
}

template <int D>
static hipError_t launch_d(const AttnCall& c, int grid, int parts, hipStream_t s, hipEvent_t start, hipEvent_t stop) {
  const size_t lds = (size_t)(128 + 4 * 16 * (D + 1)) * 4;
  if (lds > 64 * 1024) {
    hipError_t e = hipFuncSetAttribute((const void*)k_attn<D>, hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
    if (e != hipSuccess) return e;
  }
  if (!start && !stop) {
    k_attn<D><<<grid, 256, lds, s>>>(c);
    if (parts > 1) k_attn_combine<D><<<dim3(c.hkv, c.batch), 256, 0, s>>>(c);
    return hipGetLastError();
  }
  // timed: the events ride on the kernels' own dispatches
  AttnCall arg = c;
  void* args[] = {&arg};
  hipError_t e = hipExtLaunchKernel((const void*)k_attn<D>, dim3(grid), dim3(256), args, lds, s, start,
                                    parts > 1 ? nullptr : stop, 0);
  if (e != hipSuccess || parts <= 1) return e;
  return hipExtLaunchKernel((const void*)k_attn_combine<D>, dim3(c.hkv, c.batch), dim3(256), args, 0, s, nullptr, stop,
                            0);
}

hipError_t launch_attention(const AttnCall& call, hipStream_t s, hipEvent_t start, hipEvent_t stop) {
  if (call.batch <= 0) return hipSuccess;
  AttnCall c = call;
  const int max_tokens = c.max_blocks * c.kv.bs;
  c.part_tokens = attn_part_tokens_for(c.batch, c.hkv, max_tokens, c.num_cus);  // as the plan was built
  const int parts = (max_tokens + c.part_tokens - 1) / c.part_tokens;
  if (parts > c.max_parts) return hipErrorInvalidValue;
  if (c.hq / c.hkv > 16) return hipErrorInvalidValue;
  const int grid = 2 * c.num_cus;  // persistent: two 4-wave workgroups per CU
  if (c.d == 128) return launch_d<128>(c, grid, parts, s, start, stop);
  if (c.d == 64) return launch_d<64>(c, grid, parts, s, start, stop);
  return hipErrorInvalidValue;
}

}  // namespace sidp
