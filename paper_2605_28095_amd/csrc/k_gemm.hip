// Dense projections of the decoder layer on gfx950 MFMA (bf16 in, fp32 accumulate):
// QKV (+bias), O (+residual), gate/up (+SwiGLU), down (+residual).
//
// Shape of the problem: out[M, N] = X[M, K] * W[N, K]^T with M = decode batch
// (8..512) and N, K in the thousands, so the weights dominate the bytes and
// every weight byte must be read exactly once. Design:
//  * Weights are packed once (into the layer's pool blob) in MFMA B-fragment
//    order: for each 64-wide k-tile, for each group of 64 output columns, for
//    each 16-wide k step, two 32x16 fragments of 64 lanes x 8 bf16. A wave
//    that owns a column group streams its weights with 1 KB fully contiguous
//    loads straight into registers (no LDS traffic for W), and the waves of a
//    grid, which move through k together, read adjacent 8 KB pieces.
//  * Activations X are shared by the 4 waves of a workgroup: staged through
//    LDS (64-wide k tiles, double buffered). A row is 128 bytes; its 16-byte
//    chunk c is stored at slot c ^ ((row >> 1) & 7), so the 16 lanes that one
//    LDS cycle serves for a 128-bit fragment read (rows r..r+15, one chunk)
//    hit 16 distinct 16-byte bank groups of the 64 four-byte banks.
//  * A workgroup covers up to 128 rows x 256 columns with 4 waves; each wave
//    holds MF x 2 accumulators of 32x32 (up to 128 rows x 64 columns) and
//    issues v_mfma_f32_32x32x16_bf16; two workgroups fit on a CU.
//  * Loads go through raw buffer resources: addresses stay in scalar
//    registers, and an offset past the buffer reads zeros (row and K tails).
//  * When the column tiles alone cannot fill the 256 CUs (N = 8192 gives 32
//    tiles), K is split; each split writes fp32 partials, which are summed in
//    split order (deterministic, so streamed and resident runs are
//    bit-identical) with the epilogue applied, either by k_splitk_reduce here
//    or by the kernel that consumes the result (the RoPE/KV-append kernel for
//    QKV, the residual + RMSNorm reduction for O and down; LinearCall's
//    defer_reduce and norm_out select this).
//  * k_gemm_lw is the same contraction with 256-row workgroups whose weight
//    tiles are staged once per CU in LDS (direct-to-LDS loads) and shared by
//    both 128-row halves. It halves the weight loads per flop but needs twice
//    the splits at a given batch; launch_linear takes it only where k_gemm
//    would leave a quarter of the CUs idle (use_lds_weights).
#include "common.h"
#include "internal.h"

namespace sidp {

constexpr int kWaves = 4;          // waves per workgroup, one column group each
constexpr int kBK = 64;            // k per LDS stage
constexpr int kFragElems = 512;    // 64 lanes x 8 bf16

__host__ __device__ inline int round_up(int a, int b) { return (a + b - 1) / b * b; }

// ---------------------------------------------------------------- packing

// Packed order of one 16-byte chunk: [KP/64 k-tiles][NG column groups][4 k
// steps][2 column halves][64 lanes] of 8 bf16 each. A k-tile's 8 KB for every
// column group are adjacent, so the waves of a grid that all stand at the same
// k-tile read one contiguous stretch of the weights (spread over every HBM
// channel) rather than one 8 KB piece in each of NG regions a group apart.
__device__ __forceinline__ void packed_coords(int64_t chunk, int NG, int& lane, int& nf, int& kb, int& ng) {
  lane = (int)(chunk % 64);
  nf = (int)((chunk / 64) % 2);
  const int ks = (int)((chunk / 128) % 4);
  ng = (int)((chunk / 512) % NG);
  kb = (int)(chunk / (512 * (int64_t)NG)) * 4 + ks;
}

// Rows of the matrix to pack, taken from up to three sources stacked in
// order (the QKV projection packs W_q, W_k, W_v as one matrix).
struct PackRows {
  const uint16_t* w[3];
  int n[3];  // rows from each source; the packed matrix has n[0] + n[1] + n[2]
};

// W [N, K] (the stacked sources) -> packed as above, zero padded.
__global__ void k_pack_linear(PackRows src, int N, int K, int KB, int NG, uint16_t* __restrict__ out) {
  const int64_t chunk = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;  // one 8-element chunk
  const int64_t total = (int64_t)NG * KB * 2 * 64;
  if (chunk >= total) return;
  int lane, nf, kb, ng;
  packed_coords(chunk, NG, lane, nf, kb, ng);
  int n = ng * 64 + nf * 32 + (lane % 32);
  const bool in_rows = n < N;
  int seg = 0;
  while (seg < 2 && n >= src.n[seg]) n -= src.n[seg++];
  const uint16_t* w = src.w[seg];
  const int k0 = kb * 16 + (lane / 32) * 8;
  uint16_t v[8];
#pragma unroll
  for (int i = 0; i < 8; i++) v[i] = (in_rows && k0 + i < K) ? w[(int64_t)n * K + k0 + i] : (uint16_t)0;
  uint16_t* dst = out + chunk * 8;
#pragma unroll
  for (int i = 0; i < 8; i++) dst[i] = v[i];
}

// gate, up [F, K] -> packed with n-group j = {gate rows 32j..32j+31, up rows 32j..32j+31}.
__global__ void k_pack_gate_up(const uint16_t* __restrict__ wg, const uint16_t* __restrict__ wu, int F,
                               int K, int KB, int NG, uint16_t* __restrict__ out) {
  const int64_t chunk = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  const int64_t total = (int64_t)NG * KB * 2 * 64;
  if (chunk >= total) return;
  int lane, nf, kb, ng;
  packed_coords(chunk, NG, lane, nf, kb, ng);
  const int f = ng * 32 + (lane % 32);
  const int k0 = kb * 16 + (lane / 32) * 8;
  const uint16_t* src = nf == 0 ? wg : wu;
  uint16_t v[8];
#pragma unroll
  for (int i = 0; i < 8; i++) v[i] = (f < F && k0 + i < K) ? src[(int64_t)f * K + k0 + i] : (uint16_t)0;
  uint16_t* dst = out + chunk * 8;
#pragma unroll
  for (int i = 0; i < 8; i++) dst[i] = v[i];
}

// ---------------------------------------------------------------- GEMM

struct GemmArgs {
  const uint16_t* x;   // [M, K] bf16, row stride K
  const uint16_t* w;   // packed
  int M, K, KP;        // KP = K rounded up to 64
  int NG;              // packed column groups (64 columns each)
  int tiles;           // ceil(NG / waves per workgroup)
  int splits;
  int N;               // valid output columns (SWIGLU: F)
  int mblocks;         // row blocks of BM rows
  void* out;
  const uint16_t* bias;  // EPI_BF16
  const float* resid;    // EPI_RESID
  float* ws;             // split-K partials [splits][M][NG*64]
};

__device__ __forceinline__ float silu_f(float g) { return g / (1.0f + __expf(-g)); }

constexpr uint32_t kRsrcWord3 = 0x00020000u;  // gfx9 raw buffer: 32-bit data, bounds-checked
constexpr uint32_t kOutOfRange = 0x80000000u;  // any offset past num_records reads as zero

__device__ __forceinline__ __amdgpu_buffer_rsrc_t make_rsrc(const void* p, uint32_t bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(p), (short)0, (int)bytes, (int)kRsrcWord3);
}

__device__ __forceinline__ u32x4_t buf_load16(__amdgpu_buffer_rsrc_t r, uint32_t voff, uint32_t soff) {
  return __builtin_bit_cast(u32x4_t, __builtin_amdgcn_raw_buffer_load_b128(r, voff, soff, 0));
}

// Writes one wave's tile: rows row0 + [0, 32 MF), the 64 packed columns of
// group ng; acc[m][nf] holds the 32x32 block (m, nf) in the MFMA's layout
// (register r of lane l: row 8 (r / 4) + 4 (l / 32) + r % 4, column l % 32).
template <int MF, int EPI, bool PARTIAL>
__device__ __forceinline__ void store_tile(const GemmArgs& a, const f32x16_t (&acc)[MF][2], int row0, int ng,
                                           int split, int lane) {
  const int NP = a.NG * 64;
#pragma unroll
  for (int m = 0; m < MF; m++) {
#pragma unroll
    for (int r = 0; r < 16; r++) {
      const int row = row0 + m * 32 + (r >> 2) * 8 + (lane >> 5) * 4 + (r & 3);
      if (row >= a.M) continue;
      if (PARTIAL) {
        float* dst = a.ws + ((int64_t)split * a.M + row) * NP + ng * 64 + (lane & 31);
        dst[0] = acc[m][0][r];
        dst[32] = acc[m][1][r];
      } else if (EPI == SIDP_EPI_SWIGLU) {
        const int f = ng * 32 + (lane & 31);
        if (f < a.N)
          ((uint16_t*)a.out)[(int64_t)row * a.N + f] = f2bf(silu_f(acc[m][0][r]) * acc[m][1][r]);
      } else {
#pragma unroll
        for (int nf = 0; nf < 2; nf++) {
          const int n = ng * 64 + nf * 32 + (lane & 31);
          if (n >= a.N) continue;
          const int64_t o = (int64_t)row * a.N + n;
          if (EPI == SIDP_EPI_BF16) {
            float v = acc[m][nf][r];
            if (a.bias) v += bf2f(a.bias[n]);
            ((uint16_t*)a.out)[o] = f2bf(v);
          } else {
            ((float*)a.out)[o] = a.resid ? a.resid[o] + acc[m][nf][r] : acc[m][nf][r];
          }
        }
      }
    }
  }
}

// One workgroup: W waves (4, or 8 for wide unsplit launches). Wave wn
// computes rows [row0, row0 + MF*32) x the 64 packed columns of group
// tile*W + wn; the activation tile staged in LDS serves all W waves.
template <int MF, int EPI, bool PARTIAL, int W = kWaves>
__global__ void __launch_bounds__(64 * W, W > 4 ? 1 : 2) k_gemm(GemmArgs a) {
  // Issue priority over waves of lower priority on the same SIMD: in the
  // streamed step the slot-fill waves (default, lowest priority) share the
  // CUs with the projections and then take the issue slots the projection's
  // waves leave idle (0.35% more tokens/s in the step, same session).
  __builtin_amdgcn_s_setprio(3);
  constexpr int NT = 64 * W;
  constexpr int BM = MF * 32;
  constexpr int CPT = (BM * 8 + NT - 1) / NT;  // 16-byte X chunks per thread per stage (the last may be idle)
  constexpr bool kXTail = BM * 8 % NT != 0;     // 7-wave workgroups: not every thread has a last chunk
  extern __shared__ __attribute__((aligned(16))) uint16_t smem[];
  uint16_t* lds0 = smem;
  uint16_t* lds1 = smem + BM * kBK;

  // Workgroup id -> (column tile, split, row block). The row blocks of one
  // (tile, split) sit 8 ids apart: dispatch deals ids round-robin to the 8
  // XCDs, so they run together on one XCD and share its L2 for the weights.
  int pair, mblk;
  {
    const int L = blockIdx.x;
    const int per_group = 8 * a.mblocks;
    const int r = L % per_group;
    pair = (L / per_group) * 8 + (r % 8);
    mblk = r / 8;
    if (pair >= a.tiles * a.splits) return;
  }
  const int split = pair % a.splits;
  const int tile = pair / a.splits;
  const int row0 = mblk * BM;
  // wave index made provably uniform so weight offsets live in scalar registers
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6), lane = threadIdx.x & 63;
  const int wn = wave;
  const int ng = tile * W + wn;
  const bool active = ng < a.NG;
  const int KT = a.KP / kBK;
  const int kt0 = (int)((int64_t)split * KT / a.splits);
  const int kt1 = (int)((int64_t)(split + 1) * KT / a.splits);

  const __amdgpu_buffer_rsrc_t xr_rsrc = make_rsrc(a.x, (uint32_t)((size_t)a.M * a.K * 2));
  const __amdgpu_buffer_rsrc_t wr_rsrc = make_rsrc(a.w, (uint32_t)((size_t)a.NG * a.KP * 64 * 2));
  // byte offset of this wave's 8 KB piece of k-tile kt: (kt * NG + ng) * 8 KB
  const uint32_t w_base = (uint32_t)(active ? ng : 0) * 8192u;
  const uint32_t w_tile = (uint32_t)a.NG * 8192u;
  const uint32_t w_lane = (uint32_t)lane * 16u;

  // X chunks this thread stages: row r, 16-byte column chunk cc of the 64-wide k tile
  int x_row[CPT], x_cc[CPT];
#pragma unroll
  for (int i = 0; i < CPT; i++) {
    const int ci = threadIdx.x + i * NT;
    x_row[i] = (!kXTail || ci < BM * 8) ? ci >> 3 : -1;  // -1: no chunk (out of range load, no store)
    x_cc[i] = ci & 7;
  }

  f32x16_t acc[MF][2];
#pragma unroll
  for (int m = 0; m < MF; m++)
#pragma unroll
    for (int n = 0; n < 2; n++)
#pragma unroll
      for (int r = 0; r < 16; r++) acc[m][n][r] = 0.f;

  const int arow = lane & 31;
  u32x4_t xs[CPT];
  // Weight fragments of a k-tile in two halves (k steps 0-1 and 2-3). The
  // next tile's low half is fetched at the top of an iteration, its high half
  // once the current low half is consumed, so 48 registers hold weights.
  u32x4_t wlo[4], whi[4], nlo[4], nhi[4];

  auto load_x = [&](int kt) {
#pragma unroll
    for (int i = 0; i < CPT; i++) {
      const int row = row0 + x_row[i];
      const int k = kt * kBK + x_cc[i] * 8;
      const bool in = (!kXTail || x_row[i] >= 0) && row < a.M && k < a.K;  // every thread issues the load
      const uint32_t off = in ? (uint32_t)(((size_t)row * a.K + k) * 2) : kOutOfRange;
      xs[i] = buf_load16(xr_rsrc, off, 0);
    }
  };
  auto store_x = [&](uint16_t* lds) {
#pragma unroll
    for (int i = 0; i < CPT; i++) {
      const int r = x_row[i];
      if (kXTail && r < 0) continue;
      *(u32x4_t*)(lds + r * kBK + ((x_cc[i] ^ ((r >> 1) & 7)) << 3)) = xs[i];
    }
  };
  // fragments (kb, nf) of tile kt live at 1 KB * (kb * 2 + nf) in the tile's 8 KB
  auto load_w_half = [&](int kt, int half, u32x4_t (&w)[4]) {
    const uint32_t soff = w_base + (uint32_t)kt * w_tile + (uint32_t)half * 4096u;
#pragma unroll
    for (int j = 0; j < 4; j++) w[j] = buf_load16(wr_rsrc, w_lane + j * 1024u, soff);
  };
  auto mma_half = [&](const uint16_t* cur, int half, const u32x4_t (&w)[4]) {
#pragma unroll
    for (int kh = 0; kh < 2; kh++) {
      const int kb = half * 2 + kh;
      const int cc = kb * 2 + (lane >> 5);
#pragma unroll
      for (int m = 0; m < MF; m++) {
        const int r = arow + m * 32;
        const bf16x8_t af = as_bf16x8(*(const u32x4_t*)(cur + r * kBK + ((cc ^ ((r >> 1) & 7)) << 3)));
        acc[m][0] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(af, as_bf16x8(w[kh * 2 + 0]), acc[m][0], 0, 0, 0);
        acc[m][1] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(af, as_bf16x8(w[kh * 2 + 1]), acc[m][1], 0, 0, 0);
      }
    }
    if constexpr (MF == 4) {
      // Scheduling hint (mask 0x100 = LDS reads, 0x008 = MFMAs): read each
      // activation fragment two MFMA pairs ahead of its use, so that an LDS
      // read's latency hides behind matrix work instead of stalling the pipe:
      // 3 reads, then (2 MFMAs, 1 read) x 5, then the last 6 MFMAs.
      __builtin_amdgcn_sched_group_barrier(0x100, 3, 0);
#pragma unroll
      for (int i = 0; i < 5; i++) {
        __builtin_amdgcn_sched_group_barrier(0x008, 2, 0);
        __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
      }
      __builtin_amdgcn_sched_group_barrier(0x008, 6, 0);
    }
  };

  // Every load of the k loop is issued on every path (a wait count can only
  // be exact when all paths issue the same loads): the prefetch past the
  // split's last k-tile re-reads that tile (weights, an L2 hit) or reads past
  // K (activations, out of range, zeros), and is never consumed. The loop is
  // unrolled by two so the current and next weight registers swap roles
  // without copies.
  auto step = [&](int kt, const uint16_t* cur, uint16_t* nxt, u32x4_t (&clo)[4], u32x4_t (&chi)[4],
                  u32x4_t (&plo)[4], u32x4_t (&phi)[4]) {
    const int kn = min(kt + 1, kt1 - 1);
    load_x(kt + 1);
    load_w_half(kn, 0, plo);
    if (active) mma_half(cur, 0, clo);
    load_w_half(kn, 1, phi);
    if (active) mma_half(cur, 1, chi);
    store_x(nxt);
    __syncthreads();
  };
  load_x(kt0);
  load_w_half(kt0, 0, wlo);
  load_w_half(kt0, 1, whi);
  store_x(lds0);
  __syncthreads();
  // Pairs of k-tiles, then an odd last tile outside the loop: an exit from
  // the middle of the unrolled body would give the loop header a second
  // predecessor on which the first step's weight loads are still pending,
  // and the header would wait for them on every iteration.
  int kt = kt0;
  for (; kt + 1 < kt1; kt += 2) {
    step(kt, lds0, lds1, wlo, whi, nlo, nhi);
    step(kt + 1, lds1, lds0, nlo, nhi, wlo, whi);
  }
  if (kt < kt1) step(kt, lds0, lds1, wlo, whi, nlo, nhi);

  if (!active) return;
  store_tile<MF, EPI, PARTIAL>(a, acc, row0, ng, split, lane);
}

// LDS-staged weights. One 8-wave workgroup per CU covers 256 rows x 256
// columns: waves 0-3 take rows 0-127 and waves 4-7 rows 128-255 of the same
// four column groups. Each weight fragment of a stage is fetched once per
// workgroup, straight into LDS by direct-to-LDS buffer loads (no VGPR round
// trip), and read there by the two waves that use it; the 256-row activation
// tile is staged through LDS as in k_gemm. A stage is 32 k (two MFMA k steps);
// two stages (2 x 32 KB) are in LDS at once, which leaves room beside a CU's
// slot-fill workgroup. Each stage buffer is its own LDS array, so the compiler
// can tell that reading the current stage does not depend on the direct loads
// landing in the other one.
constexpr int kLwRows = 256;                 // rows per workgroup
constexpr int kLwBK = 32;                    // k per stage
constexpr int kLwA = kLwRows * kLwBK;        // bf16 elements of a stage's activations (16 KB)
constexpr int kLwW = 4 * 4 * kFragElems;     // 4 groups x 4 fragments (16 KB)

// s_waitcnt vmcnt(0): expcnt and lgkmcnt at their no-wait maxima (7, 15)
__device__ __forceinline__ void wait_vm0() { __builtin_amdgcn_s_waitcnt((7 << 4) | (15 << 8)); }

template <int EPI, bool PARTIAL>
__global__ void __launch_bounds__(512, 1) k_gemm_lw(GemmArgs a) {
  __builtin_amdgcn_s_setprio(3);  // as k_gemm: ahead of the slot-fill waves sharing the CU
  __shared__ __attribute__((aligned(1024))) uint16_t lw_a0[kLwA];
  __shared__ __attribute__((aligned(1024))) uint16_t lw_a1[kLwA];
  __shared__ __attribute__((aligned(1024))) uint16_t lw_w0[kLwW];
  __shared__ __attribute__((aligned(1024))) uint16_t lw_w1[kLwW];

  // workgroup id -> (column tile, split, row block), row blocks 8 ids apart (as k_gemm)
  int pair, mblk;
  {
    const int L = blockIdx.x;
    const int per_group = 8 * a.mblocks;
    const int r = L % per_group;
    pair = (L / per_group) * 8 + (r % 8);
    mblk = r / 8;
    if (pair >= a.tiles * a.splits) return;
  }
  const int split = pair % a.splits;
  const int tile = pair / a.splits;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6), lane = threadIdx.x & 63;
  const int half = wave >> 2, g = wave & 3;
  const int ng = tile * 4 + g;
  const bool active = ng < a.NG;
  const int row0 = mblk * kLwRows + half * 128;  // this wave's rows
  // the split's k range in 64-wide k-tiles (as k_gemm), walked in 32-wide stages
  const int KT = a.KP / kBK;
  const int st0 = 2 * (int)((int64_t)split * KT / a.splits);
  const int st1 = 2 * (int)((int64_t)(split + 1) * KT / a.splits);

  const __amdgpu_buffer_rsrc_t xr_rsrc = make_rsrc(a.x, (uint32_t)((size_t)a.M * a.K * 2));
  const __amdgpu_buffer_rsrc_t wr_rsrc = make_rsrc(a.w, (uint32_t)((size_t)a.NG * a.KP * 64 * 2));

  // Activations: stage rows r = 0..255, 16-byte chunks c = 0..3 (8 k each);
  // thread t stages chunks t and t + 512. In LDS a row is 64 bytes and chunk
  // c sits at slot c ^ ((r >> 2) & 3): the 16 rows one LDS cycle serves for a
  // fragment read (one chunk each) then fall on 16 distinct 16-byte bank groups.
  int x_row[2], x_cc[2];
#pragma unroll
  for (int i = 0; i < 2; i++) {
    const int ci = threadIdx.x + i * 512;
    x_row[i] = ci >> 2;
    x_cc[i] = ci & 3;
  }
  u32x4_t xs[2];
  auto load_x = [&](int st) {
#pragma unroll
    for (int i = 0; i < 2; i++) {
      const int row = mblk * kLwRows + x_row[i];
      const int k = st * kLwBK + x_cc[i] * 8;
      const bool in = row < a.M && k < a.K;
      const uint32_t off = in ? (uint32_t)(((size_t)row * a.K + k) * 2) : kOutOfRange;
      xs[i] = buf_load16(xr_rsrc, off, 0);
    }
  };
  auto store_x = [&](uint16_t* lds) {
#pragma unroll
    for (int i = 0; i < 2; i++) {
      const int r = x_row[i];
      *(u32x4_t*)(lds + r * kLwBK + ((x_cc[i] ^ ((r >> 2) & 3)) << 3)) = xs[i];
    }
  };
  // Weights of stage st: k-tile st / 2, k steps 2 (st % 2) and + 1, so bytes
  // [4 KB (st % 2), + 4 KB) of each group's 8 KB piece: fragments (k step,
  // column half) in packed order. Wave (half, g) fetches fragments 2 half and
  // 2 half + 1 of group g into LDS fragment slot 4 g + f (1 KB each; lane l's
  // 16 bytes land at 16 l). A group past NG re-reads group 0 (its waves skip
  // the MFMAs).
  const uint32_t w_lane = (uint32_t)lane * 16u;
  const uint32_t w_group = (uint32_t)(active ? ng : 0) * 8192u;
  auto load_w = [&](int st, uint16_t* lds) {
    const uint32_t soff = (uint32_t)(st >> 1) * (uint32_t)a.NG * 8192u + w_group + (uint32_t)(st & 1) * 4096u;
#pragma unroll
    for (int j = 0; j < 2; j++) {
      const int f = half * 2 + j;
      __builtin_amdgcn_raw_ptr_buffer_load_lds(
          wr_rsrc, (__attribute__((address_space(3))) void*)(lds + (g * 4 + f) * kFragElems), 16, w_lane,
          soff + (uint32_t)f * 1024u, 0, 0);
    }
  };

  f32x16_t acc[4][2];
#pragma unroll
  for (int m = 0; m < 4; m++)
#pragma unroll
    for (int n = 0; n < 2; n++)
#pragma unroll
      for (int r = 0; r < 16; r++) acc[m][n][r] = 0.f;

  const int arow = lane & 31;
  auto mma_stage = [&](const uint16_t* xa, const uint16_t* wl) {
#pragma unroll
    for (int ks = 0; ks < 2; ks++) {
      const bf16x8_t b0 = as_bf16x8(*(const u32x4_t*)(wl + (g * 4 + ks * 2 + 0) * kFragElems + lane * 8));
      const bf16x8_t b1 = as_bf16x8(*(const u32x4_t*)(wl + (g * 4 + ks * 2 + 1) * kFragElems + lane * 8));
      const int cc = ks * 2 + (lane >> 5);
#pragma unroll
      for (int m = 0; m < 4; m++) {
        const int r = half * 128 + m * 32 + arow;
        const bf16x8_t af = as_bf16x8(*(const u32x4_t*)(xa + r * kLwBK + ((cc ^ ((r >> 2) & 3)) << 3)));
        acc[m][0] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(af, b0, acc[m][0], 0, 0, 0);
        acc[m][1] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(af, b1, acc[m][1], 0, 0, 0);
      }
    }
  };

  // Stage st computes from (xa, wl) while stage st + 1 is fetched into (xn,
  // wn); every path issues the same loads (the prefetch past the split's last
  // stage re-reads that stage).
  auto step = [&](int st, const uint16_t* xa, const uint16_t* wl, uint16_t* xn, uint16_t* wn) {
    const int sn = min(st + 1, st1 - 1);
    load_x(sn);
    load_w(sn, wn);
    if (active) mma_stage(xa, wl);
    store_x(xn);
    wait_vm0();  // this wave's direct-to-LDS loads have landed before the barrier
    __syncthreads();
  };
  load_x(st0);
  load_w(st0, lw_w0);
  store_x(lw_a0);
  wait_vm0();
  __syncthreads();
  int st = st0;
  for (; st + 1 < st1; st += 2) {
    step(st, lw_a0, lw_w0, lw_a1, lw_w1);
    step(st + 1, lw_a1, lw_w1, lw_a0, lw_w0);
  }
  if (st < st1) step(st, lw_a0, lw_w0, lw_a1, lw_w1);

  if (!active) return;
  store_tile<4, EPI, PARTIAL>(a, acc, row0, ng, split, lane);
}

// Sum split-K partials in split order and apply the epilogue.
template <int EPI>
__global__ void k_splitk_reduce(GemmArgs a) {
  const int NP = a.NG * 64;
  const int cols = EPI == SIDP_EPI_SWIGLU ? a.N : a.N;  // output columns
  const int64_t idx = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (idx >= (int64_t)a.M * cols) return;
  const int row = (int)(idx / cols), c = (int)(idx % cols);
  if (EPI == SIDP_EPI_SWIGLU) {
    const int pc = (c / 32) * 64 + (c % 32);
    float g = 0.f, u = 0.f;
    for (int s0 = 0; s0 < a.splits; s0 += 4) {  // four partials in flight, summed in split order
      float pg[4], pu[4];
#pragma unroll
      for (int j = 0; j < 4; j++)
        if (s0 + j < a.splits) {
          const float* p = a.ws + ((int64_t)(s0 + j) * a.M + row) * NP + pc;
          pg[j] = p[0];
          pu[j] = p[32];
        }
#pragma unroll
      for (int j = 0; j < 4; j++)
        if (s0 + j < a.splits) {
          g += pg[j];
          u += pu[j];
        }
    }
    ((uint16_t*)a.out)[idx] = f2bf(silu_f(g) * u);
  } else {
    const int pc = (c / 64) * 64 + (c % 64);  // packed column of output n (identity)
    float v = 0.f;
    for (int s0 = 0; s0 < a.splits; s0 += 4) {  // four partials in flight, summed in split order
      float pv[4];
#pragma unroll
      for (int j = 0; j < 4; j++)
        if (s0 + j < a.splits) pv[j] = a.ws[((int64_t)(s0 + j) * a.M + row) * NP + pc];
#pragma unroll
      for (int j = 0; j < 4; j++)
        if (s0 + j < a.splits) v += pv[j];
    }
    if (EPI == SIDP_EPI_BF16) {
      if (a.bias) v += bf2f(a.bias[c]);
      ((uint16_t*)a.out)[idx] = f2bf(v);
    } else {
      ((float*)a.out)[idx] = a.resid ? a.resid[idx] + v : v;
    }
  }
}

// ---------------------------------------------------------------- host side

size_t packed_bytes(int n, int k) { return (size_t)round_up(n, 64) * round_up(k, 64) * 2; }

// The kernels address the packed weights and the activations through 32-bit
// buffer offsets.
bool gemm_fits(int m, int n_cols_packed, int k) {
  // the activations stay below 2^31 bytes, so the out-of-range offset 2^31
  // that rows past M and k past K read through lies past them
  constexpr size_t kLimit = (size_t)1 << 32;
  return packed_bytes(n_cols_packed, k) < kLimit && (size_t)m * round_up(k, 64) * 2 < ((size_t)1 << 31);
}


static int splits_for(int tiles, int mblocks, int KT, int num_cus);

// Whether a projection runs on k_gemm_lw (256-row workgroups, weights staged
// in LDS) rather than k_gemm (128-row blocks, weights into registers). Alone
// at B = 256 the LDS-staged kernel is slower on all four 70B projections
// (QKV 53 against 51 us, O 46 against 40, down 143-148 against 129-136,
// gate/up 318-335 against 284-309, its reductions 5 us slower with twice the
// splits); it wins where k_gemm would run a single unsplit round on under
// three quarters of the CUs, as QKV at 512 rows does (160 workgroups: 128-132
// us against 95-97 plus a 16 us reduction on 240).
static bool use_lds_weights(int M, int NG, int K, int num_cus) {
  if (M <= 128 || K % 64) return false;
  const int tiles = (NG + kWaves - 1) / kWaves, mblocks = (M + 127) / 128;
  return splits_for(tiles, mblocks, K / kBK, num_cus) == 1 && (int64_t)tiles * mblocks * 4 < 3 * (int64_t)num_cus;
}

int gemm_splits(int M, int n_cols_packed, int K, int num_cus) {
  const int NG = round_up(n_cols_packed, 64) / 64;
  const bool lw = use_lds_weights(M, NG, K, num_cus);
  const int tiles = (NG + kWaves - 1) / kWaves;
  const int mblocks = lw ? (M + kLwRows - 1) / kLwRows : (M + 127) / 128;
  const int KT = round_up(K, 64) / kBK;
  return splits_for(tiles, mblocks, KT, num_cus);
}

static int splits_for(int tiles, int mblocks, int KT, int num_cus) {
  const int base = tiles * mblocks;
  // As many splits as keep the grid at most one 4-wave workgroup per CU (two
  // fit): each split writes fp32 partials for all M x N outputs, and at decode
  // batches that traffic (O at B=256: 8 splits would write and re-read 67 MB
  // beside 134 MB of weights) costs more than the second workgroup's latency
  // hiding gains. Rounding down rather than to nearest keeps a few CUs from
  // running a second workgroup after the rest have finished (O and down at
  // M=384: 192 workgroups instead of 288, the step 2% faster).
  int s = num_cus / base;
  if (s < 1) s = 1;
  if (s > 16) s = 16;
  if (s > KT) s = KT;
  return s;
}

size_t gemm_ws_bytes(int M, int n_cols_packed, int K, int num_cus) {
  const int s = gemm_splits(M, n_cols_packed, K, num_cus);
  if (s <= 1) return 0;
  return (size_t)s * M * round_up(n_cols_packed, 64) * sizeof(float);
}

static hipError_t launch_pack_rows(const PackRows& src, int n, int k, void* packed, hipStream_t s) {
  const int NG = round_up(n, 64) / 64, KB = round_up(k, 64) / 16;
  const int64_t chunks = (int64_t)NG * KB * 128;
  k_pack_linear<<<(unsigned)((chunks + 255) / 256), 256, 0, s>>>(src, n, k, KB, NG, (uint16_t*)packed);
  return hipGetLastError();
}

hipError_t launch_pack_linear(const void* w, int n, int k, void* packed, hipStream_t s) {
  PackRows src{{(const uint16_t*)w, nullptr, nullptr}, {n, 0, 0}};
  return launch_pack_rows(src, n, k, packed, s);
}

hipError_t launch_pack_qkv(const void* wq, const void* wk, const void* wv, int nq, int nkv, int k, void* packed,
                           hipStream_t s) {
  PackRows src{{(const uint16_t*)wq, (const uint16_t*)wk, (const uint16_t*)wv}, {nq, nkv, nkv}};
  return launch_pack_rows(src, nq + 2 * nkv, k, packed, s);
}

hipError_t launch_pack_gate_up(const void* wg, const void* wu, int f, int k, void* packed, hipStream_t s) {
  const int F32 = round_up(f, 32);
  const int NG = 2 * F32 / 64, KB = round_up(k, 64) / 16;
  const int64_t chunks = (int64_t)NG * KB * 128;
  k_pack_gate_up<<<(unsigned)((chunks + 255) / 256), 256, 0, s>>>((const uint16_t*)wg, (const uint16_t*)wu, f, k, KB,
                                                                  NG, (uint16_t*)packed);
  return hipGetLastError();
}

template <int MF, int EPI, bool P, int W = kWaves>
static hipError_t launch_mf(GemmArgs a, hipStream_t s) {
  constexpr int BM = MF * 32;
  a.mblocks = (a.M + BM - 1) / BM;
  a.tiles = (a.NG + W - 1) / W;
  const size_t lds = (size_t)2 * BM * kBK * sizeof(uint16_t);
  static bool attr_set = false;
  if (!attr_set) {
    hipError_t e =
        hipFuncSetAttribute((const void*)k_gemm<MF, EPI, P, W>, hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
    if (e != hipSuccess) return e;
    attr_set = true;
  }
  const int pairs = a.tiles * a.splits;
  const int grid = (pairs + 7) / 8 * 8 * a.mblocks;
  k_gemm<MF, EPI, P, W><<<grid, 64 * W, lds, s>>>(a);
  return hipGetLastError();
}

template <int EPI, bool P>
static hipError_t launch_lw(GemmArgs a, hipStream_t s) {
  a.mblocks = (a.M + kLwRows - 1) / kLwRows;
  a.tiles = (a.NG + 3) / 4;
  const int pairs = a.tiles * a.splits;
  const int grid = (pairs + 7) / 8 * 8 * a.mblocks;
  k_gemm_lw<EPI, P><<<grid, 512, 0, s>>>(a);
  return hipGetLastError();
}

template <int EPI, bool P>
static hipError_t launch_epi(const GemmArgs& a, hipStream_t s, int wide = 0) {
  if constexpr (!P) {
    if (wide == 7) return launch_mf<4, EPI, P, 7>(a, s);
    if (wide == 8) return launch_mf<4, EPI, P, 8>(a, s);
  }
  if (wide == -1) return launch_lw<EPI, P>(a, s);
  if (a.M <= 32) return launch_mf<1, EPI, P>(a, s);
  if (a.M <= 64) return launch_mf<2, EPI, P>(a, s);
  return launch_mf<4, EPI, P>(a, s);
}

// Without a split, past 64 rows, a 7- or 8-wave workgroup (128 rows x 448 or
// 512 columns) stages each activation tile once for all its column groups, so
// a wave issues fewer loads per k step (the projections pay per load
// instruction). The width is chosen by the waves a CU runs to finish the grid:
// 4-wave workgroups go two to a CU (rounds of 8 waves), 7- and 8-wave ones one
// (rounds of 7 or 8), and a wide width is a candidate only while it gives at
// least 0.8 workgroups per CU (fewer would leave CUs idle that the model
// counts as busy); ties go to the wider one. A 70B-shaped gate/up (896 column
// groups) gets 7 waves at 256 rows, exactly 256 workgroups; a 924-group one 8.
// Returns 4, 7 or 8.
static int unsplit_width(int m, int NG, int num_cus) {
  int wide = 4;
  if (m > 64) {
    const int64_t mb = (m + 127) / 128, cus = std::max(1, num_cus);
    const int64_t n4 = (NG + 3) / 4 * mb, n7 = (NG + 6) / 7 * mb, n8 = (NG + 7) / 8 * mb;
    int64_t best = (n4 + 2 * cus - 1) / (2 * cus) * 8;
    if (n7 * 10 >= 8 * cus && (n7 + cus - 1) / cus * 7 <= best) best = (n7 + cus - 1) / cus * 7, wide = 7;
    if (n8 * 10 >= 8 * cus && (n8 + cus - 1) / cus * 8 <= best) best = (n8 + cus - 1) / cus * 8, wide = 8;
  }
  return wide;
}

GemmPlan plan_linear(int m, int n, int k, int epilogue, int num_cus) {
  const int ncols = epilogue == SIDP_EPI_SWIGLU ? 2 * round_up(n, 32) : n;
  const int NG = round_up(ncols, 64) / 64;
  GemmPlan p;
  p.splits = gemm_splits(m, ncols, k, num_cus);
  p.ws_bytes = gemm_ws_bytes(m, ncols, k, num_cus);
  if (use_lds_weights(m, NG, k, num_cus)) {
    p.kernel = 1;
    p.waves = 8;
    p.rows = kLwRows;
  } else {
    p.kernel = 0;
    p.waves = p.splits == 1 ? unsplit_width(m, NG, num_cus) : kWaves;
    p.rows = p.waves > kWaves ? 128 : m <= 32 ? 32 : m <= 64 ? 64 : 128;  // launch_epi's MF
  }
  const int cols_per_wg = p.kernel == 1 ? 4 : p.waves;  // column groups per workgroup
  const int tiles = (NG + cols_per_wg - 1) / cols_per_wg;
  const int mblocks = (m + p.rows - 1) / p.rows;
  p.workgroups = (tiles * p.splits + 7) / 8 * 8 * mblocks;
  return p;
}

hipError_t launch_linear(const LinearCall& c, hipStream_t s) {
  GemmArgs a;
  a.x = (const uint16_t*)c.x;
  a.w = (const uint16_t*)c.packed;
  a.M = c.m;
  a.K = c.k;
  a.KP = round_up(c.k, 64);
  const int ncols = c.epilogue == SIDP_EPI_SWIGLU ? 2 * round_up(c.n, 32) : c.n;
  a.NG = round_up(ncols, 64) / 64;
  a.tiles = (a.NG + kWaves - 1) / kWaves;
  a.splits = gemm_splits(c.m, ncols, c.k, c.num_cus);
  a.N = c.n;
  a.out = c.out;
  a.bias = (const uint16_t*)c.bias;
  a.resid = c.residual;
  a.ws = c.ws;
  if (!gemm_fits(c.m, ncols, c.k)) return hipErrorInvalidValue;
  if (a.splits > 1 && (size_t)a.splits * a.M * a.NG * 64 * sizeof(float) > c.ws_bytes) return hipErrorInvalidValue;
  const bool fuse_norm = c.norm_out && c.epilogue == SIDP_EPI_RESID && c.residual == c.out;
  if (c.norm_out && !fuse_norm) return hipErrorInvalidValue;
  // the kernel and width plan_linear describes: -1 the LDS-staged kernel, 7 or
  // 8 a wide unsplit k_gemm, 0 the 4-wave k_gemm
  const GemmPlan plan = plan_linear(c.m, c.n, c.k, c.epilogue, c.num_cus);
  const int wide = plan.kernel == 1 ? -1 : plan.waves > kWaves ? plan.waves : 0;
  hipError_t e;
  if (a.splits == 1) {
    if (c.epilogue == SIDP_EPI_BF16) e = launch_epi<SIDP_EPI_BF16, false>(a, s, wide);
    else if (c.epilogue == SIDP_EPI_RESID) e = launch_epi<SIDP_EPI_RESID, false>(a, s, wide);
    else e = launch_epi<SIDP_EPI_SWIGLU, false>(a, s, wide);
    if (e != hipSuccess || !fuse_norm) return e;
    return launch_rmsnorm((const float*)c.out, c.norm_gain, c.norm_eps, c.norm_out, a.M, a.N, s);
  }
  e = launch_epi<SIDP_EPI_BF16, true>(a, s, wide);  // partials only; epilogue in the reduction
  if (e != hipSuccess || c.defer_reduce) return e;
  if (fuse_norm && reduce_resid_norm_fits(a.N))
    return launch_reduce_resid_norm(a.ws, a.splits, a.M, a.NG * 64, a.N, (float*)c.out, c.norm_gain, c.norm_eps,
                                    c.norm_out, s);
  const int64_t outs = (int64_t)a.M * a.N;
  const unsigned blocks = (unsigned)((outs + 255) / 256);
  if (c.epilogue == SIDP_EPI_BF16) k_splitk_reduce<SIDP_EPI_BF16><<<blocks, 256, 0, s>>>(a);
  else if (c.epilogue == SIDP_EPI_RESID) k_splitk_reduce<SIDP_EPI_RESID><<<blocks, 256, 0, s>>>(a);
  else k_splitk_reduce<SIDP_EPI_SWIGLU><<<blocks, 256, 0, s>>>(a);
  e = hipGetLastError();
  if (e != hipSuccess || !fuse_norm) return e;
  return launch_rmsnorm((const float*)c.out, c.norm_gain, c.norm_eps, c.norm_out, a.M, a.N, s);
}

}  // namespace sidp
