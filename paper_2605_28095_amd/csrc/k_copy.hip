// Slot-fill engine of the weight cache (the WaS one-sided read, emulated
// inside one HBM): a grid-stride 16-byte copy with non-temporal loads and
// stores, so the streamed weights do not evict the compute's working set from
// L2. On this platform a same-device hipMemcpyAsync also runs as a shader
// copy on the CUs; a copy kernel of our own lets the runtime choose how many
// workgroups (CUs) the fill may occupy while compute runs beside it.
// Also: a NaN poison fill and a bounded spin, used to expose missing waits.
#include "common.h"
#include "internal.h"

namespace sidp {

typedef float f4v_t __attribute__((ext_vector_type(4)));

__global__ void __launch_bounds__(256) k_copy16(const f4v_t* __restrict__ src, f4v_t* __restrict__ dst, size_t n) {
  const size_t stride = (size_t)gridDim.x * blockDim.x;
  size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x;
  for (; i + 3 * stride < n; i += 4 * stride) {
    const f4v_t a = __builtin_nontemporal_load(src + i);
    const f4v_t b = __builtin_nontemporal_load(src + i + stride);
    const f4v_t c = __builtin_nontemporal_load(src + i + 2 * stride);
    const f4v_t d = __builtin_nontemporal_load(src + i + 3 * stride);
    __builtin_nontemporal_store(a, dst + i);
    __builtin_nontemporal_store(b, dst + i + stride);
    __builtin_nontemporal_store(c, dst + i + 2 * stride);
    __builtin_nontemporal_store(d, dst + i + 3 * stride);
  }
  for (; i < n; i += stride) __builtin_nontemporal_store(__builtin_nontemporal_load(src + i), dst + i);
}

// Background slot fill: runs beside the layer kernels instead of ahead of
// them. One 4-wave workgroup per CU with few VGPRs per wave and scalar buffer
// bases: 12, 24 or 48 allocated for 2, 4 or 8 loads per lane. Beside two
// attention waves (224 each) or two projection waves (up to 240 each, the
// 7-wave gate/up) on a SIMD there is room for the 2- and 4-load fill waves;
// the 8-load one, used only for the first tile of a layer, fits beside
// attention and beside the split projections (one wave per SIMD), which is
// what that tile runs beside. The 81 KB of LDS it requests and never touches
// keeps two fill workgroups off one CU (2 x 81 KB > 160 KB) while one still
// fits beside two projection (2 x 32 KB), two attention (2 x 34 KB) or one
// LDS-staged projection (64 KB) workgroups, so the fill never claims the
// resources a layer kernel needs. U 16-byte loads per lane are in flight per
// iteration.
constexpr int kFillLdsBytes = 81 * 1024;
constexpr uint32_t kFillRsrcWord3 = 0x00020000u;

template <int U>
__device__ __forceinline__ void fill_body(const uint8_t* __restrict__ src, uint8_t* __restrict__ dst, uint32_t n16) {
  const __amdgpu_buffer_rsrc_t rs = __builtin_amdgcn_make_buffer_rsrc(const_cast<uint8_t*>(src), (short)0,
                                                                      (int)(n16 * 16u), (int)kFillRsrcWord3);
  const __amdgpu_buffer_rsrc_t rd = __builtin_amdgcn_make_buffer_rsrc(dst, (short)0, (int)(n16 * 16u),
                                                                      (int)kFillRsrcWord3);
  const uint32_t stride = gridDim.x * 256u;
  uint32_t i = blockIdx.x * 256u + threadIdx.x;
  for (; i + (U - 1) * stride < n16; i += U * stride) {
    u32x4_t v[U];
#pragma unroll
    for (int u = 0; u < U; u++)
      v[u] = __builtin_bit_cast(u32x4_t, __builtin_amdgcn_raw_buffer_load_b128(rs, (i + u * stride) * 16u, 0, 2));
#pragma unroll
    for (int u = 0; u < U; u++) __builtin_amdgcn_raw_buffer_store_b128(v[u], rd, (i + u * stride) * 16u, 0, 2);
  }
  for (; i < n16; i += stride) {
    const u32x4_t a = __builtin_bit_cast(u32x4_t, __builtin_amdgcn_raw_buffer_load_b128(rs, i * 16u, 0, 2));
    __builtin_amdgcn_raw_buffer_store_b128(a, rd, i * 16u, 0, 2);
  }
}

__global__ void __launch_bounds__(256)
k_fill_bg2(const uint8_t* __restrict__ src, uint8_t* __restrict__ dst, uint32_t n16) {
  extern __shared__ uint8_t fill_lds_reserve[];
  fill_body<2>(src, dst, n16);
}
__global__ void __launch_bounds__(256)
k_fill_bg4(const uint8_t* __restrict__ src, uint8_t* __restrict__ dst, uint32_t n16) {
  extern __shared__ uint8_t fill_lds_reserve[];
  fill_body<4>(src, dst, n16);
}
__global__ void __launch_bounds__(256)
k_fill_bg8(const uint8_t* __restrict__ src, uint8_t* __restrict__ dst, uint32_t n16) {
  extern __shared__ uint8_t fill_lds_reserve[];
  fill_body<8>(src, dst, n16);
}

template <int U>
static hipError_t launch_fill_u(const void* src, void* dst, size_t bytes, int num_cus, hipStream_t s) {
  const void* k = U == 8 ? (const void*)k_fill_bg8 : U == 4 ? (const void*)k_fill_bg4 : (const void*)k_fill_bg2;
  static bool attr = false;
  if (!attr) {
    hipError_t e = hipFuncSetAttribute(k, hipFuncAttributeMaxDynamicSharedMemorySize, kFillLdsBytes);
    if (e != hipSuccess) return e;
    attr = true;
  }
  const uint8_t* sp = (const uint8_t*)src;
  uint8_t* dp = (uint8_t*)dst;
  const uint32_t n16 = (uint32_t)(bytes / 16);
  if (U == 8) k_fill_bg8<<<num_cus, 256, kFillLdsBytes, s>>>(sp, dp, n16);
  else if (U == 4) k_fill_bg4<<<num_cus, 256, kFillLdsBytes, s>>>(sp, dp, n16);
  else k_fill_bg2<<<num_cus, 256, kFillLdsBytes, s>>>(sp, dp, n16);
  return hipGetLastError();
}

// The kernel addresses a launch's range through a buffer resource whose size
// field is a signed 32-bit count, so a range of 2 GiB or more is filled by
// several launches just under 2 GiB each, back to back on the stream (same
// engine, same grid).
constexpr size_t kFillChunk = ((size_t)1 << 31) - 4096;

hipError_t launch_fill_bg(const void* src, void* dst, size_t bytes, int num_cus, int loads, hipStream_t s) {
  if (bytes % 16) return hipErrorInvalidValue;  // slot ranges are 256-byte aligned
  for (size_t off = 0; off < bytes; off += kFillChunk) {
    const size_t n = bytes - off < kFillChunk ? bytes - off : kFillChunk;
    const uint8_t* sp = (const uint8_t*)src + off;
    uint8_t* dp = (uint8_t*)dst + off;
    hipError_t e;
    switch (loads) {
      case 8: e = launch_fill_u<8>(sp, dp, n, num_cus, s); break;
      case 4: e = launch_fill_u<4>(sp, dp, n, num_cus, s); break;
      default: e = launch_fill_u<2>(sp, dp, n, num_cus, s); break;
    }
    if (e != hipSuccess) return e;
  }
  return hipSuccess;
}

__global__ void k_copy_tail(const uint8_t* __restrict__ src, uint8_t* __restrict__ dst, size_t n) {
  const size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i < n) dst[i] = src[i];
}

hipError_t launch_copy(const void* src, void* dst, size_t bytes, int grid, hipStream_t s) {
  if (bytes == 0) return hipSuccess;
  if (grid <= 0) grid = 1024;
  const size_t n16 = bytes / 16;
  if (n16) k_copy16<<<grid, 256, 0, s>>>((const f4v_t*)src, (f4v_t*)dst, n16);
  const size_t rem = bytes - n16 * 16;
  if (rem) k_copy_tail<<<1, 64, 0, s>>>((const uint8_t*)src + n16 * 16, (uint8_t*)dst + n16 * 16, rem);
  return hipGetLastError();
}

// One workgroup per staging row; 16-byte copies.
__global__ void __launch_bounds__(256) k_rows_move(RowMove m) {
  const int i = blockIdx.x;
  int r = 0;
  while (r + 1 < m.n && m.row_off[r + 1] <= i) r++;
  uint8_t* srow = (uint8_t*)m.staging + (size_t)i * m.row_bytes;
  uint8_t* rrow = (uint8_t*)m.rep[r] + (size_t)(i - m.row_off[r]) * m.row_bytes;
  const uint8_t* from = m.gather ? rrow : srow;
  uint8_t* to = m.gather ? srow : rrow;
  for (size_t j = (size_t)threadIdx.x * 16; j < m.row_bytes; j += 256 * 16)
    *(u32x4_t*)(to + j) = *(const u32x4_t*)(from + j);
}

hipError_t launch_rows_move(const RowMove& m, hipStream_t s) {
  if (m.n < 1 || m.n > kMaxReplicas || m.row_bytes % 16) return hipErrorInvalidValue;
  const int rows = m.row_off[m.n];
  if (rows <= 0) return hipSuccess;
  k_rows_move<<<rows, 256, 0, s>>>(m);
  return hipGetLastError();
}

__global__ void k_poison(uint32_t* __restrict__ dst, size_t n) {
  const size_t stride = (size_t)gridDim.x * blockDim.x;
  for (size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += stride) dst[i] = 0xffffffffu;
}

hipError_t launch_poison(void* dst, size_t bytes, hipStream_t s) {
  const size_t n = bytes / 4;
  if (n) k_poison<<<1024, 256, 0, s>>>((uint32_t*)dst, n);
  return hipGetLastError();
}

// Spins for `ticks` of the 100 MHz constant clock; the iteration cap bounds
// it even if the clock were not to advance.
__global__ void k_spin(int64_t ticks) {
  const uint64_t t0 = wall_clock64();
  for (int it = 0; it < (1 << 22); it++) {
    if ((int64_t)(wall_clock64() - t0) >= ticks) break;
    __builtin_amdgcn_s_sleep(8);
  }
}

hipError_t launch_spin(int64_t ticks, hipStream_t s) {
  k_spin<<<1, 64, 0, s>>>(ticks);
  return hipGetLastError();
}

}  // namespace sidp
