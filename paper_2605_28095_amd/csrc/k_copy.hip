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
