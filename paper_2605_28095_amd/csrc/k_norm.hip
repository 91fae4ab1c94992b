// RMSNorm of the fp32 residual stream into the bf16 GEMM input (K1/K6):
// out = bf16(x / sqrt(mean(x^2) + eps) * g). One workgroup per row; HBM-bound
// and tiny next to the projections.
#include "common.h"
#include "internal.h"

namespace sidp {

__global__ void __launch_bounds__(256) k_rmsnorm(const float* __restrict__ x, const uint16_t* __restrict__ g,
                                                 float eps, uint16_t* __restrict__ out, int n) {
  __shared__ float red[4];
  const int row = blockIdx.x;
  const float* xr = x + (int64_t)row * n;
  float ss = 0.f;
  for (int i = threadIdx.x * 4; i < n; i += 1024) {
    const float4 v = *(const float4*)(xr + i);
    ss += v.x * v.x + v.y * v.y + v.z * v.z + v.w * v.w;
  }
  ss = wave_sum(ss);
  if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = ss;
  __syncthreads();
  const float total = red[0] + red[1] + red[2] + red[3];
  const float r = 1.0f / sqrtf(total / (float)n + eps);
  uint16_t* orow = out + (int64_t)row * n;
  for (int i = threadIdx.x * 4; i < n; i += 1024) {
    const float4 v = *(const float4*)(xr + i);
    const uint2 gg = *(const uint2*)(g + i);
    const float g0 = bf2f((uint16_t)(gg.x & 0xffff)), g1 = bf2f((uint16_t)(gg.x >> 16));
    const float g2 = bf2f((uint16_t)(gg.y & 0xffff)), g3 = bf2f((uint16_t)(gg.y >> 16));
    uint2 o;
    o.x = pack_bf2(v.x * r * g0, v.y * r * g1);
    o.y = pack_bf2(v.z * r * g2, v.w * r * g3);
    *(uint2*)(orow + i) = o;
  }
}

hipError_t launch_rmsnorm(const float* x, const void* gain, float eps, void* out, int rows, int n, hipStream_t s) {
  if (rows <= 0) return hipSuccess;
  k_rmsnorm<<<rows, 256, 0, s>>>(x, (const uint16_t*)gain, eps, (uint16_t*)out, n);
  return hipGetLastError();
}

}  // namespace sidp
