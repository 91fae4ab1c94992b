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

// Split-K reduction of a projection with a residual epilogue, fused with the
// RMSNorm that reads its result (the O projection followed by the FFN norm):
//   x[row] += sum_s partial_s[row]          (fp32, partials summed in split order)
//   h[row]  = bf16(x[row] / sqrt(mean(x[row]^2) + eps) * g)
// One 1024-thread workgroup per row; each thread keeps its float4 chunks in
// registers between the two passes. The partials of split s are rows of NP
// floats at ws + s * M * NP.
constexpr int kRrnThreads = 1024;
constexpr int kRrnMaxChunks = 4;  // rows of up to 16384 columns

__global__ void __launch_bounds__(kRrnThreads) k_reduce_resid_norm(const float* __restrict__ ws, int splits, int M,
                                                                  int NP, int n, float* __restrict__ x,
                                                                  const uint16_t* __restrict__ g, float eps,
                                                                  uint16_t* __restrict__ h) {
  __shared__ float red[kRrnThreads / 64];
  const int row = blockIdx.x;
  float* xr = x + (int64_t)row * n;
  float4 v[kRrnMaxChunks];
  float ss = 0.f;
#pragma unroll
  for (int c = 0; c < kRrnMaxChunks; c++) {
    const int i = (threadIdx.x + c * kRrnThreads) * 4;
    if (i < n) {
      // partials four splits at a time: the loads of a group are in flight
      // together, the sum still runs in split order
      float4 acc = make_float4(0.f, 0.f, 0.f, 0.f);
      for (int sp0 = 0; sp0 < splits; sp0 += 4) {
        float4 p[4];
#pragma unroll
        for (int j = 0; j < 4; j++)
          if (sp0 + j < splits) p[j] = *(const float4*)(ws + ((int64_t)(sp0 + j) * M + row) * NP + i);
#pragma unroll
        for (int j = 0; j < 4; j++)
          if (sp0 + j < splits) {
            acc.x += p[j].x;
            acc.y += p[j].y;
            acc.z += p[j].z;
            acc.w += p[j].w;
          }
      }
      const float4 r = *(const float4*)(xr + i);
      v[c] = make_float4(r.x + acc.x, r.y + acc.y, r.z + acc.z, r.w + acc.w);
      *(float4*)(xr + i) = v[c];
      ss += v[c].x * v[c].x + v[c].y * v[c].y + v[c].z * v[c].z + v[c].w * v[c].w;
    }
  }
  ss = wave_sum(ss);
  if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = ss;
  __syncthreads();
  float total = 0.f;
#pragma unroll
  for (int w = 0; w < kRrnThreads / 64; w++) total += red[w];
  const float rs = 1.0f / sqrtf(total / (float)n + eps);
  uint16_t* hr = h + (int64_t)row * n;
#pragma unroll
  for (int c = 0; c < kRrnMaxChunks; c++) {
    const int i = (threadIdx.x + c * kRrnThreads) * 4;
    if (i < n) {
      const uint2 gg = *(const uint2*)(g + i);
      uint2 o;
      o.x = pack_bf2(v[c].x * rs * bf2f((uint16_t)(gg.x & 0xffff)), v[c].y * rs * bf2f((uint16_t)(gg.x >> 16)));
      o.y = pack_bf2(v[c].z * rs * bf2f((uint16_t)(gg.y & 0xffff)), v[c].w * rs * bf2f((uint16_t)(gg.y >> 16)));
      *(uint2*)(hr + i) = o;
    }
  }
}

bool reduce_resid_norm_fits(int n) { return n % 4 == 0 && n <= kRrnMaxChunks * kRrnThreads * 4; }

hipError_t launch_reduce_resid_norm(const float* ws, int splits, int M, int NP, int n, float* x, const void* gain,
                                    float eps, void* h, hipStream_t s) {
  if (M <= 0) return hipSuccess;
  if (!reduce_resid_norm_fits(n)) return hipErrorInvalidValue;
  k_reduce_resid_norm<<<M, kRrnThreads, 0, s>>>(ws, splits, M, NP, n, x, (const uint16_t*)gain, eps, (uint16_t*)h);
  return hipGetLastError();
}

}  // namespace sidp
