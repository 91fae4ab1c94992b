// sidp_linear_noalloc: the dense projection of sidp_linear for callers that
// cannot allocate device memory (code under HIP graph capture, serving loops
// that forbid allocation). Its split-K partials go to `scratch`, a file-scope
// device array that the code object brings with it: each device the library
// runs on holds its own copy from module load until the process ends.
//
// The array's name is a host-side stand-in in host code; the device address
// of each device's copy is taken once per device with hipGetSymbolAddress,
// with that device current, and only that address is handed to kernels.
#include <hip/hip_runtime.h>

#include <mutex>

#include "../../include/sidp.h"
#include "internal.h"

namespace {

// Every split writes its whole partial block before the reduction reads it,
// so nothing here has to start at zero.
__device__ __align__(256) unsigned char scratch[SIDP_NOALLOC_SCRATCH_BYTES];

constexpr int kMaxDevices = 64;
struct DeviceScratch {
  std::once_flag once;
  void* ptr = nullptr;   // device address of this device's `scratch`
  int num_cus = 0;
  hipError_t err = hipSuccess;
};
DeviceScratch g_dev[kMaxDevices];

// The device's scratch address and CU count, looked up on its first use.
hipError_t device_scratch(int dev, void** ptr, int* num_cus) {
  DeviceScratch& d = g_dev[dev];
  std::call_once(d.once, [&] {
    d.err = hipGetSymbolAddress(&d.ptr, HIP_SYMBOL(scratch));
    if (d.err == hipSuccess) d.err = hipDeviceGetAttribute(&d.num_cus, hipDeviceAttributeMultiprocessorCount, dev);
  });
  *ptr = d.ptr;
  *num_cus = d.num_cus;
  return d.err;
}

}  // namespace

extern "C" int sidp_linear_noalloc(const void* x, int32_t m, int32_t k, const void* packed, int32_t n,
                                   int32_t epilogue, const void* bias, const float* residual, void* out,
                                   void* stream) {
  if (!x || !packed || !out || m < 1 || m > 4096 || k < 8 || k % 8 || n < 1) return SIDP_EINVAL;
  if (k > (1 << 24) || n > (1 << 24)) return SIDP_EINVAL;
  if (epilogue < SIDP_EPI_BF16 || epilogue > SIDP_EPI_SWIGLU) return SIDP_EINVAL;
  if (epilogue == SIDP_EPI_RESID && !residual) return SIDP_EINVAL;
  if (epilogue != SIDP_EPI_BF16 && bias) return SIDP_EINVAL;
  const int ncols = epilogue == SIDP_EPI_SWIGLU ? 2 * ((n + 31) / 32 * 32) : n;
  if (!sidp::gemm_fits(m, ncols, k)) return SIDP_EINVAL;
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess) return SIDP_EHIP;
  if (dev < 0 || dev >= kMaxDevices) return SIDP_EINVAL;
  void* ws = nullptr;
  int num_cus = 0;
  if (device_scratch(dev, &ws, &num_cus) != hipSuccess) return SIDP_EHIP;
  // the same split as sidp_linear; refused if its partials outgrow the scratch
  if (sidp::gemm_ws_bytes(m, ncols, k, num_cus) > (size_t)SIDP_NOALLOC_SCRATCH_BYTES) return SIDP_EINVAL;
  sidp::LinearCall c;
  c.x = x;
  c.m = m;
  c.k = k;
  c.packed = packed;
  c.n = n;
  c.epilogue = epilogue;
  c.bias = bias;
  c.residual = residual;
  c.out = out;
  c.ws = (float*)ws;
  c.ws_bytes = SIDP_NOALLOC_SCRATCH_BYTES;
  c.num_cus = num_cus;
  return sidp::launch_linear(c, (hipStream_t)stream) == hipSuccess ? SIDP_OK : SIDP_EHIP;
}
