// noalloc.hip -- the fixed device workspace of comet_w4ax_gemm_noalloc.
//
// The tile kernels need device memory beyond their inputs and outputs: the
// schedule (work units, K-block order, split table) and, for split tiles, fp32
// partials and arrival counters.  comet_w4ax_gemm allocates these on first
// use; the no-allocation entry point takes them from one static array per
// device instead, laid out as
//     [partials: kPartialBytes][counters: kCounterBytes][plan: kPlanBytes].
// In host code the array's name is only a host-side stand-in: its device
// address comes from hipGetSymbolAddress, taken once per device with that
// device current, and only that address is ever handed to kernels or copies.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include <map>
#include <mutex>

#include "kernels.h"

namespace comet {

namespace {

__device__ __align__(256) uint8_t scratch[kNoallocBytes];

std::mutex g_scratch_mu;
std::map<int, uint8_t*> g_scratch_ptr;

__global__ void zero_ints(int* p, int n) {
  const int i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i < n) p[i] = 0;
}

}  // namespace

hipError_t noalloc_scratch(int dev, uint8_t** ptr) {
  std::lock_guard<std::mutex> lk(g_scratch_mu);
  auto it = g_scratch_ptr.find(dev);
  if (it != g_scratch_ptr.end()) {
    *ptr = it->second;
    return hipSuccess;
  }
  void* p = nullptr;
  const hipError_t e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
  if (e != hipSuccess) return e;
  g_scratch_ptr[dev] = static_cast<uint8_t*>(p);
  *ptr = static_cast<uint8_t*>(p);
  return hipSuccess;
}

hipError_t launch_zero_ints(int* p, int n, hipStream_t stream) {
  if (n <= 0) return hipSuccess;
  hipLaunchKernelGGL(zero_ints, dim3((n + 255) / 256), dim3(256), 0, stream, p, n);
  return hipGetLastError();
}

}  // namespace comet
