// Device scratch of the allocation-free GEMM entry point
// (pw_moe_paged_gemm_noalloc in include/pw.h).
//
// The paged GEMM's workspace (the SwiGLU rows of every routed slot and the
// down projection's fp32 partial sums) lives here, in one file-scope array
// per GPU, so that a caller that cannot allocate device memory still runs the
// same kernels. The array is loaded with the code object on every GPU the
// library runs on and stays until the process ends. Host code never uses the
// array's name as an address: the device address comes from
// hipGetSymbolAddress, looked up once per GPU with that GPU current, and is
// what the kernels receive.
#include <hip/hip_runtime.h>

#include <mutex>

#include "pw_internal.hpp"

static __device__ __align__(256) uint8_t scratch[pw::kStaticScratchBytes];

namespace {

constexpr int kMaxDevices = 64;
std::mutex g_mu;
void* g_ptr[kMaxDevices];   // device address of `scratch` per GPU; null until looked up

}  // namespace

namespace pw {

hipError_t static_scratch(int device, void** ptr) {
  if (device < 0 || device >= kMaxDevices) return hipErrorInvalidDevice;
  std::lock_guard<std::mutex> lock(g_mu);
  if (!g_ptr[device]) {
    int cur = -1;
    hipError_t e = hipGetDevice(&cur);
    if (e != hipSuccess) return e;
    if (cur != device && (e = hipSetDevice(device)) != hipSuccess) return e;
    void* p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (cur != device) {
      const hipError_t e2 = hipSetDevice(cur);
      if (e == hipSuccess) e = e2;
    }
    if (e != hipSuccess) return e;
    if (!p) return hipErrorInvalidSymbol;
    g_ptr[device] = p;
  }
  *ptr = g_ptr[device];
  return hipSuccess;
}

}  // namespace pw
