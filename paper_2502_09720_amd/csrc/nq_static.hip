// nq_matmul_static: nq_matmul_ex with its workspace in a fixed device array of the library
// (`scratch`), for callers that cannot allocate device memory.
//
// `scratch` is a file-scope __device__ array: every device the library runs on holds its own
// copy, at its own address, until the process ends.  In host code the array's name is only
// a host-side stand-in, never a device address, so the address each device's copy has is
// looked up once per device (hipGetSymbolAddress, with that device current) on the first
// call there and kept; kernels get that pointer as their workspace argument.
//
// The workspace needs no clearing: the decode stage writes every byte of it that the
// contraction reads (padding included) on every call.  Calls on one device share the array,
// so calls whose kernels overlap on that device (other streams, other host threads) race.
#include <mutex>

#include "nestquant.h"
#include "nq_kernels.hpp"

namespace {

static __device__ __align__(256) unsigned char scratch[NQ_STATIC_SCRATCH_BYTES];

constexpr int kDevices = 64;
std::mutex g_mu;
void* g_ptr[kDevices] = {};

// The device address of `scratch` on the device that stream st runs on.
hipError_t scratch_address(hipStream_t st, void** out) {
  hipDevice_t dev = 0;
  hipError_t e = hipStreamGetDevice(st, &dev);
  if (e != hipSuccess) return e;
  if (dev < 0 || dev >= kDevices) return hipErrorInvalidDevice;
  std::lock_guard<std::mutex> g(g_mu);
  if (!g_ptr[dev]) {
    int cur = 0;
    if ((e = hipGetDevice(&cur)) != hipSuccess) return e;
    if (cur != dev && (e = hipSetDevice(dev)) != hipSuccess) return e;
    void* p = nullptr;
    const hipError_t r = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (cur != dev && (e = hipSetDevice(cur)) != hipSuccess) return e;
    if (r != hipSuccess) return r;
    if (!p) return hipErrorInvalidSymbol;
    g_ptr[dev] = p;
  }
  *out = g_ptr[dev];
  return hipSuccess;
}

}  // namespace

extern "C" nq_status nq_matmul_static(const nq_params* pa, const uint32_t* a_codes,
                                      const uint32_t* a_beta, const float* a_scales, int64_t M,
                                      const nq_params* pw, const uint32_t* w_codes,
                                      const uint32_t* w_beta, const float* w_scales, int64_t N,
                                      int64_t K, float* c, int64_t ldc, void* hip_stream) {
  const int64_t need = nq_matmul_workspace_size(M, N, K);
  if (need > (int64_t)NQ_STATIC_SCRATCH_BYTES)
    return nq::set_error(NQ_ERR_UNSUPPORTED,
                         "nq_matmul_static: this product needs %lld bytes of workspace, more than "
                         "the library's static %lld; call nq_matmul_ex with a workspace",
                         (long long)need, (long long)NQ_STATIC_SCRATCH_BYTES);
  void* ws = nullptr;
  if (need > 0) {
    const hipError_t e = scratch_address((hipStream_t)hip_stream, &ws);
    if (e != hipSuccess)
      return nq::set_error(NQ_ERR_HIP, "nq_matmul_static: %s", hipGetErrorString(e));
  }
  // validation, then the decode-once (or skinny) product of nq_matmul_ex on the scratch
  return nq::matmul_stages(NQ_STAGE_DECODE | NQ_STAGE_CONTRACT, pa, a_codes, a_beta, a_scales,
                           M, pw, w_codes, w_beta, w_scales, N, K, c, ldc, ws,
                           need > 0 ? need : 0, hip_stream, "nq_matmul_static");
}
