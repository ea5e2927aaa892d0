// adapter_predict_static: the adapter priorities of section "Expert
// Prediction Adapter" on explicit device weights, for callers that cannot
// allocate device memory.  Its scratch -- two completion counters and the
// per-token adapter hidden units / distributions -- lives in one file-scope
// device array of fixed size instead of a context's allocation.  Each device
// the library runs on holds its own copy of the array (at its own address,
// looked up once per device) until the process ends; every call on a device
// shares it.
#include <hip/hip_runtime.h>

#include <cstdint>
#include <mutex>

#include "spp.h"
#include "spp_internal.h"

namespace {

constexpr int kCounterWords = 64;  // 256 bytes; the router kernels use the first two
constexpr size_t kScratchFloats = SPP_STATIC_SCRATCH_FLOATS;

// [counters: kCounterWords u32][hidden units / distributions: B * (n + r) floats]
static __device__ __align__(256) float scratch[kCounterWords + kScratchFloats];

constexpr int kMaxDevices = 64;
std::mutex g_mu;
void* g_scratch[kMaxDevices] = {};  // device address of `scratch` on each device, once looked up

// The counters must start at zero; a kernel clears them (no memset node in a
// captured graph).
__global__ void clear_counters(unsigned* p, int n) {
  const int i = static_cast<int>(threadIdx.x);
  if (i < n) p[i] = 0u;
}

// The array's device address on the current device (host code never passes
// the array's own name: on the host it is only a stand-in for the symbol).
hipError_t scratch_address(void** out) {
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
  std::lock_guard<std::mutex> lock(g_mu);
  if (!g_scratch[dev]) {
    void* p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return e;
    g_scratch[dev] = p;
  }
  *out = g_scratch[dev];
  return hipSuccess;
}

bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

}  // namespace

extern "C" spp_status adapter_predict_static(const void* adapter_a, const void* adapter_b, int32_t dtype, int32_t D,
                                             int32_t n, int32_t r, const float* x_dev, int32_t B, float* s_out_dev,
                                             void* hip_stream) {
  if (!adapter_a || !adapter_b || !x_dev || !s_out_dev)
    return spp::set_error(SPP_EINVAL, "adapter_a, adapter_b, x_dev and s_out_dev must not be NULL");
  if (dtype != SPP_DTYPE_F32 && dtype != SPP_DTYPE_BF16)
    return spp::set_error(SPP_EINVAL, "dtype must be 0 (f32) or 1 (bf16)");
  const int elem = dtype == SPP_DTYPE_BF16 ? 2 : 4;
  if (D < 1 || n < 1 || r < 1 || B < 1) return spp::set_error(SPP_EINVAL, "D, n, r and B must be >= 1");
  if ((static_cast<int64_t>(D) * elem) % 16 != 0 || (D * elem / 16 + 63) / 64 > 8)
    return spp::set_error(SPP_EINVAL, "D * element size must be a multiple of 16 bytes, D at most 4096 bf16 / 2048 fp32");
  if (n > spp::kMaxExpertsTopK || r > 256) return spp::set_error(SPP_EINVAL, "n must be <= 1024 and r <= 256");
  if ((static_cast<int64_t>(n) * r * elem) % 16 != 0)
    return spp::set_error(SPP_EINVAL, "n * r * element size must be a multiple of 16 bytes");
  if (B > 1 && D % 16 != 0) return spp::set_error(SPP_EINVAL, "B > 1 needs D a multiple of 16");
  if (static_cast<int64_t>(B) * (n + r) > static_cast<int64_t>(kScratchFloats))
    return spp::set_error(SPP_EINVAL, "B * (n + r) exceeds the static scratch (SPP_STATIC_SCRATCH_FLOATS)");
  if (!aligned16(adapter_a) || !aligned16(adapter_b) || !aligned16(x_dev))
    return spp::set_error(SPP_EINVAL, "adapter_a, adapter_b and x_dev must be 16-byte aligned");
  void* base = nullptr;
  hipError_t e = scratch_address(&base);
  if (e != hipSuccess) return spp::set_error(SPP_EHIP, hipGetErrorString(e));
  const hipStream_t st = static_cast<hipStream_t>(hip_stream);
  unsigned* counter = static_cast<unsigned*>(base);
  hipLaunchKernelGGL(clear_counters, dim3(1), dim3(64), 0, st, counter, 2);
  e = hipGetLastError();
  if (e != hipSuccess) return spp::set_error(SPP_EHIP, hipGetErrorString(e));
  spp::RouterArgs ra{};
  ra.u = x_dev;           // the router inputs themselves (no normalisation)
  ra.A = adapter_a;
  ra.Bm = adapter_b;
  ra.zbuf = static_cast<float*>(base) + kCounterWords;
  ra.s = s_out_dev;
  ra.counter = counter;
  ra.B = B;
  ra.D = D;
  ra.n = n;
  ra.K = 1;               // no routing: the router rows are off
  ra.r = r;
  ra.x_given = 1;
  ra.router_on = 0;
  e = spp::launch_router(ra, dtype, st);
  if (e != hipSuccess) return spp::set_error(SPP_EHIP, hipGetErrorString(e));
  return SPP_OK;
}
