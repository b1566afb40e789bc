// Device scratch of the no-allocation entry point (lionmuon_step_noalloc):
// one file-scope array per device, holding the plan tables, the per-call
// address table and the Newton-Schulz workspace of the call, plus the kernel
// that fills the tables from its own arguments (so that no pinned staging
// buffer, and no allocation of any kind, is needed to reach the device).
//
// In host code `scratch` names a host-side stand-in, not device memory: every
// host use goes through the device address scratch_address() returns.
#include <hip/hip_runtime.h>

#include <cstring>
#include <mutex>
#include <utility>
#include <vector>

#include "kernels.h"

namespace lm {

namespace {

static __device__ __align__(256) uint8_t scratch[kScratchBytes];

constexpr int kUploadWords = 512;   // 2 KB of table data per launch (kernel arguments)

struct UploadArgs {
  uint32_t* dst;
  uint32_t n;                       // words in this chunk
  uint32_t w[kUploadWords];
};

__global__ __launch_bounds__(256) void upload_kernel(UploadArgs a) {
  for (uint32_t i = threadIdx.x; i < a.n; i += 256) a.dst[i] = a.w[i];
}

}  // namespace

namespace {
// Device address of `scratch` on each device, looked up once per device (with
// that device current) and kept for the life of the process.
std::mutex g_scratch_mu;
std::vector<std::pair<int, void*>> g_scratch_ptr;
}  // namespace

hipError_t scratch_address(int device, void** out) {
  *out = nullptr;
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  for (const auto& d : g_scratch_ptr)
    if (d.first == device) {
      *out = d.second;
      return hipSuccess;
    }
  int current = -1;
  hipError_t e = hipGetDevice(&current);
  if (e != hipSuccess) return e;
  if (current != device) return hipErrorInvalidDevice;
  void* ptr = nullptr;
  e = hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch));
  if (e != hipSuccess) return e;
  if (ptr == nullptr) return hipErrorInvalidSymbol;
  g_scratch_ptr.push_back({device, ptr});
  *out = ptr;
  return hipSuccess;
}

hipError_t launch_upload(void* dst, const void* src, size_t bytes, hipStream_t stream) {
  if ((reinterpret_cast<uintptr_t>(dst) & 3u) || (bytes & 3u)) return hipErrorInvalidValue;
  const uint8_t* s = static_cast<const uint8_t*>(src);
  uint32_t* d = static_cast<uint32_t*>(dst);
  const size_t words = bytes / 4;
  for (size_t w0 = 0; w0 < words; w0 += kUploadWords) {
    UploadArgs a;
    a.dst = d + w0;
    a.n = uint32_t(words - w0 < size_t(kUploadWords) ? words - w0 : size_t(kUploadWords));
    std::memcpy(a.w, s + w0 * 4, size_t(a.n) * 4);
    hipLaunchKernelGGL(upload_kernel, dim3(1), dim3(256), 0, stream, a);
    const hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  return hipSuccess;
}

}  // namespace lm
