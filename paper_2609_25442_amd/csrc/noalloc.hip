// Device memory the library holds itself, for callers that cannot allocate
// (code under stream capture, tight serving loops, harnesses that forbid
// allocation): wb_unpack_round_noalloc stages a round's work tables and its
// pointer table here instead of in a caller workspace.
//
// The array is a file-scope device variable: every GPU the library runs on
// holds its own copy, at its own address, until the process ends. In host code
// its name denotes a host-side stand-in, not device memory, so host code never
// uses the name as an address: scratch_address() asks the runtime for the
// current device's copy once per device (hipGetSymbolAddress, with that device
// current) and every later use goes through the pointer it returns.
#include <hip/hip_runtime.h>

#include <mutex>

#include "wb_internal.hpp"

namespace wb {
namespace {

constexpr size_t kScratchBytes = size_t(32) << 20;
constexpr int kMaxDevices = 64;

static __device__ __align__(256) uint8_t scratch[kScratchBytes];

std::mutex g_mutex;
void* g_scratch[kMaxDevices];  // per device; null until first looked up

// Up to kWords table entries per launch, carried in the kernel arguments.
constexpr int kWords = 32;
struct Words {
  uint64_t w[kWords];
};

__global__ __launch_bounds__(64) void wb_store_words_kernel(uint64_t* dst, Words v, uint32_t n) {
  const uint32_t i = threadIdx.x;
  if (i < n) dst[i] = v.w[i];
}

}  // namespace

int scratch_address(void** out, size_t* bytes) {
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
  std::lock_guard<std::mutex> lock(g_mutex);
  if (!g_scratch[dev]) {
    void* p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return e;
    if (!p) return hipErrorInvalidSymbol;
    g_scratch[dev] = p;
  }
  *out = g_scratch[dev];
  *bytes = kScratchBytes;
  return hipSuccess;
}

int launch_store_table(uint64_t* dev, const void* const* ptrs, int n, void* stream) {
  // entry 0 stands for the launch's buffer argument and is never read
  for (int first = 0; first < n + 1; first += kWords) {
    Words v{};
    const int m = std::min(kWords, n + 1 - first);
    for (int i = 0; i < m; ++i) {
      const int k = first + i;
      v.w[i] = k == 0 ? 0 : reinterpret_cast<uint64_t>(ptrs[k - 1]);
    }
    hipLaunchKernelGGL(wb_store_words_kernel, dim3(1), dim3(64), 0, static_cast<hipStream_t>(stream), dev + first, v,
                       static_cast<uint32_t>(m));
    const hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  return hipSuccess;
}

}  // namespace wb
