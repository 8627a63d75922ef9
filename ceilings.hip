// Practical HBM ceilings of this GPU for 16-byte vector streams: read-only,
// write-only, copy with one contiguous 256 KiB chunk per workgroup looping over
// it, hipMemcpy, copy with one-shot one-wave workgroups (one load and one store
// per lane, the copy kernel's pattern), and a one-shot stream that reads two
// bytes per byte written (each lane loads two vectors one wave apart and
// stores one: the read/write mix of the fp32 -> bf16 and fp8 assembly), over
// 8 GiB buffers, best of five. Prints one JSON object. Used to put the
// resharding kernels' bandwidth next to what a plain stream reaches on the
// same part.
#include <hip/hip_runtime.h>

#include <cstdint>
#include <cstdio>

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));

#define CHECK(x)                                                                   \
  do {                                                                             \
    hipError_t e_ = (x);                                                           \
    if (e_ != hipSuccess) {                                                        \
      std::fprintf(stderr, "HIP error %s at line %d\n", hipGetErrorString(e_), __LINE__); \
      return 1;                                                                    \
    }                                                                              \
  } while (0)

__global__ void read_stream(const u32x4* __restrict__ s, uint64_t n, u32x4* __restrict__ out) {
  u32x4 acc = {0, 0, 0, 0};
  const uint64_t stride = uint64_t(gridDim.x) * blockDim.x;
  uint64_t i = uint64_t(blockIdx.x) * blockDim.x + threadIdx.x;
  for (; i + 3 * stride < n; i += 4 * stride) {
    u32x4 v[4];
#pragma unroll
    for (int k = 0; k < 4; ++k) v[k] = __builtin_nontemporal_load(s + i + k * stride);
#pragma unroll
    for (int k = 0; k < 4; ++k) acc ^= v[k];
  }
  for (; i < n; i += stride) acc ^= s[i];
  out[uint64_t(blockIdx.x) * blockDim.x + threadIdx.x] = acc;
}

__global__ void write_stream(u32x4* __restrict__ d, uint64_t n) {
  const uint64_t stride = uint64_t(gridDim.x) * blockDim.x;
  const u32x4 v = {1u, 2u, 3u, uint32_t(threadIdx.x)};
  for (uint64_t i = uint64_t(blockIdx.x) * blockDim.x + threadIdx.x; i < n; i += stride) d[i] = v;
}

__global__ void copy_chunks(const u32x4* __restrict__ s, u32x4* __restrict__ d, uint64_t n, uint64_t per) {
  const uint64_t a = uint64_t(blockIdx.x) * per;
  const uint64_t b = a + per < n ? a + per : n;
  uint64_t i = a + threadIdx.x;
  for (; i + 3 * blockDim.x < b; i += 4 * blockDim.x) {
    u32x4 v[4];
#pragma unroll
    for (int k = 0; k < 4; ++k) v[k] = __builtin_nontemporal_load(s + i + k * blockDim.x);
#pragma unroll
    for (int k = 0; k < 4; ++k) __builtin_nontemporal_store(v[k], d + i + k * blockDim.x);
  }
  for (; i < b; i += blockDim.x) d[i] = s[i];
}

__global__ void copy_oneshot(const u32x4* __restrict__ s, u32x4* __restrict__ d) {
  const uint64_t i = uint64_t(blockIdx.x) * blockDim.x + threadIdx.x;
  __builtin_nontemporal_store(__builtin_nontemporal_load(s + i), d + i);
}

// vectors 2 b T + l and 2 b T + T + l in, one vector out (T = blockDim.x)
__global__ void read2_write1_oneshot(const u32x4* __restrict__ s, u32x4* __restrict__ d) {
  const uint64_t i = uint64_t(blockIdx.x) * 2 * blockDim.x + threadIdx.x;
  const u32x4 a = __builtin_nontemporal_load(s + i), b = __builtin_nontemporal_load(s + i + blockDim.x);
  __builtin_nontemporal_store(a ^ b, d + uint64_t(blockIdx.x) * blockDim.x + threadIdx.x);
}

// the memory shape of the fp32 -> bf16 and fp8 assemblies: vectors 2 b T + l
// and 2 b T + T + l in, an 8-byte half of each out at the same two positions
// of an array of halves
__global__ void read2_write1_halves_oneshot(const u32x4* __restrict__ s, u32x2* __restrict__ d) {
  const uint64_t i = uint64_t(blockIdx.x) * 2 * blockDim.x + threadIdx.x;
  const u32x4 a = __builtin_nontemporal_load(s + i), b = __builtin_nontemporal_load(s + i + blockDim.x);
  __builtin_nontemporal_store(u32x2{a.x ^ a.z, a.y ^ a.w}, d + i);
  __builtin_nontemporal_store(u32x2{b.x ^ b.z, b.y ^ b.w}, d + i + blockDim.x);
}

int main() {
  const uint64_t bytes = 8ull << 30, n = bytes / 16;
  const int read_grid = 512, write_grid = 16384, threads = 256;
  const uint64_t per = 16384;  // 256 KiB per workgroup
  u32x4 *s, *d, *out;
  CHECK(hipMalloc(&s, bytes));
  CHECK(hipMalloc(&d, bytes));
  CHECK(hipMalloc(&out, uint64_t(read_grid) * threads * 16));
  CHECK(hipMemset(s, 1, bytes));
  CHECK(hipMemset(d, 0, bytes));
  hipEvent_t e0, e1;
  CHECK(hipEventCreate(&e0));
  CHECK(hipEventCreate(&e1));
  double gbs[7];
  for (int which = 0; which < 7; ++which) {
    float best = 1e30f;
    for (int r = 0; r < 6; ++r) {
      CHECK(hipEventRecord(e0));
      if (which == 0) read_stream<<<read_grid, threads>>>(s, n, out);
      if (which == 1) write_stream<<<write_grid, threads>>>(d, n);
      if (which == 2) copy_chunks<<<int((n + per - 1) / per), threads>>>(s, d, n, per);
      if (which == 3) CHECK(hipMemcpyAsync(d, s, bytes, hipMemcpyDeviceToDevice, 0));
      if (which == 4) copy_oneshot<<<int(n / 64), 64>>>(s, d);
      if (which == 5) read2_write1_oneshot<<<int(n / 2 / 64), 64>>>(s, d);  // reads n vectors, writes n / 2
      if (which == 6) read2_write1_halves_oneshot<<<int(n / 2 / 64), 64>>>(s, reinterpret_cast<u32x2*>(d));
      CHECK(hipEventRecord(e1));
      CHECK(hipEventSynchronize(e1));
      float ms;
      CHECK(hipEventElapsedTime(&ms, e0, e1));
      if (r > 0 && ms < best) best = ms;  // first run warms up
    }
    const double moved = which >= 5 ? 1.5 : which >= 2 ? 2.0 : 1.0;  // bytes read + written per buffer byte
    gbs[which] = moved * double(bytes) / (best * 1e-3) / 1e9;
  }
  std::printf("{\"read_GBps\": %.1f, \"write_GBps\": %.1f, \"copy_GBps\": %.1f, \"hipMemcpy_GBps\": %.1f, "
              "\"copy_oneshot_GBps\": %.1f, \"read2_write1_oneshot_GBps\": %.1f, "
              "\"read2_write1_halves_oneshot_GBps\": %.1f, \"bytes\": %llu}\n",
              gbs[0], gbs[1], gbs[2], gbs[3], gbs[4], gbs[5], gbs[6], (unsigned long long)bytes);
  CHECK(hipFree(s));
  CHECK(hipFree(d));
  CHECK(hipFree(out));
  return 0;
}
