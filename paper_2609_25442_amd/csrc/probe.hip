// Source-map probing kernels (WeightBridge Sec. 3.1 and App. B, Algorithm 1).
//
// wb_make_ids_kernel writes one b-bit chunk of every checkpoint element's
// identifier into a checkpoint tensor, in a form a value-preserving loader
// copies unchanged: 16-bit and 8-bit dtypes carry the chunk as their bit
// pattern, fp32 carries it as an exactly representable value.
//
// wb_diff2_kernel computes the second-order difference of a loaded chunk
// field (Eq. diff2: the outer product of [1, -2, 1] with itself, the field
// taken as 0 above and left of the tensor) and appends its non-zero entries
// to a list. A slice copy leaves at most 16 of them, so the list is short.
#include <hip/hip_runtime.h>

#include <cstdint>

#include "wb_internal.hpp"

namespace wb {
namespace {

constexpr int kThreads = 256;
constexpr int kStrip = 64;  // rows per workgroup in the stencil

__global__ __launch_bounds__(kThreads) void wb_make_ids_kernel(char* dst, int dtype, int64_t numel, int64_t first_id,
                                                               int shift, uint32_t mask) {
  const int64_t stride = int64_t(gridDim.x) * kThreads;
  for (int64_t n = int64_t(blockIdx.x) * kThreads + threadIdx.x; n < numel; n += stride) {
    const uint32_t v = uint32_t((uint64_t(first_id + n) >> shift) & mask);
    if (dtype == WB_F32)
      reinterpret_cast<float*>(dst)[n] = float(v);
    else if (dtype == WB_BF16)
      reinterpret_cast<uint16_t*>(dst)[n] = uint16_t(v);
    else
      reinterpret_cast<uint8_t*>(dst)[n] = uint8_t(v);
  }
}

__device__ __forceinline__ int load_chunk(const char* src, int dtype, int64_t k) {
  if (dtype == WB_F32) return int(reinterpret_cast<const float*>(src)[k]);
  if (dtype == WB_BF16) return int(reinterpret_cast<const uint16_t*>(src)[k]);
  return int(reinterpret_cast<const uint8_t*>(src)[k]);
}

// One thread per column, kStrip rows per workgroup (two halo rows above).
// The column's horizontal second difference h(i) = c(i,j) - 2 c(i,j-1) +
// c(i,j-2) takes the two left neighbours from the lanes to the left (the
// first two lanes of a wavefront load theirs); then D = h(i) - 2 h(i-1) + h(i-2).
__global__ __launch_bounds__(kThreads) void wb_diff2_kernel(const char* __restrict__ src, int dtype, int64_t rows,
                                                            int64_t cols, int64_t* __restrict__ index,
                                                            int32_t* __restrict__ value, int64_t capacity,
                                                            unsigned long long* __restrict__ count) {
  const int lane = threadIdx.x & 63;
  for (int64_t jb = int64_t(blockIdx.x) * kThreads; jb < cols; jb += int64_t(gridDim.x) * kThreads) {
  const int64_t j = jb + threadIdx.x;
  const bool col = j < cols;
  for (int64_t i0 = int64_t(blockIdx.y) * kStrip; i0 < rows; i0 += int64_t(gridDim.y) * kStrip) {
  const int64_t i1 = i0 + kStrip < rows ? i0 + kStrip : rows;
  int h1 = 0, h2 = 0;  // h(i-1), h(i-2)
  for (int64_t i = (i0 >= 2 ? i0 - 2 : 0); i < i1; ++i) {
    const int64_t rowbase = i * cols;
    const int c0 = col ? load_chunk(src, dtype, rowbase + j) : 0;
    int c1 = __shfl_up(c0, 1, 64), c2 = __shfl_up(c0, 2, 64);
    if (lane == 0) c1 = (col && j >= 1) ? load_chunk(src, dtype, rowbase + j - 1) : 0;
    if (lane <= 1) c2 = (col && j >= 2) ? load_chunk(src, dtype, rowbase + j - 2) : 0;
    if (j < 1) c1 = 0;
    if (j < 2) c2 = 0;
    const int h = c0 - 2 * c1 + c2;
    const int d = h - 2 * h1 + h2;
    h2 = h1;
    h1 = h;
    const bool emit = col && i >= i0 && d != 0;
    const unsigned long long m = __ballot(emit);
    if (m == 0) continue;
    unsigned long long base = 0;
    const int leader = __ffsll(static_cast<long long>(m)) - 1;
    if (lane == leader) base = atomicAdd(count, static_cast<unsigned long long>(__popcll(m)));
    base = __shfl(base, leader, 64);
    if (emit) {
      const unsigned long long below = lane ? (m & ((1ull << lane) - 1)) : 0ull;
      const int64_t slot = int64_t(base) + __popcll(below);
      if (slot < capacity) {
        index[slot] = rowbase + j;
        value[slot] = d;
      }
    }
  }
  }
  }
}

// Append the lanes' non-zero entries of one candidate position: one ballot,
// one atomic add per wavefront.
__device__ __forceinline__ void emit_entries(bool emit, int64_t pos, int d, int lane, int64_t* __restrict__ index,
                                             int32_t* __restrict__ value, int64_t capacity,
                                             unsigned long long* __restrict__ count) {
  const unsigned long long m = __ballot(emit);
  if (m == 0) return;
  unsigned long long base = 0;
  const int leader = __ffsll(static_cast<long long>(m)) - 1;
  if (lane == leader) base = atomicAdd(count, static_cast<unsigned long long>(__popcll(m)));
  base = __shfl(base, leader, 64);
  if (emit) {
    const unsigned long long below = lane ? (m & ((1ull << lane) - 1)) : 0ull;
    const int64_t slot = int64_t(base) + __popcll(below);
    if (slot < capacity) {
      index[slot] = pos;
      value[slot] = d;
    }
  }
}

constexpr int kVecStrip = 32;  // rows per workgroup in the vector stencil
constexpr int kUnroll = 4;     // row vectors in flight per lane

// V columns per lane from one 16-byte load (8 bf16 or 4 fp32 values), rows
// loaded kUnroll at a time. The two columns left of a lane's vector are the
// previous lane's last two (the first lane of each wavefront loads them). Same
// arithmetic as wb_diff2_kernel; needs cols % V == 0 and a 16-byte aligned src.
template <int V>
__global__ __launch_bounds__(kThreads) void wb_diff2_vec_kernel(const char* __restrict__ src, int64_t rows,
                                                                int64_t cols, int64_t* __restrict__ index,
                                                                int32_t* __restrict__ value, int64_t capacity,
                                                                unsigned long long* __restrict__ count) {
  const int lane = threadIdx.x & 63;
  const int64_t nvec = cols / V;
  for (int64_t vb = int64_t(blockIdx.x) * kThreads; vb < nvec; vb += int64_t(gridDim.x) * kThreads) {
    const int64_t v = vb + threadIdx.x;
    const bool live = v < nvec;
    const int64_t j0 = v * V;
    for (int64_t i0 = int64_t(blockIdx.y) * kVecStrip; i0 < rows; i0 += int64_t(gridDim.y) * kVecStrip) {
      const int64_t i1 = i0 + kVecStrip < rows ? i0 + kVecStrip : rows;
      int h1[V], h2[V];
#pragma unroll
      for (int k = 0; k < V; ++k) h1[k] = h2[k] = 0;
      for (int64_t ib = (i0 >= 2 ? i0 - 2 : 0); ib < i1; ib += kUnroll) {
        int x[kUnroll][V];
        int l1[kUnroll], l2[kUnroll];  // columns j0 - 1 and j0 - 2 of the first lane
#pragma unroll
        for (int u = 0; u < kUnroll; ++u) {
          const int64_t i = ib + u;
          l1[u] = l2[u] = 0;
          if (live && i < i1) {
            const char* row = src + i * cols * (16 / V);
            const uint4 q = *reinterpret_cast<const uint4*>(row + j0 * (16 / V));
            if (V == 8) {
              const uint32_t w[4] = {q.x, q.y, q.z, q.w};
#pragma unroll
              for (int k = 0; k < 4; ++k) {
                x[u][2 * k] = int(w[k] & 0xFFFFu);
                x[u][2 * k + 1] = int(w[k] >> 16);
              }
            } else {
              x[u][0] = int(__uint_as_float(q.x));
              x[u][1] = int(__uint_as_float(q.y));
              x[u][2] = int(__uint_as_float(q.z));
              x[u][3] = int(__uint_as_float(q.w));
            }
            if (lane == 0 && j0 >= 2) {
              if (V == 8) {
                const uint32_t pw = *reinterpret_cast<const uint32_t*>(row + (j0 - 2) * 2);
                l2[u] = int(pw & 0xFFFFu);
                l1[u] = int(pw >> 16);
              } else {
                const uint2 pw = *reinterpret_cast<const uint2*>(row + (j0 - 2) * 4);
                l2[u] = int(__uint_as_float(pw.x));
                l1[u] = int(__uint_as_float(pw.y));
              }
            }
          } else {
#pragma unroll
            for (int k = 0; k < V; ++k) x[u][k] = 0;
          }
        }
#pragma unroll
        for (int u = 0; u < kUnroll; ++u) {
          const int64_t i = ib + u;
          if (i >= i1) break;  // uniform: every lane of the workgroup has the same rows
          int p1 = __shfl_up(x[u][V - 1], 1, 64), p2 = __shfl_up(x[u][V - 2], 1, 64);
          if (lane == 0) {
            p1 = l1[u];
            p2 = l2[u];
          }
          int h[V];
          h[0] = x[u][0] - 2 * p1 + p2;
          h[1] = x[u][1] - 2 * x[u][0] + p1;
#pragma unroll
          for (int k = 2; k < V; ++k) h[k] = x[u][k] - 2 * x[u][k - 1] + x[u][k - 2];
          int d[V];
          unsigned any = 0;
#pragma unroll
          for (int k = 0; k < V; ++k) {
            d[k] = h[k] - 2 * h1[k] + h2[k];
            h2[k] = h1[k];
            h1[k] = h[k];
            any |= (live && i >= i0 && d[k] != 0) ? (1u << k) : 0u;
          }
          if (__ballot(any != 0) == 0) continue;
#pragma unroll
          for (int k = 0; k < V; ++k)
            emit_entries((any >> k) & 1u, i * cols + j0 + k, d[k], lane, index, value, capacity, count);
        }
      }
    }
  }
}

constexpr int kFlatUnroll = 8;  // vectors in flight per lane along a one-row field

// One-row fields (flat buffers): with nothing above, D is the row's second
// difference h. Each workgroup takes kFlatUnroll consecutive tiles of
// kThreads vectors; lane l of tile u holds vector (tile start + l).
template <int V>
__global__ __launch_bounds__(kThreads) void wb_diff2_flat_kernel(const char* __restrict__ src, int64_t cols,
                                                                 int64_t* __restrict__ index,
                                                                 int32_t* __restrict__ value, int64_t capacity,
                                                                 unsigned long long* __restrict__ count) {
  const int lane = threadIdx.x & 63;
  const int64_t nvec = cols / V;
  const int64_t step = int64_t(gridDim.x) * kThreads * kFlatUnroll;
  for (int64_t cb = int64_t(blockIdx.x) * kThreads * kFlatUnroll; cb < nvec; cb += step) {
    int x[kFlatUnroll][V];
    int l1[kFlatUnroll], l2[kFlatUnroll];
#pragma unroll
    for (int u = 0; u < kFlatUnroll; ++u) {
      const int64_t v = cb + int64_t(u) * kThreads + threadIdx.x;
      const int64_t j0 = v * V;
      l1[u] = l2[u] = 0;
      if (v < nvec) {
        const uint4 q = *reinterpret_cast<const uint4*>(src + j0 * (16 / V));
        if (V == 8) {
          const uint32_t w[4] = {q.x, q.y, q.z, q.w};
#pragma unroll
          for (int k = 0; k < 4; ++k) {
            x[u][2 * k] = int(w[k] & 0xFFFFu);
            x[u][2 * k + 1] = int(w[k] >> 16);
          }
        } else {
          x[u][0] = int(__uint_as_float(q.x));
          x[u][1] = int(__uint_as_float(q.y));
          x[u][2] = int(__uint_as_float(q.z));
          x[u][3] = int(__uint_as_float(q.w));
        }
        if (lane == 0 && j0 >= 2) {
          if (V == 8) {
            const uint32_t pw = *reinterpret_cast<const uint32_t*>(src + (j0 - 2) * 2);
            l2[u] = int(pw & 0xFFFFu);
            l1[u] = int(pw >> 16);
          } else {
            const uint2 pw = *reinterpret_cast<const uint2*>(src + (j0 - 2) * 4);
            l2[u] = int(__uint_as_float(pw.x));
            l1[u] = int(__uint_as_float(pw.y));
          }
        }
      } else {
#pragma unroll
        for (int k = 0; k < V; ++k) x[u][k] = 0;
      }
    }
#pragma unroll
    for (int u = 0; u < kFlatUnroll; ++u) {
      const int64_t v = cb + int64_t(u) * kThreads + threadIdx.x;
      if (cb + int64_t(u) * kThreads >= nvec) break;  // uniform over the workgroup
      int p1 = __shfl_up(x[u][V - 1], 1, 64), p2 = __shfl_up(x[u][V - 2], 1, 64);
      if (lane == 0) {
        p1 = l1[u];
        p2 = l2[u];
      }
      int d[V];
      d[0] = x[u][0] - 2 * p1 + p2;
      d[1] = x[u][1] - 2 * x[u][0] + p1;
#pragma unroll
      for (int k = 2; k < V; ++k) d[k] = x[u][k] - 2 * x[u][k - 1] + x[u][k - 2];
      unsigned any = 0;
#pragma unroll
      for (int k = 0; k < V; ++k) any |= (v < nvec && d[k] != 0) ? (1u << k) : 0u;
      if (__ballot(any != 0) == 0) continue;
#pragma unroll
      for (int k = 0; k < V; ++k) emit_entries((any >> k) & 1u, v * V + k, d[k], lane, index, value, capacity, count);
    }
  }
}

__global__ void wb_zero_count_kernel(unsigned long long* count) { *count = 0; }

}  // namespace

int launch_make_ids(void* dst, int dtype, int64_t numel, int64_t first_id, int shift, uint32_t mask, void* stream) {
  if (numel == 0) return hipSuccess;
  const int64_t want = (numel + kThreads - 1) / kThreads;
  const unsigned blocks = static_cast<unsigned>(want < 65536 ? want : 65536);
  hipLaunchKernelGGL(wb_make_ids_kernel, dim3(blocks), dim3(kThreads), 0, static_cast<hipStream_t>(stream),
                     static_cast<char*>(dst), dtype, numel, first_id, shift, mask);
  return hipGetLastError();
}

int launch_diff2(const void* src, int dtype, int64_t rows, int64_t cols, int64_t* index, int32_t* value,
                 int64_t capacity, unsigned long long* count, void* stream) {
  hipStream_t st = static_cast<hipStream_t>(stream);
  hipLaunchKernelGGL(wb_zero_count_kernel, dim3(1), dim3(1), 0, st, count);
  if (rows == 0 || cols == 0) return hipGetLastError();
  const int es = dtype == WB_F32 ? 4 : 2;
  const int V = 16 / es;
  if (rows == 1 && cols % V == 0 && reinterpret_cast<uintptr_t>(src) % 16 == 0) {
    const int64_t chunks = (cols / V + kThreads * kFlatUnroll - 1) / (kThreads * kFlatUnroll);
    const dim3 grid(static_cast<unsigned>(chunks < 65536 ? chunks : 65536));
    if (V == 8)
      hipLaunchKernelGGL(wb_diff2_flat_kernel<8>, grid, dim3(kThreads), 0, st, static_cast<const char*>(src), cols,
                         index, value, capacity, count);
    else
      hipLaunchKernelGGL(wb_diff2_flat_kernel<4>, grid, dim3(kThreads), 0, st, static_cast<const char*>(src), cols,
                         index, value, capacity, count);
    return hipGetLastError();
  }
  if (cols % V == 0 && reinterpret_cast<uintptr_t>(src) % 16 == 0) {
    const int64_t strips = (rows + kVecStrip - 1) / kVecStrip;
    const int64_t tiles = (cols / V + kThreads - 1) / kThreads;
    const int64_t ytiles = strips < 65535 ? strips : 65535;
    const int64_t xtiles = tiles < (65536 + ytiles - 1) / ytiles ? tiles : (65536 + ytiles - 1) / ytiles;
    const dim3 grid(static_cast<unsigned>(xtiles), static_cast<unsigned>(ytiles));
    if (V == 8)
      hipLaunchKernelGGL(wb_diff2_vec_kernel<8>, grid, dim3(kThreads), 0, st, static_cast<const char*>(src), rows,
                         cols, index, value, capacity, count);
    else
      hipLaunchKernelGGL(wb_diff2_vec_kernel<4>, grid, dim3(kThreads), 0, st, static_cast<const char*>(src), rows,
                         cols, index, value, capacity, count);
    return hipGetLastError();
  }
  const int64_t strips = (rows + kStrip - 1) / kStrip;
  const int64_t tiles = (cols + kThreads - 1) / kThreads;
  const int64_t ytiles = strips < 65535 ? strips : 65535;
  // about 64 K workgroups at most; each loops over further column tiles
  const int64_t xtiles = tiles < (65536 + ytiles - 1) / ytiles ? tiles : (65536 + ytiles - 1) / ytiles;
  const dim3 grid(static_cast<unsigned>(xtiles), static_cast<unsigned>(ytiles));
  hipLaunchKernelGGL(wb_diff2_kernel, grid, dim3(kThreads), 0, st, static_cast<const char*>(src), dtype, rows, cols,
                     index, value, capacity, count);
  return hipGetLastError();
}

}  // namespace wb
