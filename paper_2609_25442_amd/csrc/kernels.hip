// gfx950 kernels of the packing and assembly steps (WeightBridge Sec. 3.2:
// a packing kernel coalesces a round's tensors into per-receiver buffers in
// checkpoint format; an assembly kernel scatters them into the inference
// tensors). Both are batched across tensors: one launch walks a flat table of
// work items, each spread over one or more workgroups.
//
//  * wb_tasks_kernel  -- copy/cast work items: 16-byte vectorised row copies,
//    fp32 -> bf16 (v_cvt_pk_bf16_f32, round to nearest even), bf16 -> fp32,
//    an element-wise fallback for unaligned or odd cases, and 64 x 64 tiles
//    transposed through LDS where a trainer stores a shard transposed. Work
//    items are spread over several one-wave workgroups: a vector kind takes
//    one per chunk of kChunkVecs vectors, each issuing all of its loads, then
//    all of its stores, and exiting (no loop, so no wait on the completion of
//    earlier stores before the next loads, which caps a looping copy well
//    below the rate of these one-shot workgroups on gfx950); a transpose
//    takes one per 64 x 64 (registers) or 32 x 32 (LDS) tile.
//  * wb_qblock_kernel -- fp8 E4M3FN blocks (<= 128 x 128): two single-piece
//    bf16 blocks per workgroup (a row of the pair is one 512-byte load span),
//    other blocks one per workgroup, gathered from their wire pieces; blocks
//    held in registers, amax by wavefront shuffles plus LDS across the four
//    waves, s = amax / 448 (IEEE division),
//    q = RN(x / s) computed with one reciprocal per block and a remainder
//    correction for bf16 sources (exact in the range that reaches E4M3;
//    checked for every bf16 input pair), IEEE division otherwise, then
//    v_cvt_pk_fp8_f32. The scale is written by thread 0.
// The work is bandwidth bound: no matrix cores are involved.
#include <hip/hip_runtime.h>

#include "wb_internal.hpp"

namespace wb {
namespace {

// Tuning knobs (build-time): whether loads / stores carry the non-temporal
// hint (every byte is touched once), and dynamic LDS reserved per copy
// workgroup (a cap on workgroups per CU). The chunk size is in wb_internal.hpp.
#ifndef WB_NT_LOAD
#define WB_NT_LOAD 1
#endif
#ifndef WB_NT_STORE
#define WB_NT_STORE 1
#endif
#ifndef WB_TASK_DYN_LDS
#define WB_TASK_DYN_LDS 0
#endif
// The fp8 block kernel reserves enough dynamic LDS to hold two workgroups per
// CU (two waves per SIMD): more resident workgroups, each gathering 128 rows
// at once, were slower (measured) and the cap leaves the kernel the registers
// of every block class without costing occupancy.
#ifndef WB_QBLOCK_DYN_LDS
#define WB_QBLOCK_DYN_LDS 65536
#endif

constexpr int kThreads = kChunkThreads;

template <class T>
__device__ __forceinline__ T ld(const T* p) {
#if WB_NT_LOAD
  return __builtin_nontemporal_load(p);
#else
  return *p;
#endif
}
template <class T>
__device__ __forceinline__ void st(T v, T* p) {
#if WB_NT_STORE
  __builtin_nontemporal_store(v, p);
#else
  *p = v;
#endif
}

typedef float f32x2 __attribute__((ext_vector_type(2)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));

__device__ __forceinline__ uint32_t pack_bf16x2(float a, float b) {
  const bf16x2 h = __builtin_convertvector(f32x2{a, b}, bf16x2);
  return __builtin_bit_cast(uint32_t, h);
}

__device__ __forceinline__ u32x4 cvt8_f32_bf16(const f32x4& a, const f32x4& b) {
  return u32x4{pack_bf16x2(a.x, a.y), pack_bf16x2(a.z, a.w), pack_bf16x2(b.x, b.y), pack_bf16x2(b.z, b.w)};
}

__device__ __forceinline__ float bf16_lo(uint32_t w) { return __uint_as_float(w << 16); }
__device__ __forceinline__ float bf16_hi(uint32_t w) { return __uint_as_float(w & 0xFFFF0000u); }

// Walks the flattened (row, vector) index space of a rows x vpr block with
// stride kThreads, keeping row and column incrementally (one division per task).
struct Walker {
  uint32_t r, c, dr, dc, vpr;
  __device__ Walker(uint32_t start, uint32_t vpr_) : vpr(vpr_) {
    r = start / vpr;
    c = start % vpr;
    dr = kThreads / vpr;
    dc = kThreads % vpr;
  }
  __device__ __forceinline__ void step() {
    c += dc;
    r += dr;
    if (c >= vpr) {
      c -= vpr;
      ++r;
    }
  }
};

// Units [q0, q1) of a rows x vpr block in row-major order: lane l takes
// q0 + l + k * kThreads for k < N; on[k] says whether that unit exists.
template <int N = kChunkPerLane>
struct ChunkWalk {
  uint32_t r[N], c[N];
  bool on[N];
  __device__ ChunkWalk(uint32_t q0, uint32_t q1, uint32_t vpr) {
    Walker w(q0 + threadIdx.x, vpr);
#pragma unroll
    for (int k = 0; k < N; ++k) {
      on[k] = q0 + threadIdx.x + k * kThreads < q1;
      r[k] = w.r;
      c[k] = w.c;
      w.step();
    }
  }
};

// 16-byte row copy of one chunk; cols, strides and offsets in bytes.
__device__ void run_copy16(const Task& t, const char* src, char* dst, uint32_t q0) {
  const uint32_t vpr = t.cols >> 4;
  const uint32_t total = t.rows * vpr;
  if (q0 >= total) return;
  const uint32_t q1 = min(total, q0 + uint32_t(kChunkVecs));
  u32x4 v[kChunkPerLane];
  if (t.rows == 1) {
    const u32x4* s = reinterpret_cast<const u32x4*>(src) + q0 + threadIdx.x;
    u32x4* d = reinterpret_cast<u32x4*>(dst) + q0 + threadIdx.x;
    const uint32_t m = q1 - q0;
#pragma unroll
    for (int k = 0; k < kChunkPerLane; ++k)
      if (threadIdx.x + k * kThreads < m) v[k] = ld(s + k * kThreads);
#pragma unroll
    for (int k = 0; k < kChunkPerLane; ++k)
      if (threadIdx.x + k * kThreads < m) st(v[k], d + k * kThreads);
    return;
  }
  const ChunkWalk<> w(q0, q1, vpr);
#pragma unroll
  for (int k = 0; k < kChunkPerLane; ++k)
    if (w.on[k]) v[k] = ld(reinterpret_cast<const u32x4*>(src + uint64_t(w.r[k]) * t.src_ld) + w.c[k]);
#pragma unroll
  for (int k = 0; k < kChunkPerLane; ++k)
    if (w.on[k]) st(v[k], reinterpret_cast<u32x4*>(dst + uint64_t(w.r[k]) * t.dst_ld) + w.c[k]);
}

// fp32 -> bf16 of one chunk of 2 kThreads units of 4 elements (chunk c starts
// at unit 2 c kThreads): lane l converts units l and l + kThreads, so each load
// instruction of the wave reads 64 consecutive 16-byte vectors of a row; two
// 8-byte stores. Strides in elements.
__device__ void run_f32_bf16(const Task& t, const char* src, char* dst, uint32_t chunk) {
  const uint32_t vpr = t.cols >> 2;
  const uint32_t total = t.rows * vpr;
  const uint32_t q0 = chunk * 2 * uint32_t(kThreads);
  if (q0 >= total) return;
  const uint32_t q1 = min(total, q0 + 2 * uint32_t(kThreads));
  f32x4 a[2];
  if (t.rows == 1) {  // one run: unit q is input vector q and output half q
    const f32x4* s = reinterpret_cast<const f32x4*>(src) + q0 + threadIdx.x;
    u32x2* d = reinterpret_cast<u32x2*>(dst) + q0 + threadIdx.x;
#pragma unroll
    for (int k = 0; k < 2; ++k)
      if (q0 + threadIdx.x + k * kThreads < q1) a[k] = ld(s + k * kThreads);
#pragma unroll
    for (int k = 0; k < 2; ++k)
      if (q0 + threadIdx.x + k * kThreads < q1)
        st(u32x2{pack_bf16x2(a[k].x, a[k].y), pack_bf16x2(a[k].z, a[k].w)}, d + k * kThreads);
    return;
  }
  const ChunkWalk<2> w(q0, q1, vpr);
#pragma unroll
  for (int k = 0; k < 2; ++k)
    if (w.on[k])
      a[k] = ld(reinterpret_cast<const f32x4*>(src + (uint64_t(w.r[k]) * t.src_ld + uint64_t(w.c[k]) * 4) * 4));
#pragma unroll
  for (int k = 0; k < 2; ++k)
    if (w.on[k])
      st(u32x2{pack_bf16x2(a[k].x, a[k].y), pack_bf16x2(a[k].z, a[k].w)},
         reinterpret_cast<u32x2*>(dst + (uint64_t(w.r[k]) * t.dst_ld + uint64_t(w.c[k]) * 4) * 2));
}

// bf16 -> fp32 of one chunk of input vectors (8 elements each); strides in
// elements.
__device__ void run_bf16_f32(const Task& t, const char* src, char* dst, uint32_t q0) {
  const uint32_t vpr = t.cols >> 3;
  const uint32_t total = t.rows * vpr;
  if (q0 >= total) return;
  const uint32_t q1 = min(total, q0 + uint32_t(kChunkVecs));
  u32x4 v[kChunkPerLane];
  if (t.rows == 1) {  // one run: input vector q becomes output vectors 2q and 2q + 1
    const u32x4* s = reinterpret_cast<const u32x4*>(src) + q0 + threadIdx.x;
    f32x4* d = reinterpret_cast<f32x4*>(dst) + 2 * (q0 + threadIdx.x);
#pragma unroll
    for (int k = 0; k < kChunkPerLane; ++k)
      if (q0 + threadIdx.x + k * kThreads < q1) v[k] = ld(s + k * kThreads);
#pragma unroll
    for (int k = 0; k < kChunkPerLane; ++k)
      if (q0 + threadIdx.x + k * kThreads < q1) {
        const u32x4 x = v[k];
        st(f32x4{bf16_lo(x.x), bf16_hi(x.x), bf16_lo(x.y), bf16_hi(x.y)}, d + 2 * k * kThreads);
        st(f32x4{bf16_lo(x.z), bf16_hi(x.z), bf16_lo(x.w), bf16_hi(x.w)}, d + 2 * k * kThreads + 1);
      }
    return;
  }
  const ChunkWalk<> w(q0, q1, vpr);
#pragma unroll
  for (int k = 0; k < kChunkPerLane; ++k)
    if (w.on[k])
      v[k] = ld(reinterpret_cast<const u32x4*>(src + (uint64_t(w.r[k]) * t.src_ld + uint64_t(w.c[k]) * 8) * 2));
#pragma unroll
  for (int k = 0; k < kChunkPerLane; ++k)
    if (w.on[k]) {
      const u32x4 x = v[k];
      f32x4* dp = reinterpret_cast<f32x4*>(dst + (uint64_t(w.r[k]) * t.dst_ld + uint64_t(w.c[k]) * 8) * 4);
      st(f32x4{bf16_lo(x.x), bf16_hi(x.x), bf16_lo(x.y), bf16_hi(x.y)}, dp);
      st(f32x4{bf16_lo(x.z), bf16_hi(x.z), bf16_lo(x.w), bf16_hi(x.w)}, dp + 1);
    }
}

// Raw bits of one element, widened to 32 bits.
__device__ __forceinline__ uint32_t load_bits(const char* p, int dt) {
  if (dt == WB_F32) return *reinterpret_cast<const uint32_t*>(p);
  if (dt == WB_BF16) return *reinterpret_cast<const uint16_t*>(p);
  return *reinterpret_cast<const uint8_t*>(p);
}

__device__ __forceinline__ void store_converted(char* p, uint32_t bits, int sdt, int ddt) {
  if (ddt == WB_F32) {
    *reinterpret_cast<uint32_t*>(p) = sdt == WB_BF16 ? bits << 16 : bits;
  } else if (ddt == WB_BF16) {
    const uint32_t w = sdt == WB_F32 ? pack_bf16x2(__uint_as_float(bits), 0.0f) : bits;
    *reinterpret_cast<uint16_t*>(p) = static_cast<uint16_t>(w);
  } else {
    *reinterpret_cast<uint8_t*>(p) = static_cast<uint8_t>(bits);
  }
}

__device__ __forceinline__ int dt_bytes(int dt) { return dt == WB_F32 ? 4 : (dt == WB_BF16 ? 2 : 1); }

// Element by element; strides in elements.
__device__ void run_scalar(const Task& t, const char* src, char* dst) {
  const int ss = dt_bytes(t.sdt), ds = dt_bytes(t.ddt);
  const uint64_t total = uint64_t(t.rows) * t.cols;
  Walker w(threadIdx.x, t.cols);
  for (uint64_t q = threadIdx.x; q < total; q += kThreads) {
    const uint32_t bits = load_bits(src + (uint64_t(w.r) * t.src_ld + w.c) * ss, t.sdt);
    store_converted(dst + (uint64_t(w.r) * t.dst_ld + w.c) * ds, bits, t.sdt, t.ddt);
    w.step();
  }
}

// dst[c][r] = cvt(src[r][c]) for quarter `part` (32 x 32) of a tile of up to
// 64 x 64, through LDS (padded rows: conflict-free column reads).
__device__ void run_transpose(const Task& t, const char* src, char* dst, uint32_t part) {
  __shared__ uint32_t tile[32][33];
  const uint32_t r0 = (part >> 1) * 32, c0 = (part & 1) * 32;
  if (r0 >= t.rows || c0 >= t.cols) return;  // uniform over the workgroup
  const int ss = dt_bytes(t.sdt), ds = dt_bytes(t.ddt);
  const uint32_t R = min(32u, t.rows - r0), C = min(32u, t.cols - c0);
  src += (uint64_t(r0) * t.src_ld + c0) * ss;
  dst += (uint64_t(c0) * t.dst_ld + r0) * ds;
  for (uint32_t i = threadIdx.x; i < 32 * 32; i += kThreads) {
    const uint32_t r = i >> 5, c = i & 31;
    if (r < R && c < C) tile[r][c] = load_bits(src + (uint64_t(r) * t.src_ld + c) * ss, t.sdt);
  }
  __syncthreads();
  for (uint32_t i = threadIdx.x; i < 32 * 32; i += kThreads) {
    const uint32_t c = i >> 5, r = i & 31;
    if (r < R && c < C) store_converted(dst + (uint64_t(c) * t.dst_ld + r) * ds, tile[r][c], t.sdt, t.ddt);
  }
}

// Column j of an 8 x 8 block of 2-byte elements held as eight 16-byte rows.
__device__ __forceinline__ u32x4 column8(const u32x4 (&a)[8], int j) {
  uint32_t o[4];
#pragma unroll
  for (int k = 0; k < 4; ++k) {
    const uint32_t x = a[2 * k][j >> 1], y = a[2 * k + 1][j >> 1];
    o[k] = (j & 1) ? ((x >> 16) | (y & 0xFFFF0000u)) : ((x & 0xFFFFu) | (y << 16));
  }
  return u32x4{o[0], o[1], o[2], o[3]};
}

// dst[c][r] = src[r][c] for 2-byte elements, (64..256) rows x 64 columns: each
// wave takes one 64 x 64 tile (tile `w` of the item, counted down the rows),
// each lane an 8 x 8 sub-tile that it loads as eight 16-byte rows, transposes
// in registers and stores as eight 16-byte rows. Lanes 8i..8i+7 cover one
// 128-byte span of a row on both sides.
__device__ void run_transpose16(const Task& t, const char* src, char* dst, uint32_t w) {
  const uint32_t l = threadIdx.x & 63;
  if (w * 64 >= t.rows) return;
  const uint32_t c0 = 8 * (l & 7), r0 = w * 64 + 8 * (l >> 3);
  u32x4 a[8];
#pragma unroll
  for (int i = 0; i < 8; ++i)
    a[i] = ld(reinterpret_cast<const u32x4*>(src + (uint64_t(r0 + i) * t.src_ld + c0) * 2));
#pragma unroll
  for (int j = 0; j < 8; ++j) st(column8(a, j), reinterpret_cast<u32x4*>(dst + (uint64_t(c0 + j) * t.dst_ld + r0) * 2));
}

}  // namespace

__device__ __forceinline__ const char* base_of(uint16_t idx, const uint64_t* ptrs, const char* buf, const char* aux) {
  return idx == 0 ? buf : idx == kAuxBuffer ? aux : reinterpret_cast<const char*>(ptrs[idx]);
}

// XCD-aware order of a launch's work. The hardware hands workgroup b to XCD
// b mod 8 (round-robin over the 8 XCDs), and over a long launch the XCDs drift
// apart, so neighbouring work units (the same DRAM pages; for fp8 blocks, the
// same 128 rows of a wire payload) end up in flight at different times on
// different XCDs. Renumbered so that in each run of 8 C workgroups XCD x takes
// C consecutive units, neighbours are in flight together on one XCD, while the
// eight XCDs still work within one run (so every HBM channel stays busy). A
// bijection of [0, total); a tail shorter than 8 C keeps the plain order.
constexpr uint64_t kXcds = 8;
constexpr uint64_t kXcdRunCopy = 1024;  // copy/cast chunks (1-2 KiB of source each)
constexpr uint64_t kXcdRunPairs = 512;  // fp8 block pairs (64 KiB of wire each)
__device__ __forceinline__ uint64_t xcd_order(uint64_t b, uint64_t total, uint64_t C) {
  const uint64_t run = kXcds * C, base = b / run * run;
  if (base + run > total) return b;
  const uint64_t k = b - base;
  return base + (k % kXcds) * C + k / kXcds;
}

// Workgroups are laid out class by class: item i of class 0 takes workgroups
// [i, i + 1) * 2^s0, chunk = b mod 2^s0 (b in XCD-aware order); then class 1
// the same with s1; then one workgroup per class-2 item. A grid wider than
// kMaxGridX workgroups is folded into rows of gridDim.x.
__global__ __launch_bounds__(kThreads) void wb_tasks_kernel(const Task* __restrict__ tasks,
                                                            const uint64_t* __restrict__ ptrs, const char* buf,
                                                            const char* aux, uint32_t ntasks, uint32_t n0,
                                                            uint32_t n1, uint32_t s0, uint32_t s1) {
  uint64_t b = uint64_t(blockIdx.y) * gridDim.x + blockIdx.x;
  const uint64_t w0 = uint64_t(n0) << s0, w1 = uint64_t(n1) << s1;
  uint64_t ti;
  uint32_t chunk = 0;
  if (b < w0) {
    b = xcd_order(b, w0, kXcdRunCopy);
    ti = b >> s0;
    chunk = uint32_t(b) & ((1u << s0) - 1u);
  } else if ((b -= w0) < w1) {
    ti = n0 + (b >> s1);
    chunk = uint32_t(b) & ((1u << s1) - 1u);
  } else {
    ti = uint64_t(n0) + n1 + (b - w1);
  }
  if (ti >= ntasks) return;
  const Task t = tasks[ti];
  const char* src = base_of(t.src_idx, ptrs, buf, aux) + t.src_off;
  char* dst = const_cast<char*>(base_of(t.dst_idx, ptrs, buf, aux)) + t.dst_off;
  const uint32_t q0 = chunk * uint32_t(kChunkVecs);
  switch (t.kind) {
    case TASK_COPY16: run_copy16(t, src, dst, q0); break;
    case TASK_F32_BF16: run_f32_bf16(t, src, dst, chunk); break;
    case TASK_BF16_F32: run_bf16_f32(t, src, dst, q0); break;
    case TASK_SCALAR: if (chunk == 0) run_scalar(t, src, dst); break;
    case TASK_TRANSPOSE: run_transpose(t, src, dst, chunk); break;
    case TASK_TRANSPOSE16: run_transpose16(t, src, dst, chunk * (kThreads / 64) + (threadIdx.x >> 6)); break;
    default: break;
  }
}

// dst[c][r] = src[r][c] of one kTileRows x kTileCols tile of 2-byte elements
// per workgroup (TASK_TILE items): thread t transposes the 8 x 8 sub-tile at
// source rows 8 (t / 64) .., columns 8 (t mod 64) .. in registers (a wave
// instruction reads 1 KiB of one source row), LDS regroups the sub-tiles by
// destination row, and each thread then stores eight 16-byte pieces of
// destination rows (a wave instruction writes four whole 256-byte rows). The
// 16-byte words of destination row r sit in LDS at word w ^ ((r / 8) mod 16):
// the sub-tiles of one wave land in 16 different bank groups, and a row read
// back is a permutation of its own words.
__global__ __launch_bounds__(kTileThreads) void wb_tile_kernel(const Task* __restrict__ tasks,
                                                               const uint64_t* __restrict__ ptrs, const char* buf,
                                                               const char* aux) {
  constexpr int GR = kTileRows / 8, GC = kTileCols / 8;  // 16-byte words per destination / source row
  __shared__ u32x4 lds[kTileCols][GR];
  const Task t = tasks[blockIdx.x];
  const char* src = base_of(t.src_idx, ptrs, buf, aux) + t.src_off;
  char* dst = const_cast<char*>(base_of(t.dst_idx, ptrs, buf, aux)) + t.dst_off;
  const int cg = threadIdx.x % GC, rg = threadIdx.x / GC;
  u32x4 a[8];
#pragma unroll
  for (int i = 0; i < 8; ++i)
    a[i] = ld(reinterpret_cast<const u32x4*>(src + (uint64_t(8 * rg + i) * t.src_ld + 8 * cg) * 2));
#pragma unroll
  for (int j = 0; j < 8; ++j) {
    const int row = 8 * cg + j;  // destination row
    lds[row][rg ^ ((row >> 3) & (GR - 1))] = column8(a, j);
  }
  __syncthreads();
  const int w = threadIdx.x % GR, r0 = threadIdx.x / GR;
#pragma unroll
  for (int k = 0; k < 8; ++k) {
    const int row = r0 + (kTileThreads / GR) * k;
    st(lds[row][w ^ ((row >> 3) & (GR - 1))], reinterpret_cast<u32x4*>(dst + (uint64_t(row) * t.dst_ld + 8 * w) * 2));
  }
}

// ---- fp8 E4M3FN blocks ---------------------------------------------------

namespace {

__device__ __forceinline__ float load_f32(const char* p, int dt) {
  return dt == WB_F32 ? *reinterpret_cast<const float*>(p) : __uint_as_float(uint32_t(*reinterpret_cast<const uint16_t*>(p)) << 16);
}

// Element (r, c) of the block from its pieces (the block is exactly covered).
__device__ __forceinline__ float gather_one(const QPiece* pcs, int n, const char* recv, int r, int c) {
  for (int i = 0; i < n; ++i) {
    const QPiece& p = pcs[i];
    if (r >= p.r0 && r <= p.r1m1 && c >= p.c0 && c <= p.c1m1) {
      const int es = p.sdt == WB_F32 ? 4 : 2;
      return load_f32(recv + p.src_off + (uint64_t(r - p.r0) * p.src_ld + (c - p.c0)) * es, p.sdt);
    }
  }
  return 0.0f;
}

__device__ __forceinline__ void unpack8(const u32x4 x, float* v) {
  v[0] = bf16_lo(x.x); v[1] = bf16_hi(x.x); v[2] = bf16_lo(x.y); v[3] = bf16_hi(x.y);
  v[4] = bf16_lo(x.z); v[5] = bf16_hi(x.z); v[6] = bf16_lo(x.w); v[7] = bf16_hi(x.w);
}

constexpr int kLdsPieces = 128;

// The block's scale s = amax / 448 (IEEE division; 1 for an all-zero block)
// and the quantities RN(x / s) is computed from, s = m 2^E (m in [1, 2)):
//
// mode 2 (bf16 source, -90 <= E <= 100): r = RN(1 / s), q0 = RN(x r),
//   e = x - q0 s (exact, by FMA), q = RN(q0 + e r). A quotient that can round
//   to a non-zero E4M3 value has |x / s| >= 2^-10, so q0 >= 2^-10, e is at
//   least 2^(E - 33) in magnitude and every intermediate is a normal number;
//   r stays normal for E <= 100.
// mode 1 (bf16 source, any other normal s): the same on x' = x 2^-E and m,
//   which keeps the intermediates normal whatever E.
// In both the sign is copied from x: a quotient that rounds to zero can lose
//   it in the correction. Since |x| <= amax, |q| <= 448.00003 rounds to at most
//   448 in E4M3, so no clamp is needed. Both are verified exhaustively for
//   every bf16 (x, amax) pair.
// mode 0 (fp32 sources, subnormal s): IEEE division, clamped to +-448 (a no-op
//   that keeps the conversion away from its overflow path whatever the source).
struct QScale {
  float s, sp, rp, pw;
  int mode;
};

__device__ __forceinline__ QScale make_scale(float amax, bool bf16_source) {
  QScale q;
  q.s = amax > 0.0f ? amax / 448.0f : 1.0f;  // IEEE fp32 division
  const uint32_t sbits = __float_as_uint(q.s);
  const int sexp = int((sbits >> 23) & 0xFF);  // E + 127
  q.mode = (!bf16_source || sexp == 0) ? 0 : (sexp >= 127 - 90 && sexp <= 127 + 100) ? 2 : 1;
  q.pw = __uint_as_float(uint32_t(254 - sexp) << 23);  // 2^-E
  q.sp = q.mode == 1 ? __uint_as_float((sbits & 0x007FFFFFu) | 0x3F800000u) : q.s;  // m, or s
  q.rp = 1.0f / q.sp;
  return q;
}

template <int kMode>
__device__ __forceinline__ float quotient(float x, const QScale& q) {
  if (kMode == 0) return __builtin_amdgcn_fmed3f(x / q.s, -448.0f, 448.0f);
  const float xp = kMode == 1 ? x * q.pw : x;
  const float q0 = xp * q.rp;
  const float e = fmaf(-q0, q.sp, xp);
  return __builtin_copysignf(fmaf(e, q.rp, q0), x);
}

// E4M3FN(RN(x / s)) of this thread's R rows of 8 columns (rows rb + kStep k),
// row k's values produced by row(k, v); 8-byte stores, or bytes at a ragged
// right edge or an unaligned destination.
template <int kMode, int R, int kStep, class Row>
__device__ __forceinline__ void quantise_store(Row row, const QScale& qs, int rows, int cols, int rb, int cg,
                                               uint8_t* q8, uint32_t dst_ld, bool vec) {
#pragma unroll
  for (int k = 0; k < R; ++k) {
    const int r = rb + kStep * k;
    if (r >= rows || cg >= cols) continue;
    float v[8], q[8];
    row(k, v);
#pragma unroll
    for (int m = 0; m < 8; ++m) q[m] = quotient<kMode>(v[m], qs);
    uint32_t lo = __builtin_amdgcn_cvt_pk_fp8_f32(q[0], q[1], 0, false);
    lo = __builtin_amdgcn_cvt_pk_fp8_f32(q[2], q[3], lo, true);
    uint32_t hi = __builtin_amdgcn_cvt_pk_fp8_f32(q[4], q[5], 0, false);
    hi = __builtin_amdgcn_cvt_pk_fp8_f32(q[6], q[7], hi, true);
    uint8_t* dst = q8 + uint64_t(r) * dst_ld + cg;
    if (vec && cg + 8 <= cols) {
      st(u32x2{lo, hi}, reinterpret_cast<u32x2*>(dst));
    } else {
#pragma unroll
      for (int m = 0; m < 8; ++m)
        if (cg + m < cols) dst[m] = static_cast<uint8_t>((m < 4 ? lo : hi) >> (8 * (m & 3)));
    }
  }
}

template <int R, int kStep, class Row>
__device__ __forceinline__ void quantise_block(Row row, const QScale& qs, int rows, int cols, int rb, int cg,
                                               uint8_t* q8, uint32_t dst_ld, bool vec) {
  // the mode is uniform over the block, so this branch is taken once, outside
  // the element loops
  if (qs.mode == 2)
    quantise_store<2, R, kStep>(row, qs, rows, cols, rb, cg, q8, dst_ld, vec);
  else if (qs.mode == 1)
    quantise_store<1, R, kStep>(row, qs, rows, cols, rb, cg, q8, dst_ld, vec);
  else
    quantise_store<0, R, kStep>(row, qs, rows, cols, rb, cg, q8, dst_ld, vec);
}

typedef uint16_t u16x2 __attribute__((ext_vector_type(2)));

// Takes the word by value: __builtin_bit_cast applied to a vector element
// expression (v.y) reads the vector's first element in this compiler.
__device__ __forceinline__ u16x2 as_u16x2(uint32_t w) { return __builtin_bit_cast(u16x2, w); }

// Per-lane view of one of the two blocks of a pair.
struct PairLane {
  const char* src;   // this lane's first element (row rb, column cg)
  uint64_t src_ld2;  // wire row stride in bytes
  uint8_t* q8;       // fp8 block origin
  uint32_t dst_ld;
  int rows, cols;
  bool vec;
};

// Blocks i0 and i0 + 1 (absent when i0 + 1 == nsingle), both pairable. In
// each half-wave, lanes 0..15 take block i0 and lanes 16..31 block i0 + 1, so a
// load instruction reads 512 contiguous bytes of each of two rows when the two
// blocks are neighbours on the wire; thread t holds columns 8 (t mod 16) .. + 7
// of rows t / 32 + 8 k, k < 16, as raw bf16. kFull: both blocks present,
// 128 x 128 and with 8-byte stores, so no load or store needs a predicate.
// kBands: at least one block of the pair is QB_BANDS; each row's source is
// base + r * ld2 of the band that holds it, from the lane's own block's band
// table (registers: indexed only by unrolled constants); otherwise every row
// follows the single piece's stride.
struct PairBands {
  uint64_t base[kMaxBands];   // recv + band offset - first row * pitch (bytes)
  uint32_t ld2[kMaxBands];    // band pitch in bytes
  uint32_t start[kMaxBands];  // first row; bands past the block's last: 256
};

template <bool kFull, bool kBands>
__device__ __forceinline__ void qblock_pair_run(const PairLane& L, const PairBands& S, int h, bool on,
                                                const QBlock& b0, const QBlock& b1, const uint64_t* __restrict__ ptrs) {
  constexpr int R = 16, kStep = 8;
  static_assert(kQBlockThreads == 32 * kStep, "pair mapping");
  static_assert(kMaxBands == 4, "band selection");
  __shared__ uint32_t wave_max[kQBlockThreads / 64][2];
  const int cg = (threadIdx.x & 15) * 8, rb = threadIdx.x >> 5;
  u32x4 raw[R];
  if (kBands) {
#pragma unroll
    for (int k = 0; k < R; ++k) {
      const uint32_t r = rb + kStep * k;
      raw[k] = u32x4{0u, 0u, 0u, 0u};
      if (kFull || (int(r) < L.rows && cg < L.cols)) {
        uint64_t base = S.base[0];
        uint32_t ld2 = S.ld2[0];
#pragma unroll
        for (int j = 1; j < kMaxBands; ++j)
          if (r >= S.start[j]) {
            base = S.base[j];
            ld2 = S.ld2[j];
          }
        raw[k] = ld(reinterpret_cast<const u32x4*>(base + uint64_t(r) * ld2 + uint64_t(cg) * 2));
      }
    }
  } else if (kFull) {
    const char* p = L.src;
#pragma unroll
    for (int k = 0; k < R; ++k, p += kStep * L.src_ld2) raw[k] = ld(reinterpret_cast<const u32x4*>(p));
  } else {
#pragma unroll
    for (int k = 0; k < R; ++k) {
      const int r = rb + kStep * k;
      raw[k] = u32x4{0u, 0u, 0u, 0u};
      if (r < L.rows && cg < L.cols)
        raw[k] = ld(reinterpret_cast<const u32x4*>(L.src + uint64_t(kStep * k) * L.src_ld2));
    }
  }
  // amax: finite bf16 magnitudes order as their bit patterns with the sign
  // cleared (two per word, packed 16-bit maxima)
  u16x2 acc = {0, 0};
#pragma unroll
  for (int k = 0; k < R; ++k) {
    const u32x4 a = raw[k] & 0x7FFF7FFFu;
    acc = __builtin_elementwise_max(acc, as_u16x2(a.x));
    acc = __builtin_elementwise_max(acc, as_u16x2(a.y));
    acc = __builtin_elementwise_max(acc, as_u16x2(a.z));
    acc = __builtin_elementwise_max(acc, as_u16x2(a.w));
  }
  uint32_t m = max(uint32_t(acc.x), uint32_t(acc.y));
  // lanes of one block: xor 1..8 within a 16-lane group, xor 32 across the
  // half-waves
  m = max(m, uint32_t(__shfl_xor(int(m), 1)));
  m = max(m, uint32_t(__shfl_xor(int(m), 2)));
  m = max(m, uint32_t(__shfl_xor(int(m), 4)));
  m = max(m, uint32_t(__shfl_xor(int(m), 8)));
  m = max(m, uint32_t(__shfl_xor(int(m), 32)));
  if ((threadIdx.x & 47) == 0) wave_max[threadIdx.x >> 6][h] = m;  // lanes 0 and 16
  __syncthreads();
  m = wave_max[0][h];
#pragma unroll
  for (int w = 1; w < kQBlockThreads / 64; ++w) m = max(m, wave_max[w][h]);
  const QScale qs = make_scale(__uint_as_float(m << 16), true);
  // rows and columns past the edge are skipped by the store loop; in the full
  // case there are none
  const int rows = kFull ? 128 : L.rows, cols = kFull ? 128 : L.cols;
  quantise_block<R, kStep>([&](int k, float* v) { unpack8(raw[k], v); }, qs, rows, cols, rb, cg, L.q8, L.dst_ld,
                           kFull || L.vec);
  const QBlock& b = h ? b1 : b0;
  if (on && (threadIdx.x & ~16u) == 0) reinterpret_cast<float*>(ptrs[b.scale_idx])[b.scale_off] = qs.s;
}

// This lane's view of the block it works on in a pair (h: 0 or 1).
__device__ __forceinline__ PairLane pair_lane(const QBlock& b0, const QBlock& b1, int h, bool on,
                                              const uint64_t* __restrict__ ptrs, const char* recv) {
  const QBlock& b = h ? b1 : b0;
  const int cg = (threadIdx.x & 15) * 8, rb = threadIdx.x >> 5;
  PairLane L;
  L.src_ld2 = uint64_t(b.src_ld) * 2;
  L.src = recv + b.src_off + uint64_t(cg) * 2 + uint64_t(rb) * L.src_ld2;
  L.dst_ld = b.dst_ld;
  uint8_t* const q0 = reinterpret_cast<uint8_t*>(ptrs[b0.dst_idx]) + b0.dst_off;
  uint8_t* const q1 = reinterpret_cast<uint8_t*>(ptrs[b1.dst_idx]) + b1.dst_off;
  L.q8 = h ? q1 : q0;
  L.rows = on ? b.rows_m1 + 1 : 0;
  L.cols = b.cols_m1 + 1;
  L.vec = (b.flags & QB_VEC_STORE) != 0;
  return L;
}

// Blocks i0 and i0 + 1, both QB_SINGLE, 128 x 128, 8-byte stores (the
// planner's full pairs): no predicates, one quotient form per block.
__device__ __forceinline__ void qblock_pair_full(const QBlock* __restrict__ blocks, uint32_t i0, const uint64_t* __restrict__ ptrs,
                                 const char* recv) {
  const QBlock b0 = blocks[i0];
  const QBlock b1 = blocks[i0 + 1];
  const int h = (threadIdx.x >> 4) & 1;
  qblock_pair_run<true, false>(pair_lane(b0, b1, h, true, ptrs, recv), PairBands{}, h, true, b0, b1, ptrs);
}

// Blocks i0 and i0 + 1 (absent when i0 + 1 == n), both pairable, any extent.
__device__ __forceinline__ void qblock_pair(const QBlock* __restrict__ blocks, uint32_t i0, uint32_t n,
                            const QPiece* __restrict__ pieces, const uint64_t* __restrict__ ptrs, const char* recv) {
  // both descriptors are read at workgroup-uniform addresses; each lane then
  // selects its block's fields
  const bool has1 = i0 + 1 < n;
  const QBlock b0 = blocks[i0];
  const QBlock b1 = blocks[has1 ? i0 + 1 : i0];
  const int h = (threadIdx.x >> 4) & 1;
  const bool on = h == 0 || has1;
  const PairLane L = pair_lane(b0, b1, h, on, ptrs, recv);
  const bool full = has1 && b0.rows_m1 == 127 && b0.cols_m1 == 127 && b1.rows_m1 == 127 && b1.cols_m1 == 127 &&
                    (b0.flags & b1.flags & QB_VEC_STORE);
  const bool bands = ((b0.flags | b1.flags) & QB_BANDS) != 0;  // uniform over the workgroup
  if (bands) {
    // the band table of this lane's block (its own stride when it is a
    // single piece)
    const uint32_t flags = h ? b1.flags : b0.flags;
    const uint32_t np = h ? b1.npieces : b0.npieces, p0 = h ? b1.piece0 : b0.piece0;
    PairBands S;
#pragma unroll
    for (int j = 0; j < kMaxBands; ++j) {
      S.base[j] = 0;
      S.ld2[j] = 0;
      S.start[j] = 256;
    }
    if (flags & QB_BANDS) {
#pragma unroll
      for (int j = 0; j < kMaxBands; ++j)
        if (uint32_t(j) < np) {
          const QPiece q = pieces[p0 + j];
          S.ld2[j] = q.src_ld * 2;
          S.base[j] = reinterpret_cast<uint64_t>(recv) + q.src_off - uint64_t(q.r0) * S.ld2[j];
          S.start[j] = q.r0;
        }
    } else {
      S.ld2[0] = (h ? b1.src_ld : b0.src_ld) * 2;
      S.base[0] = reinterpret_cast<uint64_t>(recv) + (h ? b1.src_off : b0.src_off);
      S.start[0] = 0;
    }
    if (full)
      qblock_pair_run<true, true>(L, S, h, on, b0, b1, ptrs);
    else
      qblock_pair_run<false, true>(L, S, h, on, b0, b1, ptrs);
  } else if (full) {
    qblock_pair_run<true, false>(L, PairBands{}, h, on, b0, b1, ptrs);
  } else {
    qblock_pair_run<false, false>(L, PairBands{}, h, on, b0, b1, ptrs);
  }
}

// One block of any kind (several wire pieces, unaligned or fp32 ones): thread t
// holds columns 8 (t mod 16) .. + 7 of rows t / 16 + 16 k, k < 8, as fp32,
// gathered from the pieces.
__device__ __forceinline__ void qblock_one(const QBlock& b, const QPiece* __restrict__ pieces, const uint64_t* __restrict__ ptrs,
                           const char* recv) {
  constexpr int R = 8, kStep = 16;
  static_assert(kQBlockThreads == 16 * kStep, "block mapping");
  __shared__ float wave_max[kQBlockThreads / 64];
  __shared__ QPiece lds_pcs[kLdsPieces];
  __shared__ uint8_t row_piece[128];
  const int rows = b.rows_m1 + 1, cols = b.cols_m1 + 1;
  const int cg = (threadIdx.x & 15) * 8, rb = threadIdx.x >> 4;
  // stage the piece list in LDS with a row -> piece table for the pieces that
  // span the block's full width (row bands: the common case, a replicated
  // tensor split by rows among its senders); resolve each row chunk's source
  // first (the table, else a search of the list), then issue the loads
  const int n = b.npieces;
  const QPiece* pcs = pieces + b.piece0;
  bool table = false;
  if (n <= kLdsPieces) {
    for (int i = threadIdx.x; i < n; i += kQBlockThreads) lds_pcs[i] = pcs[i];
    for (int r = threadIdx.x; r < 128; r += kQBlockThreads) row_piece[r] = 0xFF;
    __syncthreads();
    for (int i = threadIdx.x; i < n; i += kQBlockThreads) {
      const QPiece& p = lds_pcs[i];
      if (p.c0 == 0 && p.c1m1 == cols - 1)
        for (int r = p.r0; r <= p.r1m1; ++r) row_piece[r] = static_cast<uint8_t>(i);
    }
    __syncthreads();
    pcs = lds_pcs;
    table = true;
  }
  const char* src[R];
#pragma unroll
  for (int k = 0; k < R; ++k) {
    const int r = rb + kStep * k;
    src[k] = nullptr;
    if (r >= rows || cg >= cols) continue;
    int i = table ? row_piece[r] : 0xFF;
    if (i == 0xFF)
      for (i = 0; i < n; ++i) {
        const QPiece& p = pcs[i];
        if (r >= p.r0 && r <= p.r1m1 && cg >= p.c0 && cg + 7 <= p.c1m1) break;
      }
    if (i < n) {
      const QPiece& p = pcs[i];
      const char* a = recv + p.src_off + (uint64_t(r - p.r0) * p.src_ld + (cg - p.c0)) * 2;
      if (p.sdt == WB_BF16 && cg + 7 <= p.c1m1 && (reinterpret_cast<uintptr_t>(a) & 15) == 0) src[k] = a;
    }
  }
  u32x4 raw[R];
#pragma unroll
  for (int k = 0; k < R; ++k) {
    raw[k] = u32x4{0u, 0u, 0u, 0u};
    if (src[k]) raw[k] = ld(reinterpret_cast<const u32x4*>(src[k]));
  }
  float v[R][8];
#pragma unroll
  for (int k = 0; k < R; ++k) {
    unpack8(raw[k], v[k]);
    const int r = rb + kStep * k;
    if (!src[k] && r < rows && cg < cols) {
#pragma unroll
      for (int m = 0; m < 8; ++m) v[k][m] = cg + m < cols ? gather_one(pcs, n, recv, r, cg + m) : 0.0f;
    }
  }
  float amax = 0.0f;
#pragma unroll
  for (int k = 0; k < R; ++k)
#pragma unroll
    for (int m = 0; m < 8; ++m) amax = fmaxf(amax, fabsf(v[k][m]));
  for (int off = 32; off > 0; off >>= 1) amax = fmaxf(amax, __shfl_xor(amax, off));
  if ((threadIdx.x & 63) == 0) wave_max[threadIdx.x >> 6] = amax;
  __syncthreads();
  amax = wave_max[0];
#pragma unroll
  for (int w = 1; w < kQBlockThreads / 64; ++w) amax = fmaxf(amax, wave_max[w]);
  const QScale qs = make_scale(amax, (b.flags & QB_BF16_SOURCE) != 0);
  uint8_t* q8 = reinterpret_cast<uint8_t*>(ptrs[b.dst_idx]) + b.dst_off;
  quantise_block<R, kStep>(
      [&](int k, float* out) {
#pragma unroll
        for (int m = 0; m < 8; ++m) out[m] = v[k][m];
      },
      qs, rows, cols, rb, cg, q8, b.dst_ld, (b.flags & QB_VEC_STORE) != 0);
  if (threadIdx.x == 0) reinterpret_cast<float*>(ptrs[b.scale_idx])[b.scale_off] = qs.s;
}

}  // namespace

// The fp8 blocks of a launch range come in three classes, taken by one launch
// (the slower classes overlap the bulk instead of trailing it in launches of
// their own): workgroup w < nfull / 2 takes the full pair 2v, 2v + 1, v = w in
// XCD-aware order; the next
// ones the other pairable blocks two at a time (the second absent past npair);
// the rest one block each.
__global__ __launch_bounds__(kQBlockThreads) void wb_qblock_kernel(const QBlock* __restrict__ blocks,
                                                                   const QPiece* __restrict__ pieces,
                                                                   const uint64_t* __restrict__ ptrs,
                                                                   const char* recv, uint32_t n, uint32_t nfull,
                                                                   uint32_t npair) {
  const uint32_t g0 = nfull / 2, g1 = (npair - nfull + 1) / 2;
  if (blockIdx.x < g0) {
    qblock_pair_full(blocks, 2 * uint32_t(xcd_order(blockIdx.x, g0, kXcdRunPairs)), ptrs, recv);
  } else if (blockIdx.x < g0 + g1) {
    qblock_pair(blocks + nfull, 2 * (blockIdx.x - g0), npair - nfull, pieces, ptrs, recv);
  } else {
    const uint32_t i = npair + (blockIdx.x - g0 - g1);
    if (i < n) qblock_one(blocks[i], pieces, ptrs, recv);
  }
}

void task_grid(uint32_t n, const TaskSplit& sp, uint32_t* gx, uint32_t* gy) {
  const uint64_t total =
      (uint64_t(sp.n[0]) << sp.s[0]) + (uint64_t(sp.n[1]) << sp.s[1]) + (n - sp.n[0] - sp.n[1] - sp.tiles);
  if (total == 0) {
    *gx = *gy = 0;
    return;
  }
  if (total <= kMaxGridX) {
    *gx = static_cast<uint32_t>(total);
    *gy = 1;
  } else {  // fewest rows, then the narrowest rows: fewer than gy idle workgroups
    *gy = static_cast<uint32_t>((total + kMaxGridX - 1) / kMaxGridX);
    *gx = static_cast<uint32_t>((total + *gy - 1) / *gy);
  }
}

int launch_tasks(const Task* tasks, uint32_t n, const TaskSplit& sp, const uint64_t* ptrs, const void* buf,
                 const void* aux, void* stream) {
  if (n == 0) return hipSuccess;
  uint32_t gx, gy;
  task_grid(n, sp, &gx, &gy);
  if (gx) {
    hipLaunchKernelGGL(wb_tasks_kernel, dim3(gx, gy), dim3(kThreads), WB_TASK_DYN_LDS,
                       static_cast<hipStream_t>(stream), tasks, ptrs, static_cast<const char*>(buf),
                       static_cast<const char*>(aux), n - sp.tiles, sp.n[0], sp.n[1], sp.s[0], sp.s[1]);
    const hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  if (sp.tiles) {
    hipLaunchKernelGGL(wb_tile_kernel, dim3(sp.tiles), dim3(kTileThreads), 0, static_cast<hipStream_t>(stream),
                       tasks + (n - sp.tiles), ptrs, static_cast<const char*>(buf), static_cast<const char*>(aux));
    return hipGetLastError();
  }
  return hipSuccess;
}

int launch_qblocks(const QBlock* blocks, uint32_t n, uint32_t nfull, uint32_t npair, const QPiece* pieces,
                   const uint64_t* ptrs, const void* buf, void* stream) {
  if (n == 0) return hipSuccess;
  hipLaunchKernelGGL(wb_qblock_kernel, dim3(qblock_workgroups(n, nfull, npair)), dim3(kQBlockThreads),
                     WB_QBLOCK_DYN_LDS, static_cast<hipStream_t>(stream), blocks, pieces, ptrs,
                     static_cast<const char*>(buf), n, nfull, npair);
  return hipGetLastError();
}

const char* hip_error_string(int err) { return hipGetErrorString(static_cast<hipError_t>(err)); }

}  // namespace wb
