// Source-map probing kernels (WeightBridge Sec. 3.1 and App. B, Algorithm 1).
//
// wb_make_ids_kernel writes one b-bit chunk of every checkpoint element's
// identifier into a checkpoint tensor, in a form a value-preserving loader
// copies unchanged: bf16 carries the chunk as its bit pattern, fp32 as an
// exactly representable value.
//
// The diff2 kernels compute the second-order difference of a loaded chunk
// field (Eq. diff2: the outer product of [1, -2, 1] with itself, the field
// taken as 0 above and left of the tensor) and append its non-zero entries to
// a list. A slice copy leaves at most 16 of them, so the list is short. The
// work is cut into tiles, each one workgroup's share of one field:
//   ELEM  64 rows x 256 columns, one element per lane (any width, any
//         element-aligned address);
//   VEC   32 rows (128 batched) x 256 vectors of 16 bytes (8 bf16 or 4 fp32
//         values), the next row's loads in flight while a row is computed
//         (cols a multiple of the vector, 16-byte aligned field);
//   FLAT  one-row fields, 8 x 256 vectors per tile (32 x 256 batched).
// Single-field launches walk one field's tiles with a strided grid; the
// batched launch takes one tile per workgroup from a table that covers many
// fields, so all of a rank's tensors take one launch.
//
// Entries are gathered per workgroup in LDS (a wavefront ballot and an LDS
// add place each lane's entry) and appended to the global list with one
// atomic add per workgroup when the workgroup ends.
//
// Carry passes (Algorithm 1, ExpandCarry and EmitCarry): a pass's field is
// one 16-bit chunk, and the chunk's wrap-arounds make diff2 non-zero every
// 2^16 identifiers. Pass k's stencil adds to each non-zero D the carry that
// pass k - 1 left at that position, emits S mod 2^16 when non-zero and
// inserts floor(S / 2^16) when non-zero into the carry table of pass k + 1;
// the last pass emits S whole. The stencil's lookups wait in LDS and are made
// together when its tile ends, and its carries are staged per tile and
// inserted by a launch of their own; another launch handles the carries at
// positions where D is zero. The sum over passes of 2^(16 k) times the
// emitted values is diff2 of the identifier field, and only its positions
// (next to slice-copy corners) are emitted: the wrap-arounds stay in the
// device carry tables, which are hash tables (key position + 1, linear
// probing, at most half full when within capacity).
#include <hip/hip_runtime.h>

#include <cstdint>
#include <vector>

#include "wb_internal.hpp"

namespace wb {
namespace {

constexpr int kThreads = 256;
constexpr int kStrip = 64;      // rows of an ELEM tile
constexpr int kVecStrip = 32;   // rows of a VEC tile
constexpr int kFlatUnroll = 8;  // vectors in flight per lane (FLAT)

__global__ __launch_bounds__(kThreads) void wb_make_ids_kernel(char* dst, int dtype, int64_t numel, int64_t first_id,
                                                               int shift, uint32_t mask) {
  const int64_t stride = int64_t(gridDim.x) * kThreads;
  for (int64_t n = int64_t(blockIdx.x) * kThreads + threadIdx.x; n < numel; n += stride) {
    const uint32_t v = uint32_t((uint64_t(first_id + n) >> shift) & mask);
    if (dtype == WB_F32)
      reinterpret_cast<float*>(dst)[n] = float(v);
    else
      reinterpret_cast<uint16_t*>(dst)[n] = uint16_t(v);
  }
}

// Where non-zero entries go: slot k of index/value, k from an atomic counter;
// slots at or past capacity are counted but not written.
template <typename T>
struct Sink {
  int64_t* __restrict__ index;
  T* __restrict__ value;
  int64_t capacity;
  unsigned long long* __restrict__ count;
  __device__ __forceinline__ void operator()(unsigned long long slot, int64_t pos, int64_t v) const {
    if (slot < static_cast<unsigned long long>(capacity)) {
      index[slot] = pos;
      value[slot] = T(v);
    }
  }
};

// The chunk fields a tile reads: element value sum over k < n of p[k] << (16 k).
// Single-field and carry launches read one pass as int; the held-pass launch
// recombines up to kMaxPasses passes as int64 (identifiers below 2^48, |diff2|
// below 2^52).
template <int P>
struct Passes {
  const char* p[P];
  int n;
};

// One workgroup's entries, in LDS; entries past kWgCap go straight to the
// global list (one atomic add per wavefront).
constexpr int kWgCap = 256;
struct WgBuf {
  unsigned n;
  unsigned long long base;
  int64_t pos[kWgCap];
  int64_t val[kWgCap];
};

__device__ __forceinline__ void wg_init(WgBuf& b) {
  if (threadIdx.x == 0) b.n = 0;
}

__device__ __forceinline__ unsigned lanes_below(unsigned long long m, int lane) {
  return lane ? unsigned(__popcll(m & ((1ull << lane) - 1))) : 0u;
}

// Place (pos, v) of the lanes with `put` in the workgroup's buffer: one
// ballot and one LDS add per wavefront. Every lane of the wavefront calls it;
// it returns true for a lane whose entry did not fit (all such lanes of the
// wavefront then call the spill path together).
__device__ __forceinline__ bool wg_place(WgBuf& b, bool put, int64_t pos, int64_t v, int lane) {
  const unsigned long long m = __ballot(put);
  if (m == 0) return false;
  const int leader = __ffsll(static_cast<long long>(m)) - 1;
  unsigned off = 0;
  if (lane == leader) off = atomicAdd(&b.n, unsigned(__popcll(m)));
  off = __shfl(off, leader, 64);
  const unsigned slot = off + lanes_below(m, lane);
  if (put && slot < unsigned(kWgCap)) {
    b.pos[slot] = pos;
    b.val[slot] = v;
    return false;
  }
  return put;
}

// Entries that did not fit the buffer: one atomic add per wavefront on the
// list's counter, then each lane writes its slot.
template <typename T>
__device__ __forceinline__ void sink_spill(const Sink<T>& w, bool spill, int64_t pos, int64_t v, int lane) {
  const unsigned long long ms = __ballot(spill);
  if (ms == 0) return;
  const int first = __ffsll(static_cast<long long>(ms)) - 1;
  unsigned long long g = 0;
  if (lane == first) g = atomicAdd(w.count, static_cast<unsigned long long>(__popcll(ms)));
  g = __shfl(g, first, 64);
  if (spill) w(g + lanes_below(ms, lane), pos, v);
}

template <typename T>
__device__ __forceinline__ void sink_append(WgBuf& b, const Sink<T>& w, bool put, int64_t pos, int64_t v, int lane) {
  sink_spill(w, wg_place(b, put, pos, v, lane), pos, v, lane);
}

// Hand the workgroup's buffered entries to the global list: one atomic add.
// Every thread of the workgroup calls it, once, at the end.
template <typename T>
__device__ __forceinline__ void sink_flush(WgBuf& b, const Sink<T>& w) {
  __syncthreads();
  const unsigned n = b.n < unsigned(kWgCap) ? b.n : unsigned(kWgCap);
  if (threadIdx.x == 0 && n) b.base = atomicAdd(w.count, static_cast<unsigned long long>(n));
  __syncthreads();
  for (unsigned t = threadIdx.x; t < n; t += blockDim.x) w(b.base + t, b.pos[t], b.val[t]);
}

// The plain entry list of a launch: put() is what a tile calls for every
// candidate position (all lanes of a wavefront together).
template <typename T>
struct ListOut {
  WgBuf* buf;
  Sink<T> sink;
  __device__ __forceinline__ void put(bool nz, int64_t pos, T d, int lane) const {
    sink_append(*buf, sink, nz, pos, int64_t(d), lane);
  }
  // the V values of a lane at pos0 .. pos0 + V - 1, bit k of `any` set where
  // value k is a candidate
  template <int V>
  __device__ __forceinline__ void put_row(unsigned any, int64_t pos0, const T* d, int lane) const {
#pragma unroll
    for (int k = 0; k < V; ++k) put((any >> k) & 1u, pos0 + k, d[k], lane);
  }
  __device__ __forceinline__ void flush() const { sink_flush(*buf, sink); }
};

// Carry tables: slot h holds key position + 1 (0 empty) and field << 32 |
// carry (as uint32). Inserts probe linearly from the position's hash, at
// most kCarryProbes slots; one that finds none sets the table's flag.
__device__ __forceinline__ uint64_t carry_hash(int64_t pos) {
  uint64_t x = static_cast<uint64_t>(pos);  // MurmurHash3 64-bit finaliser
  x ^= x >> 33;
  x *= 0xff51afd7ed558ccdull;
  x ^= x >> 33;
  x *= 0xc4ceb9fe1a85ec53ull;
  x ^= x >> 33;
  return x;
}

__device__ __forceinline__ void carry_insert(const CarryTable& t, int64_t pos, int64_t packed) {
  uint64_t h = carry_hash(pos) & t.mask;
  const unsigned long long key = static_cast<unsigned long long>(pos + 1);
  for (int n = 0; n < kCarryProbes; ++n) {
    if (atomicCAS(reinterpret_cast<unsigned long long*>(t.slot + 2 * h), 0ull, key) == 0ull) {
      t.slot[2 * h + 1] = packed;
      return;
    }
    h = (h + 1) & t.mask;
  }
  t.count[kCarryCounters] = 1;
}

__device__ __forceinline__ int carry_lookup(const CarryTable& t, int64_t pos) {
  uint64_t h = carry_hash(pos) & t.mask;
  for (int n = 0; n < kCarryProbes; ++n) {
    const int64_t key = t.slot[2 * h];
    if (key == pos + 1) return static_cast<int32_t>(static_cast<uint32_t>(t.slot[2 * h + 1]));
    if (key == 0) return 0;
    h = (h + 1) & t.mask;
  }
  return 0;
}

// Carries that do not fit the workgroup's buffer are inserted at once and
// counted on one of kCarryCounters counters (an add whose result is not
// needed).
__device__ __forceinline__ void carry_spill(const CarryTable& t, bool spill, int64_t pos, int64_t packed, int lane) {
  const unsigned long long ms = __ballot(spill);
  if (ms == 0) return;
  if (lane == __ffsll(static_cast<long long>(ms)) - 1)
    atomicAdd(t.count + blockIdx.x % kCarryCounters, static_cast<unsigned long long>(__popcll(ms)));
  if (spill) carry_insert(t, pos, packed);
}

// The workgroup's buffered carries. With kStage (a stencil tile) the first
// kCarryStage are staged for the insert launch with plain stores and their
// number stored for the tile (no atomic), the rest inserted and counted
// here; otherwise all are inserted here and counted with one add.
template <bool kStage>
__device__ __forceinline__ void carry_flush(WgBuf& b, const CarryTable& t) {
  __syncthreads();
  const unsigned n = b.n < unsigned(kWgCap) ? b.n : unsigned(kWgCap);
  const unsigned m = kStage ? (n < unsigned(kCarryStage) ? n : unsigned(kCarryStage)) : 0u;
  if (threadIdx.x == 0) {
    if (kStage) t.stage_n[blockIdx.x] = int32_t(m);
    if (n > m) atomicAdd(t.count + blockIdx.x % kCarryCounters, static_cast<unsigned long long>(n - m));
  }
  for (unsigned k = threadIdx.x; k < n; k += blockDim.x) {
    if (k < m) {
      int64_t* e = t.stage + 2 * (int64_t(blockIdx.x) * kCarryStage + k);
      e[0] = b.pos[k];
      e[1] = b.val[k];
    } else {
      carry_insert(t, b.pos[k], b.val[k]);
    }
  }
}

// A carry pass's output. The stencil's candidates (non-zero D) wait in
// `pending`, placed with one LDS add per wavefront per row, and are split
// together when the tile ends: the carry of pass k - 1 is looked up (kIn),
// S = D + carry gives an emitted value and a carry (split). Candidates that
// do not fit `pending` are split at once.
template <bool kIn, bool kLast, bool kStage>
struct CarryOut {
  WgBuf* ebuf;
  WgBuf* cbuf;
  WgBuf* pending;
  Sink<int64_t> sink;
  CarryTable in, next;
  int64_t field;
  __device__ __forceinline__ void split(bool c, int64_t pos, int s, int64_t f, int lane) const {
    if (kLast) {
      sink_append(*ebuf, sink, c && s != 0, pos, int64_t(s), lane);
    } else {
      const int r = s & 0xFFFF, q = s >> 16;  // arithmetic shift: floor(S / 2^16)
      sink_append(*ebuf, sink, c && r != 0, pos, int64_t(r), lane);
      const bool cq = c && q != 0;
      const int64_t packed = (f << 32) | int64_t(static_cast<uint32_t>(q));
      carry_spill(next, wg_place(*cbuf, cq, pos, packed, lane), pos, packed, lane);
    }
  }
  __device__ __forceinline__ int carry_in(bool c, int64_t pos) const { return kIn && c ? carry_lookup(in, pos) : 0; }
  __device__ __forceinline__ void put(bool nz, int64_t pos, int d, int lane) const {
    const bool now = wg_place(*pending, nz, pos, int64_t(d), lane);
    if (__ballot(now) == 0) return;
    split(now, pos, d + carry_in(now, pos), field, lane);
  }
  // All lanes of the wavefront call it, with at least one bit set in some
  // lane's `any`; the count of a lane (at most 8) is summed over the
  // wavefront bit by bit with four ballots.
  template <int V>
  __device__ __forceinline__ void put_row(unsigned any, int64_t pos0, const int* d, int lane) const {
    static_assert(V <= 8, "at most 8 values per lane");
    const unsigned c = __popc(any);
    const unsigned long long lt = lane ? (1ull << lane) - 1 : 0ull;
    unsigned below = 0, total = 0;
#pragma unroll
    for (int b = 0; b < 4; ++b) {
      const unsigned long long m = __ballot((c >> b) & 1u);
      below += unsigned(__popcll(m & lt)) << b;
      total += unsigned(__popcll(m)) << b;
    }
    unsigned off = 0;
    if (lane == 0) off = atomicAdd(&pending->n, total);
    off = __shfl(off, 0, 64);
    unsigned slot = off + below;
    unsigned now = 0;
#pragma unroll
    for (int k = 0; k < V; ++k) {
      if ((any >> k) & 1u) {
        if (slot < unsigned(kWgCap)) {
          pending->pos[slot] = pos0 + k;
          pending->val[slot] = d[k];
        } else {
          now |= 1u << k;
        }
        ++slot;
      }
    }
    if (__ballot(now != 0) == 0) return;
#pragma unroll
    for (int k = 0; k < V; ++k) {
      const bool c1 = (now >> k) & 1u;
      if (__ballot(c1) == 0) continue;
      split(c1, pos0 + k, d[k] + carry_in(c1, pos0 + k), field, lane);
    }
  }
  // the emitted values and the carries of the workgroup
  __device__ __forceinline__ void flush_outputs() const {
    sink_flush(*ebuf, sink);
    if (!kLast) carry_flush<kStage>(*cbuf, next);
  }
  __device__ __forceinline__ void flush() const {
    __syncthreads();
    const unsigned n = pending->n < unsigned(kWgCap) ? pending->n : unsigned(kWgCap);
    for (unsigned b0 = 0; b0 < n; b0 += blockDim.x) {
      const unsigned k = b0 + threadIdx.x;
      const bool ok = k < n;
      const int64_t pos = ok ? pending->pos[k] : 0;
      const int s = ok ? int(pending->val[k]) + carry_in(true, pos) : 0;
      split(ok, pos, s, field, threadIdx.x & 63);
    }
    flush_outputs();
  }
};

__device__ __forceinline__ int load_chunk(const char* src, int dtype, int64_t k) {
  if (dtype == WB_F32) return int(reinterpret_cast<const float*>(src)[k]);
  return int(reinterpret_cast<const uint16_t*>(src)[k]);
}

template <typename T, int P>
__device__ __forceinline__ T load_value(const Passes<P>& s, int dtype, int64_t k) {
  T v = 0;
#pragma unroll
  for (int c = 0; c < P; ++c)
    if (c < s.n) v += T(load_chunk(s.p[c], dtype, k)) << (16 * c);
  return v;
}

// ELEM tile: thread t takes column jb + t over rows [i0, i0 + kStrip), after
// two halo rows above. The horizontal difference h(i) = c(i,j) - 2 c(i,j-1) +
// c(i,j-2) takes its left neighbours from the lanes to the left (the first two
// lanes of a wavefront load theirs); then D = h(i) - 2 h(i-1) + h(i-2).
template <typename T, int P, class Out>
__device__ __forceinline__ void elem_tile(const Passes<P>& s, int dtype, int64_t rows, int64_t cols, int64_t base,
                                          int64_t i0, int64_t jb, const Out& out) {
  const int lane = threadIdx.x & 63;
  const int64_t j = jb + threadIdx.x;
  const bool col = j < cols;
  const int64_t i1 = i0 + kStrip < rows ? i0 + kStrip : rows;
  T h1 = 0, h2 = 0;  // h(i-1), h(i-2)
  for (int64_t i = (i0 >= 2 ? i0 - 2 : 0); i < i1; ++i) {
    const int64_t rowbase = i * cols;
    const T c0 = col ? load_value<T, P>(s, dtype, rowbase + j) : T(0);
    T c1 = __shfl_up(c0, 1, 64), c2 = __shfl_up(c0, 2, 64);
    if (lane == 0) c1 = (col && j >= 1) ? load_value<T, P>(s, dtype, rowbase + j - 1) : T(0);
    if (lane <= 1) c2 = (col && j >= 2) ? load_value<T, P>(s, dtype, rowbase + j - 2) : T(0);
    if (j < 1) c1 = 0;
    if (j < 2) c2 = 0;
    const T h = c0 - 2 * c1 + c2;
    const T d = h - 2 * h1 + h2;
    h2 = h1;
    h1 = h;
    out.put(col && i >= i0 && d != 0, base + rowbase + j, d, lane);
  }
}

// Add the V chunk values of one 16-byte vector, shifted, to x.
template <int V, typename T>
__device__ __forceinline__ void add_vec(const uint4 q, int shift, T* x) {
  if (V == 8) {
    const uint32_t w[4] = {q.x, q.y, q.z, q.w};
#pragma unroll
    for (int k = 0; k < 4; ++k) {
      x[2 * k] += T(w[k] & 0xFFFFu) << shift;
      x[2 * k + 1] += T(w[k] >> 16) << shift;
    }
  } else {
    x[0] += T(int(__uint_as_float(q.x))) << shift;
    x[1] += T(int(__uint_as_float(q.y))) << shift;
    x[2] += T(int(__uint_as_float(q.z))) << shift;
    x[3] += T(int(__uint_as_float(q.w))) << shift;
  }
}

// Add the values at columns j0 - 1 (l1) and j0 - 2 (l2) of a row, j0 >= 2.
template <int V, typename T>
__device__ __forceinline__ void add_left_pair(const char* row, int64_t j0, int shift, T& l1, T& l2) {
  if (V == 8) {
    const uint32_t pw = *reinterpret_cast<const uint32_t*>(row + (j0 - 2) * 2);
    l2 += T(pw & 0xFFFFu) << shift;
    l1 += T(pw >> 16) << shift;
  } else {
    const uint2 pw = *reinterpret_cast<const uint2*>(row + (j0 - 2) * 4);
    l2 += T(int(__uint_as_float(pw.x))) << shift;
    l1 += T(int(__uint_as_float(pw.y))) << shift;
  }
}

// Row i's vector at column j0 (x) and, for the first lane of a wavefront,
// the two values left of it, summed over the passes.
template <int V, typename T, int P>
__device__ __forceinline__ void load_row_vec(const Passes<P>& s, int64_t rowoff, int64_t j0, bool left, T* x, T& l1,
                                             T& l2) {
#pragma unroll
  for (int c = 0; c < P; ++c) {
    if (c >= s.n) break;
    const char* row = s.p[c] + rowoff;
    add_vec<V, T>(*reinterpret_cast<const uint4*>(row + j0 * (16 / V)), 16 * c, x);
    if (left) add_left_pair<V, T>(row, j0, 16 * c, l1, l2);
  }
}

// VEC tile: thread t takes the V columns of vector vb + t over rows [i0, i0 +
// S), after two halo rows, one row of state per lane. The two columns left of
// a lane's vector are the previous lane's last two (the first lane of each
// wavefront loads them). The next row's vectors of every pass (and, for the
// first lane, the two values left of them) are loaded before the current row
// is computed, so two rows of loads are in flight per lane. Measured against
// rows loaded and then computed: carry passes (one pass, int) 5-7 % faster
// per pass than one row and faster than two or four rows; held passes (three,
// int64) 9.56 -> 8.05 ms for 48 GB; two rows ahead gave nothing more.
template <int V, typename T, int P, int S, class Out>
__device__ __forceinline__ void vec_tile(const Passes<P>& s, int64_t rows, int64_t cols, int64_t base, int64_t i0,
                                         int64_t vb, const Out& out) {
  const int lane = threadIdx.x & 63;
  const int64_t nvec = cols / V;
  const int64_t v = vb + threadIdx.x;
  const bool live = v < nvec;
  const int64_t j0 = v * V;
  const int64_t i1 = i0 + S < rows ? i0 + S : rows;
  const int64_t rb = cols * (16 / V);
  const bool left = lane == 0 && j0 >= 2;
  T h1[V], h2[V];
#pragma unroll
  for (int k = 0; k < V; ++k) h1[k] = h2[k] = 0;
  const int64_t ist = i0 >= 2 ? i0 - 2 : 0;
  auto fetch = [&](int64_t i, uint4* qq, uint2* ll) {
#pragma unroll
    for (int c = 0; c < P; ++c) {
      qq[c] = uint4{0u, 0u, 0u, 0u};
      ll[c] = uint2{0u, 0u};
      if (c < s.n && live && i < i1) {
        qq[c] = *reinterpret_cast<const uint4*>(s.p[c] + j0 * (16 / V) + i * rb);
        if (left) {
          if (V == 8) ll[c].x = *reinterpret_cast<const uint32_t*>(s.p[c] + (j0 - 2) * 2 + i * rb);
          else ll[c] = *reinterpret_cast<const uint2*>(s.p[c] + (j0 - 2) * 4 + i * rb);
        }
      }
    }
  };
  uint4 q[P];
  uint2 lq[P];
  fetch(ist, q, lq);
  for (int64_t i = ist; i < i1; ++i) {
    uint4 qn[P];
    uint2 ln[P];
    fetch(i + 1, qn, ln);
    T x[V];
#pragma unroll
    for (int k = 0; k < V; ++k) x[k] = 0;
    T l1 = 0, l2 = 0;
#pragma unroll
    for (int c = 0; c < P; ++c) {
      if (c >= s.n) break;
      add_vec<V, T>(q[c], 16 * c, x);
      if (V == 8) {
        l2 += T(lq[c].x & 0xFFFFu) << (16 * c);
        l1 += T(lq[c].x >> 16) << (16 * c);
      } else {
        l2 += T(int(__uint_as_float(lq[c].x))) << (16 * c);
        l1 += T(int(__uint_as_float(lq[c].y))) << (16 * c);
      }
    }
    T p1 = __shfl_up(x[V - 1], 1, 64), p2 = __shfl_up(x[V - 2], 1, 64);
    if (lane == 0) {
      p1 = l1;
      p2 = l2;
    }
    T h[V];
    h[0] = x[0] - 2 * p1 + p2;
    h[1] = x[1] - 2 * x[0] + p1;
#pragma unroll
    for (int k = 2; k < V; ++k) h[k] = x[k] - 2 * x[k - 1] + x[k - 2];
    T d[V];
    unsigned any = 0;
#pragma unroll
    for (int k = 0; k < V; ++k) {
      d[k] = h[k] - 2 * h1[k] + h2[k];
      h2[k] = h1[k];
      h1[k] = h[k];
      any |= (live && i >= i0 && d[k] != 0) ? (1u << k) : 0u;
    }
    if (__ballot(any != 0) != 0) out.template put_row<V>(any, base + i * cols + j0, d, lane);
#pragma unroll
    for (int c = 0; c < P; ++c) {
      q[c] = qn[c];
      lq[c] = ln[c];
    }
  }
}

// FLAT tile of a one-row field: with nothing above, D is the row's second
// difference. Lane l of sub-tile u takes vector cb + u * kThreads + l.
template <int V, typename T, int P, int U, class Out>
__device__ __forceinline__ void flat_tile(const Passes<P>& s, int64_t cols, int64_t base, int64_t cb,
                                          const Out& out) {
  const int lane = threadIdx.x & 63;
  const int64_t nvec = cols / V;
  T x[U][V];
  T l1[U], l2[U];
#pragma unroll
  for (int u = 0; u < U; ++u) {
    const int64_t v = cb + int64_t(u) * kThreads + threadIdx.x;
    l1[u] = l2[u] = 0;
#pragma unroll
    for (int k = 0; k < V; ++k) x[u][k] = 0;
    if (v < nvec) load_row_vec<V, T, P>(s, 0, v * V, lane == 0 && v * V >= 2, x[u], l1[u], l2[u]);
  }
#pragma unroll
  for (int u = 0; u < U; ++u) {
    const int64_t v = cb + int64_t(u) * kThreads + threadIdx.x;
    if (cb + int64_t(u) * kThreads >= nvec) break;  // uniform over the workgroup
    T p1 = __shfl_up(x[u][V - 1], 1, 64), p2 = __shfl_up(x[u][V - 2], 1, 64);
    if (lane == 0) {
      p1 = l1[u];
      p2 = l2[u];
    }
    T d[V];
    d[0] = x[u][0] - 2 * p1 + p2;
    d[1] = x[u][1] - 2 * x[u][0] + p1;
#pragma unroll
    for (int k = 2; k < V; ++k) d[k] = x[u][k] - 2 * x[u][k - 1] + x[u][k - 2];
    unsigned any = 0;
#pragma unroll
    for (int k = 0; k < V; ++k) any |= (v < nvec && d[k] != 0) ? (1u << k) : 0u;
    if (__ballot(any != 0) == 0) continue;
    out.template put_row<V>(any, base + v * V, d, lane);
  }
}

// Single-field launches: one pass, int arithmetic, a strided grid over the
// field's tiles.

__global__ __launch_bounds__(kThreads) void wb_diff2_kernel(const char* __restrict__ src, int dtype, int64_t rows,
                                                            int64_t cols, Sink<int> sink) {
  __shared__ WgBuf buf;
  wg_init(buf);
  __syncthreads();
  const ListOut<int> out{&buf, sink};
  const Passes<1> s{{src}, 1};
  for (int64_t jb = int64_t(blockIdx.x) * kThreads; jb < cols; jb += int64_t(gridDim.x) * kThreads)
    for (int64_t i0 = int64_t(blockIdx.y) * kStrip; i0 < rows; i0 += int64_t(gridDim.y) * kStrip)
      elem_tile<int, 1>(s, dtype, rows, cols, 0, i0, jb, out);
  out.flush();
}

template <int V>
__global__ __launch_bounds__(kThreads) void wb_diff2_vec_kernel(const char* __restrict__ src, int64_t rows,
                                                                int64_t cols, Sink<int> sink) {
  __shared__ WgBuf buf;
  wg_init(buf);
  __syncthreads();
  const ListOut<int> out{&buf, sink};
  const Passes<1> s{{src}, 1};
  const int64_t nvec = cols / V;
  for (int64_t vb = int64_t(blockIdx.x) * kThreads; vb < nvec; vb += int64_t(gridDim.x) * kThreads)
    for (int64_t i0 = int64_t(blockIdx.y) * kVecStrip; i0 < rows; i0 += int64_t(gridDim.y) * kVecStrip)
      vec_tile<V, int, 1, kVecStrip>(s, rows, cols, 0, i0, vb, out);
  out.flush();
}

template <int V>
__global__ __launch_bounds__(kThreads) void wb_diff2_flat_kernel(const char* __restrict__ src, int64_t cols,
                                                                 Sink<int> sink) {
  __shared__ WgBuf buf;
  wg_init(buf);
  __syncthreads();
  const ListOut<int> out{&buf, sink};
  const Passes<1> s{{src}, 1};
  const int64_t nvec = cols / V;
  const int64_t step = int64_t(gridDim.x) * kThreads * kFlatUnroll;
  for (int64_t cb = int64_t(blockIdx.x) * kThreads * kFlatUnroll; cb < nvec; cb += step)
    flat_tile<V, int, 1, kFlatUnroll>(s, cols, 0, cb, out);
  out.flush();
}

// Batched launches: workgroup b takes tile b of the table, taller VEC tiles
// (vec_tile) and FLAT tiles of several sub-tiles (fewer, larger table
// rows). Held passes recombine up to kMaxPasses passes in int64; carry passes
// read one pass in int.
constexpr int kBatchVecStrip = 128;
constexpr int kBatchFlatUnroll = 4;
constexpr int kBatchFlatSub = 8;  // sub-tiles of kBatchFlatUnroll x kThreads vectors per FLAT tile

template <typename T, int P, class Out>
__device__ __forceinline__ void batch_tile(const DiffField& f, const DiffTile& t, const Out& out) {
  Passes<P> s;
#pragma unroll
  for (int c = 0; c < P; ++c) s.p[c] = static_cast<const char*>(f.src[c]);
  s.n = P == 1 ? 1 : f.passes;
  if (f.kind == DIFF_FLAT) {
    for (int q = 0; q < kBatchFlatSub; ++q) {
      const int64_t cb = t.j0 + int64_t(q) * kBatchFlatUnroll * kThreads;
      if (f.dtype == WB_F32)
        flat_tile<4, T, P, kBatchFlatUnroll>(s, f.cols, f.base, cb, out);
      else
        flat_tile<8, T, P, kBatchFlatUnroll>(s, f.cols, f.base, cb, out);
    }
  } else if (f.kind == DIFF_VEC) {
    if (f.dtype == WB_F32)
      vec_tile<4, T, P, kBatchVecStrip>(s, f.rows, f.cols, f.base, t.i0, t.j0, out);
    else
      vec_tile<8, T, P, kBatchVecStrip>(s, f.rows, f.cols, f.base, t.i0, t.j0, out);
  } else {
    elem_tile<T, P>(s, f.dtype, f.rows, f.cols, f.base, t.i0, t.j0, out);
  }
}

__global__ __launch_bounds__(kThreads) void wb_diff2_batch_kernel(const DiffField* __restrict__ fields,
                                                                  const DiffTile* __restrict__ tiles,
                                                                  Sink<int64_t> sink) {
  __shared__ WgBuf buf;
  wg_init(buf);
  __syncthreads();
  const ListOut<int64_t> out{&buf, sink};
  const DiffTile t = tiles[blockIdx.x];
  batch_tile<int64_t, kMaxPasses>(fields[t.field], t, out);
  out.flush();
}

// Carry pass, stencil part: one tile per workgroup of one pass's fields.
template <bool kIn, bool kLast>
__global__ __launch_bounds__(kThreads) void wb_diff2_carry_kernel(const DiffField* __restrict__ fields,
                                                                  const DiffTile* __restrict__ tiles, CarryTable in,
                                                                  CarryTable next, Sink<int64_t> sink) {
  __shared__ WgBuf ebuf, cbuf, pending;
  wg_init(ebuf);
  wg_init(cbuf);
  wg_init(pending);
  __syncthreads();
  const DiffTile t = tiles[blockIdx.x];
  const CarryOut<kIn, kLast, true> out{&ebuf, &cbuf, &pending, sink, in, next, int64_t(t.field)};
  batch_tile<int, 1>(fields[t.field], t, out);
  out.flush();
}

// D at local position p of a one-pass field, straight from the nine
// neighbours (Eq. diff2 as the outer product of [1, -2, 1] with itself).
__device__ __forceinline__ int diff2_at(const DiffField& f, int64_t p) {
  const int64_t i = p / f.cols, j = p - i * f.cols;
  const char* src = static_cast<const char*>(f.src[0]);
  int d = 0;
  for (int a = 0; a < 3 && a <= i; ++a) {
    const int wa = a == 1 ? -2 : 1;
    for (int b = 0; b < 3 && b <= j; ++b) {
      const int w = wa * (b == 1 ? -2 : 1);
      d += w * load_chunk(src, f.dtype, (i - a) * f.cols + (j - b));
    }
  }
  return d;
}

// Carry pass, the carries of pass k - 1 at positions where D is zero (the
// stencil took the others): S is the carry itself. A walk over the slots of
// the table; slots whose field or position does not fit the fields are
// skipped.
template <bool kLast>
__global__ __launch_bounds__(kThreads) void wb_carry_rest_kernel(const DiffField* __restrict__ fields, int nfields,
                                                                 CarryTable in, CarryTable next,
                                                                 Sink<int64_t> sink) {
  __shared__ WgBuf ebuf, cbuf;
  wg_init(ebuf);
  wg_init(cbuf);
  __syncthreads();
  const int lane = threadIdx.x & 63;
  const int64_t slots = static_cast<int64_t>(in.mask) + 1;
  const CarryOut<false, kLast, false> out{&ebuf, &cbuf, nullptr, sink, in, next, 0};
  for (int64_t b0 = int64_t(blockIdx.x) * kThreads; b0 < slots; b0 += int64_t(gridDim.x) * kThreads) {
    const int64_t h = b0 + threadIdx.x;
    int64_t pos = 0, field = 0;
    int q = 0;
    bool take = false;
    if (h < slots) {
      const int64_t key = in.slot[2 * h];
      if (key != 0) {
        pos = key - 1;
        const int64_t packed = in.slot[2 * h + 1];
        field = packed >> 32;
        q = static_cast<int32_t>(static_cast<uint32_t>(packed));
        if (field >= 0 && field < nfields) {
          const DiffField& f = fields[field];
          const int64_t p = pos - f.base;
          take = q != 0 && f.passes == 1 && p >= 0 && p < f.rows * f.cols && diff2_at(f, p) == 0;
        }
      }
    }
    out.split(take, pos, q, field, lane);
  }
  out.flush_outputs();
}

// Insert the carries the stencil workgroups staged: one thread per staging
// slot of every tile.
__global__ __launch_bounds__(kThreads) void wb_carry_insert_kernel(CarryTable next, int64_t ntiles) {
  const int64_t total = ntiles * kCarryStage;
  const int64_t stride = int64_t(gridDim.x) * kThreads;
  for (int64_t e = int64_t(blockIdx.x) * kThreads + threadIdx.x; e < total; e += stride) {
    const int64_t t = e / kCarryStage, k = e - t * kCarryStage;
    if (k < next.stage_n[t]) carry_insert(next, next.stage[2 * e], next.stage[2 * e + 1]);
  }
}

// Empty the next carry table, zero its counters and flag and the entry
// counter (a fill, not a memset: the launches may be captured).
__global__ __launch_bounds__(kThreads) void wb_carry_clear_kernel(int64_t* slot, int64_t slots,
                                                                 unsigned long long* carries,
                                                                 unsigned long long* count) {
  const int64_t stride = int64_t(gridDim.x) * kThreads;
  for (int64_t k = int64_t(blockIdx.x) * kThreads + threadIdx.x; k < slots; k += stride) slot[2 * k] = 0;
  if (blockIdx.x == 0) {
    if (threadIdx.x <= kCarryCounters) carries[threadIdx.x] = 0;
    if (threadIdx.x == 0) *count = 0;
  }
}

// The carries a pass kept: the staged counts of the ntiles stencil tiles
// plus the counters of the carries inserted directly, or past the capacity
// if an insert found no slot. One workgroup.
__global__ __launch_bounds__(kThreads) void wb_carry_report_kernel(const int32_t* stage_n, int64_t ntiles,
                                                                  const unsigned long long* counters,
                                                                  int64_t capacity, unsigned long long* out) {
  __shared__ unsigned long long part[kThreads];
  unsigned long long n = 0;
  for (int64_t t = threadIdx.x; t < ntiles; t += kThreads) n += static_cast<unsigned long long>(stage_n[t]);
  if (threadIdx.x < kCarryCounters) n += counters[threadIdx.x];
  part[threadIdx.x] = n;
  __syncthreads();
  for (int w = kThreads / 2; w > 0; w /= 2) {
    if (threadIdx.x < w) part[threadIdx.x] += part[threadIdx.x + w];
    __syncthreads();
  }
  if (threadIdx.x == 0) {
    unsigned long long total = part[0];
    if (counters[kCarryCounters] && total <= static_cast<unsigned long long>(capacity))
      total = static_cast<unsigned long long>(capacity) + 1;
    *out = total;
  }
}


__global__ void wb_zero_count_kernel(unsigned long long* count) { *count = 0; }

// VEC and FLAT tiles need whole 16-byte vectors in every pass.
int tile_kind(const void* const* src, int passes, int dtype, int64_t rows, int64_t cols) {
  const int V = dtype == WB_F32 ? 4 : 8;
  if (cols % V != 0) return DIFF_ELEM;
  for (int c = 0; c < passes; ++c)
    if (reinterpret_cast<uintptr_t>(src[c]) % 16 != 0) return DIFF_ELEM;
  return rows == 1 ? DIFF_FLAT : DIFF_VEC;
}

// A 2-D grid over (x tiles, y strips), about 64 K workgroups at most; each
// workgroup loops over further tiles.
dim3 strided_grid(int64_t xtiles, int64_t strips) {
  const int64_t y = strips < 65535 ? strips : 65535;
  const int64_t xcap = (65536 + y - 1) / y;
  return dim3(static_cast<unsigned>(xtiles < xcap ? xtiles : xcap), static_cast<unsigned>(y));
}

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
  const Sink<int> out{index, value, capacity, count};
  const char* s = static_cast<const char*>(src);
  const bool f32 = dtype == WB_F32;
  const int V = f32 ? 4 : 8;
  switch (tile_kind(&src, 1, dtype, rows, cols)) {
    case DIFF_FLAT: {
      const int64_t tiles = (cols / V + kThreads * kFlatUnroll - 1) / (kThreads * kFlatUnroll);
      const dim3 grid(static_cast<unsigned>(tiles < 65536 ? tiles : 65536));
      if (f32)
        hipLaunchKernelGGL(wb_diff2_flat_kernel<4>, grid, dim3(kThreads), 0, st, s, cols, out);
      else
        hipLaunchKernelGGL(wb_diff2_flat_kernel<8>, grid, dim3(kThreads), 0, st, s, cols, out);
      break;
    }
    case DIFF_VEC: {
      const dim3 grid = strided_grid((cols / V + kThreads - 1) / kThreads, (rows + kVecStrip - 1) / kVecStrip);
      if (f32)
        hipLaunchKernelGGL(wb_diff2_vec_kernel<4>, grid, dim3(kThreads), 0, st, s, rows, cols, out);
      else
        hipLaunchKernelGGL(wb_diff2_vec_kernel<8>, grid, dim3(kThreads), 0, st, s, rows, cols, out);
      break;
    }
    default: {
      const dim3 grid = strided_grid((cols + kThreads - 1) / kThreads, (rows + kStrip - 1) / kStrip);
      hipLaunchKernelGGL(wb_diff2_kernel, grid, dim3(kThreads), 0, st, s, dtype, rows, cols, out);
    }
  }
  return hipGetLastError();
}

void diff_tiles(int32_t fi, DiffField& f, std::vector<DiffTile>& out) {
  f.kind = static_cast<uint8_t>(tile_kind(f.src, f.passes, f.dtype, f.rows, f.cols));
  if (f.rows == 0 || f.cols == 0) return;
  const int64_t nvec = f.cols / (f.dtype == WB_F32 ? 4 : 8);
  int64_t istep = kStrip, jstep = kThreads, jend = f.cols;
  if (f.kind == DIFF_FLAT) {
    istep = 1;
    jstep = int64_t(kThreads) * kBatchFlatUnroll * kBatchFlatSub;
    jend = nvec;
  } else if (f.kind == DIFF_VEC) {
    istep = kBatchVecStrip;
    jend = nvec;
  }
  DiffTile t{};
  t.field = fi;
  for (int64_t i0 = 0; i0 < f.rows; i0 += istep)
    for (int64_t j0 = 0; j0 < jend; j0 += jstep) {
      t.i0 = i0;
      t.j0 = j0;
      out.push_back(t);
    }
}

int launch_diff2_batch(const DiffField* fields, const DiffTile* tiles, int64_t ntiles, int64_t* index, int64_t* value,
                       int64_t capacity, unsigned long long* count, void* stream) {
  hipStream_t st = static_cast<hipStream_t>(stream);
  hipLaunchKernelGGL(wb_zero_count_kernel, dim3(1), dim3(1), 0, st, count);
  if (ntiles == 0) return hipGetLastError();
  const Sink<int64_t> out{index, value, capacity, count};
  hipLaunchKernelGGL(wb_diff2_batch_kernel, dim3(static_cast<unsigned>(ntiles)), dim3(kThreads), 0, st, fields, tiles,
                     out);
  return hipGetLastError();
}

int launch_diff2_carry(const DiffField* fields, int32_t nfields, const DiffTile* tiles, int64_t ntiles, bool has_in,
                       bool last, const CarryTable& in, const CarryTable& next, int64_t* index, int64_t* value,
                       int64_t capacity, unsigned long long* count, unsigned long long* carries, void* stream) {
  hipStream_t st = static_cast<hipStream_t>(stream);
  const int64_t slots = last ? 0 : static_cast<int64_t>(next.mask) + 1;
  const int64_t clear = (slots + kThreads - 1) / kThreads;
  hipLaunchKernelGGL(wb_carry_clear_kernel, dim3(static_cast<unsigned>(clear < 1 ? 1 : clear < 4096 ? clear : 4096)),
                     dim3(kThreads), 0, st, next.slot, slots, next.count, count);
  const Sink<int64_t> sink{index, value, capacity, count};
  if (ntiles > 0) {
    const dim3 grid(static_cast<unsigned>(ntiles));
    if (has_in && last)
      hipLaunchKernelGGL((wb_diff2_carry_kernel<true, true>), grid, dim3(kThreads), 0, st, fields, tiles, in, next, sink);
    else if (has_in)
      hipLaunchKernelGGL((wb_diff2_carry_kernel<true, false>), grid, dim3(kThreads), 0, st, fields, tiles, in, next,
                         sink);
    else if (last)
      hipLaunchKernelGGL((wb_diff2_carry_kernel<false, true>), grid, dim3(kThreads), 0, st, fields, tiles, in, next,
                         sink);
    else
      hipLaunchKernelGGL((wb_diff2_carry_kernel<false, false>), grid, dim3(kThreads), 0, st, fields, tiles, in, next,
                         sink);
  }
  if (ntiles > 0 && !last) {
    const int64_t want = (ntiles * kCarryStage + kThreads - 1) / kThreads;
    hipLaunchKernelGGL(wb_carry_insert_kernel, dim3(static_cast<unsigned>(want < 8192 ? want : 8192)), dim3(kThreads),
                       0, st, next, ntiles);
  }
  if (has_in) {
    const int64_t want = (static_cast<int64_t>(in.mask) + kThreads) / kThreads;
    const dim3 grid(static_cast<unsigned>(want < 4096 ? want : 4096));
    if (last)
      hipLaunchKernelGGL(wb_carry_rest_kernel<true>, grid, dim3(kThreads), 0, st, fields, int(nfields), in, next, sink);
    else
      hipLaunchKernelGGL(wb_carry_rest_kernel<false>, grid, dim3(kThreads), 0, st, fields, int(nfields), in, next,
                         sink);
  }
  hipLaunchKernelGGL(wb_carry_report_kernel, dim3(1), dim3(kThreads), 0, st, next.stage_n, last ? 0 : ntiles,
                     next.count, next.capacity, carries);
  return hipGetLastError();
}

}  // namespace wb
