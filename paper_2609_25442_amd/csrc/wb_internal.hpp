// Internal types of libwb: layouts, the global plan, one rank's kernel work.
#pragma once

#include <cstdint>
#include <memory>
#include <stdexcept>
#include <string>
#include <unordered_map>
#include <utility>
#include <vector>

#include "../../include/wb.h"

namespace wb {

// Error carried from deep inside the planner to the C ABI boundary.
struct Error : std::runtime_error {
  int code;
  Error(int c, const std::string& m) : std::runtime_error(m), code(c) {}
};
[[noreturn]] inline void fail(int code, const std::string& msg) { throw Error(code, msg); }

// Allocator that leaves new elements of trivial types uninitialised on
// resize, so a large table is first touched by the threads that fill it
// (every element must then be written before it is read).
template <class T>
struct NoInitAlloc : std::allocator<T> {
  template <class U>
  struct rebind {
    using other = NoInitAlloc<U>;
  };
  NoInitAlloc() = default;
  template <class U>
  NoInitAlloc(const NoInitAlloc<U>&) noexcept {}
  template <class U>
  void construct(U* p) noexcept {
    ::new (static_cast<void*>(p)) U;
  }
  template <class U, class... A>
  void construct(U* p, A&&... a) {
    ::new (static_cast<void*>(p)) U(std::forward<A>(a)...);
  }
};

inline int dtype_bytes(int dt) {
  switch (dt) {
    case WB_F32: return 4;
    case WB_BF16: return 2;
    case WB_F8E4M3: return 1;
    default: return 0;
  }
}
inline const char* dtype_name(int dt) {
  switch (dt) {
    case WB_F32: return "f32";
    case WB_BF16: return "bf16";
    case WB_F8E4M3: return "f8e4m3";
    default: return "?";
  }
}

struct Tensor {
  std::string name;
  int64_t rows = 0, cols = 0;
  int64_t numel() const { return rows * cols; }
};

struct Local {
  std::string name;
  int dtype = WB_F32;
  int64_t batch = 1, rows = 1, cols = 1;
  int block = 0;    // quantisation block edge; 0 when not quantised
  int scale = -1;   // companion scale tensor of a quantised tensor
  int scales = -1;  // for a scale tensor: the tensor it serves
  int64_t numel() const { return batch * rows * cols; }
};

struct Placement {
  int t = 0, u = 0;
  int64_t r0 = 0, r1 = 0, c0 = 0, c1 = 0, base = 0, ld = 0;
  int tr = 0;
  int64_t rows() const { return r1 - r0; }
  int64_t cols() const { return c1 - c0; }
  int64_t numel() const { return rows() * cols(); }
};

struct Rank {
  std::vector<Local> locals;
  std::vector<Placement> pls;
};

}  // namespace wb

struct wb_layout_t {
  std::vector<wb::Tensor> catalog;
  std::vector<wb::Rank> ranks;
};

namespace wb {

struct Rect {
  int64_t r0, r1, c0, c1;
  int64_t rows() const { return r1 - r0; }
  int64_t cols() const { return c1 - c0; }
  int64_t numel() const { return rows() * cols(); }
};

// One piece of the routing plan: a rectangle of checkpoint tensor t that
// sender s ships to receiver d. In the receive stage (0) s is a trainer rank;
// in the external (1) and internal (2) exchange stages s is a rollout rank that
// forwards bytes it received earlier in the same round.
struct Segment {
  int s, d, t;
  Rect x;
  int src_pl, dst_pl;   // src_pl: the trainer placement (stage 0 only)
  int64_t bytes;
  int64_t send_off = 0, recv_off = 0;  // within the segment's round; recv_off spans all sections
  int round = 0;
  int stage = 0;
  int src_seg = -1;     // exchange stages: the segment whose received bytes are forwarded
  int origin = -1;      // the stage-0 segment the bytes left the trainers in
  int64_t src_off = 0;  // exchange stages: where those bytes sit in the forwarding rank's receive buffer
};

// Wire layout of one stage of one round: per-rank buffer sizes and
// per-(sender, receiver) region offsets and sizes, indexed [s * receivers + d]
// (-1 when the pair is idle). recv_region is an offset in the whole receive
// buffer (the stage's section included).
struct StageWire {
  std::vector<int64_t> send_bytes, recv_bytes;
  std::vector<int64_t> send_region, recv_region, region_bytes;
};

// Stage 0 pairs trainer and rollout ranks; stages 1 and 2 pair rollout ranks.
// A rollout rank's receive buffer holds the three stages' sections in order.
struct RoundWire {
  StageWire st[3];
  std::vector<int64_t> recv_total;
};

// Work item of the copy/cast kernel: a rows x cols block of elements.
// Offsets are bytes from pointer-table entries; strides are in elements.
enum TaskKind : uint8_t {
  TASK_COPY16 = 0,     // byte copy, 16-byte vectors (cols, lds and offsets in bytes)
  TASK_F32_BF16 = 1,   // fp32 -> bf16, 8 elements per vector
  TASK_BF16_F32 = 2,   // bf16 -> fp32, 8 elements per vector
  TASK_SCALAR = 3,     // any supported pair, element by element
  TASK_TRANSPOSE = 4,  // dst[c][r] = cvt(src[r][c]), one LDS tile of up to 64 x 64
  TASK_TRANSPOSE16 = 5,  // 2-byte dst[c][r] = src[r][c], (64..256) rows x 64 cols, in registers
  TASK_TILE = 6,       // 2-byte dst[c][r] = src[r][c], one kTileRows x kTileCols tile through LDS (a launch of its own)
};

// TASK_TILE items run one per workgroup of kTileThreads threads: each thread
// transposes one 8 x 8 sub-tile, so that a wave instruction reads 1 KiB of one
// source row and writes 256 bytes of each of four destination rows.
constexpr int kTileRows = 128, kTileCols = 512;  // of the source block
constexpr int kTileThreads = (kTileRows / 8) * (kTileCols / 8);

struct Task {
  uint64_t src_off, dst_off;
  uint32_t rows, cols;
  uint32_t src_ld, dst_ld;
  uint16_t src_idx, dst_idx;
  uint8_t kind, sdt, ddt, pad0;
  uint32_t pad1;
  uint32_t pad2;
};
static_assert(sizeof(Task) == 48, "Task layout");

// Copy kernel launch. Each launch's range of work items is ordered by class:
// class 0 (the vector kinds) takes 2^s[0] workgroups of kChunkThreads
// threads (a multiple of 64: one wave by default) per item, one per chunk of
// kChunkVecs 16-byte vectors (kChunkPerLane per lane); class 1 (transposes)
// takes 2^shift[1] per item, TASK_TRANSPOSE16 one per kChunkThreads / 64 tiles
// of 64 x 64 and TASK_TRANSPOSE one per 32 x 32 quarter of its tile; class 2
// (element-wise) one workgroup per item. Grids wider than kMaxGridX
// workgroups fold into a second dimension.
#ifndef WB_CHUNK_THREADS
#define WB_CHUNK_THREADS 64
#endif
#ifndef WB_CHUNK_PER_LANE
#define WB_CHUNK_PER_LANE 1
#endif
constexpr int kChunkThreads = WB_CHUNK_THREADS;
constexpr int kChunkPerLane = WB_CHUNK_PER_LANE;
constexpr uint32_t kChunkVecs = uint32_t(kChunkThreads) * kChunkPerLane;
constexpr uint32_t kMaxGridX = 1u << 22;
static_assert(kChunkThreads % 64 == 0 && kChunkThreads <= 256, "copy workgroup size");

inline int task_class(const Task& t) {
  if (t.kind == TASK_TILE) return 3;
  if (t.kind == TASK_TRANSPOSE || t.kind == TASK_TRANSPOSE16) return 1;
  return t.kind == TASK_SCALAR ? 2 : 0;
}

// Workgroups a work item needs (host side of the rule above).
inline uint32_t task_chunks(const Task& t) {
  uint64_t vecs = 0;
  switch (t.kind) {
    case TASK_COPY16: vecs = uint64_t(t.rows) * (t.cols >> 4); break;
    case TASK_F32_BF16: {  // units of 4 elements, 2 kChunkThreads per chunk
      const uint64_t units = uint64_t(t.rows) * (t.cols >> 2), per = 2 * uint64_t(kChunkThreads);
      return static_cast<uint32_t>(units == 0 ? 1 : (units + per - 1) / per);
    }
    case TASK_BF16_F32: vecs = uint64_t(t.rows) * (t.cols >> 3); break;
    case TASK_TRANSPOSE16: {
      const uint32_t per = kChunkThreads / 64, tiles = (t.rows + 63) / 64;
      return (tiles + per - 1) / per;
    }
    case TASK_TRANSPOSE: return 4;
    default: return 1;
  }
  return static_cast<uint32_t>(vecs == 0 ? 1 : (vecs + kChunkVecs - 1) / kChunkVecs);
}

// One launch's range: items of classes 0 and 1 at its start, class 2 after
// them, and log2 of the workgroups per item of classes 0 and 1 (fits its
// longest item); the last tiles items (class 3) go to the tile kernel.
struct TaskSplit {
  uint32_t n[2] = {0, 0};
  uint32_t s[2] = {0, 0};
  uint32_t tiles = 0;
};

// One fp8 destination block and the wire pieces that fill it. Blocks filled by
// a single 16-byte aligned bf16 piece (QB_SINGLE) carry its source address
// here and have no piece-table entry, so the kernel needs no piece lookups
// for them.
struct QBlock {
  uint64_t dst_off;     // bytes from the fp8 tensor to the block origin
  uint64_t src_off;     // QB_SINGLE: bytes from recv_buf to the block's first element
  uint32_t src_ld;      // QB_SINGLE: wire row length in elements
  uint32_t piece0;      // first piece (npieces is 0 for QB_SINGLE blocks)
  uint32_t dst_ld;      // row stride of the fp8 matrix (elements = bytes)
  uint32_t scale_off;   // element index of the block's scale
  uint16_t npieces, dst_idx, scale_idx;
  uint8_t rows_m1, cols_m1;  // block extent minus one (blocks are at most 128 x 128)
  uint8_t flags, pad0;
  uint16_t pad1;
  uint32_t pad2;        // every byte a named member: copies carry zeros, not indeterminate padding
};
static_assert(sizeof(QBlock) == 48, "QBlock layout");

struct QPiece {
  uint64_t src_off;     // bytes from recv_buf to the piece's first element
  uint32_t src_ld;      // wire row length in elements
  uint8_t r0, r1m1, c0, c1m1;  // block-local rectangle [r0, r1m1] x [c0, c1m1]
  uint8_t sdt, pad0;
  uint16_t pad1;
  uint32_t pad2;
};
static_assert(sizeof(QPiece) == 24, "QPiece layout");

// QB_BANDS: a block filled by 2..kMaxBands full-width, aligned bf16 row bands
// (its pieces, sorted by first row); such blocks take the pair path too, each
// row loaded from the band that holds it.
enum QBlockFlags : uint8_t { QB_VEC_STORE = 1, QB_BF16_SOURCE = 2, QB_SINGLE = 4, QB_BANDS = 8 };
constexpr int kMaxBands = 4;
inline bool qblock_pairable(const QBlock& b) { return (b.flags & (QB_SINGLE | QB_BANDS)) != 0; }
inline bool qblock_full_single(const QBlock& b) {
  return (b.flags & QB_SINGLE) && (b.flags & QB_VEC_STORE) && b.rows_m1 == 127 && b.cols_m1 == 127;
}

// The fp8 block kernel runs kQBlockThreads threads per workgroup. Each launch
// range of blocks starts with its full pairs (nfull, even: QB_SINGLE blocks of
// 128 x 128 with 8-byte stores), then the other pairable blocks (QB_SINGLE or
// QB_BANDS) up to npair, each pair taken by one workgroup (horizontal
// neighbours in block order, so one row of the pair is 512 contiguous bytes
// of the wire), 16 rows of 8 columns per thread; the other blocks follow, one
// per workgroup, 8 rows of 8 columns per thread.
constexpr int kQBlockThreads = 256;
inline uint32_t qblock_workgroups(uint32_t n, uint32_t nfull, uint32_t npair) {
  return nfull / 2 + (npair - nfull + 1) / 2 + (n - npair);
}

// A field of a batched diff2 launch: rows x cols values, value at (i, j) the
// sum over k < passes of src[k][i * cols + j] << (16 k); its element 0 is
// entry index base of the output. kind says how its tiles read it.
constexpr int kMaxPasses = 3;
enum DiffKind : uint8_t { DIFF_ELEM = 0, DIFF_VEC = 1, DIFF_FLAT = 2 };
struct DiffField {
  const void* src[kMaxPasses];
  int64_t rows, cols, base;
  int32_t dtype;
  uint8_t kind, passes;
  uint16_t pad;
};
static_assert(sizeof(DiffField) == 56, "DiffField layout");
// One workgroup's share: the tile of field `field` starting at row i0 and
// column (ELEM) or 16-byte vector (VEC, FLAT) j0.
struct DiffTile {
  int32_t field, pad;
  int64_t i0, j0;
};
static_assert(sizeof(DiffTile) == 24, "DiffTile layout");
// A carry table of the probing passes: `mask + 1` slots (a power of two, at
// least twice `capacity`) of two int64, key position + 1 (0 empty) and
// field << 32 | carry as uint32; `count` points to kCarryCounters counters
// whose sum is the number of carries inserted, then a flag set when an
// insert found no free slot within kCarryProbes of its hash. The stencil
// workgroup of tile t stages up to kCarryStage of its carries at
// stage[2 * (t * kCarryStage + k)] (position, packed carry) and their number
// at stage_n[t]; a later launch inserts them.
constexpr int kCarryCounters = 64;
constexpr int kCarryProbes = 256;
constexpr int kCarryStage = 64;
struct CarryTable {
  int64_t* slot;
  unsigned long long* count;
  int64_t* stage;
  int32_t* stage_n;
  int64_t capacity;
  uint64_t mask;
};

// A local tensor of a probed rank and its recombined diff2 entries.
struct ProbeLocal {
  std::string name;
  int dtype = WB_BF16;
  int64_t batch = 1, rows = 1, cols = 1;
  std::unordered_map<int64_t, __int128> z;  // flat index -> sum over passes
};

}  // namespace wb

struct wb_probe_t {
  std::vector<wb::Tensor> catalog;
  std::vector<int64_t> first;  // identifier of element (0, 0) of every tensor
  int64_t end_id = 0;          // one past the last identifier
  int dtype = WB_BF16, bits = 16, nchunks = 0;
  std::vector<wb::ProbeLocal> locals;
};

struct wb_plan_t {
  // global plan
  int n_send = 0, n_recv = 0;
  int node_size = 0;                    // rollout ranks per node; 0: no exchange stages
  std::vector<wb::Segment> segs;
  std::vector<wb::RoundWire> rounds;
  // view of one rank
  int role = WB_SENDER, rank = 0;
  int n_locals = 0;
  int64_t read_bytes = 0, write_bytes = 0;
  int64_t q_read_bytes = 0, q_write_bytes = 0;  // the fp8 launch's share
  int64_t tile_read_bytes = 0, tile_write_bytes = 0;  // the tile launch's share (pack and unpack ranges)
  std::vector<wb::Task> tasks;          // pack or unpack work by round, then forward work by stage and round
  std::vector<wb::TaskSplit> round_split;  // [k]: class sizes of round k's pack/unpack range
  std::vector<wb::TaskSplit> fwd_split[2]; // the same for the forward range of stage 1 + i, round k
  std::vector<wb::QBlock, wb::NoInitAlloc<wb::QBlock>> qblocks;  // grouped by round
  std::vector<wb::QPiece, wb::NoInitAlloc<wb::QPiece>> qpieces;
  std::vector<uint32_t> round_tasks, round_qblocks;  // [k] .. [k + 1] is round k's range
  std::vector<uint32_t> round_qfull;    // [k]: blocks of full pairs at the start of round k's block range (even)
  std::vector<uint32_t> round_qsingle;  // [k]: pairable blocks (full pairs, QB_SINGLE, QB_BANDS) at its start
  std::vector<uint32_t> round_qpieces;  // [2k], [2k + 1]: the piece-table range round k's blocks read
  std::vector<uint32_t> round_fwd[2];   // forward work of exchange stage 1 + i, round k: [k] .. [k + 1]
  int64_t fwd_bytes[2] = {0, 0};        // bytes this rank forwards in each exchange stage (all rounds)
  // copies of the two layouts used for dumps and queries
  wb_layout_t trainer, rollout;
  // device state after wb_plan_upload
  uint8_t* ws = nullptr;
  size_t ws_bytes = 0;
  size_t off_ptrs = 0, off_tasks = 0, off_qblocks = 0, off_qpieces = 0;
  // kPtrSlots pointer tables in the workspace (slot k at off_ptrs + k * (n_locals + 1) * 8),
  // each with its pinned host staging slot, the pointer set it holds, an event
  // recorded after the last work that wrote or read it and that work's stream
  static constexpr int kPtrSlots = 4;
  void* ptr_stage = nullptr;
  void* ptr_copied[kPtrSlots] = {};  // after the staging copy (the pinned slot is free again)
  void* ptr_done[kPtrSlots] = {};    // after the last copy or launches touching the table
  void* ptr_stream[kPtrSlots] = {};  // the stream ptr_done was recorded on
  std::vector<uint64_t> slot_ptrs[kPtrSlots];
  int next_slot = 0;
};

namespace wb {
// layout.cpp
void describe(const wb_model_shapes& m, const wb_parallelism& p, wb_layout_t& out);
void check_placement(const wb_layout_t& L, int rank, const Placement& p);
std::string dump_layout(const wb_layout_t& L);
// plan.cpp
void build_plan(const wb_layout_t& trainer, const wb_layout_t& rollout, int role, int rank, int64_t round_budget,
                int node_size, wb_plan_t& out);
std::string dump_plan(const wb_plan_t& P);
// kernels.hip
// ptrs[1 + u] is local tensor u; work items with index 0 use buf, with index
// kAuxBuffer aux (the second buffer of a forward launch).
constexpr uint16_t kAuxBuffer = 0xFFFF;
// n work items ordered by class, split as in `sp`: the copy kernel's grid
// (the last sp.tiles items excluded: one tile-kernel workgroup each)
void task_grid(uint32_t n, const TaskSplit& sp, uint32_t* gx, uint32_t* gy);
int launch_tasks(const Task* tasks, uint32_t n, const TaskSplit& sp, const uint64_t* ptrs,
                 const void* buf, const void* aux, void* stream);
// n blocks: nfull in full pairs, then pairable ones up to npair, then the rest
int launch_qblocks(const QBlock* blocks, uint32_t n, uint32_t nfull, uint32_t npair, const QPiece* pieces,
                   const uint64_t* ptrs, const void* buf, void* stream);
const char* hip_error_string(int err);
// noalloc.hip: the library's per-GPU scratch array for allocation-free calls
// (its address on the current device, found once per device, and its size)
int scratch_address(void** out, size_t* bytes);
// dev[0] = 0, dev[1 + i] = ptrs[i] for i < n, written by kernels whose
// arguments carry the pointers (no host buffer outlives the call)
int launch_store_table(uint64_t* dev, const void* const* ptrs, int n, void* stream);
// probe.cpp
void probe_init(wb_probe_t& P, const wb_tensor_desc* catalog, int n, int ckpt_dtype);
void probe_record(wb_probe_t& P, int local, int chunk, const int64_t* index, const int64_t* value, int64_t n);
void probe_scan(const wb_probe_t& P, wb_layout_t& out, int rank);
// probe.hip
int launch_make_ids(void* dst, int dtype, int64_t numel, int64_t first_id, int shift, uint32_t mask, void* stream);
int launch_diff2(const void* src, int dtype, int64_t rows, int64_t cols, int64_t* index, int32_t* value,
                 int64_t capacity, unsigned long long* count, void* stream);
// fills f.kind and appends the tiles of field f (index fi) to out
void diff_tiles(int32_t fi, DiffField& f, std::vector<DiffTile>& out);
int launch_diff2_batch(const DiffField* fields, const DiffTile* tiles, int64_t ntiles, int64_t* index, int64_t* value,
                       int64_t capacity, unsigned long long* count, void* stream);
// one carry pass: clears `next` (unless last), runs the stencil over the
// tiles, then (has_in) the carries of `in` at positions the stencil skipped,
// and copies next's carry count to *carries
int launch_diff2_carry(const DiffField* fields, int32_t nfields, const DiffTile* tiles, int64_t ntiles, bool has_in,
                       bool last, const CarryTable& in, const CarryTable& next, int64_t* index, int64_t* value,
                       int64_t capacity, unsigned long long* count, unsigned long long* carries, void* stream);
}  // namespace wb
