// C ABI of libwb (declared in include/wb.h): argument checks, error strings,
// work-table upload and the per-call pointer tables of wb_pack / wb_unpack.
#include <hip/hip_runtime_api.h>

#include <algorithm>
#include <climits>
#include <cstring>
#include <new>
#include <string>

#include "wb_internal.hpp"

namespace {

thread_local std::string g_error;

int set_error(int code, const std::string& msg) {
  g_error = msg;
  return code;
}

template <class F>
int guarded(F&& f) {
  try {
    g_error.clear();
    return f();
  } catch (const wb::Error& e) {
    return set_error(e.code, e.what());
  } catch (const std::bad_alloc&) {
    return set_error(WB_ENOMEM, "host allocation failed");
  } catch (const std::exception& e) {
    return set_error(WB_EINVAL, e.what());
  }
}

int hip_fail(hipError_t e, const char* what) {
  return set_error(WB_EHIP, std::string(what) + ": " + hipGetErrorString(e));
}

int copy_text(const std::string& s, char* buf, size_t cap, size_t* needed) {
  if (needed) *needed = s.size() + 1;
  if (!buf || cap < s.size() + 1) return set_error(WB_ESIZE, "buffer too small for the text");
  std::memcpy(buf, s.c_str(), s.size() + 1);
  return WB_OK;
}

size_t align256(size_t x) { return (x + 255) & ~size_t(255); }

// Refuse a pointer the GPU cannot address (pageable host memory, or an
// address the runtime does not know) and one whose device allocation is
// smaller than what the kernels will touch. Pinned host memory is accepted;
// the runtime does not size it.
int check_extent(const void* p, int64_t bytes, const char* what, int align = 16) {
  if (!p) return set_error(WB_EINVAL, std::string(what) + " is null");
  if (reinterpret_cast<uintptr_t>(p) % align != 0)
    return set_error(WB_EINVAL, std::string(what) + " is not " + std::to_string(align) + "-byte aligned");
  hipPointerAttribute_t attr;
  if (hipPointerGetAttributes(&attr, p) != hipSuccess) {
    (void)hipGetLastError();
    return set_error(WB_EINVAL, std::string(what) + " is not memory the GPU can address (device or pinned host)");
  }
  if (attr.type == hipMemoryTypeUnregistered)
    return set_error(WB_EINVAL, std::string(what) + " is pageable host memory: the kernels need device or pinned host memory");
  hipDeviceptr_t base = nullptr;
  size_t size = 0;
  if (hipMemGetAddressRange(&base, &size, const_cast<void*>(p)) != hipSuccess) {
    (void)hipGetLastError();
    return WB_OK;
  }
  const uintptr_t end = reinterpret_cast<uintptr_t>(base) + size;
  if (reinterpret_cast<uintptr_t>(p) + uint64_t(bytes) > end)
    return set_error(WB_EINVAL, std::string(what) + " is smaller than the plan needs (" + std::to_string(bytes) + " bytes)");
  return WB_OK;
}

// Stage a new pointer table into the workspace when the pointers changed.
// The device pointer table of `ptrs` for work enqueued on `stream`. A slot
// that already holds the set is reused; otherwise the least recently staged
// slot is restaged. Either way, work on another stream that last touched the
// slot is waited for on `stream` (no host wait), so a table is never
// overwritten while read, nor read before its copy; the host waits only for
// the staging copy of the slot it refills (issued kPtrSlots new sets ago).
// Returns the slot, or -1 with the error set.
int table_slot(wb_plan_t* P, const std::vector<uint64_t>& ptrs, void* stream) {
  hipError_t e;
  int k = -1;
  for (int i = 0; i < wb_plan_t::kPtrSlots && k < 0; ++i)
    if (P->slot_ptrs[i] == ptrs) k = i;
  const bool restage = k < 0;
  if (restage) {
    k = P->next_slot;
    P->next_slot = (k + 1) % wb_plan_t::kPtrSlots;
  }
  if ((restage || P->ptr_stream[k] != stream) &&
      (e = hipStreamWaitEvent(static_cast<hipStream_t>(stream), static_cast<hipEvent_t>(P->ptr_done[k]), 0)) !=
          hipSuccess)
    return hip_fail(e, "hipStreamWaitEvent"), -1;
  if (restage) {
    const size_t n = ptrs.size();
    if ((e = hipEventSynchronize(static_cast<hipEvent_t>(P->ptr_copied[k]))) != hipSuccess)
      return hip_fail(e, "hipEventSynchronize"), -1;
    uint64_t* stage = static_cast<uint64_t*>(P->ptr_stage) + k * n;
    std::memcpy(stage, ptrs.data(), n * sizeof(uint64_t));
    P->slot_ptrs[k].clear();  // holds nothing until the copy is enqueued
    if ((e = hipMemcpyAsync(P->ws + P->off_ptrs + k * n * sizeof(uint64_t), stage, n * sizeof(uint64_t),
                            hipMemcpyHostToDevice, static_cast<hipStream_t>(stream))) != hipSuccess)
      return hip_fail(e, "hipMemcpyAsync (pointer table)"), -1;
    if ((e = hipEventRecord(static_cast<hipEvent_t>(P->ptr_copied[k]), static_cast<hipStream_t>(stream))) !=
        hipSuccess)
      return hip_fail(e, "hipEventRecord"), -1;
    P->slot_ptrs[k] = ptrs;
  }
  return k;
}

// Record that the work just enqueued on stream touched slot k.
int table_done(wb_plan_t* P, int k, void* stream) {
  const hipError_t e = hipEventRecord(static_cast<hipEvent_t>(P->ptr_done[k]), static_cast<hipStream_t>(stream));
  if (e != hipSuccess) return hip_fail(e, "hipEventRecord");
  P->ptr_stream[k] = stream;
  return WB_OK;
}

const uint64_t* table_at(const wb_plan_t* P, int k) {
  return reinterpret_cast<const uint64_t*>(P->ws + P->off_ptrs) + size_t(k) * (P->n_locals + 1);
}

int64_t local_bytes(const wb::Local& l) { return l.numel() * wb::dtype_bytes(l.dtype); }

const wb::Rank& rank_of(const wb_plan_t* P) {
  return P->role == WB_SENDER ? P->trainer.ranks[P->rank] : P->rollout.ranks[P->rank];
}

}  // namespace

extern "C" {

const char* wb_last_error(void) { return g_error.c_str(); }
const char* wb_version(void) { return "wb 0.1.0 (gfx950)"; }

int wb_describe_layout(const wb_model_shapes* shapes, const wb_parallelism* par, wb_layout_t** out) {
  return guarded([&]() -> int {
    if (!shapes || !par || !out) return set_error(WB_EINVAL, "null argument");
    *out = nullptr;
    auto* L = new wb_layout_t;
    try {
      wb::describe(*shapes, *par, *L);
    } catch (...) {
      delete L;
      throw;
    }
    *out = L;
    return WB_OK;
  });
}

int wb_layout_create(const wb_tensor_desc* catalog, int32_t num_tensors, int32_t num_ranks, wb_layout_t** out) {
  return guarded([&]() -> int {
    if (!out || (num_tensors > 0 && !catalog) || num_tensors < 0 || num_ranks < 1)
      return set_error(WB_EINVAL, "bad catalog or rank count");
    *out = nullptr;
    auto* L = new wb_layout_t;
    for (int i = 0; i < num_tensors; ++i) {
      if (!catalog[i].name || catalog[i].rows < 1 || catalog[i].cols < 1) {
        delete L;
        return set_error(WB_EINVAL, "catalog tensors need a name and positive shape");
      }
      L->catalog.push_back({catalog[i].name, catalog[i].rows, catalog[i].cols});
    }
    L->ranks.resize(num_ranks);
    *out = L;
    return WB_OK;
  });
}

int wb_layout_add_local(wb_layout_t* L, int32_t rank, const char* name, int32_t dtype, int64_t batch, int64_t rows,
                        int64_t cols, int32_t quant_block, int32_t* out_index) {
  return guarded([&]() -> int {
    if (!L || !name || rank < 0 || rank >= static_cast<int>(L->ranks.size()))
      return set_error(WB_EINVAL, "bad layout, rank or name");
    if (batch < 1 || rows < 1 || cols < 1) return set_error(WB_EINVAL, "local tensor shape must be positive");
    if (dtype != WB_F32 && dtype != WB_BF16 && dtype != WB_F8E4M3) return set_error(WB_EINVAL, "bad dtype");
    if ((dtype == WB_F8E4M3) != (quant_block > 0))
      return set_error(WB_EUNSUPPORTED, "fp8 local tensors need a quant_block (and only they take one)");
    if (quant_block > 128) return set_error(WB_EUNSUPPORTED, "quant_block above 128");
    wb::Rank& R = L->ranks[rank];
    const int u = static_cast<int>(R.locals.size());
    wb::Local l;
    l.name = name;
    l.dtype = dtype;
    l.batch = batch;
    l.rows = rows;
    l.cols = cols;
    if (quant_block > 0) {
      l.block = quant_block;
      l.scale = u + 1;
      R.locals.push_back(l);
      wb::Local s;
      s.name = std::string(name) + "_scale";
      s.dtype = WB_F32;
      s.batch = batch;
      s.rows = (rows + quant_block - 1) / quant_block;
      s.cols = (cols + quant_block - 1) / quant_block;
      s.scales = u;
      R.locals.push_back(s);
    } else {
      R.locals.push_back(l);
    }
    if (out_index) *out_index = u;
    return WB_OK;
  });
}

int wb_layout_add_placement(wb_layout_t* L, int32_t rank, const wb_placement* p) {
  return guarded([&]() -> int {
    if (!L || !p) return set_error(WB_EINVAL, "null argument");
    wb::Placement q;
    q.t = p->t;
    q.u = p->u;
    q.r0 = p->r0;
    q.r1 = p->r1;
    q.c0 = p->c0;
    q.c1 = p->c1;
    q.base = p->base;
    q.ld = p->ld;
    q.tr = p->transposed;
    wb::check_placement(*L, rank, q);
    L->ranks[rank].pls.push_back(q);
    return WB_OK;
  });
}

int wb_layout_num_ranks(const wb_layout_t* L, int32_t* out) {
  if (!L || !out) return set_error(WB_EINVAL, "null argument");
  *out = static_cast<int32_t>(L->ranks.size());
  return WB_OK;
}

int wb_layout_num_tensors(const wb_layout_t* L, int32_t* out) {
  if (!L || !out) return set_error(WB_EINVAL, "null argument");
  *out = static_cast<int32_t>(L->catalog.size());
  return WB_OK;
}

int wb_layout_tensor(const wb_layout_t* L, int32_t t, wb_tensor_desc* out) {
  if (!L || !out || t < 0 || t >= static_cast<int>(L->catalog.size())) return set_error(WB_EINVAL, "bad tensor index");
  out->name = L->catalog[t].name.c_str();
  out->rows = L->catalog[t].rows;
  out->cols = L->catalog[t].cols;
  return WB_OK;
}

int wb_layout_num_locals(const wb_layout_t* L, int32_t rank, int32_t* out) {
  if (!L || !out || rank < 0 || rank >= static_cast<int>(L->ranks.size())) return set_error(WB_EINVAL, "bad rank");
  *out = static_cast<int32_t>(L->ranks[rank].locals.size());
  return WB_OK;
}

int wb_layout_local(const wb_layout_t* L, int32_t rank, int32_t index, wb_local_info* out) {
  if (!L || !out || rank < 0 || rank >= static_cast<int>(L->ranks.size())) return set_error(WB_EINVAL, "bad rank");
  const wb::Rank& R = L->ranks[rank];
  if (index < 0 || index >= static_cast<int>(R.locals.size())) return set_error(WB_EINVAL, "bad local index");
  const wb::Local& l = R.locals[index];
  out->name = l.name.c_str();
  out->dtype = l.dtype;
  out->quant_block = l.block;
  out->batch = l.batch;
  out->rows = l.rows;
  out->cols = l.cols;
  out->scale_index = l.scale;
  out->scales_index = l.scales;
  return WB_OK;
}

int wb_layout_num_placements(const wb_layout_t* L, int32_t rank, int32_t* out) {
  if (!L || !out || rank < 0 || rank >= static_cast<int>(L->ranks.size())) return set_error(WB_EINVAL, "bad rank");
  *out = static_cast<int32_t>(L->ranks[rank].pls.size());
  return WB_OK;
}

int wb_layout_placement(const wb_layout_t* L, int32_t rank, int32_t index, wb_placement* out) {
  if (!L || !out || rank < 0 || rank >= static_cast<int>(L->ranks.size())) return set_error(WB_EINVAL, "bad rank");
  const wb::Rank& R = L->ranks[rank];
  if (index < 0 || index >= static_cast<int>(R.pls.size())) return set_error(WB_EINVAL, "bad placement index");
  const wb::Placement& p = R.pls[index];
  *out = wb_placement{p.t, p.u, p.r0, p.r1, p.c0, p.c1, p.base, p.ld, p.tr, 0};
  return WB_OK;
}

int wb_layout_dump(const wb_layout_t* L, char* buf, size_t cap, size_t* needed) {
  return guarded([&]() -> int {
    if (!L) return set_error(WB_EINVAL, "null layout");
    return copy_text(wb::dump_layout(*L), buf, cap, needed);
  });
}

void wb_layout_destroy(wb_layout_t* L) { delete L; }

int wb_plan_exchange(const wb_layout_t* trainer, const wb_layout_t* rollout, int32_t role, int32_t rank,
                     int64_t round_budget, int32_t node_size, wb_plan_t** out) {
  return guarded([&]() -> int {
    if (!trainer || !rollout || !out) return set_error(WB_EINVAL, "null argument");
    if (round_budget < 0) return set_error(WB_EINVAL, "round budget must be >= 0");
    if (node_size < 0) return set_error(WB_EINVAL, "node size must be >= 0");
    *out = nullptr;
    auto* P = new wb_plan_t;
    try {
      wb::build_plan(*trainer, *rollout, role, rank, round_budget, node_size, *P);
      P->trainer = *trainer;
      P->rollout = *rollout;
      const wb::Rank& R = rank_of(P);
      if (R.locals.size() + 1 > 65535) wb::fail(WB_EUNSUPPORTED, "too many local tensors on one rank");
      if (P->tasks.size() > 0x7FFFFFFF || P->qblocks.size() > 0x7FFFFFFF)
        wb::fail(WB_EUNSUPPORTED, "too many work items for one launch");
    } catch (...) {
      delete P;
      throw;
    }
    *out = P;
    return WB_OK;
  });
}

int wb_plan_rounds(const wb_layout_t* trainer, const wb_layout_t* rollout, int32_t role, int32_t rank,
                   int64_t round_budget, wb_plan_t** out) {
  return wb_plan_exchange(trainer, rollout, role, rank, round_budget, 0, out);
}

int wb_plan(const wb_layout_t* trainer, const wb_layout_t* rollout, int32_t role, int32_t rank, wb_plan_t** out) {
  return wb_plan_exchange(trainer, rollout, role, rank, 0, 0, out);
}

int wb_plan_node_size(const wb_plan_t* P, int32_t* out) {
  if (!P || !out) return set_error(WB_EINVAL, "null argument");
  *out = P->node_size;
  return WB_OK;
}

int wb_plan_num_segments(const wb_plan_t* P, int64_t* out) {
  if (!P || !out) return set_error(WB_EINVAL, "null argument");
  *out = static_cast<int64_t>(P->segs.size());
  return WB_OK;
}

int wb_plan_num_rounds(const wb_plan_t* P, int32_t* out) {
  if (!P || !out) return set_error(WB_EINVAL, "null argument");
  *out = static_cast<int32_t>(P->rounds.size());
  return WB_OK;
}

static int64_t rank_bytes(const wb_plan_t* P, size_t k, int role, int rank) {
  return role == WB_SENDER ? P->rounds[k].st[0].send_bytes[rank] : P->rounds[k].recv_total[rank];
}

int wb_plan_round_buffer_bytes(const wb_plan_t* P, int32_t round, int64_t* out) {
  if (!P || !out) return set_error(WB_EINVAL, "null argument");
  if (round < 0 || round >= static_cast<int>(P->rounds.size())) return set_error(WB_EINVAL, "round out of range");
  *out = rank_bytes(P, round, P->role, P->rank);
  return WB_OK;
}

int wb_plan_buffer_bytes(const wb_plan_t* P, int64_t* out) {
  if (!P || !out) return set_error(WB_EINVAL, "null argument");
  int64_t m = 0;
  for (size_t k = 0; k < P->rounds.size(); ++k) m = std::max(m, rank_bytes(P, k, P->role, P->rank));
  *out = m;
  return WB_OK;
}

int wb_plan_rank_buffer_bytes(const wb_plan_t* P, int32_t role, int32_t rank, int64_t* out) {
  if (!P || !out) return set_error(WB_EINVAL, "null argument");
  if (!((role == WB_SENDER && rank >= 0 && rank < P->n_send) || (role == WB_RECEIVER && rank >= 0 && rank < P->n_recv)))
    return set_error(WB_EINVAL, "bad role or rank");
  int64_t m = 0;
  for (size_t k = 0; k < P->rounds.size(); ++k) m = std::max(m, rank_bytes(P, k, role, rank));
  *out = m;
  return WB_OK;
}

int wb_plan_num_peers(const wb_plan_t* P, int32_t* out) {
  if (!P || !out) return set_error(WB_EINVAL, "null argument");
  const wb::StageWire& W = P->rounds[0].st[0];
  int n = 0;
  const int others = P->role == WB_SENDER ? P->n_recv : P->n_send;
  for (int o = 0; o < others; ++o) {
    const size_t k = P->role == WB_SENDER ? size_t(P->rank) * P->n_recv + o : size_t(o) * P->n_recv + P->rank;
    n += W.send_region[k] >= 0;
  }
  *out = n;
  return WB_OK;
}

int wb_plan_peer(const wb_plan_t* P, int32_t i, int32_t* peer, int64_t* offset, int64_t* bytes) {
  if (!P || !peer || !offset || !bytes) return set_error(WB_EINVAL, "null argument");
  const wb::StageWire& W = P->rounds[0].st[0];
  const int others = P->role == WB_SENDER ? P->n_recv : P->n_send;
  int n = 0;
  for (int o = 0; o < others; ++o) {
    const size_t k = P->role == WB_SENDER ? size_t(P->rank) * P->n_recv + o : size_t(o) * P->n_recv + P->rank;
    if (W.send_region[k] < 0) continue;
    if (n++ == i) {
      *peer = o;
      *offset = P->role == WB_SENDER ? W.send_region[k] : W.recv_region[k];
      *bytes = W.region_bytes[k];
      return WB_OK;
    }
  }
  return set_error(WB_EINVAL, "peer index out of range");
}

int wb_plan_round_region(const wb_plan_t* P, int32_t round, int32_t s, int32_t d, int64_t* send_offset,
                         int64_t* recv_offset, int64_t* bytes) {
  if (!P || !send_offset || !recv_offset || !bytes) return set_error(WB_EINVAL, "null argument");
  if (round < 0 || round >= static_cast<int>(P->rounds.size())) return set_error(WB_EINVAL, "round out of range");
  if (s < 0 || s >= P->n_send || d < 0 || d >= P->n_recv) return set_error(WB_EINVAL, "rank out of range");
  const wb::StageWire& W = P->rounds[round].st[0];
  const size_t k = size_t(s) * P->n_recv + d;
  *send_offset = W.send_region[k] < 0 ? 0 : W.send_region[k];
  *recv_offset = W.recv_region[k] < 0 ? 0 : W.recv_region[k];
  *bytes = W.region_bytes[k];
  return WB_OK;
}

int wb_plan_stage_region(const wb_plan_t* P, int32_t round, int32_t stage, int32_t s, int32_t d,
                         int64_t* send_offset, int64_t* recv_offset, int64_t* bytes) {
  if (!P || !send_offset || !recv_offset || !bytes) return set_error(WB_EINVAL, "null argument");
  if (stage == 0) return wb_plan_round_region(P, round, s, d, send_offset, recv_offset, bytes);
  if (stage != 1 && stage != 2) return set_error(WB_EINVAL, "stage must be 0, 1 or 2");
  if (round < 0 || round >= static_cast<int>(P->rounds.size())) return set_error(WB_EINVAL, "round out of range");
  if (s < 0 || s >= P->n_recv || d < 0 || d >= P->n_recv) return set_error(WB_EINVAL, "rank out of range");
  const wb::StageWire& W = P->rounds[round].st[stage];
  const size_t k = size_t(s) * P->n_recv + d;
  *send_offset = W.send_region[k] < 0 ? 0 : W.send_region[k];
  *recv_offset = W.recv_region[k] < 0 ? 0 : W.recv_region[k];
  *bytes = W.region_bytes[k];
  return WB_OK;
}

int wb_plan_segment(const wb_plan_t* P, int64_t i, wb_segment_info* out) {
  if (!P || !out) return set_error(WB_EINVAL, "null argument");
  if (i < 0 || i >= static_cast<int64_t>(P->segs.size())) return set_error(WB_EINVAL, "segment index out of range");
  const wb::Segment& g = P->segs[i];
  *out = wb_segment_info{g.s, g.d, g.t, g.stage, g.round, g.src_pl, g.dst_pl, 0, g.x.r0, g.x.r1, g.x.c0, g.x.c1,
                         g.send_off, g.recv_off, g.src_off, g.origin, g.bytes};
  return WB_OK;
}

int wb_plan_forward_bytes(const wb_plan_t* P, int32_t round, int32_t stage, int64_t* out) {
  if (!P || !out) return set_error(WB_EINVAL, "null argument");
  if (stage != 1 && stage != 2) return set_error(WB_EINVAL, "stage must be 1 or 2");
  if (round < -1 || round >= static_cast<int>(P->rounds.size())) return set_error(WB_EINVAL, "round out of range");
  int64_t m = 0;
  if (P->role == WB_RECEIVER)
    for (size_t k = 0; k < P->rounds.size(); ++k)
      if (round < 0 || static_cast<int>(k) == round) m = std::max(m, P->rounds[k].st[stage].send_bytes[P->rank]);
  *out = m;
  return WB_OK;
}

int wb_plan_region(const wb_plan_t* P, int32_t s, int32_t d, int64_t* send_offset, int64_t* recv_offset,
                   int64_t* bytes) {
  return wb_plan_round_region(P, 0, s, d, send_offset, recv_offset, bytes);
}

int wb_plan_num_local_tensors(const wb_plan_t* P, int32_t* out) {
  if (!P || !out) return set_error(WB_EINVAL, "null argument");
  *out = P->n_locals;
  return WB_OK;
}

int wb_plan_local_tensor(const wb_plan_t* P, int32_t i, int32_t* dtype, int64_t* numel) {
  if (!P || !dtype || !numel) return set_error(WB_EINVAL, "null argument");
  if (i < 0 || i >= P->n_locals) return set_error(WB_EINVAL, "local tensor index out of range");
  const wb::Local& l = rank_of(P).locals[i];
  *dtype = l.dtype;
  *numel = l.numel();
  return WB_OK;
}

static void workspace_layout(const wb_plan_t* P, size_t* ptrs, size_t* tasks, size_t* qb, size_t* qp, size_t* total) {
  size_t off = 0;
  *ptrs = off;
  off = align256(off + wb_plan_t::kPtrSlots * sizeof(uint64_t) * (P->n_locals + 1));
  *tasks = off;
  off = align256(off + sizeof(wb::Task) * P->tasks.size());
  *qb = off;
  off = align256(off + sizeof(wb::QBlock) * P->qblocks.size());
  *qp = off;
  off = align256(off + sizeof(wb::QPiece) * P->qpieces.size());
  *total = off;
}

int wb_plan_workspace_bytes(const wb_plan_t* P, int64_t* out) {
  if (!P || !out) return set_error(WB_EINVAL, "null argument");
  size_t a, b, c, d, total;
  workspace_layout(P, &a, &b, &c, &d, &total);
  *out = static_cast<int64_t>(total);
  return WB_OK;
}

int wb_plan_traffic_bytes(const wb_plan_t* P, int64_t* read_bytes, int64_t* write_bytes) {
  if (!P || !read_bytes || !write_bytes) return set_error(WB_EINVAL, "null argument");
  *read_bytes = P->read_bytes;
  *write_bytes = P->write_bytes;
  return WB_OK;
}

int wb_plan_kernel_traffic(const wb_plan_t* P, int32_t launch, int64_t* read_bytes, int64_t* write_bytes) {
  if (!P || !read_bytes || !write_bytes || launch < 0 || launch > 4) return set_error(WB_EINVAL, "bad argument");
  if (launch == 2 || launch == 3) {
    *read_bytes = *write_bytes = P->fwd_bytes[launch - 2];
  } else if (launch == 4) {
    *read_bytes = P->tile_read_bytes;
    *write_bytes = P->tile_write_bytes;
  } else if (launch == 1) {
    *read_bytes = P->q_read_bytes;
    *write_bytes = P->q_write_bytes;
  } else {
    *read_bytes = P->read_bytes - P->q_read_bytes - P->tile_read_bytes;
    *write_bytes = P->write_bytes - P->q_write_bytes - P->tile_write_bytes;
  }
  return WB_OK;
}

int wb_plan_work_counts(const wb_plan_t* P, int64_t* tasks, int64_t* blocks, int64_t* pieces) {
  if (!P || !tasks || !blocks || !pieces) return set_error(WB_EINVAL, "null argument");
  *tasks = static_cast<int64_t>(P->tasks.size());
  *blocks = static_cast<int64_t>(P->qblocks.size());
  *pieces = static_cast<int64_t>(P->qpieces.size());
  return WB_OK;
}

int wb_plan_work_digest(const wb_plan_t* P, uint64_t* out) {
  if (!P || !out) return set_error(WB_EINVAL, "null argument");
  uint64_t h = 1469598103934665603ull;
  auto add = [&h](const void* p, size_t n) {
    const unsigned char* c = static_cast<const unsigned char*>(p);
    for (size_t i = 0; i < n; ++i) h = (h ^ c[i]) * 1099511628211ull;
  };
  auto vec = [&](const auto& v) {
    const uint64_t n = v.size();
    add(&n, sizeof n);
    if (n) add(v.data(), n * sizeof(v[0]));
  };
  vec(P->tasks);
  vec(P->qblocks);
  vec(P->qpieces);
  vec(P->round_tasks);
  vec(P->round_qblocks);
  vec(P->round_qfull);
  vec(P->round_qsingle);
  vec(P->round_qpieces);
  for (int st = 0; st < 2; ++st) vec(P->round_fwd[st]);
  vec(P->round_split);
  for (int st = 0; st < 2; ++st) vec(P->fwd_split[st]);
  const int64_t v[10] = {P->n_locals,         P->read_bytes,       P->write_bytes,  P->q_read_bytes, P->q_write_bytes,
                         P->tile_read_bytes,  P->tile_write_bytes, P->fwd_bytes[0], P->fwd_bytes[1], P->role};
  add(v, sizeof v);
  *out = h;
  return WB_OK;
}

int wb_plan_launch_grid(const wb_plan_t* P, int32_t launch, int32_t round, uint32_t* gx, uint32_t* gy,
                        uint32_t* threads) {
  if (!P || !gx || !gy || !threads) return set_error(WB_EINVAL, "null argument");
  if (launch < 0 || launch > 4) return set_error(WB_EINVAL, "launch must be 0..4");
  if (round < 0 || round >= static_cast<int>(P->rounds.size())) return set_error(WB_EINVAL, "round out of range");
  *gx = *gy = 0;
  *threads = launch == 1 ? wb::kQBlockThreads : launch == 4 ? wb::kTileThreads : wb::kChunkThreads;
  if (launch == 4) {
    if (P->round_split.size() == P->rounds.size() && P->round_split[round].tiles)
      *gx = P->round_split[round].tiles, *gy = 1;
    return WB_OK;
  }
  if (launch == 1) {
    const uint32_t n = P->round_qblocks[round + 1] - P->round_qblocks[round];
    if (n) *gx = wb::qblock_workgroups(n, P->round_qfull[round], P->round_qsingle[round]), *gy = 1;
    return WB_OK;
  }
  const std::vector<uint32_t>& r = launch == 0 ? P->round_tasks : P->round_fwd[launch - 2];
  const std::vector<wb::TaskSplit>& c = launch == 0 ? P->round_split : P->fwd_split[launch - 2];
  if (r.size() != P->rounds.size() + 1 || c.size() != P->rounds.size()) return WB_OK;
  const uint32_t n = r[round + 1] - r[round];
  if (n) wb::task_grid(n, c[round], gx, gy);
  return WB_OK;
}

int wb_plan_dump(const wb_plan_t* P, char* buf, size_t cap, size_t* needed) {
  return guarded([&]() -> int {
    if (!P) return set_error(WB_EINVAL, "null plan");
    return copy_text(wb::dump_plan(*P), buf, cap, needed);
  });
}

int wb_plan_upload(wb_plan_t* P, void* workspace, size_t bytes, void* stream) {
  return guarded([&]() -> int {
    if (!P || !workspace) return set_error(WB_EINVAL, "null argument");
    if (reinterpret_cast<uintptr_t>(workspace) % 256 != 0) return set_error(WB_EINVAL, "workspace must be 256-byte aligned");
    size_t total;
    workspace_layout(P, &P->off_ptrs, &P->off_tasks, &P->off_qblocks, &P->off_qpieces, &total);
    if (bytes < total) return set_error(WB_EINVAL, "workspace smaller than wb_plan_workspace_bytes");
    int rc = check_extent(workspace, static_cast<int64_t>(total), "workspace");
    if (rc != WB_OK) return rc;
    hipStream_t st = static_cast<hipStream_t>(stream);
    auto* ws = static_cast<uint8_t*>(workspace);
    hipError_t e;
    if (!P->tasks.empty() &&
        (e = hipMemcpyAsync(ws + P->off_tasks, P->tasks.data(), sizeof(wb::Task) * P->tasks.size(),
                            hipMemcpyHostToDevice, st)) != hipSuccess)
      return hip_fail(e, "hipMemcpyAsync (tasks)");
    if (!P->qblocks.empty() &&
        (e = hipMemcpyAsync(ws + P->off_qblocks, P->qblocks.data(), sizeof(wb::QBlock) * P->qblocks.size(),
                            hipMemcpyHostToDevice, st)) != hipSuccess)
      return hip_fail(e, "hipMemcpyAsync (fp8 blocks)");
    if (!P->qpieces.empty() &&
        (e = hipMemcpyAsync(ws + P->off_qpieces, P->qpieces.data(), sizeof(wb::QPiece) * P->qpieces.size(),
                            hipMemcpyHostToDevice, st)) != hipSuccess)
      return hip_fail(e, "hipMemcpyAsync (fp8 pieces)");
    for (int k = 0; k < wb_plan_t::kPtrSlots; ++k) {
      for (void** ev : {&P->ptr_copied[k], &P->ptr_done[k]}) {
        if (*ev) continue;
        hipEvent_t h;
        if ((e = hipEventCreateWithFlags(&h, hipEventDisableTiming)) != hipSuccess)
          return hip_fail(e, "hipEventCreateWithFlags");
        *ev = h;
      }
    }
    if (!P->ptr_stage) {
      const size_t stage_bytes = wb_plan_t::kPtrSlots * sizeof(uint64_t) * (P->n_locals + 1);
      if ((e = hipHostMalloc(&P->ptr_stage, stage_bytes, hipHostMallocDefault)) != hipSuccess) {
        P->ptr_stage = nullptr;
        return hip_fail(e, "hipHostMalloc (pointer staging)");
      }
    }
    // the host tables must stay valid until the copies above have run
    if ((e = hipStreamSynchronize(st)) != hipSuccess) return hip_fail(e, "hipStreamSynchronize");
    P->ws = ws;
    P->ws_bytes = bytes;
    for (int k = 0; k < wb_plan_t::kPtrSlots; ++k) {
      P->slot_ptrs[k].clear();
      P->ptr_stream[k] = stream;  // the new workspace's tables have not been touched yet
    }
    P->next_slot = 0;
    return WB_OK;
  });
}

// One round of a pack (sender) or unpack (receiver): check the pointers, stage
// the local-tensor table when it changed, launch the round's work items.
static int run_round(wb_plan_t* P, int round, const void* const* locals, const void* buf, void* stream, int role) {
  if (P->role != role)
    return set_error(WB_EINVAL, role == WB_SENDER ? "packing needs a sender plan" : "unpacking needs a receiver plan");
  if (!P->ws) return set_error(WB_EINVAL, "plan not uploaded (wb_plan_upload)");
  if (round < 0 || round >= static_cast<int>(P->rounds.size())) return set_error(WB_EINVAL, "round out of range");
  if (!locals && P->n_locals > 0) return set_error(WB_EINVAL, "local tensor pointer array is null");
  const wb::Rank& R = rank_of(P);
  int rc = check_extent(buf, rank_bytes(P, round, P->role, P->rank), role == WB_SENDER ? "send_buf" : "recv_buf");
  if (rc != WB_OK) return rc;
  std::vector<uint64_t> ptrs(P->n_locals + 1, 0);
  for (int i = 0; i < P->n_locals; ++i) ptrs[i + 1] = reinterpret_cast<uint64_t>(locals[i]);
  bool known = false;
  for (const auto& v : P->slot_ptrs) known = known || v == ptrs;
  if (!known) {
    for (int i = 0; rc == WB_OK && i < P->n_locals; ++i)
      rc = check_extent(locals[i], local_bytes(R.locals[i]), ("local tensor " + std::to_string(i)).c_str());
    if (rc != WB_OK) return rc;
  }
  const int slot = table_slot(P, ptrs, stream);
  if (slot < 0) return WB_EHIP;
  const uint64_t* table = table_at(P, slot);
  const auto* tasks = reinterpret_cast<const wb::Task*>(P->ws + P->off_tasks);
  int e = wb::launch_tasks(tasks + P->round_tasks[round], P->round_tasks[round + 1] - P->round_tasks[round],
                           P->round_split[round], table, buf, nullptr, stream);
  if (e != 0) return set_error(WB_EHIP, std::string("copy launch: ") + wb::hip_error_string(e));
  const auto* blocks = reinterpret_cast<const wb::QBlock*>(P->ws + P->off_qblocks);
  e = wb::launch_qblocks(blocks + P->round_qblocks[round], P->round_qblocks[round + 1] - P->round_qblocks[round],
                         P->round_qfull[round], P->round_qsingle[round], reinterpret_cast<const wb::QPiece*>(P->ws + P->off_qpieces), table,
                         buf, stream);
  if (e != 0) return set_error(WB_EHIP, std::string("fp8 launch: ") + wb::hip_error_string(e));
  return table_done(P, slot, stream);
}

int wb_pack_round(wb_plan_t* P, int32_t round, const void* const* src_ptrs, void* send_buf, void* stream) {
  return guarded([&]() -> int {
    if (!P) return set_error(WB_EINVAL, "null plan");
    return run_round(P, round, src_ptrs, send_buf, stream, WB_SENDER);
  });
}

int wb_unpack_round(wb_plan_t* P, int32_t round, const void* recv_buf, void* const* dst_ptrs, void* stream) {
  return guarded([&]() -> int {
    if (!P) return set_error(WB_EINVAL, "null plan");
    return run_round(P, round, const_cast<const void* const*>(dst_ptrs), recv_buf, stream, WB_RECEIVER);
  });
}

int wb_forward_round(wb_plan_t* P, int32_t round, int32_t stage, const void* recv_buf, void* fwd_buf, void* stream) {
  return guarded([&]() -> int {
    if (!P) return set_error(WB_EINVAL, "null plan");
    if (P->role != WB_RECEIVER) return set_error(WB_EINVAL, "forwarding needs a receiver plan");
    if (!P->ws) return set_error(WB_EINVAL, "plan not uploaded (wb_plan_upload)");
    if (round < 0 || round >= static_cast<int>(P->rounds.size())) return set_error(WB_EINVAL, "round out of range");
    if (stage != 1 && stage != 2) return set_error(WB_EINVAL, "stage must be 1 (external) or 2 (internal)");
    const uint32_t a = P->round_fwd[stage - 1][round], b = P->round_fwd[stage - 1][round + 1];
    if (a == b) return WB_OK;
    int rc = check_extent(recv_buf, P->rounds[round].recv_total[P->rank], "recv_buf");
    if (rc == WB_OK) rc = check_extent(fwd_buf, P->rounds[round].st[stage].send_bytes[P->rank], "fwd_buf");
    if (rc != WB_OK) return rc;
    // forwarding reads only the two buffers, never the local-tensor table
    const auto* table = reinterpret_cast<const uint64_t*>(P->ws + P->off_ptrs);
    const auto* tasks = reinterpret_cast<const wb::Task*>(P->ws + P->off_tasks);
    const int e = wb::launch_tasks(tasks + a, b - a, P->fwd_split[stage - 1][round], table,
                                   recv_buf, fwd_buf, stream);
    if (e != 0) return set_error(WB_EHIP, std::string("forward launch: ") + wb::hip_error_string(e));
    return WB_OK;
  });
}

int wb_unpack_round_noalloc(wb_plan_t* P, int32_t round, const void* recv_buf, void* const* dst_ptrs, void* stream) {
  return guarded([&]() -> int {
    if (!P) return set_error(WB_EINVAL, "null plan");
    if (P->role != WB_RECEIVER) return set_error(WB_EINVAL, "unpacking needs a receiver plan");
    if (round < 0 || round >= static_cast<int>(P->rounds.size())) return set_error(WB_EINVAL, "round out of range");
    // the round's tables in the scratch array: [pointer table | tasks | blocks | pieces]
    const uint32_t t0 = P->round_tasks[round], t1 = P->round_tasks[round + 1];
    const uint32_t b0 = P->round_qblocks[round], b1 = P->round_qblocks[round + 1];
    const uint32_t q0 = P->round_qpieces[2 * round], q1 = P->round_qpieces[2 * round + 1];
    const size_t off_tasks = align256(sizeof(uint64_t) * (P->n_locals + 1));
    const size_t off_blocks = align256(off_tasks + sizeof(wb::Task) * (t1 - t0));
    const size_t off_pieces = align256(off_blocks + sizeof(wb::QBlock) * (b1 - b0));
    const size_t need = off_pieces + sizeof(wb::QPiece) * (q1 - q0);
    void* base = nullptr;
    size_t cap = 0;
    hipError_t e = static_cast<hipError_t>(wb::scratch_address(&base, &cap));
    if (e != hipSuccess) return hip_fail(e, "hipGetSymbolAddress (scratch array)");
    if (need > cap)
      return set_error(WB_ESIZE, "the round's work tables need " + std::to_string(need) + " bytes; the library's scratch "
                                 "array holds " + std::to_string(cap) + ": plan with a smaller round budget");
    if (!dst_ptrs && P->n_locals > 0) return set_error(WB_EINVAL, "local tensor pointer array is null");
    const wb::Rank& R = rank_of(P);
    int rc = check_extent(recv_buf, rank_bytes(P, round, P->role, P->rank), "recv_buf");
    for (int i = 0; rc == WB_OK && i < P->n_locals; ++i)
      rc = check_extent(dst_ptrs[i], local_bytes(R.locals[i]), "local tensor");
    if (rc != WB_OK) return rc;
    hipStream_t st = static_cast<hipStream_t>(stream);
    auto* ws = static_cast<uint8_t*>(base);
    e = static_cast<hipError_t>(
        wb::launch_store_table(reinterpret_cast<uint64_t*>(ws), const_cast<const void* const*>(dst_ptrs), P->n_locals, stream));
    if (e != hipSuccess) return hip_fail(e, "pointer table launch");
    if (t1 > t0 && (e = hipMemcpyAsync(ws + off_tasks, P->tasks.data() + t0, sizeof(wb::Task) * (t1 - t0),
                                       hipMemcpyHostToDevice, st)) != hipSuccess)
      return hip_fail(e, "hipMemcpyAsync (tasks)");
    if (b1 > b0 && (e = hipMemcpyAsync(ws + off_blocks, P->qblocks.data() + b0, sizeof(wb::QBlock) * (b1 - b0),
                                       hipMemcpyHostToDevice, st)) != hipSuccess)
      return hip_fail(e, "hipMemcpyAsync (fp8 blocks)");
    if (q1 > q0 && (e = hipMemcpyAsync(ws + off_pieces, P->qpieces.data() + q0, sizeof(wb::QPiece) * (q1 - q0),
                                       hipMemcpyHostToDevice, st)) != hipSuccess)
      return hip_fail(e, "hipMemcpyAsync (fp8 pieces)");
    const auto* table = reinterpret_cast<const uint64_t*>(ws);
    int k = wb::launch_tasks(reinterpret_cast<const wb::Task*>(ws + off_tasks), t1 - t0, P->round_split[round], table,
                             recv_buf, nullptr, stream);
    if (k != 0) return set_error(WB_EHIP, std::string("copy launch: ") + wb::hip_error_string(k));
    // blocks address pieces by their index in the whole table: the staged range
    // starts at piece q0
    const auto* pieces =
        reinterpret_cast<const wb::QPiece*>(reinterpret_cast<uintptr_t>(ws + off_pieces) - sizeof(wb::QPiece) * q0);
    k = wb::launch_qblocks(reinterpret_cast<const wb::QBlock*>(ws + off_blocks), b1 - b0, P->round_qfull[round],
                           P->round_qsingle[round], pieces,
                           table, recv_buf, stream);
    if (k != 0) return set_error(WB_EHIP, std::string("fp8 launch: ") + wb::hip_error_string(k));
    return WB_OK;
  });
}

int wb_pack(wb_plan_t* P, const void* const* src_ptrs, void* send_buf, void* stream) {
  return guarded([&]() -> int {
    if (!P) return set_error(WB_EINVAL, "null plan");
    if (P->rounds.size() != 1) return set_error(WB_EINVAL, "the plan has several rounds: use wb_pack_round");
    return run_round(P, 0, src_ptrs, send_buf, stream, WB_SENDER);
  });
}

int wb_unpack(wb_plan_t* P, const void* recv_buf, void* const* dst_ptrs, void* stream) {
  return guarded([&]() -> int {
    if (!P) return set_error(WB_EINVAL, "null plan");
    if (P->rounds.size() != 1) return set_error(WB_EINVAL, "the plan has several rounds: use wb_unpack_round");
    return run_round(P, 0, const_cast<const void* const*>(dst_ptrs), recv_buf, stream, WB_RECEIVER);
  });
}

int wb_probe_create(const wb_tensor_desc* catalog, int32_t num_tensors, int32_t ckpt_dtype, wb_probe_t** out) {
  return guarded([&]() -> int {
    if (!out || !catalog || num_tensors < 1) return set_error(WB_EINVAL, "bad catalog");
    *out = nullptr;
    auto* P = new wb_probe_t;
    try {
      wb::probe_init(*P, catalog, num_tensors, ckpt_dtype);
    } catch (...) {
      delete P;
      throw;
    }
    *out = P;
    return WB_OK;
  });
}

int wb_probe_chunks(const wb_probe_t* P, int32_t* num_chunks, int32_t* chunk_bits) {
  if (!P || !num_chunks || !chunk_bits) return set_error(WB_EINVAL, "null argument");
  *num_chunks = P->nchunks;
  *chunk_bits = P->bits;
  return WB_OK;
}

int wb_probe_first_id(const wb_probe_t* P, int32_t t, int64_t* id) {
  if (!P || !id) return set_error(WB_EINVAL, "null argument");
  if (t < 0 || t >= static_cast<int>(P->first.size())) return set_error(WB_EINVAL, "tensor out of range");
  *id = P->first[t];
  return WB_OK;
}

int wb_probe_add_local(wb_probe_t* P, const char* name, int32_t dtype, int64_t batch, int64_t rows, int64_t cols,
                       int32_t* index) {
  return guarded([&]() -> int {
    if (!P || !name || !index) return set_error(WB_EINVAL, "null argument");
    if (batch < 1 || rows < 1 || cols < 1) return set_error(WB_EINVAL, "local tensor shape must be positive");
    if (dtype != P->dtype) return set_error(WB_EUNSUPPORTED, "probed local tensors take the checkpoint dtype");
    wb::ProbeLocal L;
    L.name = name;
    L.dtype = dtype;
    L.batch = batch;
    L.rows = rows;
    L.cols = cols;
    P->locals.push_back(std::move(L));
    *index = static_cast<int32_t>(P->locals.size() - 1);
    return WB_OK;
  });
}

int wb_probe_record(wb_probe_t* P, int32_t local, int32_t chunk, const int64_t* index, const int64_t* value,
                    int64_t n) {
  return guarded([&]() -> int {
    if (!P) return set_error(WB_EINVAL, "null probe");
    wb::probe_record(*P, local, chunk, index, value, n);
    return WB_OK;
  });
}

int wb_probe_scan(const wb_probe_t* P, wb_layout_t* L, int32_t rank) {
  return guarded([&]() -> int {
    if (!P || !L) return set_error(WB_EINVAL, "null argument");
    wb::probe_scan(*P, *L, rank);
    return WB_OK;
  });
}

void wb_probe_destroy(wb_probe_t* P) { delete P; }

int wb_make_ids(void* dst, int32_t dtype, int64_t numel, int64_t first_id, int32_t chunk, int32_t chunk_bits,
                void* stream) {
  return guarded([&]() -> int {
    if (dtype != WB_F32 && dtype != WB_BF16) return set_error(WB_EINVAL, "identifier chunks need f32 or bf16");
    if (chunk_bits != 16 || chunk < 0 || chunk * chunk_bits >= 64 || numel < 0 || first_id < 0)
      return set_error(WB_EINVAL, "bad chunk, width, size or first identifier");
    if (numel == 0) return WB_OK;
    const int rc = check_extent(dst, numel * wb::dtype_bytes(dtype), "dst", wb::dtype_bytes(dtype));
    if (rc != WB_OK) return rc;
    const int e = wb::launch_make_ids(dst, dtype, numel, first_id, chunk * chunk_bits, 0xFFFFu, stream);
    if (e != 0) return set_error(WB_EHIP, std::string("identifier launch: ") + wb::hip_error_string(e));
    return WB_OK;
  });
}

int wb_diff2(const void* src, int32_t dtype, int64_t rows, int64_t cols, int64_t* index, int32_t* value,
             int64_t capacity, uint64_t* count, void* stream) {
  return guarded([&]() -> int {
    if (dtype != WB_F32 && dtype != WB_BF16) return set_error(WB_EINVAL, "diff2 needs an f32 or bf16 field");
    if (rows < 1 || cols < 1 || capacity < 0) return set_error(WB_EINVAL, "bad shape or capacity");
    if (!count || reinterpret_cast<uintptr_t>(count) % 8) return set_error(WB_EINVAL, "count must be 8-byte aligned");
    int rc = check_extent(count, 8, "count", 8);
    if (rc == WB_OK) rc = check_extent(src, rows * cols * wb::dtype_bytes(dtype), "src", wb::dtype_bytes(dtype));
    if (rc == WB_OK && capacity > 0) rc = check_extent(index, capacity * 8, "index", 8);
    if (rc == WB_OK && capacity > 0) rc = check_extent(value, capacity * 4, "value", 4);
    if (rc != WB_OK) return rc;
    const int e = wb::launch_diff2(src, dtype, rows, cols, index, value, capacity,
                                   reinterpret_cast<unsigned long long*>(count), stream);
    if (e != 0) return set_error(WB_EHIP, std::string("diff2 launch: ") + wb::hip_error_string(e));
    return WB_OK;
  });
}

// Check the fields of a batched diff2 call and build its field and tile
// tables; the device extents of the fields are checked only when `memory` is
// set. The workspace holds the field table, then (8-byte aligned) the tiles.
struct Diff2Tables {
  std::vector<wb::DiffField> fields;
  std::vector<wb::DiffTile> tiles;
  size_t tiles_offset() const { return (fields.size() * sizeof(wb::DiffField) + 7) / 8 * 8; }
  size_t bytes() const { return tiles.empty() ? 0 : tiles_offset() + tiles.size() * sizeof(wb::DiffTile); }
};

static int diff2_batch_tables(const wb_field* fields, int32_t n, bool memory, Diff2Tables& T) {
  if (n < 0 || (n > 0 && !fields)) return set_error(WB_EINVAL, "fields is null or n is negative");
  int64_t base = 0;
  for (int32_t fi = 0; fi < n; ++fi) {
    const wb_field& x = fields[fi];
    const std::string what = "field " + std::to_string(fi);
    if (x.dtype != WB_F32 && x.dtype != WB_BF16) return set_error(WB_EINVAL, what + ": diff2 needs f32 or bf16");
    if (x.passes < 1 || x.passes > wb::kMaxPasses)
      return set_error(WB_EINVAL, what + ": passes must be 1.." + std::to_string(wb::kMaxPasses));
    if (x.rows < 0 || x.cols < 0 || (x.cols > 0 && x.rows > (int64_t(1) << 61) / x.cols))
      return set_error(WB_EINVAL, what + ": bad shape");
    const int64_t numel = x.rows * x.cols;
    if (base > (int64_t(1) << 61) - numel) return set_error(WB_EINVAL, "fields too large");
    wb::DiffField f{};
    f.rows = x.rows;
    f.cols = x.cols;
    f.base = base;
    f.dtype = x.dtype;
    f.passes = static_cast<uint8_t>(x.passes);
    const int es = wb::dtype_bytes(x.dtype);
    for (int c = 0; c < x.passes; ++c) {
      f.src[c] = x.data[c];
      if (numel == 0) continue;
      const std::string d = what + " data[" + std::to_string(c) + "]";
      if (!x.data[c]) return set_error(WB_EINVAL, d + " is null");
      if (reinterpret_cast<uintptr_t>(x.data[c]) % es) return set_error(WB_EINVAL, d + " is not element-aligned");
      if (memory) {
        const int rc = check_extent(x.data[c], numel * es, d.c_str(), es);
        if (rc != WB_OK) return rc;
      }
    }
    wb::diff_tiles(fi, f, T.tiles);
    T.fields.push_back(f);
    base += numel;
  }
  if (T.tiles.size() > size_t(INT32_MAX)) return set_error(WB_EINVAL, "more than 2^31 - 1 tiles");
  return WB_OK;
}

int wb_diff2_batch_workspace(const wb_field* fields, int32_t n, size_t* bytes) {
  return guarded([&]() -> int {
    if (!bytes) return set_error(WB_EINVAL, "bytes is null");
    Diff2Tables T;
    const int rc = diff2_batch_tables(fields, n, false, T);
    if (rc != WB_OK) return rc;
    *bytes = T.bytes();
    return WB_OK;
  });
}

int wb_diff2_batch(const wb_field* fields, int32_t n, void* workspace, size_t workspace_bytes, int64_t* index,
                   int64_t* value, int64_t capacity, uint64_t* count, void* stream) {
  return guarded([&]() -> int {
    if (capacity < 0) return set_error(WB_EINVAL, "negative capacity");
    if (!count || reinterpret_cast<uintptr_t>(count) % 8) return set_error(WB_EINVAL, "count must be 8-byte aligned");
    int rc = check_extent(count, 8, "count", 8);
    if (rc == WB_OK && capacity > 0) rc = check_extent(index, capacity * 8, "index", 8);
    if (rc == WB_OK && capacity > 0) rc = check_extent(value, capacity * 8, "value", 8);
    if (rc != WB_OK) return rc;
    Diff2Tables T;
    rc = diff2_batch_tables(fields, n, true, T);
    if (rc != WB_OK) return rc;
    const size_t need = T.bytes();
    if (need > workspace_bytes) return set_error(WB_EINVAL, "workspace smaller than wb_diff2_batch_workspace");
    hipStream_t st = static_cast<hipStream_t>(stream);
    char* ws = static_cast<char*>(workspace);
    if (need > 0) {
      rc = check_extent(workspace, static_cast<int64_t>(need), "workspace", 8);
      if (rc != WB_OK) return rc;
      std::vector<char> host(need);
      std::memcpy(host.data(), T.fields.data(), T.fields.size() * sizeof(wb::DiffField));
      std::memcpy(host.data() + T.tiles_offset(), T.tiles.data(), T.tiles.size() * sizeof(wb::DiffTile));
      hipError_t e = hipMemcpyAsync(ws, host.data(), need, hipMemcpyHostToDevice, st);
      if (e != hipSuccess) return hip_fail(e, "hipMemcpyAsync (diff2 tables)");
      e = hipStreamSynchronize(st);  // the host copy is freed on return
      if (e != hipSuccess) return hip_fail(e, "hipStreamSynchronize");
    }
    const int e = wb::launch_diff2_batch(reinterpret_cast<const wb::DiffField*>(ws),
                                         reinterpret_cast<const wb::DiffTile*>(ws + T.tiles_offset()),
                                         int64_t(T.tiles.size()), index, value, capacity,
                                         reinterpret_cast<unsigned long long*>(count), stream);
    if (e != 0) return set_error(WB_EHIP, std::string("diff2 launch: ") + wb::hip_error_string(e));
    return WB_OK;
  });
}

// Workspace of a carry pass: the field and tile tables, the counters of the
// two carry tables (1 KiB each), the two tables (pass k writes table k % 2
// and reads the other), each `slots` slots of 16 bytes, slots the smallest
// power of two at least twice the capacity (64 at least), then the staging
// area of the stencil's carries (kCarryStage entries of 16 bytes per tile,
// then a 4-byte count per tile).
struct CarryLayout {
  size_t counters = 0, table[2] = {0, 0}, stage = 0, stage_n = 0, bytes = 0;
  uint64_t slots = 0;
};

static constexpr int64_t kMaxCarryCapacity = int64_t(1) << 36;

static CarryLayout carry_layout(const Diff2Tables& T, int64_t capacity) {
  CarryLayout L;
  L.slots = 64;
  while (L.slots < uint64_t(2 * capacity)) L.slots <<= 1;
  const size_t tables = T.tiles_offset() + T.tiles.size() * sizeof(wb::DiffTile);
  L.counters = (tables + 255) / 256 * 256;
  const size_t one = L.slots * 16;
  L.table[0] = L.counters + 2048;
  L.table[1] = L.table[0] + one;
  L.stage = L.table[1] + one;
  L.stage_n = L.stage + T.tiles.size() * wb::kCarryStage * 16;
  L.bytes = L.stage_n + (T.tiles.size() * 4 + 255) / 256 * 256;
  return L;
}

static int carry_fields(const wb_field* fields, int32_t n, bool memory, int64_t carry_capacity, Diff2Tables& T) {
  if (carry_capacity < 1 || carry_capacity > kMaxCarryCapacity)
    return set_error(WB_EINVAL, "carry_capacity must be 1..2^36");
  const int rc = diff2_batch_tables(fields, n, memory, T);
  if (rc != WB_OK) return rc;
  for (int32_t fi = 0; fi < n; ++fi)
    if (fields[fi].passes != 1)
      return set_error(WB_EINVAL, "field " + std::to_string(fi) + ": a carry pass reads one pass per field");
  return WB_OK;
}

int wb_diff2_carry_workspace(const wb_field* fields, int32_t n, int64_t carry_capacity, size_t* bytes) {
  return guarded([&]() -> int {
    if (!bytes) return set_error(WB_EINVAL, "bytes is null");
    Diff2Tables T;
    const int rc = carry_fields(fields, n, false, carry_capacity, T);
    if (rc != WB_OK) return rc;
    *bytes = carry_layout(T, carry_capacity).bytes;
    return WB_OK;
  });
}

int wb_diff2_carry(const wb_field* fields, int32_t n, int32_t pass, int32_t last, int64_t carry_capacity,
                   void* workspace, size_t workspace_bytes, int64_t* index, int64_t* value, int64_t capacity,
                   uint64_t* count, uint64_t* carries, void* stream) {
  return guarded([&]() -> int {
    if (pass < 0) return set_error(WB_EINVAL, "negative pass");
    if (capacity < 0) return set_error(WB_EINVAL, "negative capacity");
    if (!count || reinterpret_cast<uintptr_t>(count) % 8) return set_error(WB_EINVAL, "count must be 8-byte aligned");
    if (!carries || reinterpret_cast<uintptr_t>(carries) % 8)
      return set_error(WB_EINVAL, "carries must be 8-byte aligned");
    if (!workspace || reinterpret_cast<uintptr_t>(workspace) % 8)
      return set_error(WB_EINVAL, "workspace must be 8-byte aligned");
    int rc = check_extent(count, 8, "count", 8);
    if (rc == WB_OK) rc = check_extent(carries, 8, "carries", 8);
    if (rc == WB_OK && capacity > 0) rc = check_extent(index, capacity * 8, "index", 8);
    if (rc == WB_OK && capacity > 0) rc = check_extent(value, capacity * 8, "value", 8);
    if (rc != WB_OK) return rc;
    Diff2Tables T;
    rc = carry_fields(fields, n, true, carry_capacity, T);
    if (rc != WB_OK) return rc;
    const CarryLayout L = carry_layout(T, carry_capacity);
    if (L.bytes > workspace_bytes) return set_error(WB_EINVAL, "workspace smaller than wb_diff2_carry_workspace");
    rc = check_extent(workspace, static_cast<int64_t>(L.bytes), "workspace", 8);
    if (rc != WB_OK) return rc;
    hipStream_t st = static_cast<hipStream_t>(stream);
    char* ws = static_cast<char*>(workspace);
    const size_t tables = T.tiles_offset() + T.tiles.size() * sizeof(wb::DiffTile);
    if (!T.fields.empty()) {
      std::vector<char> host(tables);
      std::memcpy(host.data(), T.fields.data(), T.fields.size() * sizeof(wb::DiffField));
      if (!T.tiles.empty())
        std::memcpy(host.data() + T.tiles_offset(), T.tiles.data(), T.tiles.size() * sizeof(wb::DiffTile));
      hipError_t e = hipMemcpyAsync(ws, host.data(), tables, hipMemcpyHostToDevice, st);
      if (e != hipSuccess) return hip_fail(e, "hipMemcpyAsync (diff2 tables)");
      e = hipStreamSynchronize(st);  // the host copy is freed on return
      if (e != hipSuccess) return hip_fail(e, "hipStreamSynchronize");
    }
    wb::CarryTable tab[2];
    for (int t = 0; t < 2; ++t) {
      tab[t].slot = reinterpret_cast<int64_t*>(ws + L.table[t]);
      tab[t].count = reinterpret_cast<unsigned long long*>(ws + L.counters + 1024 * t);
      tab[t].stage = reinterpret_cast<int64_t*>(ws + L.stage);
      tab[t].stage_n = reinterpret_cast<int32_t*>(ws + L.stage_n);
      tab[t].capacity = carry_capacity;
      tab[t].mask = L.slots - 1;
    }
    const wb::CarryTable& next = tab[pass & 1];
    const wb::CarryTable& in = tab[(pass + 1) & 1];
    const int e = wb::launch_diff2_carry(reinterpret_cast<const wb::DiffField*>(ws), n,
                                         reinterpret_cast<const wb::DiffTile*>(ws + T.tiles_offset()),
                                         int64_t(T.tiles.size()), pass > 0, last != 0, in, next, index, value,
                                         capacity, reinterpret_cast<unsigned long long*>(count),
                                         reinterpret_cast<unsigned long long*>(carries), stream);
    if (e != 0) return set_error(WB_EHIP, std::string("diff2 carry launch: ") + wb::hip_error_string(e));
    return WB_OK;
  });
}

void wb_plan_destroy(wb_plan_t* P) {
  if (!P) return;
  for (int k = 0; k < wb_plan_t::kPtrSlots; ++k) {
    for (void* ev : {P->ptr_copied[k], P->ptr_done[k]}) {
      if (!ev) continue;
      (void)hipEventSynchronize(static_cast<hipEvent_t>(ev));
      (void)hipEventDestroy(static_cast<hipEvent_t>(ev));
    }
  }
  if (P->ptr_stage) (void)hipHostFree(P->ptr_stage);
  delete P;
}

}  // extern "C"
