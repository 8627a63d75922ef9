// Routing plan (WeightBridge Sec. 3.2, "Generating an efficient routing plan")
// and the per-rank kernel work derived from it.
//
// Correspondence is the overlap of trainer and rollout source maps in the
// checkpoint index space (Sec. 3.1). Identical trainer rectangles held by
// several ranks are replicas: each region they serve is cut into distinct
// slices, one per replica, so the trainers together send a single copy, and
// slices go to the replica furthest below its even share (Sec. 3.2: no
// redundant transfer, no single-source bottleneck). This file follows the
// canonical rules stated in wb.h so that every rank derives the same plan.
#include <sched.h>

#include <algorithm>
#include <array>
#include <atomic>
#include <cstdlib>
#include <exception>
#include <map>
#include <numeric>
#include <sstream>
#include <system_error>
#include <thread>

#include "wb_internal.hpp"

namespace wb {
namespace {

constexpr int64_t kPayloadAlign = 256;
constexpr int64_t kRegionAlign = 4096;

int64_t align_up(int64_t x, int64_t a) { return (x + a - 1) / a * a; }

bool intersect(const Rect& a, const Rect& b, Rect& out) {
  out.r0 = std::max(a.r0, b.r0);
  out.r1 = std::min(a.r1, b.r1);
  out.c0 = std::max(a.c0, b.c0);
  out.c1 = std::min(a.c1, b.c1);
  return out.r0 < out.r1 && out.c0 < out.c1;
}

Rect rect_of(const Placement& p) { return {p.r0, p.r1, p.c0, p.c1}; }

// k parts of x: by rows when it has at least k rows, else by columns; part j
// spans [j n / k, (j + 1) n / k) of that axis; empty parts are left out.
void split_parts(const Rect& x, int k, std::vector<Rect>& parts) {
  const bool by_rows = x.rows() >= k;
  const int64_t n = by_rows ? x.rows() : x.cols();
  parts.clear();
  for (int j = 0; j < k; ++j) {
    const int64_t a = j * n / k, b = (j + 1) * n / k;
    if (a == b) continue;
    parts.push_back(by_rows ? Rect{x.r0 + a, x.r0 + b, x.c0, x.c1} : Rect{x.r0, x.r1, x.c0 + a, x.c0 + b});
  }
}

// Deficit hand-out over k owners (ascending ranks): every owner's counter
// drops by the region's weight, then the parts, largest first (stable), each
// go to the owner with the lowest counter (the lower rank on ties), whose
// counter rises by k times the part's weight. who[j] is an owner position.
void deal(const std::vector<Rect>& parts, std::vector<int64_t>& E, int64_t total, int64_t per_elem,
          std::vector<int>& who) {
  const int k = static_cast<int>(E.size());
  for (int64_t& e : E) e -= total;
  std::vector<int> order(parts.size());
  std::iota(order.begin(), order.end(), 0);
  std::stable_sort(order.begin(), order.end(), [&](int a, int b) { return parts[a].numel() > parts[b].numel(); });
  who.assign(parts.size(), -1);
  for (int j : order) {
    int best = 0;
    for (int o = 1; o < k; ++o)
      if (E[o] < E[best]) best = o;
    E[best] += int64_t(k) * parts[j].numel() * per_elem;
    who[j] = best;
  }
}

struct Group {
  Rect x;
  std::vector<int> owners;  // ascending ranks
  std::vector<int> pls;     // placement index of each owner
  int set = -1;             // interned owner set
  int esize = 0;
};

void validate_layout(const wb_layout_t& L, bool exact_cover, const char* side) {
  for (size_t r = 0; r < L.ranks.size(); ++r) {
    const Rank& R = L.ranks[r];
    std::vector<int64_t> covered(R.locals.size(), 0);
    for (const Placement& p : R.pls) {
      check_placement(L, static_cast<int>(r), p);
      covered[p.u] += p.numel();
    }
    if (!exact_cover) continue;
    for (size_t u = 0; u < R.locals.size(); ++u) {
      if (R.locals[u].scales >= 0) continue;
      if (covered[u] != R.locals[u].numel())
        fail(WB_EINVAL, std::string(side) + " rank " + std::to_string(r) + " tensor " + R.locals[u].name +
                            " is not exactly covered by its placements");
    }
  }
}

// ---- task builders (copy/cast kernel work) ------------------------------

struct TaskSink {
  std::vector<Task>& out;
  int64_t task_bytes;

  void push(uint8_t kind, int sidx, uint64_t soff, uint32_t sld, int sdt, int didx, uint64_t doff, uint32_t dld,
            int ddt, int64_t rows, int64_t cols) {
    Task t{};
    t.src_off = soff;
    t.dst_off = doff;
    t.rows = static_cast<uint32_t>(rows);
    t.cols = static_cast<uint32_t>(cols);
    t.src_ld = sld;
    t.dst_ld = dld;
    t.src_idx = static_cast<uint16_t>(sidx);
    t.dst_idx = static_cast<uint16_t>(didx);
    t.kind = kind;
    t.sdt = static_cast<uint8_t>(sdt);
    t.ddt = static_cast<uint8_t>(ddt);
    out.push_back(t);
  }

  // Elements per vector of a vector kind and the kind itself, or false.
  static bool vector_kind(int sdt, int ddt, uint8_t& kind, int64_t& v) {
    if (sdt == ddt) { kind = TASK_COPY16; v = 16 / dtype_bytes(sdt); return true; }
    if (sdt == WB_F32 && ddt == WB_BF16) { kind = TASK_F32_BF16; v = 8; return true; }
    if (sdt == WB_BF16 && ddt == WB_F32) { kind = TASK_BF16_F32; v = 8; return true; }
    return false;
  }

  // One vector-kind task; COPY16 tasks are expressed in bytes.
  void push_vec(uint8_t kind, int sidx, uint64_t soff, int64_t sld, int sdt, int didx, uint64_t doff, int64_t dld,
                int ddt, int64_t rows, int64_t cols) {
    if (kind == TASK_COPY16) {
      const int es = dtype_bytes(sdt);
      push(kind, sidx, soff, static_cast<uint32_t>(sld * es), sdt, didx, doff, static_cast<uint32_t>(dld * es), ddt,
           rows, cols * es);
    } else {
      push(kind, sidx, soff, static_cast<uint32_t>(sld), sdt, didx, doff, static_cast<uint32_t>(dld), ddt, rows, cols);
    }
  }

  // rows x cols elements; src/dst row strides in elements; offsets in bytes.
  void copy_rect(int sidx, uint64_t soff, int64_t sld, int sdt, int didx, uint64_t doff, int64_t dld, int ddt,
                 int64_t rows, int64_t cols) {
    const int ss = dtype_bytes(sdt), ds = dtype_bytes(ddt);
    const int64_t per_task = std::max<int64_t>(16, task_bytes / std::max(ss, ds));
    uint8_t kind;
    int64_t v;
    const bool vk = vector_kind(sdt, ddt, kind, v);
    if (rows == 1 || (cols == sld && cols == dld)) {
      // contiguous on both sides: one linear run
      const int64_t n = rows * cols;
      int64_t head = -1;
      if (vk)
        for (int64_t e = 0; e < v && e < n; ++e)
          if ((soff + e * ss) % 16 == 0 && (doff + e * ds) % 16 == 0) { head = e; break; }
      if (head < 0) {
        for (int64_t a = 0; a < n; a += per_task)
          push(TASK_SCALAR, sidx, soff + a * ss, 0, sdt, didx, doff + a * ds, 0, ddt, 1, std::min(per_task, n - a));
        return;
      }
      if (head > 0) push(TASK_SCALAR, sidx, soff, 0, sdt, didx, doff, 0, ddt, 1, head);
      const int64_t body = (n - head) / v * v;
      const int64_t chunk = std::max<int64_t>(v, per_task / v * v);
      for (int64_t a = 0; a < body; a += chunk) {
        const int64_t len = std::min(chunk, body - a);
        push_vec(kind, sidx, soff + (head + a) * ss, len, sdt, didx, doff + (head + a) * ds, len, ddt, 1, len);
      }
      const int64_t tail = n - head - body;
      if (tail > 0)
        push(TASK_SCALAR, sidx, soff + (head + body) * ss, 0, sdt, didx, doff + (head + body) * ds, 0, ddt, 1, tail);
      return;
    }
    const bool vec = vk && soff % 16 == 0 && doff % 16 == 0 && cols % v == 0 && (sld * ss) % 16 == 0 &&
                     (dld * ds) % 16 == 0;
    const int64_t unit = vec ? v : 1;
    const int64_t col_chunk = cols <= per_task ? cols : std::max(unit, per_task / unit * unit);
    const int64_t rows_per = std::max<int64_t>(1, per_task / col_chunk);
    for (int64_t r = 0; r < rows; r += rows_per) {
      const int64_t nr = std::min(rows_per, rows - r);
      for (int64_t c = 0; c < cols; c += col_chunk) {
        const int64_t nc = std::min(col_chunk, cols - c);
        const uint64_t so = soff + (r * sld + c) * ss, dof = doff + (r * dld + c) * ds;
        if (vec)
          push_vec(kind, sidx, so, sld, sdt, didx, dof, dld, ddt, nr, nc);
        else
          push(TASK_SCALAR, sidx, so, static_cast<uint32_t>(sld), sdt, didx, dof, static_cast<uint32_t>(dld), ddt, nr,
               nc);
      }
    }
  }

  // dst[c][r] = src[r][c] for an R x C source block. Aligned 2-byte data is
  // cut into tiles of 128 source rows by 512 source columns (taken along the
  // source rows, which measured fastest for these tiles), transposed by the
  // tile kernel; the edges go to transpose_small.
  void transpose_rect(int sidx, uint64_t soff, int64_t sld, int sdt, int didx, uint64_t doff, int64_t dld, int ddt,
                      int64_t R, int64_t C) {
    const int ss = dtype_bytes(sdt), ds = dtype_bytes(ddt);
    const bool fast = ss == 2 && ds == 2 && sdt == ddt && soff % 16 == 0 && doff % 16 == 0 && (sld * 2) % 16 == 0 &&
                      (dld * 2) % 16 == 0;
    const int64_t RT = fast ? R / kTileRows * kTileRows : 0, CT = fast ? C / kTileCols * kTileCols : 0;
    if (RT == 0 || CT == 0) {
      transpose_small(sidx, soff, sld, sdt, didx, doff, dld, ddt, R, C);
      return;
    }
    for (int64_t r = 0; r < RT; r += kTileRows)
      for (int64_t c = 0; c < CT; c += kTileCols)
        push(TASK_TILE, sidx, soff + (r * sld + c) * 2, static_cast<uint32_t>(sld), sdt, didx,
             doff + (c * dld + r) * 2, static_cast<uint32_t>(dld), ddt, kTileRows, kTileCols);
    if (CT < C)  // right strip of the tiled rows
      transpose_small(sidx, soff + CT * 2, sld, sdt, didx, doff + CT * dld * 2, dld, ddt, RT, C - CT);
    if (RT < R)  // bottom strip, full width
      transpose_small(sidx, soff + RT * sld * 2, sld, sdt, didx, doff + RT * 2, dld, ddt, R - RT, C);
  }

  // The same for blocks without whole tiles. Aligned 2-byte data is
  // transposed in registers, in items of up to 256 x 64 taken one 64-column
  // strip at a time, each strip top to bottom: consecutive tiles (and
  // workgroups) read down the source columns and write neighbouring 128-byte
  // spans of the same destination rows, an order that measured 9-13 % faster
  // on gfx950 than row by row. The rest (ragged edges, other dtypes) goes in
  // 64 x 64 LDS tiles.
  void transpose_small(int sidx, uint64_t soff, int64_t sld, int sdt, int didx, uint64_t doff, int64_t dld, int ddt,
                       int64_t R, int64_t C) {
    const int ss = dtype_bytes(sdt), ds = dtype_bytes(ddt);
    const bool fast = ss == 2 && ds == 2 && sdt == ddt && soff % 16 == 0 && doff % 16 == 0 && (sld * 2) % 16 == 0 &&
                      (dld * 2) % 16 == 0;
    const int64_t R64 = fast ? R / 64 * 64 : 0, C64 = fast ? C / 64 * 64 : 0;
    for (int64_t c = 0; c < C64; c += 64)
      for (int64_t r = 0; r < R64; r += 256)
        push(TASK_TRANSPOSE16, sidx, soff + (r * sld + c) * 2, static_cast<uint32_t>(sld), sdt, didx,
             doff + (c * dld + r) * 2, static_cast<uint32_t>(dld), ddt, std::min<int64_t>(256, R64 - r), 64);
    for (int64_t r = 0; r < R; r += 64)
      for (int64_t c = r < R64 ? C64 : 0; c < C; c += 64)
        push(TASK_TRANSPOSE, sidx, soff + (r * sld + c) * ss, static_cast<uint32_t>(sld), sdt, didx,
             doff + (c * dld + r) * ds, static_cast<uint32_t>(dld), ddt, std::min<int64_t>(64, R - r),
             std::min<int64_t>(64, C - c));
  }
};

bool cast_supported(int sdt, int ddt) {
  if (sdt != WB_F32 && sdt != WB_BF16) return false;
  return ddt == WB_F32 || ddt == WB_BF16 || ddt == WB_F8E4M3;
}

int64_t env_task_bytes() {
  const char* s = std::getenv("WB_TASK_BYTES");
  const int64_t v = s ? std::atoll(s) : 0;
  return v >= 1024 && v <= (int64_t(1) << 30) ? v : (int64_t(1) << 18);
}

// The dtype a segment's bytes travel in: that of the trainer placement they
// were packed from (forwarded segments keep it).
int wire_dtype(const wb_layout_t& trainer, const std::vector<Segment>& segs, const Segment& g) {
  const Segment& o = g.stage == 0 ? g : segs[g.origin];
  const Rank& S = trainer.ranks[o.s];
  return S.locals[S.pls[o.src_pl].u].dtype;
}

// One wire segment's image in a quantised local: matrix e of the stack, its
// first row and column there.
struct QSpan {
  const Segment* g;
  int64_t e, row0, col0;
};

// Host threads for a planning step over `work` items: WB_PLAN_THREADS if set
// (1..64), else one below `small` items and otherwise the CPUs this process
// may run on, at most 16. The plan does not depend on it.
int plan_threads(int64_t work, int64_t small) {
  if (const char* e = std::getenv("WB_PLAN_THREADS")) {
    const long v = std::strtol(e, nullptr, 10);
    if (v >= 1 && v <= 64) return static_cast<int>(v);
  }
  if (work < small) return 1;
  cpu_set_t set;
  const int n = sched_getaffinity(0, sizeof set, &set) == 0 ? CPU_COUNT(&set) : 1;
  return std::max(1, std::min(n, 16));
}

// fn(i, w) for every i in [0, n) on up to `threads` workers (w is the
// worker's number, below `threads`), which take indices in increasing order
// from a shared counter. After an exception no further index is started;
// every lower index was taken before it and runs to its end, so rethrowing
// the exception of the lowest index reports what one thread would have.
template <class F>
void parallel_for(size_t n, int threads, F&& fn) {
  const int nw = static_cast<int>(std::min<size_t>(n, std::max(threads, 1)));
  if (nw <= 1) {
    for (size_t i = 0; i < n; ++i) fn(i, 0);
    return;
  }
  std::atomic<size_t> next{0};
  std::atomic<bool> stop{false};
  std::vector<std::exception_ptr> err(n);
  auto work = [&](int w) {
    for (size_t i; !stop.load() && (i = next.fetch_add(1)) < n;) {
      try {
        fn(i, w);
      } catch (...) {
        err[i] = std::current_exception();
        stop = true;
      }
    }
  };
  std::vector<std::thread> pool;
  try {
    for (int w = 1; w < nw; ++w) pool.emplace_back(work, w);
  } catch (const std::system_error&) {
    // no more threads to be had: the ones started and this one take every index
  }
  work(0);
  for (auto& th : pool) th.join();
  for (auto& e : err)
    if (e) std::rethrow_exception(e);
}

// What the fp8 tables need of one quantised local, built by qlocal_blocks.
struct QLocalScratch {
  std::vector<QBlock> blocks;    // the local's blocks in id order (piece0 relative to the local)
  std::vector<int> round;        // each block's round
  std::vector<QPiece> pieces;    // the local's pieces, grouped by block in id order
  std::vector<uint32_t> count;   // pieces of block i: count[i] .. count[i + 1]
  std::vector<int64_t> area;
};

// Block class within a round's launch range: full pairs, other pairable
// blocks, the rest.
int qblock_class(const QBlock& b) { return qblock_full_single(b) ? 0 : qblock_pairable(b) ? 1 : 2; }

// The blocks and pieces of quantised local u of rank R from the wire spans
// that land in it (spans in plan order), numbered within the local: block
// (e, bi, bj) is block (e nbr + bi) nbc + bj, also its scale's index, and
// piece0 counts only this local's pieces.
void qlocal_blocks(const wb_layout_t& trainer, const Rank& R, const wb_plan_t& P, int u, const QSpan* spans,
                   size_t nspans, QLocalScratch& S) {
  const Local& l = R.locals[u];
  const int64_t B = l.block, nbr = (l.rows + B - 1) / B, nbc = (l.cols + B - 1) / B, nb = l.batch * nbr * nbc;
  S.blocks.assign(nb, QBlock{});
  S.round.assign(nb, -1);
  S.count.assign(nb + 1, 0);
  S.area.assign(nb, 0);
  auto for_pieces = [&](const QSpan& sp, auto&& fn) {
    const Segment& g = *sp.g;
    const int sdt = wire_dtype(trainer, P.segs, g), ss = dtype_bytes(sdt);
    const int64_t Rr = g.x.rows(), C = g.x.cols();
    for (int64_t bi = sp.row0 / B; bi <= (sp.row0 + Rr - 1) / B; ++bi)
      for (int64_t bj = sp.col0 / B; bj <= (sp.col0 + C - 1) / B; ++bj) {
        const int64_t a0 = std::max(sp.row0, bi * B), a1 = std::min(sp.row0 + Rr, (bi + 1) * B);
        const int64_t b0 = std::max(sp.col0, bj * B), b1 = std::min(sp.col0 + C, (bj + 1) * B);
        const int64_t rows = std::min(B, l.rows - bi * B), cols = std::min(B, l.cols - bj * B);
        QPiece pc{};
        pc.src_off = g.recv_off + uint64_t(((a0 - sp.row0) * C + (b0 - sp.col0)) * ss);
        pc.src_ld = static_cast<uint32_t>(C);
        pc.r0 = static_cast<uint8_t>(a0 - bi * B);
        pc.r1m1 = static_cast<uint8_t>(a1 - bi * B - 1);
        pc.c0 = static_cast<uint8_t>(b0 - bj * B);
        pc.c1m1 = static_cast<uint8_t>(b1 - bj * B - 1);
        pc.sdt = static_cast<uint8_t>(sdt);
        const bool single = sdt == WB_BF16 && a0 == bi * B && b0 == bj * B && a1 - a0 == rows && b1 - b0 == cols &&
                            cols % 8 == 0 && pc.src_off % 16 == 0 && (uint64_t(C) * 2) % 16 == 0;
        fn((sp.e * nbr + bi) * nbc + bj, pc, single, (a1 - a0) * (b1 - b0));
      }
  };
  for (size_t i = 0; i < nspans; ++i)
    for_pieces(spans[i], [&](int64_t id, const QPiece& pc, bool single, int64_t a) {
      S.area[id] += a;
      if (S.round[id] >= 0 && S.round[id] != spans[i].g->round) fail(WB_EINVAL, "internal: fp8 block spans rounds");
      S.round[id] = spans[i].g->round;
      if (single) {
        QBlock& b = S.blocks[id];
        b.flags |= QB_SINGLE;
        b.src_off = pc.src_off;
        b.src_ld = pc.src_ld;
      } else {
        ++S.count[id + 1];
      }
    });
  for (int64_t i = 0; i < nb; ++i) S.count[i + 1] += S.count[i];
  S.pieces.resize(S.count[nb]);
  {
    std::vector<uint32_t> fill(S.count.begin(), S.count.end() - 1);
    for (size_t i = 0; i < nspans; ++i)
      for_pieces(spans[i], [&](int64_t id, const QPiece& pc, bool single, int64_t) {
        if (!single) S.pieces[fill[id]++] = pc;
      });
  }
  for (int64_t e = 0; e < l.batch; ++e)
    for (int64_t bi = 0; bi < nbr; ++bi)
      for (int64_t bj = 0; bj < nbc; ++bj) {
        const int64_t id = (e * nbr + bi) * nbc + bj;
        const int64_t rows = std::min(B, l.rows - bi * B), cols = std::min(B, l.cols - bj * B);
        if (S.area[id] != rows * cols) fail(WB_EINVAL, "fp8 block of " + l.name + " is not exactly covered");
        const uint32_t p0 = S.count[id], np = S.count[id + 1] - p0;
        if (np > 65535) fail(WB_EUNSUPPORTED, "too many pieces in one fp8 block");
        QBlock& b = S.blocks[id];
        b.dst_off = uint64_t((e * l.rows + bi * B) * l.cols + bj * B);
        b.piece0 = p0;
        b.npieces = static_cast<uint16_t>(np);
        b.dst_ld = static_cast<uint32_t>(l.cols);
        b.scale_off = static_cast<uint32_t>(id);
        b.dst_idx = static_cast<uint16_t>(1 + u);
        b.scale_idx = static_cast<uint16_t>(1 + l.scale);
        b.rows_m1 = static_cast<uint8_t>(rows - 1);
        b.cols_m1 = static_cast<uint8_t>(cols - 1);
        if (b.dst_off % 8 == 0 && l.cols % 8 == 0 && cols % 8 == 0) b.flags |= QB_VEC_STORE;
        bool bf16 = true;
        for (uint32_t i = p0; i < p0 + np; ++i) bf16 = bf16 && S.pieces[i].sdt == WB_BF16;
        if (bf16) b.flags |= QB_BF16_SOURCE;
        // row bands: every piece spans the block's width, 16-byte aligned
        // rows; sorted by first row they tile the block from row 0
        if (bf16 && np >= 2 && np <= uint32_t(kMaxBands) && cols % 8 == 0) {
          QPiece* pc = S.pieces.data() + p0;
          std::sort(pc, pc + np, [](const QPiece& a, const QPiece& c) { return a.r0 < c.r0; });
          bool bands = true;
          for (uint32_t i = 0; i < np; ++i)
            bands = bands && pc[i].c0 == 0 && pc[i].c1m1 == cols - 1 && pc[i].src_off % 16 == 0 &&
                    (uint64_t(pc[i].src_ld) * 2) % 16 == 0 && pc[i].r0 == (i ? pc[i - 1].r1m1 + 1 : 0);
          if (bands && pc[np - 1].r1m1 == rows - 1) b.flags |= QB_BANDS;
        }
      }
}

// The fp8 block and piece tables of a rollout rank. Block ids run over the
// quantised locals, then batch, block row, block column; pieces are grouped
// by block in id order (canonical segment order within a block, row bands
// sorted by first row). A block filled whole by one aligned bf16 wire piece
// (QB_SINGLE) keeps that piece's address in its own descriptor, which is all
// the pair path reads, and takes no piece. Every piece adds to its block's
// covered area, so a block with a whole piece and any other one fails the
// exact-cover check. The blocks are then grouped by round and, within a
// round, ordered full pairs, other pairable blocks, the rest, each class in
// id order (consecutive pairable blocks are mostly horizontal neighbours).
// Locals are independent: each is built twice on the planning threads, once
// to count its pieces and its blocks per (round, class), once to write them
// where those counts place them.
void build_qblocks(const wb_layout_t& trainer, const Rank& R, wb_plan_t& P, const std::vector<QSpan>& qspans,
                   int64_t nblocks) {
  const int nrounds = static_cast<int>(P.rounds.size());
  const size_t nl = R.locals.size();
  // the spans of each local, in plan order
  std::vector<size_t> span0(nl + 1, 0);
  for (const QSpan& sp : qspans) ++span0[R.pls[sp.g->dst_pl].u + 1];
  for (size_t u = 0; u < nl; ++u) span0[u + 1] += span0[u];
  std::vector<QSpan> spans(qspans.size());
  {
    std::vector<size_t> at(span0.begin(), span0.end() - 1);
    for (const QSpan& sp : qspans) spans[at[R.pls[sp.g->dst_pl].u]++] = sp;
  }
  std::vector<int> ql;
  for (size_t u = 0; u < nl; ++u)
    if (R.locals[u].block > 0) ql.push_back(static_cast<int>(u));
  const size_t nq = ql.size();
  const int threads = plan_threads(nblocks, int64_t(1) << 15);
  // pass 1: per local, its pieces, its blocks per (round, class) and the
  // local piece range each round reads
  std::vector<uint32_t> npieces(nq);
  std::vector<uint32_t> cls(nq * nrounds * 3);
  std::vector<uint32_t> plo(nq * nrounds, UINT32_MAX), phi(nq * nrounds, 0);
  std::vector<QLocalScratch> scratch(threads);
  parallel_for(nq, threads, [&](size_t i, int w) {
    QLocalScratch& S = scratch[w];
    const int u = ql[i];
    qlocal_blocks(trainer, R, P, u, spans.data() + span0[u], span0[u + 1] - span0[u], S);
    npieces[i] = static_cast<uint32_t>(S.pieces.size());
    for (size_t b = 0; b < S.blocks.size(); ++b) {
      const int k = S.round[b];
      ++cls[(i * nrounds + k) * 3 + qblock_class(S.blocks[b])];
      if (S.blocks[b].npieces) {
        plo[i * nrounds + k] = std::min(plo[i * nrounds + k], S.blocks[b].piece0);
        phi[i * nrounds + k] = std::max(phi[i * nrounds + k], S.blocks[b].piece0 + S.blocks[b].npieces);
      }
    }
  });
  // global piece base of every local, block positions of every (local, round, class)
  std::vector<uint64_t> pbase(nq + 1, 0);
  for (size_t i = 0; i < nq; ++i) pbase[i + 1] = pbase[i] + npieces[i];
  if (pbase[nq] > UINT32_MAX) fail(WB_EUNSUPPORTED, "too many fp8 pieces");
  std::vector<uint32_t> pos(nq * nrounds * 3);
  uint32_t at = 0;
  for (int k = 0; k < nrounds; ++k) {
    P.round_qblocks[k] = at;
    uint32_t n[3] = {0, 0, 0};
    for (int c = 0; c < 3; ++c)
      for (size_t i = 0; i < nq; ++i) {
        pos[(i * nrounds + k) * 3 + c] = at;
        at += cls[(i * nrounds + k) * 3 + c];
        n[c] += cls[(i * nrounds + k) * 3 + c];
      }
    P.round_qsingle[k] = n[0] + n[1];
    P.round_qfull[k] = n[0] & ~1u;  // an odd one out stays with the other pairable blocks
    uint32_t lo = UINT32_MAX, hi = 0;
    for (size_t i = 0; i < nq; ++i)
      if (phi[i * nrounds + k]) {
        lo = std::min<uint32_t>(lo, static_cast<uint32_t>(pbase[i] + plo[i * nrounds + k]));
        hi = std::max<uint32_t>(hi, static_cast<uint32_t>(pbase[i] + phi[i * nrounds + k]));
      }
    P.round_qpieces[2 * k] = hi ? lo : 0;
    P.round_qpieces[2 * k + 1] = hi;
  }
  P.round_qblocks[nrounds] = at;
  if (at != uint64_t(nblocks)) fail(WB_EINVAL, "internal: fp8 block count");
  // pass 2: the same blocks again, written in place
  P.qblocks.resize(nblocks);
  P.qpieces.resize(pbase[nq]);
  parallel_for(nq, threads, [&](size_t i, int w) {
    QLocalScratch& S = scratch[w];
    const int u = ql[i];
    qlocal_blocks(trainer, R, P, u, spans.data() + span0[u], span0[u + 1] - span0[u], S);
    std::copy(S.pieces.begin(), S.pieces.end(), P.qpieces.begin() + pbase[i]);
    uint32_t* p = pos.data() + i * nrounds * 3;
    for (size_t b = 0; b < S.blocks.size(); ++b) {
      QBlock q = S.blocks[b];
      q.piece0 += static_cast<uint32_t>(pbase[i]);
      P.qblocks[p[S.round[b] * 3 + qblock_class(q)]++] = q;
    }
  });
}

void build_rank_view(const wb_layout_t& trainer, const wb_layout_t& rollout, wb_plan_t& P) {
  TaskSink sink{P.tasks, env_task_bytes()};
  const int nrounds = static_cast<int>(P.rounds.size());
  std::vector<std::vector<const Segment*>> by_round(nrounds);
  for (const Segment& g : P.segs) by_round[g.round].push_back(&g);
  P.round_tasks.assign(nrounds + 1, 0);
  P.round_qblocks.assign(nrounds + 1, 0);
  P.round_qsingle.assign(nrounds, 0);
  P.round_qfull.assign(nrounds, 0);
  P.round_qpieces.assign(2 * size_t(nrounds), 0);  // every plan: ranks without fp8 blocks keep empty ranges
  if (P.role == WB_SENDER) {
    const Rank& R = trainer.ranks[P.rank];
    P.n_locals = static_cast<int>(R.locals.size());
    for (int k = 0; k < nrounds; ++k) {
    for (const Segment* gp : by_round[k]) {
      const Segment& g = *gp;
      if (g.stage != 0 || g.s != P.rank) continue;
      const Placement& sp = R.pls[g.src_pl];
      const int dt = R.locals[sp.u].dtype, es = dtype_bytes(dt);
      const int64_t C = g.x.cols(), Rr = g.x.rows();
      P.read_bytes += g.bytes;
      P.write_bytes += g.bytes;
      if (!sp.tr) {
        const int64_t start = sp.base + (g.x.r0 - sp.r0) * sp.ld + (g.x.c0 - sp.c0);
        sink.copy_rect(1 + sp.u, uint64_t(start) * es, sp.ld, dt, 0, g.send_off, C, dt, Rr, C);
      } else {
        // local holds the transpose: rows are checkpoint columns
        const int64_t start = sp.base + (g.x.c0 - sp.c0) * sp.ld + (g.x.r0 - sp.r0);
        sink.transpose_rect(1 + sp.u, uint64_t(start) * es, sp.ld, dt, 0, g.send_off, C, dt, C, Rr);
      }
    }
    P.round_tasks[k + 1] = static_cast<uint32_t>(P.tasks.size());
    }
    for (auto& r : P.round_fwd) r.assign(nrounds + 1, static_cast<uint32_t>(P.tasks.size()));
    return;
  }
  const Rank& R = rollout.ranks[P.rank];
  P.n_locals = static_cast<int>(R.locals.size());
  // fp8 blocks of all quantised locals
  int64_t nblocks = 0;
  for (size_t u = 0; u < R.locals.size(); ++u) {
    const Local& l = R.locals[u];
    if (l.block <= 0) continue;
    nblocks += l.batch * ((l.rows + l.block - 1) / l.block) * ((l.cols + l.block - 1) / l.block);
    P.write_bytes += R.locals[l.scale].numel() * 4;
    P.q_write_bytes += R.locals[l.scale].numel() * 4;
  }
  std::vector<QSpan> qspans;
  for (int k = 0; k < nrounds; ++k) {
  for (const Segment* gp : by_round[k]) {
    const Segment& g = *gp;
    if (g.d != P.rank) continue;
    const Placement& q = R.pls[g.dst_pl];
    const Local& dl = R.locals[q.u];
    const int sdt = wire_dtype(trainer, P.segs, g);
    if (!cast_supported(sdt, dl.dtype))
      fail(WB_EUNSUPPORTED, std::string("unsupported cast ") + dtype_name(sdt) + " -> " + dtype_name(dl.dtype));
    const int64_t C = g.x.cols(), Rr = g.x.rows();
    P.read_bytes += g.bytes;
    if (dl.block > 0) {
      P.write_bytes += g.x.numel();
      P.q_write_bytes += g.x.numel();
      P.q_read_bytes += g.bytes;
      if (q.tr) fail(WB_EUNSUPPORTED, "fp8 destinations cannot be transposed");
      const int64_t f0 = q.base + (g.x.r0 - q.r0) * q.ld + (g.x.c0 - q.c0);
      const int64_t mat = dl.rows * dl.cols;
      const int64_t e = f0 / mat, row0 = (f0 % mat) / dl.cols, col0 = f0 % dl.cols;
      if (col0 + C > dl.cols || row0 + Rr > dl.rows || (Rr > 1 && q.ld != dl.cols))
        fail(WB_EUNSUPPORTED, "an fp8 placement must be a sub-rectangle of one matrix of its tensor");
      qspans.push_back({&g, e, row0, col0});
      continue;
    }
    const int ddt = dl.dtype, ds = dtype_bytes(ddt);
    P.write_bytes += g.x.numel() * ds;
    if (!q.tr) {
      const int64_t start = q.base + (g.x.r0 - q.r0) * q.ld + (g.x.c0 - q.c0);
      sink.copy_rect(0, g.recv_off, C, sdt, 1 + q.u, uint64_t(start) * ds, q.ld, ddt, Rr, C);
    } else {
      const int64_t start = q.base + (g.x.c0 - q.c0) * q.ld + (g.x.r0 - q.r0);
      sink.transpose_rect(0, g.recv_off, C, sdt, 1 + q.u, uint64_t(start) * ds, q.ld, ddt, Rr, C);
    }
  }
  P.round_tasks[k + 1] = static_cast<uint32_t>(P.tasks.size());
  }
  // forward work of the exchange stages: each segment this rank forwards is a
  // byte copy from where it landed in the receive buffer (buf) to its place in
  // the stage's forward buffer (aux)
  for (int st = 0; st < 2; ++st) {
    P.round_fwd[st].assign(nrounds + 1, static_cast<uint32_t>(P.tasks.size()));
    for (int k = 0; k < nrounds; ++k) {
      for (const Segment* gp : by_round[k]) {
        const Segment& g = *gp;
        if (g.stage != st + 1 || g.s != P.rank) continue;
        const int dt = wire_dtype(trainer, P.segs, g);
        sink.copy_rect(0, g.src_off, g.x.numel(), dt, kAuxBuffer, g.send_off, g.x.numel(), dt, 1, g.x.numel());
        P.fwd_bytes[st] += g.bytes;
      }
      P.round_fwd[st][k + 1] = static_cast<uint32_t>(P.tasks.size());
    }
  }
  if (nblocks > 0) build_qblocks(trainer, R, P, qspans, nblocks);
}

// Every byte a work item touches lies inside its buffer, and vector work items
// meet the alignment their loads and stores assume (base pointers are 16-byte
// aligned, which wb_pack / wb_unpack check). Run on every plan.
void check_work(const wb_plan_t& P, const Rank& R) {
  std::vector<int64_t> size(R.locals.size() + 1);
  for (size_t u = 0; u < R.locals.size(); ++u) size[u + 1] = R.locals[u].numel() * dtype_bytes(R.locals[u].dtype);
  int64_t aux_size = 0;
  auto inside = [&](int idx, uint64_t off, uint64_t len, const char* what) {
    const bool known = idx == kAuxBuffer || (idx >= 0 && idx < static_cast<int>(size.size()));
    if (!known || len == 0 || off + len > uint64_t(idx == kAuxBuffer ? aux_size : size[idx]))
      fail(WB_EINVAL, std::string("internal: ") + what + " work item out of bounds");
  };
  const size_t nr = P.rounds.size();
  bool ranges = P.round_tasks.size() == nr + 1 && P.round_qblocks.size() == nr + 1 &&
                P.round_qblocks.back() == P.qblocks.size() && P.round_qblocks[0] == 0 && P.round_tasks[0] == 0;
  uint32_t prev = ranges ? P.round_tasks.back() : 0;
  for (const auto& r : P.round_fwd) {
    ranges = ranges && r.size() == nr + 1 && r[0] == prev;
    if (ranges) prev = r.back();
  }
  ranges = ranges && prev == P.tasks.size();
  for (size_t k = 0; ranges && k < nr; ++k) {
    ranges = P.round_tasks[k] <= P.round_tasks[k + 1] && P.round_qblocks[k] <= P.round_qblocks[k + 1];
    for (const auto& r : P.round_fwd) ranges = ranges && r[k] <= r[k + 1];
  }
  if (!ranges) fail(WB_EINVAL, "internal: round ranges");
  auto check_task = [&](const Task& t) {
    if (t.rows == 0 || t.cols == 0) fail(WB_EINVAL, "internal: empty work item");
    // the kernel counts a work item's vectors and chunk offsets in 32 bits
    if (uint64_t(t.rows) * t.cols >= (uint64_t(1) << 31)) fail(WB_EINVAL, "internal: work item too large");
    const uint64_t ss = dtype_bytes(t.sdt), ds = dtype_bytes(t.ddt);
    switch (t.kind) {
      case TASK_COPY16:
        if (t.src_off % 16 || t.dst_off % 16 || t.cols % 16 || (t.rows > 1 && (t.src_ld % 16 || t.dst_ld % 16)))
          fail(WB_EINVAL, "internal: misaligned copy work item");
        inside(t.src_idx, t.src_off, uint64_t(t.rows - 1) * t.src_ld + t.cols, "copy source");
        inside(t.dst_idx, t.dst_off, uint64_t(t.rows - 1) * t.dst_ld + t.cols, "copy destination");
        break;
      case TASK_F32_BF16:
      case TASK_BF16_F32:
        if (t.src_off % 16 || t.dst_off % 16 || t.cols % 8 ||
            (t.rows > 1 && ((t.src_ld * ss) % 16 || (t.dst_ld * ds) % 16)))
          fail(WB_EINVAL, "internal: misaligned cast work item");
        [[fallthrough]];
      case TASK_SCALAR:
        inside(t.src_idx, t.src_off, (uint64_t(t.rows - 1) * t.src_ld + t.cols) * ss, "source");
        inside(t.dst_idx, t.dst_off, (uint64_t(t.rows - 1) * t.dst_ld + t.cols) * ds, "destination");
        break;
      case TASK_TRANSPOSE:
        if (t.rows > 64 || t.cols > 64) fail(WB_EINVAL, "internal: transpose tile above 64 x 64");
        inside(t.src_idx, t.src_off, (uint64_t(t.rows - 1) * t.src_ld + t.cols) * ss, "transpose source");
        inside(t.dst_idx, t.dst_off, (uint64_t(t.cols - 1) * t.dst_ld + t.rows) * ds, "transpose destination");
        break;
      case TASK_TILE:
        if (t.rows != kTileRows || t.cols != kTileCols || ss != 2 || ds != 2 || t.src_off % 16 || t.dst_off % 16 ||
            (t.src_ld * 2) % 16 || (t.dst_ld * 2) % 16)
          fail(WB_EINVAL, "internal: bad transpose tile");
        inside(t.src_idx, t.src_off, (uint64_t(t.rows - 1) * t.src_ld + t.cols) * ss, "transpose source");
        inside(t.dst_idx, t.dst_off, (uint64_t(t.cols - 1) * t.dst_ld + t.rows) * ds, "transpose destination");
        break;
      case TASK_TRANSPOSE16:
        if (t.cols != 64 || t.rows % 64 || t.rows > 256 || t.rows == 0 || ss != 2 || ds != 2 ||
            t.src_off % 16 || t.dst_off % 16 || (t.src_ld * 2) % 16 || (t.dst_ld * 2) % 16)
          fail(WB_EINVAL, "internal: bad register-transpose work item");
        inside(t.src_idx, t.src_off, (uint64_t(t.rows - 1) * t.src_ld + t.cols) * ss, "transpose source");
        inside(t.dst_idx, t.dst_off, (uint64_t(t.cols - 1) * t.dst_ld + t.rows) * ds, "transpose destination");
        break;
      default:
        fail(WB_EINVAL, "internal: unknown work item");
    }
  };
  for (size_t k = 0; k < nr; ++k) {
  const RoundWire& W = P.rounds[k];
  size[0] = P.role == WB_SENDER ? W.st[0].send_bytes[P.rank] : W.recv_total[P.rank];
  aux_size = 0;
  auto check_order = [&](uint32_t a, uint32_t b, const TaskSplit& sp) {
    if (uint64_t(sp.n[0]) + sp.n[1] + sp.tiles > b - a) fail(WB_EINVAL, "internal: work item class sizes");
    if (sp.s[0] > 24 || sp.s[1] > 24) fail(WB_EINVAL, "internal: work item class shift");
    for (uint32_t ti = a; ti < b; ++ti) {
      const int want = ti < a + sp.n[0] ? 0 : ti < a + sp.n[0] + sp.n[1] ? 1 : ti < b - sp.tiles ? 2 : 3;
      if (task_class(P.tasks[ti]) != want) fail(WB_EINVAL, "internal: work item order");
      // every chunk of an item has a workgroup
      if (want < 2 && task_chunks(P.tasks[ti]) > (1u << sp.s[want]))
        fail(WB_EINVAL, "internal: work item too large for its launch");
    }
  };
  check_order(P.round_tasks[k], P.round_tasks[k + 1], P.round_split[k]);
  for (int st = 0; st < 2; ++st) check_order(P.round_fwd[st][k], P.round_fwd[st][k + 1], P.fwd_split[st][k]);
  for (uint32_t ti = P.round_tasks[k]; ti < P.round_tasks[k + 1]; ++ti) {
    if (P.tasks[ti].src_idx == kAuxBuffer || P.tasks[ti].dst_idx == kAuxBuffer)
      fail(WB_EINVAL, "internal: pack or unpack work item on the forward buffer");
    check_task(P.tasks[ti]);
  }
  for (int st = 0; st < 2; ++st) {
    aux_size = P.role == WB_SENDER ? 0 : W.st[st + 1].send_bytes[P.rank];
    for (uint32_t ti = P.round_fwd[st][k]; ti < P.round_fwd[st][k + 1]; ++ti) {
      const Task& t = P.tasks[ti];
      if (t.kind != TASK_COPY16 && t.kind != TASK_SCALAR) fail(WB_EINVAL, "internal: forward work item kind");
      if (t.src_idx != 0 || t.dst_idx != kAuxBuffer) fail(WB_EINVAL, "internal: forward work item buffers");
      check_task(t);
    }
  }
  if (P.round_qsingle.size() != nr || P.round_qsingle[k] > P.round_qblocks[k + 1] - P.round_qblocks[k])
    fail(WB_EINVAL, "internal: single-piece fp8 block count");
  if (P.round_qfull.size() != nr || P.round_qfull[k] % 2 || P.round_qfull[k] > P.round_qsingle[k])
    fail(WB_EINVAL, "internal: full fp8 pair count");
  if (P.round_qpieces.size() != 2 * nr || P.round_qpieces[2 * k] > P.round_qpieces[2 * k + 1] ||
      P.round_qpieces[2 * k + 1] > P.qpieces.size())
    fail(WB_EINVAL, "internal: fp8 piece range of a round");
  auto check_block = [&](uint32_t bi) {
    const QBlock& b = P.qblocks[bi];
    if (qblock_pairable(b) != (bi < P.round_qblocks[k] + P.round_qsingle[k]) ||
        (bi < P.round_qblocks[k] + P.round_qfull[k] && !qblock_full_single(b)))
      fail(WB_EINVAL, "internal: fp8 block order");
    const uint64_t rows = b.rows_m1 + 1u, cols = b.cols_m1 + 1u;
    inside(b.dst_idx, b.dst_off, (rows - 1) * b.dst_ld + cols, "fp8 block");
    inside(b.scale_idx, uint64_t(b.scale_off) * 4, 4, "fp8 scale");
    if (R.locals[b.dst_idx - 1].dtype != WB_F8E4M3 || R.locals[b.scale_idx - 1].dtype != WB_F32)
      fail(WB_EINVAL, "internal: fp8 block targets the wrong tensors");
    if ((b.flags & QB_VEC_STORE) && (b.dst_off % 8 || b.dst_ld % 8)) fail(WB_EINVAL, "internal: misaligned fp8 store");
    if (b.flags & QB_SINGLE) {
      if (b.src_off % 16 || (uint64_t(b.src_ld) * 2) % 16 || cols % 8 || !(b.flags & QB_BF16_SOURCE))
        fail(WB_EINVAL, "internal: misaligned single-piece fp8 block");
      inside(0, b.src_off, ((rows - 1) * b.src_ld + cols) * 2, "fp8 single-piece source");
    }
    if (uint64_t(b.piece0) + b.npieces > P.qpieces.size() || (b.npieces == 0) != ((b.flags & QB_SINGLE) != 0))
      fail(WB_EINVAL, "internal: fp8 block pieces out of range");
    if (b.npieces && (b.piece0 < P.round_qpieces[2 * k] || b.piece0 + b.npieces > P.round_qpieces[2 * k + 1]))
      fail(WB_EINVAL, "internal: fp8 block pieces outside its round's piece range");
    if (b.flags & QB_BANDS) {
      if ((b.flags & QB_SINGLE) || b.npieces < 2 || b.npieces > kMaxBands || cols % 8 || !(b.flags & QB_BF16_SOURCE))
        fail(WB_EINVAL, "internal: fp8 band block");
      for (uint32_t i = 0; i < b.npieces; ++i) {
        const QPiece& q = P.qpieces[b.piece0 + i];
        if (q.sdt != WB_BF16 || q.c0 != 0 || q.c1m1 != cols - 1 || q.src_off % 16 || (uint64_t(q.src_ld) * 2) % 16 ||
            q.r0 != (i ? P.qpieces[b.piece0 + i - 1].r1m1 + 1u : 0u) || (i + 1 == b.npieces && q.r1m1 != rows - 1))
          fail(WB_EINVAL, "internal: fp8 bands do not tile their block");
      }
    }
    for (uint32_t i = b.piece0; i < b.piece0 + b.npieces; ++i) {
      const QPiece& q = P.qpieces[i];
      if (q.r1m1 < q.r0 || q.c1m1 < q.c0 || q.r1m1 >= rows || q.c1m1 >= cols)
        fail(WB_EINVAL, "internal: fp8 piece outside its block");
      const uint64_t es = dtype_bytes(q.sdt);
      inside(0, q.src_off, (uint64_t(q.r1m1 - q.r0) * q.src_ld + (q.c1m1 - q.c0) + 1) * es, "fp8 piece");
    }
  };
  // blocks in runs of 2^14 on the planning threads (the checks only read)
  const uint32_t b0 = P.round_qblocks[k], nb = P.round_qblocks[k + 1] - b0, run = 1u << 14;
  parallel_for((nb + run - 1) / run, plan_threads(nb, 2 * run), [&](size_t i, int) {
    const uint32_t lo = b0 + static_cast<uint32_t>(i) * run, hi = lo + std::min(run, b0 + nb - lo);
    for (uint32_t bi = lo; bi < hi; ++bi) check_block(bi);
  });
  }
}

// ---- rounds (Sec. 3.2 round-based transfer; App. D buffer budget) --------

// Unit of every checkpoint tensor: tensors whose images in one quantised
// destination matrix touch a common block share a unit, so no fp8 block is
// fed from two rounds.
std::vector<int> block_units(const wb_layout_t& rollout, int ntensors) {
  std::vector<int> parent(ntensors);
  std::iota(parent.begin(), parent.end(), 0);
  auto find = [&](int a) {
    while (parent[a] != a) a = parent[a] = parent[parent[a]];
    return a;
  };
  struct Img {
    int64_t bi0, bi1, bj0, bj1;
    int t;
  };
  for (const Rank& R : rollout.ranks) {
    std::map<std::pair<int, int64_t>, std::vector<Img>> per_matrix;
    for (const Placement& p : R.pls) {
      const Local& l = R.locals[p.u];
      if (l.block <= 0) continue;
      const int64_t mat = l.rows * l.cols;
      const int64_t e = p.base / mat, row0 = (p.base % mat) / l.cols, col0 = p.base % l.cols;
      if (p.tr || col0 + p.cols() > l.cols || row0 + p.rows() > l.rows || (p.rows() > 1 && p.ld != l.cols))
        fail(WB_EUNSUPPORTED, "an fp8 placement must be a non-transposed sub-rectangle of one matrix");
      const int64_t B = l.block;
      per_matrix[{p.u, e}].push_back({row0 / B, (row0 + p.rows() - 1) / B, col0 / B, (col0 + p.cols() - 1) / B, p.t});
    }
    for (auto& kv : per_matrix) {
      const std::vector<Img>& v = kv.second;
      for (size_t a = 0; a < v.size(); ++a)
        for (size_t b = a + 1; b < v.size(); ++b)
          if (v[a].bi0 <= v[b].bi1 && v[b].bi0 <= v[a].bi1 && v[a].bj0 <= v[b].bj1 && v[b].bj0 <= v[a].bj1)
            parent[find(v[a].t)] = find(v[b].t);
    }
  }
  std::vector<int> unit(ntensors);
  for (int t = 0; t < ntensors; ++t) unit[t] = find(t);
  return unit;
}

// Rounds: each a run of units (tensors sharing an fp8 block stay together)
// in catalog order. Filling with a cap X: a unit that would push some
// sender's send bytes or some receiver's receive bytes past X opens the next
// round, so a rank goes past X in a round only through the round's first
// unit (one larger than X on its own). The count n is what
// filling with the budget needs (App. D); the rounds are the filling with the
// smallest cap X <= budget that still needs only n rounds (bisection over
// whole bytes), so the largest round is as small as n rounds allow and the
// chunks come out about equal (Sec. 3.2). Returns n.
int assign_rounds(const wb_layout_t& trainer, const wb_layout_t& rollout, std::vector<Segment>& segs,
                  int64_t budget) {
  const int nt = static_cast<int>(trainer.catalog.size());
  const std::vector<int> unit = block_units(rollout, nt);
  std::vector<std::vector<size_t>> members(nt);  // indexed by unit root
  std::vector<int> first(nt, nt);
  for (size_t i = 0; i < segs.size(); ++i) {
    const int u = unit[segs[i].t];
    members[u].push_back(i);
    first[u] = std::min(first[u], segs[i].t);
  }
  std::vector<int> order;
  for (int u = 0; u < nt; ++u)
    if (!members[u].empty()) order.push_back(u);
  std::sort(order.begin(), order.end(), [&](int a, int b) { return first[a] < first[b]; });
  // bytes of every unit per rank: keys 0..ns-1 senders, ns.. receivers
  const size_t ns = trainer.ranks.size(), nd = rollout.ranks.size();
  std::vector<std::vector<std::pair<int, int64_t>>> size(order.size());
  std::vector<int64_t> add(ns + nd, 0), total(ns + nd, 0);
  for (size_t k = 0; k < order.size(); ++k) {
    std::vector<int> keys;
    for (size_t i : members[order[k]]) {
      const Segment& g = segs[i];
      const int ks[2] = {g.stage == 0 ? g.s : -1, static_cast<int>(ns) + g.d};
      for (int key : ks) {
        if (key < 0) continue;
        if (add[key] == 0) keys.push_back(key);
        add[key] += g.bytes;
      }
    }
    for (int key : keys) size[k].push_back({key, add[key]}), total[key] += add[key], add[key] = 0;
  }
  std::vector<int> rounds(order.size(), 0);
  std::vector<int64_t> cur(ns + nd, 0);
  auto fill = [&](int64_t cap) {  // returns the number of rounds
    std::fill(cur.begin(), cur.end(), 0);
    int r = 0;
    bool empty = true;
    for (size_t k = 0; k < order.size(); ++k) {
      bool over = false;
      for (const auto& kv : size[k]) over = over || cur[kv.first] + kv.second > cap;
      if (over && !empty) {
        ++r;
        std::fill(cur.begin(), cur.end(), 0);
      }
      for (const auto& kv : size[k]) cur[kv.first] += kv.second;
      empty = false;
      rounds[k] = r;
    }
    return r + 1;
  };
  const int n = fill(budget);
  int64_t lo = 1, hi = budget;
  for (int64_t t : total) lo = std::max(lo, (t + n - 1) / n);
  while (lo < hi) {
    const int64_t mid = lo + (hi - lo) / 2;
    if (fill(mid) <= n)
      hi = mid;
    else
      lo = mid + 1;
  }
  fill(std::min(lo, budget));
  for (size_t k = 0; k < order.size(); ++k)
    for (size_t i : members[order[k]]) segs[i].round = rounds[k];
  return order.empty() ? 1 : rounds.back() + 1;
}

// The segments of every (round, stage), each list in canonical order.
struct SegRange {
  const uint32_t *first, *last;
};
struct SegIndex {
  std::vector<uint32_t> idx, start;
  SegIndex(const std::vector<Segment>& segs, int nrounds) : idx(segs.size()), start(size_t(nrounds) * 3 + 1, 0) {
    for (const Segment& g : segs) ++start[size_t(g.round) * 3 + g.stage + 1];
    for (size_t i = 1; i < start.size(); ++i) start[i] += start[i - 1];
    std::vector<uint32_t> fill(start.begin(), start.end() - 1);
    for (size_t i = 0; i < segs.size(); ++i) idx[fill[size_t(segs[i].round) * 3 + segs[i].stage]++] = uint32_t(i);
  }
  SegRange of(int k, int stage) const {
    return {idx.data() + start[size_t(k) * 3 + stage], idx.data() + start[size_t(k) * 3 + stage + 1]};
  }
};

// Wire offsets of one stage of round k (segments in canonical order, payloads
// at multiples of 256 bytes within their region, regions at multiples of 4096
// bytes; senders' buffers by ascending receiver, receivers' by ascending
// sender). Offsets are relative to the stage's receive section.
void wire_stage(std::vector<Segment>& segs, const SegRange& in, int ns, int nd, StageWire& W) {
  std::vector<int64_t> end(size_t(ns) * nd, -1);
  for (const uint32_t* i = in.first; i != in.last; ++i) {
    Segment& g = segs[*i];
    int64_t& e = end[size_t(g.s) * nd + g.d];
    const int64_t off = e < 0 ? 0 : align_up(e, kPayloadAlign);
    g.send_off = g.recv_off = off;
    e = off + g.bytes;
  }
  W.region_bytes.assign(size_t(ns) * nd, 0);
  W.send_region.assign(size_t(ns) * nd, -1);
  W.recv_region.assign(size_t(ns) * nd, -1);
  W.send_bytes.assign(ns, 0);
  W.recv_bytes.assign(nd, 0);
  for (int s = 0; s < ns; ++s) {
    int64_t pos = 0;
    for (int d = 0; d < nd; ++d) {
      const int64_t b = end[size_t(s) * nd + d];
      if (b < 0) continue;
      pos = align_up(pos, kRegionAlign);
      W.send_region[size_t(s) * nd + d] = pos;
      W.region_bytes[size_t(s) * nd + d] = b;
      pos += b;
    }
    W.send_bytes[s] = pos;
  }
  for (int d = 0; d < nd; ++d) {
    int64_t pos = 0;
    for (int s = 0; s < ns; ++s) {
      const int64_t b = end[size_t(s) * nd + d];
      if (b < 0) continue;
      pos = align_up(pos, kRegionAlign);
      W.recv_region[size_t(s) * nd + d] = pos;
      pos += b;
    }
    W.recv_bytes[d] = pos;
  }
  for (const uint32_t* i = in.first; i != in.last; ++i) {
    Segment& g = segs[*i];
    g.send_off += W.send_region[size_t(g.s) * nd + g.d];
    g.recv_off += W.recv_region[size_t(g.s) * nd + g.d];
  }
}

// All stages of round k: the exchange sections follow the receive section in
// every rollout rank's buffer (a non-empty section starts on a 4096-byte
// boundary); forwarded segments read where their source segment landed.
void wire_round(wb_plan_t& P, int k, const SegIndex& at) {
  const int ns = P.n_send, nd = P.n_recv;
  RoundWire& W = P.rounds[k];
  wire_stage(P.segs, at.of(k, 0), ns, nd, W.st[0]);
  W.recv_total = W.st[0].recv_bytes;
  for (int stage = 1; stage <= 2; ++stage) {
    StageWire& S = W.st[stage];
    const SegRange in = at.of(k, stage);
    wire_stage(P.segs, in, nd, nd, S);
    std::vector<int64_t> base(nd);
    for (int d = 0; d < nd; ++d) {
      if (S.recv_bytes[d]) W.recv_total[d] = align_up(W.recv_total[d], kRegionAlign);
      base[d] = W.recv_total[d];
      W.recv_total[d] += S.recv_bytes[d];
    }
    for (size_t i = 0; i < S.recv_region.size(); ++i)
      if (S.recv_region[i] >= 0) S.recv_region[i] += base[i % nd];
    for (const uint32_t* i = in.first; i != in.last; ++i) {
      Segment& g = P.segs[*i];
      g.recv_off += base[g.d];
      g.src_off = P.segs[g.src_seg].recv_off;
    }
  }
}

}  // namespace

void build_plan(const wb_layout_t& trainer, const wb_layout_t& rollout, int role, int rank, int64_t round_budget,
                int node_size, wb_plan_t& P) {
  if (role != WB_SENDER && role != WB_RECEIVER) fail(WB_EINVAL, "role must be WB_SENDER or WB_RECEIVER");
  const int ns = static_cast<int>(trainer.ranks.size()), nd = static_cast<int>(rollout.ranks.size());
  if (ns < 1 || nd < 1) fail(WB_EINVAL, "layouts need at least one rank");
  if (rank < 0 || rank >= (role == WB_SENDER ? ns : nd)) fail(WB_EINVAL, "rank out of range");
  if (trainer.catalog.size() != rollout.catalog.size()) fail(WB_EINVAL, "trainer and rollout catalogs differ");
  for (size_t t = 0; t < trainer.catalog.size(); ++t) {
    const Tensor &a = trainer.catalog[t], &b = rollout.catalog[t];
    if (a.name != b.name || a.rows != b.rows || a.cols != b.cols) fail(WB_EINVAL, "trainer and rollout catalogs differ");
  }
  validate_layout(trainer, false, "trainer");
  validate_layout(rollout, true, "rollout");
  for (const Rank& R : rollout.ranks)
    for (const Local& l : R.locals)
      if (l.block > 128) fail(WB_EUNSUPPORTED, "quant_block above 128");

  // 1. trainer groups, ordered by (t, r0, c0, r1, c1), owners ascending
  struct Entry {
    int t;
    Rect x;
    int s, pl;
  };
  std::vector<Entry> entries;
  for (int s = 0; s < ns; ++s)
    for (size_t i = 0; i < trainer.ranks[s].pls.size(); ++i) {
      const Placement& p = trainer.ranks[s].pls[i];
      entries.push_back({p.t, rect_of(p), s, static_cast<int>(i)});
    }
  std::sort(entries.begin(), entries.end(), [](const Entry& a, const Entry& b) {
    if (a.t != b.t) return a.t < b.t;
    if (a.x.r0 != b.x.r0) return a.x.r0 < b.x.r0;
    if (a.x.c0 != b.x.c0) return a.x.c0 < b.x.c0;
    if (a.x.r1 != b.x.r1) return a.x.r1 < b.x.r1;
    if (a.x.c1 != b.x.c1) return a.x.c1 < b.x.c1;
    return a.s < b.s;
  });
  std::vector<std::vector<Group>> groups(trainer.catalog.size());
  std::map<std::vector<int>, int> set_ids;
  for (size_t i = 0; i < entries.size();) {
    size_t j = i;
    Group g;
    g.x = entries[i].x;
    while (j < entries.size() && entries[j].t == entries[i].t && entries[j].x.r0 == g.x.r0 &&
           entries[j].x.r1 == g.x.r1 && entries[j].x.c0 == g.x.c0 && entries[j].x.c1 == g.x.c1) {
      if (!g.owners.empty() && g.owners.back() == entries[j].s)
        fail(WB_EINVAL, "a trainer rank holds the same rectangle twice");
      g.owners.push_back(entries[j].s);
      g.pls.push_back(entries[j].pl);
      ++j;
    }
    int es = 0;
    for (size_t k = 0; k < g.owners.size(); ++k) {
      const Rank& S = trainer.ranks[g.owners[k]];
      const int e = dtype_bytes(S.locals[S.pls[g.pls[k]].u].dtype);
      if (es && e != es) fail(WB_EUNSUPPORTED, "replicas of one rectangle hold different dtypes");
      es = e;
    }
    g.esize = es;
    auto it = set_ids.emplace(g.owners, static_cast<int>(set_ids.size())).first;
    g.set = it->second;
    groups[entries[i].t].push_back(std::move(g));
    i = j;
  }
  for (auto& gl : groups)
    for (size_t a = 0; a < gl.size(); ++a)
      for (size_t b = a + 1; b < gl.size(); ++b) {
        Rect tmp;
        if (intersect(gl[a].x, gl[b].x, tmp))
          fail(WB_EUNSUPPORTED, "overlapping, non-identical trainer rectangles");
      }

  // 6. rollout groups (identical rollout rectangles, holders ascending) and
  // the hand-out of a replicated group's parts over its holders
  if (node_size < 0) fail(WB_EINVAL, "node size must be >= 0");
  const int G = node_size;
  struct RGroup {
    std::vector<int> holders, pls, who;
    std::vector<Rect> parts;
  };
  std::vector<RGroup> rgroups;
  std::vector<std::vector<int>> rg_of(nd);
  if (G > 0) {
    std::map<std::array<int64_t, 5>, int> by_key;
    for (int d = 0; d < nd; ++d) {
      const Rank& R = rollout.ranks[d];
      rg_of[d].assign(R.pls.size(), -1);
      for (size_t qi = 0; qi < R.pls.size(); ++qi) {
        const Placement& q = R.pls[qi];
        auto it = by_key.emplace(std::array<int64_t, 5>{q.t, q.r0, q.r1, q.c0, q.c1}, static_cast<int>(rgroups.size()));
        if (it.second) rgroups.emplace_back();
        RGroup& h = rgroups[it.first->second];
        if (!h.holders.empty() && h.holders.back() == d) fail(WB_EINVAL, "a rollout rank holds the same rectangle twice");
        h.holders.push_back(d);
        h.pls.push_back(static_cast<int>(qi));
        rg_of[d][qi] = it.first->second;
      }
    }
    std::map<std::vector<int>, std::vector<int64_t>> rdeficit;
    for (int d = 0; d < nd; ++d)
      for (size_t qi = 0; qi < rollout.ranks[d].pls.size(); ++qi) {
        RGroup& h = rgroups[rg_of[d][qi]];
        if (h.holders.size() == 1 || h.holders[0] != d) continue;
        const Rect x = rect_of(rollout.ranks[d].pls[qi]);
        split_parts(x, static_cast<int>(h.holders.size()), h.parts);
        std::vector<int64_t>& E = rdeficit.emplace(h.holders, std::vector<int64_t>(h.holders.size(), 0)).first->second;
        deal(h.parts, E, x.numel(), 1, h.who);
      }
  }

  // 2./3. regions and stage-0 segments in canonical order, deficit assignment
  // per owner set; with exchange stages a replicated rollout group asks the
  // trainers only for each holder's parts
  std::vector<std::vector<int64_t>> deficit(set_ids.size());
  for (const auto& kv : set_ids) deficit[kv.second].assign(kv.first.size(), 0);
  P.segs.clear();
  std::vector<Rect> parts, needs;
  std::vector<int> who;
  for (int d = 0; d < nd; ++d) {
    const Rank& R = rollout.ranks[d];
    for (size_t qi = 0; qi < R.pls.size(); ++qi) {
      const Placement& q = R.pls[qi];
      needs.clear();
      if (G > 0 && rgroups[rg_of[d][qi]].holders.size() > 1) {
        const RGroup& h = rgroups[rg_of[d][qi]];
        for (size_t j = 0; j < h.parts.size(); ++j)
          if (h.holders[h.who[j]] == d) needs.push_back(h.parts[j]);
      } else {
        needs.push_back(rect_of(q));
      }
      for (const Rect& need : needs) {
        int64_t covered = 0;
        for (const Group& g : groups[q.t]) {
          Rect x;
          if (!intersect(need, g.x, x)) continue;
          covered += x.numel();
          const int k = static_cast<int>(g.owners.size());
          if (k == 1) {
            P.segs.push_back({g.owners[0], d, q.t, x, g.pls[0], static_cast<int>(qi), x.numel() * g.esize});
            P.segs.back().origin = static_cast<int>(P.segs.size() - 1);
            continue;
          }
          split_parts(x, k, parts);
          deal(parts, deficit[g.set], x.numel() * g.esize, g.esize, who);
          for (size_t j = 0; j < parts.size(); ++j) {
            P.segs.push_back({g.owners[who[j]], d, q.t, parts[j], g.pls[who[j]], static_cast<int>(qi),
                              parts[j].numel() * g.esize});
            P.segs.back().origin = static_cast<int>(P.segs.size() - 1);
          }
        }
        if (covered != need.numel())
          fail(WB_EINVAL, "rollout rank " + std::to_string(d) + " needs elements no trainer holds");
      }
    }
  }

  // 6. exchange stages: stage 1 sends every stage-0 segment of a replicated
  // group to one holder in each other node (same position in that node's
  // holder list, modulo its length); stage 2 sends every stage-0 and stage-1
  // segment to the other holders in the receiver's node
  if (G > 0) {
    const size_t n0 = P.segs.size();
    size_t more = 0;  // every holder of a replicated group receives each of its segments once
    for (size_t gi = 0; gi < n0; ++gi) more += rgroups[rg_of[P.segs[gi].d][P.segs[gi].dst_pl]].holders.size() - 1;
    P.segs.reserve(n0 + more);
    for (size_t gi = 0; gi < n0; ++gi) {
      const Segment g = P.segs[gi];
      const RGroup& h = rgroups[rg_of[g.d][g.dst_pl]];
      if (h.holders.size() == 1) continue;
      int pos = 0;
      for (int x : h.holders) {
        if (x == g.d) break;
        if (x / G == g.d / G) ++pos;
      }
      for (size_t a = 0; a < h.holders.size();) {
        const int v = h.holders[a] / G;
        size_t b = a;
        while (b < h.holders.size() && h.holders[b] / G == v) ++b;
        if (v != g.d / G) {
          const size_t k = a + size_t(pos) % (b - a);
          Segment f{g.d, h.holders[k], g.t, g.x, -1, h.pls[k], g.bytes};
          f.stage = 1;
          f.src_seg = static_cast<int>(gi);
          f.origin = g.origin;
          P.segs.push_back(f);
        }
        a = b;
      }
    }
    const size_t n1 = P.segs.size();
    for (size_t gi = 0; gi < n1; ++gi) {
      const Segment g = P.segs[gi];
      const RGroup& h = rgroups[rg_of[g.d][g.dst_pl]];
      for (size_t k = 0; k < h.holders.size(); ++k) {
        const int z = h.holders[k];
        if (z == g.d || z / G != g.d / G) continue;
        Segment f{g.d, z, g.t, g.x, -1, h.pls[k], g.bytes};
        f.stage = 2;
        f.src_seg = static_cast<int>(gi);
        f.origin = g.origin;
        P.segs.push_back(f);
      }
    }
  }

  if (P.segs.size() > 0x7FFFFFFF) fail(WB_EUNSUPPORTED, "too many segments");

  // 5. rounds, then 4. wire offsets per round
  P.n_send = ns;
  P.n_recv = nd;
  P.node_size = G;
  const int nrounds = round_budget > 0 ? assign_rounds(trainer, rollout, P.segs, round_budget) : 1;
  P.rounds.assign(nrounds, RoundWire{});
  const SegIndex at(P.segs, nrounds);
  for (int k = 0; k < nrounds; ++k) wire_round(P, k, at);

  P.role = role;
  P.rank = rank;
  build_rank_view(trainer, rollout, P);
  // each launch range ordered by work item class (planner order within a class)
  auto partition = [&](uint32_t a, uint32_t b) {
    const auto first = P.tasks.begin() + a, last = P.tasks.begin() + b;
    const auto mid0 = std::stable_partition(first, last, [](const Task& t) { return task_class(t) == 0; });
    const auto mid1 = std::stable_partition(mid0, last, [](const Task& t) { return task_class(t) == 1; });
    const auto mid2 = std::stable_partition(mid1, last, [](const Task& t) { return task_class(t) == 2; });
    TaskSplit sp;
    sp.n[0] = static_cast<uint32_t>(mid0 - first);
    sp.n[1] = static_cast<uint32_t>(mid1 - mid0);
    sp.tiles = static_cast<uint32_t>(last - mid2);
    for (int c = 0; c < 2; ++c) {
      uint32_t most = 1;  // workgroups of the copy kernel per item of class c in this launch
      for (auto it = c == 0 ? first : mid0; it != (c == 0 ? mid0 : mid1); ++it) most = std::max(most, task_chunks(*it));
      while ((1u << sp.s[c]) < most) ++sp.s[c];
    }
    return sp;
  };
  const size_t nr = P.rounds.size();
  P.round_split.assign(nr, TaskSplit{});
  for (auto& f : P.fwd_split) f.assign(nr, TaskSplit{});
  for (size_t k = 0; k < nr; ++k) {
    P.round_split[k] = partition(P.round_tasks[k], P.round_tasks[k + 1]);
    for (int st = 0; st < 2; ++st) P.fwd_split[st][k] = partition(P.round_fwd[st][k], P.round_fwd[st][k + 1]);
    for (uint32_t ti = P.round_tasks[k + 1] - P.round_split[k].tiles; ti < P.round_tasks[k + 1]; ++ti) {
      const Task& t = P.tasks[ti];
      P.tile_read_bytes += int64_t(t.rows) * t.cols * dtype_bytes(t.sdt);
      P.tile_write_bytes += int64_t(t.rows) * t.cols * dtype_bytes(t.ddt);
    }
  }
  check_work(P, role == WB_SENDER ? trainer.ranks[rank] : rollout.ranks[rank]);
}

std::string dump_plan(const wb_plan_t& P) {
  std::ostringstream o;
  auto seg = [&](const Segment& g) {
    static const char* kTag[3] = {"seg ", "xseg ", "iseg "};
    o << kTag[g.stage] << g.s << " " << g.d << " " << g.t << " " << g.x.r0 << " " << g.x.r1 << " " << g.x.c0 << " "
      << g.x.c1 << " ";
    if (g.stage == 0)
      o << g.src_pl;
    else
      o << g.src_off;
    o << " " << g.dst_pl << " " << g.send_off << " " << g.recv_off << " " << g.bytes << "\n";
  };
  auto sizes = [&](const RoundWire& W) {
    for (int s = 0; s < P.n_send; ++s) o << "send " << s << " " << W.st[0].send_bytes[s] << "\n";
    for (int d = 0; d < P.n_recv; ++d) o << "recv " << d << " " << W.recv_total[d] << "\n";
    if (P.node_size)
      for (int st = 1; st <= 2; ++st)
        for (int d = 0; d < P.n_recv; ++d) o << "fwd" << st << " " << d << " " << W.st[st].send_bytes[d] << "\n";
  };
  o << "plan trainer_ranks=" << P.n_send << " rollout_ranks=" << P.n_recv << " segments=" << P.segs.size();
  if (P.node_size) o << " node_size=" << P.node_size;
  if (P.rounds.size() == 1) {
    o << "\n";
    sizes(P.rounds[0]);
    for (const Segment& g : P.segs) seg(g);
    return o.str();
  }
  o << " rounds=" << P.rounds.size() << "\n";
  std::vector<size_t> start(P.rounds.size() + 1, 0), idx(P.segs.size());  // segments by round, in order
  for (const Segment& g : P.segs) ++start[g.round + 1];
  for (size_t k = 0; k < P.rounds.size(); ++k) start[k + 1] += start[k];
  {
    std::vector<size_t> fill(start.begin(), start.end() - 1);
    for (size_t i = 0; i < P.segs.size(); ++i) idx[fill[P.segs[i].round]++] = i;
  }
  for (size_t k = 0; k < P.rounds.size(); ++k) {
    o << "round " << k << "\n";
    sizes(P.rounds[k]);
    for (size_t i = start[k]; i < start[k + 1]; ++i) seg(P.segs[idx[i]]);
  }
  return o.str();
}

}  // namespace wb
