// Source maps from probed identifiers (WeightBridge Sec. 3.1 and App. B,
// Algorithm 1): the recombination of the per-pass diff2 entries and the scan
// that turns them back into slice-copy placements.
//
// Identifiers are 2^24 + the element's flat position in the checkpoint; a
// local tensor is seen as a [batch * rows, cols] field A. Pass k loads chunk
// k (16 bits) of every identifier and keeps the non-zero entries of diff2 of
// that chunk field; sum_k 2^(16 k) of them is diff2(A) exactly (diff2 is
// linear). The scan never materialises A: with Z = diff2(A) sparse, A is the
// double prefix sum A(i,j) = sum_{a<=i, b<=j} Z(a,b) (i-a+1)(j-b+1), so between
// consecutive rows and columns that hold entries (a *cell*) A is a bilinear
// polynomial whose coefficients are prefix sums of four moments of Z. Inside
// one slice copy A is affine; cells are merged into maximal affine rectangles
// and each rectangle is decoded into checkpoint placements.
#include <algorithm>
#include <map>
#include <unordered_map>

#include "wb_internal.hpp"

namespace wb {
namespace {

using i128 = __int128;

constexpr int64_t kFirstId = int64_t(1) << 24;
constexpr int kChunkBits = 16;
constexpr size_t kMaxCells = size_t(1) << 22;

int64_t to_i64(i128 v) {
  if (v > i128(INT64_MAX) || v < i128(INT64_MIN)) fail(WB_EUNSUPPORTED, "identifier field out of range");
  return static_cast<int64_t>(v);
}

// One affine region: rows [r0, r0 + h), cols [c0, c0 + w); the value at
// (r0, c0) and the steps per row and per column (unknown for a single row or
// column).
struct Region {
  int64_t r0, h, c0, w;
  int64_t v0;
  bool has_di, has_dj;
  int64_t di, dj;
  bool zero() const { return v0 == 0 && (!has_di || di == 0) && (!has_dj || dj == 0); }
};

struct Decoder {
  const wb_probe_t& P;
  int u;
  int64_t C;  // local columns (of the [batch * rows, cols] view)
  std::vector<Placement>& out;

  // checkpoint tensor holding identifier id, or fail
  int tensor_of(int64_t id) const {
    if (id < kFirstId || id >= P.end_id) fail(WB_EUNSUPPORTED, "a local element holds a value that is no identifier");
    const auto it = std::upper_bound(P.first.begin(), P.first.end(), id);
    return static_cast<int>(it - P.first.begin()) - 1;
  }

  void emit(int t, int64_t r0, int64_t r1, int64_t c0, int64_t c1, int64_t base, int64_t ld, int tr) {
    Placement p;
    p.t = t;
    p.u = u;
    p.r0 = r0;
    p.r1 = r1;
    p.c0 = c0;
    p.c1 = c1;
    p.base = base;
    p.ld = ld;
    p.tr = tr;
    out.push_back(p);
  }

  // A run of len local elements starting at local flat index n0, local step
  // ls (1 along a row, C down a column), identifiers s, s + st, ...
  void run(int64_t s, int64_t st, int64_t len, int64_t n0, int64_t ls) {
    while (len > 0) {
      const int t = tensor_of(s);
      const Tensor& T = P.catalog[t];
      const int64_t off = s - P.first[t], r = off / T.cols, c = off % T.cols;
      int64_t k;
      if (st == 1 && ls == 1) {
        // contiguous on both sides: a flat run, as a partial head row, whole
        // rows and a partial tail row
        k = std::min(len, T.numel() - off);
        int64_t p = off, n = n0;
        const int64_t p1 = off + k;
        if (p % T.cols) {
          const int64_t e = std::min(p1, (p / T.cols + 1) * T.cols);
          emit(t, p / T.cols, p / T.cols + 1, p % T.cols, p % T.cols + (e - p), n, T.cols, 0);
          n += e - p;
          p = e;
        }
        if (p1 - p >= T.cols) {
          const int64_t rows = (p1 - p) / T.cols;
          emit(t, p / T.cols, p / T.cols + rows, 0, T.cols, n, T.cols, 0);
          n += rows * T.cols;
          p += rows * T.cols;
        }
        if (p < p1) emit(t, p / T.cols, p / T.cols + 1, 0, p1 - p, n, T.cols, 0);
      } else if (st == 1) {
        // consecutive identifiers down a local column: one checkpoint row
        // piece at a time, stored transposed
        k = std::min(len, T.cols - c);
        emit(t, r, r + 1, c, c + k, n0, ls, 1);
      } else if (st == T.cols) {
        // one checkpoint column, row after row
        k = std::min(len, T.rows - r);
        emit(t, r, r + k, c, c + 1, n0, ls, 0);
      } else {
        k = 1;
        emit(t, r, r + 1, c, c + 1, n0, 1, 0);
      }
      s += k * st;
      n0 += k * ls;
      len -= k;
    }
  }

  bool slab(const Region& g) {
    const size_t mark = out.size();
    int64_t s = g.v0, rr = g.r0;
    while (rr < g.r0 + g.h) {
      const int t = tensor_of(s);
      const Tensor& T = P.catalog[t];
      const int64_t off = s - P.first[t], r = off / T.cols, c = off % T.cols;
      if (g.di != T.cols || c + g.w > T.cols || tensor_of(s + g.w - 1) != t) {
        out.resize(mark);
        return false;
      }
      const int64_t k = std::min(g.r0 + g.h - rr, T.rows - r);
      emit(t, r, r + k, c, c + g.w, rr * C + g.c0, C, 0);
      s += k * g.di;
      rr += k;
    }
    return true;
  }

  bool transposed(const Region& g) {
    const int t = tensor_of(g.v0);
    const Tensor& T = P.catalog[t];
    const int64_t off = g.v0 - P.first[t], r = off / T.cols, c = off % T.cols;
    if (g.dj != T.cols || c + g.h > T.cols || r + g.w > T.rows) return false;
    emit(t, r, r + g.w, c, c + g.h, g.r0 * C + g.c0, C, 1);
    return true;
  }

  void region(const Region& g) {
    if (g.zero()) return;
    const int64_t n0 = g.r0 * C + g.c0;
    if (g.h == 1 && g.w == 1) return run(g.v0, 1, 1, n0, 1);
    if (g.h == 1) return run(g.v0, g.dj, g.w, n0, 1);
    if (g.w == 1) return run(g.v0, g.di, g.h, n0, C);
    if (g.dj == 1 && g.w == C && g.di == C) return run(g.v0, 1, g.h * g.w, n0, 1);
    if (g.dj == 1 && slab(g)) return;
    if (g.di == 1 && transposed(g)) return;
    for (int64_t k = 0; k < g.h; ++k) run(g.v0 + k * g.di, g.dj, g.w, n0 + k * C, 1);
  }
};

void scan_local(const wb_probe_t& P, int u, std::vector<Placement>& out) {
  const ProbeLocal& L = P.locals[u];
  const int64_t R = L.batch * L.rows, C = L.cols;
  struct Entry {
    int64_t i, j;
    i128 v;
  };
  std::vector<Entry> z;
  z.reserve(L.z.size());
  for (const auto& kv : L.z)
    if (kv.second != 0) z.push_back({kv.first / C, kv.first % C, kv.second});
  std::vector<int64_t> I{0}, J{0};
  for (const Entry& e : z) {
    I.push_back(e.i);
    J.push_back(e.j);
  }
  std::sort(I.begin(), I.end());
  I.erase(std::unique(I.begin(), I.end()), I.end());
  std::sort(J.begin(), J.end());
  J.erase(std::unique(J.begin(), J.end()), J.end());
  const size_t ni = I.size(), nj = J.size();
  if (ni * nj > kMaxCells) fail(WB_EUNSUPPORTED, "local tensor " + L.name + " has too many distinct slice boundaries");
  // moments of Z per coarse grid point, then prefix sums: A = M0 i j - Mb i - Ma j + Mab
  std::vector<i128> M0(ni * nj, 0), Ma(ni * nj, 0), Mb(ni * nj, 0), Mab(ni * nj, 0);
  for (const Entry& e : z) {
    const size_t p = std::lower_bound(I.begin(), I.end(), e.i) - I.begin();
    const size_t q = std::lower_bound(J.begin(), J.end(), e.j) - J.begin();
    const size_t k = p * nj + q;
    M0[k] += e.v;
    Ma[k] += e.v * i128(e.i - 1);
    Mb[k] += e.v * i128(e.j - 1);
    Mab[k] += e.v * i128(e.i - 1) * i128(e.j - 1);
  }
  for (auto* M : {&M0, &Ma, &Mb, &Mab}) {
    for (size_t p = 0; p < ni; ++p)
      for (size_t q = 1; q < nj; ++q) (*M)[p * nj + q] += (*M)[p * nj + q - 1];
    for (size_t p = 1; p < ni; ++p)
      for (size_t q = 0; q < nj; ++q) (*M)[p * nj + q] += (*M)[(p - 1) * nj + q];
  }
  auto field = [&](size_t k, int64_t i, int64_t j) -> i128 {
    return M0[k] * i128(i) * i128(j) - Mb[k] * i128(i) - Ma[k] * i128(j) + Mab[k];
  };
  Decoder dec{P, u, C, out};
  std::map<std::pair<int64_t, int64_t>, Region> open;  // by (c0, w), regions reaching the previous band
  for (size_t p = 0; p < ni; ++p) {
    const int64_t r0 = I[p], h = (p + 1 < ni ? I[p + 1] : R) - r0;
    // cells of this band, merged left to right
    std::vector<Region> band;
    for (size_t q = 0; q < nj; ++q) {
      const int64_t c0 = J[q], w = (q + 1 < nj ? J[q + 1] : C) - c0;
      const size_t k = p * nj + q;
      if (h >= 2 && w >= 2 && M0[k] != 0) fail(WB_EUNSUPPORTED, "local tensor " + L.name + " is not made of slice copies");
      Region g{r0, h, c0, w, to_i64(field(k, r0, c0)), h >= 2, w >= 2, 0, 0};
      if (g.has_di) g.di = to_i64(field(k, r0 + 1, c0) - field(k, r0, c0));
      if (g.has_dj) g.dj = to_i64(field(k, r0, c0 + 1) - field(k, r0, c0));
      if (!band.empty()) {
        Region& b = band.back();
        if (b.zero() && g.zero()) {
          b.w += g.w;
          continue;
        }
        if (!b.zero() && !g.zero() && b.has_di == g.has_di && (!b.has_di || b.di == g.di)) {
          const int64_t step = b.has_dj ? b.dj : g.v0 - b.v0;
          if (g.v0 == b.v0 + step * b.w && (!g.has_dj || g.dj == step)) {
            b.w += g.w;
            b.has_dj = true;
            b.dj = step;
            continue;
          }
        }
      }
      band.push_back(g);
    }
    // continue the regions of the previous band where the field carries on
    std::map<std::pair<int64_t, int64_t>, Region> next;
    for (const Region& g : band) {
      const auto key = std::make_pair(g.c0, g.w);
      auto it = open.find(key);
      if (it != open.end()) {
        Region& o = it->second;
        bool ok = o.zero() && g.zero();
        if (!ok && !o.zero() && !g.zero() && o.has_dj == g.has_dj && (!o.has_dj || o.dj == g.dj)) {
          const int64_t step = o.has_di ? o.di : g.v0 - o.v0;
          if (g.v0 == o.v0 + step * o.h && (!g.has_di || g.di == step)) {
            o.has_di = true;
            o.di = step;
            ok = true;
          }
        }
        if (ok) {
          o.h += g.h;
          next.emplace(key, o);
          open.erase(it);
          continue;
        }
      }
      next.emplace(key, g);
    }
    for (const auto& kv : open) dec.region(kv.second);
    open.swap(next);
  }
  for (const auto& kv : open) dec.region(kv.second);
}

}  // namespace

void probe_init(wb_probe_t& P, const wb_tensor_desc* catalog, int n, int ckpt_dtype) {
  if (ckpt_dtype != WB_F32 && ckpt_dtype != WB_BF16)
    fail(WB_EUNSUPPORTED, "probing needs an f32 or bf16 checkpoint (16 identifier bits per pass)");
  P.dtype = ckpt_dtype;
  P.bits = kChunkBits;
  int64_t id = kFirstId;
  for (int t = 0; t < n; ++t) {
    if (!catalog[t].name || catalog[t].rows < 1 || catalog[t].cols < 1) fail(WB_EINVAL, "bad catalog tensor");
    P.catalog.push_back({catalog[t].name, catalog[t].rows, catalog[t].cols});
    P.first.push_back(id);
    id += catalog[t].rows * catalog[t].cols;
  }
  P.end_id = id;
  int bits = 0;
  for (int64_t x = id - 1; x > 0; x >>= 1) ++bits;
  P.nchunks = (bits + P.bits - 1) / P.bits;
}

void probe_record(wb_probe_t& P, int local, int chunk, const int64_t* index, const int64_t* value, int64_t n) {
  if (local < 0 || local >= static_cast<int>(P.locals.size())) fail(WB_EINVAL, "local index out of range");
  if (chunk < 0 || chunk >= P.nchunks) fail(WB_EINVAL, "chunk out of range");
  if (n < 0 || (n > 0 && (!index || !value))) fail(WB_EINVAL, "bad entry arrays");
  ProbeLocal& L = P.locals[local];
  const int64_t numel = L.batch * L.rows * L.cols;
  for (int64_t k = 0; k < n; ++k) {
    if (index[k] < 0 || index[k] >= numel) fail(WB_EINVAL, "entry index outside the local tensor");
    L.z[index[k]] += i128(value[k]) << (P.bits * chunk);
  }
}

void probe_scan(const wb_probe_t& P, wb_layout_t& out, int rank) {
  if (rank < 0 || rank >= static_cast<int>(out.ranks.size())) fail(WB_EINVAL, "rank out of range");
  if (out.catalog.size() != P.catalog.size()) fail(WB_EINVAL, "layout and probe catalogs differ");
  for (size_t t = 0; t < P.catalog.size(); ++t)
    if (out.catalog[t].name != P.catalog[t].name || out.catalog[t].rows != P.catalog[t].rows ||
        out.catalog[t].cols != P.catalog[t].cols)
      fail(WB_EINVAL, "layout and probe catalogs differ");
  Rank& R = out.ranks[rank];
  if (!R.locals.empty()) fail(WB_EINVAL, "the layout rank already has local tensors");
  std::vector<Placement> pls;
  for (size_t u = 0; u < P.locals.size(); ++u) scan_local(P, static_cast<int>(u), pls);
  Rank fresh;
  for (const ProbeLocal& L : P.locals) {
    Local l;
    l.name = L.name;
    l.dtype = L.dtype;
    l.batch = L.batch;
    l.rows = L.rows;
    l.cols = L.cols;
    fresh.locals.push_back(l);
  }
  fresh.pls = std::move(pls);
  R = std::move(fresh);
  for (const Placement& p : R.pls) check_placement(out, rank, p);
}

}  // namespace wb
