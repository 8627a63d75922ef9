// Layouts: checkpoint catalogs and slice-copy placements of every rank of one
// side (WeightBridge Sec. 3.1: a worker's source map is the list of slice
// copies, each optionally transposed, that its loader performs from the full
// checkpoint; the checkpoint index space bridges trainer and rollout).
#include <algorithm>
#include <cstdio>
#include <map>
#include <sstream>

#include "wb_internal.hpp"

namespace wb {
namespace {

struct Catalog {
  std::vector<Tensor> list;
  std::map<std::string, int> index;
  void add(const std::string& n, int64_t r, int64_t c) {
    index[n] = static_cast<int>(list.size());
    list.push_back({n, r, c});
  }
  int at(const std::string& n) const {
    auto it = index.find(n);
    if (it == index.end()) fail(WB_EINVAL, "catalog has no tensor " + n);
    return it->second;
  }
};

std::string lp(int layer) { return "layers." + std::to_string(layer) + "."; }
std::string ex(int layer, int e, const char* leaf) {
  return lp(layer) + "experts." + std::to_string(e) + "." + leaf;
}

Catalog make_catalog(const wb_model_shapes& m) {
  Catalog c;
  const int64_t H = m.hidden, hd = m.head_dim;
  const bool dense = m.family == WB_FAMILY_DENSE, mix = m.family == WB_FAMILY_MIXTRAL;
  if (dense || mix) c.add("embed", m.vocab, H);
  for (int l = 0; l < m.num_layers; ++l) {
    const std::string p = lp(l);
    if (dense || mix) {
      c.add(p + "attn_norm", 1, H);
      c.add(p + "q", int64_t(m.num_heads) * hd, H);
      c.add(p + "k", int64_t(m.num_kv_heads) * hd, H);
      c.add(p + "v", int64_t(m.num_kv_heads) * hd, H);
      c.add(p + "o", H, int64_t(m.num_heads) * hd);
      c.add(p + "mlp_norm", 1, H);
    }
    if (dense) {
      c.add(p + "gate", m.ffn, H);
      c.add(p + "up", m.ffn, H);
      c.add(p + "down", H, m.ffn);
      continue;
    }
    c.add(p + "router", m.num_experts, H);
    if (m.family == WB_FAMILY_MOE_ONLY) {
      const int64_t fs = int64_t(m.ffn) * m.num_shared_experts;
      c.add(p + "shared.gate", fs, H);
      c.add(p + "shared.up", fs, H);
      c.add(p + "shared.down", H, fs);
    }
    for (int e = 0; e < m.num_experts; ++e) {
      c.add(ex(l, e, "gate"), m.ffn, H);
      c.add(ex(l, e, "up"), m.ffn, H);
      c.add(ex(l, e, "down"), H, m.ffn);
    }
  }
  if (dense || mix) {
    c.add("final_norm", 1, H);
    c.add("lm_head", m.vocab, H);
  }
  return c;
}

// Appends locals and placements of one rank.
struct RankBuilder {
  const Catalog& cat;
  Rank r;
  explicit RankBuilder(const Catalog& c) : cat(c) {}
  int local(const std::string& name, int dtype, int64_t batch, int64_t rows, int64_t cols, int block = 0) {
    const int u = static_cast<int>(r.locals.size());
    Local l;
    l.name = name;
    l.dtype = dtype;
    l.batch = batch;
    l.rows = rows;
    l.cols = cols;
    if (block > 0) {
      l.block = block;
      l.scale = u + 1;
      r.locals.push_back(l);
      Local s;
      s.name = name + "_scale";
      s.dtype = WB_F32;
      s.batch = batch;
      s.rows = (rows + block - 1) / block;
      s.cols = (cols + block - 1) / block;
      s.scales = u;
      r.locals.push_back(s);
    } else {
      r.locals.push_back(l);
    }
    return u;
  }
  void place(const std::string& t, int64_t r0, int64_t r1, int64_t c0, int64_t c1, int u, int64_t base, int64_t ld,
             int tr = 0) {
    Placement p;
    p.t = cat.at(t);
    p.r0 = r0;
    p.r1 = r1;
    p.c0 = c0;
    p.c1 = c1;
    p.u = u;
    p.base = base;
    p.ld = ld;
    p.tr = tr;
    r.pls.push_back(p);
  }
};

void need(bool ok, const char* msg) {
  if (!ok) fail(WB_EINVAL, msg);
}

void check_tp(const wb_model_shapes& m, int tp) {
  if (m.family != WB_FAMILY_MOE_ONLY) {
    need(m.vocab % tp == 0 && m.num_heads % tp == 0 && m.num_kv_heads % tp == 0, "tp must divide vocab, heads and kv heads");
    need(m.num_kv_heads > 0 && m.num_heads % m.num_kv_heads == 0, "kv heads must divide heads");
  }
  need(m.ffn % tp == 0, "tp must divide ffn");
}

// Row-major flat run [p0, p1) of a matrix with `cols` columns as at most three
// rectangles: a partial first row, whole rows, a partial last row.
template <class F>
void flat_run(int64_t p0, int64_t p1, int64_t cols, F&& emit) {
  int64_t p = p0;
  if (p < p1 && p % cols != 0) {
    const int64_t row = p / cols, c = p % cols;
    const int64_t take = std::min(p1 - p, cols - c);
    emit(p, row, row + 1, c, c + take);
    p += take;
  }
  const int64_t whole = (p1 - p) / cols;
  if (whole > 0) {
    emit(p, p / cols, p / cols + whole, 0, cols);
    p += whole * cols;
  }
  if (p < p1) emit(p, p / cols, p / cols + 1, 0, p1 - p);
}

struct Unit {
  std::string name;
  std::vector<int> tensors;
  int group;  // expert-parallel group, -1 for units every group holds
};

std::vector<Unit> fsdp_units(const wb_model_shapes& m, const Catalog& cat, int ep) {
  std::vector<Unit> units;
  const bool has_embed = m.family != WB_FAMILY_MOE_ONLY;
  if (has_embed) units.push_back({"flat.embed", {cat.at("embed")}, -1});
  for (int l = 0; l < m.num_layers; ++l) {
    const std::string p = lp(l);
    Unit layer{"flat.layers." + std::to_string(l), {}, -1};
    std::vector<Unit> groups;
    for (int g = 0; g < ep && m.family != WB_FAMILY_DENSE; ++g)
      groups.push_back({"flat.layers." + std::to_string(l) + ".experts." + std::to_string(g), {}, g});
    const int per = m.family == WB_FAMILY_DENSE ? 0 : m.num_experts / ep;
    for (size_t t = 0; t < cat.list.size(); ++t) {
      const std::string& n = cat.list[t].name;
      if (n.compare(0, p.size(), p) != 0) continue;
      const std::string rest = n.substr(p.size());
      if (m.family != WB_FAMILY_DENSE && rest.compare(0, 8, "experts.") == 0) {
        const int e = std::stoi(rest.substr(8));
        groups[e / per].tensors.push_back(static_cast<int>(t));
      } else {
        layer.tensors.push_back(static_cast<int>(t));
      }
    }
    units.push_back(layer);
    for (auto& g : groups) units.push_back(g);
  }
  if (has_embed) units.push_back({"flat.final", {cat.at("final_norm"), cat.at("lm_head")}, -1});
  return units;
}

void style_fsdp(const wb_model_shapes& m, const wb_parallelism& par, const Catalog& cat, wb_layout_t& L) {
  need(par.fsdp >= 1 && par.ep >= 1 && par.dp >= 1 && par.tp == 1, "fsdp_flat: degrees must be >= 1 and tp == 1");
  need(m.family != WB_FAMILY_DENSE || par.ep == 1, "fsdp_flat: ep > 1 needs experts");
  need(m.family == WB_FAMILY_DENSE || m.num_experts % par.ep == 0, "fsdp_flat: ep must divide experts");
  const std::vector<Unit> units = fsdp_units(m, cat, par.ep);
  for (int dpi = 0; dpi < par.dp; ++dpi)
    for (int epi = 0; epi < par.ep; ++epi)
      for (int f = 0; f < par.fsdp; ++f) {
        RankBuilder rb(cat);
        for (const Unit& unit : units) {
          if (unit.group >= 0 && unit.group != epi) continue;
          int64_t total = 0;
          for (int t : unit.tensors) total += cat.list[t].numel();
          const int64_t shard = (total + par.fsdp - 1) / par.fsdp;
          const int64_t a = f * shard, b = a + shard;
          const int u = rb.local(unit.name, par.dtype, 1, 1, shard);
          int64_t off = 0;
          for (int t : unit.tensors) {
            const Tensor& T = cat.list[t];
            const int64_t lo = std::max(a, off), hi = std::min(b, off + T.numel());
            if (lo < hi)
              flat_run(lo - off, hi - off, T.cols, [&](int64_t first, int64_t r0, int64_t r1, int64_t c0, int64_t c1) {
                rb.place(T.name, r0, r1, c0, c1, u, off + first - a, T.cols);
              });
            off += T.numel();
          }
        }
        L.ranks.push_back(std::move(rb.r));
      }
}

void style_megatron(const wb_model_shapes& m, const wb_parallelism& par, const Catalog& cat, wb_layout_t& L) {
  const int tp = par.tp, ep = par.ep;
  need(tp >= 1 && ep >= 1 && par.dp >= 1 && par.fsdp == 1, "megatron: degrees must be >= 1 and fsdp == 1");
  need(m.family != WB_FAMILY_DENSE || ep == 1, "megatron: ep > 1 needs experts");
  if (m.family != WB_FAMILY_DENSE && (tp != 1 || m.num_experts % ep != 0))
    fail(WB_EUNSUPPORTED, "megatron: MoE layouts need tp == 1 and ep dividing the experts");
  check_tp(m, tp);
  const int64_t H = m.hidden, hd = m.head_dim;
  const int dt = par.dtype;
  const bool T = par.transposed_row_parallel != 0;
  const bool attn = m.family != WB_FAMILY_MOE_ONLY;
  for (int dpi = 0; dpi < par.dp; ++dpi)
    for (int epi = 0; epi < ep; ++epi)
      for (int r = 0; r < tp; ++r) {
        RankBuilder rb(cat);
        // row-parallel shard: columns [c0, c1) of a [rows, *] tensor
        auto row_par = [&](const std::string& local, const std::string& t, int64_t rows, int64_t c0, int64_t c1) {
          if (T) {
            rb.place(t, 0, rows, c0, c1, rb.local(local, dt, 1, c1 - c0, rows), 0, rows, 1);
          } else {
            rb.place(t, 0, rows, c0, c1, rb.local(local, dt, 1, rows, c1 - c0), 0, c1 - c0, 0);
          }
        };
        const int64_t vl = attn ? m.vocab / tp : 0;
        if (attn) rb.place("embed", r * vl, (r + 1) * vl, 0, H, rb.local("embed", dt, 1, vl, H), 0, H);
        for (int l = 0; l < m.num_layers; ++l) {
          const std::string p = lp(l);
          if (attn) {
            rb.place(p + "attn_norm", 0, 1, 0, H, rb.local(p + "attn_norm", dt, 1, 1, H), 0, H);
            const int64_t groups = m.num_kv_heads / tp, qpg = m.num_heads / m.num_kv_heads;
            const int u = rb.local(p + "qkv", dt, 1, groups * (qpg + 2) * hd, H);
            for (int64_t gi = 0; gi < groups; ++gi) {
              const int64_t g = r * groups + gi, row = gi * (qpg + 2) * hd;
              rb.place(p + "q", g * qpg * hd, (g + 1) * qpg * hd, 0, H, u, row * H, H);
              rb.place(p + "k", g * hd, (g + 1) * hd, 0, H, u, (row + qpg * hd) * H, H);
              rb.place(p + "v", g * hd, (g + 1) * hd, 0, H, u, (row + (qpg + 1) * hd) * H, H);
            }
            const int64_t ql = int64_t(m.num_heads) * hd / tp;
            row_par(p + "o", p + "o", H, r * ql, (r + 1) * ql);
            rb.place(p + "mlp_norm", 0, 1, 0, H, rb.local(p + "mlp_norm", dt, 1, 1, H), 0, H);
          }
          if (m.family == WB_FAMILY_DENSE) {
            const int64_t fl = m.ffn / tp;
            const int u = rb.local(p + "gate_up", dt, 1, 2 * fl, H);
            rb.place(p + "gate", r * fl, (r + 1) * fl, 0, H, u, 0, H);
            rb.place(p + "up", r * fl, (r + 1) * fl, 0, H, u, fl * H, H);
            row_par(p + "down", p + "down", H, r * fl, (r + 1) * fl);
            continue;
          }
          rb.place(p + "router", 0, m.num_experts, 0, H, rb.local(p + "router", dt, 1, m.num_experts, H), 0, H);
          if (m.family == WB_FAMILY_MOE_ONLY) {
            const int64_t fs = int64_t(m.ffn) * m.num_shared_experts;
            rb.place(p + "shared.gate", 0, fs, 0, H, rb.local(p + "shared.w1", dt, 1, fs, H), 0, H);
            rb.place(p + "shared.up", 0, fs, 0, H, rb.local(p + "shared.w3", dt, 1, fs, H), 0, H);
            row_par(p + "shared.w2", p + "shared.down", H, 0, fs);
          }
          const int64_t el = m.num_experts / ep, F = m.ffn;
          const int u1 = rb.local(p + "experts.w1", dt, el, F, H);
          const int u3 = rb.local(p + "experts.w3", dt, el, F, H);
          const int u2 = T ? rb.local(p + "experts.w2", dt, el, F, H) : rb.local(p + "experts.w2", dt, el, H, F);
          for (int64_t j = 0; j < el; ++j) {
            const int e = static_cast<int>(epi * el + j);
            rb.place(ex(l, e, "gate"), 0, F, 0, H, u1, j * F * H, H);
            rb.place(ex(l, e, "up"), 0, F, 0, H, u3, j * F * H, H);
            if (T)
              rb.place(ex(l, e, "down"), 0, H, 0, F, u2, j * F * H, H, 1);
            else
              rb.place(ex(l, e, "down"), 0, H, 0, F, u2, j * H * F, F);
          }
        }
        if (attn) {
          rb.place("final_norm", 0, 1, 0, H, rb.local("final_norm", dt, 1, 1, H), 0, H);
          rb.place("lm_head", r * vl, (r + 1) * vl, 0, H, rb.local("lm_head", dt, 1, vl, H), 0, H);
        }
        L.ranks.push_back(std::move(rb.r));
      }
}

void style_serving(const wb_model_shapes& m, const wb_parallelism& par, const Catalog& cat, wb_layout_t& L) {
  const int tp = par.tp, ep = par.ep;
  need(tp >= 1 && ep >= 1 && par.dp >= 1 && par.fsdp == 1 && !par.transposed_row_parallel,
       "serving: degrees must be >= 1, fsdp == 1, no transposed shards");
  need(m.family != WB_FAMILY_DENSE || ep == 1, "serving: ep > 1 needs experts");
  need(m.family == WB_FAMILY_DENSE || m.num_experts % ep == 0, "serving: ep must divide experts");
  const bool quant = par.quant_dtype == WB_F8E4M3;
  need(quant || par.quant_dtype == WB_DTYPE_NONE, "serving: quant_dtype must be none or f8e4m3");
  if (quant && (par.quant_block < 1 || par.quant_block > 128))
    fail(WB_EUNSUPPORTED, "serving: quant_block must be in 1..128");
  check_tp(m, tp);
  const int64_t H = m.hidden, hd = m.head_dim;
  const int dt = par.dtype, qdt = quant ? WB_F8E4M3 : par.dtype, qb = quant ? par.quant_block : 0;
  const bool attn = m.family != WB_FAMILY_MOE_ONLY;
  for (int dpi = 0; dpi < par.dp; ++dpi)
    for (int epi = 0; epi < ep; ++epi)
      for (int r = 0; r < tp; ++r) {
        RankBuilder rb(cat);
        const int64_t vl = attn ? m.vocab / tp : 0;
        if (attn) rb.place("embed", r * vl, (r + 1) * vl, 0, H, rb.local("embed", dt, 1, vl, H), 0, H);
        for (int l = 0; l < m.num_layers; ++l) {
          const std::string p = lp(l);
          if (attn) {
            rb.place(p + "attn_norm", 0, 1, 0, H, rb.local(p + "attn_norm", dt, 1, 1, H), 0, H);
            const int64_t ql = int64_t(m.num_heads) * hd / tp, kl = int64_t(m.num_kv_heads) * hd / tp;
            int u = rb.local(p + "qkv", qdt, 1, ql + 2 * kl, H, qb);
            rb.place(p + "q", r * ql, (r + 1) * ql, 0, H, u, 0, H);
            rb.place(p + "k", r * kl, (r + 1) * kl, 0, H, u, ql * H, H);
            rb.place(p + "v", r * kl, (r + 1) * kl, 0, H, u, (ql + kl) * H, H);
            u = rb.local(p + "o", qdt, 1, H, ql, qb);
            rb.place(p + "o", 0, H, r * ql, (r + 1) * ql, u, 0, ql);
            rb.place(p + "mlp_norm", 0, 1, 0, H, rb.local(p + "mlp_norm", dt, 1, 1, H), 0, H);
          }
          const int64_t fl = m.ffn / tp;
          if (m.family == WB_FAMILY_DENSE) {
            int u = rb.local(p + "gate_up", qdt, 1, 2 * fl, H, qb);
            rb.place(p + "gate", r * fl, (r + 1) * fl, 0, H, u, 0, H);
            rb.place(p + "up", r * fl, (r + 1) * fl, 0, H, u, fl * H, H);
            u = rb.local(p + "down", qdt, 1, H, fl, qb);
            rb.place(p + "down", 0, H, r * fl, (r + 1) * fl, u, 0, fl);
            continue;
          }
          rb.place(p + "router", 0, m.num_experts, 0, H, rb.local(p + "router", dt, 1, m.num_experts, H), 0, H);
          if (m.family == WB_FAMILY_MOE_ONLY) {
            const int64_t fsl = int64_t(m.ffn) * m.num_shared_experts / tp;
            int u = rb.local(p + "shared.w13", qdt, 1, 2 * fsl, H, qb);
            rb.place(p + "shared.gate", r * fsl, (r + 1) * fsl, 0, H, u, 0, H);
            rb.place(p + "shared.up", r * fsl, (r + 1) * fsl, 0, H, u, fsl * H, H);
            u = rb.local(p + "shared.w2", qdt, 1, H, fsl, qb);
            rb.place(p + "shared.down", 0, H, r * fsl, (r + 1) * fsl, u, 0, fsl);
          }
          const int64_t el = m.num_experts / ep;
          const int u13 = rb.local(p + "experts.w13", qdt, el, 2 * fl, H, qb);
          const int u2 = rb.local(p + "experts.w2", qdt, el, H, fl, qb);
          for (int64_t j = 0; j < el; ++j) {
            const int e = static_cast<int>(epi * el + j);
            rb.place(ex(l, e, "gate"), r * fl, (r + 1) * fl, 0, H, u13, j * 2 * fl * H, H);
            rb.place(ex(l, e, "up"), r * fl, (r + 1) * fl, 0, H, u13, (2 * j + 1) * fl * H, H);
            rb.place(ex(l, e, "down"), 0, H, r * fl, (r + 1) * fl, u2, j * H * fl, fl);
          }
        }
        if (attn) {
          rb.place("final_norm", 0, 1, 0, H, rb.local("final_norm", dt, 1, 1, H), 0, H);
          rb.place("lm_head", r * vl, (r + 1) * vl, 0, H, rb.local("lm_head", dt, 1, vl, H), 0, H);
        }
        L.ranks.push_back(std::move(rb.r));
      }
}

}  // namespace

void describe(const wb_model_shapes& m, const wb_parallelism& par, wb_layout_t& out) {
  need(m.family >= WB_FAMILY_DENSE && m.family <= WB_FAMILY_MOE_ONLY, "unknown model family");
  need(m.num_layers >= 1 && m.hidden >= 1 && m.ffn >= 1, "model dimensions must be positive");
  if (m.family != WB_FAMILY_MOE_ONLY)
    need(m.num_heads >= 1 && m.num_kv_heads >= 1 && m.head_dim >= 1 && m.vocab >= 1, "attention dimensions must be positive");
  if (m.family != WB_FAMILY_DENSE) need(m.num_experts >= 1, "MoE families need experts");
  if (m.family == WB_FAMILY_MOE_ONLY) need(m.num_shared_experts >= 0, "shared experts must be >= 0");
  need(par.dtype == WB_F32 || par.dtype == WB_BF16, "local parameter dtype must be f32 or bf16");
  const Catalog cat = make_catalog(m);
  out.catalog = cat.list;
  out.ranks.clear();
  switch (par.style) {
    case WB_STYLE_FSDP_FLAT: style_fsdp(m, par, cat, out); break;
    case WB_STYLE_MEGATRON: style_megatron(m, par, cat, out); break;
    case WB_STYLE_SERVING: style_serving(m, par, cat, out); break;
    default: fail(WB_EINVAL, "unknown layout style");
  }
}

void check_placement(const wb_layout_t& L, int rank, const Placement& p) {
  need(rank >= 0 && rank < static_cast<int>(L.ranks.size()), "rank out of range");
  need(p.t >= 0 && p.t < static_cast<int>(L.catalog.size()), "placement tensor out of range");
  const Tensor& T = L.catalog[p.t];
  need(0 <= p.r0 && p.r0 < p.r1 && p.r1 <= T.rows && 0 <= p.c0 && p.c0 < p.c1 && p.c1 <= T.cols,
       "placement rectangle outside its checkpoint tensor");
  const Rank& R = L.ranks[rank];
  need(p.u >= 0 && p.u < static_cast<int>(R.locals.size()), "placement local tensor out of range");
  const Local& lc = R.locals[p.u];
  need(lc.scales < 0, "placements cannot target a scale tensor");
  need(p.tr == 0 || p.tr == 1, "transposed must be 0 or 1");
  need(p.base >= 0 && p.ld >= 1, "placement base must be >= 0 and ld >= 1");
  // extent along the strided axis and the contiguous axis
  const int64_t strided = p.tr ? p.cols() : p.rows();
  const int64_t contig = p.tr ? p.rows() : p.cols();
  need(strided == 1 || contig <= p.ld, "placement rows overlap (ld smaller than the contiguous extent)");
  const int64_t last = p.base + (strided - 1) * p.ld + (contig - 1);
  need(last < lc.numel(), "placement addresses elements past its local tensor");
}

std::string dump_layout(const wb_layout_t& L) {
  std::ostringstream o;
  o << "layout ranks=" << L.ranks.size() << " tensors=" << L.catalog.size() << "\n";
  for (size_t r = 0; r < L.ranks.size(); ++r) {
    const Rank& R = L.ranks[r];
    o << "rank " << r << " locals=" << R.locals.size() << " placements=" << R.pls.size() << "\n";
    for (size_t u = 0; u < R.locals.size(); ++u) {
      const Local& l = R.locals[u];
      o << "local " << u << " " << l.name << " " << dtype_name(l.dtype) << " " << l.batch << " " << l.rows << " "
        << l.cols << " " << l.block << " " << l.scale << " " << l.scales << "\n";
    }
    for (const Placement& p : R.pls)
      o << "pl " << p.t << " " << p.r0 << " " << p.r1 << " " << p.c0 << " " << p.c1 << " " << p.u << " " << p.base
        << " " << p.ld << " " << p.tr << "\n";
  }
  return o.str();
}

}  // namespace wb
