"""Source maps as slice-copies (WeightBridge Sec. 3.1 and App. B).

The paper represents what a worker holds as the sequence of slice-copy
operations that its weight loader performs, each an affine copy of a
rectangle of one checkpoint tensor into one local tensor, with or without
transposition. A *placement* is one such slice-copy:

    (t, rows r0:r1, cols c0:c1) of checkpoint tensor t  ->  local tensor u at
    local[u][base + (i - r0) * ld + (j - c0)] = T_t[i, j]     (not transposed)
    local[u][base + (j - c0) * ld + (i - r0)] = T_t[i, j]     (transposed)

The paper recovers placements by probing the loader; here they are declared
(``describe_layout``) for the layouts its workloads use. A layout covers every
rank of one side (all trainer ranks, or all rollout ranks).

Quantised local tensors (dtype ``f8e4m3``) carry a block edge and a companion
fp32 scale tensor of shape [batch, ceil(rows/B), ceil(cols/B)]; the scale
tensor has no placements, it is produced by the blockwise quantiser.
"""

from __future__ import annotations

from dataclasses import dataclass, field

from .catalog import CkptTensor, ModelShapes, checkpoint_catalog, index_of

DTYPE_BYTES = {"f32": 4, "bf16": 2, "f8e4m3": 1}


@dataclass(frozen=True)
class Local:
    name: str
    dtype: str
    batch: int
    rows: int
    cols: int
    block: int = 0       # quantisation block edge (0: not quantised)
    scale: int = -1      # index of the companion scale tensor (quantised tensors)
    scales: int = -1     # index of the quantised tensor this scale tensor serves

    @property
    def numel(self) -> int:
        return self.batch * self.rows * self.cols


@dataclass(frozen=True)
class Placement:
    t: int
    r0: int
    r1: int
    c0: int
    c1: int
    u: int
    base: int
    ld: int
    tr: int = 0

    @property
    def rows(self) -> int:
        return self.r1 - self.r0

    @property
    def cols(self) -> int:
        return self.c1 - self.c0

    @property
    def numel(self) -> int:
        return self.rows * self.cols


@dataclass
class RankLayout:
    locals: list[Local] = field(default_factory=list)
    placements: list[Placement] = field(default_factory=list)


@dataclass
class Layout:
    catalog: list[CkptTensor]
    ranks: list[RankLayout]

    @property
    def nranks(self) -> int:
        return len(self.ranks)


@dataclass(frozen=True)
class Parallelism:
    style: str                 # "fsdp_flat" | "megatron" | "serving"
    dtype: str                 # local parameter dtype
    tp: int = 1
    ep: int = 1
    fsdp: int = 1
    dp: int = 1
    transposed_row_parallel: bool = False
    quant: str = ""            # serving style: "" or "f8e4m3" for linear weights
    quant_block: int = 128


class _Rank:
    """Helper that appends locals and placements of one rank."""

    def __init__(self, cat_index: dict[str, int]):
        self.r = RankLayout()
        self.ix = cat_index

    def local(self, name, dtype, batch, rows, cols, block=0) -> int:
        u = len(self.r.locals)
        if block:
            self.r.locals.append(Local(name, dtype, batch, rows, cols, block, scale=u + 1))
            self.r.locals.append(Local(name + "_scale", "f32", batch, -(-rows // block), -(-cols // block), scales=u))
        else:
            self.r.locals.append(Local(name, dtype, batch, rows, cols))
        return u

    def place(self, tname, r0, r1, c0, c1, u, base, ld, tr=0):
        self.r.placements.append(Placement(self.ix[tname], r0, r1, c0, c1, u, base, ld, tr))


def flat_run_rects(p0: int, p1: int, cols: int):
    """Split the row-major flat run [p0, p1) of a matrix with ``cols`` columns
    into at most three rectangles: a partial head row, whole rows, a partial
    tail row. Yields (first flat index, r0, r1, c0, c1)."""
    p = p0
    if p < p1 and p % cols:
        end = min(p1, (p // cols + 1) * cols)
        yield p, p // cols, p // cols + 1, p % cols, p % cols + (end - p)
        p = end
    if p1 - p >= cols:
        n = (p1 - p) // cols
        yield p, p // cols, p // cols + n, 0, cols
        p += n * cols
    if p < p1:
        yield p, p // cols, p // cols + 1, 0, p1 - p


def _fsdp_units(m: ModelShapes, cat: list[CkptTensor], ep: int):
    """FSDP1-style flat-parameter units: (name, tensor names, ep group or None)."""
    units = []
    names = [t.name for t in cat]
    if m.family in ("dense", "mixtral"):
        units.append(("flat.embed", ["embed"], None))
    for layer in range(m.num_layers):
        p = f"layers.{layer}."
        mine = [n for n in names if n.startswith(p)]
        if m.family == "dense":
            units.append((f"flat.layers.{layer}", mine, None))
            continue
        non_expert = [n for n in mine if not n.startswith(p + "experts.")]
        units.append((f"flat.layers.{layer}", non_expert, None))
        per = m.num_experts // ep
        for g in range(ep):
            grp = [n for e in range(g * per, (g + 1) * per) for n in
                   (f"{p}experts.{e}.gate", f"{p}experts.{e}.up", f"{p}experts.{e}.down")]
            units.append((f"flat.layers.{layer}.experts.{g}", grp, g))
    if m.family in ("dense", "mixtral"):
        units.append(("flat.final", ["final_norm", "lm_head"], None))
    return units


def _fsdp_flat(m, par, cat, ix):
    if par.fsdp < 1 or par.ep < 1 or par.dp < 1 or par.tp != 1:
        raise ValueError("fsdp_flat: bad degrees")
    if m.family == "dense" and par.ep != 1:
        raise ValueError("fsdp_flat: ep > 1 needs experts")
    if m.family != "dense" and m.num_experts % par.ep:
        raise ValueError("fsdp_flat: experts not divisible by ep")
    units = _fsdp_units(m, cat, par.ep)
    shape = {t.name: t for t in cat}
    ranks = []
    for dp_i in range(par.dp):
        for ep_i in range(par.ep):
            for f in range(par.fsdp):
                rk = _Rank(ix)
                for uname, tnames, grp in units:
                    if grp is not None and grp != ep_i:
                        continue
                    total = sum(shape[n].numel for n in tnames)
                    per = -(-total // par.fsdp)
                    a, b = f * per, (f + 1) * per
                    u = rk.local(uname, par.dtype, 1, 1, per)
                    off = 0
                    for n in tnames:
                        t = shape[n]
                        lo, hi = max(a, off), min(b, off + t.numel)
                        if lo < hi:
                            for first, r0, r1, c0, c1 in flat_run_rects(lo - off, hi - off, t.cols):
                                rk.place(n, r0, r1, c0, c1, u, off + first - a, t.cols)
                        off += t.numel
                ranks.append(rk.r)
    return ranks


def _check_tp(m, tp):
    if m.family in ("dense", "mixtral"):
        if m.vocab % tp or m.num_heads % tp or m.num_kv_heads % tp or m.num_heads % m.num_kv_heads:
            raise ValueError("tp does not divide vocab / heads / kv heads")
    if m.ffn % tp:
        raise ValueError("tp does not divide ffn")


def _megatron(m, par, cat, ix):
    tp, ep = par.tp, par.ep
    if tp < 1 or ep < 1 or par.dp < 1 or par.fsdp != 1:
        raise ValueError("megatron: bad degrees")
    if m.family == "dense" and ep != 1:
        raise ValueError("megatron: ep > 1 needs experts")
    if m.family != "dense" and (tp != 1 or m.num_experts % ep):
        raise ValueError("megatron: MoE layouts need tp == 1 and ep | experts")
    _check_tp(m, tp)
    h, hd, dt, T = m.hidden, m.head_dim, par.dtype, 1 if par.transposed_row_parallel else 0
    ranks = []
    for dp_i in range(par.dp):
        for ep_i in range(ep):
            for r in range(tp):
                rk = _Rank(ix)

                def row_parallel(name, tname, rows, cols_total, c0, c1):
                    # shard T[:, c0:c1]; stored [rows, c1-c0] or transposed [c1-c0, rows]
                    if T:
                        u = rk.local(name, dt, 1, c1 - c0, rows)
                        rk.place(tname, 0, rows, c0, c1, u, 0, rows, 1)
                    else:
                        u = rk.local(name, dt, 1, rows, c1 - c0)
                        rk.place(tname, 0, rows, c0, c1, u, 0, c1 - c0, 0)

                if m.family in ("dense", "mixtral"):
                    vl = m.vocab // tp
                    u = rk.local("embed", dt, 1, vl, h)
                    rk.place("embed", r * vl, (r + 1) * vl, 0, h, u, 0, h)
                for layer in range(m.num_layers):
                    p = f"layers.{layer}."
                    if m.family in ("dense", "mixtral"):
                        u = rk.local(p + "attn_norm", dt, 1, 1, h)
                        rk.place(p + "attn_norm", 0, 1, 0, h, u, 0, h)
                        ng = m.num_kv_heads // tp
                        qpg = m.num_heads // m.num_kv_heads
                        u = rk.local(p + "qkv", dt, 1, ng * (qpg + 2) * hd, h)
                        for gi in range(ng):
                            g = r * ng + gi
                            off = gi * (qpg + 2) * hd
                            rk.place(p + "q", g * qpg * hd, (g + 1) * qpg * hd, 0, h, u, off * h, h)
                            rk.place(p + "k", g * hd, (g + 1) * hd, 0, h, u, (off + qpg * hd) * h, h)
                            rk.place(p + "v", g * hd, (g + 1) * hd, 0, h, u, (off + (qpg + 1) * hd) * h, h)
                        ql = m.num_heads * hd // tp
                        row_parallel(p + "o", p + "o", h, m.num_heads * hd, r * ql, (r + 1) * ql)
                        u = rk.local(p + "mlp_norm", dt, 1, 1, h)
                        rk.place(p + "mlp_norm", 0, 1, 0, h, u, 0, h)
                    if m.family == "dense":
                        fl = m.ffn // tp
                        u = rk.local(p + "gate_up", dt, 1, 2 * fl, h)
                        rk.place(p + "gate", r * fl, (r + 1) * fl, 0, h, u, 0, h)
                        rk.place(p + "up", r * fl, (r + 1) * fl, 0, h, u, fl * h, h)
                        row_parallel(p + "down", p + "down", h, m.ffn, r * fl, (r + 1) * fl)
                        continue
                    u = rk.local(p + "router", dt, 1, m.num_experts, h)
                    rk.place(p + "router", 0, m.num_experts, 0, h, u, 0, h)
                    if m.family == "moe_only":
                        fs = m.ffn * m.num_shared_experts
                        u = rk.local(p + "shared.w1", dt, 1, fs, h)
                        rk.place(p + "shared.gate", 0, fs, 0, h, u, 0, h)
                        u = rk.local(p + "shared.w3", dt, 1, fs, h)
                        rk.place(p + "shared.up", 0, fs, 0, h, u, 0, h)
                        row_parallel(p + "shared.w2", p + "shared.down", h, fs, 0, fs)
                    el, f = m.num_experts // ep, m.ffn
                    u1 = rk.local(p + "experts.w1", dt, el, f, h)
                    u3 = rk.local(p + "experts.w3", dt, el, f, h)
                    u2 = rk.local(p + "experts.w2", dt, el, f, h) if T else rk.local(p + "experts.w2", dt, el, h, f)
                    for j in range(el):
                        e = ep_i * el + j
                        rk.place(f"{p}experts.{e}.gate", 0, f, 0, h, u1, j * f * h, h)
                        rk.place(f"{p}experts.{e}.up", 0, f, 0, h, u3, j * f * h, h)
                        if T:
                            rk.place(f"{p}experts.{e}.down", 0, h, 0, f, u2, j * f * h, h, 1)
                        else:
                            rk.place(f"{p}experts.{e}.down", 0, h, 0, f, u2, j * h * f, f)
                if m.family in ("dense", "mixtral"):
                    u = rk.local("final_norm", dt, 1, 1, h)
                    rk.place("final_norm", 0, 1, 0, h, u, 0, h)
                    u = rk.local("lm_head", dt, 1, vl, h)
                    rk.place("lm_head", r * vl, (r + 1) * vl, 0, h, u, 0, h)
                ranks.append(rk.r)
    return ranks


def _serving(m, par, cat, ix):
    tp, ep = par.tp, par.ep
    if tp < 1 or ep < 1 or par.dp < 1 or par.fsdp != 1 or par.transposed_row_parallel:
        raise ValueError("serving: bad degrees")
    if m.family == "dense" and ep != 1:
        raise ValueError("serving: ep > 1 needs experts")
    if m.family != "dense" and m.num_experts % ep:
        raise ValueError("serving: ep must divide experts")
    if par.quant not in ("", "f8e4m3") or (par.quant and par.quant_block < 1):
        raise ValueError("serving: bad quantisation")
    _check_tp(m, tp)
    h, hd, dt = m.hidden, m.head_dim, par.dtype
    qdt = par.quant or dt
    qb = par.quant_block if par.quant else 0
    ranks = []
    for dp_i in range(par.dp):
        for ep_i in range(ep):
            for r in range(tp):
                rk = _Rank(ix)
                if m.family in ("dense", "mixtral"):
                    vl = m.vocab // tp
                    u = rk.local("embed", dt, 1, vl, h)
                    rk.place("embed", r * vl, (r + 1) * vl, 0, h, u, 0, h)
                for layer in range(m.num_layers):
                    p = f"layers.{layer}."
                    if m.family in ("dense", "mixtral"):
                        u = rk.local(p + "attn_norm", dt, 1, 1, h)
                        rk.place(p + "attn_norm", 0, 1, 0, h, u, 0, h)
                        ql, kl = m.num_heads * hd // tp, m.num_kv_heads * hd // tp
                        u = rk.local(p + "qkv", qdt, 1, ql + 2 * kl, h, qb)
                        rk.place(p + "q", r * ql, (r + 1) * ql, 0, h, u, 0, h)
                        rk.place(p + "k", r * kl, (r + 1) * kl, 0, h, u, ql * h, h)
                        rk.place(p + "v", r * kl, (r + 1) * kl, 0, h, u, (ql + kl) * h, h)
                        u = rk.local(p + "o", qdt, 1, h, ql, qb)
                        rk.place(p + "o", 0, h, r * ql, (r + 1) * ql, u, 0, ql)
                        u = rk.local(p + "mlp_norm", dt, 1, 1, h)
                        rk.place(p + "mlp_norm", 0, 1, 0, h, u, 0, h)
                    if m.family == "dense":
                        fl = m.ffn // tp
                        u = rk.local(p + "gate_up", qdt, 1, 2 * fl, h, qb)
                        rk.place(p + "gate", r * fl, (r + 1) * fl, 0, h, u, 0, h)
                        rk.place(p + "up", r * fl, (r + 1) * fl, 0, h, u, fl * h, h)
                        u = rk.local(p + "down", qdt, 1, h, fl, qb)
                        rk.place(p + "down", 0, h, r * fl, (r + 1) * fl, u, 0, fl)
                        continue
                    u = rk.local(p + "router", dt, 1, m.num_experts, h)
                    rk.place(p + "router", 0, m.num_experts, 0, h, u, 0, h)
                    fl = m.ffn // tp
                    if m.family == "moe_only":
                        fsl = m.ffn * m.num_shared_experts // tp
                        u = rk.local(p + "shared.w13", qdt, 1, 2 * fsl, h, qb)
                        rk.place(p + "shared.gate", r * fsl, (r + 1) * fsl, 0, h, u, 0, h)
                        rk.place(p + "shared.up", r * fsl, (r + 1) * fsl, 0, h, u, fsl * h, h)
                        u = rk.local(p + "shared.w2", qdt, 1, h, fsl, qb)
                        rk.place(p + "shared.down", 0, h, r * fsl, (r + 1) * fsl, u, 0, fsl)
                    el = m.num_experts // ep
                    u13 = rk.local(p + "experts.w13", qdt, el, 2 * fl, h, qb)
                    u2 = rk.local(p + "experts.w2", qdt, el, h, fl, qb)
                    for j in range(el):
                        e = ep_i * el + j
                        rk.place(f"{p}experts.{e}.gate", r * fl, (r + 1) * fl, 0, h, u13, j * 2 * fl * h, h)
                        rk.place(f"{p}experts.{e}.up", r * fl, (r + 1) * fl, 0, h, u13, (j * 2 + 1) * fl * h, h)
                        rk.place(f"{p}experts.{e}.down", 0, h, r * fl, (r + 1) * fl, u2, j * h * fl, fl)
                if m.family in ("dense", "mixtral"):
                    u = rk.local("final_norm", dt, 1, 1, h)
                    rk.place("final_norm", 0, 1, 0, h, u, 0, h)
                    u = rk.local("lm_head", dt, 1, vl, h)
                    rk.place("lm_head", r * vl, (r + 1) * vl, 0, h, u, 0, h)
                ranks.append(rk.r)
    return ranks


def describe_layout(m: ModelShapes, par: Parallelism) -> Layout:
    """Placements of every rank of one side for model ``m`` under ``par``."""
    if par.dtype not in ("f32", "bf16"):
        raise ValueError("local parameter dtype must be f32 or bf16")
    cat = checkpoint_catalog(m)
    ix = index_of(cat)
    style = {"fsdp_flat": _fsdp_flat, "megatron": _megatron, "serving": _serving}.get(par.style)
    if style is None:
        raise ValueError(f"unknown style {par.style!r}")
    return Layout(cat, style(m, par, cat, ix))


def validate(layout: Layout, require_full_cover: bool) -> None:
    """Check every placement against its checkpoint tensor and local tensor,
    element by element (small layouts only). With ``require_full_cover`` each
    non-scale local element must be written by exactly one placement."""
    import numpy as np

    for rk in layout.ranks:
        cover = [np.zeros(lc.numel, dtype=np.int64) for lc in rk.locals]
        for p in rk.placements:
            t = layout.catalog[p.t]
            assert 0 <= p.r0 < p.r1 <= t.rows and 0 <= p.c0 < p.c1 <= t.cols, p
            lc = rk.locals[p.u]
            assert lc.scales < 0, "placement into a scale tensor"
            i = np.arange(p.r0, p.r1)[:, None]
            j = np.arange(p.c0, p.c1)[None, :]
            idx = p.base + ((j - p.c0) * p.ld + (i - p.r0) if p.tr else (i - p.r0) * p.ld + (j - p.c0))
            assert idx.min() >= 0 and idx.max() < lc.numel, p
            np.add.at(cover[p.u], idx.ravel(), 1)
        for lc, c in zip(rk.locals, cover):
            assert c.max(initial=0) <= 1, f"{lc.name}: element placed twice"
            if require_full_cover and lc.scales < 0:
                assert c.min(initial=1) == 1, f"{lc.name}: element not covered"


def layout_from_spec(model: dict, par: dict) -> Layout:
    """Layout from plain-data model and parallelism specs."""
    from .catalog import ModelShapes as _MS

    return describe_layout(_MS(**model), Parallelism(**par))
