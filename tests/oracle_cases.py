"""Small hand-built and random layouts shared by the plan tests (oracle types)."""

from __future__ import annotations

import numpy as np

from oracle.catalog import CkptTensor, ModelShapes
from oracle.layout import Layout, Local, Parallelism, Placement, RankLayout, describe_layout


def hand_replicated_pair():
    """The layout pair of tests/golden/hand_plan_replicated.txt."""
    cat = [CkptTensor("T0", 4, 6), CkptTensor("T1", 1, 10)]
    full = RankLayout([Local("a", "f32", 1, 4, 6), Local("b", "f32", 1, 1, 10)],
                      [Placement(0, 0, 4, 0, 6, 0, 0, 6), Placement(1, 0, 1, 0, 10, 1, 0, 10)])
    only_t1 = RankLayout([Local("b", "f32", 1, 1, 10)], [Placement(1, 0, 1, 0, 10, 0, 0, 10)])
    trainer = Layout(cat, [full, RankLayout(list(full.locals), list(full.placements)), only_t1])
    r0 = RankLayout([Local("x", "bf16", 1, 2, 6), Local("y", "bf16", 1, 1, 10)],
                    [Placement(0, 0, 2, 0, 6, 0, 0, 6), Placement(1, 0, 1, 0, 10, 1, 0, 10)])
    r1 = RankLayout([Local("x", "bf16", 1, 6, 2), Local("y", "bf16", 1, 1, 5)],
                    [Placement(0, 2, 4, 0, 6, 0, 0, 2, 1), Placement(1, 0, 1, 5, 10, 1, 0, 5)])
    rollout = Layout(cat, [r0, r1])
    return trainer, rollout


def random_model(rng) -> ModelShapes:
    fam = ["dense", "mixtral", "moe_only"][int(rng.integers(0, 3))]
    nkv = int(rng.choice([1, 2, 4]))
    qpg = int(rng.choice([1, 2]))
    return ModelShapes(fam, num_layers=int(rng.integers(1, 3)), hidden=int(rng.choice([8, 12, 16, 20])),
                       num_heads=nkv * qpg, num_kv_heads=nkv, head_dim=int(rng.choice([2, 4])),
                       ffn=int(rng.choice([8, 12, 24])), vocab=int(rng.choice([8, 16, 24])),
                       num_experts=int(rng.choice([2, 4, 8])), num_shared_experts=1)


def random_medium_model(rng) -> ModelShapes:
    """Like random_model, with shapes that span several 16-byte vectors,
    64 x 64 transpose tiles and 128 x 128 fp8 blocks, and ragged tails."""
    fam = ["dense", "mixtral", "moe_only"][int(rng.integers(0, 3))]
    nkv = int(rng.choice([1, 2, 4]))
    qpg = int(rng.choice([1, 2]))
    return ModelShapes(fam, num_layers=int(rng.integers(1, 3)), hidden=int(rng.choice([128, 200, 256, 384])),
                       num_heads=nkv * qpg, num_kv_heads=nkv, head_dim=int(rng.choice([32, 64])),
                       ffn=int(rng.choice([256, 320, 512])), vocab=int(rng.choice([256, 500])),
                       num_experts=int(rng.choice([2, 4])), num_shared_experts=1)


def random_par(rng, m: ModelShapes, side: str, blocks=(4, 8)) -> Parallelism:
    """A random parallelism valid for model m (trainer or rollout side); fp8
    rollouts take a block edge from ``blocks``."""
    dtype = ["f32", "bf16"][int(rng.integers(0, 2))]
    while True:
        style = ["fsdp_flat", "megatron"][int(rng.integers(0, 2))] if side == "trainer" else "serving"
        tp = int(rng.choice([1, 2, 4]))
        ep = int(rng.choice([1, 2, 4])) if m.family != "dense" else 1
        dp = int(rng.choice([1, 1, 2]))
        try:
            if style == "fsdp_flat":
                p = Parallelism(style, dtype, fsdp=int(rng.integers(1, 6)), ep=ep, dp=dp)
            elif style == "megatron":
                p = Parallelism(style, dtype, tp=tp if m.family == "dense" else 1, ep=ep, dp=dp,
                                transposed_row_parallel=bool(rng.integers(0, 2)))
            else:
                q = "f8e4m3" if rng.integers(0, 3) == 0 else ""
                p = Parallelism(style, "bf16" if q else dtype, tp=tp, ep=ep, dp=dp, quant=q,
                                quant_block=int(rng.choice(list(blocks))))
            describe_layout(m, p)
            return p
        except ValueError:
            continue


def id_values(catalog):
    """Checkpoint tensors whose elements hold unique identifiers (1-based)."""
    out, off = [], 1
    for t in catalog:
        out.append(np.arange(off, off + t.numel, dtype=np.int64).reshape(t.rows, t.cols))
        off += t.numel
    return out


def hand_rounds_pair():
    """The layout pair of tests/golden/hand_plan_rounds.txt."""
    cat = [CkptTensor("T0", 4, 6), CkptTensor("T1", 2, 8), CkptTensor("T2", 1, 16), CkptTensor("A", 1, 4),
           CkptTensor("B", 2, 4)]
    tl = [Local("t0", "f32", 1, 4, 6), Local("t1", "f32", 1, 2, 8), Local("t2", "f32", 1, 1, 16),
          Local("a", "f32", 1, 1, 4), Local("b", "f32", 1, 2, 4)]
    tp = [Placement(0, 0, 4, 0, 6, 0, 0, 6), Placement(1, 0, 2, 0, 8, 1, 0, 8), Placement(2, 0, 1, 0, 16, 2, 0, 16),
          Placement(3, 0, 1, 0, 4, 3, 0, 4), Placement(4, 0, 2, 0, 4, 4, 0, 4)]
    trainer = Layout(cat, [RankLayout(tl, tp)])
    rl = [Local("x0", "bf16", 1, 4, 6), Local("x1", "bf16", 1, 2, 8), Local("x2", "bf16", 1, 1, 16),
          Local("q", "f8e4m3", 1, 3, 4, 2, scale=4), Local("q_scale", "f32", 1, 2, 2, scales=3)]
    rp = [Placement(0, 0, 4, 0, 6, 0, 0, 6), Placement(1, 0, 2, 0, 8, 1, 0, 8), Placement(2, 0, 1, 0, 16, 2, 0, 16),
          Placement(3, 0, 1, 0, 4, 3, 0, 4), Placement(4, 0, 2, 0, 4, 3, 4, 4)]
    rollout = Layout(cat, [RankLayout(rl, rp)])
    return trainer, rollout


def hand_exchange_pair():
    """The layout pair of tests/golden/hand_plan_exchange.txt (node size 2)."""
    cat = [CkptTensor("T0", 4, 4), CkptTensor("T1", 1, 8)]
    tr = []
    for r0 in (0, 2):
        tr.append(RankLayout([Local("a", "f32", 1, 2, 4), Local("b", "f32", 1, 1, 8)],
                             [Placement(0, r0, r0 + 2, 0, 4, 0, 0, 4), Placement(1, 0, 1, 0, 8, 1, 0, 8)]))
    both = RankLayout([Local("x", "bf16", 1, 4, 4), Local("y", "bf16", 1, 1, 8)],
                      [Placement(0, 0, 4, 0, 4, 0, 0, 4), Placement(1, 0, 1, 0, 8, 1, 0, 8)])
    only_x = RankLayout([Local("x", "bf16", 1, 4, 4)], [Placement(0, 0, 4, 0, 4, 0, 0, 4)])
    return Layout(cat, tr), Layout(cat, [both, only_x, RankLayout(list(both.locals), list(both.placements))])


def overlapping_rollout_pair():
    """Rollout ranks holding overlapping but non-identical rectangles of one
    tensor (rows 0:4 and 2:6 of T), each replicated on two ranks in different
    nodes of two, and a replicated vector; trainer FSDP-like row halves."""
    cat = [CkptTensor("T", 6, 4), CkptTensor("v", 1, 6)]
    tr = [RankLayout([Local("a", "f32", 1, 3, 4), Local("b", "f32", 1, 1, 6)],
                     [Placement(0, r0, r0 + 3, 0, 4, 0, 0, 4), Placement(1, 0, 1, 0, 6, 1, 0, 6)])
          for r0 in (0, 3)]
    ro = []
    for r0 in (0, 2, 0, 2):
        ro.append(RankLayout([Local("x", "bf16", 1, 4, 4), Local("y", "bf16", 1, 1, 6)],
                             [Placement(0, r0, r0 + 4, 0, 4, 0, 0, 4), Placement(1, 0, 1, 0, 6, 1, 0, 6)]))
    return Layout(cat, tr), Layout(cat, ro)


def hand_rounds_balanced_pair():
    """The layout pair of tests/golden/hand_plan_rounds_balanced.txt."""
    sizes = [38, 10, 10, 10, 38]
    cat = [CkptTensor(f"T{i}", 1, n) for i, n in enumerate(sizes)]
    tl = [Local(f"t{i}", "f32", 1, 1, n) for i, n in enumerate(sizes)]
    pl = [Placement(i, 0, 1, 0, n, i, 0, n) for i, n in enumerate(sizes)]
    rl = [Local(f"x{i}", "bf16", 1, 1, n) for i, n in enumerate(sizes)]
    return Layout(cat, [RankLayout(tl, pl)]), Layout(cat, [RankLayout(rl, list(pl))])
