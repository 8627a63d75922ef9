"""Pins for oracle.plan.

* a plan derived by hand from the rules (tests/golden/hand_plan_replicated.txt);
* brute-force enumeration on random tiny layouts, using unique element
  identifiers: every element a rollout rank needs arrives exactly once, from a
  trainer rank that holds it (Sec. 3.2: trainers collectively send one copy);
* balance: each sender's bytes stay within one segment of its ideal share, and
  the total sent equals the total needed;
* the shape of the correspondence described in the text about Figure 2
  (identical layouts map one-to-one; re-sharding makes every rollout worker
  need data from every trainer).
"""

import os

import numpy as np
import pytest

from oracle.catalog import ModelShapes
from oracle.layout import DTYPE_BYTES, Parallelism, describe_layout, layout_from_spec
from oracle.plan import PlanError, build_plan, dump, sender_loads
from oracle.transfer import local_index
from synthetic_checkpoint.workloads import ORDER, WORKLOADS, scaled

from oracle_cases import hand_replicated_pair, id_values, random_model, random_par

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _golden(name):
    return "".join(l for l in open(os.path.join(GOLDEN, name)) if not l.startswith("#"))


def test_hand_plan_matches_golden():
    tr, ro = hand_replicated_pair()
    assert dump(build_plan(tr, ro)) == _golden("hand_plan_replicated.txt")


def brute_force_check(trainer, rollout, plan):
    """Enumerate every element; raise AssertionError on any violation."""
    ids = id_values(trainer.catalog)
    held = []
    for s, rk in enumerate(trainer.ranks):
        loc = [np.zeros(lc.numel, dtype=np.int64) for lc in rk.locals]
        for p in rk.placements:
            i = np.arange(p.r0, p.r1)[:, None]
            j = np.arange(p.c0, p.c1)[None, :]
            loc[p.u][local_index(p, i, j)] = ids[p.t][p.r0:p.r1, p.c0:p.c1]
        held.append(loc)
    got = [[np.zeros(lc.numel, dtype=np.int64) for lc in rk.locals] for rk in rollout.ranks]
    count = [[np.zeros(lc.numel, dtype=np.int64) for lc in rk.locals] for rk in rollout.ranks]
    for g in plan.segments:
        sp = trainer.ranks[g.s].placements[g.src_pl]
        q = rollout.ranks[g.d].placements[g.dst_pl]
        assert sp.t == g.t == q.t
        r = g.rect
        i = np.arange(r.r0, r.r1)[:, None]
        j = np.arange(r.c0, r.c1)[None, :]
        # the sender holds exactly these checkpoint elements where its placement says
        assert np.array_equal(held[g.s][sp.u][local_index(sp, i, j)], ids[g.t][r.r0:r.r1, r.c0:r.c1])
        idx = local_index(q, i, j)
        got[g.d][q.u][idx] = held[g.s][sp.u][local_index(sp, i, j)]
        np.add.at(count[g.d][q.u], idx.ravel(), 1)
    for d, rk in enumerate(rollout.ranks):
        want = [np.zeros(lc.numel, dtype=np.int64) for lc in rk.locals]
        for q in rk.placements:
            i = np.arange(q.r0, q.r1)[:, None]
            j = np.arange(q.c0, q.c1)[None, :]
            want[q.u][local_index(q, i, j)] = ids[q.t][q.r0:q.r1, q.c0:q.c1]
        for u, lc in enumerate(rk.locals):
            if lc.scales >= 0:
                continue
            assert np.all(count[d][u] == 1), (d, lc.name)
            assert np.array_equal(got[d][u], want[u]), (d, lc.name)


def balance_check(plan, global_bound=False):
    """Per owner set, every owner's bytes stay within one part of its even
    share; with ``global_bound`` the same holds for each sender's total."""
    per = {}
    for g in plan.segments:
        reg = plan.regions[g.region]
        key = reg.owners
        acc = per.setdefault(key, {"load": {s: 0 for s in key}, "share": 0.0, "max": 0})
        acc["load"][g.s] += g.nbytes
        acc["max"] = max(acc["max"], g.nbytes)
    for reg in plan.regions:
        per[reg.owners]["share"] += reg.nbytes / len(reg.owners)
    for key, acc in per.items():
        for s, b in acc["load"].items():
            assert b <= acc["share"] + acc["max"], (key, s, b, acc["share"], acc["max"])
    if global_bound:
        load, ideal = sender_loads(plan)
        mx = max(g.nbytes for g in plan.segments)
        for s in range(len(load)):
            assert load[s] <= ideal[s] + mx, (s, load[s], ideal[s], mx)
    elems_sent = sum(g.rect.numel for g in plan.segments)
    elems_needed = sum(q.numel for rk in plan.rollout.ranks for q in rk.placements)
    assert elems_sent == elems_needed
    load, ideal = sender_loads(plan)
    assert abs(sum(load) - sum(ideal)) < 1e-6 * max(1, sum(load))


def wire_check(plan):
    """Payloads are 256-byte aligned, disjoint, inside the buffers, and each
    (sender, receiver) region sits at the same relative offsets on both sides."""
    for side, key, total in (("send", "s", plan.send_bytes), ("recv", "d", plan.recv_bytes)):
        spans = {}
        for g in plan.segments:
            off = g.send_off if side == "send" else g.recv_off
            assert off % 256 == 0
            who = g.s if side == "send" else g.d
            spans.setdefault(who, []).append((off, off + g.nbytes))
        for who, sp in spans.items():
            sp.sort()
            for (a0, a1), (b0, b1) in zip(sp, sp[1:]):
                assert a1 <= b0
            assert sp[-1][1] <= total[who]
    base = {}
    for g in plan.segments:
        key = (g.s, g.d)
        delta = g.send_off - g.recv_off
        assert base.setdefault(key, delta) == delta


@pytest.mark.parametrize("seed", range(40))
def test_random_tiny_layouts_brute_force(seed):
    rng = np.random.default_rng(seed)
    m = random_model(rng)
    tr = describe_layout(m, random_par(rng, m, "trainer"))
    ro = describe_layout(m, random_par(rng, m, "rollout"))
    plan = build_plan(tr, ro)
    brute_force_check(tr, ro, plan)
    balance_check(plan)
    wire_check(plan)


@pytest.mark.parametrize("name", ORDER)
def test_scaled_workloads_brute_force(name):
    w = scaled(name)
    tr = layout_from_spec(w["model"], w["trainer"])
    ro = layout_from_spec(w["model"], w["rollout"])
    plan = build_plan(tr, ro)
    brute_force_check(tr, ro, plan)
    balance_check(plan, global_bound=True)
    wire_check(plan)


@pytest.mark.parametrize("name", ORDER)
def test_full_size_workloads_invariants(name):
    w = WORKLOADS[name]
    tr = layout_from_spec(w["model"], w["trainer"])
    ro = layout_from_spec(w["model"], w["rollout"])
    plan = build_plan(tr, ro)
    balance_check(plan, global_bound=True)
    wire_check(plan)
    # bytes needed by the unpacked rank, in the trainer dtype
    d = w["unpack_rank"]
    es = DTYPE_BYTES[w["trainer"]["dtype"]]
    need = sum(q.numel for q in ro.ranks[d].placements) * es
    assert sum(g.nbytes for g in plan.segments if g.d == d) == need


def test_figure2_correspondence_shapes():
    m = ModelShapes("dense", num_layers=2, hidden=16, num_heads=4, num_kv_heads=2, head_dim=4, ffn=16, vocab=16)
    a = describe_layout(m, Parallelism("fsdp_flat", "bf16", fsdp=2))
    plan = build_plan(a, describe_layout(m, Parallelism("fsdp_flat", "bf16", fsdp=2)))
    pairs = {(g.s, g.d) for g in plan.segments}
    assert pairs == {(0, 0), (1, 1)}          # same layout: one-to-one
    plan = build_plan(a, describe_layout(m, Parallelism("serving", "bf16", tp=1, dp=2)))
    pairs = {(g.s, g.d) for g in plan.segments}
    assert pairs == {(s, d) for s in range(2) for d in range(2)}   # every rollout needs every trainer
    # with replicated tensors (norms under TP), each replica sends a distinct slice
    b = describe_layout(m, Parallelism("serving", "bf16", tp=2))
    plan = build_plan(b, describe_layout(m, Parallelism("serving", "bf16", tp=2)))
    norm = [i for i, t in enumerate(b.catalog) if t.name.endswith("norm")]
    for d in range(2):
        for t in norm:
            senders = sorted(g.s for g in plan.segments if g.d == d and g.t == t)
            assert senders == [0, 1]
    assert all(g.s == g.d for g in plan.segments if g.t not in norm)


def test_overlapping_trainer_rectangles_rejected():
    from oracle.layout import Layout, Local, Placement, RankLayout
    from oracle.catalog import CkptTensor
    cat = [CkptTensor("T", 4, 4)]
    tr = Layout(cat, [RankLayout([Local("a", "f32", 1, 2, 4)], [Placement(0, 0, 2, 0, 4, 0, 0, 4)]),
                      RankLayout([Local("a", "f32", 1, 3, 4)], [Placement(0, 1, 4, 0, 4, 0, 0, 4)])])
    ro = Layout(cat, [RankLayout([Local("x", "f32", 1, 4, 4)], [Placement(0, 0, 4, 0, 4, 0, 0, 4)])])
    with pytest.raises(PlanError):
        build_plan(tr, ro)


def test_uncovered_need_rejected():
    from oracle.layout import Layout, Local, Placement, RankLayout
    from oracle.catalog import CkptTensor
    cat = [CkptTensor("T", 4, 4)]
    tr = Layout(cat, [RankLayout([Local("a", "f32", 1, 2, 4)], [Placement(0, 0, 2, 0, 4, 0, 0, 4)])])
    ro = Layout(cat, [RankLayout([Local("x", "f32", 1, 4, 4)], [Placement(0, 0, 4, 0, 4, 0, 0, 4)])])
    with pytest.raises(PlanError):
        build_plan(tr, ro)
