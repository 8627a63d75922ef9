"""Pins for the three-stage plan (rollout-side de-duplication, external and
internal exchange; Sec. 3.2 and Figure 5).

* Figure 5's caption: with a TP2 trainer and four DP rollout workers on two
  nodes of two, the exchange stages cut each node's ingress from six squares
  (receive stage plus a flat all-to-all exchange) to four; without rollout
  de-duplication it is eight (every worker fetches the whole model).
* Eq. 1's traffic: the trainers send exactly one copy of what the rollout side
  needs, and every rollout node receives over the inter-node network exactly
  one copy of what its ranks need (M_v), brute-forced on random layouts.
* Element-level brute force with unique identifiers: every element of every
  rollout placement is written exactly once, with the right identifier, by a
  chain of forwards that starts at a trainer rank holding it.
* A plan derived by hand (tests/golden/hand_plan_exchange.txt).
"""

import os

import numpy as np
import pytest

from oracle.catalog import ModelShapes
from oracle.layout import DTYPE_BYTES, Parallelism, describe_layout, layout_from_spec
from oracle.plan import PlanError, build_plan, dump
from oracle.transfer import expected_rollout, local_index, materialize, run_stages, unpack
from synthetic_checkpoint.workloads import ORDER, scaled

from oracle_cases import hand_exchange_pair, hand_replicated_pair, id_values, random_model, random_par

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _golden(name):
    return "".join(l for l in open(os.path.join(GOLDEN, name)) if not l.startswith("#"))


def test_hand_exchange_plan_matches_golden():
    tr, ro = hand_exchange_pair()
    assert dump(build_plan(tr, ro, node_size=2)) == _golden("hand_plan_exchange.txt")


def test_direct_plan_unchanged_by_option():
    tr, ro = hand_replicated_pair()
    assert dump(build_plan(tr, ro, node_size=0)) == _golden("hand_plan_replicated.txt")
    with pytest.raises(PlanError):
        build_plan(tr, ro, node_size=-1)


def _wire_bytes(plan, g):
    o = plan.segments[g.origin]
    sp = plan.trainer.ranks[o.s].placements[o.src_pl]
    return g.rect.numel * DTYPE_BYTES[plan.trainer.ranks[o.s].locals[sp.u].dtype]


def node_ingress(plan, node_size):
    """Bytes entering each node (of ``node_size`` consecutive rollout ranks)
    from outside it: every receive-stage segment, and exchange segments whose
    sender sits in another node."""
    nn = -(-plan.rollout.nranks // node_size)
    ing = [0] * nn
    for g in plan.segments:
        if g.stage == 0 or g.s // node_size != g.d // node_size:
            ing[g.d // node_size] += g.nbytes
    return ing


def needed_per_node(rollout, trainer, node_size):
    """M_v: wire bytes of one copy of every distinct rollout rectangle that some
    rank of node v holds (computed from the layouts alone)."""
    esize = {}
    for rk in trainer.ranks:
        for p in rk.placements:
            esize[p.t] = DTYPE_BYTES[rk.locals[p.u].dtype]
    nn = -(-rollout.nranks // node_size)
    seen = [set() for _ in range(nn)]
    for d, rk in enumerate(rollout.ranks):
        for q in rk.placements:
            seen[d // node_size].add((q.t, q.r0, q.r1, q.c0, q.c1))
    return [sum((k[2] - k[1]) * (k[4] - k[3]) * esize[k[0]] for k in s) for s in seen]


def test_figure5_ingress_six_to_four():
    m = ModelShapes("dense", num_layers=2, hidden=16, num_heads=4, num_kv_heads=4, head_dim=4, ffn=32, vocab=32)
    tr = describe_layout(m, Parallelism("megatron", "bf16", tp=2))
    ro = describe_layout(m, Parallelism("serving", "bf16", tp=1, dp=4))
    M = sum(t.numel for t in tr.catalog) * 2
    square = M // 4
    assert M % 4 == 0
    three = build_plan(tr, ro, node_size=2)
    flat = build_plan(tr, ro, node_size=1)
    direct = build_plan(tr, ro)
    assert node_ingress(three, 2) == [4 * square, 4 * square]
    assert node_ingress(flat, 2) == [6 * square, 6 * square]
    assert node_ingress(direct, 2) == [8 * square, 8 * square]
    # each worker receives a distinct quarter from the trainers
    recv0 = [0] * 4
    for g in three.segments:
        if g.stage == 0:
            recv0[g.d] += g.nbytes
    assert recv0 == [square] * 4
    # the trainers send one copy of the model instead of four
    assert sum(g.nbytes for g in three.segments if g.stage == 0) == M
    assert sum(g.nbytes for g in direct.segments) == 4 * M


def brute_force_exchange(trainer, rollout, plan):
    """Replay the three stages on unique identifiers; every rollout placement
    element must be written exactly once with its identifier."""
    ids = id_values(trainer.catalog)
    G = plan.node_size
    held = {}
    for s, rk in enumerate(trainer.ranks):
        loc = [np.zeros(lc.numel, dtype=np.int64) for lc in rk.locals]
        for p in rk.placements:
            i = np.arange(p.r0, p.r1)[:, None]
            j = np.arange(p.c0, p.c1)[None, :]
            loc[p.u][local_index(p, i, j)] = ids[p.t][p.r0:p.r1, p.c0:p.c1]
        held[s] = loc
    got = [[np.zeros(lc.numel, dtype=np.int64) for lc in rk.locals] for rk in rollout.ranks]
    count = [[np.zeros(lc.numel, dtype=np.int64) for lc in rk.locals] for rk in rollout.ranks]
    payload = {}
    for gi, g in enumerate(plan.segments):
        r = g.rect
        i = np.arange(r.r0, r.r1)[:, None]
        j = np.arange(r.c0, r.c1)[None, :]
        if g.stage == 0:
            sp = trainer.ranks[g.s].placements[g.src_pl]
            assert sp.t == g.t
            data = held[g.s][sp.u][local_index(sp, i, j)]
        else:
            src = plan.segments[g.src_seg]
            # forwarded by the rank that received it, in an earlier stage
            assert src.d == g.s and src.stage < g.stage and src.rect == g.rect and src.t == g.t
            assert g.origin == src.origin and g.nbytes == src.nbytes
            if g.stage == 1:
                assert g.s // G != g.d // G
            else:
                assert g.s // G == g.d // G and g.s != g.d
            data = payload[g.src_seg]
        payload[gi] = data
        q = rollout.ranks[g.d].placements[g.dst_pl]
        assert q.t == g.t
        idx = local_index(q, i, j)
        got[g.d][q.u][idx] = data
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


def traffic_check(trainer, rollout, plan):
    G = plan.node_size
    assert node_ingress(plan, G) == needed_per_node(rollout, trainer, G)
    # trainers send one copy of every distinct rollout rectangle
    distinct = needed_per_node(rollout, trainer, rollout.nranks)[0]
    assert sum(g.nbytes for g in plan.segments if g.stage == 0) == distinct
    for g in plan.segments:
        assert g.nbytes == _wire_bytes(plan, g)


def stage_wire_check(plan):
    """Within every stage of every round: payloads 256-byte aligned, disjoint and
    inside the buffers; receive sections do not overlap across stages."""
    for k, rd in enumerate(plan.rounds):
        spans_recv = {}
        for stage in (0, 1, 2):
            mine = [g for g in plan.segments if g.round == k and g.stage == stage]
            sends = {}
            for g in mine:
                assert g.send_off % 256 == 0 and g.recv_off % 256 == 0
                sends.setdefault(g.s, []).append((g.send_off, g.send_off + g.nbytes))
                spans_recv.setdefault(g.d, []).append((g.recv_off, g.recv_off + g.nbytes))
                if stage:
                    src = plan.segments[g.src_seg]
                    assert g.src_off == src.recv_off and src.round == k
            limit = rd.send_bytes if stage == 0 else rd.fwd_bytes[stage - 1]
            for who, sp in sends.items():
                sp.sort()
                assert all(a1 <= b0 for (_, a1), (b0, _) in zip(sp, sp[1:]))
                assert sp[-1][1] <= limit[who]
        for who, sp in spans_recv.items():
            sp.sort()
            assert all(a1 <= b0 for (_, a1), (b0, _) in zip(sp, sp[1:]))
            assert sp[-1][1] <= rd.recv_bytes[who]


@pytest.mark.parametrize("seed", range(40))
def test_random_exchange_plans(seed):
    rng = np.random.default_rng(900 + seed)
    m = random_model(rng)
    tr = describe_layout(m, random_par(rng, m, "trainer"))
    ro = describe_layout(m, random_par(rng, m, "rollout"))
    G = int(rng.integers(1, ro.nranks + 1))
    budget = int(rng.choice([0, 0, 256, 2048]))
    plan = build_plan(tr, ro, round_budget=budget, node_size=G)
    brute_force_exchange(tr, ro, plan)
    traffic_check(tr, ro, plan)
    stage_wire_check(plan)


@pytest.mark.parametrize("name", ORDER)
def test_scaled_workloads_exchange(name):
    w = scaled(name)
    tr = layout_from_spec(w["model"], w["trainer"])
    ro = layout_from_spec(w["model"], w["rollout"])
    for G in sorted({1, 2, ro.nranks}):
        plan = build_plan(tr, ro, node_size=G)
        brute_force_exchange(tr, ro, plan)
        traffic_check(tr, ro, plan)
        stage_wire_check(plan)


@pytest.mark.parametrize("seed", range(12))
def test_three_stage_transfer_equals_expectation(seed):
    """Byte level: pack, receive, forward twice, unpack equals the plan-free
    expectation on every rollout rank (casts and fp8 blocks included)."""
    rng = np.random.default_rng(1300 + seed)
    m = random_model(rng)
    tr = describe_layout(m, random_par(rng, m, "trainer"))
    ro = describe_layout(m, random_par(rng, m, "rollout"))
    G = int(rng.integers(1, ro.nranks + 1))
    budget = int(rng.choice([0, 512]))
    plan = build_plan(tr, ro, round_budget=budget, node_size=G)
    dt = tr.ranks[0].locals[0].dtype
    vals = {}
    for t, c in enumerate(tr.catalog):
        x = rng.standard_normal((c.rows, c.cols)).astype(np.float32)
        codes = x.view(np.uint32)
        vals[t] = codes if dt == "f32" else (codes >> 16).astype(np.uint16)
    locs = {s: materialize(tr, s, lambda t: vals[t]) for s in range(tr.nranks)}
    bufs = [run_stages(plan, locs, k) for k in range(len(plan.rounds))]
    for d in range(ro.nranks):
        got = unpack(plan, d, [b[d] for b in bufs])
        want = expected_rollout(ro, d, lambda t: vals[t], dt)
        for a, b in zip(got, want):
            assert np.array_equal(a, b)


@pytest.mark.parametrize("G", [1, 2, 4])
def test_overlapping_rollout_rectangles(G):
    """Overlapping, non-identical rollout rectangles are separate groups: still
    every element of every placement exactly once, byte-exact after casts."""
    from oracle_cases import overlapping_rollout_pair
    tr, ro = overlapping_rollout_pair()
    plan = build_plan(tr, ro, node_size=G)
    brute_force_exchange(tr, ro, plan)
    stage_wire_check(plan)
    rng = np.random.default_rng(G)
    vals = {t: rng.standard_normal((c.rows, c.cols)).astype(np.float32).view(np.uint32) for t, c in enumerate(tr.catalog)}
    locs = {s: materialize(tr, s, lambda t: vals[t]) for s in range(tr.nranks)}
    bufs = run_stages(plan, locs)
    for d in range(ro.nranks):
        for a, b in zip(unpack(plan, d, bufs[d]), expected_rollout(ro, d, lambda t: vals[t], "f32")):
            assert np.array_equal(a, b)
