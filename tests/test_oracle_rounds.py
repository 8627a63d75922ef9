"""Pins for the oracle's rounds (Sec. 3.2 round-based transfer; App. D budget):
a hand-derived golden, budget and block invariants on random layouts, and the
unique unpack result through every round's buffers."""

import os

import numpy as np
import pytest

import synthetic_checkpoint as sc
from oracle.layout import describe_layout, layout_from_spec
from oracle.plan import build_plan, dump
from oracle.transfer import expected_rollout, local_index, materialize, network, pack, unpack
from synthetic_checkpoint.workloads import ORDER, WORKLOADS, scaled

from oracle_cases import hand_rounds_balanced_pair, hand_rounds_pair, random_model, random_par
from test_oracle_plan import wire_check

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def test_hand_rounds_match_golden():
    tr, ro = hand_rounds_pair()
    want = "".join(l for l in open(os.path.join(GOLDEN, "hand_plan_rounds.txt")) if not l.startswith("#"))
    assert dump(build_plan(tr, ro, round_budget=160)) == want
    # a budget of zero means one round and the single-round form
    assert "rounds=" not in dump(build_plan(tr, ro))


def test_hand_balanced_rounds_match_golden():
    tr, ro = hand_rounds_balanced_pair()
    want = "".join(l for l in open(os.path.join(GOLDEN, "hand_plan_rounds_balanced.txt")) if not l.startswith("#"))
    assert dump(build_plan(tr, ro, round_budget=200)) == want


def _partitions(k, parts):
    """Every split of k units in order into ``parts`` non-empty runs, as run
    boundaries [0, b1, ..., k]."""
    import itertools
    for cuts in itertools.combinations(range(1, k), parts - 1):
        yield [0, *cuts, k]


@pytest.mark.parametrize("seed", range(30))
def test_rounds_are_min_max_balanced(seed):
    """Brute force over every way to cut a few units into runs: the plan takes
    the fewest rounds whose runs fit the budget, and among cuts into that
    many rounds its largest run is the smallest possible, or at most the even
    share ceil(total / rounds) of the busiest rank. A run's size is the most
    bytes it gives a rank that some unit after its first touches (a rank may
    go past the cap only through the first unit of its round, which can be
    larger than the cap on its own)."""
    from oracle.catalog import CkptTensor
    from oracle.layout import Layout, Local, Placement, RankLayout
    rng = np.random.default_rng(700 + seed)
    k = int(rng.integers(3, 9))
    sizes = [int(x) for x in rng.integers(1, 40, k)]
    cat = [CkptTensor(f"T{i}", 1, n) for i, n in enumerate(sizes)]
    # two trainer ranks: a tensor held by one of them or by both (then split)
    held = [int(rng.integers(0, 3)) for _ in range(k)]
    trs = []
    for r in range(2):
        ts = [i for i in range(k) if held[i] in (r, 2)]
        trs.append(RankLayout([Local(f"t{i}", "f32", 1, 1, sizes[i]) for i in ts],
                              [Placement(i, 0, 1, 0, sizes[i], j, 0, sizes[i]) for j, i in enumerate(ts)]))
    # two rollout ranks: every tensor wanted by one or both
    want = [int(rng.integers(0, 3)) for _ in range(k)]
    ros = []
    for d in range(2):
        ts = [i for i in range(k) if want[i] in (d, 2)]
        ros.append(RankLayout([Local(f"x{i}", "bf16", 1, 1, sizes[i]) for i in ts],
                              [Placement(i, 0, 1, 0, sizes[i], j, 0, sizes[i]) for j, i in enumerate(ts)]))
    tr, ro = Layout(cat, trs), Layout(cat, ros)
    one = build_plan(tr, ro)
    unit_bytes = []
    for i in range(k):
        b = {}
        for g in one.segments:
            if g.t == i:
                b[("s", g.s)] = b.get(("s", g.s), 0) + g.nbytes
                b[("d", g.d)] = b.get(("d", g.d), 0) + g.nbytes
        unit_bytes.append(b)
    largest = max(max(b.values()) for b in unit_bytes)
    total = sum(sum(b.values()) for b in unit_bytes)
    budget = int(rng.integers(largest // 2 + 1, max(largest // 2 + 2, total // 3)))

    def cost(bounds):  # the largest run: bytes of ranks that a unit after its first touches
        worst = 0
        for a, z in zip(bounds, bounds[1:]):
            per, later = {}, set()
            for j, b in enumerate(unit_bytes[a:z]):
                for key, v in b.items():
                    per[key] = per.get(key, 0) + v
                    if j:
                        later.add(key)
            worst = max([worst] + [per[key] for key in later])
        return worst

    n = next(p for p in range(1, k + 1) if any(cost(c) <= budget for c in _partitions(k, p)))
    best = min(cost(c) for p in range(1, n + 1) for c in _partitions(k, p))
    plan = build_plan(tr, ro, round_budget=budget)
    assert len(plan.rounds) == n
    rounds = [min(g.round for g in plan.segments if g.t == i) for i in range(k)]
    assert rounds == sorted(rounds) and all(g.round == rounds[g.t] for g in plan.segments)
    bounds = [0] + [i for i in range(1, k) if rounds[i] != rounds[i - 1]] + [k]
    share = max(-(-sum(b.get(key, 0) for b in unit_bytes) // n) for key in set().union(*unit_bytes))
    got = cost(bounds)
    assert got <= budget and (got == best or got <= share), (got, best, share, bounds)


def _round_checks(plan, budget):
    tr, ro = plan.trainer, plan.rollout
    nr = len(plan.rounds)
    assert sorted({g.round for g in plan.segments}) == list(range(nr))
    # canonical order is kept: rounds never go back
    rs = [g.round for g in plan.segments]
    # per-rank bytes per round within budget unless the round is one unit
    for k in range(nr):
        segs = [g for g in plan.segments if g.round == k]
        per = {}
        for g in segs:
            per[("s", g.s)] = per.get(("s", g.s), 0) + g.nbytes
            per[("d", g.d)] = per.get(("d", g.d), 0) + g.nbytes
        if max(per.values()) > budget:
            tensors = {g.t for g in segs}
            # over budget only when everything in the round had to travel together
            assert len(tensors) == 1 or all(g.round == k for g in plan.segments if g.t in tensors)
    # no fp8 block is fed from two rounds (element by element)
    for d, rk in enumerate(ro.ranks):
        for u, lc in enumerate(rk.locals):
            if not lc.block:
                continue
            owner = np.full(lc.numel, -1, dtype=np.int64)
            for g in plan.segments:
                q = rk.placements[g.dst_pl] if g.d == d else None
                if q is None or q.u != u:
                    continue
                i = np.arange(g.rect.r0, g.rect.r1)[:, None]
                j = np.arange(g.rect.c0, g.rect.c1)[None, :]
                owner[local_index(q, i, j).ravel()] = g.round
            o = owner.reshape(lc.batch, lc.rows, lc.cols)
            B = lc.block
            for bi in range(0, lc.rows, B):
                for bj in range(0, lc.cols, B):
                    blk = o[:, bi:bi + B, bj:bj + B].reshape(lc.batch, -1)
                    assert np.all(blk == blk[:, :1]), (lc.name, bi, bj)


@pytest.mark.parametrize("seed", range(30))
def test_random_rounds_invariants(seed):
    rng = np.random.default_rng(500 + seed)
    m = random_model(rng)
    tr = describe_layout(m, random_par(rng, m, "trainer"))
    ro = describe_layout(m, random_par(rng, m, "rollout"))
    single = build_plan(tr, ro)
    budget = int(rng.integers(64, 4096))
    plan = build_plan(tr, ro, round_budget=budget)
    # same segments and owners as the single-round plan, only regrouped
    key = lambda g: (g.s, g.d, g.t, g.rect, g.src_pl, g.dst_pl, g.nbytes)
    assert [key(g) for g in plan.segments] == [key(g) for g in single.segments]
    _round_checks(plan, budget)
    for k in range(len(plan.rounds)):
        sub = type(plan)(plan.trainer, plan.rollout, [g for g in plan.segments if g.round == k], plan.regions,
                         plan.rounds[k].send_bytes, plan.rounds[k].recv_bytes)
        wire_check(sub)


@pytest.mark.parametrize("name", ORDER)
def test_scaled_workload_rounds_unpack(name):
    w = scaled(name)
    tr = layout_from_spec(w["model"], w["trainer"])
    ro = layout_from_spec(w["model"], w["rollout"])
    dt = w["trainer"]["dtype"]
    budget = max(4096, sum(g.nbytes for g in build_plan(tr, ro).segments) // (5 * ro.nranks))
    plan = build_plan(tr, ro, round_budget=budget)
    assert len(plan.rounds) > 1
    _round_checks(plan, budget)
    cache = {}

    def vals(t):
        if t not in cache:
            c = tr.catalog[t]
            cache[t] = sc.values_numpy(t, np.arange(c.numel), dt).reshape(c.rows, c.cols)
        return cache[t]

    locs = {s: materialize(tr, s, vals) for s in range(tr.nranks)}
    for d in range(ro.nranks):
        bufs = []
        for k in range(len(plan.rounds)):
            sends = {s: pack(plan, s, locs[s], k) for s in range(tr.nranks)}
            bufs.append(network(plan, d, sends, k))
        got = unpack(plan, d, bufs)
        for g, e in zip(got, expected_rollout(ro, d, vals, dt)):
            assert np.array_equal(g, e)


def test_full_size_round_counts():
    # 4 GiB per rank per round (the paper's default registered-buffer budget)
    w = WORKLOADS["llama3_8b_fsdp8_to_tp1"]
    plan = build_plan(layout_from_spec(w["model"], w["trainer"]), layout_from_spec(w["model"], w["rollout"]),
                      round_budget=4 << 30)
    assert len(plan.rounds) == 4
    assert all(max(r.recv_bytes) <= 4 << 30 for r in plan.rounds)
