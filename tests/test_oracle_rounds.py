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

from oracle_cases import hand_rounds_pair, random_model, random_par
from test_oracle_plan import wire_check

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def test_hand_rounds_match_golden():
    tr, ro = hand_rounds_pair()
    want = "".join(l for l in open(os.path.join(GOLDEN, "hand_plan_rounds.txt")) if not l.startswith("#"))
    assert dump(build_plan(tr, ro, round_budget=160)) == want
    # a budget of zero means one round and the single-round form
    assert "rounds=" not in dump(build_plan(tr, ro))


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
