"""The library's source-map scan without a GPU (App. B, Algorithm 1): the
oracle's per-pass diff2 entries of every local tensor go through
wb_probe_record / wb_probe_scan, and the placements the library recovers must
reproduce the exact identifier field of the declared layout, element by
element, on every workload (scaled) and on random layouts; a loader that is
not made of slice copies is refused."""

import numpy as np
import pytest

import paper_2609_25442_amd as wb
from oracle.catalog import CkptTensor
from oracle.diff2 import (FIRST_ID, carry_passes, diff2, id_chunk, id_fields, nonzeros, num_chunks, probe_fields,
                          recombine)
from oracle.layout import Layout, Local, Placement, RankLayout, describe_layout, layout_from_spec
from synthetic_checkpoint.workloads import ORDER, scaled

from oracle_cases import random_model, random_par


def to_oracle_rank(L: "wb.Layout", rank: int) -> RankLayout:
    locs = [Local(x["name"], x["dtype"], x["batch"], x["rows"], x["cols"]) for x in L.locals(rank)]
    pls = [Placement(t, r0, r1, c0, c1, u, base, ld, tr) for (t, r0, r1, c0, c1, u, base, ld, tr) in L.placements(rank)]
    return RankLayout(locs, pls)


def probe_via_library(layout, rank, dtype="bf16", combined=False, carried=False):
    """Feed the oracle's passes of one declared rank into the library scan,
    pass by pass, or (combined) recombined first and recorded as chunk 0, as
    the batched diff2 over held passes hands them over, or (carried) the
    entries the carry passes keep, pass by pass."""
    cat = [(c.name, c.rows, c.cols) for c in layout.catalog]
    P = wb.Probe(cat, dtype)
    assert P.num_chunks == num_chunks(layout.catalog, 16)
    fields = id_fields(layout, rank)
    per_chunk, _ = probe_fields(fields, 16, P.num_chunks)
    if carried:
        per_chunk = [carry_passes([id_chunk(A, k, 16) for k in range(P.num_chunks)], 16)[0] for A in fields]
    rk = layout.ranks[rank]
    for u, lc in enumerate(rk.locals):
        assert P.add_local(lc.name, dtype, lc.batch, lc.rows, lc.cols) == u
        C = lc.cols
        if combined:
            z = recombine(per_chunk[u], 16)
            P.record(u, 0, np.array([i * C + j for (i, j) in z], dtype=np.int64),
                     np.array(list(z.values()), dtype=np.int64))
            continue
        for k, z in enumerate(per_chunk[u]):
            idx = np.array([i * C + j for (i, j) in z], dtype=np.int64)
            val = np.array(list(z.values()), dtype=np.int32)
            P.record(u, k, idx, val)
    out = wb.Layout.create(cat, 1)
    P.scan(out, 0)
    return out, fields


def check(layout, rank, combined=False, carried=False):
    out, fields = probe_via_library(layout, rank, combined=combined, carried=carried)
    got = id_fields(Layout(layout.catalog, [to_oracle_rank(out, 0)]), 0)
    for A, B in zip(fields, got):
        assert np.array_equal(A, B)
    return out


@pytest.mark.parametrize("name", ORDER)
def test_workload_ranks_recovered(name):
    w = scaled(name)
    for side in ("trainer", "rollout"):
        L = layout_from_spec(w["model"], w[side])
        for r in sorted({0, L.nranks - 1}):
            out = check(L, r)
            # on these layouts the scan gives back exactly the declared slice copies
            want = [(p.t, p.r0, p.r1, p.c0, p.c1, p.u, p.base, p.ld, p.tr) for p in L.ranks[r].placements]
            assert sorted(out.placements(0)) == sorted(want), (name, side, r)


@pytest.mark.parametrize("seed", range(30))
def test_random_ranks_recovered(seed):
    rng = np.random.default_rng(4000 + seed)
    m = random_model(rng)
    for side in ("trainer", "rollout"):
        L = describe_layout(m, random_par(rng, m, side))
        check(L, int(rng.integers(0, L.nranks)))


def test_odd_slices_recovered():
    """Strided, reversed and scattered copies fall back to rows or single
    elements but still name every element."""
    cat = [CkptTensor("T", 6, 10), CkptTensor("U", 3, 10)]
    lc = [Local("x", "bf16", 1, 5, 7), Local("y", "bf16", 2, 3, 4)]
    pl = [Placement(0, 0, 5, 0, 3, 0, 0, 7),                 # slab
          Placement(0, 1, 5, 5, 9, 0, 3, 7, 1),              # transposed 4 x 4 -> local cols 3..6
          Placement(1, 0, 1, 0, 4, 1, 0, 4),                 # batch 0 row 0
          Placement(1, 2, 3, 6, 10, 1, 12, 4),               # batch 1 row 0
          Placement(0, 5, 6, 0, 8, 1, 16, 4),                # a flat run over two local rows
          ]
    check(Layout(cat, [RankLayout(lc, pl)]), 0)


def test_not_slice_copies_refused():
    cat = [("T", 4, 4)]
    P = wb.Probe(cat, "bf16")
    P.add_local("x", "bf16", 1, 4, 4)
    A = np.arange(16, dtype=np.int64).reshape(4, 4) ** 2 + FIRST_ID      # not affine
    for k in range(P.num_chunks):
        z = nonzeros(diff2(id_chunk(A, k, 16)))
        P.record(0, k, np.array([i * 4 + j for i, j in z], dtype=np.int64), np.array(list(z.values()), dtype=np.int32))
    out = wb.Layout.create(cat, 1)
    with pytest.raises(wb.WbError) as e:
        P.scan(out, 0)
    assert e.value.code == wb.WB_EUNSUPPORTED


def test_probe_errors():
    with pytest.raises(wb.WbError):
        wb.Probe([("T", 4, 4)], "f8e4m3")
    P = wb.Probe([("T", 4, 4)], "bf16")
    with pytest.raises(wb.WbError):
        P.add_local("x", "f32", 1, 4, 4)
    P.add_local("x", "bf16", 1, 4, 4)
    with pytest.raises(wb.WbError):
        P.record(0, 0, np.array([16], dtype=np.int64), np.array([1], dtype=np.int32))
    with pytest.raises(wb.WbError):
        P.record(0, P.num_chunks, np.array([0], dtype=np.int64), np.array([1], dtype=np.int32))


@pytest.mark.parametrize("name", ORDER)
def test_workload_ranks_recovered_from_recombined_entries(name):
    w = scaled(name)
    for side in ("trainer", "rollout"):
        L = layout_from_spec(w["model"], w[side])
        for r in sorted({0, L.nranks - 1}):
            check(L, r, combined=True)


def test_diff2_batch_workspace():
    """The workspace query runs on the host: field and tile tables, and the
    argument checks (device pointers are not touched)."""
    A = 1 << 20                      # a 16-byte aligned stand-in address

    def ws(fields):
        return wb.diff2_batch_workspace(fields)

    assert ws([]) == 0
    assert ws([(0, "bf16", 0, 7), (0, "f32", 5, 0)]) == 0          # no elements, no tiles
    one = ws([(A, "bf16", 1, 1 << 20)])
    two = ws([(A, "bf16", 300, 4096)])
    assert one > 56 and two > 56 and (one - 56) % 24 == 0 and (two - 56) % 24 == 0
    assert ws([(A, "bf16", 1, 1 << 20), (A, "bf16", 300, 4096)]) == 112 + (one - 56) + (two - 56)
    assert ws([([A, A + 64, A + 128], "bf16", 300, 4096)]) == two   # passes share the tiles
    assert ws([(A, "bf16", 1, 1 << 20), (A + 2, "bf16", 1, 1 << 20)]) > 2 * one - 56   # unaligned: element tiles
    for bad in ([(A, "f8e4m3", 4, 4)], [(A + 1, "bf16", 4, 4)], [(0, "bf16", 4, 4)], [(A, "bf16", -1, 4)],
                [([A, 0], "bf16", 4, 4)], [([A] * 4, "bf16", 4, 4)]):
        with pytest.raises((wb.WbError, ValueError)):
            ws(bad)
    arr = wb._field_array([(A, "bf16", 4, 4)])
    arr[0].passes = 0
    assert wb.lib.wb_diff2_batch_workspace(arr, 1, wb.byref(wb.c_size_t())) == wb.WB_EINVAL


@pytest.mark.parametrize("name", ORDER)
def test_workload_ranks_recovered_from_carried_passes(name):
    w = scaled(name)
    for side in ("trainer", "rollout"):
        L = layout_from_spec(w["model"], w[side])
        for r in sorted({0, L.nranks - 1}):
            check(L, r, carried=True)


def test_diff2_carry_workspace():
    """The carry pass's workspace: the field and tile tables of
    wb_diff2_batch, 256-byte aligned, 2 KiB of counters, two carry tables of
    16-byte slots, slots the smallest power of two at least twice the
    capacity and at least 64, then 64 staged carries of 16 bytes and a 4-byte
    count per tile."""
    A = 1 << 20

    def tables(cap):
        slots = 64
        while slots < 2 * cap:
            slots *= 2
        return 2 * slots * 16

    def ws(fields, cap):
        return wb.diff2_carry_workspace(fields, cap)

    assert ws([], 1) == 2048 + tables(1)
    assert ws([], 100) == 2048 + tables(100) == 2048 + 2 * 256 * 16
    f = [(A, "bf16", 300, 4096), (A, "f32", 1, 1 << 20)]
    head = wb.diff2_batch_workspace(f)
    ntiles = (head - 2 * 56) // 24
    stage = ntiles * 64 * 16 + -(-ntiles * 4 // 256) * 256
    for cap in (1, 33, 1000, 1 << 20):
        assert ws(f, cap) == -(-head // 256) * 256 + 2048 + tables(cap) + stage
    for bad_cap in (0, -1, (1 << 36) + 1):
        with pytest.raises(wb.WbError):
            ws(f, bad_cap)
    with pytest.raises(wb.WbError):
        ws([([A, A + 64], "bf16", 4, 4)], 10)       # a carry pass reads one pass per field


def test_diff2_carry_argument_checks():
    """Refusals decided on the host before any device access."""
    A = 1 << 20
    arr = wb._field_array([(A, "bf16", 4, 4)])
    d = wb.c_void_p(A)

    def call(pass_=0, cap=10, ws=d, nbytes=1 << 20, count=d, carries=d, capacity=4):
        return wb.lib.wb_diff2_carry(arr, 1, pass_, 0, cap, ws, nbytes, d, d, capacity, count, carries, None)

    assert call(pass_=-1) == wb.WB_EINVAL
    assert call(capacity=-1) == wb.WB_EINVAL
    assert call(count=None) == wb.WB_EINVAL
    assert call(count=wb.c_void_p(A + 4)) == wb.WB_EINVAL
    assert call(carries=None) == wb.WB_EINVAL
    assert call(carries=wb.c_void_p(A + 4)) == wb.WB_EINVAL
    assert call(ws=None) == wb.WB_EINVAL
    assert call(ws=wb.c_void_p(A + 4)) == wb.WB_EINVAL


def test_identifier_checkpoint_is_made_on_demand(monkeypatch):
    """The checkpoint a probed loader reads makes a tensor the first time it is
    read and fills it once per pass; membership tests, iteration and len make
    nothing (make_ids replaced by a recorder: no GPU needed)."""
    import torch

    made = []
    monkeypatch.setattr(wb, "make_ids", lambda x, dt, first, k: made.append((x.shape, first, k)))
    cat = [("a", 2, 3), ("b", 1, 4), ("c", 5, 1)]
    probe = wb.Probe(cat, "bf16")
    ck = wb._IdCheckpoint(cat, "bf16", torch.bfloat16, "cpu")
    ck.start_pass(probe, 0)
    assert "b" in ck and "z" not in ck and list(ck) == ["a", "b", "c"] and len(ck) == 3 and made == []
    x = ck["b"]
    assert x.shape == (1, 4) and x.dtype == torch.bfloat16 and made == [((1, 4), probe.first_id(1), 0)]
    assert ck["b"] is x and len(made) == 1           # read again in the same pass: not refilled
    ck.start_pass(probe, 1)
    assert ck["b"] is x and made[-1] == ((1, 4), probe.first_id(1), 1)
    ck["a"]
    assert [m[0] for m in made] == [(1, 4), (1, 4), (2, 3)]
    with pytest.raises(KeyError):
        ck["z"]
