"""The C ABI without a GPU: the library loads, exports every declared call, and
its host planner (layouts, plan, wire offsets) equals the oracle's, line for
line, on every workload at scaled and full size, on random tiny layouts and on
the hand-derived golden plan. Error paths return error codes."""

import os
import re

import numpy as np
import pytest

import paper_2609_25442_amd as wb
from oracle.catalog import CkptTensor
from oracle.layout import Layout, Local, Placement, RankLayout, describe_layout, layout_from_spec
from oracle.plan import build_plan, dump, dump_layout
from synthetic_checkpoint.workloads import ORDER, WORKLOADS, scaled

from oracle_cases import hand_replicated_pair, random_model, random_par
from wb_cases import to_wb

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def test_library_exports_every_declared_call():
    names = set()
    for h in os.listdir(os.path.join(ROOT, "include")):
        if h.endswith(".h"):
            text = open(os.path.join(ROOT, "include", h)).read()
            names |= set(re.findall(r"^\s*(?:int|void|const char\*)\s+(wb_\w+)\s*\(", text, re.M))
    assert len(names) >= 30
    for n in sorted(names):
        assert hasattr(wb.lib, n), n


def test_version():
    assert "gfx950" in wb.version()


@pytest.mark.parametrize("full", [False, True], ids=["scaled", "full"])
@pytest.mark.parametrize("name", ORDER)
def test_layouts_and_plans_equal_oracle(name, full):
    w = WORKLOADS[name] if full else scaled(name)
    tr = wb.Layout.describe(w["model"], w["trainer"])
    ro = wb.Layout.describe(w["model"], w["rollout"])
    otr = layout_from_spec(w["model"], w["trainer"])
    oro = layout_from_spec(w["model"], w["rollout"])
    assert tr.dump() == dump_layout(otr)
    assert ro.dump() == dump_layout(oro)
    want = dump(build_plan(otr, oro))
    for role, rank in ((wb.SENDER, w["pack_rank"]), (wb.RECEIVER, w["unpack_rank"])):
        assert wb.Plan(tr, ro, role, rank).dump() == want


def test_generic_builder_hand_plan():
    tr, ro = hand_replicated_pair()
    golden = "".join(l for l in open(os.path.join(ROOT, "tests", "golden", "hand_plan_replicated.txt"))
                     if not l.startswith("#"))
    p = wb.Plan(to_wb(tr), to_wb(ro), wb.RECEIVER, 1)
    assert p.dump() == golden
    assert p.buffer_bytes == 8200
    assert p.peers() == [(0, 0, 260), (1, 4096, 264), (2, 8192, 8)]
    assert p.region(2, 1) == (4096, 8192, 8)
    s = wb.Plan(to_wb(tr), to_wb(ro), wb.SENDER, 0)
    assert s.buffer_bytes == 4356 and s.peers() == [(0, 0, 272), (1, 4096, 260)]


def test_hand_balanced_rounds_golden():
    from oracle_cases import hand_rounds_balanced_pair
    tr, ro = hand_rounds_balanced_pair()
    golden = "".join(l for l in open(os.path.join(ROOT, "tests", "golden", "hand_plan_rounds_balanced.txt"))
                     if not l.startswith("#"))
    p = wb.Plan(to_wb(tr), to_wb(ro), wb.RECEIVER, 0, round_budget=200)
    assert p.dump() == golden
    assert [p.round_buffer_bytes(k) for k in range(3)] == [152, 552, 152]


@pytest.mark.parametrize("seed", range(25))
def test_random_tiny_plans_equal_oracle(seed):
    rng = np.random.default_rng(seed)
    m = random_model(rng)
    otr = describe_layout(m, random_par(rng, m, "trainer"))
    oro = describe_layout(m, random_par(rng, m, "rollout"))
    want = dump(build_plan(otr, oro))
    tr, ro = to_wb(otr), to_wb(oro)
    assert tr.dump() == dump_layout(otr) and ro.dump() == dump_layout(oro)
    for d in range(oro.nranks):
        assert wb.Plan(tr, ro, wb.RECEIVER, d).dump() == want
    assert wb.Plan(tr, ro, wb.SENDER, otr.nranks - 1).dump() == want


def test_traffic_counts():
    w = WORKLOADS["llama3_8b_fsdp8_to_tp1"]
    tr = wb.Layout.describe(w["model"], w["trainer"])
    ro = wb.Layout.describe(w["model"], w["rollout"])
    p = wb.Plan(tr, ro, wb.RECEIVER, 0)
    assert p.traffic() == (2 * 8030261248, 2 * 8030261248)
    s = wb.Plan(tr, ro, wb.SENDER, 0)
    r, wr = s.traffic()
    assert r == wr and abs(r - 2 * 8030261248 / 8) < 8 * 4096
    w = WORKLOADS["dsv3_ep64_to_ep8_fp8"]
    tr = wb.Layout.describe(w["model"], w["trainer"])
    ro = wb.Layout.describe(w["model"], w["rollout"])
    p = wb.Plan(tr, ro, wb.RECEIVER, 0)
    n = 16 * (33 * 3 * 2048 * 7168 + 256 * 7168)
    scales = 16 * (32 * 32 * 56 + 32 * 56 * 16 + 32 * 56 + 56 * 16)
    assert p.traffic() == (2 * n, n - 16 * 256 * 7168 + 2 * 16 * 256 * 7168 + 4 * scales)
    assert p.work_counts()[1] == scales


@pytest.mark.parametrize("name", ORDER)
def test_copy_launch_grid_is_dense(name):
    """The copy kernel's grid at full size: chunked items take one workgroup per
    chunk (one 16-byte vector per lane: 1 KiB for one-wave workgroups, so an
    item of up to 256 KiB spans at most 256), transposes one per tile, the
    element-wise items one workgroup each, so no launch is dominated by
    workgroups that find no work: each moves at least half a chunk's
    read-plus-write bytes on average, also where most items are transposes
    (the TP4 trainer's pack) or element-wise (fp8 unpack copies)."""
    w = WORKLOADS[name]
    tr = wb.Layout.describe(w["model"], w["trainer"])
    ro = wb.Layout.describe(w["model"], w["rollout"])
    for role, rank in ((wb.SENDER, w["pack_rank"]), (wb.RECEIVER, w["unpack_rank"])):
        p = wb.Plan(tr, ro, role, rank)
        # whole transpose tiles of 128 source rows x 512 columns: one tile-kernel workgroup each
        tiles, ty, tt = p.launch_grid(4)
        tr_, tw_ = p.kernel_traffic(4)
        assert tt == 1024 and ty == (1 if tiles else 0) and tr_ == tw_ == tiles * 128 * 512 * 2
        if (name, role) == ("llama3_8b_tp4_to_tp2", wb.SENDER):
            # the row-parallel o and down slabs, [1024, 4096] and [3584, 4096] per layer
            assert tiles == 32 * (8 + 28) * 8
        items = p.work_counts()[0] - tiles
        x, y, threads = p.launch_grid(0)
        assert threads in (64, 128, 256) and x <= 1 << 22
        chunk = 16 * threads
        wgs = x * y
        r, wr = p.kernel_traffic(0)
        assert items <= wgs < (256 << 10) // chunk * items + y
        assert (r + wr) / wgs >= chunk, (name, role, wgs, r + wr)
    fx, fy, ft = p.launch_grid(1)
    # fp8 blocks: pairable ones (single-piece, row bands) two per workgroup,
    # the others one each
    nb = p.work_counts()[1]
    assert ft == 256 and fy == (1 if nb else 0) and (nb + 1) // 2 <= fx <= nb
    # the launches' algorithmic bytes add up to the rank's
    parts = [p.kernel_traffic(k) for k in (0, 1, 4)]
    assert tuple(map(sum, zip(*parts))) == p.traffic()
    if name == "dsv3_ep64_to_ep8_fp8":
        # routed-expert blocks (97 %) are single-piece and the shared expert's
        # are row bands: all pair up
        assert fx == (nb + 1) // 2
    _expect(wb.WB_EINVAL, p.launch_grid, 5, 0)
    _expect(wb.WB_EINVAL, p.launch_grid, 0, 1)


def _expect(code, fn, *a):
    with pytest.raises(wb.WbError) as e:
        fn(*a)
    assert e.value.code == code, str(e.value)


def test_error_paths():
    m = dict(WORKLOADS["llama3_8b_fsdp8_to_tp1"]["model"])
    _expect(wb.WB_EINVAL, wb.Layout.describe, m, dict(style="serving", dtype="bf16", tp=3))
    _expect(wb.WB_EINVAL, wb.Layout.describe, m, dict(style="fsdp_flat", dtype="bf16", fsdp=0))
    _expect(wb.WB_EINVAL, wb.Layout.describe, m, dict(style="serving", dtype="f8e4m3"))
    _expect(wb.WB_EUNSUPPORTED, wb.Layout.describe, dict(WORKLOADS["mixtral_ep8fsdp2_to_ep2"]["model"]),
            dict(style="megatron", dtype="bf16", tp=2, ep=2))
    _expect(wb.WB_EUNSUPPORTED, wb.Layout.describe, m,
            dict(style="serving", dtype="bf16", quant="f8e4m3", quant_block=256))
    tr = wb.Layout.describe(m, dict(style="fsdp_flat", dtype="bf16", fsdp=8))
    ro = wb.Layout.describe(m, dict(style="serving", dtype="bf16"))
    _expect(wb.WB_EINVAL, wb.Plan, tr, ro, wb.SENDER, 8)
    _expect(wb.WB_EINVAL, wb.Plan, tr, ro, wb.RECEIVER, 1)
    _expect(wb.WB_EINVAL, wb.Plan, tr, ro, 7, 0)
    other = wb.Layout.describe(dict(m, num_layers=2), dict(style="serving", dtype="bf16"))
    _expect(wb.WB_EINVAL, wb.Plan, tr, other, wb.RECEIVER, 0)
    # a placement outside its tensor / local
    L = wb.Layout.create([("T", 4, 4)], 1)
    L.add_local(0, "a", "f32", 1, 4, 4)
    _expect(wb.WB_EINVAL, L.add_placement, 0, 0, 0, 5, 0, 4, 0, 0, 4)
    _expect(wb.WB_EINVAL, L.add_placement, 0, 0, 0, 4, 0, 4, 0, 1, 4)
    _expect(wb.WB_EINVAL, L.add_placement, 0, 0, 0, 4, 0, 4, 1, 0, 4)
    _expect(wb.WB_EUNSUPPORTED, L.add_local, 0, "q", "f8e4m3", 1, 4, 4, 0)
    # overlapping, non-identical trainer rectangles
    T = wb.Layout.create([("T", 4, 4)], 2)
    for r, (a, b) in enumerate([(0, 2), (1, 4)]):
        T.add_local(r, "a", "f32", 1, b - a, 4)
        T.add_placement(r, 0, a, b, 0, 4, 0, 0, 4)
    R = wb.Layout.create([("T", 4, 4)], 1)
    R.add_local(0, "x", "f32", 1, 4, 4)
    R.add_placement(0, 0, 0, 4, 0, 4, 0, 0, 4)
    _expect(wb.WB_EUNSUPPORTED, wb.Plan, T, R, wb.RECEIVER, 0)
    # rollout element held by no trainer
    T2 = wb.Layout.create([("T", 4, 4)], 1)
    T2.add_local(0, "a", "f32", 1, 2, 4)
    T2.add_placement(0, 0, 0, 2, 0, 4, 0, 0, 4)
    _expect(wb.WB_EINVAL, wb.Plan, T2, R, wb.RECEIVER, 0)
    # rollout tensor not exactly covered
    R2 = wb.Layout.create([("T", 4, 4)], 1)
    R2.add_local(0, "x", "f32", 1, 5, 4)
    R2.add_placement(0, 0, 0, 4, 0, 4, 0, 0, 4)
    _expect(wb.WB_EINVAL, wb.Plan, T2, R2, wb.RECEIVER, 0)
    # pack/unpack before upload, or with the wrong role
    p = wb.Plan(tr, ro, wb.RECEIVER, 0)
    _expect(wb.WB_EINVAL, p.unpack, 0, [0] * p.num_local_tensors, 0)
    _expect(wb.WB_EINVAL, p.pack, [0] * p.num_local_tensors, 0, 0)
    # queries with null arguments
    assert wb.lib.wb_plan_work_digest(p._h, None) == wb.WB_EINVAL
    assert wb.lib.wb_plan_work_digest(None, wb.byref(wb.c_uint64())) == wb.WB_EINVAL


def test_hand_rounds_golden():
    from oracle_cases import hand_rounds_pair
    tr, ro = hand_rounds_pair()
    golden = "".join(l for l in open(os.path.join(ROOT, "tests", "golden", "hand_plan_rounds.txt"))
                     if not l.startswith("#"))
    p = wb.Plan(to_wb(tr), to_wb(ro), wb.RECEIVER, 0, round_budget=160)
    assert p.dump() == golden
    assert p.num_rounds == 2 and p.round_buffer_bytes(0) == 320 and p.round_buffer_bytes(1) == 544
    assert p.buffer_bytes == 544
    assert p.round_region(1, 0, 0) == (0, 0, 544)


@pytest.mark.parametrize("seed", range(25))
def test_random_round_plans_equal_oracle(seed):
    rng = np.random.default_rng(700 + seed)
    m = random_model(rng)
    otr = describe_layout(m, random_par(rng, m, "trainer"))
    oro = describe_layout(m, random_par(rng, m, "rollout"))
    budget = int(rng.integers(64, 8192))
    want = dump(build_plan(otr, oro, round_budget=budget))
    tr, ro = to_wb(otr), to_wb(oro)
    assert wb.Plan(tr, ro, wb.RECEIVER, int(rng.integers(0, oro.nranks)), round_budget=budget).dump() == want
    assert wb.Plan(tr, ro, wb.SENDER, int(rng.integers(0, otr.nranks)), round_budget=budget).dump() == want


@pytest.mark.parametrize("name", ORDER)
def test_workload_round_plans_equal_oracle(name):
    for w, budgets in ((scaled(name), (3000, 50000)), (WORKLOADS[name], (1 << 30, 4 << 30))):
        tr = wb.Layout.describe(w["model"], w["trainer"])
        ro = wb.Layout.describe(w["model"], w["rollout"])
        otr = layout_from_spec(w["model"], w["trainer"])
        oro = layout_from_spec(w["model"], w["rollout"])
        for b in budgets:
            want = dump(build_plan(otr, oro, round_budget=b))
            p = wb.Plan(tr, ro, wb.RECEIVER, w["unpack_rank"], round_budget=b)
            assert p.dump() == want, (name, b)
            assert wb.Plan(tr, ro, wb.SENDER, w["pack_rank"], round_budget=b).dump() == want


def test_round_calls_need_round_plans():
    w = scaled("llama3_8b_fsdp8_to_tp1")
    tr = wb.Layout.describe(w["model"], w["trainer"])
    ro = wb.Layout.describe(w["model"], w["rollout"])
    p = wb.Plan(tr, ro, wb.RECEIVER, 0, round_budget=50000)
    assert p.num_rounds > 1
    _expect(wb.WB_EINVAL, p.unpack, 0, [0] * p.num_local_tensors, 0)       # not uploaded, and several rounds
    _expect(wb.WB_EINVAL, p.unpack_round, p.num_rounds, 0, [0] * p.num_local_tensors, 0)
    _expect(wb.WB_EINVAL, wb.Plan, tr, ro, wb.RECEIVER, 0, -1)


def test_hand_exchange_golden():
    from oracle_cases import hand_exchange_pair
    tr, ro = hand_exchange_pair()
    golden = "".join(l for l in open(os.path.join(ROOT, "tests", "golden", "hand_plan_exchange.txt"))
                     if not l.startswith("#"))
    for d in range(3):
        p = wb.Plan(to_wb(tr), to_wb(ro), wb.RECEIVER, d, node_size=2)
        assert p.dump() == golden
        assert p.node_size == 2
    p = wb.Plan(to_wb(tr), to_wb(ro), wb.RECEIVER, 0, node_size=2)
    assert p.buffer_bytes == 12304
    assert p.forward_bytes(1) == 520 and p.forward_bytes(2) == 272
    assert p.stage_region(0, 1, 2, 0) == (0, 8192, 520)
    assert p.stage_region(0, 2, 1, 0) == (0, 12288, 16)
    assert p.stage_region(0, 0, 1, 0) == (0, 4096, 264)
    assert p.kernel_traffic(2) == (8 + 8 + 32, 48) and p.kernel_traffic(3) == (32 + 16, 48)
    s = wb.Plan(to_wb(tr), to_wb(ro), wb.SENDER, 1, node_size=2)
    assert s.forward_bytes(1) == 0 and s.buffer_bytes == 4104


@pytest.mark.parametrize("seed", range(30))
def test_random_exchange_plans_equal_oracle(seed):
    rng = np.random.default_rng(1900 + seed)
    m = random_model(rng)
    otr = describe_layout(m, random_par(rng, m, "trainer"))
    oro = describe_layout(m, random_par(rng, m, "rollout"))
    G = int(rng.integers(1, oro.nranks + 1))
    budget = int(rng.choice([0, 0, 300, 3000]))
    want = dump(build_plan(otr, oro, round_budget=budget, node_size=G))
    tr, ro = to_wb(otr), to_wb(oro)
    for d in range(oro.nranks):
        assert wb.Plan(tr, ro, wb.RECEIVER, d, round_budget=budget, node_size=G).dump() == want
    assert wb.Plan(tr, ro, wb.SENDER, int(rng.integers(0, otr.nranks)), round_budget=budget,
                   node_size=G).dump() == want


@pytest.mark.parametrize("name", ORDER)
def test_workload_exchange_plans_equal_oracle(name):
    for w, full in ((scaled(name), False), (WORKLOADS[name], True)):
        tr = wb.Layout.describe(w["model"], w["trainer"])
        ro = wb.Layout.describe(w["model"], w["rollout"])
        otr = layout_from_spec(w["model"], w["trainer"])
        oro = layout_from_spec(w["model"], w["rollout"])
        for G in sorted({1, max(1, oro.nranks // 2)}):
            budget = (4 << 30) if full else 0
            want = dump(build_plan(otr, oro, round_budget=budget, node_size=G))
            p = wb.Plan(tr, ro, wb.RECEIVER, w["unpack_rank"], round_budget=budget, node_size=G)
            assert p.dump() == want, (name, G)
            assert wb.Plan(tr, ro, wb.SENDER, w["pack_rank"], round_budget=budget, node_size=G).dump() == want


def test_exchange_errors():
    tr, ro = hand_replicated_pair()
    _expect(wb.WB_EINVAL, wb.Plan, to_wb(tr), to_wb(ro), wb.RECEIVER, 0, 0, -1)
    p = wb.Plan(to_wb(tr), to_wb(ro), wb.RECEIVER, 0, node_size=1)
    _expect(wb.WB_EINVAL, p.forward_round, 0, 1, 0, 0, 0)        # not uploaded
    _expect(wb.WB_EINVAL, p.stage_region, 0, 3, 0, 0)
    _expect(wb.WB_EINVAL, p.forward_bytes, 0)
    s = wb.Plan(to_wb(tr), to_wb(ro), wb.SENDER, 0, node_size=1)
    _expect(wb.WB_EINVAL, s.forward_round, 0, 1, 0, 0, 0)        # senders do not forward
    # a rollout rank holding one rectangle twice
    R = wb.Layout.create([("T", 2, 4)], 1)
    R.add_local(0, "x", "f32", 1, 2, 4)
    R.add_local(0, "y", "f32", 1, 2, 4)
    R.add_placement(0, 0, 0, 2, 0, 4, 0, 0, 4)
    R.add_placement(0, 0, 0, 2, 0, 4, 1, 0, 4)
    T = wb.Layout.create([("T", 2, 4)], 1)
    T.add_local(0, "a", "f32", 1, 2, 4)
    T.add_placement(0, 0, 0, 2, 0, 4, 0, 0, 4)
    assert wb.Plan(T, R, wb.RECEIVER, 0).num_segments == 2
    _expect(wb.WB_EINVAL, wb.Plan, T, R, wb.RECEIVER, 0, 0, 1)


def test_segment_query_matches_the_oracle():
    from oracle_cases import hand_exchange_pair
    tr, ro = hand_exchange_pair()
    op = build_plan(tr, ro, node_size=2)
    p = wb.Plan(to_wb(tr), to_wb(ro), wb.RECEIVER, 2, node_size=2)
    segs = p.segments()
    assert len(segs) == len(op.segments) == 17
    for a, g in zip(segs, op.segments):
        assert (a["sender"], a["receiver"], a["tensor"], a["stage"], a["round"]) == (g.s, g.d, g.t, g.stage, g.round)
        assert (a["r0"], a["r1"], a["c0"], a["c1"]) == (g.rect.r0, g.rect.r1, g.rect.c0, g.rect.c1)
        assert (a["send_offset"], a["recv_offset"], a["bytes"], a["origin"]) == (g.send_off, g.recv_off, g.nbytes, g.origin)
        assert a["src_offset"] == g.src_off and a["dst_placement"] == g.dst_pl
        assert a["src_placement"] == (g.src_pl if g.stage == 0 else -1)
    import ctypes
    info = wb.SegmentInfo()
    assert wb.lib.wb_plan_segment(p._h, 17, ctypes.byref(info)) == wb.WB_EINVAL
    assert wb.lib.wb_plan_segment(p._h, -1, ctypes.byref(info)) == wb.WB_EINVAL


def test_local_tensor_query():
    w = WORKLOADS["dsv3_ep64_to_ep8_fp8"]
    tr = wb.Layout.describe(w["model"], w["trainer"])
    ro = wb.Layout.describe(w["model"], w["rollout"])
    p = wb.Plan(tr, ro, wb.RECEIVER, 0)
    locs = ro.locals(0)
    assert p.num_local_tensors == len(locs)
    for i, lc in enumerate(locs):
        assert p.local_tensor(i) == (lc["dtype"], lc["numel"])
    _expect(wb.WB_EINVAL, p.local_tensor, len(locs))


@pytest.mark.parametrize("G", [1, 2, 4])
def test_overlapping_rollout_exchange_equals_oracle(G):
    from oracle_cases import overlapping_rollout_pair
    tr, ro = overlapping_rollout_pair()
    want = dump(build_plan(tr, ro, node_size=G))
    for d in range(4):
        assert wb.Plan(to_wb(tr), to_wb(ro), wb.RECEIVER, d, node_size=G).dump() == want


def test_degenerate_layouts_are_refused_by_both_sides():
    """A zero-sized checkpoint tensor and a rollout rank needing elements no
    trainer holds are errors for the library (WB_EINVAL) and for the oracle
    (ValueError); a trainer rank that holds nothing gets an empty plan with an
    empty grid."""
    with pytest.raises(wb.WbError) as e:
        wb.Layout.create([("Z", 0, 8), ("A", 4, 8)], 1)
    assert e.value.code == wb.WB_EINVAL
    with pytest.raises(ValueError):
        CkptTensor("Z", 0, 8)
    cat = [CkptTensor("A", 4, 4)]
    tr = Layout(cat, [RankLayout([Local("a", "bf16", 1, 2, 4)], [Placement(0, 0, 2, 0, 4, 0, 0, 4)])])
    ro = Layout(cat, [RankLayout([Local("a", "bf16", 1, 4, 4)], [Placement(0, 0, 4, 0, 4, 0, 0, 4)])])
    _expect(wb.WB_EINVAL, wb.Plan, to_wb(tr), to_wb(ro), wb.RECEIVER, 0)
    with pytest.raises(ValueError):
        build_plan(tr, ro)
    cat = [CkptTensor("A", 1, 1)]
    tr = Layout(cat, [RankLayout([Local("a", "bf16", 1, 1, 1)], [Placement(0, 0, 1, 0, 1, 0, 0, 1)]),
                      RankLayout([], [])])
    ro = Layout(cat, [RankLayout([Local("a", "bf16", 1, 1, 1)], [Placement(0, 0, 1, 0, 1, 0, 0, 1)])])
    s1 = wb.Plan(to_wb(tr), to_wb(ro), wb.SENDER, 1)
    assert s1.buffer_bytes == 0 and s1.work_counts() == (0, 0, 0) and s1.launch_grid(0)[:2] == (0, 0)
    r0 = wb.Plan(to_wb(tr), to_wb(ro), wb.RECEIVER, 0)
    assert r0.work_counts()[0] == 1 and r0.traffic() == (2, 2)
    assert build_plan(tr, ro).send_bytes[1] == 0


@pytest.mark.parametrize("name", ORDER)
def test_work_item_size_changes_only_the_grid(name, monkeypatch):
    """WB_TASK_BYTES only re-cuts the kernels' work: the canonical plan, the
    buffer sizes and each launch's algorithmic bytes are the same for 1 KiB,
    4 KiB, the default and 1 GiB items, and every grid has a workgroup for each
    chunk of its longest item class (the planner's bounds proof runs on every
    plan)."""
    w = scaled(name)
    tr = wb.Layout.describe(w["model"], w["trainer"])
    ro = wb.Layout.describe(w["model"], w["rollout"])
    seen = None
    items = {}
    for tb in ("1024", "4096", "", str(1 << 30)):
        monkeypatch.setenv("WB_TASK_BYTES", tb)
        rp = wb.Plan(tr, ro, wb.RECEIVER, w["unpack_rank"])
        sp = wb.Plan(tr, ro, wb.SENDER, w["pack_rank"])
        items[tb] = rp.work_counts()[0]
        facts = (rp.dump(), rp.buffer_bytes, sp.buffer_bytes, rp.kernel_traffic(0), rp.kernel_traffic(1),
                 sp.kernel_traffic(0))
        assert seen is None or facts == seen, (name, tb)
        seen = facts
        for p in (rp, sp):
            x, y, _ = p.launch_grid(0)
            n = p.work_counts()[0]
            assert (x * y >= n) if n else (x, y) == (0, 0)
    assert items["1024"] > items[""]  # the setting reached the planner


def test_binding_refuses_bad_tensors_before_the_library():
    """The binding checks every tensor of a pack or unpack against the plan
    (count, dtype, element count, contiguity, device or pinned memory) and the
    buffers' size before anything reaches the library: all refused here on a
    machine without a GPU, so nothing could have been launched."""
    import torch

    tr, ro = hand_replicated_pair()
    T, R = to_wb(tr), to_wb(ro)
    rp = wb.Plan(T, R, wb.RECEIVER, 1)
    sp = wb.Plan(T, R, wb.SENDER, 0)
    dst = [torch.empty(12, dtype=torch.bfloat16), torch.empty(5, dtype=torch.bfloat16)]
    recv = torch.empty(rp.buffer_bytes, dtype=torch.uint8)

    def refused(fn, *a, word):
        with pytest.raises(wb.WbError) as e:
            fn(*a)
        assert e.value.code == wb.WB_EINVAL and word in str(e.value), str(e.value)

    refused(rp.unpack, recv, dst[:1], word="2 local tensors")
    refused(rp.unpack, recv, dst, word="pinned")                                   # pageable host tensors
    refused(rp.unpack, recv, [dst[0].float(), dst[1]], word="dtype float32")
    refused(rp.unpack, recv, [torch.empty(11, dtype=torch.bfloat16), dst[1]], word="smaller")
    refused(rp.unpack, recv, [torch.empty(13, dtype=torch.int16), dst[1]], word="larger")
    refused(rp.unpack, recv, [torch.empty(6, 4, dtype=torch.bfloat16)[:, ::2], dst[1]], word="contiguous")
    refused(rp.unpack_round, 0, recv, dst[:1], word="2 local tensors")
    # raw pointers pass to the library, which refuses the unuploaded plan
    refused(rp.unpack, 0, [0, 0], 0, word="uploaded")
    src = [torch.empty(24, dtype=torch.float32), torch.empty(10, dtype=torch.float32)]
    refused(sp.pack, src, torch.empty(sp.buffer_bytes, dtype=torch.uint8), word="pinned")
    refused(sp.pack, [0, 0], torch.empty(sp.buffer_bytes - 1, dtype=torch.uint8), word="pinned")
    refused(sp.pack_round, 0, [0, 0, 0], 0, word="2 local tensors")
    refused(sp.upload, torch.empty(sp.workspace_bytes, dtype=torch.uint8), word="pinned")


@pytest.mark.parametrize("name", ORDER)
def test_noalloc_entry_reads_only_planned_tables(name):
    """wb_unpack_round_noalloc reads the round's table ranges before anything
    else; on a machine without a GPU it must then stop at the device lookup
    with an error, for plans with and without fp8 blocks and in every round
    (a plan without fp8 blocks once had no piece ranges, and the call read
    past an empty table)."""
    w = scaled(name)
    tr = wb.Layout.describe(w["model"], w["trainer"])
    ro = wb.Layout.describe(w["model"], w["rollout"])
    for budget in (0, 4096):
        p = wb.Plan(tr, ro, wb.RECEIVER, w["unpack_rank"], round_budget=budget)
        ptrs = (wb.c_void_p * max(1, p.num_local_tensors))()
        for k in range(p.num_rounds):
            rc = wb.lib.wb_unpack_round_noalloc(p._h, k, None, ptrs, None)
            assert rc == wb.WB_EHIP, (rc, wb.lib.wb_last_error())
        assert wb.lib.wb_unpack_round_noalloc(p._h, p.num_rounds, None, ptrs, None) == wb.WB_EINVAL
    s = wb.Plan(tr, ro, wb.SENDER, w["pack_rank"])
    assert wb.lib.wb_unpack_round_noalloc(s._h, 0, None, ptrs, None) == wb.WB_EINVAL


@pytest.mark.parametrize("budget,G", [(0, 0), (1 << 30, 0), (0, 2)])
def test_plan_threads_change_nothing(budget, G, monkeypatch):
    """The full DeepSeek-V3 rollout rank's fp8 tables (1.4 M blocks, built local
    by local on the planning threads and checked in runs of 2^14 blocks) and
    every other work table are the same for 1, 3 and 16 planning threads, with
    rounds and with exchange stages; the digest does see the tables (1 KiB work
    items change it)."""
    w = WORKLOADS["dsv3_ep64_to_ep8_fp8"]
    tr = wb.Layout.describe(w["model"], w["trainer"])
    ro = wb.Layout.describe(w["model"], w["rollout"])
    seen = set()
    for n in ("1", "3", "16"):
        monkeypatch.setenv("WB_PLAN_THREADS", n)
        p = wb.Plan(tr, ro, wb.RECEIVER, w["unpack_rank"], round_budget=budget, node_size=G)
        assert p.work_counts()[1] > 1 << 20
        seen.add((p.work_digest(), p.dump()))
    assert len(seen) == 1
    monkeypatch.setenv("WB_TASK_BYTES", "1024")
    p = wb.Plan(tr, ro, wb.RECEIVER, w["unpack_rank"], round_budget=budget, node_size=G)
    assert p.work_digest() != next(iter(seen))[0]


def test_c_client_compiles_and_plans(tmp_path):
    """include/wb.h is a C header: a C99 program using it (tests/c_abi_plan.c)
    compiles without warnings under -pedantic, links against libwb.so and, on
    a machine without a GPU, plans the tiny workload's rollout rank 1 exactly
    as the Python binding does (buffer bytes, work counts, canonical dump)."""
    import shutil
    import subprocess

    cc = shutil.which("gcc") or shutil.which("cc")
    if cc is None:
        pytest.skip("no C compiler")
    libdir = os.path.dirname(os.path.abspath(wb.LIB_PATH))
    exe = str(tmp_path / "c_abi_plan")
    rocm = os.environ.get("ROCM_PATH", "/opt/rocm")
    subprocess.run([cc, "-std=c99", "-Wall", "-Wextra", "-Werror", "-pedantic", "-I", os.path.join(ROOT, "include"),
                    os.path.join(ROOT, "tests", "c_abi_plan.c"), "-o", exe, "-L", libdir, "-l:" + os.path.basename(wb.LIB_PATH),
                    "-Wl,-rpath," + libdir, "-Wl,-rpath-link," + os.path.join(rocm, "lib")],
                   check=True, capture_output=True, text=True)
    out = subprocess.run([exe], check=True, capture_output=True, text=True, timeout=60).stdout
    version, counts, dump = out.split("\n", 2)
    w = WORKLOADS["tiny_fsdp2_to_tp2"]
    p = wb.Plan(wb.Layout.describe(w["model"], w["trainer"]), wb.Layout.describe(w["model"], w["rollout"]),
                wb.RECEIVER, 1)
    assert version == wb.version()
    assert [int(x) for x in counts.split()] == [p.buffer_bytes, *p.work_counts()]
    assert dump == p.dump()


@pytest.mark.parametrize("seed", range(40))
def test_plan_threads_change_nothing_on_random_fp8_layouts(seed, monkeypatch):
    """Random layouts with fp8 rollouts of 4 x 4 blocks (ragged, multi-piece
    and row-band blocks), rounds and exchange stages: with WB_PLAN_THREADS set
    every plan builds its fp8 tables on that many threads, and 1 and 7 threads
    give the same work tables and dump on every rollout rank."""
    rng = np.random.default_rng(5000 + seed)
    m = random_model(rng)
    otr = describe_layout(m, random_par(rng, m, "trainer"))
    oro = describe_layout(m, random_par(rng, m, "rollout", blocks=(4,)))
    tr, ro = to_wb(otr), to_wb(oro)
    budget = int(rng.choice([0, 0, 300, 3000]))
    G = int(rng.integers(0, oro.nranks + 1))
    for d in range(oro.nranks):
        seen = set()
        for n in ("1", "7"):
            monkeypatch.setenv("WB_PLAN_THREADS", n)
            p = wb.Plan(tr, ro, wb.RECEIVER, d, round_budget=budget, node_size=G)
            seen.add((p.work_digest(), p.dump()))
        assert len(seen) == 1, (seed, d)
