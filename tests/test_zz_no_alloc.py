"""The allocation-free unpack (wb_unpack_round_noalloc, for callers that cannot
allocate) against wb_unpack_round through an uploaded workspace: the rollout
tensors agree byte for byte on consecutive calls (a larger plan, then a
smaller one, so the second call finds the first call's tables in the
library's array), over every round of multi-round plans on plans that were
never uploaded, with whole transpose tiles, and a round whose tables exceed
the array is refused before any pointer is looked at."""

import pytest
import torch

import paper_2609_25442_amd as wb
from oracle.catalog import CkptTensor
from oracle.layout import Layout, Local, Placement, RankLayout, layout_from_spec
from oracle.plan import build_plan
from synthetic_checkpoint.workloads import ORDER, WORKLOADS, scaled

from gpu_util import say, workspace_for
from wb_cases import to_wb

pytestmark = pytest.mark.gpu


def _layouts(w):
    return wb.Layout.describe(w["model"], w["trainer"]), wb.Layout.describe(w["model"], w["rollout"])


def _receive_buffers(plan, dtype, seed):
    """Each round's receive buffer, filled with finite random values of the wire
    dtype (every payload starts at a multiple of 256 bytes)."""
    g = torch.Generator(device="cuda").manual_seed(seed)
    out = []
    for k in range(plan.num_rounds):
        n = plan.round_buffer_bytes(k)
        es = 4 if dtype == "f32" else 2
        x = torch.randn(max(1, (n + es - 1) // es), generator=g, device="cuda") * 0.02
        x = x if dtype == "f32" else x.to(torch.bfloat16)
        out.append(x.view(torch.uint8)[:max(1, n)])
    return out


def _raw(t):
    return t.reshape(-1).view(torch.uint8)


def _compare(name, w, budget, seed):
    tr, ro = _layouts(w)
    return _compare_layouts(name, tr, ro, w["unpack_rank"], w["trainer"]["dtype"], budget, seed)


def _compare_layouts(name, tr, ro, d, dtype, budget, seed):
    up = wb.Plan(tr, ro, wb.RECEIVER, d, round_budget=budget)
    free = wb.Plan(tr, ro, wb.RECEIVER, d, round_budget=budget)     # never uploaded
    ws = workspace_for(up)
    up.upload(ws)
    recvs = _receive_buffers(up, dtype, seed)
    want = wb.allocate_locals(ro, d)
    got = wb.allocate_locals(ro, d)
    for a, b in zip(want, got):
        _raw(a).fill_(0x11)
        _raw(b).fill_(0x22)
    say(f"[noalloc] {name}: {up.num_rounds} rounds, {len(got)} tensors")
    for k in range(up.num_rounds):
        up.unpack_round(k, recvs[k], want)
        free.unpack_round_noalloc(k, recvs[k], got)
    torch.cuda.synchronize()
    for u, (a, b) in enumerate(zip(want, got)):
        assert torch.equal(_raw(a), _raw(b)), f"{name}: local tensor {u} differs"
    return up.num_rounds


def test_noalloc_matches_uploaded_unpack_on_consecutive_calls():
    # the fp8 workload first (copy tasks, single-piece and multi-piece blocks),
    # then a smaller one: the second call overwrites only part of the array
    _compare("dsv3 scaled", scaled("dsv3_ep64_to_ep8_fp8"), 0, 1)
    _compare("tiny", WORKLOADS["tiny_fsdp2_to_tp2"], 0, 2)


@pytest.mark.parametrize("name", ORDER)
def test_noalloc_every_round(name):
    w = scaled(name)
    otr = layout_from_spec(w["model"], w["trainer"])
    oro = layout_from_spec(w["model"], w["rollout"])
    total = sum(g.nbytes for g in build_plan(otr, oro).segments)
    budget = max(4096, total // (4 * oro.nranks))
    assert _compare(name, w, budget, 3) > 2


@pytest.mark.parametrize("rows,cols", [(256, 1024), (600, 1096)])
def test_noalloc_transposed_rollout_tiles(rows, cols):
    # a rollout that stores T transposed: whole transpose tiles (a launch of
    # their own) and, for 600 x 1096, ragged strips and unaligned payloads
    cat = [CkptTensor("T", rows, cols)]
    h = rows // 2
    tr = Layout(cat, [RankLayout([Local("a", "bf16", 1, h, cols)], [Placement(0, 0, h, 0, cols, 0, 0, cols)]),
                      RankLayout([Local("b", "bf16", 1, rows - h, cols)], [Placement(0, h, rows, 0, cols, 0, 0, cols)])])
    ro = Layout(cat, [RankLayout([Local("x", "bf16", 1, cols, rows)], [Placement(0, 0, rows, 0, cols, 0, 0, rows, 1)])])
    tr, ro = to_wb(tr), to_wb(ro)
    assert wb.Plan(tr, ro, wb.RECEIVER, 0).launch_grid(4)[0] > 0
    _compare_layouts(f"transposed {rows}x{cols}", tr, ro, 0, "bf16", 0, 4)


def test_noalloc_refuses_tables_beyond_the_array():
    # the DeepSeek-V3 receiver in one round needs ~72 MB of tables: refused
    # before its (null) pointers are looked at; in 4 GiB rounds it fits
    w = WORKLOADS["dsv3_ep64_to_ep8_fp8"]
    tr, ro = _layouts(w)
    p = wb.Plan(tr, ro, wb.RECEIVER, 0)
    assert p.workspace_bytes > (32 << 20)
    ptrs = (wb.c_void_p * p.num_local_tensors)()
    rc = wb.lib.wb_unpack_round_noalloc(p._h, 0, None, ptrs, None)
    assert rc == wb.WB_ESIZE, wb.lib.wb_last_error().decode()
    assert "round budget" in wb.lib.wb_last_error().decode()
    q = wb.Plan(tr, ro, wb.RECEIVER, 0, round_budget=4 << 30)
    assert q.num_rounds > 1
    rc = wb.lib.wb_unpack_round_noalloc(q._h, 0, None, ptrs, None)
    assert rc == wb.WB_EINVAL and "null" in wb.lib.wb_last_error().decode()
