"""The local-tensor pointer tables of a plan on the GPU: a plan keeps the
device tables of its last four pointer sets. Alternating sets must not block
the host, and a table refilled for a new set on one stream must not change
under work on another stream that still reads it (nor be read before its copy
has landed). Checked on the full-size Llama-3-8B FSDP8 -> TP1 receiver, whose
unpack takes milliseconds, so that work on two streams overlaps."""

import time

import pytest
import torch

import paper_2609_25442_amd as wb
from synthetic_checkpoint.workloads import WORKLOADS

from gpu_util import say, workspace_for

pytestmark = pytest.mark.gpu

W = WORKLOADS["llama3_8b_fsdp8_to_tp1"]


def _receiver():
    tr = wb.Layout.describe(W["model"], W["trainer"])
    ro = wb.Layout.describe(W["model"], W["rollout"])
    d = W["unpack_rank"]
    rp = wb.Plan(tr, ro, wb.RECEIVER, d)
    ws = workspace_for(rp)
    rp.upload(ws)
    # any bytes will do: every rollout tensor is a bf16 copy of wire bytes
    recv = torch.randint(0, 256, (rp.buffer_bytes,), dtype=torch.uint8, device="cuda")
    ref = wb.allocate_locals(ro, d)
    rp.unpack(recv, ref)
    torch.cuda.synchronize()
    return rp, ws, ro, d, recv, ref


def _fill(sets, value):
    for t in sets:
        t.view(torch.uint8).fill_(value)


def _same(a, b):
    return all(torch.equal(x.view(torch.uint8), y.view(torch.uint8)) for x, y in zip(a, b))


@pytest.mark.timeout(300)
def test_pointer_tables_across_streams():
    rp, ws, ro, d, recv, ref = _receiver()
    sets = [wb.allocate_locals(ro, d) for _ in range(5)]
    A, B = torch.cuda.Stream(), torch.cuda.Stream()
    torch.cuda.synchronize()
    say("[tables] stream A refills and unpacks set 0 ten times; stream B meanwhile takes sets 1-4")
    # B's fourth new set refills the table of set 0 (the least recently
    # staged); the library must make B wait for A's unpacks that read it.
    # Were the table rewritten under them, A's last unpacks would write set 4
    # and leave set 0 as filled.
    with torch.cuda.stream(A):
        for _ in range(10):
            _fill(sets[0], 0x7F)
            rp.unpack(recv, sets[0], A)
    with torch.cuda.stream(B):
        for j in range(1, 5):
            _fill(sets[j], 0x7F)
            rp.unpack(recv, sets[j], B)
    torch.cuda.synchronize()
    for j, s in enumerate(sets):
        assert _same(s, ref), j
    say("[tables] back to set 0 on stream B, then set 1 on stream A (tables reused across streams)")
    _fill(sets[0], 0x11)
    _fill(sets[1], 0x22)
    torch.cuda.synchronize()
    with torch.cuda.stream(B):
        rp.unpack(recv, sets[0], B)
    with torch.cuda.stream(A):
        rp.unpack(recv, sets[1], A)
    torch.cuda.synchronize()
    assert _same(sets[0], ref) and _same(sets[1], ref)


@pytest.mark.timeout(300)
def test_alternating_pointer_sets_do_not_block_the_host():
    rp, ws, ro, d, recv, ref = _receiver()
    sets = [wb.allocate_locals(ro, d) for _ in range(2)]
    rp.unpack(recv, sets[0])
    rp.unpack(recv, sets[1])
    torch.cuda.synchronize()
    n = 12
    t0 = time.perf_counter()
    for i in range(n):
        rp.unpack(recv, sets[i % 2])
    t1 = time.perf_counter()
    torch.cuda.synchronize()
    t2 = time.perf_counter()
    say(f"[tables] {n} alternating unpacks: enqueued in {1e3 * (t1 - t0):.1f} ms, ran in {1e3 * (t2 - t0):.1f} ms")
    # each unpack moves 32 GB (about 5 ms); enqueueing must not wait for them
    assert (t1 - t0) < 0.25 * (t2 - t0)
    assert _same(sets[0], ref) and _same(sets[1], ref)
