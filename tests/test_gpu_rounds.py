"""Round-based transfer on the GPU (Sec. 3.2; App. D): every round's pack
output equals the oracle's pack of that round, byte for byte; the receiver
assembles round after round from two alternating receive buffers (double
buffering); the final rollout tensors equal the oracle's expectation. At full
size the Llama-3-8B and DeepSeek-V3 workloads run in 4 GiB rounds and are
checked in full against torch."""

import numpy as np
import pytest
import torch

import paper_2609_25442_amd as wb
import synthetic_checkpoint as sc
from oracle.layout import layout_from_spec
from oracle.plan import build_plan
from oracle.transfer import expected_rollout, materialize
from oracle.transfer import pack as o_pack
from synthetic_checkpoint.workloads import ORDER, WORKLOADS, scaled

from gpu_util import FILL, codes_to_gpu, gpu_to_codes, say, workspace_for

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("name", ORDER)
def test_scaled_rounds_parity(name):
    w = scaled(name)
    otr = layout_from_spec(w["model"], w["trainer"])
    oro = layout_from_spec(w["model"], w["rollout"])
    dt = w["trainer"]["dtype"]
    total = sum(g.nbytes for g in build_plan(otr, oro).segments)
    budget = max(4096, total // (4 * oro.nranks))
    oplan = build_plan(otr, oro, round_budget=budget)
    nr = len(oplan.rounds)
    assert nr > 2
    tr = wb.Layout.describe(w["model"], w["trainer"])
    ro = wb.Layout.describe(w["model"], w["rollout"])
    cache = {}

    def vals(t):
        if t not in cache:
            c = otr.catalog[t]
            cache[t] = sc.values_numpy(t, np.arange(c.numel), dt).reshape(c.rows, c.cols)
        return cache[t]

    splans, srcs, o_locals = {}, {}, {}
    for s in range(otr.nranks):
        p = wb.Plan(tr, ro, wb.SENDER, s, round_budget=budget)
        assert p.num_rounds == nr
        ws = workspace_for(p)
        p.upload(ws)
        o_locals[s] = materialize(otr, s, vals)
        srcs[s] = [codes_to_gpu(c, lc.dtype) for c, lc in zip(o_locals[s], otr.ranks[s].locals)]
        splans[s] = (p, ws)
    for d in range(oro.nranks):
        rp = wb.Plan(tr, ro, wb.RECEIVER, d, round_budget=budget)
        rws = workspace_for(rp)
        rp.upload(rws)
        recv = [torch.empty(max(1, rp.buffer_bytes), dtype=torch.uint8, device="cuda") for _ in range(2)]
        dst = wb.allocate_locals(ro, d)
        for t in dst:
            t.view(torch.uint8).fill_(0x7F)
        for k in range(nr):
            say(f"[rounds {name}] receiver {d} round {k}/{nr}")
            buf = recv[k % 2]
            for s in range(otr.nranks):
                so, ro_off, nb = rp.round_region(k, s, d)
                if not nb:
                    continue
                p, _ = splans[s]
                send = torch.full((max(1, p.round_buffer_bytes(k)),), FILL, dtype=torch.uint8, device="cuda")
                p.pack_round(k, srcs[s], send)
                torch.cuda.synchronize()
                if d == 0:
                    want = o_pack(oplan, s, o_locals[s], k)
                    got = send.cpu().numpy()[:len(want)]
                    for g in oplan.segments:
                        if g.s == s and g.round == k:
                            assert np.array_equal(got[g.send_off:g.send_off + g.nbytes],
                                                  want[g.send_off:g.send_off + g.nbytes]), (s, k)
                buf[ro_off:ro_off + nb] = send[so:so + nb]
            rp.unpack_round(k, buf, dst)
        torch.cuda.synchronize()
        want = expected_rollout(oro, d, vals, dt)
        for u, (t, e) in enumerate(zip(dst, want)):
            lc = oro.ranks[d].locals[u]
            assert np.array_equal(gpu_to_codes(t, lc.dtype), e), (d, lc.name)


@pytest.mark.timeout(900)
@pytest.mark.parametrize("name", ["llama3_8b_fsdp8_to_tp1", "dsv3_ep64_to_ep8_fp8"])
def test_full_size_rounds(name):
    """4 GiB rounds at full size: every round's receive buffer is filled by the
    senders' round packs, then assembled round by round into the same
    rollout tensors; checked in full against torch."""
    from test_gpu_full import SENTINEL, _check_unpack_full, _sender_locals

    w = WORKLOADS[name]
    budget = 4 << 30
    dt = w["trainer"]["dtype"]
    d = w["unpack_rank"]
    otr = layout_from_spec(w["model"], w["trainer"])
    oro = layout_from_spec(w["model"], w["rollout"])
    tr = wb.Layout.describe(w["model"], w["trainer"])
    ro = wb.Layout.describe(w["model"], w["rollout"])
    rp = wb.Plan(tr, ro, wb.RECEIVER, d, round_budget=budget)
    rws = workspace_for(rp)
    rp.upload(rws)
    nr = rp.num_rounds
    assert nr > 1 and rp.buffer_bytes <= budget
    recv = [torch.empty(max(1, rp.round_buffer_bytes(k)), dtype=torch.uint8, device="cuda") for k in range(nr)]
    senders = [s for s in range(otr.nranks) if any(rp.round_region(k, s, d)[2] for k in range(nr))]
    say(f"[{name}] {nr} rounds of at most {budget >> 30} GiB, {len(senders)} senders")
    for g0 in range(0, len(senders), 16):
        group = senders[g0:g0 + 16]
        say(f"[{name}] senders {group[0]}..{group[-1]}")
        for s in group:
            locs = _sender_locals(otr, s, dt)
            p = wb.Plan(tr, ro, wb.SENDER, s, round_budget=budget)
            ws = workspace_for(p)
            p.upload(ws)
            send = torch.empty(max(1, p.buffer_bytes), dtype=torch.uint8, device="cuda")
            for k in range(nr):
                so, ro_off, nb = rp.round_region(k, s, d)
                if nb:
                    p.pack_round(k, locs, send)
                    recv[k][ro_off:ro_off + nb] = send[so:so + nb]
            torch.cuda.synchronize()
            del locs, send, p, ws
    dst = wb.allocate_locals(ro, d)
    for t, lc in zip(dst, oro.ranks[d].locals):
        t.view(torch.uint8).fill_(SENTINEL[lc.dtype])
    for k in range(nr):
        rp.unpack_round(k, recv[k], dst)
    torch.cuda.synchronize()
    say(f"[{name}] full check")
    _check_unpack_full(oro, d, dst, otr.catalog, dt)


@pytest.mark.parametrize("name", ["llama3_8b_fsdp8_to_tp1", "mixtral_ep8fsdp2_to_ep2", "dsv3_ep64_to_ep8_fp8"])
def test_two_stream_pipeline(name):
    """Depth-2 pipeline (Sec. 3.2 rounds; the two-buffer design of Sec. 4.6): the packs of
    round k+1 run on one stream while the receiver's stream moves round k's
    regions out of the senders' send buffers and assembles round k. Each sender
    alternates between two send buffers and the receiver between two receive
    buffers; events order only what the buffers require. The rollout tensors
    must equal the oracle's expectation."""
    w = scaled(name)
    otr = layout_from_spec(w["model"], w["trainer"])
    oro = layout_from_spec(w["model"], w["rollout"])
    dt = w["trainer"]["dtype"]
    d = w["unpack_rank"]
    total = sum(g.nbytes for g in build_plan(otr, oro).segments if g.d == d)
    budget = max(4096, total // 6)
    tr = wb.Layout.describe(w["model"], w["trainer"])
    ro = wb.Layout.describe(w["model"], w["rollout"])
    rp = wb.Plan(tr, ro, wb.RECEIVER, d, round_budget=budget)
    rws = workspace_for(rp)
    rp.upload(rws)
    nr = rp.num_rounds
    assert nr > 3
    cache = {}

    def vals(t):
        if t not in cache:
            c = otr.catalog[t]
            cache[t] = sc.values_numpy(t, np.arange(c.numel), dt).reshape(c.rows, c.cols)
        return cache[t]

    senders = [s for s in range(otr.nranks) if any(rp.round_region(k, s, d)[2] for k in range(nr))]
    keep = []
    plans, srcs, sends = {}, {}, {}
    for s in senders:
        p = wb.Plan(tr, ro, wb.SENDER, s, round_budget=budget)
        ws = workspace_for(p)
        p.upload(ws)
        keep.append(ws)
        plans[s] = p
        srcs[s] = [codes_to_gpu(c, lc.dtype) for c, lc in zip(materialize(otr, s, vals), otr.ranks[s].locals)]
        sends[s] = [torch.full((max(1, p.buffer_bytes),), FILL, dtype=torch.uint8, device="cuda") for _ in range(2)]
    recv = [torch.full((max(1, rp.buffer_bytes),), FILL, dtype=torch.uint8, device="cuda") for _ in range(2)]
    dst = wb.allocate_locals(ro, d)
    for t in dst:
        t.view(torch.uint8).fill_(0x7F)
    torch.cuda.synchronize()
    P, U = torch.cuda.Stream(), torch.cuda.Stream()
    packed = [torch.cuda.Event() for _ in range(nr)]
    moved = [torch.cuda.Event() for _ in range(nr)]
    say(f"[pipeline {name}] {nr} rounds, {len(senders)} senders")
    for k in range(nr):
        if k >= 2:
            P.wait_event(moved[k - 2])          # send buffers k % 2 drained
        for s in senders:
            if rp.round_region(k, s, d)[2]:
                plans[s].pack_round(k, srcs[s], sends[s][k % 2], P)
        packed[k].record(P)
        U.wait_event(packed[k])
        with torch.cuda.stream(U):              # the network stand-in, then assembly
            for s in senders:
                so, roff, nb = rp.round_region(k, s, d)
                if nb:
                    recv[k % 2][roff:roff + nb].copy_(sends[s][k % 2][so:so + nb])
        moved[k].record(U)
        rp.unpack_round(k, recv[k % 2], dst, U)
    torch.cuda.synchronize()
    want = expected_rollout(oro, d, vals, dt)
    for u, (t, e) in enumerate(zip(dst, want)):
        lc = oro.ranks[d].locals[u]
        assert np.array_equal(gpu_to_codes(t, lc.dtype), e), (d, lc.name)
