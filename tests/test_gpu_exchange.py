"""Three-stage transfer on the GPU (Sec. 3.2; Figure 5): trainer packs, the
receive stage, the forward packings of the external and internal exchanges
(wb_forward_round) and assembly, all through the C ABI. Every forward buffer
and every receive buffer equals the oracle's byte for byte where the plan puts
payloads, and every rollout tensor equals the plan-free expectation."""

import numpy as np
import pytest
import torch

import paper_2609_25442_amd as wb
import synthetic_checkpoint as sc
from oracle.layout import describe_layout, layout_from_spec
from oracle.plan import build_plan
from oracle.transfer import expected_rollout, forward, materialize, network
from oracle.transfer import pack as o_pack
from synthetic_checkpoint.workloads import ORDER, scaled

from gpu_util import FILL, codes_to_gpu, gpu_to_codes, say, workspace_for
from oracle_cases import random_medium_model, random_model, random_par
from wb_cases import to_wb

pytestmark = pytest.mark.gpu


def _payload_mask(n, spans):
    m = np.zeros(n, dtype=bool)
    for a, b in spans:
        m[a:b] = True
    return m


def three_stage(otr, oro, values, G, budget=0, tr=None, ro=None, label=""):
    tr = tr or to_wb(otr)
    ro = ro or to_wb(oro)
    oplan = build_plan(otr, oro, round_budget=budget, node_size=G)
    nr = len(oplan.rounds)
    ns, nd = otr.nranks, oro.nranks
    keep = []
    splans, srcs, o_locals = {}, {}, {}
    for s in range(ns):
        p = wb.Plan(tr, ro, wb.SENDER, s, round_budget=budget, node_size=G)
        ws = workspace_for(p)
        p.upload(ws)
        keep.append(ws)
        splans[s] = p
        o_locals[s] = materialize(otr, s, values)
        srcs[s] = [codes_to_gpu(c, lc.dtype) for c, lc in zip(o_locals[s], otr.ranks[s].locals)]
    rplans, dsts = {}, {}
    for d in range(nd):
        p = wb.Plan(tr, ro, wb.RECEIVER, d, round_budget=budget, node_size=G)
        assert p.num_rounds == nr and p.node_size == G
        ws = workspace_for(p)
        p.upload(ws)
        keep.append(ws)
        rplans[d] = p
        dsts[d] = wb.allocate_locals(ro, d)
        for t in dsts[d]:
            t.view(torch.uint8).fill_(0x7F)
    for k in range(nr):
        say(f"[{label}] round {k}/{nr}")
        sends = {}
        o_sends = {s: o_pack(oplan, s, o_locals[s], k) for s in range(ns)}
        for s in range(ns):
            sends[s] = torch.full((max(1, splans[s].round_buffer_bytes(k)),), FILL, dtype=torch.uint8, device="cuda")
            splans[s].pack_round(k, srcs[s], sends[s])
        recv = {d: torch.full((max(1, rplans[d].round_buffer_bytes(k)),), FILL, dtype=torch.uint8, device="cuda")
                for d in range(nd)}
        o_recv = {d: network(oplan, d, o_sends, k) for d in range(nd)}
        for d in range(nd):
            for s in range(ns):
                so, roff, nb = rplans[d].stage_region(k, 0, s, d)
                if nb:
                    recv[d][roff:roff + nb] = sends[s][so:so + nb]
        for stage in (1, 2):
            fwd, o_fwd = {}, {}
            for r in range(nd):
                nbytes = rplans[r].forward_bytes(stage, k)
                fwd[r] = torch.full((max(1, nbytes),), FILL, dtype=torch.uint8, device="cuda")
                rplans[r].forward_round(k, stage, recv[r], fwd[r])
                o_fwd[r] = forward(oplan, r, o_recv[r], stage, k)
            torch.cuda.synchronize()
            for r in range(nd):
                got = fwd[r].cpu().numpy()[:len(o_fwd[r])]
                spans = [(g.send_off, g.send_off + g.nbytes) for g in oplan.segments
                         if g.round == k and g.stage == stage and g.s == r]
                m = _payload_mask(len(o_fwd[r]), spans)
                assert np.array_equal(got[m], o_fwd[r][m]), (label, k, stage, r)
            for d in range(nd):
                network(oplan, d, o_fwd, k, stage, into=o_recv[d])
                for r in range(nd):
                    so, roff, nb = rplans[d].stage_region(k, stage, r, d)
                    if nb:
                        recv[d][roff:roff + nb] = fwd[r][so:so + nb]
        torch.cuda.synchronize()
        for d in range(nd):
            got = recv[d].cpu().numpy()[:len(o_recv[d])]
            spans = [(g.recv_off, g.recv_off + g.nbytes) for g in oplan.segments if g.round == k and g.d == d]
            m = _payload_mask(len(o_recv[d]), spans)
            assert np.array_equal(got[m], o_recv[d][m]), (label, k, d)
            rplans[d].unpack_round(k, recv[d], dsts[d])
        torch.cuda.synchronize()
    src_dtype = otr.ranks[0].locals[0].dtype
    for d in range(nd):
        want = expected_rollout(oro, d, values, src_dtype)
        for t, e, lc in zip(dsts[d], want, oro.ranks[d].locals):
            assert np.array_equal(gpu_to_codes(t, lc.dtype), e), (label, d, lc.name)
    return oplan


def _values(otr):
    dt = otr.ranks[0].locals[0].dtype
    cache = {}

    def vals(t):
        if t not in cache:
            c = otr.catalog[t]
            cache[t] = sc.values_numpy(t, np.arange(c.numel), dt).reshape(c.rows, c.cols)
        return cache[t]
    return vals


@pytest.mark.parametrize("name", ORDER)
def test_scaled_workloads_three_stage(name):
    w = scaled(name)
    otr = layout_from_spec(w["model"], w["trainer"])
    oro = layout_from_spec(w["model"], w["rollout"])
    tr = wb.Layout.describe(w["model"], w["trainer"])
    ro = wb.Layout.describe(w["model"], w["rollout"])
    for G in sorted({1, max(1, oro.nranks // 2)}):
        plan = three_stage(otr, oro, _values(otr), G, tr=tr, ro=ro, label=f"{name} G={G}")
        assert any(g.stage for g in plan.segments) == (oro.nranks > 1)


@pytest.mark.parametrize("seed", range(10))
def test_random_three_stage(seed):
    rng = np.random.default_rng(2700 + seed)
    m = random_model(rng)
    otr = describe_layout(m, random_par(rng, m, "trainer"))
    oro = describe_layout(m, random_par(rng, m, "rollout"))
    G = int(rng.integers(1, oro.nranks + 1))
    budget = int(rng.choice([0, 400]))
    three_stage(otr, oro, _values(otr), G, budget, label=f"random {seed} G={G} budget={budget}")


@pytest.mark.parametrize("seed", range(8))
def test_random_medium_three_stage(seed):
    """The same on random models with hidden sizes of 128 to 384 (vector work
    items, transposed slabs, fp8 blocks of 64 and 128), in one round or in 1 MiB
    rounds."""
    rng = np.random.default_rng(2900 + seed)
    m = random_medium_model(rng)
    otr = describe_layout(m, random_par(rng, m, "trainer"))
    oro = describe_layout(m, random_par(rng, m, "rollout", blocks=(64, 128)))
    G = int(rng.integers(1, oro.nranks + 1))
    budget = int(rng.choice([0, 1 << 20]))
    three_stage(otr, oro, _values(otr), G, budget, label=f"random-medium {seed} G={G} budget={budget}")


def test_figure5_dp4_three_stage():
    """TP2 trainer, four DP rollout workers on two nodes of two."""
    from oracle.catalog import ModelShapes
    from oracle.layout import Parallelism

    m = ModelShapes("dense", num_layers=2, hidden=64, num_heads=4, num_kv_heads=2, head_dim=16, ffn=128, vocab=96)
    otr = describe_layout(m, Parallelism("megatron", "bf16", tp=2, transposed_row_parallel=True))
    oro = describe_layout(m, Parallelism("serving", "bf16", tp=1, dp=4))
    plan = three_stage(otr, oro, _values(otr), 2, label="figure 5")
    assert {g.stage for g in plan.segments} == {0, 1, 2}


@pytest.mark.timeout(900)
@pytest.mark.parametrize("name,G", [("mixtral_ep8fsdp2_to_ep2", 1), ("dsv3_ep64_to_ep8_fp8", 4),
                                    ("llama3_8b_tp4_to_tp2", 1)])
def test_full_size_three_stage(name, G):
    """Full size, in the benchmark's configuration for the exchange stages: the
    unpack rank's receive buffer holds its stage-0 regions and the payloads
    forwarded to it (each the bytes its origin segment left a trainer with);
    its forward packings must copy exactly the bytes they forward, and its
    tensors, assembled from all three sections, are checked in full against
    torch and sampled against the oracle."""
    from synthetic_checkpoint.workloads import WORKLOADS
    from test_gpu_full import SENTINEL, _check_unpack_full, _check_unpack_sampled, _sender_locals

    w = WORKLOADS[name]
    dt = w["trainer"]["dtype"]
    d = w["unpack_rank"]
    otr = layout_from_spec(w["model"], w["trainer"])
    oro = layout_from_spec(w["model"], w["rollout"])
    tr = wb.Layout.describe(w["model"], w["trainer"])
    ro = wb.Layout.describe(w["model"], w["rollout"])
    rp = wb.Plan(tr, ro, wb.RECEIVER, d, node_size=G)
    rws = workspace_for(rp)
    rp.upload(rws)
    segs = rp.segments()
    forwarded = {}
    for f in segs:
        if f["stage"] and f["receiver"] == d:
            o = segs[f["origin"]]
            forwarded.setdefault(o["sender"], []).append((o, f))
    assert forwarded, "the unpack rank must receive forwarded payloads"
    recv = torch.full((rp.buffer_bytes,), FILL, dtype=torch.uint8, device="cuda")
    say(f"[{name} G={G}] receive buffer {rp.buffer_bytes / 1e9:.2f} GB, "
        f"{sum(len(v) for v in forwarded.values())} forwarded payloads")
    for s in range(otr.nranks):
        so, roff, nb = rp.region(s, d)
        if not nb and s not in forwarded:
            continue
        locs = _sender_locals(otr, s, dt)
        p = wb.Plan(tr, ro, wb.SENDER, s, node_size=G)
        ws = workspace_for(p)
        p.upload(ws)
        send = torch.empty(max(1, p.buffer_bytes), dtype=torch.uint8, device="cuda")
        p.pack(locs, send)
        if nb:
            recv[roff:roff + nb] = send[so:so + nb]
        for o, f in forwarded.get(s, []):
            recv[f["recv_offset"]:f["recv_offset"] + f["bytes"]] = send[o["send_offset"]:o["send_offset"] + o["bytes"]]
        torch.cuda.synchronize()
        del locs, send, p, ws
    for st in (1, 2):
        fwd = torch.full((max(1, rp.forward_bytes(st)),), FILL, dtype=torch.uint8, device="cuda")
        rp.forward_round(0, st, recv, fwd)
        torch.cuda.synchronize()
        mine = [f for f in segs if f["stage"] == st and f["sender"] == d]
        say(f"[{name} G={G}] stage {st}: {len(mine)} forwarded payloads checked")
        for f in mine:
            a = fwd[f["send_offset"]:f["send_offset"] + f["bytes"]]
            b = recv[f["src_offset"]:f["src_offset"] + f["bytes"]]
            assert torch.equal(a, b), (st, f)
        del fwd
    dst = wb.allocate_locals(ro, d)
    for t, lc in zip(dst, oro.ranks[d].locals):
        t.view(torch.uint8).fill_(SENTINEL[lc.dtype])
    rp.unpack(recv, dst)
    torch.cuda.synchronize()
    say(f"[{name} G={G}] full check against torch")
    _check_unpack_full(oro, d, dst, otr.catalog, dt)
    _check_unpack_sampled(oro, d, dst, otr.catalog, dt, np.random.default_rng(12))
    del recv, dst
    torch.cuda.empty_cache()
