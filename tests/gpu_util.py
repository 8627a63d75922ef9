"""Helpers of the GPU tests: moving raw codes between numpy and torch, and
driving pack -> network -> unpack through the C ABI against the oracle."""

from __future__ import annotations

import sys

import numpy as np
import torch

import paper_2609_25442_amd as wb
from oracle.plan import build_plan
from oracle.transfer import CODE_DTYPE, expected_rollout, materialize
from oracle.transfer import network as o_network
from oracle.transfer import pack as o_pack

SIGNED = {"f32": (np.int32, torch.int32), "bf16": (np.int16, torch.int16), "f8e4m3": (np.uint8, torch.uint8)}
FILL = 0x5A


def say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


def codes_to_gpu(codes: np.ndarray, dtype: str, device="cuda") -> torch.Tensor:
    np_t, t_t = SIGNED[dtype]
    t = torch.from_numpy(np.ascontiguousarray(codes).view(np_t)).to(device)
    return t.view(wb.torch_dtype(dtype)) if dtype != "f8e4m3" else t.view(torch.float8_e4m3fn)


def gpu_to_codes(t: torch.Tensor, dtype: str) -> np.ndarray:
    np_t, t_t = SIGNED[dtype]
    return t.reshape(-1).view(t_t).cpu().numpy().view(CODE_DTYPE[dtype])


def workspace_for(plan: "wb.Plan") -> torch.Tensor:
    return torch.empty(max(256, plan.workspace_bytes), dtype=torch.uint8, device="cuda")


def _buffer(nbytes, fill, staged):
    """A send or receive buffer in device memory, or in pinned host memory
    that the kernels reach over PCIe (the host-staged modes)."""
    if staged:
        return torch.full((max(1, nbytes),), fill, dtype=torch.uint8, pin_memory=True)
    return torch.full((max(1, nbytes),), fill, dtype=torch.uint8, device="cuda")


def roundtrip(otr, oro, values, tr=None, ro=None, label="", staged=False):
    """Pack every trainer rank and unpack every rollout rank on the GPU through
    the C ABI; compare every payload byte with the oracle's pack, check that
    padding between payloads is untouched, and compare every rollout tensor
    with the oracle's plan-free expectation. ``staged`` puts buffers in pinned
    host memory: "send" the send buffers (sender staging), "recv" the receive
    buffers (receiver staging), True both."""
    stage_send = staged in (True, "send")
    stage_recv = staged in (True, "recv")
    from wb_cases import to_wb

    tr = tr or to_wb(otr)
    ro = ro or to_wb(oro)
    oplan = build_plan(otr, oro)
    src_dtype = otr.ranks[0].locals[0].dtype
    sends = {}
    o_sends = {}
    for s in range(otr.nranks):
        say(f"[{label}] pack sender {s}")
        o_locals = materialize(otr, s, values)
        o_sends[s] = o_pack(oplan, s, o_locals)
        p = wb.Plan(tr, ro, wb.SENDER, s)
        ws = workspace_for(p)
        p.upload(ws)
        src = [codes_to_gpu(c, lc.dtype) for c, lc in zip(o_locals, otr.ranks[s].locals)]
        buf = _buffer(p.buffer_bytes, FILL, stage_send)
        p.pack(src, buf)
        torch.cuda.synchronize()
        got = buf.cpu().numpy()[:p.buffer_bytes]
        want = o_sends[s]
        mask = np.zeros(len(want), dtype=bool)
        for g in oplan.segments:
            if g.s == s:
                mask[g.send_off:g.send_off + g.nbytes] = True
        assert np.array_equal(got[mask], want[mask]), f"{label}: pack payload of sender {s}"
        assert np.all(got[~mask] == FILL), f"{label}: pack wrote outside payloads of sender {s}"
        sends[s] = buf
    for d in range(oro.nranks):
        say(f"[{label}] unpack receiver {d}")
        p = wb.Plan(tr, ro, wb.RECEIVER, d)
        ws = workspace_for(p)
        p.upload(ws)
        recv = _buffer(p.buffer_bytes, 0, stage_recv)
        for s in range(otr.nranks):
            so, ro_off, nb = p.region(s, d)
            if nb:
                recv[ro_off:ro_off + nb] = sends[s][so:so + nb]
        # the network stand-in gives the same bytes as the oracle's
        o_recv = o_network(oplan, d, o_sends)
        got_recv = recv.cpu().numpy()[:p.buffer_bytes]
        for g in oplan.segments:
            if g.d == d:
                assert np.array_equal(got_recv[g.recv_off:g.recv_off + g.nbytes], o_recv[g.recv_off:g.recv_off + g.nbytes])
        dst = wb.allocate_locals(ro, d)
        for t in dst:
            t.view(torch.uint8).fill_(0x7F)
        p.unpack(recv, dst)
        torch.cuda.synchronize()
        want = expected_rollout(oro, d, values, src_dtype)
        for u, (t, e) in enumerate(zip(dst, want)):
            lc = oro.ranks[d].locals[u]
            got = gpu_to_codes(t, lc.dtype)
            if not np.array_equal(got, e):
                bad = np.nonzero(got != e)[0]
                raise AssertionError(f"{label}: receiver {d} tensor {lc.name}: {len(bad)} mismatches, first at {bad[:5]}: "
                                     f"got {got[bad[:5]]} want {e[bad[:5]]}")
    return oplan
