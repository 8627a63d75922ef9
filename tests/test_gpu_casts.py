"""Exhaustive cast domains through wb_unpack on the GPU.

* fp32 -> bf16: all 2^32 fp32 bit patterns through the assembly kernel,
  against torch's own conversion on the GPU, and the rounding-relevant
  structured set against the oracle;
* bf16 -> fp8 E4M3FN with a block scale: every pair (x, amax) of bf16 values
  with |x| <= amax (amax > 0), i.e. every quantiser input the workloads can
  produce, against torch's formula (amax / 448, x / s, E4M3FN cast) on the
  GPU, plus all-zero blocks; a sample of blocks against the oracle.
"""

import numpy as np
import pytest
import torch

import paper_2609_25442_amd as wb
from oracle import casts

from gpu_util import say, workspace_for

pytestmark = pytest.mark.gpu


def _one_tensor_plan(rows, cols, sdt, ddt, block=0):
    tr = wb.Layout.create([("X", rows, cols)], 1)
    tr.add_local(0, "x", sdt, 1, rows, cols)
    tr.add_placement(0, 0, 0, rows, 0, cols, 0, 0, cols)
    ro = wb.Layout.create([("X", rows, cols)], 1)
    ro.add_local(0, "y", ddt, 1, rows, cols, block)
    ro.add_placement(0, 0, 0, rows, 0, cols, 0, 0, cols)
    p = wb.Plan(tr, ro, wb.RECEIVER, 0)
    assert p.region(0, 0)[1] == 0  # the single payload starts the receive buffer
    ws = workspace_for(p)
    p.upload(ws)
    return p, ws


def test_f32_to_bf16_all_patterns():
    rows, cols = 1 << 16, 4096          # 2^28 patterns per launch
    p, ws = _one_tensor_plan(rows, cols, "f32", "bf16")
    dst = torch.empty(rows, cols, dtype=torch.bfloat16, device="cuda")
    step = rows * cols
    for k in range((1 << 32) // step):
        if k % 4 == 0:
            say(f"f32->bf16 patterns from {k * step:#x}")
        x = torch.arange(k * step, (k + 1) * step, dtype=torch.int64, device="cuda").to(torch.int32)
        recv = x.view(torch.float32)
        p.unpack(recv, [dst])
        ref = recv.to(torch.bfloat16)
        same = (dst.view(-1).view(torch.int16) == ref.view(torch.int16)) | (torch.isnan(dst.view(-1)) & torch.isnan(ref))
        assert bool(same.all()), f"mismatch in chunk {k}"
        del x, recv, ref, same
    torch.cuda.synchronize()


def test_f32_to_bf16_structured_vs_oracle():
    hi = np.arange(1 << 16, dtype=np.uint32) << 16
    lows = np.array([0, 1, 0x7FFF, 0x8000, 0x8001, 0xFFFF, 0x4000, 0xC000], dtype=np.uint32)
    u = (hi[:, None] | lows[None, :]).ravel()
    u = u[(u & 0x7F800000) != 0x7F800000]
    cols = 512
    n = len(u) // cols * cols
    u = u[:n]
    p, ws = _one_tensor_plan(n // cols, cols, "f32", "bf16")
    recv = torch.from_numpy(u.view(np.int32)).cuda().view(torch.float32)
    dst = torch.empty(n // cols, cols, dtype=torch.bfloat16, device="cuda")
    p.unpack(recv, [dst])
    got = dst.view(-1).view(torch.int16).cpu().numpy().view(np.uint16)
    assert np.array_equal(got, casts.f32_to_bf16(u))


def test_bf16_to_f32_all_codes():
    p, ws = _one_tensor_plan(64, 1024, "bf16", "f32")
    codes = torch.arange(0, 1 << 16, dtype=torch.int32, device="cuda").to(torch.int16)
    dst = torch.empty(64, 1024, dtype=torch.float32, device="cuda")
    p.unpack(codes.view(torch.bfloat16), [dst])
    want = (codes.to(torch.int32) & 0xFFFF) << 16
    assert torch.equal(dst.view(-1).view(torch.int32), want)


def _domain_chunk(a0, a1):
    """Blocks of 16384 bf16 codes: for each amax code a in [a0, a1), four blocks
    holding every code c with |c| <= a (others zero) and +a, rotated."""
    a = torch.arange(a0, a1, dtype=torch.int32, device="cuda")
    c = torch.arange(0, 1 << 16, dtype=torch.int32, device="cuda")
    keep = (c & 0x7FFF)[None, :] <= a[:, None]
    x = torch.where(keep, c[None, :], torch.zeros_like(c)[None, :])
    x = x.view(-1, 16384)
    x[:, 0] = a.repeat_interleave(4)
    # rotate each block by its own offset, so that the amax (and every other
    # code) sits at a different row, column, lane and word from block to block
    nb = x.shape[0]
    shift = (torch.arange(nb, device="cuda") * 4099 + a0 * 61) % 16384
    idx = (torch.arange(16384, device="cuda")[None, :] + shift[:, None]) % 16384
    x = torch.gather(x, 1, idx)
    return x.to(torch.int16).view(torch.bfloat16).reshape(-1, 128)


def _split_fp8_plan(rows, split):
    """rows x 128 bf16 held by `split` trainer ranks, one column slab each, so
    every 128 x 128 destination block is filled from `split` wire pieces (the
    fp8 kernel's general path; one piece takes its single-piece path)."""
    if split == 1:
        p, ws = _one_tensor_plan(rows, 128, "bf16", "f8e4m3", block=128)
        return p, ws, lambda x: x
    w = 128 // split
    tr = wb.Layout.create([("X", rows, 128)], split)
    for r in range(split):
        tr.add_local(r, "x", "bf16", 1, rows, w)
        tr.add_placement(r, 0, 0, rows, r * w, (r + 1) * w, 0, 0, w)
    ro = wb.Layout.create([("X", rows, 128)], 1)
    ro.add_local(0, "y", "f8e4m3", 1, rows, 128, 128)
    ro.add_placement(0, 0, 0, rows, 0, 128, 0, 0, 128)
    p = wb.Plan(tr, ro, wb.RECEIVER, 0)
    ws = workspace_for(p)
    p.upload(ws)
    recv = torch.empty(p.buffer_bytes, dtype=torch.uint8, device="cuda")
    regions = [p.region(s, 0) for s in range(split)]

    def to_wire(x):
        for s, (_, off, nb) in enumerate(regions):
            assert nb == rows * w * 2
            recv[off:off + nb].view(torch.bfloat16).view(rows, w).copy_(x[:, s * w:(s + 1) * w])
        return recv

    return p, ws, to_wire


@pytest.mark.parametrize("split", [1, 2])
def test_fp8_quantiser_all_pairs(split):
    amax_max = 0x7F7F + 1
    per = 2048                                    # amax codes per launch -> 8192 blocks
    rows = per * 4 * 128
    p, ws, to_wire = _split_fp8_plan(rows, split)
    q = torch.empty(rows, 128, dtype=torch.float8_e4m3fn, device="cuda")
    s = torch.empty(rows // 128, 1, dtype=torch.float32, device="cuda")
    rng = np.random.default_rng(7)
    for a0 in range(1, amax_max, per):
        a1 = min(amax_max, a0 + per)
        if (a0 - 1) % (per * 4) == 0:
            say(f"fp8 pairs amax codes {a0:#x}..")
        x = _domain_chunk(a0, a1)
        if x.shape[0] < rows:
            x = torch.cat([x, torch.zeros(rows - x.shape[0], 128, dtype=torch.bfloat16, device="cuda")])
        p.unpack(to_wire(x), [q, s])
        xf = x.float().view(-1, 16384)
        amax = xf.abs().amax(dim=1)
        # divide by a tensor: torch turns division by a CPU scalar into a
        # multiplication by its reciprocal, which is not correctly rounded
        sref = torch.where(amax > 0, amax / torch.full_like(amax, 448.0), torch.ones_like(amax))
        qref = (xf / sref[:, None]).to(torch.float8_e4m3fn)
        se = s.view(-1).view(torch.int32) == sref.view(torch.int32)
        if not bool(se.all()):
            i = torch.nonzero(~se)[:4].view(-1)
            raise AssertionError(f"scales from amax {a0:#x}: blocks {i.tolist()} got {s.view(-1)[i].tolist()} "
                                 f"want {sref[i].tolist()} amax {amax[i].tolist()}")
        eq = q.view(-1, 16384).view(torch.uint8) == qref.view(torch.uint8)
        if not bool(eq.all()):
            bad = torch.nonzero(~eq)[:5].cpu().numpy()
            raise AssertionError(f"codes differ from amax {a0:#x}: first (block, elem) {bad}")
        # a few blocks straight against the oracle
        for b in rng.integers(0, (a1 - a0) * 4, 3):
            xb = x.view(-1, 16384)[b].view(torch.int16).cpu().numpy().view(np.uint16)
            codes, sc = casts.quantize_block(casts.bf16_to_f32(xb).view(np.float32))
            assert np.array_equal(q.view(-1, 16384)[b].view(torch.uint8).cpu().numpy(), codes)
            assert np.float32(s.view(-1)[b].item()) == sc
        del x, xf, amax, sref, qref, eq
    # all-zero blocks (scale 1) and signed zeros
    x = torch.zeros(rows, 128, dtype=torch.bfloat16, device="cuda")
    x.view(-1, 16384)[1::2] = -0.0
    p.unpack(to_wire(x), [q, s])
    assert bool((s == 1.0).all())
    qb = q.view(torch.uint8).view(-1, 16384)
    assert bool((qb[0::2] == 0).all()) and bool((qb[1::2] == 0x80).all())
