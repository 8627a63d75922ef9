"""The XCD-aware workgroup order at its edges: the copy/cast launches renumber
class-0 workgroups in runs of 8 x 1024 and the fp8 launch its full block pairs
in runs of 8 x 512, a shorter tail keeping the plain order. Launches just
below, at and past whole runs (and several runs plus a tail) must move every
element exactly as before: a bf16 copy and an fp32 -> bf16 cast of one tensor
(pack, then unpack of the packed payload) against the source and torch's
cast, and fp8 blocks of one [128, 128 nb] matrix against torch's blockwise
amax / 448, x / s, E4M3FN."""

import pytest
import torch

import paper_2609_25442_amd as wb

from gpu_util import say, workspace_for

pytestmark = pytest.mark.gpu


def _identity(rows, cols, dt_tr, dt_ro, block=0):
    cat = [("W", rows, cols)]
    tr = wb.Layout.create(cat, 1)
    u = tr.add_local(0, "W", dt_tr, 1, rows, cols)
    tr.add_placement(0, 0, 0, rows, 0, cols, u, 0, cols)
    ro = wb.Layout.create(cat, 1)
    v = ro.add_local(0, "W", dt_ro, 1, rows, cols, block)
    ro.add_placement(0, 0, 0, rows, 0, cols, v, 0, cols)
    return tr, ro


def _transfer(tr, ro, src):
    sp = wb.Plan(tr, ro, wb.SENDER, 0)
    rp = wb.Plan(tr, ro, wb.RECEIVER, 0)
    sws, rws = workspace_for(sp), workspace_for(rp)
    sp.upload(sws)
    rp.upload(rws)
    send = torch.zeros(max(1, sp.buffer_bytes), dtype=torch.uint8, device="cuda")
    sp.pack([src], send)
    so, roff, nb = rp.region(0, 0)
    recv = torch.zeros(max(1, rp.buffer_bytes), dtype=torch.uint8, device="cuda")
    recv[roff:roff + nb] = send[so:so + nb]
    dst = wb.allocate_locals(ro, 0)
    rp.unpack(recv, dst)
    torch.cuda.synchronize()
    gx, gy, _ = rp.launch_grid(0)
    return send[so:so + nb], dst, gx * max(gy, 1)


# 256 KiB work items: a bf16 copy item takes 256 one-KiB chunks (32 items per
# run of 8192 workgroups), an fp32 -> bf16 item 128 two-KiB chunks (64 items)
@pytest.mark.parametrize("items", [31, 32, 33, 64, 97])
def test_copy_runs_and_tails(items):
    rows, cols = items * 128, 1024                      # 256 KiB of bf16 per 128 rows
    g = torch.Generator(device="cuda").manual_seed(items)
    src = torch.randn(rows, cols, generator=g, device="cuda").to(torch.bfloat16)
    tr, ro = _identity(rows, cols, "bf16", "bf16")
    wire, dst, wgs = _transfer(tr, ro, src)
    say(f"[xcd] bf16 copy, {items} items, {wgs} workgroups ({wgs / 8192:.3f} runs)")
    assert torch.equal(wire.view(torch.bfloat16).view(rows, cols), src)
    assert torch.equal(dst[0].view(rows, cols), src)


@pytest.mark.parametrize("items", [63, 64, 65, 129])
def test_cast_runs_and_tails(items):
    rows, cols = items * 64, 1024                       # 256 KiB of fp32 per 64 rows
    g = torch.Generator(device="cuda").manual_seed(100 + items)
    src = torch.randn(rows, cols, generator=g, device="cuda")
    tr, ro = _identity(rows, cols, "f32", "bf16")
    wire, dst, wgs = _transfer(tr, ro, src)
    say(f"[xcd] fp32 -> bf16, {items} items, {wgs} workgroups ({wgs / 8192:.3f} runs)")
    assert torch.equal(wire.view(torch.float32).view(rows, cols), src)
    assert torch.equal(dst[0].view(rows, cols), src.to(torch.bfloat16))


@pytest.mark.parametrize("nb", [8190, 8192, 8194, 16386])
def test_fp8_pair_runs_and_tails(nb):
    rows, cols = 128, 128 * nb                          # nb full blocks, nb / 2 full pairs
    g = torch.Generator(device="cuda").manual_seed(200 + nb)
    src = (torch.randn(rows, cols, generator=g, device="cuda") *
           torch.exp2(torch.randint(-20, 20, (1, cols), generator=g, device="cuda").float())).to(torch.bfloat16)
    tr, ro = _identity(rows, cols, "bf16", "f8e4m3", 128)
    _, dst, _ = _transfer(tr, ro, src)
    say(f"[xcd] fp8, {nb} blocks ({nb // 2 / 4096:.3f} runs of pairs)")
    xb = src.float().view(1, 128, nb, 128)
    amax = xb.abs().amax(dim=(1, 3))
    s = torch.where(amax > 0, amax / torch.full_like(amax, 448.0), torch.ones_like(amax))
    q = (xb / s[:, None, :, None]).to(torch.float8_e4m3fn).view(rows, cols)
    assert torch.equal(dst[0].view(torch.uint8).view(rows, cols), q.view(torch.uint8))
    assert torch.equal(dst[1].view(-1), s.view(-1))
