"""Single tensors past 2^32 elements or bytes, through pack and unpack: element
indices and byte offsets beyond 32 bits in the work items, the copy, cast and
fp8 kernels and the folded launch grids. One trainer rank holds the tensor
whole and one rollout rank receives it whole; outputs are compared in full
with the source, torch's fp32 -> bf16 cast and torch's blockwise quantiser
(amax / 448, x / s, E4M3FN)."""

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
    """Pack src on the trainer rank, move the payload, unpack on the rollout
    rank; returns the rollout tensors (the wire is freed on the way)."""
    sp = wb.Plan(tr, ro, wb.SENDER, 0)
    sws = workspace_for(sp)
    sp.upload(sws)
    send = torch.empty(sp.buffer_bytes, dtype=torch.uint8, device="cuda")
    sp.pack([src], send)
    rp = wb.Plan(tr, ro, wb.RECEIVER, 0)
    rws = workspace_for(rp)
    rp.upload(rws)
    so, roff, nb = rp.region(0, 0)
    assert roff == 0 and nb == rp.buffer_bytes
    recv = send[so:so + nb]           # the payload is the receive buffer (one sender)
    dst = wb.allocate_locals(ro, 0)
    rp.unpack(recv, dst)
    torch.cuda.synchronize()
    gx, gy, _ = rp.launch_grid(0)
    del send, recv
    return dst, (gx, gy)


@pytest.mark.timeout(300)
def test_bf16_copy_past_2_32_elements():
    rows, cols = 35000, 131072                          # 4.59e9 elements, 9.2 GB
    g = torch.Generator(device="cuda").manual_seed(4)
    src = torch.randint(-32768, 32767, (rows, cols), generator=g, device="cuda", dtype=torch.int16).view(torch.bfloat16)
    tr, ro = _identity(rows, cols, "bf16", "bf16")
    dst, grid = _transfer(tr, ro, src)
    say(f"[large] bf16 copy {rows}x{cols}, unpack grid {grid}")
    assert torch.equal(dst[0].view(rows, cols).view(torch.int16), src.view(torch.int16))


@pytest.mark.timeout(300)
def test_fp32_to_bf16_past_2_32_bytes():
    rows, cols = 20000, 131072                          # 2.6e9 elements, 10.5 GB of fp32
    g = torch.Generator(device="cuda").manual_seed(5)
    src = torch.randn(rows, cols, generator=g, device="cuda")
    tr, ro = _identity(rows, cols, "f32", "bf16")
    dst, grid = _transfer(tr, ro, src)
    say(f"[large] fp32 -> bf16 {rows}x{cols}, unpack grid {grid}")
    assert torch.equal(dst[0].view(rows, cols), src.to(torch.bfloat16))


@pytest.mark.timeout(300)
def test_fp8_blocks_past_2_32_elements():
    rows, cols = 65536, 65664                           # 4.30e9 elements, 262,656 blocks (513 per block row)
    g = torch.Generator(device="cuda").manual_seed(6)
    src = torch.randn(rows, cols, generator=g, device="cuda", dtype=torch.bfloat16)
    tr, ro = _identity(rows, cols, "bf16", "f8e4m3", 128)
    dst, grid = _transfer(tr, ro, src)
    say(f"[large] fp8 {rows}x{cols}")
    nbr, nbc = rows // 128, cols // 128
    for r0 in range(0, nbr, 64):                        # 64 block rows (8192 rows) at a time
        r1 = min(nbr, r0 + 64)
        xb = src[r0 * 128:r1 * 128].float().view(r1 - r0, 128, nbc, 128)
        amax = xb.abs().amax(dim=(1, 3))
        s = torch.where(amax > 0, amax / torch.full_like(amax, 448.0), torch.ones_like(amax))
        q = (xb / s[:, None, :, None]).to(torch.float8_e4m3fn).view((r1 - r0) * 128, cols)
        got = dst[0].view(rows, cols)[r0 * 128:r1 * 128]
        assert torch.equal(got.view(torch.uint8), q.view(torch.uint8)), r0
        assert torch.equal(dst[1].view(nbr, nbc)[r0:r1], s), r0
