"""Pins for oracle.transfer.

* pack -> network -> unpack with identical trainer and rollout layouts and
  dtypes is the identity on every rank's tensors;
* unpack through the plan equals the rollout tensors computed straight from
  the rollout layout and the checkpoint (the result is unique: any correct
  routing gives it), for every scaled workload, including the fp32 -> bf16 and
  bf16 -> fp8 casts;
* the wire holds checkpoint row-major rectangles in the sender dtype.
* fp8 blocks tile each expert matrix of a stacked tensor on its own, with
  scales in [expert][block row][block column] order, against a torch
  construction (pad to whole blocks, per-block amax, amax / 448, x / s,
  float8_e4m3fn).
"""

import numpy as np
import pytest

import synthetic_checkpoint as sc
from oracle.layout import Parallelism, describe_layout, layout_from_spec
from oracle.plan import build_plan
from oracle.transfer import CODE_DTYPE, expected_rollout, materialize, network, pack, unpack
from synthetic_checkpoint.workloads import ORDER, scaled

from oracle_cases import hand_replicated_pair, random_model


def _values(catalog, dtype):
    cache = {}

    def get(t):
        if t not in cache:
            c = catalog[t]
            cache[t] = sc.values_numpy(t, np.arange(c.numel), dtype).reshape(c.rows, c.cols)
        return cache[t]
    return get


def _run(trainer, rollout, dtype):
    plan = build_plan(trainer, rollout)
    vals = _values(trainer.catalog, dtype)
    sends = {s: pack(plan, s, materialize(trainer, s, vals)) for s in range(trainer.nranks)}
    return plan, vals, sends


@pytest.mark.parametrize("seed", range(6))
def test_identity_on_identical_layouts(seed):
    rng = np.random.default_rng(100 + seed)
    m = random_model(rng)
    for par in (Parallelism("serving", "bf16", tp=2), Parallelism("serving", "bf16", tp=1),
                Parallelism("fsdp_flat", "f32", fsdp=3),
                Parallelism("megatron", "bf16", ep=2 if m.family != "dense" else 1, transposed_row_parallel=True)):
        try:
            lay = describe_layout(m, par)
        except ValueError:
            continue
        plan, vals, sends = _run(lay, lay, par.dtype)
        for d in range(lay.nranks):
            got = unpack(plan, d, network(plan, d, sends))
            want = materialize(lay, d, vals)
            for g, w in zip(got, want):
                assert np.array_equal(g, w)


@pytest.mark.parametrize("name", ORDER)
def test_unpack_equals_direct_expectation(name):
    w = scaled(name)
    tr = layout_from_spec(w["model"], w["trainer"])
    ro = layout_from_spec(w["model"], w["rollout"])
    src_dtype = w["trainer"]["dtype"]
    plan, vals, sends = _run(tr, ro, src_dtype)
    for d in range(ro.nranks):
        got = unpack(plan, d, network(plan, d, sends))
        want = expected_rollout(ro, d, vals, src_dtype)
        for u, (g, e) in enumerate(zip(got, want)):
            assert g.dtype == e.dtype and np.array_equal(g, e), (d, ro.ranks[d].locals[u].name)


def test_wire_holds_row_major_rectangles():
    tr, ro = hand_replicated_pair()
    plan, vals, sends = _run(tr, ro, "f32")
    # segment 0: T0 row 0 from sender 0 at offset 0; segment 4: T1 cols 6..10 from sender 0 at 256
    assert np.array_equal(sends[0][0:24].view(np.uint32), vals(0)[0, :])
    assert np.array_equal(sends[0][256:272].view(np.uint32), vals(1)[0, 6:10])
    # receiver 1 gets T0 rows 2..4 transposed into a [6, 2] tensor, cast to bf16
    got = unpack(plan, 1, network(plan, 1, sends))
    from oracle.casts import f32_to_bf16
    assert np.array_equal(got[0].reshape(6, 2), f32_to_bf16(vals(0)[2:4, :]).T)


def test_quantised_scales_cover_every_block():
    w = scaled("dsv3_ep64_to_ep8_fp8")
    tr = layout_from_spec(w["model"], w["trainer"])
    ro = layout_from_spec(w["model"], w["rollout"])
    plan, vals, sends = _run(tr, ro, "bf16")
    got = unpack(plan, 0, network(plan, 0, sends))
    for u, lc in enumerate(ro.ranks[0].locals):
        if lc.scales >= 0:
            s = got[u].view(np.float32)
            assert s.size == lc.numel and np.all(s > 0) and np.all(np.isfinite(s))
        if lc.block:
            assert got[u].dtype == CODE_DTYPE["f8e4m3"] and not np.any((got[u] & 0x7F) == 0x7F)


def _stacked_fp8_pair(rows, cols, block, dtype):
    """Three experts [rows, cols] stacked into one fp8 rollout tensor
    [3, rows, cols] with its [3, ceil(rows/B), ceil(cols/B)] scales; the
    trainer holds them in two ranks cut at a row that is not a block edge."""
    from oracle.catalog import CkptTensor
    from oracle.layout import Layout, Local, Placement, RankLayout

    cat = [CkptTensor(f"w{e}", rows, cols) for e in range(3)]
    h = rows // 2 + 3
    r0 = RankLayout([Local("a", dtype, 1, rows, cols), Local("b", dtype, 1, h, cols)],
                    [Placement(0, 0, rows, 0, cols, 0, 0, cols), Placement(1, 0, h, 0, cols, 1, 0, cols)])
    r1 = RankLayout([Local("c", dtype, 1, rows - h, cols), Local("d", dtype, 1, rows, cols)],
                    [Placement(1, h, rows, 0, cols, 0, 0, cols), Placement(2, 0, rows, 0, cols, 1, 0, cols)])
    nbr, nbc = -(-rows // block), -(-cols // block)
    ro = RankLayout([Local("w", "f8e4m3", 3, rows, cols, block, scale=1), Local("w_scale", "f32", 3, nbr, nbc, scales=0)],
                    [Placement(e, 0, rows, 0, cols, 0, e * rows * cols, cols) for e in range(3)])
    return Layout(cat, [r0, r1]), Layout(cat, [ro])


def _block_scaled_values(rows, cols, block, dtype, seed):
    """Checkpoint codes whose magnitude changes from block to block (every
    block of every expert has its own amax), with one all-zero block of
    signed zeros in expert 1."""
    import torch

    g = torch.Generator().manual_seed(seed)
    out = []
    for e in range(3):
        x = torch.randn(rows, cols, generator=g, dtype=torch.float64)
        for bi in range(-(-rows // block)):
            for bj in range(-(-cols // block)):
                f = 10.0 ** (4.0 * torch.rand((), generator=g, dtype=torch.float64).item() - 2.0)
                x[bi * block:(bi + 1) * block, bj * block:(bj + 1) * block] *= f
        if e == 1:
            z = x[-(rows % block or block):, -(cols % block or block):]
            z.copy_(torch.where(z < 0, -0.0, 0.0))
        x = x.to(torch.float32 if dtype == "f32" else torch.bfloat16)
        codes = x.view(torch.int32 if dtype == "f32" else torch.int16).numpy()
        out.append(codes.view(np.uint32 if dtype == "f32" else np.uint16))
    return out


def _torch_stacked_quantise(codes, rows, cols, block, dtype):
    """Independent construction with torch on the CPU: pad each expert to whole
    blocks, view as [E, nbr, B, nbc, B], amax per block, s = amax / 448 (a
    division by a tensor: IEEE), q = float8_e4m3fn(x / s)."""
    import torch

    tdt = torch.float32 if dtype == "f32" else torch.bfloat16
    idt = torch.int32 if dtype == "f32" else torch.int16
    x = torch.stack([torch.from_numpy(c.view(np.int32 if dtype == "f32" else np.int16)).view(idt).view(tdt).float()
                     for c in codes])
    nbr, nbc = -(-rows // block), -(-cols // block)
    pad = torch.zeros(3, nbr * block, nbc * block, dtype=torch.float32)
    pad[:, :rows, :cols] = x
    blocks = pad.view(3, nbr, block, nbc, block)
    amax = blocks.abs().amax(dim=(2, 4))
    s = torch.where(amax > 0, amax / torch.full_like(amax, 448.0), torch.ones_like(amax))
    q = (blocks / s[:, :, None, :, None]).to(torch.float8_e4m3fn).view(torch.uint8)
    q = q.view(3, nbr * block, nbc * block)[:, :rows, :cols]
    return q.contiguous().numpy().ravel(), s.numpy().ravel().view(np.uint32)


@pytest.mark.parametrize("rows,cols,block,dtype", [(272, 328, 128, "bf16"), (272, 328, 128, "f32"),
                                                   (130, 200, 64, "bf16")])
def test_stacked_fp8_blocks_tile_each_expert(rows, cols, block, dtype):
    """fp8 blocks tile every expert matrix of a stacked tensor on its own
    (rows and cols not multiples of the block, so tiling the flattened
    [E * rows, cols] matrix gives other blocks), scales in [e][bi][bj]
    order; checked through the plan-free expectation and through
    pack -> network -> unpack against a torch construction."""
    tr, ro = _stacked_fp8_pair(rows, cols, block, dtype)
    codes = _block_scaled_values(rows, cols, block, dtype, seed=rows + cols + block + len(dtype))
    vals = lambda t: codes[t]
    want_q, want_s = _torch_stacked_quantise(codes, rows, cols, block, dtype)
    plan = build_plan(tr, ro)
    sends = {s: pack(plan, s, materialize(tr, s, vals)) for s in range(tr.nranks)}
    for got in (expected_rollout(ro, 0, vals, dtype), unpack(plan, 0, network(plan, 0, sends))):
        assert got[0].dtype == np.uint8 and np.array_equal(got[0], want_q)
        assert np.array_equal(got[1], want_s)
    # the signed-zero block: scale 1, each zero's sign kept
    nbr, nbc = -(-rows // block), -(-cols // block)
    assert want_s.view(np.float32).reshape(3, nbr, nbc)[1, -1, -1] == 1.0
