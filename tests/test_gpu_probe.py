"""Source-map probing on the GPU (Sec. 3.1; App. B, Algorithm 1): the
identifier-chunk kernel and the diff2 stencil against the oracle, and whole
ranks probed through torch-slicing weight loaders (the black box) recovering
exactly the declared slice copies."""

import numpy as np
import pytest
import torch

import paper_2609_25442_amd as wb
from oracle.diff2 import diff2, id_chunk, nonzeros
from oracle.layout import layout_from_spec
from synthetic_checkpoint.workloads import ORDER, scaled

from synthetic_checkpoint import loaders as ref
from gpu_util import say

pytestmark = pytest.mark.gpu

TORCH = {"bf16": torch.bfloat16, "f32": torch.float32}


def _codes(t, dtype):
    if dtype == "bf16":
        return t.view(torch.int16).cpu().numpy().view(np.uint16).astype(np.int64)
    return t.cpu().numpy().astype(np.int64)


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
def test_make_ids_matches_oracle(dtype):
    n = 1_000_003
    first = (1 << 24) + 123_456_789_012
    t = torch.empty(n, dtype=TORCH[dtype], device="cuda")
    ids = first + np.arange(n, dtype=np.int64)
    for k in range(3):
        wb.make_ids(t, dtype, first, k)
        torch.cuda.synchronize()
        assert np.array_equal(_codes(t, dtype), id_chunk(ids, k, 16)), k


def _field(rng, R, C, kind):
    if kind == "random":
        return rng.integers(0, 1 << 16, size=(R, C))
    # chunk 0 of a few affine slices: the wraps of a real pass
    A = np.zeros((R, C), dtype=np.int64)
    for _ in range(3):
        a = int(rng.integers(0, R)); b = int(rng.integers(a + 1, R + 1))
        c = int(rng.integers(0, C)); d = int(rng.integers(c + 1, C + 1))
        base = int(rng.integers(1 << 24, 1 << 40))
        i = np.arange(a, b)[:, None]; j = np.arange(c, d)[None, :]
        A[a:b, c:d] = base + i * int(rng.integers(1, 5000)) + j
    return id_chunk(A, 0, 16)


def _to_gpu(codes, dtype):
    if dtype == "bf16":
        return torch.from_numpy(codes.astype(np.uint16).view(np.int16)).cuda().view(torch.bfloat16)
    return torch.from_numpy(codes.astype(np.float32)).cuda()


# vector path (cols a multiple of 8 bf16 / 4 f32 values, aligned) and element path
SHAPES = [(1, 1), (1, 1000), (1000, 1), (3, 257), (130, 300), (65, 64), (64, 513), (200, 1), (2, 70000),
          (97, 2048), (33, 4104), (1, 300000), (1, 8), (1, 2056)]


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
@pytest.mark.parametrize("kind", ["random", "slices"])
def test_diff2_matches_oracle(dtype, kind):
    rng = np.random.default_rng(7)
    count = torch.zeros(1, dtype=torch.int64, device="cuda")
    for R, C in SHAPES:
        say(f"[diff2] {dtype} {kind} {R}x{C}")
        F = _field(rng, R, C, kind)
        want = nonzeros(diff2(F))
        x = _to_gpu(F, dtype)
        cap = R * C
        idx = torch.full((cap,), -1, dtype=torch.int64, device="cuda")
        val = torch.zeros(cap, dtype=torch.int32, device="cuda")
        wb.diff2(x, dtype, R, C, idx, val, count)
        torch.cuda.synchronize()
        n = int(count.item())
        assert n == len(want), (R, C)
        got = {(int(i) // C, int(i) % C): int(v) for i, v in zip(idx[:n].cpu().numpy(), val[:n].cpu().numpy())}
        assert got == want, (R, C)


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
def test_diff2_unaligned_view(dtype):
    """A tensor starting one element into its allocation takes the element path."""
    rng = np.random.default_rng(9)
    R, C = 40, 512
    F = _field(rng, R, C, "slices")
    big = _to_gpu(np.concatenate([[7], F.ravel(), [9]]), dtype)
    x = big[1:1 + R * C]
    want = nonzeros(diff2(F))
    idx = torch.full((R * C,), -1, dtype=torch.int64, device="cuda")
    val = torch.zeros(R * C, dtype=torch.int32, device="cuda")
    count = torch.zeros(1, dtype=torch.int64, device="cuda")
    wb.diff2(x, dtype, R, C, idx, val, count)
    torch.cuda.synchronize()
    n = int(count.item())
    got = {(int(i) // C, int(i) % C): int(v) for i, v in zip(idx[:n].cpu().numpy(), val[:n].cpu().numpy())}
    assert got == want


def test_diff2_capacity_overflow_reports_the_count():
    rng = np.random.default_rng(8)
    F = rng.integers(0, 1 << 16, size=(50, 90))
    want = nonzeros(diff2(F))
    x = _to_gpu(F, "bf16")
    idx = torch.full((10,), -1, dtype=torch.int64, device="cuda")
    val = torch.zeros(10, dtype=torch.int32, device="cuda")
    count = torch.zeros(1, dtype=torch.int64, device="cuda")
    wb.diff2(x, "bf16", 50, 90, idx, val, count)
    torch.cuda.synchronize()
    assert int(count.item()) == len(want)
    for i, v in zip(idx.cpu().numpy(), val.cpu().numpy()):
        assert want[(int(i) // 90, int(i) % 90)] == int(v)


def _loaders(w, side, ranks):
    par = w[side]
    fn = ref.STYLES[par["style"]]
    return [lambda T, r=r: [x.contiguous() for x in fn(w["model"], par, T, r) if x is not None] for r in ranks]


@pytest.mark.parametrize("name", ORDER)
def test_probe_recovers_declared_layouts(name):
    w = scaled(name)
    shapes = ref.ckpt_shapes(w["model"])
    for side in ("trainer", "rollout"):
        L = layout_from_spec(w["model"], w[side])
        cat = [(c.name, c.rows, c.cols) for c in L.catalog]
        assert all(shapes[n] == (r, c) for n, r, c in cat)
        ranks = sorted({0, L.nranks - 1})
        say(f"[probe] {name} {side} ranks {ranks}")
        dtype = w["trainer"]["dtype"]
        got = wb.probe_layout(cat, dtype, _loaders(w, side, ranks))
        for k, r in enumerate(ranks):
            rk = L.ranks[r]
            keep = [u for u, lc in enumerate(rk.locals) if lc.scales < 0]
            remap = {u: i for i, u in enumerate(keep)}
            want = sorted((p.t, p.r0, p.r1, p.c0, p.c1, remap[p.u], p.base, p.ld, p.tr) for p in rk.placements)
            assert sorted(got.placements(k)) == want, (name, side, r)
            assert [x["numel"] for x in got.locals(k)] == [rk.locals[u].numel for u in keep]


@pytest.mark.timeout(600)
@pytest.mark.parametrize("name,side", [("llama3_8b_fsdp8_to_tp1", "trainer"), ("llama3_8b_fsdp8_to_tp1", "rollout"),
                                       ("llama3_8b_tp4_to_tp2", "trainer")])
def test_probe_full_size(name, side):
    """The benchmark ranks at full size (16 GB identifier checkpoint), probed
    through the torch loaders: the recovered placements equal the declared."""
    from synthetic_checkpoint.workloads import WORKLOADS

    w = WORKLOADS[name]
    rank = w["pack_rank"] if side == "trainer" else w["unpack_rank"]
    L = layout_from_spec(w["model"], w[side])
    cat = [(c.name, c.rows, c.cols) for c in L.catalog]
    say(f"[probe full] {name} {side} rank {rank}")
    got = wb.probe_layout(cat, w["trainer"]["dtype"], _loaders(w, side, [rank]))
    rk = L.ranks[rank]
    keep = [u for u, lc in enumerate(rk.locals) if lc.scales < 0]
    remap = {u: i for i, u in enumerate(keep)}
    want = sorted((p.t, p.r0, p.r1, p.c0, p.c1, remap[p.u], p.base, p.ld, p.tr) for p in rk.placements)
    assert sorted(got.placements(0)) == want
    del got
    torch.cuda.empty_cache()
