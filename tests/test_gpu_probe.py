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


def _batch(fields, cap):
    """Run wb_diff2_batch; returns (count, {index: value})."""
    idx = torch.full((cap,), -1, dtype=torch.int64, device="cuda")
    val = torch.zeros(cap, dtype=torch.int64, device="cuda")
    count = torch.zeros(1, dtype=torch.int64, device="cuda")
    ws = torch.empty(max(wb.diff2_batch_workspace(fields), 8), dtype=torch.uint8, device="cuda")
    wb.diff2_batch(fields, idx, val, count, ws)
    torch.cuda.synchronize()
    n = int(count.item())
    m = min(n, cap)
    got = dict(zip(idx[:m].cpu().numpy().tolist(), val[:m].cpu().numpy().tolist()))
    assert len(got) == m
    return n, got


def _expected(fields_np):
    """Oracle entries of a batch: diff2 of every field's value (sum of 2^(16 k)
    times pass k), at the field's offset in the concatenation."""
    want, off = {}, 0
    for passes, R, C in fields_np:
        A = sum((p.astype(np.int64) << (16 * k)) for k, p in enumerate(passes))
        for (i, j), v in nonzeros(diff2(np.asarray(A, dtype=np.int64).reshape(R, C))).items():
            want[off + i * C + j] = v
        off += R * C
    return want


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
@pytest.mark.parametrize("kind", ["random", "slices"])
def test_diff2_batch_one_pass_matches_oracle(dtype, kind):
    """Every shape above in one launch, plus empty fields and an unaligned view
    (element tiles): entries at each field's offset in the concatenation."""
    rng = np.random.default_rng(11)
    shapes = SHAPES + [(0, 5), (4, 0), (40, 512)]
    fields, fields_np, keep = [], [], []
    for n, (R, C) in enumerate(shapes):
        F = _field(rng, R, C, kind) if R * C else np.zeros((R, C), dtype=np.int64)
        if n == len(shapes) - 1:   # one element into its allocation
            big = _to_gpu(np.concatenate([[7], F.ravel(), [9]]), dtype)
            x = big[1:1 + R * C]
            keep.append(big)
        else:
            x = _to_gpu(F, dtype)
        fields.append((x, dtype, R, C))
        fields_np.append(([F], R, C))
    say(f"[diff2 batch] {dtype} {kind} {len(fields)} fields")
    want = _expected(fields_np)
    n, got = _batch(fields, sum(R * C for R, C in shapes) + 16)
    assert n == len(want)
    assert got == want


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
@pytest.mark.parametrize("passes", [2, 3])
def test_diff2_batch_recombines_passes(dtype, passes):
    """Fields given as several passes: random chunks (every entry survives,
    values up to 2^52), and the chunks of real identifier slices, whose
    wrap-around entries cancel inside the launch so that only diff2 of the
    identifier field itself comes out."""
    rng = np.random.default_rng(12 + passes)
    fields, fields_np = [], []
    for R, C in SHAPES:
        if rng.random() < 0.5:
            chunks = [rng.integers(0, 1 << 16, size=(R, C)) for _ in range(passes)]
        else:
            A = np.zeros((R, C), dtype=np.int64)
            for _ in range(3):
                a = int(rng.integers(0, R)); b = int(rng.integers(a + 1, R + 1))
                c = int(rng.integers(0, C)); d = int(rng.integers(c + 1, C + 1))
                base = int(rng.integers(1 << 24, 1 << (16 * passes - 2)))
                i = np.arange(a, b)[:, None]; j = np.arange(c, d)[None, :]
                A[a:b, c:d] = base + i * int(rng.integers(1, 5000)) + j
            chunks = [id_chunk(A, k, 16) for k in range(passes)]
            # the chunk fields alone have many more entries than the identifiers
            assert sum(len(nonzeros(diff2(ch))) for ch in chunks) >= len(nonzeros(diff2(A)))
        fields.append(([_to_gpu(ch, dtype) for ch in chunks], dtype, R, C))
        fields_np.append((chunks, R, C))
    say(f"[diff2 batch] {dtype} passes={passes}")
    want = _expected(fields_np)
    n, got = _batch(fields, sum(R * C for R, C in SHAPES) + 16)
    assert n == len(want)
    assert got == want


def test_diff2_batch_capacity_overflow_reports_the_count():
    rng = np.random.default_rng(13)
    F = [rng.integers(0, 1 << 16, size=(50, 90)) for _ in range(2)]
    fields = [([_to_gpu(f, "bf16") for f in F], "bf16", 50, 90), (_to_gpu(F[0], "bf16"), "bf16", 50, 90)]
    want = _expected([(F, 50, 90), ([F[0]], 50, 90)])
    n, got = _batch(fields, 10)
    assert n == len(want)
    assert len(got) == 10 and all(want[i] == v for i, v in got.items())


def _loaders(w, side, ranks):
    par = w[side]
    fn = ref.STYLES[par["style"]]
    return [lambda T, r=r: [x.contiguous() for x in fn(w["model"], par, T, r) if x is not None] for r in ranks]


@pytest.mark.parametrize("hold", [True, False])
@pytest.mark.parametrize("name", ORDER)
def test_probe_recovers_declared_layouts(name, hold):
    w = scaled(name)
    shapes = ref.ckpt_shapes(w["model"])
    for side in ("trainer", "rollout"):
        L = layout_from_spec(w["model"], w[side])
        cat = [(c.name, c.rows, c.cols) for c in L.catalog]
        assert all(shapes[n] == (r, c) for n, r, c in cat)
        ranks = sorted({0, L.nranks - 1})
        say(f"[probe] {name} {side} ranks {ranks} hold_passes={hold}")
        dtype = w["trainer"]["dtype"]
        stats = {}
        got = wb.probe_layout(cat, dtype, _loaders(w, side, ranks), stats=stats, hold_passes=hold)
        assert stats["hold_passes"] == [hold] * len(ranks)
        for k, r in enumerate(ranks):
            rk = L.ranks[r]
            keep = [u for u, lc in enumerate(rk.locals) if lc.scales < 0]
            remap = {u: i for i, u in enumerate(keep)}
            want = sorted((p.t, p.r0, p.r1, p.c0, p.c1, remap[p.u], p.base, p.ld, p.tr) for p in rk.placements)
            assert sorted(got.placements(k)) == want, (name, side, r)
            assert [x["numel"] for x in got.locals(k)] == [rk.locals[u].numel for u in keep]


@pytest.mark.timeout(600)
@pytest.mark.parametrize("name,side,hold", [("llama3_8b_fsdp8_to_tp1", "trainer", True),
                                            ("llama3_8b_fsdp8_to_tp1", "rollout", True),
                                            ("llama3_8b_fsdp8_to_tp1", "rollout", False),
                                            ("llama3_8b_tp4_to_tp2", "trainer", True)])
def test_probe_full_size(name, side, hold):
    """The benchmark ranks at full size (16 GB identifier checkpoint), probed
    through the torch loaders, with the passes held on the device or recorded
    one by one: the recovered placements equal the declared."""
    from synthetic_checkpoint.workloads import WORKLOADS

    w = WORKLOADS[name]
    rank = w["pack_rank"] if side == "trainer" else w["unpack_rank"]
    L = layout_from_spec(w["model"], w[side])
    cat = [(c.name, c.rows, c.cols) for c in L.catalog]
    say(f"[probe full] {name} {side} rank {rank} hold_passes={hold}")
    got = wb.probe_layout(cat, w["trainer"]["dtype"], _loaders(w, side, [rank]), hold_passes=hold)
    rk = L.ranks[rank]
    keep = [u for u, lc in enumerate(rk.locals) if lc.scales < 0]
    remap = {u: i for i, u in enumerate(keep)}
    want = sorted((p.t, p.r0, p.r1, p.c0, p.c1, remap[p.u], p.base, p.ld, p.tr) for p in rk.placements)
    assert sorted(got.placements(0)) == want
    del got
    torch.cuda.empty_cache()
