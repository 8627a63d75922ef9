"""Source-map probing on the GPU (Sec. 3.1; App. B, Algorithm 1): the
identifier-chunk kernel and the diff2 stencils (single field, batched, and
carry passes) against the oracle, and whole ranks probed through
torch-slicing weight loaders (the black box) recovering exactly the declared
slice copies, with passes held or carried one at a time."""

import numpy as np
import pytest
import torch

import paper_2609_25442_amd as wb
from oracle.diff2 import carry_passes, diff2, id_chunk, nonzeros
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


def _carry_fields(rng, kind, passes):
    """Chunk fields of every shape (and a few empty ones): random chunks (a
    carry at nearly every position), or identifier slices whose bases sit
    near multiples of 2^32 so that chunk 1 wraps too."""
    out = []
    for R, C in SHAPES + [(0, 5), (4, 0), (40, 512)]:
        if R * C == 0:
            out.append(([np.zeros((R, C), dtype=np.int64)] * passes, R, C))
            continue
        if kind == "random":
            out.append(([rng.integers(0, 1 << 16, size=(R, C)) for _ in range(passes)], R, C))
            continue
        A = np.zeros((R, C), dtype=np.int64)
        for _ in range(3):
            a = int(rng.integers(0, R)); b = int(rng.integers(a + 1, R + 1))
            c = int(rng.integers(0, C)); d = int(rng.integers(c + 1, C + 1))
            step = int(rng.integers(1, 5000))
            top = int(rng.integers(1, 1 << (16 * passes - 33))) << 32
            base = top - int(rng.integers(0, (b - a) * step + (d - c) + 1))
            i = np.arange(a, b)[:, None]; j = np.arange(c, d)[None, :]
            A[a:b, c:d] = base + i * step + j
        out.append(([id_chunk(A, k, 16) for k in range(passes)], R, C))
    return out


def _carry_expected(fields_np, passes):
    """Oracle entries of every pass (carry_passes) at each field's offset, and
    the number of carries every pass keeps."""
    want = [{} for _ in range(passes)]
    carried = [0] * passes
    off = 0
    for chunks, R, C in fields_np:
        if R * C:
            kept, carries = carry_passes(chunks, 16)
            for k in range(passes):
                for (i, j), v in kept[k].items():
                    want[k][off + i * C + j] = v
                carried[k] += len(carries[k])
        off += R * C
    return want, carried


class _CarryRun:
    def __init__(self, fields0, carry_cap, cap):
        self.cap_c = carry_cap
        self.ws = torch.empty(wb.diff2_carry_workspace(fields0, carry_cap), dtype=torch.uint8, device="cuda")
        self.idx = torch.full((cap,), -1, dtype=torch.int64, device="cuda")
        self.val = torch.zeros(cap, dtype=torch.int64, device="cuda")
        self.count = torch.zeros(1, dtype=torch.int64, device="cuda")
        self.carries = torch.zeros(1, dtype=torch.int64, device="cuda")

    def run(self, fields, k, last):
        wb.diff2_carry(fields, k, last, self.cap_c, self.idx, self.val, self.count, self.carries, self.ws)
        torch.cuda.synchronize()
        n, c = int(self.count.item()), int(self.carries.item())
        m = min(n, self.idx.numel())
        got = dict(zip(self.idx[:m].cpu().numpy().tolist(), self.val[:m].cpu().numpy().tolist()))
        assert len(got) == m
        return n, c, got


def _carry_gpu_fields(fields_np, k, dtype, keep):
    """Pass k's fields on the device; the last field starts one element into
    its allocation (element tiles)."""
    fields = []
    for n, (chunks, R, C) in enumerate(fields_np):
        if n == len(fields_np) - 1:
            big = _to_gpu(np.concatenate([[7], chunks[k].ravel(), [9]]), dtype)
            keep.append(big)
            fields.append((big[1:1 + R * C], dtype, R, C))
        else:
            fields.append((_to_gpu(chunks[k], dtype), dtype, R, C))
    return fields


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
@pytest.mark.parametrize("kind", ["random", "slices"])
def test_diff2_carry_matches_oracle(dtype, kind):
    """Three passes one at a time, carries kept on the device between them:
    every pass's entries equal the oracle's kept entries, element by element,
    and the carries kept equal the oracle's in number. Identifier slices
    leave entries only where diff2 of the identifiers is non-zero."""
    passes = 3
    rng = np.random.default_rng(31 + (kind == "slices"))
    fields_np = _carry_fields(rng, kind, passes)
    want, carried = _carry_expected(fields_np, passes)
    numel = sum(R * C for _, R, C in fields_np)
    keep = []
    runner = None
    for k in range(passes):
        fields = _carry_gpu_fields(fields_np, k, dtype, keep)
        if runner is None:
            runner = _CarryRun(fields, numel + 16, numel + 16)
        say(f"[diff2 carry] {dtype} {kind} pass {k}: {len(fields)} fields, {numel} elements")
        n, c, got = runner.run(fields, k, k == passes - 1)
        assert n == len(want[k]), k
        assert got == want[k], k
        assert c == carried[k], k
    if kind == "slices":
        full = {}
        off = 0
        for chunks, R, C in fields_np:
            A = sum(ch.astype(np.int64) << (16 * k) for k, ch in enumerate(chunks))
            for (i, j), v in nonzeros(diff2(A)).items():
                full[off + i * C + j] = v
            off += R * C
        assert all(set(w) <= set(full) for w in want)
        assert sum(carried) > 0


def test_diff2_carry_reruns_and_reports_overflow():
    """Too few carry slots: the count of carries says so. Too little entry
    room: the pass is run again on the same workspace with more, and the
    next pass still gets the right carries."""
    rng = np.random.default_rng(33)
    F = [rng.integers(0, 1 << 16, size=(50, 90)) for _ in range(2)]
    fields_np = [(F, 50, 90)]
    want, carried = _carry_expected(fields_np, 2)
    f0 = [(_to_gpu(F[0], "bf16"), "bf16", 50, 90)]
    f1 = [(_to_gpu(F[1], "bf16"), "bf16", 50, 90)]
    small = _CarryRun(f0, 10, 4500)
    say("[diff2 carry] overflow of the carry table")
    n, c, got = small.run(f0, 0, False)
    assert c == carried[0] > 10
    assert n == len(want[0]) and got == want[0]
    room = _CarryRun(f0, 4500, 10)
    say("[diff2 carry] overflow of the entries, then the pass again")
    n, c, got = room.run(f0, 0, False)
    assert n == len(want[0]) > 10 and len(got) == 10 and all(want[0][i] == v for i, v in got.items())
    room.idx = torch.full((4500,), -1, dtype=torch.int64, device="cuda")
    room.val = torch.zeros(4500, dtype=torch.int64, device="cuda")
    n, c, got = room.run(f0, 0, False)
    assert got == want[0] and c == carried[0]
    n, c, got = room.run(f1, 1, True)
    assert got == want[1] and c == 0


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
            if not hold:
                # every pass hands over only entries next to slice-copy corners
                assert all(p["entries"] <= 16 * len(rk.placements) for p in stats[k]), stats[k]
            keep = [u for u, lc in enumerate(rk.locals) if lc.scales < 0]
            remap = {u: i for i, u in enumerate(keep)}
            want = sorted((p.t, p.r0, p.r1, p.c0, p.c1, remap[p.u], p.base, p.ld, p.tr) for p in rk.placements)
            assert sorted(got.placements(k)) == want, (name, side, r)
            assert [x["numel"] for x in got.locals(k)] == [rk.locals[u].numel for u in keep]


@pytest.mark.timeout(600)
@pytest.mark.parametrize("name,side,hold", [("llama3_8b_fsdp8_to_tp1", "trainer", True),
                                            ("llama3_8b_fsdp8_to_tp1", "rollout", True),
                                            ("llama3_8b_fsdp8_to_tp1", "rollout", False),
                                            ("llama3_8b_tp4_to_tp2", "trainer", True),
                                            ("mixtral_ep8fsdp2_to_ep2", "trainer", False),
                                            ("dsv3_ep64_to_ep8_fp8", "trainer", True),
                                            ("dsv3_ep64_to_ep8_fp8", "rollout", False)])
def test_probe_full_size(name, side, hold):
    """The benchmark ranks at full size, probed through the torch loaders, with
    the passes held on the device or carried one at a time (each pass handing
    over only corner entries): the recovered placements equal the declared.
    The identifier checkpoint is made on demand, tensor by tensor as the loader
    reads it: the DeepSeek-V3 checkpoint (1.8 x 10^11 elements, 362 GB in bf16)
    is larger than the GPU, and its expert-parallel rollout rank reads 47 GB of
    it per pass (the fp8 tensors are probed in the checkpoint's bf16, before
    quantisation)."""
    from synthetic_checkpoint.workloads import WORKLOADS

    w = WORKLOADS[name]
    rank = w["pack_rank"] if side == "trainer" else w["unpack_rank"]
    L = layout_from_spec(w["model"], w[side])
    cat = [(c.name, c.rows, c.cols) for c in L.catalog]
    say(f"[probe full] {name} {side} rank {rank} hold_passes={hold}")
    stats = {}
    got = wb.probe_layout(cat, w["trainer"]["dtype"], _loaders(w, side, [rank]), hold_passes=hold, stats=stats)
    rk = L.ranks[rank]
    if not hold:
        say(f"[probe full] passes: {[(p['entries'], p['carries']) for p in stats[0]]}")
        assert all(p["entries"] <= 16 * len(rk.placements) for p in stats[0])
        assert stats[0][0]["carries"] > 0 and "carry_retries" not in stats
    keep = [u for u, lc in enumerate(rk.locals) if lc.scales < 0]
    remap = {u: i for i, u in enumerate(keep)}
    want = sorted((p.t, p.r0, p.r1, p.c0, p.c1, remap[p.u], p.base, p.ld, p.tr) for p in rk.placements)
    assert sorted(got.placements(0)) == want
    del got
    torch.cuda.empty_cache()
