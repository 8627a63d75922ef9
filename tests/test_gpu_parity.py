"""GPU parity through the C ABI: pack -> network stand-in -> unpack, bit for bit
against the oracle, on every scaled workload (several tiles, ragged tails,
partial and multi-piece fp8 blocks), random tiny layouts with odd shapes and
unaligned flat-shard boundaries, a transposed destination, and a sender with
nothing to send."""

import numpy as np
import pytest
import torch

import synthetic_checkpoint as sc
import paper_2609_25442_amd as wb
from oracle.catalog import CkptTensor
from oracle.layout import Layout, Local, Placement, RankLayout, describe_layout, layout_from_spec
from synthetic_checkpoint.workloads import ORDER, scaled

from gpu_util import roundtrip, say
from oracle_cases import hand_replicated_pair, random_medium_model, random_model, random_par
from wb_cases import to_wb

pytestmark = pytest.mark.gpu


def _values(catalog, dtype):
    cache = {}

    def get(t):
        if t not in cache:
            c = catalog[t]
            cache[t] = sc.values_numpy(t, np.arange(c.numel), dtype).reshape(c.rows, c.cols)
        return cache[t]
    return get


@pytest.mark.parametrize("name", ORDER)
def test_scaled_workload_parity(name):
    w = scaled(name)
    otr = layout_from_spec(w["model"], w["trainer"])
    oro = layout_from_spec(w["model"], w["rollout"])
    tr = wb.Layout.describe(w["model"], w["trainer"])
    ro = wb.Layout.describe(w["model"], w["rollout"])
    roundtrip(otr, oro, _values(otr.catalog, w["trainer"]["dtype"]), tr, ro, label=name)


@pytest.mark.parametrize("seed", range(16))
def test_random_tiny_layout_parity(seed):
    rng = np.random.default_rng(1000 + seed)
    m = random_model(rng)
    otr = describe_layout(m, random_par(rng, m, "trainer"))
    oro = describe_layout(m, random_par(rng, m, "rollout"))
    dtype = otr.ranks[0].locals[0].dtype
    roundtrip(otr, oro, _values(otr.catalog, dtype), label=f"random{seed}")


@pytest.mark.parametrize("seed", range(16))
def test_random_medium_layout_parity(seed):
    """Random models with hidden sizes of 128 to 384 under random trainer and
    rollout parallelism: vector copies and casts, register-transposed slabs,
    fp8 blocks of 64 and 128 (two-block and general paths), odd flat-shard
    boundaries and ragged tails, each through every rank."""
    rng = np.random.default_rng(2000 + seed)
    m = random_medium_model(rng)
    otr = describe_layout(m, random_par(rng, m, "trainer"))
    oro = describe_layout(m, random_par(rng, m, "rollout", blocks=(64, 128)))
    dtype = otr.ranks[0].locals[0].dtype
    roundtrip(otr, oro, _values(otr.catalog, dtype), label=f"random-medium{seed}")


def test_hand_layout_with_transposed_destination():
    tr, ro = hand_replicated_pair()
    roundtrip(tr, ro, _values(tr.catalog, "f32"), label="hand")


def test_sender_with_nothing_to_send():
    cat = [CkptTensor("T0", 3, 5), CkptTensor("T1", 2, 7)]
    tr = Layout(cat, [RankLayout([Local("a", "bf16", 1, 3, 5)], [Placement(0, 0, 3, 0, 5, 0, 0, 5)]),
                      RankLayout([Local("b", "bf16", 1, 2, 7)], [Placement(1, 0, 2, 0, 7, 0, 0, 7)])])
    ro = Layout(cat, [RankLayout([Local("x", "bf16", 1, 5, 3)], [Placement(0, 0, 3, 0, 5, 0, 0, 3, 1)])])
    roundtrip(tr, ro, _values(cat, "bf16"), label="idle-sender")


def test_odd_widths_and_unaligned_runs():
    # FSDP flat shards of odd-width tensors: runs start at every offset mod 8
    from oracle.catalog import ModelShapes
    from oracle.layout import Parallelism
    m = ModelShapes("dense", num_layers=2, hidden=13, num_heads=2, num_kv_heads=1, head_dim=3, ffn=11, vocab=7)
    for fsdp, dt in ((3, "f32"), (5, "bf16"), (7, "f32")):
        otr = describe_layout(m, Parallelism("fsdp_flat", dt, fsdp=fsdp))
        for rp in (Parallelism("serving", "bf16"), Parallelism("serving", "f32"),
                   Parallelism("serving", "bf16", quant="f8e4m3", quant_block=4)):
            oro = describe_layout(m, rp)
            roundtrip(otr, oro, _values(otr.catalog, dt), label=f"odd-fsdp{fsdp}-{dt}-{rp.dtype}{rp.quant}")


def test_generator_matches_on_gpu():
    for t, (r, c) in [(0, (129, 4097)), (5000, (7, 33))]:
        for dt in ("f32", "bf16"):
            x = sc.values_torch(t, r, c, dt, device="cuda").reshape(-1)
            bits = x.view(torch.int32 if dt == "f32" else torch.int16).cpu().numpy()
            bits = bits.view(np.uint32 if dt == "f32" else np.uint16)
            assert np.array_equal(bits, sc.values_numpy(t, np.arange(r * c), dt))


@pytest.mark.parametrize("rows,cols,split", [(520, 200, 1), (640, 264, 2), (130, 77, 1), (1024, 512, 3), (384, 1100, 2),
                                            (768, 1536, 2), (1000, 1296, 2), (1024, 4096, 4), (1536, 1024, 4)])
def test_transposed_trainer_shards(rows, cols, split):
    """Trainer ranks hold column slabs of T stored transposed (row-parallel
    shards); the rollout wants T row-major in one tensor. Whole tiles of 128
    slab rows x 512 slab columns of aligned slabs (16-byte rows on both sides)
    go to the tile kernel: 1536 x 1024 in four slabs gives 2 x 3 tiles each and
    nothing else; 520 x 200 one tile and strips for the register transposes
    (64-column strips of up to 256 rows) and the LDS tiles; 1000 x 1296 gives
    648 x 1000 slabs, 5 tiles each, a right and a bottom strip;
    1024 x 4096 in four slabs is the shape of a Llama-3-8B o slab. Slabs whose
    rows are not 16-byte multiples (384 x 1100: 1100-byte rows) and odd widths
    go to the LDS tiles."""
    cat = [CkptTensor("T", rows, cols)]
    cuts = [cols * k // split for k in range(split + 1)]
    ranks = []
    for a, b in zip(cuts, cuts[1:]):
        ranks.append(RankLayout([Local("t", "bf16", 1, b - a, rows)], [Placement(0, 0, rows, a, b, 0, 0, rows, 1)]))
    tr = Layout(cat, ranks)
    ro = Layout(cat, [RankLayout([Local("x", "bf16", 1, rows, cols)], [Placement(0, 0, rows, 0, cols, 0, 0, cols)])])
    p = wb.Plan(to_wb(tr), to_wb(ro), wb.SENDER, 0)
    slab = cuts[1] - cuts[0]
    aligned = (slab * 2) % 16 == 0 and (rows * 2) % 16 == 0
    assert p.launch_grid(4)[0] == ((slab // 128) * (rows // 512) if aligned else 0)
    roundtrip(tr, ro, _values(cat, "bf16"), label=f"transposed-{rows}x{cols}/{split}")


@pytest.mark.parametrize("rows,cols", [(600, 520), (512, 768), (256, 300), (600, 1096), (256, 1024)])
def test_transposed_rollout_tiles(rows, cols):
    """The unpack direction: the rollout stores T transposed, so its
    assembly transposes whole tiles of 128 payload rows x 512 columns (and the
    ragged strips) out of the row-major wire payloads of two trainer ranks
    (row halves of T)."""
    cat = [CkptTensor("T", rows, cols)]
    h = rows // 2
    tr = Layout(cat, [RankLayout([Local("a", "bf16", 1, h, cols)], [Placement(0, 0, h, 0, cols, 0, 0, cols)]),
                      RankLayout([Local("b", "bf16", 1, rows - h, cols)], [Placement(0, h, rows, 0, cols, 0, 0, cols)])])
    ro = Layout(cat, [RankLayout([Local("x", "bf16", 1, cols, rows)], [Placement(0, 0, rows, 0, cols, 0, 0, rows, 1)])])
    p = wb.Plan(to_wb(tr), to_wb(ro), wb.RECEIVER, 0)
    # whole tiles where the payload's rows and its place in x are 16-byte aligned
    aligned = (cols * 2) % 16 == 0 and (rows * 2) % 16 == 0
    tiles = [(n // 128) * (cols // 512) if aligned and (r0 * 2) % 16 == 0 else 0 for r0, n in ((0, h), (h, rows - h))]
    assert p.launch_grid(4)[0] == sum(tiles)
    roundtrip(tr, ro, _values(cat, "bf16"), label=f"transposed-rollout-{rows}x{cols}")


def test_fp8_paired_and_general_blocks():
    """fp8 blocks of one unpack on all three paths of the block kernel: 19 single-piece
    blocks, of which 9 are full 128 x 128 (8 taken as full pairs, the odd one
    out with the other 10: ragged right and bottom edges, pairs that straddle
    tensors and block rows, the last one alone), and blocks filled from two
    wire pieces or from an unaligned one (one per workgroup)."""
    cat = [CkptTensor("T", 300, 392), CkptTensor("V", 130, 264), CkptTensor("W", 128, 128), CkptTensor("U", 200, 136)]
    r0 = RankLayout([Local("t0", "bf16", 1, 256, 392), Local("v", "bf16", 1, 130, 264), Local("u0", "bf16", 1, 200, 60)],
                    [Placement(0, 0, 256, 0, 392, 0, 0, 392), Placement(1, 0, 130, 0, 264, 1, 0, 264),
                     Placement(3, 0, 200, 0, 60, 2, 0, 60)])
    r1 = RankLayout([Local("t1", "bf16", 1, 44, 392), Local("w", "bf16", 1, 128, 128), Local("u1", "bf16", 1, 200, 76)],
                    [Placement(0, 256, 300, 0, 392, 0, 0, 392), Placement(2, 0, 128, 0, 128, 1, 0, 128),
                     Placement(3, 0, 200, 60, 136, 2, 0, 76)])
    tr = Layout(cat, [r0, r1])
    locs, pls = [], []
    for t, c in enumerate(cat):
        nbr, nbc = -(-c.rows // 128), -(-c.cols // 128)
        u = len(locs)
        locs += [Local("q" + c.name, "f8e4m3", 1, c.rows, c.cols, 128, scale=u + 1),
                 Local("s" + c.name, "f32", 1, nbr, nbc, scales=u)]
        pls.append(Placement(t, 0, c.rows, 0, c.cols, u, 0, c.cols))
    ro = Layout(cat, [RankLayout(locs, pls)])
    p = wb.Plan(to_wb(tr), to_wb(ro), wb.RECEIVER, 0)
    nb = p.work_counts()[1]
    gx = p.launch_grid(1)[0]
    assert nb == 12 + 6 + 1 + 4 and gx == 8 // 2 + (19 - 8 + 1) // 2 + 4, (nb, gx)
    roundtrip(tr, ro, _values(cat, "bf16"), label="fp8-paths")


@pytest.mark.parametrize("copies", [2, 3, 5, 8, 10])
def test_fp8_row_band_blocks(copies):
    """A tensor replicated on ``copies`` trainer ranks is cut into row bands
    among them, so each fp8 block of a rollout rank's copy is filled by up to
    four full-width bands (paired with other blocks, each row read from its
    band) or, with more bands, by the one-block path; ragged bottom and right
    edges, and a single-piece tensor beside it."""
    cat = [CkptTensor("S", 300, 264), CkptTensor("P", 128, 384)]
    ranks = []
    for r in range(copies):
        locs = [Local("s", "bf16", 1, 300, 264)] + ([Local("p", "bf16", 1, 128, 384)] if r == 0 else [])
        pls = [Placement(0, 0, 300, 0, 264, 0, 0, 264)] + ([Placement(1, 0, 128, 0, 384, 1, 0, 384)] if r == 0 else [])
        ranks.append(RankLayout(locs, pls))
    tr = Layout(cat, ranks)
    locs, pls = [], []
    for t, c in enumerate(cat):
        u = len(locs)
        locs += [Local("q" + c.name, "f8e4m3", 1, c.rows, c.cols, 128, scale=u + 1),
                 Local("s" + c.name, "f32", 1, -(-c.rows // 128), -(-c.cols // 128), scales=u)]
        pls.append(Placement(t, 0, c.rows, 0, c.cols, u, 0, c.cols))
    ro = Layout(cat, [RankLayout(locs, pls)])
    p = wb.Plan(to_wb(tr), to_wb(ro), wb.RECEIVER, 0)
    gx = p.launch_grid(1)[0]
    # rows of S split as floor(j * 300 / copies): pieces per block row of S
    # (3 block columns each, the last 8 wide; the last block row 44 high)
    cuts = [j * 300 // copies for j in range(copies + 1)]
    pieces = [sum(1 for a, b in zip(cuts, cuts[1:]) if a < min(300, 128 * (i + 1)) and b > 128 * i) for i in range(3)]
    full = 3 + sum(2 for i, n in enumerate(pieces) if n == 1 and i < 2)   # P's blocks, then S's whole ones
    pairable = 3 + sum(3 for n in pieces if n <= 4)
    assert gx == full // 2 + (pairable - full // 2 * 2 + 1) // 2 + 3 + 9 - pairable, (pieces, gx)
    assert pairable > full and (copies < 10 or pairable < 12)
    roundtrip(tr, ro, _values(cat, "bf16"), label=f"fp8-bands-{copies}")


def _tiny_catalog_layouts(tdtype, rdtype, block=0):
    """[A 1 x 1, B 1 x 3, C 3 x 1, Z 2 x 2] held by two trainer ranks (B split
    by columns, rank 1 holding none of A and Z), wanted whole by one rollout
    rank in ``rdtype`` (fp8 with one block per tensor when ``block``)."""
    cat = [CkptTensor("A", 1, 1), CkptTensor("B", 1, 3), CkptTensor("C", 3, 1), CkptTensor("Z", 2, 2)]
    r0 = RankLayout([Local("a", tdtype, 1, 1, 1), Local("b0", tdtype, 1, 1, 2), Local("z", tdtype, 1, 2, 2)],
                    [Placement(0, 0, 1, 0, 1, 0, 0, 1), Placement(1, 0, 1, 0, 2, 1, 0, 2),
                     Placement(3, 0, 2, 0, 2, 2, 0, 2)])
    r1 = RankLayout([Local("c", tdtype, 1, 3, 1), Local("b1", tdtype, 1, 1, 1)],
                    [Placement(2, 0, 3, 0, 1, 0, 0, 1), Placement(1, 0, 1, 2, 3, 1, 0, 1)])
    locs, pls = [], []
    for t, c in enumerate(cat):
        u = len(locs)
        if block:
            locs += [Local("q" + c.name, rdtype, 1, c.rows, c.cols, block, scale=u + 1),
                     Local("s" + c.name, "f32", 1, 1, 1, scales=u)]
        else:
            locs.append(Local(c.name.lower(), rdtype, 1, c.rows, c.cols))
        pls.append(Placement(t, 0, c.rows, 0, c.cols, u, 0, c.cols))
    return cat, Layout(cat, [r0, r1]), Layout(cat, [RankLayout(locs, pls)])


@pytest.mark.parametrize("tdtype,rdtype,block", [("bf16", "bf16", 0), ("f32", "bf16", 0), ("bf16", "f8e4m3", 128),
                                                 ("f32", "f8e4m3", 128)])
def test_single_elements_and_zero_blocks(tdtype, rdtype, block):
    """Degenerate shapes through each cast path: 1 x 1, 1 x 3 and 3 x 1 tensors
    and a 2 x 2 block of signed zeros. As fp8, every tensor is one partial
    block: a one-element block quantises to +-448 exactly with s = |x| / 448,
    and the all-zero block takes s = 1 and keeps each zero's sign."""
    cat, tr, ro = _tiny_catalog_layouts(tdtype, rdtype, block)
    base = _values(cat, tdtype)
    neg0 = 0x80000000 if tdtype == "f32" else 0x8000

    def values(t):
        if cat[t].name != "Z":
            return base(t)
        return np.array([[0, neg0], [neg0, 0]], dtype=np.uint32 if tdtype == "f32" else np.uint16)

    roundtrip(tr, ro, values, label=f"tiny-{tdtype}-{rdtype}")


@pytest.mark.parametrize("task_bytes", [1024, 4096, 1 << 30])
@pytest.mark.parametrize("name", ORDER)
def test_work_item_size_leaves_results_unchanged(name, task_bytes, monkeypatch):
    """The planner cuts contiguous runs into work items of WB_TASK_BYTES
    (default 256 KiB) and each launch maps workgroups to items by class shifts
    fitted to its longest item. One-chunk items (1 KiB), ragged multi-chunk
    items (4 KiB) and one item per run (1 GiB: the longest shifts and the most
    idle workgroups) give the oracle's bytes on every scaled workload."""
    monkeypatch.setenv("WB_TASK_BYTES", str(task_bytes))
    w = scaled(name)
    otr = layout_from_spec(w["model"], w["trainer"])
    oro = layout_from_spec(w["model"], w["rollout"])
    tr = wb.Layout.describe(w["model"], w["trainer"])
    ro = wb.Layout.describe(w["model"], w["rollout"])
    roundtrip(otr, oro, _values(otr.catalog, w["trainer"]["dtype"]), tr, ro, label=f"{name}/{task_bytes}")
