"""Pins for oracle.catalog and oracle.layout.

* catalogs against published parameter counts and hand closed forms;
* every layout style against an independent torch-slicing construction
  (synthetic_checkpoint/loaders.py), using unique element identifiers, the same
  device the paper uses to reveal a loader's source map (Sec. 3.1);
* full coverage of rollout tensors and in-bounds placements.
"""

import os

import numpy as np
import pytest
import torch

from oracle import catalog as C
from oracle.layout import Parallelism, describe_layout, flat_run_rects, layout_from_spec, validate
from oracle.transfer import materialize
from synthetic_checkpoint.workloads import ORDER, WORKLOADS, scaled

from synthetic_checkpoint.loaders import STYLES, ckpt_shapes

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _counts():
    out = {}
    for line in open(os.path.join(GOLDEN, "param_counts.txt")):
        if line.strip() and not line.startswith("#"):
            name, n = line.split()[:2]
            out[name] = int(n)
    return out


@pytest.mark.parametrize("name,shapes", [("llama3_8b", C.LLAMA3_8B), ("mixtral_8x7b", C.MIXTRAL_8X7B),
                                         ("tiny_dense", C.TINY), ("dsv3_16moe", C.DSV3_16MOE)])
def test_parameter_counts(name, shapes):
    cat = C.checkpoint_catalog(shapes)
    assert sum(t.numel for t in cat) == _counts()[name]


def test_catalog_tensor_counts():
    assert len(C.checkpoint_catalog(C.DSV3_16MOE)) == 16 * (1 + 3 + 3 * 256)
    assert len(C.checkpoint_catalog(C.LLAMA3_8B)) == 3 + 32 * 9
    assert len(C.checkpoint_catalog(C.MIXTRAL_8X7B)) == 3 + 32 * (7 + 24)


def test_flat_run_rects_brute_force():
    rng = np.random.default_rng(0)
    for _ in range(500):
        cols = int(rng.integers(1, 9))
        rows = int(rng.integers(1, 6))
        p0 = int(rng.integers(0, rows * cols))
        p1 = int(rng.integers(p0 + 1, rows * cols + 1))
        got = []
        rects = list(flat_run_rects(p0, p1, cols))
        assert 1 <= len(rects) <= 3
        for first, r0, r1, c0, c1 in rects:
            assert first == r0 * cols + c0
            got += [i * cols + j for i in range(r0, r1) for j in range(c0, c1)]
        assert got == list(range(p0, p1))


def _id_tensors(model):
    shapes = ckpt_shapes(model)
    T, off = {}, 0
    for n, (r, c) in shapes.items():
        T[n] = torch.arange(off, off + r * c, dtype=torch.int64).reshape(r, c) + 1
        off += r * c
    return T


EXTRA = [
    (scaled("llama3_8b_tp4_to_tp2")["model"], dict(style="megatron", dtype="bf16", tp=2, dp=2)),
    (scaled("llama3_8b_tp4_to_tp2")["model"], dict(style="serving", dtype="bf16", tp=4, dp=2)),
    (scaled("llama3_8b_tp4_to_tp2")["model"], dict(style="fsdp_flat", dtype="f32", fsdp=3, dp=2)),
    (scaled("mixtral_ep8fsdp2_to_ep2")["model"], dict(style="megatron", dtype="bf16", ep=4, transposed_row_parallel=True)),
    (scaled("mixtral_ep8fsdp2_to_ep2")["model"], dict(style="serving", dtype="bf16", ep=2, tp=2)),
    (scaled("dsv3_ep64_to_ep8_fp8")["model"], dict(style="fsdp_flat", dtype="bf16", fsdp=5, ep=4)),
    (scaled("dsv3_ep64_to_ep8_fp8")["model"], dict(style="serving", dtype="bf16", ep=2, tp=2, quant="f8e4m3",
                                                  quant_block=64)),
]


def _cases():
    for name in ORDER:
        w = scaled(name)
        yield name + ":trainer", w["model"], w["trainer"]
        yield name + ":rollout", w["model"], w["rollout"]
    for k, (m, p) in enumerate(EXTRA):
        yield f"extra{k}", m, p


@pytest.mark.parametrize("label,model,par", list(_cases()), ids=[c[0] for c in _cases()])
def test_layout_matches_torch_slicing(label, model, par):
    lay = layout_from_spec(model, par)
    validate(lay, require_full_cover=par["style"] != "fsdp_flat")
    T = _id_tensors(model)
    cat_t = [T[t.name].numpy() for t in lay.catalog]
    for rank in range(lay.nranks):
        got = materialize(lay, rank, lambda t: cat_t[t], dtype=np.int64)
        want = STYLES[par["style"]](model, par, T, rank)
        assert len(got) == len(want), (rank, len(got), len(want))
        for u, (g, w) in enumerate(zip(got, want)):
            lc = lay.ranks[rank].locals[u]
            if w is None:            # scale tensor: shape only
                q = lay.ranks[rank].locals[lc.scales]
                assert (lc.batch, lc.rows, lc.cols) == (q.batch, -(-q.rows // q.block), -(-q.cols // q.block))
                continue
            assert g.size == w.numel(), (rank, lc.name)
            assert np.array_equal(g, w.reshape(-1).numpy()), (rank, lc.name)


def test_rank_counts_full_size():
    for name in ORDER:
        w = WORKLOADS[name]
        tr = layout_from_spec(w["model"], w["trainer"])
        ro = layout_from_spec(w["model"], w["rollout"])
        want_t = {"tiny_fsdp2_to_tp2": 2, "llama3_8b_fsdp8_to_tp1": 8, "llama3_8b_tp4_to_tp2": 4,
                  "mixtral_ep8fsdp2_to_ep2": 16, "dsv3_ep64_to_ep8_fp8": 64}[name]
        want_r = {"tiny_fsdp2_to_tp2": 2, "llama3_8b_fsdp8_to_tp1": 1, "llama3_8b_tp4_to_tp2": 2,
                  "mixtral_ep8fsdp2_to_ep2": 2, "dsv3_ep64_to_ep8_fp8": 8}[name]
        assert (tr.nranks, ro.nranks) == (want_t, want_r)


def test_full_size_rollout_shapes():
    # the rollout tensors of one rank at the published shapes
    w = WORKLOADS["dsv3_ep64_to_ep8_fp8"]
    ro = layout_from_spec(w["model"], w["rollout"])
    loc = {lc.name: lc for lc in ro.ranks[0].locals}
    assert (loc["layers.0.experts.w13"].batch, loc["layers.0.experts.w13"].rows, loc["layers.0.experts.w13"].cols) == (32, 4096, 7168)
    assert (loc["layers.0.experts.w13_scale"].rows, loc["layers.0.experts.w13_scale"].cols) == (32, 56)
    assert (loc["layers.0.experts.w2"].rows, loc["layers.0.experts.w2"].cols) == (7168, 2048)
    assert (loc["layers.0.experts.w2_scale"].rows, loc["layers.0.experts.w2_scale"].cols) == (56, 16)
    assert loc["layers.0.router"].dtype == "bf16" and loc["layers.0.experts.w13"].dtype == "f8e4m3"
    w = WORKLOADS["llama3_8b_fsdp8_to_tp1"]
    tr = layout_from_spec(w["model"], w["trainer"])
    # per-layer flat unit 218,112,000 elements -> 27,264,000 per rank
    assert tr.ranks[0].locals[1].numel == 27264000


def test_bad_degrees_rejected():
    m = C.LLAMA3_8B
    for par in [Parallelism("serving", "bf16", tp=3), Parallelism("megatron", "bf16", tp=16),
                Parallelism("fsdp_flat", "bf16", fsdp=0), Parallelism("serving", "f8e4m3", tp=1),
                Parallelism("serving", "bf16", ep=2)]:
        with pytest.raises(ValueError):
            describe_layout(m, par)
