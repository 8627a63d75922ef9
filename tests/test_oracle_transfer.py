"""Pins for oracle.transfer.

* pack -> network -> unpack with identical trainer and rollout layouts and
  dtypes is the identity on every rank's tensors;
* unpack through the plan equals the rollout tensors computed straight from
  the rollout layout and the checkpoint (the result is unique: any correct
  routing gives it), for every scaled workload, including the fp32 -> bf16 and
  bf16 -> fp8 casts;
* the wire holds checkpoint row-major rectangles in the sender dtype.
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
