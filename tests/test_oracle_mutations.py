"""The oracle's pins catch plausible mistakes. Each case plants one mistake in
the oracle (a dropped rounding step, a wrong constant, sign or index, a
transposed operand, a changed tie-break), on the CPU only, and requires that a
named pin test then fails. Nothing here touches the library."""

import numpy as np
import pytest

from oracle import casts, diff2, layout, plan, transfer

import test_oracle_casts as T_casts
import test_oracle_diff2 as T_diff2
import test_oracle_exchange as T_exchange
import test_oracle_layout as T_layout
import test_oracle_plan as T_plan
import test_oracle_rounds as T_rounds
import test_oracle_transfer as T_transfer


def _truncating_bf16(bits32):
    u = np.asarray(bits32, dtype=np.uint32)
    return (u >> 16).astype(np.uint16)


def _ties_away_bf16(bits32):
    u = np.asarray(bits32, dtype=np.uint32)
    return ((u + np.uint32(0x8000)) >> 16).astype(np.uint16)


def _scale_447(amax):
    a = np.float32(amax)
    return np.float32(1.0) if a == 0 else np.float32(a / np.float32(447.0))


def _quantize_by_reciprocal(x_f32):
    x = np.asarray(x_f32, dtype=np.float32)
    amax = np.float32(np.max(np.abs(x))) if x.size else np.float32(0)
    s = casts.block_scale(amax)
    q = (x * (np.float32(1.0) / s)).astype(np.float32)
    return casts.f64_to_e4m3(q.astype(np.float64)), s


def _e4m3_ties_up(x):
    x = np.asarray(x, dtype=np.float64)
    a = np.abs(x)
    v = casts.E4M3_VALUES
    lo = np.clip(np.searchsorted(v, a, side="right") - 1, 0, 0x7E)
    hi = np.minimum(lo + 1, 0x7E)
    up = (v[hi] - a) <= (a - v[lo])
    code = np.where(up & (a > v[lo]), hi, lo).astype(np.uint8)
    return code | (np.signbit(x).astype(np.uint8) << 7)


def _ignores_transpose(p, i, j):
    return p.base + (i - p.r0) * p.ld + (j - p.c0)


def _split_always_columns(x, k):
    n = x.c1 - x.c0
    out = []
    for j in range(k):
        a, b = j * n // k, (j + 1) * n // k
        if a < b:
            out.append(plan.Rect(x.r0, x.r1, x.c0 + a, x.c0 + b))
    return out


def _deal_reversed_ties(pieces, owners, e, total, weight):
    k = len(owners)
    for q in owners:
        e[q] -= total
    who = [None] * len(pieces)
    for j in sorted(range(len(pieces)), key=lambda j: (-pieces[j].numel, j)):
        q = min(owners, key=lambda q: (e[q], -q))
        e[q] += k * weight(pieces[j])
        who[j] = q
    return who


def _diff1_wrong_corner(A):
    P = np.zeros((A.shape[0] + 1, A.shape[1] + 1), dtype=A.dtype)
    P[1:, 1:] = A
    return P[1:, 1:] - P[:-1, 1:] - P[1:, :-1] - P[:-1, :-1]


def _recombine_shifted(per_chunk, b):
    out = {}
    for k, z in enumerate(per_chunk):
        for pos, v in z.items():
            out[pos] = out.get(pos, 0) + (v << (b * (k + 1)))
    return {pos: v for pos, v in out.items() if v}


def _carry_passes_variant(drop=False, trunc=False, last_low=False):
    def run(chunk_fields, b):
        K = len(chunk_fields)
        kept, carries = [], []
        Q = np.zeros(chunk_fields[0].shape, dtype=np.int64)
        for k, C in enumerate(chunk_fields):
            D = diff2.diff2(np.asarray(C, dtype=np.int64)) + (0 if drop else Q)
            if k == K - 1 and not last_low:
                kept.append(diff2.nonzeros(D))
                Q = np.zeros_like(D)
            else:
                Q = (np.trunc(D / (1 << b)).astype(np.int64) if trunc else np.floor_divide(D, 1 << b))
                kept.append(diff2.nonzeros(D - (Q << b)))
            carries.append(diff2.nonzeros(Q))
        return kept, carries
    return run


_orig_flat_run_rects = layout.flat_run_rects


def _flat_run_short_tail(p0, p1, cols):
    for first, r0, r1, c0, c1 in _orig_flat_run_rects(p0, p1, cols):
        if c1 - c0 > 1 and r1 - r0 == 1 and c0 == 0 and c1 < cols:
            c1 -= 1
        yield first, r0, r1, c0, c1


_orig_rollout_groups = plan._rollout_groups


def _groups_lowest_holder_only(rollout):
    return {k: {min(v): v[min(v)]} for k, v in _orig_rollout_groups(rollout).items()}


def _wire_align_128(mine, ns, nd):
    old = plan.PAYLOAD_ALIGN
    plan.PAYLOAD_ALIGN = 128
    try:
        return _orig_wire(mine, ns, nd)
    finally:
        plan.PAYLOAD_ALIGN = old


_orig_wire = plan._wire


def _rounds_filled_to_budget(trainer, rollout, segments, budget):
    # rounds filled greedily up to the budget, not re-cut into equal chunks
    unit = plan._block_units(rollout, len(trainer.catalog))
    order = sorted({unit[g.t] for g in segments}, key=lambda u: min(g.t for g in segments if unit[g.t] == u))
    r, cur = 0, {}
    for u in order:
        mine = [g for g in segments if unit[g.t] == u]
        add = {}
        for g in mine:
            if g.stage == 0:
                add[("s", g.s)] = add.get(("s", g.s), 0) + g.nbytes
            add[("d", g.d)] = add.get(("d", g.d), 0) + g.nbytes
        if cur and any(cur.get(k, 0) + v > budget for k, v in add.items()):
            r, cur = r + 1, {}
        for k, v in add.items():
            cur[k] = cur.get(k, 0) + v
        for g in mine:
            g.round = r
    return r + 1


def _quantize_flattened(lc, staged):
    # blocks tiled over the flattened [batch * rows, cols] matrix (scales kept right)
    x = staged.view(np.float32)
    codes, _ = casts.quantize_matrix(x.reshape(lc.batch * lc.rows, lc.cols), lc.block)
    scales = [casts.quantize_matrix(m, lc.block)[1] for m in x.reshape(lc.batch, lc.rows, lc.cols)]
    return codes.ravel(), np.stack(scales).ravel().view(np.uint32)


def _quantize_scales_transposed(lc, staged):
    # each expert's scales written [bj][bi]
    out_c, out_s = [], []
    for m in staged.view(np.float32).reshape(lc.batch, lc.rows, lc.cols):
        c, s = casts.quantize_matrix(m, lc.block)
        out_c.append(c)
        out_s.append(np.ascontiguousarray(s.T))
    return np.stack(out_c).ravel(), np.concatenate([s.ravel() for s in out_s]).view(np.uint32)


MUTANTS = {
    # casts
    "bf16 truncates": (casts, "f32_to_bf16", _truncating_bf16, [T_casts.test_hand_worked_rounding_cases]),
    "bf16 ties away from zero": (casts, "f32_to_bf16", _ties_away_bf16, [T_casts.test_hand_worked_rounding_cases]),
    "fp8 scale amax/447": (casts, "block_scale", _scale_447, [T_casts.test_quantize_block_matches_torch_formula]),
    "fp8 divides by multiplying the reciprocal": (casts, "quantize_block", _quantize_by_reciprocal,
                                                  [T_casts.test_quantize_divides_rather_than_multiplying_by_the_reciprocal]),
    "fp8 ties round up": (casts, "f64_to_e4m3", _e4m3_ties_up, [T_casts.test_hand_worked_rounding_cases]),
    "stacked fp8 tiled over the flattened experts": (transfer, "_quantize_local", _quantize_flattened,
                                                      [lambda: T_transfer.test_stacked_fp8_blocks_tile_each_expert(
                                                          272, 328, 128, "bf16")]),
    "stacked fp8 scales written [e][bj][bi]": (transfer, "_quantize_local", _quantize_scales_transposed,
                                               [lambda: T_transfer.test_stacked_fp8_blocks_tile_each_expert(
                                                   130, 200, 64, "bf16")]),
    # placements
    "transposed placement read as plain": (transfer, "local_index", _ignores_transpose,
                                           [lambda: T_layout.test_layout_matches_torch_slicing(
                                               *[c for c in T_layout._cases() if c[0] == "extra3"][0])]),
    "flat run drops the tail's last column": (layout, "flat_run_rects", _flat_run_short_tail,
                                              [T_layout.test_flat_run_rects_brute_force,
                                               lambda: T_layout.test_layout_matches_torch_slicing(
                                                   *[c for c in T_layout._cases()
                                                     if c[0] == "llama3_8b_fsdp8_to_tp1:trainer"][0])]),
    # plan
    "replicas always split by columns": (plan, "_split", _split_always_columns,
                                         [T_plan.test_hand_plan_matches_golden]),
    "deficit ties go to the higher rank": (plan, "_deal", _deal_reversed_ties, [T_plan.test_hand_plan_matches_golden]),
    "payloads 128-byte aligned": (plan, "_wire", _wire_align_128, [T_plan.test_hand_plan_matches_golden]),
    "rounds ignore the budget": (plan, "_assign_rounds", lambda tr, ro, segs, budget: 1,
                                 [T_rounds.test_hand_rounds_match_golden]),
    "rounds filled up to the budget, not balanced": (plan, "_assign_rounds", _rounds_filled_to_budget,
                                                     [T_rounds.test_hand_balanced_rounds_match_golden]),
    # exchange stages
    "rollout groups keep only their lowest holder": (plan, "_rollout_groups", _groups_lowest_holder_only,
                                                     [T_exchange.test_hand_exchange_plan_matches_golden]),
    # diff2
    "diff1 corner term with the wrong sign": (diff2, "diff1", _diff1_wrong_corner, [T_diff2.test_hand_worked_example]),
    "passes recombined one chunk too high": (diff2, "recombine", _recombine_shifted,
                                             [lambda: T_diff2.test_chunked_passes_recombine_exactly(16, 0),
                                              lambda: T_diff2.test_workloads_probe_recovers_fields(
                                                  "llama3_8b_fsdp8_to_tp1")]),
    "carries not added to the next pass": (diff2, "carry_passes", _carry_passes_variant(drop=True),
                                           [T_diff2.test_carry_hand_worked_examples,
                                            lambda: T_diff2.test_carries_closed_form_on_random_fields(16, 0)]),
    "carries truncated toward zero": (diff2, "carry_passes", _carry_passes_variant(trunc=True),
                                      [T_diff2.test_carry_hand_worked_examples,
                                       lambda: T_diff2.test_carries_closed_form_on_random_fields(16, 0)]),
    "last pass keeps only its low bits": (diff2, "carry_passes", _carry_passes_variant(last_low=True),
                                          [T_diff2.test_carry_hand_worked_examples,
                                           lambda: T_diff2.test_carries_keep_only_corner_entries_of_slice_copies(0)]),
}


@pytest.mark.parametrize("name", list(MUTANTS))
def test_pins_catch_planted_mistake(name, monkeypatch):
    mod, attr, mutant, pins = MUTANTS[name]
    original = getattr(mod, attr)
    monkeypatch.setattr(mod, attr, mutant)
    # test modules that imported the oracle function by name hold the same object
    for T in (T_casts, T_diff2, T_exchange, T_layout, T_plan, T_rounds, T_transfer):
        if getattr(T, attr, None) is original:
            monkeypatch.setattr(T, attr, mutant)
    caught = 0
    for pin in pins:
        try:
            pin()
        except Exception:
            caught += 1
    assert caught, f"no pin caught: {name}"


def test_pins_pass_without_mistakes():
    for _, _, _, pins in MUTANTS.values():
        for pin in pins:
            pin()
