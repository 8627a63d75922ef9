"""Pins for oracle.diff2 (App. B, Algorithm 1, Eqs. diff1 and diff2).

* a worked example derived by hand from the separable closed form
  (tests/golden/diff2_example.txt);
* the closed form itself on random rectangles and affine fields: diff2 of one
  slice copy is the sum of three outer products of one-dimensional second
  differences, supported on at most 16 points (the paper's bound);
* diff1 is inverted by a two-dimensional prefix sum, so diff2 is lossless;
* chunked passes recombine exactly to diff2 of the full identifiers;
* the per-pass carries (Algorithm 1, ExpandCarry and EmitCarry): two worked
  examples derived by hand (tests/golden/diff2_carries_b4.txt); the carries
  of pass k equal floor(diff2(A mod M) / M) and the entries kept up to pass k
  sum to diff2(A mod M) mod M, M = 2^(b (k + 1)) (A mod M is what the first
  k + 1 chunks hold, and diff2 is linear); the kept entries recombine to
  diff2(A), lie where diff2(A) is non-zero, and are below 2^b except in the
  last pass;
* on every workload (scaled) and on random layouts, the recombined entries of
  every local tensor number at most 16 per placement and give back the exact
  identifier field of the declared placements.
"""

import os

import numpy as np
import pytest

from oracle.catalog import CkptTensor
from oracle.diff2 import (FIRST_ID, carry_passes, chunk_bits, decode, dense, diff1, diff2, field_from_nonzeros,
                          first_ids, id_chunk, id_fields, nonzeros, num_chunks, probe_fields, recombine, undiff2)
from oracle.layout import Layout, Local, Placement, RankLayout, describe_layout, layout_from_spec
from synthetic_checkpoint.workloads import ORDER, scaled

from oracle_cases import random_model, random_par

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def test_hand_worked_example():
    cat = [CkptTensor("T0", 4, 5)]
    L = Layout(cat, [RankLayout([Local("x", "f32", 1, 3, 6)], [Placement(0, 1, 3, 2, 5, 0, 1, 6)])])
    (A,) = id_fields(L, 0)
    want = {}
    for line in open(os.path.join(GOLDEN, "diff2_example.txt")):
        if line.startswith("#") or not line.strip():
            continue
        i, j, v = map(int, line.split())
        want[(i, j)] = v
    assert nonzeros(diff2(A)) == want
    assert A[0, 1] == FIRST_ID + 5 * 1 + 2


def _d2_indicator(a, b):
    """Second difference of 1[a, b) and of x 1[a, b), written out by hand."""
    u0, u1 = {}, {}
    for x, w0, w1 in ((a, 1, a), (a + 1, -1, 1 - a), (b, -1, -b), (b + 1, 1, b - 1)):
        u0[x] = u0.get(x, 0) + w0
        u1[x] = u1.get(x, 0) + w1
    return u0, u1


@pytest.mark.parametrize("seed", range(40))
def test_closed_form_of_one_slice_copy(seed):
    rng = np.random.default_rng(seed)
    R, C = int(rng.integers(1, 14)), int(rng.integers(1, 14))
    a = int(rng.integers(0, R)); b = int(rng.integers(a + 1, R + 1))
    c = int(rng.integers(0, C)); d = int(rng.integers(c + 1, C + 1))
    al, be, ga = (int(x) for x in rng.integers(-10**9, 10**9, 3))
    A = np.zeros((R, C), dtype=np.int64)
    i = np.arange(a, b)[:, None]
    j = np.arange(c, d)[None, :]
    A[a:b, c:d] = al + be * i + ga * j
    u0, u1 = _d2_indicator(a, b)
    v0, v1 = _d2_indicator(c, d)
    want = {}
    for x in u0:
        for y in v0:
            v = al * u0[x] * v0[y] + be * u1[x] * v0[y] + ga * u0[x] * v1[y]
            if v and x < R and y < C:
                want[(x, y)] = v
    got = nonzeros(diff2(A))
    assert got == want
    assert len(got) <= 16


@pytest.mark.parametrize("seed", range(10))
def test_diff1_inverted_by_prefix_sums(seed):
    rng = np.random.default_rng(100 + seed)
    A = rng.integers(-2**40, 2**40, size=(int(rng.integers(1, 30)), int(rng.integers(1, 30))))
    assert np.array_equal(np.cumsum(np.cumsum(diff1(A), 0), 1), A)
    assert np.array_equal(undiff2(diff2(A)), A)


@pytest.mark.parametrize("b", [8, 16])
@pytest.mark.parametrize("seed", range(8))
def test_chunked_passes_recombine_exactly(b, seed):
    rng = np.random.default_rng(200 + seed)
    A = rng.integers(0, 2**50, size=(int(rng.integers(1, 20)), int(rng.integers(1, 20))))
    A[rng.random(A.shape) < 0.3] = 0
    chunks = [nonzeros(diff2(id_chunk(A, k, b))) for k in range(-(-50 // b))]
    assert recombine(chunks, b) == nonzeros(diff2(A))
    assert np.array_equal(sum(id_chunk(A, k, b) << (b * k) for k in range(-(-50 // b))), A)


def _golden_carries():
    cases, kept, carried = {}, {}, {}
    for line in open(os.path.join(GOLDEN, "diff2_carries_b4.txt")):
        if line.startswith("#") or not line.strip():
            continue
        w = line.split()
        if w[0] == "field":
            b, K, R, C = map(int, w[2:6])
            cases[w[1]] = (b, K, np.array(list(map(int, w[6:])), dtype=np.int64).reshape(R, C))
            kept[w[1]] = [{} for _ in range(K)]
            carried[w[1]] = [{} for _ in range(K)]
        else:
            k, i, j, v = map(int, w[2:])
            (kept if w[0] == "kept" else carried)[w[1]][k][(i, j)] = v
    return cases, kept, carried


def test_carry_hand_worked_examples():
    cases, kept, carried = _golden_carries()
    assert set(cases) == {"row", "slab"}
    for name, (b, K, A) in cases.items():
        got_kept, got_carries = carry_passes([id_chunk(A, k, b) for k in range(K)], b)
        assert got_kept == kept[name], name
        assert got_carries == carried[name], name
        assert recombine(got_kept, b) == nonzeros(diff2(A))


def _check_carries(A, b, K):
    kept, carries = carry_passes([id_chunk(A, k, b) for k in range(K)], b)
    assert recombine(kept, b) == nonzeros(diff2(A))
    support = nonzeros(diff2(A))
    for k in range(K):
        assert set(kept[k]) <= set(support), k
        if k < K - 1:
            assert all(0 < v < (1 << b) for v in kept[k].values())
            M = 1 << (b * (k + 1))
            P = diff2(np.mod(A, M))
            assert carries[k] == nonzeros(np.floor_divide(P, M)), k
            low = sum((dense(kept[j], *A.shape) << (b * j)) for j in range(k + 1))
            assert np.array_equal(low, np.mod(P, M)), k
        else:
            assert carries[k] == {}
    return kept, carries


@pytest.mark.parametrize("b", [4, 8, 16])
@pytest.mark.parametrize("seed", range(8))
def test_carries_closed_form_on_random_fields(b, seed):
    rng = np.random.default_rng(400 + seed)
    A = rng.integers(0, 2**40, size=(int(rng.integers(1, 24)), int(rng.integers(1, 24))))
    A[rng.random(A.shape) < 0.3] = 0
    _check_carries(A, b, -(-40 // b))


@pytest.mark.parametrize("seed", range(6))
def test_carries_keep_only_corner_entries_of_slice_copies(seed):
    # identifiers of random layouts, shifted so that 4-bit chunks wrap many
    # times inside every slice copy and 16-bit chunks wrap across 2^32
    rng = np.random.default_rng(500 + seed)
    m = random_model(rng)
    L = describe_layout(m, random_par(rng, m, "rollout"))
    r = int(rng.integers(0, L.nranks))
    for A in id_fields(L, r):
        for b, shift in ((4, 0), (16, (1 << 32) - int(rng.integers(1, max(2, A.size))))):
            B = np.where(A > 0, A + shift, 0)
            K = -(-int(B.max()).bit_length() // b) if B.max() > 0 else 1
            kept, carries = _check_carries(B, b, K)
            # the wrap-arounds leave many carries but no kept entries of their own
            if b == 4 and A.size >= 64 and np.count_nonzero(A) == A.size:
                assert sum(map(len, carries)) > 0


def _check_rank(layout, rank):
    fields = id_fields(layout, rank)
    b = chunk_bits("bf16")
    per_chunk, combined = probe_fields(fields, b, num_chunks(layout.catalog, b))
    rk = layout.ranks[rank]
    npl = [0] * len(rk.locals)
    for p in rk.placements:
        npl[p.u] += 1
    for u, (A, Z) in enumerate(zip(fields, combined)):
        assert len(Z) <= 16 * npl[u], (rk.locals[u].name, len(Z), npl[u])
        assert np.array_equal(field_from_nonzeros(Z, *A.shape), A)
    return fields


@pytest.mark.parametrize("name", ORDER)
def test_workloads_probe_recovers_fields(name):
    w = scaled(name)
    for side in ("trainer", "rollout"):
        L = layout_from_spec(w["model"], w[side])
        for r in sorted({0, L.nranks - 1}):
            _check_rank(L, r)


@pytest.mark.parametrize("seed", range(20))
def test_random_layouts_probe_recovers_fields(seed):
    rng = np.random.default_rng(300 + seed)
    m = random_model(rng)
    for side in ("trainer", "rollout"):
        L = describe_layout(m, random_par(rng, m, side))
        fields = _check_rank(L, int(rng.integers(0, L.nranks)))
        # decoding an identifier gives back the element the placement names
        rk = L.ranks[0]
        for A in fields:
            dec = decode(A, L.catalog)
            assert np.all((dec[:, 0] >= 0) == (A.ravel() > 0))


def test_identifier_layout():
    cat = [CkptTensor("a", 2, 3), CkptTensor("b", 4, 5)]
    assert first_ids(cat) == [FIRST_ID, FIRST_ID + 6]
    assert num_chunks(cat, 16) == 2 and num_chunks(cat, 8) == 4
    assert chunk_bits("f8e4m3") == 8 and chunk_bits("bf16") == 16 and chunk_bits("f32") == 16
