"""Source maps from probed identifiers and their second-order differences.

Test infrastructure: only the tests, the smoke check and the benchmark's CPU
baseline use this package.

WeightBridge Sec. 3.1 and App. B (Algorithm 1): every checkpoint element gets
a unique identifier; a black-box weight loader run on a checkpoint holding
those identifiers leaves, in every local tensor, the identifier field A of the
elements it copied there. Because identifiers need more bits than a parameter
holds, the checkpoint is loaded several times, pass k carrying the k-th b-bit
chunk floor(p / 2^(b k)) mod 2^b of every identifier. Each pass keeps only the
non-zero entries of diff2 of the chunk field, and the passes are recombined
as sum_k 2^(b k) diff2(C_k), which equals diff2(A) exactly because diff2 is
linear. diff2 of a field made of slice copies is zero except next to the
corners of the copied rectangles, and A is recovered from it by prefix sums.

Readings (the paper leaves these open):
* identifiers are 2^24 + the element's flat position in the checkpoint
  (catalog order, row-major); 0 marks an element no loader wrote. Every step
  of an affine run of identifiers is below 2^24 (at most a row length), so no
  run can continue into a 0;
* local tensors are seen as 2-D [batch * rows, cols] fields (a flat buffer is
  one row), and diff2 keeps the tensor's own extent (A = 0 above and to the
  left, nothing is stored past the end);
* the carry (Algorithm 1: ExpandCarry, EmitCarry, with D <- D + carries
  before NonZeros): pass k's field S_k = diff2(C_k) + Q_(k-1) is split into
  the entries kept, R_k = S_k mod 2^b (in [0, 2^b)), and the carry into the
  next pass, Q_k = floor(S_k / 2^b); the last pass keeps S_k whole. Then
  sum_k 2^(b k) R_k = diff2(A) exactly, and R_k is zero wherever diff2(A) is
  (the chunk wrap-arounds move into the carries), so every pass keeps only
  entries next to slice-copy corners. The carries are a sparse field of their
  own; how they travel between passes is not modelled here.

Everything is computed densely on small tensors with plain integer numpy.
"""

from __future__ import annotations

import numpy as np

from .layout import Layout
from .transfer import local_index

FIRST_ID = 1 << 24


def first_ids(catalog) -> list[int]:
    """Identifier of element (0, 0) of every checkpoint tensor."""
    out, p = [], FIRST_ID
    for t in catalog:
        out.append(p)
        p += t.rows * t.cols
    return out


def chunk_bits(dtype: str) -> int:
    """Identifier bits one parameter element carries per loading pass."""
    return 8 if dtype == "f8e4m3" else 16


def num_chunks(catalog, b: int) -> int:
    last = first_ids(catalog)[-1] + catalog[-1].rows * catalog[-1].cols - 1
    return -(-last.bit_length() // b)


def id_chunk(ids: np.ndarray, k: int, b: int) -> np.ndarray:
    """Chunk k of width b of every identifier (Algorithm 1, MakeIdChunk)."""
    return (ids.astype(np.int64) >> (b * k)) & ((1 << b) - 1)


def diff1(A: np.ndarray) -> np.ndarray:
    """Eq. (diff1): A[i,j] - A[i-1,j] - A[i,j-1] + A[i-1,j-1], A = 0 outside."""
    P = np.zeros((A.shape[0] + 1, A.shape[1] + 1), dtype=A.dtype)
    P[1:, 1:] = A
    return P[1:, 1:] - P[:-1, 1:] - P[1:, :-1] + P[:-1, :-1]


def diff2(A: np.ndarray) -> np.ndarray:
    """Eq. (diff2): diff1 applied twice."""
    return diff1(diff1(A))


def prefix2(D: np.ndarray) -> np.ndarray:
    """Two-dimensional prefix sum, the inverse of diff1."""
    return np.cumsum(np.cumsum(D, axis=0), axis=1)


def undiff2(Z: np.ndarray) -> np.ndarray:
    return prefix2(prefix2(Z))


def nonzeros(D: np.ndarray) -> dict:
    """{(i, j): value} of the non-zero entries (Algorithm 1, NonZeros)."""
    ii, jj = np.nonzero(D)
    return {(int(i), int(j)): int(D[i, j]) for i, j in zip(ii, jj)}


def recombine(per_chunk: list[dict], b: int) -> dict:
    """Algorithm 1, Recombine: sum over passes of 2^(b k) times pass k's
    entries, exactly (Python integers), zeros dropped."""
    out: dict = {}
    for k, z in enumerate(per_chunk):
        for pos, v in z.items():
            out[pos] = out.get(pos, 0) + (v << (b * k))
    return {pos: v for pos, v in out.items() if v}


def carry_passes(chunk_fields: list[np.ndarray], b: int) -> tuple[list[dict], list[dict]]:
    """Algorithm 1 with carries, on the chunk fields C_0 .. C_(K-1) of one
    tensor: for k = 0 .. K-1, D = diff2(C_k) plus the carries of pass k - 1
    (ExpandCarry; none before pass 0); the entries kept for pass k are
    NonZeros of D mod 2^b, and D's carry part floor(D / 2^b) goes to pass k + 1
    (EmitCarry); the last pass keeps D itself. Returns the kept entries and
    the carries of every pass (the last pass's carries are empty)."""
    K = len(chunk_fields)
    kept, carries = [], []
    Q = np.zeros(chunk_fields[0].shape, dtype=np.int64)
    for k, C in enumerate(chunk_fields):
        D = diff2(np.asarray(C, dtype=np.int64)) + Q
        if k == K - 1:
            kept.append(nonzeros(D))
            Q = np.zeros_like(D)
        else:
            kept.append(nonzeros(np.mod(D, 1 << b)))
            Q = np.floor_divide(D, 1 << b)
        carries.append(nonzeros(Q))
    return kept, carries


def dense(Z: dict, R: int, C: int) -> np.ndarray:
    D = np.zeros((R, C), dtype=np.int64)
    for (i, j), v in Z.items():
        D[i, j] = v
    return D


def id_fields(layout: Layout, rank: int) -> list[np.ndarray]:
    """Identifier field of every local tensor of one rank, from its placements
    (what a loader run on the identifier checkpoint leaves), as
    [batch * rows, cols] int64 arrays."""
    firsts = first_ids(layout.catalog)
    rk = layout.ranks[rank]
    out = [np.zeros(lc.numel, dtype=np.int64) for lc in rk.locals]
    for p in rk.placements:
        cols = layout.catalog[p.t].cols
        i = np.arange(p.r0, p.r1, dtype=np.int64)[:, None]
        j = np.arange(p.c0, p.c1, dtype=np.int64)[None, :]
        out[p.u][local_index(p, i, j)] = firsts[p.t] + i * cols + j
    return [a.reshape(lc.batch * lc.rows, lc.cols) for a, lc in zip(out, rk.locals)]


def probe_fields(fields: list[np.ndarray], b: int, nchunks: int) -> tuple[list[list[dict]], list[dict]]:
    """Algorithm 1 on given identifier fields: per local tensor, the non-zero
    entries of diff2 of every chunk field, and their recombination."""
    per_local, combined = [], []
    for A in fields:
        chunks = [nonzeros(diff2(id_chunk(A, k, b))) for k in range(nchunks)]
        per_local.append(chunks)
        combined.append(recombine(chunks, b))
    return per_local, combined


def field_from_nonzeros(Z: dict, R: int, C: int) -> np.ndarray:
    """The identifier field recovered from the recombined entries."""
    return undiff2(dense(Z, R, C))


def decode(ids: np.ndarray, catalog) -> np.ndarray:
    """(tensor, row, col) of every identifier (-1 rows for 0 = not loaded)."""
    firsts = np.array(first_ids(catalog), dtype=np.int64)
    flat = ids.ravel()
    out = np.full((flat.size, 3), -1, dtype=np.int64)
    hit = flat > 0
    t = np.searchsorted(firsts, flat[hit], side="right") - 1
    cols = np.array([c.cols for c in catalog], dtype=np.int64)
    off = flat[hit] - firsts[t]
    out[hit, 0] = t
    out[hit, 1] = off // cols[t]
    out[hit, 2] = off % cols[t]
    return out
