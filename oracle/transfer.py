"""Pack, the network stand-in, unpack, and the plan-independent expectation.

WeightBridge Sec. 3.2: on the trainer side a packing kernel transforms the
tensors planned for a round into checkpoint format and coalesces them into one
contiguous buffer per receiver; on the rollout side an assembly kernel gathers
the shards from different senders, transforms them into inference format and
writes them into the model parameters. Here each step is spelled out element
by element with explicit index arithmetic (placement semantics from
``layout``), one segment at a time.

Tensors are numpy arrays of raw codes: uint32 for f32, uint16 for bf16, uint8
for f8e4m3 (fp32 values for scale tensors are uint32 codes too).
"""

from __future__ import annotations

import numpy as np

from . import casts
from .layout import DTYPE_BYTES, Layout, Placement
from .plan import Plan

CODE_DTYPE = {"f32": np.uint32, "bf16": np.uint16, "f8e4m3": np.uint8}


def local_index(p: Placement, i, j):
    """Flat local index of checkpoint element (i, j) under placement p."""
    if p.tr:
        return p.base + (j - p.c0) * p.ld + (i - p.r0)
    return p.base + (i - p.r0) * p.ld + (j - p.c0)


def _grid(r0, r1, c0, c1):
    return np.arange(r0, r1, dtype=np.int64)[:, None], np.arange(c0, c1, dtype=np.int64)[None, :]


def materialize(layout: Layout, rank: int, values, dtype=None) -> list[np.ndarray]:
    """Local tensors of one rank filled from the checkpoint (what a weight
    loader does). ``values(t)`` returns checkpoint tensor t as a [rows, cols]
    array of codes in the local dtype (or of ``dtype`` when given, e.g. element
    identifiers). Unplaced elements are zero."""
    rk = layout.ranks[rank]
    out = [np.zeros(lc.numel, dtype=dtype or CODE_DTYPE[lc.dtype]) for lc in rk.locals]
    for p in rk.placements:
        i, j = _grid(p.r0, p.r1, p.c0, p.c1)
        out[p.u][local_index(p, i, j)] = values(p.t)[p.r0:p.r1, p.c0:p.c1]
    return out


def pack(plan: Plan, s: int, trainer_locals: list[np.ndarray], rnd: int = 0) -> np.ndarray:
    """Send buffer of trainer rank s in round ``rnd``: every segment's
    rectangle, read through the sender's placement, written row-major at its
    send offset."""
    rounds = plan.rounds or [None]
    buf = np.zeros((rounds[rnd].send_bytes if rounds[rnd] else plan.send_bytes)[s], dtype=np.uint8)
    rk = plan.trainer.ranks[s]
    for g in plan.segments:
        if g.s != s or g.round != rnd or g.stage != 0:
            continue
        p = rk.placements[g.src_pl]
        lc = rk.locals[p.u]
        r = g.rect
        i, j = _grid(r.r0, r.r1, r.c0, r.c1)
        vals = trainer_locals[p.u][local_index(p, i, j)]          # [rows, cols] codes
        buf[g.send_off:g.send_off + g.nbytes] = np.ascontiguousarray(vals).view(np.uint8).ravel()
        assert vals.dtype == CODE_DTYPE[lc.dtype]
    return buf


def network(plan: Plan, d: int, send_bufs: dict[int, np.ndarray], rnd: int = 0, stage: int = 0,
            into: np.ndarray | None = None) -> np.ndarray:
    """Receive buffer of rollout rank d in round ``rnd`` after ``stage``: each
    sender's region for d in that stage copied into its section (into
    ``into`` when given, else into a new zeroed buffer). Stage 0 senders are
    trainer ranks; exchange-stage senders are rollout ranks and ``send_bufs``
    holds their forward buffers of that stage."""
    rounds = plan.rounds or [None]
    buf = into if into is not None else np.zeros(
        (rounds[rnd].recv_bytes if rounds[rnd] else plan.recv_bytes)[d], dtype=np.uint8)
    for g in plan.segments:
        if g.d == d and g.round == rnd and g.stage == stage:
            buf[g.recv_off:g.recv_off + g.nbytes] = send_bufs[g.s][g.send_off:g.send_off + g.nbytes]
    return buf


def forward(plan: Plan, r: int, recv_buf: np.ndarray, stage: int, rnd: int = 0) -> np.ndarray:
    """Forward buffer of rollout rank r for exchange ``stage`` (1 external, 2
    internal) in round ``rnd``: each forwarded segment's bytes, copied from
    where r received them, at the segment's send offset."""
    buf = np.zeros(plan.rounds[rnd].fwd_bytes[stage - 1][r], dtype=np.uint8)
    for g in plan.segments:
        if g.s == r and g.round == rnd and g.stage == stage:
            buf[g.send_off:g.send_off + g.nbytes] = recv_buf[g.src_off:g.src_off + g.nbytes]
    return buf


def run_stages(plan: Plan, trainer_locals: dict[int, list[np.ndarray]], rnd: int = 0) -> dict[int, np.ndarray]:
    """Every rollout rank's receive buffer for round ``rnd`` after the receive
    stage and, for plans with exchange stages, the external and internal
    exchanges, each stage starting when the previous one has landed."""
    nd = plan.rollout.nranks
    sends = {s: pack(plan, s, trainer_locals[s], rnd) for s in trainer_locals}
    recv = {d: network(plan, d, sends, rnd) for d in range(nd)}
    if plan.node_size:
        for stage in (1, 2):
            fwd = {r: forward(plan, r, recv[r], stage, rnd) for r in range(nd)}
            for d in range(nd):
                network(plan, d, fwd, rnd, stage, into=recv[d])
    return recv


def _convert(codes: np.ndarray, src: str, dst: str) -> np.ndarray:
    if src == dst:
        return codes
    if src == "f32" and dst == "bf16":
        return casts.f32_to_bf16(codes)
    if src == "bf16" and dst == "f32":
        return casts.bf16_to_f32(codes)
    raise ValueError(f"unsupported cast {src} -> {dst}")


def _to_f32(codes: np.ndarray, src: str) -> np.ndarray:
    return codes.astype(np.uint32) if src == "f32" else casts.bf16_to_f32(codes)


def _quantize_local(lc, staged_f32_codes: np.ndarray):
    """Blockwise quantisation of one staged local tensor (per batch matrix)."""
    x = staged_f32_codes.view(np.float32).reshape(lc.batch, lc.rows, lc.cols)
    codes = np.empty((lc.batch, lc.rows, lc.cols), dtype=np.uint8)
    nbr, nbc = -(-lc.rows // lc.block), -(-lc.cols // lc.block)
    scales = np.empty((lc.batch, nbr, nbc), dtype=np.float32)
    for e in range(lc.batch):
        codes[e], scales[e] = casts.quantize_matrix(x[e], lc.block)
    return codes.ravel(), scales.ravel().view(np.uint32)


def _finish(rk, staged, dst_locals):
    for u, lc in enumerate(rk.locals):
        if lc.block:
            codes, scales = _quantize_local(lc, staged[u])
            dst_locals[u] = codes
            dst_locals[lc.scale] = scales
    return dst_locals


def unpack(plan: Plan, d: int, recv_buf, rounds=None) -> list[np.ndarray]:
    """Rollout rank d's tensors from its receive buffer(s): each segment's
    payload is read row-major and written through the receiver's placement,
    cast to the local dtype; quantised tensors are staged in fp32 and quantised
    blockwise. With rounds, ``recv_buf`` is the list of the rounds' buffers."""
    rk = plan.rollout.ranks[d]
    dst = [np.zeros(lc.numel, dtype=CODE_DTYPE[lc.dtype]) for lc in rk.locals]
    staged = {u: np.zeros(lc.numel, dtype=np.uint32) for u, lc in enumerate(rk.locals) if lc.block}
    bufs = recv_buf if isinstance(recv_buf, list) else [recv_buf]
    for g in plan.segments:
        if g.d != d:
            continue
        recv_buf = bufs[g.round]
        q = rk.placements[g.dst_pl]
        lc = rk.locals[q.u]
        src_dtype = g.wire                                       # the trainer dtype the bytes travel in
        r = g.rect
        payload = recv_buf[g.recv_off:g.recv_off + g.nbytes].view(CODE_DTYPE[src_dtype])
        payload = payload.reshape(r.r1 - r.r0, r.c1 - r.c0)
        i, j = _grid(r.r0, r.r1, r.c0, r.c1)
        idx = local_index(q, i, j)
        if lc.block:
            staged[q.u][idx] = _to_f32(payload, src_dtype)
        else:
            dst[q.u][idx] = _convert(payload, src_dtype, lc.dtype)
    return _finish(rk, staged, dst)


def expected_rollout(rollout: Layout, d: int, values, src_dtype: str) -> list[np.ndarray]:
    """What rollout rank d must hold, straight from its layout and the
    checkpoint (no plan involved): dst = cast(checkpoint slice)."""
    rk = rollout.ranks[d]
    dst = [np.zeros(lc.numel, dtype=CODE_DTYPE[lc.dtype]) for lc in rk.locals]
    staged = {u: np.zeros(lc.numel, dtype=np.uint32) for u, lc in enumerate(rk.locals) if lc.block}
    for q in rk.placements:
        lc = rk.locals[q.u]
        i, j = _grid(q.r0, q.r1, q.c0, q.c1)
        idx = local_index(q, i, j)
        src = values(q.t)[q.r0:q.r1, q.c0:q.c1]
        if lc.block:
            staged[q.u][idx] = _to_f32(src, src_dtype)
        else:
            dst[q.u][idx] = _convert(src, src_dtype, lc.dtype)
    return _finish(rk, staged, dst)


def bytes_of(layout: Layout, rank: int) -> int:
    return sum(lc.numel * DTYPE_BYTES[lc.dtype] for lc in layout.ranks[rank].locals)
