"""Full-size parity of the five workloads, in the launch configuration the
benchmark times (same plans, same kernels, same buffers).

For each workload every sender that feeds the unpacked rollout rank is
packed for real and its region copied into the receive buffer; then:
* pack output of the benchmarked sender: every payload byte equals the
  checkpoint rectangle built with torch slicing on the GPU, and no byte
  between payloads is written;
* unpack output: every element of every rollout tensor equals the cast of its
  checkpoint slice built with torch on the GPU (torch's fp32 -> bf16 cast; for
  fp8 tensors torch's blockwise amax / 448, x / s, E4M3FN formula), so no
  element is left unwritten;
* unpack output against the oracle, every element of every tensor that is
  not fp8: the oracle's placement formula (local_index) evaluated on index
  tensors on the GPU gives each element's position, and its value is the
  checkpoint element (copies) or the oracle's fp32 -> bf16 rounding, which is
  elementwise and so is evaluated once per distinct fp32 value of the tensor;
* fp8 tensors against the oracle: every expert matrix of every layer
  (routed w13 and w2, the shared expert's) staged through the oracle's
  placement formula and quantised by the oracle's quantize_matrix in a pool
  of host processes, codes and scales compared in full;
* sampled elements and whole fp8 blocks are computed one by one by the CPU
  oracle from the numpy generator and compared.
"""

import os

import numpy as np
import pytest
import torch

import paper_2609_25442_amd as wb
import synthetic_checkpoint as sc
from oracle import casts
from oracle.layout import layout_from_spec
from oracle.plan import build_plan
from oracle.transfer import CODE_DTYPE, local_index
from synthetic_checkpoint.workloads import ORDER, WORKLOADS

from gpu_util import FILL, SIGNED, say, workspace_for

pytestmark = pytest.mark.gpu

SENTINEL = {"f32": 0xFF, "bf16": 0xFF, "f8e4m3": 0x7F}


def _rect(cat, t, r0, r1, c0, c1, dtype):
    rows, cols = cat[t].rows, cat[t].cols
    block = sc.values_torch(t, rows, cols, dtype, device="cuda", start=r0 * cols, count=(r1 - r0) * cols)
    return block.view(r1 - r0, cols)[:, c0:c1]


def _view(flat, p):
    if p.tr:
        return torch.as_strided(flat, (p.r1 - p.r0, p.c1 - p.c0), (1, p.ld), p.base)
    return torch.as_strided(flat, (p.r1 - p.r0, p.c1 - p.c0), (p.ld, 1), p.base)


def _sender_locals(otr, s, dtype):
    rk = otr.ranks[s]
    locs = [torch.zeros(lc.numel, dtype=wb.torch_dtype(lc.dtype), device="cuda") for lc in rk.locals]
    for p in rk.placements:
        _view(locs[p.u], p).copy_(_rect(otr.catalog, p.t, p.r0, p.r1, p.c0, p.c1, dtype))
    return locs


def _check_pack(oplan, s, send, dtype, cat):
    mask = torch.zeros(send.numel(), dtype=torch.bool, device="cuda")
    es = {"f32": 4, "bf16": 2}[dtype]
    for g in oplan.segments:
        if g.s != s:
            continue
        r = g.rect
        got = send[g.send_off:g.send_off + g.nbytes].view(wb.torch_dtype(dtype)).view(r.r1 - r.r0, r.c1 - r.c0)
        want = _rect(cat, g.t, r.r0, r.r1, r.c0, r.c1, dtype)
        assert torch.equal(got.view(SIGNED[dtype][1]), want.contiguous().view(SIGNED[dtype][1])), f"payload t={g.t}"
        mask[g.send_off:g.send_off + g.nbytes] = True
        assert g.nbytes == r.numel * es
    assert not bool(((send != FILL) & ~mask).any()), "pack wrote outside its payloads"


def _torch_quant(staged, lc):
    B = lc.block
    x = staged.view(lc.batch, lc.rows, lc.cols)
    pr, pc = (-lc.rows) % B, (-lc.cols) % B
    if pr or pc:
        x = torch.nn.functional.pad(x, (0, pc, 0, pr))
    nbr, nbc = x.shape[1] // B, x.shape[2] // B
    xb = x.view(lc.batch, nbr, B, nbc, B)
    amax = xb.abs().amax(dim=(2, 4))
    s = torch.where(amax > 0, amax / torch.full_like(amax, 448.0), torch.ones_like(amax))
    q = (xb / s[:, :, None, :, None]).to(torch.float8_e4m3fn).view(lc.batch, nbr * B, nbc * B)
    return q[:, :lc.rows, :lc.cols].contiguous(), s


def _check_unpack_full(oro, d, dst, cat, src_dtype):
    rk = oro.ranks[d]
    staged = {}
    for p in rk.placements:
        lc = rk.locals[p.u]
        want = _rect(cat, p.t, p.r0, p.r1, p.c0, p.c1, src_dtype)
        if lc.block:
            st = staged.setdefault(p.u, torch.zeros(lc.numel, dtype=torch.float32, device="cuda"))
            _view(st, p).copy_(want.float())
            continue
        got = _view(dst[p.u].view(-1), p)
        want = want.to(wb.torch_dtype(lc.dtype))
        assert torch.equal(got.view(SIGNED[lc.dtype][1]), want.contiguous().view(SIGNED[lc.dtype][1])), lc.name
    for u, st in staged.items():
        lc = rk.locals[u]
        q, s = _torch_quant(st, lc)
        assert torch.equal(dst[u].view(-1).view(torch.uint8), q.view(-1).view(torch.uint8)), f"{lc.name} codes"
        assert torch.equal(dst[lc.scale].view(-1).view(torch.int32), s.reshape(-1).view(torch.int32)), f"{lc.name} scales"


class _OracleCast:
    """The oracle's elementwise cast applied to GPU tensors of codes: each
    distinct code is cast once by the oracle on the host, and the results are
    kept (sorted by code) and gathered back on the GPU."""

    def __init__(self, src, dst, device="cuda"):
        if (src, dst) == ("f32", "bf16"):
            self.fn = casts.f32_to_bf16
        elif (src, dst) == ("bf16", "f32"):
            self.fn = casts.bf16_to_f32
        else:
            raise ValueError(f"no cast {src} -> {dst}")
        self.src, self.dst = src, dst
        self.keys = torch.empty(0, dtype=SIGNED[src][1], device=device)
        self.vals = torch.empty(0, dtype=SIGNED[dst][1], device=device)

    def __call__(self, codes):
        uniq = torch.unique(codes.reshape(-1))
        new = uniq[~torch.isin(uniq, self.keys)]
        if new.numel():
            out = self.fn(new.cpu().numpy().view(CODE_DTYPE[self.src]))
            out = torch.from_numpy(np.ascontiguousarray(out).view(SIGNED[self.dst][0])).to(self.keys.device)
            keys = torch.cat([self.keys, new])
            order = torch.argsort(keys)
            self.keys, self.vals = keys[order], torch.cat([self.vals, out])[order]
        return self.vals[torch.searchsorted(self.keys, codes.reshape(-1))].view(codes.shape)


def _oracle_index(p, device="cuda"):
    """Flat local positions of a placement's rectangle by the oracle's formula,
    evaluated on GPU index tensors."""
    i = torch.arange(p.r0, p.r1, dtype=torch.int64, device=device)[:, None]
    j = torch.arange(p.c0, p.c1, dtype=torch.int64, device=device)[None, :]
    return local_index(p, i, j)


def _check_unpack_oracle(oro, d, dst, cat, src_dtype, device="cuda"):
    """Every element of every non-fp8 rollout tensor against the oracle (the
    placements cover each tensor exactly, so this is every element)."""
    rk = oro.ranks[d]
    by_t = {}
    for p in rk.placements:
        if not rk.locals[p.u].block:
            by_t.setdefault(p.t, []).append(p)
    n = 0
    cast = {}
    for t, pls in sorted(by_t.items()):
        T = sc.values_torch(t, cat[t].rows, cat[t].cols, src_dtype, device=device).view(cat[t].rows, cat[t].cols)
        T = T.view(SIGNED[src_dtype][1])
        for p in pls:
            lc = rk.locals[p.u]
            want = T[p.r0:p.r1, p.c0:p.c1].contiguous()
            if lc.dtype != src_dtype:
                want = cast.setdefault(lc.dtype, _OracleCast(src_dtype, lc.dtype, device))(want)
            got = dst[p.u].reshape(-1).view(SIGNED[lc.dtype][1])[_oracle_index(p, device)]
            if not torch.equal(got, want):
                bad = torch.nonzero(got != want)[:5].tolist()
                raise AssertionError(f"{lc.name}: placement of tensor {t} rows {p.r0}:{p.r1} cols {p.c0}:{p.c1}: "
                                     f"first mismatches at {bad}")
            n += p.numel
        del T
    return n


def _check_fp8_oracle(oro, d, dst, cat, src_dtype, prefixes, workers, device="cuda"):
    """Every fp8 tensor whose name starts with one of ``prefixes`` (one layer
    each, taken in turn to bound host memory) against the oracle: each batch
    matrix staged in fp32 through the oracle's placement formula, quantised by
    casts.quantize_matrix in host processes, codes and scales compared in
    full. Returns the number of matrices compared."""
    import concurrent.futures as cf
    import multiprocessing as mp

    rk = oro.ranks[d]
    done = 0
    with cf.ProcessPoolExecutor(max_workers=workers, mp_context=mp.get_context("spawn")) as pool:
        for prefix in prefixes:
            futs = []
            for u, lc in enumerate(rk.locals):
                if not lc.block or not lc.name.startswith(prefix):
                    continue
                staged = torch.zeros(lc.numel, dtype=torch.float32, device=device)
                for p in rk.placements:
                    if p.u == u:
                        x = sc.values_torch(p.t, cat[p.t].rows, cat[p.t].cols, src_dtype, device=device,
                                            start=p.r0 * cat[p.t].cols, count=(p.r1 - p.r0) * cat[p.t].cols)
                        staged[_oracle_index(p, device)] = x.view(p.r1 - p.r0, cat[p.t].cols)[:, p.c0:p.c1].float()
                staged = staged.view(lc.batch, lc.rows, lc.cols)
                for e in range(lc.batch):
                    futs.append((u, e, pool.submit(casts.quantize_matrix, staged[e].cpu().numpy(), lc.block)))
                del staged
            assert futs, f"no fp8 tensors under {prefix}"
            for u, e, f in futs:
                codes, scales = f.result()
                lc = rk.locals[u]
                got = dst[u][e] if lc.batch > 1 else dst[u]
                got = got.reshape(-1).view(torch.uint8).cpu().numpy()
                assert np.array_equal(got, codes.ravel()), f"{lc.name}[{e}] codes differ from the oracle"
                sl = dst[lc.scale][e] if lc.batch > 1 else dst[lc.scale]
                assert np.array_equal(sl.reshape(-1).view(torch.int32).cpu().numpy(),
                                      np.ascontiguousarray(scales).ravel().view(np.int32)), f"{lc.name}[{e}] scales"
            done += len(futs)
            say(f"  {prefix}: {len(futs)} fp8 matrices equal the oracle's")
    return done


def _oracle_value(t, i, j, cat, src_dtype):
    return sc.values_numpy(t, np.asarray(i) * cat[t].cols + np.asarray(j), src_dtype)


def _check_unpack_sampled(oro, d, dst, cat, src_dtype, rng, n_pl=120, per_pl=16, n_blocks=6):
    rk = oro.ranks[d]
    plain = [k for k, p in enumerate(rk.placements) if not rk.locals[p.u].block]
    for k in rng.choice(plain, min(n_pl, len(plain)), replace=False) if plain else []:
        p = rk.placements[k]
        lc = rk.locals[p.u]
        i = rng.integers(p.r0, p.r1, per_pl)
        j = rng.integers(p.c0, p.c1, per_pl)
        src = _oracle_value(p.t, i, j, cat, src_dtype)
        if lc.dtype == src_dtype:
            want = src
        elif src_dtype == "f32" and lc.dtype == "bf16":
            want = casts.f32_to_bf16(src)
        else:
            want = casts.bf16_to_f32(src)
        idx = torch.from_numpy(local_index(p, i, j)).cuda()
        got = dst[p.u].view(-1).view(SIGNED[lc.dtype][1])[idx].cpu().numpy().view(CODE_DTYPE[lc.dtype])
        assert np.array_equal(got, want), (lc.name, p)
    qlocals = [u for u, lc in enumerate(rk.locals) if lc.block]
    for _ in range(n_blocks if qlocals else 0):
        u = int(rng.choice(qlocals))
        lc = rk.locals[u]
        B = lc.block
        e = int(rng.integers(0, lc.batch))
        bi = int(rng.integers(0, -(-lc.rows // B)))
        bj = int(rng.integers(0, -(-lc.cols // B)))
        rr = np.arange(bi * B, min(lc.rows, (bi + 1) * B))
        cc = np.arange(bj * B, min(lc.cols, (bj + 1) * B))
        f = (e * lc.rows + rr[:, None]) * lc.cols + cc[None, :]
        vals = np.zeros(f.shape, dtype=np.uint32)
        seen = np.zeros(f.shape, dtype=bool)
        for p in rk.placements:
            if p.u != u or p.tr:
                continue
            rel = f - p.base
            i = rel // p.ld + p.r0
            j = rel % p.ld + p.c0
            hit = (rel >= 0) & (i < p.r1) & (j < p.c1)
            if hit.any():
                src = _oracle_value(p.t, i[hit], j[hit], cat, src_dtype)
                vals[hit] = src.astype(np.uint32) if src_dtype == "f32" else casts.bf16_to_f32(src)
                seen |= hit
        assert seen.all()
        codes, s = casts.quantize_block(vals.view(np.float32))
        fi = torch.from_numpy(f.ravel()).cuda()
        got = dst[u].view(-1).view(torch.uint8)[fi].cpu().numpy().reshape(f.shape)
        assert np.array_equal(got, codes), (lc.name, e, bi, bj)
        sidx = (e * -(-lc.rows // B) + bi) * -(-lc.cols // B) + bj
        assert np.float32(dst[lc.scale].view(-1)[sidx].item()) == s


@pytest.mark.timeout(900)
@pytest.mark.parametrize("name", ORDER)
def test_full_size_workload(name):
    w = WORKLOADS[name]
    src_dtype = w["trainer"]["dtype"]
    s0, d = w["pack_rank"], w["unpack_rank"]
    otr = layout_from_spec(w["model"], w["trainer"])
    oro = layout_from_spec(w["model"], w["rollout"])
    oplan = build_plan(otr, oro)
    cat = otr.catalog
    tr = wb.Layout.describe(w["model"], w["trainer"])
    ro = wb.Layout.describe(w["model"], w["rollout"])
    rplan = wb.Plan(tr, ro, wb.RECEIVER, d)
    rws = workspace_for(rplan)
    rplan.upload(rws)
    recv = torch.empty(rplan.buffer_bytes, dtype=torch.uint8, device="cuda")
    say(f"[{name}] receive buffer {rplan.buffer_bytes / 1e9:.2f} GB")
    for s in range(otr.nranks):
        so, roff, nb = rplan.region(s, d)
        if nb == 0 and s != s0:
            continue
        say(f"[{name}] pack sender {s}")
        locs = _sender_locals(otr, s, src_dtype)
        p = wb.Plan(tr, ro, wb.SENDER, s)
        ws = workspace_for(p)
        p.upload(ws)
        send = torch.full((p.buffer_bytes,), FILL, dtype=torch.uint8, device="cuda")
        p.pack(locs, send)
        torch.cuda.synchronize()
        if s == s0:
            say(f"[{name}] check pack of sender {s} ({p.buffer_bytes / 1e9:.2f} GB)")
            _check_pack(oplan, s, send, src_dtype, cat)
        if nb:
            recv[roff:roff + nb] = send[so:so + nb]
        del locs, send, p, ws
        torch.cuda.synchronize()
    dst = wb.allocate_locals(ro, d)
    for t, lc in zip(dst, oro.ranks[d].locals):
        t.view(torch.uint8).fill_(SENTINEL[lc.dtype])
    say(f"[{name}] unpack receiver {d}")
    rplan.unpack(recv, dst)
    torch.cuda.synchronize()
    say(f"[{name}] full check against torch")
    _check_unpack_full(oro, d, dst, cat, src_dtype)
    say(f"[{name}] every non-fp8 element against the oracle")
    n = _check_unpack_oracle(oro, d, dst, cat, src_dtype)
    say(f"[{name}] {n} elements equal the oracle's")
    if any(lc.block for lc in oro.ranks[d].locals):
        workers = max(1, min(15, (os.cpu_count() or 2) - 1))
        nl = w["model"]["num_layers"]
        say(f"[{name}] fp8 tensors of all {nl} layers against the oracle ({workers} host processes)")
        m = _check_fp8_oracle(oro, d, dst, cat, src_dtype, [f"layers.{k}." for k in range(nl)], workers)
        say(f"[{name}] {m} fp8 matrices equal the oracle's")
    say(f"[{name}] sampled check against the oracle")
    _check_unpack_sampled(oro, d, dst, cat, src_dtype, np.random.default_rng(11))
    del recv, dst
    torch.cuda.empty_cache()
