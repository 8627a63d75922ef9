"""Benchmark of the resharding hot path on one MI355X.

One step = pack of one trainer rank's shards (wb_pack) followed by the
assembly of one rollout rank's tensors (wb_unpack), on synthetic seeded
parameters already resident in HBM. The headline workload is the largest
one that fits one GPU, Mixtral-8x7B-shaped (trainer EP=8 x FSDP=2 flat fp32
shards -> rollout EP=2 bf16 with stacked experts; pack trainer rank 0,
unpack rollout rank 0 from the sixteen senders' regions: 169 GB per step).
Other workloads: --workload NAME.

Prints one JSON line: effective GB/s of the step (algorithmic bytes: each
element read once in the source dtype and written once in the destination
dtype, plus fp8 scales), the HBM roofline of the dominant kernel from HIP
events on the launch stream, wb_plan time, this GPU's stream ceilings
(measured first, in a child process) with the dominant kernel's fraction of the
one-shot stream of its read/write mix, the CPU oracle timed on bounded
samples of the same workload (unpack and pack), and ``per_config``: every
workload timed in the same run (fewer steps each), its pack and unpack rates,
roofline fraction and plan time.
"""

from __future__ import annotations

import argparse
import hashlib
import json
import os
import statistics
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0          # MI355X HBM3E, 8 TB/s
DEFAULT_WORKLOAD = "mixtral_ep8fsdp2_to_ep2"


def log(*a):
    print(*a, file=sys.stderr, flush=True)


def build_sender_locals(wb, torch, sc, layout, rank, dtype):
    """Trainer rank's local tensors filled from the synthetic checkpoint through
    its placements (plain torch slicing; what a trainer's weights look like)."""
    cat = layout.tensors()
    locs = wb.allocate_locals(layout, rank, zero=True)
    flat = [t.view(-1) for t in locs]
    for (t, r0, r1, c0, c1, u, base, ld, tr) in layout.placements(rank):
        _, rows, cols = cat[t]
        block = sc.values_torch(t, rows, cols, dtype, device="cuda", start=r0 * cols, count=(r1 - r0) * cols)
        block = block.view(r1 - r0, cols)[:, c0:c1]
        if tr:
            view = torch.as_strided(flat[u], (r1 - r0, c1 - c0), (1, ld), base)
        else:
            view = torch.as_strided(flat[u], (r1 - r0, c1 - c0), (ld, 1), base)
        view.copy_(block)
    return locs


def work_fingerprint(workload):
    """What the committed HBM-traffic counters of a workload depend on: the
    kernels' source and the benchmarked plans' work tables (work-item counts and
    algorithmic bytes of every launch, under the current task size). The
    counters are reported only while this is unchanged."""
    from synthetic_checkpoint.workloads import WORKLOADS

    h = hashlib.sha256()
    h.update(open(os.path.join(ROOT, "paper_2609_25442_amd", "csrc", "kernels.hip"), "rb").read())
    grids, _ = _launch_grids(WORKLOADS[workload])
    h.update(repr(sorted(grids.items())).encode())
    h.update(os.environ.get("WB_TASK_BYTES", "").encode())
    return h.hexdigest()[:16]


def stored_traffic(workload, kernel, why=None):
    """HBM bytes per launch from committed rocprofv3 counter runs, if they were
    taken on the current kernel source (else None, with the reason appended to
    the list ``why`` when given)."""
    path = os.path.join(ROOT, "profiles", f"traffic-{workload}.txt")
    if not os.path.exists(path):
        if why is not None:
            why.append(f"no profiles/traffic-{workload}.txt")
        return None
    rec = json.load(open(path))
    fp = work_fingerprint(workload)
    if rec.get("work_fingerprint") != fp or kernel not in rec.get("kernels", {}):
        if why is not None:
            why.append(f"{kernel}: stored fingerprint {rec.get('work_fingerprint')} != current {fp}"
                       if rec.get("work_fingerprint") != fp else f"{kernel}: not in the stored counters")
        return None
    return rec["kernels"][kernel]["hbm_bytes_per_launch"]


def cpu_baseline(w, recv_host_fn, src_host_fn, unpack_budget_s=12.0, pack_budget_s=8.0,
                 max_tensor_bytes=256 << 20, wall_cap_s=90.0):
    """The oracle as it stands, on time-bounded samples of the workload: its
    planner, its element-by-element unpack of the receiver's tensors and its
    pack of the sender's segments.

    Unpack: one destination tensor at a time in layout order (every segment
    that feeds it, then its blockwise quantisation when it is fp8) until the
    unpack calls have taken ``unpack_budget_s`` seconds (or ``wall_cap_s`` of
    wall time have passed). Tensors above ``max_tensor_bytes`` (embeddings and
    output heads) are left out: the oracle's index arrays for them take
    gigabytes. Each segment's wire bytes are copied back to back into one
    reused, pre-touched host buffer by ``recv_host_fn(offset, nbytes, out)``
    (the segments re-based onto it), so the rate counts the oracle and not
    first-touch page faults.

    Pack: the sender's segments in send-buffer order, one oracle pack call
    per segment (re-based to offset 0), until ``pack_budget_s``; the local
    tensors they read are fetched once by ``src_host_fn(u)`` (not timed)."""
    import dataclasses

    import numpy as np

    from oracle.layout import DTYPE_BYTES, Layout
    from oracle.layout import layout_from_spec
    from oracle.plan import build_plan
    from oracle.transfer import pack as o_pack
    from oracle.transfer import unpack as o_unpack

    t0 = time.perf_counter()
    otr = layout_from_spec(w["model"], w["trainer"])
    oro = layout_from_spec(w["model"], w["rollout"])
    oplan = build_plan(otr, oro)
    plan_ms = (time.perf_counter() - t0) * 1e3
    d = w["unpack_rank"]
    rk = oro.ranks[d]
    by_local = {}
    for g in oplan.segments:
        if g.d == d:
            by_local.setdefault(rk.placements[g.dst_pl].u, []).append(g)
    sample, skipped = [], 0
    for u, lc in enumerate(rk.locals):
        segs = by_local.get(u)
        if not segs:
            continue
        if lc.numel * DTYPE_BYTES[lc.dtype] > max_tensor_bytes:
            skipped += 1
            continue
        sample.append((u, lc, segs))
    buf = np.ones(max(sum(g.nbytes for g in segs) for _, _, segs in sample), dtype=np.uint8)   # touched once
    done_bytes, spent, n_t, n_seg = 0, 0.0, 0, 0
    wall0 = time.perf_counter()
    for u, lc, segs in sample:
        # a receiver layout holding just this tensor (and its scale companion),
        # its segments re-based onto the reused buffer
        keep = [u] + ([lc.scale] if lc.block else [])
        sub_locals = [rk.locals[k] if k in keep else dataclasses.replace(rk.locals[k], batch=0) for k in range(len(rk.locals))]
        sub_rank = dataclasses.replace(rk, locals=sub_locals)
        sub_ro = Layout(oro.catalog, [sub_rank if r == d else oro.ranks[r] for r in range(oro.nranks)])
        segs0, pos = [], 0
        for g in segs:
            recv_host_fn(g.recv_off, g.nbytes, buf[pos:pos + g.nbytes])
            segs0.append(dataclasses.replace(g, recv_off=pos))
            pos += g.nbytes
        sub = dataclasses.replace(oplan, rollout=sub_ro, segments=segs0)
        t1 = time.perf_counter()
        o_unpack(sub, d, buf[:pos])
        spent += time.perf_counter() - t1
        done_bytes += sum(g.nbytes for g in segs) + lc.numel * DTYPE_BYTES[lc.dtype]
        if lc.block:
            done_bytes += rk.locals[lc.scale].numel * 4
        n_t += 1
        n_seg += len(segs)
        log(f"[cpu_baseline] {lc.name}: {n_t} tensors, {done_bytes / 1e9:.2f} GB in {spent:.1f} s")
        if spent >= unpack_budget_s or time.perf_counter() - wall0 >= wall_cap_s:
            break
    del buf
    # pack: the sender's segments in send order
    s0 = w["pack_rank"]
    mine = sorted((g for g in oplan.segments if g.s == s0 and g.stage == 0), key=lambda g: g.send_off)
    trk = otr.ranks[s0]
    host = [np.zeros(0, dtype=np.uint8)] * len(trk.locals)
    p_bytes, p_spent, p_seg, fetched = 0, 0.0, 0, set()
    wall1 = time.perf_counter()
    for g in mine:
        u = trk.placements[g.src_pl].u
        if u not in fetched:
            host = list(host)
            host[u] = src_host_fn(u)
            fetched.add(u)
        sub = dataclasses.replace(oplan, segments=[dataclasses.replace(g, send_off=0)], rounds=None,
                                  send_bytes=[g.nbytes if r == s0 else 0 for r in range(otr.nranks)])
        t1 = time.perf_counter()
        o_pack(sub, s0, host)
        p_spent += time.perf_counter() - t1
        p_bytes += 2 * g.nbytes
        p_seg += 1
        if p_spent >= pack_budget_s or time.perf_counter() - wall1 >= wall_cap_s:
            break
    log(f"[cpu_baseline] pack: {p_seg} segments, {p_bytes / 1e9:.2f} GB in {p_spent:.1f} s")
    try:
        affinity = len(os.sched_getaffinity(0))
    except AttributeError:
        affinity = None
    total = done_bytes + p_bytes
    return {"value": round(total / (spent + p_spent) / 1e9, 4), "unit": "GB/s", "cores": 1, "kind": "oracle",
            "sample": f"oracle unpack of the first {n_t} rollout tensors of rank {d} of at most "
                      f"{max_tensor_bytes >> 20} MiB ({skipped} larger ones left out; {n_seg} segments, "
                      f"{done_bytes / 1e9:.2f} GB read+written in {spent:.1f} s) and oracle pack of the first "
                      f"{p_seg} of trainer rank {s0}'s {len(mine)} segments ({p_bytes / 1e9:.2f} GB read+written "
                      f"in {p_spent:.1f} s), single-threaded numpy; oracle plan {plan_ms:.0f} ms",
            "unpack": {"GB/s": round(done_bytes / spent / 1e9, 4), "bytes": done_bytes, "s": round(spent, 2)},
            "pack": {"GB/s": round(p_bytes / p_spent / 1e9, 4) if p_spent else None, "bytes": p_bytes,
                     "s": round(p_spent, 2)},
            "host_cpu_count": os.cpu_count(), "host_affinity_cpus": affinity,
            "plan_ms": round(plan_ms, 1)}


def _read_csv(path):
    import csv

    with open(path, newline="") as f:
        return list(csv.DictReader(f))


def _launch_grids(w):
    """Grid sizes (threads) of the pack and unpack launches of a workload,
    from the library's host planner (no GPU needed)."""
    import paper_2609_25442_amd as wb

    tr = wb.Layout.describe(w["model"], w["trainer"])
    ro = wb.Layout.describe(w["model"], w["rollout"])
    rp = wb.Plan(tr, ro, wb.RECEIVER, w["unpack_rank"])
    sp = wb.Plan(tr, ro, wb.SENDER, w["pack_rank"])
    def threads_x(plan, launch):
        # rocprofv3 reports grid sizes in threads: the kernel trace per
        # dimension (Grid_Size_X), the counter collection the product (Grid_Size)
        x, y, t = plan.launch_grid(launch)
        return x * t, x * max(y, 1) * t

    return {"pack": (threads_x(sp, 0), "wb_tasks_kernel", sp.kernel_traffic(0)),
            "pack_tiles": (threads_x(sp, 4), "wb_tile_kernel", sp.kernel_traffic(4)),
            "unpack": (threads_x(rp, 0), "wb_tasks_kernel", rp.kernel_traffic(0)),
            "unpack_tiles": (threads_x(rp, 4), "wb_tile_kernel", rp.kernel_traffic(4)),
            "unpack_fp8": (threads_x(rp, 1), "wb_qblock_kernel", rp.kernel_traffic(1))}, rp.buffer_bytes


def summarize_counters(workload, fetch_csv, write_csv):
    """HBM bytes per launch of the pack and unpack kernels from two rocprofv3
    --pmc runs of this benchmark (FETCH_SIZE, then WRITE_SIZE, KiB per
    dispatch), each scaled by what the counter reads for the benchmark's plain
    device copy of known size."""
    from synthetic_checkpoint.workloads import WORKLOADS

    grids, recv_bytes = _launch_grids(WORKLOADS[workload])
    copy_bytes = min(recv_bytes, 16 << 30)
    out = {"workload": workload, "work_fingerprint": work_fingerprint(workload), "kernels": {}, "calibration": {}}
    per = {}
    for counter, path in (("FETCH_SIZE", fetch_csv), ("WRITE_SIZE", write_csv)):
        rows = [r for r in _read_csv(path) if r["Counter_Name"] == counter]
        copies = [float(r["Counter_Value"]) for r in rows if "copyBuffer" in r["Kernel_Name"]]
        copies = sorted(copies)[-3:]                       # the timed reference copies
        factor = statistics.mean(copies) * 1024 / copy_bytes
        out["calibration"][counter] = {"copy_bytes": copy_bytes, "copy_kib": statistics.mean(copies),
                                       "factor": round(factor, 5)}
        for label, ((_, total), kname, _) in grids.items():
            vals = [float(r["Counter_Value"]) for r in rows
                    if kname in r["Kernel_Name"] and int(r["Grid_Size"]) == total and total > 0]
            if vals:
                per.setdefault(label, {})[counter] = (statistics.mean(vals), len(vals), factor)
    for label, c in per.items():
        if "FETCH_SIZE" not in c or "WRITE_SIZE" not in c:
            continue
        fk, n, ff = c["FETCH_SIZE"]
        wk, _, wf = c["WRITE_SIZE"]
        rd, wr = fk * 1024 / ff, wk * 1024 / wf
        alg = grids[label][2]
        out["kernels"][label] = {"dispatches": n, "fetch_kib": fk, "write_kib": wk, "hbm_read_bytes": round(rd),
                                 "hbm_write_bytes": round(wr), "hbm_bytes_per_launch": round(rd + wr),
                                 "algorithmic_bytes": (alg[0] + alg[1]) if alg else None}
    return out


# kernel-trace columns that describe a launch's resources (registers, LDS,
# workgroup size), reported with its durations
_RESOURCE_COLUMNS = ("Workgroup_Size", "Workgroup_Size_X", "VGPR_Count", "Arch_VGPR_Count", "Accum_VGPR_Count",
                     "SGPR_Count", "LDS_Block_Size", "Scratch_Size")


def summarize_metric(workload, name, csv_path):
    """Mean of one rocprofv3 --pmc counter or derived metric (e.g.
    MeanOccupancyPerCU) per pack and unpack launch of this benchmark."""
    from synthetic_checkpoint.workloads import WORKLOADS

    grids, _ = _launch_grids(WORKLOADS[workload])
    rows = [r for r in _read_csv(csv_path) if r["Counter_Name"] == name]
    out = {"workload": workload, "metric": name, "kernels": {}}
    for label, ((_, total), kname, _) in grids.items():
        vals = [float(r["Counter_Value"]) for r in rows
                if kname in r["Kernel_Name"] and int(r["Grid_Size"]) == total and total > 0]
        if vals:
            out["kernels"][label] = {"dispatches": len(vals), "mean": round(statistics.mean(vals), 3)}
    return out


def summarize_trace(workload, trace_csv):
    """Per-launch durations of the pack, unpack and reference-copy kernels from
    a rocprofv3 --kernel-trace run of this benchmark."""
    from synthetic_checkpoint.workloads import WORKLOADS

    grids, recv_bytes = _launch_grids(WORKLOADS[workload])
    rows = _read_csv(trace_csv)
    res = {}
    for label, ((gx, _), kname, alg) in grids.items():
        ds = [(int(r["End_Timestamp"]) - int(r["Start_Timestamp"])) for r in rows
              if kname in r["Kernel_Name"] and int(r["Grid_Size_X"]) == gx and gx > 0]
        if ds:
            res[label] = {"launches": len(ds), "avg_us": round(statistics.mean(ds) / 1e3, 2),
                          "min_us": round(min(ds) / 1e3, 2), "max_us": round(max(ds) / 1e3, 2),
                          "GB/s_at_avg": round((alg[0] + alg[1]) / statistics.mean(ds), 1) if alg else None}
            first = next(r for r in rows if kname in r["Kernel_Name"] and int(r["Grid_Size_X"]) == gx)
            used = {k: int(first[k]) for k in _RESOURCE_COLUMNS if first.get(k, "").strip().isdigit()}
            if used:
                res[label]["resources"] = used
    copies = [(int(r["End_Timestamp"]) - int(r["Start_Timestamp"])) for r in rows if "copyBuffer" in r["Kernel_Name"]]
    if copies:
        top = sorted(copies)[-3:]
        res["device_copy"] = {"launches": len(top), "avg_us": round(statistics.mean(top) / 1e3, 2)}
    return res


def run_ceilings():
    """This GPU's stream ceilings (wb_ceilings, built from ceilings.hip by
    __graft_entry__.build(); a separate process: 2 x 8 GiB of device memory
    while it runs)."""
    import subprocess

    exe = os.path.join(ROOT, "wb_ceilings")
    return subprocess.run([exe], capture_output=True, text=True, timeout=300)


def run_plan_stress():
    """Host planning time on a DeepSeek-V3-like catalog of 58 MoE layers
    (44,776 checkpoint tensors), EP64 bf16 trainer -> EP8 fp8 rollout: median of
    five plans per role, with and without the exchange stages."""
    import paper_2609_25442_amd as wb
    from synthetic_checkpoint.workloads import WORKLOADS

    w = WORKLOADS["dsv3_ep64_to_ep8_fp8"]
    m = dict(w["model"], num_layers=58)
    tr = wb.Layout.describe(m, w["trainer"])
    ro = wb.Layout.describe(m, w["rollout"])
    out = {"metric": "wb_plan ms (58-layer DeepSeek-V3-like catalog)", "tensors": len(tr.tensors()), "plan_ms": {},
           "host_cpu_count": os.cpu_count(), "host_affinity_cpus": len(os.sched_getaffinity(0)),
           "plan_threads": os.environ.get("WB_PLAN_THREADS", "default (allowed CPUs, at most 16)")}
    for label, role, G in (("receiver", wb.RECEIVER, 0), ("sender", wb.SENDER, 0), ("receiver_exchange_G4", wb.RECEIVER, 4)):
        ts = []
        for _ in range(5):
            t0 = time.perf_counter()
            p = wb.Plan(tr, ro, role, 0, node_size=G)
            ts.append((time.perf_counter() - t0) * 1e3)
        out["plan_ms"][label] = {"median": round(statistics.median(ts), 1), "segments": p.num_segments,
                                 "work": p.work_counts()}
    print(json.dumps(out), flush=True)


def run_probe(args):
    """Source-map probing (App. B, Algorithm 1) of the benchmark's trainer and
    rollout ranks at full size, through the torch-slicing stand-in loaders;
    the recovered placements must equal the declared ones. Prints one JSON
    line: per-rank probe time, the passes, and the diff2 stencil's own rate
    (HIP events around its launches over every loaded local tensor)."""
    import torch

    import paper_2609_25442_amd as wb
    from synthetic_checkpoint import loaders
    from synthetic_checkpoint.workloads import WORKLOADS

    w = WORKLOADS[args.workload]
    dtype = w["trainer"]["dtype"]
    torch.cuda.set_device(0)
    out = {"metric": "source-map probe of one rank (ms); diff2 stencil GB/s", "workload": args.workload,
           "dtype": dtype, "data": "synthetic", "ranks": {}}
    for side, rank in (("trainer", w["pack_rank"]), ("rollout", w["unpack_rank"])):
        par = w[side]
        fn = loaders.STYLES[par["style"]]

        def load(T, fn=fn, par=par, rank=rank):
            return [x.contiguous() for x in fn(w["model"], par, T, rank) if x is not None]

        declared = wb.Layout.describe(w["model"], par)
        cat = declared.tensors()
        keep = [u for u, lc in enumerate(declared.locals(rank)) if lc["scales"] < 0]
        remap = {u: i for i, u in enumerate(keep)}
        want = sorted((t, r0, r1, c0, c1, remap[u], b, ld, tr)
                      for (t, r0, r1, c0, c1, u, b, ld, tr) in declared.placements(rank))
        modes = {}
        wb.probe_layout(cat, dtype, [load])  # untimed: loads the code objects of every launch
        # holding the passes needs the rank's loaded tensors once per pass
        # (and the identifier tensors it reads, about as large)
        es = {"f32": 4, "bf16": 2, "f8e4m3": 1}
        local_bytes = sum(lc["numel"] * es[dtype] for u, lc in enumerate(declared.locals(rank)) if u in keep)
        hold_fits = local_bytes * (wb.Probe(cat, dtype).num_chunks + 1) * 4 <= torch.cuda.mem_get_info()[0] * 3
        for hold in (True, False):
            if hold and not hold_fits:
                modes["held_passes"] = None
                log(f"[probe] {side} rank {rank} held_passes: skipped ({local_bytes / 1e9:.1f} GB per pass)")
                continue
            stats = {}
            torch.cuda.synchronize()
            t0 = time.perf_counter()
            got = wb.probe_layout(cat, dtype, [load], stats=stats, hold_passes=hold)
            ms = (time.perf_counter() - t0) * 1e3
            same = sorted(got.placements(0)) == want
            label = "held_passes" if hold else "carried_passes"
            log(f"[probe] {side} rank {rank} {label}: {ms:.0f} ms, recovered == declared: {same}")
            modes[label] = {"probe_ms": round(ms, 1), "recovered_equals_declared": same, "passes": stats[0],
                            "scan_ms": round(stats["scan_s"][0] * 1e3, 1),
                            "carry_retries": len(stats.get("carry_retries", []))}
            del got
        # the stencils alone: each carry pass over the loaded tensors of that
        # pass (pass by pass, since a pass reads the carries of the one before;
        # repeating a pass rewrites the same table from the same input), and,
        # when all passes fit on the device, one launch over all of them held;
        # a timed call includes the library's host work (tile table, its
        # upload and the wait for it), the field arrays are built beforehand
        probe = wb.Probe(cat, dtype)
        ids = wb._IdCheckpoint(cat, dtype, wb.torch_dtype(dtype), "cuda")
        cap = 1 << 21
        idx = torch.empty(cap, dtype=torch.int64, device="cuda")
        val = torch.empty(cap, dtype=torch.int64, device="cuda")
        count = torch.zeros(1, dtype=torch.int64, device="cuda")
        carries = torch.zeros(1, dtype=torch.int64, device="cuda")
        ev = [torch.cuda.Event(enable_timing=True) for _ in range(2)]
        stencil, held, ws = {}, [], None
        for k in range(probe.num_chunks):
            ids.start_pass(probe, k)
            locs = load(ids)  # may hold views of the identifier tensors: cloned only to be held
            if k == 0:
                shapes = [wb._view_shape(x) for x in locs]
                nbytes = sum(x.numel() * x.element_size() for x in locs)
                numel = sum(x.numel() for x in locs)
                ccap = 16 * (numel >> 16) + 64 * len(shapes) + 4096
                hold_all = nbytes * probe.num_chunks * 4 <= torch.cuda.mem_get_info()[0] * 3
            fields = wb._field_array([(x, dtype, b * rr, cc) for x, (b, rr, cc) in zip(locs, shapes)])
            if ws is None:
                ws = torch.empty(wb.diff2_carry_workspace(fields, ccap), dtype=torch.uint8, device="cuda")
            times = []
            for rep in range(4):
                ev[0].record()
                wb.diff2_carry(fields, k, k + 1 == probe.num_chunks, ccap, idx, val, count, carries, ws)
                ev[1].record()
                torch.cuda.synchronize()
                times.append(ev[0].elapsed_time(ev[1]))
            best = min(times[1:])
            rate = nbytes / (best * 1e-3) / 1e9
            got = (int(count.item()), int(carries.item()))
            stencil[f"carry_pass_{k}"] = {"bytes": nbytes, "entries": got[0], "carries": got[1],
                                          "carry_capacity": ccap, "workspace_bytes": ws.numel(),
                                          "ms": round(best, 3), "GB/s": round(rate, 1),
                                          "frac_of_hbm_peak": round(rate / HBM_PEAK_GBS, 4)}
            log(f"[probe] {side} diff2 carry pass {k}: {best:.3f} ms, {rate:.0f} GB/s, "
                f"{got[0]} entries, {got[1]} carries")
            if hold_all:
                held.append([x.clone() for x in locs])
            del fields, locs
        del ws, ids
        if hold_all:
            every = wb._field_array([([h[u] for h in held], dtype, b * rr, cc) for u, (b, rr, cc) in enumerate(shapes)])
            ws = torch.empty(wb.diff2_batch_workspace(every), dtype=torch.uint8, device="cuda")
            times = []
            for rep in range(4):
                ev[0].record()
                wb.diff2_batch(every, idx, val, count, ws)
                ev[1].record()
                torch.cuda.synchronize()
                times.append(ev[0].elapsed_time(ev[1]))
            best = min(times[1:])
            rate = nbytes * len(held) / (best * 1e-3) / 1e9
            stencil["all_passes"] = {"launches": 1, "bytes": nbytes * len(held), "entries": int(count.item()),
                                     "table_bytes": ws.numel(), "ms": round(best, 3), "GB/s": round(rate, 1),
                                     "frac_of_hbm_peak": round(rate / HBM_PEAK_GBS, 4)}
            log(f"[probe] {side} diff2 all_passes: {best:.3f} ms, {rate:.0f} GB/s, {int(count.item())} entries")
            del every, ws
        else:
            stencil["all_passes"] = None
            log(f"[probe] {side} diff2 all_passes: skipped ({probe.num_chunks} passes of {nbytes / 1e9:.1f} GB "
                f"do not fit on the device together)")
        out["ranks"][side] = {"rank": rank, "placements": len(want), "local_tensors": len(keep), **modes,
                              "diff2": stencil}
        del held, idx, val
        torch.cuda.empty_cache()
    print(json.dumps(out), flush=True)


def run_workload(args, name, steps, warmup, ceilings=None, with_cpu=False):
    """Build one workload's inputs in HBM, time ``steps`` steps after
    ``warmup``, and return its JSON record (with the CPU oracle's samples
    when ``with_cpu``). Frees the workload's device memory before returning."""
    import torch

    import paper_2609_25442_amd as wb
    import synthetic_checkpoint as sc
    from synthetic_checkpoint.workloads import WORKLOADS

    w = WORKLOADS[name]
    src_dtype = w["trainer"]["dtype"]
    s0, d = w["pack_rank"], w["unpack_rank"]
    torch.cuda.set_device(0)

    tr = wb.Layout.describe(w["model"], w["trainer"])
    ro = wb.Layout.describe(w["model"], w["rollout"])
    plan_ms = {}
    for label, role, rank in (("unpack", wb.RECEIVER, d), ("pack", wb.SENDER, s0)):
        # median of 20 plans (global plan plus rank view), fewer if they pass 3 s
        ts = []
        while len(ts) < 20 and (len(ts) < 3 or sum(ts) < 3000):
            t0 = time.perf_counter()
            p = wb.Plan(tr, ro, role, rank)
            ts.append((time.perf_counter() - t0) * 1e3)
            del p
        plan_ms[label] = round(statistics.median(ts), 2)
    rb, G = args.round_budget, args.node_size
    rplan = wb.Plan(tr, ro, wb.RECEIVER, d, round_budget=rb, node_size=G)
    splan = wb.Plan(tr, ro, wb.SENDER, s0, round_budget=rb, node_size=G)
    nr = rplan.num_rounds
    rws = torch.empty(rplan.workspace_bytes, dtype=torch.uint8, device="cuda")
    sws = torch.empty(splan.workspace_bytes, dtype=torch.uint8, device="cuda")
    rplan.upload(rws)
    splan.upload(sws)
    log(f"[bench] {name}: plan ms {plan_ms}; recv {rplan.buffer_bytes / 1e9:.2f} GB")

    # inputs: every sender's region for the receiver, through real packs. With
    # rounds, each round has its receive buffer (what the network delivers) and
    # the sender alternates between two send buffers.
    def alloc(n):
        if args.staged:
            return torch.empty(max(1, n), dtype=torch.uint8, pin_memory=True)
        return torch.empty(max(1, n), dtype=torch.uint8, device="cuda")

    recvs = [alloc(rplan.round_buffer_bytes(k)) for k in range(nr)]
    sends = [alloc(splan.buffer_bytes) for _ in range(min(2, nr))]
    recv, send0 = recvs[0], sends[0]
    fwds = {st: alloc(rplan.forward_bytes(st)) for st in (1, 2)} if G else {}
    # with exchange stages, the payloads forwarded to the unpack rank are the
    # bytes their origin segment left a trainer with: copied out of that
    # trainer's send buffer into their section of the receive buffer
    forwarded = {}
    if G:
        segs = rplan.segments()
        for f in segs:
            if f["stage"] and f["receiver"] == d:
                o = segs[f["origin"]]
                forwarded.setdefault(o["sender"], []).append((o, f))
    src0 = None
    for s in range(tr.nranks):
        if s != s0 and s not in forwarded and not any(rplan.round_region(k, s, d)[2] for k in range(nr)):
            continue
        locs = build_sender_locals(wb, torch, sc, tr, s, src_dtype)
        p = splan if s == s0 else wb.Plan(tr, ro, wb.SENDER, s, round_budget=rb, node_size=G)
        if s != s0:
            ws = torch.empty(p.workspace_bytes, dtype=torch.uint8, device="cuda")
            p.upload(ws)
        buf = send0 if s == s0 else alloc(p.buffer_bytes)
        for k in range(nr):
            so, roff, nb = rplan.round_region(k, s, d)
            mine = [(o, f) for o, f in forwarded.get(s, []) if o["round"] == k]
            if nb or mine:
                (p.pack_round(k, locs, buf) if nr > 1 else p.pack(locs, buf))
            if nb:
                recvs[k][roff:roff + nb] = buf[so:so + nb]
            for o, f in mine:
                recvs[k][f["recv_offset"]:f["recv_offset"] + f["bytes"]] = \
                    buf[o["send_offset"]:o["send_offset"] + o["bytes"]]
        if s == s0:
            src0 = locs
        else:
            del locs, buf, p, ws
        torch.cuda.synchronize()
    dst = wb.allocate_locals(ro, d)
    torch.cuda.synchronize()
    log("[bench] inputs resident")

    pr, pw = splan.traffic()
    ur, uw = rplan.traffic()
    pack_bytes, unpack_bytes = pr + pw, ur + uw
    fwd_bytes = {st: sum(rplan.kernel_traffic(1 + st)) for st in (1, 2)} if G else {}
    stream = torch.cuda.current_stream()
    if args.pipeline and nr < 2:
        sys.exit("--pipeline needs a round budget that gives more than one round")
    pstream, ustream = torch.cuda.Stream(), torch.cuda.Stream()
    packed = [torch.cuda.Event() for _ in range(nr)]
    done = [torch.cuda.Event() for _ in range(nr)]

    def step(ev=None):
        if nr == 1:
            if ev:
                ev[0].record(stream)
            splan.pack(src0, send0, stream)
            if ev:
                ev[1].record(stream)
            for st in fwds:
                rplan.forward_round(0, st, recv, fwds[st], stream)
                if ev:
                    ev[1 + st].record(stream)
            rplan.unpack(recv, dst, stream)
            if ev:
                ev[-1].record(stream)
            return
        if args.pipeline:
            # depth 2: round k+2 reuses the send buffer of round k, so its pack
            # waits for round k's assembly; otherwise the streams run freely.
            # Steps do not overlap: both streams start after the previous step.
            pstream.wait_stream(stream)
            ustream.wait_stream(stream)
            for k in range(nr):
                if k >= 2:
                    pstream.wait_event(done[k - 2])
                splan.pack_round(k, src0, sends[k % 2], pstream)
                packed[k].record(pstream)
                ustream.wait_event(packed[k])
                # the receiver's exchange stages of round k, then its assembly
                for st in fwds:
                    rplan.forward_round(k, st, recvs[k], fwds[st], ustream)
                rplan.unpack_round(k, recvs[k], dst, ustream)
                done[k].record(ustream)
            stream.wait_stream(ustream)
            stream.wait_stream(pstream)
            return
        for k in range(nr):
            splan.pack_round(k, src0, sends[k % 2], stream)
            for st in fwds:
                rplan.forward_round(k, st, recvs[k], fwds[st], stream)
            rplan.unpack_round(k, recvs[k], dst, stream)

    for _ in range(warmup):
        step()
    torch.cuda.synchronize()
    events = [[torch.cuda.Event(enable_timing=True) for _ in range(3 + len(fwds))] for _ in range(steps)]
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for k in range(steps):
        step(events[k])
    torch.cuda.synchronize()
    elapsed = time.perf_counter() - t0
    ms_per_step = elapsed * 1e3 / steps
    fwd_ms = {}
    spread = {}
    if nr == 1:
        pack_steps = [e[0].elapsed_time(e[1]) for e in events]
        unpack_steps = [e[-2].elapsed_time(e[-1]) for e in events]
        pack_ms = statistics.mean(pack_steps)
        for st in fwds:
            fwd_ms[st] = statistics.mean(e[st].elapsed_time(e[1 + st]) for e in events)
        unpack_ms = statistics.mean(unpack_steps)
        # per-step spread of the two launches (the mean is what the line reports)
        for step, xs in (("pack", pack_steps), ("unpack", unpack_steps)):
            spread[step] = {"ms_min": round(min(xs), 4), "ms_median": round(statistics.median(xs), 4),
                            "ms_max": round(max(xs), 4)}
        log("unpack ms per step: " + " ".join(f"{x:.3f}" for x in unpack_steps))
    else:
        # per-kernel times of a round-based step: one more pass timing the
        # packs and the unpacks of all rounds separately
        e = [torch.cuda.Event(enable_timing=True) for _ in range(3)]
        e[0].record(stream)
        for k in range(nr):
            splan.pack_round(k, src0, sends[k % 2], stream)
        e[1].record(stream)
        for k in range(nr):
            rplan.unpack_round(k, recvs[k], dst, stream)
        e[2].record(stream)
        torch.cuda.synchronize()
        pack_ms, unpack_ms = e[0].elapsed_time(e[1]), e[1].elapsed_time(e[2])
    value = (pack_bytes + sum(fwd_bytes.values()) + unpack_bytes) / (ms_per_step * 1e-3) / 1e9

    # practical ceiling: a plain device copy of the receive buffer (also the
    # known-size copy that calibrates the HBM byte counters)
    csrc = recv[:min(recv.numel(), 16 << 30)].cuda() if args.staged else recv[:min(recv.numel(), 16 << 30)]
    scratch = torch.empty_like(csrc)
    scratch.copy_(csrc)
    torch.cuda.synchronize()
    c0, c1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    c0.record(stream)
    for _ in range(3):
        scratch.copy_(csrc)
    c1.record(stream)
    torch.cuda.synchronize()
    copy_ms = c0.elapsed_time(c1) / 3
    del scratch

    # the launches of one wb_unpack, all timed together: the copy/cast kernel
    # and the fp8 block kernels that have work
    launches = [(k, lab, kern) for k, lab, kern in
                ((0, "unpack", "wb::wb_tasks_kernel"), (4, "unpack_tiles", "wb::wb_tile_kernel"),
                 (1, "unpack_fp8", "wb::wb_qblock_kernel"))
                if rplan.launch_grid(k)[0]]
    dom = " + ".join(kern for _, _, kern in launches) + (
        " (one wb_unpack, timed together)" if len(launches) > 1 else " (unpack)")
    achieved = unpack_bytes / (unpack_ms * 1e-3) / 1e9
    # HBM bytes of the launches the roofline times (every launch of the unpack)
    why = []
    parts = [stored_traffic(name, lab, why) for _, lab, _ in launches]
    traffic = sum(parts) if all(x is not None for x in parts) and not G and nr == 1 and not args.staged else None
    out = {
        "metric": "pack+unpack effective GB/s per GPU (% of HBM peak); wb_plan ms",
        "value": round(value, 1),
        "unit": "GB/s",
        "n_gpus": 1,
        "steps": steps,
        "warmup": warmup,
        "ms_per_step": round(ms_per_step, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": src_dtype if src_dtype == w["rollout"]["dtype"] and not w["rollout"].get("quant")
        else f"{src_dtype}->{w['rollout'].get('quant') or w['rollout']['dtype']}",
        "data": "synthetic",
        "config": {"workload": name, "trainer": w["trainer"], "rollout": w["rollout"],
                   "pack_rank": s0, "unpack_rank": d, "bytes_per_step": pack_bytes + unpack_bytes,
                   "buffers": "pinned host (PCIe)" if args.staged else "device",
                   "rounds": nr, "round_budget": rb, "pipeline": bool(args.pipeline), "node_size": G},
        "pct_of_hbm_peak": round(100 * value / HBM_PEAK_GBS, 2),
        "plan_ms": plan_ms,
        "pack": {"ms": round(pack_ms, 4), "GB/s": round(pack_bytes / (pack_ms * 1e-3) / 1e9, 1), "bytes": pack_bytes,
                 **spread.get("pack", {})},
        "unpack": {"ms": round(unpack_ms, 4), "GB/s": round(achieved, 1), "bytes": unpack_bytes,
                   **spread.get("unpack", {})},
        "device_copy": {"GB/s": round(2 * csrc.numel() / (copy_ms * 1e-3) / 1e9, 1), "bytes": 2 * csrc.numel(),
                        "what": "torch copy_ of (up to 16 GiB of) the receive buffer: hipMemcpy device to device"},
        "roofline": {"bound": "hbm", "kernel": dom, "achieved": round(achieved, 1),
                     "peak": HBM_PEAK_GBS, "unit": "GB/s", "frac": round(achieved / HBM_PEAK_GBS, 4),
                     "traffic": traffic,
                     "traffic_source": (f"stored: profiles/traffic-{name}.txt, two rocprofv3 --pmc runs (FETCH_SIZE, "
                                        "then WRITE_SIZE) of this benchmark scaled by a device copy of known size; "
                                        "used only while the kernels' source and the plans' launch grids match its "
                                        "fingerprint") if traffic is not None else
                     ("; ".join(why) or "not the one-round device-buffer step the counters were taken on")},
    }
    if ceilings:
        # the one-shot stream with the dominant kernel's read/write mix: a same-
        # dtype copy reads one byte per byte written, a cast assembly two (the
        # faster of the two 2 : 1 shapes: one 16-byte store per lane, or two
        # 8-byte halves one wave apart as the cast kernels store)
        if ur < 1.5 * uw:
            mix = "copy_oneshot_GBps"
        else:
            mix = max(("read2_write1_oneshot_GBps", "read2_write1_halves_oneshot_GBps"),
                      key=lambda k: ceilings.get(k) or 0.0)
        out["stream_ceilings"] = dict(ceilings, matching=mix,
                                      frac_of_matching=round(achieved / ceilings[mix], 4) if ceilings.get(mix) else None)
    if fwds:
        out["forward"] = {f"stage{st}": {"bytes": fwd_bytes[st], "ms": round(fwd_ms[st], 4) if st in fwd_ms else None,
                                         "GB/s": round(fwd_bytes[st] / (fwd_ms[st] * 1e-3) / 1e9, 1)
                                         if fwd_ms.get(st) else None} for st in fwds}
        out["config"]["bytes_per_step"] = pack_bytes + sum(fwd_bytes.values()) + unpack_bytes
    if with_cpu and nr == 1 and not G:
        import numpy as np

        def recv_host(off, nb, out):
            torch.from_numpy(out[:nb]).copy_(recv[off:off + nb])

        def src_host(u):
            x = src0[u].reshape(-1)
            return x.view(torch.int32 if x.element_size() == 4 else torch.int16).cpu().numpy().view(
                np.uint32 if x.element_size() == 4 else np.uint16)

        out["cpu_baseline"] = cpu_baseline(w, recv_host, src_host)
    # free the workload's device memory before the next one
    locs = buf = p = ws = None
    del recvs, sends, recv, send0, fwds, src0, dst, rws, sws, rplan, splan, csrc
    torch.cuda.synchronize()
    torch.cuda.empty_cache()
    return out



def per_config_entry(rec):
    """The part of a workload's record that the headline line repeats for
    every workload."""
    ent = {"value_GBps": rec["value"], "pct_of_hbm_peak": rec["pct_of_hbm_peak"], "ms_per_step": rec["ms_per_step"],
           "steps": rec["steps"], "dtype": rec["dtype"], "bytes_per_step": rec["config"]["bytes_per_step"],
           "pack": {k: rec["pack"][k] for k in ("ms", "GB/s", "bytes")},
           "unpack": {k: rec["unpack"][k] for k in ("ms", "GB/s", "bytes")},
           "roofline_kernel": rec["roofline"]["kernel"], "roofline_frac": rec["roofline"]["frac"],
           "pack_frac": round(rec["pack"]["GB/s"] / HBM_PEAK_GBS, 4),
           "plan_ms": rec["plan_ms"], "stored_traffic_applies": rec["roofline"]["traffic"] is not None,
           "traffic": rec["roofline"]["traffic"]}
    sc = rec.get("stream_ceilings")
    if sc:
        ent["frac_of_matching_ceiling"] = sc.get("frac_of_matching")
    return ent


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--workload", default=DEFAULT_WORKLOAD)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-per-config", action="store_true",
                    help="time only --workload (by default every workload is timed after it, fewer steps each)")
    ap.add_argument("--no-ceilings", action="store_true",
                    help="skip measuring this GPU's stream ceilings before the benchmark")
    ap.add_argument("--round-budget", type=int, default=0,
                    help="bytes per rank per round (0: one round); each step packs and unpacks every round")
    ap.add_argument("--node-size", type=int, default=0,
                    help="rollout ranks per node: plan with rollout de-duplication and the two exchange stages; "
                         "each step also runs the unpack rank's forward packings")
    ap.add_argument("--pipeline", action="store_true",
                    help="with rounds: pack round k+1 on one stream while round k is forwarded (with --node-size) "
                         "and assembled on another")
    ap.add_argument("--plan-stress", action="store_true",
                    help="wb_plan time on a 58-MoE-layer DeepSeek-V3-like catalog (44,776 tensors, EP64 -> EP8 fp8)")
    ap.add_argument("--probe", action="store_true",
                    help="discover the trainer and rollout ranks' layouts by probing torch loaders (diff2 kernels)")
    ap.add_argument("--staged", action="store_true",
                    help="send and receive buffers in pinned host memory (PCIe-bound; not the headline value)")
    ap.add_argument("--summarize-counters", nargs=2, metavar=("FETCH_CSV", "WRITE_CSV"),
                    help="print HBM traffic per launch from two rocprofv3 --pmc runs of this benchmark")
    ap.add_argument("--ceilings", action="store_true",
                    help="print this GPU's read, write and copy stream ceilings (wb_ceilings, from ceilings.hip)")
    ap.add_argument("--summarize-trace", metavar="KERNEL_TRACE_CSV",
                    help="print per-launch kernel durations from a rocprofv3 --kernel-trace run of this benchmark")
    ap.add_argument("--summarize-metric", nargs=2, metavar=("NAME", "COUNTER_CSV"),
                    help="print the mean of one rocprofv3 --pmc counter or derived metric per launch")
    args = ap.parse_args()
    if args.summarize_counters:
        print(json.dumps(summarize_counters(args.workload, *args.summarize_counters), indent=1))
        return
    if args.ceilings:
        r = run_ceilings()
        sys.stderr.write(r.stderr)
        print(r.stdout.strip())
        sys.exit(r.returncode)
    if args.summarize_trace:
        print(json.dumps(summarize_trace(args.workload, args.summarize_trace), indent=1))
        return
    if args.summarize_metric:
        print(json.dumps(summarize_metric(args.workload, *args.summarize_metric), indent=1))
        return
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py measures one GPU: the resharding hot path here runs on a single MI355X "
              "(pack of one trainer rank, unpack of one rollout rank); --gpus above 1 is not supported.",
              file=sys.stderr)
        sys.exit(2)

    if args.probe:
        run_probe(args)
        return
    if args.plan_stress:
        run_plan_stress()
        return

    # the practical ceilings of this GPU, measured before the benchmark
    # allocates anything, for reading the roofline fraction against
    ceilings = None
    if not args.no_ceilings and not args.staged:
        r = run_ceilings()
        if r.returncode == 0:
            ceilings = json.loads(r.stdout.strip().splitlines()[-1])
            ceilings.pop("bytes", None)
        else:
            log(f"[bench] stream ceilings failed ({r.returncode}): {r.stderr.strip()[-300:]}")

    out = run_workload(args, args.workload, args.steps, args.warmup, ceilings, with_cpu=not args.no_cpu_baseline)
    plain = not (args.round_budget or args.node_size or args.pipeline or args.staged)
    if plain and not args.no_per_config:
        # every workload in the same run: its pack and unpack rates and roofline
        from synthetic_checkpoint.workloads import ORDER

        per = {}
        for other in ORDER:
            rec = out if other == args.workload else run_workload(args, other, min(args.steps, 10), 2, ceilings)
            per[other] = per_config_entry(rec)
            log(f"[bench] {other}: {per[other]['value_GBps']} GB/s, unpack frac {per[other]['roofline_frac']}")
        out["per_config"] = per
    print(json.dumps(out), flush=True)

if __name__ == "__main__":
    main()
