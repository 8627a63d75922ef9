"""Routing plan: correspondence, de-duplication, balance, wire format.

Follows WeightBridge Sec. 3.1 (correspondence is the overlap of two workers'
source maps in the checkpoint index space) and Sec. 3.2 ("Generating an
efficient routing plan": a tensor replicated on the trainer side is split into
distinct slices, one per replica, so the trainers together send one copy and
no replica becomes a single-source bottleneck). Without rule 6 each rollout
rank receives everything it needs from the trainers; with it, replicated
rollout tensors are also split and completed by two exchange stages.
The canonical choices below are the reading taken here; the paper fixes none of
them:

1. Trainer *groups*: placements of one checkpoint tensor with identical
   rectangles form one group whose owner set is the sorted list of ranks that
   hold it. Distinct groups of a tensor must be disjoint.
2. Visit rollout rank d ascending, then d's placements Q in layout order, then
   the groups of Q's tensor ordered by (r0, c0, r1, c1). Each non-empty
   X = Q.rect & g.rect is a *region*; together the regions of Q must cover Q.
3. A region with one owner is one segment. Otherwise it is split into k equal
   parts (k = number of owners): by rows when it has at least k rows, else by
   columns; part j spans [floor(j n / k), floor((j+1) n / k)) of that axis.
   Empty parts are dropped. Parts are handed out per owner set by deficit:
   each owner q of the set keeps E_q = k * (bytes assigned to q) - (bytes of
   all regions of the set so far); the region's bytes are first added to the
   total, then its parts, largest first (ties: lower part index), each go to
   the owner with the smallest E_q (ties: lower rank). Since the E_q of a set
   sum to zero after every region and a part always goes to a negative E_q,
   no owner ever exceeds its even share of the set by more than one part.
4. Wire format (Sec. 3.2, the packing kernel coalesces the tensors for one
   receiver into one contiguous buffer): the payloads of sender s for receiver
   d follow the canonical order, each a row-major copy of its rectangle in the
   sender's dtype, each starting at a multiple of 256 bytes of its region. A
   sender's buffer holds its regions by ascending receiver; a receiver's
   buffer holds the regions by ascending sender; every region starts at a
   multiple of 4096 bytes. Forwarding rollout ranks build one forward buffer
   per exchange stage the same way. A rollout rank's receive buffer holds the
   stage-0 section, then the stage-1 section, then the stage-2 section; a
   non-empty later section starts at the next multiple of 4096 bytes.
5. Rounds (Sec. 3.2: the model is cut into roughly equal chunks, one per
   round; App. D: the round count follows from the registered-buffer budget).
   With a budget B > 0 the checkpoint tensors are grouped into *units*: two
   tensors share a unit when their images in one fp8 destination matrix touch
   a common quantisation block (so no block spans two rounds). Units are
   visited in order of their first tensor; a unit joins the current round
   unless that would take some sender's or receiver's bytes in the round above
   B, in which case it opens the next round (a unit larger than B is a round of
   its own). Segments keep their canonical order; each round has its own wire
   offsets, computed by rule 4 over that round's segments.
6. Rollout-side de-duplication and the exchange stages (Sec. 3.2, the second
   principle and the three-stage plan; Figure 5), with rollout ranks grouped
   into nodes of G consecutive ranks (G = 0: the direct plan of rule 2).
   Rollout placements of one tensor with identical rectangles form a rollout
   group with holder set D (ascending ranks). A group with m = |D| > 1 is
   split into m parts by the rule of 3, the parts handed out over D by the
   deficit rule of 3 counted in elements (one counter set per holder set,
   groups visited when their first holder's placement is visited in the order
   of rule 2). In the *receive* stage (stage 0) each holder asks the trainers
   only for its parts; rule 2 then runs over these parts instead of the whole
   rectangle. In the *external exchange* (stage 1) each stage-0 segment that
   rank r received for a group is forwarded, byte for byte, to one holder in
   every other node v that holds the group: the holder at position
   (i mod |H_v|) of H_v, where H_v lists the group's holders in node v and i
   is r's position in its own node's list. In the *internal exchange* (stage
   2) every segment a holder received in stage 0 or stage 1 is forwarded to
   each other holder of the group in its node. Stage-1 segments follow the
   stage-0 segments they forward; stage-2 segments follow the stage-0 and then
   the stage-1 segments they forward. Each node thus receives over the
   inter-node network exactly one copy of what its ranks need.
"""

from __future__ import annotations

from dataclasses import dataclass

from .layout import DTYPE_BYTES, Layout

PAYLOAD_ALIGN = 256
REGION_ALIGN = 4096


@dataclass(frozen=True)
class Rect:
    r0: int
    r1: int
    c0: int
    c1: int

    @property
    def numel(self) -> int:
        return (self.r1 - self.r0) * (self.c1 - self.c0)

    def intersect(self, o: "Rect"):
        r0, r1, c0, c1 = max(self.r0, o.r0), min(self.r1, o.r1), max(self.c0, o.c0), min(self.c1, o.c1)
        return Rect(r0, r1, c0, c1) if r0 < r1 and c0 < c1 else None


@dataclass
class Segment:
    s: int          # sender (trainer rank)
    d: int          # receiver (rollout rank)
    t: int          # checkpoint tensor
    rect: Rect
    src_pl: int     # placement index in the sender's layout
    dst_pl: int     # placement index in the receiver's layout
    nbytes: int     # payload bytes (sender dtype)
    region: int = -1  # index of the region the segment was cut from
    round: int = 0
    send_off: int = 0
    recv_off: int = 0
    stage: int = 0    # 0 receive (trainer -> rollout); 1, 2 exchange (rollout -> rollout)
    src_seg: int = -1  # exchange stages: the segment whose received bytes are forwarded
    origin: int = -1   # the stage-0 segment the bytes came from (its own index in stage 0)
    src_off: int = 0   # exchange stages: offset of the forwarded bytes in the sender's receive buffer
    wire: str = ""     # dtype of the payload: the trainer dtype it was packed in


@dataclass
class Region:
    owners: tuple
    nbytes: int     # bytes of the whole region (sender dtype)


@dataclass
class Round:
    send_bytes: list[int]
    recv_bytes: list[int]
    fwd_bytes: list = None   # [stage 1 bytes per rollout rank, stage 2 bytes per rollout rank]


@dataclass
class Plan:
    trainer: Layout
    rollout: Layout
    segments: list[Segment]
    regions: list[Region]
    send_bytes: list[int]
    recv_bytes: list[int]
    rounds: list[Round] = None
    node_size: int = 0


def _align(x: int, a: int) -> int:
    return -(-x // a) * a


class PlanError(ValueError):
    pass


def _split(x: Rect, k: int) -> list[Rect]:
    """Rule 3: k parts by rows when x has at least k rows, else by columns;
    empty parts dropped."""
    by_rows = (x.r1 - x.r0) >= k
    n = (x.r1 - x.r0) if by_rows else (x.c1 - x.c0)
    pieces = []
    for j in range(k):
        a, b = j * n // k, (j + 1) * n // k
        if a < b:
            pieces.append(Rect(x.r0 + a, x.r0 + b, x.c0, x.c1) if by_rows
                          else Rect(x.r0, x.r1, x.c0 + a, x.c0 + b))
    return pieces


def _deal(pieces: list[Rect], owners: tuple, e: dict, total: int, weight) -> list:
    """Rule 3's deficit hand-out: returns the owner of every piece."""
    k = len(owners)
    for q in owners:
        e[q] -= total
    who = [None] * len(pieces)
    for j in sorted(range(len(pieces)), key=lambda j: (-pieces[j].numel, j)):
        q = min(owners, key=lambda q: (e[q], q))
        e[q] += k * weight(pieces[j])
        who[j] = q
    return who


def _rollout_groups(rollout: Layout) -> dict:
    """Rule 6: (t, r0, r1, c0, c1) -> {rollout rank: placement index}."""
    holders: dict[tuple, dict] = {}
    for d, rk in enumerate(rollout.ranks):
        for qi, q in enumerate(rk.placements):
            h = holders.setdefault((q.t, q.r0, q.r1, q.c0, q.c1), {})
            if d in h:
                raise PlanError("a rollout rank holds the same rectangle twice")
            h[d] = qi
    return holders


def build_plan(trainer: Layout, rollout: Layout, round_budget: int = 0, node_size: int = 0) -> Plan:
    cat = trainer.catalog
    if [(t.name, t.rows, t.cols) for t in cat] != [(t.name, t.rows, t.cols) for t in rollout.catalog]:
        raise PlanError("trainer and rollout catalogs differ")

    # 1. trainer groups: rect -> owners (ascending rank) and their placement index
    by_rect: dict[tuple, dict] = {}
    for s, rk in enumerate(trainer.ranks):
        for pi, p in enumerate(rk.placements):
            key = (p.t, p.r0, p.r1, p.c0, p.c1)
            owners = by_rect.setdefault(key, {})
            if s in owners:
                raise PlanError("a trainer rank holds the same rectangle twice")
            owners[s] = pi
    groups: dict[int, list] = {}
    for (t, r0, r1, c0, c1), owners in by_rect.items():
        groups.setdefault(t, []).append((Rect(r0, r1, c0, c1), tuple(sorted(owners)), owners))
    for t, gl in groups.items():
        gl.sort(key=lambda g: (g[0].r0, g[0].c0, g[0].r1, g[0].c1))
        for a in range(len(gl)):
            for b in range(a + 1, len(gl)):
                if gl[a][0].intersect(gl[b][0]) is not None:
                    raise PlanError(f"overlapping, non-identical trainer rectangles in tensor {t}")

    if node_size < 0:
        raise PlanError("node size must be >= 0")
    G = node_size
    holders = _rollout_groups(rollout) if G else {}

    # 6. rollout parts: a replicated rollout group is dealt out over its holders
    assign: dict[tuple, list] = {}
    rdeficit: dict[tuple, dict[int, int]] = {}
    for d, rk in enumerate(rollout.ranks):
        for q in rk.placements if G else ():
            key = (q.t, q.r0, q.r1, q.c0, q.c1)
            D = tuple(sorted(holders[key]))
            if len(D) == 1 or D[0] != d:
                continue
            rect = Rect(q.r0, q.r1, q.c0, q.c1)
            pieces = _split(rect, len(D))
            e = rdeficit.setdefault(D, {x: 0 for x in D})
            assign[key] = list(zip(pieces, _deal(pieces, D, e, rect.numel, lambda p: p.numel)))

    # 2./3. regions and stage-0 segments in canonical order
    deficit: dict[tuple, dict[int, int]] = {}
    segments: list[Segment] = []
    regions: list[Region] = []
    for d, rk in enumerate(rollout.ranks):
        for qi, q in enumerate(rk.placements):
            qrect = Rect(q.r0, q.r1, q.c0, q.c1)
            key = (q.t, q.r0, q.r1, q.c0, q.c1)
            needs = [p for p, x in assign[key] if x == d] if key in assign else [qrect]
            for need in needs:
                covered = 0
                for grect, owners, pl_of in groups.get(q.t, []):
                    x = need.intersect(grect)
                    if x is None:
                        continue
                    covered += x.numel
                    esizes = {DTYPE_BYTES[trainer.ranks[s].locals[trainer.ranks[s].placements[pl_of[s]].u].dtype]
                              for s in owners}
                    if len(esizes) != 1:
                        raise PlanError("replicas of one rectangle hold different dtypes")
                    esize = esizes.pop()
                    wire = trainer.ranks[owners[0]].locals[trainer.ranks[owners[0]].placements[pl_of[owners[0]]].u].dtype
                    if len(owners) == 1:
                        parts = [(x, owners[0])]
                    else:
                        pieces = _split(x, len(owners))
                        e = deficit.setdefault(owners, {s: 0 for s in owners})
                        parts = list(zip(pieces, _deal(pieces, owners, e, x.numel * esize,
                                                       lambda p: p.numel * esize)))
                    for part, s in parts:
                        segments.append(Segment(s, d, q.t, part, pl_of[s], qi, part.numel * esize, len(regions),
                                                origin=len(segments), wire=wire))
                    regions.append(Region(owners, x.numel * esize))
                if covered != need.numel:
                    raise PlanError(f"rollout rank {d} placement {qi} is not fully held by the trainers")

    # 6. exchange stages
    if G:
        def group_of(g):
            q = rollout.ranks[g.d].placements[g.dst_pl]
            key = (q.t, q.r0, q.r1, q.c0, q.c1)
            return key, sorted(holders[key])

        n0 = len(segments)
        for gi in range(n0):
            g = segments[gi]
            key, D = group_of(g)
            if len(D) == 1:
                continue
            mine = [x for x in D if x // G == g.d // G]
            i = mine.index(g.d)
            for v in sorted({x // G for x in D}):
                if v == g.d // G:
                    continue
                hv = [x for x in D if x // G == v]
                x = hv[i % len(hv)]
                segments.append(Segment(g.d, x, g.t, g.rect, -1, holders[key][x], g.nbytes, -1,
                                        stage=1, src_seg=gi, origin=g.origin, wire=g.wire))
        n1 = len(segments)
        for gi in range(n1):
            g = segments[gi]
            key, D = group_of(g)
            for z in D:
                if z != g.d and z // G == g.d // G:
                    segments.append(Segment(g.d, z, g.t, g.rect, -1, holders[key][z], g.nbytes, -1,
                                            stage=2, src_seg=gi, origin=g.origin, wire=g.wire))

    # 5. rounds, then 4. wire offsets per round
    ns, nd = trainer.nranks, rollout.nranks
    nrounds = _assign_rounds(trainer, rollout, segments, round_budget) if round_budget > 0 else 1
    rounds = [_wire_round(segments, r, ns, nd) for r in range(nrounds)]
    return Plan(trainer, rollout, segments, regions, rounds[0].send_bytes, rounds[0].recv_bytes, rounds, G)


def _wire_round(segments, r, ns, nd) -> Round:
    """Rule 4 for round r: stage 0 between trainers and rollout ranks, then
    each exchange stage between rollout ranks, its section placed after the
    earlier ones in every receive buffer; forwarded segments read the bytes
    their source segment received."""
    send0, recv0 = _wire([g for g in segments if g.round == r and g.stage == 0], ns, nd)
    pos = list(recv0)
    fwd = []
    for stage in (1, 2):
        mine = [g for g in segments if g.round == r and g.stage == stage]
        fsend, frecv = _wire(mine, nd, nd)
        base = []
        for d in range(nd):
            if frecv[d]:
                pos[d] = _align(pos[d], REGION_ALIGN)
            base.append(pos[d])
            pos[d] += frecv[d]
        for g in mine:
            g.recv_off += base[g.d]
            g.src_off = segments[g.src_seg].recv_off
        fwd.append(fsend)
    return Round(send0, pos, fwd)


def _wire(mine, ns, nd):
    """Rule 4 over one stage's segments of one round (offsets set in place);
    returns (send bytes per sender, receive bytes per receiver)."""
    payload_end: dict[tuple, int] = {}
    for sg in mine:
        off = _align(payload_end.get((sg.s, sg.d), 0), PAYLOAD_ALIGN)
        sg.send_off = off
        sg.recv_off = off
        payload_end[(sg.s, sg.d)] = off + sg.nbytes
    send_region, send_bytes = {}, []
    for s in range(ns):
        pos = 0
        for d in range(nd):
            if (s, d) in payload_end:
                pos = _align(pos, REGION_ALIGN)
                send_region[(s, d)] = pos
                pos += payload_end[(s, d)]
        send_bytes.append(pos)
    recv_region, recv_bytes = {}, []
    for d in range(nd):
        pos = 0
        for s in range(ns):
            if (s, d) in payload_end:
                pos = _align(pos, REGION_ALIGN)
                recv_region[(s, d)] = pos
                pos += payload_end[(s, d)]
        recv_bytes.append(pos)
    for sg in mine:
        sg.send_off += send_region[(sg.s, sg.d)]
        sg.recv_off += recv_region[(sg.s, sg.d)]
    return send_bytes, recv_bytes


def _block_units(rollout: Layout, ntensors: int) -> list[int]:
    """Unit id of every checkpoint tensor: tensors whose images in one
    quantised destination matrix share a block are joined (union-find)."""
    parent = list(range(ntensors))

    def find(a):
        while parent[a] != a:
            parent[a] = parent[parent[a]]
            a = parent[a]
        return a

    for rk in rollout.ranks:
        per_matrix: dict[tuple, list] = {}
        for p in rk.placements:
            lc = rk.locals[p.u]
            if not lc.block:
                continue
            mat = lc.rows * lc.cols
            e, row0, col0 = p.base // mat, (p.base % mat) // lc.cols, p.base % lc.cols
            if p.tr or col0 + p.cols > lc.cols or row0 + p.rows > lc.rows or (p.rows > 1 and p.ld != lc.cols):
                raise PlanError("an fp8 placement must be a non-transposed sub-rectangle of one matrix")
            B = lc.block
            per_matrix.setdefault((p.u, e), []).append(
                (row0 // B, (row0 + p.rows - 1) // B, col0 // B, (col0 + p.cols - 1) // B, p.t))
        for items in per_matrix.values():
            for a in range(len(items)):
                for b in range(a + 1, len(items)):
                    x, y = items[a], items[b]
                    if x[0] <= y[1] and y[0] <= x[1] and x[2] <= y[3] and y[2] <= x[3]:
                        parent[find(x[4])] = find(y[4])
    return [find(t) for t in range(ntensors)]


def _assign_rounds(trainer: Layout, rollout: Layout, segments, budget: int) -> int:
    """Cut the transfer into rounds, each a run of units (tensors that share
    an fp8 block stay together) visited in catalog order.

    Filling with a cap X means: a unit that would push some sender's send
    bytes or some receiver's receive bytes past X opens the next round, so a
    rank goes past X in a round only through the round's first unit (one
    larger than X on its own). The number of rounds n is what
    filling with the budget needs (App. D: the round count follows from the
    registered-buffer budget). The rounds are then the filling with the
    smallest cap X <= budget that still needs only n rounds (found by
    bisection over whole bytes): the largest round is as small as n rounds
    allow, so the model moves in chunks of about equal size (Sec. 3.2)."""
    unit = _block_units(rollout, len(trainer.catalog))
    members: dict[int, list] = {}
    for sg in segments:
        members.setdefault(unit[sg.t], []).append(sg)
    order = sorted(members, key=lambda u: min(sg.t for sg in members[u]))
    # bytes of each unit per rank: ("s", sender) and ("d", receiver)
    size = []
    for u in order:
        b = {}
        for sg in members[u]:
            if sg.stage == 0:
                b[("s", sg.s)] = b.get(("s", sg.s), 0) + sg.nbytes
            b[("d", sg.d)] = b.get(("d", sg.d), 0) + sg.nbytes
        size.append(b)

    def fill(cap):
        rounds, cur, r = [], {}, 0
        for b in size:
            if cur and any(cur.get(k, 0) + v > cap for k, v in b.items()):
                r, cur = r + 1, {}
            for k, v in b.items():
                cur[k] = cur.get(k, 0) + v
            rounds.append(r)
        return rounds

    rounds = fill(budget)
    n = rounds[-1] + 1 if rounds else 1
    total = {}
    for b in size:
        for k, v in b.items():
            total[k] = total.get(k, 0) + v
    lo = max([1] + [-(-t // n) for t in total.values()])
    hi = budget
    while lo < hi:
        mid = lo + (hi - lo) // 2
        cut = fill(mid)
        if (cut[-1] + 1 if cut else 1) <= n:
            hi = mid
        else:
            lo = mid + 1
    rounds = fill(lo) if lo < budget else rounds
    for r, u in zip(rounds, order):
        for sg in members[u]:
            sg.round = r
    return (rounds[-1] + 1) if rounds else 1


def dump(plan: Plan) -> str:
    """Canonical text form of a plan, one line per segment (grouped by round
    when there are several)."""
    def segline(g):
        r = g.rect
        if g.stage == 0:
            return (f"seg {g.s} {g.d} {g.t} {r.r0} {r.r1} {r.c0} {r.c1} {g.src_pl} {g.dst_pl} "
                    f"{g.send_off} {g.recv_off} {g.nbytes}")
        return (f"{'xseg' if g.stage == 1 else 'iseg'} {g.s} {g.d} {g.t} {r.r0} {r.r1} {r.c0} {r.c1} "
                f"{g.src_off} {g.dst_pl} {g.send_off} {g.recv_off} {g.nbytes}")

    def sizes(rd):
        out = [f"send {s} {b}" for s, b in enumerate(rd.send_bytes)]
        out += [f"recv {d} {b}" for d, b in enumerate(rd.recv_bytes)]
        if plan.node_size:
            for stage in (1, 2):
                out += [f"fwd{stage} {d} {b}" for d, b in enumerate(rd.fwd_bytes[stage - 1])]
        return out

    head = f"plan trainer_ranks={plan.trainer.nranks} rollout_ranks={plan.rollout.nranks} segments={len(plan.segments)}"
    if plan.node_size:
        head += f" node_size={plan.node_size}"
    rounds = plan.rounds or [Round(plan.send_bytes, plan.recv_bytes)]
    if len(rounds) == 1:
        return "\n".join([head] + sizes(rounds[0]) + [segline(g) for g in plan.segments]) + "\n"
    out = [head + f" rounds={len(rounds)}"]
    for k, rd in enumerate(rounds):
        out.append(f"round {k}")
        out += sizes(rd)
        out += [segline(g) for g in plan.segments if g.round == k]
    return "\n".join(out) + "\n"


def dump_layout(layout: Layout) -> str:
    """Canonical text form of a layout."""
    out = [f"layout ranks={layout.nranks} tensors={len(layout.catalog)}"]
    for r, rk in enumerate(layout.ranks):
        out.append(f"rank {r} locals={len(rk.locals)} placements={len(rk.placements)}")
        for u, lc in enumerate(rk.locals):
            out.append(f"local {u} {lc.name} {lc.dtype} {lc.batch} {lc.rows} {lc.cols} {lc.block} {lc.scale} {lc.scales}")
        for p in rk.placements:
            out.append(f"pl {p.t} {p.r0} {p.r1} {p.c0} {p.c1} {p.u} {p.base} {p.ld} {p.tr}")
    return "\n".join(out) + "\n"


def sender_loads(plan: Plan):
    """(load, ideal) bytes per sender: ideal counts each region's bytes split
    evenly over its owners."""
    ns = plan.trainer.nranks
    load = [0] * ns
    ideal = [0.0] * ns
    for g in plan.segments:
        if g.stage == 0:
            load[g.s] += g.nbytes
    for reg in plan.regions:
        for s in reg.owners:
            ideal[s] += reg.nbytes / len(reg.owners)
    return load, ideal
