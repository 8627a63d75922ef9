"""Marshal oracle layouts into the library's generic layout builder (tests only).

A layout is an input description (which checkpoint rectangles each rank holds
and where), so feeding the oracle's description to the library is how the
tests give both sides the same problem; the arithmetic of each side stays its
own.
"""

from __future__ import annotations

import paper_2609_25442_amd as wb


def to_wb(layout) -> "wb.Layout":
    L = wb.Layout.create([(t.name, t.rows, t.cols) for t in layout.catalog], layout.nranks)
    for r, rk in enumerate(layout.ranks):
        for u, lc in enumerate(rk.locals):
            if lc.scales >= 0:
                continue  # added by the library with its quantised tensor
            got = L.add_local(r, lc.name, lc.dtype, lc.batch, lc.rows, lc.cols, lc.block)
            assert got == u
        for p in rk.placements:
            L.add_placement(r, p.t, p.r0, p.r1, p.c0, p.c1, p.u, p.base, p.ld, p.tr)
    return L
