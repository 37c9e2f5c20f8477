"""Arena planner (oracle side): Section 3 "Memory Allocation and Management",
Alg. 4 (Greedy-by-Size) and the naive sequential plan it is compared with.

All activations live in one caller-allocated buffer; the planner assigns a
byte offset to every tensor ahead of time from tensor lifetimes.

  * Buffers: a Transpose/Reshape whose layouts make it a view owns no bytes;
    its output is an alias of its input's root.  Every other node output is a
    buffer, except graph outputs (written straight into the caller's buffer).
    Graph inputs are caller-owned too.
  * size = elements * dtype bytes rounded up to the alignment (256 B).
  * lifetime = [def, last]: def the producing node, last the largest id of a
    node reading any edge rooted at the buffer (def if never read).  Two
    buffers conflict iff their closed lifetimes intersect, so an operator's
    output never shares bytes with its own inputs (no in-place reuse).
  * Greedy-by-Size: take buffers by size descending (ties: def ascending,
    then edge id); among the already placed buffers whose lifetime overlaps,
    walk the gaps in offset order and choose the smallest gap that fits
    (lowest offset on ties) -- the text asks for "the most suitable slot";
    if none fits, place it at the end of the overlapping buffers ("increase
    and allocate the last free available block").
  * Naive plan: one slice per buffer of the row-major plan, offsets the
    prefix sums of the sizes in edge-id order, no reuse.
  * Lower bound: the largest total size of buffers live at one node.
  * Fused chains of the layout plan (fuse[m] = t: the MatMul m performs
    nodes m+1 .. m+t in its launch): the intermediate results never reach
    memory and get no buffer; the launch reads the MatMul's operands while
    it writes node m+t's output, so their lifetimes run at least to m+t.
"""
from __future__ import annotations

import numpy as np

from . import fusion, numerics
from .layouts import node_is_view


def align_up(x, a):
    return (x + a - 1) // a * a


class ArenaPlan:
    def __init__(self, root, buffers, size, defn, last, offset, peak):
        self.root = root          # per edge: root edge (itself if not a view)
        self.buffers = buffers    # arena buffer edge ids
        self.size = size          # dict edge -> bytes
        self.defn = defn
        self.last = last
        self.offset = offset      # dict edge -> byte offset
        self.peak = peak


def buffers_and_lifetimes(g, layout_of_edge, align=256, fuse=None):
    """Roots, arena buffers, sizes and lifetimes under the given layouts
    (and the plan's fused chains, if any)."""
    isz = numerics.itemsize(g.dtype)
    root = list(range(g.n_edges))
    view = [False] * len(g.nodes)
    for n in range(len(g.nodes)):
        if node_is_view(g, n, layout_of_edge):
            view[n] = True
            root[g.out_edge(n)] = root[g.act_inputs(n)[0]]
    outs = set(g.outputs)
    on_chip, until = set(), {}
    for m, t in enumerate(fuse or []):
        if t:
            on_chip.update(fusion.on_chip_edges(g, m, t))
            until[m] = m + t
    buffers = [g.out_edge(n) for n in range(len(g.nodes))
               if not view[n] and g.out_edge(n) not in outs and g.out_edge(n) not in on_chip]
    size = {b: align_up(int(np.prod(g.edge_shape(b))) * isz, align) for b in buffers}
    defn = {b: g.producer(b) for b in buffers}
    last = dict(defn)
    for n, nd in enumerate(g.nodes):
        for v in nd.ins:
            if v >= 0:
                r = root[v]
                if r in last:
                    last[r] = max(last[r], until.get(n, n))
    return root, buffers, size, defn, last


def overlaps(defn, last, a, b):
    return defn[a] <= last[b] and defn[b] <= last[a]


def greedy_by_size(buffers, size, defn, last):
    order = sorted(buffers, key=lambda b: (-size[b], defn[b], b))
    offset = {}
    placed = []
    for b in order:
        O = sorted((o for o in placed if overlaps(defn, last, o, b)),
                   key=lambda o: (offset[o], o))
        cursor = 0
        best = None          # (gap size, offset)
        for o in O:
            gap = offset[o] - cursor
            if gap >= size[b]:
                if best is None or gap < best[0]:
                    best = (gap, cursor)
            cursor = max(cursor, offset[o] + size[o])
        offset[b] = best[1] if best is not None else cursor
        placed.append(b)
    peak = max((offset[b] + size[b] for b in buffers), default=0)
    return offset, peak


def plan_arena(g, layout_of_edge, align=256, fuse=None):
    root, buffers, size, defn, last = buffers_and_lifetimes(g, layout_of_edge, align, fuse)
    offset, peak = greedy_by_size(buffers, size, defn, last)
    return ArenaPlan(root, buffers, size, defn, last, offset, peak)


def naive_plan(g, align=256):
    """Row-major layouts, every buffer its own slice, edge-id order."""
    ident = {e: tuple(range(len(g.edge_shape(e)))) for e in range(g.n_edges)}
    root, buffers, size, defn, last = buffers_and_lifetimes(g, ident, align)
    offset, cur = {}, 0
    for b in sorted(buffers):
        offset[b] = cur
        cur += size[b]
    return ArenaPlan(root, buffers, size, defn, last, offset, cur)


def lower_bound(buffers, size, defn, last, n_nodes):
    best = 0
    for t in range(n_nodes):
        best = max(best, sum(size[b] for b in buffers if defn[b] <= t <= last[b]))
    return best


def check_disjoint(plan):
    """True iff no two lifetime-overlapping buffers share a byte."""
    bs = plan.buffers
    for i in range(len(bs)):
        for j in range(i + 1, len(bs)):
            a, b = bs[i], bs[j]
            if overlaps(plan.defn, plan.last, a, b):
                if plan.offset[a] < plan.offset[b] + plan.size[b] and \
                        plan.offset[b] < plan.offset[a] + plan.size[a]:
                    return False
    return True
