"""Exhaustive searches used to pin the oracle on tiny inputs.

* ``view_by_offsets``: the definition of a zero-copy view written out --
  every element of the output has the same byte offset as the input element
  it equals -- checked element by element.
* ``best_arena_peak``: the optimal peak of a static placement of at most ~8
  buffers.  For every order of the buffers, each one goes to the lowest
  offset that clears all lifetime-overlapping buffers placed before it
  (candidates: 0 and the ends of those buffers); the minimum peak over all
  orders is the optimum (order any optimal packing by offset and place in
  that order: no buffer lands above its optimal offset).
* ``best_layouts``: the minimum total cost over every assignment of
  candidate layouts to the non-pinned edges (the paper's brute-force
  "optimal schedule", Section 5.3); ties go to the lexicographically
  smallest assignment in edge order.
"""
from __future__ import annotations

import itertools

import numpy as np

from .costtable import INF
from .layouts import strides


def view_by_offsets(op, perm, xs, ys, lin, lout):
    xs, ys = tuple(xs), tuple(ys)
    n = int(np.prod(xs))
    sx = strides(xs, lin)
    sy = strides(ys, lout)
    # byte (element) offset of every logical element of X, in X's row-major order
    idx_x = np.indices(xs).reshape(len(xs), -1)
    off_x = (np.asarray(sx)[:, None] * idx_x).sum(0).reshape(xs)
    if op == "transpose":
        off_x_as_y = np.transpose(off_x, perm)
    else:
        off_x_as_y = off_x.reshape(ys)
    idx_y = np.indices(ys).reshape(len(ys), -1)
    off_y = (np.asarray(sy)[:, None] * idx_y).sum(0).reshape(ys)
    return n == int(np.prod(ys)) and bool(np.array_equal(off_x_as_y, off_y))


def best_arena_peak(buffers, size, defn, last):
    def ov(a, b):
        return defn[a] <= last[b] and defn[b] <= last[a]
    best = None
    for order in itertools.permutations(buffers):
        off = {}
        for b in order:
            cands = sorted({0} | {off[o] + size[o] for o in off if ov(o, b)})
            for c in cands:
                if all(not ov(o, b) or c + size[b] <= off[o] or off[o] + size[o] <= c
                       for o in off):
                    off[b] = c
                    break
        peak = max((off[b] + size[b] for b in buffers), default=0)
        if best is None or peak < best:
            best = peak
    return best if best is not None else 0


def best_layouts(g, ct, use_v0=False):
    """(total, layout index per edge) minimising the summed node cost."""
    free = [e for e in range(g.n_edges) if len(ct.L[e]) > 1]
    best = None
    lay = [0] * g.n_edges
    for assign in itertools.product(*[range(len(ct.L[e])) for e in free]):
        for e, l in zip(free, assign):
            lay[e] = l
        tot = 0
        for n in range(len(g.nodes)):
            C = ct.nodes[n].v0 if use_v0 else ct.nodes[n].best
            key = tuple(lay[e] for e in g.act_inputs(n)) + (lay[g.out_edge(n)],)
            tot = min(tot + int(C[key]), INF)
            if tot >= INF:
                break
        if best is None or tot < best[0]:
            best = (tot, list(lay))
    return best


def best_layouts_fused(g, ct, use_v0=False):
    """The minimum total cost over every layout assignment of the
    non-pinned edges and every set of non-overlapping fusion chains with
    measured costs (ct.fused): a chain (m, t) costs its fused entry at the
    layouts of its slots and of node m+t's output, every other node its own
    entry.  Returns the minimum total."""
    chains = sorted(ct.fused)
    choices = []
    for k in range(len(chains) + 1):
        for sel in itertools.combinations(chains, k):
            spans = [set(range(m, m + t + 1)) for m, t in sel]
            if all(not (a & b) for i, a in enumerate(spans) for b in spans[i + 1:]):
                choices.append(sel)
    free = [e for e in range(g.n_edges) if len(ct.L[e]) > 1]
    best = None
    lay = [0] * g.n_edges
    for assign in itertools.product(*[range(len(ct.L[e])) for e in free]):
        for e, l in zip(free, assign):
            lay[e] = l
        for sel in choices:
            covered = {n for m, t in sel for n in range(m, m + t + 1)}
            tot = 0
            for m, t in sel:
                C = ct.fused[(m, t)].v0 if use_v0 else ct.fused[(m, t)].best
                slots = list(g.act_inputs(m))
                last = g.nodes[m + t]
                if last.op in ("add", "mul"):
                    other = [v for v in last.ins if v >= 0 and v != g.out_edge(m + t - 1)]
                    slots += other[:1]
                key = tuple(lay[e] for e in slots) + (lay[g.out_edge(m + t)],)
                c = int(C[key])
                # a residual sum read also after its norm is stored by the
                # launch, in the norm output's layout
                e0, eo = g.out_edge(m), g.out_edge(m + t)
                if g.nodes[m].op == "add" and sum(1 for x in g.nodes if e0 in x.ins) > 1 and \
                        ct.L[e0][lay[e0]] != ct.L[eo][lay[eo]]:
                    c = INF
                tot = min(tot + c, INF)
            for n in range(len(g.nodes)):
                if n in covered:
                    continue
                C = ct.nodes[n].v0 if use_v0 else ct.nodes[n].best
                key = tuple(lay[e] for e in g.act_inputs(n)) + (lay[g.out_edge(n)],)
                tot = min(tot + int(C[key]), INF)
            if best is None or tot < best:
                best = tot
    return best
