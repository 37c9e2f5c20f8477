"""Candidate layouts, strides and the view predicate (oracle side).

A layout of a tensor with logical shape ``d`` is a permutation ``pi`` of its
dimensions listed outermost -> innermost; the tensor is stored densely in
that order, i.e. as ``X.transpose(pi)`` made contiguous.  The paper
schedules "all possible layouts" of each edge (Alg. 3) without defining
them; here they are all r! permutations in lexicographic order, with
physically identical ones (equal once extent-1 dimensions are deleted)
merged into the first.  Graph inputs and outputs are fixed to row-major.

A Transpose or Reshape node costs nothing when its output layout makes the
output a relabelling of the input's bytes; that is how a chosen layout
removes an explicit transpose.
"""
from __future__ import annotations

import itertools


def physical_key(shape, perm):
    return tuple(d for d in perm if shape[d] != 1)


def layout_list(shape):
    """All layouts of ``shape``, lexicographic, deduplicated; identity first."""
    r = len(shape)
    seen, out = set(), []
    for p in itertools.permutations(range(r)):
        k = physical_key(shape, p)
        if k not in seen:
            seen.add(k)
            out.append(tuple(p))
    return out


def identity(r):
    return tuple(range(r))


def edge_layouts(g):
    """L(e) for every activation edge; graph inputs/outputs pinned to identity."""
    pinned = set(range(g.n_inputs)) | set(g.outputs)
    L = []
    for e in range(g.n_edges):
        s = g.edge_shape(e)
        L.append([identity(len(s))] if e in pinned else layout_list(s))
    return L


def strides(shape, perm):
    """Element strides per logical dim for a dense tensor stored in ``perm`` order."""
    st = [0] * len(shape)
    acc = 1
    for d in reversed(perm):
        st[d] = acc
        acc *= shape[d]
    return st


def reshape_kind(xs, ys):
    """('split', a): X dim a -> Y dims (a, a+1);  ('merge', a): X dims (a, a+1)
    -> Y dim a;  ('same', -1) for equal shapes;  ('other', -1) otherwise."""
    xs, ys = tuple(xs), tuple(ys)
    if xs == ys:
        return "same", -1
    if len(ys) == len(xs) + 1:
        for a in range(len(xs)):
            if ys[:a] == xs[:a] and ys[a] * ys[a + 1] == xs[a] and ys[a + 2:] == xs[a + 1:]:
                return "split", a
    if len(ys) == len(xs) - 1:
        for a in range(len(ys)):
            if xs[:a] == ys[:a] and xs[a] * xs[a + 1] == ys[a] and xs[a + 2:] == ys[a + 1:]:
                return "merge", a
    return "other", -1


def _collapse(seq, shape, a):
    """Physical dim sequence ``seq`` of a tensor in which dims (a, a+1) are the
    two halves of one coarser dim: drop extent-1 dims, require a immediately
    followed by a+1 when both remain, merge them, renumber.  None if they are
    not adjacent in that order."""
    s = [d for d in seq if shape[d] != 1]
    both = shape[a] != 1 and shape[a + 1] != 1
    out, i = [], 0
    while i < len(s):
        d = s[i]
        if d in (a, a + 1):
            if both:
                if d != a or i + 1 >= len(s) or s[i + 1] != a + 1:
                    return None
                i += 2
            else:
                i += 1
            out.append(a)
            continue
        out.append(d if d < a else d - 1)
        i += 1
    return out


def is_view(op, perm, xs, ys, lin, lout):
    """True iff output layout ``lout`` makes the node's output a relabelling of
    its input stored in layout ``lin`` (identical byte offsets for every
    element).  Only Transpose and split/merge Reshape can be views."""
    xs, ys = tuple(xs), tuple(ys)
    if op == "transpose":
        mapped = [perm[s] for s in lout if ys[s] != 1]
        return mapped == [d for d in lin if xs[d] != 1]
    if op == "reshape":
        kind, a = reshape_kind(xs, ys)
        if kind == "same":
            return physical_key(xs, lin) == physical_key(ys, lout)
        if kind == "split":
            c = _collapse(lout, ys, a)
            return c is not None and c == [d for d in lin if xs[d] != 1]
        if kind == "merge":
            c = _collapse(lin, xs, a)
            return c is not None and c == [s for s in lout if ys[s] != 1]
    return False


def node_is_view(g, n, layout_of_edge):
    """View test for node n under an edge->layout mapping.  A node whose output
    is a graph output is never a view (the caller's buffer must be written)."""
    nd = g.nodes[n]
    if nd.op not in ("transpose", "reshape"):
        return False
    if g.out_edge(n) in g.outputs:
        return False
    e_in = g.act_inputs(n)[0]
    return is_view(nd.op, nd.perm, g.edge_shape(e_in), nd.out_shape,
                   layout_of_edge[e_in], layout_of_edge[g.out_edge(n)])
