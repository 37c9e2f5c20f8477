"""Layout planner (oracle side): Section 3, Alg. 1-3, Eq. 1 and the merge rule.

Steps, in the paper's order:
  1. ``split``: take the longest operator path of the graph (Alg. 1), remove
     it, and recurse on each weakly connected component of what remains
     (Alg. 2) until every node lies on exactly one path.
  2. ``dp_path``: on each path, a dynamic program over the output layout of
     every node (Eq. 1 / Alg. 3): the best total time to produce a node's
     output in layout b is the best over the previous output's layout a of
     (time so far) + (the node's measured time for those layouts).
  3. Conflicts on edges shared between paths are settled by majority vote;
     the losing paths are then re-optimised with the voted layouts fixed.

Readings where the paper is silent or ambiguous (all deterministic so that
two implementations agree bit for bit):
  * Alg. 1 is described as a Dijkstra-like walk recording the longest
    distance; it is computed as a longest path over the DAG in topological
    order.  Ties: the first input slot whose producer attains the distance,
    and the smallest node id among the path ends.
  * Alg. 2: full recursion; components ordered by their smallest node id.
  * Eq. 1 minimises over the chain predecessor's layout; inputs coming from
    other paths ("boundary" inputs) are minimised per node, ties broken by
    the lexicographically smallest choice.  Back-pointers are kept and the
    path is traced back from the cheapest final layout (smallest index on
    ties), as the text describes.
  * Vote: one ballot per path touching a shared edge (the producing path
    votes its own state, a reading path the layout its best plan assumed at
    its first reading node).  The paper breaks vote ties at random; here the
    tied layout with the lowest summed re-optimised cost of the touching
    paths wins, then the smallest index.
  * Re-optimisation: one more DP of every path with all shared edges fixed.
  * Guard (an addition): if the result costs more than the all-row-major
    plan on the same table, the row-major plan is returned.
Costs are integers (nanoseconds); +infinity is 2**62 with saturating sums.
"""
from __future__ import annotations

import itertools

import numpy as np

from .costtable import INF
from .layouts import node_is_view

NO_DP = 1
NO_VARIANTS = 2
NO_GUARD = 4


class Infeasible(Exception):
    pass


def sat_add(a, b):
    """Saturating add on non-negative int64 values bounded by INF."""
    a = np.minimum(np.asarray(a, dtype=np.int64), INF).astype(np.uint64)
    b = np.minimum(np.asarray(b, dtype=np.int64), INF).astype(np.uint64)
    return np.minimum(a + b, np.uint64(INF)).astype(np.int64)


# ---------------------------------------------------------------- Alg. 1 / 2
def longest_path(g, S):
    """Longest path (in nodes) inside node set S, head first."""
    Sset = set(S)
    dist, pred = {}, {}
    for n in sorted(S):
        preds = []
        for e in g.act_inputs(n):
            p = g.producer(e)
            if p is not None and p in Sset:
                preds.append(p)
        if not preds:
            dist[n], pred[n] = 1, None
        else:
            dist[n] = 1 + max(dist[p] for p in preds)
            pred[n] = next(p for p in preds if dist[p] == dist[n] - 1)
    top = max(dist.values())
    end = min(n for n in S if dist[n] == top)
    path = []
    while end is not None:
        path.append(end)
        end = pred[end]
    return path[::-1]


def _components(g, R):
    Rset = set(R)
    parent = {n: n for n in R}

    def find(n):
        while parent[n] != n:
            parent[n] = parent[parent[n]]
            n = parent[n]
        return n

    for n in R:
        for e in g.act_inputs(n):
            p = g.producer(e)
            if p is not None and p in Rset:
                a, b = find(n), find(p)
                if a != b:
                    parent[max(a, b)] = min(a, b)
    groups = {}
    for n in sorted(R):
        groups.setdefault(find(n), []).append(n)
    return sorted(groups.values(), key=lambda c: c[0])


def split(g, S=None):
    if S is None:
        S = list(range(len(g.nodes)))
    if not S:
        return []
    P = longest_path(g, S)
    Pset = set(P)
    R = [n for n in S if n not in Pset]
    out = [P]
    for c in _components(g, R):
        out.extend(split(g, c))
    return out


# ---------------------------------------------------------------- path info
class PathInfo:
    """Chain slot and boundary edges of every node on a path."""

    def __init__(self, g, path):
        self.path = path
        self.chain_slot = []      # per step: slot index of the chain input or None
        self.bnd_edges = []       # per step: distinct boundary edges, by first slot
        for j, n in enumerate(path):
            slots = g.act_inputs(n)
            cs = None
            if j > 0:
                prev = path[j - 1]
                cs = next(s for s, e in enumerate(slots) if g.producer(e) == prev)
            chain_edge = slots[cs] if cs is not None else None
            be = []
            for s, e in enumerate(slots):
                if s == cs or e == chain_edge:
                    continue
                if e not in be:
                    be.append(e)
            self.chain_slot.append(cs)
            self.bnd_edges.append(be)


def _allowed(L, FIX, e):
    return [FIX[e]] if e in FIX else list(range(len(L[e])))


def _node_gain(g, ct, use_v0, info, j, FIX):
    """G[a, b] = min over boundary layouts beta of C[n][...], and the argmin
    beta (lexicographically smallest on ties).  a ranges over the chain
    edge's full candidate list (size 1 axis when j == 0)."""
    n = info.path[j]
    slots = g.act_inputs(n)
    L = ct.L
    C = ct.nodes[n].v0 if use_v0 else ct.nodes[n].best
    cs = info.chain_slot[j]
    chain_edge = slots[cs] if cs is not None else None
    be = info.bnd_edges[j]
    eo = g.out_edge(n)
    A = len(L[chain_edge]) if chain_edge is not None else 1
    Bn = len(L[eo])
    allowed_b = [_allowed(L, FIX, e) for e in be]
    G = np.full((A, Bn), INF, dtype=np.int64)
    arg = np.full((A, Bn), -1, dtype=np.int64)
    betas = list(itertools.product(*allowed_b))   # lexicographic
    for bi, beta in enumerate(betas):
        lay = {e: beta[i] for i, e in enumerate(be)}
        # index into C: one axis per slot, then the out axis
        idx = []
        for s, e in enumerate(slots):
            if chain_edge is not None and e == chain_edge:
                idx.append(slice(None))
            else:
                idx.append(lay[e])
        sub = C[tuple(idx) + (slice(None),)]
        if chain_edge is None:
            sub = sub.reshape(1, Bn)
        else:
            # several slots may carry the chain edge: take the diagonal
            k = sum(1 for e in slots if e == chain_edge)
            if k > 1:
                sub = np.stack([sub[(a,) * k] for a in range(A)])
            sub = sub.reshape(A, Bn)
        better = sub < G
        G = np.where(better, sub, G)
        arg = np.where(better, bi, arg)
    return G, arg, betas, be


def dp_path(g, ct, use_v0, info, FIX):
    """Viterbi over one path.  Returns (total, states, betas) where states[j]
    is the chosen layout index of the output of step j and betas[j] maps each
    boundary edge of step j to its chosen layout index."""
    L = ct.L
    m = len(info.path)
    Vs, backs, gains = [], [], []
    V = None
    for j in range(m):
        n = info.path[j]
        eo = g.out_edge(n)
        G, arg, betas, be = _node_gain(g, ct, use_v0, info, j, FIX)
        allowed_out = _allowed(L, FIX, eo)
        mask_b = np.full(len(L[eo]), True)
        mask_b[allowed_out] = False
        G = np.where(mask_b[None, :], INF, G)
        if j == 0:
            Vn = G[0].copy()
            back = np.full(len(L[eo]), -1, dtype=np.int64)
        else:
            tot = sat_add(V[:, None], G)                # [a, b]
            back = np.argmin(tot, axis=0)               # first = smallest a
            Vn = tot[back, np.arange(tot.shape[1])]
        Vs.append(Vn)
        backs.append(back)
        gains.append((arg, betas, be))
        V = Vn
    total = int(V.min())
    b = int(np.argmin(V))
    states = [0] * m
    chosen_a = [0] * m
    for j in range(m - 1, -1, -1):
        states[j] = b
        a = int(backs[j][b]) if j > 0 else 0
        chosen_a[j] = a
        b = a
    bsel = []
    for j in range(m):
        arg, betas, be = gains[j]
        bi = int(arg[chosen_a[j] if j > 0 else 0, states[j]])
        beta = betas[bi] if bi >= 0 else tuple(0 for _ in be)
        bsel.append({e: beta[i] for i, e in enumerate(be)})
    return total, states, bsel


# ---------------------------------------------------------------- full plan
class LayoutPlan:
    def __init__(self, layout_idx, variant, total, guard_used, paths):
        self.layout_idx = layout_idx    # per edge
        self.variant = variant          # per node
        self.total = total
        self.guard_used = guard_used
        self.paths = paths


def _node_key(g, n, lay):
    return tuple(lay[e] for e in g.act_inputs(n)) + (lay[g.out_edge(n)],)


def plan_cost(g, ct, use_v0, lay):
    total = 0
    for n in range(len(g.nodes)):
        C = ct.nodes[n].v0 if use_v0 else ct.nodes[n].best
        total = int(sat_add(total, C[_node_key(g, n, lay)]))
    return total


def _variants(g, ct, use_v0, lay):
    perm_of = {e: ct.L[e][lay[e]] for e in range(g.n_edges)}
    out = []
    for n in range(len(g.nodes)):
        if node_is_view(g, n, perm_of):
            out.append(-1)
        elif use_v0:
            out.append(0)
        else:
            out.append(int(ct.nodes[n].var[_node_key(g, n, lay)]))
    return out


def plan_layouts(g, ct, flags=0):
    use_v0 = bool(flags & NO_VARIANTS)
    paths = split(g)
    ident = [0] * g.n_edges
    ident_cost = plan_cost(g, ct, use_v0, ident)
    if ident_cost >= INF:
        raise Infeasible("the all-row-major plan has no cost entry")
    if flags & NO_DP:
        return LayoutPlan(ident, _variants(g, ct, use_v0, ident), ident_cost, 0, paths)

    infos = [PathInfo(g, p) for p in paths]
    owner = {}
    for pi, p in enumerate(paths):
        for n in p:
            owner[g.out_edge(n)] = pi
    readers = {}    # edge -> {path index: lowest step reading it in a boundary slot}
    for pi, info in enumerate(infos):
        for j, be in enumerate(info.bnd_edges):
            for e in be:
                readers.setdefault(e, {})
                readers[e].setdefault(pi, j)
    pinned = set(range(g.n_inputs)) | set(g.outputs)

    FIX = {}
    first = [dp_path(g, ct, use_v0, info, FIX) for info in infos]
    for pi, (tot, _, _) in enumerate(first):
        if tot >= INF:
            raise Infeasible(f"path {pi} has no feasible layout")

    for e in sorted(readers):
        if e in pinned:
            continue
        ballots = []
        touch = []
        if e in owner:
            po = owner[e]
            step = paths[po].index(g.producer(e))
            ballots.append(first[po][1][step])
            touch.append(po)
        for pi in sorted(readers[e]):
            if e in owner and pi == owner[e]:
                continue
            ballots.append(first[pi][2][readers[e][pi]][e])
            touch.append(pi)
        counts = {}
        for b in ballots:
            counts[b] = counts.get(b, 0) + 1
        top = max(counts.values())
        tied = sorted(l for l, c in counts.items() if c == top)
        if len(tied) == 1:
            win = tied[0]
        else:
            best, win = None, None
            for l in tied:
                F2 = dict(FIX)
                F2[e] = l
                c = 0
                for pi in touch:
                    c = int(sat_add(c, dp_path(g, ct, use_v0, infos[pi], F2)[0]))
                if best is None or c < best:
                    best, win = c, l
        FIX[e] = win

    lay = list(ident)
    for pi, info in enumerate(infos):
        tot, states, _ = dp_path(g, ct, use_v0, info, FIX)
        if tot >= INF:
            if flags & NO_GUARD:
                raise Infeasible(f"path {pi} infeasible after the vote")
            return LayoutPlan(ident, _variants(g, ct, use_v0, ident), ident_cost, 1, paths)
        for j, n in enumerate(info.path):
            lay[g.out_edge(n)] = states[j]
    total = plan_cost(g, ct, use_v0, lay)
    if not (flags & NO_GUARD) and total > ident_cost:
        return LayoutPlan(ident, _variants(g, ct, use_v0, ident), ident_cost, 1, paths)
    return LayoutPlan(lay, _variants(g, ct, use_v0, lay), total, 0, paths)
