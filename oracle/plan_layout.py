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
  * Fusion chains (an addition, see fusion.py), when the table prices them:
    the path DP may also step over a chain, the chain's fused entry standing
    in for its nodes' own.  After the vote, the chains are chosen anew for
    the final layouts, exactly: chains are runs of consecutive node ids, so
    the cheapest set of disjoint chains is an interval DP over node ids
    (ties: a node on its own, then the shorter chain).  Two voted layout
    assignments compete -- the one from the fusion-aware DP and the one
    from the plain DP (the paper's) -- each with its best chains; the
    cheaper total wins, the fusion-aware one on ties.  The guard compares
    with the row-major plan with its best chains.
Costs are integers (nanoseconds); +infinity is 2**62 with saturating sums.
"""
from __future__ import annotations

import itertools

import numpy as np

from . import fusion
from .costtable import INF
from .layouts import node_is_view

NO_DP = 1
NO_VARIANTS = 2
NO_GUARD = 4
NO_FUSION = 8


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


def _gain(L, C, slots, chain_edge, be, eo, FIX):
    """G[a, b] = min over boundary layouts beta of C[slot layouts..., b] with
    the chain edge in layout a, and the argmin beta (lexicographically
    smallest on ties).  a ranges over the chain edge's full candidate list
    (a size-1 axis when there is no chain edge)."""
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
        for e in slots:
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


def _node_gain(g, ct, use_v0, info, j, FIX):
    """The gain of step j run as its own node."""
    n = info.path[j]
    slots = g.act_inputs(n)
    C = ct.nodes[n].v0 if use_v0 else ct.nodes[n].best
    cs = info.chain_slot[j]
    chain_edge = slots[cs] if cs is not None else None
    return _gain(ct.L, C, slots, chain_edge, info.bnd_edges[j], g.out_edge(n), FIX)


def fused_options(g, ct, info, j):
    """Chain lengths t for which steps j .. j+t of the path form a fusion
    chain with measured costs (the MatMul at step j, nodes m+1 .. m+t)."""
    m = info.path[j]
    out = []
    for t in (1, 2, 3):
        if (m, t) in ct.fused and j + t < len(info.path) and \
                all(info.path[j + i] == m + i for i in range(1, t + 1)):
            out.append(t)
    return out


def store_index(L, e_store, e_out, b):
    """The index in L(e_store) of the permutation L(e_out)[b] -- the layout
    a chain's stored intermediate takes when the chain's output takes b --
    or None when e_store has no such candidate."""
    p = L[e_out][b]
    return L[e_store].index(p) if p in L[e_store] else None


def chain_layouts_ok(g, L, m, t, lay):
    """Whether every intermediate the chain (m, t) stores has the layout of
    the chain's output under the assignment lay."""
    eo = g.out_edge(m + t)
    return all(lay[e] == store_index(L, e, eo, lay[eo]) for e in fusion.stored_edges(g, m, t))


def _fused_gain(g, ct, use_v0, info, j, t, FIX):
    """The gain of steps j .. j+t run as one fused launch: a virtual node
    whose slots are the chain's (the MatMul's activation inputs, then R) and
    whose output is the last node's.  An output layout b that a stored
    intermediate cannot take (no such candidate, or fixed otherwise) is
    infeasible."""
    m = info.path[j]
    slots = fusion.chain_slots(g, m, t)
    cs = info.chain_slot[j]
    chain_edge = g.act_inputs(m)[cs] if cs is not None else None
    be = []
    for e in slots:
        if e != chain_edge and e not in be:
            be.append(e)
    NC = ct.fused[(m, t)]
    eo = g.out_edge(m + t)
    G, arg, betas, be = _gain(ct.L, NC.v0 if use_v0 else NC.best, slots, chain_edge, be, eo, FIX)
    for e in fusion.stored_edges(g, m, t):
        for b in range(len(ct.L[eo])):
            k = store_index(ct.L, e, eo, b)
            if k is None or (e in FIX and FIX[e] != k):
                G[:, b] = INF
                arg[:, b] = -1
    return G, arg, betas, be


def dp_path(g, ct, use_v0, info, FIX, fuse=True):
    """Viterbi over one path.  Returns (total, states, betas, fused) where
    states[j] is the chosen layout index of the output of step j (0 for a
    result a fused launch keeps on chip), betas[j] maps each boundary edge
    of step j to its chosen layout index, and fused[j] is the length t of
    the fused chain starting at step j (0 when step j runs on its own).

    A step's output layout b is reached either by the step's own node from
    the previous step's layout a, or -- when fusion chains are priced -- by
    the fused launch of the chain ending there, from the layout a of the
    step before the chain.  Ties: the lower cost, then the shorter
    transition (a node on its own first), then the smaller a."""
    L = ct.L
    m = len(info.path)
    opts = [fused_options(g, ct, info, j) if fuse else [] for j in range(m)]
    Vs, backs, choices = [], [], []
    for j in range(m):
        n = info.path[j]
        eo = g.out_edge(n)
        allowed_out = _allowed(L, FIX, eo)
        mask_b = np.full(len(L[eo]), True)
        mask_b[allowed_out] = False
        cands = []   # (t, start, G, arg, betas, be)
        G, arg, betas, be = _node_gain(g, ct, use_v0, info, j, FIX)
        cands.append((0, j, G, arg, betas, be))
        for s in range(j - 1, max(0, j - 3) - 1, -1):    # t = 1, 2, 3
            t = j - s
            if t in opts[s]:
                Gf, argf, betasf, bef = _fused_gain(g, ct, use_v0, info, s, t, FIX)
                cands.append((t, s, Gf, argf, betasf, bef))
        Vn = np.full(len(L[eo]), INF, dtype=np.int64)
        back = [(0, 0)] * len(L[eo])
        for t, s, G, arg, betas, be in cands:
            G = np.where(mask_b[None, :], INF, G)
            if s == 0:
                tot = G[0]
                aa = np.zeros(len(L[eo]), dtype=np.int64)
            else:
                full = sat_add(Vs[s - 1][:, None], G)     # [a, b]
                aa = np.argmin(full, axis=0)               # first = smallest a
                tot = full[aa, np.arange(full.shape[1])]
            for b in range(len(L[eo])):
                # the node on its own always sets the state (also at +inf);
                # a fused launch replaces it only when strictly cheaper
                if t == 0 or tot[b] < Vn[b]:
                    Vn[b] = tot[b]
                    back[b] = (t, int(aa[b]))
        Vs.append(Vn)
        backs.append(back)
        choices.append({t: (s, arg, betas, be) for t, s, G, arg, betas, be in cands})
    total = int(Vs[-1].min())
    b = int(np.argmin(Vs[-1]))
    states = [0] * m
    fused = [0] * m
    bsel = [dict() for _ in range(m)]
    j = m - 1
    while j >= 0:
        t, a = backs[j][b]
        s, arg, betas, be = choices[j][t]
        states[j] = b
        bi = int(arg[a if s > 0 else 0, b])
        beta = betas[bi] if bi >= 0 else tuple(0 for _ in be)
        chosen = {e: beta[i] for i, e in enumerate(be)}
        if s > 0:   # a boundary read of the launch's chain edge sees layout a
            chosen.setdefault(g.act_inputs(info.path[s])[info.chain_slot[s]], a)
        # a boundary edge's layout is recorded at every step of the launch
        # that reads it as a boundary edge
        for k in range(s, j + 1):
            bsel[k] = {e: chosen[e] for e in info.bnd_edges[k] if e in chosen}
        if t:
            # an intermediate the launch stores takes the output's layout
            m0 = info.path[s]
            for e in fusion.stored_edges(g, m0, t):
                states[s + (g.producer(e) - m0)] = store_index(ct.L, e, g.out_edge(m0 + t), b)
        fused[s] = t
        j = s - 1
        b = a
    return total, states, bsel, fused


# ---------------------------------------------------------------- full plan
class LayoutPlan:
    def __init__(self, layout_idx, variant, total, guard_used, paths, fuse=None):
        self.layout_idx = layout_idx    # per edge
        self.variant = variant          # per node (-1 view, -2 performed in a MatMul's fused launch)
        self.total = total
        self.guard_used = guard_used
        self.paths = paths
        self.fuse = fuse or [0] * len(variant)   # per node: chain length of a fused MatMul, else 0


def _node_key(g, n, lay):
    return tuple(lay[e] for e in g.act_inputs(n)) + (lay[g.out_edge(n)],)


def _chain_key(g, m, t, lay):
    return tuple(lay[e] for e in fusion.chain_slots(g, m, t)) + (lay[g.out_edge(m + t)],)


def plan_cost(g, ct, use_v0, lay, fuse=None):
    """Summed table cost of a plan: every node on its own, except the fused
    chains (fuse[m] = t), which cost their fused entry."""
    fuse = fuse or [0] * len(g.nodes)
    total = 0
    n = 0
    while n < len(g.nodes):
        if fuse[n]:
            NC = ct.fused[(n, fuse[n])]
            C = NC.v0 if use_v0 else NC.best
            c = int(C[_chain_key(g, n, fuse[n], lay)]) if chain_layouts_ok(g, ct.L, n, fuse[n], lay) else INF
            total = int(sat_add(total, c))
            n += fuse[n] + 1
            continue
        C = ct.nodes[n].v0 if use_v0 else ct.nodes[n].best
        total = int(sat_add(total, C[_node_key(g, n, lay)]))
        n += 1
    return total


def _variants(g, ct, use_v0, lay, fuse=None):
    fuse = fuse or [0] * len(g.nodes)
    perm_of = {e: ct.L[e][lay[e]] for e in range(g.n_edges)}
    out = []
    absorbed = set()
    for m, t in enumerate(fuse):
        absorbed.update(range(m + 1, m + t + 1))
    for n in range(len(g.nodes)):
        if n in absorbed:
            out.append(-2)
        elif node_is_view(g, n, perm_of):
            out.append(-1)
        elif use_v0:
            out.append(0)
        elif fuse[n]:
            out.append(int(ct.fused[(n, fuse[n])].var[_chain_key(g, n, fuse[n], lay)]))
        else:
            out.append(int(ct.nodes[n].var[_node_key(g, n, lay)]))
    return out


def plan_layouts(g, ct, flags=0):
    use_v0 = bool(flags & NO_VARIANTS)
    fz = not (flags & NO_FUSION)
    paths = split(g)
    ident = [0] * g.n_edges
    ident_cost = plan_cost(g, ct, use_v0, ident)
    if ident_cost >= INF:
        raise Infeasible("the all-row-major plan has no cost entry")
    if flags & NO_DP:
        return LayoutPlan(ident, _variants(g, ct, use_v0, ident), ident_cost, 0, paths)

    priced = fz and bool(ct.fused)
    if priced:
        ident_fuse = best_chains(g, ct, use_v0, ident)
        ident_cost = plan_cost(g, ct, use_v0, ident, ident_fuse)
    else:
        ident_fuse = None
    infos = [PathInfo(g, p) for p in paths]
    cands = []
    for fz_dp in ((True, False) if priced else (False,)):
        lay = _voted_layouts(g, ct, use_v0, paths, infos, fz_dp)
        if lay is None:
            continue
        fuse = best_chains(g, ct, use_v0, lay) if priced else None
        cands.append((plan_cost(g, ct, use_v0, lay, fuse), lay, fuse))
    if not cands:
        if flags & NO_GUARD:
            raise Infeasible("every path plan is infeasible after the vote")
        return LayoutPlan(ident, _variants(g, ct, use_v0, ident, ident_fuse), ident_cost, 1, paths, ident_fuse)
    total, lay, fuse = min(cands, key=lambda c: c[0])   # the first on ties
    if not (flags & NO_GUARD) and total > ident_cost:
        return LayoutPlan(ident, _variants(g, ct, use_v0, ident, ident_fuse), ident_cost, 1, paths, ident_fuse)
    return LayoutPlan(lay, _variants(g, ct, use_v0, lay, fuse), total, 0, paths, fuse)


def best_chains(g, ct, use_v0, lay):
    """The cheapest set of disjoint fusion chains for fixed layouts: per
    node, fuse[m] = t for a chain (m, t) run as one launch, else 0.  Chains
    cover consecutive node ids, so this is an interval DP from the last node
    back: f(n) = min(cost of n on its own + f(n+1), min over chains (n, t) of
    their fused entry + f(n+t+1)); ties keep the node on its own, then the
    shorter chain."""
    N = len(g.nodes)
    f = [0] * (N + 1)
    pick = [0] * N
    for n in range(N - 1, -1, -1):
        C = ct.nodes[n].v0 if use_v0 else ct.nodes[n].best
        f[n] = int(sat_add(C[_node_key(g, n, lay)], f[n + 1]))
        t = 1
        while (n, t) in ct.fused:
            if chain_layouts_ok(g, ct.L, n, t, lay):
                NC = ct.fused[(n, t)]
                c = int(sat_add((NC.v0 if use_v0 else NC.best)[_chain_key(g, n, t, lay)], f[n + t + 1]))
                if c < f[n]:
                    f[n], pick[n] = c, t
            t += 1
    fuse = [0] * N
    n = 0
    while n < N:
        fuse[n] = pick[n]
        n += pick[n] + 1
    return fuse


def _voted_layouts(g, ct, use_v0, paths, infos, fz):
    """The first DP of every path, the vote on shared edges and the
    re-optimisation with the voted layouts fixed: the layout index per edge,
    or None when a path has no feasible plan after the vote."""
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
    first = [dp_path(g, ct, use_v0, info, FIX, fz) for info in infos]
    for pi, (tot, _, _, _) in enumerate(first):
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
                    c = int(sat_add(c, dp_path(g, ct, use_v0, infos[pi], F2, fz)[0]))
                if best is None or c < best:
                    best, win = c, l
        FIX[e] = win

    lay = [0] * g.n_edges
    for info in infos:
        tot, states, _, _ = dp_path(g, ct, use_v0, info, FIX, fz)
        if tot >= INF:
            return None
        for j, n in enumerate(info.path):
            lay[g.out_edge(n)] = states[j]
    return lay
