"""Reader for the JSON cost-table file (oracle side).

The paper's planner calls ``eval(node, layouts)`` for the real-world time of
a node under given input and output layouts (Alg. 3).  Here those times are
frozen in a file so that two independent planners can be run on identical
numbers.  Format ("fluid-cost-table/1"):

  edges     : for every activation edge e, the list L(e) of candidate
              layouts (permutations), identity first
  sigs      : operator signatures, each with "entries" =
              [[slot_perms...], out_perm, [cost_ns per kernel variant]]
              (a cost of -1 means that variant is unavailable)
  node_sig  : the signature index of every node
  fused_sigs, fused (optional): measured costs of fusion chains (see
              oracle/fusion.py) -- fused_sigs holds signatures like sigs,
              whose entries list the layouts of the chain's slots (the
              MatMul's activation inputs, then R of an Add / Mul step) and of
              the last node's output; fused lists [m, t, signature index]
              for the chain of the MatMul node m and length t

A node's activation slots (constants excluded) are listed in slot order.
Missing combinations cost +infinity.  Layout-only (view) combinations carry
the single cost 0.
"""
from __future__ import annotations

import json

import numpy as np

from . import fusion

INF = 1 << 62


class NodeCosts:
    """Dense per-node arrays over (slot layout idx..., out layout idx)."""

    def __init__(self, best, var, v0):
        self.best = best      # int64, min over variants (INF if none)
        self.var = var        # int32, argmin variant (lowest on ties), -1 if none
        self.v0 = v0          # int64, variant-0 cost (INF if unavailable)


class CostTable:
    def __init__(self, L, nodes, fused=None):
        self.L = L            # list of lists of perms
        self.nodes = nodes    # list of NodeCosts
        self.fused = fused or {}   # (m, t) -> NodeCosts over the chain's slots + output


def load(path_or_obj, g):
    obj = path_or_obj
    if isinstance(path_or_obj, str):
        with open(path_or_obj) as f:
            obj = json.load(f)
    if obj.get("format") != "fluid-cost-table/1":
        raise ValueError("bad format tag")
    L = [[tuple(p) for p in lst] for lst in obj["edges"]]
    if len(L) != g.n_edges:
        raise ValueError("edge count mismatch")
    for e, lst in enumerate(L):
        r = len(g.edge_shape(e))
        if not lst or lst[0] != tuple(range(r)):
            raise ValueError(f"L({e}) must start with the identity layout")
    if len(obj["node_sig"]) != len(g.nodes):
        raise ValueError("node count mismatch")
    def dense(slots, eo, entries, what):
        dims = [len(L[e]) for e in slots] + [len(L[eo])]
        best = np.full(dims, INF, dtype=np.int64)
        var = np.full(dims, -1, dtype=np.int32)
        v0 = np.full(dims, INF, dtype=np.int64)
        index = [{p: i for i, p in enumerate(L[e])} for e in slots + [eo]]
        for ent in entries:
            perms = [tuple(p) for p in ent[0]] + [tuple(ent[1])]
            if len(perms) != len(dims):
                raise ValueError(f"{what}: entry arity mismatch")
            try:
                key = tuple(index[i][p] for i, p in enumerate(perms))
            except KeyError:
                continue  # a layout outside this node's candidate lists
            costs = list(ent[2])
            ok = [(c, v) for v, c in enumerate(costs) if c >= 0]
            if ok:
                c, v = min(ok)   # lowest cost, then lowest variant id
                best[key] = c
                var[key] = v
            if costs and costs[0] >= 0:
                v0[key] = costs[0]
        return NodeCosts(best, var, v0)

    nodes = [dense(g.act_inputs(n), g.out_edge(n), obj["sigs"][sig]["entries"], f"node {n}")
             for n, sig in enumerate(obj["node_sig"])]
    fused = {}
    chains = fusion.all_chains(g)
    for m, t, si in obj.get("fused", []):
        if (m, t) not in chains:
            raise ValueError(f"fused entry ({m}, {t}) is not a fusion chain of this graph")
        if (m, t) in fused:
            raise ValueError(f"fused entry ({m}, {t}) listed twice")
        if not 0 <= si < len(obj.get("fused_sigs", [])):
            raise ValueError(f"fused entry ({m}, {t}): no signature {si}")
        fused[(m, t)] = dense(fusion.chain_slots(g, m, t), g.out_edge(m + t), obj["fused_sigs"][si]["entries"],
                              f"chain ({m}, {t})")
    return CostTable(L, nodes, fused)
