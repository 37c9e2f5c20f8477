"""Synthetic cost tables for planner tests (test helper; uses the oracle).

The tables are seeded inputs to both planners.  Candidate layout lists and
the view predicate come from the oracle; costs are random integers, so the
same file can be handed to the oracle planner and to the C++ planner.
"""
from __future__ import annotations

import json

import numpy as np

from oracle import layouts


def _sig_key(g, n):
    nd = g.nodes[n]
    ins = [tuple(g.edge_shape(e)) for e in g.act_inputs(n)]
    cs = [tuple(g.consts[~v][1]) for v in nd.ins if v < 0]
    return (nd.op, tuple(ins), tuple(cs), tuple(nd.out_shape), nd.perm,
            nd.fattr, nd.iattr)


def synthetic_table(g, seed, mode="random", n_variants=3, lo=1, hi=1000,
                    drop_identity_node=None):
    """Build a cost table dict.  Modes:
      random    -- uniform integer costs in [lo, hi] per variant (some -1)
      ties      -- every non-view cost equal (ties everywhere)
      identity  -- identity combination cheapest for every node
      distinct  -- all costs distinct (no ties anywhere in sums is likely)
    """
    rng = np.random.default_rng(seed)
    L = layouts.edge_layouts(g)
    sig_index, sigs, node_sig = {}, [], []
    for n, nd in enumerate(g.nodes):
        key = _sig_key(g, n)
        if key in sig_index and n != drop_identity_node:
            node_sig.append(sig_index[key])
            continue
        slot_shapes = [g.edge_shape(e) for e in g.act_inputs(n)]
        lists = [layouts.layout_list(s) for s in slot_shapes]
        out_list = layouts.layout_list(nd.out_shape)
        entries = []
        for combo in __import__("itertools").product(*lists, out_list):
            ins, out = combo[:-1], combo[-1]
            if nd.op in ("transpose", "reshape") and layouts.is_view(
                    nd.op, nd.perm, slot_shapes[0], nd.out_shape, ins[0], out):
                entries.append([[list(p) for p in ins], list(out), [0]])
                continue
            ident = all(p == tuple(range(len(p))) for p in combo)
            if n == drop_identity_node and ident:
                continue
            if mode == "ties":
                costs = [100] * n_variants
            elif mode == "identity":
                costs = [10 if ident else int(rng.integers(11, hi + 1))
                         for _ in range(n_variants)]
            elif mode == "distinct":
                costs = [int(rng.integers(0, 1 << 40)) for _ in range(n_variants)]
            else:
                costs = [int(rng.integers(lo, hi + 1)) for _ in range(n_variants)]
                for v in range(1, n_variants):
                    if rng.random() < 0.2:
                        costs[v] = -1
            entries.append([[list(p) for p in ins], list(out), costs])
        sig_index.setdefault(key, len(sigs))
        node_sig.append(len(sigs))
        sigs.append({"op": nd.op, "in_shapes": [list(s) for s in slot_shapes],
                     "out_shape": list(nd.out_shape), "entries": entries})
    return {"format": "fluid-cost-table/1",
            "edges": [[list(p) for p in lst] for lst in L],
            "sigs": sigs, "node_sig": node_sig}


def write_table(obj, path):
    with open(path, "w") as f:
        json.dump(obj, f)
    return str(path)


def rank2_table(g, costs):
    """A hand-written table for a graph of [2,3] tensors.  costs[n] is a dict
    {(slot layout idx ..., out idx): cost}; the layouts of a [2,3] tensor are
    (0,1) row-major = 0 and (1,0) = 1; graph inputs and outputs keep only
    row-major.  A combination absent from costs[n] has no entry (+inf)."""
    P = [[0, 1], [1, 0]]
    L = []
    for e in range(g.n_edges):
        pinned = e < g.n_inputs or e in g.outputs
        L.append([P[0]] if pinned else P)
    sigs = []
    for n in range(len(g.nodes)):
        ents = [[[P[i] for i in key[:-1]], P[key[-1]], [c]] for key, c in costs[n].items()]
        sigs.append({"op": g.nodes[n].op, "in_shapes": [], "out_shape": [2, 3], "entries": ents})
    return {"format": "fluid-cost-table/1", "edges": L, "sigs": sigs,
            "node_sig": list(range(len(g.nodes)))}


def fanout_costs(infeasible_after_vote=False):
    """Costs for tinygraphs.fanout_graph where the majority vote hurts.
    Node order: a, b, b2, c, d, s, y.  Path [a b b2 s y] pays 100 more on b
    when a is column-major; paths [c] and [d] each save 1 with a
    column-major.  With infeasible_after_vote, b has no entry at all for a
    column-major a, so the path that owns a cannot follow the vote."""
    same = {(0, 0): 10, (1, 1): 10, (0, 1): 50, (1, 0): 50}
    if infeasible_after_vote:
        b = {(0, 0): 10, (0, 1): 110}
    else:
        b = {(0, 0): 10, (1, 0): 110, (0, 1): 110, (1, 1): 110}
    reader = {(0, 0): 10, (1, 0): 9, (0, 1): 50, (1, 1): 50}
    import itertools
    add3 = {k: (10 if k == (0, 0, 0) else 100) for k in itertools.product((0, 1), repeat=3)}
    return [
        {(0, 0): 10, (0, 1): 10},                                # a (x pinned)
        b,                                                       # b
        dict(same),                                              # b2
        dict(reader),                                            # c
        dict(reader),                                            # d
        add3,                                                    # s
        {k: v for k, v in add3.items() if k[2] == 0},            # y (pinned)
    ]


def add_fused(obj, g, seed, n_variants=3, lo=1, hi=1000, scale=1.0):
    """Adds random fused entries for every fusion chain of g (oracle's
    chain rules) to a synthetic table: costs over the chain's slots and the
    last node's output, drawn like the node entries (times `scale`)."""
    from oracle import fusion
    rng = np.random.default_rng(seed + 12345)
    L = layouts.edge_layouts(g)
    obj["fused_sigs"], obj["fused"] = [], []
    for (m, t), nodes in sorted(fusion.all_chains(g).items()):
        slots = fusion.chain_slots(g, m, t)
        eo = g.out_edge(m + t)
        entries = []
        for combo in __import__("itertools").product(*[L[e] for e in slots], L[eo]):
            costs = [int(scale * rng.integers(lo, hi + 1)) for _ in range(n_variants)]
            entries.append([[list(p) for p in combo[:-1]], list(combo[-1]), costs])
        obj["fused"].append([m, t, len(obj["fused_sigs"])])
        obj["fused_sigs"].append({"op": g.nodes[m].op, "steps": t, "in_shapes": [list(g.edge_shape(e)) for e in slots],
                                  "out_shape": list(g.edge_shape(eo)), "entries": entries})
    return obj
