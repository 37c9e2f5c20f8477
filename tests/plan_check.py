"""Plan parity on one cost table: the C++ layout and arena plans against the
oracle planners run on the same table file (test helper; uses the oracle).

Checks, in order:
  * layout plan (Alg. 1-3 and the vote): layout index per edge, kernel
    variant per node, summed table cost and guard flag;
  * arena plan with the paper's lifetimes (Alg. 4): roots, offsets, peak,
    max-live bound;
  * arena plan with the fusion lifetimes (a MatMul that absorbs the nodes
    after it keeps its operands until the last of them): the same buffers,
    sizes and producers as the paper's plan, every lifetime at least the
    paper's, and offsets and peak equal to the oracle's Greedy-by-Size run on
    exactly those lifetimes, with no two lifetime-overlapping buffers sharing
    a byte.
When the table prices fusion chains, the layout plan's chosen chains
(per MatMul) must match too, and both arena requests must equal the
oracle's arena planned with exactly those chains (their intermediates get
no buffer).
"""
from __future__ import annotations

import json

from oracle import costtable, plan_arena as PA, plan_layout as PL


def assert_plans_match_oracle(og, g, table_obj, lp, flags=0):
    """og: oracle graph; g: the library's graph of the same description;
    table_obj: the cost table (parsed JSON) both planners read; lp: the
    library's layout plan on that table.  Returns a short summary."""
    from paper_2411_09242_amd import fluid as F
    ct = costtable.load(table_obj, og)
    ref = PL.plan_layouts(og, ct, flags)
    assert lp.layout_idx == ref.layout_idx, "layout index per edge"
    assert lp.variant == ref.variant, "kernel variant per node"
    assert lp.total_ns == ref.total, (lp.total_ns, ref.total)
    assert lp.guard_used == ref.guard_used
    lay = {e: ct.L[e][ref.layout_idx[e]] for e in range(og.n_edges)}
    assert lp.fusion_priced == (bool(ct.fused) and not flags & (PL.NO_FUSION | PL.NO_DP))
    if lp.fusion_priced:
        assert lp.fuse == ref.fuse, "fusion chain length per MatMul"
        oap = PA.plan_arena(og, lay, fuse=ref.fuse)
        for epi in (False, True):
            ap = F.ArenaPlan(g, lp, epilogue=epi)
            assert ap.peak == oap.peak
            for e in range(og.n_edges):
                assert ap.root[e] == oap.root[e], e
                r = oap.root[e]
                assert ap.offset[e] == (oap.offset[r] if r in oap.offset else -1), e
            assert ap.lower_bound == PA.lower_bound(oap.buffers, oap.size, oap.defn, oap.last, len(og.nodes))
        return {"total_ns": ref.total, "guard_used": ref.guard_used, "peak": oap.peak,
                "peak_fusion_lifetimes": oap.peak, "extended_lifetimes": 0,
                "fused_chains": sum(1 for t in ref.fuse if t)}

    # the paper's lifetimes
    oap = PA.plan_arena(og, lay)
    ap = F.ArenaPlan(g, lp)
    assert ap.peak == oap.peak
    for e in range(og.n_edges):
        assert ap.root[e] == oap.root[e], e
        r = oap.root[e]
        assert ap.offset[e] == (oap.offset[r] if r in oap.offset else -1), e
    assert ap.lower_bound == PA.lower_bound(oap.buffers, oap.size, oap.defn, oap.last, len(og.nodes))
    lt = ap.lifetimes()
    assert sorted(lt) == sorted(oap.buffers)
    for b, (size, d, last) in lt.items():
        assert (size, d, last) == (oap.size[b], oap.defn[b], oap.last[b]), b

    # the fusion lifetimes
    ape = F.ArenaPlan(g, lp, epilogue=True)
    lte = ape.lifetimes()
    assert sorted(lte) == sorted(oap.buffers)
    last_e = {}
    extended = 0
    for b, (size, d, last) in lte.items():
        assert size == oap.size[b] and d == oap.defn[b], b
        assert oap.last[b] <= last < len(og.nodes), (b, oap.last[b], last)
        extended += last > oap.last[b]
        last_e[b] = last
    off, peak = PA.greedy_by_size(oap.buffers, oap.size, oap.defn, last_e)
    assert ape.peak == peak
    for e in range(og.n_edges):
        assert ape.root[e] == oap.root[e], e
        r = oap.root[e]
        assert ape.offset[e] == (off[r] if r in off else -1), e
    assert PA.check_disjoint(PA.ArenaPlan(oap.root, oap.buffers, oap.size, oap.defn, last_e, off, peak))
    assert ape.lower_bound == PA.lower_bound(oap.buffers, oap.size, oap.defn, last_e, len(og.nodes))
    return {"total_ns": ref.total, "guard_used": ref.guard_used, "peak": oap.peak,
            "peak_fusion_lifetimes": peak, "extended_lifetimes": extended}


def load_json(path):
    with open(path) as f:
        return json.load(f)
