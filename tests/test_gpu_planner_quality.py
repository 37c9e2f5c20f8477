"""Planner quality on cost tables measured on the GPU (the paper's
comparison of the heuristic plan with the brute-force optimum, Section 5.3,
here on real kernel timings instead of synthetic costs).

For small graphs whose every layout assignment can be enumerated: the
library measures a cost table on the GPU; the C++ planner's plan must be
identical to the oracle planner's on that same table (layouts, variants,
total); on a pure chain it must equal the brute-force optimum (Eq. 1 is an
exact dynamic program on one path); on branched graphs it must lie between
the optimum and the row-major plan.  The gap to the optimum is printed.
"""
import json

import pytest

from gpu_util import say
from oracle import brute, costtable, plan_layout as PL
from tinygraphs import chain_graph, diamond_graph, ffn_block, t1_graph, t2_graph

pytestmark = pytest.mark.gpu

GRAPHS = {
    "chain": lambda: chain_graph(5, (3, 40, 64)),
    "diamond": lambda: diamond_graph((2, 48, 64)),
    "t1": t1_graph,
    "t2": t2_graph,
    "ffn": lambda: ffn_block(1, 32, 64, 128),
}


@pytest.mark.parametrize("name", list(GRAPHS))
def test_plan_on_measured_table_vs_brute_force(name, tmp_path):
    from paper_2411_09242_amd import fluid as F
    og = GRAPHS[name]()
    g = F.Graph.from_desc(og.export())
    t = F.CostTable.measure(g, reps=3)
    path = tmp_path / "table.json"
    t.save(str(path))
    ct = costtable.load(json.loads(path.read_text()), og)

    lp = F.LayoutPlan(g, t)
    ref = PL.plan_layouts(og, ct)
    assert list(lp.layout_idx) == list(ref.layout_idx)
    assert list(lp.variant) == list(ref.variant)
    assert lp.total_ns == ref.total

    # with priced fusion chains the optimum also ranges over the chains
    opt = brute.best_layouts_fused(og, ct) if ct.fused else brute.best_layouts(og, ct)[0]
    ident = PL.plan_cost(og, ct, False, [0] * og.n_edges)
    say(f"{name}: plan {lp.total_ns} ns, optimum {opt} ns, row-major {ident} ns, "
        f"plan/optimum {lp.total_ns / max(opt, 1):.4f}")
    assert opt <= lp.total_ns <= ident
    if name == "chain":
        nog = PL.plan_layouts(og, ct, PL.NO_GUARD)
        assert nog.total == opt
