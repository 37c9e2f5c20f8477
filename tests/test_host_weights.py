"""Weight layouts planned with their MatMul (CPU, host-only library).

MatMul variants 10-19 run the kernels of 0-9 on the weight stored
K-contiguous.  The planners treat variants alike (the table's minimum over
variants per layout combination), so the weight's layout follows from the
plan's variant; fluid_constant_layout reports it, and a packed variant is
refused for a weight that another node also reads."""
import pytest

from oracle import costtable, plan_layout as PL
from oracle.graph import Graph
from paper_2411_09242_amd import fluid as F
from tables import synthetic_table, write_table
from tinygraphs import ffn_block


@pytest.fixture(scope="module", autouse=True)
def host_lib():
    return F.load(host_only=True)


def _favour(obj, og, node_variant):
    """Make variant v the cheapest for the listed MatMul nodes, everywhere;
    the other operators keep variant 0 (which every one of them has)."""
    for sig in obj["sigs"]:
        if sig["op"] != "matmul":
            for ent in sig["entries"]:
                ent[2] = ent[2][:1]
    for n, v in node_variant.items():
        sig = obj["sigs"][obj["node_sig"][n]]
        for ent in sig["entries"]:
            ent[2] = [5 if i == v else 50 for i in range(20)]
    return obj


def _plan(og, obj, tmp_path):
    g = F.Graph.from_desc(og.export())
    t = F.CostTable.load(write_table(obj, tmp_path / "t.json"), g)
    return g, F.LayoutPlan(g, t)


def test_packed_variant_sets_the_weight_layout(tmp_path):
    og = ffn_block()
    mms = [n for n, nd in enumerate(og.nodes) if nd.op == "matmul"]
    obj = synthetic_table(og, seed=1, mode="random", n_variants=20)
    # distinct signatures per MatMul so that each can be favoured alone
    obj = _favour(obj, og, {mms[0]: 12, mms[1]: 3})
    g, lp = _plan(og, obj, tmp_path)
    ref = PL.plan_layouts(og, costtable.load(obj, og))
    assert lp.variant == ref.variant
    assert lp.variant[mms[0]] == 12 and lp.variant[mms[1]] == 3
    w = {~og.nodes[m].ins[1]: m for m in mms}
    for c, (role, shape, _) in enumerate(og.consts):
        want = (1, 0) if w.get(c) == mms[0] else tuple(range(len(shape)))
        assert lp.constant_layout(c) == want, c
    assert lp.kernel(mms[0]).startswith("gemm_f32_sk32w4_") and "_bk_" in lp.kernel(mms[0])
    assert "_bmn_" in lp.kernel(mms[1])
    ap = F.ArenaPlan(g, lp)
    assert F.fluid_run_launches(g.h, lp.h, ap.h) > 0


def test_packed_variant_refused_for_a_shared_weight(tmp_path):
    """One weight read by two MatMuls cannot be stored in two layouts."""
    og = Graph(dtype="f32")
    x = og.add_input((1, 6, 8))
    w = og.add_const("weight", (8, 8))
    a = og.add_node("matmul", [x, w], (1, 6, 8))
    b = og.add_node("matmul", [a, w], (1, 6, 8))
    og.outputs = [b]
    obj = _favour(synthetic_table(og, seed=2, n_variants=20), og, {0: 11})
    g, lp = _plan(og, obj, tmp_path)
    assert lp.variant[0] == 11
    with pytest.raises(F.FluidError, match="read by this node only"):
        F.ArenaPlan(g, lp, epilogue=True)
