"""Causal attention products (host library, no GPU).

A batched MatMul whose only reader is a causal Softmax never has the
entries above that Softmax's diagonal read (the softmax takes only key <=
query); a MatMul whose A operand is a causal Softmax's output has exact zeros
there.  The graph marks both and the kernels skip the corresponding tiles
and K ranges; the mark shows in the kernel name.  The skipped products are
exact zeros (or never read), so the outputs do not change -- the GPU parity
tests check that against the oracle.
"""
import pytest

from oracle.graph import Graph
from tables import synthetic_table, write_table


def attention(causal=1, s_is_output=False, extra_reader=False):
    g = Graph(dtype="f32")
    q = g.add_input((1, 2, 40, 16))
    kt = g.add_input((1, 2, 16, 40))
    v = g.add_input((1, 2, 40, 16))
    s = g.add_node("matmul", [q, kt], (1, 2, 40, 40))
    p = g.add_node("softmax", [s], (1, 2, 40, 40), fattr=0.25, iattr=causal)
    o = g.add_node("matmul", [p, v], (1, 2, 40, 16))
    g.outputs = [o]
    if s_is_output:
        g.outputs.append(s)
    if extra_reader:
        g.outputs.append(g.add_node("gelu", [s], (1, 2, 40, 40)))
    return g


def names(og, tmp_path):
    from paper_2411_09242_amd import fluid as F
    F.load(host_only=True)
    g = F.Graph.from_desc(og.export())
    t = F.CostTable.load(write_table(synthetic_table(og, seed=1, mode="identity", n_variants=1), tmp_path / "t.json"), g)
    lp = F.LayoutPlan(g, t)
    return [lp.kernel(n) for n in range(g.n_nodes)]


@pytest.mark.parametrize("case,qk,pv", [
    (dict(), "_causal1", "_causal2"),
    (dict(causal=0), None, None),
    (dict(s_is_output=True), None, "_causal2"),
    (dict(extra_reader=True), None, "_causal2"),
])
def test_causal_marks(case, qk, pv, tmp_path):
    k = names(attention(**case), tmp_path)
    assert k[0].startswith("gemm_") and k[2].startswith("gemm_")
    for name, want in ((k[0], qk), (k[2], pv)):
        if want is None:
            assert "_causal" not in name, name
        else:
            assert name.endswith(want), name
