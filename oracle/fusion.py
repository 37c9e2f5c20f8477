"""Fusion chains (oracle side): which operators a MatMul may perform in its
own launch, so that the layout planner can price them.

The paper's compiler fuses operators and then plans layouts over the fused
graph (Section 4, "Compiler").  Here a fusion is an alternative the planner
weighs: a MatMul m and the t nodes right after it (ids m+1 .. m+t) form a
chain when, step by step,
  * the previous result has exactly one reader, the next node, and is not a
    graph output;
  * the steps come in this order, each optional: an Add of a bias constant
    [N] (N the product's last dim; first step only), one GELU or SiLU, and
    an Add or Mul of the chain value with another activation R of the
    product's shape, produced before m (last step).
A second kind of chain starts at an Add of two activations of its own
output's shape (a residual sum) read by the next node, a LayerNorm or
RMSNorm over it (with constant scale and shift), and is not a graph output:
the normalisation launch then also forms the sum (t = 1).
A MatMul chain's launch writes only the last node's output: the
intermediate results never reach memory.  A residual sum that has further
readers (a pre-norm block's next residual) is stored by the launch as well,
in the layout of the normalisation's output ("norm_store"); otherwise it
stays on chip ("norm").  t is 1..3; every prefix of a chain is a chain.
"""
from __future__ import annotations


def _readers(g, e):
    return sorted({n for n, nd in enumerate(g.nodes) if e in nd.ins})


def chain_steps(g, m):
    """The longest fusion chain starting at node m, as a list of
    (node, kind, R) with kind in {"bias", "act", "add_r", "mul_r", "norm"}
    and R the other activation of an Add / Mul step (None otherwise).  Empty
    when m heads no chain."""
    nd = g.nodes[m]
    if nd.op == "add":
        return _norm_chain(g, m)
    if nd.op != "matmul" or len(nd.ins) != 2:
        return []
    out_shape = tuple(nd.out_shape)
    cur = g.out_edge(m)
    steps = []
    act = False
    for i in range(1, 4):
        n = m + i
        if n >= len(g.nodes) or cur in g.outputs or _readers(g, cur) != [n]:
            break
        x = g.nodes[n]
        if x.op in ("add", "mul") and len(x.ins) == 2:
            slot = 0 if x.ins[0] == cur else 1
            other = x.ins[1 - slot]
            if other == cur:
                break
            if other < 0:
                role, cshape, cdt = g.consts[~other]
                if x.op != "add" or steps or cshape != (out_shape[-1],) or cdt != g.dtype:
                    break
                steps.append((n, "bias", None))
            else:
                p = g.producer(other)
                if tuple(g.edge_shape(other)) != out_shape or (p is not None and p >= m):
                    break
                steps.append((n, "add_r" if x.op == "add" else "mul_r", other))
                break
        elif x.op in ("gelu", "silu") and not act:
            act = True
            steps.append((n, "act", None))
        else:
            break
        cur = g.out_edge(n)
    return steps


def _norm_chain(g, m):
    """Add m of two activations followed by the normalisation of its sum."""
    nd = g.nodes[m]
    out_shape = tuple(nd.out_shape)
    if len(nd.ins) != 2 or min(nd.ins) < 0 or nd.ins[0] == nd.ins[1] or \
            any(tuple(g.edge_shape(e)) != out_shape for e in nd.ins):
        return []
    cur, n = g.out_edge(m), m + 1
    if n >= len(g.nodes) or cur in g.outputs or n not in _readers(g, cur):
        return []
    x = g.nodes[n]
    if x.op not in ("layernorm", "rmsnorm") or x.ins[0] != cur or cur in x.ins[1:] or min(x.ins[1:]) >= 0:
        return []
    return [(n, "norm" if _readers(g, cur) == [n] else "norm_store", None)]


def stored_edges(g, m, t):
    """Intermediate results of the chain (m, t) that its launch stores (in
    the layout of the last node's output): a residual sum with further
    readers."""
    steps = chain_steps(g, m)[:t]
    return [g.out_edge(m)] if steps and steps[0][1] == "norm_store" else []


def on_chip_edges(g, m, t):
    """Intermediate results of the chain (m, t) that never reach memory."""
    st = stored_edges(g, m, t)
    return [g.out_edge(m + i) for i in range(t) if g.out_edge(m + i) not in st]


def chain_slots(g, m, t):
    """Activation edges a fused launch of the chain (m, t) reads, in slot
    order: the MatMul's activation inputs, then R of an Add / Mul step."""
    steps = chain_steps(g, m)[:t]
    slots = g.act_inputs(m)
    if steps and steps[-1][2] is not None:
        slots = slots + [steps[-1][2]]
    return slots


def all_chains(g):
    """{(m, t): [node ids m .. m+t]} for every chain head m and length t."""
    out = {}
    for m in range(len(g.nodes)):
        steps = chain_steps(g, m)
        for t in range(1, len(steps) + 1):
            out[(m, t)] = [m] + [s[0] for s in steps[:t]]
    return out
