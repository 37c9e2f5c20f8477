"""Tiny graphs for exhaustive oracle checks (built with the oracle's IR)."""
from __future__ import annotations

from oracle.graph import Graph


def t1_graph():
    """x[1,4,6] -> MatMul -> Reshape[1,4,2,3] -> Transpose[0,2,1,3] -> Softmax
    -> Transpose back -> Reshape[1,4,6] -> Add(., x) -> LayerNorm.  Distinct
    extents so that a dimension mix-up cannot hide."""
    g = Graph(dtype="f32")
    x = g.add_input((1, 4, 6))
    w = g.add_const("weight", (6, 6))
    m = g.add_node("matmul", [x, w], (1, 4, 6))
    r = g.add_node("reshape", [m], (1, 4, 2, 3))
    t = g.add_node("transpose", [r], (1, 2, 4, 3), perm=(0, 2, 1, 3))
    s = g.add_node("softmax", [t], (1, 2, 4, 3), fattr=0.5, iattr=0)
    t2 = g.add_node("transpose", [s], (1, 4, 2, 3), perm=(0, 2, 1, 3))
    r2 = g.add_node("reshape", [t2], (1, 4, 6))
    a = g.add_node("add", [r2, x], (1, 4, 6))
    gm = g.add_const("gamma", (6,)); bt = g.add_const("beta", (6,))
    y = g.add_node("layernorm", [a, gm, bt], (1, 4, 6), fattr=1e-5)
    g.outputs = [y]
    return g


def t2_graph():
    """Batched attention MatMuls: r = Reshape(x[1,4,6] -> [1,4,2,3]);
    q = Transpose(r,[0,2,1,3]); kT = Transpose(r,[0,2,3,1]); s = MatMul(q,kT);
    o = MatMul(Softmax(s), q) is the (row-major) graph output."""
    g = Graph(dtype="f32")
    x = g.add_input((1, 4, 6))
    r = g.add_node("reshape", [x], (1, 4, 2, 3))
    q = g.add_node("transpose", [r], (1, 2, 4, 3), perm=(0, 2, 1, 3))
    kt = g.add_node("transpose", [r], (1, 2, 3, 4), perm=(0, 2, 3, 1))
    s = g.add_node("matmul", [q, kt], (1, 2, 4, 4))
    p = g.add_node("softmax", [s], (1, 2, 4, 4), fattr=0.5, iattr=1)
    o = g.add_node("matmul", [p, q], (1, 2, 4, 3))
    g.outputs = [o]
    return g


def chain_graph(n_ops=5, shape=(3, 4, 5)):
    """A pure chain of unary ops on a rank-3 tensor (one path, no sharing)."""
    g = Graph(dtype="f32")
    e = g.add_input(shape)
    ops = ["gelu", "silu", "gelu", "silu", "gelu", "silu", "gelu", "silu"]
    for i in range(n_ops):
        e = g.add_node(ops[i], [e], shape)
    g.outputs = [e]
    return g


def diamond_graph(shape=(2, 3, 4)):
    """x -> a -> {b, c} -> d = Add(b, c) -> y: a shared edge with two readers."""
    g = Graph(dtype="f32")
    x = g.add_input(shape)
    a = g.add_node("gelu", [x], shape)
    b = g.add_node("silu", [a], shape)
    c = g.add_node("gelu", [a], shape)
    b2 = g.add_node("silu", [b], shape)
    d = g.add_node("add", [b2, c], shape)
    y = g.add_node("gelu", [d], shape)
    g.outputs = [y]
    return g


def mlp_graph(layers=3, B=2, S=5, H=8, F=12):
    """Row-major MLP chain (MatMul, Add, GELU per layer): few buffers."""
    g = Graph(dtype="f32")
    e = g.add_input((B, S, H))
    for i in range(layers):
        K, N = (H, F) if i % 2 == 0 else (F, H)
        w = g.add_const("weight", (K, N)); b = g.add_const("bias", (N,))
        e = g.add_node("matmul", [e, w], (B, S, N))
        e = g.add_node("add", [e, b], (B, S, N))
        e = g.add_node("gelu", [e], (B, S, N))
    g.outputs = [e]
    return g


def ffn_block(B=1, S=4, H=8, F=16):
    """One residual FFN block + LayerNorm (a skip edge)."""
    g = Graph(dtype="f32")
    x = g.add_input((B, S, H))
    w1 = g.add_const("weight", (H, F)); b1 = g.add_const("bias", (F,))
    f0 = g.add_node("matmul", [x, w1], (B, S, F))
    f1 = g.add_node("add", [f0, b1], (B, S, F))
    f2 = g.add_node("gelu", [f1], (B, S, F))
    w2 = g.add_const("weight", (F, H)); b2 = g.add_const("bias", (H,))
    f3 = g.add_node("matmul", [f2, w2], (B, S, H))
    f4 = g.add_node("add", [f3, b2], (B, S, H))
    r = g.add_node("add", [f4, x], (B, S, H))
    gm = g.add_const("gamma", (H,)); bt = g.add_const("beta", (H,))
    y = g.add_node("layernorm", [r, gm, bt], (B, S, H), fattr=1e-5)
    g.outputs = [y]
    return g


def fanout_graph():
    """x -> a=gelu(x) -> b=silu(a) -> b2=silu(b); c=gelu(a); d=gelu(a);
    s=add(b2, c); y=add(s, d).  Paths: [a b b2 s y], [c], [d]; edge a is
    produced on the first path and read in boundary slots by the other two,
    so three ballots decide it."""
    g = Graph(dtype="f32")
    x = g.add_input((2, 3))
    a = g.add_node("gelu", [x], (2, 3))
    b = g.add_node("silu", [a], (2, 3))
    b2 = g.add_node("silu", [b], (2, 3))
    c = g.add_node("gelu", [a], (2, 3))
    d = g.add_node("gelu", [a], (2, 3))
    s = g.add_node("add", [b2, c], (2, 3))
    y = g.add_node("add", [s, d], (2, 3))
    g.outputs = [y]
    return g


def prenorm_graph(B=2, S=3, H=4):
    """A residual sum read by its LayerNorm and again by a later Add (the
    pre-norm pattern): x -> a = GELU(x), b = SiLU(x); s = a + b;
    n = LN(s); y = GELU(n) + s."""
    g = Graph(dtype="f32")
    x = g.add_input((B, S, H))
    a = g.add_node("gelu", [x], (B, S, H))
    b = g.add_node("silu", [x], (B, S, H))
    s = g.add_node("add", [a, b], (B, S, H))
    gm = g.add_const("gamma", (H,)); bt = g.add_const("beta", (H,))
    n = g.add_node("layernorm", [s, gm, bt], (B, S, H), fattr=1e-5)
    y1 = g.add_node("gelu", [n], (B, S, H))
    y = g.add_node("add", [y1, s], (B, S, H))
    g.outputs = [y]
    return g
