"""Operator graph IR and transformer graph builders (oracle side).

The paper's compiler turns the model into a built-in graph whose nodes are
operators and whose edges are tensors, then linearises it into one operator
sequence (Section 4, "Compiler").  Here the builder's insertion order is that
sequence and must be topological.

Edge numbering: graph inputs are edges 0..n_inputs-1, the output of node n is
edge n_inputs + n (every operator has one output).  Constants (weights,
biases, norm scales, rotary tables) are not edges: they have no layout choice
and never live in the arena.  A node input is an int: >= 0 an edge id,
< 0 the constant ``~v``.
"""
from __future__ import annotations

import json
from dataclasses import dataclass, field

import numpy as np

OPS = ("matmul", "add", "mul", "transpose", "reshape", "softmax",
       "layernorm", "rmsnorm", "gelu", "silu", "rope",
       "pad", "conv", "relu", "maxpool")


@dataclass
class Node:
    op: str
    ins: list
    out_shape: tuple
    perm: tuple = ()
    fattr: float = 0.0     # Softmax scale / norm eps (a float32 value)
    iattr: int = 0         # Softmax causal flag; Pad width; MaxPool window


@dataclass
class Graph:
    dtype: str                               # "f32" or "bf16"
    input_shapes: list = field(default_factory=list)
    consts: list = field(default_factory=list)   # (role, shape, dtype)
    nodes: list = field(default_factory=list)
    outputs: list = field(default_factory=list)

    @property
    def n_inputs(self):
        return len(self.input_shapes)

    @property
    def n_edges(self):
        return self.n_inputs + len(self.nodes)

    def out_edge(self, n):
        return self.n_inputs + n

    def producer(self, e):
        """Node id producing edge e, or None for a graph input."""
        return None if e < self.n_inputs else e - self.n_inputs

    def edge_shape(self, e):
        if e < self.n_inputs:
            return tuple(self.input_shapes[e])
        return tuple(self.nodes[e - self.n_inputs].out_shape)

    def act_inputs(self, n):
        """Activation input edges of node n, in slot order (constants skipped)."""
        return [v for v in self.nodes[n].ins if v >= 0]

    def consumers(self, e):
        return [n for n, nd in enumerate(self.nodes) if e in nd.ins]

    # --- builder helpers --------------------------------------------------
    def add_input(self, shape):
        self.input_shapes.append(tuple(shape))
        return len(self.input_shapes) - 1

    def add_const(self, role, shape, dtype=None):
        self.consts.append((role, tuple(shape), dtype or self.dtype))
        return ~(len(self.consts) - 1)

    def add_node(self, op, ins, out_shape, perm=(), fattr=0.0, iattr=0):
        assert op in OPS, op
        for v in ins:
            if v >= 0:
                assert v < self.n_edges, "inputs must already exist (topological)"
        self.nodes.append(Node(op, list(ins), tuple(int(s) for s in out_shape),
                               tuple(perm), float(np.float32(fattr)), int(iattr)))
        return self.out_edge(len(self.nodes) - 1)

    def const_specs(self):
        return [(role, shape) for role, shape, _ in self.consts]

    def export(self):
        """Canonical JSON-able description (compared with the C++ builder's)."""
        return {
            "dtype": self.dtype,
            "inputs": [list(s) for s in self.input_shapes],
            "consts": [{"role": r, "shape": list(s), "dtype": d}
                       for r, s, d in self.consts],
            "nodes": [{"op": nd.op, "ins": list(nd.ins),
                       "out_shape": list(nd.out_shape), "perm": list(nd.perm),
                       "fattr": nd.fattr, "iattr": nd.iattr}
                      for nd in self.nodes],
            "outputs": list(self.outputs),
        }

    def export_json(self):
        return json.dumps(self.export(), sort_keys=True)


def _attention_block(g, h, B, S, H, NH, causal, biases, rope, cos_c, sin_c):
    """q/k/v projections, scores, softmax, context, head merge.

    Node order per projection p in (q, k, v): MatMul -> [Add bias] -> Reshape
    [B,S,NH,D] -> [RoPE, q and k only] -> Transpose ([0,2,1,3] for q and v,
    [0,2,3,1] for k so that the key operand is already [B,NH,D,S]).
    """
    D = H // NH
    heads = {}
    for p in ("q", "k", "v"):
        w = g.add_const("weight", (H, H))
        e = g.add_node("matmul", [h, w], (B, S, H))
        if biases:
            b = g.add_const("bias", (H,))
            e = g.add_node("add", [e, b], (B, S, H))
        e = g.add_node("reshape", [e], (B, S, NH, D))
        if rope and p != "v":
            e = g.add_node("rope", [e, cos_c, sin_c], (B, S, NH, D))
        if p == "k":
            e = g.add_node("transpose", [e], (B, NH, D, S), perm=(0, 2, 3, 1))
        else:
            e = g.add_node("transpose", [e], (B, NH, S, D), perm=(0, 2, 1, 3))
        heads[p] = e
    scale = np.float32(1.0 / np.sqrt(np.float64(D)))
    s = g.add_node("matmul", [heads["q"], heads["k"]], (B, NH, S, S))
    pr = g.add_node("softmax", [s], (B, NH, S, S), fattr=scale, iattr=causal)
    c = g.add_node("matmul", [pr, heads["v"]], (B, NH, S, D))
    c1 = g.add_node("transpose", [c], (B, S, NH, D), perm=(0, 2, 1, 3))
    c2 = g.add_node("reshape", [c1], (B, S, H))
    return c2


def build_vgg(cfg: dict) -> Graph:
    """VGG-shaped convolutional network (the paper's VGG and ConvBERT models
    in Section 5 carry Conv and Pad operators).  Per stage (width, n): n
    times zero Pad of 1 on H and W, 3x3 Conv with bias (no padding of its
    own, stride 1), ReLU; then a 2x2 MaxPool.  Then the feature map
    [B, C, h, w] is flattened by two Reshapes (merge h, w; merge C, h*w)
    and classified: MatMul, bias Add, ReLU twice (width fc), MatMul and bias
    Add to `classes`, Softmax (scale 1)."""
    B, C, S = cfg["batch"], cfg["channels"], cfg["image"]
    g = Graph(dtype=cfg["dtype"])
    e = g.add_input((B, C, S, S))
    for width, n in cfg["stages"]:
        for _ in range(n):
            p = g.add_node("pad", [e], (B, C, S + 2, S + 2), iattr=1)
            w = g.add_const("weight", (width, C, 3, 3)); b = g.add_const("bias", (width,))
            c = g.add_node("conv", [p, w, b], (B, width, S, S))
            e = g.add_node("relu", [c], (B, width, S, S))
            C = width
        e = g.add_node("maxpool", [e], (B, C, S // 2, S // 2), iattr=2)
        S //= 2
    e = g.add_node("reshape", [e], (B, C, S * S))
    e = g.add_node("reshape", [e], (B, C * S * S))
    K = C * S * S
    for i, N in enumerate((cfg["fc"], cfg["fc"], cfg["classes"])):
        w = g.add_const("weight", (K, N)); b = g.add_const("bias", (N,))
        e = g.add_node("matmul", [e, w], (B, N))
        e = g.add_node("add", [e, b], (B, N))
        if i < 2:
            e = g.add_node("relu", [e], (B, N))
        K = N
    e = g.add_node("softmax", [e], (B, cfg["classes"]), fattr=1.0, iattr=0)
    g.outputs = [e]
    return g


def build_transformer(cfg: dict) -> Graph:
    """Build one of the three layer stacks (post-LN encoder, pre-LN decoder,
    Llama-style decoder) as an explicit operator graph (or, for
    arch "vgg", the convolutional network of build_vgg).

    The chain operand always comes first in a binary node (e.g. the residual
    add is Add(o1, x)), which fixes the chain slot used by the planner.
    """
    arch = cfg["arch"]
    if arch == "vgg":
        return build_vgg(cfg)
    B, S, H, NH, F = (cfg["batch"], cfg["seq"], cfg["hidden"], cfg["heads"],
                      cfg["ffn"])
    L = cfg["layers"]
    eps = np.float32(cfg.get("eps", 1e-5))
    g = Graph(dtype=cfg["dtype"])
    x = g.add_input((B, S, H))
    cos_c = sin_c = None
    if arch == "llama":
        D = H // NH
        cos_c = g.add_const("rope_cos", (S, D // 2), "f32")
        sin_c = g.add_const("rope_sin", (S, D // 2), "f32")
    for _ in range(L):
        if arch == "post_ln":
            c2 = _attention_block(g, x, B, S, H, NH, 0, True, False, None, None)
            w = g.add_const("weight", (H, H)); b = g.add_const("bias", (H,))
            o0 = g.add_node("matmul", [c2, w], (B, S, H))
            o1 = g.add_node("add", [o0, b], (B, S, H))
            r1 = g.add_node("add", [o1, x], (B, S, H))
            gm = g.add_const("gamma", (H,)); bt = g.add_const("beta", (H,))
            h1 = g.add_node("layernorm", [r1, gm, bt], (B, S, H), fattr=eps)
            w1 = g.add_const("weight", (H, F)); b1 = g.add_const("bias", (F,))
            f0 = g.add_node("matmul", [h1, w1], (B, S, F))
            f1 = g.add_node("add", [f0, b1], (B, S, F))
            f2 = g.add_node("gelu", [f1], (B, S, F))
            w2 = g.add_const("weight", (F, H)); b2 = g.add_const("bias", (H,))
            f3 = g.add_node("matmul", [f2, w2], (B, S, H))
            f4 = g.add_node("add", [f3, b2], (B, S, H))
            r2 = g.add_node("add", [f4, h1], (B, S, H))
            gm2 = g.add_const("gamma", (H,)); bt2 = g.add_const("beta", (H,))
            x = g.add_node("layernorm", [r2, gm2, bt2], (B, S, H), fattr=eps)
        elif arch == "pre_ln":
            gm = g.add_const("gamma", (H,)); bt = g.add_const("beta", (H,))
            h0 = g.add_node("layernorm", [x, gm, bt], (B, S, H), fattr=eps)
            c2 = _attention_block(g, h0, B, S, H, NH, 1, True, False, None, None)
            w = g.add_const("weight", (H, H)); b = g.add_const("bias", (H,))
            o0 = g.add_node("matmul", [c2, w], (B, S, H))
            o1 = g.add_node("add", [o0, b], (B, S, H))
            r1 = g.add_node("add", [o1, x], (B, S, H))
            gm2 = g.add_const("gamma", (H,)); bt2 = g.add_const("beta", (H,))
            h1 = g.add_node("layernorm", [r1, gm2, bt2], (B, S, H), fattr=eps)
            w1 = g.add_const("weight", (H, F)); b1 = g.add_const("bias", (F,))
            f0 = g.add_node("matmul", [h1, w1], (B, S, F))
            f1 = g.add_node("add", [f0, b1], (B, S, F))
            f2 = g.add_node("gelu", [f1], (B, S, F))
            w2 = g.add_const("weight", (F, H)); b2 = g.add_const("bias", (H,))
            f3 = g.add_node("matmul", [f2, w2], (B, S, H))
            f4 = g.add_node("add", [f3, b2], (B, S, H))
            x = g.add_node("add", [f4, r1], (B, S, H))
        elif arch == "llama":
            gm = g.add_const("gamma", (H,))
            h0 = g.add_node("rmsnorm", [x, gm], (B, S, H), fattr=eps)
            c2 = _attention_block(g, h0, B, S, H, NH, 1, False, True, cos_c, sin_c)
            w = g.add_const("weight", (H, H))
            o0 = g.add_node("matmul", [c2, w], (B, S, H))
            r1 = g.add_node("add", [o0, x], (B, S, H))
            gm2 = g.add_const("gamma", (H,))
            h1 = g.add_node("rmsnorm", [r1, gm2], (B, S, H), fattr=eps)
            wg = g.add_const("weight", (H, F))
            wu = g.add_const("weight", (H, F))
            gg = g.add_node("matmul", [h1, wg], (B, S, F))
            sg = g.add_node("silu", [gg], (B, S, F))
            uu = g.add_node("matmul", [h1, wu], (B, S, F))
            m = g.add_node("mul", [sg, uu], (B, S, F))
            wd = g.add_const("weight", (F, H))
            d = g.add_node("matmul", [m, wd], (B, S, H))
            x = g.add_node("add", [d, r1], (B, S, H))
        else:
            raise ValueError(arch)
    if arch == "pre_ln":
        gm = g.add_const("gamma", (H,)); bt = g.add_const("beta", (H,))
        x = g.add_node("layernorm", [x, gm, bt], (B, S, H), fattr=eps)
    elif arch == "llama":
        gm = g.add_const("gamma", (H,))
        x = g.add_node("rmsnorm", [x, gm], (B, S, H), fattr=eps)
    g.outputs = [x]
    return g
