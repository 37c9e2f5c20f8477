"""Oracle executors.

``run_canonical`` is the plain definition of what the hot path computes:
the operator graph evaluated in logical index space, each operator in
float64 and its result rounded to the edge dtype (float32, or bfloat16 via
float32), in row-major storage.  Layout and arena choices transform only the
execution blueprint of a fixed graph, so the planned execution must reach
this same result.

``run_in_arena`` executes the same graph with every edge stored in its own
layout inside one byte arena at its planned offset (views aliasing their
root's bytes).  It uses the same operator functions, so for any valid layout
assignment and any valid arena plan it must return bit-identical outputs;
the arena is filled with NaN bytes first, so reading a byte before it is
written, or a buffer overwritten while still live, shows up as a mismatch.

Operator semantics follow ONNX, the paper's front-end format:
  MatMul      numpy matmul (batch broadcast; weights are 2-D [K, N])
  Add / Mul   elementwise with numpy broadcasting (bias [N])
  Transpose   Y = X.transpose(perm);  Reshape: row-major reinterpretation
  Softmax     over the last axis of scale*x; with causal, key k > query q is
              excluded and its probability is exactly 0
  LayerNorm   (x - mean) / sqrt(biased var + eps) * gamma + beta, last axis
  RMSNorm     x / sqrt(mean(x^2) + eps) * gamma, last axis
  GELU        0.5 x (1 + erf(x / sqrt 2));  SiLU: x / (1 + exp(-x))
  RoPE        rotate-half on the last axis of [B, S, NH, D] with tables
              cos/sin [S, D/2] indexed by the position (axis 1)
  Pad         zero padding of width p on both sides of H and W ([N,C,H,W])
  Conv        y[n,o,i,j] = sum_{c,u,v} x[n,c,i+u,j+v] w[o,c,u,v] + b[o]
              (ONNX Conv with no padding, stride 1, one group)
  ReLU        max(x, 0);  MaxPool: maximum over k x k windows, stride k
"""
from __future__ import annotations

import numpy as np
from scipy.special import erf

from . import fusion
from . import numerics
from .layouts import node_is_view


def op_matmul(a, b):
    return np.matmul(a, b)


def op_softmax(x, scale, causal, dt=np.float64):
    z = dt(scale) * x
    if causal:
        q, k = x.shape[-2], x.shape[-1]
        mask = np.arange(k)[None, :] > np.arange(q)[:, None]
        z = np.where(mask, -np.inf, z)
    m = z.max(axis=-1, keepdims=True)
    e = np.exp(z - m)
    return e / e.sum(axis=-1, keepdims=True)


def op_layernorm(x, gamma, beta, eps, dt=np.float64):
    mu = x.mean(axis=-1, keepdims=True)
    var = ((x - mu) ** 2).mean(axis=-1, keepdims=True)
    return (x - mu) / np.sqrt(var + dt(eps)) * gamma + beta


def op_rmsnorm(x, gamma, eps, dt=np.float64):
    ms = (x * x).mean(axis=-1, keepdims=True)
    return x / np.sqrt(ms + dt(eps)) * gamma


def op_gelu(x):
    return 0.5 * x * (1.0 + erf(x / np.sqrt(2.0)))


def op_silu(x):
    return x / (1.0 + np.exp(-x))


def op_rope(x, cos, sin):
    h = x.shape[-1] // 2
    c = cos[None, :, None, :]
    s = sin[None, :, None, :]
    x1, x2 = x[..., :h], x[..., h:]
    return np.concatenate([x1 * c - x2 * s, x2 * c + x1 * s], axis=-1)


def op_pad(x, p):
    return np.pad(x, ((0, 0), (0, 0), (p, p), (p, p)))


def op_conv(x, w, b=None):
    """The convolution sum written as one matrix product over the unfolded
    input windows (im2col): rows (n, i, j), columns (c, u, v)."""
    N, C, H, W = x.shape
    Co, Ci, KH, KW = w.shape
    OH, OW = H - KH + 1, W - KW + 1
    win = np.lib.stride_tricks.sliding_window_view(x, (KH, KW), axis=(2, 3))   # [N, C, OH, OW, KH, KW]
    cols = np.ascontiguousarray(win.transpose(0, 2, 3, 1, 4, 5)).reshape(N * OH * OW, C * KH * KW)
    y = (cols @ w.reshape(Co, Ci * KH * KW).T).reshape(N, OH, OW, Co).transpose(0, 3, 1, 2)
    if b is not None:
        y = y + b[None, :, None, None]
    return y


def op_relu(x):
    return np.maximum(x, 0)


def op_maxpool(x, k):
    N, C, H, W = x.shape
    return x.reshape(N, C, H // k, k, W // k, k).max(axis=(3, 5))


def eval_node(nd, args, dt=np.float64):
    """Result of one operator on arguments of the arithmetic type dt (float64
    unless a caller asks for float32 arithmetic), not yet rounded."""
    op = nd.op
    if op == "matmul":
        return op_matmul(args[0], args[1])
    if op == "add":
        return args[0] + args[1]
    if op == "mul":
        return args[0] * args[1]
    if op == "transpose":
        return np.transpose(args[0], nd.perm)
    if op == "reshape":
        return args[0].reshape(nd.out_shape)
    if op == "softmax":
        return op_softmax(args[0], nd.fattr, nd.iattr, dt)
    if op == "layernorm":
        return op_layernorm(args[0], args[1], args[2], nd.fattr, dt)
    if op == "rmsnorm":
        return op_rmsnorm(args[0], args[1], nd.fattr, dt)
    if op == "gelu":
        return op_gelu(args[0])
    if op == "silu":
        return op_silu(args[0])
    if op == "rope":
        return op_rope(args[0], args[1], args[2])
    if op == "pad":
        return op_pad(args[0], nd.iattr)
    if op == "conv":
        return op_conv(args[0], args[1], args[2] if len(args) > 2 else None)
    if op == "relu":
        return op_relu(args[0])
    if op == "maxpool":
        return op_maxpool(args[0], nd.iattr)
    raise ValueError(op)


def _const_values(g, consts):
    out = []
    for (role, shape, dt), a in zip(g.consts, consts):
        a = np.asarray(a, dtype=np.float64).reshape(shape)
        out.append(numerics.round_to(a, dt))
    return out


def run_canonical(g, inputs, consts, keep=False, arith=np.float64, on_chip=()):
    """Row-major reference execution.  Returns the graph outputs (float64
    arrays of dtype-representable values); with ``keep`` also every edge.
    Edges in ``on_chip`` keep their unrounded values (results that a fused
    launch never stores).

    ``arith`` is the type every operator computes in before its result is
    rounded to the edge dtype: float64 is the definition; float32 gives a
    second, equally valid pipeline for bfloat16 graphs (the rounding points
    are the same, only the arithmetic between them differs), used to measure
    how far two valid bfloat16 executions drift apart."""
    cv = _const_values(g, consts)
    vals = {}
    for e, a in enumerate(inputs):
        vals[e] = numerics.round_to(np.asarray(a, np.float64).reshape(g.input_shapes[e]), g.dtype)
    for n, nd in enumerate(g.nodes):
        args = [vals[v] if v >= 0 else cv[~v] for v in nd.ins]
        if arith is not np.float64:
            args = [a.astype(arith) for a in args]
        y = eval_node(nd, args, arith)
        assert tuple(y.shape) == tuple(nd.out_shape), (n, nd.op, y.shape, nd.out_shape)
        e = g.out_edge(n)
        vals[e] = y if e in on_chip else numerics.round_to(y, g.dtype)
    outs = [vals[e] for e in g.outputs]
    return (outs, vals) if keep else outs


def run_in_arena(g, layout_of_edge, root_of_edge, offset_of_root, peak,
                 inputs, consts, poison=True, fuse=None):
    """Execute with each edge stored permuted inside one uint8 arena.

    ``layout_of_edge[e]`` is a permutation; ``root_of_edge[e]`` the buffer
    edge e lives in; ``offset_of_root[r]`` the byte offset of arena buffer r.
    Graph inputs and outputs live in separate caller buffers (row-major).
    ``fuse[m] = t`` marks a fused chain: the results of nodes m .. m+t-1
    never reach memory (they are held outside the arena, as a fused launch
    holds them on chip).
    """
    isz = numerics.itemsize(g.dtype)
    arena = np.full(max(int(peak), 1), 0xFF if poison else 0, dtype=np.uint8)
    ext = {}
    for e, a in enumerate(inputs):
        v = numerics.round_to(np.asarray(a, np.float64).reshape(g.input_shapes[e]), g.dtype)
        ext[e] = numerics.to_bytes(v, g.dtype).copy()
    for e in g.outputs:
        ext[e] = np.full(int(np.prod(g.edge_shape(e))) * isz, 0xFF, np.uint8)

    on_chip = {}
    for m, t in enumerate(fuse or []):
        for e in fusion.on_chip_edges(g, m, t):
            on_chip[e] = None

    def buf(e):
        r = root_of_edge[e]
        if r in ext:
            return ext[r], 0
        return arena, int(offset_of_root[r])

    def load(e):
        if e in on_chip:
            return on_chip[e]
        shape = g.edge_shape(e)
        perm = tuple(layout_of_edge[e])
        cnt = int(np.prod(shape))
        b, off = buf(e)
        flat = numerics.from_bytes(b[off: off + cnt * isz], g.dtype, cnt)
        phys = flat.reshape([shape[d] for d in perm])
        return phys.transpose(np.argsort(perm))

    def store(e, val):
        if e in on_chip:
            on_chip[e] = val
            return
        perm = tuple(layout_of_edge[e])
        phys = np.ascontiguousarray(val.transpose(perm))
        raw = numerics.to_bytes(phys, g.dtype)
        b, off = buf(e)
        b[off: off + raw.size] = raw

    cv = _const_values(g, consts)
    for n, nd in enumerate(g.nodes):
        if node_is_view(g, n, layout_of_edge):
            continue
        args = [load(v) if v >= 0 else cv[~v] for v in nd.ins]
        y = numerics.round_to(eval_node(nd, args), g.dtype)
        store(g.out_edge(n), y)
    return [load(e) for e in g.outputs]
