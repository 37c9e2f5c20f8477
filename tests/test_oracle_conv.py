"""Pins for the oracle's convolutional operators and the VGG-shaped graph
(the paper's VGG and ConvBERT models carry Conv and Pad, Section 5)."""
import itertools

import numpy as np
import pytest

import synth_inputs
from oracle import execute, graph, layouts, plan_arena
from oracle.graph import Node


def _conv_loops(x, w, b):
    N, C, H, W = x.shape
    Co, Ci, KH, KW = w.shape
    y = np.zeros((N, Co, H - KH + 1, W - KW + 1))
    for n, o, i, j in itertools.product(range(N), range(Co), range(H - KH + 1), range(W - KW + 1)):
        s = 0.0
        for c, u, v in itertools.product(range(C), range(KH), range(KW)):
            s += x[n, c, i + u, j + v] * w[o, c, u, v]
        y[n, o, i, j] = s + (b[o] if b is not None else 0.0)
    return y


@pytest.mark.parametrize("shape,kernel,bias", [((1, 3, 7, 6), (4, 3, 3, 3), True), ((2, 2, 5, 9), (3, 2, 2, 4), False),
                                               ((1, 1, 4, 4), (1, 1, 4, 4), True)])
def test_conv_equals_the_summation(shape, kernel, bias):
    rng = np.random.default_rng(sum(shape) + sum(kernel))
    x = rng.standard_normal(shape)
    w = rng.standard_normal(kernel)
    b = rng.standard_normal(kernel[0]) if bias else None
    got = execute.op_conv(x, w, b)
    want = _conv_loops(x, w, b)
    assert got.shape == want.shape
    assert np.allclose(got, want, rtol=1e-12, atol=1e-12)


def test_conv_special_cases():
    rng = np.random.default_rng(3)
    x = rng.standard_normal((1, 4, 6, 6))
    # a 1x1 kernel is a matrix product over channels at every pixel
    w = rng.standard_normal((5, 4, 1, 1))
    assert np.allclose(execute.op_conv(x, w), np.einsum("nchw,oc->nohw", x, w[:, :, 0, 0]), atol=1e-12)
    # a kernel with one 1 picks a shifted input channel
    w = np.zeros((1, 4, 3, 3))
    w[0, 2, 1, 0] = 1.0
    assert np.array_equal(execute.op_conv(x, w), x[:, 2:3, 1:5, 0:4])


def test_pad_and_maxpool_definitions():
    rng = np.random.default_rng(4)
    x = rng.standard_normal((2, 3, 4, 6))
    p = execute.op_pad(x, 2)
    assert p.shape == (2, 3, 8, 10)
    assert np.array_equal(p[:, :, 2:6, 2:8], x)
    mask = np.ones(p.shape, bool)
    mask[:, :, 2:6, 2:8] = False
    assert not p[mask].any()
    m = execute.op_maxpool(x, 2)
    assert m.shape == (2, 3, 2, 3)
    for n, c, i, j in itertools.product(range(2), range(3), range(2), range(3)):
        assert m[n, c, i, j] == max(x[n, c, 2 * i + u, 2 * j + v] for u in range(2) for v in range(2))
    r = execute.op_relu(np.array([-1.0, 0.0, 2.5]))
    assert list(r) == [0.0, 0.0, 2.5]


def small_vgg(**kw):
    c = dict(name="vgg-small", arch="vgg", batch=1, channels=3, image=8, stages=((4, 1), (6, 2)), fc=10, classes=5,
             dtype="f32")
    c.update(kw)
    return c


def test_vgg_graph_shape():
    g = graph.build_transformer(synth_inputs.config(6))
    ops = [nd.op for nd in g.nodes]
    assert ops.count("conv") == 13 and ops.count("pad") == 13 and ops.count("maxpool") == 5
    assert ops.count("matmul") == 3 and ops[-1] == "softmax"
    assert g.edge_shape(g.outputs[0]) == (1, 1000)
    flat = [e for e in range(g.n_edges) if g.edge_shape(e) == (1, 512 * 7 * 7)]
    assert len(flat) == 1


def test_vgg_zero_weights_closed_form():
    """All weights and biases zero: every convolution and product gives 0,
    so the logits are 0 and the Softmax is uniform over the classes."""
    cfg = small_vgg()
    g = graph.build_transformer(cfg)
    x, consts = synth_inputs.make_inputs(cfg, g.const_specs(), 1)
    (y,) = execute.run_canonical(g, [x], [np.zeros_like(c) for c in consts])
    assert np.array_equal(y, np.full((1, 5), np.float32(0.2)))


def test_vgg_layout_invariance():
    """Random layout assignments of a small conv net (batch 2 so that every
    permutation of [N, C, H, W] is distinct), run permuted in a poisoned
    arena placed by Greedy-by-Size: identical to the row-major result."""
    cfg = small_vgg(batch=2)
    g = graph.build_transformer(cfg)
    x, cs = synth_inputs.make_inputs(cfg, g.const_specs(), 2)
    ref = execute.run_canonical(g, [x], cs)
    L = layouts.edge_layouts(g)
    rng = np.random.default_rng(5)
    for _ in range(60):
        lay = {e: L[e][int(rng.integers(0, len(L[e])))] for e in range(g.n_edges)}
        ap = plan_arena.plan_arena(g, lay)
        assert plan_arena.check_disjoint(ap)
        out = execute.run_in_arena(g, lay, ap.root, ap.offset, ap.peak, [x], cs)
        assert np.array_equal(out[0], ref[0])
