"""The convolutional operators on the GPU through the C ABI (Pad, Conv as an
implicit GEMM on MFMA, ReLU, MaxPool), per operator in forced layouts and
end to end on VGG-shaped networks planned on GPU-measured tables, against
the oracle."""
import itertools

import numpy as np
import pytest

import synth_inputs
from gpu_util import assert_close, forced_table, random_inputs, run_device, say
from oracle import execute, graph as OG, layouts
from oracle.graph import Graph
from plan_check import assert_plans_match_oracle, load_json

pytestmark = pytest.mark.gpu


def _pairs(la, lc, n, seed):
    pairs = list(itertools.product(la, lc))
    if len(pairs) <= n:
        return pairs
    rng = np.random.default_rng(seed)
    return [pairs[i] for i in sorted(rng.choice(len(pairs), size=n, replace=False))]


def _check(og, want, variants, tmp_path, seed):
    xs, cs = random_inputs(og, seed)
    ref = execute.run_canonical(og, xs, cs)
    out, lp, _ = run_device(og, forced_table(og, want, variants), xs, cs, tmp_path)
    assert_close(out[0], ref[0], "f32", f"want={want} variants={variants}")
    return lp


def conv_graph(x_shape, w_shape, bias):
    g = Graph(dtype="f32")
    x = g.add_input(x_shape)
    a = g.add_node("relu", [x], x_shape)
    w = g.add_const("weight", w_shape)
    ins = [a, w] + ([g.add_const("bias", (w_shape[0],))] if bias else [])
    out = (x_shape[0], w_shape[0], x_shape[2] - w_shape[2] + 1, x_shape[3] - w_shape[3] + 1)
    c = g.add_node("conv", ins, out)
    y = g.add_node("relu", [c], out)
    g.outputs = [y]
    return g, a, c


CONV_CASES = [((1, 3, 9, 7), (5, 3, 3, 3), True), ((2, 8, 10, 12), (16, 8, 3, 3), True),
              ((1, 16, 6, 6), (70, 16, 1, 1), True), ((1, 5, 8, 9), (3, 5, 2, 4), False),
              ((1, 64, 14, 14), (130, 64, 3, 3), True)]


@pytest.mark.parametrize("case", CONV_CASES, ids=str)
@pytest.mark.parametrize("variant", [0, 1, 2, 3, 4, 5])
def test_conv_layouts(case, variant, tmp_path):
    """Input and output of the convolution in (a sample of) every layout
    pair; both reduction orders, with and without the K split over wave
    groups (64 x 64 tiles over 4 groups, 32 x 32 tiles over 8; K-tiles past
    the end in the last round); ragged pixel and channel tiles."""
    xs_, ws_, bias = case
    og, a, c = conv_graph(xs_, ws_, bias)
    for pa, pc in _pairs(layouts.layout_list(og.edge_shape(a)), layouts.layout_list(og.edge_shape(c)), 24,
                         sum(xs_)):
        say(f"conv {case} v{variant} x{pa} y{pc}")
        _check(og, {a: pa, c: pc}, {og.producer(c): variant}, tmp_path, sum(xs_) + variant)


def window_graph(op, shape, k):
    g = Graph(dtype="f32")
    x = g.add_input(shape)
    a = g.add_node("relu", [x], shape)
    N, C, H, W = shape
    out = (N, C, H + 2 * k, W + 2 * k) if op == "pad" else (N, C, H // k, W // k)
    b = g.add_node(op, [a], out, iattr=k)
    y = g.add_node("relu", [b], out)
    g.outputs = [y]
    return g, a, b


@pytest.mark.parametrize("op,shape,k", [("pad", (1, 3, 7, 5), 1), ("pad", (2, 4, 6, 6), 2),
                                        ("maxpool", (1, 5, 8, 6), 2), ("maxpool", (2, 3, 9, 12), 3)])
def test_pad_and_pool_layouts(op, shape, k, tmp_path):
    og, a, b = window_graph(op, shape, k)
    for pa, pb in _pairs(layouts.layout_list(shape), layouts.layout_list(og.edge_shape(b)), 36, sum(shape)):
        say(f"{op} {shape} k{k} x{pa} y{pb}")
        _check(og, {a: pa, b: pb}, {}, tmp_path, sum(shape) + k)


def _vgg_run(cfg, seed, tmp_path):
    import torch
    from paper_2411_09242_amd import fluid as F
    og = OG.build_transformer(cfg)
    x, consts = synth_inputs.make_inputs(cfg, og.const_specs(), seed)
    (ref,) = execute.run_canonical(og, [x], consts)
    g = F.Graph.transformer(cfg)
    t = F.CostTable.measure(g, reps=2)
    lp = F.LayoutPlan(g, t)
    t.save(str(tmp_path / "measured.json"))
    summary = assert_plans_match_oracle(og, g, load_json(tmp_path / "measured.json"), lp)
    outs = []
    for epi in (False, True):
        ap = F.ArenaPlan(g, lp, epilogue=epi)
        assert ap.lower_bound <= ap.peak < ap.naive
        ex = F.Executor(g, lp, ap, consts, [x])
        ex.arena.fill_(0xFF)
        ex.outputs[0].fill_(float("nan"))
        y = ex.run()[0]
        torch.cuda.synchronize()
        outs.append(y.float().cpu().numpy().astype(np.float64))
        assert_close(outs[-1], ref, "f32", f"{cfg['name']} fusion lifetimes={epi}")
    kinds = sorted({lp.kernel(n).split("_t")[0] for n in range(g.n_nodes) if lp.kernel(n).startswith("conv")})
    say(f"{cfg['name']}: plan {lp.total_ns} ns, arena {ap.peak / 2**20:.2f} MiB (naive {ap.naive / 2**20:.1f}), "
        f"conv kernels {kinds}; {summary}")
    return outs


def test_small_vgg_planned_matches_oracle(tmp_path):
    cfg = dict(synth_inputs.config(6), name="vgg-ragged", batch=2, channels=5, image=12, stages=((7, 1), (9, 2)),
               fc=13, classes=11)
    _vgg_run(cfg, 3, tmp_path)


def test_vgg16_planned_matches_oracle(tmp_path):
    """The full VGG-16-shaped network (224 x 224, 13 convolutions, 138 M
    parameters), planned on its measured table: every output element within
    the fp32 tolerance of the oracle."""
    _vgg_run(synth_inputs.config(6), 6, tmp_path)
