"""Pins for the oracle executors.

* Layout invariance: every layout assignment of two tiny graphs, executed
  permuted inside a NaN-poisoned arena placed by Greedy-by-Size, returns
  exactly the canonical row-major result.
* Closed forms: with all projection weights zero, the post-LN layer reduces
  to LN(LN(x)), the pre-LN stack to the final LN of x and the Llama stack to
  the final RMSNorm of x (checked against torch's own norms in float64).
"""
import itertools

import numpy as np
import pytest
import torch

import synth_inputs
from oracle import execute, graph, layouts, numerics, plan_arena
from tinygraphs import t1_graph, t2_graph


def _inputs(g, seed):
    rng = np.random.default_rng(seed)
    xs = [rng.standard_normal(s).astype(np.float32) for s in g.input_shapes]
    cs = []
    for role, shape, _ in g.consts:
        if role == "gamma":
            cs.append((1 + 0.1 * rng.standard_normal(shape)).astype(np.float32))
        else:
            cs.append((0.3 * rng.standard_normal(shape)).astype(np.float32))
    return xs, cs


def _all_assignments(g):
    L = layouts.edge_layouts(g)
    free = [e for e in range(g.n_edges) if len(L[e]) > 1]
    for combo in itertools.product(*[L[e] for e in free]):
        lay = {e: L[e][0] for e in range(g.n_edges)}
        lay.update(dict(zip(free, combo)))
        yield lay


def _run_permuted(g, lay, xs, cs):
    ap = plan_arena.plan_arena(g, lay)
    assert plan_arena.check_disjoint(ap)
    return execute.run_in_arena(g, lay, ap.root, ap.offset, ap.peak, xs, cs)


@pytest.mark.parametrize("builder,expected", [(t1_graph, 2 * 6 ** 4 * 2 * 2), (t2_graph, 6 ** 5)])
def test_every_layout_assignment_gives_identical_outputs(builder, expected):
    g = builder()
    xs, cs = _inputs(g, 11)
    ref = execute.run_canonical(g, xs, cs)
    n = 0
    for lay in _all_assignments(g):
        out = _run_permuted(g, lay, xs, cs)
        for a, b in zip(out, ref):
            assert np.array_equal(a, b), lay
        n += 1
    assert n == expected


def test_random_assignments_on_one_encoder_layer():
    cfg = synth_inputs.config(1)
    g = graph.build_transformer(cfg)
    x, cs = synth_inputs.make_inputs(cfg, g.const_specs(), 1)
    ref = execute.run_canonical(g, [x], cs)
    L = layouts.edge_layouts(g)
    rng = np.random.default_rng(7)
    for _ in range(300):
        lay = {e: L[e][int(rng.integers(0, len(L[e])))] for e in range(g.n_edges)}
        out = _run_permuted(g, lay, [x], cs)
        assert np.array_equal(out[0], ref[0])


def test_poisoned_arena_detects_a_bad_plan():
    """A plan that lets two live buffers share bytes must change the output
    (the NaN poison or the overwrite shows up) -- the check has teeth."""
    cfg = synth_inputs.config(1)
    g = graph.build_transformer(cfg)
    x, cs = synth_inputs.make_inputs(cfg, g.const_specs(), 1)
    ref = execute.run_canonical(g, [x], cs)
    lay = {e: tuple(range(len(g.edge_shape(e)))) for e in range(g.n_edges)}
    ap = plan_arena.plan_arena(g, lay)
    bad = dict(ap.offset)
    for b in ap.buffers:
        bad[b] = 0                      # everything at offset 0
    out = execute.run_in_arena(g, lay, ap.root, bad, ap.peak, [x], cs)
    assert not np.array_equal(out[0], ref[0])


def _ln(t, eps=1e-5):
    return torch.nn.functional.layer_norm(t, (t.shape[-1],), eps=eps)


def _rms(t, eps=1e-5):
    return torch.nn.functional.rms_norm(t, (t.shape[-1],), eps=eps)


def _zero_weight_consts(g, cs):
    return [np.zeros_like(a) if role == "weight" else a
            for a, (role, _, _) in zip(cs, g.consts)]


def _r32(t):
    return t.to(torch.float32).to(torch.float64)


@pytest.mark.parametrize("arch,layers", [("post_ln", 1), ("post_ln", 2), ("pre_ln", 2), ("llama", 2)])
def test_zero_weight_closed_forms(arch, layers):
    cfg = dict(synth_inputs.config(1), arch=arch, layers=layers, dtype="f32")
    g = graph.build_transformer(cfg)
    x, cs = synth_inputs.make_inputs(cfg, g.const_specs(), 3)
    (y,) = execute.run_canonical(g, [x], _zero_weight_consts(g, cs))
    t = torch.from_numpy(x.astype(np.float64))
    if arch == "post_ln":
        ref = t
        for _ in range(layers):
            ref = _r32(_ln(_r32(_ln(ref))))
    elif arch == "pre_ln":
        ref = _r32(_ln(t))
    else:
        ref = _r32(_rms(t))
    assert np.allclose(y, ref.numpy(), rtol=3e-7, atol=1e-7)


def test_bf16_edges_hold_bf16_values():
    cfg = dict(synth_inputs.config(1), arch="llama", layers=1, dtype="bf16")
    g = graph.build_transformer(cfg)
    x, cs = synth_inputs.make_inputs(cfg, g.const_specs(), 5)
    _, vals = execute.run_canonical(g, [x], cs, keep=True)
    for e, v in vals.items():
        f = v.astype(np.float32)
        assert np.array_equal(numerics.bf16_bits_to_f32(numerics.f32_to_bf16_bits(f)), f)


def test_float32_arithmetic_pipeline():
    """The float32-arithmetic option (used only to measure how far two valid
    bfloat16 executions drift apart) computes every operator in float32 --
    no operand or constant upcasts it -- and rounds at the same edges: on a
    small bf16 Llama stack every edge lands within one bfloat16 ulp of the
    definition (relative to the edge's largest value) and most edges differ
    from it somewhere."""
    cfg = synth_inputs.config(1, arch="llama", layers=2, seq=64, hidden=256, heads=4, ffn=512, dtype="bf16")
    g = graph.build_transformer(cfg)
    x, consts = synth_inputs.make_inputs(cfg, g.const_specs(), 4)
    _, vals = execute.run_canonical(g, [x], consts, keep=True)
    cv = [numerics.round_to(np.asarray(a, np.float64).reshape(s), dt) for (_, s, dt), a in zip(g.consts, consts)]
    for nd in g.nodes:
        args = [(vals[v] if v >= 0 else cv[~v]).astype(np.float32) for v in nd.ins]
        assert execute.eval_node(nd, args, np.float32).dtype == np.float32, nd.op
    (y64,), v64 = execute.run_canonical(g, [x], consts, keep=True)
    (y32,), v32 = execute.run_canonical(g, [x], consts, keep=True, arith=np.float32)
    assert np.array_equal(numerics.round_bf16(y32), y32)
    assert sum(not np.array_equal(v32[e], v64[e]) for e in v64) > len(v64) // 2
    for e in v64:
        assert np.abs(v32[e] - v64[e]).max() <= 2.0 ** -8 * max(np.abs(v64[e]).max(), 1e-3), e
