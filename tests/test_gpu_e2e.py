"""End-to-end parity on the GPU: whole transformer graphs, layout plan from a
cost table measured on the GPU, Greedy-by-Size arena, run through fluid_run,
compared with the oracle's row-major execution of the same seeded inputs."""
import numpy as np
import pytest

import synth_inputs
from gpu_util import assert_close, forced_table, say
from plan_check import assert_plans_match_oracle, load_json
from oracle import execute, graph as OG, layouts

pytestmark = pytest.mark.gpu


def _device_run(cfg, x, consts, table=None, flags=0, no_reuse=False, graph=None, epilogue=False):
    import torch
    from paper_2411_09242_amd import fluid as F
    g = graph if graph is not None else F.Graph.transformer(cfg)
    t = table(g) if callable(table) else (table or F.CostTable.measure(g, reps=3))
    lp = F.LayoutPlan(g, t, flags)
    ap = F.ArenaPlan(g, lp, no_reuse=no_reuse, epilogue=epilogue)
    assert ap.lower_bound <= ap.peak <= (ap.naive if not no_reuse else ap.peak)
    ex = F.Executor(g, lp, ap, consts, [x])
    ex.arena.fill_(0xFF)
    ex.outputs[0].fill_(float("nan"))
    out = ex.run()[0]
    torch.cuda.synchronize()
    return out.float().cpu().numpy().astype(np.float64), g, lp, ap, t


@pytest.mark.parametrize("idx", [1, 2, 3])
def test_config_planned_and_naive_match_oracle(idx, tmp_path):
    cfg = synth_inputs.config(idx)
    og = OG.build_transformer(cfg)
    x, consts = synth_inputs.make_inputs(cfg, og.const_specs(), idx)
    say(f"cfg{idx}: oracle")
    (ref,) = execute.run_canonical(og, [x], consts)
    say(f"cfg{idx}: measure + plan + run")
    out, g, lp, ap, t = _device_run(cfg, x, consts)
    say(f"cfg{idx}: planned total {lp.total_ns} ns guard {lp.guard_used} peak {ap.peak} naive {ap.naive}")
    err = assert_close(out, ref, cfg["dtype"], f"cfg{idx} planned")
    say(f"cfg{idx}: planned max abs err {err:.3g}")
    # the plans on the GPU-measured table equal the oracle planners' on it
    t.save(str(tmp_path / "measured.json"))
    summary = assert_plans_match_oracle(og, g, load_json(tmp_path / "measured.json"), lp)
    say(f"cfg{idx}: plans equal the oracle's on the measured table: {summary}")
    from paper_2411_09242_amd import fluid as F
    out2, *_ = _device_run(cfg, x, consts, table=t, graph=g, flags=F.NO_DP, no_reuse=True)
    assert_close(out2, ref, cfg["dtype"], f"cfg{idx} naive")
    # the arena that lets every epilogue fuse (what the benchmark runs)
    out3, _, lp3, ap3, _ = _device_run(cfg, x, consts, table=t, graph=g, epilogue=True)
    assert F.fluid_run_launches(g.h, lp3.h, ap3.h) <= F.fluid_run_launches(g.h, lp.h, ap.h)
    assert_close(out3, ref, cfg["dtype"], f"cfg{idx} planned, fusion lifetimes")


@pytest.mark.parametrize("arch,dtype", [("post_ln", "f32"), ("pre_ln", "f32"), ("llama", "f32"), ("llama", "bf16")])
@pytest.mark.parametrize("epilogue", [False, True])
def test_ragged_small_stacks(arch, dtype, epilogue):
    cfg = synth_inputs.config(1, arch=arch, dtype=dtype, layers=2, batch=2, seq=37, hidden=72, heads=3, ffn=100)
    og = OG.build_transformer(cfg)
    x, consts = synth_inputs.make_inputs(cfg, og.const_specs(), 11)
    (ref,) = execute.run_canonical(og, [x], consts)
    out, *_ = _device_run(cfg, x, consts, epilogue=epilogue)
    assert_close(out, ref, dtype, f"{arch} {dtype}")


@pytest.mark.parametrize("idx", [1, 2])
def test_hip_graph_replay_matches_eager(idx):
    """fluid_run captured into a HIP graph: every replay, with eager work and
    synchronisation between replays (arena re-poisoned each time), gives the
    eager result bit for bit."""
    import torch
    from paper_2411_09242_amd import fluid as F
    cfg = synth_inputs.config(idx)
    g = F.Graph.transformer(cfg)
    x, consts = synth_inputs.make_inputs(cfg, g.const_specs(), idx)
    t = F.CostTable.measure(g, reps=2)
    lp = F.LayoutPlan(g, t)
    ap = F.ArenaPlan(g, lp)
    ex = F.Executor(g, lp, ap, consts, [x])
    ref = ex.run()[0].clone()
    torch.cuda.synchronize()
    graph = ex.capture(steps=2)
    for rep in range(4):
        ex.arena.fill_(0xFF)
        ex.outputs[0].fill_(float("nan"))
        torch.cuda.synchronize()
        graph.replay()
        torch.cuda.synchronize()
        assert torch.equal(ex.outputs[0], ref), f"replay {rep}"
        # eager run in between
        ex.run()
        torch.cuda.synchronize()
        assert torch.equal(ex.outputs[0], ref)


def test_random_forced_layouts_on_one_layer(tmp_path):
    """Many random layout assignments of the one-layer encoder: every kernel
    family meets many stride patterns inside the real graph."""
    import json
    from paper_2411_09242_amd import fluid as F
    cfg = synth_inputs.config(1)
    og = OG.build_transformer(cfg)
    x, consts = synth_inputs.make_inputs(cfg, og.const_specs(), 1)
    (ref,) = execute.run_canonical(og, [x], consts)
    L = layouts.edge_layouts(og)
    rng = np.random.default_rng(3)
    for trial in range(40):
        want = {e: L[e][int(rng.integers(0, len(L[e])))] for e in range(og.n_edges) if len(L[e]) > 1}
        obj = forced_table(og, want)
        path = tmp_path / f"t{trial}.json"
        path.write_text(json.dumps(obj))
        say(f"forced trial {trial}")
        out, *_ = _device_run(cfg, x, consts, table=lambda gg: F.CostTable.load(str(path), gg))
        assert_close(out, ref, "f32", f"trial {trial}")


def test_run_nodes_replays_the_run_bit_for_bit():
    """fluid_run_nodes over every non-view node, in node order, is the same
    computation as fluid_run: the output matches bit for bit; a view node or
    an empty list is rejected before any launch."""
    import torch
    from paper_2411_09242_amd import fluid as F
    cfg = synth_inputs.config(1)
    g = F.Graph.transformer(cfg)
    x, consts = synth_inputs.make_inputs(cfg, g.const_specs(), 1)
    t = F.CostTable.measure(g, reps=2)
    lp = F.LayoutPlan(g, t)
    ap = F.ArenaPlan(g, lp)
    ex = F.Executor(g, lp, ap, consts, [x])
    ref = ex.run()[0].clone()
    torch.cuda.synchronize()
    launched = [n for n in range(g.n_nodes) if lp.variant[n] != -1]
    ex.arena.fill_(0xFF)
    ex.outputs[0].fill_(float("nan"))
    ex.run_nodes(launched, repeat=2)
    torch.cuda.synchronize()
    assert torch.equal(ex.outputs[0], ref)
    views = [n for n in range(g.n_nodes) if lp.variant[n] == -1]
    if views:
        with pytest.raises(F.FluidError, match="view"):
            ex.run_nodes([views[0]])
    with pytest.raises(F.FluidError):
        ex.run_nodes([])


def test_run_rejects_bad_arguments_before_any_launch():
    """fluid_run validates everything before it enqueues: an arena below the
    plan's peak (ARENA_TOO_SMALL), a misaligned or NULL arena, a NULL or
    misaligned constant, input or output, and plans of another graph
    (INVALID) -- and the caller's output is untouched; a correct call then
    still gives the planned result."""
    import torch
    from paper_2411_09242_amd import fluid as F
    cfg = synth_inputs.config(1)
    og = OG.build_transformer(cfg)
    x, consts = synth_inputs.make_inputs(cfg, og.const_specs(), 1)
    (ref,) = execute.run_canonical(og, [x], consts)
    g = F.Graph.transformer(cfg)
    t = F.CostTable.measure(g, reps=2)
    lp = F.LayoutPlan(g, t)
    ap = F.ArenaPlan(g, lp)
    ex = F.Executor(g, lp, ap, consts, [x])
    s = torch.cuda.current_stream().cuda_stream
    ex.outputs[0].fill_(float("nan"))
    torch.cuda.synchronize()
    args = dict(arena=ex.arena_ptr, nbytes=ap.peak, consts=list(ex._cp), inputs=list(ex._ip),
                outputs=list(ex._op), lp=lp, ap=ap)

    def run(**kw):
        a = dict(args, **kw)
        F.fluid_run(g.h, a["lp"].h, a["ap"].h, a["arena"], a["nbytes"], a["consts"], a["inputs"],
                    a["outputs"], s)

    other = F.Graph.transformer(synth_inputs.config(1, seq=16))
    lp_other = F.LayoutPlan(other, F.CostTable.measure(other, reps=1))
    bad = [
        (dict(nbytes=ap.peak - 1), -4, "plan needs"),
        (dict(arena=ex.arena_ptr + 16), -1, "aligned"),
        (dict(arena=None), -1, "NULL arena"),
        (dict(consts=[None] + args["consts"][1:]), -1, "const 0"),
        (dict(consts=[args["consts"][0] + 4] + args["consts"][1:]), -1, "const 0"),
        (dict(inputs=[None]), -1, "input 0"),
        (dict(outputs=[args["outputs"][0] + 8]), -1, "output 0"),
        (dict(lp=lp_other), -1, "another graph"),
    ]
    for kw, status, msg in bad:
        with pytest.raises(F.FluidError, match=msg) as ei:
            run(**kw)
        assert ei.value.status == status, (kw, ei.value)
    torch.cuda.synchronize()
    assert torch.isnan(ex.outputs[0]).all()
    run()
    torch.cuda.synchronize()
    assert_close(ex.outputs[0].float().cpu().numpy(), ref, "f32", "after rejected calls")


PRICED = [("post_ln", "f32"), ("pre_ln", "f32"), ("llama", "f32"), ("llama", "bf16")]


@pytest.mark.parametrize("arch,dtype", PRICED)
@pytest.mark.parametrize("seed", [0, 1])
def test_priced_fusion_chains_run_to_parity(arch, dtype, seed, tmp_path):
    """Plans whose layout DP chose fusion chains (random tables that price
    every chain, for MatMul variant 1, whose tile performs every step): the
    run -- each chosen chain one launch that stores only its last output --
    matches the oracle.  fluid_run_nodes replays it bit for bit when the
    list holds each chain whole, and refuses, before any launch, a list that
    splits a chain (the chain's intermediate results have no buffer)."""
    import torch
    from paper_2411_09242_amd import fluid as F
    from tables import add_fused, synthetic_table, write_table
    cfg = synth_inputs.config(1, arch=arch, dtype=dtype, layers=2, batch=2, seq=37, hidden=72, heads=3, ffn=100)
    og = OG.build_transformer(cfg)
    x, consts = synth_inputs.make_inputs(cfg, og.const_specs(), 11 + seed)
    (ref,) = execute.run_canonical(og, [x], consts)
    tab = synthetic_table(og, seed=seed, mode="random", lo=1, hi=1000, n_variants=1)
    # fused entries mostly below the sum of the chain's separate nodes, so
    # that the DP chooses chains on every configuration here
    add_fused(tab, og, seed, n_variants=2, lo=1, hi=200)
    for fs in tab["fused_sigs"]:
        for ent in fs["entries"]:
            ent[2][0] = -1
    path = write_table(tab, tmp_path / "t.json")
    out, g, lp, ap, _ = _device_run(cfg, x, consts, table=lambda gg: F.CostTable.load(str(path), gg))
    assert lp.fusion_priced and any(lp.fuse)
    say(f"{arch} {dtype} seed {seed}: {sum(1 for t in lp.fuse if t)} priced chains")
    assert_close(out, ref, dtype, f"{arch} {dtype} priced fusion")
    ex = F.Executor(g, lp, ap, consts, [x])
    want = ex.run()[0].clone()
    torch.cuda.synchronize()
    ex.outputs[0].fill_(float("nan"))
    ex.run_nodes([n for n in range(g.n_nodes) if lp.variant[n] != -1])
    torch.cuda.synchronize()
    assert torch.equal(ex.outputs[0], want)
    m = next(i for i, t in enumerate(lp.fuse) if t)
    before = ex.outputs[0].clone()
    for bad in ([m], [m + lp.fuse[m]], list(range(m, m + lp.fuse[m]))):
        with pytest.raises(F.FluidError, match="fusion chain"):
            ex.run_nodes(bad)
    torch.cuda.synchronize()
    assert torch.equal(ex.outputs[0], before)


@pytest.mark.parametrize("arch,dtype", [("pre_ln", "f32"), ("llama", "bf16")])
@pytest.mark.parametrize("seed", [0, 1])
def test_stored_residual_sums_run_to_parity(arch, dtype, seed, tmp_path):
    """Pre-norm stacks with residual-norm chains priced well below their
    nodes (and MatMul chains, which compete for the same Adds, well above):
    the plan fuses residual sums that the next residual reads too, each
    launch storing the sum in the norm output's layout, and the run matches
    the oracle; fluid_run_nodes replays it bit for bit."""
    import torch
    from oracle import fusion
    from paper_2411_09242_amd import fluid as F
    from tables import add_fused, synthetic_table, write_table
    cfg = synth_inputs.config(1, arch=arch, dtype=dtype, layers=2, batch=2, seq=37, hidden=72, heads=3, ffn=100)
    og = OG.build_transformer(cfg)
    x, consts = synth_inputs.make_inputs(cfg, og.const_specs(), 21 + seed)
    (ref,) = execute.run_canonical(og, [x], consts)
    tab = synthetic_table(og, seed=seed, mode="random", lo=50, hi=100, n_variants=1)
    add_fused(tab, og, seed, n_variants=2, lo=1, hi=20)
    for fs in tab["fused_sigs"]:
        for ent in fs["entries"]:
            ent[2][0] = -1
            if fs["op"] == "matmul":
                ent[2] = [c * 50 if c > 0 else c for c in ent[2]]
    path = write_table(tab, tmp_path / "t.json")
    out, g, lp, ap, _ = _device_run(cfg, x, consts, table=lambda gg: F.CostTable.load(str(path), gg))
    stored = [(m, t) for m, t in enumerate(lp.fuse) if t and fusion.stored_edges(og, m, t)]
    assert stored
    for m, t in stored:
        (e,) = fusion.stored_edges(og, m, t)
        assert ap.offset[e] >= 0 and lp.perm(e) == lp.perm(og.out_edge(m + t))
    say(f"{arch} {dtype} seed {seed}: stored sums at {stored}")
    assert_close(out, ref, dtype, f"{arch} {dtype} stored residual sums")
    ex = F.Executor(g, lp, ap, consts, [x])
    want = ex.run()[0].clone()
    torch.cuda.synchronize()
    ex.outputs[0].fill_(float("nan"))
    ex.run_nodes([n for n in range(g.n_nodes) if lp.variant[n] != -1])
    torch.cuda.synchronize()
    assert torch.equal(ex.outputs[0], want)
