"""fluid_run_static (the entry point that allocates nothing: its arena is a
static device array inside the library) against fluid_run on the same plans
and inputs, through the C ABI: two calls in a row, the second on a smaller
graph, each bit-identical to fluid_run (same kernels, same arena offsets);
and a plan above the static arena's size is refused before any launch."""
import numpy as np
import pytest

import synth_inputs
from gpu_util import assert_close, say
from oracle import execute, graph as OG

pytestmark = pytest.mark.gpu


def _setup(idx, **over):
    from paper_2411_09242_amd import fluid as F
    cfg = synth_inputs.config(idx, **over)
    g = F.Graph.transformer(cfg)
    x, consts = synth_inputs.make_inputs(cfg, g.const_specs(), idx)
    t = F.CostTable.measure(g, reps=2)
    lp = F.LayoutPlan(g, t)
    ap = F.ArenaPlan(g, lp, epilogue=True)
    return cfg, g, lp, ap, F.Executor(g, lp, ap, consts, [x]), x, consts


def _static_run(ex, stream):
    from paper_2411_09242_amd import fluid as F
    F.fluid_run_static(ex.graph.h, ex.lplan.h, ex.aplan.h, ex._cp, ex._ip, ex._op, stream)


def test_static_arena_run_matches_fluid_run():
    import torch
    from paper_2411_09242_amd import fluid as F
    s = torch.cuda.current_stream().cuda_stream
    for idx in (2, 1):      # the second call: a smaller graph in the same array
        cfg, g, lp, ap, ex, x, consts = _setup(idx)
        say(f"static arena: workload {idx}, peak {ap.peak} of {64 << 20} bytes")
        assert 0 < ap.peak <= 64 << 20
        ref = ex.run(s)[0].clone()
        torch.cuda.synchronize()
        ex.outputs[0].fill_(float("nan"))
        torch.cuda.synchronize()
        _static_run(ex, s)
        torch.cuda.synchronize()
        assert torch.equal(ex.outputs[0], ref), f"workload {idx}"
        og = OG.build_transformer(cfg)
        (want,) = execute.run_canonical(og, [x], consts)
        assert_close(ex.outputs[0].float().cpu().numpy(), want, cfg["dtype"], f"workload {idx} vs oracle")


def test_static_arena_refuses_a_plan_above_its_size():
    import torch
    from paper_2411_09242_amd import fluid as F
    cfg = synth_inputs.config(4, layers=1, batch=8)   # 288 MiB of live activations
    g = F.Graph.transformer(cfg)
    t = F.CostTable.measure(g, reps=1)
    lp = F.LayoutPlan(g, t)
    ap = F.ArenaPlan(g, lp)
    assert ap.peak > 64 << 20
    x = torch.zeros((cfg["batch"], cfg["seq"], cfg["hidden"]), device="cuda")
    y = torch.full_like(x, float("nan"))
    cs = [torch.zeros(c["shape"], device="cuda") for c in g.desc["consts"]]
    with pytest.raises(F.FluidError, match="static arena") as ei:
        F.fluid_run_static(g.h, lp.h, ap.h, [c.data_ptr() for c in cs], [x.data_ptr()], [y.data_ptr()],
                           torch.cuda.current_stream().cuda_stream)
    assert ei.value.status == -4
    torch.cuda.synchronize()
    assert torch.isnan(y).all()
