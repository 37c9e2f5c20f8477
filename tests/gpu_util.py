"""Helpers for GPU parity tests: forced-layout cost tables, device runs
through the C ABI, and the tolerance check against the oracle."""
from __future__ import annotations

import itertools
import json
import sys

import numpy as np

from oracle import costtable, layouts, plan_layout as PL

# Tolerances of the workloads: fp32 |g - o| <= 1e-5 + 1e-4 |o|;
# bf16 rtol 2e-2 with atol 1e-2.
TOL = {"f32": (1e-4, 1e-5), "bf16": (2e-2, 1e-2)}


def say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


def assert_close(got, ref, dtype, what=""):
    got = np.asarray(got, dtype=np.float64)
    ref = np.asarray(ref, dtype=np.float64)
    assert got.shape == ref.shape, (what, got.shape, ref.shape)
    rtol, atol = TOL[dtype]
    err = np.abs(got - ref)
    # written as "not within" so that a NaN (or an infinity where the
    # reference is finite) counts as out of tolerance
    bad = ~(err <= atol + rtol * np.abs(ref))
    if bad.any():
        i = np.unravel_index(np.argmax(np.where(bad, np.nan_to_num(err, nan=np.inf), -1.0)), ref.shape)
        raise AssertionError(f"{what}: {int(bad.sum())} of {ref.size} elements out of tolerance; "
                             f"worst at {i}: got {got[i]!r} want {ref[i]!r}; "
                             f"max abs err {err.max():.3g}")
    return float(err.max())


def forced_table(og, want, variants=None):
    """A cost table under which the only cheap plan gives every edge in
    ``want`` (edge -> perm) that layout, and every node in ``variants`` that
    kernel variant.  Unlisted edges stay row-major.  The all-row-major
    combination of every node is present (required) but expensive."""
    variants = variants or {}
    L = layouts.edge_layouts(og)
    lay = {e: tuple(want.get(e, tuple(range(len(og.edge_shape(e)))))) for e in range(og.n_edges)}
    for e, p in lay.items():
        if e < og.n_inputs or e in og.outputs:
            assert p == tuple(range(len(p))), "graph inputs/outputs are row-major"
        else:
            assert p in L[e], (e, p, "not a candidate (use the first of equivalent layouts)")
    sigs, node_sig = [], []
    nvar = {"matmul": 20, "gelu": 2, "silu": 2, "relu": 2, "conv": 6, "transpose": 2, "reshape": 2,
            "softmax": 3, "layernorm": 3, "rmsnorm": 3}
    for n, nd in enumerate(og.nodes):
        slots = og.act_inputs(n)
        eo = og.out_edge(n)
        ins = [lay[e] for e in slots]
        out = lay[eo]
        ident = [tuple(range(len(og.edge_shape(e)))) for e in slots]
        ident_out = tuple(range(len(nd.out_shape)))
        entries = []
        nv = nvar.get(nd.op, 1)

        def costs_for(i_perms, o_perm, cheap):
            if nd.op in ("transpose", "reshape") and layouts.is_view(
                    nd.op, nd.perm, og.edge_shape(slots[0]), nd.out_shape, i_perms[0], o_perm):
                return [0]
            c = 1 if cheap else 1000
            if n in variants:
                return [c if v == variants[n] else -1 for v in range(nv)]
            return [c] * nv
        entries.append([[list(p) for p in ins], list(out), costs_for(ins, out, True)])
        if (ins, out) != (ident, ident_out):
            entries.append([[list(p) for p in ident], list(ident_out), costs_for(ident, ident_out, False)])
        sigs.append({"op": nd.op, "in_shapes": [list(og.edge_shape(e)) for e in slots],
                     "out_shape": list(nd.out_shape), "entries": entries})
        node_sig.append(n)
    obj = {"format": "fluid-cost-table/1", "edges": [[list(p) for p in l] for l in L],
           "sigs": sigs, "node_sig": node_sig}
    # the oracle planner must pick exactly the requested plan
    ct = costtable.load(obj, og)
    plan = PL.plan_layouts(og, ct)
    for e in range(og.n_edges):
        assert ct.L[e][plan.layout_idx[e]] == lay[e], ("forced plan not taken", e)
    return obj


def random_inputs(og, seed, scale=1.0):
    """Seeded inputs for a small test graph: activations N(0, scale^2),
    weights N(0, 1/K), norm scales around 1, rotary tables from positions."""
    import synth_inputs
    rng = np.random.default_rng(seed)
    xs = [synth_inputs.random_tensor(s, seed + 17 * i, scale, og.dtype) for i, s in enumerate(og.input_shapes)]
    cs = []
    for i, (role, shape, dt) in enumerate(og.consts):
        if role == "weight":
            a = synth_inputs.random_tensor(shape, seed + 1000 + i, 1.0 / np.sqrt(shape[0]), dt)
        elif role == "gamma":
            a = (1.0 + 0.1 * rng.standard_normal(shape)).astype(np.float32)
            a = synth_inputs._to_bf16_exact(a) if dt == "bf16" else a
        elif role in ("bias", "beta"):
            a = synth_inputs.random_tensor(shape, seed + 2000 + i, 0.1, dt)
        elif role == "rope_cos":
            a = synth_inputs.rope_tables(shape[0], 2 * shape[1])[0]
        elif role == "rope_sin":
            a = synth_inputs.rope_tables(shape[0], 2 * shape[1])[1]
        else:
            a = synth_inputs.random_tensor(shape, seed + 3000 + i, 1.0, dt)
        cs.append(a)
    return xs, cs


def run_device(og, table_obj, xs, cs, tmp_path, flags=0, no_reuse=False, poison=True, epilogue=False):
    """Build the graph in the C library, load the table, plan, run on the GPU
    and return (outputs as float64 numpy, layout plan, arena plan)."""
    import torch
    from paper_2411_09242_amd import fluid as F
    g = F.Graph.from_desc(og.export())
    path = tmp_path / "table.json"
    with open(path, "w") as f:
        json.dump(table_obj, f)
    t = F.CostTable.load(str(path), g)
    lp = F.LayoutPlan(g, t, flags)
    ap = F.ArenaPlan(g, lp, no_reuse=no_reuse, epilogue=epilogue)
    ex = F.Executor(g, lp, ap, cs, xs)
    if poison:
        ex.arena.fill_(0xFF)     # NaN bytes: reads of unwritten bytes show up
        for o in ex.outputs:
            o.fill_(float("nan"))
    outs = ex.run()
    torch.cuda.synchronize()
    return [o.float().cpu().numpy().astype(np.float64) for o in outs], lp, ap
