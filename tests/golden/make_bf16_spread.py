"""Measure how far two valid bfloat16 executions of the 8-layer Llama-style
workload drift apart, to set the deep-stack tolerance of its GPU test.

Both runs are the oracle (oracle/) on the seeded inputs (synth_inputs): the
definition (every operator in float64, then rounded to bfloat16 at every
edge) and the same graph with every operator computed in float32 before the
same roundings.  Nothing else differs, yet rounding flips compound through
the layers.  The statistics are taken on the rows that
oracle_rows_cfg5.npz samples (the rows the GPU test compares) and on the
whole output, and written to bf16_spread_cfg5.json.

With --one-layer, the same comparison on every edge of one layer at the
workload's full width (bf16_spread_cfg5_layer.json): the spread the GPU test
of that layer allows when it compares each stored edge with the oracle's
own edge (rather than with the oracle applied to the device's inputs).

Usage: python tests/golden/make_bf16_spread.py [--one-layer]
"""
import json
import os
import sys
import time

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(os.path.dirname(HERE))
sys.path.insert(0, ROOT)

import synth_inputs  # noqa: E402
from oracle import execute, graph  # noqa: E402

ATOL, RTOL = 1e-2, 2e-2     # the per-element bfloat16 bound of the single-layer tests


def stats(a, b):
    """a: the float32-arithmetic run, b: the definition."""
    d = np.abs(a - b)
    return {"rel_l2": float(np.linalg.norm(a - b) / np.linalg.norm(b)),
            "max_abs": float(d.max()),
            "frac_outside_per_element_bound": float((d > ATOL + RTOL * np.abs(b)).mean()),
            "p99_abs": float(np.quantile(d, 0.99))}


def main():
    idx = 5
    cfg = synth_inputs.config(idx)
    og = graph.build_transformer(cfg)
    x, consts = synth_inputs.make_inputs(cfg, og.const_specs(), idx)
    gold = np.load(os.path.join(HERE, f"oracle_rows_cfg{idx}.npz"), allow_pickle=False)
    rows = gold["rows"]
    t0 = time.time()
    (y64,) = execute.run_canonical(og, [x], consts)
    t1 = time.time()
    (y32,) = execute.run_canonical(og, [x], consts, arith=np.float32)
    t2 = time.time()
    # the stored rows are the definition's
    assert np.array_equal(y64[rows[:, 0], rows[:, 1], :].astype(np.float32), gold["values"])
    out = {
        "workload": cfg["name"],
        "what": "oracle with float32 arithmetic before each bfloat16 rounding vs the float64 oracle",
        "sampled_rows": stats(y32[rows[:, 0], rows[:, 1], :], y64[rows[:, 0], rows[:, 1], :]),
        "whole_output": stats(y32, y64),
        "oracle_f64_s": round(t1 - t0, 1), "oracle_f32_s": round(t2 - t1, 1),
    }
    path = os.path.join(HERE, f"bf16_spread_cfg{idx}.json")
    with open(path, "w") as f:
        json.dump(out, f, indent=1)
        f.write("\n")
    print(json.dumps(out), flush=True)


def one_layer():
    idx = 5
    cfg = synth_inputs.config(idx, layers=1)
    og = graph.build_transformer(cfg)
    x, consts = synth_inputs.make_inputs(cfg, og.const_specs(), idx)
    _, v64 = execute.run_canonical(og, [x], consts, keep=True)
    _, v32 = execute.run_canonical(og, [x], consts, keep=True, arith=np.float32)
    edges = {}
    for n, nd in enumerate(og.nodes):
        e = og.out_edge(n)
        if nd.op in ("transpose", "reshape"):
            continue
        edges[str(e)] = dict(stats(v32[e], v64[e]), node=n, op=nd.op)
    out = {"workload": cfg["name"], "layers": 1,
           "what": "per edge: oracle with float32 arithmetic before each bfloat16 rounding vs the float64 "
                   "oracle, each on its own inputs",
           "edges": edges}
    path = os.path.join(HERE, f"bf16_spread_cfg{idx}_layer.json")
    with open(path, "w") as f:
        json.dump(out, f, indent=1)
        f.write("\n")
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    if "--one-layer" in sys.argv[1:]:
        one_layer()
    else:
        main()
