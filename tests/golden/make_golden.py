"""Write oracle reference samples for the two largest workloads.

Runs only the oracle (oracle/) on the seeded inputs (synth_inputs) and stores,
per workload, a fixed sample of output rows (one row = all H features of one
token) plus whole-output statistics.  The GPU parity tests compare the
device output with these rows element by element and with the statistics.

Usage: python tests/golden/make_golden.py [4] [5]
"""
import os
import sys
import time

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(os.path.dirname(HERE))
sys.path.insert(0, ROOT)

import synth_inputs  # noqa: E402
from oracle import execute, graph  # noqa: E402


def sample_rows(B, S, n, seed):
    rng = np.random.default_rng(1000 + seed)
    tok = np.sort(rng.choice(B * S, size=n, replace=False))
    tok[0] = 0                      # first token of the first sequence
    tok[-1] = B * S - 1             # last token of the last sequence
    return np.stack([tok // S, tok % S], axis=1)


def make(idx, n_rows):
    cfg = synth_inputs.config(idx)
    og = graph.build_transformer(cfg)
    t0 = time.time()
    x, consts = synth_inputs.make_inputs(cfg, og.const_specs(), idx)
    t1 = time.time()
    (y,) = execute.run_canonical(og, [x], consts)
    t2 = time.time()
    rows = sample_rows(cfg["batch"], cfg["seq"], n_rows, idx)
    vals = y[rows[:, 0], rows[:, 1], :].astype(np.float32)
    out = os.path.join(HERE, f"oracle_rows_cfg{idx}.npz")
    np.savez_compressed(out, rows=rows.astype(np.int32), values=vals,
                        mean=np.float64(y.mean()), mean_abs=np.float64(np.abs(y).mean()),
                        sumsq=np.float64((y * y).sum()), shape=np.array(y.shape, np.int64),
                        gen_s=np.float64(t1 - t0), oracle_s=np.float64(t2 - t1))
    print(f"cfg{idx}: wrote {out} ({len(rows)} rows); inputs {t1 - t0:.1f}s, oracle {t2 - t1:.1f}s",
          flush=True)


if __name__ == "__main__":
    which = [int(a) for a in sys.argv[1:]] or [4, 5]
    for i in which:
        make(i, 64 if i == 4 else 32)
