"""Oracle for the layout-planned transformer hot path -- TEST INFRASTRUCTURE ONLY.

A plain, slow, obviously-correct CPU implementation written from the FluidML
paper (arXiv 2411.09242).  Only the tests, the smoke check and the benchmark's
CPU-baseline leg may import it; the product path never does, and this package
imports nothing from the product package.

Modules:
  graph        -- operator graph IR and the three transformer graph builders
  numerics     -- float32 / bfloat16 round-to-nearest-even helpers
  execute      -- canonical row-major executor (every edge rounded to its
                  dtype) and the layout-permuted single-arena executor
  layouts      -- candidate layouts per edge, strides, view predicate
  plan_layout  -- longest-path decomposition (Alg. 1-2), per-path dynamic
                  program (Eq. 1 / Alg. 3), majority vote and re-optimisation
  plan_arena   -- Greedy-by-Size arena placement (Alg. 4), naive plan,
                  max-live lower bound
  brute        -- exhaustive searches used as pins on tiny inputs
  costtable    -- reader for the JSON cost-table file format

Every function is pinned by a CPU test against something other than itself
(closed forms, brute force, library routines); see tests/test_oracle_*.py.
"""
