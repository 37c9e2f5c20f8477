"""Pins for the oracle arena planner (Alg. 4, Greedy-by-Size)."""
import numpy as np
import pytest

import synth_inputs
from oracle import brute, graph, layouts, plan_arena as pa
from tinygraphs import ffn_block, mlp_graph


def test_hand_worked_best_fit_example():
    """Five buffers worked by hand.  Sizes 600/400/300/200 are placed first
    (0, 600, 1000, 1300); the 100-byte buffer [4,6] then sees two gaps among
    the buffers alive with it: [0,600) and [1000,1300).  The smallest gap that
    fits is chosen (offset 1000); a first-fit rule would have taken 0."""
    size = {0: 100, 1: 600, 2: 300, 3: 200, 4: 400}
    defn = {0: 4, 1: 0, 2: 2, 3: 2, 4: 2}
    last = {0: 6, 1: 3, 2: 3, 3: 6, 4: 6}
    off, peak = pa.greedy_by_size(list(size), size, defn, last)
    assert off == {1: 0, 4: 600, 2: 1000, 3: 1300, 0: 1000}
    assert peak == 1500
    # max-live bound by hand: at nodes 2 and 3 buffers 1, 2, 3, 4 are live
    # (600 + 300 + 200 + 400); at 4..6 only 0, 3, 4 (700); at 0..1 only 1
    assert pa.lower_bound(list(size), size, defn, last, 7) == 1500


def test_lower_bound_below_optimum_hand_worked():
    """Seven buffers (in units of 256 B) whose max-live bound is 5 units while
    no placement fits in 5.  Live sets: node 1 {4:2, 2:3}, node 2 {2:3, 1:1,
    5:1}, node 3 {1:1, 3:2, 5:1}, node 4 {0:2, 3:2, 5:1}, node 5 {0:2, 6:3}:
    at most 5 units.  In 5 units, node 1 forces buffer 2 to one end (the two
    units of buffer 4 must be contiguous), say the bottom [0,3) (the other
    case is its mirror image); node 2 then puts buffers 1 and 5 in units 3
    and 4; node 3 leaves buffer 3 inside [0,3); node 5 forces buffer 0 to an
    end; at node 4 buffer 0 cannot take [0,2) (buffer 3 overlaps it) nor
    [3,5) (buffer 5 sits in unit 3 or 4).  So the optimum is 6 units, which
    Greedy-by-Size reaches.  With half-open lifetimes the bound would be only
    3 units (buffers ending at a node would not count there)."""
    u = 256
    items = {0: (2, 4, 5), 1: (1, 2, 3), 2: (3, 1, 2), 3: (2, 3, 4), 4: (2, 0, 1), 5: (1, 2, 4), 6: (3, 5, 6)}
    bs = sorted(items)
    size = {b: items[b][0] * u for b in bs}
    defn = {b: items[b][1] for b in bs}
    last = {b: items[b][2] for b in bs}
    assert pa.lower_bound(bs, size, defn, last, 7) == 5 * u
    assert brute.best_arena_peak(bs, size, defn, last) == 6 * u
    off, peak = pa.greedy_by_size(bs, size, defn, last)
    assert peak == 6 * u
    assert pa.check_disjoint(pa.ArenaPlan(None, bs, size, defn, last, off, peak))


def test_no_reuse_when_all_lifetimes_overlap():
    size = {0: 256, 1: 512, 2: 768}
    defn = {0: 0, 1: 0, 2: 0}
    last = {0: 5, 1: 5, 2: 5}
    off, peak = pa.greedy_by_size([0, 1, 2], size, defn, last)
    assert peak == sum(size.values())
    assert off == {2: 0, 1: 768, 0: 1280}


def test_random_interval_sets_bounds_and_brute_force():
    rng = np.random.default_rng(0)
    gaps = []
    for _ in range(300):
        n = int(rng.integers(1, 7))
        bs = list(range(n))
        size = {b: int(rng.integers(1, 9)) * 256 for b in bs}
        defn, last = {}, {}
        for b in bs:
            a = int(rng.integers(0, 8))
            defn[b], last[b] = a, int(rng.integers(a, 9))
        off, peak = pa.greedy_by_size(bs, size, defn, last)
        plan = pa.ArenaPlan(None, bs, size, defn, last, off, peak)
        assert pa.check_disjoint(plan)
        lb = pa.lower_bound(bs, size, defn, last, 9)
        opt = brute.best_arena_peak(bs, size, defn, last)
        assert lb <= opt <= peak <= sum(size.values())
        gaps.append(peak - opt)
    assert max(gaps) >= 0


@pytest.mark.parametrize("builder", [lambda: mlp_graph(3), lambda: mlp_graph(2), ffn_block])
def test_greedy_is_optimal_on_small_builder_graphs(builder):
    g = builder()
    ident = {e: tuple(range(len(g.edge_shape(e)))) for e in range(g.n_edges)}
    ap = pa.plan_arena(g, ident)
    assert len(ap.buffers) <= 8
    opt = brute.best_arena_peak(ap.buffers, ap.size, ap.defn, ap.last)
    assert ap.peak == opt
    assert pa.check_disjoint(ap)


@pytest.mark.parametrize("idx", [1, 2, 3])
def test_config_graphs_bounds(idx):
    g = graph.build_transformer(synth_inputs.config(idx))
    L = layouts.edge_layouts(g)
    rng = np.random.default_rng(idx)
    naive = pa.naive_plan(g)
    for trial in range(3):
        lay = {e: (L[e][0] if trial == 0 else L[e][int(rng.integers(0, len(L[e])))])
               for e in range(g.n_edges)}
        ap = pa.plan_arena(g, lay)
        assert pa.check_disjoint(ap)
        lb = pa.lower_bound(ap.buffers, ap.size, ap.defn, ap.last, len(g.nodes))
        assert lb <= ap.peak
        if trial == 0:
            assert ap.peak <= naive.peak
            assert ap.peak < naive.peak       # these graphs do have reusable buffers


def test_naive_plan_is_prefix_sum_and_views_share_roots():
    g = graph.build_transformer(synth_inputs.config(1))
    nv = pa.naive_plan(g)
    cur = 0
    for b in sorted(nv.buffers):
        assert nv.offset[b] == cur
        cur += nv.size[b]
    assert nv.peak == cur
    # row-major: every split/merge Reshape is a view, every Transpose a copy
    for n, nd in enumerate(g.nodes):
        e = g.out_edge(n)
        if nd.op == "reshape":
            assert nv.root[e] != e
        elif nd.op == "transpose":
            assert nv.root[e] == e
