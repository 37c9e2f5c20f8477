"""Pins for the oracle layout planner (Alg. 1-3, Eq. 1, vote)."""
import itertools

import numpy as np
import pytest

import synth_inputs
from oracle import brute, costtable, graph, plan_layout as PL
from oracle.graph import Graph
from tables import fanout_costs, rank2_table, synthetic_table
from tinygraphs import chain_graph, diamond_graph, fanout_graph, t1_graph, t2_graph


def _all_paths_len(g, S):
    """Brute force: the largest node count of any producer->consumer path in S."""
    Sset = set(S)
    succ = {n: [] for n in S}
    for n in S:
        for e in g.act_inputs(n):
            p = g.producer(e)
            if p is not None and p in Sset:
                succ[p].append(n)
    best = 0

    def dfs(n, k):
        nonlocal best
        best = max(best, k)
        for m in succ[n]:
            dfs(m, k + 1)
    for n in S:
        dfs(n, 1)
    return best


def _random_dag(rng, n):
    g = Graph(dtype="f32")
    g.add_input((2, 3))
    for i in range(n):
        k = int(rng.integers(1, 3))
        ins = sorted({int(rng.integers(0, g.n_edges)) for _ in range(k)})
        if len(ins) == 1:
            g.add_node("gelu", ins, (2, 3))
        else:
            g.add_node("add", ins[:2], (2, 3))
    g.outputs = [g.n_edges - 1]
    return g


def test_longest_path_is_longest_and_split_partitions():
    rng = np.random.default_rng(0)
    for _ in range(200):
        g = _random_dag(rng, int(rng.integers(1, 12)))
        S = list(range(len(g.nodes)))
        p = PL.longest_path(g, S)
        assert len(p) == _all_paths_len(g, S)
        for a, b in zip(p, p[1:]):
            assert a in [g.producer(e) for e in g.act_inputs(b)]
        paths = PL.split(g)
        flat = sorted(n for q in paths for n in q)
        assert flat == S
        for q in paths:
            for a, b in zip(q, q[1:]):
                assert a in [g.producer(e) for e in g.act_inputs(b)]


def test_post_ln_layer_paths():
    g = graph.build_transformer(synth_inputs.config(1))
    paths = PL.split(g)
    assert paths[0] == [0, 1, 2, 3, 12, 13, 14, 15, 16, 17, 18, 19, 20, 21, 22, 23, 24, 25, 26, 27]
    assert paths[1:] == [[4, 5, 6, 7], [8, 9, 10, 11]]


def _ct(g, **kw):
    return costtable.load(synthetic_table(g, **kw), g)


@pytest.mark.parametrize("seed", range(12))
def test_dp_on_pure_chain_equals_brute_force(seed):
    g = chain_graph(4, (2, 3, 4))
    mode = "distinct" if seed % 2 else "random"
    ct = _ct(g, seed=seed, mode=mode, lo=1, hi=20)
    plan = PL.plan_layouts(g, ct, PL.NO_GUARD)
    opt_total, opt_lay = brute.best_layouts(g, ct)
    assert plan.total == opt_total
    if mode == "distinct":
        assert plan.layout_idx == opt_lay
    # the variant-0 column is an independent table for the same check
    plan0 = PL.plan_layouts(g, ct, PL.NO_GUARD | PL.NO_VARIANTS)
    assert plan0.total == brute.best_layouts(g, ct, use_v0=True)[0]


@pytest.mark.parametrize("builder", [diamond_graph, t1_graph, t2_graph])
@pytest.mark.parametrize("seed", range(4))
def test_branched_plan_between_optimum_and_identity(builder, seed):
    g = builder()
    ct = _ct(g, seed=seed, mode="random", lo=1, hi=50)
    plan = PL.plan_layouts(g, ct)
    ident = PL.plan_cost(g, ct, False, [0] * g.n_edges)
    opt, _ = brute.best_layouts(g, ct)
    assert opt <= plan.total <= ident
    assert plan.total == PL.plan_cost(g, ct, False, plan.layout_idx)


def _rank2_table(g, costs):
    return rank2_table(g, costs)


def _hand_diamond():
    """x -> a=gelu(x) -> {b=silu(a), c=gelu(a)}; b2=silu(b); d=add(b2,c);
    y=gelu(d).  Paths: [a b b2 d y] and [c]; shared edges a and c."""
    g = Graph(dtype="f32")
    x = g.add_input((2, 3))
    a = g.add_node("gelu", [x], (2, 3))
    b = g.add_node("silu", [a], (2, 3))
    c = g.add_node("gelu", [a], (2, 3))
    b2 = g.add_node("silu", [b], (2, 3))
    d = g.add_node("add", [b2, c], (2, 3))
    y = g.add_node("gelu", [d], (2, 3))
    g.outputs = [y]
    same = {(0, 0): 10, (1, 1): 10, (0, 1): 50, (1, 0): 50}
    costs = [
        {(0, 0): 10, (0, 1): 10},                           # a
        dict(same),                                         # b
        {(0, 0): 25, (1, 1): 1, (0, 1): 50, (1, 0): 50},    # c
        dict(same),                                         # b2
        {k: (10 if k[0] == k[1] == k[2] else 100)
         for k in itertools.product((0, 1), repeat=3)},     # d
        {(0, 0): 10, (1, 0): 30},                           # y (output pinned)
    ]
    return g, costs


def test_hand_worked_vote_with_cost_tie_breaks():
    """Worked by hand.  Alone, path [a b b2 d y] is cheapest all row-major
    (50) and path [c] prefers a, c column-major (cost 1), so edges a and c
    each get one ballot per layout.  Tie on a: fixing a row-major costs
    50 + 25 = 75 over the two paths, column-major 70 + 1 = 71 -> column.
    Tie on c (a fixed column): row 90 + 50 = 140, column 70 + 1 = 71 -> column.
    Re-optimised plan: a b c b2 d all column-major, total 71 < row-major 75."""
    g, costs = _hand_diamond()
    ct = costtable.load(_rank2_table(g, costs), g)
    paths = PL.split(g)
    assert paths == [[0, 1, 3, 4, 5], [2]]
    infos = [PL.PathInfo(g, p) for p in paths]
    t0, s0, b0, _ = PL.dp_path(g, ct, False, infos[0], {})
    t1, s1, b1, _ = PL.dp_path(g, ct, False, infos[1], {})
    assert (t0, s0) == (50, [0, 0, 0, 0, 0]) and b0[3] == {3: 0}
    assert (t1, s1) == (1, [1]) and b1[0] == {1: 1}
    plan = PL.plan_layouts(g, ct)
    assert plan.layout_idx == [0, 1, 1, 1, 1, 1, 0]
    assert plan.total == 71 and plan.guard_used == 0
    assert PL.plan_cost(g, ct, False, [0] * 7) == 75


def test_guard_returns_identity_when_vote_hurts():
    """Worked by hand on the fan-out graph (paths [a b b2 s y], [c], [d]).
    Alone, the first path costs 50 all row-major (a column-major would add
    100 on b); [c] and [d] each cost 9 with a column-major a (10 row-major).
    Ballots on a: row (owner), column, column -> column wins 2:1.  Edges c
    and d get their owners' row-major states.  Re-optimised with a column:
    150 + 9 + 9 = 168 > 70, the all-row-major cost (seven nodes at 10), so
    the guard returns the row-major plan."""
    g = fanout_graph()
    ct = costtable.load(rank2_table(g, fanout_costs()), g)
    paths = PL.split(g)
    assert paths == [[0, 1, 2, 5, 6], [3], [4]]
    infos = [PL.PathInfo(g, p) for p in paths]
    firsts = [PL.dp_path(g, ct, False, i, {}) for i in infos]
    assert [f[0] for f in firsts] == [50, 9, 9]
    assert firsts[0][1][0] == 0 and firsts[1][2][0] == {1: 1} and firsts[2][2][0] == {1: 1}
    assert PL.plan_cost(g, ct, False, [0] * g.n_edges) == 70
    voted = PL.plan_layouts(g, ct, PL.NO_GUARD)
    assert voted.layout_idx == [0, 1, 0, 0, 0, 0, 0, 0]
    assert voted.total == 168 and voted.guard_used == 0
    assert PL.plan_cost(g, ct, False, voted.layout_idx) == 168
    plan = PL.plan_layouts(g, ct)
    assert plan.layout_idx == [0] * g.n_edges
    assert plan.total == 70 and plan.guard_used == 1
    assert plan.variant == [0] * len(g.nodes)


def test_guard_catches_a_path_infeasible_after_the_vote():
    """Same ballots, but b has no entry for a column-major a: after the vote
    fixes a column-major, the first path has no feasible layout.  With the
    guard the row-major plan is returned (guard_used 1); without it the
    planner reports the path as infeasible."""
    g = fanout_graph()
    ct = costtable.load(rank2_table(g, fanout_costs(infeasible_after_vote=True)), g)
    plan = PL.plan_layouts(g, ct)
    assert plan.layout_idx == [0] * g.n_edges
    assert plan.total == 70 and plan.guard_used == 1
    with pytest.raises(PL.Infeasible, match="after the vote"):
        PL.plan_layouts(g, ct, PL.NO_GUARD)


def test_missing_identity_entry_is_infeasible():
    g = chain_graph(3, (2, 3, 4))
    obj = synthetic_table(g, seed=0, drop_identity_node=1)
    ct = costtable.load(obj, g)
    with pytest.raises(PL.Infeasible):
        PL.plan_layouts(g, ct)


def test_no_dp_returns_identity_and_ties_prefer_identity():
    g = graph.build_transformer(synth_inputs.config(1))
    ct = _ct(g, seed=3)
    p = PL.plan_layouts(g, ct, PL.NO_DP)
    assert p.layout_idx == [0] * g.n_edges and p.guard_used == 0
    pt = PL.plan_layouts(g, _ct(g, seed=3, mode="ties"))
    # with every copy costing the same, the plan removes transposes (views
    # cost 0) and never costs more than row-major
    ident = PL.plan_cost(g, _ct(g, seed=3, mode="ties"), False, [0] * g.n_edges)
    assert pt.total <= ident


def test_identity_favouring_table_gives_identity_plan():
    g = graph.build_transformer(synth_inputs.config(1))
    ct = _ct(g, seed=4, mode="identity")
    p = PL.plan_layouts(g, ct)
    assert p.total <= PL.plan_cost(g, ct, False, [0] * g.n_edges)


@pytest.mark.parametrize("seed", range(6))
@pytest.mark.parametrize("layers", [1, 2])
def test_fused_dp_on_pure_chain_equals_brute_force(seed, layers):
    """With fusion chains priced (MatMul + bias Add + GELU per layer), the
    per-path DP has skip transitions; on a pure chain it is still exact: its
    total equals the minimum over every layout assignment and every set of
    non-overlapping chains, searched exhaustively."""
    from tables import add_fused
    g = __import__("tinygraphs").mlp_graph(layers)
    obj = add_fused(synthetic_table(g, seed=seed, mode="random", lo=1, hi=30), g, seed, lo=1, hi=60)
    ct = costtable.load(obj, g)
    plan = PL.plan_layouts(g, ct, PL.NO_GUARD)
    assert plan.total == brute.best_layouts_fused(g, ct)
    assert plan.total == PL.plan_cost(g, ct, False, plan.layout_idx, plan.fuse)
    # the plan's variants: the fused entry's on the MatMul, -2 on the absorbed nodes
    for m, t in enumerate(plan.fuse):
        if t:
            assert all(plan.variant[m + i] == -2 for i in range(1, t + 1))
            assert plan.variant[m] >= 0


def test_fusion_priced_against_running_alone():
    """Fused entries far more expensive than the separate nodes: no chain is
    fused and the plan is the plain DP's; far cheaper: every MatMul fuses
    its whole chain.  NO_FUSION ignores the fused entries."""
    from tables import add_fused
    g = __import__("tinygraphs").mlp_graph(2)
    base = synthetic_table(g, seed=3, mode="random", lo=1, hi=30)
    plain = PL.plan_layouts(g, costtable.load(base, g))
    dear = costtable.load(add_fused(json_copy(base), g, 3, lo=10 ** 6, hi=10 ** 6 + 10), g)
    p1 = PL.plan_layouts(g, dear)
    assert p1.fuse == [0] * len(g.nodes) and p1.total == plain.total and p1.layout_idx == plain.layout_idx
    cheap = costtable.load(add_fused(json_copy(base), g, 3, lo=1, hi=1), g)
    p2 = PL.plan_layouts(g, cheap)
    assert p2.fuse == [2, 0, 0, 2, 0, 0] and p2.total == 2
    p3 = PL.plan_layouts(g, cheap, PL.NO_FUSION)
    assert p3.fuse == [0] * len(g.nodes) and p3.total == plain.total


def json_copy(o):
    import json
    return json.loads(json.dumps(o))


def test_fused_plan_arena_and_permuted_execution():
    """A fused plan's arena holds no buffer for the results kept on chip,
    keeps each fused MatMul's operands live to the chain's end, places no two
    live buffers over each other, and the permuted execution in the poisoned
    arena equals the row-major result."""
    from oracle import execute, plan_arena
    from tables import add_fused
    import synth_inputs
    cfg = synth_inputs.config(1, arch="post_ln", layers=1, batch=2, seq=5, hidden=6, heads=2, ffn=8)
    g = graph.build_transformer(cfg)
    obj = add_fused(synthetic_table(g, seed=5, mode="random", lo=1, hi=40), g, 5, lo=1, hi=40)
    ct = costtable.load(obj, g)
    plan = PL.plan_layouts(g, ct)
    assert any(plan.fuse)
    lay = {e: ct.L[e][plan.layout_idx[e]] for e in range(g.n_edges)}
    ap = plan_arena.plan_arena(g, lay, fuse=plan.fuse)
    assert plan_arena.check_disjoint(ap)
    for m, t in enumerate(plan.fuse):
        for i in range(t):
            assert g.out_edge(m + i) not in ap.buffers
        for v in g.act_inputs(m):
            if v in ap.last:
                assert ap.last[v] >= m + t
    x, cs = synth_inputs.make_inputs(cfg, g.const_specs(), 9)
    ref = execute.run_canonical(g, [x], cs)
    out = execute.run_in_arena(g, lay, ap.root, ap.offset, ap.peak, [x], cs, fuse=plan.fuse)
    assert np.array_equal(out[0], ref[0])


@pytest.mark.parametrize("seed", range(6))
@pytest.mark.parametrize("builder", ["mlp2", "mlp3", "ffn_block"])
def test_best_chains_is_the_cheapest_chain_set(seed, builder):
    """For fixed layouts the chain choice is exact: best_chains' set costs
    the minimum over every set of disjoint chains (enumerated), and no
    plan the planner returns could lower its total by choosing its chains
    differently."""
    import tinygraphs
    from oracle import fusion
    from tables import add_fused
    g = {"mlp2": lambda: tinygraphs.mlp_graph(2), "mlp3": lambda: tinygraphs.mlp_graph(3),
         "ffn_block": tinygraphs.ffn_block}[builder]()
    obj = add_fused(synthetic_table(g, seed=seed, mode="random", lo=1, hi=40), g, seed, lo=1, hi=70)
    ct = costtable.load(obj, g)
    chains = sorted(ct.fused)
    assert chains
    rng = np.random.default_rng(seed)

    def brute_min(lay):
        best = None
        for k in range(len(chains) + 1):
            for sel in itertools.combinations(chains, k):
                spans = [set(range(m, m + t + 1)) for m, t in sel]
                if any(a & b for i, a in enumerate(spans) for b in spans[i + 1:]):
                    continue
                fz = [0] * len(g.nodes)
                for m, t in sel:
                    fz[m] = t
                c = PL.plan_cost(g, ct, False, lay, fz)
                best = c if best is None else min(best, c)
        return best

    for _ in range(4):
        lay = [int(rng.integers(0, len(ct.L[e]))) for e in range(g.n_edges)]
        fz = PL.best_chains(g, ct, False, lay)
        assert PL.plan_cost(g, ct, False, lay, fz) == brute_min(lay)
        # every chosen chain is a chain of the graph, disjoint from the others
        assert all((m, t) in fusion.all_chains(g) for m, t in enumerate(fz) if t)
    plan = PL.plan_layouts(g, ct)
    assert plan.total == brute_min(plan.layout_idx)


@pytest.mark.parametrize("arch", ["post_ln", "pre_ln", "llama"])
def test_fusion_chains_of_transformer_layers(arch):
    """The chain rules on one layer of each block kind, enumerated by hand
    from the builder's node order: a MatMul with its bias, activation and
    residual steps, and the residual Add with the normalisation right after
    it -- on chip where the sum has that norm as its only reader (post-LN;
    the last sum of pre-LN / Llama, before the final norm), stored by the
    launch where the next residual reads it too (pre-LN, Llama)."""
    from oracle import fusion
    cfg = synth_inputs.config(1, arch=arch, layers=1, seq=8, hidden=32, heads=2, ffn=48)
    g = graph.build_transformer(cfg)
    ops = [nd.op for nd in g.nodes]
    got = {k: [ops[n] for n in v] for k, v in fusion.all_chains(g).items()}
    norm_heads = sorted(m for (m, t), v in got.items() if v[0] == "add" and t == 1)
    kinds = []
    for m in norm_heads:
        assert got[(m, 1)][1] in ("layernorm", "rmsnorm")
        (step,) = fusion.chain_steps(g, m)
        readers = [n for n, x in enumerate(g.nodes) if g.out_edge(m) in x.ins]
        assert step == (m + 1, "norm" if readers == [m + 1] else "norm_store", None)
        assert fusion.chain_slots(g, m, 1) == list(g.nodes[m].ins)
        assert fusion.stored_edges(g, m, 1) == ([] if step[1] == "norm" else [g.out_edge(m)])
        assert fusion.on_chip_edges(g, m, 1) == ([g.out_edge(m)] if step[1] == "norm" else [])
        kinds.append(step[1])
    # residual sums (two activations) with a norm right after them
    expect = [m for m, nd in enumerate(g.nodes) if nd.op == "add" and min(nd.ins) >= 0 and m + 1 < len(ops)
              and ops[m + 1] in ("layernorm", "rmsnorm") and g.nodes[m + 1].ins[0] == g.out_edge(m)]
    assert norm_heads == expect
    assert kinds == {"post_ln": ["norm", "norm"], "pre_ln": ["norm_store", "norm"],
                     "llama": ["norm_store", "norm"]}[arch]
    # MatMul chains: the FFN up-projection with bias and GELU (post/pre-LN),
    # the down-projection with bias and the residual (post/pre-LN) or with
    # the residual alone (Llama)
    mm = {m: v for (m, t), v in got.items() if v[0] == "matmul"}
    if arch in ("post_ln", "pre_ln"):
        assert ["matmul", "add", "gelu"] in mm.values()
        assert ["matmul", "add", "add"] in mm.values()
    else:
        assert ["matmul", "silu"] in mm.values() and ["matmul", "add"] in mm.values()
        # SiLU's product meets the up-projection only after another MatMul
        assert ["matmul", "silu", "mul"] not in mm.values()


@pytest.mark.parametrize("arch", ["pre_ln", "llama"])
@pytest.mark.parametrize("seed", [0, 1, 2])
def test_stored_residual_sums(arch, seed):
    """Pre-norm stacks: a residual sum read by its norm and by the next
    residual.  When the plan fuses such a sum with its norm, the launch
    stores the sum too, in the norm output's layout: the sum keeps its
    arena buffer (live to its last reader), its layout equals the norm's,
    the plan's total is its recomputed cost, and the permuted execution in
    the poisoned arena equals the row-major result."""
    from oracle import execute, fusion, plan_arena
    from tables import add_fused
    cfg = synth_inputs.config(1, arch=arch, layers=1, batch=2, seq=5, hidden=8, heads=2, ffn=8)
    g = graph.build_transformer(cfg)
    # residual-norm entries well below the separate nodes, MatMul chains
    # (which would take the same Add) well above, so that sums are fused
    obj = add_fused(synthetic_table(g, seed=seed, mode="random", lo=50, hi=100), g, seed, lo=1, hi=20)
    for fs in obj["fused_sigs"]:
        if fs["op"] == "matmul":
            for ent in fs["entries"]:
                ent[2] = [c * 50 for c in ent[2]]
    ct = costtable.load(obj, g)
    plan = PL.plan_layouts(g, ct)
    stored = [(m, t) for m, t in enumerate(plan.fuse) if t and fusion.stored_edges(g, m, t)]
    assert stored
    assert plan.total == PL.plan_cost(g, ct, False, plan.layout_idx, plan.fuse)
    lay = {e: ct.L[e][plan.layout_idx[e]] for e in range(g.n_edges)}
    ap = plan_arena.plan_arena(g, lay, fuse=plan.fuse)
    assert plan_arena.check_disjoint(ap)
    for m, t in stored:
        (e,) = fusion.stored_edges(g, m, t)
        assert e in ap.buffers and lay[e] == lay[g.out_edge(m + t)]
        # live to its last reader (to that reader's chain end if it heads one)
        last = max(n + plan.fuse[n] for n, x in enumerate(g.nodes) if e in x.ins)
        assert ap.last[e] == last > m + t
    for m, t in enumerate(plan.fuse):
        for e in fusion.on_chip_edges(g, m, t) if t else []:
            assert e not in ap.buffers
    x, cs = synth_inputs.make_inputs(cfg, g.const_specs(), 9)
    ref = execute.run_canonical(g, [x], cs)
    out = execute.run_in_arena(g, lay, ap.root, ap.offset, ap.peak, [x], cs, fuse=plan.fuse)
    assert np.array_equal(out[0], ref[0])


@pytest.mark.parametrize("seed", range(4))
def test_stored_sum_chain_choice_and_optimum(seed):
    """A residual sum with a second reader (tiny pre-norm graph): its chain
    with the LayerNorm is the stored kind; for random layout assignments the
    chosen chain set costs what the definition gives -- the separate nodes,
    or, when the sum's layout equals the norm output's, the cheaper of that
    and the fused entry -- and the plan costs no less than the exhaustive
    optimum over every layout assignment and chain set."""
    from oracle import fusion
    from tables import add_fused
    from tinygraphs import prenorm_graph
    g = prenorm_graph()
    sm = next(m for m, nd in enumerate(g.nodes) if nd.op == "add" and g.nodes[m + 1].op == "layernorm")
    assert fusion.chain_steps(g, sm) == [(sm + 1, "norm_store", None)]
    obj = add_fused(synthetic_table(g, seed=seed, mode="random", lo=10, hi=60), g, seed, lo=1, hi=70)
    ct = costtable.load(obj, g)
    rng = np.random.default_rng(seed)
    es, eo = g.out_edge(sm), g.out_edge(sm + 1)
    for _ in range(60):
        lay = [int(rng.integers(0, len(ct.L[e]))) for e in range(g.n_edges)]
        if rng.random() < 0.5:    # often put the sum in the norm output's layout
            lay[es] = ct.L[es].index(ct.L[eo][lay[eo]])
        own = [int(ct.nodes[n].best[tuple(lay[e] for e in g.act_inputs(n)) + (lay[g.out_edge(n)],)])
               for n in range(len(g.nodes))]
        want = sum(own)
        if ct.L[es][lay[es]] == ct.L[eo][lay[eo]]:
            fz = int(ct.fused[(sm, 1)].best[tuple(lay[e] for e in g.nodes[sm].ins) + (lay[eo],)])
            want = min(want, want - own[sm] - own[sm + 1] + fz)
        assert PL.plan_cost(g, ct, False, lay, PL.best_chains(g, ct, False, lay)) == want
    plan = PL.plan_layouts(g, ct, PL.NO_GUARD)
    assert plan.total >= brute.best_layouts_fused(g, ct)
    if plan.fuse[sm]:
        assert ct.L[es][plan.layout_idx[es]] == ct.L[eo][plan.layout_idx[eo]]
