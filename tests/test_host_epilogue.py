"""Epilogue fusion decisions on the CPU (host-only library): how many
launches a run of a plan enqueues, and the arena option that keeps a fused
MatMul's operands live until the end of the nodes it absorbs."""
import os

import pytest

import synth_inputs
from gpu_util import forced_table
from oracle import fusion, graph as OG, plan_arena as PA
from paper_2411_09242_amd import fluid as F
from tables import synthetic_table, write_table
from test_gpu_ops import EPILOGUES, epilogue_graph, fusable_steps


@pytest.fixture(scope="module", autouse=True)
def host_lib():
    return F.load(host_only=True)


def _plan(og, table_obj, tmp_path, flags=0):
    g = F.Graph.from_desc(og.export())
    path = os.path.join(tmp_path, "t.json")
    write_table(table_obj, path)
    t = F.CostTable.load(path, g)
    return g, F.LayoutPlan(g, t, flags)


def _launches(g, lp, **kw):
    ap = F.ArenaPlan(g, lp, **kw)
    return F.fluid_run_launches(g.h, lp.h, ap.h), ap


@pytest.mark.parametrize("chain", sorted(EPILOGUES))
@pytest.mark.parametrize("v", [0, 2, 7, 9])
@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_epilogue_arena_lets_every_chain_fuse(chain, v, dtype, tmp_path):
    """Without keep-alive readers, the default arena may put the chain's
    output over the MatMul's input (its lifetime ends at the MatMul), which
    refuses the fusion; with FLUID_ARENA_EPILOGUE the chain always fuses, as
    far as the variant's epilogue reaches."""
    if dtype == "f32" and v >= 8:
        pytest.skip("variants 8 and 9 are bf16 only")
    og, a, r, edges = epilogue_graph(2, 24, 32, 32, dtype, keep_a=False, chain=chain)
    mm = [i for i, nd in enumerate(og.nodes) if nd.op == "matmul"][0]
    g, lp = _plan(og, forced_table(og, {}, {mm: v}), tmp_path)
    nonview = sum(1 for n in range(g.n_nodes) if lp.kernel(n) != "view")
    n_def, _ = _launches(g, lp)
    n_epi, ap = _launches(g, lp, epilogue=True)
    n_nr, _ = _launches(g, lp, no_reuse=True)
    assert n_epi == n_nr == nonview - fusable_steps(chain, v, dtype)
    assert n_def >= n_epi


@pytest.mark.parametrize("chained", [False, True])
@pytest.mark.parametrize("variant,dtype,grouped", [(6, "f32", True), (7, "f32", True), (2, "f32", False),
                                                   (6, "bf16", False)])
def test_grouped_launch_count(chained, variant, dtype, grouped, tmp_path):
    """Sibling products of the fp32 direct-load tiles share one launch
    unless one reads another's output; other tiles launch one by one."""
    from test_gpu_ops import siblings_graph
    og, prods, outs = siblings_graph(1, 37, 64, 64, dtype, chained)
    mms = [i for i, nd in enumerate(og.nodes) if nd.op == "matmul"]
    g, lp = _plan(og, forced_table(og, {}, {m: variant for m in mms}), tmp_path)
    nonview = sum(1 for n in range(g.n_nodes) if lp.kernel(n) != "view")
    n, _ = _launches(g, lp, epilogue=True)
    saved = (1 if chained else 2) if grouped else 0
    assert n == nonview - 3 - saved


@pytest.mark.parametrize("T,D,extra", [(128, 64, False), (40, 32, True)])
def test_attention_runs_as_its_three_operators(T, D, extra, tmp_path):
    """Q K^T, Softmax and P V each run their own launch (the scores and
    probabilities are arena tensors, as in the paper's operator chain); only
    the GELU after P V goes into that product's epilogue."""
    from test_gpu_ops import chain_attn_graph
    og, q, k, v, s, p, o = chain_attn_graph(1, 2, 40, T, D, False, extra)
    g, lp = _plan(og, forced_table(og, {}), tmp_path)
    nonview = sum(1 for n in range(g.n_nodes) if lp.kernel(n) != "view")
    n, ap = _launches(g, lp, epilogue=True)
    assert n == nonview - 1
    launch, written, names = F.fluid_run_schedule(g.h, lp.h, ap.h, g.n_nodes)
    sn, pn, on = og.producer(s), og.producer(p), og.producer(o)
    assert len({launch[sn], launch[pn], launch[on]}) == 3
    assert written[sn] and written[pn] and not written[on]
    assert launch[on + 1] == launch[on] and written[on + 1]
    assert names[launch[on]].endswith("_eg") and names[launch[pn]].startswith("softmax")


CFGS = [synth_inputs.config(1, arch="post_ln", layers=2, seq=17, hidden=40, heads=5, ffn=72),
        synth_inputs.config(1, arch="pre_ln", layers=2, seq=19, hidden=36, heads=3, ffn=52),
        synth_inputs.config(1, arch="llama", layers=2, seq=21, hidden=48, heads=4, ffn=40, dtype="bf16")]


@pytest.mark.parametrize("cfg", CFGS, ids=lambda c: c["arch"])
@pytest.mark.parametrize("seed", [0, 1, 2])
def test_epilogue_arena_on_transformers(cfg, seed, tmp_path):
    """Transformer stacks planned on random tables: with the option every
    fusion that a no-reuse arena allows happens, and the plan is still a
    valid arena under the paper's lifetimes (no two buffers live at the same
    node share a byte), no smaller than their max-live bound."""
    og = OG.build_transformer(cfg)
    tab = synthetic_table(og, seed=seed, mode="random", lo=1, hi=1000)
    # MatMul variants 0-2 run with any layouts; other operators keep
    # variant 0, which does too
    for sig in tab["sigs"]:
        for ent in sig["entries"]:
            ent[2] = [c if v == 0 or sig["op"] == "matmul" else -1 for v, c in enumerate(ent[2])]
            if max(ent[2]) < 0:
                ent[2][0] = 1
    g, lp = _plan(og, tab, tmp_path)
    n_def, ap_def = _launches(g, lp)
    n_epi, ap = _launches(g, lp, epilogue=True)
    n_nr, _ = _launches(g, lp, no_reuse=True)
    assert n_epi == n_nr <= n_def
    lay = {e: lp.perm(e) for e in range(og.n_edges)}
    ref = PA.plan_arena(og, lay)
    for b in ref.buffers:
        assert ap.offset[b] >= 0 and ap.offset[b] + ref.size[b] <= ap.peak
    for i, x in enumerate(ref.buffers):
        for y in ref.buffers[i + 1:]:
            if ref.defn[x] <= ref.last[y] and ref.defn[y] <= ref.last[x]:
                assert (ap.offset[x] + ref.size[x] <= ap.offset[y] or
                        ap.offset[y] + ref.size[y] <= ap.offset[x]), (x, y)
    assert ap.peak >= ap_def.lower_bound
    # the launch schedule: every non-view node is performed by one launch;
    # a node whose output no launch stores is read only inside its own launch
    launch, written, names = F.fluid_run_schedule(g.h, lp.h, ap.h, g.n_nodes)
    assert len(names) == n_epi == max(launch) + 1
    for n, nd in enumerate(og.nodes):
        is_view = lp.kernel(n) == "view"
        assert (launch[n] < 0) == is_view and not (is_view and written[n])
        e = og.out_edge(n)
        if e in og.outputs:
            assert written[n]
        if launch[n] >= 0 and not written[n]:
            readers = [m for m, md in enumerate(og.nodes) if e in md.ins]
            assert readers and all(launch[m] == launch[n] for m in readers), (n, readers)


@pytest.mark.parametrize("cfg", CFGS, ids=lambda c: c["arch"])
@pytest.mark.parametrize("seed", [0, 1])
def test_priced_fusions_are_the_launches(cfg, seed, tmp_path):
    """A table that prices fusion chains: the run performs exactly the chains
    the layout DP chose -- each in one launch that stores the chain's last
    output and the intermediates with further readers (a pre-norm block's
    residual sum, in the layout of the chain's output), the others without
    an arena buffer -- and no other fusion; without pricing (FLUID_NO_FUSION) the epilogue fusion by
    adjacency is back."""
    from tables import add_fused
    og = OG.build_transformer(cfg)
    tab = synthetic_table(og, seed=seed, mode="random", lo=1, hi=1000, n_variants=1)
    # chains priced for variant 1 only (a MatMul's: its tile performs every
    # epilogue step, variant 0 has no R operand; a residual norm's: the
    # column reduction, which runs on any layouts)
    add_fused(tab, og, seed, n_variants=2, lo=1, hi=1500)
    for fs in tab["fused_sigs"]:
        for ent in fs["entries"]:
            ent[2][0] = -1
    g, lp = _plan(og, tab, tmp_path)
    assert lp.fusion_priced and any(lp.fuse)
    n, ap = _launches(g, lp, epilogue=True)
    launch, written, names = F.fluid_run_schedule(g.h, lp.h, ap.h, g.n_nodes)
    kernels = [lp.kernel(i) for i in range(g.n_nodes)]
    assert n == len(names) == sum(1 for k in kernels if k not in ("view", "fused"))
    covered = set()
    for m, t in enumerate(lp.fuse):
        if not t:
            continue
        assert og.nodes[m].op in ("matmul", "add") and lp.variant[m] == 1
        chain = list(range(m, m + t + 1))
        covered.update(chain)
        assert all(lp.variant[k] == -2 and kernels[k] == "fused" for k in chain[1:])
        assert {launch[k] for k in chain} == {launch[m]}
        stored = fusion.stored_edges(og, m, t)
        assert written[chain[-1]]
        assert all(bool(written[k]) == (og.out_edge(k) in stored) for k in chain[:-1])
        assert all((ap.offset[og.out_edge(k)] >= 0) == (og.out_edge(k) in stored) for k in chain[:-1])
        for e in stored:
            assert lp.perm(e) == lp.perm(og.out_edge(m + t))
        if og.nodes[m].op == "matmul":
            assert "_e" in names[launch[m]]
        else:
            assert names[launch[m]] == kernels[m] and names[launch[m]].startswith("add_" + og.nodes[m + 1].op)
    for k in range(g.n_nodes):
        if k not in covered and kernels[k] != "view":
            assert written[k] and list(launch).count(launch[k]) == 1, k
    # without pricing: no -2, and adjacency fusion performs at least one chain
    g2, lp2 = _plan(og, tab, tmp_path, F.NO_FUSION)
    assert not lp2.fusion_priced and not any(lp2.fuse) and -2 not in lp2.variant
    n2, _ = _launches(g2, lp2, epilogue=True)
    assert n2 < sum(1 for i in range(g2.n_nodes) if lp2.kernel(i) != "view")
