"""Kernel parity on the GPU, per operator, through the C ABI.

Each case is a small graph whose interior edges are forced (by a cost table
that makes only that plan cheap) into chosen layouts and whose nodes are
forced onto chosen kernel variants; the run goes through fluid_run and the
output is compared element by element with the oracle's row-major result.
Sizes span several tiles and ragged tails.
"""
import itertools

import numpy as np
import pytest

from gpu_util import assert_close, forced_table, random_inputs, run_device, say
from oracle import execute, layouts
from oracle.graph import Graph

pytestmark = pytest.mark.gpu


def _check_gemm(og, want, variants, tmp_path, seed, dtype):
    """_check for a forced GEMM variant (tile = variant % 10; variants 10-19
    read the weight packed K-contiguous); the fp32 direct-load tiles (6, 7,
    8) need unit-stride K or M/N operands, the bf16 tiles 8 and 9 (9 is bf16
    only) a K-contiguous A and a K- or N-contiguous B (9 also K <= 128):
    they are skipped where they cannot run."""
    try:
        return _check(og, want, variants, tmp_path, seed=seed)
    except Exception as ex:  # noqa: BLE001
        t = max(variants.values()) % 10
        if (t >= 8 or (dtype == "f32" and t >= 6)) and "cannot run with these layouts" in str(ex):
            return None
        raise


def row_block_ok(shape, dtype, *perms):
    """Whether reduction variant 2 (a workgroup per row, 16-byte pieces)
    runs: the reduced (last) dim innermost in every layout, rows a multiple
    of 16 bytes and at most 4096 values."""
    R, vec = shape[-1], (8 if dtype == "bf16" else 4)
    return R % vec == 0 and R <= 4096 and all(p[-1] == len(shape) - 1 for p in perms)


def _check(og, want, variants, tmp_path, seed=0, scale=1.0):
    xs, cs = random_inputs(og, seed, scale)
    ref = execute.run_canonical(og, xs, cs)
    obj = forced_table(og, want, variants)
    out, lp, _ = run_device(og, obj, xs, cs, tmp_path)
    for a, b in zip(out, ref):
        assert_close(a, b, og.dtype, f"want={want} variants={variants}")
    return lp


# ------------------------------------------------------------------ GEMM
def proj_graph(B, S, K, N, dtype):
    g = Graph(dtype=dtype)
    x = g.add_input((B, S, K))
    a = g.add_node("gelu", [x], (B, S, K))
    w = g.add_const("weight", (K, N))
    c = g.add_node("matmul", [a, w], (B, S, N))
    y = g.add_node("gelu", [c], (B, S, N))
    g.outputs = [y]
    return g, a, c


PROJ_SHAPES = [(1, 37, 29, 53), (1, 130, 64, 70), (2, 65, 96, 40), (1, 256, 128, 256), (3, 8, 16, 200),
               (1, 300, 200, 264)]


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("shape", PROJ_SHAPES, ids=str)
@pytest.mark.parametrize("variant", list(range(20)))
def test_projection_gemm_all_layouts(dtype, shape, variant, tmp_path):
    """Every tile, with the weight row-major (variants 0-9) and packed
    K-contiguous by fluid_pack_constant (10-19), for every layout of A and C."""
    B, S, K, N = shape
    og, a, c = proj_graph(B, S, K, N, dtype)
    mm = 1
    La = layouts.layout_list((B, S, K))
    Lc = layouts.layout_list((B, S, N))
    for pa, pc in itertools.product(La, Lc):
        say(f"gemm proj {dtype} {shape} v{variant} A{pa} C{pc}")
        lp = _check_gemm(og, {a: pa, c: pc}, {mm: variant}, tmp_path, B * S + K, dtype)
        if lp is not None:
            assert lp.constant_layout(0) == ((1, 0) if variant >= 10 else (0, 1))


@pytest.mark.parametrize("shape", [(1, 37, 1000, 70), (2, 65, 3100, 40)], ids=str)
@pytest.mark.parametrize("variant", [6, 7, 8, 9, 16, 17, 18, 19])
def test_projection_gemm_long_k(shape, variant, tmp_path):
    """The fp32 direct-load tiles on K slices of more than six 16-k groups
    (the rotating K loop), group counts not divisible by 4 and K not
    divisible by 16, and the fp32 128 x 128 tiles on odd counts of 32-k
    tiles with a partial last one, with A in every layout and the weight
    row-major (6-9) or K-contiguous (16-19)."""
    B, S, K, N = shape
    og, a, c = proj_graph(B, S, K, N, "f32")
    for pa, pc in itertools.product(layouts.layout_list((B, S, K)), layouts.layout_list((B, S, N))[:2]):
        say(f"gemm long K {shape} v{variant} A{pa} C{pc}")
        _check_gemm(og, {a: pa, c: pc}, {1: variant}, tmp_path, B * S + K, "f32")


# epilogue chains after the MatMul: Add of a bias [N], GELU, SiLU, and the
# Add / Mul with another activation tensor r of the output's shape
EPILOGUES = {"bias": ["bias"], "bias_gelu": ["bias", "gelu"], "silu": ["silu"], "bias_silu": ["bias", "silu"],
             "res": ["add_r"], "bias_res": ["bias", "add_r"], "gate": ["mul_r"],
             "bias_gelu_gate": ["bias", "gelu", "mul_r"]}


def epilogue_graph(B, S, K, N, dtype, keep_a, chain="bias_gelu"):
    """gelu -> MatMul -> the chain's nodes; r = silu(second input) is the
    chain's other tensor (the residual of an Add, the gate of a Mul).  With
    keep_a the chain's output goes through a softmax (which no MatMul
    absorbs) and the MatMul's input stays live to the end (multiplied into
    the result), so the chain's output is an arena buffer that cannot share
    bytes with that input, and the whole chain always runs inside the
    MatMul.  Returns the graph, the MatMul's input edge, r (or None) and the
    edges of the product and of each chain node."""
    g = Graph(dtype=dtype)
    x = g.add_input((B, S, K))
    two = any(st.endswith("_r") for st in EPILOGUES[chain])
    x2 = g.add_input((B, S, N)) if two else None   # inputs before nodes
    a = g.add_node("gelu", [x], (B, S, K))
    r = g.add_node("silu", [x2], (B, S, N)) if two else None
    w = g.add_const("weight", (K, N))
    c = g.add_node("matmul", [a, w], (B, S, N))
    edges = [c]
    y = c
    for step in EPILOGUES[chain]:
        if step == "bias":
            y = g.add_node("add", [y, g.add_const("bias", (N,))], (B, S, N))
        elif step == "add_r":
            y = g.add_node("add", [y, r], (B, S, N))
        elif step == "mul_r":
            y = g.add_node("mul", [r, y], (B, S, N))   # chain operand second
        else:
            y = g.add_node(step, [y], (B, S, N))
        edges.append(y)
    if keep_a:
        assert K == N
        y = g.add_node("softmax", [y], (B, S, N), fattr=0.5)
        y = g.add_node("mul", [y, a], (B, S, N))
    else:
        y = g.add_node("mul", [y, y], (B, S, N))
    g.outputs = [y]
    return g, a, r, edges


def fusable_steps(chain, v, dtype):
    """How many of the chain's steps a MatMul of variant v absorbs when
    nothing else stops it: the bf16 variants 6, 8 and 9 (short-K attention
    products) take a bias only; the Add / Mul with another tensor is taken
    by variants 1-5, and by the fp32 variants 6-9."""
    bias_only = dtype == "bf16" and v in (6, 8, 9)
    rop = 1 <= v <= 5 or (dtype == "f32" and v in (6, 7, 8, 9))
    n = 0
    for step in EPILOGUES[chain]:
        if step == "bias" or (step in ("gelu", "silu") and not bias_only) or (step.endswith("_r") and rop):
            n += 1
        else:
            break
    return n


def reference_rounding_except(og, xs, cs, unrounded):
    """The oracle's operators in graph order, every edge rounded to the graph
    dtype except those in ``unrounded``: the intermediates of a fused launch,
    which never leave fp32 (so one rounding where separate nodes round after
    each)."""
    from oracle import numerics
    cv = [numerics.round_to(np.asarray(a, np.float64).reshape(shape), dt)
          for (role, shape, dt), a in zip(og.consts, cs)]
    vals = {e: numerics.round_to(np.asarray(a, np.float64).reshape(og.input_shapes[e]), og.dtype)
            for e, a in enumerate(xs)}
    for n, nd in enumerate(og.nodes):
        y = execute.eval_node(nd, [vals[v] if v >= 0 else cv[~v] for v in nd.ins])
        e = og.out_edge(n)
        vals[e] = y if e in unrounded else numerics.round_to(y, og.dtype)
    return [vals[e] for e in og.outputs]


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("shape", [(1, 37, 64, 64), (2, 130, 96, 96)], ids=str)
@pytest.mark.parametrize("keep_a", [True, False])
@pytest.mark.parametrize("chain", sorted(EPILOGUES))
def test_matmul_epilogue(dtype, shape, keep_a, chain, tmp_path):
    """The chain of nodes that fluid_run performs inside the MatMul's launch,
    for every GEMM variant and layouts of the MatMul's input and output, of
    r and of the chain's output: the oracle's result with the fused
    intermediates left unrounded."""
    from paper_2411_09242_amd import fluid as F
    og, a, r, edges = epilogue_graph(*shape, dtype, keep_a, chain)
    c, d = edges[0], edges[-1]
    mm = [i for i, nd in enumerate(og.nodes) if nd.op == "matmul"][0]
    L = layouts.layout_list(og.edge_shape(c))
    total = 0
    for v in range(10):
        for ia, ic, id_ in ((0, 0, 0), (1, 1, 0), (0, 1, 1), (1, 0, 1)):
            want = {a: L[ia], c: L[ic], d: L[id_]}
            if r is not None:
                want[r] = L[ia]
            seed = ia + 2 * ic + 4 * id_
            say(f"epilogue {chain} {dtype} {shape} keep_a={keep_a} v{v} {want}")
            xs, cs = random_inputs(og, seed)
            try:
                out, lp, ap = run_device(og, forced_table(og, want, {mm: v}), xs, cs, tmp_path)
            except Exception as ex:  # noqa: BLE001
                if (v >= 8 or (dtype == "f32" and v >= 6)) and "cannot run with these layouts" in str(ex):
                    continue
                raise
            nonview = sum(1 for x in lp.variant if x >= 0)
            n = F.fluid_run_launches(lp.graph.h, lp.h, ap.h)
            fused = nonview - n
            full = fusable_steps(chain, v, dtype)
            assert 0 <= fused <= full
            if keep_a:
                assert fused == full, "epilogue not fused"
            total += fused
            # the fused steps are a prefix of the chain: the product and the
            # outputs of all but the last fused node stayed in fp32
            ref = reference_rounding_except(og, xs, cs, set(edges[:fused]))
            assert_close(out[0], ref[0], dtype, f"want={want} v{v} fused={fused}")
    if keep_a:
        assert total > 0


def siblings_graph(B, S, K, N, dtype, chained=False):
    """gelu -> three MatMuls of the same input, each + bias (the Q, K, V
    projections), combined as (q * k) + v.  With chained the second product
    reads the first's output instead, so the two may not share a launch.
    Returns the graph, the product edges and the bias-Add edges."""
    g = Graph(dtype=dtype)
    x = g.add_input((B, S, K))
    a = g.add_node("gelu", [x], (B, S, K))
    prods, outs = [], []
    for i in range(3):
        src = outs[0] if (chained and i == 1) else a
        c = g.add_node("matmul", [src, g.add_const("weight", (K if src == a else N, N))], (B, S, N))
        prods.append(c)
        outs.append(g.add_node("add", [c, g.add_const("bias", (N,))], (B, S, N)))
    y = g.add_node("mul", [outs[0], outs[1]], (B, S, N))
    y = g.add_node("add", [y, outs[2]], (B, S, N))
    g.outputs = [y]
    return g, prods, outs


@pytest.mark.parametrize("shape", [(1, 37, 64, 64), (2, 130, 96, 96)], ids=str)
@pytest.mark.parametrize("variant", [6, 7])
@pytest.mark.parametrize("chained", [False, True])
def test_grouped_products(shape, variant, chained, tmp_path):
    """Sibling fp32 products launched as one grouped launch (each with its
    fused bias and its own output layout): same result as the oracle with
    the fused intermediates unrounded, and one launch for the group unless a
    member reads another's output."""
    from paper_2411_09242_amd import fluid as F
    og, prods, outs = siblings_graph(*shape, "f32", chained)
    L = layouts.layout_list(og.edge_shape(outs[0]))
    mms = [i for i, nd in enumerate(og.nodes) if nd.op == "matmul"]
    for lays in ((0, 0, 0), (1, 0, 1), (0, 1, 1)):
        want = {e: L[l] for e, l in zip(outs, lays)}
        say(f"grouped {shape} v{variant} chained={chained} {want}")
        xs, cs = random_inputs(og, sum(lays))
        try:
            out, lp, ap = run_device(og, forced_table(og, want, {m: variant for m in mms}), xs, cs, tmp_path,
                                     epilogue=True)
        except Exception as ex:  # noqa: BLE001
            # chained: the second product reads the first's output, which in
            # an M-contiguous layout with M % 4 != 0 no direct-load tile takes
            if chained and "cannot run with these layouts" in str(ex):
                continue
            raise
        nonview = sum(1 for x in lp.variant if x >= 0)
        n = F.fluid_run_launches(lp.graph.h, lp.h, ap.h)
        # three bias Adds fused; the products grouped into one launch (two
        # when the second reads the first: it then waits for it)
        assert n == nonview - 3 - (1 if chained else 2)
        ref = reference_rounding_except(og, xs, cs, set(prods))
        assert_close(out[0], ref[0], "f32", f"want={want} v{variant}")


def chain_attn_graph(B, NH, S, T, D, causal, extra_reader=False):
    """q = gelu, k = silu, v = gelu of three inputs; O = softmax(Q K^T / 8,
    causal) V, then gelu.  With extra_reader the scores are also an output
    (read by a second node)."""
    g = Graph(dtype="f32")
    xq = g.add_input((B, NH, S, D))
    xk = g.add_input((B, NH, D, T))
    xv = g.add_input((B, NH, T, D))
    q = g.add_node("gelu", [xq], (B, NH, S, D))
    k = g.add_node("silu", [xk], (B, NH, D, T))
    v = g.add_node("gelu", [xv], (B, NH, T, D))
    s = g.add_node("matmul", [q, k], (B, NH, S, T))
    p = g.add_node("softmax", [s], (B, NH, S, T), fattr=0.125, iattr=int(causal))
    o = g.add_node("matmul", [p, v], (B, NH, S, D))
    y = g.add_node("gelu", [o], (B, NH, S, D))
    g.outputs = [y]
    if extra_reader:
        g.outputs.append(g.add_node("silu", [s], (B, NH, S, T)))
    return g, q, k, v, s, p, o


def attn_graph(B, NH, S, D, dtype, pv=False):
    g = Graph(dtype=dtype)
    if not pv:
        x1 = g.add_input((B, NH, S, D))
        x2 = g.add_input((B, NH, D, S))
        out = (B, NH, S, S)
    else:
        x1 = g.add_input((B, NH, S, S))
        x2 = g.add_input((B, NH, S, D))
        out = (B, NH, S, D)
    q = g.add_node("gelu", [x1], g.edge_shape(x1))
    k = g.add_node("silu", [x2], g.edge_shape(x2))
    s = g.add_node("matmul", [q, k], out)
    y = g.add_node("gelu", [s], out)
    g.outputs = [y]
    return g, q, k, s


ATTN_SHAPES = [(1, 2, 37, 16), (2, 3, 64, 32), (1, 4, 130, 64)]


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("shape", ATTN_SHAPES, ids=str)
@pytest.mark.parametrize("pv", [False, True])
def test_attention_gemm_sampled_layouts(dtype, shape, pv, tmp_path):
    og, q, k, s = attn_graph(*shape, dtype, pv)
    Lq = layouts.layout_list(og.edge_shape(q))
    Lk = layouts.layout_list(og.edge_shape(k))
    Ls = layouts.layout_list(og.edge_shape(s))
    rng = np.random.default_rng(sum(shape) + pv)
    combos = list(itertools.product(range(len(Lq)), range(len(Lk)), range(len(Ls))))
    pick = [combos[0]] + [combos[i] for i in rng.choice(len(combos), size=min(10, len(combos)), replace=False)]
    for iq, ik, is_ in pick:
        for v in range(10):
            say(f"gemm attn {dtype} {shape} pv={pv} v{v} {Lq[iq]} {Lk[ik]} {Ls[is_]}")
            _check_gemm(og, {q: Lq[iq], k: Lk[ik], s: Ls[is_]}, {2: v}, tmp_path, iq + ik + is_, dtype)


def causal_attn_graph(B, NH, S, D, dtype):
    g = Graph(dtype=dtype)
    x1 = g.add_input((B, NH, S, D))
    x2 = g.add_input((B, NH, D, S))
    x3 = g.add_input((B, NH, S, D))
    q = g.add_node("gelu", [x1], (B, NH, S, D))
    k = g.add_node("silu", [x2], (B, NH, D, S))
    s = g.add_node("matmul", [q, k], (B, NH, S, S))
    p = g.add_node("softmax", [s], (B, NH, S, S), fattr=0.3, iattr=1)
    o = g.add_node("matmul", [p, x3], (B, NH, S, D))
    y = g.add_node("gelu", [o], (B, NH, S, D))
    g.outputs = [y]
    return g, q, k, s, p, o


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("shape", [(1, 2, 37, 16), (1, 2, 300, 64), (2, 1, 520, 32)], ids=str)
def test_causal_attention_skips(dtype, shape, tmp_path):
    """Q K^T read only by a causal softmax (tiles above the diagonal are
    skipped) and P V with P from it (K stops at the tile's last row), every
    GEMM variant on both, a few layouts of S and P: same output as the
    oracle's full products."""
    og, q, k, s, p, o = causal_attn_graph(*shape, dtype)
    Ls = layouts.layout_list(og.edge_shape(s))
    rng = np.random.default_rng(sum(shape))
    picks = [(0, 0)] + [tuple(int(v) for v in rng.integers(0, len(Ls), 2)) for _ in range(2)]
    for i_s, i_p in picks:
        for v in range(10):
            say(f"causal attn {dtype} {shape} v{v} S{Ls[i_s]} P{Ls[i_p]}")
            _check_gemm(og, {s: Ls[i_s], p: Ls[i_p]}, {2: v, 4: v}, tmp_path, i_s + i_p, dtype)


# ------------------------------------------------------------------ elementwise
def ew_graph(B, S, H, dtype):
    g = Graph(dtype=dtype)
    x = g.add_input((B, S, H))
    a = g.add_node("gelu", [x], (B, S, H))
    bias = g.add_const("bias", (H,))
    b = g.add_node("add", [a, bias], (B, S, H))
    c = g.add_node("add", [b, a], (B, S, H))
    d = g.add_node("mul", [c, a], (B, S, H))
    e = g.add_node("silu", [d], (B, S, H))
    g.outputs = [e]
    return g, [a, b, c, d]


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("shape", [(1, 33, 40), (2, 17, 24), (3, 64, 128), (2, 5, 7)], ids=str)
def test_elementwise_layouts(dtype, shape, tmp_path):
    og, edges = ew_graph(*shape, dtype)
    L = layouts.layout_list(shape)
    rng = np.random.default_rng(len(L) + shape[1])
    for trial in range(12):
        want = {e: L[int(rng.integers(0, len(L)))] for e in edges}
        if trial == 0:
            want = {e: L[0] for e in edges}
        for v in (0, 1):
            say(f"ew {dtype} {shape} gelu-v{v} {want}")
            try:
                _check(og, want, {0: v}, tmp_path, seed=trial)
            except Exception as ex:  # noqa: BLE001
                # the tiled variant needs differing unit-stride dims
                if v == 1 and "cannot run with these layouts" in str(ex):
                    continue
                raise


def relayout_graph(B, S, NH, D, dtype):
    g = Graph(dtype=dtype)
    x = g.add_input((B, S, NH * D))
    a = g.add_node("gelu", [x], (B, S, NH * D))
    r = g.add_node("reshape", [a], (B, S, NH, D))
    t = g.add_node("transpose", [r], (B, NH, S, D), perm=(0, 2, 1, 3))
    t2 = g.add_node("transpose", [t], (B, S, NH, D), perm=(0, 2, 1, 3))
    m = g.add_node("reshape", [t2], (B, S, NH * D))
    y = g.add_node("silu", [m], (B, S, NH * D))
    g.outputs = [y]
    return g, [a, r, t, t2, m]


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("shape", [(1, 37, 3, 16), (2, 70, 4, 32), (1, 130, 2, 64)], ids=str)
def test_transpose_reshape_copies_and_views(dtype, shape, tmp_path):
    og, edges = relayout_graph(*shape, dtype)
    Ls = [layouts.layout_list(og.edge_shape(e)) for e in edges]
    rng = np.random.default_rng(shape[1])
    for trial in range(16):
        want = {e: L[int(rng.integers(0, len(L)))] for e, L in zip(edges, Ls)}
        for v in (0, 1):
            var = {}
            for n in (1, 2, 3, 4):   # reshape, transpose, transpose, reshape
                var[n] = v
            # the tiled variant needs differing unit-stride dims; fall back to 0
            say(f"relayout {dtype} {shape} v{v} {want}")
            try:
                _check(og, want, var, tmp_path, seed=trial)
            except Exception as ex:  # noqa: BLE001
                if v == 1 and "cannot run with these layouts" in str(ex):
                    continue
                raise


# ------------------------------------------------------------------ reductions
def softmax_graph(B, NH, S, T, dtype, causal, scale):
    g = Graph(dtype=dtype)
    x = g.add_input((B, NH, S, T))
    a = g.add_node("gelu", [x], (B, NH, S, T))
    p = g.add_node("softmax", [a], (B, NH, S, T), fattr=scale, iattr=causal)
    y = g.add_node("silu", [p], (B, NH, S, T))
    g.outputs = [y]
    return g, a, p


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("shape", [(1, 2, 37, 37), (2, 3, 64, 64), (1, 2, 130, 130), (1, 1, 5, 300), (1, 1, 9, 1024)], ids=str)
@pytest.mark.parametrize("causal", [0, 1])
def test_softmax_layouts_and_variants(dtype, shape, causal, tmp_path):
    og, a, p = softmax_graph(*shape, dtype, causal, 0.125)
    L = layouts.layout_list(shape)
    rng = np.random.default_rng(shape[2] + causal)
    combos = [(0, 0)] + [tuple(int(v) for v in rng.integers(0, len(L), 2)) for _ in range(8)]
    for ia, ip in combos:
        for v in (0, 1, 2):
            if v == 2 and not row_block_ok(shape, dtype, L[ia], L[ip]):
                continue
            say(f"softmax {dtype} {shape} causal={causal} v{v} {L[ia]} {L[ip]}")
            _check(og, {a: L[ia], p: L[ip]}, {1: v}, tmp_path, seed=ia * 7 + ip, scale=3.0)


def norm_graph(B, S, H, dtype, op):
    g = Graph(dtype=dtype)
    x = g.add_input((B, S, H))
    a = g.add_node("gelu", [x], (B, S, H))
    gm = g.add_const("gamma", (H,))
    if op == "layernorm":
        bt = g.add_const("beta", (H,))
        n = g.add_node("layernorm", [a, gm, bt], (B, S, H), fattr=1e-5)
    else:
        n = g.add_node("rmsnorm", [a, gm], (B, S, H), fattr=1e-5)
    y = g.add_node("silu", [n], (B, S, H))
    g.outputs = [y]
    return g, a, n


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("op", ["layernorm", "rmsnorm"])
@pytest.mark.parametrize("shape", [(1, 37, 64), (2, 19, 130), (1, 8, 768), (2, 5, 1024), (1, 5, 3000), (1, 3, 4096),
                                   (2, 32, 96), (1, 48, 1024), (2, 8, 2048)], ids=str)
def test_norm_layouts_and_variants(dtype, op, shape, tmp_path):
    """Every pair of input / output layouts and every variant."""
    og, a, n = norm_graph(*shape, dtype, op)
    L = layouts.layout_list(shape)
    for ia, ib in itertools.product(range(len(L)), range(len(L))):
        for v in (0, 1, 2):
            if v == 2 and not row_block_ok(shape, dtype, L[ia], L[ib]):
                continue
            say(f"{op} {dtype} {shape} v{v} {L[ia]} {L[ib]}")
            _check(og, {a: L[ia], n: L[ib]}, {1: v}, tmp_path, seed=ia + 3 * ib, scale=2.0)


def sum_norm_graph(B, S, H, dtype, op, store=False):
    """x -> a = GELU(x), b = SiLU(x); s = a + b; n = norm(s); y = GELU(n):
    the residual Add (node 2) and its normalisation (node 3) form a chain.
    With store, y = GELU(n) + s: the sum has a second reader (the pre-norm
    residual), so the chain's launch stores it."""
    g = Graph(dtype=dtype)
    x = g.add_input((B, S, H))
    a = g.add_node("gelu", [x], (B, S, H))
    b = g.add_node("silu", [x], (B, S, H))
    sm = g.add_node("add", [a, b], (B, S, H))
    gm = g.add_const("gamma", (H,))
    if op == "layernorm":
        bt = g.add_const("beta", (H,))
        n = g.add_node("layernorm", [sm, gm, bt], (B, S, H), fattr=1e-5)
    else:
        n = g.add_node("rmsnorm", [sm, gm], (B, S, H), fattr=1e-5)
    y = g.add_node("gelu", [n], (B, S, H))
    if store:
        y = g.add_node("add", [y, sm], (B, S, H))
    g.outputs = [y]
    return g, a, b, sm, n


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("op", ["layernorm", "rmsnorm"])
@pytest.mark.parametrize("shape", [(1, 37, 64), (2, 19, 130), (1, 8, 768), (2, 5, 1024), (1, 3, 4096), (2, 32, 1024),
                                   (1, 8, 4096)], ids=str)
def test_residual_norm_one_launch(dtype, op, shape, tmp_path):
    """A residual Add and the LayerNorm / RMSNorm of its sum as one planned
    launch (a table that prices the chain below the two nodes): both
    summands and the output in many layouts, every reduction variant; the
    sum is never stored, so the oracle keeps it unrounded too."""
    og, a, b, sm, n = sum_norm_graph(*shape, dtype, op)
    L = layouts.layout_list(shape)
    combos = [(0, 0, 0)] + [(i, (5 * i + 1) % len(L), (2 * i + 3) % len(L)) for i in range(len(L))]
    for ia, ib, io in combos:
        for v in (0, 1, 2):
            if v == 2 and not row_block_ok(shape, dtype, L[ia], L[ib], L[io]):
                continue
            say(f"sum-{op} {dtype} {shape} v{v} {L[ia]} {L[ib]} -> {L[io]}")
            xs, cs = random_inputs(og, ia + 7 * ib + io, 2.0)
            (ref,) = execute.run_canonical(og, xs, cs, on_chip={sm})
            obj = forced_table(og, {a: L[ia], b: L[ib], n: L[io]}, {3: v})
            obj["fused_sigs"] = [{"op": "add", "in_shapes": [list(shape)] * 2, "out_shape": list(shape),
                                  "entries": [[[list(L[ia]), list(L[ib])], list(L[io]),
                                               [1 if w == v else -1 for w in range(3)]]]}]
            obj["fused"] = [[2, 1, 0]]
            (out,), lp, ap = run_device(og, obj, xs, cs, tmp_path)
            assert lp.fusion_priced and lp.fuse[2] == 1 and lp.variant[2] == v and lp.variant[3] == -2
            assert ap.offset[sm] == -1
            assert lp.kernel(2).startswith("add_" + op)
            assert_close(out, ref, dtype, f"sum-{op} v{v} {L[ia]} {L[ib]} {L[io]}")


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("op", ["layernorm", "rmsnorm"])
@pytest.mark.parametrize("shape", [(1, 37, 64), (2, 19, 130), (2, 5, 1024), (1, 3, 4096), (2, 32, 1024)], ids=str)
def test_stored_residual_norm_one_launch(dtype, op, shape, tmp_path):
    """The sum of a residual-norm chain with a second reader (a pre-norm
    block's next residual): the one launch also stores the sum, in the norm
    output's layout, and normalises the stored (rounded) values -- the
    oracle rounds the sum like any stored tensor."""
    og, a, b, sm, n = sum_norm_graph(*shape, dtype, op, store=True)
    L = layouts.layout_list(shape)
    combos = [(0, 0, 0)] + [(i, (5 * i + 1) % len(L), (2 * i + 3) % len(L)) for i in range(1, min(len(L), 4))]
    for ia, ib, io in combos:
        for v in (0, 1, 2):
            if v == 2 and not row_block_ok(shape, dtype, L[ia], L[ib], L[io]):
                continue
            say(f"stored sum-{op} {dtype} {shape} v{v} {L[ia]} {L[ib]} -> {L[io]}")
            xs, cs = random_inputs(og, ia + 7 * ib + io, 2.0)
            (ref,) = execute.run_canonical(og, xs, cs)
            obj = forced_table(og, {a: L[ia], b: L[ib], sm: L[io], n: L[io]}, {3: v})
            obj["fused_sigs"] = [{"op": "add", "in_shapes": [list(shape)] * 2, "out_shape": list(shape),
                                  "entries": [[[list(L[ia]), list(L[ib])], list(L[io]),
                                               [1 if w == v else -1 for w in range(3)]]]}]
            obj["fused"] = [[2, 1, 0]]
            (out,), lp, ap = run_device(og, obj, xs, cs, tmp_path)
            assert lp.fusion_priced and lp.fuse[2] == 1 and lp.variant[2] == v and lp.variant[3] == -2
            assert ap.offset[sm] >= 0 and lp.perm(sm) == lp.perm(n)
            assert lp.kernel(2).startswith("add_" + op)
            assert_close(out, ref, dtype, f"stored sum-{op} v{v} {L[ia]} {L[ib]} {L[io]}")


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("op", ["layernorm", "rmsnorm", "softmax"])
def test_column_reduction_many_rows(dtype, op, tmp_path):
    """More than 32704 short rows: the column variant's 64-row tiles (fewer
    rows take 16- or 8-row tiles), with a row length that leaves masked k."""
    if op == "softmax":
        shape = (1, 1, 32775, 40)
        L = layouts.layout_list(shape)
        for causal in (0, 1):
            og, a, n = softmax_graph(*shape, dtype, causal, 0.5)
            for ia, ib in ((0, 0), (1, 1), (0, 1)):
                say(f"{op} {dtype} {shape} causal={causal} v1 {L[ia]} {L[ib]}")
                _check(og, {a: L[ia], n: L[ib]}, {1: 1}, tmp_path, seed=ia + 3 * ib, scale=3.0)
        return
    shape = (1, 32775, 40)
    og, a, n = norm_graph(*shape, dtype, op)
    L = layouts.layout_list(shape)
    for ia, ib in ((0, 0), (1, 1), (0, 1), (1, 0)):
        say(f"{op} {dtype} {shape} v1 {L[ia]} {L[ib]}")
        _check(og, {a: L[ia], n: L[ib]}, {1: 1}, tmp_path, seed=ia + 3 * ib, scale=2.0)


# ------------------------------------------------------------------ RoPE
def rope_graph(B, S, NH, D, dtype):
    g = Graph(dtype=dtype)
    x = g.add_input((B, S, NH, D))
    a = g.add_node("gelu", [x], (B, S, NH, D))
    cc = g.add_const("rope_cos", (S, D // 2), "f32")
    ss = g.add_const("rope_sin", (S, D // 2), "f32")
    r = g.add_node("rope", [a, cc, ss], (B, S, NH, D))
    y = g.add_node("silu", [r], (B, S, NH, D))
    g.outputs = [y]
    return g, a, r


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("shape", [(1, 37, 3, 16), (2, 20, 2, 64), (1, 130, 4, 128)], ids=str)
def test_rope_layouts(dtype, shape, tmp_path):
    og, a, r = rope_graph(*shape, dtype)
    L = layouts.layout_list(shape)
    rng = np.random.default_rng(shape[1])
    combos = [(0, 0)] + [tuple(int(v) for v in rng.integers(0, len(L), 2)) for _ in range(8)]
    for ia, ir in combos:
        say(f"rope {dtype} {shape} {L[ia]} {L[ir]}")
        _check(og, {a: L[ia], r: L[ir]}, {}, tmp_path, seed=ia + ir)
