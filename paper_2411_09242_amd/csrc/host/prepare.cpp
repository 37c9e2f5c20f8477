#include "prepare.h"

#include <algorithm>
#include <string>

#include "fusion.h"
#include "handles.h"
#include "layouts.h"

namespace fluid {

namespace {

// Bases are validated to be 256-byte (arena) or 16-byte (caller tensors)
// aligned, so preparing with base address 0 keeps every alignment decision
// valid for the real addresses.
const void* fake_ptr(const Bind& b) { return (const void*)(uintptr_t)(b.off < 0 ? 0 : b.off); }

Bind bind_edge(const Graph& g, const ArenaPlan* ap, int e) {
  Bind b;
  const int r = ap ? ap->root[e] : e;
  if (r < g.n_inputs()) {
    b.kind = BK_INPUT;
    b.index = r;
  } else if (g.is_output[r]) {
    b.kind = BK_OUTPUT;
    b.index = (int)(std::find(g.outputs.begin(), g.outputs.end(), r) - g.outputs.begin());
  } else {
    b.kind = BK_ARENA;
    b.off = ap ? ap->offset[e] : 0;
  }
  return b;
}

// Bytes [lo, hi) an arena-bound edge occupies (empty for caller tensors and
// for results a planned fused launch keeps on chip, offset -1).
std::pair<int64_t, int64_t> arena_range(const Graph& g, const ArenaPlan* ap, int e, const Bind& b) {
  if (!ap || b.kind != BK_ARENA || b.off < 0) return {0, 0};
  const int64_t bytes = numel(g.edge_shape(e)) * (g.dtype == FLUID_BF16 ? 2 : 4);
  return {b.off, b.off + bytes};
}

}  // namespace

NodeKernel fused_gemm_kernel(const Node& mn, int variant, int dtype, const std::vector<Operand>& mm_ops,
                             const Operand& out, uint32_t act, uint32_t rop, const Operand* r) {
  NodeKernel kf = prepare_node(mn, variant, dtype, mm_ops, out);
  if (!kf.available) return kf;
  const int caps = gemm_epilogue_caps(variant, dtype);
  if ((act && !(caps & EPI_ACT)) || (rop && !(caps & EPI_ROP))) {
    kf.available = false;
    kf.why = "this tile does not perform that epilogue";
    return kf;
  }
  if (rop) {
    // R's strides in the output's batch / row decomposition: prepare the
    // product as if it wrote R
    const NodeKernel kr = prepare_node(mn, variant, dtype, mm_ops, *r);
    if (!kr.available) {
      kf.available = false;
      kf.why = kr.why;
      return kf;
    }
    kf.gemm.r_g1 = kr.gemm.c_g1;
    kf.gemm.r_g2 = kr.gemm.c_g2;
    kf.gemm.r_m1 = kr.gemm.c_m1;
    kf.gemm.r_m2 = kr.gemm.c_m2;
    kf.gemm.r_n = kr.gemm.c_n;
    kf.gemm.r_m2div = kf.gemm.m2div;
  }
  kf.gemm.epi_bf16 = dtype == FLUID_BF16 ? 1u : 0u;
  kf.gemm.act = act;
  kf.gemm.rop = rop;
  return kf;
}

namespace {

// Epilogue fusion.  A MatMul absorbs the node `nx` launched right after the
// chain it already performs when nx is the chain output's only reader (which
// is no graph output) and is, in this order of steps: an Add of a bias
// constant [N] (first step only), a GELU / SiLU, or an Add / Mul of the chain
// output and another activation tensor R of the same shape (the last step).
// The MatMul is then re-prepared to write nx's output, in nx's output layout,
// with every step applied in fp32 before the one rounding.  Not when nx's
// output shares arena bytes with a MatMul operand: that output only becomes
// live after the MatMul has read its operands, so the arena may have placed
// it over them.  R is produced before the MatMul (the chain's intermediates
// have no other reader, so R is none of them) and is live, and not written,
// until nx; nx's output never shares bytes with R, both being live at nx.
// `tail` is the output edge of the chain's last node.
void try_fuse_epilogue(const Graph& g, const LayoutPlan& lp, const ArenaPlan* ap, PreparedNode& mm, int tail,
                       PreparedNode& nx, const Operand& nx_out) {
  if (mm.k.family != KF_GEMM || mm.fused_away || (mm.fuse_n && mm.kf.family != KF_GEMM)) return;
  const Node& xn = g.nodes[nx.node];
  const Node& mn = g.nodes[mm.node];
  const uint32_t act_now = mm.fuse_n ? mm.kf.gemm.act : 0u;
  const uint32_t rop_now = mm.fuse_n ? mm.kf.gemm.rop : 0u;
  const int caps = gemm_epilogue_caps(lp.variant[mm.node], g.dtype);
  if (mn.ins.size() != 2 || rop_now) return;
  if (g.is_output[tail] || g.readers[tail].size() != 1 || g.readers[tail][0] != nx.node) return;
  int bias = mm.fbias;
  uint32_t act = act_now, rop = 0;
  int rslot = -1;
  if ((xn.op == FLUID_OP_ADD || xn.op == FLUID_OP_MUL) && xn.ins.size() == 2) {
    const int slot = xn.ins[0] == tail ? 0 : 1;
    const int o = xn.ins[1 - slot];
    if (o == tail) return;
    if (o < 0) {
      const int c = ~o;
      const Shape& cs = g.consts[c].shape;
      if (xn.op != FLUID_OP_ADD || mm.fuse_n != 0 || cs.size() != 1 || cs[0] != mn.out_shape.back() ||
          g.consts[c].dtype != g.dtype)
        return;
      bias = c;
    } else {
      if (g.edge_shape(o) != mn.out_shape || !(caps & EPI_ROP)) return;
      rop = xn.op == FLUID_OP_ADD ? 1u : 2u;
      rslot = 1 - slot;
    }
  } else if ((xn.op == FLUID_OP_GELU || xn.op == FLUID_OP_SILU) && act_now == 0 && (caps & EPI_ACT)) {
    act = xn.op == FLUID_OP_GELU ? 1u : 2u;
  } else {
    return;
  }
  const auto ro = arena_range(g, ap, g.out_edge(nx.node), nx.out);
  for (int i = 0; i < 2; ++i) {
    if (mn.ins[i] < 0) continue;
    const auto ri = arena_range(g, ap, mn.ins[i], mm.in[i]);
    if (ro.first < ro.second && ri.first < ri.second && ro.first < ri.second && ri.first < ro.second) return;
  }
  NodeKernel kf = fused_gemm_kernel(mn, lp.variant[mm.node], g.dtype, mm.ops, nx_out, act, rop,
                                    rop ? &nx.ops[rslot] : nullptr);
  if (!kf.available) return;
  if (rop) {
    mm.fr = nx.in[rslot];
    mm.fr_edge = xn.ins[rslot];
  }
  // a placeholder until each run binds the constant (fused_kernel): the
  // launch's name shows the bias step
  if (bias >= 0) kf.gemm.bias = (const void*)(uintptr_t)256;
  mm.fuse_n += 1;
  mm.kf = kf;
  mm.fout = nx.out;
  mm.fbias = bias;
  nx.fused_away = true;
}

// A planned residual-norm chain: the normalisation nx of the sum that the
// Add h forms, run as one reduction over h's two operands (the sum never
// stored; nx's output lies apart from both operands in the arena, the
// chain's lifetimes keeping them live until nx).
void fuse_norm(const Graph& g, const LayoutPlan& lp, PreparedNode& h, PreparedNode& nx, const Operand& nx_out) {
  const Node& xn = g.nodes[nx.node];
  std::vector<Operand> ops = nx.ops;
  ops[0] = h.ops[0];
  NodeKernel kf = prepare_sum_norm(xn, lp.variant[h.node], g.dtype, ops, h.ops[1], nx_out);
  if (!kf.available) return;
  // a sum with further readers is stored with the normalisation's offsets:
  // the plan gives it the layout of the normalisation's output
  const bool store = !stored_edges(g, h.node, 1).empty();
  if (store && dense_strides(g.nodes[h.node].out_shape, lp.perm[g.out_edge(h.node)]) != nx_out.stride) return;
  h.fstore = store;
  h.kf = kf;
  h.fuse_n = 1;
  h.fout = nx.out;
  h.fgamma = xn.ins.size() > 1 ? ~xn.ins[1] : -1;
  h.fbeta = xn.ins.size() > 2 ? ~xn.ins[2] : -1;
  nx.fused_away = true;
}

// The output edge and binding a prepared launch writes.
int written_edge(const Graph& g, const Prepared& P, size_t i) {
  return g.out_edge(P.nodes[i + P.nodes[i].fuse_n].node);
}
const Bind& written_bind(const Prepared& P, size_t i) {
  return P.nodes[i].fuse_n ? P.nodes[i].fout : P.nodes[i].out;
}

// Whether two bindings may share bytes: arena ranges that intersect, or the
// same caller tensor.
bool may_alias(const Graph& g, const ArenaPlan* ap, int e1, const Bind& b1, int e2, const Bind& b2) {
  if (b1.kind == BK_ARENA && b2.kind == BK_ARENA) {
    const auto r1 = arena_range(g, ap, e1, b1), r2 = arena_range(g, ap, e2, b2);
    return r1.first < r2.second && r2.first < r1.second;
  }
  return b1.kind == b2.kind && b1.kind != BK_CONST && b1.index == b2.index;
}

// Activation operands (edge, binding) a prepared launch reads.
std::vector<std::pair<int, Bind>> read_operands(const Graph& g, const Prepared& P, size_t i) {
  const PreparedNode& pn = P.nodes[i];
  std::vector<std::pair<int, Bind>> r;
  const Node& nd = g.nodes[pn.node];
  for (size_t s = 0; s < nd.ins.size(); ++s)
    if (nd.ins[s] >= 0) r.push_back({nd.ins[s], pn.in[s]});
  if (pn.fr_edge >= 0) r.push_back({pn.fr_edge, pn.fr});
  return r;
}

// Grouped launches.  Consecutive launches of fp32 products with the same
// direct-load tile (6 or 7), operand modes and epilogue instance -- the Q,
// K and V projections of a layer once their bias Adds are fused and their
// head reshapes are views -- go out as one launch when none reads or
// overwrites what another writes (they run concurrently).
void group_launches(const Graph& g, const ArenaPlan* ap, Prepared& P) {
  auto kern = [&](size_t i) -> const NodeKernel& { return P.nodes[i].fuse_n ? P.nodes[i].kf : P.nodes[i].k; };
  auto eligible = [&](size_t i) {
    const NodeKernel& k = kern(i);
    return !P.nodes[i].fused_away && k.family == KF_GEMM && k.dtype == DT_F32 &&
           (k.gemm_tile == 6 || k.gemm_tile == 7);
  };
  auto next_launch = [&](size_t i) {
    size_t j = i + 1;
    while (j < P.nodes.size() && P.nodes[j].fused_away) ++j;
    return j;
  };
  for (size_t i = 0; i < P.nodes.size(); i = next_launch(i)) {
    if (!eligible(i)) continue;
    std::vector<size_t> mem = {i};
    for (size_t j = next_launch(i); j < P.nodes.size() && mem.size() < (size_t)kMaxGroup; j = next_launch(j)) {
      const NodeKernel &a = kern(i), &b = kern(j);
      if (!eligible(j) || b.gemm_tile != a.gemm_tile || b.amode != a.amode || b.bmode != a.bmode ||
          (b.gemm.rop != 0) != (a.gemm.rop != 0))
        break;
      bool indep = true;
      for (size_t m : mem) {
        const int we = written_edge(g, P, j), wm = written_edge(g, P, m);
        if (may_alias(g, ap, we, written_bind(P, j), wm, written_bind(P, m))) indep = false;
        for (const auto& [e, bd] : read_operands(g, P, j))
          if (may_alias(g, ap, e, bd, wm, written_bind(P, m))) indep = false;
        for (const auto& [e, bd] : read_operands(g, P, m))
          if (may_alias(g, ap, e, bd, we, written_bind(P, j))) indep = false;
      }
      if (!indep) break;
      mem.push_back(j);
    }
    if (mem.size() < 2) continue;
    for (size_t t = 1; t < mem.size(); ++t) {
      P.nodes[i].group.push_back((int)mem[t]);
      P.nodes[mem[t]].grouped = true;
    }
    i = mem.back();
  }
}

}  // namespace

std::shared_ptr<Prepared> prepare(const Graph& g, const LayoutPlan& lp, const ArenaPlan* ap) {
  auto P = std::make_shared<Prepared>();
  for (int n = 0; n < g.n_nodes(); ++n) {
    const int v = lp.variant[n];
    if (v == -1) continue;  // view: no kernel
    const Node& nd = g.nodes[n];
    PreparedNode pn;
    pn.node = n;
    if (v >= 0 && packs_weight(nd.op, v) && nd.ins.size() == 2 && nd.ins[1] < 0 &&
        g.const_readers[~nd.ins[1]].size() != 1)
      fail(FLUID_E_INVALID, "node " + std::to_string(n) + ": a packed-weight variant needs a weight read by this "
                                                          "node only");
    std::vector<Operand> ins;
    for (size_t slot = 0; slot < nd.ins.size(); ++slot) {
      const int vin = nd.ins[slot];
      Operand o;
      Bind b;
      if (vin >= 0) {
        b = bind_edge(g, ap, vin);
        o.shape = g.edge_shape(vin);
        o.stride = dense_strides(o.shape, lp.perm[vin]);
        o.dtype = g.dtype;
      } else {
        b.kind = BK_CONST;
        b.index = ~vin;
        o.shape = g.consts[~vin].shape;
        o.stride = const_strides(nd, (int)slot, v >= 0 ? v : 0, o.shape);
        o.dtype = g.consts[~vin].dtype;
      }
      o.ptr = fake_ptr(b);
      ins.push_back(o);
      pn.in.push_back(b);
    }
    const int eo = g.out_edge(n);
    pn.out = bind_edge(g, ap, eo);
    Operand out;
    out.shape = nd.out_shape;
    out.stride = dense_strides(out.shape, lp.perm[eo]);
    out.dtype = g.dtype;
    out.ptr = fake_ptr(pn.out);
    pn.ops = ins;
    if (lp.fusion_priced && lp.fuse[n] > 0 && nd.op == FLUID_OP_ADD) {
      // heads a residual-norm chain: variant v is the normalisation's, and
      // the sum is formed in its launch (fuse_norm)
      pn.k.why = "performed in the launch of the normalisation after it";
      P->nodes.push_back(std::move(pn));
      continue;
    }
    if (v == -2) {
      // performed by the fused MatMul before it (the plan priced that launch)
      size_t j = P->nodes.empty() ? 0 : P->nodes.size() - 1;
      while (j > 0 && P->nodes[j].fused_away) --j;
      require(!P->nodes.empty() && j + P->nodes[j].fuse_n == P->nodes.size() - 1 &&
                  lp.fuse[P->nodes[j].node] >= n - P->nodes[j].node,
              "node " + std::to_string(n) + ": marked fused, but no fused MatMul launch precedes it");
      if (g.nodes[P->nodes[j].node].op == FLUID_OP_ADD)
        fuse_norm(g, lp, P->nodes[j], pn, out);
      else
        try_fuse_epilogue(g, lp, ap, P->nodes[j], g.out_edge(P->nodes.back().node), pn, out);
      require(pn.fused_away, "node " + std::to_string(n) + ": the plan fuses it into node " +
                                 std::to_string(P->nodes[j].node) + ", which cannot perform it with variant " +
                                 std::to_string(lp.variant[P->nodes[j].node]));
      P->nodes.push_back(std::move(pn));
      continue;
    }
    pn.k = prepare_node(nd, v, g.dtype, ins, out);
    if (!pn.k.available)
      fail(FLUID_E_INVALID, "node " + std::to_string(n) + ": variant " + std::to_string(v) +
                                " cannot run with these layouts (" + pn.k.why + ")");
    if (!lp.fusion_priced && !P->nodes.empty()) {
      // the MatMul whose fused chain ends at the previous launch, if any
      size_t j = P->nodes.size() - 1;
      while (j > 0 && P->nodes[j].fused_away) --j;
      if (j + P->nodes[j].fuse_n == P->nodes.size() - 1)
        try_fuse_epilogue(g, lp, ap, P->nodes[j], g.out_edge(P->nodes.back().node), pn, out);
    }
    P->nodes.push_back(std::move(pn));
  }
  if (ap) group_launches(g, ap, *P);
  return P;
}

std::vector<int> epilogue_reads_until(const Graph& g, const LayoutPlan& lp) {
  std::vector<int> until(g.n_nodes());
  for (int n = 0; n < g.n_nodes(); ++n) until[n] = n;
  const auto P = prepare(g, lp, nullptr);
  for (size_t i = 0; i < P->nodes.size(); ++i)
    if (P->nodes[i].fuse_n > 0) until[P->nodes[i].node] = P->nodes[i + P->nodes[i].fuse_n].node;
  return until;
}

Perm constant_layout(const Graph& g, const LayoutPlan& lp, int c) {
  const auto& rd = g.const_readers[c];
  if (rd.size() == 1) {
    const Node& nd = g.nodes[rd[0]];
    if (packs_weight(nd.op, lp.variant[rd[0]]) && nd.ins.size() == 2 && nd.ins[1] == ~c) return {1, 0};
  }
  return identity_perm((int)g.consts[c].shape.size());
}

int prepared_launches(const Prepared& P) {
  int n = 0;
  for (const PreparedNode& pn : P.nodes) n += (pn.fused_away || pn.grouped) ? 0 : 1;
  return n;
}

}  // namespace fluid
