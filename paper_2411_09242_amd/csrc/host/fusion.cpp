#include "fusion.h"

#include <algorithm>

namespace fluid {

namespace {

// Add m of two activations followed by the normalisation of its sum.
std::vector<ChainStep> norm_chain(const Graph& g, int m) {
  const Node& nd = g.nodes[m];
  if (nd.ins.size() != 2 || nd.ins[0] < 0 || nd.ins[1] < 0 || nd.ins[0] == nd.ins[1]) return {};
  for (int e : nd.ins)
    if (g.edge_shape(e) != nd.out_shape) return {};
  const int cur = g.out_edge(m), n = m + 1;
  const auto& rd = g.readers[cur];
  if (n >= g.n_nodes() || g.is_output[cur] || std::find(rd.begin(), rd.end(), n) == rd.end()) return {};
  const Node& x = g.nodes[n];
  if ((x.op != FLUID_OP_LAYERNORM && x.op != FLUID_OP_RMSNORM) || x.ins[0] != cur) return {};
  for (size_t i = 1; i < x.ins.size(); ++i)
    if (x.ins[i] >= 0) return {};
  const bool alone = std::all_of(rd.begin(), rd.end(), [&](int r) { return r == n; });
  return {{n, alone ? CH_NORM : CH_NORM_STORE, -1, -1}};
}

}  // namespace

std::vector<ChainStep> chain_steps(const Graph& g, int m) {
  std::vector<ChainStep> steps;
  const Node& nd = g.nodes[m];
  if (nd.op == FLUID_OP_ADD) return norm_chain(g, m);
  if (nd.op != FLUID_OP_MATMUL || nd.ins.size() != 2) return steps;
  const Shape& out_shape = nd.out_shape;
  int cur = g.out_edge(m);
  bool act = false;
  for (int i = 1; i <= 3; ++i) {
    const int n = m + i;
    if (n >= g.n_nodes() || g.is_output[cur] || g.readers[cur].size() != 1 || g.readers[cur][0] != n) break;
    const Node& x = g.nodes[n];
    if ((x.op == FLUID_OP_ADD || x.op == FLUID_OP_MUL) && x.ins.size() == 2) {
      const int slot = x.ins[0] == cur ? 0 : 1;
      const int other = x.ins[1 - slot];
      if (other == cur) break;
      if (other < 0) {
        const Const& c = g.consts[~other];
        if (x.op != FLUID_OP_ADD || !steps.empty() || c.shape != Shape({out_shape.back()}) || c.dtype != g.dtype)
          break;
        steps.push_back({n, CH_BIAS, -1, ~other});
      } else {
        const int p = g.producer(other);
        if (g.edge_shape(other) != out_shape || (p >= 0 && p >= m)) break;
        steps.push_back({n, x.op == FLUID_OP_ADD ? CH_ADD_R : CH_MUL_R, other, -1});
        break;
      }
    } else if ((x.op == FLUID_OP_GELU || x.op == FLUID_OP_SILU) && !act) {
      act = true;
      steps.push_back({n, CH_ACT, -1, -1});
    } else {
      break;
    }
    cur = g.out_edge(n);
  }
  return steps;
}

std::vector<int> stored_edges(const Graph& g, int m, int t) {
  const auto steps = chain_steps(g, m);
  if (t >= 1 && !steps.empty() && steps[0].kind == CH_NORM_STORE) return {g.out_edge(m)};
  return {};
}

std::vector<int> on_chip_edges(const Graph& g, int m, int t) {
  const std::vector<int> st = stored_edges(g, m, t);
  std::vector<int> out;
  for (int i = 0; i < t; ++i) {
    const int e = g.out_edge(m + i);
    if (std::find(st.begin(), st.end(), e) == st.end()) out.push_back(e);
  }
  return out;
}

std::vector<int> chain_slots(const Graph& g, int m, int t) {
  std::vector<int> slots = g.act_in[m];
  const auto steps = chain_steps(g, m);
  if (t >= 1 && t <= (int)steps.size() && steps[t - 1].r >= 0) slots.push_back(steps[t - 1].r);
  return slots;
}

}  // namespace fluid
