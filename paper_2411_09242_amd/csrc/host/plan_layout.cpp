// Layout planner: Section 3, Alg. 1 (longest sequence), Alg. 2 (recursive
// extraction), Eq. 1 / Alg. 3 (dynamic programming on a sequence over
// measured kernel times) and the majority-vote conflict resolution.
//
// Readings of the points the paper leaves open (every tie is deterministic
// so that independent implementations agree exactly):
//  * Alg. 1's walk "recording the longest distance" is a longest path over
//    the DAG in topological order; a node's predecessor is the producer of
//    its first input slot that attains the distance; the path ends at the
//    smallest node id of maximal distance.
//  * Alg. 2 recurses fully; components are visited by smallest node id.
//  * Eq. 1: the state of step j is the layout b of the step's output; the
//    minimum runs over the chain predecessor's layout a; inputs produced on
//    other paths ("boundary" inputs) are minimised inside the node's cost,
//    lexicographically smallest choice on ties; back-pointers keep the
//    smallest a, and the trace-back starts at the smallest cheapest b.
//  * Vote: per shared edge, in edge order, one ballot per touching path;
//    vote ties (random in the paper) go to the layout whose re-optimised
//    touching paths cost least, then the smallest index; the winner is fixed
//    before the next edge.  Then every path is re-optimised once with all
//    shared edges fixed.  Guard: the row-major plan if it is cheaper.
#include <algorithm>
#include <map>
#include <numeric>

#include "layouts.h"
#include "planner.h"

namespace fluid {

std::vector<int> longest_path(const Graph& g, const std::vector<int>& S) {
  std::vector<char> in(g.n_nodes(), 0);
  for (int n : S) in[n] = 1;
  std::vector<int> dist(g.n_nodes(), 0), pred(g.n_nodes(), -1);
  std::vector<int> order = S;
  std::sort(order.begin(), order.end());
  int top = 0;
  for (int n : order) {
    int best = 0, bp = -1;
    for (int e : g.act_in[n]) {
      int p = g.producer(e);
      if (p >= 0 && in[p] && dist[p] > best) { best = dist[p]; bp = p; }
    }
    // first slot attaining the maximum
    if (bp >= 0) {
      for (int e : g.act_in[n]) {
        int p = g.producer(e);
        if (p >= 0 && in[p] && dist[p] == best) { bp = p; break; }
      }
    }
    dist[n] = best + 1;
    pred[n] = bp;
    top = std::max(top, dist[n]);
  }
  int end = -1;
  for (int n : order)
    if (dist[n] == top) { end = n; break; }
  std::vector<int> path;
  for (int n = end; n >= 0; n = pred[n]) path.push_back(n);
  std::reverse(path.begin(), path.end());
  return path;
}

namespace {

void split_rec(const Graph& g, std::vector<int> S, std::vector<std::vector<int>>& out) {
  if (S.empty()) return;
  std::sort(S.begin(), S.end());
  std::vector<int> P = longest_path(g, S);
  std::vector<char> onp(g.n_nodes(), 0), inR(g.n_nodes(), 0);
  for (int n : P) onp[n] = 1;
  std::vector<int> R;
  for (int n : S)
    if (!onp[n]) { R.push_back(n); inR[n] = 1; }
  out.push_back(P);
  // weakly connected components of R (union-find, root = smallest id)
  std::vector<int> parent(g.n_nodes());
  std::iota(parent.begin(), parent.end(), 0);
  auto find = [&](int x) {
    while (parent[x] != x) { parent[x] = parent[parent[x]]; x = parent[x]; }
    return x;
  };
  for (int n : R)
    for (int e : g.act_in[n]) {
      int p = g.producer(e);
      if (p >= 0 && inR[p]) {
        int a = find(n), b = find(p);
        if (a != b) parent[std::max(a, b)] = std::min(a, b);
      }
    }
  std::map<int, std::vector<int>> comps;
  for (int n : R) comps[find(n)].push_back(n);
  std::vector<std::vector<int>> cs;
  for (auto& kv : comps) cs.push_back(kv.second);
  std::sort(cs.begin(), cs.end(), [](const std::vector<int>& a, const std::vector<int>& b) { return a[0] < b[0]; });
  for (auto& c : cs) split_rec(g, c, out);
}

struct PathInfo {
  std::vector<int> path;
  std::vector<int> chain_slot;             // -1 at step 0
  std::vector<std::vector<int>> bnd;       // distinct boundary edges by first slot
};

PathInfo make_info(const Graph& g, const std::vector<int>& path) {
  PathInfo in;
  in.path = path;
  for (size_t j = 0; j < path.size(); ++j) {
    const auto& slots = g.act_in[path[j]];
    int cs = -1;
    if (j > 0)
      for (size_t s = 0; s < slots.size(); ++s)
        if (g.producer(slots[s]) == path[j - 1]) { cs = (int)s; break; }
    const int ce = cs >= 0 ? slots[cs] : -1;
    std::vector<int> be;
    for (size_t s = 0; s < slots.size(); ++s) {
      if ((int)s == cs || slots[s] == ce) continue;
      if (std::find(be.begin(), be.end(), slots[s]) == be.end()) be.push_back(slots[s]);
    }
    in.chain_slot.push_back(cs);
    in.bnd.push_back(std::move(be));
  }
  return in;
}

using Fix = std::map<int, int>;

struct Planner {
  const Graph& g;
  const CostTable& t;
  bool use_v0;

  const std::vector<int64_t>& costs(int n) const { return use_v0 ? t.nodes[n].v0 : t.nodes[n].best; }

  std::vector<int> allowed(const Fix& F, int e) const {
    auto it = F.find(e);
    if (it != F.end()) return {it->second};
    std::vector<int> v(t.L[e].size());
    std::iota(v.begin(), v.end(), 0);
    return v;
  }

  struct Gain {
    int A = 1, Bn = 0;
    std::vector<int64_t> G;                 // [A][Bn]
    std::vector<int> arg;                   // beta index
    std::vector<std::vector<int>> betas;    // lexicographic
    std::vector<int> be;
  };

  Gain node_gain(const PathInfo& info, size_t j, const Fix& F) const {
    Gain r;
    const int n = info.path[j];
    const auto& slots = g.act_in[n];
    const NodeCost& nc = t.nodes[n];
    const auto& C = costs(n);
    const int cs = info.chain_slot[j];
    const int ce = cs >= 0 ? slots[cs] : -1;
    r.be = info.bnd[j];
    const int eo = g.out_edge(n);
    r.A = ce >= 0 ? (int)t.L[ce].size() : 1;
    r.Bn = (int)t.L[eo].size();
    r.G.assign((size_t)r.A * r.Bn, kInf);
    r.arg.assign((size_t)r.A * r.Bn, -1);
    // strides of the dense array: slots then out (last, stride 1)
    const int k = (int)slots.size();
    std::vector<int64_t> stride(k + 1, 1);
    for (int i = k - 1; i >= 0; --i) stride[i] = stride[i + 1] * nc.dims[i + 1];
    int64_t chain_stride = 0;
    for (int s = 0; s < k; ++s)
      if (ce >= 0 && slots[s] == ce) chain_stride += stride[s];
    // enumerate beta lexicographically
    std::vector<std::vector<int>> al;
    for (int e : r.be) al.push_back(allowed(F, e));
    std::vector<size_t> cur(al.size(), 0);
    bool done = false;
    for (const auto& a : al)
      if (a.empty()) done = true;
    while (!done) {
      std::vector<int> beta(al.size());
      for (size_t i = 0; i < al.size(); ++i) beta[i] = al[i][cur[i]];
      int64_t base = 0;
      for (int s = 0; s < k; ++s) {
        if (ce >= 0 && slots[s] == ce) continue;
        size_t bi = std::find(r.be.begin(), r.be.end(), slots[s]) - r.be.begin();
        base += (int64_t)beta[bi] * stride[s];
      }
      const int bidx = (int)r.betas.size();
      r.betas.push_back(beta);
      for (int a = 0; a < r.A; ++a)
        for (int b = 0; b < r.Bn; ++b) {
          int64_t c = C[(size_t)(base + a * chain_stride + b)];
          size_t o = (size_t)a * r.Bn + b;
          if (c < r.G[o]) { r.G[o] = c; r.arg[o] = bidx; }
        }
      // next beta (last index fastest)
      int i = (int)al.size() - 1;
      for (; i >= 0; --i) {
        if (++cur[i] < al[i].size()) break;
        cur[i] = 0;
      }
      if (i < 0) done = true;
    }
    return r;
  }

  struct DP {
    int64_t total = kInf;
    std::vector<int> states;
    std::vector<std::map<int, int>> betas;
  };

  DP dp_path(const PathInfo& info, const Fix& F) const {
    const size_t m = info.path.size();
    std::vector<std::vector<int>> backs(m);
    std::vector<Gain> gains(m);
    std::vector<int64_t> V;
    for (size_t j = 0; j < m; ++j) {
      const int n = info.path[j];
      const int eo = g.out_edge(n);
      gains[j] = node_gain(info, j, F);
      Gain& gn = gains[j];
      std::vector<char> ok(gn.Bn, 0);
      for (int b : allowed(F, eo)) ok[b] = 1;
      std::vector<int64_t> Vn(gn.Bn, kInf);
      std::vector<int> back(gn.Bn, -1);
      for (int b = 0; b < gn.Bn; ++b) {
        if (j == 0) {
          Vn[b] = ok[b] ? gn.G[b] : kInf;
          continue;
        }
        int64_t best = kInf + 1;  // so that an all-INF column keeps a = 0
        int ba = 0;
        for (int a = 0; a < gn.A; ++a) {
          int64_t gab = ok[b] ? gn.G[(size_t)a * gn.Bn + b] : kInf;
          int64_t v = sat_add(V[a], gab);
          if (v < best) { best = v; ba = a; }
        }
        Vn[b] = best > kInf ? kInf : best;
        back[b] = ba;
      }
      backs[j] = std::move(back);
      V = std::move(Vn);
    }
    DP r;
    int b = 0;
    int64_t best = kInf + 1;
    for (int i = 0; i < (int)V.size(); ++i)
      if (V[i] < best) { best = V[i]; b = i; }
    r.total = best > kInf ? kInf : best;
    r.states.assign(m, 0);
    std::vector<int> chosen_a(m, 0);
    for (int j = (int)m - 1; j >= 0; --j) {
      r.states[j] = b;
      int a = j > 0 ? backs[j][b] : 0;
      chosen_a[j] = a;
      b = a;
    }
    r.betas.resize(m);
    for (size_t j = 0; j < m; ++j) {
      const Gain& gn = gains[j];
      int bi = gn.arg[(size_t)(j > 0 ? chosen_a[j] : 0) * gn.Bn + r.states[j]];
      for (size_t i = 0; i < gn.be.size(); ++i) r.betas[j][gn.be[i]] = bi >= 0 ? gn.betas[bi][i] : 0;
    }
    return r;
  }

  int64_t plan_cost(const std::vector<int>& lay) const {
    int64_t total = 0;
    for (int n = 0; n < g.n_nodes(); ++n) {
      const NodeCost& nc = t.nodes[n];
      size_t flat = 0;
      const auto& slots = g.act_in[n];
      for (size_t s = 0; s < slots.size(); ++s) flat = flat * nc.dims[s] + lay[slots[s]];
      flat = flat * nc.dims[slots.size()] + lay[g.out_edge(n)];
      total = sat_add(total, costs(n)[flat]);
    }
    return total;
  }

  LayoutPlan finish(const std::vector<int>& lay, int64_t total, int guard, const std::vector<std::vector<int>>& paths) const {
    LayoutPlan p;
    p.layout_idx = lay;
    p.total = total;
    p.guard_used = guard;
    p.paths = paths;
    for (int e = 0; e < g.n_edges(); ++e) p.perm.push_back(t.L[e][lay[e]]);
    for (int n = 0; n < g.n_nodes(); ++n) {
      if (node_is_view(g, n, p.perm)) { p.variant.push_back(-1); continue; }
      if (use_v0) { p.variant.push_back(0); continue; }
      const NodeCost& nc = t.nodes[n];
      size_t flat = 0;
      const auto& slots = g.act_in[n];
      for (size_t s = 0; s < slots.size(); ++s) flat = flat * nc.dims[s] + lay[slots[s]];
      flat = flat * nc.dims[slots.size()] + lay[g.out_edge(n)];
      p.variant.push_back(nc.var[flat]);
    }
    return p;
  }
};

}  // namespace

std::vector<std::vector<int>> split_paths(const Graph& g) {
  std::vector<int> all(g.n_nodes());
  std::iota(all.begin(), all.end(), 0);
  std::vector<std::vector<int>> out;
  split_rec(g, all, out);
  return out;
}

LayoutPlan plan_layouts(const Graph& g, const CostTable& t, uint32_t flags) {
  Planner P{g, t, (flags & FLUID_NO_VARIANTS) != 0};
  auto paths = split_paths(g);
  std::vector<int> ident(g.n_edges(), 0);
  const int64_t ident_cost = P.plan_cost(ident);
  if (ident_cost >= kInf) fail(FLUID_E_INFEASIBLE, "the all-row-major plan has no cost entry");
  if (flags & FLUID_NO_DP) return P.finish(ident, ident_cost, 0, paths);

  std::vector<PathInfo> infos;
  for (auto& p : paths) infos.push_back(make_info(g, p));
  std::vector<int> owner(g.n_edges(), -1), step_of(g.n_nodes(), -1);
  for (size_t pi = 0; pi < paths.size(); ++pi)
    for (size_t j = 0; j < paths[pi].size(); ++j) {
      owner[g.out_edge(paths[pi][j])] = (int)pi;
      step_of[paths[pi][j]] = (int)j;
    }
  // readers[e]: path -> lowest step reading e in a boundary slot
  std::map<int, std::map<int, int>> readers;
  for (size_t pi = 0; pi < infos.size(); ++pi)
    for (size_t j = 0; j < infos[pi].bnd.size(); ++j)
      for (int e : infos[pi].bnd[j]) {
        auto& m = readers[e];
        if (!m.count((int)pi)) m[(int)pi] = (int)j;
      }

  Fix F;
  std::vector<Planner::DP> first;
  for (size_t pi = 0; pi < infos.size(); ++pi) {
    first.push_back(P.dp_path(infos[pi], F));
    if (first.back().total >= kInf) fail(FLUID_E_INFEASIBLE, "path " + std::to_string(pi) + " has no feasible layout");
  }
  for (auto& kv : readers) {
    const int e = kv.first;
    if (g.pinned(e)) continue;
    std::vector<int> ballots, touch;
    if (owner[e] >= 0) {
      const int po = owner[e];
      ballots.push_back(first[po].states[step_of[g.producer(e)]]);
      touch.push_back(po);
    }
    for (auto& rv : kv.second) {
      if (rv.first == owner[e]) continue;
      ballots.push_back(first[rv.first].betas[rv.second].at(e));
      touch.push_back(rv.first);
    }
    std::map<int, int> counts;
    for (int b : ballots) counts[b]++;
    int top = 0;
    for (auto& c : counts) top = std::max(top, c.second);
    std::vector<int> tied;
    for (auto& c : counts)
      if (c.second == top) tied.push_back(c.first);  // ascending (map order)
    int win = tied[0];
    if (tied.size() > 1) {
      int64_t best = -1;
      for (int l : tied) {
        Fix F2 = F;
        F2[e] = l;
        int64_t c = 0;
        for (int pi : touch) c = sat_add(c, P.dp_path(infos[pi], F2).total);
        if (best < 0 || c < best) { best = c; win = l; }
      }
    }
    F[e] = win;
  }
  std::vector<int> lay(ident);
  for (size_t pi = 0; pi < infos.size(); ++pi) {
    Planner::DP d = P.dp_path(infos[pi], F);
    if (d.total >= kInf) {
      if (flags & FLUID_NO_GUARD) fail(FLUID_E_INFEASIBLE, "path " + std::to_string(pi) + " infeasible after the vote");
      return P.finish(ident, ident_cost, 1, paths);
    }
    for (size_t j = 0; j < infos[pi].path.size(); ++j) lay[g.out_edge(infos[pi].path[j])] = d.states[j];
  }
  const int64_t total = P.plan_cost(lay);
  if (!(flags & FLUID_NO_GUARD) && total > ident_cost) return P.finish(ident, ident_cost, 1, paths);
  return P.finish(lay, total, 0, paths);
}

LayoutPlan identity_plan(const Graph& g) {
  LayoutPlan p;
  p.layout_idx.assign(g.n_edges(), 0);
  for (int e = 0; e < g.n_edges(); ++e) p.perm.push_back(identity_perm((int)g.edge_shape(e).size()));
  for (int n = 0; n < g.n_nodes(); ++n) p.variant.push_back(node_is_view(g, n, p.perm) ? -1 : 0);
  return p;
}

}  // namespace fluid
