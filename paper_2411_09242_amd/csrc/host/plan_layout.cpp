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

#include "fusion.h"
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

  // G[a, b] = min over boundary layouts beta of C[slot layouts..., b] with
  // the chain edge ce in layout a; argmin beta lexicographically smallest.
  Gain gain(const std::vector<int>& slots, int ce, const std::vector<int>& be, int eo, const NodeCost& nc,
            const std::vector<int64_t>& C, const Fix& F) const {
    Gain r;
    r.be = be;
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

  Gain node_gain(const PathInfo& info, size_t j, const Fix& F) const {
    const int n = info.path[j];
    const auto& slots = g.act_in[n];
    const int cs = info.chain_slot[j];
    return gain(slots, cs >= 0 ? slots[cs] : -1, info.bnd[j], g.out_edge(n), t.nodes[n], costs(n), F);
  }

  // chain lengths t with measured costs whose nodes m+1 .. m+t follow the
  // MatMul at step j on this path
  std::vector<int> fused_options(const PathInfo& info, size_t j) const {
    std::vector<int> out;
    const int m = info.path[j];
    for (int tt = 1; tt <= 3; ++tt) {
      if (!t.fused.count({m, tt}) || j + tt >= info.path.size()) continue;
      bool ok = true;
      for (int i = 1; i <= tt; ++i) ok = ok && info.path[j + i] == m + i;
      if (ok) out.push_back(tt);
    }
    return out;
  }

  // The index in L(e_store) of the permutation L(e_out)[b] -- the layout a
  // chain's stored intermediate takes when the chain's output takes b --
  // or -1 when e_store has no such candidate.
  int store_index(int e_store, int e_out, int b) const {
    const auto& ls = t.L[e_store];
    auto it = std::find(ls.begin(), ls.end(), t.L[e_out][b]);
    return it == ls.end() ? -1 : (int)(it - ls.begin());
  }

  // whether every intermediate the chain (m, tt) stores has the layout of
  // the chain's output under lay
  bool chain_layouts_ok(int m, int tt, const std::vector<int>& lay) const {
    const int eo = g.out_edge(m + tt);
    for (int e : stored_edges(g, m, tt))
      if (lay[e] != store_index(e, eo, lay[eo])) return false;
    return true;
  }

  // the fused launch of steps j .. j+tt as one virtual node; an output
  // layout b that a stored intermediate cannot take (no such candidate, or
  // fixed otherwise) is infeasible
  Gain fused_gain(const PathInfo& info, size_t j, int tt, const Fix& F) const {
    const int m = info.path[j];
    const std::vector<int> slots = chain_slots(g, m, tt);
    const int cs = info.chain_slot[j];
    const int ce = cs >= 0 ? g.act_in[m][cs] : -1;
    std::vector<int> be;
    for (int e : slots)
      if (e != ce && std::find(be.begin(), be.end(), e) == be.end()) be.push_back(e);
    const NodeCost& nc = t.fused.at({m, tt});
    const int eo = g.out_edge(m + tt);
    Gain r = gain(slots, ce, be, eo, nc, use_v0 ? nc.v0 : nc.best, F);
    for (int e : stored_edges(g, m, tt))
      for (int b = 0; b < r.Bn; ++b) {
        const int k = store_index(e, eo, b);
        auto it = F.find(e);
        if (k >= 0 && (it == F.end() || it->second == k)) continue;
        for (int a = 0; a < r.A; ++a) {
          r.G[(size_t)a * r.Bn + b] = kInf;
          r.arg[(size_t)a * r.Bn + b] = -1;
        }
      }
    return r;
  }

  struct DP {
    int64_t total = kInf;
    std::vector<int> states;
    std::vector<std::map<int, int>> betas;
    std::vector<int> fused;  // per step: length of the fused chain starting there
  };

  // Viterbi over one path; with fusion priced, a step's output layout is
  // also reached by the fused launch of the chain ending there, from the
  // layout of the step before the chain (ties: the node on its own, then
  // the shorter chain, then the smaller predecessor layout).
  DP dp_path(const PathInfo& info, const Fix& F, bool fuse) const {
    const size_t m = info.path.size();
    struct Cand {
      int tt;
      size_t s;
      Gain gn;
    };
    std::vector<std::vector<int>> opts(m);
    if (fuse)
      for (size_t j = 0; j < m; ++j) opts[j] = fused_options(info, j);
    std::vector<std::vector<std::pair<int, int>>> backs(m);  // (t, a)
    std::vector<std::vector<Cand>> cands(m);
    std::vector<std::vector<int64_t>> Vs(m);
    for (size_t j = 0; j < m; ++j) {
      const int eo = g.out_edge(info.path[j]);
      cands[j].push_back({0, j, node_gain(info, j, F)});
      for (int s = (int)j - 1; s >= std::max(0, (int)j - 3); --s) {
        const int tt = (int)j - s;
        if (std::find(opts[s].begin(), opts[s].end(), tt) != opts[s].end())
          cands[j].push_back({tt, (size_t)s, fused_gain(info, (size_t)s, tt, F)});
      }
      const int Bn = (int)t.L[eo].size();
      std::vector<char> ok(Bn, 0);
      for (int b : allowed(F, eo)) ok[b] = 1;
      std::vector<int64_t> Vn(Bn, kInf);
      std::vector<std::pair<int, int>> back(Bn, {0, 0});
      for (const Cand& c : cands[j]) {
        const Gain& gn = c.gn;
        for (int b = 0; b < Bn; ++b) {
          int64_t tot;
          int ba = 0;
          if (c.s == 0) {
            tot = ok[b] ? gn.G[b] : kInf;
          } else {
            int64_t best = kInf + 1;  // so that an all-INF column keeps a = 0
            const auto& V = Vs[c.s - 1];
            for (int a = 0; a < gn.A; ++a) {
              int64_t gab = ok[b] ? gn.G[(size_t)a * gn.Bn + b] : kInf;
              int64_t v = sat_add(V[a], gab);
              if (v < best) { best = v; ba = a; }
            }
            tot = best > kInf ? kInf : best;
          }
          // the node on its own always sets the state; a fused launch
          // replaces it only when strictly cheaper
          if (c.tt == 0 || tot < Vn[b]) { Vn[b] = tot; back[b] = {c.tt, ba}; }
        }
      }
      backs[j] = std::move(back);
      Vs[j] = std::move(Vn);
    }
    DP r;
    const auto& V = Vs[m - 1];
    int b = 0;
    int64_t best = kInf + 1;
    for (int i = 0; i < (int)V.size(); ++i)
      if (V[i] < best) { best = V[i]; b = i; }
    r.total = best > kInf ? kInf : best;
    r.states.assign(m, 0);
    r.fused.assign(m, 0);
    r.betas.assign(m, {});
    for (int j = (int)m - 1; j >= 0;) {
      const auto [tt, a] = backs[j][b];
      const Cand* c = nullptr;
      for (const Cand& x : cands[j])
        if (x.tt == tt) c = &x;
      const Gain& gn = c->gn;
      const int s = (int)c->s;
      r.states[j] = b;
      const int bi = gn.arg[(size_t)(s > 0 ? a : 0) * gn.Bn + b];
      std::map<int, int> chosen;
      for (size_t i = 0; i < gn.be.size(); ++i) chosen[gn.be[i]] = bi >= 0 ? gn.betas[bi][i] : 0;
      if (s > 0) chosen.emplace(g.act_in[info.path[s]][info.chain_slot[s]], a);
      // a boundary edge's layout is recorded at every step of the launch
      // that reads it as a boundary edge
      for (int k = s; k <= j; ++k)
        for (int e : info.bnd[k]) {
          auto it = chosen.find(e);
          if (it != chosen.end()) r.betas[k][e] = it->second;
        }
      if (tt) {  // an intermediate the launch stores takes the output's layout
        const int m0 = info.path[s];
        for (int e : stored_edges(g, m0, tt))
          r.states[s + (g.producer(e) - m0)] = store_index(e, g.out_edge(m0 + tt), b);
      }
      r.fused[s] = tt;
      j = s - 1;
      b = a;
    }
    return r;
  }

  // flat index of (slot layouts..., out layout) into a dense cost array
  static size_t flat_of(const NodeCost& nc, const std::vector<int>& slots, int eo, const std::vector<int>& lay) {
    size_t flat = 0;
    for (size_t s = 0; s < slots.size(); ++s) flat = flat * nc.dims[s] + lay[slots[s]];
    return flat * nc.dims[slots.size()] + lay[eo];
  }

  // summed table cost: every node on its own, except the fused chains
  // (fuse[m] = t), which cost their fused entry
  int64_t plan_cost(const std::vector<int>& lay, const std::vector<int>& fuse = {}) const {
    int64_t total = 0;
    for (int n = 0; n < g.n_nodes();) {
      const int tt = fuse.empty() ? 0 : fuse[n];
      if (tt) {
        const NodeCost& nc = t.fused.at({n, tt});
        const auto& C = use_v0 ? nc.v0 : nc.best;
        total = sat_add(total, chain_layouts_ok(n, tt, lay)
                                   ? C[flat_of(nc, chain_slots(g, n, tt), g.out_edge(n + tt), lay)]
                                   : kInf);
        n += tt + 1;
        continue;
      }
      total = sat_add(total, costs(n)[flat_of(t.nodes[n], g.act_in[n], g.out_edge(n), lay)]);
      ++n;
    }
    return total;
  }

  // The cheapest set of disjoint fusion chains for fixed layouts (fuse[m] =
  // t for a chain run as one launch): chains cover consecutive node ids, so
  // an interval DP from the last node back -- f(n) = min(n on its own +
  // f(n+1), min over chains (n, t) of their fused entry + f(n+t+1)); ties
  // keep the node on its own, then the shorter chain.
  std::vector<int> best_chains(const std::vector<int>& lay) const {
    const int N = g.n_nodes();
    std::vector<int64_t> f(N + 1, 0);
    std::vector<int> pick(N, 0);
    for (int n = N - 1; n >= 0; --n) {
      f[n] = sat_add(costs(n)[flat_of(t.nodes[n], g.act_in[n], g.out_edge(n), lay)], f[n + 1]);
      for (int tt = 1;; ++tt) {
        auto it = t.fused.find({n, tt});
        if (it == t.fused.end()) break;
        if (!chain_layouts_ok(n, tt, lay)) continue;
        const NodeCost& nc = it->second;
        const auto& C = use_v0 ? nc.v0 : nc.best;
        const int64_t c = sat_add(C[flat_of(nc, chain_slots(g, n, tt), g.out_edge(n + tt), lay)], f[n + tt + 1]);
        if (c < f[n]) { f[n] = c; pick[n] = tt; }
      }
    }
    std::vector<int> fuse(N, 0);
    for (int n = 0; n < N; n += pick[n] + 1) fuse[n] = pick[n];
    return fuse;
  }

  LayoutPlan finish(const std::vector<int>& lay, int64_t total, int guard, const std::vector<std::vector<int>>& paths,
                    const std::vector<int>& fuse = {}) const {
    LayoutPlan p;
    p.layout_idx = lay;
    p.total = total;
    p.guard_used = guard;
    p.paths = paths;
    p.fuse = fuse.empty() ? std::vector<int>(g.n_nodes(), 0) : fuse;
    std::vector<char> absorbed(g.n_nodes(), 0);
    for (int m = 0; m < g.n_nodes(); ++m)
      for (int i = 1; i <= p.fuse[m]; ++i) absorbed[m + i] = 1;
    for (int e = 0; e < g.n_edges(); ++e) p.perm.push_back(t.L[e][lay[e]]);
    for (int n = 0; n < g.n_nodes(); ++n) {
      if (absorbed[n]) { p.variant.push_back(-2); continue; }
      if (node_is_view(g, n, p.perm)) { p.variant.push_back(-1); continue; }
      if (use_v0) { p.variant.push_back(0); continue; }
      if (p.fuse[n]) {
        const NodeCost& nc = t.fused.at({n, p.fuse[n]});
        p.variant.push_back(nc.var[flat_of(nc, chain_slots(g, n, p.fuse[n]), g.out_edge(n + p.fuse[n]), lay)]);
        continue;
      }
      p.variant.push_back(t.nodes[n].var[flat_of(t.nodes[n], g.act_in[n], g.out_edge(n), lay)]);
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
  LayoutPlan p = plan_layouts_dp(g, t, flags);
  p.fusion_priced = !(flags & FLUID_NO_FUSION) && !(flags & FLUID_NO_DP) && !t.fused.empty();
  return p;
}

namespace {

// The first DP of every path, the vote on shared edges and the
// re-optimisation with the voted layouts fixed: the layout index per edge;
// false when a path has no feasible plan after the vote.
bool voted_layouts(const Graph& g, const Planner& P, const std::vector<std::vector<int>>& paths,
                   const std::vector<PathInfo>& infos, bool fz, std::vector<int>& lay) {
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
    first.push_back(P.dp_path(infos[pi], F, fz));
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
        for (int pi : touch) c = sat_add(c, P.dp_path(infos[pi], F2, fz).total);
        if (best < 0 || c < best) { best = c; win = l; }
      }
    }
    F[e] = win;
  }
  lay.assign(g.n_edges(), 0);
  for (size_t pi = 0; pi < infos.size(); ++pi) {
    Planner::DP d = P.dp_path(infos[pi], F, fz);
    if (d.total >= kInf) return false;
    for (size_t j = 0; j < infos[pi].path.size(); ++j) lay[g.out_edge(infos[pi].path[j])] = d.states[j];
  }
  return true;
}

}  // namespace

// Sections 3.1-3.3 (Alg. 1-3, Eq. 1, the vote), with the row-major guard;
// when the table prices fusion chains, two voted layout assignments compete
// (from the fusion-aware path DP and from the plain one), each with the
// cheapest chains for its layouts (Planner::best_chains); the cheaper total
// wins, the fusion-aware one on ties.
LayoutPlan plan_layouts_dp(const Graph& g, const CostTable& t, uint32_t flags) {
  Planner P{g, t, (flags & FLUID_NO_VARIANTS) != 0};
  const bool priced = !(flags & FLUID_NO_FUSION) && !t.fused.empty();
  auto paths = split_paths(g);
  std::vector<int> ident(g.n_edges(), 0);
  if (P.plan_cost(ident) >= kInf) fail(FLUID_E_INFEASIBLE, "the all-row-major plan has no cost entry");
  if (flags & FLUID_NO_DP) return P.finish(ident, P.plan_cost(ident), 0, paths);
  const std::vector<int> ident_fuse = priced ? P.best_chains(ident) : std::vector<int>{};
  const int64_t ident_cost = P.plan_cost(ident, ident_fuse);

  std::vector<PathInfo> infos;
  for (auto& p : paths) infos.push_back(make_info(g, p));
  bool have = false;
  int64_t total = 0;
  std::vector<int> lay, fuse;
  for (bool fz : priced ? std::vector<bool>{true, false} : std::vector<bool>{false}) {
    std::vector<int> l;
    if (!voted_layouts(g, P, paths, infos, fz, l)) continue;
    std::vector<int> f = priced ? P.best_chains(l) : std::vector<int>{};
    const int64_t c = P.plan_cost(l, f);
    if (!have || c < total) {
      have = true;
      total = c;
      lay = std::move(l);
      fuse = std::move(f);
    }
  }
  if (!have) {
    if (flags & FLUID_NO_GUARD) fail(FLUID_E_INFEASIBLE, "every path plan is infeasible after the vote");
    return P.finish(ident, ident_cost, 1, paths, ident_fuse);
  }
  if (!(flags & FLUID_NO_GUARD) && total > ident_cost) return P.finish(ident, ident_cost, 1, paths, ident_fuse);
  return P.finish(lay, total, 0, paths, fuse);
}

LayoutPlan identity_plan(const Graph& g) {
  LayoutPlan p;
  p.layout_idx.assign(g.n_edges(), 0);
  for (int e = 0; e < g.n_edges(); ++e) p.perm.push_back(identity_perm((int)g.edge_shape(e).size()));
  for (int n = 0; n < g.n_nodes(); ++n) p.variant.push_back(node_is_view(g, n, p.perm) ? -1 : 0);
  p.fuse.assign(g.n_nodes(), 0);
  return p;
}

}  // namespace fluid
