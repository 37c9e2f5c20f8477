#include "costtable.h"
#include "fusion.h"

#include <algorithm>
#include <map>
#include <sstream>

#include "layouts.h"

namespace fluid {

namespace {

int op_from_name(const std::string& s) {
  for (int op = 0; op <= FLUID_OP_MAXPOOL; ++op)
    if (s == op_name(op)) return op;
  fail(FLUID_E_INVALID, "cost table: unknown op '" + s + "'");
}

Perm perm_of(const Json& j) {
  Perm p;
  for (const Json& v : j.arr()) p.push_back((int)v.as_int());
  return p;
}

Shape shape_of(const Json& j) {
  Shape s;
  for (const Json& v : j.arr()) s.push_back(v.as_int());
  return s;
}

bool valid_perm(const Perm& p, size_t rank) {
  if (p.size() != rank) return false;
  std::vector<int> seen(rank, 0);
  for (int d : p) {
    if (d < 0 || d >= (int)rank || seen[d]) return false;
    seen[d] = 1;
  }
  return true;
}

}  // namespace

CostTable cost_table_from_json(const Json& j) {
  CostTable t;
  if (j.at("format").kind != Json::Str || j.at("format").s != "fluid-cost-table/1")
    fail(FLUID_E_INVALID, "cost table: format must be \"fluid-cost-table/1\"");
  for (const Json& lst : j.at("edges").arr()) {
    std::vector<Perm> ls;
    for (const Json& p : lst.arr()) ls.push_back(perm_of(p));
    t.L.push_back(std::move(ls));
  }
  auto parse_sig = [&](const Json& sj) {
    Sig s;
    s.op = op_from_name(sj.at("op").s);
    if (sj.has("in_shapes"))
      for (const Json& x : sj.at("in_shapes").arr()) s.in_shapes.push_back(shape_of(x));
    if (sj.has("out_shape")) s.out_shape = shape_of(sj.at("out_shape"));
    for (const Json& ej : sj.at("entries").arr()) {
      const auto& a = ej.arr();
      require(a.size() == 3, "cost table: entry must be [slot perms, out perm, costs]");
      SigEntry e;
      for (const Json& p : a[0].arr()) e.in.push_back(perm_of(p));
      e.out = perm_of(a[1]);
      for (const Json& c : a[2].arr()) e.costs.push_back(c.as_int());
      s.entries.push_back(std::move(e));
    }
    return s;
  };
  for (const Json& sj : j.at("sigs").arr()) t.sigs.push_back(parse_sig(sj));
  if (j.has("fused_sigs"))
    for (const Json& sj : j.at("fused_sigs").arr()) t.fused_sigs.push_back(parse_sig(sj));
  if (j.has("fused"))
    for (const Json& f : j.at("fused").arr()) {
      const auto& a = f.arr();
      require(a.size() == 3, "cost table: a fused reference is [m, t, signature]");
      t.fused_refs.push_back({(int)a[0].as_int(), (int)a[1].as_int(), (int)a[2].as_int()});
    }
  for (const Json& v : j.at("node_sig").arr()) t.node_sig.push_back((int)v.as_int());
  return t;
}

void CostTable::bind(const Graph& g) {
  const int E = g.n_edges();
  require((int)L.size() == E, "cost table: has " + std::to_string(L.size()) + " edges, graph has " + std::to_string(E));
  for (int e = 0; e < E; ++e) {
    const size_t r = g.edge_shape(e).size();
    require(!L[e].empty() && L[e][0] == identity_perm((int)r),
            "cost table: L(" + std::to_string(e) + ") must start with the identity layout");
    for (const Perm& p : L[e]) require(valid_perm(p, r), "cost table: bad layout for edge " + std::to_string(e));
    std::vector<Perm> sorted = L[e];
    std::sort(sorted.begin(), sorted.end());
    require(std::adjacent_find(sorted.begin(), sorted.end()) == sorted.end(), "cost table: duplicate layout");
    if (g.pinned(e)) require(L[e].size() == 1, "cost table: graph input/output edges must be row-major only");
  }
  require((int)node_sig.size() == g.n_nodes(), "cost table: node count mismatch");
  // dense costs over (slot layout index..., out layout index)
  auto dense = [&](const std::vector<int>& slots, int eo, const Sig& s, const std::string& what, const Node* nd) {
    NodeCost nc;
    std::vector<std::map<Perm, int>> index;
    for (size_t i = 0; i <= slots.size(); ++i) {
      const int e = i < slots.size() ? slots[i] : eo;
      nc.dims.push_back((int)L[e].size());
      std::map<Perm, int> m;
      for (size_t k = 0; k < L[e].size(); ++k) m[L[e][k]] = (int)k;
      index.push_back(std::move(m));
    }
    size_t total = 1;
    for (int d : nc.dims) total *= (size_t)d;
    nc.best.assign(total, kInf);
    nc.var.assign(total, -1);
    nc.v0.assign(total, kInf);
    for (const SigEntry& en : s.entries) {
      require(en.in.size() == slots.size(), "cost table: " + what + " entry arity");
      size_t flat = 0;
      bool ok = true;
      for (size_t i = 0; i <= slots.size() && ok; ++i) {
        const Perm& p = i < slots.size() ? en.in[i] : en.out;
        auto it = index[i].find(p);
        if (it == index[i].end()) { ok = false; break; }
        flat = flat * nc.dims[i] + it->second;
      }
      if (!ok) continue;  // a layout outside this node's candidates
      if (nd && (nd->op == FLUID_OP_TRANSPOSE || nd->op == FLUID_OP_RESHAPE)) {
        if (is_view(nd->op, nd->perm, g.edge_shape(slots[0]), nd->out_shape, en.in[0], en.out))
          for (int64_t c : en.costs) require(c <= 0, "cost table: " + what + ": a view combination must cost 0");
      }
      int64_t best = kInf;
      int var = -1;
      for (size_t v = 0; v < en.costs.size(); ++v) {
        int64_t c = en.costs[v];
        if (c >= 0 && c < best) { best = std::min(c, kInf); var = (int)v; }
      }
      nc.best[flat] = best;
      nc.var[flat] = var;
      nc.v0[flat] = (!en.costs.empty() && en.costs[0] >= 0) ? std::min(en.costs[0], kInf) : kInf;
    }
    return nc;
  };
  nodes.assign(g.n_nodes(), {});
  for (int n = 0; n < g.n_nodes(); ++n) {
    const int si = node_sig[n];
    require(si >= 0 && si < (int)sigs.size(), "cost table: bad signature index");
    const Sig& s = sigs[si];
    const Node& nd = g.nodes[n];
    const auto& slots = g.act_in[n];
    require(s.op == nd.op, "cost table: node " + std::to_string(n) + " op mismatch");
    if (!s.in_shapes.empty()) {
      require(s.in_shapes.size() == slots.size(), "cost table: node " + std::to_string(n) + " slot count");
      for (size_t i = 0; i < slots.size(); ++i)
        require(s.in_shapes[i] == g.edge_shape(slots[i]), "cost table: node " + std::to_string(n) + " input shape");
    }
    if (!s.out_shape.empty()) require(s.out_shape == nd.out_shape, "cost table: node " + std::to_string(n) + " output shape");
    nodes[n] = dense(slots, g.out_edge(n), s, "node " + std::to_string(n), &nd);
  }
  fused.clear();
  for (const FusedRef& f : fused_refs) {
    const std::string what = "chain (" + std::to_string(f.m) + ", " + std::to_string(f.t) + ")";
    require(f.m >= 0 && f.m < g.n_nodes() && f.t >= 1 && f.t <= (int)chain_steps(g, f.m).size(),
            "cost table: " + what + " is not a fusion chain of this graph");
    require(f.sig >= 0 && f.sig < (int)fused_sigs.size(), "cost table: bad fused signature index");
    require(!fused.count({f.m, f.t}), "cost table: " + what + " listed twice");
    fused[{f.m, f.t}] = dense(chain_slots(g, f.m, f.t), g.out_edge(f.m + f.t), fused_sigs[f.sig], what, nullptr);
  }
  graph_serial = 0;
}

std::string cost_table_to_json(const CostTable& t) {
  std::ostringstream o;
  auto perm = [&](const Perm& p) {
    o << '[';
    for (size_t i = 0; i < p.size(); ++i) o << (i ? "," : "") << p[i];
    o << ']';
  };
  o << "{\"format\": \"fluid-cost-table/1\",\n\"edges\": [";
  for (size_t e = 0; e < t.L.size(); ++e) {
    o << (e ? ",\n" : "") << '[';
    for (size_t i = 0; i < t.L[e].size(); ++i) { if (i) o << ','; perm(t.L[e][i]); }
    o << ']';
  }
  auto write_sigs = [&](const std::vector<Sig>& sigs) {
    for (size_t si = 0; si < sigs.size(); ++si) {
      const Sig& s = sigs[si];
      o << (si ? ",\n" : "") << "{\"op\": \"" << op_name(s.op) << "\", \"in_shapes\": [";
      for (size_t i = 0; i < s.in_shapes.size(); ++i) {
        if (i) o << ',';
        o << '[';
        for (size_t k = 0; k < s.in_shapes[i].size(); ++k) o << (k ? "," : "") << s.in_shapes[i][k];
        o << ']';
      }
      o << "], \"out_shape\": [";
      for (size_t k = 0; k < s.out_shape.size(); ++k) o << (k ? "," : "") << s.out_shape[k];
      o << "], \"entries\": [";
      for (size_t k = 0; k < s.entries.size(); ++k) {
        const SigEntry& en = s.entries[k];
        o << (k ? ",\n" : "") << "[[";
        for (size_t i = 0; i < en.in.size(); ++i) { if (i) o << ','; perm(en.in[i]); }
        o << "],";
        perm(en.out);
        o << ",[";
        for (size_t i = 0; i < en.costs.size(); ++i) o << (i ? "," : "") << en.costs[i];
        o << "]]";
      }
      o << "]}";
    }
  };
  o << "],\n\"sigs\": [";
  write_sigs(t.sigs);
  o << "],\n\"node_sig\": [";
  for (size_t n = 0; n < t.node_sig.size(); ++n) o << (n ? "," : "") << t.node_sig[n];
  o << "]";
  if (!t.fused_refs.empty()) {
    o << ",\n\"fused_sigs\": [";
    write_sigs(t.fused_sigs);
    o << "],\n\"fused\": [";
    for (size_t i = 0; i < t.fused_refs.size(); ++i)
      o << (i ? "," : "") << '[' << t.fused_refs[i].m << ',' << t.fused_refs[i].t << ',' << t.fused_refs[i].sig << ']';
    o << "]";
  }
  o << "}\n";
  return o.str();
}

}  // namespace fluid
