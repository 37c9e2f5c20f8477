// Host-side entry points of the C ABI (graph, cost table, planners).
#include <algorithm>
#include <atomic>
#include <memory>
#include <cstring>
#include <fstream>
#include <sstream>

#include "fluid.h"
#include "handles.h"
#include "dispatch.h"
#include "layouts.h"
#include "prepare.h"

namespace fluid {

namespace {
thread_local std::string g_last_error;
std::atomic<uint64_t> g_serial{1};
}  // namespace

void set_last_error(const std::string& msg) { g_last_error = msg; }
uint64_t next_serial() { return g_serial.fetch_add(1); }

uint64_t measure_scratch_bytes(const Graph& g) {
  uint64_t best = 0;
  const uint64_t isz = (uint64_t)dtype_bytes(g.dtype);
  for (int n = 0; n < g.n_nodes(); ++n) {
    uint64_t s = 0;
    for (int v : g.nodes[n].ins) {
      const Shape& sh = v >= 0 ? g.edge_shape(v) : g.consts[~v].shape;
      const uint64_t b = v >= 0 ? isz : (uint64_t)dtype_bytes(g.consts[~v].dtype);
      s += (uint64_t)numel(sh) * b + 256;
    }
    s += (uint64_t)numel(g.nodes[n].out_shape) * isz + 256;
    // a fused launch also reads R (the output's shape) and a bias [N], or
    // (a residual Add and its normalisation) the norm's constants and
    // writes a second output (a stored sum)
    if (g.nodes[n].op == FLUID_OP_MATMUL)
      s += (uint64_t)numel(g.nodes[n].out_shape) * isz + 256 + (uint64_t)g.nodes[n].out_shape.back() * isz + 256;
    if (g.nodes[n].op == FLUID_OP_ADD && n + 1 < g.n_nodes()) {
      for (int v : g.nodes[n + 1].ins)
        if (v < 0) s += (uint64_t)numel(g.consts[~v].shape) * dtype_bytes(g.consts[~v].dtype) + 256;
      s += (uint64_t)numel(g.nodes[n].out_shape) * isz + 256;
    }
    // the copies of a constant weight the timed launches rotate over
    const Node& nd = g.nodes[n];
    if ((nd.op == FLUID_OP_MATMUL || nd.op == FLUID_OP_CONV) && nd.ins.size() > 1 && nd.ins[1] < 0) {
      const Const& w = g.consts[~nd.ins[1]];
      const uint64_t wb = (uint64_t)numel(w.shape) * dtype_bytes(w.dtype);
      s += (uint64_t)(cold_weight_copies(wb) - 1) * ((wb + 255) & ~uint64_t(255)) + 256;
    }
    best = std::max(best, s);
  }
  return best;
}

}  // namespace fluid

using namespace fluid;

extern "C" {

const char* fluid_last_error(void) { return g_last_error.c_str(); }

fluid_status fluid_build_graph(const fluid_graph_desc* d, fluid_graph** out) {
  return call_guarded([&] {
    require(d && out, "fluid_build_graph: NULL argument");
    auto h = std::make_unique<fluid_graph>();
    Graph& g = h->g;
    g.dtype = d->dtype;
    require(d->n_inputs >= 0 && d->n_consts >= 0 && d->n_nodes >= 0 && d->n_outputs >= 0, "negative count");
    require(d->n_inputs == 0 || (d->input_rank && d->input_shapes), "NULL input shape arrays");
    require(d->n_consts == 0 || (d->const_rank && d->const_shapes && d->const_dtype), "NULL const arrays");
    require(d->n_nodes == 0 || d->nodes, "NULL node array");
    require(d->n_outputs == 0 || d->output_edges, "NULL output array");
    for (int i = 0; i < d->n_inputs; ++i) {
      int r = d->input_rank[i];
      require(r >= 1 && r <= FLUID_MAX_RANK, "input rank out of range");
      g.inputs.emplace_back(d->input_shapes + (size_t)i * FLUID_MAX_RANK, d->input_shapes + (size_t)i * FLUID_MAX_RANK + r);
    }
    for (int i = 0; i < d->n_consts; ++i) {
      int r = d->const_rank[i];
      require(r >= 1 && r <= FLUID_MAX_RANK, "const rank out of range");
      Const c;
      c.shape.assign(d->const_shapes + (size_t)i * FLUID_MAX_RANK, d->const_shapes + (size_t)i * FLUID_MAX_RANK + r);
      c.dtype = d->const_dtype[i];
      c.role = d->const_role ? d->const_role[i] : FLUID_ROLE_OTHER;
      g.consts.push_back(std::move(c));
    }
    for (int n = 0; n < d->n_nodes; ++n) {
      const fluid_node_desc& nd = d->nodes[n];
      require(nd.n_in >= 1 && nd.n_in <= FLUID_MAX_IN, "node " + std::to_string(n) + ": n_in out of range");
      require(nd.out_rank >= 1 && nd.out_rank <= FLUID_MAX_RANK, "node " + std::to_string(n) + ": out_rank out of range");
      Node x;
      x.op = nd.op;
      x.ins.assign(nd.in, nd.in + nd.n_in);
      x.out_shape.assign(nd.out_shape, nd.out_shape + nd.out_rank);
      if (nd.op == FLUID_OP_TRANSPOSE) x.perm.assign(nd.perm, nd.perm + nd.out_rank);
      x.fattr = nd.f_attr[0];
      x.iattr = nd.i_attr[0];
      g.nodes.push_back(std::move(x));
    }
    g.outputs.assign(d->output_edges, d->output_edges + d->n_outputs);
    g.finalize();
    h->serial = next_serial();
    *out = h.release();
  });
}

fluid_status fluid_build_transformer(const fluid_model_cfg* cfg, fluid_graph** out) {
  return call_guarded([&] {
    require(cfg && out, "fluid_build_transformer: NULL argument");
    auto h = std::make_unique<fluid_graph>();
    h->g = build_transformer(*cfg);
    h->serial = next_serial();
    *out = h.release();
  });
}

fluid_status fluid_graph_info(const fluid_graph* g, int32_t* ni, int32_t* nc, int32_t* nn, int32_t* ne, int32_t* dt) {
  return call_guarded([&] {
    require(g, "NULL graph");
    if (ni) *ni = g->g.n_inputs();
    if (nc) *nc = (int32_t)g->g.consts.size();
    if (nn) *nn = g->g.n_nodes();
    if (ne) *ne = g->g.n_edges();
    if (dt) *dt = g->g.dtype;
  });
}

fluid_status fluid_graph_export_json(const fluid_graph* g, char* buf, uint64_t cap, uint64_t* len) {
  return call_guarded([&] {
    require(g && len, "NULL argument");
    std::string s = g->g.export_json();
    *len = s.size();
    if (buf && cap > 0) {
      size_t n = std::min<uint64_t>(cap - 1, s.size());
      std::memcpy(buf, s.data(), n);
      buf[n] = '\0';
    }
  });
}

fluid_status fluid_cost_table_load(const char* path, const fluid_graph* g, fluid_cost_table** out) {
  return call_guarded([&] {
    require(path && g && out, "NULL argument");
    std::ifstream f(path, std::ios::binary);
    require((bool)f, std::string("cannot open ") + path);
    std::stringstream ss;
    ss << f.rdbuf();
    auto h = std::make_unique<fluid_cost_table>();
    h->t = cost_table_from_json(json_parse(ss.str()));
    h->t.bind(g->g);
    h->serial = g->serial;
    *out = h.release();
  });
}

fluid_status fluid_cost_table_save(const fluid_cost_table* t, const char* path) {
  return call_guarded([&] {
    require(t && path, "NULL argument");
    std::ofstream f(path, std::ios::binary);
    require((bool)f, std::string("cannot write ") + path);
    f << cost_table_to_json(t->t);
    require((bool)f, std::string("write failed: ") + path);
  });
}

fluid_status fluid_measure_scratch_bytes(const fluid_graph* g, uint64_t* bytes) {
  return call_guarded([&] {
    require(g && bytes, "NULL argument");
    *bytes = measure_scratch_bytes(g->g);
  });
}

fluid_status fluid_plan_layouts(const fluid_graph* g, const fluid_cost_table* t, uint32_t flags, fluid_layout_plan** out) {
  return call_guarded([&] {
    require(g && t && out, "NULL argument");
    require(t->serial == g->serial, "cost table was loaded for another graph");
    require((flags & ~15u) == 0, "unknown flags");
    auto h = std::make_unique<fluid_layout_plan>();
    h->p = plan_layouts(g->g, t->t, flags);
    h->p.graph_serial = g->serial;
    h->serial = next_serial();
    *out = h.release();
  });
}

fluid_status fluid_layout_plan_get(const fluid_layout_plan* lp, int32_t* lay, int32_t* var, int64_t* total, int32_t* guard) {
  return call_guarded([&] {
    require(lp, "NULL plan");
    if (lay) for (size_t e = 0; e < lp->p.layout_idx.size(); ++e) lay[e] = lp->p.layout_idx[e];
    if (var) for (size_t n = 0; n < lp->p.variant.size(); ++n) var[n] = lp->p.variant[n];
    if (total) *total = lp->p.total;
    if (guard) *guard = lp->p.guard_used;
  });
}

fluid_status fluid_layout_plan_fusion(const fluid_layout_plan* lp, int32_t* fuse, int32_t* priced) {
  return call_guarded([&] {
    require(lp, "NULL plan");
    if (fuse)
      for (size_t n = 0; n < lp->p.fuse.size(); ++n) fuse[n] = lp->p.fuse[n];
    if (priced) *priced = lp->p.fusion_priced ? 1 : 0;
  });
}

fluid_status fluid_edge_layout(const fluid_graph* g, const fluid_layout_plan* lp, int32_t edge, int32_t* perm_out) {
  return call_guarded([&] {
    require(g && lp && perm_out, "NULL argument");
    require(lp->p.graph_serial == g->serial, "plan belongs to another graph");
    require(edge >= 0 && edge < g->g.n_edges(), "edge out of range");
    const Perm& p = lp->p.perm[edge];
    for (size_t i = 0; i < p.size(); ++i) perm_out[i] = p[i];
  });
}

fluid_status fluid_plan_arena(const fluid_graph* g, const fluid_layout_plan* lp, uint64_t align, uint32_t flags,
                              fluid_arena_plan** out) {
  return call_guarded([&] {
    require(g && lp && out, "NULL argument");
    require(lp->p.graph_serial == g->serial, "plan belongs to another graph");
    require(align >= 16 && (align & (align - 1)) == 0, "align must be a power of two >= 16");
    require((flags & ~3u) == 0, "unknown flags");
    auto h = std::make_unique<fluid_arena_plan>();
    // a plan that priced fusion chains fixes the fusions and their
    // lifetimes; otherwise FLUID_ARENA_EPILOGUE extends the lifetimes for
    // the executor's own fusion rule
    std::vector<int> until;
    if (!lp->p.fusion_priced && (flags & FLUID_ARENA_EPILOGUE)) until = epilogue_reads_until(g->g, lp->p);
    h->a = plan_arena(g->g, lp->p.perm, align, (flags & FLUID_ARENA_NO_REUSE) != 0, until,
                      lp->p.fusion_priced ? lp->p.fuse : std::vector<int>{});
    h->a.graph_serial = g->serial;
    h->serial = next_serial();
    *out = h.release();
  });
}

fluid_status fluid_run_launches(const fluid_graph* gh, const fluid_layout_plan* lh, const fluid_arena_plan* ah,
                                int32_t* launches) {
  return call_guarded([&] {
    require(gh && lh && ah && launches, "fluid_run_launches: NULL argument");
    require(lh->p.graph_serial == gh->serial && ah->a.graph_serial == gh->serial,
            "fluid_run_launches: plans belong to another graph");
    *launches = prepared_launches(*prepare(gh->g, lh->p, &ah->a));
  });
}

fluid_status fluid_arena_plan_get(const fluid_arena_plan* ap, uint64_t* peak, uint64_t* naive, uint64_t* lb,
                                  int64_t* offset, int32_t* root) {
  return call_guarded([&] {
    require(ap, "NULL plan");
    if (peak) *peak = ap->a.peak;
    if (naive) *naive = ap->a.naive;
    if (lb) *lb = ap->a.lower_bound;
    if (offset) for (size_t e = 0; e < ap->a.offset.size(); ++e) offset[e] = ap->a.offset[e];
    if (root) for (size_t e = 0; e < ap->a.root.size(); ++e) root[e] = ap->a.root[e];
  });
}

fluid_status fluid_run_schedule(const fluid_graph* gh, const fluid_layout_plan* lh, const fluid_arena_plan* ah,
                                int32_t* launch_of_node, uint8_t* output_written, char* names, uint64_t names_cap,
                                uint64_t* names_len, int32_t* n_launches) {
  return call_guarded([&] {
    require(gh && lh && ah, "fluid_run_schedule: NULL argument");
    require(lh->p.graph_serial == gh->serial && ah->a.graph_serial == gh->serial,
            "fluid_run_schedule: plans belong to another graph");
    const Graph& g = gh->g;
    const auto P = prepare(g, lh->p, &ah->a);
    std::vector<int32_t> launch(g.n_nodes(), -1);
    std::vector<uint8_t> written(g.n_nodes(), 0);
    std::string all;
    int32_t L = 0;
    // a prepared launch performs its node and the fuse_n nodes after it, and
    // writes the output of the last of them (and a residual sum it stores)
    auto claim = [&](size_t i, int32_t l) {
      const PreparedNode& pn = P->nodes[i];
      for (int f = 0; f <= pn.fuse_n; ++f) {
        launch[P->nodes[i + f].node] = l;
        written[P->nodes[i + f].node] = f == pn.fuse_n || (f == 0 && pn.fstore) ? 1 : 0;
      }
    };
    for (size_t i = 0; i < P->nodes.size(); ++i) {
      const PreparedNode& pn = P->nodes[i];
      if (pn.fused_away || pn.grouped) continue;
      claim(i, L);
      for (int m : pn.group) claim((size_t)m, L);
      std::string nm = (pn.fuse_n ? pn.kf : pn.k).name();
      if (!pn.group.empty()) nm += "_x" + std::to_string(1 + pn.group.size());
      all += (L ? "\n" : "") + nm;
      ++L;
    }
    if (names_len) *names_len = all.size() + 1;
    if (names) {
      require(names_cap >= all.size() + 1, "fluid_run_schedule: names buffer too small");
      std::memcpy(names, all.c_str(), all.size() + 1);
    }
    for (int n = 0; n < g.n_nodes(); ++n) {
      if (launch_of_node) launch_of_node[n] = launch[n];
      if (output_written) output_written[n] = written[n];
    }
    if (n_launches) *n_launches = L;
  });
}

fluid_status fluid_constant_layout(const fluid_graph* gh, const fluid_layout_plan* lh, int32_t c, int32_t* perm_out) {
  return call_guarded([&] {
    require(gh && lh && perm_out, "fluid_constant_layout: NULL argument");
    require(lh->p.graph_serial == gh->serial, "plan belongs to another graph");
    require(c >= 0 && c < (int32_t)gh->g.consts.size(), "constant id out of range");
    const Perm p = constant_layout(gh->g, lh->p, c);
    for (size_t i = 0; i < p.size(); ++i) perm_out[i] = p[i];
  });
}

fluid_status fluid_arena_plan_lifetimes(const fluid_arena_plan* ap, int32_t n_edges, uint64_t* size,
                                        int32_t* def, int32_t* last) {
  return call_guarded([&] {
    require(ap, "NULL plan");
    const auto& a = ap->a;
    require(n_edges == (int32_t)a.root.size(), "n_edges is not the plan's edge count");
    std::vector<char> is_buf(a.root.size(), 0);
    for (int b : a.buffers) is_buf[b] = 1;
    for (int32_t e = 0; e < n_edges; ++e) {
      if (size) size[e] = is_buf[e] ? a.size[e] : 0;
      if (def) def[e] = is_buf[e] ? a.def[e] : -1;
      if (last) last[e] = is_buf[e] ? a.last[e] : -1;
    }
  });
}

fluid_status fluid_node_kernel(const fluid_graph* gh, const fluid_layout_plan* lh, int32_t node, char* buf, uint64_t cap) {
  return call_guarded([&] {
    require(gh && lh && buf && cap > 0, "fluid_node_kernel: bad argument");
    require(lh->p.graph_serial == gh->serial, "plan belongs to another graph");
    const Graph& g = gh->g;
    require(node >= 0 && node < g.n_nodes(), "node out of range");
    std::string name = lh->p.variant[node] == -2 ? "fused" : "view";
    if (lh->p.variant[node] >= 0) {
      // a residual Add heading a planned chain names the normalisation's
      // summed kernel (its variant is that kernel's)
      const bool sum_head = lh->p.fusion_priced && lh->p.fuse[node] > 0 && g.nodes[node].op == FLUID_OP_ADD;
      const Node& nd = g.nodes[sum_head ? node + 1 : node];
      auto operand = [&](int v, int slot) {
        Operand o;
        o.shape = v >= 0 ? g.edge_shape(v) : g.consts[~v].shape;
        o.stride = v >= 0 ? dense_strides(o.shape, lh->p.perm[v])
                          : const_strides(nd, slot, lh->p.variant[node], o.shape);
        o.dtype = v >= 0 ? g.dtype : g.consts[~v].dtype;
        return o;
      };
      std::vector<Operand> ins;
      for (size_t slot = 0; slot < nd.ins.size(); ++slot) ins.push_back(operand(nd.ins[slot], (int)slot));
      Operand ou;
      ou.shape = nd.out_shape;
      ou.stride = dense_strides(ou.shape, lh->p.perm[g.out_edge(sum_head ? node + 1 : node)]);
      NodeKernel k;
      if (sum_head) {
        ins[0] = operand(g.nodes[node].ins[0], 0);
        k = prepare_sum_norm(nd, lh->p.variant[node], g.dtype, ins, operand(g.nodes[node].ins[1], 1), ou);
      } else {
        k = prepare_node(nd, lh->p.variant[node], g.dtype, ins, ou);
      }
      name = k.name();
    }
    size_t n = std::min<size_t>(cap - 1, name.size());
    std::memcpy(buf, name.data(), n);
    buf[n] = '\0';
  });
}

void fluid_graph_free(fluid_graph* g) { delete g; }
void fluid_cost_table_free(fluid_cost_table* t) { delete t; }
void fluid_layout_plan_free(fluid_layout_plan* lp) { delete lp; }
void fluid_arena_plan_free(fluid_arena_plan* ap) { delete ap; }

}  // extern "C"
