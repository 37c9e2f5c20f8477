// Arena planner: Alg. 4 (Greedy-by-Size) over tensor lifetimes, the naive
// one-slice-per-tensor plan it improves on, and the max-live lower bound.
//
// Readings: buffers are the outputs of non-view nodes other than graph
// outputs; lifetimes are closed intervals [producer, last reader] over node
// ids (so no operator writes over its own inputs); buffers are taken by size
// descending, then producer, then edge id; each goes into the smallest gap,
// among the placed buffers whose lifetimes overlap its own, that fits it
// (lowest offset on ties) -- the text's "most suitable slot" -- else right
// after those buffers ("increase and allocate the last free block").
#include <algorithm>

#include "fusion.h"
#include "layouts.h"
#include "planner.h"

namespace fluid {

bool node_is_view(const Graph& g, int n, const std::vector<Perm>& perm_of_edge) {
  const Node& nd = g.nodes[n];
  if (nd.op != FLUID_OP_TRANSPOSE && nd.op != FLUID_OP_RESHAPE) return false;
  const int eo = g.out_edge(n);
  if (g.is_output[eo]) return false;
  const int ei = g.act_in[n][0];
  return is_view(nd.op, nd.perm, g.edge_shape(ei), nd.out_shape, perm_of_edge[ei], perm_of_edge[eo]);
}

namespace {

uint64_t align_up(uint64_t x, uint64_t a) { return (x + a - 1) / a * a; }

struct Buffers {
  std::vector<int> root, list, def, last;
  std::vector<uint64_t> size;
};

Buffers collect(const Graph& g, const std::vector<Perm>& perm, uint64_t align, const std::vector<int>& until_in,
                const std::vector<int>& fuse) {
  Buffers B;
  const int E = g.n_edges();
  B.root.resize(E);
  for (int e = 0; e < E; ++e) B.root[e] = e;
  // fused chains: results kept on chip (a stored one is an ordinary buffer),
  // operands read until the chain's end
  std::vector<char> on_chip(E, 0);
  std::vector<int> until = until_in;
  if (!fuse.empty()) {
    if (until.empty()) {
      until.resize(g.n_nodes());
      for (int n = 0; n < g.n_nodes(); ++n) until[n] = n;
    }
    for (int m = 0; m < g.n_nodes(); ++m)
      if (fuse[m]) {
        for (int e : on_chip_edges(g, m, fuse[m])) on_chip[e] = 1;
        until[m] = std::max(until[m], m + fuse[m]);
      }
  }
  std::vector<char> is_buf(E, 0);
  for (int n = 0; n < g.n_nodes(); ++n) {
    const int eo = g.out_edge(n);
    if (node_is_view(g, n, perm)) {
      B.root[eo] = B.root[g.act_in[n][0]];
    } else if (!g.is_output[eo] && !on_chip[eo]) {
      is_buf[eo] = 1;
      B.list.push_back(eo);
    }
  }
  const uint64_t isz = (uint64_t)dtype_bytes(g.dtype);
  B.size.assign(E, 0);
  B.def.assign(E, -1);
  B.last.assign(E, -1);
  for (int b : B.list) {
    B.size[b] = align_up((uint64_t)numel(g.edge_shape(b)) * isz, align);
    B.def[b] = B.last[b] = g.producer(b);
  }
  for (int n = 0; n < g.n_nodes(); ++n)
    for (int e : g.act_in[n]) {
      int r = B.root[e];
      if (is_buf[r]) B.last[r] = std::max(B.last[r], until.empty() ? n : until[n]);
    }
  return B;
}

bool overlaps(const Buffers& B, int a, int b) { return B.def[a] <= B.last[b] && B.def[b] <= B.last[a]; }

}  // namespace

ArenaPlan plan_arena(const Graph& g, const std::vector<Perm>& perm, uint64_t align, bool no_reuse,
                     const std::vector<int>& reads_until, const std::vector<int>& fuse) {
  Buffers B = collect(g, perm, align, reads_until, fuse);
  ArenaPlan ap;
  const int E = g.n_edges();
  ap.root = B.root;
  ap.buffers = B.list;
  ap.size = B.size;
  ap.def = B.def;
  ap.last = B.last;
  std::vector<int64_t> off(E, -1);
  if (no_reuse) {
    uint64_t cur = 0;
    std::vector<int> sorted = B.list;
    std::sort(sorted.begin(), sorted.end());
    for (int b : sorted) { off[b] = (int64_t)cur; cur += B.size[b]; }
  } else {
    std::vector<int> order = B.list;
    std::sort(order.begin(), order.end(), [&](int a, int b) {
      if (B.size[a] != B.size[b]) return B.size[a] > B.size[b];
      if (B.def[a] != B.def[b]) return B.def[a] < B.def[b];
      return a < b;
    });
    std::vector<int> placed;
    for (int b : order) {
      std::vector<int> O;
      for (int o : placed)
        if (overlaps(B, o, b)) O.push_back(o);
      std::sort(O.begin(), O.end(), [&](int x, int y) { return off[x] != off[y] ? off[x] < off[y] : x < y; });
      int64_t cursor = 0, best_gap = -1, best_off = -1;
      for (int o : O) {
        int64_t gap = off[o] - cursor;
        if (gap >= (int64_t)B.size[b] && (best_gap < 0 || gap < best_gap)) { best_gap = gap; best_off = cursor; }
        cursor = std::max(cursor, off[o] + (int64_t)B.size[o]);
      }
      off[b] = best_gap >= 0 ? best_off : cursor;
      placed.push_back(b);
    }
  }
  uint64_t peak = 0;
  for (int b : B.list) peak = std::max(peak, (uint64_t)off[b] + B.size[b]);
  ap.peak = peak;
  // per-edge offsets: views resolve to their root's offset
  ap.offset.assign(E, -1);
  for (int e = 0; e < E; ++e)
    if (off[B.root[e]] >= 0) ap.offset[e] = off[B.root[e]];
  // max-live lower bound over node ids
  uint64_t lb = 0;
  for (int t = 0; t < g.n_nodes(); ++t) {
    uint64_t s = 0;
    for (int b : B.list)
      if (B.def[b] <= t && t <= B.last[b]) s += B.size[b];
    lb = std::max(lb, s);
  }
  ap.lower_bound = lb;
  // naive: row-major layouts, no reuse
  {
    std::vector<Perm> ident;
    for (int e = 0; e < E; ++e) ident.push_back(identity_perm((int)g.edge_shape(e).size()));
    Buffers N = collect(g, ident, align, {}, {});
    uint64_t s = 0;
    for (int b : N.list) s += N.size[b];
    ap.naive = s;
  }
  return ap;
}

}  // namespace fluid
