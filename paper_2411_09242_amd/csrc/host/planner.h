// Layout planner (Section 3: Alg. 1-3, Eq. 1, majority vote) and arena
// planner (Alg. 4, Greedy-by-Size).
#pragma once

#include <vector>

#include "costtable.h"
#include "graph.h"

namespace fluid {

struct LayoutPlan {
  std::vector<int> layout_idx;     // per edge, index into the table's L(e)
  std::vector<Perm> perm;          // per edge, the chosen permutation
  std::vector<int> variant;        // per node, -1 = view, -2 = performed in a fused MatMul's launch
  std::vector<int> fuse;           // per node: length t of the fusion chain a MatMul runs, else 0
  bool fusion_priced = false;      // the table priced fusion chains (the plan's fusions are the run's)
  int64_t total = 0;
  int guard_used = 0;
  std::vector<std::vector<int>> paths;
  uint64_t graph_serial = 0;
};

std::vector<int> longest_path(const Graph& g, const std::vector<int>& S);
std::vector<std::vector<int>> split_paths(const Graph& g);
LayoutPlan plan_layouts(const Graph& g, const CostTable& t, uint32_t flags);
LayoutPlan plan_layouts_dp(const Graph& g, const CostTable& t, uint32_t flags);
LayoutPlan identity_plan(const Graph& g);  // row-major everywhere, variant 0

struct ArenaPlan {
  std::vector<int> root;            // per edge
  std::vector<int64_t> offset;      // per edge (-1 = not in the arena)
  std::vector<int> buffers;         // arena buffer edge ids
  std::vector<uint64_t> size;       // per edge (0 if not a buffer)
  std::vector<int> def, last;       // per edge (buffers only)
  uint64_t peak = 0, naive = 0, lower_bound = 0;
  uint64_t graph_serial = 0;
};

bool node_is_view(const Graph& g, int n, const std::vector<Perm>& perm_of_edge);
// reads_until (empty: each node itself): per node, the last node id until
// which that node's inputs must stay live.  fuse (empty: none): the layout
// plan's fusion chains, whose intermediate results get no buffer and whose
// MatMul reads its operands until the chain's end.
ArenaPlan plan_arena(const Graph& g, const std::vector<Perm>& perm_of_edge, uint64_t align, bool no_reuse,
                     const std::vector<int>& reads_until = {}, const std::vector<int>& fuse = {});

}  // namespace fluid
