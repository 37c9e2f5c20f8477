// Cost table: measured time per node for each combination of input and
// output layouts (Alg. 3's eval), per kernel variant.
#pragma once

#include <map>
#include <string>
#include <utility>
#include <vector>

#include "graph.h"
#include "json.h"

namespace fluid {

struct SigEntry {
  std::vector<Perm> in;          // one layout per activation slot
  Perm out;
  std::vector<int64_t> costs;    // ns per variant; -1 = unavailable
};

struct Sig {
  int op = 0;
  std::vector<Shape> in_shapes;  // activation slots
  Shape out_shape;
  std::vector<SigEntry> entries;
};

// Dense costs of one node over (slot layout index..., out layout index),
// indices into the table's candidate lists of the node's edges.
struct NodeCost {
  std::vector<int> dims;
  std::vector<int64_t> best;     // min over variants, kInf if none
  std::vector<int32_t> var;      // argmin variant (lowest id on ties), -1 if none
  std::vector<int64_t> v0;       // variant-0 cost, kInf if unavailable
};

// A fused entry: the chain of MatMul node m and length t (fusion.h) costs
// fused_sigs[sig], whose entries list the chain's slot layouts and the
// layout of node m+t's output.
struct FusedRef {
  int m = 0, t = 0, sig = 0;
};

struct CostTable {
  std::vector<std::vector<Perm>> L;  // candidate layouts per edge, identity first
  std::vector<Sig> sigs;
  std::vector<int> node_sig;
  std::vector<Sig> fused_sigs;
  std::vector<FusedRef> fused_refs;
  std::vector<NodeCost> nodes;                    // filled by bind()
  std::map<std::pair<int, int>, NodeCost> fused;  // (m, t) -> costs, filled by bind()
  uint64_t graph_serial = 0;

  // Validates against g and builds the dense per-node arrays.
  void bind(const Graph& g);
};

CostTable cost_table_from_json(const Json& j);
std::string cost_table_to_json(const CostTable& t);

}  // namespace fluid
