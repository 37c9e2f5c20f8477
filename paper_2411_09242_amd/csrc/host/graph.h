// Operator graph IR: nodes are operators, edges are tensors (one output per
// node); the node array order is the execution order.
#pragma once

#include <string>
#include <vector>

#include "common.h"

namespace fluid {

struct Node {
  int op = 0;
  std::vector<int> ins;  // >= 0 edge id, < 0 constant ~id
  Shape out_shape;
  Perm perm;             // TRANSPOSE
  float fattr = 0.f;
  int iattr = 0;
  // derived by Graph::finalize, for a batched MatMul: bit 0, a causal
  // Softmax is the only reader of the output (entries above its diagonal
  // are never read); bit 1, input A is a causal Softmax's output (exactly
  // zero above the diagonal)
  int causal = 0;
};

struct Const {
  Shape shape;
  int dtype = FLUID_F32;
  int role = FLUID_ROLE_OTHER;
};

// Reshape classification: split X dim a into Y dims (a, a+1), merge X dims
// (a, a+1) into Y dim a, identical shapes, or anything else.
enum class ReshapeKind { Same, Split, Merge, Other };
ReshapeKind reshape_kind(const Shape& xs, const Shape& ys, int* axis);

struct Graph {
  int dtype = FLUID_F32;
  std::vector<Shape> inputs;
  std::vector<Const> consts;
  std::vector<Node> nodes;
  std::vector<int> outputs;

  // derived (filled by finalize)
  std::vector<std::vector<int>> act_in;   // per node: activation input edges, slot order
  std::vector<std::vector<int>> readers;  // per edge: nodes reading it (ascending, unique)
  std::vector<std::vector<int>> const_readers;  // per constant: nodes reading it (ascending, unique)
  std::vector<char> is_output;            // per edge
  std::vector<std::vector<Perm>> cand;    // per edge: candidate layouts L(e)

  int n_inputs() const { return (int)inputs.size(); }
  int n_nodes() const { return (int)nodes.size(); }
  int n_edges() const { return n_inputs() + n_nodes(); }
  int out_edge(int n) const { return n_inputs() + n; }
  int producer(int e) const { return e < n_inputs() ? -1 : e - n_inputs(); }
  const Shape& edge_shape(int e) const {
    return e < n_inputs() ? inputs[e] : nodes[e - n_inputs()].out_shape;
  }
  bool pinned(int e) const { return e < n_inputs() || is_output[e]; }

  // Validates every node and fills the derived fields; throws fluid::Error.
  void finalize();
  std::string export_json() const;
};

Graph build_transformer(const fluid_model_cfg& cfg);
const char* op_name(int op);

}  // namespace fluid
