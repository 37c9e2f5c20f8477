// Fusion chains: the operators a MatMul may perform in its own launch, as
// alternatives the layout planner prices (Section 4: the compiler fuses
// operators before planning layouts).  A MatMul m and the nodes m+1 .. m+t
// form a chain when, step by step, the previous result has exactly one
// reader (the next node) and is no graph output, and the steps are, in this
// order and each optional: an Add of a bias constant [N] (first step only),
// one GELU or SiLU, and an Add or Mul with another activation R of the
// product's shape produced before m (last step).  A second kind starts at
// an Add of two activations of its output's shape (a residual sum) whose
// result is read by the next node, a LayerNorm / RMSNorm over it (with
// constant scale and shift), and is no graph output: the normalisation
// launch also forms the sum (t = 1).  A MatMul chain's intermediates never
// reach memory; a residual sum with further readers (a pre-norm block's
// next residual) is stored by the launch too, in the layout of the norm's
// output (CH_NORM_STORE), else it stays on chip (CH_NORM).
// t = 1..3; every prefix of a chain is a chain.
#pragma once

#include <vector>

#include "graph.h"

namespace fluid {

enum ChainKind : int { CH_BIAS = 0, CH_ACT = 1, CH_ADD_R = 2, CH_MUL_R = 3, CH_NORM = 4, CH_NORM_STORE = 5 };

struct ChainStep {
  int node;
  int kind;
  int r;      // R's edge for CH_ADD_R / CH_MUL_R, else -1
  int bias;   // the bias constant id for CH_BIAS, else -1
};

// The longest chain starting at node m (empty if none).
std::vector<ChainStep> chain_steps(const Graph& g, int m);
// Edges a fused launch of (m, t) reads, in slot order: the MatMul's
// activation inputs, then R of a last Add / Mul step.
std::vector<int> chain_slots(const Graph& g, int m, int t);
// Intermediate results of (m, t) its launch stores (in the layout of node
// m+t's output), and those that never reach memory.
std::vector<int> stored_edges(const Graph& g, int m, int t);
std::vector<int> on_chip_edges(const Graph& g, int m, int t);

}  // namespace fluid
