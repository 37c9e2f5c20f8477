// Launch preparation for the executor: per non-view node, the kernel
// parameters of its variant under the layout plan, where each operand lives
// (arena offset, caller input / output, constant), and the epilogue fusion
// of a MatMul with the nodes launched right after it.  HIP-free, so that
// the host-only build reports the same launches and the arena planner can
// see which MatMuls will absorb which nodes.
#pragma once

#include <memory>
#include <utility>
#include <vector>

#include "dispatch.h"
#include "planner.h"

namespace fluid {

enum BindKind : int { BK_ARENA = 0, BK_INPUT = 1, BK_OUTPUT = 2, BK_CONST = 3 };

struct Bind {
  int kind = BK_ARENA;
  int index = 0;
  int64_t off = 0;  // bytes from the base
};

struct PreparedNode {
  int node = 0;
  NodeKernel k;
  std::vector<Bind> in;  // one per node input (activations and constants)
  Bind out;
  std::vector<Operand> ops;  // the inputs as prepared (for re-preparing a fused launch)
  // Epilogue fusion: this MatMul also performs the fuse_n nodes after it (in
  // this order, each optional: a bias Add, a GELU / SiLU, an Add or Mul with
  // another tensor) and writes the last one's output (fout) directly; those
  // nodes are then not launched by fluid_run.  A residual Add that heads a
  // planned chain is instead performed by the LayerNorm / RMSNorm after it
  // (kf a RED_SUM_* reduction, fuse_n 1); when the sum has further readers
  // that launch also stores it at out (fstore), in the layout of fout.
  int fuse_n = 0;
  NodeKernel kf;
  Bind fout;
  int fbias = -1;           // constant id of the bias, -1 when none
  int fgamma = -1, fbeta = -1;  // a summed normalisation's scale / shift constants
  bool fstore = false;          // the summed normalisation also stores the sum
  Bind fr;                  // the other tensor of the Add / Mul (kf.gemm.rop set)
  int fr_edge = -1;         // its edge
  // Grouped launch: this product also launches the products of these nodes
  // (indices into Prepared::nodes, launched right after it), which are then
  // not launched on their own (grouped set).
  std::vector<int> group;
  bool grouped = false;
  bool fused_away = false;  // this node is performed by a MatMul before it
};

struct Prepared {
  std::vector<PreparedNode> nodes;
};

// The prepared launches of (graph, layout plan, arena plan).  With ap null
// the arena is ignored: every activation is bound at offset 0 (alignment
// decisions are the same, arena offsets being 256-byte aligned) and no
// fusion is refused for sharing arena bytes -- the fusion a run will do
// when the arena keeps those bytes apart (epilogue_reads_until).
std::shared_ptr<Prepared> prepare(const Graph& g, const LayoutPlan& lp, const ArenaPlan* ap);

// Per node, the last node whose execution reads that node's inputs: the
// node itself, or for a MatMul that absorbs the nodes after it (as prepared
// with the arena ignored) the last of them, since the fused launch is only
// done with its operands once it has written that node's output.
std::vector<int> epilogue_reads_until(const Graph& g, const LayoutPlan& lp);

// The fused launch of MatMul mn (variant, operands as prepared) writing out
// with the epilogue steps act (0 none, 1 GELU, 2 SiLU) and rop (0 none,
// 1 Add, 2 Mul of R); unavailable when the tile lacks a step.  The bias and
// R pointers are bound at launch.
NodeKernel fused_gemm_kernel(const Node& mn, int variant, int dtype, const std::vector<Operand>& mm_ops,
                             const Operand& out, uint32_t act, uint32_t rop, const Operand* r);

// The layout constant c must be stored in for a run of this plan: the
// identity (row-major as supplied), or (1, 0) -- K-contiguous -- for a
// weight whose one reader runs a packed-weight MatMul variant.
Perm constant_layout(const Graph& g, const LayoutPlan& lp, int c);

// Kernel launches of a prepared run.
int prepared_launches(const Prepared& P);

}  // namespace fluid
