// Node -> kernel translation: given the layouts of a node's operands, pick
// the kernel family for a variant id and fill its parameter block.  Shared by
// the executor, the cost measurement and fluid_node_kernel; HIP-free.
//
// Variant ids per operator:
//   MATMUL                      0: 128x128 tile, 1: 64x64 tile (LDS-staged);
//                               2, 3, 5: 32x32 tile with K split over 4, 8,
//                               16 wavefronts; 4: 64x32 tile, K over 4;
//                               bf16 6: 256x128, 7: 128x128 tile, loads K
//                               tiles ahead; 8: 256x128, two workgroups per
//                               CU; 9: 128x128, whole K (<= 128) in LDS;
//                               fp32 6: 16x32, 7: 32x32 tiles, operands
//                               straight into registers
//   ADD MUL                     0: streaming elementwise in output order
//   GELU SILU TRANSPOSE RESHAPE 0: streaming; 1: LDS-tiled (input and output
//                               unit-stride dims differ)
//   SOFTMAX LAYERNORM RMSNORM   0: one wavefront per row; 1: one lane per row
//   ROPE                        0: streaming
#pragma once

#include <string>
#include <vector>

#include "graph.h"
#include "kparams.h"

namespace fluid {

struct Operand {
  const void* ptr = nullptr;
  Shape shape;
  std::vector<int64_t> stride;  // elements, per logical dim
  int dtype = FLUID_F32;
};

enum KernelFamily : int { KF_VIEW, KF_EW, KF_EW_TILED, KF_ROPE, KF_RED_ROW, KF_RED_COL, KF_GEMM, KF_WIN, KF_CONV };

enum GemmMode : int { GM_GENERIC = 0, GM_K = 1, GM_MN = 2 };  // A: K-/M-contig; B: K-/N-contig

struct NodeKernel {
  int family = KF_VIEW;
  bool available = false;
  std::string why;              // reason when not available
  int dtype = DT_F32;
  int vec = 1;                  // EW vector width (1, 4 or 8)
  bool vin0 = false, vin1 = false;
  EwParams ew{};
  RopeParams rope{};
  RedParams red{};
  GemmParams gemm{};
  WinParams win{};
  ConvParams conv{};
  int conv_kord = 0, conv_ks = 1, conv_tile = 64;  // conv: reduction order; K groups per workgroup; tile width
  bool red_block = false;       // row reduction: one 256-thread workgroup per row (variant 2)
  int gemm_tile = 0, amode = 0, bmode = 0, cmode = 0;  // cmode 0 generic, 1 N-contig, 2 M-contig
  std::string name() const;
};

int num_variants(int op);
// MatMul variants come in two halves: tile t (0 .. kGemmTiles-1) with the
// weight (a constant B operand [K, N]) stored row-major, and variant
// kGemmTiles + t, the same tile with the weight stored K-contiguous
// (physically [N, K]).  A weight is read by one MatMul, so its layout is a
// choice local to that node, made with the node's kernel: the cost table's
// minimum over variants picks the weight layout too.
constexpr int kGemmTiles = 10;
inline int gemm_tile_of(int variant) { return variant % kGemmTiles; }
inline bool packs_weight(int op, int variant) { return op == FLUID_OP_MATMUL && variant >= kGemmTiles; }
// Element strides of constant operand `slot` (shape `shape`) of node nd
// under `variant`: row-major, or K-contiguous for a packed weight.
std::vector<int64_t> const_strides(const Node& nd, int slot, int variant, const Shape& shape);
// Epilogue steps the kernels of MatMul variant `variant` perform after the
// product for a graph of dtype `dtype` (GemmParams): bit 0 bias, bit 1
// activation, bit 2 the Add / Mul with another tensor.
enum : int { EPI_BIAS = 1, EPI_ACT = 2, EPI_ROP = 4 };
int gemm_epilogue_caps(int variant, int dtype);
NodeKernel prepare_node(const Node& nd, int variant, int dtype, const std::vector<Operand>& ins,
                        const Operand& out);
// The LayerNorm / RMSNorm node nd (variant, operands as for prepare_node)
// applied to ins[0] + x1, the sum formed on load in fp32 (x1 of ins[0]'s
// shape, any layout): the kernel of a residual Add and its normalisation.
NodeKernel prepare_sum_norm(const Node& nd, int variant, int dtype, const std::vector<Operand>& ins, const Operand& x1,
                            const Operand& out);

// Cost measurement: the copies of a MatMul's or Conv's constant weight
// (bytes each) that the timed launches rotate over, so that each launch
// reads its weight from HBM, as in a run, where the layers in between have
// evicted it: copies totalling at least twice the 256 MiB last-level cache,
// at most 64.
int cold_weight_copies(uint64_t bytes);

// Row-major strides of a shape.
std::vector<int64_t> row_major_strides(const Shape& s);

}  // namespace fluid
