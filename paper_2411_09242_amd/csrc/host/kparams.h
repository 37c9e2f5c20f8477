// Kernel parameter blocks, filled on the host and passed by value to the
// HIP kernels.  Plain C++ (no HIP types) so host code and tests can build
// them without a GPU toolchain.  All offsets are in elements; every tensor
// handed to a kernel has fewer than 2^31 elements.
#pragma once

#include <cstdint>

namespace fluid {

// Exact unsigned division by a runtime constant (Granlund-Montgomery):
// q = (umulhi(n, m) + n) >> s for every n < 2^32.
struct FastDiv {
  uint32_t d = 1, m = 1, s = 0;
};
FastDiv make_fastdiv(uint32_t d);

constexpr int kMaxDims = 6;

enum EwOp : int { EW_COPY = 0, EW_ADD = 1, EW_MUL = 2, EW_GELU = 3, EW_SILU = 4, EW_RELU = 5 };
enum DType : int { DT_F32 = 0, DT_BF16 = 1 };

// Elementwise / relayout over a canonical iteration space: dims ordered
// outer -> inner with the output's unit-stride dim last.
struct EwParams {
  int rank;
  uint32_t ext[kMaxDims];
  FastDiv div[kMaxDims];      // div[d] divides by ext[d] (div[rank-1] by ext/VEC)
  int32_t os[kMaxDims];       // output strides
  int32_t is0[kMaxDims];      // input 0 strides
  int32_t is1[kMaxDims];      // input 1 strides (0 = broadcast)
  uint32_t total;             // elements (or vectors) to produce
  const void* x0;
  const void* x1;
  void* y;
  int op;
  int in1_dtype;              // dtype of input 1 (a bias constant may differ)
  // tiled variant: the input's unit-stride dim and the grid decomposition
  int tdim;                   // index of the input-contiguous dim (!= rank-1)
  uint32_t tiles_inner, tiles_t;
  FastDiv div_ti, div_tt;     // over tiles of dim rank-1 and of dim tdim
};

// RoPE over the iteration space [B, S, NH, D/2] (dims reordered by output
// stride); pos_dim / half_dim give where S and D/2 landed.
struct RopeParams {
  int rank;
  uint32_t ext[4];
  FastDiv div[4];
  int32_t xs[4], ys[4];       // strides of x and y for the 4 iteration dims
  int32_t x_half, y_half;     // stride of D in x / y, times D/2
  int pos_dim, half_dim;
  uint32_t half;              // D/2 (row length of the tables)
  uint32_t total;
  const void* x;
  void* y;
  const float* cos_t;
  const float* sin_t;
};

// RED_SUM_*: the normalisation of x + x1 (a residual sum formed on load,
// in fp32, never rounded or stored).
enum RedOp : int { RED_SOFTMAX = 0, RED_LAYERNORM = 1, RED_RMSNORM = 2, RED_SUM_LAYERNORM = 3, RED_SUM_RMSNORM = 4 };
constexpr int red_base_op(int op) { return op >= RED_SUM_LAYERNORM ? op - 2 : op; }
constexpr bool red_has_sum(int op) { return op >= RED_SUM_LAYERNORM; }

// Row reductions over the last logical dim (length R).  Row dims are
// ordered by input stride, outer -> inner.
struct RedParams {
  int nrd;
  uint32_t rext[kMaxDims];
  FastDiv rdiv[kMaxDims];
  int32_t ris[kMaxDims], ros[kMaxDims];
  int qdim;                   // row-dim index of the query dim (causal), -1 otherwise
  uint32_t nrows;
  uint32_t R;
  int32_t irs, ors;           // input / output stride of the reduced dim
  int32_t ris1[kMaxDims];     // the second summand's strides (RED_SUM_*)
  int32_t irs1;
  const void* x1;
  void* h;                    // RED_SUM_*: the sum's own output (y's layout), or null
  const void* x;
  void* y;
  const void* gamma;
  const void* beta;
  float attr;                 // softmax scale or norm eps
  int causal;
  int op;
};

// Zero Pad and MaxPool over [N, C, H, W]: one thread per output element; the
// four output dims are walked outer -> inner in the output's physical order
// (dims sorted by output stride), each with its input stride (N and C) or
// its role (H, W), whose input coordinate the op derives.
struct WinParams {
  uint32_t ext[4];
  FastDiv div[4];
  int32_t os[4], is[4];       // output strides; input strides of N / C dims
  int32_t role[4];            // 0 batch or channel, 1 H, 2 W
  int32_t in_h, in_w;         // input extents of H and W
  int32_t is_h, is_w;         // input strides of H and W
  uint32_t total;
  int32_t op;                 // 0 pad, 1 maxpool
  int32_t k;                  // pad width / pool window
  const void* x;
  void* y;
};

// Convolution (no padding, stride 1) as an implicit GEMM: row m = (n, i, j)
// an output pixel, column o an output channel, reduction index k over
// (c, u, v) -- in the weight's row-major order (KORD 0) or as (u, v, c)
// (KORD 1, channel fastest) -- so that x[n, c, i+u, j+v] sits at
// row_offset(m) + col_offset(k) for any layout of x.
struct ConvParams {
  const float* x;
  const float* w;             // [Co, C, KH, KW] row-major
  const float* bias;          // [Co] or null
  float* y;
  uint32_t M, Co, K, C;       // M = N*OH*OW, K = C*KH*KW
  uint32_t OHW, OW, KHW, KW, KWC;
  FastDiv ohw_div, ow_div, khw_div, kw_div, kwc_div, c_div;
  int32_t x_n, x_c, x_h, x_w;
  int32_t y_n, y_c, y_h, y_w;
  uint32_t tiles_n;
};

// C[g, m, n] = sum_k A[g, m, k] * B[g, k, n]; g = g1 * G2 + g2 and
// m = m1 * M2 + m2 (two-level decomposition of batch and row indices).
struct GemmParams {
  const void* A;
  const void* B;
  void* C;
  uint32_t M, N, K, G;
  uint32_t G2, M2;
  FastDiv g2div, m2div;
  int32_t a_g1, a_g2, a_m1, a_m2, a_k;
  int32_t b_g1, b_g2, b_k, b_n;
  int32_t c_g1, c_g2, c_m1, c_m2, c_n;
  int32_t cmode;              // 0 scalar stores, 1 N-contiguous, 2 M-contiguous (4 rows)
  uint32_t tiles_m, tiles_n;
  uint32_t a_bytes, b_bytes;  // byte span of A and B from their base pointers
  // Causal attention (rows m are query positions, columns or k key
  // positions): bit 0, only C[m][n] with n <= m is ever read, so tiles with
  // every n > m may be skipped; bit 1, A[m][k] = 0 for k > m, so the K loop
  // of rows m0 .. m0 + BM - 1 may stop at m0 + BM.
  uint32_t causal;
  // Epilogue: C[m][n] = act(sum_k A B + bias[n]) (rop 0), that plus R[m][n]
  // (rop 1) or times R[m][n] (rop 2); bias a dense [N] vector or none when
  // null; act 0 none, 1 GELU (erf form), 2 SiLU; R a tensor of C's shape
  // with its own strides (batch and row decomposition as C's).  Bias and R
  // hold bf16 when epi_bf16, else fp32.
  const void* bias;
  uint32_t epi_bf16;
  uint32_t act;
  const void* R;
  int32_t r_g1, r_g2, r_m1, r_m2, r_n;
  FastDiv r_m2div;            // a copy of m2div
  uint32_t rop;
};

// Up to kMaxGroup independent products of one kernel shape in one launch
// (the Q, K and V projections of a layer): workgroups [tiles[i],
// tiles[i+1]) run member i.
constexpr int kMaxGroup = 4;
struct GemmGroup {
  GemmParams p[kMaxGroup];
  uint32_t n;
  uint32_t tiles[kMaxGroup + 1];
};

}  // namespace fluid
