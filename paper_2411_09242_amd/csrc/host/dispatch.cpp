#include "dispatch.h"

#include <algorithm>

namespace fluid {

FastDiv make_fastdiv(uint32_t d) {
  FastDiv f;
  f.d = d ? d : 1;
  uint32_t s = 0;
  while ((uint64_t(1) << s) < f.d) ++s;
  f.s = s;
  f.m = (uint32_t)(((uint64_t(1) << 32) * ((uint64_t(1) << s) - f.d)) / f.d + 1);
  return f;
}

std::vector<int64_t> row_major_strides(const Shape& s) {
  std::vector<int64_t> st(s.size(), 1);
  for (int i = (int)s.size() - 2; i >= 0; --i) st[i] = st[i + 1] * s[i + 1];
  return st;
}

int num_variants(int op) {
  switch (op) {
    case FLUID_OP_MATMUL: return 2 * kGemmTiles;
    case FLUID_OP_GELU:
    case FLUID_OP_SILU:
    case FLUID_OP_RELU:
    case FLUID_OP_TRANSPOSE:
    case FLUID_OP_RESHAPE: return 2;
    case FLUID_OP_CONV: return 6;
    case FLUID_OP_SOFTMAX:
    case FLUID_OP_LAYERNORM:
    case FLUID_OP_RMSNORM: return 3;
    default: return 1;
  }
}

int cold_weight_copies(uint64_t bytes) {
  const uint64_t target = 512ull << 20;
  if (bytes == 0) return 1;
  return (int)std::min<uint64_t>(64, std::max<uint64_t>(1, (target + bytes - 1) / bytes));
}

std::vector<int64_t> const_strides(const Node& nd, int slot, int variant, const Shape& shape) {
  if (packs_weight(nd.op, variant) && slot == 1 && shape.size() == 2) return {1, shape[0]};
  return row_major_strides(shape);
}

namespace {

struct IterDim {
  int64_t ext, os, s0, s1;
};

bool aligned16(const void* p) { return ((uintptr_t)p & 15u) == 0; }

std::vector<IterDim> canonicalize(std::vector<IterDim> d) {
  std::vector<IterDim> k;
  for (auto& x : d)
    if (x.ext != 1) k.push_back(x);
  std::stable_sort(k.begin(), k.end(), [](const IterDim& a, const IterDim& b) { return a.os > b.os; });
  std::vector<IterDim> m;
  for (int i = (int)k.size() - 1; i >= 0; --i) {
    const IterDim& o = k[i];
    if (!m.empty()) {
      IterDim& in = m.back();
      if (o.os == in.os * in.ext && o.s0 == in.s0 * in.ext && o.s1 == in.s1 * in.ext) {
        in.ext *= o.ext;
        continue;
      }
    }
    m.push_back(o);
  }
  std::reverse(m.begin(), m.end());
  if (m.empty()) m.push_back({1, 1, 0, 0});
  return m;
}

void check_small(const Operand& o, const char* what) {
  if (numel(o.shape) >= (int64_t(1) << 31))
    fail(FLUID_E_UNSUPPORTED, std::string(what) + ": tensors of 2^31 or more elements are not supported");
}

int ew_op_of(int op) {
  switch (op) {
    case FLUID_OP_ADD: return EW_ADD;
    case FLUID_OP_MUL: return EW_MUL;
    case FLUID_OP_GELU: return EW_GELU;
    case FLUID_OP_SILU: return EW_SILU;
    case FLUID_OP_RELU: return EW_RELU;
    default: return EW_COPY;
  }
}

NodeKernel prepare_ew(const Node& nd, int variant, int dtype, const std::vector<Operand>& ins, const Operand& out) {
  NodeKernel k;
  k.dtype = dtype == FLUID_BF16 ? DT_BF16 : DT_F32;
  const Operand& x = ins[0];
  const bool binary = nd.op == FLUID_OP_ADD || nd.op == FLUID_OP_MUL;
  std::vector<IterDim> dims;
  if (nd.op == FLUID_OP_TRANSPOSE) {
    for (size_t i = 0; i < out.shape.size(); ++i)
      dims.push_back({out.shape[i], out.stride[i], x.stride[nd.perm[i]], 0});
  } else if (nd.op == FLUID_OP_RESHAPE) {
    int a;
    ReshapeKind rk = reshape_kind(x.shape, out.shape, &a);
    if (rk == ReshapeKind::Same) {
      for (size_t i = 0; i < out.shape.size(); ++i) dims.push_back({out.shape[i], out.stride[i], x.stride[i], 0});
    } else if (rk == ReshapeKind::Split) {  // iterate the output's (finer) dims
      for (int i = 0; i < (int)out.shape.size(); ++i) {
        int64_t s0;
        if (i < a) s0 = x.stride[i];
        else if (i == a) s0 = x.stride[a] * out.shape[a + 1];
        else if (i == a + 1) s0 = x.stride[a];
        else s0 = x.stride[i - 1];
        dims.push_back({out.shape[i], out.stride[i], s0, 0});
      }
    } else if (rk == ReshapeKind::Merge) {  // iterate the input's (finer) dims
      for (int i = 0; i < (int)x.shape.size(); ++i) {
        int64_t os;
        if (i < a) os = out.stride[i];
        else if (i == a) os = out.stride[a] * x.shape[a + 1];
        else if (i == a + 1) os = out.stride[a];
        else os = out.stride[i - 1];
        dims.push_back({x.shape[i], os, x.stride[i], 0});
      }
    } else {
      fail(FLUID_E_UNSUPPORTED, "reshape kind");
    }
  } else {
    const size_t r = out.shape.size();
    for (size_t i = 0; i < r; ++i) {
      int64_t s1 = 0;
      if (binary) {
        const Operand& y = ins[1];
        if (y.shape.size() == r) s1 = y.stride[i];
        else s1 = (i == r - 1) ? y.stride[0] : 0;  // bias [N] broadcast
      }
      dims.push_back({out.shape[i], out.stride[i], x.stride[i], s1});
    }
  }
  check_small(out, "elementwise");
  std::vector<IterDim> c = canonicalize(dims);
  const int R = (int)c.size();
  if (R > kMaxDims) fail(FLUID_E_UNSUPPORTED, "elementwise rank");
  EwParams& p = k.ew;
  p.rank = R;
  for (int d = 0; d < R; ++d) {
    p.ext[d] = (uint32_t)c[d].ext;
    p.os[d] = (int32_t)c[d].os;
    p.is0[d] = (int32_t)c[d].s0;
    p.is1[d] = (int32_t)c[d].s1;
  }
  p.x0 = x.ptr;
  p.x1 = binary ? ins[1].ptr : nullptr;
  p.y = const_cast<void*>(out.ptr);
  p.op = ew_op_of(nd.op);
  p.in1_dtype = binary ? (ins[1].dtype == FLUID_BF16 ? DT_BF16 : DT_F32) : k.dtype;
  const uint32_t total = (uint32_t)numel(out.shape);
  if (variant == 0) {
    k.family = KF_EW;
    const int VEC = k.dtype == DT_F32 ? 4 : 8;
    const uint32_t inner = p.ext[R - 1];
    int vec = (inner % VEC == 0 && aligned16(out.ptr)) ? VEC : 1;
    auto vec_ok = [&](const int32_t* s, const void* ptr) {
      if (vec == 1 || s[R - 1] != 1 || !aligned16(ptr)) return false;
      for (int d = 0; d < R - 1; ++d)
        if (s[d] % vec != 0) return false;
      return true;
    };
    k.vec = vec;
    k.vin0 = vec_ok(p.is0, p.x0);
    k.vin1 = binary && p.in1_dtype == k.dtype && vec_ok(p.is1, p.x1);
    for (int d = 0; d < R - 1; ++d) p.div[d] = make_fastdiv(p.ext[d]);
    p.div[R - 1] = make_fastdiv(inner / vec);
    p.total = total / vec;
    k.available = true;
    return k;
  }
  // variant 1: LDS-tiled relayout for unary ops whose input is contiguous
  // along a dim other than the output's innermost one
  k.family = KF_EW_TILED;
  if (binary) { k.why = "tiled variant is unary only"; return k; }
  int t = -1;
  for (int d = 0; d < R - 1; ++d)
    if (p.is0[d] == 1) t = d;
  if (t < 0) { k.why = "input and output share the unit-stride dim"; return k; }
  p.tdim = t;
  p.tiles_inner = (p.ext[R - 1] + 63) / 64;
  p.tiles_t = (p.ext[t] + 63) / 64;
  p.div_ti = make_fastdiv(p.tiles_inner);
  p.div_tt = make_fastdiv(p.tiles_t);
  uint32_t other = 1;
  for (int d = 0; d < R - 1; ++d)
    if (d != t) { p.div[d] = make_fastdiv(p.ext[d]); other *= p.ext[d]; }
  p.total = p.tiles_inner * p.tiles_t * other;  // blocks
  k.available = true;
  return k;
}

NodeKernel prepare_rope(const Node&, int dtype, const std::vector<Operand>& ins, const Operand& out) {
  NodeKernel k;
  k.family = KF_ROPE;
  k.dtype = dtype == FLUID_BF16 ? DT_BF16 : DT_F32;
  const Operand& x = ins[0];
  check_small(out, "rope");
  const int64_t half = x.shape[3] / 2;
  struct D { int64_t ext, xs, ys; int logical; };
  std::vector<D> d = {{x.shape[0], x.stride[0], out.stride[0], 0},
                      {x.shape[1], x.stride[1], out.stride[1], 1},
                      {x.shape[2], x.stride[2], out.stride[2], 2},
                      {half, x.stride[3], out.stride[3], 3}};
  std::stable_sort(d.begin(), d.end(), [](const D& a, const D& b) { return a.ys > b.ys; });
  RopeParams& p = k.rope;
  p.rank = 4;
  for (int i = 0; i < 4; ++i) {
    p.ext[i] = (uint32_t)d[i].ext;
    p.div[i] = make_fastdiv(p.ext[i]);
    p.xs[i] = (int32_t)d[i].xs;
    p.ys[i] = (int32_t)d[i].ys;
    if (d[i].logical == 1) p.pos_dim = i;
    if (d[i].logical == 3) p.half_dim = i;
  }
  p.x_half = (int32_t)(x.stride[3] * half);
  p.y_half = (int32_t)(out.stride[3] * half);
  p.half = (uint32_t)half;
  p.total = (uint32_t)(numel(out.shape) / 2);
  p.x = x.ptr;
  p.y = const_cast<void*>(out.ptr);
  p.cos_t = (const float*)ins[1].ptr;
  p.sin_t = (const float*)ins[2].ptr;
  // 16-byte pieces along D/2 when D is unit-stride in x and y
  const int VEC = k.dtype == DT_BF16 ? 8 : 4;
  bool vec_ok = p.half_dim == 3 && p.xs[3] == 1 && p.ys[3] == 1 && half % VEC == 0 && aligned16(p.x) &&
                aligned16(p.y) && aligned16(p.cos_t) && aligned16(p.sin_t) && p.x_half % VEC == 0 && p.y_half % VEC == 0;
  for (int i = 0; i < 3; ++i) vec_ok = vec_ok && p.xs[i] % VEC == 0 && p.ys[i] % VEC == 0;
  if (vec_ok) {
    k.vec = VEC;
    p.ext[3] = (uint32_t)(half / VEC);
    p.div[3] = make_fastdiv(p.ext[3]);
    p.xs[3] = p.ys[3] = VEC;
    p.total /= (uint32_t)VEC;
  }
  k.available = true;
  return k;
}

NodeKernel prepare_red(const Node& nd, int variant, int dtype, const std::vector<Operand>& ins, const Operand& out,
                       const Operand* x1 = nullptr) {
  NodeKernel k;
  k.family = variant == 1 ? KF_RED_COL : KF_RED_ROW;
  k.dtype = dtype == FLUID_BF16 ? DT_BF16 : DT_F32;
  const Operand& x = ins[0];
  check_small(out, "reduction");
  const int r = (int)x.shape.size();
  RedParams& p = k.red;
  p.op = nd.op == FLUID_OP_SOFTMAX ? RED_SOFTMAX : nd.op == FLUID_OP_LAYERNORM ? RED_LAYERNORM : RED_RMSNORM;
  if (x1) {
    if (p.op == RED_SOFTMAX || x1->shape != x.shape) fail(FLUID_E_INVALID, "summed reduction: bad second summand");
    p.op += 2;
  }
  p.causal = nd.op == FLUID_OP_SOFTMAX ? nd.iattr : 0;
  p.attr = nd.fattr;
  p.R = (uint32_t)x.shape[r - 1];
  p.irs = (int32_t)x.stride[r - 1];
  p.ors = (int32_t)out.stride[r - 1];
  p.irs1 = x1 ? (int32_t)x1->stride[r - 1] : 0;
  p.x1 = x1 ? x1->ptr : nullptr;
  struct D { int64_t ext, is, os, is1; bool q; };
  std::vector<D> rows;
  for (int i = 0; i < r - 1; ++i) {
    bool q = p.causal && i == r - 2;
    if (x.shape[i] != 1 || q) rows.push_back({x.shape[i], x.stride[i], out.stride[i], x1 ? x1->stride[i] : 0, q});
  }
  std::stable_sort(rows.begin(), rows.end(), [](const D& a, const D& b) { return a.is > b.is; });
  if (rows.size() > (size_t)kMaxDims) fail(FLUID_E_UNSUPPORTED, "reduction rank");
  p.nrd = (int)rows.size();
  p.qdim = -1;
  uint32_t nrows = 1;
  for (int i = 0; i < p.nrd; ++i) {
    p.rext[i] = (uint32_t)rows[i].ext;
    p.rdiv[i] = make_fastdiv(p.rext[i]);
    p.ris[i] = (int32_t)rows[i].is;
    p.ros[i] = (int32_t)rows[i].os;
    p.ris1[i] = (int32_t)rows[i].is1;
    if (rows[i].q) p.qdim = i;
    nrows *= p.rext[i];
  }
  p.nrows = nrows;
  p.x = x.ptr;
  p.y = const_cast<void*>(out.ptr);
  p.gamma = ins.size() > 1 ? ins[1].ptr : nullptr;
  p.beta = ins.size() > 2 ? ins[2].ptr : nullptr;
  if (variant != 1 && p.R > 4096) { k.why = "row variants hold at most 4096 values per row"; return k; }
  if (variant != 1) {
    // 16-byte pieces: unit-stride rows starting on 16-byte boundaries
    const int VEC = k.dtype == DT_BF16 ? 8 : 4;
    bool ok = p.irs == 1 && p.ors == 1 && p.R % VEC == 0 && aligned16(p.x) && aligned16(p.y);
    for (int i = 0; i < p.nrd; ++i) ok = ok && p.ris[i] % VEC == 0 && p.ros[i] % VEC == 0;
    if (x1) {
      ok = ok && p.irs1 == 1 && aligned16(p.x1);
      for (int i = 0; i < p.nrd; ++i) ok = ok && p.ris1[i] % VEC == 0;
    }
    if (p.op != RED_SOFTMAX)
      ok = ok && aligned16(p.gamma) && (red_base_op(p.op) != RED_LAYERNORM || aligned16(p.beta));
    if (ok) k.vec = VEC;
    if (variant == 2) {
      // a workgroup per row: 16-byte pieces only, at most 4 per thread
      if (!ok) { k.why = "the workgroup-per-row variant needs unit-stride, 16-byte aligned rows"; return k; }
      k.red_block = true;
    }
  }
  k.available = true;
  return k;
}

NodeKernel prepare_gemm(const Node& nd, int variant, int dtype, const std::vector<Operand>& ins, const Operand& out) {
  NodeKernel k;
  if (packs_weight(nd.op, variant) && (nd.ins.size() != 2 || nd.ins[1] >= 0 || ins[1].shape.size() != 2)) {
    k.why = "a packed-weight variant needs a 2-D constant B operand";
    return k;
  }
  const int tile = gemm_tile_of(variant);
  k.family = KF_GEMM;
  k.dtype = dtype == FLUID_BF16 ? DT_BF16 : DT_F32;
  const Operand& A = ins[0];
  const Operand& B = ins[1];
  const Operand& C = out;
  check_small(A, "matmul");
  check_small(B, "matmul");
  check_small(C, "matmul");
  const int rA = (int)A.shape.size(), rB = (int)B.shape.size();
  GemmParams& p = k.gemm;
  p.bias = nullptr;
  p.epi_bf16 = 0;
  p.act = 0;
  p.R = nullptr;
  p.r_g1 = p.r_g2 = p.r_m1 = p.r_m2 = p.r_n = 0;
  p.rop = 0;
  p.A = A.ptr;
  p.B = B.ptr;
  p.C = const_cast<void*>(C.ptr);
  p.K = (uint32_t)A.shape[rA - 1];
  p.N = (uint32_t)B.shape[rB - 1];
  p.a_k = (int32_t)A.stride[rA - 1];
  p.b_k = (int32_t)B.stride[rB - 2];
  p.b_n = (int32_t)B.stride[rB - 1];
  p.c_n = (int32_t)C.stride[rA - 1];
  uint32_t G1 = 1, G2 = 1, M1 = 1, M2 = 1;
  p.a_g1 = p.a_g2 = p.a_m1 = p.b_g1 = p.b_g2 = p.c_g1 = p.c_g2 = p.c_m1 = 0;
  if (rB == 2) {
    if (rA == 2) {
      M2 = (uint32_t)A.shape[0];
      p.a_m2 = (int32_t)A.stride[0]; p.c_m2 = (int32_t)C.stride[0];
    } else if (rA == 3) {
      M1 = (uint32_t)A.shape[0]; M2 = (uint32_t)A.shape[1];
      p.a_m1 = (int32_t)A.stride[0]; p.a_m2 = (int32_t)A.stride[1];
      p.c_m1 = (int32_t)C.stride[0]; p.c_m2 = (int32_t)C.stride[1];
    } else if (rA == 4) {
      G1 = (uint32_t)A.shape[0]; G2 = (uint32_t)A.shape[1]; M2 = (uint32_t)A.shape[2];
      p.a_g1 = (int32_t)A.stride[0]; p.a_g2 = (int32_t)A.stride[1]; p.a_m2 = (int32_t)A.stride[2];
      p.c_g1 = (int32_t)C.stride[0]; p.c_g2 = (int32_t)C.stride[1]; p.c_m2 = (int32_t)C.stride[2];
    } else {
      fail(FLUID_E_UNSUPPORTED, "matmul rank");
    }
  } else {
    M2 = (uint32_t)A.shape[rA - 2];
    p.a_m2 = (int32_t)A.stride[rA - 2];
    p.c_m2 = (int32_t)C.stride[rA - 2];
    if (rA == 3) {
      G2 = (uint32_t)A.shape[0];
      p.a_g2 = (int32_t)A.stride[0]; p.b_g2 = (int32_t)B.stride[0]; p.c_g2 = (int32_t)C.stride[0];
    } else if (rA == 4) {
      G1 = (uint32_t)A.shape[0]; G2 = (uint32_t)A.shape[1];
      p.a_g1 = (int32_t)A.stride[0]; p.a_g2 = (int32_t)A.stride[1];
      p.b_g1 = (int32_t)B.stride[0]; p.b_g2 = (int32_t)B.stride[1];
      p.c_g1 = (int32_t)C.stride[0]; p.c_g2 = (int32_t)C.stride[1];
    } else if (rA != 2) {
      fail(FLUID_E_UNSUPPORTED, "matmul rank");
    }
  }
  p.G = G1 * G2;
  p.G2 = G2;
  p.M2 = M2;
  p.M = M1 * M2;
  // batched products only: rows are then the query dim, unmerged
  p.causal = rB >= 3 ? (uint32_t)nd.causal : 0u;
  p.g2div = make_fastdiv(G2);
  p.m2div = make_fastdiv(M2);
  const int VEC = k.dtype == DT_F32 ? 4 : 8;
  auto mult = [&](std::initializer_list<int32_t> s) {
    for (int32_t v : s)
      if (v % VEC != 0) return false;
    return true;
  };
  k.amode = GM_GENERIC;
  if (aligned16(p.A)) {
    if (p.a_k == 1 && p.K % VEC == 0 && mult({p.a_g1, p.a_g2, p.a_m1, p.a_m2})) k.amode = GM_K;
    else if (p.a_m2 == 1 && p.M2 % VEC == 0 && mult({p.a_g1, p.a_g2, p.a_m1, p.a_k})) k.amode = GM_MN;
  }
  k.bmode = GM_GENERIC;
  if (aligned16(p.B)) {
    if (p.b_n == 1 && p.N % VEC == 0 && mult({p.b_g1, p.b_g2, p.b_k})) k.bmode = GM_MN;
    else if (p.b_k == 1 && p.K % VEC == 0 && mult({p.b_g1, p.b_g2, p.b_n})) k.bmode = GM_K;
  }
  k.cmode = 0;
  if (p.c_n == 1) k.cmode = 1;
  else if (p.c_m2 == 1 && p.M2 % 4 == 0 && aligned16(p.C) && (p.c_m1 % 4 == 0) && (p.c_g1 % 4 == 0) &&
           (p.c_g2 % 4 == 0) && (p.c_n % 4 == 0))
    k.cmode = 2;
  p.cmode = k.cmode;
  const int64_t esz = k.dtype == DT_F32 ? 4 : 2;
  auto span_bytes = [&](const Operand& o) {
    int64_t s = 1;
    for (size_t d = 0; d < o.shape.size(); ++d) {
      if (o.shape[d] == 0) return int64_t(0);
      s += (o.shape[d] - 1) * o.stride[d];
    }
    return s * esz;
  };
  const int64_t sa = span_bytes(A), sb = span_bytes(B);
  p.a_bytes = (uint32_t)std::min<int64_t>(sa, 0x7fffffff);
  p.b_bytes = (uint32_t)std::min<int64_t>(sb, 0x7fffffff);
  k.gemm_tile = tile;
  // tile sizes: 0: 128x128, 1: 64x64 (LDS-staged); 2, 3: 32x32 and 4: 64x32
  // with the K range split over the workgroup's wavefronts
  // bf16 6: 256x128 and 7: 128x128, loads two or more K-tiles ahead, 8:
  // 256x128 with a three-stage ring, two workgroups per CU, 9: 128x128
  // persistent with the whole K (at most 128) in LDS;
  // fp32 6: 16x32 with K split over 8 wavefronts, 7: 32x32 over 4, operands
  // loaded straight into MFMA registers, 8 and 9: 128x128 double-buffered
  // in LDS with the next K-tile in flight in registers, over sixteen or
  // eight wavefronts
  static const uint32_t TM[] = {128, 64, 32, 32, 64, 32, 256, 128, 256, 128};
  static const uint32_t TN[] = {128, 64, 32, 32, 32, 32, 128, 128, 128, 128};
  uint32_t tm = TM[tile], tn = TN[tile];
  const bool f32 = k.dtype != DT_BF16;
  if (tile >= 8 && !f32 && (k.amode != GM_K || (k.bmode != GM_K && k.bmode != GM_MN))) {
    k.available = false;
    k.why = "bf16 tiles 8 and 9 need a K-contiguous A and a K- or N-contiguous B";
    return k;
  }
  if (tile == 9 && !f32 && p.K > 128) {
    k.available = false;
    k.why = "tile 9 holds the whole K (at most 128) in LDS";
    return k;
  }
  if (tile >= 6 && f32) {
    tm = tile == 6 ? 16 : tile == 7 ? 32 : 128;
    tn = tile >= 8 ? 128 : 32;
    if ((k.amode != GM_K && k.amode != GM_MN) || (k.bmode != GM_K && k.bmode != GM_MN)) {
      k.available = false;
      k.why = "the direct-load tiles need unit-stride K or M/N operands";
      return k;
    }
  }
  if (tile >= 6 && (sa >= 0x7fffffff || sb >= 0x7fffffff)) {
    k.available = false;
    k.why = "buffer-load tiles address at most 2 GiB per operand";
    return k;
  }
  p.tiles_m = (p.M + tm - 1) / tm;
  p.tiles_n = (p.N + tn - 1) / tn;
  k.available = true;
  return k;
}

// Pad / MaxPool: the output's four dims ordered by output stride (outermost
// first) so that consecutive threads write consecutive addresses.
NodeKernel prepare_window(const Node& nd, int dtype, const std::vector<Operand>& ins, const Operand& out) {
  NodeKernel k;
  k.family = KF_WIN;
  k.dtype = dtype == FLUID_BF16 ? DT_BF16 : DT_F32;
  const Operand& x = ins[0];
  check_small(out, "window");
  check_small(x, "window");
  WinParams& p = k.win;
  int order[4] = {0, 1, 2, 3};
  std::stable_sort(order, order + 4, [&](int a, int b) { return out.stride[a] > out.stride[b]; });
  for (int d = 0; d < 4; ++d) {
    const int l = order[d];
    p.ext[d] = (uint32_t)out.shape[l];
    p.div[d] = make_fastdiv(p.ext[d]);
    p.os[d] = (int32_t)out.stride[l];
    p.is[d] = l < 2 ? (int32_t)x.stride[l] : 0;
    p.role[d] = l < 2 ? 0 : (l == 2 ? 1 : 2);
  }
  p.in_h = (int32_t)x.shape[2];
  p.in_w = (int32_t)x.shape[3];
  p.is_h = (int32_t)x.stride[2];
  p.is_w = (int32_t)x.stride[3];
  p.total = (uint32_t)numel(out.shape);
  p.op = nd.op == FLUID_OP_PAD ? 0 : 1;
  p.k = nd.iattr;
  p.x = x.ptr;
  p.y = const_cast<void*>(out.ptr);
  k.available = true;
  return k;
}

// Conv: variant 0 reduces over (c, u, v) with wavefronts along pixels, 1
// over (u, v, c) with wavefronts along channels; variants 2 and 3 are 0 and
// 1 with the K-tiles of a tile split over 4 groups of wavefronts in one
// workgroup; variants 4 and 5 take 32 x 32 tiles with the K-tiles split
// over 8 single-wavefront groups (k_conv.hip).
NodeKernel prepare_conv(const Node& nd, int variant, int dtype, const std::vector<Operand>& ins, const Operand& out) {
  NodeKernel k;
  k.family = KF_CONV;
  k.dtype = dtype == FLUID_BF16 ? DT_BF16 : DT_F32;
  if (k.dtype != DT_F32) { k.why = "the convolution kernel is fp32"; return k; }
  const Operand& x = ins[0];
  const Operand& w = ins[1];
  check_small(x, "conv");
  check_small(out, "conv");
  check_small(w, "conv");
  const bool row_major_w = w.stride == row_major_strides(w.shape);
  if (!row_major_w || (ins.size() > 2 && ins[2].stride[0] != 1)) { k.why = "weights must be row-major"; return k; }
  ConvParams& p = k.conv;
  const uint32_t C = (uint32_t)x.shape[1], KH = (uint32_t)w.shape[2], KW = (uint32_t)w.shape[3];
  const uint32_t OH = (uint32_t)out.shape[2], OW = (uint32_t)out.shape[3];
  p.x = (const float*)x.ptr;
  p.w = (const float*)w.ptr;
  p.bias = ins.size() > 2 ? (const float*)ins[2].ptr : nullptr;
  p.y = (float*)out.ptr;
  p.M = (uint32_t)out.shape[0] * OH * OW;
  p.Co = (uint32_t)out.shape[1];
  p.C = C;
  p.K = C * KH * KW;
  p.OHW = OH * OW;
  p.OW = OW;
  p.KHW = KH * KW;
  p.KW = KW;
  p.KWC = KW * C;
  p.ohw_div = make_fastdiv(p.OHW);
  p.ow_div = make_fastdiv(OW);
  p.khw_div = make_fastdiv(p.KHW);
  p.kw_div = make_fastdiv(KW);
  p.kwc_div = make_fastdiv(p.KWC);
  p.c_div = make_fastdiv(C);
  p.x_n = (int32_t)x.stride[0]; p.x_c = (int32_t)x.stride[1]; p.x_h = (int32_t)x.stride[2]; p.x_w = (int32_t)x.stride[3];
  p.y_n = (int32_t)out.stride[0]; p.y_c = (int32_t)out.stride[1]; p.y_h = (int32_t)out.stride[2];
  p.y_w = (int32_t)out.stride[3];
  k.conv_kord = variant & 1;
  k.conv_ks = variant >= 4 ? 8 : variant >= 2 ? 4 : 1;
  k.conv_tile = variant >= 4 ? 32 : 64;
  p.tiles_n = (p.Co + k.conv_tile - 1) / k.conv_tile;
  k.available = true;
  return k;
}

}  // namespace

// Which steps pay off inside the product's launch was measured per tile
// against the product followed by separate elementwise kernels.  bf16 tile 9
// (the whole-K-in-LDS kernel for short-K attention products) has no
// registers to spare: bias only.  On the large bf16 tiles (6, 8) the epilogue runs after
// the last MFMA with nothing left to overlap it: a GELU or SiLU there costs
// 13-41 us on a 2048 x 11008 output, more than its own kernel (17-21 us),
// and the per-element reads of an Add / Mul tensor 15-75 us: bias only.  The
// Add / Mul also stays out of the 128 x 128 tiles (an instance with its
// reads drops from three to two workgroups per SIMD); on the 64 x 64, the
// split-K and the fp32 direct-load tiles every step is faster fused.
int gemm_epilogue_caps(int variant, int dtype) {
  variant = gemm_tile_of(variant);
  const bool bf16 = dtype == FLUID_BF16;
  if (bf16 && (variant == 6 || variant == 8 || variant == 9)) return EPI_BIAS;
  const bool rop = (variant >= 1 && variant <= 5) || (!bf16 && variant >= 6);
  return EPI_BIAS | EPI_ACT | (rop ? EPI_ROP : 0);
}

NodeKernel prepare_sum_norm(const Node& nd, int variant, int dtype, const std::vector<Operand>& ins, const Operand& x1,
                            const Operand& out) {
  if (nd.op != FLUID_OP_LAYERNORM && nd.op != FLUID_OP_RMSNORM) fail(FLUID_E_INVALID, "summed reduction: not a norm");
  if (variant < 0 || variant >= num_variants(nd.op)) {
    NodeKernel k;
    k.why = "no such variant";
    return k;
  }
  return prepare_red(nd, variant, dtype, ins, out, &x1);
}

NodeKernel prepare_node(const Node& nd, int variant, int dtype, const std::vector<Operand>& ins, const Operand& out) {
  if (variant < 0 || variant >= num_variants(nd.op)) {
    NodeKernel k;
    k.why = "no such variant";
    return k;
  }
  switch (nd.op) {
    case FLUID_OP_MATMUL: return prepare_gemm(nd, variant, dtype, ins, out);
    case FLUID_OP_SOFTMAX:
    case FLUID_OP_LAYERNORM:
    case FLUID_OP_RMSNORM: return prepare_red(nd, variant, dtype, ins, out);
    case FLUID_OP_ROPE: return prepare_rope(nd, dtype, ins, out);
    case FLUID_OP_PAD:
    case FLUID_OP_MAXPOOL: return prepare_window(nd, dtype, ins, out);
    case FLUID_OP_CONV: return prepare_conv(nd, variant, dtype, ins, out);
    default: return prepare_ew(nd, variant, dtype, ins, out);
  }
}

std::string NodeKernel::name() const {
  static const char* ew_names[] = {"copy", "add", "mul", "gelu", "silu", "relu"};
  static const char* red_names[] = {"softmax", "layernorm", "rmsnorm", "add_layernorm", "add_rmsnorm"};
  static const char* gm[] = {"g", "k", "mn"};
  const std::string dt = dtype == DT_BF16 ? "bf16" : "f32";
  switch (family) {
    case KF_VIEW: return "view";
    case KF_EW: return "ew_" + std::string(ew_names[ew.op]) + "_" + dt + "_v" + std::to_string(vec);
    case KF_EW_TILED: return "ew_tiled_" + std::string(ew_names[ew.op]) + "_" + dt;
    case KF_ROPE: return "rope_" + dt + (vec > 1 ? "_v" + std::to_string(vec) : "");
    case KF_RED_ROW:
      return std::string(red_names[red.op]) + (red_block ? "_rowblock_" : "_row_") + dt +
             (vec > 1 ? "_v" + std::to_string(vec) : "");
    case KF_RED_COL: return std::string(red_names[red.op]) + "_col_" + dt;
    case KF_WIN: return std::string(win.op == 0 ? "pad_" : "maxpool_") + dt;
    case KF_CONV:
      return "conv_" + dt + "_t" + std::to_string(conv_tile) + (conv_kord == 0 ? "_kcuv" : "_kuvc") +
             (conv_ks > 1 ? "_ks" + std::to_string(conv_ks) : "");
    case KF_GEMM: {
      // fused epilogue steps: b bias, g GELU, s SiLU, a / m Add / Mul of R
      auto epi_suffix = [&]() {
        std::string e = std::string(gemm.bias ? "b" : "") + (gemm.act == 1 ? "g" : gemm.act == 2 ? "s" : "") +
                        (gemm.rop == 1 ? "a" : gemm.rop == 2 ? "m" : "");
        return e.empty() ? e : "_e" + e;
      };
      static const char* tiles[] = {"t128", "t64", "sk32w4", "sk32w8", "sk64x32w4", "sk32w16", "p256x128", "p128", "p256x128s3", "q128"};
      static const char* tiles_f32[] = {"t128", "t64", "sk32w4", "sk32w8", "sk64x32w4", "sk32w16", "dl16x32w8", "dl32w4", "r128", "r128w8"};
      return "gemm_" + dt + "_" + (dtype == DT_BF16 ? tiles : tiles_f32)[gemm_tile] + "_a" + gm[amode] + "_b" + gm[bmode] + "_c" +
             (cmode == 1 ? "n" : cmode == 2 ? "m" : "g") + (gemm.causal ? "_causal" + std::to_string(gemm.causal) : "") +
             epi_suffix();
    }
  }
  return "?";
}

}  // namespace fluid
