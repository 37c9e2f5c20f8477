// Graph validation, shape checks, transformer builders and canonical export.
#include "graph.h"

#include <algorithm>
#include <cmath>
#include <cstdio>
#include <sstream>

#include "layouts.h"

namespace fluid {

std::string shape_str(const Shape& s) {
  std::string r = "[";
  for (size_t i = 0; i < s.size(); ++i) r += (i ? "," : "") + std::to_string(s[i]);
  return r + "]";
}

const char* op_name(int op) {
  static const char* names[] = {"matmul", "add",     "mul",     "transpose", "reshape", "softmax", "layernorm",
                                "rmsnorm", "gelu",    "silu",    "rope",      "pad",     "conv",    "relu",
                                "maxpool"};
  return (op >= 0 && op <= FLUID_OP_MAXPOOL) ? names[op] : "?";
}

ReshapeKind reshape_kind(const Shape& xs, const Shape& ys, int* axis) {
  *axis = -1;
  if (xs == ys) return ReshapeKind::Same;
  size_t rx = xs.size(), ry = ys.size();
  if (ry == rx + 1) {
    for (size_t a = 0; a < rx; ++a) {
      bool ok = ys[a] * ys[a + 1] == xs[a];
      for (size_t i = 0; ok && i < a; ++i) ok = ys[i] == xs[i];
      for (size_t i = a + 1; ok && i < rx; ++i) ok = ys[i + 1] == xs[i];
      if (ok) { *axis = (int)a; return ReshapeKind::Split; }
    }
  }
  if (rx == ry + 1) {
    for (size_t a = 0; a < ry; ++a) {
      bool ok = xs[a] * xs[a + 1] == ys[a];
      for (size_t i = 0; ok && i < a; ++i) ok = xs[i] == ys[i];
      for (size_t i = a + 1; ok && i < ry; ++i) ok = xs[i + 1] == ys[i];
      if (ok) { *axis = (int)a; return ReshapeKind::Merge; }
    }
  }
  return ReshapeKind::Other;
}

namespace {

void check_shape(const Shape& s, const std::string& what) {
  require(!s.empty() && s.size() <= FLUID_MAX_RANK, what + ": rank must be 1.." + std::to_string(FLUID_MAX_RANK));
  for (int64_t d : s) require(d >= 1, what + ": dims must be >= 1, got " + shape_str(s));
  require(numel(s) < (int64_t(1) << 40), what + ": tensor too large");
}

}  // namespace

void Graph::finalize() {
  require(dtype == FLUID_F32 || dtype == FLUID_BF16, "graph dtype must be F32 or BF16");
  require(!inputs.empty(), "graph needs at least one input");
  require(!nodes.empty(), "graph needs at least one node");
  for (size_t i = 0; i < inputs.size(); ++i) check_shape(inputs[i], "input " + std::to_string(i));
  for (size_t i = 0; i < consts.size(); ++i) {
    check_shape(consts[i].shape, "const " + std::to_string(i));
    require(consts[i].dtype == FLUID_F32 || consts[i].dtype == FLUID_BF16, "const dtype");
  }
  const int E = n_edges();
  act_in.assign(nodes.size(), {});
  for (size_t n = 0; n < nodes.size(); ++n) {
    const Node& nd = nodes[n];
    std::string where = "node " + std::to_string(n) + " (" + op_name(nd.op) + ")";
    require(nd.op >= 0 && nd.op <= FLUID_OP_MAXPOOL, where + ": unknown op");
    check_shape(nd.out_shape, where + " output");
    const int self = out_edge((int)n);
    std::vector<const Shape*> in_shapes;
    std::vector<bool> in_const;
    for (int v : nd.ins) {
      if (v >= 0) {
        require(v < self, where + ": input edge " + std::to_string(v) + " is not produced earlier");
        act_in[n].push_back(v);
        in_shapes.push_back(&edge_shape(v));
        in_const.push_back(false);
      } else {
        int c = ~v;
        require(c < (int)consts.size(), where + ": constant id out of range");
        in_shapes.push_back(&consts[c].shape);
        in_const.push_back(true);
      }
    }
    auto arity = [&](size_t k) {
      require(nd.ins.size() == k, where + ": expects " + std::to_string(k) + " inputs");
    };
    auto act = [&](size_t i) { require(!in_const[i], where + ": input " + std::to_string(i) + " must be an activation"); };
    auto cst = [&](size_t i) { require(in_const[i], where + ": input " + std::to_string(i) + " must be a constant"); };
    const Shape& y = nd.out_shape;
    switch (nd.op) {
      case FLUID_OP_MATMUL: {
        arity(2); act(0);
        const Shape& a = *in_shapes[0];
        const Shape& b = *in_shapes[1];
        require(a.size() >= 2 && b.size() >= 2, where + ": operands need rank >= 2");
        require(a[a.size() - 1] == b[b.size() - 2], where + ": inner dims differ");
        if (b.size() != 2) {
          act(1);
          require(b.size() == a.size(), where + ": batched B must have A's rank");
          for (size_t i = 0; i + 2 < a.size(); ++i) require(a[i] == b[i], where + ": batch dims differ");
        }
        Shape want(a.begin(), a.end() - 1);
        want.push_back(b.back());
        require(y == want, where + ": output shape must be " + shape_str(want));
        break;
      }
      case FLUID_OP_ADD:
      case FLUID_OP_MUL: {
        arity(2); act(0);
        const Shape& a = *in_shapes[0];
        const Shape& b = *in_shapes[1];
        require(y == a, where + ": output shape must equal input 0");
        bool bias = b.size() == 1 && b[0] == a.back();
        if (nd.op == FLUID_OP_MUL || b.size() != 1 || a.size() == 1) {
          act(1);
          require(b == a, where + ": operands must have equal shapes");
        } else {
          cst(1);
          require(bias, where + ": bias must be [last dim]");
        }
        break;
      }
      case FLUID_OP_TRANSPOSE: {
        arity(1); act(0);
        const Shape& a = *in_shapes[0];
        require(nd.perm.size() == a.size(), where + ": perm rank");
        std::vector<int> seen(a.size(), 0);
        for (int p : nd.perm) {
          require(p >= 0 && p < (int)a.size() && !seen[p], where + ": perm must be a permutation");
          seen[p] = 1;
        }
        for (size_t i = 0; i < a.size(); ++i) require(y[i] == a[nd.perm[i]], where + ": output shape");
        require(y.size() == a.size(), where + ": output rank");
        break;
      }
      case FLUID_OP_RESHAPE: {
        arity(1); act(0);
        require(numel(y) == numel(*in_shapes[0]), where + ": element count differs");
        int ax;
        if (reshape_kind(*in_shapes[0], y, &ax) == ReshapeKind::Other)
          fail(FLUID_E_UNSUPPORTED, where + ": only split-one-dim / merge-two-adjacent-dims reshapes");
        break;
      }
      case FLUID_OP_SOFTMAX:
        arity(1); act(0);
        require(y == *in_shapes[0], where + ": output shape");
        require(y.size() >= 2 || nd.iattr == 0, where + ": causal needs rank >= 2");
        require(std::isfinite(nd.fattr), where + ": scale must be finite");
        break;
      case FLUID_OP_LAYERNORM:
      case FLUID_OP_RMSNORM: {
        size_t k = nd.op == FLUID_OP_LAYERNORM ? 3 : 2;
        arity(k); act(0);
        require(y == *in_shapes[0], where + ": output shape");
        for (size_t i = 1; i < k; ++i) {
          cst(i);
          require(in_shapes[i]->size() == 1 && (*in_shapes[i])[0] == y.back(), where + ": scale/shift must be [H]");
        }
        require(nd.fattr > 0.f && std::isfinite(nd.fattr), where + ": eps must be positive");
        break;
      }
      case FLUID_OP_GELU:
      case FLUID_OP_SILU:
      case FLUID_OP_RELU:
        arity(1); act(0);
        require(y == *in_shapes[0], where + ": output shape");
        break;
      case FLUID_OP_PAD: {
        arity(1); act(0);
        const Shape& a = *in_shapes[0];
        require(a.size() == 4, where + ": input must be [N, C, H, W]");
        require(nd.iattr >= 0, where + ": pad width must be >= 0");
        const int64_t p = nd.iattr;
        require(y == Shape({a[0], a[1], a[2] + 2 * p, a[3] + 2 * p}), where + ": output shape");
        break;
      }
      case FLUID_OP_CONV: {
        require(nd.ins.size() == 2 || nd.ins.size() == 3, where + ": expects 2 or 3 inputs");
        act(0); cst(1);
        const Shape& a = *in_shapes[0];
        const Shape& w = *in_shapes[1];
        require(a.size() == 4 && w.size() == 4, where + ": input [N, C, H, W] and weight [Co, C, KH, KW]");
        require(w[1] == a[1] && w[2] <= a[2] && w[3] <= a[3], where + ": weight does not fit the input");
        require(consts[~nd.ins[1]].dtype == dtype, where + ": weight dtype must be the graph's");
        if (nd.ins.size() == 3) {
          cst(2);
          require(*in_shapes[2] == Shape({w[0]}), where + ": bias must be [Co]");
          require(consts[~nd.ins[2]].dtype == dtype, where + ": bias dtype must be the graph's");
        }
        require(y == Shape({a[0], w[0], a[2] - w[2] + 1, a[3] - w[3] + 1}), where + ": output shape");
        break;
      }
      case FLUID_OP_MAXPOOL: {
        arity(1); act(0);
        const Shape& a = *in_shapes[0];
        const int64_t k = nd.iattr;
        require(a.size() == 4 && k >= 1 && a[2] % k == 0 && a[3] % k == 0,
                where + ": input [N, C, H, W] with H and W multiples of the window");
        require(y == Shape({a[0], a[1], a[2] / k, a[3] / k}), where + ": output shape");
        break;
      }
      case FLUID_OP_ROPE: {
        arity(3); act(0); cst(1); cst(2);
        const Shape& a = *in_shapes[0];
        require(a.size() == 4 && a[3] % 2 == 0, where + ": input must be [B,S,NH,D] with even D");
        require(y == a, where + ": output shape");
        Shape tab = {a[1], a[3] / 2};
        for (int i = 1; i <= 2; ++i) {
          require(*in_shapes[i] == tab, where + ": tables must be [S, D/2]");
          require(consts[~nd.ins[i]].dtype == FLUID_F32, where + ": tables must be fp32");
        }
        break;
      }
    }
  }
  require(!outputs.empty(), "graph needs at least one output");
  is_output.assign(E, 0);
  for (int e : outputs) {
    require(e >= n_inputs() && e < E, "outputs must be node outputs");
    require(!is_output[e], "duplicate output edge");
    is_output[e] = 1;
  }
  readers.assign(E, {});
  for (size_t n = 0; n < nodes.size(); ++n)
    for (int e : act_in[n])
      if (readers[e].empty() || readers[e].back() != (int)n) readers[e].push_back((int)n);
  const_readers.assign(consts.size(), {});
  for (size_t n = 0; n < nodes.size(); ++n)
    for (int v : nodes[n].ins)
      if (v < 0 && (const_readers[~v].empty() || const_readers[~v].back() != (int)n)) const_readers[~v].push_back((int)n);
  cand.assign(E, {});
  for (int e = 0; e < E; ++e)
    cand[e] = pinned(e) ? std::vector<Perm>{identity_perm((int)edge_shape(e).size())} : layout_list(edge_shape(e));
  // Causal attention products.  A causal softmax reads only the entries of
  // its input on or below the diagonal (key <= query, the last two dims),
  // and writes exact zeros above it.
  auto causal_softmax = [&](int m) { return m >= 0 && nodes[m].op == FLUID_OP_SOFTMAX && nodes[m].iattr != 0; };
  for (size_t n = 0; n < nodes.size(); ++n) {
    Node& nd = nodes[n];
    nd.causal = 0;
    if (nd.op != FLUID_OP_MATMUL || nd.ins[0] < 0 || nd.ins[1] < 0 || edge_shape(nd.ins[1]).size() < 3) continue;
    const int e = out_edge((int)n);
    if (!is_output[e] && readers[e].size() == 1 && causal_softmax(readers[e][0])) nd.causal |= 1;
    if (causal_softmax(producer(nd.ins[0]))) nd.causal |= 2;
  }
}

// ------------------------------------------------------------ transformers
namespace {

struct Builder {
  Graph& g;
  int add_const(int role, Shape s, int dt) {
    g.consts.push_back({std::move(s), dt, role});
    return ~(int)(g.consts.size() - 1);
  }
  int add(int op, std::vector<int> ins, Shape out, Perm perm = {}, float f = 0.f, int i = 0) {
    Node nd;
    nd.op = op;
    nd.ins = std::move(ins);
    nd.out_shape = std::move(out);
    nd.perm = std::move(perm);
    nd.fattr = f;
    nd.iattr = i;
    g.nodes.push_back(std::move(nd));
    return g.out_edge((int)g.nodes.size() - 1);
  }
};

}  // namespace

namespace {

// VGG-shaped convolutional network (arch 3): Pad, 3x3 Conv with bias, ReLU
// per convolution; MaxPool(2) per stage; flatten; three classifier layers.
Graph build_vgg(const fluid_model_cfg& c) {
  require(c.batch >= 1 && c.channels >= 1 && c.image >= 1 && c.fc >= 1 && c.classes >= 1,
          "model sizes must be positive");
  require(c.n_stages >= 1 && c.n_stages <= FLUID_MAX_STAGES, "n_stages must be 1..FLUID_MAX_STAGES");
  require(c.dtype == FLUID_F32, "the convolutional network is fp32");
  Graph g;
  g.dtype = c.dtype;
  Builder b{g};
  const int dt = c.dtype;
  const int64_t B = c.batch;
  int64_t C = c.channels, S = c.image;
  g.inputs.push_back({B, C, S, S});
  int e = 0;
  for (int s = 0; s < c.n_stages; ++s) {
    const int64_t Wd = c.stage_width[s];
    require(Wd >= 1 && c.stage_convs[s] >= 1, "stage widths and counts must be positive");
    for (int k = 0; k < c.stage_convs[s]; ++k) {
      int p = b.add(FLUID_OP_PAD, {e}, {B, C, S + 2, S + 2}, {}, 0.f, 1);
      int w = b.add_const(FLUID_ROLE_WEIGHT, {Wd, C, 3, 3}, dt);
      int bi = b.add_const(FLUID_ROLE_BIAS, {Wd}, dt);
      int cv = b.add(FLUID_OP_CONV, {p, w, bi}, {B, Wd, S, S});
      e = b.add(FLUID_OP_RELU, {cv}, {B, Wd, S, S});
      C = Wd;
    }
    require(S % 2 == 0, "every stage's image size must be even");
    e = b.add(FLUID_OP_MAXPOOL, {e}, {B, C, S / 2, S / 2}, {}, 0.f, 2);
    S /= 2;
  }
  e = b.add(FLUID_OP_RESHAPE, {e}, {B, C, S * S});
  e = b.add(FLUID_OP_RESHAPE, {e}, {B, C * S * S});
  int64_t K = C * S * S;
  const int64_t widths[3] = {c.fc, c.fc, c.classes};
  for (int i = 0; i < 3; ++i) {
    const int64_t N = widths[i];
    e = b.add(FLUID_OP_MATMUL, {e, b.add_const(FLUID_ROLE_WEIGHT, {K, N}, dt)}, {B, N});
    e = b.add(FLUID_OP_ADD, {e, b.add_const(FLUID_ROLE_BIAS, {N}, dt)}, {B, N});
    if (i < 2) e = b.add(FLUID_OP_RELU, {e}, {B, N});
    K = N;
  }
  e = b.add(FLUID_OP_SOFTMAX, {e}, {B, (int64_t)c.classes}, {}, 1.0f, 0);
  g.outputs = {e};
  g.finalize();
  return g;
}

}  // namespace

Graph build_transformer(const fluid_model_cfg& c) {
  if (c.arch == 3) return build_vgg(c);
  require(c.arch >= 0 && c.arch <= 2, "arch must be 0 (post-LN), 1 (pre-LN), 2 (Llama) or 3 (VGG-shaped)");
  require(c.layers >= 1 && c.batch >= 1 && c.seq >= 1 && c.hidden >= 1 && c.heads >= 1 && c.ffn >= 1,
          "model sizes must be positive");
  require(c.hidden % c.heads == 0, "hidden must be a multiple of heads");
  require(c.dtype == FLUID_F32 || c.dtype == FLUID_BF16, "dtype");
  const int64_t B = c.batch, S = c.seq, H = c.hidden, NH = c.heads, F = c.ffn, D = H / NH;
  require(c.arch != 2 || D % 2 == 0, "RoPE needs an even head dim");
  Graph g;
  g.dtype = c.dtype;
  Builder b{g};
  const int dt = c.dtype;
  g.inputs.push_back({B, S, H});
  int x = 0;
  int cosc = 0, sinc = 0;
  if (c.arch == 2) {
    cosc = b.add_const(FLUID_ROLE_ROPE_COS, {S, D / 2}, FLUID_F32);
    sinc = b.add_const(FLUID_ROLE_ROPE_SIN, {S, D / 2}, FLUID_F32);
  }
  const float scale = (float)(1.0 / std::sqrt((double)D));
  const float eps = c.eps;
  auto attention = [&](int h, int causal, bool bias, bool rope) {
    int heads[3];
    for (int p = 0; p < 3; ++p) {
      int w = b.add_const(FLUID_ROLE_WEIGHT, {H, H}, dt);
      int e = b.add(FLUID_OP_MATMUL, {h, w}, {B, S, H});
      if (bias) e = b.add(FLUID_OP_ADD, {e, b.add_const(FLUID_ROLE_BIAS, {H}, dt)}, {B, S, H});
      e = b.add(FLUID_OP_RESHAPE, {e}, {B, S, NH, D});
      if (rope && p != 2) e = b.add(FLUID_OP_ROPE, {e, cosc, sinc}, {B, S, NH, D});
      if (p == 1)
        e = b.add(FLUID_OP_TRANSPOSE, {e}, {B, NH, D, S}, {0, 2, 3, 1});
      else
        e = b.add(FLUID_OP_TRANSPOSE, {e}, {B, NH, S, D}, {0, 2, 1, 3});
      heads[p] = e;
    }
    int s = b.add(FLUID_OP_MATMUL, {heads[0], heads[1]}, {B, NH, S, S});
    int pr = b.add(FLUID_OP_SOFTMAX, {s}, {B, NH, S, S}, {}, scale, causal);
    int cx = b.add(FLUID_OP_MATMUL, {pr, heads[2]}, {B, NH, S, D});
    int c1 = b.add(FLUID_OP_TRANSPOSE, {cx}, {B, S, NH, D}, {0, 2, 1, 3});
    return b.add(FLUID_OP_RESHAPE, {c1}, {B, S, H});
  };
  auto ffn_gelu = [&](int h) {
    int f0 = b.add(FLUID_OP_MATMUL, {h, b.add_const(FLUID_ROLE_WEIGHT, {H, F}, dt)}, {B, S, F});
    int f1 = b.add(FLUID_OP_ADD, {f0, b.add_const(FLUID_ROLE_BIAS, {F}, dt)}, {B, S, F});
    int f2 = b.add(FLUID_OP_GELU, {f1}, {B, S, F});
    int f3 = b.add(FLUID_OP_MATMUL, {f2, b.add_const(FLUID_ROLE_WEIGHT, {F, H}, dt)}, {B, S, H});
    return b.add(FLUID_OP_ADD, {f3, b.add_const(FLUID_ROLE_BIAS, {H}, dt)}, {B, S, H});
  };
  auto layernorm = [&](int e) {
    int gm = b.add_const(FLUID_ROLE_GAMMA, {H}, dt);
    int bt = b.add_const(FLUID_ROLE_BETA, {H}, dt);
    return b.add(FLUID_OP_LAYERNORM, {e, gm, bt}, {B, S, H}, {}, eps);
  };
  auto rmsnorm = [&](int e) {
    return b.add(FLUID_OP_RMSNORM, {e, b.add_const(FLUID_ROLE_GAMMA, {H}, dt)}, {B, S, H}, {}, eps);
  };
  for (int l = 0; l < c.layers; ++l) {
    if (c.arch == 0) {
      int c2 = attention(x, 0, true, false);
      int o0 = b.add(FLUID_OP_MATMUL, {c2, b.add_const(FLUID_ROLE_WEIGHT, {H, H}, dt)}, {B, S, H});
      int o1 = b.add(FLUID_OP_ADD, {o0, b.add_const(FLUID_ROLE_BIAS, {H}, dt)}, {B, S, H});
      int r1 = b.add(FLUID_OP_ADD, {o1, x}, {B, S, H});
      int h1 = layernorm(r1);
      int f4 = ffn_gelu(h1);
      int r2 = b.add(FLUID_OP_ADD, {f4, h1}, {B, S, H});
      x = layernorm(r2);
    } else if (c.arch == 1) {
      int h0 = layernorm(x);
      int c2 = attention(h0, 1, true, false);
      int o0 = b.add(FLUID_OP_MATMUL, {c2, b.add_const(FLUID_ROLE_WEIGHT, {H, H}, dt)}, {B, S, H});
      int o1 = b.add(FLUID_OP_ADD, {o0, b.add_const(FLUID_ROLE_BIAS, {H}, dt)}, {B, S, H});
      int r1 = b.add(FLUID_OP_ADD, {o1, x}, {B, S, H});
      int h1 = layernorm(r1);
      int f4 = ffn_gelu(h1);
      x = b.add(FLUID_OP_ADD, {f4, r1}, {B, S, H});
    } else {
      int h0 = rmsnorm(x);
      int c2 = attention(h0, 1, false, true);
      int o0 = b.add(FLUID_OP_MATMUL, {c2, b.add_const(FLUID_ROLE_WEIGHT, {H, H}, dt)}, {B, S, H});
      int r1 = b.add(FLUID_OP_ADD, {o0, x}, {B, S, H});
      int h1 = rmsnorm(r1);
      const int wg = b.add_const(FLUID_ROLE_WEIGHT, {H, F}, dt);
      const int wu = b.add_const(FLUID_ROLE_WEIGHT, {H, F}, dt);
      int gg = b.add(FLUID_OP_MATMUL, {h1, wg}, {B, S, F});
      int sg = b.add(FLUID_OP_SILU, {gg}, {B, S, F});
      int uu = b.add(FLUID_OP_MATMUL, {h1, wu}, {B, S, F});
      int m = b.add(FLUID_OP_MUL, {sg, uu}, {B, S, F});
      int d = b.add(FLUID_OP_MATMUL, {m, b.add_const(FLUID_ROLE_WEIGHT, {F, H}, dt)}, {B, S, H});
      x = b.add(FLUID_OP_ADD, {d, r1}, {B, S, H});
    }
  }
  if (c.arch == 1) x = layernorm(x);
  if (c.arch == 2) x = rmsnorm(x);
  g.outputs = {x};
  g.finalize();
  return g;
}

// ------------------------------------------------------------ export
namespace {

const char* role_name(int r) {
  static const char* names[] = {"other", "weight", "bias", "gamma", "beta", "rope_cos", "rope_sin"};
  return (r >= 0 && r <= 6) ? names[r] : "other";
}

void put_shape(std::ostringstream& o, const Shape& s) {
  o << '[';
  for (size_t i = 0; i < s.size(); ++i) o << (i ? ", " : "") << s[i];
  o << ']';
}

void put_float(std::ostringstream& o, float f) {
  // shortest round-trip text of the float32 value as a double
  char buf[64];
  double d = (double)f;
  for (int prec = 1; prec <= 17; ++prec) {
    std::snprintf(buf, sizeof buf, "%.*g", prec, d);
    if (std::strtod(buf, nullptr) == d) break;
  }
  std::string s = buf;
  if (s.find_first_of(".eEn") == std::string::npos) s += ".0";
  o << s;
}

}  // namespace

std::string Graph::export_json() const {
  std::ostringstream o;
  o << "{\"dtype\": \"" << (dtype == FLUID_BF16 ? "bf16" : "f32") << "\", \"inputs\": [";
  for (size_t i = 0; i < inputs.size(); ++i) { if (i) o << ", "; put_shape(o, inputs[i]); }
  o << "], \"consts\": [";
  for (size_t i = 0; i < consts.size(); ++i) {
    if (i) o << ", ";
    o << "{\"role\": \"" << role_name(consts[i].role) << "\", \"shape\": ";
    put_shape(o, consts[i].shape);
    o << ", \"dtype\": \"" << (consts[i].dtype == FLUID_BF16 ? "bf16" : "f32") << "\"}";
  }
  o << "], \"nodes\": [";
  for (size_t n = 0; n < nodes.size(); ++n) {
    const Node& nd = nodes[n];
    if (n) o << ", ";
    o << "{\"op\": \"" << op_name(nd.op) << "\", \"ins\": [";
    for (size_t i = 0; i < nd.ins.size(); ++i) o << (i ? ", " : "") << nd.ins[i];
    o << "], \"out_shape\": ";
    put_shape(o, nd.out_shape);
    o << ", \"perm\": [";
    for (size_t i = 0; i < nd.perm.size(); ++i) o << (i ? ", " : "") << nd.perm[i];
    o << "], \"fattr\": ";
    put_float(o, nd.fattr);
    o << ", \"iattr\": " << nd.iattr << "}";
  }
  o << "], \"outputs\": [";
  for (size_t i = 0; i < outputs.size(); ++i) o << (i ? ", " : "") << outputs[i];
  o << "], \"layouts\": [";
  for (size_t e = 0; e < cand.size(); ++e) {
    if (e) o << ", ";
    o << '[';
    for (size_t k = 0; k < cand[e].size(); ++k) {
      if (k) o << ", ";
      o << '[';
      for (size_t i = 0; i < cand[e][k].size(); ++i) o << (i ? ", " : "") << cand[e][k][i];
      o << ']';
    }
    o << ']';
  }
  o << "]}";
  return o.str();
}

}  // namespace fluid
