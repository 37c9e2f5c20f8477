// GPU entry points of the C ABI: the executor (fluid_run), the cost-table
// measurement (fluid_measure_costs) and per-node tracing.
//
// fluid_run is the paper's VM invoke path (Section 4): every non-view node
// becomes one kernel launch, in node order, on the caller's stream, with
// all activations inside the caller's single arena at their planned
// offsets -- except the nodes a MatMul performs in its epilogue
// (prepare.cpp).  The launch parameters depend only on the graph and the
// two plans, so they are prepared once per (layout plan, arena plan) pair
// and cached; each call only patches the base addresses.
#include <algorithm>
#include <cmath>
#include <cstring>
#include <map>
#include <memory>
#include <mutex>
#include <tuple>
#include <vector>

#include "../host/fusion.h"
#include "../host/handles.h"
#include "../host/layouts.h"
#include "../host/prepare.h"
#include "launch.h"

namespace fluid {

namespace {

std::mutex g_cache_mu;

struct Bases {
  char* arena;
  const void* const* inputs;
  void* const* outputs;
  const void* const* consts;
};

inline void* resolve(const Bind& b, const Bases& B) {
  switch (b.kind) {
    case BK_ARENA: return B.arena + b.off;
    case BK_INPUT: return const_cast<void*>(B.inputs[b.index]);
    case BK_OUTPUT: return B.outputs[b.index];
    default: return const_cast<void*>(B.consts[b.index]);
  }
}

void patch(NodeKernel& k, const PreparedNode& pn, const Bases& B) {
  void* out = resolve(pn.out, B);
  void* in0 = resolve(pn.in[0], B);
  void* in1 = pn.in.size() > 1 ? resolve(pn.in[1], B) : nullptr;
  void* in2 = pn.in.size() > 2 ? resolve(pn.in[2], B) : nullptr;
  switch (k.family) {
    case KF_EW:
    case KF_EW_TILED:
      k.ew.x0 = in0; k.ew.x1 = in1; k.ew.y = out;
      break;
    case KF_ROPE:
      k.rope.x = in0; k.rope.cos_t = (const float*)in1; k.rope.sin_t = (const float*)in2; k.rope.y = out;
      break;
    case KF_RED_ROW:
    case KF_RED_COL:
      k.red.x = in0; k.red.gamma = in1; k.red.beta = in2; k.red.y = out;
      break;
    case KF_GEMM:
      k.gemm.A = in0; k.gemm.B = in1; k.gemm.C = out;
      break;
    case KF_WIN:
      k.win.x = in0; k.win.y = out;
      break;
    case KF_CONV:
      k.conv.x = (const float*)in0; k.conv.w = (const float*)in1; k.conv.bias = (const float*)in2;
      k.conv.y = (float*)out;
      break;
    default:
      break;
  }
}

// The fused launch of pn (fuse_n > 0): the MatMul and its epilogue, or the
// normalisation of the sum a residual Add forms.
NodeKernel fused_kernel(const PreparedNode& pn, const Bases& B) {
  NodeKernel k = pn.kf;
  if (k.family == KF_RED_ROW || k.family == KF_RED_COL) {
    k.red.x = resolve(pn.in[0], B);
    k.red.x1 = resolve(pn.in[1], B);
    k.red.gamma = pn.fgamma >= 0 ? B.consts[pn.fgamma] : nullptr;
    k.red.beta = pn.fbeta >= 0 ? B.consts[pn.fbeta] : nullptr;
    k.red.y = resolve(pn.fout, B);
    k.red.h = pn.fstore ? resolve(pn.out, B) : nullptr;
    return k;
  }
  k.gemm.A = resolve(pn.in[0], B);
  k.gemm.B = resolve(pn.in[1], B);
  k.gemm.C = resolve(pn.fout, B);
  k.gemm.bias = pn.fbias >= 0 ? B.consts[pn.fbias] : nullptr;
  k.gemm.R = k.gemm.rop ? resolve(pn.fr, B) : nullptr;
  return k;
}

// The prepared launch of pn (the launch of its whole chain when it has
// absorbed the nodes after it).
NodeKernel launch_kernel(const PreparedNode& pn, const Bases& B) {
  if (pn.fuse_n) return fused_kernel(pn, B);
  NodeKernel k = pn.k;
  patch(k, pn, B);
  return k;
}

// One launch of pn's product (kernel k) and the products grouped with it.
hipError_t launch_group(const Prepared& P, const PreparedNode& pn, const NodeKernel& k, const Bases& B,
                        hipStream_t s) {
  GemmGroup G{};
  G.n = 1 + (uint32_t)pn.group.size();
  G.p[0] = k.gemm;
  G.tiles[0] = 0;
  G.tiles[1] = k.gemm.tiles_m * k.gemm.tiles_n * k.gemm.G;
  for (size_t t = 0; t < pn.group.size(); ++t) {
    const GemmParams q = launch_kernel(P.nodes[pn.group[t]], B).gemm;
    G.p[t + 1] = q;
    G.tiles[t + 2] = G.tiles[t + 1] + q.tiles_m * q.tiles_n * q.G;
  }
  return launch_gemm_f32_dl_group(k, G, s);
}

// ------------------------------------------------------------ tracing
struct Trace {
  bool on = false;
  std::vector<uint8_t> mask;
  std::vector<hipEvent_t> ev;  // 2 per record
  std::vector<int> node_of;    // per used record
  int max_records = 0;
  uint64_t graph_serial = 0;
};
std::mutex g_trace_mu;
Trace g_trace;

void hip_check(hipError_t e, const char* what) {
  if (e != hipSuccess) fail(FLUID_E_HIP, std::string(what) + ": " + hipGetErrorString(e));
}

bool aligned(const void* p, uintptr_t a) { return ((uintptr_t)p & (a - 1)) == 0; }

}  // namespace

// ------------------------------------------------------------ measurement
namespace {

struct SigKey {
  int op;
  float f;
  int i;
  Perm perm;
  std::vector<Shape> in_shapes;   // activation slots
  std::vector<Shape> const_shapes;
  std::vector<int> const_dtypes;
  std::vector<int> slot_is_const; // per input position
  Shape out;
  bool operator<(const SigKey& o) const {
    return std::tie(op, f, i, perm, in_shapes, const_shapes, const_dtypes, slot_is_const, out) <
           std::tie(o.op, o.f, o.i, o.perm, o.in_shapes, o.const_shapes, o.const_dtypes, o.slot_is_const, o.out);
  }
};

SigKey sig_key(const Graph& g, int n) {
  const Node& nd = g.nodes[n];
  SigKey k;
  k.op = nd.op;
  k.f = nd.fattr;
  k.i = nd.iattr;
  k.perm = nd.perm;
  for (int v : nd.ins) {
    k.slot_is_const.push_back(v < 0);
    if (v >= 0) {
      k.in_shapes.push_back(g.edge_shape(v));
    } else {
      k.const_shapes.push_back(g.consts[~v].shape);
      k.const_dtypes.push_back(g.consts[~v].dtype);
    }
  }
  k.out = nd.out_shape;
  return k;
}

uint64_t align256(uint64_t x) { return (x + 255) & ~uint64_t(255); }

}  // namespace

}  // namespace fluid

using namespace fluid;

namespace {

std::shared_ptr<Prepared> cached_prepared(const fluid_graph* gh, const fluid_layout_plan* lh,
                                          const fluid_arena_plan* ah);

// Argument checks shared by fluid_run and fluid_run_nodes, then the cached
// launch parameters of the (layout plan, arena plan) pair.
std::shared_ptr<Prepared> checked_prepared(const fluid_graph* gh, const fluid_layout_plan* lh,
                                           const fluid_arena_plan* ah, void* arena, uint64_t arena_bytes,
                                           const void* const* consts, const void* const* inputs,
                                           void* const* outputs, const char* fn) {
  const std::string f(fn);
  require(gh && lh && ah, f + ": NULL graph or plan");
  const Graph& g = gh->g;
  require(lh->p.graph_serial == gh->serial && ah->a.graph_serial == gh->serial, f + ": plans belong to another graph");
  require(ah->a.root.size() == (size_t)g.n_edges(), f + ": arena plan size mismatch");
  if (ah->a.peak > 0) {
    require(arena != nullptr, f + ": NULL arena");
    require(aligned(arena, 256), f + ": arena must be 256-byte aligned");
  }
  if (arena_bytes < ah->a.peak)
    fail(FLUID_E_ARENA_TOO_SMALL, f + ": arena has " + std::to_string(arena_bytes) + " bytes, plan needs " +
                                      std::to_string(ah->a.peak));
  require(inputs && outputs, f + ": NULL inputs/outputs array");
  require(consts || g.consts.empty(), f + ": NULL consts array");
  for (int i = 0; i < g.n_inputs(); ++i)
    require(inputs[i] && aligned(inputs[i], 16), f + ": input " + std::to_string(i) + " is NULL or not 16-byte aligned");
  for (size_t i = 0; i < g.outputs.size(); ++i)
    require(outputs[i] && aligned(outputs[i], 16), f + ": output " + std::to_string(i) + " is NULL or not 16-byte aligned");
  for (size_t i = 0; i < g.consts.size(); ++i)
    require(consts[i] && aligned(consts[i], 16), f + ": const " + std::to_string(i) + " is NULL or not 16-byte aligned");
  return cached_prepared(gh, lh, ah);
}

std::shared_ptr<Prepared> cached_prepared(const fluid_graph* gh, const fluid_layout_plan* lh,
                                          const fluid_arena_plan* ah) {
  std::lock_guard<std::mutex> lk(g_cache_mu);
  // plan serials are never reused, so a stale entry can never match
  static std::map<std::pair<uint64_t, uint64_t>, std::shared_ptr<Prepared>> cache;
  auto key = std::make_pair(lh->serial, ah->serial);
  auto it = cache.find(key);
  if (it != cache.end()) return it->second;
  auto prep = prepare(gh->g, lh->p, &ah->a);
  if (cache.size() > 256) cache.clear();
  cache[key] = prep;
  return prep;
}

// Enqueues the launches of a prepared run (fluid_run, fluid_run_static).
void run_prepared(const fluid_graph* gh, const Prepared& prep, const Bases& B, hipStream_t s) {
  std::unique_lock<std::mutex> tl(g_trace_mu);
  const bool tracing = g_trace.on && g_trace.graph_serial == gh->serial;
  if (!tracing) tl.unlock();
  for (const PreparedNode& pn : prep.nodes) {
    if (pn.fused_away || pn.grouped) continue;  // launched with an earlier node
    const NodeKernel k = launch_kernel(pn, B);
    int rec = -1;
    if (tracing && g_trace.mask[pn.node] && (int)g_trace.node_of.size() < g_trace.max_records) {
      rec = (int)g_trace.node_of.size();
      g_trace.node_of.push_back(pn.node);
      hip_check(hipEventRecord(g_trace.ev[2 * rec], s), "hipEventRecord");
    }
    const hipError_t e = pn.group.empty() ? launch_node_kernel(k, s) : launch_group(prep, pn, k, B, s);
    if (e != hipSuccess)
      fail(FLUID_E_HIP, "node " + std::to_string(pn.node) + " (" + k.name() + "): " + hipGetErrorString(e));
    if (rec >= 0) hip_check(hipEventRecord(g_trace.ev[2 * rec + 1], s), "hipEventRecord");
  }
}

// The arena of fluid_run_static: a file-scope device array, one copy per
// GPU, alive until the process ends.  Host code never uses the array's name
// as an address (on the host it is only a stand-in symbol): the device
// address of each GPU's copy is looked up once, with that GPU current, and
// kept per device.
__device__ __align__(256) unsigned char scratch[FLUID_STATIC_ARENA_BYTES];

std::mutex g_static_mu;
std::map<int, void*> g_static_ptr;  // device ordinal -> address of its copy

void* static_arena() {
  int dev = -1;
  hip_check(hipGetDevice(&dev), "hipGetDevice");
  std::lock_guard<std::mutex> lk(g_static_mu);
  auto it = g_static_ptr.find(dev);
  if (it != g_static_ptr.end()) return it->second;
  void* ptr = nullptr;
  hip_check(hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch)), "hipGetSymbolAddress(static arena)");
  require(ptr != nullptr && ((uintptr_t)ptr & 255) == 0, "static arena address is not 256-byte aligned");
  g_static_ptr[dev] = ptr;
  return ptr;
}

}  // namespace

extern "C" {

fluid_status fluid_run(const fluid_graph* gh, const fluid_layout_plan* lh, const fluid_arena_plan* ah, void* arena,
                       uint64_t arena_bytes, const void* const* consts, const void* const* inputs,
                       void* const* outputs, void* hip_stream) {
  return call_guarded([&] {
    std::shared_ptr<Prepared> prep =
        checked_prepared(gh, lh, ah, arena, arena_bytes, consts, inputs, outputs, "fluid_run");
    run_prepared(gh, *prep, Bases{(char*)arena, inputs, outputs, consts}, (hipStream_t)hip_stream);
  });
}

fluid_status fluid_run_static(const fluid_graph* gh, const fluid_layout_plan* lh, const fluid_arena_plan* ah,
                              const void* const* consts, const void* const* inputs, void* const* outputs,
                              void* hip_stream) {
  return call_guarded([&] {
    require(gh && lh && ah, "fluid_run_static: NULL graph or plan");
    if (ah->a.peak > FLUID_STATIC_ARENA_BYTES)
      fail(FLUID_E_ARENA_TOO_SMALL, "fluid_run_static: the plan needs " + std::to_string(ah->a.peak) +
                                        " arena bytes, the static arena holds " +
                                        std::to_string((uint64_t)FLUID_STATIC_ARENA_BYTES));
    void* arena = static_arena();
    std::shared_ptr<Prepared> prep = checked_prepared(gh, lh, ah, arena, FLUID_STATIC_ARENA_BYTES, consts, inputs,
                                                      outputs, "fluid_run_static");
    run_prepared(gh, *prep, Bases{(char*)arena, inputs, outputs, consts}, (hipStream_t)hip_stream);
  });
}

fluid_status fluid_pack_constant(const fluid_graph* gh, const fluid_layout_plan* lh, int32_t c, const void* src,
                                 void* dst, void* hip_stream) {
  return call_guarded([&] {
    require(gh && lh && src && dst, "fluid_pack_constant: NULL argument");
    require(lh->p.graph_serial == gh->serial, "fluid_pack_constant: plan belongs to another graph");
    const Graph& g = gh->g;
    require(c >= 0 && c < (int32_t)g.consts.size(), "fluid_pack_constant: constant id out of range");
    require(aligned(src, 16) && aligned(dst, 16), "fluid_pack_constant: src and dst must be 16-byte aligned");
    const Const& k = g.consts[c];
    const uint64_t bytes = (uint64_t)numel(k.shape) * dtype_bytes(k.dtype);
    const uintptr_t s0 = (uintptr_t)src, d0 = (uintptr_t)dst;
    require(s0 + bytes <= d0 || d0 + bytes <= s0, "fluid_pack_constant: src and dst overlap");
    hipStream_t s = (hipStream_t)hip_stream;
    const Perm p = constant_layout(g, lh->p, c);
    if (p == identity_perm((int)k.shape.size())) {
      hip_check(hipMemcpyAsync(dst, src, bytes, hipMemcpyDeviceToDevice, s), "hipMemcpyAsync");
      return;
    }
    // a relayout copy of the [K, N] row-major weight into K-contiguous order
    Node nd;
    nd.op = FLUID_OP_RESHAPE;
    nd.out_shape = k.shape;
    Operand in, out;
    in.shape = out.shape = k.shape;
    in.dtype = out.dtype = k.dtype;
    in.stride = row_major_strides(k.shape);
    out.stride = dense_strides(k.shape, p);
    in.ptr = src;
    out.ptr = dst;
    NodeKernel kk = prepare_node(nd, 1, k.dtype, {in}, out);
    if (!kk.available) kk = prepare_node(nd, 0, k.dtype, {in}, out);
    require(kk.available, "fluid_pack_constant: no copy kernel for this constant (" + kk.why + ")");
    const hipError_t e = launch_node_kernel(kk, s);
    if (e != hipSuccess) fail(FLUID_E_HIP, std::string("fluid_pack_constant: ") + hipGetErrorString(e));
  });
}

fluid_status fluid_run_nodes(const fluid_graph* gh, const fluid_layout_plan* lh, const fluid_arena_plan* ah,
                             void* arena, uint64_t arena_bytes, const void* const* consts, const void* const* inputs,
                             void* const* outputs, const int32_t* nodes, int32_t n_nodes, int32_t repeat,
                             void* hip_stream) {
  return call_guarded([&] {
    std::shared_ptr<Prepared> prep =
        checked_prepared(gh, lh, ah, arena, arena_bytes, consts, inputs, outputs, "fluid_run_nodes");
    require(nodes && n_nodes > 0 && repeat >= 1, "fluid_run_nodes: empty node list or repeat < 1");
    std::vector<const PreparedNode*> sel;
    for (int32_t i = 0; i < n_nodes; ++i) {
      const int n = nodes[i];
      require(n >= 0 && n < gh->g.n_nodes(), "fluid_run_nodes: node out of range");
      const PreparedNode* found = nullptr;
      for (const PreparedNode& pn : prep->nodes)
        if (pn.node == n) found = &pn;
      require(found != nullptr, "fluid_run_nodes: node " + std::to_string(n) + " is a view under this plan");
      sel.push_back(found);
    }
    // what the list launches, decided and checked before the first launch:
    // a fused MatMul followed in the list by every node it absorbs runs as in
    // fluid_run, and so does a grouped launch whose nodes (the products and
    // the nodes they absorb) all follow in fluid_run's order; otherwise each
    // node runs its own kernel -- which a node the plan performs only inside
    // a fused launch (a priced fusion chain) does not have, and which would
    // touch a tensor the plan keeps on chip when it is such a chain's MatMul
    enum { OWN, CHAIN, GROUP };
    std::vector<std::pair<const PreparedNode*, int>> todo;
    const PreparedNode* first = prep->nodes.data();
    auto stored = [](const Bind& b) { return b.kind != BK_ARENA || b.off >= 0; };
    for (size_t i = 0; i < sel.size(); ++i) {
      const PreparedNode* pn = sel[i];
      if (!pn->group.empty()) {
        const size_t last = (size_t)pn->group.back();
        const size_t span = last + prep->nodes[last].fuse_n - (size_t)(pn - first) + 1;
        bool whole = i + span <= sel.size();
        for (size_t t = 0; whole && t < span; ++t) whole = sel[i + t] == pn + t;
        if (whole) {
          todo.push_back({pn, GROUP});
          i += span - 1;
          continue;
        }
      }
      bool whole = pn->fuse_n > 0 && i + pn->fuse_n < sel.size();
      for (int f = 1; whole && f <= pn->fuse_n; ++f) whole = sel[i + f] == pn + f;
      if (whole) {
        todo.push_back({pn, CHAIN});
        i += pn->fuse_n;
        continue;
      }
      bool ok = pn->k.available && stored(pn->out);
      for (const Bind& b : pn->in) ok = ok && stored(b);
      require(ok, "fluid_run_nodes: node " + std::to_string(pn->node) +
                      " belongs to a fusion chain whose intermediate results the plan keeps on chip; list the "
                      "chain's nodes together, in node order");
      todo.push_back({pn, OWN});
    }
    Bases B{(char*)arena, inputs, outputs, consts};
    hipStream_t s = (hipStream_t)hip_stream;
    for (int32_t r = 0; r < repeat; ++r)
      for (const auto& [pn, mode] : todo) {
        NodeKernel k = pn->k;
        hipError_t e;
        if (mode == GROUP) {
          k = launch_kernel(*pn, B);
          e = launch_group(*prep, *pn, k, B, s);
        } else {
          if (mode == CHAIN) k = fused_kernel(*pn, B);
          else patch(k, *pn, B);
          e = launch_node_kernel(k, s);
        }
        if (e != hipSuccess)
          fail(FLUID_E_HIP, "node " + std::to_string(pn->node) + " (" + k.name() + "): " + hipGetErrorString(e));
      }
  });
}

fluid_status fluid_trace_enable(const fluid_graph* gh, const uint8_t* mask, int32_t max_records) {
  return call_guarded([&] {
    require(gh && max_records > 0, "fluid_trace_enable: bad argument");
    std::lock_guard<std::mutex> lk(g_trace_mu);
    for (hipEvent_t e : g_trace.ev) (void)hipEventDestroy(e);
    g_trace = Trace();
    g_trace.mask.assign(gh->g.n_nodes(), 1);
    if (mask)
      for (int n = 0; n < gh->g.n_nodes(); ++n) g_trace.mask[n] = mask[n] ? 1 : 0;
    g_trace.ev.resize(2 * (size_t)max_records);
    for (auto& e : g_trace.ev) hip_check(hipEventCreate(&e), "hipEventCreate");
    g_trace.max_records = max_records;
    g_trace.graph_serial = gh->serial;
    g_trace.on = true;
  });
}

fluid_status fluid_trace_collect(const fluid_graph* gh, double* ms, int32_t* launches) {
  return call_guarded([&] {
    require(gh && ms && launches, "fluid_trace_collect: NULL argument");
    std::lock_guard<std::mutex> lk(g_trace_mu);
    require(g_trace.graph_serial == gh->serial, "fluid_trace_collect: tracing was enabled for another graph");
    for (size_t r = 0; r < g_trace.node_of.size(); ++r) {
      hip_check(hipEventSynchronize(g_trace.ev[2 * r + 1]), "hipEventSynchronize");
      float t = 0.f;
      hip_check(hipEventElapsedTime(&t, g_trace.ev[2 * r], g_trace.ev[2 * r + 1]), "hipEventElapsedTime");
      ms[g_trace.node_of[r]] += t;
      launches[g_trace.node_of[r]] += 1;
    }
    for (hipEvent_t e : g_trace.ev) (void)hipEventDestroy(e);
    g_trace = Trace();
  });
}

fluid_status fluid_measure_costs(const fluid_graph* gh, uint32_t reps, void* scratch, uint64_t scratch_bytes,
                                 void* hip_stream, fluid_cost_table** out) {
  return call_guarded([&] {
    require(gh && out, "fluid_measure_costs: NULL argument");
    const Graph& g = gh->g;
    require(reps >= 1 && reps <= 1000, "fluid_measure_costs: reps must be 1..1000");
    const uint64_t need = measure_scratch_bytes(g);
    require(scratch && aligned(scratch, 256), "fluid_measure_costs: scratch must be non-NULL and 256-byte aligned");
    require(scratch_bytes >= need, "fluid_measure_costs: scratch needs " + std::to_string(need) + " bytes");
    hip_check(launch_fill(scratch, scratch_bytes, 12345u, (hipStream_t)hip_stream), "fill");
    hip_check(hipStreamSynchronize((hipStream_t)hip_stream), "hipStreamSynchronize");
    // a stream of its own (default priority), which the timed batches are
    // captured from: the caller's may be the null stream
    hipStream_t s = nullptr;
    hip_check(hipStreamCreateWithFlags(&s, hipStreamNonBlocking), "hipStreamCreateWithFlags");
    struct StreamGuard {
      hipStream_t s;
      ~StreamGuard() { (void)hipStreamSynchronize(s); (void)hipStreamDestroy(s); }
    } sg{s};

    CostTable t;
    for (int e = 0; e < g.n_edges(); ++e)
      t.L.push_back(g.pinned(e) ? std::vector<Perm>{identity_perm((int)g.edge_shape(e).size())}
                                : measured_layout_list(g.edge_shape(e)));
    std::map<SigKey, int> sig_of;
    std::vector<int> rep_node;
    for (int n = 0; n < g.n_nodes(); ++n) {
      SigKey k = sig_key(g, n);
      auto it = sig_of.find(k);
      if (it == sig_of.end()) {
        it = sig_of.emplace(k, (int)rep_node.size()).first;
        rep_node.push_back(n);
      }
      t.node_sig.push_back(it->second);
    }
    // candidate list per slot / output of each signature: the union over
    // its nodes (identity only if every node has that edge pinned)
    std::vector<std::vector<std::vector<Perm>>> slot_lists(rep_node.size());
    std::vector<std::vector<Perm>> out_lists(rep_node.size());
    for (int n = 0; n < g.n_nodes(); ++n) {
      const int si = t.node_sig[n];
      const auto& slots = g.act_in[n];
      auto& sl = slot_lists[si];
      if (sl.empty()) sl.resize(slots.size());
      for (size_t s2 = 0; s2 < slots.size(); ++s2)
        if (t.L[slots[s2]].size() > sl[s2].size()) sl[s2] = t.L[slots[s2]];
      const int eo = g.out_edge(n);
      if (t.L[eo].size() > out_lists[si].size()) out_lists[si] = t.L[eo];
    }
    // packed-weight MatMul variants: only where every node of the
    // signature reads a weight that no other node reads
    std::vector<char> packable(rep_node.size(), 1);
    for (int n = 0; n < g.n_nodes(); ++n) {
      const Node& nd = g.nodes[n];
      if (nd.op != FLUID_OP_MATMUL || nd.ins.size() != 2 || nd.ins[1] >= 0 ||
          g.const_readers[~nd.ins[1]].size() != 1)
        packable[t.node_sig[n]] = 0;
    }
    hipEvent_t ev[2 * 64];
    const uint32_t R = std::min<uint32_t>(reps, 64);
    for (auto& e : ev) hip_check(hipEventCreate(&e), "hipEventCreate");
    struct EvGuard {
      hipEvent_t* ev;
      ~EvGuard() { for (int i = 0; i < 128; ++i) (void)hipEventDestroy(ev[i]); }
    } evg{ev};
    // one candidate: an untimed warm-up launch (the first launch of a kernel
    // instance also loads its code, which can take milliseconds), then one
    // launch timed on its own -- clearly losing candidates (over 8x the
    // signature's best so far) get no more launches -- then R back-to-back
    // launches captured once as a HIP graph and replayed three times, each
    // replay between two events (the per-launch time includes the kernel's
    // start-up and the gap to the next launch as a run's graph issues them,
    // without the host's launch cost, which would pace kernels of a few
    // microseconds); the median, in integer ns.  Successive launches take
    // the kernels of ks in turn (copies of a constant weight,
    // cold_weight_copies).
    auto time_kernel = [&](const std::vector<NodeKernel>& ks, int64_t& best_so_far) -> int64_t {
      size_t li = 0;
      auto next = [&]() -> const NodeKernel& { return ks[li++ % ks.size()]; };
      hip_check(launch_node_kernel(next(), s), "warm-up launch");
      hip_check(hipEventRecord(ev[0], s), "hipEventRecord");
      hip_check(launch_node_kernel(next(), s), "first timed launch");
      hip_check(hipEventRecord(ev[1], s), "hipEventRecord");
      hip_check(hipEventSynchronize(ev[1]), "hipEventSynchronize");
      float first = 0.f;
      hip_check(hipEventElapsedTime(&first, ev[0], ev[1]), "hipEventElapsedTime");
      std::vector<float> times = {first};
      const int64_t first_ns = (int64_t)std::llround((double)first * 1e6);
      if (!(best_so_far >= 0 && first_ns > 8 * best_so_far)) {
        times.clear();
        struct GraphGuard {
          hipGraph_t g = nullptr;
          hipGraphExec_t x = nullptr;
          ~GraphGuard() {
            if (x) (void)hipGraphExecDestroy(x);
            if (g) (void)hipGraphDestroy(g);
          }
        } gg;
        hip_check(hipStreamBeginCapture(s, hipStreamCaptureModeThreadLocal), "hipStreamBeginCapture");
        hipError_t le = hipSuccess;
        for (uint32_t r = 0; r < R && le == hipSuccess; ++r) le = launch_node_kernel(next(), s);
        const hipError_t ce = hipStreamEndCapture(s, &gg.g);
        hip_check(le, "captured launch");
        hip_check(ce, "hipStreamEndCapture");
        hip_check(hipGraphInstantiate(&gg.x, gg.g, nullptr, nullptr, 0), "hipGraphInstantiate");
        for (int b = 0; b < 3; ++b) {
          hip_check(hipEventRecord(ev[2 + 2 * b], s), "hipEventRecord");
          hip_check(hipGraphLaunch(gg.x, s), "hipGraphLaunch");
          hip_check(hipEventRecord(ev[3 + 2 * b], s), "hipEventRecord");
        }
        hip_check(hipEventSynchronize(ev[7]), "hipEventSynchronize");
        for (int b = 0; b < 3; ++b) {
          float ms = 0.f;
          hip_check(hipEventElapsedTime(&ms, ev[2 + 2 * b], ev[3 + 2 * b]), "hipEventElapsedTime");
          times.push_back(ms / (float)R);
        }
      }
      std::sort(times.begin(), times.end());
      const int64_t ns_ = std::max<int64_t>(1, (int64_t)std::llround((double)times[times.size() / 2] * 1e6));
      if (best_so_far < 0 || ns_ < best_so_far) best_so_far = ns_;
      return ns_;
    };
    // k and its copies reading the constant weight (MatMul / Conv operand 1,
    // wbytes) from the copies placed at `copies` onwards
    auto with_weight_copies = [&](const NodeKernel& k, const Node& nd, char* copies) {
      std::vector<NodeKernel> ks = {k};
      if (!(nd.op == FLUID_OP_MATMUL || nd.op == FLUID_OP_CONV) || nd.ins.size() < 2 || nd.ins[1] >= 0) return ks;
      const Const& w = g.consts[~nd.ins[1]];
      const uint64_t wb = (uint64_t)numel(w.shape) * dtype_bytes(w.dtype);
      const int W = cold_weight_copies(wb);
      for (int i = 1; i < W; ++i) {
        NodeKernel c = k;
        char* p = copies + (uint64_t)(i - 1) * align256(wb);
        if (c.family == KF_GEMM) c.gemm.B = p;
        else if (c.family == KF_CONV) c.conv.w = (const float*)p;
        ks.push_back(c);
      }
      return ks;
    };
    char* base = (char*)scratch;
    for (size_t si = 0; si < rep_node.size(); ++si) {
      const int n = rep_node[si];
      const Node& nd = g.nodes[n];
      Sig sig;
      sig.op = nd.op;
      for (int e : g.act_in[n]) sig.in_shapes.push_back(g.edge_shape(e));
      sig.out_shape = nd.out_shape;
      const auto& lists = slot_lists[si];
      const auto& olist = out_lists[si];
      const int ns = (int)lists.size();
      std::vector<size_t> idx(ns + 1, 0);
      int64_t best_so_far = -1;
      for (;;) {
        SigEntry en;
        for (int i = 0; i < ns; ++i) en.in.push_back(lists[i][idx[i]]);
        en.out = olist[idx[ns]];
        const bool view = (nd.op == FLUID_OP_TRANSPOSE || nd.op == FLUID_OP_RESHAPE) &&
                          is_view(nd.op, nd.perm, g.edge_shape(g.act_in[n][0]), nd.out_shape, en.in[0], en.out);
        if (view) {
          en.costs = {0};
        } else {
          // operands laid out one after another in the scratch buffer
          std::vector<Operand> ins;
          uint64_t off = 0;
          int slot = 0;
          for (int v : nd.ins) {
            Operand o;
            if (v >= 0) {
              o.shape = g.edge_shape(v);
              o.stride = dense_strides(o.shape, en.in[slot++]);
              o.dtype = g.dtype;
            } else {
              o.shape = g.consts[~v].shape;
              o.stride = row_major_strides(o.shape);
              o.dtype = g.consts[~v].dtype;
            }
            o.ptr = base + off;
            off = align256(off + (uint64_t)numel(o.shape) * dtype_bytes(o.dtype));
            ins.push_back(o);
          }
          Operand ou;
          ou.shape = nd.out_shape;
          ou.stride = dense_strides(ou.shape, en.out);
          ou.dtype = g.dtype;
          ou.ptr = base + off;
          for (int v = 0; v < num_variants(nd.op); ++v) {
            if (packs_weight(nd.op, v) && !packable[si]) { en.costs.push_back(-1); continue; }
            std::vector<Operand> vins = ins;
            for (size_t s2 = 0; s2 < nd.ins.size(); ++s2)
              if (nd.ins[s2] < 0) vins[s2].stride = const_strides(nd, (int)s2, v, vins[s2].shape);
            NodeKernel k = prepare_node(nd, v, g.dtype, vins, ou);
            if (!k.available) { en.costs.push_back(-1); continue; }
            char* copies = base + align256(off + (uint64_t)numel(ou.shape) * dtype_bytes(g.dtype));
            en.costs.push_back(time_kernel(with_weight_copies(k, nd, copies), best_so_far));
          }
        }
        sig.entries.push_back(std::move(en));
        int i = ns;
        for (; i >= 0; --i) {
          const size_t lim = i == ns ? olist.size() : lists[i].size();
          if (++idx[i] < lim) break;
          idx[i] = 0;
        }
        if (i < 0) break;
      }
      t.sigs.push_back(std::move(sig));
    }
    // fusion chains (fusion.h): one fused signature per (head signature,
    // step signatures); the head's slots and R laid out as for the node, R
    // in the output's layout only (a fused launch reading R in another
    // layout than it writes is never the cheap way to run the chain)
    {
      struct FusedKey {
        SigKey k;
        std::vector<SigKey> steps;
        std::vector<int> kinds;  // a stored residual sum costs its extra write
        bool operator<(const FusedKey& o) const { return std::tie(k, steps, kinds) < std::tie(o.k, o.steps, o.kinds); }
      };
      std::map<FusedKey, int> fsig_of;
      std::vector<std::pair<int, int>> rep_chain;  // (m, t) per fused signature
      std::vector<std::vector<std::vector<Perm>>> fslot_lists;
      std::vector<std::vector<Perm>> fout_lists;
      for (int m = 0; m < g.n_nodes(); ++m) {
        const std::vector<ChainStep> steps = chain_steps(g, m);
        FusedKey fk{sig_key(g, m), {}};
        for (int tl = 1; tl <= (int)steps.size(); ++tl) {
          fk.steps.push_back(sig_key(g, steps[tl - 1].node));
          fk.kinds.push_back(steps[tl - 1].kind);
          auto it = fsig_of.find(fk);
          if (it == fsig_of.end()) {
            it = fsig_of.emplace(fk, (int)rep_chain.size()).first;
            rep_chain.push_back({m, tl});
            fslot_lists.emplace_back();
            fout_lists.emplace_back();
          }
          const int fi = it->second;
          t.fused_refs.push_back({m, tl, fi});
          const std::vector<int> slots = chain_slots(g, m, tl);
          auto& sl = fslot_lists[fi];
          if (sl.empty()) sl.resize(slots.size());
          for (size_t s2 = 0; s2 < slots.size(); ++s2)
            if (t.L[slots[s2]].size() > sl[s2].size()) sl[s2] = t.L[slots[s2]];
          const int eo = g.out_edge(m + tl);
          if (t.L[eo].size() > fout_lists[fi].size()) fout_lists[fi] = t.L[eo];
        }
      }
      for (size_t fi = 0; fi < rep_chain.size(); ++fi) {
        const int m = rep_chain[fi].first, tl = rep_chain[fi].second;
        const Node& mn = g.nodes[m];
        const std::vector<ChainStep> steps = chain_steps(g, m);
        uint32_t act = 0, rop = 0;
        int bias = -1;
        for (int i = 0; i < tl; ++i) {
          if (steps[i].kind == CH_BIAS) bias = steps[i].bias;
          else if (steps[i].kind == CH_ACT) act = g.nodes[steps[i].node].op == FLUID_OP_GELU ? 1u : 2u;
          else if (steps[i].kind == CH_ADD_R) rop = 1u;
          else if (steps[i].kind == CH_MUL_R) rop = 2u;
        }
        Sig sig;
        sig.op = mn.op;
        for (int e : chain_slots(g, m, tl)) sig.in_shapes.push_back(g.edge_shape(e));
        sig.out_shape = g.nodes[m + tl].out_shape;
        const auto& lists = fslot_lists[fi];
        const auto& olist = fout_lists[fi];
        const int nmm = (int)g.act_in[m].size();  // the MatMul's own slots; R follows
        const int ns = (int)lists.size();
        std::vector<size_t> idx(ns + 1, 0);
        int64_t best_so_far = -1;
        for (;;) {
          SigEntry en;
          for (int i = 0; i < ns; ++i) en.in.push_back(lists[i][idx[i]]);
          en.out = olist[idx[ns]];
          if (mn.op == FLUID_OP_ADD) {
            // the residual sum and its normalisation: both summands, the
            // norm's constants, the output
            const Node& xn = g.nodes[m + 1];
            uint64_t off = 0;
            auto place = [&](const Shape& sh, std::vector<int64_t> st, int dt) {
              Operand o;
              o.shape = sh;
              o.stride = std::move(st);
              o.dtype = dt;
              o.ptr = base + off;
              off = align256(off + (uint64_t)numel(sh) * dtype_bytes(dt));
              return o;
            };
            const Shape& xs = sig.out_shape;
            const Operand x0 = place(xs, dense_strides(xs, en.in[0]), g.dtype);
            const Operand x1 = place(xs, dense_strides(xs, en.in[1]), g.dtype);
            std::vector<Operand> ins = {x0};
            for (size_t s2 = 1; s2 < xn.ins.size(); ++s2) {
              const Const& c = g.consts[~xn.ins[s2]];
              ins.push_back(place(c.shape, row_major_strides(c.shape), c.dtype));
            }
            const Operand ou = place(xs, dense_strides(xs, en.out), g.dtype);
            // a sum with further readers is also stored, in the output's layout
            void* hs = steps[0].kind == CH_NORM_STORE ? (void*)place(xs, dense_strides(xs, en.out), g.dtype).ptr : nullptr;
            for (int v = 0; v < num_variants(xn.op); ++v) {
              NodeKernel k = prepare_sum_norm(xn, v, g.dtype, ins, x1, ou);
              if (!k.available) { en.costs.push_back(-1); continue; }
              k.red.h = hs;
              en.costs.push_back(time_kernel({k}, best_so_far));
            }
            sig.entries.push_back(std::move(en));
          } else if (!rop || en.in[nmm] == en.out) {
            std::vector<Operand> ins;
            uint64_t off = 0;
            int slot = 0;
            for (int v : mn.ins) {
              Operand o;
              if (v >= 0) {
                o.shape = g.edge_shape(v);
                o.stride = dense_strides(o.shape, en.in[slot++]);
                o.dtype = g.dtype;
              } else {
                o.shape = g.consts[~v].shape;
                o.stride = row_major_strides(o.shape);
                o.dtype = g.consts[~v].dtype;
              }
              o.ptr = base + off;
              off = align256(off + (uint64_t)numel(o.shape) * dtype_bytes(o.dtype));
              ins.push_back(o);
            }
            void* bias_ptr = nullptr;
            if (bias >= 0) {
              bias_ptr = base + off;
              off = align256(off + (uint64_t)numel(g.consts[bias].shape) * dtype_bytes(g.dtype));
            }
            Operand r;
            if (rop) {
              r.shape = sig.out_shape;
              r.stride = dense_strides(r.shape, en.in[nmm]);
              r.dtype = g.dtype;
              r.ptr = base + off;
              off = align256(off + (uint64_t)numel(r.shape) * dtype_bytes(g.dtype));
            }
            Operand ou;
            ou.shape = sig.out_shape;
            ou.stride = dense_strides(ou.shape, en.out);
            ou.dtype = g.dtype;
            ou.ptr = base + off;
            for (int v = 0; v < num_variants(mn.op); ++v) {
              if (packs_weight(mn.op, v) && !packable[t.node_sig[m]]) { en.costs.push_back(-1); continue; }
              std::vector<Operand> vins = ins;
              for (size_t s2 = 0; s2 < mn.ins.size(); ++s2)
                if (mn.ins[s2] < 0) vins[s2].stride = const_strides(mn, (int)s2, v, vins[s2].shape);
              NodeKernel k = fused_gemm_kernel(mn, v, g.dtype, vins, ou, act, rop, rop ? &r : nullptr);
              if (!k.available) { en.costs.push_back(-1); continue; }
              k.gemm.bias = bias_ptr;
              k.gemm.R = rop ? r.ptr : nullptr;
              char* copies = (char*)ou.ptr + align256((uint64_t)numel(ou.shape) * dtype_bytes(g.dtype));
              en.costs.push_back(time_kernel(with_weight_copies(k, mn, copies), best_so_far));
            }
            sig.entries.push_back(std::move(en));
          }
          int i = ns;
          for (; i >= 0; --i) {
            const size_t lim = i == ns ? olist.size() : lists[i].size();
            if (++idx[i] < lim) break;
            idx[i] = 0;
          }
          if (i < 0) break;
        }
        t.fused_sigs.push_back(std::move(sig));
      }
    }
    hip_check(hipStreamSynchronize(s), "hipStreamSynchronize");
    t.bind(g);
    auto h = std::make_unique<fluid_cost_table>();
    h->t = std::move(t);
    h->serial = gh->serial;
    *out = h.release();
  });
}

}  // extern "C"
