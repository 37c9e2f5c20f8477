"""ctypes binding of include/fluid.h (argument marshalling only).

Every function named ``fluid_*`` here calls the C entry point of the same
name; all computation happens in the native library.  ``load()`` picks the
GPU library (lib/libfluid.so) or, with ``host_only=True``, the planner-only
library (lib/libfluid_host.so).  A missing library raises immediately: there
is no fallback implementation.

The small classes at the end (Graph, CostTable, LayoutPlan, ArenaPlan,
Executor) own handles and, for the executor, the torch device tensors that
hold constants, inputs, outputs and the arena.
"""
from __future__ import annotations

import ctypes as C
import json
import os

_PKG = os.path.dirname(os.path.abspath(__file__))
# FLUID_LIBDIR: load the libraries from another directory (e.g. a
# sanitizer build of the host library)
LIBDIR = os.environ.get("FLUID_LIBDIR") or os.path.join(_PKG, "lib")

MAX_RANK = 6
MAX_IN = 4

F32, BF16 = 0, 1
OPS = {"matmul": 0, "add": 1, "mul": 2, "transpose": 3, "reshape": 4, "softmax": 5,
       "layernorm": 6, "rmsnorm": 7, "gelu": 8, "silu": 9, "rope": 10,
       "pad": 11, "conv": 12, "relu": 13, "maxpool": 14}
ROLES = {"other": 0, "weight": 1, "bias": 2, "gamma": 3, "beta": 4, "rope_cos": 5, "rope_sin": 6}
ARCH = {"post_ln": 0, "pre_ln": 1, "llama": 2, "vgg": 3}
MAX_STAGES = 8
NO_DP, NO_VARIANTS, NO_GUARD, NO_FUSION = 1, 2, 4, 8
ARENA_NO_REUSE, ARENA_EPILOGUE = 1, 2
STATUS = {0: "OK", -1: "INVALID", -2: "UNSUPPORTED", -3: "INFEASIBLE", -4: "ARENA_TOO_SMALL",
          -5: "HIP", -6: "NOMEM"}


class FluidError(RuntimeError):
    def __init__(self, status, msg):
        super().__init__(f"{STATUS.get(status, status)}: {msg}")
        self.status = status


class NodeDesc(C.Structure):
    _fields_ = [("op", C.c_int32), ("n_in", C.c_int32), ("in_", C.c_int32 * MAX_IN),
                ("out_rank", C.c_int32), ("out_shape", C.c_int64 * MAX_RANK),
                ("perm", C.c_int32 * MAX_RANK), ("f_attr", C.c_float * 2), ("i_attr", C.c_int32 * 2)]


class GraphDesc(C.Structure):
    _fields_ = [("dtype", C.c_int32),
                ("n_inputs", C.c_int32), ("input_rank", C.POINTER(C.c_int32)),
                ("input_shapes", C.POINTER(C.c_int64)),
                ("n_consts", C.c_int32), ("const_rank", C.POINTER(C.c_int32)),
                ("const_shapes", C.POINTER(C.c_int64)), ("const_dtype", C.POINTER(C.c_int32)),
                ("const_role", C.POINTER(C.c_int32)),
                ("n_nodes", C.c_int32), ("nodes", C.POINTER(NodeDesc)),
                ("n_outputs", C.c_int32), ("output_edges", C.POINTER(C.c_int32))]


class ModelCfg(C.Structure):
    _fields_ = [("arch", C.c_int32), ("layers", C.c_int32), ("batch", C.c_int32), ("seq", C.c_int32),
                ("hidden", C.c_int32), ("heads", C.c_int32), ("ffn", C.c_int32), ("dtype", C.c_int32),
                ("eps", C.c_float), ("rope_base", C.c_float),
                ("channels", C.c_int32), ("image", C.c_int32), ("fc", C.c_int32), ("classes", C.c_int32),
                ("n_stages", C.c_int32), ("stage_width", C.c_int32 * MAX_STAGES),
                ("stage_convs", C.c_int32 * MAX_STAGES)]


_VP = C.c_void_p
_PROTOS = {
    "fluid_last_error": (C.c_char_p, []),
    "fluid_build_graph": (C.c_int, [C.POINTER(GraphDesc), C.POINTER(_VP)]),
    "fluid_build_transformer": (C.c_int, [C.POINTER(ModelCfg), C.POINTER(_VP)]),
    "fluid_graph_info": (C.c_int, [_VP] + [C.POINTER(C.c_int32)] * 5),
    "fluid_graph_export_json": (C.c_int, [_VP, C.c_char_p, C.c_uint64, C.POINTER(C.c_uint64)]),
    "fluid_cost_table_load": (C.c_int, [C.c_char_p, _VP, C.POINTER(_VP)]),
    "fluid_cost_table_save": (C.c_int, [_VP, C.c_char_p]),
    "fluid_measure_scratch_bytes": (C.c_int, [_VP, C.POINTER(C.c_uint64)]),
    "fluid_measure_costs": (C.c_int, [_VP, C.c_uint32, _VP, C.c_uint64, _VP, C.POINTER(_VP)]),
    "fluid_plan_layouts": (C.c_int, [_VP, _VP, C.c_uint32, C.POINTER(_VP)]),
    "fluid_layout_plan_get": (C.c_int, [_VP, C.POINTER(C.c_int32), C.POINTER(C.c_int32),
                                        C.POINTER(C.c_int64), C.POINTER(C.c_int32)]),
    "fluid_edge_layout": (C.c_int, [_VP, _VP, C.c_int32, C.POINTER(C.c_int32)]),
    "fluid_layout_plan_fusion": (C.c_int, [_VP, C.POINTER(C.c_int32), C.POINTER(C.c_int32)]),
    "fluid_plan_arena": (C.c_int, [_VP, _VP, C.c_uint64, C.c_uint32, C.POINTER(_VP)]),
    "fluid_arena_plan_get": (C.c_int, [_VP, C.POINTER(C.c_uint64), C.POINTER(C.c_uint64),
                                       C.POINTER(C.c_uint64), C.POINTER(C.c_int64), C.POINTER(C.c_int32)]),
    "fluid_arena_plan_lifetimes": (C.c_int, [_VP, C.c_int32, C.POINTER(C.c_uint64), C.POINTER(C.c_int32),
                                             C.POINTER(C.c_int32)]),
    "fluid_run": (C.c_int, [_VP, _VP, _VP, _VP, C.c_uint64, C.POINTER(_VP), C.POINTER(_VP),
                            C.POINTER(_VP), _VP]),
    "fluid_constant_layout": (C.c_int, [_VP, _VP, C.c_int32, C.POINTER(C.c_int32)]),
    "fluid_pack_constant": (C.c_int, [_VP, _VP, C.c_int32, _VP, _VP, _VP]),
    "fluid_run_static": (C.c_int, [_VP, _VP, _VP, C.POINTER(_VP), C.POINTER(_VP), C.POINTER(_VP), _VP]),
    "fluid_run_nodes": (C.c_int, [_VP, _VP, _VP, _VP, C.c_uint64, C.POINTER(_VP), C.POINTER(_VP),
                                  C.POINTER(_VP), C.POINTER(C.c_int32), C.c_int32, C.c_int32, _VP]),
    "fluid_run_launches": (C.c_int, [_VP, _VP, _VP, C.POINTER(C.c_int32)]),
    "fluid_run_schedule": (C.c_int, [_VP, _VP, _VP, C.POINTER(C.c_int32), C.POINTER(C.c_uint8), C.c_char_p,
                                     C.c_uint64, C.POINTER(C.c_uint64), C.POINTER(C.c_int32)]),
    "fluid_trace_enable": (C.c_int, [_VP, C.POINTER(C.c_uint8), C.c_int32]),
    "fluid_trace_collect": (C.c_int, [_VP, C.POINTER(C.c_double), C.POINTER(C.c_int32)]),
    "fluid_node_kernel": (C.c_int, [_VP, _VP, C.c_int32, C.c_char_p, C.c_uint64]),
    "fluid_graph_free": (None, [_VP]),
    "fluid_cost_table_free": (None, [_VP]),
    "fluid_layout_plan_free": (None, [_VP]),
    "fluid_arena_plan_free": (None, [_VP]),
}
SYMBOLS = tuple(_PROTOS)

_libs = {}
_lib = None


def load(host_only=False):
    """Load (once) and return the native library; raises if it is not built."""
    global _lib
    name = "libfluid_host.so" if host_only else "libfluid.so"
    if name in _libs:
        _lib = _libs[name]
        return _lib
    path = os.path.join(LIBDIR, name)
    if not os.path.exists(path):
        raise FileNotFoundError(f"{path} is not built; run `python -m paper_2411_09242_amd.build`")
    if not host_only:
        # torch carries its own HIP runtime; loading it first makes the
        # library bind to that same runtime instead of bringing a second one
        # into the process (two runtimes do not share devices or memory)
        import torch  # noqa: F401
    lib = C.CDLL(path)
    for sym, (res, args) in _PROTOS.items():
        f = getattr(lib, sym)
        f.restype = res
        f.argtypes = args
    _libs[name] = lib
    _lib = lib
    return lib


def _L():
    if _lib is None:
        load()
    return _lib


def _check(st):
    if st != 0:
        raise FluidError(st, _L().fluid_last_error().decode())


# ----------------------------------------------------------------- raw calls
def fluid_build_transformer(cfg: dict):
    c = ModelCfg()
    c.arch = ARCH[cfg["arch"]]
    c.batch = cfg["batch"]
    c.dtype = BF16 if cfg["dtype"] == "bf16" else F32
    c.eps = cfg.get("eps", 1e-5)
    c.rope_base = cfg.get("rope_base", 10000.0)
    if cfg["arch"] == "vgg":
        c.channels, c.image, c.fc, c.classes = cfg["channels"], cfg["image"], cfg["fc"], cfg["classes"]
        c.n_stages = len(cfg["stages"])
        for i, (w, n) in enumerate(cfg["stages"]):
            c.stage_width[i], c.stage_convs[i] = w, n
    else:
        c.layers, c.seq, c.hidden, c.heads, c.ffn = (cfg["layers"], cfg["seq"], cfg["hidden"], cfg["heads"],
                                                     cfg["ffn"])
    h = _VP()
    _check(_L().fluid_build_transformer(C.byref(c), C.byref(h)))
    return h


def fluid_build_graph(desc: dict):
    """desc: the canonical dict form (dtype, inputs, consts, nodes, outputs)."""
    ni, nc, nn = len(desc["inputs"]), len(desc["consts"]), len(desc["nodes"])
    irank = (C.c_int32 * max(ni, 1))(*[len(s) for s in desc["inputs"]])
    ishape = (C.c_int64 * (max(ni, 1) * MAX_RANK))()
    for i, s in enumerate(desc["inputs"]):
        for j, d in enumerate(s):
            ishape[i * MAX_RANK + j] = d
    crank = (C.c_int32 * max(nc, 1))(*[len(c["shape"]) for c in desc["consts"]])
    cshape = (C.c_int64 * (max(nc, 1) * MAX_RANK))()
    cdt = (C.c_int32 * max(nc, 1))(*[BF16 if c["dtype"] == "bf16" else F32 for c in desc["consts"]])
    crole = (C.c_int32 * max(nc, 1))(*[ROLES.get(c.get("role", "other"), 0) for c in desc["consts"]])
    for i, c in enumerate(desc["consts"]):
        for j, d in enumerate(c["shape"]):
            cshape[i * MAX_RANK + j] = d
    nodes = (NodeDesc * max(nn, 1))()
    for i, nd in enumerate(desc["nodes"]):
        x = nodes[i]
        x.op = OPS[nd["op"]]
        x.n_in = len(nd["ins"])
        for j, v in enumerate(nd["ins"]):
            x.in_[j] = v
        x.out_rank = len(nd["out_shape"])
        for j, d in enumerate(nd["out_shape"]):
            x.out_shape[j] = d
        for j, p in enumerate(nd.get("perm", [])):
            x.perm[j] = p
        x.f_attr[0] = nd.get("fattr", 0.0)
        x.i_attr[0] = nd.get("iattr", 0)
    outs = (C.c_int32 * max(len(desc["outputs"]), 1))(*desc["outputs"])
    gd = GraphDesc(BF16 if desc["dtype"] == "bf16" else F32, ni, irank, ishape, nc, crank, cshape,
                   cdt, crole, nn, nodes, len(desc["outputs"]), outs)
    h = _VP()
    _check(_L().fluid_build_graph(C.byref(gd), C.byref(h)))
    return h


def fluid_graph_info(g):
    v = [C.c_int32() for _ in range(5)]
    _check(_L().fluid_graph_info(g, *[C.byref(x) for x in v]))
    return tuple(x.value for x in v)


def fluid_graph_export_json(g):
    n = C.c_uint64()
    _check(_L().fluid_graph_export_json(g, None, 0, C.byref(n)))
    buf = C.create_string_buffer(n.value + 1)
    _check(_L().fluid_graph_export_json(g, buf, n.value + 1, C.byref(n)))
    return buf.value.decode()


def fluid_cost_table_load(path, g):
    h = _VP()
    _check(_L().fluid_cost_table_load(str(path).encode(), g, C.byref(h)))
    return h


def fluid_cost_table_save(t, path):
    _check(_L().fluid_cost_table_save(t, str(path).encode()))


def fluid_measure_scratch_bytes(g):
    n = C.c_uint64()
    _check(_L().fluid_measure_scratch_bytes(g, C.byref(n)))
    return n.value


def fluid_measure_costs(g, reps, scratch_ptr, scratch_bytes, stream):
    h = _VP()
    _check(_L().fluid_measure_costs(g, reps, scratch_ptr, scratch_bytes, stream, C.byref(h)))
    return h


def fluid_plan_layouts(g, t, flags=0):
    h = _VP()
    _check(_L().fluid_plan_layouts(g, t, flags, C.byref(h)))
    return h


def fluid_layout_plan_get(lp, n_edges, n_nodes):
    lay = (C.c_int32 * n_edges)()
    var = (C.c_int32 * n_nodes)()
    tot = C.c_int64()
    gu = C.c_int32()
    _check(_L().fluid_layout_plan_get(lp, lay, var, C.byref(tot), C.byref(gu)))
    return list(lay), list(var), tot.value, gu.value


def fluid_edge_layout(g, lp, edge, rank):
    p = (C.c_int32 * MAX_RANK)()
    _check(_L().fluid_edge_layout(g, lp, edge, p))
    return tuple(p[:rank])


def fluid_plan_arena(g, lp, align=256, flags=0):
    h = _VP()
    _check(_L().fluid_plan_arena(g, lp, align, flags, C.byref(h)))
    return h


def fluid_arena_plan_get(ap, n_edges):
    peak, naive, lb = C.c_uint64(), C.c_uint64(), C.c_uint64()
    off = (C.c_int64 * n_edges)()
    root = (C.c_int32 * n_edges)()
    _check(_L().fluid_arena_plan_get(ap, C.byref(peak), C.byref(naive), C.byref(lb), off, root))
    return peak.value, naive.value, lb.value, list(off), list(root)


def fluid_arena_plan_lifetimes(ap, n_edges):
    size = (C.c_uint64 * n_edges)()
    d = (C.c_int32 * n_edges)()
    last = (C.c_int32 * n_edges)()
    _check(_L().fluid_arena_plan_lifetimes(ap, n_edges, size, d, last))
    return list(size), list(d), list(last)


def _ptr_array(ptrs):
    arr = (_VP * max(len(ptrs), 1))()
    for i, p in enumerate(ptrs):
        arr[i] = p
    return arr


def fluid_run(g, lp, ap, arena_ptr, arena_bytes, const_ptrs, input_ptrs, output_ptrs, stream):
    _check(_L().fluid_run(g, lp, ap, arena_ptr, arena_bytes, _ptr_array(const_ptrs),
                          _ptr_array(input_ptrs), _ptr_array(output_ptrs), stream))


def fluid_constant_layout(g, lp, c, rank):
    p = (C.c_int32 * max(rank, 1))()
    _check(_L().fluid_constant_layout(g, lp, c, p))
    return tuple(p[:rank])


def fluid_pack_constant(g, lp, c, src_ptr, dst_ptr, stream):
    _check(_L().fluid_pack_constant(g, lp, c, src_ptr, dst_ptr, stream))


def fluid_run_static(g, lp, ap, const_ptrs, input_ptrs, output_ptrs, stream):
    _check(_L().fluid_run_static(g, lp, ap, _ptr_array(const_ptrs), _ptr_array(input_ptrs),
                                 _ptr_array(output_ptrs), stream))


def fluid_run_nodes(g, lp, ap, arena_ptr, arena_bytes, const_ptrs, input_ptrs, output_ptrs, nodes, repeat,
                    stream):
    arr = (C.c_int32 * len(nodes))(*nodes)
    _check(_L().fluid_run_nodes(g, lp, ap, arena_ptr, arena_bytes, _ptr_array(const_ptrs),
                                _ptr_array(input_ptrs), _ptr_array(output_ptrs), arr, len(nodes), repeat,
                                stream))


def fluid_run_launches(g, lp, ap):
    n = C.c_int32(0)
    _check(_L().fluid_run_launches(g, lp, ap, C.byref(n)))
    return n.value


def fluid_run_schedule(g, lp, ap, n_nodes):
    """(launch index per node, output-written flag per node, kernel name per
    launch)."""
    need = C.c_uint64(0)
    _check(_L().fluid_run_schedule(g, lp, ap, None, None, None, 0, C.byref(need), None))
    launch = (C.c_int32 * n_nodes)()
    written = (C.c_uint8 * n_nodes)()
    buf = C.create_string_buffer(need.value)
    n = C.c_int32(0)
    _check(_L().fluid_run_schedule(g, lp, ap, launch, written, buf, need.value, None, C.byref(n)))
    names = buf.value.decode().split("\n") if n.value else []
    return list(launch), [bool(w) for w in written], names


def fluid_trace_enable(g, mask, max_records):
    m = None
    if mask is not None:
        m = (C.c_uint8 * len(mask))(*[1 if x else 0 for x in mask])
    _check(_L().fluid_trace_enable(g, m, max_records))


def fluid_trace_collect(g, n_nodes):
    ms = (C.c_double * n_nodes)()
    cnt = (C.c_int32 * n_nodes)()
    _check(_L().fluid_trace_collect(g, ms, cnt))
    return list(ms), list(cnt)


def fluid_node_kernel(g, lp, node):
    buf = C.create_string_buffer(128)
    _check(_L().fluid_node_kernel(g, lp, node, buf, 128))
    return buf.value.decode()


# ----------------------------------------------------------------- handles
class Graph:
    def __init__(self, handle):
        self.h = handle
        self.n_inputs, self.n_consts, self.n_nodes, self.n_edges, dt = fluid_graph_info(handle)
        self.dtype = "bf16" if dt == BF16 else "f32"
        self.desc = json.loads(fluid_graph_export_json(handle))

    @classmethod
    def transformer(cls, cfg):
        return cls(fluid_build_transformer(cfg))

    @classmethod
    def from_desc(cls, desc):
        return cls(fluid_build_graph(desc))

    def edge_shape(self, e):
        if e < self.n_inputs:
            return tuple(self.desc["inputs"][e])
        return tuple(self.desc["nodes"][e - self.n_inputs]["out_shape"])

    def const_specs(self):
        return [(c["role"], tuple(c["shape"])) for c in self.desc["consts"]]

    def __del__(self):
        if getattr(self, "h", None) and _lib is not None:
            _lib.fluid_graph_free(self.h)
            self.h = None


class CostTable:
    def __init__(self, handle, graph):
        self.h, self.graph = handle, graph

    @classmethod
    def load(cls, path, graph):
        return cls(fluid_cost_table_load(path, graph.h), graph)

    @classmethod
    def measure(cls, graph, reps=7, device="cuda"):
        import torch
        nbytes = fluid_measure_scratch_bytes(graph.h)
        scratch = torch.empty(nbytes + 256, dtype=torch.uint8, device=device)
        ptr = (scratch.data_ptr() + 255) // 256 * 256
        h = fluid_measure_costs(graph.h, reps, ptr, nbytes, torch.cuda.current_stream().cuda_stream)
        del scratch
        return cls(h, graph)

    def save(self, path):
        fluid_cost_table_save(self.h, path)

    def __del__(self):
        if getattr(self, "h", None) and _lib is not None:
            _lib.fluid_cost_table_free(self.h)
            self.h = None


class LayoutPlan:
    def __init__(self, graph, table, flags=0):
        self.graph = graph
        self.h = fluid_plan_layouts(graph.h, table.h, flags)
        self.layout_idx, self.variant, self.total_ns, self.guard_used = fluid_layout_plan_get(
            self.h, graph.n_edges, graph.n_nodes)
        fz = (C.c_int32 * max(graph.n_nodes, 1))()
        priced = C.c_int32(0)
        _check(_L().fluid_layout_plan_fusion(self.h, fz, C.byref(priced)))
        self.fuse = list(fz)[:graph.n_nodes]
        self.fusion_priced = bool(priced.value)

    def perm(self, e):
        return fluid_edge_layout(self.graph.h, self.h, e, len(self.graph.edge_shape(e)))

    def kernel(self, n):
        return fluid_node_kernel(self.graph.h, self.h, n)

    def constant_layout(self, c):
        """The permutation constant c is stored in for runs of this plan."""
        return fluid_constant_layout(self.graph.h, self.h, c, len(self.graph.desc["consts"][c]["shape"]))

    def __del__(self):
        if getattr(self, "h", None) and _lib is not None:
            _lib.fluid_layout_plan_free(self.h)
            self.h = None


class ArenaPlan:
    def __init__(self, graph, lplan, align=256, no_reuse=False, epilogue=False):
        self.graph = graph
        flags = (ARENA_NO_REUSE if no_reuse else 0) | (ARENA_EPILOGUE if epilogue else 0)
        self.h = fluid_plan_arena(graph.h, lplan.h, align, flags)
        self.peak, self.naive, self.lower_bound, self.offset, self.root = fluid_arena_plan_get(
            self.h, graph.n_edges)

    def lifetimes(self):
        """{buffer edge: (bytes, producer node, last reader node)}."""
        size, d, last = fluid_arena_plan_lifetimes(self.h, self.graph.n_edges)
        return {e: (size[e], d[e], last[e]) for e in range(self.graph.n_edges) if d[e] >= 0}

    def __del__(self):
        if getattr(self, "h", None) and _lib is not None:
            _lib.fluid_arena_plan_free(self.h)
            self.h = None


class Executor:
    """Device buffers (torch) for one graph + plans, and the fluid_run call."""

    def __init__(self, graph, lplan, aplan, consts, inputs, device="cuda"):
        import torch
        self.torch = torch
        self.graph, self.lplan, self.aplan = graph, lplan, aplan
        dt = torch.bfloat16 if graph.dtype == "bf16" else torch.float32
        self.consts = []
        for c, a in zip(graph.desc["consts"], consts):
            cdt = torch.bfloat16 if c["dtype"] == "bf16" else torch.float32
            self.consts.append(torch.as_tensor(a).to(device=device, dtype=cdt).contiguous())
        # weights the plan packs (fluid_constant_layout) are rewritten once,
        # by the library, into buffers of their own
        s = torch.cuda.current_stream().cuda_stream
        for c, t in enumerate(self.consts):
            perm = lplan.constant_layout(c)
            if perm != tuple(range(len(perm))):
                packed = torch.empty_like(t)
                fluid_pack_constant(graph.h, lplan.h, c, t.data_ptr(), packed.data_ptr(), s)
                self.consts[c] = packed
        torch.cuda.synchronize()
        self.inputs = [torch.as_tensor(a).to(device=device, dtype=dt).contiguous() for a in inputs]
        self.outputs = [torch.empty(graph.edge_shape(e), dtype=dt, device=device)
                        for e in graph.desc["outputs"]]
        self.arena = torch.empty(max(aplan.peak, 1) + 256, dtype=torch.uint8, device=device)
        self.arena_ptr = (self.arena.data_ptr() + 255) // 256 * 256
        self._cp = [t.data_ptr() for t in self.consts]
        self._ip = [t.data_ptr() for t in self.inputs]
        self._op = [t.data_ptr() for t in self.outputs]

    def run(self, stream=None):
        s = stream if stream is not None else self.torch.cuda.current_stream().cuda_stream
        fluid_run(self.graph.h, self.lplan.h, self.aplan.h, self.arena_ptr, self.aplan.peak,
                  self._cp, self._ip, self._op, s)
        return self.outputs

    def launches(self):
        """Kernel launches one run enqueues (nodes performed in a MatMul's
        epilogue, and products launched together with an earlier one, are
        not counted)."""
        return fluid_run_launches(self.graph.h, self.lplan.h, self.aplan.h)

    def schedule(self):
        """(launch index per node, output-written flag per node, kernel name
        per launch) of one run."""
        return fluid_run_schedule(self.graph.h, self.lplan.h, self.aplan.h, self.graph.n_nodes)

    def run_nodes(self, nodes, repeat=1, stream=None):
        """Launch only the kernels of ``nodes`` (in list order), ``repeat``
        times over, with the bindings of a full run (profiling aid)."""
        s = stream if stream is not None else self.torch.cuda.current_stream().cuda_stream
        fluid_run_nodes(self.graph.h, self.lplan.h, self.aplan.h, self.arena_ptr, self.aplan.peak,
                        self._cp, self._ip, self._op, list(nodes), repeat, s)

    def capture(self, steps=1):
        """Record ``steps`` consecutive fluid_run calls into one HIP graph
        (torch.cuda.CUDAGraph); replaying it re-issues the same launches
        with one submission.  fluid_run only launches kernels, so the graph
        holds kernel nodes (plus event nodes while tracing)."""
        torch = self.torch
        graph = torch.cuda.CUDAGraph()
        s = torch.cuda.Stream()
        s.wait_stream(torch.cuda.current_stream())
        with torch.cuda.graph(graph, stream=s):
            for _ in range(steps):
                self.run(s.cuda_stream)
        torch.cuda.current_stream().wait_stream(s)
        return graph
