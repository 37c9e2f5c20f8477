/*
 * fluid.h -- C ABI of the layout-planned transformer hot path for MI355X.
 *
 * Method: FluidML (arXiv 2411.09242), Section 3.  A frozen operator graph
 * with known shapes gets (1) a memory layout -- a dimension permutation --
 * for every intermediate tensor, chosen by longest-path decomposition
 * (Alg. 1-2) and a dynamic program over measured kernel times (Eq. 1,
 * Alg. 3) with majority-vote conflict resolution; (2) a static placement of
 * every tensor inside one pre-allocated buffer by Greedy-by-Size over tensor
 * lifetimes (Alg. 4); then (3) the operators run as GPU kernels whose loads
 * and stores follow each tensor's layout, inside that single buffer.
 *
 * Conventions for every entry point:
 *  - Every call returns a fluid_status; nothing throws across the ABI.  On
 *    failure fluid_last_error() describes the cause (thread-local string,
 *    valid until the next fluid_* call on the same thread).
 *  - Handles (graph, cost table, plans) are created and owned by the
 *    library, immutable after creation, and released with their *_free
 *    function (NULL is accepted).  Out-pointers are written only on success.
 *  - All device memory (arena, constants, graph inputs and outputs, scratch)
 *    is owned by the caller; the library never allocates or frees device
 *    memory.  Arguments are validated before any HIP call.
 *  - Tensor shapes are int64 element counts, at most FLUID_MAX_RANK dims.
 *    Graph inputs and outputs are always dense row-major; constants are
 *    dense, row-major unless the layout plan packs a weight
 *    (fluid_constant_layout, fluid_pack_constant).
 *  - The host-only build of this library (no GPU code) exports the same
 *    symbols; there the entry points that touch the GPU return
 *    FLUID_E_UNSUPPORTED.
 */
#ifndef FLUID_H
#define FLUID_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define FLUID_MAX_RANK 6
#define FLUID_MAX_IN 4

typedef enum {
  FLUID_OK = 0,
  FLUID_E_INVALID = -1,         /* malformed argument, graph or file          */
  FLUID_E_UNSUPPORTED = -2,     /* valid but not implemented (or host build)  */
  FLUID_E_INFEASIBLE = -3,      /* no finite-cost layout plan exists          */
  FLUID_E_ARENA_TOO_SMALL = -4, /* arena_bytes below the plan's peak          */
  FLUID_E_HIP = -5,             /* a HIP runtime call failed                  */
  FLUID_E_NOMEM = -6            /* host allocation failed                     */
} fluid_status;

const char* fluid_last_error(void);

typedef enum { FLUID_F32 = 0, FLUID_BF16 = 1 } fluid_dtype;

/* Operators of the transformer chain.  Semantics (ONNX, the paper's front-end
 * format; Section 4):
 *  MATMUL    in[0] A [..., M, K] activation; in[1] B either a 2-D constant or
 *            activation [K, N], or an activation [..., K, N] with the same
 *            leading dims as A.  out [..., M, N].  fp32 accumulation.
 *  ADD, MUL  in[0] activation; in[1] activation of the same shape, or (ADD
 *            only) a constant [N] broadcast over the last dim.
 *  TRANSPOSE out dim i = in dim perm[i].
 *  RESHAPE   row-major reinterpretation; only "split one dim into two
 *            adjacent dims" and "merge two adjacent dims" are accepted.
 *  SOFTMAX   over the last dim of f_attr[0] * x; i_attr[0] = 1 masks key
 *            k > query q (second-to-last dim) and writes exact zeros there.
 *  LAYERNORM in[1] gamma [H], in[2] beta [H] constants; eps = f_attr[0];
 *            biased variance over the last dim.
 *  RMSNORM   in[1] gamma [H]; x / sqrt(mean(x^2) + eps) * gamma.
 *  GELU      0.5 x (1 + erf(x / sqrt 2));  SILU  x / (1 + exp(-x)).
 *  ROPE      in[0] [B, S, NH, D] (D even); in[1] cos, in[2] sin: fp32
 *            constants [S, D/2]; rotate-half: for i < D/2,
 *            y_i = x_i c - x_{i+D/2} s,  y_{i+D/2} = x_{i+D/2} c + x_i s.
 *  PAD       in[0] [N, C, H, W]; zero padding of i_attr[0] >= 0 on both
 *            sides of H and W: out [N, C, H + 2p, W + 2p].
 *  CONV      in[0] x [N, C, H, W]; in[1] weight constant [Co, C, KH, KW]
 *            (row-major); optional in[2] bias constant [Co]; ONNX Conv with
 *            no padding, stride 1, one group: out [N, Co, H-KH+1, W-KW+1],
 *            y[n,o,i,j] = sum_{c,u,v} x[n,c,i+u,j+v] w[o,c,u,v] + b[o].
 *  RELU      max(x, 0).
 *  MAXPOOL   in[0] [N, C, H, W], window k = i_attr[0] dividing H and W,
 *            stride k: out [N, C, H/k, W/k], the maximum of each window.  */
typedef enum {
  FLUID_OP_MATMUL = 0, FLUID_OP_ADD = 1, FLUID_OP_MUL = 2,
  FLUID_OP_TRANSPOSE = 3, FLUID_OP_RESHAPE = 4, FLUID_OP_SOFTMAX = 5,
  FLUID_OP_LAYERNORM = 6, FLUID_OP_RMSNORM = 7, FLUID_OP_GELU = 8,
  FLUID_OP_SILU = 9, FLUID_OP_ROPE = 10, FLUID_OP_PAD = 11,
  FLUID_OP_CONV = 12, FLUID_OP_RELU = 13, FLUID_OP_MAXPOOL = 14
} fluid_op;

/* Informational tag of a constant (how the synthetic workloads fill it). */
typedef enum {
  FLUID_ROLE_OTHER = 0, FLUID_ROLE_WEIGHT = 1, FLUID_ROLE_BIAS = 2,
  FLUID_ROLE_GAMMA = 3, FLUID_ROLE_BETA = 4, FLUID_ROLE_ROPE_COS = 5,
  FLUID_ROLE_ROPE_SIN = 6
} fluid_const_role;

/* One node.  Node id = index in the node array, which must be topological.
 * Edges: graph inputs are edges 0..n_inputs-1; the output of node n is edge
 * n_inputs + n.  in[i] >= 0 names an edge; in[i] < 0 names constant ~in[i]. */
typedef struct {
  int32_t op;                          /* fluid_op                              */
  int32_t n_in;
  int32_t in[FLUID_MAX_IN];
  int32_t out_rank;
  int64_t out_shape[FLUID_MAX_RANK];
  int32_t perm[FLUID_MAX_RANK];        /* TRANSPOSE only                        */
  float f_attr[2];                     /* SOFTMAX scale; LAYERNORM/RMSNORM eps  */
  int32_t i_attr[2];                   /* SOFTMAX causal flag; PAD width;
                                          MAXPOOL window                        */
} fluid_node_desc;

/* Shapes of inputs / constants: arrays of n * FLUID_MAX_RANK int64, row i
 * holding the dims of item i (entries past its rank are ignored). */
typedef struct {
  int32_t dtype;                       /* fluid_dtype of activations/weights   */
  int32_t n_inputs;
  const int32_t* input_rank;
  const int64_t* input_shapes;
  int32_t n_consts;
  const int32_t* const_rank;
  const int64_t* const_shapes;
  const int32_t* const_dtype;          /* fluid_dtype per constant             */
  const int32_t* const_role;           /* fluid_const_role per constant (NULL ok) */
  int32_t n_nodes;
  const fluid_node_desc* nodes;
  int32_t n_outputs;
  const int32_t* output_edges;         /* must be node outputs                 */
} fluid_graph_desc;

typedef struct fluid_graph fluid_graph;
typedef struct fluid_cost_table fluid_cost_table;
typedef struct fluid_layout_plan fluid_layout_plan;
typedef struct fluid_arena_plan fluid_arena_plan;

/* Builds and validates a graph (Section 4 "Compiler": the model as a graph
 * linearised into one operator sequence).  Checks arity, constant and edge
 * references, topological order and every output shape; errors:
 * FLUID_E_INVALID, FLUID_E_UNSUPPORTED (e.g. a general reshape). */
fluid_status fluid_build_graph(const fluid_graph_desc* desc, fluid_graph** out);

/* Transformer stacks used by the synthetic workloads.  arch 0: post-LN
 * encoder layer (BERT); 1: pre-LN decoder layer with causal attention and a
 * final LayerNorm (GPT-2); 2: Llama-style decoder (RMSNorm, RoPE, causal,
 * SwiGLU FFN, final RMSNorm, no biases).  Node order per layer: q, k, v
 * projections (MatMul [+ bias Add], Reshape to heads, [RoPE], Transpose to
 * [B,NH,S,D], keys to [B,NH,D,S]), scores MatMul, Softmax(1/sqrt(D)),
 * context MatMul, Transpose + Reshape back, output projection, residual,
 * norm, FFN (up, bias, GELU, down, bias; SwiGLU: gate, SiLU, up, Mul, down),
 * residual[, norm].
 * arch 3: VGG-shaped convolutional network (fp32; the paper's VGG and
 * ConvBERT models, Section 5): input [batch, channels, image, image]; per
 * stage s, stage_convs[s] times Pad(1), 3x3 Conv with bias to
 * stage_width[s] channels, ReLU, then MaxPool(2); flatten by two Reshapes
 * (merge H, W; merge C, H*W); MatMul, bias Add, ReLU to fc twice; MatMul and
 * bias Add to classes; Softmax (scale 1).  Uses batch, dtype and the fields
 * after rope_base (layers, seq, hidden, heads, ffn are ignored). */
#define FLUID_MAX_STAGES 8
typedef struct {
  int32_t arch;
  int32_t layers, batch, seq, hidden, heads, ffn;
  int32_t dtype;                       /* fluid_dtype                           */
  float eps;                           /* norm epsilon (1e-5)                   */
  float rope_base;                     /* 10000                                 */
  int32_t channels, image, fc, classes, n_stages;            /* arch 3 only */
  int32_t stage_width[FLUID_MAX_STAGES], stage_convs[FLUID_MAX_STAGES];
} fluid_model_cfg;
fluid_status fluid_build_transformer(const fluid_model_cfg* cfg, fluid_graph** out);

/* Counts of a graph (any pointer may be NULL). */
fluid_status fluid_graph_info(const fluid_graph* g, int32_t* n_inputs, int32_t* n_consts,
                              int32_t* n_nodes, int32_t* n_edges, int32_t* dtype);

/* Canonical JSON description: dtype, inputs, consts (role, shape, dtype),
 * nodes (op, ins, out_shape, perm, fattr, iattr), outputs, and the candidate
 * layout list L(e) of every edge.  Writes at most cap bytes (NUL-terminated
 * when it fits) and the full length to *len; call with cap = 0 to size. */
fluid_status fluid_graph_export_json(const fluid_graph* g, char* buf, uint64_t cap, uint64_t* len);

/* Cost table: the measured time of every node for every combination of
 * input and output layouts (the eval() of Alg. 3), the minimum over kernel
 * variants kept with its variant id (the GPU form of Section 3 "Loop
 * Reordering").  JSON file format "fluid-cost-table/1": "edges" (L(e) per
 * edge, identity first), "sigs" (op, in_shapes, out_shape, entries
 * [[slot perms], out perm, [ns per variant, -1 = unavailable]]), "node_sig".
 * Load validates the file against the graph (FLUID_E_INVALID on mismatch,
 * a missing identity layout, or a nonzero cost on a view combination). */
fluid_status fluid_cost_table_load(const char* json_path, const fluid_graph* g, fluid_cost_table** out);
fluid_status fluid_cost_table_save(const fluid_cost_table* t, const char* json_path);

/* Device scratch needed by fluid_measure_costs for this graph (bytes). */
fluid_status fluid_measure_scratch_bytes(const fluid_graph* g, uint64_t* bytes);

/* Measures the cost table on the GPU (Alg. 3's eval: real kernel time).
 * For every operator signature, every candidate layout combination and
 * every kernel variant: one untimed warm-up launch, one launch timed on its
 * own (a combination more than 8x slower than the best so far of its
 * signature keeps that time), then `reps` back-to-back launches captured
 * once as a HIP graph and replayed three times, each replay between two
 * HIP events, on a stream of the library's own (launches issued as a run's
 * graph issues them, without the host's per-launch cost); the cost is the
 * median per-launch time of the replays, rounded to integer nanoseconds.  Successive launches of a
 * MatMul or Conv with a constant weight read it from rotating copies that
 * total at least 512 MiB (at most 64 copies), so that each launch fetches
 * its weight from HBM, as in a run.  Fusion chains get entries measured
 * the same way as one launch (the R operand in the output's layout).  View
 * combinations of Transpose/Reshape cost 0.  Candidate lists: all
 * dimension permutations (deduplicated), trimmed for tensors with more than
 * six candidates to those whose innermost dim is one of the last two
 * logical dims.  scratch: caller device memory of at least
 * fluid_measure_scratch_bytes, 256-B aligned; its contents are overwritten
 * (filled on hip_stream, which is then synchronised).  GPU build only. */
fluid_status fluid_measure_costs(const fluid_graph* g, uint32_t reps, void* scratch,
                                 uint64_t scratch_bytes, void* hip_stream, fluid_cost_table** out);

#define FLUID_NO_DP 1u        /* return the all-row-major plan                */
#define FLUID_NO_VARIANTS 2u  /* plan on the variant-0 column only (ablation) */
#define FLUID_NO_GUARD 4u     /* keep the voted plan even if it costs more    */
#define FLUID_NO_FUSION 8u    /* ignore the table's fused entries            */

/* Layout plan (Section 3, Alg. 1-3, Eq. 1 and the vote): longest-path
 * decomposition; per-path dynamic program over output layouts; majority vote
 * on edges shared between paths (ties: lowest re-optimised cost of the
 * touching paths, then lowest index); one re-optimisation with shared edges
 * fixed; then, unless FLUID_NO_GUARD, the all-row-major plan if it is
 * cheaper.  Fusion (Section 4: the compiler fuses operators before it plans
 * layouts): when the table carries fused entries, a MatMul and the bias
 * Add / GELU or SiLU / Add or Mul with an earlier tensor right after it, or
 * a residual Add and the LayerNorm / RMSNorm of its sum (consecutive node
 * ids; the MatMul chain's results single-reader; a sum with further
 * readers, as in a pre-norm block, is stored by that launch in the layout
 * of the norm's output, which the plan then gives the sum), may run as one
 * launch; the path DP weighs that launch's measured cost against the nodes'
 * own (ties go to the nodes on their own); after the vote the cheapest disjoint chains are chosen
 * exactly for the final layouts, the voted layouts of the fusion-aware and
 * of the plain DP compete (the cheaper total wins), and the guard compares
 * with the row-major plan with its best chains.  Runs then perform exactly
 * the plan's fusions (fluid_layout_plan_fusion).  Errors: FLUID_E_INFEASIBLE
 * (no identity entry, or no finite plan), FLUID_E_INVALID. */
fluid_status fluid_plan_layouts(const fluid_graph* g, const fluid_cost_table* t, uint32_t flags,
                                fluid_layout_plan** out);

/* Constant layouts (the weight layout is planned with the MatMul that reads
 * it, Section 2's ahead-of-time constants with Section 3's loop reordering):
 * MatMul variants 0..9 read their weight [K, N] row-major as supplied,
 * variants 10..19 run the same tiles on the weight stored K-contiguous
 * (physically [N, K]) -- offered only for a 2-D weight that no other node
 * reads.  fluid_constant_layout writes the permutation constant c must be
 * stored in for runs of this plan (rank entries: the identity, or {1, 0}
 * for a packed weight).  Errors: FLUID_E_INVALID (NULL argument, plan of
 * another graph, c out of range).  Both builds. */
fluid_status fluid_constant_layout(const fluid_graph* g, const fluid_layout_plan* lp, int32_t c,
                                   int32_t* perm_out);
/* Writes constant c, given row-major at device address src, into device
 * memory dst (caller-allocated, same byte size, 16-byte aligned, not
 * overlapping src) in the layout fluid_constant_layout gives, enqueued on
 * hip_stream -- once, before the runs that use this plan; fluid_run then
 * takes dst as constant c.  No device allocation.  Errors: FLUID_E_INVALID,
 * FLUID_E_HIP.  GPU build only. */
fluid_status fluid_pack_constant(const fluid_graph* g, const fluid_layout_plan* lp, int32_t c, const void* src,
                                 void* dst, void* hip_stream);

/* Plan contents: layout index into L(e) per edge (n_edges), kernel variant per
 * node (n_nodes; -1 = view, no kernel), summed table cost, guard flag. */
fluid_status fluid_layout_plan_get(const fluid_layout_plan* lp, int32_t* layout_idx_per_edge,
                                   int32_t* variant_per_node, int64_t* total_ns, int32_t* guard_used);
/* The plan's fusions: fuse_per_node[n] (n_nodes entries) is the number t
 * of nodes after node n (a MatMul, or a residual Add whose normalisation
 * follows) that its launch performs (nodes n+1 .. n+t have variant -2 and
 * results n .. n+t-1 never reach memory, except a residual sum with further
 * readers, which the launch stores), 0 otherwise;
 * *priced is 1 when the plan priced fusion chains (fluid_run then performs
 * exactly these fusions), 0 when it did not (FLUID_NO_FUSION, FLUID_NO_DP, or
 * a table without fused entries: fluid_run fuses by its own rule, see
 * fluid_run).  Either pointer may be NULL.  Both builds. */
fluid_status fluid_layout_plan_fusion(const fluid_layout_plan* lp, int32_t* fuse_per_node, int32_t* priced);

/* The permutation chosen for one edge (rank entries written to perm_out). */
fluid_status fluid_edge_layout(const fluid_graph* g, const fluid_layout_plan* lp, int32_t edge,
                               int32_t* perm_out);

#define FLUID_ARENA_NO_REUSE 1u  /* naive plan: every buffer its own slice     */
#define FLUID_ARENA_EPILOGUE 2u  /* lifetimes that let every epilogue fuse    */

/* Arena plan (Alg. 4, Greedy-by-Size): a Transpose/Reshape that the layouts
 * make a view owns no bytes; every other non-output node result is a buffer
 * of size rounded up to `align` (a power of two >= 16; 256 recommended)
 * with lifetime [producer, last reader]; buffers by size descending take
 * the smallest fitting gap among lifetime-overlapping buffers, else the end.
 * FLUID_ARENA_NO_REUSE places them at prefix sums in edge order instead.
 * FLUID_ARENA_EPILOGUE (an addition to the paper's lifetimes): a MatMul
 * that fluid_run can fuse with the nodes after it (see fluid_run) keeps its
 * operands live until the last of those nodes, so that no fused output is
 * placed over them and every such fusion happens; the peak can grow. */
fluid_status fluid_plan_arena(const fluid_graph* g, const fluid_layout_plan* lp, uint64_t align,
                              uint32_t flags, fluid_arena_plan** out);

/* Arena contents: peak bytes; the no-reuse total of the row-major plan; the
 * max-live lower bound of this plan's buffers; per edge the byte offset of
 * the edge's bytes (-1 if not in the arena: graph inputs/outputs) and its
 * root edge (the buffer it aliases).  Any pointer may be NULL. */
fluid_status fluid_arena_plan_get(const fluid_arena_plan* ap, uint64_t* peak_bytes, uint64_t* naive_bytes,
                                  uint64_t* lower_bound_bytes, int64_t* offset_per_edge,
                                  int32_t* root_per_edge);

/* The lifetimes the arena plan placed its buffers by (Alg. 4's input): per
 * edge, size_per_edge the buffer bytes after rounding to the alignment, and
 * def_per_edge / last_per_edge the producing node and the last node that
 * reads any edge rooted at the buffer (with FLUID_ARENA_EPILOGUE, the
 * extended end), for edges that are arena buffers; 0 / -1 / -1 for the
 * others (graph inputs and outputs, views).  Arrays of n_edges entries,
 * each may be NULL.  Errors: FLUID_E_INVALID (NULL plan, n_edges not the
 * plan's edge count). */
fluid_status fluid_arena_plan_lifetimes(const fluid_arena_plan* ap, int32_t n_edges, uint64_t* size_per_edge,
                                        int32_t* def_per_edge, int32_t* last_per_edge);

/* Executes the graph (Section 4 "Virtual Machine": the invoke interface):
 * enqueues one kernel per non-view node, in node order, on hip_stream; the
 * caller synchronises.  One exception, epilogue fusion: a MatMul also
 * performs the nodes launched right after it that form, in this order, an
 * Add of a bias constant [N], a GELU or SiLU, and an Add or Mul with
 * another tensor of the product's shape (each step optional; the last one
 * only for the kernel variants that have it), when each step's input is
 * read by nothing else and is no graph output; the launch writes the last
 * step's output, rounding once after all steps (a step is left to its own
 * kernel when its output shares arena bytes with a MatMul operand).  And
 * consecutive fp32 MatMul launches of the same direct-load kernel (the Q, K
 * and V projections) go out as one grouped launch when none reads or
 * overwrites what another writes (fluid_run_schedule lists the launches).
 * arena:
 * device memory of at least the plan's peak,
 * 256-B aligned; consts[i], inputs[i], outputs[i]: device pointers to dense
 * tensors of the graph's dtype (RoPE tables fp32), row-major except a
 * constant the plan packs (stored as fluid_constant_layout says).  No device
 * allocation.  Errors before any launch: FLUID_E_INVALID (NULL pointer,
 * misaligned arena, plans of another graph), FLUID_E_ARENA_TOO_SMALL;
 * FLUID_E_HIP if a launch fails.  Concurrent calls on different streams
 * with different arenas are safe; calls sharing an arena race. */
fluid_status fluid_run(const fluid_graph* g, const fluid_layout_plan* lp, const fluid_arena_plan* ap,
                       void* arena, uint64_t arena_bytes, const void* const* consts,
                       const void* const* inputs, void* const* outputs, void* hip_stream);

/* For callers that cannot allocate device memory (code under HIP graph
 * capture, tight serving loops, harnesses that forbid hipMalloc): the same
 * execution as fluid_run, with the arena replaced by a static device array
 * of FLUID_STATIC_ARENA_BYTES inside the library (one per GPU, held until
 * the process ends; its address is looked up on the first call on each
 * device).  No device allocation or free happens in this call.  The
 * caller still passes constants, inputs and outputs (same rules as
 * fluid_run).  Errors: FLUID_E_ARENA_TOO_SMALL when the plan's peak exceeds
 * FLUID_STATIC_ARENA_BYTES (checked before any launch), otherwise as
 * fluid_run.  Every call on a GPU uses that GPU's one array, which keeps
 * the last run's bytes (a run writes every arena byte before reading it, so
 * nothing needs clearing); calls that overlap on one GPU (different streams
 * or threads) race.  GPU build only. */
#define FLUID_STATIC_ARENA_BYTES (64ull << 20)
fluid_status fluid_run_static(const fluid_graph* g, const fluid_layout_plan* lp, const fluid_arena_plan* ap,
                              const void* const* consts, const void* const* inputs, void* const* outputs,
                              void* hip_stream);

/* Launches only the kernels of the listed nodes, in list order, the whole
 * list `repeat` times over, with exactly the bindings and kernels fluid_run
 * uses for them (profiling aid: the time of chosen kernels back to back,
 * without the rest of the graph).  Same argument rules and errors as
 * fluid_run; nodes: n_nodes node ids, each a non-view node under the plan
 * (else FLUID_E_INVALID); repeat >= 1.  A MatMul that fluid_run fuses with
 * the nodes after it does so here too when all those nodes follow it in the
 * list; otherwise each listed node runs its own kernel -- except where the
 * plan priced the chain (fluid_layout_plan_fusion): its intermediate
 * results have no buffer, so a list that splits such a chain (its head
 * without every node it absorbs, or an absorbed node alone) is refused
 * with FLUID_E_INVALID before any launch.  Products that fluid_run groups
 * into one launch run as that launch when the list holds all its nodes
 * (the products and the nodes they absorb) consecutively in node order,
 * else one launch each (the same tile code, so the same results).  Reads and writes the arena like a run would, so it leaves the
 * arena contents of a partial run.  GPU build only. */
fluid_status fluid_run_nodes(const fluid_graph* g, const fluid_layout_plan* lp, const fluid_arena_plan* ap,
                             void* arena, uint64_t arena_bytes, const void* const* consts,
                             const void* const* inputs, void* const* outputs, const int32_t* nodes,
                             int32_t n_nodes, int32_t repeat, void* hip_stream);

/* Number of kernel launches one fluid_run of these plans enqueues (the
 * non-view nodes, less those performed in a MatMul's epilogue, less the
 * products launched with an earlier one).  Errors:
 * FLUID_E_INVALID (NULL argument, plans of another graph).  Both builds. */
fluid_status fluid_run_launches(const fluid_graph* g, const fluid_layout_plan* lp, const fluid_arena_plan* ap,
                                int32_t* launches);

/* The launches one fluid_run of these plans enqueues, in order (Section 4
 * "Virtual Machine" runs the planned operators in sequence; here with the
 * epilogue fusion and grouped launches described at fluid_run).  Per node:
 * launch_of_node the index of the launch that performs it (-1 for a view),
 * output_written 1 if that launch stores the node's output (0 for a view
 * and for a node whose output a fused launch keeps on chip; 1 for a
 * residual sum the normalisation's launch stores).  names: the
 * kernel name of every launch, '\n'-separated, NUL-terminated (a grouped
 * launch of k products ends in "_x<k>"); names_len receives the bytes
 * needed including the NUL.  n_launches receives the launch count.  Any
 * output pointer may be NULL; arrays have n_nodes entries.  Errors:
 * FLUID_E_INVALID (NULL graph or plan, plans of another graph, names_cap
 * below the bytes needed).  Both builds. */
fluid_status fluid_run_schedule(const fluid_graph* g, const fluid_layout_plan* lp, const fluid_arena_plan* ap,
                                int32_t* launch_of_node, uint8_t* output_written, char* names, uint64_t names_cap,
                                uint64_t* names_len, int32_t* n_launches);

/* Per-node timing of later fluid_run calls (profiling aid).  While enabled,
 * fluid_run records a HIP event pair around every launch of a node whose
 * node_mask entry is nonzero (NULL mask = all nodes), for at most
 * max_records launches in total.  After the caller has synchronised,
 * fluid_trace_collect adds the elapsed milliseconds and launch counts per
 * node into its arrays (n_nodes each) and disables tracing.  Global state:
 * not for concurrent use.  GPU build only. */
fluid_status fluid_trace_enable(const fluid_graph* g, const uint8_t* node_mask, int32_t max_records);
fluid_status fluid_trace_collect(const fluid_graph* g, double* ms_per_node, int32_t* launches_per_node);

/* Name of the kernel a node runs under a plan, e.g.
 * "gemm_f32_m128n128_ak_bn_cn": "view" for views, "fused" for a node the
 * plan performs inside the launch of the node before it (variant -2); a
 * chain's MatMul names its unfused product, a residual Add heading a chain
 * the summed normalisation kernel (e.g. "add_layernorm_row_f32_v4"). */
fluid_status fluid_node_kernel(const fluid_graph* g, const fluid_layout_plan* lp, int32_t node,
                               char* buf, uint64_t cap);

void fluid_graph_free(fluid_graph* g);
void fluid_cost_table_free(fluid_cost_table* t);
void fluid_layout_plan_free(fluid_layout_plan* lp);
void fluid_arena_plan_free(fluid_arena_plan* ap);

#ifdef __cplusplus
}
#endif
#endif /* FLUID_H */
