/*
 * dirigo_rocm.h -- batched backward dataflow enumeration on MI355X (gfx950).
 *
 * For a fixed-shape tensor-op graph in SSA form and a list of output
 * locations, each call returns the exact input-element footprint of every
 * location together with per-element path counts (Sec. 3.4 of "The
 * Output-Space Hypothesis: Enumerative Equivalence Checking for Tensor
 * Programs", "Per-element equations" and "Back-projection"):
 *
 *   res(y[l]) substitutes each op's per-element equation f_k backwards until
 *   only input (leaf) elements remain; the footprint of l is the set of leaf
 *   elements occurring in res(y[l]) and the path count of a leaf element is
 *   its number of occurrences.
 *
 * Conventions shared by every call:
 *  - A location is a flat row-major index into the output's logical shape
 *    (Sec. 3.3 "Setup": R_y maps flat indices of y).
 *  - A leaf element's global id is base[leaf] + its row-major flat index,
 *    where base is the running element count in leaf declaration order.
 *  - A row lists its leaf elements by ascending global id.  Rows are stored
 *    as CSR: offsets[n+1] (int64) plus two parallel arrays ids[] and
 *    counts[] (uint32, structure of arrays).
 *  - Values never matter: footprints are data independent (Sec. 2, Sec. 3.4
 *    "Flipping the quantifiers"); tensors have shapes only.
 *  - The dataflow reading of each op (which elements it reads and how
 *    often) follows the Torch lowerings of Sec. 3.3: each tensor element is
 *    one variable; activations are uninterpreted functions of their operand;
 *    selects (max, min, clamp) read each operand once; constants (padding,
 *    eps, 1/n) are not variables; softmax reads its slice once and l once
 *    more; a normalisation with statistics set S reads x[s] |S| + 2 times,
 *    x[l] once more, and its affine parameters once.
 *
 * Memory and streams: every device pointer argument is caller-owned device
 * memory (for example a torch tensor's data pointer); `stream` is a
 * hipStream_t passed as void* (NULL = the default stream).  Scratch space is
 * the caller's workspace, sized by dg_workspace_size.  The calls allocate
 * no other device memory, with two exceptions, both made once per graph and
 * device on the graph's first device call there and both released by
 * dg_graph_destroy:
 *  - the graph's compiled plan (a few KB; its expression-DAG program too,
 *    on the first DAG call), copied to the device with hipMalloc;
 *  - with specialisation on, the code object of the graph's kernels
 *    (hipModuleLoadData), shared by graphs whose plans are identical; a
 *    comparison loads one for the pair, released when either graph of the
 *    pair is destroyed; DAG calls that take the specialised DAG kernels
 *    load one for the graph's DAG program.
 *
 * Sizes: a call takes at most 2^31 locations (DG_E_INVALID_ARG beyond);
 * the library splits its launches so that no grid exceeds the device's
 * limit.
 *
 * Errors: every call returns a dg_status; 0 is success, negative values are
 * errors and dg_last_error() returns a message for the calling thread.  No
 * C++ exception crosses this interface.
 *
 * Specialisation: on its first device call, a graph compiles kernels
 * specialised to its plan (hipRTC in a helper process, lib/dirigo_jitc; a
 * few seconds, cached per process); setting the environment variable
 * DIRIGO_JIT=0 keeps the precompiled kernels, which run the same code on
 * the plan as data, and DIRIGO_JIT_INPROC=1 compiles in the calling
 * process.  Expression-DAG calls take DAG kernels specialised to the
 * graph's DAG program by the rule given with dg_graph_info_t
 * (dag_specialized).
 *
 * Thread safety: a dg_graph is immutable after construction and may be used
 * from several host threads and streams at once.  Calls that share one
 * workspace buffer must not overlap in time.
 */
#ifndef DIRIGO_ROCM_H
#define DIRIGO_ROCM_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef int32_t dg_status;

#define DG_OK 0
#define DG_E_INVALID_ARG (-1)    /* null pointer, negative size, bad index */
#define DG_E_PARSE (-2)          /* malformed dgir text */
#define DG_E_SHAPE (-3)          /* inconsistent shapes or attributes */
#define DG_E_UNSUPPORTED_OP (-4) /* op kind, or a form of it, not handled */
#define DG_E_RANGE (-5)          /* a location outside [0, output numel) */
#define DG_E_OVERFLOW (-6)       /* leaf elements beyond 2^62 or a static
                                    path-count bound beyond 2^63; in the
                                    32-bit calls, ids or a path count that
                                    do not fit 32 bits */
#define DG_E_SIGNATURE (-7)      /* compare: leaves or output shape differ */
#define DG_E_WORKSPACE (-8)      /* workspace missing or too small */
#define DG_E_HIP (-9)            /* HIP runtime error (message attached) */
#define DG_E_CAPACITY (-10)      /* the per-location plan of this graph does
                                    not fit the device's local data share */
#define DG_E_BUFFER (-11)        /* dg_enumerate: the rows need more entries
                                    than the output buffers hold */
#define DG_E_STOPPED (-12)       /* dg_enumerate_stream: the chunk consumer
                                    returned nonzero */

#define DG_MAX_RANK 8
#define DG_NAME_LEN 64

typedef struct dg_graph dg_graph;

/* ------------------------------------------------------------------------
 * Graph construction.
 * ------------------------------------------------------------------------
 * dg_graph_parse: builds a graph from dgir v1 text (`len` bytes, not
 * necessarily NUL-terminated):
 *
 *     dgir 1
 *     leaf <name> <d0,d1,...>
 *     op <name> <kind> <operand> [<operand> ...] [; key=value ...]
 *     output <name> <d0,d1,...>
 *
 * Ops are in SSA order (each writes one new tensor and reads earlier ones,
 * Sec. 3.4 "Per-element equations"); the output line names the checked
 * tensor and states its shape, which must equal the inferred one.  Op kinds:
 *   matmul A B                     batched, NumPy-broadcast batch dims
 *   linear x W [b]                 y = x W^T + b, W is [out, in]
 *   conv x W [b]                   stride= pad= dilation= groups=
 *   conv_transpose x W [b]         stride= pad= output_padding= dilation= groups=
 *   max_pool x | avg_pool x        kernel= stride= pad= dilation=
 *   relu gelu gelu_tanh hardtanh clamp sigmoid tanh exp log log1p square sqrt
 *   rsqrt neg abs identity contiguous silu softplus erf scale leaky_relu elu
 *   reciprocal x                   elementwise unary
 *   add sub mul div maximum minimum pow a b   broadcasting binary
 *   sum mean amax amin prod max min x        dims= keepdim=
 *   softmax x | log_softmax x      dim=
 *   group_norm x [g b] groups= | batch_norm x [g b] | layer_norm x [g b] ndims=
 *   channel_affine x scale shift   x * scale[c] + shift[c], c = dim 1
 *   slice x dim= start= end= step= | permute x dims= | reshape x shape= |
 *   expand x shape=
 *   affine_gather a [b ...]        shape= window= flat=lo,hi idx0=... mult=...
 *     the inverted affine write set of a custom kernel (Sec. 3.4: with the
 *     written location fixed, every read index is affine): for every window
 *     point w whose row-major flat index lies in [lo, hi), operand j is read
 *     at index idxj(o, w) with multiplicity mult[j], provided every operand
 *     index of that point is in range (and exactly divisible where written
 *     "(expr)/s"; "(expr)//s" floors).  Expressions are sums of c*o<k>,
 *     c*w<k> and integers.
 * Returns DG_E_PARSE, DG_E_SHAPE, DG_E_UNSUPPORTED_OP or DG_E_OVERFLOW
 * (leaf elements beyond 2^62, or a static path-count bound beyond 2^63) on
 * failure; *out is set only on success and is owned by the caller, who
 * releases it with dg_graph_destroy.
 */
dg_status dg_graph_parse(const char* text, size_t len, dg_graph** out);

/* dg_graph_build: the same graph from descriptors instead of text.
 * tensors[0..nt) are the leaves in declaration order (name, rank, shape);
 * ops[0..nops) are in SSA order; op i writes tensor nt + i, and operand
 * indices refer to that numbering; `attrs` is the text after ';' in the
 * dgir form (may be NULL).  output_tensor indexes the same numbering. */
typedef struct {
  const char* name;
  int32_t rank;
  const int64_t* shape;
} dg_tensor_desc;

typedef struct {
  const char* name;   /* name of the tensor the op writes */
  const char* kind;
  int32_t n_inputs;
  const int32_t* inputs;
  const char* attrs;
} dg_op_desc;

dg_status dg_graph_build(const dg_tensor_desc* tensors, int32_t nt, const dg_op_desc* ops, int32_t nops,
                         int32_t output_tensor, dg_graph** out);

/* Releases a graph and its per-device copies; NULL is ignored.  Must not
 * be called while work using the graph is still queued on a stream. */
void dg_graph_destroy(dg_graph* g);

/* ------------------------------------------------------------------------
 * Introspection (host only; no device work).
 * ------------------------------------------------------------------------ */
typedef struct {
  int32_t n_leaves;
  int32_t output_rank;
  int64_t output_shape[DG_MAX_RANK];
  int64_t output_numel;
  uint64_t leaf_total;        /* total leaf elements (global id space) */
  int64_t max_row_size;       /* static upper bound on one row's entries */
  uint64_t count_bound;       /* static upper bound on one path count
                                 (exact integer arithmetic; below 2^63) */
  int32_t n_instructions;     /* per-location plan length */
  int32_t lds_bytes;          /* local data share one location needs */
  int32_t lds_wide_bytes;     /* the same with 64-bit ids and counts */
  int32_t block_threads;      /* threads working on one location */
  int32_t max_leaf_terms;     /* separable terms of the busiest leaf */
  int32_t n_tensors;          /* leaves and op outputs (dg_graph_tensor) */
  int32_t specialized;        /* kernels specialised for this graph on the
                                 current device: 1 loaded, 0 off or failed
                                 (the precompiled kernels run the plan),
                                 -1 not used on this device yet */
  int32_t dag_specialized;    /* expression-DAG kernels specialised for this
                                 graph on the current device: 1 loaded, 0
                                 failed or off, -1 none yet (every DAG call
                                 so far ran the precompiled kernels).  By
                                 default calls over at least 2^26 edges
                                 (static bound: locations times
                                 dag_edge_bound) take them; the environment
                                 variable DIRIGO_DAG_JIT=1 makes every call
                                 take them, DIRIGO_DAG_JIT=0 none */
  int32_t dag_block_threads;  /* threads working on one location's DAG, and */
  int32_t dag_lds_bytes;      /* the LDS one location's DAG needs (both 0
                                 until the graph's first DAG call compiles
                                 its DAG program) */
  int64_t dag_edge_bound;     /* static bound on one location's DAG edges
                                 (0 until then) */
} dg_graph_info_t;

dg_status dg_graph_info(const dg_graph* g, dg_graph_info_t* out);

typedef struct {
  char name[DG_NAME_LEN];
  int32_t rank;
  int64_t shape[DG_MAX_RANK];
  uint64_t base;   /* global id of the leaf's element 0 */
  int64_t numel;
} dg_leaf_info_t;

/* Leaf i in declaration order, 0 <= i < n_leaves. */
dg_status dg_graph_leaf(const dg_graph* g, int32_t i, dg_leaf_info_t* out);

typedef struct {
  char name[DG_NAME_LEN];
  int32_t rank;
  int64_t shape[DG_MAX_RANK];
  int64_t numel;
  uint64_t gid;       /* element id of element 0 in expression DAGs: a
                         leaf's base, or for an op output the total leaf
                         elements plus the elements of all earlier ops'
                         outputs (SSA order) */
  int32_t leaf;       /* leaf index, or -1 for an op output */
  int32_t producer;   /* index of the op writing it (SSA order), or -1 */
  char kind[32];      /* that op's kind ("" for a leaf) */
} dg_tensor_info_t;

/* Tensor i in declaration order (leaves and op outputs), 0 <= i < n_tensors. */
dg_status dg_graph_tensor(const dg_graph* g, int32_t i, dg_tensor_info_t* out);

/* ------------------------------------------------------------------------
 * Enumeration.
 * ------------------------------------------------------------------------
 * dg_workspace_size: bytes of device workspace that dg_enumerate_sizes,
 * dg_enumerate_fill, dg_compare and the expression-DAG calls need for
 * n_locs locations (the same buffer serves them all; for dg_compare pass
 * the larger of the two graphs' sizes). */
dg_status dg_workspace_size(const dg_graph* g, int64_t n_locs, size_t* bytes);

/* dg_enumerate_sizes: row sizes and CSR offsets.
 *   d_locs[n]        device, int64 flat output locations (any order,
 *                    duplicates allowed: each gets its own row)
 *   d_offsets[n+1]   device, written: d_offsets[0] = 0 and d_offsets[i+1]
 *                    = d_offsets[i] + |row i|
 *   d_ws             device workspace of dg_workspace_size bytes
 *   h_total          host, written: d_offsets[n] (the number of entries)
 * Synchronous: returns after the stream has finished this work.  Returns
 * DG_E_RANGE if a location is outside the output and DG_E_OVERFLOW if a
 * path count does not fit 32 bits; d_offsets is then unspecified.
 * n == 0 writes d_offsets[0] = 0 and *h_total = 0. */
dg_status dg_enumerate_sizes(const dg_graph* g, const int64_t* d_locs, int64_t n, int64_t* d_offsets,
                             void* d_ws, int64_t* h_total, void* stream);

/* dg_enumerate_fill: writes row i to d_ids / d_counts at positions
 * [d_offsets[i], d_offsets[i+1]).  d_offsets must come from
 * dg_enumerate_sizes on the same graph and locations (a caller chunking a
 * large list passes a slice of d_locs and that slice's own offsets, which
 * start at 0).  d_ids and d_counts hold d_offsets[n] entries each.
 * Asynchronous on `stream`. */
dg_status dg_enumerate_fill(const dg_graph* g, const int64_t* d_locs, int64_t n, const int64_t* d_offsets,
                            uint32_t* d_ids, uint32_t* d_counts, void* d_ws, void* stream);

/* dg_enumerate: sizes, offsets and rows in one pass over the locations.
 * Each location's plan runs once; a block finds its row offset by a
 * decoupled look-back over its predecessors' row sizes.
 *   d_locs[n]        device, int64 flat output locations (as above)
 *   d_offsets[n+1]   device, written as by dg_enumerate_sizes
 *   d_ids, d_counts  device, `capacity` uint32 entries each; row i is written
 *                    at [d_offsets[i], d_offsets[i+1]) when that range lies
 *                    below `capacity`
 *   h_total          host, written: d_offsets[n]
 * Synchronous.  Returns DG_E_BUFFER when *h_total > capacity: the offsets
 * and *h_total are then valid, the rows past `capacity` are not written,
 * and the call can be repeated with larger buffers.  DG_E_RANGE and
 * DG_E_OVERFLOW as for dg_enumerate_sizes.  A caller that knows the total
 * (the same graph and locations as an earlier call) needs this one call. */
dg_status dg_enumerate(const dg_graph* g, const int64_t* d_locs, int64_t n, int64_t* d_offsets, uint32_t* d_ids,
                       uint32_t* d_counts, int64_t capacity, void* d_ws, int64_t* h_total, void* stream);

/* dg_enumerate_noalloc: dg_enumerate for callers that cannot allocate
 * device memory (code under HIP graph capture, tight serving loops,
 * harnesses that forbid hipMalloc).  Takes no workspace and allocates and
 * loads nothing: its workspace is a library-owned device array of about
 * 16 MiB, one per GPU the library runs on, held until the process ends.
 *  - n <= DG_NOALLOC_MAX_LOCATIONS, else DG_E_WORKSPACE.
 *  - The graph must already be resident on the current device: its plan
 *    copied there and, with specialisation on, its kernels loaded, which
 *    any earlier enumeration call with the graph on that device does (for
 *    example dg_enumerate with n = 0 or a few locations); else
 *    DG_E_INVALID_ARG.
 *  - Every call on one GPU shares that GPU's array: calls that overlap in
 *    time on one GPU (from several host threads or streams) race and must
 *    not be made.  Each call clears what it needs first, so one call's
 *    leftovers never affect the next.
 * Arguments, results and errors otherwise as dg_enumerate; synchronous. */
#define DG_NOALLOC_MAX_LOCATIONS 2097152
dg_status dg_enumerate_noalloc(const dg_graph* g, const int64_t* d_locs, int64_t n, int64_t* d_offsets,
                               uint32_t* d_ids, uint32_t* d_counts, int64_t capacity, int64_t* h_total,
                               void* stream);

/* dg_enumerate_wide: dg_enumerate with 64-bit ids and path counts, for
 * graphs whose leaves hold 2^32 elements or more (global ids up to 2^62)
 * or whose path counts reach 2^32 (the static bound is below 2^63, so
 * 64-bit counts never overflow).  d_ids and d_counts hold `capacity`
 * uint64 entries each.  The 32-bit calls (dg_enumerate_fill, dg_enumerate,
 * dg_enumerate_range, dg_enumerate_stream) return DG_E_OVERFLOW for a graph
 * whose ids need 64 bits, and for a path count of 2^32 or more.
 * Otherwise as dg_enumerate. */
dg_status dg_enumerate_wide(const dg_graph* g, const int64_t* d_locs, int64_t n, int64_t* d_offsets,
                            uint64_t* d_ids, uint64_t* d_counts, int64_t capacity, void* d_ws, int64_t* h_total,
                            void* stream);

/* ------------------------------------------------------------------------
 * Expression DAGs of res(y[l]) (Sec. 3.4, "Back-projection": substituting
 * the per-element equations backwards from y[l]).  Every element of the
 * cone of y[l] is one node, shared wherever it occurs.  A leaf element is a
 * variable; every other node is its op (dg_tensor_info_t.kind) applied to
 * the element references of its per-element equation, in the equation's
 * order: read groups in order, window points in row-major order, a group's
 * operands in order at each point (a point with any operand index outside
 * its tensor, or not exactly divisible, reads nothing).  So a conv node's
 * references are x, W pairs over (input channel, taps...) followed by its
 * bias; a matmul node's are A, B pairs over k; a norm node's are its
 * statistics set (multiplicity |S| + 2 each), its own element, then gamma
 * and beta.  Elements are named by global ids (dg_tensor_info_t.gid plus
 * the row-major flat index), which must fit 32 bits (DG_E_OVERFLOW).
 *
 * Per location i, CSR over CSR:
 *   nodes      [d_node_offsets[i], d_node_offsets[i+1]): the non-leaf cone
 *              elements, ops in reverse SSA order (y[l] first), elements
 *              ascending within an op;
 *   node_edge  per node, its first edge relative to d_edge_offsets[i]; its
 *              edges end where the next node's begin (the last node's at
 *              d_edge_offsets[i+1]);
 *   edges, mults [d_edge_offsets[i], d_edge_offsets[i+1]): child id and
 *              multiplicity of each reference.
 * Leaf elements appear only as children (ids below leaf_total).  The
 * per-location frontiers live in LDS; a graph whose static frontier bound
 * does not fit returns DG_E_CAPACITY.
 * ------------------------------------------------------------------------ */

/* dg_dag_sizes: node and edge counts of every location as running totals
 * (d_node_offsets[n+1], d_edge_offsets[n+1], device int64, written; [0] = 0)
 * and the totals on the host.  Synchronous.  DG_E_RANGE for a location
 * outside the output; the workspace is dg_workspace_size(g, n). */
dg_status dg_dag_sizes(const dg_graph* g, const int64_t* d_locs, int64_t n, int64_t* d_node_offsets,
                       int64_t* d_edge_offsets, void* d_ws, int64_t* h_nodes, int64_t* h_edges, void* stream);

/* dg_dag_fill: writes the DAGs with offsets from dg_dag_sizes on the same
 * graph and locations: d_nodes and d_node_edge hold d_node_offsets[n]
 * uint32 entries, d_edges and d_mults d_edge_offsets[n].  Synchronous;
 * DG_E_INVALID_ARG if the offsets do not match. */
dg_status dg_dag_fill(const dg_graph* g, const int64_t* d_locs, int64_t n, const int64_t* d_node_offsets,
                      const int64_t* d_edge_offsets, uint32_t* d_nodes, uint32_t* d_node_edge, uint32_t* d_edges,
                      uint32_t* d_mults, void* d_ws, void* stream);

/* dg_dag: dg_dag_sizes and dg_dag_fill in one call, with output buffers
 * sized beforehand (Sec. 3.4, "Back-projection", as above).  A call of at
 * most 2,048 locations whose DAG, at the program's static node and edge
 * bounds, fits in LDS beside the walk's frontiers (64 KiB at most) walks
 * each location once: its DAG is staged in LDS, its node and edge offsets
 * come from decoupled look-backs over its predecessors' counts, and the
 * stage is copied out, with no host round trip between passes.  Larger
 * calls, where that costs more per location than the two passes, make the
 * two passes (DIRIGO_DAG_ONEPASS=1 takes the one pass whenever the stage
 * fits, DIRIGO_DAG_ONEPASS=0 never).
 *   d_locs[n]            device, int64 flat output locations
 *   d_node_offsets[n+1]  device, written as by dg_dag_sizes
 *   d_edge_offsets[n+1]  device, written as by dg_dag_sizes
 *   d_nodes, d_node_edge device, node_capacity uint32 entries each
 *   d_edges, d_mults     device, edge_capacity uint32 entries each
 *   h_nodes, h_edges     host, written: the totals
 * Location i's DAG is written where its nodes and edges fit the capacities.
 * Synchronous.  Returns DG_E_BUFFER when a total exceeds its capacity: the
 * offsets and totals are then valid, the DAGs past a capacity are not
 * written, and the call can be repeated with larger buffers.  DG_E_RANGE,
 * DG_E_CAPACITY and DG_E_OVERFLOW as for dg_dag_sizes; the workspace is
 * dg_workspace_size(g, n). */
dg_status dg_dag(const dg_graph* g, const int64_t* d_locs, int64_t n, int64_t* d_node_offsets, int64_t* d_edge_offsets,
                 uint32_t* d_nodes, uint32_t* d_node_edge, uint32_t* d_edges, uint32_t* d_mults, int64_t node_capacity,
                 int64_t edge_capacity, void* d_ws, int64_t* h_nodes, int64_t* h_edges, void* stream);

/* dg_enumerate_range: dg_enumerate over the contiguous flat locations
 * first, first + 1, ..., first + n - 1 (row i belongs to location
 * first + i), with no location list: a whole output, or a chunk of it, is
 * enumerated by walking [0, numel) in ranges.  DG_E_RANGE if the range
 * leaves the output (checked before any work).  Otherwise as dg_enumerate;
 * the workspace is dg_workspace_size(g, n). */
dg_status dg_enumerate_range(const dg_graph* g, int64_t first, int64_t n, int64_t* d_offsets, uint32_t* d_ids,
                             uint32_t* d_counts, int64_t capacity, void* d_ws, int64_t* h_total, void* stream);

/* dg_enumerate_stream: the rows of the flat locations [first, first + n)
 * streamed in chunks through two halves of one caller-owned device buffer,
 * so that a whole output whose CSR does not fit in memory (the full
 * verification of Sec. 5, RQ4) is produced with bounded memory.  A first
 * pass computes the row sizes and offsets of the whole range (kept at the
 * start of the buffer); chunks are then cut exactly where the rows stop
 * fitting a half, and filled alternately into the two halves on stream_a
 * and stream_b without waiting for each other: while the consumer's work
 * on one chunk runs on its stream, the next chunk is written on the other.
 *   d_buf, buf_bytes  device buffer: the range's offsets (8 * (n + 1) bytes)
 *                     and the workspace of n locations, then two halves,
 *                     each with the offsets and workspace of max_chunk
 *                     locations and as many (id, count) entries as the rest
 *                     of the half allows
 *   max_chunk         most locations per chunk (> 0)
 *   fn(user, first, n, d_offsets, d_ids, d_counts, total, stream)
 *                     called on the calling thread once per chunk, in
 *                     location order, right after the chunk's work has been
 *                     enqueued on `stream`: rows of locations first ..
 *                     first + n - 1 in CSR form (device pointers into the
 *                     buffer, offsets start at 0, `total` entries).  Work
 *                     the consumer enqueues on `stream` sees the finished
 *                     chunk; the half is not reused until that stream has
 *                     finished.  A nonzero return stops the stream
 *                     (DG_E_STOPPED).
 * Returns after all chunk and consumer work has finished.  DG_E_RANGE if
 * the range leaves the output; DG_E_BUFFER if the buffer cannot hold the
 * offsets and two chunks, or one location's row alone does not fit a half;
 * DG_E_OVERFLOW as for dg_enumerate_sizes. */
typedef int32_t (*dg_chunk_fn)(void* user, int64_t first, int64_t n, const int64_t* d_offsets, const uint32_t* d_ids,
                               const uint32_t* d_counts, int64_t total, void* stream);
dg_status dg_enumerate_stream(const dg_graph* g, int64_t first, int64_t n, void* d_buf, size_t buf_bytes,
                              int64_t max_chunk, dg_chunk_fn fn, void* user, void* stream_a, void* stream_b);

/* dg_compare: footprints of two graphs, location by location (Sec. 3.4:
 * e_A and e_B at the same l; the two programs read the same leaves and
 * write outputs of the same shape, as MERGE's input/output matching of
 * Sec. 3.2 requires, else DG_E_SIGNATURE).
 *   d_status[n]      device, written: 0 rows equal, 1 the id sets differ,
 *                    2 same ids but some count differs
 *   d_mismatch[n]    device, written: the positions i (into d_locs) with
 *                    d_status[i] != 0, ascending
 *   h_n_mismatch     host, written: how many positions were written
 * Synchronous.  DG_E_RANGE / DG_E_OVERFLOW as for dg_enumerate_sizes.
 * The two graphs may have at most 16 leaves (DG_E_UNSUPPORTED_OP beyond:
 * the comparison keeps one emission shape per leaf in a fixed table), and
 * both plans plus the comparison's tables must fit the device's LDS
 * (DG_E_CAPACITY). */
dg_status dg_compare(const dg_graph* a, const dg_graph* b, const int64_t* d_locs, int64_t n, uint8_t* d_status,
                     int64_t* d_mismatch, int64_t* h_n_mismatch, void* d_ws, void* stream);

/* dg_compare_range: dg_compare over the contiguous flat locations first,
 * ..., first + n - 1 (the full-output verification of Sec. 5, RQ4, is
 * first = 0, n = numel), with a budget (Sec. 3.4, "Enumeration and
 * budgets": stop once a bug is found).
 *   max_mismatch     0: compare every location.  k > 0: once k mismatching
 *                    locations have been found, locations whose comparison
 *                    has not started yet are skipped and get status 3; at
 *                    least min(k, number of mismatching locations) are
 *                    reported, which ones depends on scheduling
 *   d_status[n]      device, written: 0, 1, 2 as for dg_compare, 3 skipped
 *   d_mismatch[n]    device, written: positions i (location first + i) with
 *                    status 1 or 2, ascending
 *   h_n_mismatch     host, written: how many positions were written
 * DG_E_RANGE if the range leaves the output (checked before any work).
 * Synchronous.  The workspace is dg_workspace_size(a, n). */
dg_status dg_compare_range(const dg_graph* a, const dg_graph* b, int64_t first, int64_t n, int64_t max_mismatch,
                           uint8_t* d_status, int64_t* d_mismatch, int64_t* h_n_mismatch, void* d_ws,
                           void* stream);

/* dg_graph_text: the graph as dgir v1 text (leaves, ops in SSA order,
 * output); writes at most cap - 1 characters and a terminating NUL to buf
 * (host; may be NULL when cap is 0) and the full length to *len. */
dg_status dg_graph_text(const dg_graph* g, char* buf, size_t cap, size_t* len);

/* dg_graph_merge: MERGE of two programs (Sec. 3.2) into one obligation.
 *  - Inputs are matched: a leaf of b pairs with the leaf of a of the same
 *    name and shape, the rest pair in declaration order among leaves of the
 *    same shape; an input without a partner, or different output shapes,
 *    give DG_E_SIGNATURE.
 *  - With trim_prefix nonzero, the longest common prefix of ops is
 *    trimmed: op i of a and op i of b
 *    match when kind, attributes and (matched) operands agree.  The prefix
 *    results that later ops of either graph read, or that are an output,
 *    become leaves, appended after a's leaves in prefix order.  A common
 *    suffix is never trimmed.
 * *a_out and *b_out receive two new graphs (owned by the caller, free with
 * dg_graph_destroy) over the same leaves in the same order under a's names,
 * ready for dg_compare; *n_trimmed (may be NULL) the number of prefix ops.
 * The trimming keeps equivalence when the prefix is surjective; in any case
 * a location that compares equal after trimming compares equal before
 * (rows compose through the shared prefix). */
dg_status dg_graph_merge(const dg_graph* a, const dg_graph* b, int32_t trim_prefix, dg_graph** a_out,
                         dg_graph** b_out, int32_t* n_trimmed);

/*
 * Location order (Sec. 4, "Search Heuristic": candidate locations ranked in
 * tiers, then a random permutation of the unchecked ones).  The tier that
 * needs an SMT solver (path-condition coverage) is not part of this path;
 * the other two are:
 *
 *   corners -- every op is taken as one kernel launch writing its output in
 *     row-major order, one element per thread, block_threads threads per
 *     block.  Its corner threads are the first and last thread of the first
 *     and last block and lanes warp-1 and warp of block 0.  A corner
 *     thread's element is mapped to an output location through reads that
 *     only permute dims (each consumer element reads exactly that element
 *     and every other operand of the read is in range everywhere); the
 *     smallest location over such paths is taken, and corners with no such
 *     path give none.  Ops rank in reverse SSA order (later launches
 *     first); per op: (thread 0, block 0), (last thread, block 0),
 *     (thread 0, last block), (last thread, last block), lane warp-1,
 *     lane warp.
 *   boundaries -- the first and the last output location.
 *
 * Each location appears once, at its first rank.  The rest of [0, numel)
 * follows in the order of a keyed permutation pi of [0, numel): a balanced
 * four-round Feistel network on 2h bits, h the smallest with 4^h >= numel,
 * round keys the first four outputs of SplitMix64 (Steele, Lea and Flood,
 * 2014) seeded with `seed`, round function the SplitMix64 output mix of
 * (right half XOR key) masked to h bits, new halves (R, L XOR F(R)); values
 * at or past numel are encrypted again until below numel (cycle walking,
 * Black and Rogaway, 2002).  The full order is the prefix followed by
 * pi(0), pi(1), ... with the prefix's locations left out.
 */

/* dg_order_prefix: the ranked prefix (corners, then boundaries) of g's
 * output for the given launch shape (block_threads >= 1, warp >= 1).  Host
 * only, no device work.  Writes min(count, cap) locations to h_prefix
 * (host memory; may be NULL when cap is 0) and the full count to
 * *h_count. */
dg_status dg_order_prefix(const dg_graph* g, int32_t block_threads, int32_t warp, int64_t* h_prefix, int64_t cap,
                          int64_t* h_count);

/* dg_order_workspace_size: bytes of device workspace dg_order_permute needs
 * for up to n_exclude excluded values. */
dg_status dg_order_workspace_size(int64_t n_exclude, size_t* bytes);

/* dg_order_permute: pi(first), ..., pi(first + count - 1) of the keyed
 * permutation of [0, n_out) (n_out <= 2^62), leaving out the values listed
 * in h_exclude, written in position order to d_out (device; room for count
 * values less those excluded values whose positions fall in the range, at
 * most count).  h_exclude: n_exclude host int64 values in [0, n_out) (any order,
 * repeats allowed; a value outside gives DG_E_INVALID_ARG).  The library
 * finds each excluded value's position by the inverse permutation, so the
 * device pass computes pi once per position.  Synchronous: *h_written
 * receives the number of values written.  Concatenating the calls over
 * consecutive position ranges gives the permutation part of the order; with
 * h_exclude = the prefix it completes the order. */
dg_status dg_order_permute(int64_t n_out, uint64_t seed, const int64_t* h_exclude, int64_t n_exclude, int64_t first,
                           int64_t count, int64_t* d_out, int64_t* h_written, void* d_ws, size_t ws_bytes,
                           void* stream);

/* Message of the calling thread's last failed call ("" if none). */
const char* dg_last_error(void);

#ifdef __cplusplus
}
#endif

#endif /* DIRIGO_ROCM_H */
