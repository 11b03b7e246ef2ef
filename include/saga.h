/*
 * saga.h -- SAGA-NN message-passing layer for AMD Instinct MI355X (gfx950).
 *
 * A GNN layer takes the graph (an adjacency matrix), the vertex embedding
 * matrix and optionally an edge embedding matrix, and produces the next
 * layer's embeddings (Zhang et al., "Architectural Implications of Graph
 * Neural Networks", IEEE CAL 2020, Sec. 2 "Model Survey").  It is
 * decomposed into four stages -- Scatter, ApplyEdge, Gather, ApplyVertex
 * (Sec. 2 "Model Decomposition"; the GGNN walk-through of Fig. 2).  This
 * library runs that layer on one GPU:
 *
 *   saga_plan_build                 graph layout: degrees, degree-sorted row
 *                                   order, row segments and row blocks
 *                                   (saga_plan_build_split: the out-degree
 *                                   and row-order branches on two streams)
 *   saga_scatter_apply_edge_gather  fused Scatter + ApplyEdge + Gather: a
 *                                   per-destination segment reduction over
 *                                   the in-CSR (the fused Gather is the
 *                                   sparse adjacency x embedding product,
 *                                   Sec. 3.2 "Gather", Fig. 7b)
 *   saga_scatter_gather_unfused     the same, unfused: materialised edge
 *                                   tensor, then a segment reduction (the
 *                                   baseline of Fig. 7a)
 *   saga_lstm_gather                GraphSAGE's LSTM Gather: a recurrence
 *                                   along each row's in-edges
 *   saga_rel_plan_build             typed-edge layout of R-GCN: the distinct
 *                                   (relation, source) pairs, grouped by
 *                                   relation, and per-edge pair rows / norms
 *   saga_rel_transform              R-GCN ApplyEdge on the matrix cores: one
 *                                   grouped GEMM, every pair's source row
 *                                   times its relation's weight
 *   saga_apply_vertex               dense per-vertex transform on the matrix
 *                                   cores, with fused epilogues (Sec. 3.2
 *                                   "ApplyVertex", Table III)
 *   saga_layer                      one whole layer of a Table I model
 *
 * Conventions (all entry points):
 *   - Every pointer argument except the host-side structs (saga_plan_opts,
 *     saga_plan, saga_rel_plan, saga_edge_op, saga_edge_inputs, saga_gemm_op,
 *     saga_layer_desc) is a DEVICE pointer.  The caller allocates, owns and
 *     frees all device memory; the library allocates nothing, ever.  Scratch
 *     space comes from a caller-provided workspace whose size the matching
 *     *_workspace_size call reports.
 *   - Matrices are row-major.  `ld` is the leading dimension in ELEMENTS.
 *     Feature matrices must have a 16-byte-aligned base and ld*elem_size a
 *     multiple of 16 bytes; columns [cols, ld) are never read as data and
 *     never written.
 *   - float32 ("f32") or bfloat16 ("bf16") storage; accumulation is always
 *     float32.  Biases, attention vectors, gate weights and degree scalings
 *     are float32.
 *   - All work is enqueued on `stream` (a hipStream_t; NULL = the null
 *     stream) and is asynchronous.  The returned status covers argument
 *     validation and kernel launch only; no call blocks except
 *     saga_plan_check.
 *   - Outputs must not overlap any input (checked on address ranges;
 *     SAGA_EINVAL).  Every output row is written, including rows with no
 *     in-edges.
 *   - Results are deterministic: the same inputs give byte-identical outputs
 *     from run to run (no floating-point atomics).
 *   - Functions never throw, abort or print.  On error they return a status
 *     and saga_last_error() gives a detail string (thread-local).
 */
#ifndef SAGA_H
#define SAGA_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum saga_status {
  SAGA_OK = 0,
  SAGA_EINVAL = 1,        /* bad argument: null, size, alignment, ld, overlap */
  SAGA_EGRAPH = 2,        /* CSR arrays violate the CSR rules */
  SAGA_EUNSUPPORTED = 3,  /* valid but not supported combination */
  SAGA_EDEVICE = 4,       /* HIP runtime error */
  SAGA_EWORKSPACE = 5,    /* workspace missing or too small */
  SAGA_EINTERNAL = 6
} saga_status;

typedef enum saga_dtype { SAGA_F32 = 0, SAGA_BF16 = 1 } saga_dtype;

/* Gather reductions (Table I "Gather" column; the simple sum/mean/max
 * reductions and the attention reduction of Sec. 2 "Survey Result"). */
typedef enum saga_reduce {
  SAGA_RED_SUM = 0,
  SAGA_RED_MEAN = 1,     /* sum / d_in(v) */
  SAGA_RED_MAX = 2,      /* elementwise maximum */
  SAGA_RED_SOFTMAX = 3   /* attention: per-destination softmax-weighted sum */
} saga_reduce;

/* Scatter + ApplyEdge message kinds (Table I "Scatter"/"ApplyEdge"). */
typedef enum saga_msg {
  SAGA_MSG_COPY = 0,      /* message of edge u->v = src row u              */
  SAGA_MSG_SRC_NORM = 1,  /* src row u * d_out(u)^-1/2  (GCN normalisation) */
  SAGA_MSG_GAT = 2,       /* score LeakyReLU(el[u,k] + er[v,k]); SOFTMAX only */
  SAGA_MSG_GATED = 3,     /* sigmoid(gs[u] + gd[v] + b_e + e_uv W_ee) * src[u] */
  SAGA_MSG_TYPED = 4      /* R-GCN: edge_norm[e] * src[edge_pair[e]] (rel plan) */
} saga_msg;

typedef enum saga_act {
  SAGA_ACT_NONE = 0,
  SAGA_ACT_RELU = 1,     /* x > 0 ? x : +0 */
  SAGA_ACT_ELU = 2,      /* x > 0 ? x : exp(x) - 1 */
  SAGA_ACT_SIGMOID = 3,
  SAGA_ACT_TANH = 4
} saga_act;

/* A device matrix view.  ptr == NULL means "absent" where an input is
 * optional. */
typedef struct saga_cmat { const void* ptr; int64_t rows, cols, ld; } saga_cmat;
typedef struct saga_mat { void* ptr; int64_t rows, cols, ld; } saga_mat;

/* ======================================================================
 * Graph layout (plan)
 * ======================================================================
 *
 * The graph is a destination-major CSR ("in-CSR"): row v of the adjacency
 * lists the sources of v's in-edges (the edge-to-vertex adjacency of
 * Sec. 3.2 "Gather", where a nonzero is an in-edge of the row's vertex).
 * row_ptr is int32[num_dst + 1], col_idx is int32[num_edges]; multi-edges
 * and self-loops are allowed and count once per copy.
 *
 * The plan holds, on the device:
 *   d_in[v]  = row_ptr[v+1] - row_ptr[v]                    (int32[num_dst])
 *   d_out[u] = number of entries of col_idx equal to u      (int32[num_src])
 *   perm     = rows sorted by d_in descending, then id ascending (power-law
 *              degree skew, Sec. 3.2 / Fig. 8a)              (int32[num_dst])
 *   segments: each row, taken in perm order, is cut into pieces of at most
 *              seg_len edges (a row with d_in <= seg_len, or an empty row,
 *              is one piece).  Segment s covers CSR entries
 *              [seg_beg[s], seg_end[s]) of row seg_row[s]; the segments of
 *              perm position i are row_seg_first[i] .. row_seg_first[i+1]-1.
 *              Rows with d_in > seg_len ("split rows") are perm positions
 *              0 .. n_split-1 and own segments 0 .. s_split-1.
 *   blocks:   segment s costs (seg_end - seg_beg) + row_cost; with P(s) the
 *              total cost of the segments before s, block b holds the
 *              segments with floor(P(s) / block_cost) == b;
 *              block_ptr[b] = its first segment, block_ptr[num_blocks] = S.
 * All of it is integer and reproducible bit for bit.
 */
typedef struct saga_plan_opts {
  int32_t seg_len;     /* > 0; default (0): min(512, block_cost / 2) */
  int32_t block_cost;  /* >= seg_len + row_cost; default (0): the power of two at
                          or below (num_edges + row_cost * num_dst) / 2048, clamped
                          to [256, 4096] (about 2048 row blocks on small graphs;
                          4096 and seg_len 512 on large ones) */
  int32_t row_cost;    /* >= 1; default 4 */
} saga_plan_opts;

/* Filled by saga_plan_build.  Plain data: copy it freely; it stays valid as
 * long as the workspace and the caller's CSR arrays live. */
typedef struct saga_plan {
  int32_t num_dst, num_src;
  int64_t num_edges;
  const int32_t* row_ptr;   /* the caller's arrays, referenced not copied */
  const int32_t* col_idx;
  int32_t seg_len, block_cost, row_cost;
  int64_t max_segments;     /* capacity of the segment arrays */
  int64_t max_blocks;       /* capacity of block_ptr (minus one) */
  int64_t max_split;        /* upper bound on split rows */
  int64_t max_split_segments;
  /* device arrays inside the workspace */
  int32_t* d_in;
  int32_t* d_out;
  int32_t* perm;
  int32_t* row_seg_first;   /* [num_dst + 1] */
  int32_t* seg_row;         /* [max_segments] */
  int32_t* seg_beg;
  int32_t* seg_end;
  int32_t* block_ptr;       /* [max_blocks + 1] */
  int32_t* counts;          /* [8]: see saga_plan_counts */
  void* scratch;            /* sort / scan temporaries */
  size_t scratch_bytes;
} saga_plan;

typedef struct saga_plan_counts {
  int64_t num_segments;
  int64_t num_blocks;
  int64_t n_split;          /* rows with d_in > seg_len */
  int64_t s_split;          /* segments owned by split rows */
  int32_t error_flags;      /* bit 0: row_ptr[0] != 0, bit 1: row_ptr not
                               non-decreasing, bit 2: row_ptr[num_dst] !=
                               num_edges, bit 3: col_idx out of range */
  int32_t max_in_degree;
} saga_plan_counts;

/* Bytes of workspace saga_plan_build needs for this graph size.
 * Errors: SAGA_EINVAL on null `bytes`, negative sizes, num_edges >= 2^31,
 * a total segment cost num_edges + row_cost * (num_dst + ceil(num_edges /
 * seg_len)) of 2^31 - 1 or more (with the options in effect: every edge
 * offset and cost prefix is an int32), or invalid options (opts may be NULL
 * for the defaults). */
saga_status saga_plan_workspace_size(int32_t num_dst, int32_t num_src, int64_t num_edges,
                                     const saga_plan_opts* opts, size_t* bytes);

/* Build the plan of a device-resident in-CSR on `stream`.  The CSR arrays
 * are read, validated on the device and referenced by the plan (they must
 * stay alive and unchanged while the plan is used).  `workspace` (device,
 * 256-byte aligned, caller-owned) receives every plan array.  Returns after
 * enqueuing; an invalid CSR is reported by saga_plan_check, and every later
 * kernel that uses a plan whose validation failed leaves its outputs
 * unwritten instead of reading out of bounds.
 * Errors: SAGA_EINVAL (null pointers, sizes, options, alignment),
 * SAGA_EWORKSPACE (too small), SAGA_EDEVICE (launch failure). */
saga_status saga_plan_build(int32_t num_dst, int32_t num_src, int64_t num_edges,
                            const int32_t* row_ptr, const int32_t* col_idx,
                            const saga_plan_opts* opts, void* workspace,
                            size_t workspace_bytes, void* stream, saga_plan* plan);

/* The same plan built as two concurrent branches, so that the stage that
 * follows the out-degrees can overlap the row order (the paper's outlook of
 * pipelining stages instead of running them one after another, Sec. 3
 * "Forward Looking"):
 *   - on `stream`: the counters are cleared, then the out-degree count
 *     (d_out); a d_out-scaled transform enqueued on `stream` after this call
 *     waits for d_out only;
 *   - on `order_stream` (made to wait for the cleared counters through
 *     fork_event): in-degrees, CSR validation, the degree order, segments and
 *     row blocks; join_event is recorded on order_stream when they are done.
 * Before anything that uses perm, segments or blocks (every Gather) runs on
 * `stream`, the caller makes `stream` wait for join_event
 * (hipStreamWaitEvent).  fork_event and join_event are caller-created
 * hipEvent_t; order_stream must differ from `stream`; keep both streams at
 * the same priority.  Graphs whose out-degrees the degree kernel counts
 * with atomics in the same pass (no edges, or more than 2^23 source
 * vertices) run entirely on `stream` (join_event is then recorded there).
 * The arrays are the same, bit for bit, as saga_plan_build's.  Errors as
 * saga_plan_build, and SAGA_EINVAL if a stream or event is missing. */
saga_status saga_plan_build_split(int32_t num_dst, int32_t num_src, int64_t num_edges,
                                  const int32_t* row_ptr, const int32_t* col_idx,
                                  const saga_plan_opts* opts, void* workspace,
                                  size_t workspace_bytes, void* stream, void* order_stream,
                                  void* fork_event, void* join_event, saga_plan* plan);

/* Synchronise `stream` and read the plan's counters.  Returns SAGA_EGRAPH
 * if the device validation found a CSR error (details in counts->error_flags
 * and saga_last_error), SAGA_EDEVICE if the stream reported a fault. */
saga_status saga_plan_check(const saga_plan* plan, void* stream, saga_plan_counts* counts);

/* ======================================================================
 * Typed edges (R-GCN)
 * ======================================================================
 * Table I, R-GCN row: Scatter takes the edge and its source, ApplyEdge is an
 * MLP picked by the edge's type, Gather sums the in-edges and adds the
 * vertex itself.  Sec. 3.2 "ApplyEdge": every edge carries a type attribute,
 * and the edges of one type are selected and batched into one GEMM.
 *
 * etype is int32[num_edges], aligned with the CSR entries, values in
 * [0, num_rel).  The message of CSR entry e = u -> v of type r is
 * x_u W_r / c(v, r), where c(v, r) counts the in-edges of v of type r.
 * x_u W_r depends only on the pair (r, u), so it is computed once per
 * distinct pair.  The rel plan holds, on the device:
 *   rel_count[r]  number of distinct sources of relation r
 *   rel_ptr[r]    first pair row of relation r: rel_ptr[0] = 0,
 *                 rel_ptr[r+1] = rel_ptr[r] + rel_count[r] rounded up to a
 *                 multiple of SAGA_REL_TILE (int32[num_rel + 1])
 *   pair_src[q]   source vertex of pair row q: the sources of relation r in
 *                 ascending order at rows rel_ptr[r] .. rel_ptr[r] +
 *                 rel_count[r] - 1, then -1 up to rel_ptr[r+1]
 *                 (int32[max_pairs]; rows from rel_ptr[num_rel] on unused)
 *   edge_pair[e]  pair row of (etype[e], col_idx[e])      (int32[num_edges])
 *   edge_norm[e]  1 / c(v, etype[e]) in float32, correctly rounded
 *                                                        (float[num_edges])
 * All integers are reproducible bit for bit.
 */
#define SAGA_REL_TILE 128
#define SAGA_REL_MAX_RELATIONS 2048

typedef struct saga_rel_plan {
  int32_t num_rel;
  int32_t num_src;
  int64_t num_edges;
  int64_t max_pairs;          /* rows of pair_src and of a transform output */
  const int32_t* etype;       /* the caller's array, referenced not copied */
  const int32_t* plan_counts; /* counters of the plan it was built on */
  /* device arrays inside the workspace */
  int32_t* rel_ptr;
  int32_t* rel_count;
  int32_t* pair_src;
  int32_t* edge_pair;
  float* edge_norm;
  int32_t* counts;            /* [4]: see saga_rel_counts */
  void* scratch;
  size_t scratch_bytes;
} saga_rel_plan;

typedef struct saga_rel_counts {
  int64_t pair_rows;          /* rel_ptr[num_rel]: pair rows incl. padding */
  int64_t pairs;              /* distinct (relation, source) pairs */
  int32_t error_flags;        /* bit 0: an etype value outside [0, num_rel) */
} saga_rel_counts;

/* Workspace bytes of saga_rel_plan_build for this plan and relation count.
 * Errors: SAGA_EINVAL (null, num_rel outside [1, SAGA_REL_MAX_RELATIONS],
 * more than 2^31 pair rows). */
saga_status saga_rel_plan_workspace_size(const saga_plan* plan, int32_t num_rel, size_t* bytes);

/* Build the typed layout of a built plan's graph on `stream`.  etype is
 * referenced (it must stay alive and unchanged while the rel plan is used);
 * workspace (device, 256-byte aligned, caller-owned) receives every array.
 * If the plan's CSR was invalid, nothing is computed; an out-of-range etype
 * is reported by saga_rel_plan_check as SAGA_EGRAPH, and every later call on
 * this rel plan then leaves its outputs unwritten.  Errors: SAGA_EINVAL,
 * SAGA_EWORKSPACE, SAGA_EDEVICE. */
saga_status saga_rel_plan_build(const saga_plan* plan, const int32_t* etype, int32_t num_rel,
                                void* workspace, size_t workspace_bytes, void* stream,
                                saga_rel_plan* rel);

/* Synchronise `stream` and read the rel plan's counters; SAGA_EGRAPH if the
 * plan's CSR or an edge type was invalid. */
saga_status saga_rel_plan_check(const saga_rel_plan* rel, void* stream, saga_rel_counts* counts);

/* R-GCN ApplyEdge hoisted to the distinct pairs, on the matrix cores:
 *     out[q] = x[pair_src[q]] w_{r(q)}     for pair rows q < rel_ptr[num_rel]
 * where r(q) is the relation whose range holds q; padding rows are written
 * as 0; rows from rel_ptr[num_rel] on are not written.  One grouped GEMM:
 * each tile of SAGA_REL_TILE rows lies in one relation and uses its weight.
 * x: num_src x K (dtype, 16-byte rows); w: the num_rel weights stacked,
 * (num_rel * K) x N (rows r*K .. r*K+K-1 are W_r; dtype); out: max_pairs x
 * N (dtype).  N <= 4096.  Workspace: saga_rel_transform_workspace_size()
 * bytes, 256-byte aligned (the packed, transposed weights). */
saga_status saga_rel_transform_workspace_size(const saga_rel_plan* rel, int32_t dtype,
                                              int64_t k, int64_t n, size_t* bytes);

saga_status saga_rel_transform(const saga_rel_plan* rel, int32_t dtype, saga_cmat x,
                               saga_cmat w, saga_mat out, void* workspace,
                               size_t workspace_bytes, void* stream);

/* ======================================================================
 * Scatter + ApplyEdge + Gather (fused)
 * ======================================================================
 * For every destination v, reduce the messages of its in-edges (Sec. 3.2
 * "Scatter", "ApplyEdge", "Gather"; Table I), then apply the epilogue
 *     out[v] = act(post(agg_v) + bias)
 * where post() is:  SUM/MAX: agg (times d_in(v)^-1/2 if dst_norm);
 * MEAN: agg / d_in(v); SOFTMAX: the per-head weighted sum, heads
 * concatenated (head_mean = 0) or averaged (head_mean = 1).  A row with no
 * in-edges has agg = 0.  No E x F edge tensor is ever materialised.
 *
 * Inputs by message kind (feature width F = src.cols):
 *   COPY, SRC_NORM: src  (num_src x F, f32 or bf16)
 *   GAT:   src = z (num_src x F, f32), el (num_src x heads), er (num_dst x
 *          heads), F % heads == 0, F/heads a multiple of 4; score of edge
 *          u->v for head k is LeakyReLU(el[u,k] + er[v,k], neg_slope).
 *   GATED: src = h (num_src x F, f32), gate_src (num_src x F), gate_dst
 *          (num_dst x F), edge_feat (num_edges x Fe, row e = CSR entry e),
 *          w_edge (Fe x F, dense), gate_bias (F); message of edge e = u->v
 *          is sigmoid(gate_src[u] + gate_dst[v] + gate_bias +
 *          edge_feat[e] w_edge) * h[u] elementwise.  F == 64, Fe <= 16.
 *   TYPED: rel (a rel plan built on this plan), src = the pair rows of
 *          saga_rel_transform (rel->max_pairs x F); message of CSR entry e
 *          is rel->edge_norm[e] * src[rel->edge_pair[e]].
 * self (optional; COPY, SRC_NORM and TYPED): num_dst x out cols, same dtype,
 * added before the bias: out[v] = act(post(agg_v) + self[v] + bias).
 * Output: num_dst x F (x F/heads if head_mean), same dtype as src.
 * Supported: COPY/SRC_NORM with SUM/MEAN/MAX in f32 and bf16, GAT with
 * SOFTMAX in f32, GATED with SUM in f32, TYPED with SUM in f32 and bf16,
 * F <= 1024 (GAT: F <= 256, GATED: F == 64); others give
 * SAGA_EUNSUPPORTED.
 */
typedef struct saga_edge_op {
  /* enumerated fields are plain int32_t (the enum named in the comment), so
     that the library can range-check whatever value a caller stores */
  int32_t msg;         /* saga_msg */
  int32_t reduce;      /* saga_reduce */
  int32_t dtype;       /* saga_dtype */
  int32_t heads;       /* GAT: number of heads; else ignored */
  int32_t head_mean;   /* GAT: 1 = average over heads */
  int32_t dst_norm;    /* 1 = multiply SUM/MAX aggregate by d_in(v)^-1/2 */
  float neg_slope;     /* GAT LeakyReLU slope (0.2 in GAT) */
  int32_t act;         /* saga_act */
} saga_edge_op;

typedef struct saga_edge_inputs {
  saga_cmat src;
  saga_cmat el, er;                /* GAT (4-byte aligned) */
  saga_cmat gate_src, gate_dst;    /* GATED */
  saga_cmat edge_feat;             /* GATED */
  const float* w_edge;             /* GATED */
  const float* gate_bias;          /* GATED, nullable */
  const float* bias;               /* nullable, length = output cols */
  const saga_rel_plan* rel;        /* TYPED */
  saga_cmat self;                  /* nullable: added to each output row */
} saga_edge_inputs;

saga_status saga_gather_workspace_size(const saga_plan* plan, const saga_edge_op* op,
                                       int64_t feat, size_t* bytes);

saga_status saga_scatter_apply_edge_gather(const saga_plan* plan, const saga_edge_op* op,
                                           const saga_edge_inputs* in, saga_mat out,
                                           void* workspace, size_t workspace_bytes,
                                           void* stream);

/* ----------------------------------------------------------------------
 * Gather with the next layer's transform fused in (the paper's outlook of
 * pipelining stages finely instead of running them one after another,
 * Sec. 4 "Forward Looking"; here the next layer's ApplyVertex transform
 * starts on a row block as soon as the Gather has finished it): with h_v
 * the row that saga_scatter_apply_edge_gather would write for v,
 *     out[v] = rs(v) * (h_v next->w)      rs(v) = next->row_scale_deg ?
 *                                          deg[v]^-1/2 (0 for deg 0) : 1
 * h lives in the workspace only: the Gather runs one 128-byte column slice
 * of the source per pass, and in the last pass each workgroup, once its
 * rows are whole, multiplies them by w on the matrix cores (16 rows at a
 * time); rows split into segments are multiplied after their combine.  For
 * bfloat16, h takes its bfloat16 storage rounding before the product, as
 * when it is stored and transformed by saga_apply_vertex; the product
 * accumulates in float32.
 * Supported: COPY messages with SUM or MEAN (dst_norm, bias, act and self
 * as in saga_scatter_apply_edge_gather); src 1 to 4 whole 128-byte lines
 * wide (32..128 float32 or 64..256 bfloat16 columns) and under 4 GiB;
 * w: F x N dense (ld == N), the op's dtype, 1 <= N <= 64; split_col (0, or
 * a multiple of 16 bytes of columns in (0, N)) sends columns from split_col
 * on to `tail`, as saga_apply_vertex's split output does.  out: num_dst x
 * (split_col ? split_col : N), 16-byte rows.  Workspace:
 * saga_gather_transform_workspace_size(plan, op, F) bytes, 256-byte aligned
 * (the split-row partials, h and w packed for the matrix cores).  Errors as
 * saga_scatter_apply_edge_gather,
 * SAGA_EUNSUPPORTED outside the supported shapes. */
typedef struct saga_next_transform {
  saga_cmat w;                    /* F x N weights */
  const int32_t* row_scale_deg;   /* nullable, int32[num_dst] */
  int32_t split_col;              /* 0 = one output matrix */
  saga_mat tail;                  /* num_dst x (N - split_col) when split_col > 0 */
} saga_next_transform;

saga_status saga_gather_transform_workspace_size(const saga_plan* plan, const saga_edge_op* op,
                                                 int64_t feat, size_t* bytes);

saga_status saga_scatter_apply_edge_gather_transform(const saga_plan* plan, const saga_edge_op* op,
                                                     const saga_edge_inputs* in,
                                                     const saga_next_transform* next,
                                                     saga_mat out, void* workspace,
                                                     size_t workspace_bytes, void* stream);

/* The same Gather for callers that cannot allocate device memory (code
 * under HIP graph capture, tight serving loops, harnesses that forbid
 * hipMalloc): no workspace argument.  The split-row partials go to a fixed
 * 64 MiB device array inside the library; each GPU the library runs on
 * holds its own copy from the first call on that GPU until the process
 * ends.  The call allocates nothing and reads the device of `stream` (the
 * current device for the null stream).  Same arguments, validation,
 * results (bit for bit) and errors as saga_scatter_apply_edge_gather, plus
 * SAGA_EUNSUPPORTED when the partials could exceed 64 MiB (bound:
 * saga_gather_workspace_size's value for this plan and op).  The array is
 * shared by every call on one GPU and keeps the last call's contents (no
 * call reads what an earlier call left): calls that overlap on one GPU
 * (different streams without ordering) race and must not be issued. */
saga_status saga_scatter_apply_edge_gather_noalloc(const saga_plan* plan, const saga_edge_op* op,
                                                   const saga_edge_inputs* in, saga_mat out,
                                                   void* stream);

/* ----------------------------------------------------------------------
 * Unfused baseline (Sec. 3.2 "Gather", Fig. 7a): the same operation as
 * saga_scatter_apply_edge_gather, computed the way a framework without a
 * fused kernel does it.  Scatter + ApplyEdge first materialise the edge
 * tensor msg[e] = w(u) * src[u] for every in-edge e = (u -> v) in CSR order
 * (an index-select; w(u) = d_out(u)^-1/2 for SAGA_MSG_SRC_NORM, else 1),
 * written into the workspace; Gather then reduces each destination's
 * contiguous run of msg rows.  Supported: msg COPY or SRC_NORM, reduce SUM,
 * MEAN or MAX, with the same dst_norm / bias / act epilogue; anything else
 * is SAGA_EUNSUPPORTED.  The result matches the fused call up to the order
 * of floating-point additions (MAX and float32 COPY are identical); for
 * bfloat16 with SRC_NORM the message is rounded to bfloat16 before the sum.
 * Workspace: saga_unfused_workspace_size() bytes, 256-byte aligned, not
 * overlapping src or out -- num_edges x (feat padded to whole 16-byte or
 * 64-byte units) elements of the op's dtype plus the split-row partials.
 * ---------------------------------------------------------------------- */
saga_status saga_unfused_workspace_size(const saga_plan* plan, const saga_edge_op* op,
                                        int64_t feat, size_t* bytes);

saga_status saga_scatter_gather_unfused(const saga_plan* plan, const saga_edge_op* op,
                                        const saga_edge_inputs* in, saga_mat out,
                                        void* workspace, size_t workspace_bytes,
                                        void* stream);

/* ----------------------------------------------------------------------
 * LSTM Gather (GraphSAGE row of Table I; Sec. 3.2 "Gather": the reduction
 * that treats a vertex's in-edges as a sequence and cannot be fused).  For
 * destination v with sources u_1 .. u_d in CSR order, from h = c = 0:
 *     z = gates_x[u_t] + h w_hh        (gate blocks i | f | g | o, width H)
 *     i, f, o = sigmoid(z_i, z_f, z_o);  g = tanh(z_g)
 *     c = f * c + i * g;  h = o * tanh(c)
 * out[v] = h after step d (0 for an empty row).  gates_x is the input part
 * of the gates, computed once per source vertex: x_u W_ih + b_ih + b_hh
 * (saga_apply_vertex with bias and bias2), num_src x 4H.  w_hh: H x 4H.
 * out: num_dst x H.  All float32; H = 32, 64 or 128 (SAGA_EUNSUPPORTED
 * otherwise).  Rows run longest first on a persistent grid (one workgroup
 * per CU); the time is bounded below by the longest row's d sequential
 * steps.
 * Workspace: saga_lstm_gather_workspace_size() bytes (a work-queue counter,
 * cleared by the call itself), 256-byte aligned.
 * ---------------------------------------------------------------------- */
saga_status saga_lstm_gather_workspace_size(const saga_plan* plan, int64_t hidden,
                                            size_t* bytes);

saga_status saga_lstm_gather(const saga_plan* plan, saga_cmat gates_x, saga_cmat w_hh,
                             saga_mat out, void* workspace, size_t workspace_bytes,
                             void* stream);

/* The LSTM Gather of the rows at perm positions [perm_begin, perm_end) only
 * (0 <= perm_begin <= perm_end <= num_dst, else SAGA_EINVAL); the other
 * output rows are not written.  perm lists rows by in-degree, largest
 * first, so a run of equal in-degrees is a range: one call per distinct
 * degree is the degree traversal of Sec. 3.2 (Fig. 8b), kept for
 * comparison with the single persistent call.  Calls that share a
 * workspace must be ordered (same stream). */
saga_status saga_lstm_gather_rows(const saga_plan* plan, int32_t perm_begin, int32_t perm_end,
                                  saga_cmat gates_x, saga_cmat w_hh, saga_mat out,
                                  void* workspace, size_t workspace_bytes, void* stream);

/* ======================================================================
 * ApplyVertex: dense transform on the matrix cores
 * ======================================================================
 * Sec. 3.2 "ApplyVertex" (all vertices batched into one GEMM), Table III.
 * mode PLAIN:  out = act(rs * (a w) + bias + bias2)
 * mode CONCAT: out = act(rs * (a w + a2 w2) + bias + bias2)   ([a | a2] [w ; w2])
 *              (bias, bias2 nullable; two vectors so that e.g. an LSTM's
 *              b_ih + b_hh need not be summed by the caller)
 * mode GRU:    GRU cell with input a and hidden state a2 (Fig. 2, GGNN):
 *              gi = a w + bias, gh = a2 w2 + bias2 (column blocks r, z, n of
 *              width F = a2.cols), r = s(gi_r + gh_r), z = s(gi_z + gh_z),
 *              n = tanh(gi_n + r * gh_n), out = (1 - z) n + z a2.
 * rs = row_scale_deg ? (deg[i] > 0 ? deg[i]^-1/2 : 0) : 1  (row i).
 * Split output (split_col = s > 0, PLAIN and CONCAT): the result is written
 * as two matrices, columns [0, s) to out and [s, N) to op->tail.  A result
 * that a Gather reads by rows can so be cut at a 128-byte boundary (s = 32
 * float32 or 64 bfloat16 columns) into a part of whole L2 lines and a
 * narrow rest, each gathered by its own call (e.g. N = 41: 32 + 9 columns
 * instead of one 192-byte row that spans two lines).
 * a: M x K, w: K x N (dense weights, ld may exceed N), out: M x N; bf16 or
 * f32 storage per op->dtype, float32 accumulation; N <= 4096 per call.
 *
 * Workspace: device memory of at least saga_apply_vertex_workspace_size()
 * bytes, 256-byte aligned, owned by the caller and not overlapping any
 * argument.  Each call first writes w (and w2) into it transposed and
 * zero-padded to whole tiles, the layout the matrix-core kernel streams;
 * its contents are scratch afterwards.  Calls that share one workspace
 * must be ordered (same stream).  Missing or too small: SAGA_EWORKSPACE.
 */
typedef enum saga_gemm_mode { SAGA_GEMM_PLAIN = 0, SAGA_GEMM_CONCAT = 1, SAGA_GEMM_GRU = 2 } saga_gemm_mode;

typedef struct saga_gemm_op {
  int32_t dtype;                  /* saga_dtype */
  int32_t mode;                   /* saga_gemm_mode */
  int32_t act;                    /* saga_act; PLAIN / CONCAT */
  const int32_t* row_scale_deg;   /* nullable, int32[M] */
  int32_t split_col;              /* PLAIN / CONCAT: 0 = one output matrix; s > 0: columns
                                     [0, s) go to `out` (M x s) and [s, N) to `tail` */
  saga_mat tail;                  /* M x (N - s), same dtype; used when split_col > 0 */
} saga_gemm_op;

/* Workspace bytes for saga_apply_vertex with op's dtype and mode, k =
 * a.cols, k2 = a2.cols (CONCAT and GRU; ignored for PLAIN), n = w.cols. */
saga_status saga_apply_vertex_workspace_size(const saga_gemm_op* op, int64_t k, int64_t k2,
                                             int64_t n, size_t* bytes);

saga_status saga_apply_vertex(const saga_gemm_op* op, saga_cmat a, saga_cmat w,
                              saga_cmat a2, saga_cmat w2, const float* bias,
                              const float* bias2, saga_mat out, void* workspace,
                              size_t workspace_bytes, void* stream);

/* ======================================================================
 * One whole layer (Table I models)
 * ======================================================================
 * GCN       out = act(d_in^-1/2 A d_out^-1/2 X W + b), evaluated
 *           transform-first: Z = d_out^-1/2 (X W) on the matrix cores, then
 *           the fused sum-Gather with d_in^-1/2, bias and act.
 * GAT       [z | el | er] = X [W | W a_l | W a_r], softmax Gather, then
 *           act(concat + b) or mean over heads + b.
 * SAGE_POOL P = ReLU(X W_pool + b_pool); A = max-Gather of P;
 *           out = [X | A] W + b   (W is 2 F_in x F_out).
 * SAGE_LSTM P = X W_ih + b_ih + b_hh; A = LSTM Gather of P with W_hh
 *           (saga_lstm_gather); out = [X | A] W + b (W is (F_in + H) x
 *           F_out).  float32 only.
 * GATED_GRU [S_src, S_dst] = X [W_e,src, W_e,dst]; gated sum-Gather with
 *           W_e,edge and b_e; out = GRU(a, X) with W_ih, W_hh, b_ih, b_hh.
 *           (W_e rows: [0,F) src part, [F,2F) dst part, [2F,2F+Fe) edge.)
 * RGCN      T = saga_rel_transform(X, W) (W: the num_rel weights stacked,
 *           (num_rel * F_in) x F_out); S = X W_self + b; typed sum-Gather
 *           with self = S: out = act(S_v + sum_e edge_norm[e] T[edge_pair[e]])
 *           (rel: a rel plan of the same graph).
 * Weights are dense device matrices (ld = cols) in the layer dtype; biases
 * and attention vectors f32.  x: num_src x F_in (num_src == num_dst).
 * act applies to GCN, GAT and RGCN.  GCN and RGCN take f32 or bf16; GAT,
 * SAGE_POOL, SAGE_LSTM and GATED_GRU are float32 only (SAGA_EUNSUPPORTED
 * for bf16).
 */
typedef enum saga_layer_kind {
  SAGA_LAYER_GCN = 0,
  SAGA_LAYER_GAT = 1,
  SAGA_LAYER_SAGE_POOL = 2,
  SAGA_LAYER_GATED_GRU = 3,
  SAGA_LAYER_SAGE_LSTM = 4,
  SAGA_LAYER_RGCN = 5
} saga_layer_kind;

typedef struct saga_layer_desc {
  int32_t kind;                   /* saga_layer_kind */
  int32_t dtype;                  /* saga_dtype */
  int32_t in_feat, out_feat;
  int32_t heads, head_mean;       /* GAT */
  float neg_slope;                /* GAT */
  int32_t act;                    /* saga_act; GCN, GAT, RGCN */
  int32_t edge_feat;              /* GATED_GRU: Fe */
  const void* w;  const float* b;             /* GCN, GAT, SAGE_POOL */
  const void* w_pool; const float* b_pool;    /* SAGE_POOL */
  const float* attn_l; const float* attn_r;   /* GAT: heads x (F/heads) */
  const float* w_e; const float* b_e;         /* GATED_GRU: (2F + Fe) x F, F */
  const float* w_ih; const float* b_ih;       /* GATED_GRU: F x 3F, 3F; SAGE_LSTM: F x 4H, 4H */
  const float* w_hh; const float* b_hh;       /* GATED_GRU: F x 3F;  SAGE_LSTM: H x 4H, 4H */
  int32_t hidden;                             /* SAGE_LSTM: H (32, 64 or 128) */
  const void* w_self;                         /* RGCN: F_in x F_out (w: stacked W_r) */
  const saga_rel_plan* rel;                   /* RGCN */
} saga_layer_desc;

saga_status saga_layer_workspace_size(const saga_plan* plan, const saga_layer_desc* desc,
                                      size_t* bytes);

saga_status saga_layer(const saga_plan* plan, const saga_layer_desc* desc, saga_cmat x,
                       saga_cmat edge_feat, saga_mat out, void* workspace,
                       size_t workspace_bytes, void* stream);

/* Stage tracing, for timing and profiling the stages inside saga_layer.
 * After each of its stages, saga_layer records the next of these caller-
 * created hipEvent_t on its stream (events[0] after the first stage, ...;
 * stages past n_events record nothing), and with markers != 0 launches an
 * empty kernel named k_stage_mark there (and k_stage_begin before the first
 * stage), which delimit the stages in a counter profile's list of
 * dispatches; with markers the host side of each call is also bracketed by
 * roctx ranges, "saga_layer" around the call and "saga stage k" around the
 * enqueue of stage k (k from 0, in the order below), for a timeline trace.
 * The stages, in order:
 *   GCN (transform first)   transform, gather (a split output: transform,
 *                           gather of the whole-line columns, gather of the
 *                           rest)
 *   GCN (aggregate first)   gather, transform
 *   GAT                     transform (with the folded attention columns),
 *                           gather
 *   SAGE_POOL               pool transform, max gather, concat transform
 *   SAGE_LSTM               input transform, LSTM gather, concat transform
 *   GATED_GRU               source-gate transform, destination-gate
 *                           transform, gated gather, GRU transform
 *   RGCN                    relation transform, self transform, typed gather
 * Each saga_layer call starts again from events[0].  The setting is
 * thread-local and copied (the array may be freed after the call); pass
 * NULL, 0, 0 to stop.  Errors: SAGA_EINVAL (n_events < 0, a null array or
 * event). */
saga_status saga_trace_stages(void* const* events, int32_t n_events, int32_t markers);

/* ====================================================================== */
/* Every compute call is asynchronous on the caller's stream: its status
 * covers argument checks and the launch only.  saga_sync_check waits for
 * all work enqueued on `stream` (NULL: the null stream) and returns
 * SAGA_EDEVICE, with the HIP error in saga_last_error, if the device
 * reported one; else SAGA_OK.  It allocates nothing. */
saga_status saga_sync_check(void* stream);

const char* saga_status_str(saga_status s);
const char* saga_last_error(void);
/* Library version string. */
const char* saga_version(void);

#ifdef __cplusplus
}
#endif
#endif /* SAGA_H */
