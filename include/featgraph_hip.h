/*
 * featgraph_hip.h -- C ABI of the gfx950 (MI355X) library for FeatGraph's two
 * feature-dimension sparse templates (Hu et al., "FeatGraph: A Flexible and
 * Efficient Backend for Graph Neural Network Systems", SC20):
 *
 *   generalized SpMM   (vertex-wise, Sec. II-A Eq. 1 and Eq. 3; the spmm
 *                       template of Sec. III-B / Fig. 3)
 *   generalized SDDMM  (edge-wise, Sec. II-A Eq. 2 and Eq. 4; the sddmm
 *                       template of Sec. III-B / Fig. 4, multi-head Fig. 4b)
 *   edge softmax       (per-destination normalisation of edge scores that
 *                       sits between the two in an attention layer)
 *   backward of gSpMM-max and of edge softmax (training; the backward of
 *                       gSpMM-sum and gSDDMM are themselves gSDDMM and gSpMM
 *                       calls, Sec. II-A)
 *   MLP aggregation    (Fig. 1 / Fig. 3b: a dense vertex transform on the
 *                       matrix cores, then a gSpMM with a relu(u + v) message)
 *
 * The paper's user-defined message / edge functions become a closed set of
 * operators (the builtin message functions it supports, Sec. III-B): copy the
 * source feature, or multiply it by an edge value (one scalar per edge and
 * head); reducers sum and max (with the edge id of the maximum).
 *
 * ---------------------------------------------------------------------------
 * Conventions shared by every entry point
 * ---------------------------------------------------------------------------
 * Graph      CSR with rows = DESTINATION vertices (row v lists the in-edges of
 *            v, so Eq. 1 reduces over in-neighbours).  indptr/indices/edge_ids
 *            are int32 DEVICE arrays.  The edge id of stored entry p is
 *            edge_ids[p], or p when edge_ids is NULL.  A transposed graph (CSC:
 *            rows = source vertices) is passed the same way with edge_ids set
 *            to the CSR positions, so edge data keeps one indexing.
 * Features   fp32, row-major, DEVICE memory.  Vertex data is [vertices, H, dh]
 *            (H heads of head_dim dh, F = H*dh floats per vertex); edge data is
 *            [edge id, H].  All offsets are computed in 64-bit.
 * Streams    `stream` is a hipStream_t passed as void* (NULL = null stream).
 *            Every compute call only enqueues work on it and returns; device
 *            faults surface at the caller's next synchronisation.
 * Ownership  The caller owns every array and the stream.  The library allocates
 *            device memory only in fg_plan_create (freed by fg_plan_destroy);
 *            fg_gspmm_noalloc uses a fixed device array the library holds.
 * Errors     The return code is the only error channel.  Argument checks run on
 *            the host before anything is enqueued; on failure nothing is
 *            written.  FG_ERR_HIP means a HIP call failed (launch or copy).
 *            Indices are NOT range-checked on the device: a graph whose
 *            indices/edge_ids lie outside [0, num_cols) / [0, nnz_total) is
 *            undefined behaviour (check it on the host first).
 * Aliasing   Outputs must not overlap inputs (checked where sizes are known).
 * Limits     nnz <= INT32_MAX; F = H*dh <= FG_MAX_WIDTH.
 * Precision  fp32 in, fp32 accumulate, fp32 out; no fast-math.  Max compares
 *            the fp32 message values exactly (IEEE ==, so -0 == +0).
 */
#ifndef FEATGRAPH_HIP_H_
#define FEATGRAPH_HIP_H_

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define FG_ABI_VERSION 4
#define FG_MAX_WIDTH (1 << 16) /* largest supported F = H*dh */

typedef enum fg_status {
  FG_OK = 0,
  FG_ERR_INVALID_ARG = -1, /* a host-side argument check failed */
  FG_ERR_UNSUPPORTED = -2, /* valid but not implemented combination */
  FG_ERR_HIP = -3,         /* a HIP runtime call failed */
  FG_ERR_NO_MEMORY = -4,   /* device or host allocation failed (plan only) */
  FG_ERR_SCRATCH_LIMIT = -5 /* fg_gspmm_noalloc: the call needs more than its
                               fixed scratch (FG_NOALLOC_SCRATCH_BYTES)      */
} fg_status;

/* Message function phi of Eq. 1 (Sec. III-B builtins). */
typedef enum fg_msg_op {
  FG_MSG_COPY_SRC = 0,    /* m = x_src[u, h, :]                            */
  FG_MSG_SRC_MUL_EDGE = 1 /* m = edge_val[e, h] * x_src[u, h, :]           */
} fg_msg_op;

/* Aggregator of Eq. 1 (any commutative reducer; sum as in GCN, Eq. 3; max as
 * in GraphSage-style and MLP aggregation, Fig. 1). */
typedef enum fg_reduce_op {
  FG_REDUCE_SUM = 0, /* out = sum of messages; empty row -> 0                 */
  FG_REDUCE_MAX = 1  /* out = max of messages and arg = the smallest edge id
                        attaining it; empty row -> out 0, arg -1              */
} fg_reduce_op;

/* Edge function psi of Eq. 2. */
typedef enum fg_edge_op {
  FG_EDGE_DOT = 0 /* out[e, h] = sum_k x_src[u, h, k] * x_dst[v, h, k] (Eq. 4,
                     per head as in Fig. 4b)                                 */
} fg_edge_op;

typedef struct fg_graph {
  int64_t num_rows; /* destination vertices (CSR rows)                          */
  int64_t num_cols; /* source vertices                                          */
  int64_t nnz;      /* stored edges = indptr[num_rows]                          */
  int64_t nnz_total;/* size of the edge-id space edge data is indexed by; 0
                       means nnz (set it to the CSR's nnz for a transposed graph) */
  const int32_t* indptr;   /* [num_rows+1], indptr[0] = 0, nondecreasing        */
  const int32_t* indices;  /* [nnz] source vertex of each stored edge           */
  const int32_t* edge_ids; /* [nnz] edge id of each stored edge, or NULL        */
} fg_graph;

/* ---------------------------------------------------------------------------
 * Plan: the degree-aware work decomposition of one graph, built once per
 * graph like the per-topology kernels the paper amortises over training
 * epochs (Sec. IV-B).  It replaces the paper's per-block row assignment
 * (Sec. III-C, adaptive parallelization) with one that stays balanced on
 * power-law graphs, and revives its 1D source partitioning (Sec. III-C, graph
 * partitioning) for the caches of each MI355X die.
 *
 * A plan holds two schedules over one workspace, and a third for the SDDMM
 * on some graphs:
 *  - plain (edge softmax): rows with more than S edges are cut into
 *    k = min(ceil(deg / S), max_row_segments) equal segments, S =
 *    softmax_segment_edges if given, else segment_edges if given, else 16384
 *    (a whole row of up to 16384 scores is streamed by one wavefront; a cut
 *    row is read once more by a merge pass); long items first
 *    (fg_plan_options.item_order), rows without edges last;
 *  - gather (gSpMM, gSDDMM, the fused SDDMM + edge softmax, fused
 *    attention): as plain with S =
 *    segment_edges if given, else 1536, unless source
 *    partitioning applies (by default once the num_cols x max_width source
 *    features exceed 128 MiB, half the Infinity Cache, or 32 MiB when the
 *    gathers are spread; see fg_plan_options.source_slab_rows).  With it,
 *    rows with at least
 *    partition_min_degree edges (if given; else max(64, 8 * ceil(num_cols /
 *    source_slab_rows)), so that pieces average 8 edges or more) and sorted
 *    source ids are cut where their sources change slab (slabs:
 *    consecutive source ids, at most source_slab_rows of them and about equal
 *    shares of these rows' edges), then into pieces of at most S edges; each
 *    slab runs on one die (slabs dealt in order to the least-loaded die), so
 *    each die gathers from a narrow band of the feature matrix at a time
 *    (more hits in its L2 and the Infinity Cache, at the price of more
 *    pieces to merge).  This pays on graphs whose gathers have no locality
 *    of their own (sources spread uniformly, or features beyond the Infinity
 *    Cache) and costs more than it saves on graphs with hubs or communities
 *    whose features the caches hold, hence the size threshold.
 *  - the SDDMM's own (only on spread graphs with source slabs, a max_width
 *    of 256 floats or more and num_cols x max_width features of at most
 *    256 MiB, the Infinity Cache): every row cut where its sources change
 *    slab (16 slabs of about equal edge shares), no partial-result slots;
 *    fg_gsddmm runs it for H * head_dim >= 256, the gather schedule
 *    otherwise.
 * Items of rows cut in several pieces write partial results that a second
 * pass merges in a fixed order, so results are deterministic for a plan.
 * ------------------------------------------------------------------------- */
typedef struct fg_plan fg_plan; /* opaque; owns device schedules + workspace */

typedef struct fg_plan_options {
  int32_t segment_edges;        /* S: target edges per item; 0 -> default (1536 for
                                   the gather schedule, 16384 for the plain one)    */
  int32_t max_row_segments;     /* cap on items per row (plain cut); 0 -> 128        */
  int32_t source_slab_rows;     /* source ids per slab of the gather schedule;
                                   0 -> automatic slabs if the num_cols x
                                   max_width features exceed 128 MiB, or exceed
                                   32 MiB with spread gathers (the most used 4 MB
                                   of source rows take under 45% of the edges,
                                   and rows with neighbouring ids do not share
                                   sources), else none (default); -1 ->
                                   automatic slabs if they exceed 32 MiB (the
                                   dies' L2s together);
                                   -2 -> no source partitioning; automatic
                                   slabs: the larger of 8 MiB of features at
                                   max_width and num_cols / 16 ids              */
  int32_t partition_min_degree; /* smallest row cut by slabs; 0 -> max(64, 8 *
                                   number of id slabs)                              */
  int32_t item_order;           /* order of the work items: 0 -> automatic (2 if rows
                                   with neighbouring ids share sources, judged on
                                   64 windows of 32 rows, else 1, and then 3 if
                                   some row is cut into 8 or more pieces; 1 or 3
                                   without indices); 1 -> longest first; 2 -> by
                                   power-of-two length class, longest first, rows
                                   in id order within a class; 3 -> die-banded
                                   gather schedule (unless source slabs apply):
                                   the items of 1, except that rows of more than
                                   band_row_edges edges are cut into at least 8
                                   pieces; piece k of a row cut into K pieces
                                   runs on die floor(8 (k + 1/2) / K) if K >= 8,
                                   else on one of the dies [floor(8k / K),
                                   ceil(8(k + 1) / K)) (the pieces sharing such
                                   a span take its dies in turn), so each die
                                   gathers from one eighth of those rows'
                                   sources; whole rows balance the dies' edges
                                   (edge softmax keeps order 1); with
                                   band_row_edges = -1 results equal those of 1 */
  int32_t max_backward;         /* 1 -> also reserve the workspace of the binned
                                   gSpMM-max backward: 8 bytes per element of a
                                   num_rows x max_width gradient (that product must
                                   not exceed 2^31 - 1, else FG_ERR_UNSUPPORTED)
                                   plus bin tables (128 KiB, and 1 KiB per source
                                   tile, at most 8 MiB); 0 -> none (default)       */
  int32_t softmax_segment_edges;/* S of the plain schedule; 0 -> segment_edges if that
                                   is given, else 16384                             */
  int32_t band_row_edges;       /* die-banded gather schedule (item_order 3): rows
                                   of more edges are cut into at least
                                   min(8, max_row_segments) pieces, so that every
                                   die takes a share of them; 0 -> 256; -1 -> no
                                   such cut (the items of order 1)                  */
  int32_t reserved[2];          /* must be zero                                      */
} fg_plan_options;

typedef struct fg_plan_info {
  int64_t num_rows, nnz;
  int64_t num_segments;         /* gather schedule: work items (with padding)        */
  int64_t num_split_rows;       /* gather schedule: rows with several items          */
  int64_t num_slots;            /* gather schedule: partial-result slots             */
  int64_t num_partitioned_rows; /* rows cut at source-slab boundaries                */
  int64_t plain_segments, plain_split_rows, plain_slots; /* edge-softmax schedule    */
  int64_t max_width;            /* largest F the workspace holds                     */
  int64_t workspace_bytes;
  int32_t segment_edges, max_row_segments, source_slab_rows, partition_min_degree;
  int32_t item_order;           /* the order used: 1, 2 or 3 (see fg_plan_options)   */
  int32_t max_backward;         /* 1 if the binned max-backward workspace is held    */
  uint64_t indptr_checksum;     /* fg_indptr_checksum of the indptr it was built for */
  int64_t sddmm_segments;       /* the SDDMM's own schedule: work items; 0: none (the
                                   gather schedule serves it)                       */
} fg_plan_info;

/* One work item of a schedule (host view; the device tables hold the same). */
typedef struct fg_segment {
  int32_t row;   /* destination row; -1: empty padding item                    */
  int32_t begin; /* first stored edge (CSR position)                           */
  int32_t end;   /* one past the last stored edge                              */
  int32_t slot;  /* -1: whole row, results go to the output directly;
                    >= 0: partial-result slot of a row cut in several pieces   */
} fg_segment;

/* Builds a schedule on the host (which = 0: gather, 1: plain, 2: the SDDMM's,
 * which is the gather schedule where the plan has no schedule of its own for
 * it) from HOST
 * copies of indptr and (optional; NULL: no source partitioning) indices.
 * Writes at most `capacity` items to `segs` (may be NULL to only count) and
 * the counts to the optional out-pointers.  Pure host function: no HIP call. */
fg_status fg_schedule_host(const int32_t* indptr_host, const int32_t* indices_host,
                           int64_t num_rows, int64_t num_cols, int64_t max_width,
                           const fg_plan_options* opt, int32_t which, fg_segment* segs,
                           int64_t capacity, int64_t* num_segments, int64_t* num_split_rows,
                           int64_t* num_slots);

/* Creates a plan for graph `g` and features up to `max_width` = H*dh floats.
 * indptr_host / indices_host: optional HOST copies of g->indptr / g->indices
 * (without them the plan copies what it needs from the device: indptr, the
 * indices when source slabs may apply, else 64 windows of them for the item
 * order).  opt may be NULL.  Validates indptr, and the indices whenever it
 * holds them all on the host (FG_ERR_INVALID_ARG), allocates device memory,
 * synchronises `stream`.  The plan is bound to g->indptr, num_rows and
 * nnz: calls with another graph are rejected with FG_ERR_INVALID_ARG; it
 * also keeps the checksum of indptr (fg_plan_validate re-checks it).  Its
 * workspace is mutable: calls that share a plan must be ordered on one
 * stream. */
fg_status fg_plan_create(const fg_graph* g, const int32_t* indptr_host,
                         const int32_t* indices_host, int64_t max_width,
                         const fg_plan_options* opt, fg_plan** out, void* stream);
fg_status fg_plan_destroy(fg_plan* plan);
fg_status fg_plan_get_info(const fg_plan* plan, fg_plan_info* info);

/* Checksum of a HOST indptr array [num_rows + 1]: 64-bit FNV-1a over the
 * little-endian bytes of its int32 entries (offset basis 14695981039346656037,
 * prime 1099511628211).  Pure host function: no HIP call. */
fg_status fg_indptr_checksum(const int32_t* indptr_host, int64_t num_rows, uint64_t* out);

/* Re-validates a plan against graph `g`: the bindings every call checks
 * (indptr pointer, num_rows, nnz) and the checksum of indptr's current
 * contents against the one taken when the plan was built, so that a plan is
 * not reused after indptr was edited in place or another graph of the same
 * shape was placed at the same address.  indptr_host: an optional HOST copy
 * of g->indptr; without it indptr is copied from the device on `stream`,
 * which is synchronised.  FG_OK if the plan fits, FG_ERR_INVALID_ARG if not.
 * (The compute calls check only the pointer and sizes: the checksum costs a
 * pass over indptr, so callers that edit graphs in place call this.) */
fg_status fg_plan_validate(const fg_plan* plan, const fg_graph* g, const int32_t* indptr_host,
                           void* stream);

/* ---------------------------------------------------------------------------
 * Generalized SpMM (Sec. II-A Eq. 1; Sec. III-B featgraph.spmm):
 *   out[v, h, k] = (+)_{stored edges p of row v} phi(p)[h, k]
 * x_src    [num_cols, H, dh]
 * edge_val [nnz_total, H] indexed by edge id; required iff msg = SRC_MUL_EDGE
 * out      [num_rows, H, dh]; every element is written
 * arg_eid  [num_rows, H, dh] int32; required iff red = MAX, else must be NULL
 * plan     NULL -> one wavefront per row (no load balancing); else a plan of
 *          this graph with max_width >= H*dh
 * Sums are fp32 in an order that depends on the schedule (deterministic for a
 * given plan).  Max/argmax is exact and schedule-independent.  A NaN message
 * competes as -inf: it never beats a number, and a row whose messages are all
 * NaN or -inf gives -inf with its smallest edge id.
 * ------------------------------------------------------------------------- */
fg_status fg_gspmm(const fg_graph* g, fg_msg_op msg, fg_reduce_op red, int32_t num_heads,
                   int64_t head_dim, const float* x_src, const float* edge_val, float* out,
                   int32_t* arg_eid, fg_plan* plan, void* stream);

/* ---------------------------------------------------------------------------
 * fg_gspmm without any allocation, for callers that cannot allocate device
 * memory at call time (code recorded into a HIP graph, tight serving loops,
 * harnesses that forbid hipMalloc).  Same arguments, checks and results as
 * fg_gspmm: with the same plan it runs the same kernels in the same order,
 * so its results are bitwise those of fg_gspmm.  The difference is where
 * the partial results of rows the plan cuts into several items live: not in
 * the plan's workspace but in a fixed device array of
 * FG_NOALLOC_SCRATCH_BYTES that the library holds on every device it runs on
 * until the process ends.
 * Limit     the plan's gather schedule needs num_slots * H * dh * 4 bytes
 *           for sum, and twice that (rounded up to 256 bytes) for max
 *           (values and edge ids); larger calls return FG_ERR_SCRATCH_LIMIT
 *           before anything is enqueued.  (The power-law benchmark graph at
 *           d = 128, 18,203 slots: 9.3 MB for sum, 18.6 MB for max.)
 *           Without a plan, or with a plan that cuts no row, no scratch is
 *           used.
 * Sharing   every call on one device uses the same array: calls that can
 *           overlap in time on one device (different streams, or host
 *           threads) race and must be ordered by the caller.  Each call
 *           writes every slot it reads, so nothing needs clearing between
 *           calls.
 * Set-up    the first call on a device (with that device current) looks up
 *           the array's device address (hipGetSymbolAddress) and keeps it;
 *           make that first call before capturing later ones into a graph.
 * Nothing is allocated: no hipMalloc, no hipFree, no allocating library call.
 * ------------------------------------------------------------------------- */
#define FG_NOALLOC_SCRATCH_BYTES (32 << 20)
fg_status fg_gspmm_noalloc(const fg_graph* g, fg_msg_op msg, fg_reduce_op red, int32_t num_heads,
                           int64_t head_dim, const float* x_src, const float* edge_val,
                           float* out, int32_t* arg_eid, fg_plan* plan, void* stream);

/* ---------------------------------------------------------------------------
 * Generalized SDDMM (Sec. II-A Eq. 2 and Eq. 4; Sec. III-B featgraph.sddmm;
 * multi-head edge function of Fig. 4b):
 *   out[e, h] = sum_k x_src[indices[p], h, k] * x_dst[v, h, k]
 * for every stored edge p of every row v, e = its edge id.
 * x_src [num_cols, H, dh]; x_dst [num_rows, H, dh]; out [nnz_total, H]
 * (entries of edge ids not stored in g are left untouched).
 * fp32 accumulation, tree reduction across the lanes that hold one head.
 * ------------------------------------------------------------------------- */
fg_status fg_gsddmm(const fg_graph* g, fg_edge_op op, int32_t num_heads, int64_t head_dim,
                    const float* x_src, const float* x_dst, float* out, fg_plan* plan,
                    void* stream);

/* ---------------------------------------------------------------------------
 * Edge softmax over each row's stored edges, per head, optionally after a
 * leaky ReLU:  s' = s > 0 ? s : negative_slope * s;
 *              out[e, h] = exp(s'_e - m) / sum_row exp(s' - m),  m = row max.
 * scores, out [nnz_total, H] indexed by edge id; rows without edges write
 * nothing.  `out` may equal `scores` only if no two stored edges share an id.
 * ------------------------------------------------------------------------- */
fg_status fg_edge_softmax(const fg_graph* g, int32_t num_heads, const float* scores,
                          int32_t apply_leaky_relu, float negative_slope, float* out,
                          fg_plan* plan, void* stream);

/* ---------------------------------------------------------------------------
 * Fused attention aggregation: the three steps above in one pass, without
 * materialising per-edge scores (the paper's point that UDFs are inlined into
 * the template instead of messages being materialised on every edge,
 * Sec. III-B and Sec. IV-A).  For every row v and head h:
 *   s_e  = sum_k x_src[u, h, k] * x_dst[v, h, k]          (Eq. 4 per head, Fig. 4b)
 *   a_e  = softmax over the row of leaky_relu(s_e)         (optional leaky ReLU)
 *   out[v, h, :] = sum_e a_e * x_src[u, h, :]              (Eq. 1, src_mul_edge + sum)
 * equal, up to rounding, to fg_gsddmm -> fg_edge_softmax -> fg_gspmm.  Each
 * source row is gathered once per edge; rows without edges give 0.
 * x_src [num_cols, H, dh]; x_dst [num_rows, H, dh]; out [num_rows, H, dh].
 * Supported shapes: dh % 4 == 0, dh / 4 a power of two, H * dh <= 256, and
 * 16-byte aligned feature arrays; otherwise FG_ERR_UNSUPPORTED (compose the
 * three calls instead).  A plan must have max_width >= H * dh.
 * ------------------------------------------------------------------------- */
fg_status fg_gat_aggregate(const fg_graph* g, int32_t num_heads, int64_t head_dim,
                           const float* x_src, const float* x_dst, int32_t apply_leaky_relu,
                           float negative_slope, float* out, fg_plan* plan, void* stream);

/* ---------------------------------------------------------------------------
 * SDDMM dot followed by edge softmax in one call (the attention scores of
 * Eq. 4 and their normalisation, fused where the scores are produced, as the
 * paper fuses UDFs into its templates, Sec. III-B):
 *   scores[e, h] = fg_gsddmm's output;  out[e, h] = fg_edge_softmax(scores)
 * One head with dh % 4 == 0, dh <= 1024 and 16-byte aligned features runs as
 * one pass (plus the merge of split rows), unless the plan's items average
 * 128 edges or more: there, and for other shapes, the two operators run one
 * after the other (the SDDMM's batches of 256 edges and the streaming softmax
 * are faster on such plans than the fused pass).  Both arrays are [nnz_total, H], written for
 * the edges of g.  A plan must have max_width >= max(H * dh, H).
 * ------------------------------------------------------------------------- */
fg_status fg_gsddmm_edge_softmax(const fg_graph* g, int32_t num_heads, int64_t head_dim,
                                 const float* x_src, const float* x_dst, int32_t apply_leaky_relu,
                                 float negative_slope, float* scores, float* out, fg_plan* plan,
                                 void* stream);

/* ---------------------------------------------------------------------------
 * Gradient of gSpMM with the max aggregator, for training with max
 * aggregation (GraphSage, Sec. V-E).  Sec. II-A derives the backward of the
 * templates by the chain rule; for (+) = max each output element took its
 * value from one edge, so only that edge's message receives the upstream
 * gradient.  For every (v, h, k) with e = arg_eid[v, h, k] >= 0 and u the
 * source of edge e:
 *   grad_src[u, h, k] += (src_mul_edge ? edge_val[e, h] : 1) * grad_out[v, h, k]
 *   grad_edge[e, h]   += x_src[u, h, k] * grad_out[v, h, k]      (src_mul_edge)
 * x_src     [num_cols, H, dh]; needed iff grad_edge != NULL
 * edge_val  [nnz_total, H]; required iff msg = SRC_MUL_EDGE, else NULL
 * arg_eid   [num_rows, H, dh] int32, as written by fg_gspmm(..., FG_REDUCE_MAX)
 * grad_out  [num_rows, H, dh]
 * grad_src  [num_cols, H, dh] or NULL; grad_edge [nnz_total, H] or NULL (must
 *           be NULL for copy_src).  Both are fully overwritten (zeros where
 *           nothing arrives).
 * plan      required when g->edge_ids != NULL: a plan created for this graph
 *           with these edge ids (it maps ids back to storage positions; ids
 *           must be distinct); otherwise optional and unused.
 * Entries of arg_eid that are not edge ids of g are skipped.
 * With a plan that holds the binned workspace (fg_plan_options.max_backward)
 * and H * dh <= max_width, <= 16384, and num_cols / (source rows per 64 KiB
 * tile) <= 8192 tiles, grad_src is built by binning: every element becomes
 * an 8-byte record in the bin of its source tile (a counting sort), and one
 * workgroup per piece of up to 16384 records sums a bin in LDS and writes the
 * tile's rows.  Otherwise, and for grad_edge always, contributions go to
 * zero-filled arrays with fp32 atomics.  Either way the order of the adds
 * into one element is not fixed, so a sum of several contributions may
 * differ in the last bits between calls, and the adds may flush subnormal
 * results to zero.
 * ------------------------------------------------------------------------- */
fg_status fg_gspmm_max_backward(const fg_graph* g, fg_msg_op msg, int32_t num_heads,
                                int64_t head_dim, const float* x_src, const float* edge_val,
                                const int32_t* arg_eid, const float* grad_out, float* grad_src,
                                float* grad_edge, fg_plan* plan, void* stream);

/* ---------------------------------------------------------------------------
 * Gradient of fg_edge_softmax w.r.t. its scores, for training attention
 * layers (GAT, Sec. V-E).  With a = the forward's output and G = dL/da, per
 * row v and head h:
 *   c = sum_{edges p of v} a_p * G_p
 *   grad_scores[e, h] = a_e * (G_e - c) * (leaky && !(s_e > 0) ? slope : 1)
 * (softmax Jacobian diag(a) - a a^T; the leaky ReLU's derivative is the slope
 * for s <= 0, as in its forward).
 * out        [nnz_total, H] the forward's result a
 * grad_out   [nnz_total, H] G
 * scores     [nnz_total, H] the forward's input s; required iff
 *            apply_leaky_relu, else ignored
 * grad_scores [nnz_total, H]; entries of edges of g are written, others left
 *            untouched.  It may be the same array as grad_out (in place); it
 *            must not overlap out or scores.
 * Sums are fp32 in a fixed order for a given plan (deterministic).
 * ------------------------------------------------------------------------- */
fg_status fg_edge_softmax_backward(const fg_graph* g, int32_t num_heads, const float* out,
                                   const float* grad_out, const float* scores,
                                   int32_t apply_leaky_relu, float negative_slope,
                                   float* grad_scores, fg_plan* plan, void* stream);

/* ---------------------------------------------------------------------------
 * The score gradient of an attention layer in one call: the gSDDMM dot of
 * x_src and x_dst per head (Sec. II-A: the gradient of the SpMM y = A(s) x
 * w.r.t. its edge values is an SDDMM of the upstream gradient with x), fed
 * straight into fg_edge_softmax_backward.  Per row v and head h:
 *   g_e = sum_k x_src[u_e, h, k] * x_dst[v, h, k]
 *   c   = sum_{edges p of v} out_p * g_p
 *   grad_scores[e, h] = out_e * (g_e - c) * (leaky && !(s_e > 0) ? slope : 1)
 * x_src      [num_cols, H, dh] (the layer's source features)
 * x_dst      [num_rows, H, dh] (the upstream gradient of the aggregation)
 * out        [nnz_total, H] the forward softmax's result
 * scores     [nnz_total, H] the forward softmax's input; required iff
 *            apply_leaky_relu
 * grad_scores [nnz_total, H]; entries of edges of g are written.  It must not
 *            overlap any input.
 * One fused pass when 2 <= H <= 16, head_dim is 16, 32 or 64, H * head_dim
 * <= 256, the feature arrays are 16-byte aligned and the plan (if any) cuts
 * no row of its softmax schedule; otherwise the same results through
 * fg_gsddmm into grad_scores followed by fg_edge_softmax_backward in place.
 * Sums are fp32 in a fixed order for a given plan (deterministic).
 * ------------------------------------------------------------------------- */
fg_status fg_gsddmm_edge_softmax_backward(const fg_graph* g, int32_t num_heads, int64_t head_dim,
                                          const float* x_src, const float* x_dst,
                                          const float* out, const float* scores,
                                          int32_t apply_leaky_relu, float negative_slope,
                                          float* grad_scores, fg_plan* plan, void* stream);

/* ---------------------------------------------------------------------------
 * Dense vertex transform y = x w (fp32 on the matrix cores): the vector-matrix
 * product of the MLP aggregation's message function (Fig. 3b), applied once
 * per vertex.  x [n, d_in], w [d_in, d_out], y [n, d_out] row-major; y must
 * not overlap x or w.  fp32 products and sums (order fixed by the kernel).
 * ------------------------------------------------------------------------- */
fg_status fg_dense_matmul(int64_t n, int64_t d_in, int64_t d_out, const float* x, const float* w,
                          float* y, void* stream);

/* ---------------------------------------------------------------------------
 * MLP aggregation (Fig. 1, message function of Fig. 3b) with the max
 * aggregator:
 *   out[v, i]     = max over stored edges (u -> v, id e) of
 *                   relu( sum_k (x_src[u, k] + x_dst[v, k]) * weight[k, i] )
 *   arg_eid[v, i] = the edge that supplies it;  empty row -> 0 / -1
 * where relu(t) = t > 0 ? t : 0.  Computed as P_src = x_src weight and
 * P_dst = x_dst weight (fg_dense_matmul) followed by a gSpMM whose message is
 * relu(P_src[u] + P_dst[v]): equal to the per-edge form in exact arithmetic
 * (the product distributes over the sum), without d_in * d_out multiply-adds
 * per edge.  The edges compete by their fp32 P_src[u, i]: arg_eid is the
 * smallest edge id among the edges with the largest P_src[u, i], and out is
 * relu(that P_src + P_dst[v, i]) rounded once (fp32 rounding is monotone, so
 * this is the largest rounded message); when that is not positive every
 * message is 0 and arg_eid is the row's smallest edge id.  Every schedule,
 * width and edge-id layout follows this rule, so results do not depend on
 * the plan.  Rounding differs from the per-edge form, and so may the argmax
 * between messages closer than that rounding.
 * x_src     [num_cols, d_in];  x_dst [num_rows, d_in] (may be x_src itself
 *           when num_rows == num_cols: one transform);  weight [d_in, d_out]
 * out, arg_eid [num_rows, d_out]
 * workspace caller-owned device scratch of (num_cols + num_rows) * d_out
 *           floats (16-byte aligned for the vector path); clobbered
 * plan      as for fg_gspmm, with max_width >= d_out
 * Nothing is allocated; calls sharing a workspace must be ordered on one
 * stream.
 * ------------------------------------------------------------------------- */
fg_status fg_mlp_aggregate(const fg_graph* g, int64_t d_in, int64_t d_out, const float* x_src,
                           const float* x_dst, const float* weight, float* out, int32_t* arg_eid,
                           float* workspace, fg_plan* plan, void* stream);

const char* fg_status_string(fg_status s); /* static storage, never NULL */
int32_t fg_abi_version(void);              /* == FG_ABI_VERSION */

#ifdef __cplusplus
}
#endif

#endif /* FEATGRAPH_HIP_H_ */
