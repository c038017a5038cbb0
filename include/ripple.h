/*
 * ripple.h -- C ABI of the MI355X library for exact incremental propagation of
 * GNN embeddings on a streaming graph (Ripple, arXiv 2505.12112).
 *
 * The problem statement (Sec. IV-A, "Assumptions") has four parts, one call each:
 *   1. a graph G(V,E) and a trained L-layer GNN with a linear aggregator
 *      ............................................. ripple_load_graph, ripple_init_embeddings
 *   2. initial embeddings H^1..H^L of every vertex, computed before updates arrive
 *      ............................................. ripple_init_embeddings
 *   3. a stream of edge inserts, edge deletes and vertex-feature replacements,
 *      applied in fixed-size batches (no vertex inserts or deletes)
 *      ............................................. ripple_apply_updates
 *   4. after each batch, the exact embeddings of every affected vertex are
 *      available at once (trigger-based inference, Sec. II-B; exact within
 *      floating-point precision, Sec. VI)
 *      ............................................. ripple_get_embeddings, ripple_get_affected
 *
 * The GNN layer is Eq. (1)-(2) of Sec. II-A with one of the linear aggregators of
 * Sec. II-C: x_v = Aggregate({h_u : u in N_in(v)}), h_v = sigma(Update(h_v, x_v)).
 *   RIPPLE_AGG_SUM   GraphSAGE-sum : h = sigma(W_self h_v + W_neigh sum_u h_u + b)
 *   RIPPLE_AGG_MEAN  GraphSAGE-mean: h = sigma(W_self h_v + W_neigh mean_u h_u + b),
 *                    the mean is 0 for a vertex without in-neighbours
 *   RIPPLE_AGG_GCN   GCN, symmetric normalisation with an implicit self-loop:
 *                    h = sigma(W sum_{u in N_in(v) + v} h_u / sqrt((dout(u)+1)(din(v)+1)) + b)
 *   RIPPLE_AGG_GC_SUM, RIPPLE_AGG_GC_MEAN  GraphConv with sum or mean (the
 *                    evaluation's GC-S and GC-M workloads, Sec. VII-A):
 *                    h = sigma(W agg_u h_u + b), no self term; a vertex whose own
 *                    embedding changed is affected at the next hop only through a
 *                    changed in-neighbour or arc
 *   RIPPLE_AGG_GIN   GINConv with sum (GI-S): h = sigma(W2 ReLU(W1 ((1 + eps) h_v
 *                    + sum_u h_u) + b1) + b2)
 *   RIPPLE_AGG_GC_WSUM  GraphConv with weighted sum (GC-W): h = sigma(W sum_u
 *                    alpha_uv h_u + b), alpha_uv the arc's stored weight (each
 *                    message is scaled by the weight of its arc, Sec. IV-C.1)
 *
 * Graph semantics: a simple directed graph on vertices 0..n-1 (int32 ids).
 * Inserting a present arc, deleting an absent arc, and inserting or deleting a
 * self-loop are counted no-ops. A batch has sequential semantics: its net effect
 * is what applying its ops in order leaves (an insert sets an arc present, a
 * delete sets it absent, the last feature write to a vertex wins). On an
 * undirected graph every edge op acts on both arcs u->v and v->u.
 *
 * Conventions for every call:
 *   - Every call returns a ripple_status; nothing else crosses the ABI. On an
 *     error the message is in ripple_last_error(ctx), valid until the next call
 *     on that context.
 *   - Pointer arguments are HOST pointers owned by the caller. The library
 *     copies what it needs during the call and keeps no caller pointer.
 *   - The library owns all device memory (hipMalloc on the context's device).
 *   - Inputs are validated before any state changes: RIPPLE_E_INVALID leaves the
 *     context exactly as it was.
 *   - A HIP runtime error, or a failed device-side consistency check (a deleted
 *     arc missing from its row, a row length mismatch, a compaction wait that
 *     timed out, a row move that would end past its column buffer), poisons the
 *     context: that call returns RIPPLE_E_DEVICE and every
 *     later call except ripple_last_error / ripple_device_bytes / ripple_destroy
 *     returns RIPPLE_E_STATE. For tests of this path, the environment variable
 *     RIPPLE_DEBUG_FAIL_BATCH=k, read by ripple_load_graph, makes the k-th batch
 *     that completes on that context report a failed device-side check (after
 *     all of its kernels have finished normally).
 *   - A context is used by one host thread at a time. Calls are synchronous:
 *     they return after the device work they issued has finished.
 */
#ifndef RIPPLE_H
#define RIPPLE_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#if defined(__GNUC__) || defined(__clang__)
#define RIPPLE_API __attribute__((visibility("default")))
#else
#define RIPPLE_API
#endif

#define RIPPLE_MAX_LAYERS 8
#define RIPPLE_MAX_DIM 1024

typedef struct ripple_ctx ripple_ctx;

typedef enum {
  RIPPLE_OK = 0,
  RIPPLE_E_INVALID = 1, /* bad argument; state unchanged */
  RIPPLE_E_STATE = 2,   /* call out of order (e.g. apply before init) or poisoned context */
  RIPPLE_E_OOM = 3,     /* device allocation failed or would exceed max_device_bytes */
  RIPPLE_E_DEVICE = 4   /* HIP error or device-side check failed; the context is now poisoned */
} ripple_status;

typedef enum {
  RIPPLE_AGG_SUM = 0,     /* GraphSAGE-sum */
  RIPPLE_AGG_MEAN = 1,    /* GraphSAGE-mean */
  RIPPLE_AGG_GCN = 2,     /* GCN, symmetric normalisation, implicit self-loop */
  RIPPLE_AGG_GC_SUM = 3,  /* GraphConv-sum (no self term) */
  RIPPLE_AGG_GC_MEAN = 4, /* GraphConv-mean (no self term) */
  RIPPLE_AGG_GIN = 5,     /* GINConv-sum with a two-layer MLP */
  RIPPLE_AGG_GC_WSUM = 6  /* GraphConv with the arcs' stored weights (a graph loaded with weights) */
} ripple_agg;

typedef enum { RIPPLE_GEMM_FP32 = 0, RIPPLE_GEMM_BF16 = 1 } ripple_gemm_prec;

enum { RIPPLE_OP_INSERT = 1, RIPPLE_OP_DELETE = 2, RIPPLE_OP_FEATURE = 3 };

/* One update (16 bytes). Edge ops: (kind, u, v, -1). Feature replacement:
 * (RIPPLE_OP_FEATURE, u, -1, feat_row): vertex u's features become row feat_row
 * of the batch's feature block. On a graph loaded with weights an insert carries
 * the arc's weight in the last field, (RIPPLE_OP_INSERT, u, v, weight), and an
 * insert of a present arc sets its weight (the last op on an arc fixes both its
 * presence and its weight; an unchanged weight is a no-op). */
typedef struct {
  int32_t kind;
  int32_t u;
  int32_t v;
  union {
    int32_t feat_row;  /* feature ops */
    float weight;      /* inserts on a weighted graph (finite) */
  };
} ripple_op;

/* Graph snapshot (Sec. IV-A: the graph before any update arrives). */
typedef struct {
  int64_t num_vertices;   /* n >= 1; ids are int32 in [0, n) */
  int64_t num_edges;      /* entries in src/dst */
  const int32_t *src;     /* host, [num_edges] */
  const int32_t *dst;     /* host, [num_edges] */
  int32_t undirected;     /* 1: entry (u,v) stands for arcs u->v and v->u */
  float slack;            /* spare slots per adjacency row, as a fraction of its degree (>= 0) */
  int32_t min_slack;      /* spare slots per row at least (>= 0) */
  int32_t device;         /* HIP device ordinal */
  void *stream;           /* hipStream_t to run on, or NULL for a library-owned stream */
  int64_t max_device_bytes; /* 0 = no cap; else allocations beyond it fail with RIPPLE_E_OOM */
  int64_t arena_slots;    /* spare slots per direction for rows that outgrow their own;
                             0 = max(65536, half the laid-out slots). When the arena runs out,
                             the direction is re-laid out (on the device if the fresh layout
                             leaves a quarter of its buffer free, else into larger buffers). */
  const float *weight;    /* [num_edges] arc weights (finite; an undirected edge's weight is both
                             arcs'), or NULL for an unweighted graph. Only RIPPLE_AGG_GC_WSUM uses
                             them; host memory, copied. */
} ripple_graph_desc;

/* Trained model (Sec. IV-A: a trained L-layer GNN with a linear aggregator). */
typedef struct {
  int32_t num_layers;            /* L in [1, RIPPLE_MAX_LAYERS] */
  int32_t agg;                   /* ripple_agg */
  const int32_t *dims;           /* [L+1]: d_0 (feature width) .. d_L, each in [1, RIPPLE_MAX_DIM] */
  const float *const *w_self;    /* [L] row-major [d_l][d_{l-1}]; GraphSAGE only (may be NULL otherwise) */
  const float *const *w_neigh;   /* [L] row-major [d_l][d_{l-1}]; GCN, GraphConv: the single W;
                                    GIN: the MLP's first layer W1 */
  const float *const *bias;      /* [L] [d_l]; NULL array or NULL entry = zero bias (GIN: b1) */
  const int32_t *relu;           /* [L] 1 = ReLU after layer l, 0 = identity */
  int32_t gemm_prec;             /* ripple_gemm_prec. RIPPLE_GEMM_FP32: the transforms' MFMA takes fp32
                                    operands. RIPPLE_GEMM_BF16: it takes bf16 operands (the gathered rows
                                    and the weights rounded to nearest even), accumulating in fp32;
                                    results within about 1e-2 of the fp32 path's. Needs the widths
                                    d_0 .. d_{L-1} (GIN: d_0 .. d_L) to be multiples of 4, else
                                    RIPPLE_E_INVALID. */
  int32_t transform_first;       /* per-layer choice of what the aggregate cache holds (see
                                    ripple_get_aggregates): -1 = for layers with d_l < d_{l-1} when the
                                    graph has at least 2^24 arcs (on smaller graphs the message step is
                                    latency-bound and the extra transform does not pay), 0 = never,
                                    1 = every layer. Results are the same up to rounding. GraphSAGE and
                                    GCN only: GraphConv and GIN models require -1 or 0 (never). */
  const float *const *w_out;     /* GIN: [L] row-major [d_l][d_l], the MLP's second layer W2; else NULL */
  const float *const *b_out;     /* GIN: [L] [d_l] b2; NULL array or NULL entry = zero */
  float gin_eps;                 /* GIN: the own embedding enters as (1 + gin_eps) h_v */
  int32_t reserved;              /* 0 */
} ripple_model_desc;

/* What one ripple_apply_updates call did. Arc counts count directed arcs (an
 * undirected edge is two arcs). */
typedef struct {
  int64_t num_ops;              /* ops in the batch */
  int64_t edge_keys;            /* distinct non-loop edges the batch named */
  int64_t noop_edge_ops;        /* self-loop edge ops + named edges whose state did not change */
  int64_t ins_arcs;             /* net inserted arcs */
  int64_t del_arcs;             /* net deleted arcs */
  int64_t features;             /* vertices whose features were replaced (|A^0|) */
  int64_t dirty[RIPPLE_MAX_LAYERS + 1];     /* [l], l=1..L: vertices whose layer-(l-1) contribution changed */
  int64_t affected[RIPPLE_MAX_LAYERS + 1];  /* [l]: |A^l|, l = 0..L */
  int64_t pushed_arcs[RIPPLE_MAX_LAYERS + 1]; /* [l]: out-arcs of the dirty set pushed at layer l */
  int64_t dest_rows[RIPPLE_MAX_LAYERS + 1];   /* [l]: distinct sinks of those arcs */
  int64_t relocated_rows;       /* adjacency rows moved to the spare arena */
  int64_t repacks;              /* adjacency re-layouts this call needed (spare arena full) */
  int64_t in_arcs[RIPPLE_MAX_LAYERS + 1];   /* [l]: in-arcs of A^l (the pull form's work) */
  int32_t pull_layers;          /* bit l set: layer l pulled over the in-arcs of A^l */
  int32_t dense_layers;         /* bit l set: layer l pulled over every in-arc of the graph */
  int64_t reweighted_arcs;      /* weighted graphs: arcs present before and after whose weight changed */
  int64_t graph_replay;         /* 1: the batch ran as one replay of a captured HIP graph (see
                                   ripple_set_graphs); 0: its kernels were queued one by one */
  int64_t long_rows;            /* adjacency rows of at least 16384 entries whose deletes were swept by
                                   many waves in chunks (graphs whose snapshot has rows of 8192 or more) */
  int32_t recompute_layers;     /* bit l set: layer l recomputed the aggregate rows of A^l from the
                                   current embeddings (re-anchoring; see ripple_set_reanchor) */
  int32_t bucket_layers;        /* bit l set: layer l summed its messages per sink bucket */
} ripple_batch_stats;

/* Part 1 of the problem statement: copies the snapshot to the device as an
 * out-adjacency (CSR) and in-adjacency (CSC) with spare slots per row.
 * Rejects (RIPPLE_E_INVALID) out-of-range ids, self-loops and repeated arcs
 * (for undirected graphs also (u,v) together with (v,u)). On success *out owns
 * a new context; on failure *out is NULL. */
RIPPLE_API ripple_status ripple_load_graph(const ripple_graph_desc *g, ripple_ctx **out);

/* Parts 1-2: uploads features X = H^0 (host [n][d_0] row-major) and the model,
 * then computes H^1..H^L of every vertex layer by layer and caches, per layer,
 * the un-normalised neighbour aggregate that the incremental path updates.
 * May be called again to restart from new features or weights. */
RIPPLE_API ripple_status ripple_init_embeddings(ripple_ctx *ctx, const float *x, const ripple_model_desc *model);

/* Part 3-4: applies one batch (Sec. IV-A batching; Sec. IV-C incremental
 * propagation) and returns when H^0..H^L are updated for every affected vertex.
 * ops: host [num_ops]; feat_rows: host [num_feat_rows][d_0] (may be NULL when
 * there is no feature op). Rejects the whole batch, with no state change, for an
 * unknown op kind, a vertex id outside [0, n), or a feat_row outside
 * [0, num_feat_rows). stats may be NULL. num_ops = 0 is a valid empty batch. */
RIPPLE_API ripple_status ripple_apply_updates(ripple_ctx *ctx, const ripple_op *ops, int64_t num_ops,
                                   const float *feat_rows, int64_t num_feat_rows,
                                   ripple_batch_stats *stats);

/* The same as ripple_apply_updates for a batch already resident in device
 * memory: ops [num_ops] and feat_rows [num_feat_rows][d_0] are DEVICE pointers
 * on the context's device, owned by the caller and only read during the call (no
 * copy through host memory). The batch is checked on the device with the same
 * rules before anything is mutated; a rejected batch returns RIPPLE_E_INVALID
 * naming the first bad op and leaves the state unchanged. Pointers that are not
 * device memory of the context's device are rejected. */
RIPPLE_API ripple_status ripple_apply_updates_device(ripple_ctx *ctx, const ripple_op *ops, int64_t num_ops,
                                                     const float *feat_rows, int64_t num_feat_rows,
                                                     ripple_batch_stats *stats);

/* Part 4: copies rows of H^layer (layer 0 = current features) to host out
 * [count][d_layer]. ids: host [count] vertex ids, or NULL for all n rows in id
 * order (count must then be n). */
RIPPLE_API ripple_status ripple_get_embeddings(ripple_ctx *ctx, int32_t layer, const int32_t *ids,
                                    int64_t count, float *out);

/* ripple_get_embeddings for callers that cannot allocate device memory (code
 * under HIP graph capture, serving loops, harnesses that forbid allocation): the
 * same rows, with the same arguments and errors, staged through a file-scope
 * device array of 32 MiB instead of buffers allocated per call (ripple_get_embeddings
 * allocates two per call with ids). The ids and gathered rows must fit in it:
 * count * 4 bytes (rounded up to 256) + count * d_layer * 4 bytes <= 32 MiB, else
 * RIPPLE_E_INVALID naming the limit. Each GPU the library runs on holds its own
 * copy of the array until the process ends; every call on that GPU, from any
 * context, stages through it, so calls that overlap on one GPU (other threads,
 * other contexts) race and must be serialised by the caller. Allocates nothing:
 * no hipMalloc, hipFree or allocating library routine. */
RIPPLE_API ripple_status ripple_get_embeddings_static(ripple_ctx *ctx, int32_t layer, const int32_t *ids,
                                                      int64_t count, float *out);

/* Trigger output of the last batch: A^layer, the vertices whose layer-`layer`
 * embedding the batch recomputed, in ascending id order (A^0 = vertices whose
 * features were replaced). Writes min(|A^layer|, capacity) ids to `ids` and
 * |A^layer| to *count (always). */
RIPPLE_API ripple_status ripple_get_affected(ripple_ctx *ctx, int32_t layer, int32_t *ids, int64_t capacity,
                                  int64_t *count);

/* The cached aggregate of layer `layer` (1..L) the incremental path maintains:
 * S^l_v = sum over in-neighbours u of c_u h^{l-1}_u, with c_u = 1 (sum, mean)
 * or 1/sqrt(dout(u)+1) (GCN), width d_{l-1}; or, for a layer cached transformed
 * (transform_first), T^l_v = W_neigh^l S^l_v (GCN: W^l S^l_v), width d_l. The
 * messages of such a layer carry W_neigh times the change of the source's row,
 * which is exact by linearity of the aggregators. Host out [count][width]; ids
 * as in ripple_get_embeddings; *width (nullable) receives the row width. For
 * checking only. */
RIPPLE_API ripple_status ripple_get_aggregates(ripple_ctx *ctx, int32_t layer, const int32_t *ids,
                                    int64_t count, float *out, int32_t *width);

/* Copies the current arc set as (src, dst) pairs read from the out-adjacency
 * (direction 0) or the in-adjacency (direction 1), grouped by row in row order.
 * Writes min(arcs, capacity) pairs and the arc count to *count (always). */
RIPPLE_API ripple_status ripple_get_arcs(ripple_ctx *ctx, int32_t direction, int32_t *src, int32_t *dst,
                              int64_t capacity, int64_t *count);

/* Weighted graphs: the arcs' weights in the order ripple_get_arcs lists them
 * (same direction); *count always receives the arc count. RIPPLE_E_INVALID on an
 * unweighted graph. */
RIPPLE_API ripple_status ripple_get_arc_weights(ripple_ctx *ctx, int32_t direction, float *weights, int64_t capacity,
                                                int64_t *count);

/* How each layer adds its messages to the cached aggregate (results agree up to
 * rounding): RIPPLE_SCATTER_PUSH, one row of fp32 atomics per pushed arc;
 * RIPPLE_SCATTER_PULL, each affected vertex sums the messages of its dirty
 * in-neighbours and adds them once; RIPPLE_SCATTER_DENSE, the pull form over every
 * in-arc of the graph, which also finds the sinks (no per-arc marks; for layers
 * where most arcs carry a message); RIPPLE_SCATTER_RECOMPUTE, no messages: each
 * affected vertex's aggregate row is summed afresh over all its in-arcs from the
 * current embeddings (reads only, summed in fp64 and rounded once: the
 * layer-wise recompute of Sec. IV-B, to which the incremental path degrades when
 * a hop covers the graph, Sec. VII-C; it also re-anchors the cached rows);
 * RIPPLE_SCATTER_BUCKET, the pushed arcs sorted by sink (into bins of consecutive
 * sinks, then by sink within each bin) and each sink's bucket summed and added to
 * its row once (the messages of Sec. IV-C.1 combined per sink before they reach
 * the aggregate; the first batch that uses the form allocates 12 bytes per
 * out-arc slot, 20 under the weighted-sum model, a counter per vertex and 258 per
 * bin of 8192 vertices; graphs of at most 2^25 vertices, a batch asking
 * for the form on a larger one fails with RIPPLE_E_INVALID);
 * RIPPLE_SCATTER_AUTO (default), per layer from the previous batch's counts, or
 * for the first batch from an estimate based on the snapshot's degrees. */
enum {
  RIPPLE_SCATTER_AUTO = 0,
  RIPPLE_SCATTER_PUSH = 1,
  RIPPLE_SCATTER_PULL = 2,
  RIPPLE_SCATTER_DENSE = 3,
  RIPPLE_SCATTER_RECOMPUTE = 4,
  RIPPLE_SCATTER_BUCKET = 5
};
RIPPLE_API ripple_status ripple_set_scatter_mode(ripple_ctx *ctx, int32_t mode);

/* Drift budget of the cached aggregates. Messages add fp32 rounding to a cached
 * row every time they reach it; with every = k >= 1, every k-th batch (counted
 * from ripple_init_embeddings) runs each layer in the RIPPLE_SCATTER_RECOMPUTE
 * form, whatever form ripple_set_scatter_mode asks for, so every row that batch
 * affects is recomputed afresh. every = 0: never. Default 256. RIPPLE_E_INVALID
 * for every < 0. */
RIPPLE_API ripple_status ripple_set_reanchor(ripple_ctx *ctx, int64_t every);

/* How a batch's kernels reach the GPU. enable = 1: the first batch of each launch
 * plan (message form and GEMM tile per layer) is captured as a HIP graph on the
 * context's stream and later batches with that plan replay it, so the host
 * thread queues one graph instead of some fifteen kernels. Batch sizes and input
 * pointers are not part of a plan: the first kernel reads them from a pinned block
 * the library fills per call. enable = 0 (default, the lower batch latency on
 * MI355X): every kernel is queued on its own, as are batches that record phase
 * events. A capture that the runtime refuses switches the context to direct
 * launches for good. The same kernels run either way. RIPPLE_E_INVALID for other
 * values. */
RIPPLE_API ripple_status ripple_set_graphs(ripple_ctx *ctx, int32_t enable);

/* Device bytes the context holds. */
RIPPLE_API ripple_status ripple_device_bytes(ripple_ctx *ctx, int64_t *bytes);

/* Kernel timing (for measurement). ripple_set_profiling(ctx, mask) makes every
 * later ripple_apply_updates time each kernel of each phase p whose bit (1 << p)
 * is set in mask: the kernel is launched with a start / stop event pair that takes
 * its own start and end (hipExtLaunchKernelGGL), so the times are kernel
 * durations as a profiler's kernel trace gives them, without the dispatch gaps
 * between kernels. Bit RIPPLE_PHASE_TOTAL instead brackets the whole batch with
 * an event pair on the context's stream (first to last kernel, gaps included).
 * mask 0 stops recording; batches that record run kernel by kernel, never as
 * graph replays. Per phase the library accumulates the milliseconds, kernel
 * launches, and the phase's algorithmic HBM bytes and flops computed from the
 * batch's own counts (each input row read once, each output row written once):
 *   SCATTER, per layer l with dirty set D, pushed arcs E_D, distinct sinks R,
 *            width d = d_{l-1}:  4 E_D + 8 |D| + 4 d |D| + 8 d R  bytes
 *   GEMM,    per layer l with |A^l| rows, K = 2 d_{l-1} (SAGE) or d_{l-1} (GCN),
 *            N = d_l:  flops 2 |A^l| K N; bytes 4 |A^l| K + 4 N K
 *            + 4 |A^l| N (2 if the layer is the last, else 3: old row, new row, delta)
 *   COMPACT, per compaction over n vertices with W = ceil(n/32) bitmap words and
 *            c ids out:  24 W + 4 c bytes
 * Other phases report bytes = flops = 0. ripple_get_phase_stats copies
 * min(capacity, RIPPLE_NUM_PHASES) entries and resets the sums. */
#define RIPPLE_NUM_PHASES 8
enum {
  RIPPLE_PHASE_NET = 0,      /* op netting (hash + membership) */
  RIPPLE_PHASE_TOPO = 1,     /* pre-batch corrections + adjacency update */
  RIPPLE_PHASE_LAYER0 = 2,   /* feature writes and layer-0 deltas */
  RIPPLE_PHASE_SCATTER = 3,  /* delta scatter-add + frontier marking (and listing, for small push
                                frontiers), all layers */
  RIPPLE_PHASE_COMPACT = 4,  /* frontier bitmaps -> sorted lists (pulls, large frontiers), all layers */
  RIPPLE_PHASE_GEMM = 5,     /* gather + transform + epilogue, all layers */
  RIPPLE_PHASE_OTHER = 6,    /* scratch clean-up */
  RIPPLE_PHASE_TOTAL = 7     /* first to last kernel of the batch */
};
typedef struct {
  double ms;
  int64_t launches;
  double bytes;          /* algorithmic bytes: each row the phase needs read or written once */
  double flops;
  double bytes_no_reuse; /* the same work with no on-chip reuse: in the message step every
                            message row is read once per arc that carries it and, in the push
                            form, every arc's row of atomics goes to memory; other phases: bytes */
} ripple_phase_stats;
RIPPLE_API ripple_status ripple_set_profiling(ripple_ctx *ctx, int32_t mask);
RIPPLE_API ripple_status ripple_get_phase_stats(ripple_ctx *ctx, ripple_phase_stats *out, int32_t capacity);
RIPPLE_API const char *ripple_phase_name(int32_t phase);

/* Message of the last failed call on ctx ("" after a success). With ctx NULL:
 * the message of this thread's last failed ripple_load_graph. */
RIPPLE_API const char *ripple_last_error(const ripple_ctx *ctx);

/* Frees the context and its device memory. NULL is a no-op. */
RIPPLE_API void ripple_destroy(ripple_ctx *ctx);

#ifdef __cplusplus
}
#endif

#endif /* RIPPLE_H */
