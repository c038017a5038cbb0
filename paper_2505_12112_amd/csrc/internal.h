// Internal declarations shared by the HIP translation units of libripple.
//
// Device state of one context (all in HBM, fp32 rows row-major, int32 vertex ids):
//   adj[0]  out-adjacency (CSR by source), adj[1] in-adjacency (CSC by sink). Each
//           row u owns slots col[off[u] .. off[u]+cap[u]) of which len[u] are used;
//           rows that outgrow their slots move to a spare arena at the end of col.
//   H[l]    embeddings, l = 0..L (H[0] = features), [n][d_l].
//   S[l]    cached neighbour aggregate of layer l = 1..L, [n][d_{l-1}]:
//           S^l_v = sum_{u in N_in(v)} c_u h^{l-1}_u with c_u = 1, or 1/sqrt(dout(u)+1)
//           under GCN. Mean divides by the in-degree when the row is read.
//   lists[l] sorted vertex lists: lists[0] = dirty set of layer 1, lists[l] = A^l.
//   delta[2] ping-pong [n][max d] rows of c'_u h'_u - c_u h_u aligned with lists[l].
#pragma once

#include <hip/hip_ext.h>
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "ripple.h"

namespace rp {

// Kernel timing for measurement (ripple_set_profiling). While a batch records the
// kernels of a phase, launch_timer hands out a fresh start / stop event pair for
// each launch (and counts it for that phase), and the launch goes through
// hipExtLaunchKernelGGL, whose events take the kernel's own start and end, as a
// profiler's kernel trace does, without the dispatch gap before it. Otherwise it
// returns false and the launch is a plain one.
bool launch_timer(hipEvent_t *start, hipEvent_t *stop);

#define RP_LAUNCH(K, G, B, SHM, S, ...)                                        \
  do {                                                                         \
    hipEvent_t rp_ev_a_, rp_ev_b_;                                             \
    if (::rp::launch_timer(&rp_ev_a_, &rp_ev_b_))                              \
      hipExtLaunchKernelGGL(K, G, B, SHM, S, rp_ev_a_, rp_ev_b_, 0, __VA_ARGS__); \
    else                                                                       \
      hipLaunchKernelGGL(K, G, B, SHM, S, __VA_ARGS__);                        \
  } while (0)

constexpr int kWave = 64;
constexpr int kMaxL = RIPPLE_MAX_LAYERS;
constexpr unsigned long long kEmptyKey = ~0ull;

typedef unsigned long long u64;

// Per-batch device counters, zeroed at the start of every batch.
struct Counters {
  u64 edge_keys;          // distinct non-loop edge keys named by the batch
  u64 noop_edge;          // self-loop edge ops + keys whose state did not change
  u64 n_ins;              // net inserted arcs
  u64 n_del;              // net deleted arcs
  u64 n_feat;             // vertices with a feature write
  u64 abort;              // 1: the spare arena cannot hold this batch; nothing was mutated
  u64 n_reloc;            // rows to move to the arena
  u64 arena_need[2];      // arena slots those moves need, per direction
  u64 err;                // device-side check failed: bit 0 deleted arc not found, bit 1 row length
                          // mismatch, bit 2 compaction wait timed out, bit 3 row move past the buffer
  u64 plan_done;          // blocks of the plan kernel that finished (last one checks the arena)
  u64 count[kMaxL + 1];   // [0] = |dirty set of layer 1|, [l] = |A^l|
  u64 pushed[kMaxL + 1];  // [l] = out-arcs pushed at layer l
  u64 dest[kMaxL + 1];    // [l] = distinct sinks of those arcs
  u64 indeg[kMaxL + 1];   // [l] = sum of in-degrees over A^l (pull work), when computed
  u64 count_all;          // vertices listed by a full compaction (dense layers)
  u64 bad_op;             // B - i for the first op i that failed the device-side check, else 0
  u64 n_rew;              // reweighted arcs (weighted graphs; each also counted in n_ins and n_del)
  u64 zero;               // never written: an arc count of zero for kernels that only mark
  u64 long_rows;          // long rows swept in chunks: count << 40 | chunks handed out
  u64 long_pool;          // pool slots handed out to them
  u64 app[kMaxL + 1];     // [l]: A^l listed by its scatter: count << 40 | sum of out-degrees
  u64 app_sinks[kMaxL + 1];  // [l]: and its distinct sinks << 40 | sum of in-degrees
  u64 maxlen[2];          // per direction: the largest new row length above RewriteBounds::maxlen, else 0
  u64 top_end[2];         // per direction: the arena top after this batch's row moves (0: none moved)
};
constexpr int kAppShift = 40;
constexpr u64 kAppMask = (1ull << kAppShift) - 1;

// Rows at least kLongRow entries long from which a batch deletes entries (and that
// keep their slots) are swept by many waves, kLongChunk entries each: the sweeps
// record the positions of deleted entries below the row's new length (holes) and
// of kept entries at or above it (movers), and a fill pass moves the movers into
// the holes (rows are unordered, so a swap-remove keeps them valid).
constexpr int kLongRow = 16384;
constexpr int kLongChunk = 4096;
struct LongRow {
  int dir, row, len0, k;  // direction, row, pre-batch length, entries deleted
  long long off;          // the row's first slot
  long long chunk0;       // its first chunk number
  long long pool;         // holes at pool[0 .. k), movers at pool[k .. 2k)
  int holes, movers, found;  // filled in by the sweeps (found: deleted entries seen)
  int pad;
};

// One batch's inputs as the host hands them over. The first kernel of the batch
// takes them as an argument, or, in a launch captured for replay, reads them from
// pinned host memory written before each replay (system scope, so a replay sees
// the new values); it keeps a device copy for the later kernels. Every other
// launch of a batch is therefore the same for batches of any size up to the
// scratch capacity, which lets a batch be replayed as one graph.
struct BatchIn {
  const ripple_op *ops;    // pinned host or device memory
  const float *feat;       // feature rows, [num_feat_rows][d_0], pinned host or device memory
  long long num_ops;
  long long num_feat_rows;
};

// Survives batches.
struct Persist {
  u64 top[2];             // next free arena slot per direction
};

struct Adj {
  long long *off;
  int *len;
  int *cap;
  int *col;
  float *wt;              // weighted graphs: the weight of the arc in each slot of col; else nullptr
  int *inscnt;            // per-row scratch, zero between batches
  int *delcnt;
};

// Per layer l = 1..L: the rows whose contributions the aggregate S[l] sums
// (src[l], width sw[l]): H[l-1] for a plain layer, or the cached P = W_neigh
// H[l-1] (width d_l) for a transform-first layer.
struct LayerPtrs {
  const float *src[kMaxL + 1];
  float *S[kMaxL + 1];
  int sw[kMaxL + 1];
  int L;
};

// True if the batch aborted (ab = its abort flag). The counts a kernel loads with
// the flag join the test (callers pass only values that cannot be negative, so
// they never change its outcome):
// then every one of those loads is issued before the branch and the kernel waits
// for them once, instead of waiting for the flag before it loads the rest.
template <typename... T>
__device__ inline bool aborted_with(u64 ab, T... counts) {
  return (ab | static_cast<u64>((static_cast<long long>(counts) | ... | 0LL)) >> 63) != 0;
}

// The per-batch scratch a batch touched, reset by its last kernel (see
// batch_cleanup).
struct CleanupArgs {
  const BatchIn *in;  // device copy of the batch's inputs
  const ripple_op *ops;
  const int *op_slot;
  u64 *ht_key;
  int *ht_val;
  int *ht_net;
  int *fop;
  int *out_inscnt, *out_delcnt, *in_inscnt, *in_delcnt;
  const int *ins_src, *ins_dst, *del_src, *del_dst;
  int *ddeg;
  const int *flist;   // the batch's feature-written vertices (A^0), n_feat of them
  int *flist_done;    // A^0 of the last batch that completed: flist is copied here unless the batch aborted
  const Counters *c;  // this batch's counters, copied to host
  Counters *next;     // the other counter buffer, zeroed for the next batch
  Counters *host;     // pinned
};

// Resets every per-batch scratch word the batch touched (also after an abort),
// copies the batch's counters to pinned host memory and clears the other counter
// buffer. A batch that did not abort also leaves its A^0 in flist_done, so a
// rejected batch (whose netting rewrote flist) cannot change the sets that the
// last completed batch returns. Thread t of `threads` (t = 0 also copies the counters, with the rest of
// its block: block is the calling block's index among the cleanup blocks). Runs in
// the batch's last kernel beside work that reads none of this scratch.
__device__ inline void batch_cleanup(const CleanupArgs &a, int block, long long t0, long long threads) {
  if (block == 0) {
    constexpr int words = static_cast<int>(sizeof(Counters) / sizeof(u64));
    const u64 *src = reinterpret_cast<const u64 *>(a.c);
    u64 *dst = reinterpret_cast<u64 *>(a.host);
    u64 *nxt = reinterpret_cast<u64 *>(a.next);
    for (int w = threadIdx.x; w < words; w += blockDim.x) {
      dst[w] = src[w];
      nxt[w] = 0ull;
    }
  }
  // item w = 2 * arc + direction (0: the source's out-row, 1: the sink's in-row)
  const long long ni = 2 * static_cast<long long>(a.c->n_ins);
  const long long nd = 2 * static_cast<long long>(a.c->n_del);
  const long long B = a.in->num_ops;
  for (long long w = t0; w < ni; w += threads) {
    if (w & 1) {
      a.in_inscnt[a.ins_dst[w >> 1]] = 0;
    } else {
      const int u = a.ins_src[w >> 1];
      a.out_inscnt[u] = 0;
      a.ddeg[u] = 0;
    }
  }
  for (long long w = t0; w < nd; w += threads) {
    if (w & 1) {
      a.in_delcnt[a.del_dst[w >> 1]] = 0;
    } else {
      const int u = a.del_src[w >> 1];
      a.out_delcnt[u] = 0;
      a.ddeg[u] = 0;
    }
  }
  if (a.c->abort == 0) {
    const long long nf = static_cast<long long>(a.c->n_feat);
    for (long long i = t0; i < nf; i += threads) a.flist_done[i] = a.flist[i];
  }
  for (long long i = t0; i < B; i += threads) {
    const int s = a.op_slot[i];
    if (s >= 0) {
      a.ht_key[s] = kEmptyKey;
      a.ht_val[s] = -1;
      a.ht_net[s] = 0;
    }
    if (a.ops[i].kind == RIPPLE_OP_FEATURE) a.fop[a.ops[i].u] = -1;
  }
}

// Same values as ripple_agg. GraphConv (kGcSum, kGcMean) has no self term; GIN's
// update is a two-layer MLP on (1 + eps) h_v + S_v.
// kGcWsum: GraphConv with the arcs' stored weights (weighted graphs).
enum Agg { kSum = 0, kMean = 1, kGcn = 2, kGcSum = 3, kGcMean = 4, kGin = 5, kGcWsum = 6 };
inline bool has_self_term(int agg) { return agg != kGcSum && agg != kGcMean && agg != kGcWsum; }

// --- launchers (each defined in the translation unit that holds its kernel) ---

// netting: after these, the net arcs are listed and every (arc, direction) item
// knows its rank among the row's inserts (ins_rank) or deletes (del_rank); the
// hash slot of every named edge holds +1 (net insert), -1 (net delete) or 0.
// The batch's inputs are `now`, or, when host_in (pinned host memory) is set,
// whatever it holds when the kernel runs (graph replays); dev_in receives a copy
// for the later kernels. The ops are copied to ops (device) on the way and
// checked (ids and feature rows in range, known kind, finite insert weights on a
// weighted graph): a failing op sets bad_op and abort, and is copied as a
// self-loop no-op. On a weighted graph (out.wt set) an insert of a present arc
// with another weight is a reweight: listed as a delete (old weight, del_w) and an
// insert (new weight, ins_w) of the same arc, counted in n_rew.
// cap_ops bounds num_ops (the grids are sized for it).
void launch_net_hash(hipStream_t s, int cap_ops, const BatchIn *host_in, const BatchIn &now, BatchIn *dev_in,
                     ripple_op *ops,
                     int undirected, int weighted, long long n, u64 *ht_key, int *ht_val, unsigned mask, int *op_slot,
                     int *fop, Counters *c);
// Both netting steps in one launch, for a batch of at most kNetDirectMax ops: the
// same outputs, except that only net-deleted edge keys enter the hash table (tagged
// -1, their slots in op_slot; every other op's op_slot is -1) and ht_val is unused.
constexpr int kNetDirectMax = 1024;
void launch_net_direct(hipStream_t s, int cap_ops, const BatchIn *host_in, const BatchIn &now, BatchIn *dev_in,
                       ripple_op *ops, int undirected, int weighted, long long n, u64 *ht_key, int *ht_net,
                       unsigned mask, int *op_slot, int *fop, Adj out, Adj in_adj, int *ins_src, int *ins_dst,
                       int *del_src, int *del_dst, int *ins_rank, int *del_rank, float *ins_w, float *del_w,
                       int *flist, int *frow, Counters *c);
void launch_net_decide(hipStream_t s, int cap_ops, const BatchIn *in, const ripple_op *ops, int undirected,
                       const int *ht_val, int *ht_net, const int *op_slot, const int *fop, Adj out, Adj in_adj,
                       int *ins_src, int *ins_dst, int *del_src, int *del_dst, int *ins_rank, int *del_rank,
                       float *ins_w, float *del_w, int *flist, int *frow, Counters *c);

// topology (cap_arcs bounds n_ins and n_del): plan row moves and check the arena
// (aborting before any mutation), then one owner wave per touched row removes its
// deleted entries, moves the row if it must grow, and sets its new length (the
// inserts are written at their ranks by launch_corr_mark).
// long_ok: rows may be long (tab / pool hold up to 2 cap_arcs rows / 4 cap_arcs
// slots); then the plan lists the long rows, the rewrite's waves also sweep their
// chunks, and launch_topo_fill must follow the rewrite.
void launch_topo_plan(hipStream_t s, int cap_arcs, Adj out, Adj in, const int *ins_src, const int *ins_dst,
                      const int *del_src, const int *del_dst, const int *ins_rank, const int *del_rank,
                      int long_ok, LongRow *tab, Counters *c, const Persist *p, long long cap_out, long long cap_in);
// The host's view of the adjacency for the rewrite: per direction, a bound on every
// row's length (rows that grow past it report their new length in Counters::maxlen)
// and the column buffer's size (a row move that would end past it sets check bit 3
// and writes nothing).
struct RewriteBounds {
  long long maxlen[2];
  long long capacity[2];
};
void launch_topo_rewrite(hipStream_t s, int cap_arcs, int undirected, long long n, Adj out, Adj in,
                         const int *ins_src, const int *ins_dst, const int *del_src, const int *del_dst,
                         const int *ins_rank, const int *del_rank, const u64 *ht_key, const int *ht_net,
                         unsigned mask, Persist *p, int *ddeg, int long_ok, LongRow *tab, int *pool, Counters *c,
                         const RewriteBounds &rb);
void launch_topo_fill(hipStream_t s, int cap_arcs, Adj out, Adj in, const LongRow *tab, const int *pool,
                      Counters *c);

// frontier. Pre-batch corrections of every layer's aggregate (an inserted arc
// (u,v) adds u's pre-batch contribution to S^l_v, a deleted one removes it) run
// after the adjacency update, with pre-batch coefficients recovered from ddeg;
// the same kernel marks the layer-1 dirty set (feature writes; GCN: vertices whose
// out-degree changed) and writes every inserted arc into the slot of its row given
// by its rank among the row's inserts (with arc_w[arc], the slot's weight, when
// the adjacency keeps weights).
// ins_w / del_w (nullable): the arcs' weights as the corrections use them
// (weighted-sum model).
// direct.list != nullptr: the layer-1 dirty set is the feature-written vertices
// alone (no GCN term; flist holds each once) and at most kDirectListMax of them.
// Then they are not marked: the kernel lists them itself, in flist's order, with
// their out-degree prefix (the compaction's list, doff, count and out_total
// outputs; a larger count sets check bit 2).
// direct.delta != nullptr as well: it also writes their layer-0 deltas (x' - x at
// list position j, row stride ld) and stages x' at row j of stage (stride ld);
// X keeps x, which the corrections read, until the layer-1 scatter copies the
// staged rows in (ScatterCopy).
constexpr int kDirectListMax = 1024;
struct DirectList {
  int *list;
  long long *doff;
  u64 *count;
  u64 *out_total;
  float *delta;
  float *stage;
  int ld;
  int d0;
  const float *X;
  const int *frow;  // feature row of each listed vertex (flist order)
  const BatchIn *in;
};
// Rows the layer-1 scatter copies after the direct listing: X[list[j]] = stage[j]
// for every listed j (dst == nullptr: none).
struct ScatterCopy {
  float *dst;
  const float *stage;
  int d;
  int ld;
};
void launch_corr_mark(hipStream_t s, int cap_feat, int cap_arcs, int agg, LayerPtrs lp, Adj out, Adj in,
                      const int *ins_rank, const float *arc_w, const int *ddeg, const int *flist, const int *ins_src,
                      const int *ins_dst, const int *del_src, const int *del_dst, const float *ins_w,
                      const float *del_w, unsigned *bm, Counters *c, const DirectList &direct);
int compact_blocks(long long n);
// Entries of the bucket form's counter array for n vertices: every vertex of every
// compaction tile (the compaction reads whole tiles of counters).
long long bucket_counter_slots(long long n);
// Outputs of one compaction of bitmaps (a | b) into an ascending list. Optional
// (nullptr = skipped): list, doff[j] = sum of out_deg over list[0..j) (doff[count]
// = total), ioff likewise over in_deg, memb[w] = (the compacted bitmap word w,
// listed vertices in words before w), so the list position of a member u is
// memb[u / 32].y + the member bits of its word below u, and one 8-byte load
// answers both questions. Both input bitmaps are cleared. full_n > 0: list all of 0..full_n-1 instead (the bitmaps are not read).
struct CompactOut {
  long long full_n;
  int *list;
  u64 *count;
  const int *out_deg;
  long long *doff;
  const int *in_deg;
  long long *ioff;
  u64 *in_total;       // receives the sum of in_deg over the list
  u64 *out_total;      // receives the sum of out_deg over the list (the next scatter's arcs)
  u64 *sinks_a;        // receives the number of bits set in the first bitmap
  uint2 *memb;
  // zero_rows (nullable, with ioff): rows zero_w floats wide of every listed vertex
  // whose in-degree exceeds kRecomputeSeg are zeroed (the recompute form adds such
  // rows up from several segments)
  float *zero_rows;
  int zero_w;
  // bucket form (all three set, or none): a vertex with bkt_cnt[v] > 0 counts as
  // marked in the first bitmap (the sinks are not marked there); boff receives the
  // prefix of bkt_cnt over the list (boff[count] = the total), and bkt_start[v] the
  // start of v's bucket for every listed v with bkt_cnt[v] > 0 (bkt_start may alias
  // bkt_cnt: each count is read before its start is written over it)
  const int *bkt_cnt;
  long long *boff;
  int *bkt_start;
};
// Floats allocated past the last row of every row table (H, S, P, the delta and
// message rows). Kernels that gather rows with lane groups read a group's whole
// span (up to 1024 floats) from each row start, masking the columns past the row's
// width afterwards, so that every lane's offsets are compile-time immediates;
// the tail keeps those reads inside the allocation for the table's last row.
constexpr long long kRowTail = 1024;
// The recompute form (launch_recompute) sums an in-row of more than kRecomputeSeg
// arcs in segments of that many, each added to the row with fp32 atomics.
constexpr int kRecomputeSeg = 64;
// Tile sums published by the single-pass compaction: compact_scratch_words(n)
// words, zero when first used, then owned by the compactions of one vertex count
// (each launch finds its epoch from a ticket counter kept there).
struct CompactScratch {
  u64 *words;
  u64 *err;  // bit 2 set if a wait for a predecessor tile timed out
};
long long compact_scratch_words(long long n);
// Layer-0 deltas of the listed (dirty) vertices u at list position j:
// delta[j] = c'_u x'_u - c_u x_u (c = 1, or 1/sqrt(dout+1) post/pre batch under
// GCN), where x'_u is u's last feature row of the batch (in->feat, which may be
// pinned host memory, row ops[fop[u]].feat_row) or x_u when u has none; then
// X[u] = x'_u. Skipped when the batch aborted.
struct Delta0Args {
  int agg;
  int d0;
  int ld;  // row stride of delta (floats)
  const ripple_op *ops;
  const BatchIn *in;
  const int *fop;
  float *X;
  const int *out_len;
  const int *ddeg;
  float *delta;
  const Counters *c;
};
// Compacts bm_a | bm_b (both cleared) into o. in_total / out_total (nullable)
// receive the degree sums over the list even when the prefix arrays are not wanted.
void launch_compact(hipStream_t s, long long n, unsigned *bm_a, unsigned *bm_b, const CompactScratch &cs,
                    const CompactOut &o);
// The layer-0 deltas of list[0 .. *count) (n bounds the count).
void launch_delta0(hipStream_t s, long long n, const Delta0Args &z, const int *list, const u64 *count);

// scatter: S^l[v] += delta[j] for every post-batch out-arc (list[j] -> v) (doff
// gives each listed vertex's first arc); marks the sinks in bm_out, and the
// listed vertices and the sinks of net arcs in bm_x. With push = false it only
// marks (the pull kernel then adds the messages).
// pushed = the number of arcs to push (the out-degree sum over the list, written
// by the compaction that built the list).
// mark_list: also mark the listed (dirty) vertices themselves in bm_x (models with
// a self term).
// A^l listed by the push scatter itself (list != nullptr), for a layer whose list
// needs no order and no membership words: the first wave to set a vertex's bit in
// bm_x (every mark also goes there) appends it to list at a position taken with
// one 64-bit atomic on *app (count << kAppShift | out-degree sum), which also gives
// its doff entry (doff nullable: not wanted). Sinks are marked in bm_out as well;
// *sinks receives the distinct sinks (first setters of a bit there) << kAppShift |
// the members' in-degree sum. The bitmaps stay set; the next transform of the list
// clears them (GemmArgs::clear_a / clear_b).
struct ScatterList {
  int *list;
  long long *doff;
  u64 *app;
  u64 *sinks;
  const int *out_len;
  const int *in_len;
};
// packed_in: count points at a scatter-built list's packed counter (count and arc
// total in one word; pushed is then not read).
// The bucket form's arrays. The pushed arcs are sorted by sink in two levels:
// into bins of 2^shift consecutive sinks (nbins bins), then by sink within each
// bin. cnt: a counter per vertex (bucket_counter_slots(n) of them, zero between
// batches); bin_total, bin_base: per bin its arc count (zero between batches) and
// its first slot; block_off: per counting block and bin the block's place in the
// bin; tv, tj, tw: the arcs grouped by bin (sink, source list position, weight);
// idx, wt: the same grouped by sink, each sink's bucket contiguous and the buckets
// in vertex order. Slots number the pushed arcs (fewer than 2^31); tw and wt only
// under the weighted-sum model, else null.
struct Buckets {
  int *cnt;
  int *bin_total;
  int *bin_base;
  int *block_off;
  int *tv;
  int *tj;
  float *tw;
  int *idx;
  float *wt;
  int shift;
  int nbins;
};
// the counting and scatter passes' grid (blocks of kBinThreads threads; per block
// and bin one atomic), and the most bins (one counter each per block in LDS)
constexpr int kBinBlocks = 256, kBinThreads = 1024, kMaxBins = 4096;
// log2 of the sinks per bin for n vertices (bins of 8192 sinks, at most kMaxBins
// bins); -1 when n needs more (the bucket form then is not available)
int bin_shift(long long n);
void launch_scatter(hipStream_t s, long long n, int d, int ld, const int *list, const u64 *count, const long long *doff,
                    const float *delta, Adj out, float *S, unsigned *bm_out, unsigned *bm_x, const int *ins_dst,
                    const int *del_dst, const u64 *pushed, const Counters *c, bool push, bool mark_list,
                    const ScatterCopy &copy = ScatterCopy{}, const ScatterList &lo = ScatterList{},
                    bool packed_in = false);
// bucket counting pass (in place of the marks-only scatter): marks the net arcs'
// heads and, with mark_list, the list in bm_x; counts the arcs pushed from the
// sorted list (numbered as the scatter numbers them) per bin and adds the counts
// to b.bin_total, recording each block's place in b.block_off. Sinks are not
// marked (the compaction finds them from the counts k_bin_sort leaves in b.cnt).
void launch_bin_count(hipStream_t s, const int *list, const u64 *count, const long long *doff, Adj out,
                      const u64 *pushed, const Buckets &b, unsigned *bm_x, const int *ins_dst, const int *del_dst,
                      bool mark_list, const Counters *c);
// bucket scatter pass: the same arcs, in the same blocks, into their bins (b.tv,
// b.tj, b.tw from each bin's first slot, stored in b.bin_base).
void launch_bin_scatter(hipStream_t s, const int *list, const u64 *count, const long long *doff, Adj out,
                        const u64 *pushed, const Buckets &b, const Counters *c);
// bucket sort within the bins: per sink its count into b.cnt (for the compaction)
// and its arcs' source positions (and weights) into its bucket in b.idx (b.wt);
// the bins' totals back to zero. n: vertices.
void launch_bin_sort(hipStream_t s, long long n, const u64 *pushed, const Buckets &b, const Counters *c);

// pull: for every vertex v of the sorted list A (in-arc prefix ioff; list null =
// the identity), S[v] += sum of msg[rank(u)] over in-arcs (u -> v) whose source u
// is a member by memb, its rank from memb too (see CompactOut). One flush (row of fp32
// atomics) per sink and lane group; each in-arc is read once. mark (nullable):
// set the bit of every sink that received a message (the dense form's frontier).
void launch_pull_msgs(hipStream_t s, long long n, int d, int ld, const int *list, const u64 *count, const long long *ioff,
                      Adj in, const uint2 *memb, const float *msg, float *S, unsigned *mark, const Counters *c);

// recompute (re-anchoring) form of the message step: for every vertex v of the
// sorted list A (in-arc prefix ioff), S[v] = sum over in-arcs (u -> v) of c'_u
// src[u] (c' = 1, or 1/sqrt(dout'(u)+1) under GCN, times the arc's weight when
// in.wt is set), with the post-batch graph and the current source rows: reads
// only, summed in fp64 and rounded once, a plain store per row. Rows of more than
// kRecomputeSeg in-arcs are summed in segments added with fp32 atomics (the
// compaction that listed A zeroed them, see CompactOut::zero_rows). d is the row
// width of src and S.
void launch_recompute(hipStream_t s, long long n, int d, int gcn, const int *list, const u64 *count,
                      const long long *ioff, Adj in, const int *out_len, const float *src, float *S, const Counters *c);
// The bucket form's sums, with the recompute's work split: for every vertex v of
// the sorted list A (bucket-slot prefix boff), S[v] += the sum over its bucket's
// slots e of bk.wt[e] (or 1) times message row bk.idx[e] of msg (row stride ld), in
// fp32; a bucket of at most kRecomputeSeg slots is added with a plain load and
// store, longer ones in segments with fp32 atomics. Each sink's counter bk.cnt[v]
// is reset to zero.
void launch_bucket_sum(hipStream_t s, int d, int ld, const int *list, const u64 *count, const long long *boff,
                       const Buckets &bk, const float *msg, float *S, const Counters *c);

// bootstrap pull: S[v] = sum over in-arcs c_u H[u]
void launch_pull(hipStream_t s, long long n, int d, int agg, const float *Hprev, Adj in, const int *out_len,
                 float *S);

// transform: for rows r < M (M = *count or count_fixed), v = rows ? rows[r] : r:
//   y = act(W [h_v || t_v S_v] + b)      (SAGE; t_v = 1 or 1/din(v))
//   y = act(W t_v (S_v + s_v h_v) + b)   (GCN; t_v = 1/sqrt(din+1), s_v = 1/sqrt(dout+1))
// then, when delta != nullptr, delta[r] = c'_v y - c_v H[v] (c = 1, or s_v post/pre
// batch under GCN), and H[v] = y.
// mode kLayer: the layer as above. kTransformFirst: S holds T = W_neigh S (width
// N), Z = h_v (K = dprev), W = W_self (SAGE) or W (GCN), and the epilogue adds
// t_v T_v (SAGE) or forms t_v (T_v + s_v y) (GCN). kPlain: y = h_v W^T (K =
// dprev); with bias nullptr and relu 0 this computes the rows P_v = W_neigh h_v a
// transform-first layer caches (H = P) and, with delta set, their messages
// c'_v P'_v - c_v P_v.
// GraphConv layers (agg kGcSum / kGcMean) use kLayer with Z = t_v S_v (K = dprev).
// GIN layers run two GEMMs: kGin1, Z = S_v + eps1 h_v (K = dprev), y = ReLU(Z W1^T
// + b1) written to H[m] (a row buffer indexed by list position, no delta); then
// kGin2, Z = Hprev[m] (that buffer, K = dprev = its width), the epilogue of kLayer.
enum GemmMode { kLayer = 0, kTransformFirst = 1, kPlain = 2, kGin1 = 3, kGin2 = 4 };
// Row stride (floats) of message and delta rows of width w: rows start on 64-byte
// boundaries, so a row read touches the fewest memory segments.
inline int row_ld(int w) { return (w + 15) / 16 * 16; }

struct GemmArgs {
  int mode;
  const int *rows;
  const u64 *count;
  long long count_fixed;
  const float *Hprev;
  int dprev;
  const float *S;
  const int *in_len;
  const int *out_len;
  const int *ddeg;
  const float *W;   // [N][K]
  const unsigned short *Wb;  // bf16 transforms: W rounded to bf16 (RN-even) as raw bits, [N][K]
  int bf16;         // 1: the MFMA takes bf16 operands (rounded RN-even at the gather), fp32 accumulation
  int K;
  int N;
  const float *bias;
  int relu;
  float *H;
  float *delta;
  int dld;  // row stride of delta (floats)
  int agg;
  const u64 *abort;
  float eps1;  // GIN: 1 + eps
  // cleanup_blocks > 0: the launch has that many extra blocks which run
  // batch_cleanup(cleanup) instead (the batch's last GEMM)
  int cleanup_blocks;
  CleanupArgs cleanup;
  long long max_rows;  // rows (list entries) the launch may read; set by launch_gemm
  int count_shift;     // the row count is *count >> count_shift (a scatter's packed list counter)
  // clear_a / clear_b (nullable): bitmaps whose words holding a listed row are
  // zeroed (a scatter-built list leaves its marks for the next transform to clear)
  unsigned *clear_a, *clear_b;
};
// Blocks a batch's clean-up takes for cap_ops ops.
int cleanup_blocks_for(long long cap_ops);
// expected_rows picks the kernel: 0 = 16-row tiles split over eight waves (short
// lists), 2 = the same over four waves, 1 = 128-row tiles (many rows);
// gemm_variant(expected_rows, N) names the choice (launches with the same variant
// and arguments are the same launch).
void launch_gemm(hipStream_t s, const GemmArgs &a, long long max_rows, long long expected_rows);
int gemm_variant(long long expected_rows, int n_cols);

// re-layout of one adjacency direction
// old_wt / new_wt (nullable): the slots' weights move with them.
void launch_repack_copy(hipStream_t s, long long n, const int *old_col, const long long *old_off, const int *len,
                        int *new_col, const long long *new_off, const float *old_wt, float *new_wt);

// Device-side re-layout of one direction. relayout_sums leaves in blocksums[nb]
// (nb = relayout_blocks(n)) the total slots a fresh layout needs (len + spare
// slots per row); once the caller has checked that total + arena fits new_col,
// relayout_apply writes the new offsets/capacities (scratch new_off[n],
// new_cap[n]), copies the rows into new_col, installs the row table and sets the
// arena top. The caller then swaps a.col and new_col.
int relayout_blocks(long long n);
void launch_relayout_sums(hipStream_t s, long long n, float slack, int min_slack, const int *len,
                          long long *blocksums);
void launch_relayout_apply(hipStream_t s, long long n, float slack, int min_slack, Adj a, int *new_col,
                           float *new_wt, const long long *blocksums, long long *new_off, int *new_cap, u64 *top);

// utilities
void launch_fill_i32(hipStream_t s, int *p, long long count, int value);
void launch_fill_u64(hipStream_t s, u64 *p, long long count, u64 value);
void launch_gather_rows(hipStream_t s, const float *src, int d, const int *ids, long long count, float *out);

}  // namespace rp
