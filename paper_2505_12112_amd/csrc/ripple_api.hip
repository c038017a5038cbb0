// Host side of libripple: the context, argument validation, the adjacency build,
// the bootstrap forward pass and the per-batch kernel pipeline.
//
// Batch pipeline (one stream, counts stay on the device, one host sync at the end):
//   net:     hash ops, decide winners against the pre-batch adjacency, count
//            per-row inserts/deletes
//   topo:    plan arena moves and check the arena, then per touched row: deletes,
//            row move, new length
//   layer 0: inserts into their slots, pre-batch corrections of every layer's
//            aggregate, mark the dirty set (feature writes; GCN: out-degree
//            changes), compact, form layer-0 deltas and write the new feature rows
//   layer l: scatter deltas along post-batch out-arcs + mark A^l, compact A^l,
//            gather + MFMA transform + epilogue (new rows, next deltas)
//   cleanup: reset per-batch scratch
// An aborted batch (arena too small) changes nothing; the host re-lays the
// adjacency out with fresh spare slots and runs the batch again.
// Every launch of a batch depends only on its plan (message form and GEMM tile
// per layer, counter parity): the batch's own sizes and input pointers reach the
// kernels through a pinned block the first kernel reads. So a batch can be
// captured once per plan as a HIP graph and later batches with that plan replay
// it (ripple_set_graphs), which takes the queueing of some fifteen dependent
// kernels off the host thread.
#include <algorithm>
#include <limits>
#include <chrono>
#include <cmath>
#include <cstdio>
#include <cstdlib>
#include <cstring>
#include <mutex>
#include <numeric>
#include <string>
#include <thread>
#include <unordered_map>
#include <vector>

#include "internal.h"

using rp::u64;

namespace {

// Batches between two re-anchoring batches by default (see ripple_set_reanchor).
constexpr long long kDefaultReanchor = 256;

struct PhaseEv {
  int phase;
  hipEvent_t a;
  hipEvent_t b;
};

// One captured batch: the executable graph of the plan with this key.
struct GraphSlot {
  unsigned long long key;
  unsigned long long key2;
  hipGraphExec_t exec;
  unsigned long long used;  // last use, for eviction
};

}  // namespace

struct ripple_ctx {
  int device = 0;
  hipStream_t stream = nullptr;
  bool own_stream = false;
  long long n = 0;
  int undirected = 0;
  float slack = 0.25f;
  int min_slack = 4;
  long long max_bytes = 0;
  long long arena_slots = 0;  // 0 = default sizing
  long long arcs_loaded = 0;  // arcs of the snapshot
  long long arcs_now = 0;     // arcs stored now (snapshot + net inserts - net deletes)
  std::vector<std::pair<uintptr_t, uintptr_t>> dev_ranges;  // device allocations seen by apply_updates_device
  long long bytes = 0;
  std::unordered_map<void *, size_t> allocs;
  std::string err;
  bool poisoned = false;
  bool inited = false;
  // test hook (RIPPLE_DEBUG_FAIL_BATCH=k, read by ripple_load_graph): the k-th batch
  // that completes on the device reports a failed device-side check (err bit 4),
  // set in the host copy of its counters after every kernel has exited normally
  long long debug_fail_batch = 0;
  long long batches_checked = 0;

  // adjacency: [0] out (CSR by source), [1] in (CSC by sink)
  rp::Adj adj[2] = {};
  long long col_capacity[2] = {0, 0};
  long long row_max[2] = {0, 0};     // per direction: no row is longer
  long long arena_top[2] = {0, 0};   // per direction: first free arena slot (as of the last batch)
  int *col_alt[2] = {nullptr, nullptr};   // spare column buffer per direction (same capacity)
  float *wt_alt[2] = {nullptr, nullptr};  // weighted graphs: the spare buffer of the slots' weights
  bool weighted = false;                  // the arcs carry weights
  long long *rl_blocksums = nullptr;      // re-layout scratch
  long long *rl_off = nullptr;
  int *rl_cap = nullptr;

  // model
  int L = 0, agg = 0;
  int dims[rp::kMaxL + 1] = {};
  int relu[rp::kMaxL] = {};
  int K[rp::kMaxL] = {};
  float *W[rp::kMaxL] = {};     // main transform [d_l][K]
  float *Wn[rp::kMaxL] = {};    // transform-first layers: W_neigh [d_l][d_{l-1}] (GCN: W)
  float *P[rp::kMaxL + 1] = {};  // [l], transform-first layers: P = W_neigh H^{l-1}, [n][d_l]
  float *bias[rp::kMaxL] = {};
  // bf16 transforms (gemm_prec RIPPLE_GEMM_BF16): the same matrices rounded to bf16
  bool gemm_bf16 = false;
  unsigned short *Wb[rp::kMaxL] = {};
  unsigned short *Wnb[rp::kMaxL] = {};
  unsigned short *W2b[rp::kMaxL] = {};
  float *W2[rp::kMaxL] = {};     // GIN: the MLP's second layer [d_l][d_l]
  float *b2[rp::kMaxL] = {};
  float gin_eps1 = 1.0f;         // GIN: 1 + eps
  float *gin_rows = nullptr;     // GIN: the MLP's hidden rows, one per list position [n][max d_l]
  int tf[rp::kMaxL + 1] = {};   // [l]: layer l caches T = W_neigh S (width d_l)
  int sw[rp::kMaxL + 1] = {};   // [l]: width of the cached aggregate rows
  float *msg = nullptr;         // [n][max d_l of transform-first layers]: message rows
  float *H[rp::kMaxL + 1] = {};
  float *S[rp::kMaxL + 1] = {};
  int dmax_delta = 0;

  // persistent scratch (n-sized)
  int *fop = nullptr;
  int *ddeg = nullptr;
  unsigned *bm_out = nullptr;
  unsigned *bm_x = nullptr;
  rp::u64 *compact_lb = nullptr;  // tile sums of the single-pass compaction
  int *lists[rp::kMaxL + 1] = {};
  long long *doff[rp::kMaxL + 1] = {};  // out-degree prefix of lists[l] (first arc index per vertex)
  long long *ioff = nullptr;            // in-degree prefix of the current layer's A^l (pull form)
  // per bitmap word of lists[k], k = 0, 1 mod 2: (member bits, members before the
  // word); the pull form's membership test and message row in one load
  uint2 *memb[2] = {nullptr, nullptr};
  int scatter_mode = RIPPLE_SCATTER_AUTO;
  // drift budget: every reanchor_every-th batch recomputes each layer's aggregate
  // rows of A^l from the current embeddings (0: never)
  long long reanchor_every = kDefaultReanchor;
  long long batches_done = 0;  // batches completed since the model was set up
  // snapshot degrees, kept to plan the first batch (no earlier batch's counts exist)
  std::vector<int> snap_out, snap_in;
  const ripple_op *plan_ops = nullptr;  // host copy of the first batch's ops, for its plan
  std::vector<ripple_op> plan_buf;
  long long last_pushed[rp::kMaxL + 1] = {};
  long long last_in[rp::kMaxL + 1] = {};
  int last_pull = 0;   // layers that pulled over A^l's in-arcs (bit l)
  int last_dense = 0;  // layers that pulled over every in-arc (bit l)
  int last_recompute = 0;  // layers whose aggregate rows of A^l were recomputed (bit l)
  int last_bucket = 0;     // layers that summed their messages per sink bucket (bit l)
  int last_app = 0;    // layers whose A^l its scatter listed, unordered (bit l), as of the last completed batch
  int run_app = 0;     // the same for the batch in flight (it becomes last_app once that batch completes)
  float *delta[2] = {nullptr, nullptr};
  rp::Counters *d_counters = nullptr;  // two buffers; batch parity picks one
  int parity = 0;
  rp::Persist *d_persist = nullptr;
  rp::Counters *h_counters = nullptr;  // pinned
  rp::BatchIn *h_in = nullptr;         // pinned: the batch's sizes and input pointers
  rp::BatchIn *d_in = nullptr;         // device copy made by the first kernel of a batch

  // batches replayed from captured graphs, one per plan key; dropped whenever a
  // device buffer is allocated or freed or the adjacency's row table moves
  bool use_graphs = false;
  bool graphs_failed = false;  // a capture failed: launch kernel by kernel from then on
  std::vector<GraphSlot> graphs;
  unsigned long long graph_clock = 0;
  bool last_graph = false;     // the last batch ran as a graph replay

  // per-batch scratch, sized for cap_ops ops
  long long cap_ops = 0;
  long long cap_feat_rows = 0;
  ripple_op *d_ops = nullptr;
  ripple_op *h_ops = nullptr;  // pinned
  float *h_feat = nullptr;     // pinned
  u64 *ht_key = nullptr;
  int *ht_val = nullptr;
  int *ht_net = nullptr;
  unsigned ht_mask = 0;
  int *op_slot = nullptr;
  int *ins_src = nullptr, *ins_dst = nullptr, *del_src = nullptr, *del_dst = nullptr;
  int *ins_rank = nullptr, *del_rank = nullptr;
  float *ins_w = nullptr, *del_w = nullptr;  // the net arcs' weights (weighted graphs)
  int *flist = nullptr;
  int *frow = nullptr;  // feature row of each flist entry
  int *flist_done = nullptr;  // [n]: A^0 of the last completed batch (written by its clean-up)
  // the bucket form's arrays, allocated when a plan first uses the form: per-vertex
  // counters and per-bin totals (zero between batches), and slots for as many arcs
  // as the out-direction has slots, which bounds the arcs any layer pushes
  rp::Buckets bkt{};
  long long bkt_cap = 0;
  bool bkt_off = false;  // the arrays could not be allocated: the time model leaves the form out
  // rows long enough for the chunked delete sweep exist (or may, once rows grow):
  // the plan lists such rows in long_tab, their sweeps record positions in long_pool
  int long_ok = 0;
  rp::LongRow *long_tab = nullptr;
  int *long_pool = nullptr;

  // last batch
  bool has_batch = false;
  long long last_count[rp::kMaxL + 1] = {};
  long long last_nfeat = 0;

  // profiling: bit p of prof_mask records phase p
  unsigned prof_mask = 0;
  bool prof = false;
  std::vector<hipEvent_t> ev_pool;
  size_t ev_used = 0;
  std::vector<PhaseEv> ev_log;
  double ph_ms[RIPPLE_NUM_PHASES] = {};
  long long ph_launch[RIPPLE_NUM_PHASES] = {};
  double ph_bytes[RIPPLE_NUM_PHASES] = {};
  double ph_extra[RIPPLE_NUM_PHASES] = {};  // bytes_no_reuse - bytes
  double ph_flops[RIPPLE_NUM_PHASES] = {};
};

namespace {

const char *kNullCtxMsg = "ripple: context is NULL";
thread_local std::string g_load_err;  // message of the last failed ripple_load_graph

ripple_status fail(ripple_ctx *c, ripple_status st, const std::string &msg) {
  c->err = msg;
  return st;
}

ripple_status device_fail(ripple_ctx *c, hipError_t e, const char *what) {
  c->poisoned = true;
  c->err = std::string("ripple: HIP error in ") + what + ": " + hipGetErrorString(e);
  return RIPPLE_E_DEVICE;
}

#define RP_HIP(ctx, expr)                                    \
  do {                                                       \
    hipError_t _e = (expr);                                  \
    if (_e != hipSuccess) return device_fail(ctx, _e, #expr); \
  } while (0)

#define RP_TRY(expr)                      \
  do {                                    \
    ripple_status _s = (expr);            \
    if (_s != RIPPLE_OK) return _s;       \
  } while (0)

void drop_graphs(ripple_ctx *c) {
  for (GraphSlot &g : c->graphs) (void)hipGraphExecDestroy(g.exec);
  c->graphs.clear();
}

// Device allocation counted against the context's byte cap. Temporary buffers that
// no batch launch names (keep_graphs) leave the captured graphs alone; any other
// allocation or free may change an address a captured launch holds.
ripple_status dalloc(ripple_ctx *c, void **p, size_t size, bool keep_graphs = false) {
  if (!keep_graphs) drop_graphs(c);
  *p = nullptr;
  if (size == 0) size = 4;
  if (c->max_bytes > 0 && c->bytes + static_cast<long long>(size) > c->max_bytes)
    return fail(c, RIPPLE_E_OOM, "ripple: device byte cap reached (requested " + std::to_string(size) +
                                     " bytes, holding " + std::to_string(c->bytes) + ")");
  hipError_t e = hipMalloc(p, size);
  if (e == hipErrorOutOfMemory || e == hipErrorMemoryAllocation) {
    (void)hipGetLastError();
    *p = nullptr;
    return fail(c, RIPPLE_E_OOM, "ripple: hipMalloc of " + std::to_string(size) + " bytes failed");
  }
  if (e != hipSuccess) return device_fail(c, e, "hipMalloc");
  c->allocs[*p] = size;
  c->bytes += static_cast<long long>(size);
  return RIPPLE_OK;
}

template <typename T>
ripple_status dalloc_n(ripple_ctx *c, T **p, long long count, bool keep_graphs = false) {
  return dalloc(c, reinterpret_cast<void **>(p), static_cast<size_t>(count) * sizeof(T), keep_graphs);
}

void dfree(ripple_ctx *c, void *p, bool keep_graphs = false) {
  if (p == nullptr) return;
  if (!keep_graphs) drop_graphs(c);
  auto it = c->allocs.find(p);
  if (it != c->allocs.end()) {
    c->bytes -= static_cast<long long>(it->second);
    c->allocs.erase(it);
  }
  (void)hipFree(p);
}

template <typename T>
void dfree_t(ripple_ctx *c, T *&p) {
  dfree(c, reinterpret_cast<void *>(p));
  p = nullptr;
}

ripple_status check_ctx(ripple_ctx *c) {
  if (c == nullptr) return RIPPLE_E_INVALID;
  if (c->poisoned) {
    if (c->err.empty()) c->err = "ripple: context poisoned by an earlier device error";
    return RIPPLE_E_STATE;
  }
  c->err.clear();
  hipError_t e = hipSetDevice(c->device);
  if (e != hipSuccess) return device_fail(c, e, "hipSetDevice");
  return RIPPLE_OK;
}

long long row_cap(int len, float slack, int min_slack) {
  long long extra = static_cast<long long>(std::ceil(static_cast<double>(len) * slack));
  if (extra < min_slack) extra = min_slack;
  return len + extra;
}

long long arena_for(const ripple_ctx *c, long long total) {
  return c->arena_slots > 0 ? c->arena_slots : std::max<long long>(65536, total / 2);
}

// Uploads one adjacency direction laid out with spare slots per row and a spare
// arena at the end.
ripple_status upload_adj(ripple_ctx *c, int dir, const std::vector<int> &len, const std::vector<int> &col_packed,
                         const std::vector<long long> &packed_off, const std::vector<float> &wt_packed) {
  const long long n = c->n;
  std::vector<long long> off(n);
  std::vector<int> cap(n);
  long long total = 0;
  for (long long u = 0; u < n; ++u) {
    off[u] = total;
    const long long cp = row_cap(len[u], c->slack, c->min_slack);
    if (cp > INT32_MAX) return fail(c, RIPPLE_E_INVALID, "ripple: adjacency row too long");
    cap[u] = static_cast<int>(cp);
    total += cp;
  }
  const long long arena = arena_for(c, total);
  const long long capacity = total + arena;
  std::vector<int> col(static_cast<size_t>(total), -1);
  for (long long u = 0; u < n; ++u)
    std::copy(col_packed.begin() + packed_off[u], col_packed.begin() + packed_off[u] + len[u], col.begin() + off[u]);
  std::vector<float> wt;
  if (c->weighted) {
    wt.assign(static_cast<size_t>(total), 0.0f);
    for (long long u = 0; u < n; ++u)
      std::copy(wt_packed.begin() + packed_off[u], wt_packed.begin() + packed_off[u] + len[u], wt.begin() + off[u]);
  }
  rp::Adj &a = c->adj[dir];
  RP_TRY(dalloc_n(c, &a.off, n));
  RP_TRY(dalloc_n(c, &a.len, n));
  RP_TRY(dalloc_n(c, &a.cap, n));
  RP_TRY(dalloc_n(c, &a.col, capacity));
  RP_TRY(dalloc_n(c, &c->col_alt[dir], capacity));
  if (c->weighted) {
    RP_TRY(dalloc_n(c, &a.wt, capacity));
    RP_TRY(dalloc_n(c, &c->wt_alt[dir], capacity));
    if (total > 0)
      RP_HIP(c, hipMemcpyAsync(a.wt, wt.data(), total * sizeof(float), hipMemcpyHostToDevice, c->stream));
  }
  RP_TRY(dalloc_n(c, &a.inscnt, n));
  RP_TRY(dalloc_n(c, &a.delcnt, n));
  RP_HIP(c, hipMemcpyAsync(a.off, off.data(), n * sizeof(long long), hipMemcpyHostToDevice, c->stream));
  RP_HIP(c, hipMemcpyAsync(a.len, len.data(), n * sizeof(int), hipMemcpyHostToDevice, c->stream));
  RP_HIP(c, hipMemcpyAsync(a.cap, cap.data(), n * sizeof(int), hipMemcpyHostToDevice, c->stream));
  if (total > 0)
    RP_HIP(c, hipMemcpyAsync(a.col, col.data(), total * sizeof(int), hipMemcpyHostToDevice, c->stream));
  rp::launch_fill_i32(c->stream, a.col + total, arena, -1);
  RP_HIP(c, hipMemsetAsync(a.inscnt, 0, n * sizeof(int), c->stream));
  RP_HIP(c, hipMemsetAsync(a.delcnt, 0, n * sizeof(int), c->stream));
  u64 top = static_cast<u64>(total);
  RP_HIP(c, hipMemcpyAsync(&c->d_persist->top[dir], &top, sizeof(u64), hipMemcpyHostToDevice, c->stream));
  RP_HIP(c, hipStreamSynchronize(c->stream));
  c->col_capacity[dir] = capacity;
  c->arena_top[dir] = total;
  c->row_max[dir] = len.empty() ? 0 : *std::max_element(len.begin(), len.end());
  return RIPPLE_OK;
}

// Re-lays one direction out with fresh spare slots into new, larger buffers (when the
// device re-layout would not leave room for the arena).
ripple_status repack_adj_grow(ripple_ctx *c, int dir) {
  const long long n = c->n;
  rp::Adj &a = c->adj[dir];
  std::vector<int> len(n);
  RP_HIP(c, hipMemcpyAsync(len.data(), a.len, n * sizeof(int), hipMemcpyDeviceToHost, c->stream));
  RP_HIP(c, hipStreamSynchronize(c->stream));
  std::vector<long long> off(n);
  std::vector<int> cap(n);
  long long total = 0;
  for (long long u = 0; u < n; ++u) {
    off[u] = total;
    cap[u] = static_cast<int>(row_cap(len[u], c->slack, std::max(c->min_slack, 4)));
    total += cap[u];
  }
  const long long arena = arena_for(c, total);
  const long long capacity = total + arena;
  int *new_col = nullptr;
  float *new_wt = nullptr;
  long long *new_off = nullptr;
  dfree_t(c, c->col_alt[dir]);
  RP_TRY(dalloc_n(c, &c->col_alt[dir], capacity));
  RP_TRY(dalloc_n(c, &new_col, capacity));
  if (c->weighted) {
    dfree_t(c, c->wt_alt[dir]);
    RP_TRY(dalloc_n(c, &c->wt_alt[dir], capacity));
    RP_TRY(dalloc_n(c, &new_wt, capacity));
  }
  RP_TRY(dalloc_n(c, &new_off, n));
  RP_HIP(c, hipMemcpyAsync(new_off, off.data(), n * sizeof(long long), hipMemcpyHostToDevice, c->stream));
  rp::launch_fill_i32(c->stream, new_col, capacity, -1);
  rp::launch_repack_copy(c->stream, n, a.col, a.off, a.len, new_col, new_off, a.wt, new_wt);
  RP_HIP(c, hipMemcpyAsync(a.cap, cap.data(), n * sizeof(int), hipMemcpyHostToDevice, c->stream));
  RP_HIP(c, hipGetLastError());
  RP_HIP(c, hipStreamSynchronize(c->stream));
  dfree(c, a.col);
  dfree(c, a.off);
  a.col = new_col;
  a.off = new_off;
  if (c->weighted) {
    dfree(c, a.wt);
    a.wt = new_wt;
  }
  u64 top = static_cast<u64>(total);
  RP_HIP(c, hipMemcpyAsync(&c->d_persist->top[dir], &top, sizeof(u64), hipMemcpyHostToDevice, c->stream));
  RP_HIP(c, hipStreamSynchronize(c->stream));
  c->col_capacity[dir] = capacity;
  c->arena_top[dir] = total;
  return RIPPLE_OK;
}

// Re-lays one direction out with fresh spare slots (after the spare arena ran out):
// on the device, into the spare column buffer, when the fresh layout leaves at
// least a quarter of the buffer as arena; otherwise into new, larger buffers.
ripple_status repack_adj(ripple_ctx *c, int dir) {
  const long long n = c->n;
  rp::Adj &a = c->adj[dir];
  const int smin = std::max(c->min_slack, 4);
  rp::launch_relayout_sums(c->stream, n, c->slack, smin, a.len, c->rl_blocksums);
  long long total = 0;
  RP_HIP(c, hipMemcpyAsync(&total, c->rl_blocksums + rp::relayout_blocks(n), sizeof(long long),
                           hipMemcpyDeviceToHost, c->stream));
  RP_HIP(c, hipStreamSynchronize(c->stream));
  if (total + c->col_capacity[dir] / 4 > c->col_capacity[dir]) return repack_adj_grow(c, dir);
  rp::launch_relayout_apply(c->stream, n, c->slack, smin, a, c->col_alt[dir], c->wt_alt[dir], c->rl_blocksums,
                            c->rl_off, c->rl_cap, &c->d_persist->top[dir]);
  RP_HIP(c, hipGetLastError());
  drop_graphs(c);  // the launches name the row table's buffers
  std::swap(a.col, c->col_alt[dir]);
  if (c->weighted) std::swap(a.wt, c->wt_alt[dir]);
  c->arena_top[dir] = total;  // the new layout's rows end there
  return RIPPLE_OK;
}

void free_batch_scratch(ripple_ctx *c) {
  dfree_t(c, c->long_tab);
  dfree_t(c, c->long_pool);
  dfree_t(c, c->d_ops);
  dfree_t(c, c->ht_key);
  dfree_t(c, c->ht_val);
  dfree_t(c, c->ht_net);
  dfree_t(c, c->op_slot);
  dfree_t(c, c->ins_src);
  dfree_t(c, c->ins_dst);
  dfree_t(c, c->del_src);
  dfree_t(c, c->del_dst);
  dfree_t(c, c->ins_rank);
  dfree_t(c, c->del_rank);
  dfree_t(c, c->ins_w);
  dfree_t(c, c->del_w);
  dfree_t(c, c->flist);
  dfree_t(c, c->frow);
  if (c->h_ops) (void)hipHostFree(c->h_ops);
  if (c->h_feat) (void)hipHostFree(c->h_feat);
  c->h_ops = nullptr;
  c->h_feat = nullptr;
  c->cap_ops = 0;
  c->cap_feat_rows = 0;
}

// Grows per-batch scratch to hold `ops` ops and `frows` feature rows.
ripple_status ensure_batch_scratch(ripple_ctx *c, long long ops, long long frows) {
  if (ops <= c->cap_ops && frows <= c->cap_feat_rows && c->d_ops != nullptr) return RIPPLE_OK;
  long long cap = std::max<long long>({ops, c->cap_ops, 256});
  long long fcap = std::max<long long>({frows, c->cap_feat_rows, 64});
  if (ops > c->cap_ops) cap = std::max(cap, 2 * c->cap_ops);
  RP_HIP(c, hipStreamSynchronize(c->stream));
  free_batch_scratch(c);
  const long long arcs = 2 * cap;           // net arcs (undirected edges give two)
  // at most 1/64 full up to 4M slots (64 MB), else at most an eighth: the topology
  // pass probes every entry of a row that loses arcs, and a probe that meets an
  // occupied slot costs another dependent round
  const unsigned long long sparse = 64 * static_cast<unsigned long long>(cap);
  const unsigned long long want = sparse <= (1ull << 22) ? sparse : 8 * static_cast<unsigned long long>(cap);
  unsigned ht = 64;
  while (ht < want) ht <<= 1;
  RP_TRY(dalloc_n(c, &c->d_ops, cap));
  RP_TRY(dalloc_n(c, &c->ht_key, ht));
  RP_TRY(dalloc_n(c, &c->ht_val, ht));
  RP_TRY(dalloc_n(c, &c->ht_net, ht));
  RP_TRY(dalloc_n(c, &c->op_slot, cap));
  RP_TRY(dalloc_n(c, &c->ins_src, arcs));
  RP_TRY(dalloc_n(c, &c->ins_dst, arcs));
  RP_TRY(dalloc_n(c, &c->del_src, arcs));
  RP_TRY(dalloc_n(c, &c->del_dst, arcs));
  RP_TRY(dalloc_n(c, &c->ins_rank, 2 * arcs));
  RP_TRY(dalloc_n(c, &c->ins_w, arcs));
  RP_TRY(dalloc_n(c, &c->del_w, arcs));
  RP_TRY(dalloc_n(c, &c->del_rank, 2 * arcs));
  RP_TRY(dalloc_n(c, &c->flist, cap));
  RP_TRY(dalloc_n(c, &c->frow, cap));
  if (c->long_ok) {  // at most one long row per (net arc, direction), and two slots per deleted entry
    RP_TRY(dalloc_n(c, &c->long_tab, 2 * arcs));
    RP_TRY(dalloc_n(c, &c->long_pool, 4 * arcs));
  }
  RP_HIP(c, hipHostMalloc(reinterpret_cast<void **>(&c->h_ops), cap * sizeof(ripple_op), hipHostMallocDefault));
  RP_HIP(c, hipHostMalloc(reinterpret_cast<void **>(&c->h_feat), fcap * c->dims[0] * sizeof(float),
                          hipHostMallocDefault));
  rp::launch_fill_u64(c->stream, c->ht_key, ht, rp::kEmptyKey);
  rp::launch_fill_i32(c->stream, c->ht_val, ht, -1);
  rp::launch_fill_i32(c->stream, c->ht_net, ht, 0);
  RP_HIP(c, hipGetLastError());
  RP_HIP(c, hipStreamSynchronize(c->stream));
  c->ht_mask = ht - 1;
  c->cap_ops = cap;
  c->cap_feat_rows = fcap;
  return RIPPLE_OK;
}

// The bucket form's arrays (allocated again when a plan next uses the form).
void free_buckets(ripple_ctx *c) {
  dfree_t(c, c->bkt.cnt);
  dfree_t(c, c->bkt.bin_total);
  dfree_t(c, c->bkt.bin_base);
  dfree_t(c, c->bkt.block_off);
  dfree_t(c, c->bkt.tv);
  dfree_t(c, c->bkt.tj);
  dfree_t(c, c->bkt.tw);
  dfree_t(c, c->bkt.idx);
  dfree_t(c, c->bkt.wt);
  c->bkt_cap = 0;
}

void free_model(ripple_ctx *c) {
  for (int l = 0; l < rp::kMaxL; ++l) {
    dfree_t(c, c->W[l]);
    dfree_t(c, c->Wn[l]);
    dfree_t(c, c->bias[l]);
    dfree_t(c, c->W2[l]);
    dfree_t(c, c->b2[l]);
    dfree_t(c, c->Wb[l]);
    dfree_t(c, c->Wnb[l]);
    dfree_t(c, c->W2b[l]);
  }
  dfree_t(c, c->gin_rows);
  dfree_t(c, c->msg);
  for (int l = 0; l <= rp::kMaxL; ++l) dfree_t(c, c->P[l]);
  for (int l = 0; l <= rp::kMaxL; ++l) {
    dfree_t(c, c->H[l]);
    dfree_t(c, c->S[l]);
    dfree_t(c, c->lists[l]);
    dfree_t(c, c->doff[l]);
  }
  dfree_t(c, c->delta[0]);
  dfree_t(c, c->delta[1]);
  dfree_t(c, c->ioff);
  dfree_t(c, c->flist_done);
  free_buckets(c);
  for (int k = 0; k < 2; ++k) {
    dfree_t(c, c->memb[k]);
  }
  free_batch_scratch(c);
  c->inited = false;
}

rp::LayerPtrs layer_ptrs(const ripple_ctx *c) {
  rp::LayerPtrs lp{};
  for (int l = 1; l <= c->L; ++l) {
    lp.src[l] = c->tf[l] ? c->P[l] : c->H[l - 1];
    lp.S[l] = c->S[l];
    lp.sw[l] = c->sw[l];
  }
  lp.L = c->L;
  return lp;
}

// abort: the current batch's abort flag (nullptr outside a batch).
rp::GemmArgs gemm_args(const ripple_ctx *c, int l, const int *rows, const u64 *count, long long count_fixed,
                       float *delta, const u64 *abort) {
  rp::GemmArgs g{};
  g.mode = c->tf[l] ? rp::kTransformFirst : rp::kLayer;
  g.rows = rows;
  g.count = count;
  g.count_fixed = count_fixed;
  g.Hprev = c->H[l - 1];
  g.dprev = c->dims[l - 1];
  g.S = c->S[l];
  g.in_len = c->adj[1].len;
  g.out_len = c->adj[0].len;
  g.ddeg = c->ddeg;
  g.W = c->W[l - 1];
  g.Wb = c->Wb[l - 1];
  g.bf16 = c->gemm_bf16 ? 1 : 0;
  g.K = c->K[l - 1];
  g.N = c->dims[l];
  g.bias = c->bias[l - 1];
  g.relu = c->relu[l - 1];
  g.H = c->H[l];
  g.delta = delta;
  g.dld = rp::row_ld(c->dims[l]);
  g.agg = c->agg == rp::kGcWsum ? rp::kGcSum : c->agg;  // the weights are already in S
  g.abort = abort;
  g.eps1 = c->gin_eps1;
  return g;
}

// P rows of transform-first layer l: P_v = W_neigh h^{l-1}_v for the vertices of
// `rows` (nullptr: all, count_fixed of them); with msg set, also the messages
// msg[r] = c'_v P'_v - c_v P_v (c = 1, or the GCN source coefficient after / before
// the batch), aligned with `rows`.
rp::GemmArgs p_gemm_args(const ripple_ctx *c, int l, const int *rows, const u64 *count, long long count_fixed,
                         float *msg, const u64 *abort) {
  rp::GemmArgs g{};
  g.mode = rp::kPlain;
  g.rows = rows;
  g.count = count;
  g.count_fixed = count_fixed;
  g.Hprev = c->H[l - 1];
  g.dprev = c->dims[l - 1];
  g.S = nullptr;
  g.in_len = c->adj[1].len;
  g.out_len = c->adj[0].len;
  g.ddeg = c->ddeg;
  g.W = c->Wn[l - 1];
  g.Wb = c->Wnb[l - 1];
  g.bf16 = c->gemm_bf16 ? 1 : 0;
  g.K = c->dims[l - 1];
  g.N = c->dims[l];
  g.bias = nullptr;
  g.relu = 0;
  g.H = c->P[l];
  g.delta = msg;
  g.dld = rp::row_ld(c->dims[l]);
  g.agg = c->agg;
  g.abort = abort;
  return g;
}

// Layer l's transform on `rows` (nullptr: all, count_fixed of them): one GEMM, or
// GIN's two (the MLP's hidden rows go through gin_rows). cleanup (nullable): the
// batch's clean-up, run by extra blocks of the last launch. Returns the launches.
int launch_layer_gemm(const ripple_ctx *c, hipStream_t s, int l, const int *rows, const u64 *count,
                      long long count_fixed, float *delta, const u64 *abort, long long max_rows,
                      long long expected_rows, const rp::CleanupArgs *cleanup = nullptr, bool packed = false) {
  rp::GemmArgs g = gemm_args(c, l, rows, count, count_fixed, delta, abort);
  if (packed) g.count_shift = rp::kAppShift;
  if (c->agg != rp::kGin) {
    if (packed) {  // the scatter left the list's marks set
      g.clear_a = c->bm_out;
      g.clear_b = c->bm_x;
    }
    if (cleanup != nullptr) {
      g.cleanup = *cleanup;
      g.cleanup_blocks = rp::cleanup_blocks_for(c->cap_ops);
    }
    rp::launch_gemm(s, g, max_rows, expected_rows);
    return 1;
  }
  rp::GemmArgs g1 = g;  // hidden = ReLU(W1 ((1 + eps) h + S) + b1), one row per list position
  g1.mode = rp::kGin1;
  g1.relu = 1;
  g1.H = c->gin_rows;
  g1.delta = nullptr;
  if (packed) {  // the scatter left the list's marks set
    g1.clear_a = c->bm_out;
    g1.clear_b = c->bm_x;
  }
  rp::launch_gemm(s, g1, max_rows, expected_rows);
  rp::GemmArgs g2 = g;  // y = W2 hidden + b2, then the layer's activation, delta and write-back
  g2.mode = rp::kGin2;
  g2.Hprev = c->gin_rows;
  g2.dprev = c->dims[l];
  g2.S = nullptr;
  g2.W = c->W2[l - 1];
  g2.Wb = c->W2b[l - 1];
  g2.K = c->dims[l];
  g2.bias = c->b2[l - 1];
  if (cleanup != nullptr) {
    g2.cleanup = *cleanup;
    g2.cleanup_blocks = rp::cleanup_blocks_for(c->cap_ops);
  }
  rp::launch_gemm(s, g2, max_rows, expected_rows);
  return 2;
}

// --- profiling helpers ---

hipEvent_t next_event(ripple_ctx *c) {
  if (c->ev_used == c->ev_pool.size()) {
    hipEvent_t e;
    if (hipEventCreate(&e) != hipSuccess) return nullptr;
    c->ev_pool.push_back(e);
  }
  return c->ev_pool[c->ev_used++];
}

// The phase whose launches are being timed on this thread (see rp::launch_timer).
thread_local ripple_ctx *t_timed_ctx = nullptr;
thread_local int t_timed_phase = -1;

// Records the kernel times of one phase of a profiled batch: the launches made in
// its scope take an event pair each (rp::launch_timer). The whole batch
// (RIPPLE_PHASE_TOTAL) is bracketed by an event pair on the stream instead, from
// before its first kernel to after its last.
struct PhaseScope {
  ripple_ctx *c;
  int phase;
  hipEvent_t a = nullptr;
  ripple_ctx *prev_ctx = nullptr;
  int prev_phase = -1;
  bool timing = false;
  PhaseScope(ripple_ctx *cc, int ph) : c(cc), phase(ph) {
    if (!c->prof || !(c->prof_mask >> ph & 1u)) return;
    if (ph == RIPPLE_PHASE_TOTAL) {
      a = next_event(c);
      if (a) (void)hipEventRecord(a, c->stream);
      return;
    }
    prev_ctx = t_timed_ctx;
    prev_phase = t_timed_phase;
    t_timed_ctx = c;
    t_timed_phase = ph;
    timing = true;
  }
  void close() {
    if (a) {
      hipEvent_t b = next_event(c);
      if (b) {
        (void)hipEventRecord(b, c->stream);
        c->ev_log.push_back(PhaseEv{phase, a, b});
      }
      a = nullptr;
    }
    if (timing) {
      t_timed_ctx = prev_ctx;
      t_timed_phase = prev_phase;
      timing = false;
    }
  }
  ~PhaseScope() { close(); }
};

void add_launches(ripple_ctx *c, int phase, int k) {
  if (c->prof) c->ph_launch[phase] += k;
}

// How layer l adds its messages to S^l. Forced modes aside, the form with the
// least estimated time for the layer's expected counts (pushed arcs, affected rows,
// their in-arcs: the previous batch's, or for the first batch an estimate from the
// snapshot's degrees). The rates are fits to MI355X kernel traces of the forms on
// the dense_large and stress workloads, and to row micro-benchmarks:
//   push       per pushed arc: a fixed 90 ps plus its row of fp32 atomics at 1.3 TB/s;
//   pull       a bit atomic per pushed arc to mark its sink (38 ps), 35 ps per in-arc
//              of A^l scanned (its source's membership looked up), every message
//              read once at 10 TB/s (the rows are mostly cache hits), one row of
//              atomics per affected vertex at 1.3 TB/s;
//   dense      25 ps per in-arc of the whole graph and 20 ps per vertex (the full
//              listing) instead of the marks and A^l's in-arcs, reads and flushes as
//              pull;
//   recompute  the pull's marks, then every in-arc of A^l carries its source's row
//              (15 ps per arc plus the row at 6 TB/s, the rate of random row reads
//              from a table larger than the caches), one plain row store per
//              affected vertex at 5 TB/s;
//   bucket     35 ps per pushed arc for its trip through the bins (counted,
//              placed, sorted into its sink's bucket), its message row read by the
//              sums at 10 TB/s while the dirty rows' table stays within 32 MB (it
//              is then served by the caches; 4 TB/s beyond), each affected row
//              read and written once at 2.5 TB/s, and 20 us for the three extra
//              launches (fitted to the form's kernels on dense_large_2l's second
//              layer at batch 1000, stress's first and dense_large's second at
//              batch 100); it is taken only when its estimate is a quarter below
//              every other form's.
// Every reanchor_every-th batch recomputes every layer (the drift budget), whatever
// the form.
enum LayerMode { kPushLayer = 0, kPullLayer = 1, kDenseLayer = 2, kRecomputeLayer = 3, kBucketLayer = 4 };

int layer_mode(const ripple_ctx *c, int l, double dirty, double pushed, double count, double in_arcs, bool reanchor) {
  if (reanchor || c->scatter_mode == RIPPLE_SCATTER_RECOMPUTE) return kRecomputeLayer;
  if (c->scatter_mode == RIPPLE_SCATTER_PUSH) return kPushLayer;
  if (c->scatter_mode == RIPPLE_SCATTER_PULL) return kPullLayer;
  if (c->scatter_mode == RIPPLE_SCATTER_DENSE) return kDenseLayer;
  if (c->scatter_mode == RIPPLE_SCATTER_BUCKET) return kBucketLayer;
  const bool bucket_ok = !c->bkt_off && rp::bin_shift(c->n) >= 0;
  constexpr double kArc = 90e-12, kAtomicRate = 1.3e12, kMark = 38e-12, kPullScan = 35e-12;
  constexpr double kBinArc = 35e-12, kBucketRmwRate = 2.5e12, kBucketFixed = 20e-6;
  constexpr double kDenseScan = 25e-12, kDenseVertex = 20e-12, kReadRate = 10e12;
  constexpr double kRecScan = 15e-12, kGatherRate = 6e12, kStoreRate = 5e12;
  const double w = 4.0 * c->sw[l];  // message row bytes
  const double push = pushed * (kArc + w / kAtomicRate);
  const double settle = pushed * w / kReadRate + count * w / kAtomicRate;
  const double pull = pushed * kMark + in_arcs * kPullScan + settle;
  const double dense = static_cast<double>(c->arcs_now) * kDenseScan + static_cast<double>(c->n) * kDenseVertex + settle;
  const double recompute = pushed * kMark + in_arcs * (kRecScan + w / kGatherRate) + count * w / kStoreRate;
  const double gather = dirty * w <= 32e6 ? 10e12 : 4e12;
  const double bucket = pushed * (kBinArc + w / gather) + count * 2.0 * w / kBucketRmwRate + kBucketFixed;
  int best = kPushLayer;
  double t = push;
  if (pull < t) best = kPullLayer, t = pull;
  if (dense < t) best = kDenseLayer, t = dense;
  if (recompute < t) best = kRecomputeLayer, t = recompute;
  if (bucket_ok && 1.25 * bucket < t) best = kBucketLayer, t = bucket;
  return best;
}

// Expected counts of the first batch (no earlier batch to learn from), from the
// snapshot's degree sequences: layer 1's dirty set is the batch's feature-written
// vertices (under GCN also the tails of its edge ops), which push their out-degrees;
// a pushed arc reaches a sink with probability proportional to the sink's
// in-degree, so x pushed arcs reach sink v with probability 1 - exp(-x din(v)/m).
// Summed over (a sample of) the vertices this gives the affected rows, their
// in-arcs and their out-arcs, which the next layer pushes. The heads of the edge
// ops are affected at every layer, and under a self term the dirty set too.
void first_batch_counts(const ripple_ctx *c, const ripple_op *ops, long long B, double (&pushed)[rp::kMaxL + 1],
                        double (&count)[rp::kMaxL + 1], double (&in_arcs)[rp::kMaxL + 1]) {
  const long long n = c->n;
  const double m = std::max<double>(1.0, static_cast<double>(c->arcs_loaded));
  const double mean = m / static_cast<double>(n);
  const bool gcn = c->agg == rp::kGcn;
  std::vector<int> dirty;
  double heads = 0.0;
  for (long long i = 0; i < B && ops != nullptr; ++i) {
    const ripple_op &o = ops[i];
    if (o.kind == RIPPLE_OP_FEATURE) {
      dirty.push_back(o.u);
    } else if (o.u != o.v) {
      heads += c->undirected ? 2.0 : 1.0;
      if (gcn) dirty.push_back(o.u);
      if (gcn && c->undirected) dirty.push_back(o.v);
    }
  }
  std::sort(dirty.begin(), dirty.end());
  dirty.erase(std::unique(dirty.begin(), dirty.end()), dirty.end());
  double x = 0.0;
  for (int u : dirty) x += u >= 0 && u < n ? c->snap_out[u] : 0;
  double prev = static_cast<double>(dirty.size());
  const long long stride = std::max<long long>(1, n / 65536);
  const bool self = rp::has_self_term(c->agg);
  for (int l = 1; l <= c->L; ++l) {
    double a = 0.0, ia = 0.0, oa = 0.0;
    for (long long v = 0; v < n; v += stride) {
      const double p = 1.0 - std::exp(-x * static_cast<double>(c->snap_in[v]) / m);
      a += p;
      ia += p * c->snap_in[v];
      oa += p * c->snap_out[v];
    }
    const double extra = heads + (self ? prev : 0.0);  // rows affected without a pushed arc
    pushed[l] = x;
    count[l] = std::min(static_cast<double>(n), a * stride + extra);
    in_arcs[l] = ia * stride + extra * mean;
    x = oa * stride + extra * mean;
    prev = count[l];
  }
}

rp::CompactScratch compact_scratch(ripple_ctx *c, rp::Counters *dc) {
  return rp::CompactScratch{c->compact_lb, &dc->err};
}

// The launch plan of the next batch: every host decision its launches depend on.
struct BatchPlan {
  int mode[rp::kMaxL + 1];             // [l]: message form of layer l
  long long tf_rows[rp::kMaxL + 1];    // [l]: expected rows of layer l's transform-first GEMM
  long long rows[rp::kMaxL + 1];       // [l]: expected rows of layer l's GEMM
  bool direct0;                        // the corrections kernel lists the layer-1 dirty set
  int app;                             // bit l: layer l's scatter lists A^l (see ScatterList)
  bool arena_plan;                     // the arena check runs (else every possible row move fits)
  bool net_direct;                     // netting in one launch (small batches)
  unsigned long long key;              // the above as GEMM variants, and the counter parity
  unsigned long long key2;             // bit l: layer l takes the bucket form (its mode bits in key read push)
};

// Pushed arcs up to which a layer's scatter lists A^l itself, and that the next
// layer may push from such a list.
constexpr double kAppMaxArcs = 65536.0;
constexpr double kAppMaxNextArcs = 1048576.0;

BatchPlan make_plan(const ripple_ctx *c) {
  BatchPlan p{};
  unsigned long long key = static_cast<unsigned long long>(c->parity);
  int bit = 1;
  // expected counts per layer: the previous batch's, or an estimate for the first
  double pushed[rp::kMaxL + 1] = {}, count[rp::kMaxL + 1] = {}, in_arcs[rp::kMaxL + 1] = {};
  if (c->has_batch) {
    for (int l = 0; l <= c->L; ++l) {
      pushed[l] = static_cast<double>(c->last_pushed[l]);
      count[l] = static_cast<double>(c->last_count[l]);
      in_arcs[l] = static_cast<double>(c->last_in[l]);
    }
  } else {
    first_batch_counts(c, c->plan_ops, c->h_in->num_ops, pushed, count, in_arcs);
    count[0] = static_cast<double>(std::min<long long>(c->h_in->num_ops, c->n));
  }
  const bool reanchor = c->reanchor_every > 0 && (c->batches_done + 1) % c->reanchor_every == 0;
  long long guess[rp::kMaxL + 1];
  for (int l = 0; l <= c->L; ++l) guess[l] = static_cast<long long>(count[l]);
  for (int l = 1; l <= c->L; ++l) {
    p.mode[l] = layer_mode(c, l, count[l - 1], pushed[l], count[l], in_arcs[l], reanchor);
    p.tf_rows[l] = guess[l - 1];
    p.rows[l] = guess[l];
    if (p.mode[l] == kBucketLayer) p.key2 |= 1ull << l;
    key |= static_cast<unsigned long long>(p.mode[l] & 3) << bit;
    key |= static_cast<unsigned long long>(rp::gemm_variant(p.tf_rows[l], c->dims[l])) << (bit + 2);
    key |= static_cast<unsigned long long>(rp::gemm_variant(p.rows[l], c->dims[l])) << (bit + 4);
    bit += 6;  // up to bit 48 for 8 layers
  }
  // the layer-1 dirty set is the feature-written vertices alone unless GCN adds
  // the sources whose out-degree changed; listed directly when layer 1 pushes (a
  // pull needs the compaction's membership words) and the ops bound its size
  p.direct0 = c->agg != rp::kGcn && p.mode[1] == kPushLayer && c->h_in->num_ops <= rp::kDirectListMax;
  key |= static_cast<unsigned long long>(p.direct0) << 62;
  // a pushing layer lists A^l in its scatter unless the next layer pulls (a pull
  // reads the sorted list's membership words), it is expected to push many arcs
  // (the appends then queue on one counter and a compaction is cheaper), or the
  // next layer pushes many arcs from the list (its row reads keep their locality
  // in vertex order)
  p.app = 0;
  double arcs[rp::kMaxL + 2] = {};
  for (int l = 1; l <= c->L; ++l) arcs[l] = pushed[l];
  for (int l = 1; l <= c->L; ++l) {
    const bool next_ok = l == c->L || (p.mode[l + 1] == kPushLayer && arcs[l + 1] <= kAppMaxNextArcs);
    if (p.mode[l] == kPushLayer && arcs[l] <= kAppMaxArcs && next_ok) p.app |= 1 << l;
  }
  key |= static_cast<unsigned long long>(p.app) << 49;  // bits 50-57
  // The plan launch sums the arena slots that growing rows need and aborts the
  // batch if they do not fit. Only rows that gain arcs move: at most (2 for
  // undirected graphs) x ops rows per direction, each to grow_cap of at most its
  // length bound + as many arcs. When that fits in every direction's free arena the
  // check cannot fail and is left out (the rewrite still refuses a move past the
  // buffer). Rows swept in chunks are listed by the plan, so it always runs then.
  p.arena_plan = true;
  if (!c->long_ok) {
    const long long grow = (c->undirected ? 2LL : 1LL) * c->h_in->num_ops;
    bool fits = true;
    for (int d = 0; d < 2; ++d) {
      const long long newlen = c->row_max[d] + grow;
      const long long g = newlen + newlen / 2 + 4;  // the rewrite's grow_cap
      const long long worst = grow * ((g + 3) / 4 * 4);
      fits = fits && worst <= c->col_capacity[d] - c->arena_top[d];
    }
    p.arena_plan = !fits;
  }
  key |= static_cast<unsigned long long>(p.arena_plan) << 61;
  p.net_direct = c->h_in->num_ops <= rp::kNetDirectMax;
  key |= static_cast<unsigned long long>(p.net_direct) << 60;
  p.key = key;
  return p;
}

// Issues one batch's launches (the inputs are in c->h_in). Returns after queuing;
// the caller syncs. Launches only: the same calls are captured as a graph, and
// then (replay) the first kernel reads the inputs from c->h_in when it runs.
void issue_batch(ripple_ctx *c, const BatchPlan &p, bool replay) {
  hipStream_t s = c->stream;
  const int cap_ops = static_cast<int>(c->cap_ops);
  rp::Counters *dc = c->d_counters + c->parity;  // zeroed by the previous batch's clean-up
  rp::Counters *dnext = c->d_counters + (c->parity ^ 1);
  const int cap_arcs = static_cast<int>(2 * c->cap_ops);
  rp::Adj out = c->adj[0], in = c->adj[1];
  // the message kernels see the arcs' weights only under the weighted-sum model
  // (the topology kernels always keep them)
  rp::Adj out_msg = out, in_msg = in;
  if (c->agg != rp::kGcWsum) out_msg.wt = in_msg.wt = nullptr;
  rp::CleanupArgs cleanup{c->d_in,      c->d_ops,      c->op_slot,   c->ht_key,    c->ht_val,    c->ht_net,
                          c->fop,       out.inscnt,    out.delcnt,   in.inscnt,    in.delcnt,    c->ins_src,
                          c->ins_dst,   c->del_src,    c->del_dst,   c->ddeg,      c->flist,     c->flist_done,
                          dc,           dnext,         c->h_counters};
  PhaseScope total(c, RIPPLE_PHASE_TOTAL);
  {
    PhaseScope ps(c, RIPPLE_PHASE_NET);
    if (p.net_direct) {
      rp::launch_net_direct(s, cap_ops, replay ? c->h_in : nullptr, *c->h_in, c->d_in, c->d_ops, c->undirected,
                            c->weighted ? 1 : 0, c->n, c->ht_key, c->ht_net, c->ht_mask, c->op_slot, c->fop, out, in,
                            c->ins_src, c->ins_dst, c->del_src, c->del_dst, c->ins_rank, c->del_rank, c->ins_w,
                            c->del_w, c->flist, c->frow, dc);
    } else {
      rp::launch_net_hash(s, cap_ops, replay ? c->h_in : nullptr, *c->h_in, c->d_in, c->d_ops, c->undirected,
                          c->weighted ? 1 : 0, c->n, c->ht_key, c->ht_val, c->ht_mask, c->op_slot, c->fop, dc);
      rp::launch_net_decide(s, cap_ops, c->d_in, c->d_ops, c->undirected, c->ht_val, c->ht_net, c->op_slot, c->fop,
                            out, in, c->ins_src, c->ins_dst, c->del_src, c->del_dst, c->ins_rank, c->del_rank,
                            c->ins_w, c->del_w, c->flist, c->frow, dc);
    }
    add_launches(c, RIPPLE_PHASE_NET, p.net_direct ? 1 : 2);
  }
  {
    PhaseScope ps(c, RIPPLE_PHASE_TOPO);
    if (p.arena_plan)
      rp::launch_topo_plan(s, cap_arcs, out, in, c->ins_src, c->ins_dst, c->del_src, c->del_dst, c->ins_rank,
                           c->del_rank, c->long_ok, c->long_tab, dc, c->d_persist, c->col_capacity[0],
                           c->col_capacity[1]);
    const rp::RewriteBounds rb{{c->row_max[0], c->row_max[1]}, {c->col_capacity[0], c->col_capacity[1]}};
    rp::launch_topo_rewrite(s, cap_arcs, c->undirected, c->n, out, in, c->ins_src, c->ins_dst, c->del_src,
                            c->del_dst, c->ins_rank, c->del_rank, c->ht_key, c->ht_net, c->ht_mask, c->d_persist,
                            c->ddeg, c->long_ok, c->long_tab, c->long_pool, dc, rb);
    if (c->long_ok) rp::launch_topo_fill(s, cap_arcs, out, in, c->long_tab, c->long_pool, dc);
    add_launches(c, RIPPLE_PHASE_TOPO, (p.arena_plan ? 1 : 0) + 1 + (c->long_ok ? 1 : 0));
  }
  {
    PhaseScope ps(c, RIPPLE_PHASE_LAYER0);
    // also writes the inserted arcs into their slots
    // listed directly, the layer-0 deltas come with the list unless layer 1
    // transforms first (its GEMM reads the new rows of X before the scatter); x'
    // is staged in delta[1], which layer 1's GEMM fills only after the scatter
    rp::DirectList direct{};
    if (p.direct0)
      direct = rp::DirectList{c->lists[0], c->doff[0], &dc->count[0],           &dc->pushed[1],
                              nullptr,     nullptr,    rp::row_ld(c->dims[0]), c->dims[0],
                              c->H[0],     c->frow,    c->d_in};
    const bool direct_delta = p.direct0 && !c->tf[1];
    if (direct_delta) {
      direct.delta = c->delta[0];
      direct.stage = c->delta[1];
    }
    rp::launch_corr_mark(s, cap_ops, cap_arcs, c->agg, layer_ptrs(c), out, in, c->ins_rank, c->ins_w, c->ddeg,
                         c->flist, c->ins_src, c->ins_dst, c->del_src, c->del_dst,
                         c->agg == rp::kGcWsum ? c->ins_w : nullptr, c->del_w, c->bm_x, dc, direct);
    if (!p.direct0) {
      rp::CompactOut co{};
      co.list = c->lists[0];
      co.count = &dc->count[0];
      co.out_deg = c->adj[0].len;
      co.doff = c->doff[0];
      co.out_total = &dc->pushed[1];
      // layer 1 pulls messages: it looks up A^0's membership
      const bool members = p.mode[1] == kPullLayer || p.mode[1] == kDenseLayer;
      co.memb = members ? c->memb[0] : nullptr;
      rp::launch_compact(s, c->n, c->bm_out, c->bm_x, compact_scratch(c, dc), co);
    }
    if (!direct_delta) {
      const rp::Delta0Args z{c->agg, c->dims[0], rp::row_ld(c->dims[0]), c->d_ops, c->d_in, c->fop, c->H[0],
                             c->adj[0].len, c->ddeg, c->delta[0], dc};
      rp::launch_delta0(s, c->n, z, c->lists[0], &dc->count[0]);
    }
    add_launches(c, RIPPLE_PHASE_LAYER0, 1 + (p.direct0 ? 0 : 1) + (direct_delta ? 0 : 1));
  }
  for (int l = 1; l <= c->L; ++l) {
    float *din = c->delta[(l - 1) & 1];
    // the next layer's messages: this layer's delta rows, unless it transforms first
    // (its messages then come from its own P rows)
    float *dout = l < c->L && !c->tf[l + 1] ? c->delta[l & 1] : nullptr;
    const float *msg = din;
    // A^{l-1} listed by its scatter: its count and arc total are one packed word
    const bool packed_in = p.app >> (l - 1) & 1;
    const u64 *count_in = packed_in ? &dc->app[l - 1] : &dc->count[l - 1];
    const bool app = p.app >> l & 1;
    if (c->tf[l]) {
      // transform-first layer: refresh P = W_neigh h for the dirty rows and form
      // their messages c' P' - c P
      PhaseScope ps(c, RIPPLE_PHASE_GEMM);
      rp::GemmArgs pg = p_gemm_args(c, l, c->lists[l - 1], count_in, 0, c->msg, &dc->abort);
      if (packed_in) pg.count_shift = rp::kAppShift;
      rp::launch_gemm(s, pg, c->n, p.tf_rows[l]);
      add_launches(c, RIPPLE_PHASE_GEMM, 1);
      msg = c->msg;
    }
    const int mode = p.mode[l];
    const int ld = rp::row_ld(c->sw[l]);  // message row stride
    const uint2 *memb = c->memb[(l - 1) & 1];
    if (mode == kDenseLayer) {
      // dense: mark the net arcs' heads and D (no arcs), list every vertex with its
      // in-arc prefix, pull over every in-arc and mark the sinks that received a
      // message (the listing is timed with the compactions)
      {
        PhaseScope ps(c, RIPPLE_PHASE_SCATTER);
        rp::launch_scatter(s, c->n, c->sw[l], ld, c->lists[l - 1], &dc->count[l - 1], c->doff[l - 1], msg, out_msg,
                           c->S[l], c->bm_out, c->bm_x, c->ins_dst, c->del_dst, &dc->zero, dc, false,
                           rp::has_self_term(c->agg));
        add_launches(c, RIPPLE_PHASE_SCATTER, 1);
      }
      {
        PhaseScope ps(c, RIPPLE_PHASE_COMPACT);
        rp::CompactOut all{};
        all.full_n = c->n;
        all.count = &dc->count_all;
        all.in_deg = c->adj[1].len;
        all.ioff = c->ioff;
        rp::launch_compact(s, c->n, nullptr, nullptr, compact_scratch(c, dc), all);
        add_launches(c, RIPPLE_PHASE_COMPACT, 1);
      }
      PhaseScope ps(c, RIPPLE_PHASE_SCATTER);
      rp::launch_pull_msgs(s, c->n, c->sw[l], ld, nullptr, &dc->count_all, c->ioff, in_msg, memb, msg,
                           c->S[l], c->bm_out, dc);
      add_launches(c, RIPPLE_PHASE_SCATTER, 1);
    } else {
      // push: marks + atomic adds; pull: marks only (the adds follow the compaction)
      PhaseScope ps(c, RIPPLE_PHASE_SCATTER);
      // after a direct listing with its deltas, layer 1's scatter also moves the
      // staged x' rows into X
      rp::ScatterCopy copy{};
      if (l == 1 && p.direct0 && !c->tf[1]) copy = rp::ScatterCopy{c->H[0], c->delta[1], c->dims[0], rp::row_ld(c->dims[0])};
      rp::ScatterList lo{};
      if (app)
        lo = rp::ScatterList{c->lists[l],       l < c->L ? c->doff[l] : nullptr, &dc->app[l], &dc->app_sinks[l],
                             c->adj[0].len, c->adj[1].len};
      if (mode == kBucketLayer) {
        // the pushed arcs sorted by sink (D is a compacted list here: a scatter lists
        // A^{l-1} only when layer l pushes, and the corrections kernel lists A^0 only
        // when layer 1 does); the compaction below lists the sinks from their counts
        rp::Buckets b = c->bkt;
        if (out_msg.wt == nullptr) b.tw = b.wt = nullptr;
        rp::launch_bin_count(s, c->lists[l - 1], &dc->count[l - 1], c->doff[l - 1], out_msg, &dc->pushed[l], b,
                             c->bm_x, c->ins_dst, c->del_dst, rp::has_self_term(c->agg), dc);
        rp::launch_bin_scatter(s, c->lists[l - 1], &dc->count[l - 1], c->doff[l - 1], out_msg, &dc->pushed[l], b, dc);
        rp::launch_bin_sort(s, c->n, &dc->pushed[l], b, dc);
        add_launches(c, RIPPLE_PHASE_SCATTER, 2);
      } else {
        rp::launch_scatter(s, c->n, c->sw[l], ld, c->lists[l - 1], count_in, c->doff[l - 1], msg, out_msg, c->S[l],
                           c->bm_out, c->bm_x, c->ins_dst, c->del_dst, &dc->pushed[l], dc, mode == kPushLayer,
                           rp::has_self_term(c->agg), copy, lo, packed_in);
      }
      add_launches(c, RIPPLE_PHASE_SCATTER, 1);
    }
    if (!app) {
      PhaseScope ps(c, RIPPLE_PHASE_COMPACT);
      rp::CompactOut co{};
      co.list = c->lists[l];
      co.count = &dc->count[l];
      co.out_deg = c->adj[0].len;
      co.doff = l < c->L ? c->doff[l] : nullptr;
      co.in_deg = c->adj[1].len;
      co.ioff = mode == kPullLayer || mode == kRecomputeLayer ? c->ioff : nullptr;
      if (mode == kRecomputeLayer) {  // rows summed in segments start from zero
        co.zero_rows = c->S[l];
        co.zero_w = c->sw[l];
      }
      if (mode == kBucketLayer) {  // the sinks from their counts; the buckets' offsets (in ioff) and starts
        co.bkt_cnt = c->bkt.cnt;
        co.boff = c->ioff;
        co.bkt_start = c->bkt.cnt;
      }
      co.in_total = &dc->indeg[l];
      co.out_total = l < c->L ? &dc->pushed[l + 1] : nullptr;
      co.sinks_a = &dc->dest[l];  // distinct sinks of the arcs pushed at layer l
      const bool members = l < c->L && (p.mode[l + 1] == kPullLayer || p.mode[l + 1] == kDenseLayer);
      co.memb = members ? c->memb[l & 1] : nullptr;
      rp::launch_compact(s, c->n, c->bm_out, c->bm_x, compact_scratch(c, dc), co);
      add_launches(c, RIPPLE_PHASE_COMPACT, 1);
    }
    if (mode == kPullLayer) {
      PhaseScope ps(c, RIPPLE_PHASE_SCATTER);
      rp::launch_pull_msgs(s, c->n, c->sw[l], ld, c->lists[l], &dc->count[l], c->ioff, in_msg, memb, msg,
                           c->S[l], nullptr, dc);
      add_launches(c, RIPPLE_PHASE_SCATTER, 1);
    } else if (mode == kRecomputeLayer) {
      // re-anchoring: every aggregate row of A^l summed afresh from the current
      // source rows (the messages and the layer-0 corrections of these rows are
      // superseded)
      PhaseScope ps(c, RIPPLE_PHASE_SCATTER);
      rp::launch_recompute(s, c->n, c->sw[l], c->agg == rp::kGcn ? 1 : 0, c->lists[l], &dc->count[l], c->ioff,
                           in_msg, c->adj[0].len, layer_ptrs(c).src[l], c->S[l], dc);
      add_launches(c, RIPPLE_PHASE_SCATTER, 1);
    } else if (mode == kBucketLayer) {
      // each sink's bucket summed into its row
      PhaseScope ps(c, RIPPLE_PHASE_SCATTER);
      rp::Buckets b = c->bkt;
      if (out_msg.wt == nullptr) b.tw = b.wt = nullptr;
      rp::launch_bucket_sum(s, c->sw[l], ld, c->lists[l], &dc->count[l], c->ioff, b, msg, c->S[l], dc);
      add_launches(c, RIPPLE_PHASE_SCATTER, 1);
    }
    {
      // the last layer's GEMM also resets the batch's scratch (extra blocks)
      PhaseScope ps(c, RIPPLE_PHASE_GEMM);
      add_launches(c, RIPPLE_PHASE_GEMM,
                   launch_layer_gemm(c, s, l, c->lists[l], app ? &dc->app[l] : &dc->count[l], 0, dout, &dc->abort,
                                     c->n, p.rows[l], l == c->L ? &cleanup : nullptr, app));
    }
  }
  total.close();
}

// The executable graph of plan p: a cached one, else a new capture of the batch's
// launches (nullptr if capturing fails; the caller then launches directly).
hipGraphExec_t plan_graph(ripple_ctx *c, const BatchPlan &p) {
  constexpr size_t kMaxGraphs = 16;
  for (GraphSlot &g : c->graphs) {
    if (g.key == p.key && g.key2 == p.key2) {
      g.used = ++c->graph_clock;
      return g.exec;
    }
  }
  hipGraph_t graph = nullptr;
  hipGraphExec_t exec = nullptr;
  hipError_t e = hipStreamBeginCapture(c->stream, hipStreamCaptureModeThreadLocal);
  if (e == hipSuccess) {
    issue_batch(c, p, true);
    e = hipStreamEndCapture(c->stream, &graph);
  }
  if (e == hipSuccess) e = hipGraphInstantiate(&exec, graph, nullptr, nullptr, 0);
  if (e == hipSuccess) e = hipGraphUpload(exec, c->stream);
  if (graph != nullptr) (void)hipGraphDestroy(graph);
  if (e != hipSuccess) {
    (void)hipGetLastError();
    if (exec != nullptr) (void)hipGraphExecDestroy(exec);
    c->graphs_failed = true;
    return nullptr;
  }
  if (c->graphs.size() >= kMaxGraphs) {
    auto old = std::min_element(c->graphs.begin(), c->graphs.end(),
                                [](const GraphSlot &a, const GraphSlot &b) { return a.used < b.used; });
    (void)hipGraphExecDestroy(old->exec);
    c->graphs.erase(old);
  }
  c->graphs.push_back(GraphSlot{p.key, p.key2, exec, ++c->graph_clock});
  return exec;
}

// The bucket form's arrays, allocated (or grown with the out-direction's slots) when
// a plan first needs them; the counters start at zero and every batch leaves them
// so.
ripple_status ensure_buckets(ripple_ctx *c) {
  const int shift = rp::bin_shift(c->n);
  if (shift < 0)
    return fail(c, RIPPLE_E_INVALID, "ripple: the bucket form takes graphs of at most 2^25 vertices");
  if (c->bkt.cnt == nullptr || c->bkt.bin_total == nullptr || c->bkt.bin_base == nullptr ||
      c->bkt.block_off == nullptr) {
    // all four or none: an allocation that failed before leaves no part of them in
    // use (the kernels take every one)
    dfree_t(c, c->bkt.cnt);
    dfree_t(c, c->bkt.bin_total);
    dfree_t(c, c->bkt.bin_base);
    dfree_t(c, c->bkt.block_off);
    const long long slots = rp::bucket_counter_slots(c->n);
    const int nbins = static_cast<int>((c->n + (1LL << shift) - 1) >> shift);
    c->bkt.shift = shift;
    c->bkt.nbins = nbins;
    RP_TRY(dalloc_n(c, &c->bkt.cnt, slots));
    RP_HIP(c, hipMemsetAsync(c->bkt.cnt, 0, static_cast<size_t>(slots) * sizeof(int), c->stream));
    RP_TRY(dalloc_n(c, &c->bkt.bin_total, nbins));
    RP_HIP(c, hipMemsetAsync(c->bkt.bin_total, 0, static_cast<size_t>(nbins) * sizeof(int), c->stream));
    RP_TRY(dalloc_n(c, &c->bkt.bin_base, nbins));
    RP_TRY(dalloc_n(c, &c->bkt.block_off, static_cast<long long>(rp::kBinBlocks) * nbins));
  }
  const long long need = std::max<long long>(1, c->col_capacity[0]);
  if (need > std::numeric_limits<int32_t>::max())  // bucket slots are int32
    return fail(c, RIPPLE_E_OOM, "ripple: the bucket form needs fewer than 2^31 out-arc slots");
  if (c->bkt_cap < need) {
    dfree_t(c, c->bkt.tv);
    dfree_t(c, c->bkt.tj);
    dfree_t(c, c->bkt.tw);
    dfree_t(c, c->bkt.idx);
    dfree_t(c, c->bkt.wt);
    c->bkt_cap = 0;
    RP_TRY(dalloc_n(c, &c->bkt.tv, need));
    RP_TRY(dalloc_n(c, &c->bkt.tj, need));
    RP_TRY(dalloc_n(c, &c->bkt.idx, need));
    if (c->agg == rp::kGcWsum) {
      RP_TRY(dalloc_n(c, &c->bkt.tw, need));
      RP_TRY(dalloc_n(c, &c->bkt.wt, need));
    }
    c->bkt_cap = need;
  }
  return RIPPLE_OK;
}

// Queues one batch whose inputs are in c->h_in: as a graph replay unless graphs
// are off or this batch records phase events.
ripple_status launch_batch(ripple_ctx *c) {
  BatchPlan p = make_plan(c);
  if (p.key2 != 0) {
    const ripple_status st = ensure_buckets(c);
    if (st == RIPPLE_E_OOM && c->scatter_mode != RIPPLE_SCATTER_BUCKET) {
      // chosen by the time model, not asked for: plan again without the form (and
      // give back what was allocated of its arrays)
      c->bkt_off = true;
      c->err.clear();
      free_buckets(c);
      p = make_plan(c);
    } else if (st != RIPPLE_OK) {
      return st;
    }
  }
  c->last_bucket = static_cast<int>(p.key2);
  c->last_pull = 0;
  c->last_dense = 0;
  c->last_recompute = 0;
  for (int l = 1; l <= c->L; ++l) {
    if (p.mode[l] == kPullLayer) c->last_pull |= 1 << l;
    if (p.mode[l] == kDenseLayer) c->last_dense |= 1 << l;
    if (p.mode[l] == kRecomputeLayer) c->last_recompute |= 1 << l;
  }
  c->run_app = p.app;
  c->last_graph = false;
  hipGraphExec_t g = c->use_graphs && !c->graphs_failed && !c->prof ? plan_graph(c, p) : nullptr;
  if (g != nullptr) {
    RP_HIP(c, hipGraphLaunch(g, c->stream));
    c->last_graph = true;
  } else {
    issue_batch(c, p, false);
    RP_HIP(c, hipGetLastError());
  }
  c->parity ^= 1;
  return RIPPLE_OK;
}

void account_phases(ripple_ctx *c) {
  if (!c->prof) return;
  const rp::Counters &k = *c->h_counters;
  for (const PhaseEv &p : c->ev_log) {
    float ms = 0.0f;
    if (hipEventElapsedTime(&ms, p.a, p.b) == hipSuccess) c->ph_ms[p.phase] += ms;
  }
  c->ph_launch[RIPPLE_PHASE_TOTAL] += 1;
  const double words = static_cast<double>((c->n + 31) / 32);
  for (int l = 1; l <= c->L; ++l) {
    const double d = c->sw[l];
    const double nd = static_cast<double>(k.count[l - 1]);
    const double per_arc = static_cast<double>(k.pushed[l]);
    const double sinks = static_cast<double>(k.dest[l]);
    if (c->last_recompute >> l & 1) {
      // recompute: the marks (arc ids and row offsets of D), every in-arc id of A^l and
      // its in-row offset, each source row read once (at most n of them) and each row
      // of A^l written once; without reuse, a source row per in-arc
      const double in_l = static_cast<double>(k.indeg[l]);
      const double rows = std::min(in_l, static_cast<double>(c->n));
      c->ph_bytes[RIPPLE_PHASE_SCATTER] +=
          4.0 * per_arc + 8.0 * nd + 4.0 * in_l + 12.0 * k.count[l] + 4.0 * d * rows + 4.0 * d * k.count[l];
      c->ph_extra[RIPPLE_PHASE_SCATTER] += 4.0 * d * (in_l - rows);
    } else {
      c->ph_bytes[RIPPLE_PHASE_SCATTER] += 4.0 * per_arc + 8.0 * nd + 4.0 * d * nd + 8.0 * d * sinks;
      // without on-chip reuse: a message row read per arc that carries it, and under
      // push a row of atomics per arc rather than per sink
      c->ph_extra[RIPPLE_PHASE_SCATTER] += 4.0 * d * std::max(per_arc - nd, 0.0);
      if (!((c->last_pull | c->last_dense | c->last_bucket) >> l & 1))
        c->ph_extra[RIPPLE_PHASE_SCATTER] += 8.0 * d * std::max(per_arc - sinks, 0.0);
    }
    if (c->last_pull >> l & 1)  // pull: every in-arc id of A^l and its in-row offset
      c->ph_bytes[RIPPLE_PHASE_SCATTER] += 4.0 * k.indeg[l] + 12.0 * k.count[l];
    if (c->last_dense >> l & 1) {
      // dense: every in-arc id and every vertex's in-row offset (the pull); the
      // listing reads every in-degree and writes the offsets
      c->ph_bytes[RIPPLE_PHASE_SCATTER] += 4.0 * static_cast<double>(c->arcs_now) + 8.0 * static_cast<double>(c->n);
      c->ph_bytes[RIPPLE_PHASE_COMPACT] += 12.0 * static_cast<double>(c->n);
    }
    if (c->tf[l]) {
      const double dp = c->dims[l - 1];
      c->ph_flops[RIPPLE_PHASE_GEMM] += 2.0 * nd * dp * d;
      c->ph_bytes[RIPPLE_PHASE_GEMM] += 4.0 * nd * dp + 4.0 * d * dp + 12.0 * nd * d;  // h rows, W, P old/new, msg
    }
    const double m = static_cast<double>(k.count[l]);
    const double K = c->K[l - 1], N = c->dims[l];
    c->ph_flops[RIPPLE_PHASE_GEMM] += 2.0 * m * K * N;
    if (c->agg == rp::kGin) {  // the MLP's second layer: hidden rows in and out once more
      c->ph_flops[RIPPLE_PHASE_GEMM] += 2.0 * m * N * N;
      c->ph_bytes[RIPPLE_PHASE_GEMM] += 8.0 * m * N + 4.0 * N * N;
    }
    c->ph_bytes[RIPPLE_PHASE_GEMM] += 4.0 * m * K + 4.0 * N * K + 4.0 * m * N * (l < c->L && !c->tf[l + 1] ? 3.0 : 2.0);
    if (c->last_app >> l & 1)  // listed by the scatter: each member's id, offset and degrees
      c->ph_bytes[RIPPLE_PHASE_SCATTER] += 20.0 * m;
    else
      c->ph_bytes[RIPPLE_PHASE_COMPACT] += 24.0 * words + 4.0 * m;
  }
  c->ev_log.clear();
  c->ev_used = 0;
}

// Waits for the batch: polls the stream for up to ~20 ms (a batch usually takes
// well under a millisecond, and polling keeps the thread from being descheduled
// while it waits), then blocks.
ripple_status wait_stream(ripple_ctx *c) {
  const auto t0 = std::chrono::steady_clock::now();
  while (true) {
    const hipError_t e = hipStreamQuery(c->stream);
    if (e == hipSuccess) return RIPPLE_OK;
    if (e != hipErrorNotReady) return device_fail(c, e, "hipStreamQuery");
    if (std::chrono::steady_clock::now() - t0 > std::chrono::milliseconds(20)) break;
  }
  RP_HIP(c, hipStreamSynchronize(c->stream));
  return RIPPLE_OK;
}

bool validate_ops(ripple_ctx *c, const ripple_op *ops, long long num_ops, long long num_feat_rows) {
  for (long long i = 0; i < num_ops; ++i) {
    const ripple_op &o = ops[i];
    if (o.kind == RIPPLE_OP_INSERT || o.kind == RIPPLE_OP_DELETE) {
      if (o.u < 0 || o.u >= c->n || o.v < 0 || o.v >= c->n) {
        c->err = "ripple: op " + std::to_string(i) + ": vertex id out of range";
        return false;
      }
      if (c->weighted && o.kind == RIPPLE_OP_INSERT && !std::isfinite(o.weight)) {
        c->err = "ripple: op " + std::to_string(i) + ": insert weight is not finite";
        return false;
      }
    } else if (o.kind == RIPPLE_OP_FEATURE) {
      if (o.u < 0 || o.u >= c->n) {
        c->err = "ripple: op " + std::to_string(i) + ": vertex id out of range";
        return false;
      }
      if (o.feat_row < 0 || o.feat_row >= num_feat_rows) {
        c->err = "ripple: op " + std::to_string(i) + ": feat_row out of range";
        return false;
      }
    } else {
      c->err = "ripple: op " + std::to_string(i) + ": unknown kind " + std::to_string(o.kind);
      return false;
    }
  }
  return true;
}

// Staging memory of ripple_get_embeddings_static: a file-scope device array, so the
// call allocates nothing. Each device holds its own copy (at its own address, found
// once per device with hipGetSymbolAddress; host code never uses the array's name
// as an address). Calls that overlap on one device race for it.
constexpr size_t kStaticStageBytes = size_t{32} << 20;
static __device__ __align__(256) unsigned char scratch[kStaticStageBytes];

constexpr int kMaxDevices = 64;
std::mutex g_stage_mu;
void *g_stage_ptr[kMaxDevices] = {};

// This device's copy of the staging array (the device must be current).
hipError_t static_stage(int device, void **ptr) {
  *ptr = nullptr;
  if (device < 0 || device >= kMaxDevices) return hipErrorInvalidDevice;
  std::lock_guard<std::mutex> lock(g_stage_mu);
  if (g_stage_ptr[device] == nullptr) {
    void *p = nullptr;
    const hipError_t e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return e;
    g_stage_ptr[device] = p;
  }
  *ptr = g_stage_ptr[device];
  return hipSuccess;
}

ripple_status read_rows(ripple_ctx *c, const float *src, int d, const int32_t *ids, long long count, float *out) {
  if (count < 0) return fail(c, RIPPLE_E_INVALID, "ripple: negative count");
  if (count == 0) return RIPPLE_OK;
  if (out == nullptr) return fail(c, RIPPLE_E_INVALID, "ripple: out is NULL");
  if (ids == nullptr) {
    if (count != c->n) return fail(c, RIPPLE_E_INVALID, "ripple: ids NULL requires count == n");
    RP_HIP(c, hipMemcpyAsync(out, src, static_cast<size_t>(count) * d * sizeof(float), hipMemcpyDeviceToHost,
                             c->stream));
    RP_HIP(c, hipStreamSynchronize(c->stream));
    return RIPPLE_OK;
  }
  for (long long i = 0; i < count; ++i)
    if (ids[i] < 0 || ids[i] >= c->n) return fail(c, RIPPLE_E_INVALID, "ripple: vertex id out of range");
  int *d_ids = nullptr;
  float *d_out = nullptr;
  RP_TRY(dalloc_n(c, &d_ids, count, true));
  ripple_status st = dalloc_n(c, &d_out, count * d, true);
  if (st != RIPPLE_OK) {
    dfree(c, d_ids, true);
    return st;
  }
  hipError_t e = hipMemcpyAsync(d_ids, ids, count * sizeof(int), hipMemcpyHostToDevice, c->stream);
  if (e == hipSuccess) {
    rp::launch_gather_rows(c->stream, src, d, d_ids, count, d_out);
    e = hipGetLastError();
  }
  if (e == hipSuccess)
    e = hipMemcpyAsync(out, d_out, static_cast<size_t>(count) * d * sizeof(float), hipMemcpyDeviceToHost, c->stream);
  if (e == hipSuccess) e = hipStreamSynchronize(c->stream);
  dfree(c, d_ids, true);
  dfree(c, d_out, true);
  if (e != hipSuccess) return device_fail(c, e, "read_rows");
  return RIPPLE_OK;
}

}  // namespace

namespace rp {

bool launch_timer(hipEvent_t *start, hipEvent_t *stop) {
  ripple_ctx *c = t_timed_ctx;
  if (c == nullptr) return false;
  *start = next_event(c);
  *stop = next_event(c);
  if (*start == nullptr || *stop == nullptr) return false;
  c->ev_log.push_back(PhaseEv{t_timed_phase, *start, *stop});
  return true;
}

}  // namespace rp

extern "C" {

ripple_status ripple_load_graph(const ripple_graph_desc *g, ripple_ctx **out) {
  if (out == nullptr) return RIPPLE_E_INVALID;
  *out = nullptr;
  if (g == nullptr) return RIPPLE_E_INVALID;
  ripple_ctx *c = new ripple_ctx();
  g_load_err.clear();
  auto bail = [&](ripple_status st) {
    g_load_err = c->err;
    ripple_destroy(c);
    return st;
  };
  const long long n = g->num_vertices, m = g->num_edges;
  if (n < 1 || n > INT32_MAX) {
    c->err = "ripple: num_vertices must be in [1, 2^31)";
    return bail(RIPPLE_E_INVALID);
  }
  if (m < 0 || (m > 0 && (g->src == nullptr || g->dst == nullptr))) {
    c->err = "ripple: bad edge arrays";
    return bail(RIPPLE_E_INVALID);
  }
  if (!(g->slack >= 0.0f) || g->min_slack < 0 || g->arena_slots < 0) {
    c->err = "ripple: slack must be >= 0";
    return bail(RIPPLE_E_INVALID);
  }
  c->n = n;
  c->undirected = g->undirected ? 1 : 0;
  c->weighted = g->weight != nullptr;
  for (long long i = 0; c->weighted && i < m; ++i)
    if (!std::isfinite(g->weight[i])) {
      c->err = "ripple: edge " + std::to_string(i) + ": weight is not finite";
      return bail(RIPPLE_E_INVALID);
    }
  c->slack = g->slack;
  c->min_slack = g->min_slack;
  if (const char *hook = std::getenv("RIPPLE_DEBUG_FAIL_BATCH")) c->debug_fail_batch = std::atoll(hook);
  c->device = g->device;
  c->max_bytes = g->max_device_bytes;
  c->arena_slots = g->arena_slots;
  // host-side validation and counting sort into CSR (by source) and CSC (by sink)
  const long long arcs = c->undirected ? 2 * m : m;
  c->arcs_loaded = arcs;
  c->arcs_now = arcs;
  std::vector<int> outdeg(n, 0), indeg(n, 0);
  for (long long i = 0; i < m; ++i) {
    const int u = g->src[i], v = g->dst[i];
    if (u < 0 || u >= n || v < 0 || v >= n) {
      c->err = "ripple: edge " + std::to_string(i) + ": vertex id out of range";
      return bail(RIPPLE_E_INVALID);
    }
    if (u == v) {
      c->err = "ripple: edge " + std::to_string(i) + ": self-loop";
      return bail(RIPPLE_E_INVALID);
    }
    outdeg[u]++;
    indeg[v]++;
    if (c->undirected) {
      outdeg[v]++;
      indeg[u]++;
    }
  }
  std::vector<long long> ooff(n + 1, 0), ioff(n + 1, 0);
  for (long long u = 0; u < n; ++u) {
    ooff[u + 1] = ooff[u] + outdeg[u];
    ioff[u + 1] = ioff[u] + indeg[u];
  }
  std::vector<int> ocol(arcs), icol(arcs);
  std::vector<float> ow, iw;  // weighted graphs: the arcs' weights in the same order
  // weighted rows are sorted as (column, weight bits) pairs packed in 64 bits
  std::vector<unsigned long long> okey;
  auto pack = [](int v, float w) {
    unsigned bits;
    std::memcpy(&bits, &w, sizeof(bits));
    return static_cast<unsigned long long>(static_cast<unsigned>(v)) << 32 | bits;
  };
  {
    std::vector<long long> fo(ooff.begin(), ooff.end() - 1);
    if (c->weighted) okey.resize(arcs);
    for (long long i = 0; i < m; ++i) {
      const int u = g->src[i], v = g->dst[i];
      if (c->weighted) {
        okey[fo[u]] = pack(v, g->weight[i]);
        if (c->undirected) okey[fo[v]] = pack(u, g->weight[i]);
      }
      ocol[fo[u]++] = v;
      if (c->undirected) ocol[fo[v]++] = u;
    }
  }
  {
    // sort every out-row (host threads over row ranges of equal arc counts) and
    // look for repeated arcs
    const int nt = static_cast<int>(std::max(1u, std::min(16u, std::thread::hardware_concurrency())));
    std::vector<long long> bad(nt, -1);
    std::vector<std::thread> pool;
    long long row0 = 0;
    for (int t = 0; t < nt; ++t) {
      const long long goal = arcs * (t + 1) / nt;
      long long row1 = t == nt - 1 ? n : std::lower_bound(ooff.begin() + row0, ooff.end() - 1, goal) - ooff.begin();
      if (row1 < row0) row1 = row0;
      pool.emplace_back([&, t, row0, row1]() {
        for (long long u = row0; u < row1; ++u) {
          if (c->weighted) {
            std::sort(okey.begin() + ooff[u], okey.begin() + ooff[u + 1]);
            for (long long e = ooff[u]; e < ooff[u + 1]; ++e) ocol[e] = static_cast<int>(okey[e] >> 32);
          } else {
            std::sort(ocol.begin() + ooff[u], ocol.begin() + ooff[u + 1]);
          }
          for (long long e = ooff[u] + 1; e < ooff[u + 1]; ++e)
            if (ocol[e] == ocol[e - 1]) {
              bad[t] = u;
              return;
            }
        }
      });
      row0 = row1;
    }
    for (auto &th : pool) th.join();
    for (int t = 0; t < nt; ++t)
      if (bad[t] >= 0) {
        c->err = "ripple: repeated arc out of vertex " + std::to_string(bad[t]);
        return bail(RIPPLE_E_INVALID);
      }
  }
  {
    // stable over CSR order, so every in-row is sorted by source
    std::vector<long long> fi(ioff.begin(), ioff.end() - 1);
    if (c->weighted) {
      ow.resize(arcs);
      iw.resize(arcs);
      for (long long e = 0; e < arcs; ++e) {
        const unsigned bits = static_cast<unsigned>(okey[e] & 0xffffffffull);
        std::memcpy(&ow[e], &bits, sizeof(float));
      }
      std::vector<unsigned long long>().swap(okey);
    }
    for (long long u = 0; u < n; ++u)
      for (long long e = ooff[u]; e < ooff[u + 1]; ++e) {
        if (c->weighted) iw[fi[ocol[e]]] = ow[e];
        icol[fi[ocol[e]]++] = static_cast<int>(u);
      }
  }
  hipError_t e = hipSetDevice(c->device);
  if (e != hipSuccess) return bail(device_fail(c, e, "hipSetDevice"));
  if (g->stream != nullptr) {
    c->stream = static_cast<hipStream_t>(g->stream);
  } else {
    e = hipStreamCreateWithFlags(&c->stream, hipStreamNonBlocking);
    if (e != hipSuccess) return bail(device_fail(c, e, "hipStreamCreate"));
    c->own_stream = true;
  }
  ripple_status st;
  if ((st = dalloc_n(c, &c->d_persist, 1)) != RIPPLE_OK) return bail(st);
  if ((st = dalloc_n(c, &c->d_counters, 2)) != RIPPLE_OK) return bail(st);
  if ((st = dalloc_n(c, &c->d_in, 1)) != RIPPLE_OK) return bail(st);
  e = hipHostMalloc(reinterpret_cast<void **>(&c->h_counters), sizeof(rp::Counters), hipHostMallocDefault);
  if (e == hipSuccess) e = hipHostMalloc(reinterpret_cast<void **>(&c->h_in), sizeof(rp::BatchIn), hipHostMallocDefault);
  if (e != hipSuccess) return bail(device_fail(c, e, "hipHostMalloc"));
  *c->h_in = rp::BatchIn{};
  std::vector<int> olen(outdeg), ilen(indeg);
  c->snap_out = outdeg;
  c->snap_in = indeg;
  // hubs of half the long-row length or more: their rows may need the chunked sweep
  const int max_len = std::max(olen.empty() ? 0 : *std::max_element(olen.begin(), olen.end()),
                               ilen.empty() ? 0 : *std::max_element(ilen.begin(), ilen.end()));
  c->long_ok = max_len >= rp::kLongRow / 2 ? 1 : 0;
  if ((st = upload_adj(c, 0, olen, ocol, ooff, ow)) != RIPPLE_OK) return bail(st);
  if ((st = upload_adj(c, 1, ilen, icol, ioff, iw)) != RIPPLE_OK) return bail(st);
  // persistent per-vertex scratch
  const long long words = (n + 31) / 32;
  if ((st = dalloc_n(c, &c->fop, n)) != RIPPLE_OK) return bail(st);
  if ((st = dalloc_n(c, &c->ddeg, n)) != RIPPLE_OK) return bail(st);
  if ((st = dalloc_n(c, &c->bm_out, words)) != RIPPLE_OK) return bail(st);
  if ((st = dalloc_n(c, &c->bm_x, words)) != RIPPLE_OK) return bail(st);
  if ((st = dalloc_n(c, &c->compact_lb, rp::compact_scratch_words(n))) != RIPPLE_OK) return bail(st);
  if ((st = dalloc_n(c, &c->rl_blocksums, rp::relayout_blocks(n) + 1)) != RIPPLE_OK) return bail(st);
  if ((st = dalloc_n(c, &c->rl_off, n)) != RIPPLE_OK) return bail(st);
  if ((st = dalloc_n(c, &c->rl_cap, n)) != RIPPLE_OK) return bail(st);
  rp::launch_fill_i32(c->stream, c->fop, n, -1);
  e = hipMemsetAsync(c->ddeg, 0, n * sizeof(int), c->stream);
  if (e == hipSuccess) e = hipMemsetAsync(c->bm_out, 0, words * sizeof(unsigned), c->stream);
  if (e == hipSuccess) e = hipMemsetAsync(c->bm_x, 0, words * sizeof(unsigned), c->stream);
  if (e == hipSuccess)
    e = hipMemsetAsync(c->compact_lb, 0, rp::compact_scratch_words(n) * sizeof(rp::u64), c->stream);
  if (e == hipSuccess) e = hipMemsetAsync(c->d_counters, 0, 2 * sizeof(rp::Counters), c->stream);
  if (e == hipSuccess) e = hipGetLastError();
  if (e == hipSuccess) e = hipStreamSynchronize(c->stream);
  if (e != hipSuccess) return bail(device_fail(c, e, "load_graph init"));
  *out = c;
  return RIPPLE_OK;
}

namespace {

// x rounded to bf16, round to nearest even (NaN kept a quiet NaN), as raw bits.
unsigned short bf16_bits(float x) {
  unsigned u;
  std::memcpy(&u, &x, sizeof(u));
  if ((u & 0x7f800000u) == 0x7f800000u && (u & 0x007fffffu) != 0) return static_cast<unsigned short>((u >> 16) | 0x40);
  u += 0x7fffu + ((u >> 16) & 1u);
  return static_cast<unsigned short>(u >> 16);
}

// A device copy of host matrix w (count floats) rounded to bf16.
ripple_status upload_bf16(ripple_ctx *c, unsigned short **dst, const float *w, long long count) {
  std::vector<unsigned short> b(static_cast<size_t>(count));
  for (long long i = 0; i < count; ++i) b[i] = bf16_bits(w[i]);
  RP_TRY(dalloc_n(c, dst, count));
  RP_HIP(c, hipMemcpy(*dst, b.data(), static_cast<size_t>(count) * sizeof(unsigned short), hipMemcpyHostToDevice));
  return RIPPLE_OK;
}

}  // namespace

ripple_status ripple_init_embeddings(ripple_ctx *c, const float *x, const ripple_model_desc *md) {
  RP_TRY(check_ctx(c));
  if (x == nullptr || md == nullptr) return fail(c, RIPPLE_E_INVALID, "ripple: x and model must be non-NULL");
  drop_graphs(c);  // a new model changes the launches of every plan
  const int L = md->num_layers;
  if (L < 1 || L > rp::kMaxL) return fail(c, RIPPLE_E_INVALID, "ripple: num_layers out of range");
  if (md->agg < RIPPLE_AGG_SUM || md->agg > RIPPLE_AGG_GC_WSUM)
    return fail(c, RIPPLE_E_INVALID, "ripple: unknown aggregator");
  if (md->agg == RIPPLE_AGG_GC_WSUM && !c->weighted)
    return fail(c, RIPPLE_E_INVALID, "ripple: RIPPLE_AGG_GC_WSUM needs a graph loaded with weights");
  const bool sage = md->agg == RIPPLE_AGG_SUM || md->agg == RIPPLE_AGG_MEAN;
  const bool gin = md->agg == RIPPLE_AGG_GIN;
  if (!sage && md->agg != RIPPLE_AGG_GCN && md->transform_first == 1)
    return fail(c, RIPPLE_E_INVALID, "ripple: transform_first = 1 needs a GraphSAGE or GCN model");
  if (gin && md->w_out == nullptr) return fail(c, RIPPLE_E_INVALID, "ripple: w_out must be non-NULL for GIN");
  if (md->gemm_prec != RIPPLE_GEMM_FP32 && md->gemm_prec != RIPPLE_GEMM_BF16)
    return fail(c, RIPPLE_E_INVALID, "ripple: unknown gemm_prec");
  if (md->dims == nullptr || md->w_neigh == nullptr || md->relu == nullptr)
    return fail(c, RIPPLE_E_INVALID, "ripple: dims, w_neigh and relu must be non-NULL");
  if (sage && md->w_self == nullptr) return fail(c, RIPPLE_E_INVALID, "ripple: w_self must be non-NULL for GraphSAGE");
  for (int l = 0; l <= L; ++l)
    if (md->dims[l] < 1 || md->dims[l] > RIPPLE_MAX_DIM) return fail(c, RIPPLE_E_INVALID, "ripple: dim out of range");
  if (md->gemm_prec == RIPPLE_GEMM_BF16)  // every transform input is gathered in float4 chunks
    for (int l = 0; l < L + (md->agg == RIPPLE_AGG_GIN ? 1 : 0); ++l)
      if (md->dims[l] % 4 != 0)
        return fail(c, RIPPLE_E_INVALID,
                    "ripple: RIPPLE_GEMM_BF16 needs the widths of the transforms' inputs to be multiples of 4");
  for (int l = 0; l < L; ++l) {
    if (md->w_neigh[l] == nullptr || (sage && md->w_self[l] == nullptr) || (gin && md->w_out[l] == nullptr))
      return fail(c, RIPPLE_E_INVALID, "ripple: missing weight matrix");
  }
  if (md->transform_first < -1 || md->transform_first > 1)
    return fail(c, RIPPLE_E_INVALID, "ripple: transform_first must be -1, 0 or 1");
  free_model(c);
  c->L = L;
  c->agg = md->agg;
  c->gemm_bf16 = md->gemm_prec == RIPPLE_GEMM_BF16;
  for (int l = 0; l <= L; ++l) c->dims[l] = md->dims[l];
  c->dmax_delta = 0;
  for (int l = 0; l < L; ++l) c->dmax_delta = std::max(c->dmax_delta, c->dims[l]);
  const long long n = c->n;
  int msg_width = 0;
  for (int l = 1; l <= L; ++l) {
    const int dp = c->dims[l - 1], dn = c->dims[l];
    const long long arcs = c->arcs_loaded;
    c->tf[l] = (sage || md->agg == RIPPLE_AGG_GCN) &&
               (md->transform_first == 1 || (md->transform_first == -1 && dn < dp && arcs >= (1LL << 24)));
    c->sw[l] = c->tf[l] ? dn : dp;
    if (c->tf[l]) msg_width = std::max(msg_width, dn);
  }
  // weights. Plain layers: SAGE W = [W_self | W_neigh] (K = 2 d_{l-1}); GCN and
  // GraphConv W, GIN W1 (K = d_{l-1}). Transform-first layers: W = W_self (SAGE)
  // or W (GCN), K = d_{l-1}, plus W_neigh (GCN: W) for the messages and
  // corrections. GIN also keeps W2 [d_l][d_l] and b2.
  c->gin_eps1 = 1.0f + (gin ? md->gin_eps : 0.0f);
  for (int l = 1; l <= L; ++l) {
    const int dp = c->dims[l - 1], dn = c->dims[l];
    const int K = (!sage || c->tf[l]) ? dp : 2 * dp;
    c->K[l - 1] = K;
    c->relu[l - 1] = md->relu[l - 1] ? 1 : 0;
    const float *wmain = sage ? md->w_self[l - 1] : md->w_neigh[l - 1];
    std::vector<float> w(static_cast<size_t>(dn) * K);
    for (int j = 0; j < dn; ++j) {
      std::memcpy(&w[static_cast<size_t>(j) * K], wmain + static_cast<size_t>(j) * dp, dp * sizeof(float));
      if (K == 2 * dp)
        std::memcpy(&w[static_cast<size_t>(j) * K + dp], md->w_neigh[l - 1] + static_cast<size_t>(j) * dp,
                    dp * sizeof(float));
    }
    std::vector<float> b(dn, 0.0f);
    if (md->bias != nullptr && md->bias[l - 1] != nullptr) std::memcpy(b.data(), md->bias[l - 1], dn * sizeof(float));
    RP_TRY(dalloc_n(c, &c->W[l - 1], static_cast<long long>(dn) * K));
    RP_TRY(dalloc_n(c, &c->bias[l - 1], dn));
    RP_HIP(c, hipMemcpyAsync(c->W[l - 1], w.data(), w.size() * sizeof(float), hipMemcpyHostToDevice, c->stream));
    RP_HIP(c, hipMemcpyAsync(c->bias[l - 1], b.data(), dn * sizeof(float), hipMemcpyHostToDevice, c->stream));
    if (c->gemm_bf16) RP_TRY(upload_bf16(c, &c->Wb[l - 1], w.data(), static_cast<long long>(w.size())));
    if (c->tf[l]) {
      RP_TRY(dalloc_n(c, &c->Wn[l - 1], static_cast<long long>(dn) * dp));
      RP_HIP(c, hipMemcpyAsync(c->Wn[l - 1], md->w_neigh[l - 1], static_cast<size_t>(dn) * dp * sizeof(float),
                               hipMemcpyHostToDevice, c->stream));
      if (c->gemm_bf16) RP_TRY(upload_bf16(c, &c->Wnb[l - 1], md->w_neigh[l - 1], static_cast<long long>(dn) * dp));
    }
    if (gin) {
      std::vector<float> b2(dn, 0.0f);
      if (md->b_out != nullptr && md->b_out[l - 1] != nullptr) std::memcpy(b2.data(), md->b_out[l - 1], dn * sizeof(float));
      RP_TRY(dalloc_n(c, &c->W2[l - 1], static_cast<long long>(dn) * dn));
      RP_TRY(dalloc_n(c, &c->b2[l - 1], dn));
      RP_HIP(c, hipMemcpyAsync(c->W2[l - 1], md->w_out[l - 1], static_cast<size_t>(dn) * dn * sizeof(float),
                               hipMemcpyHostToDevice, c->stream));
      if (c->gemm_bf16) RP_TRY(upload_bf16(c, &c->W2b[l - 1], md->w_out[l - 1], static_cast<long long>(dn) * dn));
      RP_HIP(c, hipMemcpyAsync(c->b2[l - 1], b2.data(), dn * sizeof(float), hipMemcpyHostToDevice, c->stream));
    }
    RP_HIP(c, hipStreamSynchronize(c->stream));
  }
  for (int l = 0; l <= L; ++l) {
    // row tables get rp::kRowTail floats past their last row (see there)
    RP_TRY(dalloc_n(c, &c->H[l], n * c->dims[l] + rp::kRowTail));
    RP_TRY(dalloc_n(c, &c->lists[l], n));
    RP_TRY(dalloc_n(c, &c->doff[l], n + 1));
    if (l >= 1) RP_TRY(dalloc_n(c, &c->S[l], n * c->sw[l] + rp::kRowTail));
  }
  RP_TRY(dalloc_n(c, &c->delta[0], n * rp::row_ld(c->dmax_delta) + rp::kRowTail));
  RP_TRY(dalloc_n(c, &c->delta[1], n * rp::row_ld(c->dmax_delta) + rp::kRowTail));
  RP_TRY(dalloc_n(c, &c->ioff, n + 1));
  RP_TRY(dalloc_n(c, &c->flist_done, n));
  for (int k = 0; k < 2; ++k) {
    RP_TRY(dalloc_n(c, &c->memb[k], (n + 31) / 32));
  }
  if (msg_width > 0) RP_TRY(dalloc_n(c, &c->msg, n * rp::row_ld(msg_width) + rp::kRowTail));
  if (gin) {
    int dmax = 0;
    for (int l = 1; l <= L; ++l) dmax = std::max(dmax, c->dims[l]);
    RP_TRY(dalloc_n(c, &c->gin_rows, n * dmax));
  }
  for (int l = 1; l <= L; ++l)
    if (c->tf[l]) RP_TRY(dalloc_n(c, &c->P[l], n * c->dims[l] + rp::kRowTail));
  RP_HIP(c, hipMemcpyAsync(c->H[0], x, static_cast<size_t>(n) * c->dims[0] * sizeof(float), hipMemcpyHostToDevice,
                           c->stream));
  rp::Adj pull_adj = c->adj[1];  // arc weights only under the weighted-sum model
  if (c->agg != rp::kGcWsum) pull_adj.wt = nullptr;
  // bootstrap: layer-wise full forward pass. Plain layers pull the previous
  // layer's rows over the in-rows, then transform; transform-first layers
  // transform every row by W_neigh first and pull the narrower result.
  for (int l = 1; l <= L; ++l) {
    if (c->tf[l]) {
      rp::launch_gemm(c->stream, p_gemm_args(c, l, nullptr, nullptr, n, nullptr, nullptr), n, n);
      rp::launch_pull(c->stream, n, c->dims[l], c->agg, c->P[l], pull_adj, c->adj[0].len, c->S[l]);
    } else {
      rp::launch_pull(c->stream, n, c->dims[l - 1], c->agg, c->H[l - 1], pull_adj, c->adj[0].len, c->S[l]);
    }
    launch_layer_gemm(c, c->stream, l, nullptr, nullptr, n, nullptr, nullptr, n, n);
    RP_HIP(c, hipGetLastError());
  }
  RP_HIP(c, hipStreamSynchronize(c->stream));
  c->inited = true;
  c->has_batch = false;
  c->batches_done = 0;
  return RIPPLE_OK;
}

namespace {

// Runs one batch whose ops and feature rows the kernels read from src_ops /
// src_feat (pinned host or device memory). The kernels check every op again; a
// batch they reject is invalid, reported from caller_ops (the caller's device
// copy; nullptr when src_ops is the pinned host copy), and nothing was mutated.
ripple_status run_batch(ripple_ctx *c, int B, long long num_feat_rows, const ripple_op *src_ops,
                        const float *src_feat, const ripple_op *caller_ops, ripple_batch_stats *stats) {
  long long repacks = 0;
  // the previous call has synchronised, so no kernel still reads the block
  c->h_in->ops = src_ops;
  c->h_in->feat = src_feat;
  c->h_in->num_ops = B;
  c->h_in->num_feat_rows = num_feat_rows;
  if (!c->has_batch) {
    // the first batch's plan estimates its frontiers from its ops (see
    // first_batch_counts): a batch in device memory is copied to host once
    if (caller_ops == nullptr) {
      c->plan_ops = src_ops;
    } else {
      c->plan_buf.resize(static_cast<size_t>(B));
      if (B > 0)
        RP_HIP(c, hipMemcpy(c->plan_buf.data(), caller_ops, static_cast<size_t>(B) * sizeof(ripple_op),
                            hipMemcpyDeviceToHost));
      c->plan_ops = c->plan_buf.data();
    }
  }
  for (int attempt = 0;; ++attempt) {
    RP_TRY(launch_batch(c));
    RP_TRY(wait_stream(c));
    if (c->h_counters->bad_op) {
      // rejected on the device before anything was mutated: name the first bad op
      c->ev_log.clear();
      c->ev_used = 0;
      const long long i = B - static_cast<long long>(c->h_counters->bad_op);
      ripple_op o{};
      if (caller_ops != nullptr)
        RP_HIP(c, hipMemcpy(&o, caller_ops + i, sizeof(o), hipMemcpyDeviceToHost));
      else
        o = src_ops[i];  // the batch came through pinned host memory
      if (validate_ops(c, &o, 1, num_feat_rows)) c->err = "ripple: op 0: failed the device-side check";
      const size_t at = c->err.find("op 0:");
      if (at != std::string::npos) c->err.replace(at, 5, "op " + std::to_string(i) + ":");
      return RIPPLE_E_INVALID;
    }
    if (!c->h_counters->abort) break;
    // the spare arena cannot take this batch's row moves: nothing was mutated
    c->ev_log.clear();
    c->ev_used = 0;
    if (attempt >= 2) {
      c->poisoned = true;
      return fail(c, RIPPLE_E_DEVICE, "ripple: adjacency re-layout did not make room for the batch");
    }
    RP_TRY(repack_adj(c, 0));
    RP_TRY(repack_adj(c, 1));
    ++repacks;
  }
  rp::Counters &k = *c->h_counters;
  // lists built by a scatter keep their count and out-arc total in one word
  for (int l = 1; l <= c->L; ++l) {
    if (!(c->run_app >> l & 1)) continue;
    k.count[l] = k.app[l] >> rp::kAppShift;
    if (l < c->L) k.pushed[l + 1] = k.app[l] & rp::kAppMask;
    k.dest[l] = k.app_sinks[l] >> rp::kAppShift;
    k.indeg[l] = k.app_sinks[l] & rp::kAppMask;
  }
  if (c->debug_fail_batch > 0 && ++c->batches_checked == c->debug_fail_batch) k.err |= 16ull;
  if (k.err) {
    c->poisoned = true;
    // bit 0: a net-deleted arc was not found; bit 1: a rewritten row's length did not
    // match; bit 2: the compaction's wait for a predecessor tile timed out; bit 3: a
    // row move would have ended past the column buffer; bit 4: set by the test hook
    return fail(c, RIPPLE_E_DEVICE, "ripple: device-side check failed (err bits " + std::to_string(k.err) + ")");
  }
  c->last_app = c->run_app;  // the lists now hold this batch's sets
  c->arcs_now += static_cast<long long>(k.n_ins) - static_cast<long long>(k.n_del);
  for (int d = 0; d < 2; ++d) {
    c->row_max[d] = std::max(c->row_max[d], static_cast<long long>(k.maxlen[d]));
    if (k.top_end[d] != 0) c->arena_top[d] = static_cast<long long>(k.top_end[d]);
  }
  account_phases(c);
  c->has_batch = true;
  ++c->batches_done;
  c->plan_ops = nullptr;
  c->last_nfeat = static_cast<long long>(k.n_feat);
  for (int l = 0; l <= c->L; ++l) {
    c->last_count[l] = static_cast<long long>(k.count[l]);
    c->last_pushed[l] = static_cast<long long>(k.pushed[l]);
    c->last_in[l] = static_cast<long long>(k.indeg[l]);
  }
  if (stats != nullptr) {
    std::memset(stats, 0, sizeof(*stats));
    stats->num_ops = B;
    stats->edge_keys = static_cast<int64_t>(k.edge_keys);
    stats->noop_edge_ops = static_cast<int64_t>(k.noop_edge);
    stats->ins_arcs = static_cast<int64_t>(k.n_ins - k.n_rew);
    stats->del_arcs = static_cast<int64_t>(k.n_del - k.n_rew);
    stats->reweighted_arcs = static_cast<int64_t>(k.n_rew);
    stats->features = static_cast<int64_t>(k.n_feat);
    stats->affected[0] = static_cast<int64_t>(k.n_feat);
    for (int l = 1; l <= c->L; ++l) {
      stats->dirty[l] = static_cast<int64_t>(k.count[l - 1]);
      stats->affected[l] = static_cast<int64_t>(k.count[l]);
      stats->pushed_arcs[l] = static_cast<int64_t>(k.pushed[l]);
      stats->dest_rows[l] = static_cast<int64_t>(k.dest[l]);
    }
    stats->relocated_rows = static_cast<int64_t>(k.n_reloc);
    stats->repacks = repacks;
    for (int l = 1; l <= c->L; ++l) stats->in_arcs[l] = static_cast<int64_t>(k.indeg[l]);
    stats->pull_layers = c->last_pull;
    stats->dense_layers = c->last_dense;
    stats->recompute_layers = c->last_recompute;
    stats->bucket_layers = c->last_bucket;
    stats->graph_replay = c->last_graph ? 1 : 0;
    stats->long_rows = static_cast<int64_t>(k.long_rows >> 40);
  }
  return RIPPLE_OK;
}

// True if [p, p + bytes) lies inside one device allocation of the context's
// device. Allocations already seen are remembered (the runtime query costs
// microseconds, and callers reuse their buffers), so a repeat check is a lookup.
// This refuses host pointers; it cannot tell a freed device range.
bool device_range(ripple_ctx *c, const void *p, long long bytes) {
  if (p == nullptr || bytes <= 0) return true;
  const uintptr_t lo = reinterpret_cast<uintptr_t>(p), hi = lo + static_cast<uintptr_t>(bytes);
  for (const auto &r : c->dev_ranges)
    if (lo >= r.first && hi <= r.second) return true;
  hipPointerAttribute_t at{};
  if (hipPointerGetAttributes(&at, p) != hipSuccess || at.type != hipMemoryTypeDevice || at.device != c->device) {
    (void)hipGetLastError();
    return false;
  }
  void *base = nullptr;
  size_t size = 0;
  if (hipMemGetAddressRange(reinterpret_cast<hipDeviceptr_t *>(&base), &size, const_cast<void *>(p)) != hipSuccess) {
    (void)hipGetLastError();
    return false;
  }
  const uintptr_t b = reinterpret_cast<uintptr_t>(base);
  if (hi > b + size) return false;
  if (c->dev_ranges.size() >= 64) c->dev_ranges.erase(c->dev_ranges.begin());
  c->dev_ranges.emplace_back(b, b + size);
  return true;
}

ripple_status check_batch_args(ripple_ctx *c, const ripple_op *ops, int64_t num_ops, const float *feat_rows,
                               int64_t num_feat_rows) {
  RP_TRY(check_ctx(c));
  if (!c->inited) return fail(c, RIPPLE_E_STATE, "ripple: ripple_init_embeddings has not run");
  if (num_ops < 0 || num_feat_rows < 0) return fail(c, RIPPLE_E_INVALID, "ripple: negative count");
  if (num_ops > (1LL << 26)) return fail(c, RIPPLE_E_INVALID, "ripple: batch larger than 2^26 ops");
  if (num_ops > 0 && ops == nullptr) return fail(c, RIPPLE_E_INVALID, "ripple: ops is NULL");
  if (num_feat_rows > 0 && feat_rows == nullptr) return fail(c, RIPPLE_E_INVALID, "ripple: feat_rows is NULL");
  return RIPPLE_OK;
}

}  // namespace

ripple_status ripple_apply_updates(ripple_ctx *c, const ripple_op *ops, int64_t num_ops, const float *feat_rows,
                                   int64_t num_feat_rows, ripple_batch_stats *stats) {
  RP_TRY(check_batch_args(c, ops, num_ops, feat_rows, num_feat_rows));
  if (!validate_ops(c, ops, num_ops, num_feat_rows)) return RIPPLE_E_INVALID;
  RP_TRY(ensure_batch_scratch(c, num_ops, num_feat_rows));
  // the kernels read the batch straight from these pinned buffers (the previous
  // call has synchronised, so nothing still reads them)
  const int B = static_cast<int>(num_ops);
  if (B > 0) std::memcpy(c->h_ops, ops, static_cast<size_t>(B) * sizeof(ripple_op));
  if (num_feat_rows > 0)
    std::memcpy(c->h_feat, feat_rows, static_cast<size_t>(num_feat_rows) * c->dims[0] * sizeof(float));
  return run_batch(c, B, num_feat_rows, c->h_ops, c->h_feat, nullptr, stats);
}

ripple_status ripple_apply_updates_device(ripple_ctx *c, const ripple_op *ops, int64_t num_ops,
                                          const float *feat_rows, int64_t num_feat_rows, ripple_batch_stats *stats) {
  RP_TRY(check_batch_args(c, ops, num_ops, feat_rows, num_feat_rows));
  if (!device_range(c, ops, num_ops * sizeof(ripple_op)) ||
      !device_range(c, feat_rows, num_feat_rows * c->dims[0] * sizeof(float)))
    return fail(c, RIPPLE_E_INVALID, "ripple: ops / feat_rows must be device memory of the context's device");
  RP_TRY(ensure_batch_scratch(c, num_ops, num_feat_rows));
  return run_batch(c, static_cast<int>(num_ops), num_feat_rows, ops, feat_rows, ops, stats);
}

ripple_status ripple_get_embeddings(ripple_ctx *c, int32_t layer, const int32_t *ids, int64_t count, float *out) {
  RP_TRY(check_ctx(c));
  if (!c->inited) return fail(c, RIPPLE_E_STATE, "ripple: ripple_init_embeddings has not run");
  if (layer < 0 || layer > c->L) return fail(c, RIPPLE_E_INVALID, "ripple: layer out of range");
  return read_rows(c, c->H[layer], c->dims[layer], ids, count, out);
}

ripple_status ripple_get_embeddings_static(ripple_ctx *c, int32_t layer, const int32_t *ids, int64_t count,
                                           float *out) {
  RP_TRY(check_ctx(c));
  if (!c->inited) return fail(c, RIPPLE_E_STATE, "ripple: ripple_init_embeddings has not run");
  if (layer < 0 || layer > c->L) return fail(c, RIPPLE_E_INVALID, "ripple: layer out of range");
  if (count < 0) return fail(c, RIPPLE_E_INVALID, "ripple: negative count");
  if (count == 0) return RIPPLE_OK;
  if (out == nullptr) return fail(c, RIPPLE_E_INVALID, "ripple: out is NULL");
  const int d = c->dims[layer];
  if (ids == nullptr) {  // every row, straight from the embedding buffer
    if (count != c->n) return fail(c, RIPPLE_E_INVALID, "ripple: ids NULL requires count == n");
    RP_HIP(c, hipMemcpyAsync(out, c->H[layer], static_cast<size_t>(count) * d * sizeof(float),
                             hipMemcpyDeviceToHost, c->stream));
    RP_HIP(c, hipStreamSynchronize(c->stream));
    return RIPPLE_OK;
  }
  const size_t id_bytes = (static_cast<size_t>(count) * sizeof(int) + 255) / 256 * 256;
  const size_t row_bytes = static_cast<size_t>(count) * d * sizeof(float);
  if (id_bytes + row_bytes > kStaticStageBytes)
    return fail(c, RIPPLE_E_INVALID, "ripple: " + std::to_string(count) + " rows of width " + std::to_string(d) +
                                         " exceed the " + std::to_string(kStaticStageBytes >> 20) +
                                         " MiB staging array of ripple_get_embeddings_static");
  for (long long i = 0; i < count; ++i)
    if (ids[i] < 0 || ids[i] >= c->n) return fail(c, RIPPLE_E_INVALID, "ripple: vertex id out of range");
  void *stage = nullptr;
  RP_HIP(c, static_stage(c->device, &stage));
  int *d_ids = static_cast<int *>(stage);
  float *d_out = reinterpret_cast<float *>(static_cast<unsigned char *>(stage) + id_bytes);
  RP_HIP(c, hipMemcpyAsync(d_ids, ids, static_cast<size_t>(count) * sizeof(int), hipMemcpyHostToDevice, c->stream));
  rp::launch_gather_rows(c->stream, c->H[layer], d, d_ids, count, d_out);
  RP_HIP(c, hipGetLastError());
  RP_HIP(c, hipMemcpyAsync(out, d_out, row_bytes, hipMemcpyDeviceToHost, c->stream));
  RP_HIP(c, hipStreamSynchronize(c->stream));
  return RIPPLE_OK;
}

ripple_status ripple_get_aggregates(ripple_ctx *c, int32_t layer, const int32_t *ids, int64_t count, float *out,
                                    int32_t *width) {
  RP_TRY(check_ctx(c));
  if (!c->inited) return fail(c, RIPPLE_E_STATE, "ripple: ripple_init_embeddings has not run");
  if (layer < 1 || layer > c->L) return fail(c, RIPPLE_E_INVALID, "ripple: layer out of range");
  if (width != nullptr) *width = c->sw[layer];
  return read_rows(c, c->S[layer], c->sw[layer], ids, count, out);
}

ripple_status ripple_get_affected(ripple_ctx *c, int32_t layer, int32_t *ids, int64_t capacity, int64_t *count) {
  RP_TRY(check_ctx(c));
  if (count == nullptr) return fail(c, RIPPLE_E_INVALID, "ripple: count is NULL");
  *count = 0;
  if (!c->inited) return fail(c, RIPPLE_E_STATE, "ripple: ripple_init_embeddings has not run");
  if (layer < 0 || layer > c->L) return fail(c, RIPPLE_E_INVALID, "ripple: layer out of range");
  if (capacity < 0 || (capacity > 0 && ids == nullptr)) return fail(c, RIPPLE_E_INVALID, "ripple: bad ids buffer");
  if (!c->has_batch) return RIPPLE_OK;
  if (layer == 0) {
    const long long nf = c->last_nfeat;
    std::vector<int> f(nf);
    if (nf > 0) {
      RP_HIP(c, hipMemcpyAsync(f.data(), c->flist_done, nf * sizeof(int), hipMemcpyDeviceToHost, c->stream));
      RP_HIP(c, hipStreamSynchronize(c->stream));
    }
    std::sort(f.begin(), f.end());
    *count = nf;
    const long long w = std::min<long long>(nf, capacity);
    if (w > 0) std::memcpy(ids, f.data(), w * sizeof(int));
    return RIPPLE_OK;
  }
  const long long cnt = c->last_count[layer];
  *count = cnt;
  const long long w = std::min<long long>(cnt, capacity);
  if (c->last_app >> layer & 1) {
    // listed by its scatter in no particular order: sort the whole list
    std::vector<int> all(cnt);
    if (cnt > 0) {
      RP_HIP(c, hipMemcpyAsync(all.data(), c->lists[layer], cnt * sizeof(int), hipMemcpyDeviceToHost, c->stream));
      RP_HIP(c, hipStreamSynchronize(c->stream));
    }
    std::sort(all.begin(), all.end());
    if (w > 0) std::memcpy(ids, all.data(), w * sizeof(int));
    return RIPPLE_OK;
  }
  if (w > 0) {
    RP_HIP(c, hipMemcpyAsync(ids, c->lists[layer], w * sizeof(int), hipMemcpyDeviceToHost, c->stream));
    RP_HIP(c, hipStreamSynchronize(c->stream));
  }
  return RIPPLE_OK;
}

ripple_status ripple_get_arcs(ripple_ctx *c, int32_t direction, int32_t *src, int32_t *dst, int64_t capacity,
                              int64_t *count) {
  RP_TRY(check_ctx(c));
  if (count == nullptr) return fail(c, RIPPLE_E_INVALID, "ripple: count is NULL");
  *count = 0;
  if (direction != 0 && direction != 1) return fail(c, RIPPLE_E_INVALID, "ripple: direction must be 0 or 1");
  if (capacity < 0 || (capacity > 0 && (src == nullptr || dst == nullptr)))
    return fail(c, RIPPLE_E_INVALID, "ripple: bad output buffers");
  const long long n = c->n;
  const rp::Adj &a = c->adj[direction];
  std::vector<long long> off(n);
  std::vector<int> len(n);
  std::vector<int> col(c->col_capacity[direction]);
  RP_HIP(c, hipMemcpyAsync(off.data(), a.off, n * sizeof(long long), hipMemcpyDeviceToHost, c->stream));
  RP_HIP(c, hipMemcpyAsync(len.data(), a.len, n * sizeof(int), hipMemcpyDeviceToHost, c->stream));
  RP_HIP(c, hipMemcpyAsync(col.data(), a.col, col.size() * sizeof(int), hipMemcpyDeviceToHost, c->stream));
  RP_HIP(c, hipStreamSynchronize(c->stream));
  long long k = 0;
  for (long long u = 0; u < n; ++u) {
    for (int e = 0; e < len[u]; ++e, ++k) {
      if (k < capacity) {
        const int w = col[off[u] + e];
        src[k] = direction == 0 ? static_cast<int>(u) : w;
        dst[k] = direction == 0 ? w : static_cast<int>(u);
      }
    }
  }
  *count = k;
  return RIPPLE_OK;
}

ripple_status ripple_get_arc_weights(ripple_ctx *c, int32_t direction, float *weights, int64_t capacity,
                                     int64_t *count) {
  RP_TRY(check_ctx(c));
  if (count == nullptr) return fail(c, RIPPLE_E_INVALID, "ripple: count is NULL");
  *count = 0;
  if (!c->weighted) return fail(c, RIPPLE_E_INVALID, "ripple: the graph has no weights");
  if (direction != 0 && direction != 1) return fail(c, RIPPLE_E_INVALID, "ripple: direction must be 0 or 1");
  if (capacity < 0 || (capacity > 0 && weights == nullptr)) return fail(c, RIPPLE_E_INVALID, "ripple: bad output buffer");
  const long long n = c->n;
  const rp::Adj &a = c->adj[direction];
  std::vector<long long> off(n);
  std::vector<int> len(n);
  std::vector<float> wt(c->col_capacity[direction]);
  RP_HIP(c, hipMemcpyAsync(off.data(), a.off, n * sizeof(long long), hipMemcpyDeviceToHost, c->stream));
  RP_HIP(c, hipMemcpyAsync(len.data(), a.len, n * sizeof(int), hipMemcpyDeviceToHost, c->stream));
  RP_HIP(c, hipMemcpyAsync(wt.data(), a.wt, wt.size() * sizeof(float), hipMemcpyDeviceToHost, c->stream));
  RP_HIP(c, hipStreamSynchronize(c->stream));
  long long k = 0;
  for (long long u = 0; u < n; ++u)
    for (int e = 0; e < len[u]; ++e, ++k)
      if (k < capacity) weights[k] = wt[off[u] + e];
  *count = k;
  return RIPPLE_OK;
}

ripple_status ripple_set_scatter_mode(ripple_ctx *c, int32_t mode) {
  RP_TRY(check_ctx(c));
  if (mode < RIPPLE_SCATTER_AUTO || mode > RIPPLE_SCATTER_BUCKET) return fail(c, RIPPLE_E_INVALID, "ripple: bad mode");
  c->scatter_mode = mode;
  return RIPPLE_OK;
}

ripple_status ripple_set_reanchor(ripple_ctx *c, int64_t every) {
  RP_TRY(check_ctx(c));
  if (every < 0) return fail(c, RIPPLE_E_INVALID, "ripple: every must be >= 0");
  c->reanchor_every = every;
  return RIPPLE_OK;
}

ripple_status ripple_set_graphs(ripple_ctx *c, int32_t enable) {
  RP_TRY(check_ctx(c));
  if (enable != 0 && enable != 1) return fail(c, RIPPLE_E_INVALID, "ripple: enable must be 0 or 1");
  c->use_graphs = enable == 1;
  if (!c->use_graphs) drop_graphs(c);
  return RIPPLE_OK;
}

ripple_status ripple_device_bytes(ripple_ctx *c, int64_t *bytes) {
  if (c == nullptr || bytes == nullptr) return RIPPLE_E_INVALID;
  *bytes = c->bytes;
  return RIPPLE_OK;
}

ripple_status ripple_set_profiling(ripple_ctx *c, int32_t mask) {
  RP_TRY(check_ctx(c));
  c->prof_mask = static_cast<unsigned>(mask) & ((1u << RIPPLE_NUM_PHASES) - 1u);
  c->prof = c->prof_mask != 0;
  // create the events now so that the first recorded batch does not pay for it
  const size_t want = 2 * (8 + 8 * static_cast<size_t>(rp::kMaxL));  // every timed launch of a batch
  while (c->prof && c->ev_pool.size() < want) {
    hipEvent_t e;
    RP_HIP(c, hipEventCreate(&e));
    c->ev_pool.push_back(e);
  }
  c->ev_log.clear();
  c->ev_used = 0;
  return RIPPLE_OK;
}

ripple_status ripple_get_phase_stats(ripple_ctx *c, ripple_phase_stats *out, int32_t capacity) {
  RP_TRY(check_ctx(c));
  if (capacity < 0 || (capacity > 0 && out == nullptr)) return fail(c, RIPPLE_E_INVALID, "ripple: bad buffer");
  for (int p = 0; p < RIPPLE_NUM_PHASES && p < capacity; ++p) {
    out[p].ms = c->ph_ms[p];
    out[p].launches = c->ph_launch[p];
    out[p].bytes = c->ph_bytes[p];
    out[p].bytes_no_reuse = c->ph_bytes[p] + c->ph_extra[p];
    out[p].flops = c->ph_flops[p];
  }
  for (int p = 0; p < RIPPLE_NUM_PHASES; ++p) {
    c->ph_ms[p] = 0.0;
    c->ph_launch[p] = 0;
    c->ph_bytes[p] = 0.0;
    c->ph_extra[p] = 0.0;
    c->ph_flops[p] = 0.0;
  }
  return RIPPLE_OK;
}

const char *ripple_phase_name(int32_t phase) {
  static const char *names[RIPPLE_NUM_PHASES] = {"net", "topo", "layer0", "scatter", "compact", "gemm", "other",
                                                 "total"};
  if (phase < 0 || phase >= RIPPLE_NUM_PHASES) return "";
  return names[phase];
}

const char *ripple_last_error(const ripple_ctx *c) {
  if (c == nullptr) return g_load_err.empty() ? kNullCtxMsg : g_load_err.c_str();
  return c->err.c_str();
}

void ripple_destroy(ripple_ctx *c) {
  if (c == nullptr) return;
  (void)hipSetDevice(c->device);
  if (c->stream) (void)hipStreamSynchronize(c->stream);
  drop_graphs(c);
  for (hipEvent_t e : c->ev_pool) (void)hipEventDestroy(e);
  free_model(c);
  for (int d = 0; d < 2; ++d) {
    dfree_t(c, c->adj[d].off);
    dfree_t(c, c->adj[d].len);
    dfree_t(c, c->adj[d].cap);
    dfree_t(c, c->adj[d].col);
    dfree_t(c, c->col_alt[d]);
    dfree_t(c, c->adj[d].wt);
    dfree_t(c, c->wt_alt[d]);
    dfree_t(c, c->adj[d].inscnt);
    dfree_t(c, c->adj[d].delcnt);
  }
  dfree_t(c, c->fop);
  dfree_t(c, c->ddeg);
  dfree_t(c, c->bm_out);
  dfree_t(c, c->bm_x);
  dfree_t(c, c->compact_lb);
  dfree_t(c, c->rl_blocksums);
  dfree_t(c, c->rl_off);
  dfree_t(c, c->rl_cap);
  dfree_t(c, c->d_counters);
  dfree_t(c, c->d_persist);
  dfree_t(c, c->d_in);
  if (c->h_counters) (void)hipHostFree(c->h_counters);
  if (c->h_in) (void)hipHostFree(c->h_in);
  if (c->own_stream && c->stream) (void)hipStreamDestroy(c->stream);
  delete c;
}

}  // extern "C"
