// Batch netting and the dynamic adjacency update.
//
// Netting (sequential semantics of a batch): an insert sets an arc present and a
// delete sets it absent, so the last op naming an edge decides its final state.
// One pass hashes every edge op and keeps the largest op index per edge; a second
// pass lets each winning op compare the final state with the pre-batch adjacency,
// emit the net inserted / deleted arcs, tag the edge's hash slot (+1 insert,
// -1 delete) and take a rank among its rows' inserts or deletes. The last feature
// write per vertex is found the same way with a per-vertex atomicMax. Batches of
// up to kNetDirectMax ops are netted in one pass instead: each op is compared with
// every later op, and only net-deleted keys are hashed (for the row rewrite).
//
// Adjacency update: row slots are [off, off+cap), the first len used, in no
// particular order. A plan pass sums the spare-arena slots that growing rows need
// and the last block to finish checks them against the arena: a batch that does
// not fit is aborted before anything is mutated (the host then re-lays the rows
// out and runs the batch again). The host leaves the plan out when the free arena
// holds every move the batch could cause. Then one owner wave per touched row
// drops its net-deleted entries (hash lookups; a lone delete is found by a search
// and swap-removed), moves the row to the arena if it must grow, and sets the new
// length; finally every insert is written at its rank.
#include "internal.h"

namespace rp {

namespace {

__device__ inline unsigned hash_slot(u64 key, unsigned mask) {
  key *= 0x9E3779B97F4A7C15ull;
  return static_cast<unsigned>(key >> 33) & mask;
}

__device__ inline int lane_id() { return threadIdx.x & (kWave - 1); }

__device__ inline long long global_wave() {
  return (static_cast<long long>(blockIdx.x) * blockDim.x + threadIdx.x) / kWave;
}

__device__ inline long long num_waves() {
  return static_cast<long long>(gridDim.x) * blockDim.x / kWave;
}

__device__ inline u64 edge_key(int a, int b, int undirected, long long n) {
  if (undirected && a > b) {
    const int t = a;
    a = b;
    b = t;
  }
  return static_cast<u64>(a) * static_cast<u64>(n) + static_cast<u64>(b);
}

// Position of `target` in row[0, len) or -1; all lanes of the wave get the answer.
// Reads kFindU entries per lane per round, all in flight together, so a row of up
// to 1024 entries costs one round trip.
constexpr int kFindU = 16;

__device__ inline int wave_find(const int *row, int len, int target) {
  const int lane = lane_id();
  for (int base = 0; base < len; base += kWave * kFindU) {
    int x[kFindU];
#pragma unroll
    for (int u = 0; u < kFindU; ++u) {
      const int e = base + u * kWave + lane;
      x[u] = e < len ? row[e] : -1;
    }
#pragma unroll
    for (int u = 0; u < kFindU; ++u) {
      const u64 m = __ballot(x[u] == target);
      if (m) return base + u * kWave + __ffsll(static_cast<long long>(m)) - 1;
    }
  }
  return -1;
}

__device__ inline int lanes_below(u64 mask) {
  return static_cast<int>(__builtin_amdgcn_mbcnt_hi(static_cast<unsigned>(mask >> 32),
                                                    __builtin_amdgcn_mbcnt_lo(static_cast<unsigned>(mask), 0u)));
}

__device__ inline int grow_cap(int newlen) {
  const long long g = static_cast<long long>(newlen) + newlen / 2 + 4;
  return static_cast<int>(((g + 3) / 4) * 4);
}

// Work items over arcs x directions: item w -> arc w >> 1, direction w & 1.
// Direction 0 (out-adjacency): row = src, entry = dst; direction 1: row = dst, entry = src.
__device__ inline void item_row(long long w, const int *src, const int *dst, int &dir, int &row, int &entry) {
  const long long arc = w >> 1;
  dir = static_cast<int>(w & 1);
  row = dir == 0 ? src[arc] : dst[arc];
  entry = dir == 0 ? dst[arc] : src[arc];
}

// Takes the batch's inputs from `now` (a launch for this batch alone) or, when
// host_in is set (a launch replayed for later batches), from pinned host memory
// at system scope (the host rewrites them before every replay, so no cached copy
// may be used); hands them to the later kernels in dev_in, and keeps a device
// copy of the ops.
__global__ void k_net_hash(const BatchIn *host_in, BatchIn now, BatchIn *dev_in, ripple_op *ops, int undirected,
                           int weighted, long long n, u64 *ht_key, int *ht_val, unsigned mask, int *op_slot, int *fop,
                           Counters *c) {
  if (host_in != nullptr) {
    const auto word = [&](const void *f) {
      return __hip_atomic_load(static_cast<const u64 *>(f), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_SYSTEM);
    };
    now.ops = reinterpret_cast<const ripple_op *>(word(&host_in->ops));
    now.feat = reinterpret_cast<const float *>(word(&host_in->feat));
    now.num_ops = static_cast<long long>(word(&host_in->num_ops));
    now.num_feat_rows = static_cast<long long>(word(&host_in->num_feat_rows));
  }
  const ripple_op *src_ops = now.ops;
  const long long B = now.num_ops;
  const long long num_feat_rows = now.num_feat_rows;
  const int i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i == 0) *dev_in = now;
  if (i >= B) return;
  ripple_op op = src_ops[i];
  // the same checks as the host's: an op that fails them aborts the batch before
  // anything is mutated, and is replaced by a harmless self-loop so that no kernel
  // indexes with its fields
  bool bad;
  if (op.kind == RIPPLE_OP_INSERT || op.kind == RIPPLE_OP_DELETE)
    bad = op.u < 0 || op.u >= n || op.v < 0 || op.v >= n ||
          (weighted && op.kind == RIPPLE_OP_INSERT && !isfinite(op.weight));
  else if (op.kind == RIPPLE_OP_FEATURE)
    bad = op.u < 0 || op.u >= n || op.feat_row < 0 || op.feat_row >= num_feat_rows;
  else
    bad = true;
  if (bad) {
    atomicMax(&c->bad_op, static_cast<u64>(B - i));
    c->abort = 1;
    op = ripple_op{RIPPLE_OP_INSERT, 0, 0, -1};
  }
  ops[i] = op;
  if (op.kind == RIPPLE_OP_FEATURE) {
    atomicMax(&fop[op.u], i);
    op_slot[i] = -1;
    return;
  }
  if (op.u == op.v) {
    atomicAdd(&c->noop_edge, 1ull);
    op_slot[i] = -1;
    return;
  }
  const u64 key = edge_key(op.u, op.v, undirected, n);
  unsigned s = hash_slot(key, mask);
  while (true) {
    const u64 prev = atomicCAS(&ht_key[s], kEmptyKey, key);
    if (prev == kEmptyKey || prev == key) break;
    s = (s + 1) & mask;
  }
  atomicMax(&ht_val[s], i);
  op_slot[i] = static_cast<int>(s);
}

// The decision of edge (a, b)'s deciding op (a <= b on undirected graphs; a's
// out-row and b's in-row have lengths la, lb and offsets oa, ob): is the edge present
// before the batch (searched in the shorter row), and then either a no-op or the net
// arcs with their ranks among their rows' inserts or deletes. Returns the edge's net
// change on every lane: +1 inserted, -1 deleted or reweighted, 0 none.
// ht_key != nullptr: a net-deleted key is also entered into the hash table, its
// slot tagged -1 in ht_net and written to *slot (-1 otherwise); the first probe
// goes out with the emission's atomics.
__device__ inline int emit_edge(const ripple_op &op, int a, int b, int la, int lb, long long oa, long long ob,
                                int undirected, Adj out, Adj in, int *ins_src, int *ins_dst, int *del_src,
                                int *del_dst, int *ins_rank, int *del_rank, float *ins_w, float *del_w, Counters *c,
                                u64 *ht_key = nullptr, int *ht_net = nullptr, unsigned mask = 0, u64 key = 0,
                                int *slot = nullptr) {
  const int lane = lane_id();
  const bool use_out = la <= lb;
  const long long row0 = use_out ? oa : ob;
  const int pos = wave_find((use_out ? out.col : in.col) + row0, use_out ? la : lb, use_out ? b : a);
  const bool present = pos >= 0;
  const bool want = op.kind == RIPPLE_OP_INSERT;
  const bool weighted = out.wt != nullptr;
  const float w_old = weighted && present ? (use_out ? out.wt : in.wt)[row0 + pos] : 1.0f;
  const float w_new = weighted ? op.weight : 1.0f;
  const bool reweight = want && present && w_old != w_new;
  const bool noop = want == present && !reweight;
  const int net = noop ? 0 : want && !reweight ? 1 : -1;
  const bool probe = ht_key != nullptr && net == -1;
  unsigned sl = 0;
  u64 prev = kEmptyKey;
  if (lane == 0 && probe) {
    sl = hash_slot(key, mask);
    prev = atomicCAS(&ht_key[sl], kEmptyKey, key);
  }
  if (lane == 0) {
    atomicAdd(&c->edge_keys, 1ull);
    if (noop) {
      atomicAdd(&c->noop_edge, 1ull);
    } else {
      // a reweight drops the old entry (as a delete) and puts the arc back with its
      // new weight (as an insert)
      const int narcs = undirected ? 2 : 1;
      if (reweight) atomicAdd(&c->n_rew, static_cast<u64>(narcs));
      for (int kind = 0; kind < 2; ++kind) {  // 0: delete item, 1: insert item
        if (kind == 0 ? !present : !want) continue;
        const bool ins = kind == 1;
        int *ps = ins ? ins_src : del_src;
        int *pd = ins ? ins_dst : del_dst;
        int *rank = ins ? ins_rank : del_rank;
        const u64 j = atomicAdd(ins ? &c->n_ins : &c->n_del, static_cast<u64>(narcs));
        for (int t = 0; t < narcs; ++t) {
          const int su = t == 0 ? a : b, sv = t == 0 ? b : a;
          ps[j + t] = su;
          pd[j + t] = sv;
          (ins ? ins_w : del_w)[j + t] = ins ? w_new : w_old;
          rank[2 * (j + t)] = atomicAdd(ins ? &out.inscnt[su] : &out.delcnt[su], 1);
          rank[2 * (j + t) + 1] = atomicAdd(ins ? &in.inscnt[sv] : &in.delcnt[sv], 1);
        }
      }
    }
    if (ht_key != nullptr) {
      if (probe) {  // walk on from the first probe to the key's slot
        while (prev != kEmptyKey && prev != key) {
          sl = (sl + 1) & mask;
          prev = atomicCAS(&ht_key[sl], kEmptyKey, key);
        }
        ht_net[sl] = -1;
      }
      *slot = probe ? static_cast<int>(sl) : -1;
    }
  }
  return net;
}

__global__ void k_net_decide(const BatchIn *bin, const ripple_op *ops, int undirected, const int *ht_val,
                             int *ht_net, const int *op_slot, const int *fop, Adj out, Adj in, int *ins_src,
                             int *ins_dst, int *del_src, int *del_dst, int *ins_rank, int *del_rank, float *ins_w,
                             float *del_w, int *flist, int *frow, Counters *c) {
  const int lane = lane_id();
  const long long B = bin->num_ops;
  for (long long i = global_wave(); i < B; i += num_waves()) {
    const ripple_op op = ops[i];
    const int s = op_slot[i];
    if (op.kind == RIPPLE_OP_FEATURE) {
      if (lane == 0 && fop[op.u] == i) {
        const u64 j = atomicAdd(&c->n_feat, 1ull);
        flist[j] = op.u;
        frow[j] = op.feat_row;
      }
      continue;
    }
    int a = op.u, b = op.v;
    if (undirected && a > b) {
      const int t = a;
      a = b;
      b = t;
    }
    // what the decision needs from the op's slot and rows, in one round of loads
    // (ids are in range: failing ops became self-loops); the non-negative values
    // join the test so that no load waits behind it
    const int winner = s >= 0 ? ht_val[s] : -1;
    const int la = out.len[a], lb = in.len[b];
    const long long oa = out.off[a], ob = in.off[b];
    if (static_cast<int>(s < 0 || winner != i) |
        (la | lb | static_cast<int>(oa >> 32) | static_cast<int>(ob >> 32)) >> 31)
      continue;  // self-loop, or a later op names this edge
    const int net = emit_edge(op, a, b, la, lb, oa, ob, undirected, out, in, ins_src, ins_dst, del_src, del_dst,
                              ins_rank, del_rank, ins_w, del_w, c);
    if (lane == 0) ht_net[s] = net;
  }
}

// Netting in one launch for batches of at most kNetDirectMax ops (see
// launch_net_direct). Wave i takes op i: it checks the op as k_net_hash does, and
// compares it with every later op of the batch (64 per round, all rounds' loads in
// flight together). An op that no later op overrides (same edge key; for feature
// writes, same vertex) decides: a feature write sets fop and lists its vertex, an
// edge op runs the decision of k_net_decide. Only net-deleted keys enter the hash
// table (the row rewrite looks up nothing else; an absent key is kept), tagged -1,
// and op_slot names their slots for the clean-up.
constexpr int kNetDirectRounds = kNetDirectMax / kWave;
static_assert(kNetDirectRounds * kWave == kNetDirectMax, "whole rounds");

__global__ void k_net_direct(const BatchIn *host_in, BatchIn now, BatchIn *dev_in, ripple_op *ops, int undirected,
                             int weighted, long long n, u64 *ht_key, int *ht_net, unsigned mask, int *op_slot,
                             int *fop, Adj out, Adj in, int *ins_src, int *ins_dst, int *del_src, int *del_dst,
                             int *ins_rank, int *del_rank, float *ins_w, float *del_w, int *flist, int *frow,
                             Counters *c) {
  if (host_in != nullptr) {
    const auto word = [&](const void *f) {
      return __hip_atomic_load(static_cast<const u64 *>(f), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_SYSTEM);
    };
    now.ops = reinterpret_cast<const ripple_op *>(word(&host_in->ops));
    now.feat = reinterpret_cast<const float *>(word(&host_in->feat));
    now.num_ops = static_cast<long long>(word(&host_in->num_ops));
    now.num_feat_rows = static_cast<long long>(word(&host_in->num_feat_rows));
  }
  const ripple_op *src_ops = now.ops;
  const long long B = now.num_ops;
  const long long i = global_wave();
  const int lane = lane_id();
  if (i == 0 && lane == 0) *dev_in = now;
  if (i >= B) return;
  ripple_op op = src_ops[i];
  ripple_op later[kNetDirectRounds];
#pragma unroll
  for (int t = 0; t < kNetDirectRounds; ++t) {
    const long long j = i + 1 + lane + static_cast<long long>(t) * kWave;
    later[t] = j < B ? src_ops[j] : ripple_op{-1, 0, 0, 0};
  }
  bool bad;
  if (op.kind == RIPPLE_OP_INSERT || op.kind == RIPPLE_OP_DELETE)
    bad = op.u < 0 || op.u >= n || op.v < 0 || op.v >= n ||
          (weighted && op.kind == RIPPLE_OP_INSERT && !isfinite(op.weight));
  else if (op.kind == RIPPLE_OP_FEATURE)
    bad = op.u < 0 || op.u >= n || op.feat_row < 0 || op.feat_row >= now.num_feat_rows;
  else
    bad = true;
  if (bad) {
    // the batch aborts before anything is mutated; the later kernels see a harmless self-loop
    if (lane == 0) {
      atomicMax(&c->bad_op, static_cast<u64>(B - i));
      c->abort = 1;
      ops[i] = ripple_op{RIPPLE_OP_INSERT, 0, 0, -1};
      op_slot[i] = -1;
    }
    return;
  }
  if (lane == 0) ops[i] = op;
  if (op.kind == RIPPLE_OP_FEATURE) {
    bool over = false;
#pragma unroll
    for (int t = 0; t < kNetDirectRounds; ++t) over = over || (later[t].kind == RIPPLE_OP_FEATURE && later[t].u == op.u);
    const bool decides = __ballot(over) == 0;
    if (lane == 0) {
      op_slot[i] = -1;
      if (decides) {
        fop[op.u] = static_cast<int>(i);
        const u64 j = atomicAdd(&c->n_feat, 1ull);
        flist[j] = op.u;
        frow[j] = op.feat_row;
      }
    }
    return;
  }
  if (op.u == op.v) {
    if (lane == 0) {
      atomicAdd(&c->noop_edge, 1ull);
      op_slot[i] = -1;
    }
    return;
  }
  int a = op.u, b = op.v;
  if (undirected && a > b) {
    const int t = a;
    a = b;
    b = t;
  }
  const u64 key = edge_key(a, b, undirected, n);
  bool over = false;
#pragma unroll
  for (int t = 0; t < kNetDirectRounds; ++t) {
    const bool edge = later[t].kind == RIPPLE_OP_INSERT || later[t].kind == RIPPLE_OP_DELETE;
    over = over || (edge && later[t].u != later[t].v && edge_key(later[t].u, later[t].v, undirected, n) == key);
  }
  // the rows the decision reads go out with the comparison (ids are checked)
  const int la = out.len[a], lb = in.len[b];
  const long long oa = out.off[a], ob = in.off[b];
  if (__ballot(over) != 0) {
    if (lane == 0) op_slot[i] = -1;
    return;
  }
  emit_edge(op, a, b, la, lb, oa, ob, undirected, out, in, ins_src, ins_dst, del_src, del_dst, ins_rank, del_rank,
            ins_w, del_w, c, ht_key, ht_net, mask, key, op_slot + i);
}

__global__ void k_topo_plan(Adj out, Adj in, const int *ins_src, const int *ins_dst, const int *del_src,
                            const int *del_dst, const int *ins_rank, const int *del_rank, int long_ok, LongRow *tab,
                            Counters *c, const Persist *p, long long cap_out, long long cap_in) {
  const long long ni = 2 * static_cast<long long>(c->n_ins);
  const long long nd = long_ok ? 2 * static_cast<long long>(c->n_del) : 0;
  const long long stride = static_cast<long long>(gridDim.x) * blockDim.x;
  for (long long w = blockIdx.x * blockDim.x + threadIdx.x; w < ni + nd; w += stride) {
    // one planner per touched row: its first insert item, else its first delete item
    const bool ins_item = w < ni;
    const long long x = ins_item ? w : w - ni;
    int dir, row, entry;
    item_row(x, ins_item ? ins_src : del_src, ins_item ? ins_dst : del_dst, dir, row, entry);
    if (((ins_item ? ins_rank : del_rank)[x] | row >> 31) != 0) continue;  // (row >= 0: see k_topo_rewrite)
    const Adj &a = dir ? in : out;
    const int len0 = a.len[row], k = a.delcnt[row], nins = a.inscnt[row], cap = a.cap[row];
    if (!ins_item && nins != 0) continue;
    const int need = len0 - k + nins;
    if (need > cap) {
      atomicAdd(&c->arena_need[dir], static_cast<u64>(grow_cap(need)));
    } else if (long_ok && k > 0 && len0 >= kLongRow) {
      // a long row that keeps its slots: list it for the chunked sweep
      const long long chunks = (len0 + kLongChunk - 1) / kLongChunk;
      const u64 old = atomicAdd(&c->long_rows, (1ull << 40) | static_cast<u64>(chunks));
      const long long at = static_cast<long long>(old >> 40);
      LongRow t{};
      t.dir = dir;
      t.row = row;
      t.len0 = len0;
      t.k = k;
      t.off = a.off[row];
      t.chunk0 = static_cast<long long>(old & ((1ull << 40) - 1));
      t.pool = static_cast<long long>(atomicAdd(&c->long_pool, 2ull * static_cast<u64>(k)));
      tab[at] = t;
    }
  }
  // the last block to finish compares the arena demand with the free arena
  __threadfence();
  __syncthreads();
  __shared__ bool last;
  if (threadIdx.x == 0) last = atomicAdd(&c->plan_done, 1ull) == gridDim.x - 1;
  __syncthreads();
  if (last && threadIdx.x == 0) {
    __threadfence();
    const u64 need0 = atomicAdd(&c->arena_need[0], 0ull);
    const u64 need1 = atomicAdd(&c->arena_need[1], 0ull);
    if (p->top[0] + need0 > static_cast<u64>(cap_out) || p->top[1] + need1 > static_cast<u64>(cap_in))
      c->abort = 1;
  }
}

constexpr int kRewriteU = 16;  // row entries per lane per step: 1024 per wave
// Rows up to this long whose only change is one delete are fixed by a search and a
// swap-remove (at most two rounds of wave_find) instead of a full rewrite.
constexpr int kSoloDeleteMax = 2048;

// Clears keep[u] for the entries x[u] of `row` (direction dir) that the batch
// deletes. Each entry's edge-key slot is probed together with the slot's net
// decision; probes that meet another key walk their chains one slot per round, all
// of a lane's chains in the same round (the table is at most an eighth full, so
// every chain meets an empty slot).
__device__ inline void drop_deleted(const int (&x)[kRewriteU], bool (&keep)[kRewriteU], int row, int dir,
                                    int undirected, long long n, const u64 *ht_key, const int *ht_net,
                                    unsigned mask) {
  u64 key[kRewriteU], got[kRewriteU];
  unsigned sl[kRewriteU];
  int net[kRewriteU];
#pragma unroll
  for (int u = 0; u < kRewriteU; ++u) {
    key[u] = edge_key(dir ? x[u] : row, dir ? row : x[u], undirected, n);
    sl[u] = hash_slot(key[u], mask);
  }
#pragma unroll
  for (int u = 0; u < kRewriteU; ++u) {
    got[u] = keep[u] ? ht_key[sl[u]] : kEmptyKey;
    net[u] = keep[u] ? ht_net[sl[u]] : 0;
  }
  unsigned pend = 0;
#pragma unroll
  for (int u = 0; u < kRewriteU; ++u) {
    if (!keep[u] || got[u] == kEmptyKey) continue;
    if (got[u] == key[u]) keep[u] = net[u] != -1;
    else pend |= 1u << u;
  }
  for (unsigned j = 1; pend != 0; ++j) {
#pragma unroll
    for (int u = 0; u < kRewriteU; ++u) {
      if (pend >> u & 1u) {
        const unsigned s2 = (sl[u] + j) & mask;
        got[u] = ht_key[s2];
        net[u] = ht_net[s2];
      }
    }
#pragma unroll
    for (int u = 0; u < kRewriteU; ++u) {
      if (!(pend >> u & 1u)) continue;
      if (got[u] == key[u]) {
        keep[u] = net[u] != -1;
        pend &= ~(1u << u);
      } else if (got[u] == kEmptyKey) {
        pend &= ~(1u << u);  // not named by the batch: kept
      }
    }
  }
}

// The entry of tab[0 .. n_long) holding chunk j (the last one whose chunk0 <= j;
// chunk0 grows with the index): at most two rounds of 64 loads for up to 4096 rows,
// then a plain search.
__device__ inline long long find_long(const LongRow *tab, long long n_long, long long j) {
  const int lane = lane_id();
  long long lo = 0, hi = n_long;  // answer in [lo, hi)
  while (hi - lo > 1) {
    const long long step = (hi - lo + kWave - 1) / kWave;
    const long long at = lo + lane * step;
    const bool le = at < hi && tab[at].chunk0 <= j;
    const int cnt = __popcll(__ballot(le));  // entries lo, lo + step, ... up to cnt - 1 qualify
    const long long nlo = lo + (cnt - 1) * step;
    hi = nlo + step < hi ? nlo + step : hi;
    lo = nlo;
  }
  return lo;
}

// Appends position e of every lane with flag set to list[*count ..] (at most cap
// entries; past that the check bit is set instead).
__device__ inline void append_positions(bool flag, int e, int *list, int *count, int cap, Counters *c) {
  const u64 m = __ballot(flag);
  if (m == 0) return;
  int b0 = 0;
  if (lane_id() == 0) b0 = atomicAdd(count, __popcll(m));
  b0 = __shfl(b0, 0);
  const int at = b0 + lanes_below(m);
  if (flag) {
    if (at < cap) list[at] = e;
    else atomicOr(&c->err, 2ull);
  }
}

// One wave per touched (row, direction): the row's owner is its rank-0 insert
// item, or its rank-0 delete item when it has no inserts. Long rows listed by the
// plan are left to the chunk sweeps, which follow the items in the same grid.
__global__ __launch_bounds__(256) void k_topo_rewrite(int undirected, long long n, Adj out, Adj in, const int *ins_src,
                               const int *ins_dst, const int *del_src, const int *del_dst, const int *ins_rank,
                               const int *del_rank, const u64 *ht_key, const int *ht_net, unsigned mask,
                               Persist *p, int *ddeg, int long_ok, LongRow *tab, int *pool, Counters *c,
                               RewriteBounds rb) {
  const long long ni = 2 * static_cast<long long>(c->n_ins);
  const long long nd = 2 * static_cast<long long>(c->n_del);
  const u64 lr = c->long_rows;
  if (aborted_with(c->abort, ni, nd, static_cast<long long>(lr >> 1))) return;
  const long long n_long = static_cast<long long>(lr >> 40);
  const long long chunks = static_cast<long long>(lr & ((1ull << 40) - 1));
  const int lane = lane_id();
  for (long long w = global_wave(); w < ni + nd + chunks; w += num_waves()) {
    if (w >= ni + nd) {
      // chunk sweep of a long row: its deleted entries below the new length are
      // holes, its kept entries at or above it are movers
      const long long j = w - ni - nd;
      const long long at = find_long(tab, n_long, j);
      const LongRow t = tab[at];
      const Adj &a = t.dir ? in : out;
      const int *src = a.col + t.off;
      const int e0 = static_cast<int>((j - t.chunk0) * kLongChunk);
      const int e1 = e0 + kLongChunk < t.len0 ? e0 + kLongChunk : t.len0;
      const int new_len = t.len0 - t.k;
      int found = 0;
      for (int base = e0; base < e1; base += kWave * kRewriteU) {
        int x[kRewriteU];
        bool keep[kRewriteU], live[kRewriteU];
#pragma unroll
        for (int u = 0; u < kRewriteU; ++u) {
          const int e = base + u * kWave + lane;
          live[u] = e < e1;
          keep[u] = live[u];
          x[u] = live[u] ? src[e] : -1;
        }
        drop_deleted(x, keep, t.row, t.dir, undirected, n, ht_key, ht_net, mask);
#pragma unroll
        for (int u = 0; u < kRewriteU; ++u) {
          const int e = base + u * kWave + lane;
          found += live[u] && !keep[u] ? 1 : 0;
          append_positions(live[u] && !keep[u] && e < new_len, e, pool + t.pool, &tab[at].holes, t.k, c);
          append_positions(live[u] && keep[u] && e >= new_len, e, pool + t.pool + t.k, &tab[at].movers, t.k, c);
        }
      }
#pragma unroll
      for (int o = kWave / 2; o > 0; o >>= 1) found += __shfl_xor(found, o);
      if (lane == 0 && found != 0) atomicAdd(&tab[at].found, found);
      continue;
    }
    const bool ins_item = w < ni;
    const long long x = ins_item ? w : w - ni;
    int dir, row, entry;
    item_row(x, ins_item ? ins_src : del_src, ins_item ? ins_dst : del_dst, dir, row, entry);
    const int rank = (ins_item ? ins_rank : del_rank)[x];
    if ((rank | row >> 31) != 0) continue;  // not the row's first item (row >= 0 joins the test,
                                            // so its load is not held back behind the rank's)
    const Adj &a = dir ? in : out;
    const int len0 = a.len[row], k = a.delcnt[row], nins = a.inscnt[row], cap0 = a.cap[row];
    const long long src_off = a.off[row];
    // a row with inserts belongs to its first insert item (cap0, src_off >= 0 join
    // the test so that their loads go out with the others)
    if (static_cast<int>(!ins_item && nins != 0) | (cap0 | static_cast<int>(src_off >> 32)) >> 31) continue;
    const int need = len0 - k + nins;
    const bool move = nins > 0 && need > cap0;
    const bool swept = long_ok && k > 0 && !move && len0 >= kLongRow;  // listed by the plan
    if (!ins_item && k == 1 && nins == 0 && len0 > 0 && len0 <= kSoloDeleteMax) {
      // this delete is the row's only change: find its entry (the row's last entry is
      // read in the same round) and move the last entry into its slot; rows are
      // unordered, so the swap-remove keeps the row valid
      int *rc = a.col + src_off;
      float *rw = a.wt != nullptr ? a.wt + src_off : nullptr;
      const int last = rc[len0 - 1];
      const float last_w = rw != nullptr ? rw[len0 - 1] : 0.0f;
      const int pos = wave_find(rc, len0, entry);
      if (lane == 0) {
        if (pos < 0) {
          atomicOr(&c->err, 1ull);  // a net-deleted arc that is not in its row
        } else if (pos != len0 - 1) {
          rc[pos] = last;
          if (rw != nullptr) rw[pos] = last_w;
        }
        a.len[row] = need;
        if (dir == 0) ddeg[row] = -1;
      }
      continue;
    }
    const int nc = move ? grow_cap(need) : 0;
    // a moving row's arena slots: the returning atomic stays in flight while the
    // row is read (its value is needed only for the writes)
    long long moved_to = 0;
    if (move && lane == 0) moved_to = static_cast<long long>(atomicAdd(&p->top[dir], static_cast<u64>(nc)));
    if (lane == 0 && need > rb.maxlen[dir]) atomicMax(&c->maxlen[dir], static_cast<u64>(need));
    long long dst_off = src_off;
    // a move past the arena's end (possible only if the plan did not run and the
    // host's bound was wrong) writes nothing and fails the batch
    const long long arena_end = rb.capacity[dir];
    bool overflow = false;
    if (!swept && (k > 0 || move)) {
      const int *src = a.col + src_off;
      const float *srcw = a.wt != nullptr ? a.wt + src_off : nullptr;  // weights move with their slots
      int wpos = 0;
      // kRewriteU entries per lane per step (rows up to 1024 entries take one step):
      // the step's row reads, then its hash probes, are all in flight at once; all
      // reads of a step precede its writes, and a kept entry is written at or below
      // its own position, so the in-place case is safe.
      for (int base = 0; base < len0; base += kWave * kRewriteU) {
        int x[kRewriteU];
        float xw[kRewriteU];
        bool keep[kRewriteU];
#pragma unroll
        for (int u = 0; u < kRewriteU; ++u) {
          const int e = base + u * kWave + lane;
          keep[u] = e < len0;
          x[u] = keep[u] ? src[e] : -1;
          xw[u] = keep[u] && srcw != nullptr ? srcw[e] : 0.0f;
        }
        if (k > 0) drop_deleted(x, keep, row, dir, undirected, n, ht_key, ht_net, mask);
        if (base == 0 && move) {
          dst_off = __shfl(moved_to, 0);
          overflow = dst_off + nc > arena_end;
        }
        int *dst = a.col + dst_off;
        float *dstw = a.wt != nullptr ? a.wt + dst_off : nullptr;
#pragma unroll
        for (int u = 0; u < kRewriteU; ++u) {
          const u64 m = __ballot(keep[u]);
          if (keep[u] && !overflow) {
            dst[wpos + lanes_below(m)] = x[u];
            if (dstw != nullptr) dstw[wpos + lanes_below(m)] = xw[u];
          }
          wpos += __popcll(m);
        }
      }
      if (move && len0 == 0) {  // no step ran
        dst_off = __shfl(moved_to, 0);
        overflow = dst_off + nc > arena_end;
      }
      if (lane == 0 && wpos != len0 - k) atomicOr(&c->err, 2ull);
    }
    if (overflow) {
      if (lane == 0) atomicOr(&c->err, 8ull);
      continue;
    }
    if (lane == 0) {
      if (move) {
        a.off[row] = dst_off;
        a.cap[row] = nc;
        atomicAdd(&c->n_reloc, 1ull);
        atomicMax(&c->top_end[dir], static_cast<u64>(dst_off + nc));
      }
      a.len[row] = need;
      if (dir == 0) ddeg[row] = nins - k;
    }
  }
}

// The fill pass of the long rows: each hole takes one mover's entry (and weight).
// The sweeps found as many holes as movers and every deleted entry, else the
// check bit is set.
__global__ void k_topo_fill(Adj out, Adj in, const LongRow *tab, const int *pool, Counters *c) {
  const u64 lr = c->long_rows;
  if (aborted_with(c->abort, static_cast<long long>(lr >> 1))) return;
  const long long n_long = static_cast<long long>(lr >> 40);
  const int lane = lane_id();
  for (long long r = global_wave(); r < n_long; r += num_waves()) {
    const LongRow t = tab[r];
    if (lane == 0 && (t.holes != t.movers || t.found != t.k)) atomicOr(&c->err, 2ull);
    int pairs = t.holes < t.movers ? t.holes : t.movers;
    if (pairs > t.k) pairs = t.k;  // the sweeps record at most k of each
    const Adj &a = t.dir ? in : out;
    for (int i = lane; i < pairs; i += kWave) {
      const long long hole = t.off + pool[t.pool + i], mover = t.off + pool[t.pool + t.k + i];
      a.col[hole] = a.col[mover];
      if (a.wt != nullptr) a.wt[hole] = a.wt[mover];
    }
  }
}

// Re-layout: row u's used entries move from old_col[old_off[u]..] to new_col[new_off[u]..].
__global__ void k_repack_copy(long long n, const int *old_col, const long long *old_off, const int *len,
                              int *new_col, const long long *new_off, const float *old_wt, float *new_wt) {
  const int lane = lane_id();
  for (long long u = global_wave(); u < n; u += num_waves()) {
    const int *src = old_col + old_off[u];
    int *dst = new_col + new_off[u];
    const int l = len[u];
    for (int e = lane; e < l; e += kWave) dst[e] = src[e];
    if (new_wt != nullptr)
      for (int e = lane; e < l; e += kWave) new_wt[new_off[u] + e] = old_wt[old_off[u] + e];
  }
}

inline int blocks_for(long long items, int threads, int cap = 4096) {
  long long b = (items + threads - 1) / threads;
  if (b < 1) b = 1;
  if (b > cap) b = cap;
  return static_cast<int>(b);
}

}  // namespace

void launch_net_hash(hipStream_t s, int cap_ops, const BatchIn *host_in, const BatchIn &now, BatchIn *dev_in,
                     ripple_op *ops,
                     int undirected, int weighted, long long n, u64 *ht_key, int *ht_val, unsigned mask, int *op_slot,
                     int *fop, Counters *c) {
  RP_LAUNCH(k_net_hash, dim3(blocks_for(cap_ops, 256, 1 << 20)), dim3(256), 0, s, host_in, now, dev_in, ops,
                     undirected, weighted, n, ht_key, ht_val, mask, op_slot, fop, c);
}

void launch_net_direct(hipStream_t s, int cap_ops, const BatchIn *host_in, const BatchIn &now, BatchIn *dev_in,
                       ripple_op *ops, int undirected, int weighted, long long n, u64 *ht_key, int *ht_net,
                       unsigned mask, int *op_slot, int *fop, Adj out, Adj in_adj, int *ins_src, int *ins_dst,
                       int *del_src, int *del_dst, int *ins_rank, int *del_rank, float *ins_w, float *del_w,
                       int *flist, int *frow, Counters *c) {
  const int ops_cap = cap_ops < kNetDirectMax ? cap_ops : kNetDirectMax;
  RP_LAUNCH(k_net_direct, dim3(blocks_for(static_cast<long long>(ops_cap) * kWave, 256)), dim3(256), 0, s,
                     host_in, now, dev_in, ops, undirected, weighted, n, ht_key, ht_net, mask, op_slot, fop, out,
                     in_adj, ins_src, ins_dst, del_src, del_dst, ins_rank, del_rank, ins_w, del_w, flist, frow, c);
}

void launch_net_decide(hipStream_t s, int cap_ops, const BatchIn *in, const ripple_op *ops, int undirected,
                       const int *ht_val, int *ht_net, const int *op_slot, const int *fop, Adj out, Adj in_adj,
                       int *ins_src, int *ins_dst, int *del_src, int *del_dst, int *ins_rank, int *del_rank,
                       float *ins_w, float *del_w, int *flist, int *frow, Counters *c) {
  RP_LAUNCH(k_net_decide, dim3(blocks_for(static_cast<long long>(cap_ops) * kWave, 256)), dim3(256), 0, s,
                     in, ops, undirected, ht_val, ht_net, op_slot, fop, out, in_adj, ins_src, ins_dst, del_src,
                     del_dst, ins_rank, del_rank, ins_w, del_w, flist, frow, c);
}

void launch_topo_plan(hipStream_t s, int cap_arcs, Adj out, Adj in, const int *ins_src, const int *ins_dst,
                      const int *del_src, const int *del_dst, const int *ins_rank, const int *del_rank,
                      int long_ok, LongRow *tab, Counters *c, const Persist *p, long long cap_out, long long cap_in) {
  RP_LAUNCH(k_topo_plan, dim3(blocks_for((long_ok ? 4LL : 2LL) * cap_arcs, 256, 1024)), dim3(256), 0, s,
                     out, in, ins_src, ins_dst, del_src, del_dst, ins_rank, del_rank, long_ok, tab, c, p, cap_out,
                     cap_in);
}

void launch_topo_rewrite(hipStream_t s, int cap_arcs, int undirected, long long n, Adj out, Adj in,
                         const int *ins_src, const int *ins_dst, const int *del_src, const int *del_dst,
                         const int *ins_rank, const int *del_rank, const u64 *ht_key, const int *ht_net,
                         unsigned mask, Persist *p, int *ddeg, int long_ok, LongRow *tab, int *pool, Counters *c,
                         const RewriteBounds &rb) {
  RP_LAUNCH(k_topo_rewrite, dim3(blocks_for(4LL * cap_arcs * kWave, 256)), dim3(256), 0, s, undirected,
                     n, out, in, ins_src, ins_dst, del_src, del_dst, ins_rank, del_rank, ht_key, ht_net, mask, p,
                     ddeg, long_ok, tab, pool, c, rb);
}

void launch_topo_fill(hipStream_t s, int cap_arcs, Adj out, Adj in, const LongRow *tab, const int *pool,
                      Counters *c) {
  RP_LAUNCH(k_topo_fill, dim3(blocks_for(2LL * cap_arcs * kWave, 256, 1024)), dim3(256), 0, s, out, in,
                     tab, pool, c);
}

void launch_repack_copy(hipStream_t s, long long n, const int *old_col, const long long *old_off, const int *len,
                        int *new_col, const long long *new_off, const float *old_wt, float *new_wt) {
  RP_LAUNCH(k_repack_copy, dim3(blocks_for(n * kWave, 256, 8192)), dim3(256), 0, s, n, old_col, old_off,
                     len, new_col, new_off, old_wt, new_wt);
}

}  // namespace rp

// Device-side re-layout of one adjacency direction: new capacities from the
// current lengths, an exclusive scan for the new offsets, the rows copied into
// the spare column buffer, then the row table and the arena top updated.
namespace rp {

namespace {

constexpr int kScanThreads = 1024;
constexpr int kScanPerThread = 4;
constexpr int kScanPerBlock = kScanThreads * kScanPerThread;

__device__ inline long long block_scan_excl(long long v, long long *lds, long long *total) {
  const int lane = threadIdx.x & (kWave - 1), wave = threadIdx.x / kWave;
  constexpr int waves = kScanThreads / kWave;
  long long x = v;
#pragma unroll
  for (int o = 1; o < kWave; o <<= 1) {
    const long long y = __shfl_up(x, o);
    if (lane >= o) x += y;
  }
  if (lane == kWave - 1) lds[wave] = x;
  __syncthreads();
  if (threadIdx.x == 0) {
    long long run = 0;
    for (int w = 0; w < waves; ++w) {
      const long long t = lds[w];
      lds[w] = run;
      run += t;
    }
    lds[waves] = run;
  }
  __syncthreads();
  const long long excl = x - v + lds[wave];
  *total = lds[waves];
  __syncthreads();
  return excl;
}

__device__ inline int relayout_cap(int len, float slack, int min_slack) {
  long long extra = static_cast<long long>(ceilf(static_cast<float>(len) * slack));
  if (extra < min_slack) extra = min_slack;
  return static_cast<int>(len + extra);
}

// pass 1: per-block sums of the new capacities
__global__ __launch_bounds__(kScanThreads) void k_relayout_sums(long long n, const int *len, float slack,
                                                                int min_slack, long long *blocksums) {
  __shared__ long long lds[kScanThreads / kWave + 1];
  long long s = 0;
  const long long base = static_cast<long long>(blockIdx.x) * kScanPerBlock + threadIdx.x * kScanPerThread;
  for (int i = 0; i < kScanPerThread; ++i)
    if (base + i < n) s += relayout_cap(len[base + i], slack, min_slack);
  long long total;
  block_scan_excl(s, lds, &total);
  if (threadIdx.x == 0) blocksums[blockIdx.x] = total;
}

// pass 2: one block scans the block sums in place (exclusive); total to blocksums[nb]
__global__ __launch_bounds__(kScanThreads) void k_relayout_scan_sums(long long *blocksums, int nb) {
  __shared__ long long lds[kScanThreads / kWave + 1];
  long long carry = 0;
  for (int base = 0; base < nb; base += kScanThreads) {
    const int i = base + threadIdx.x;
    const long long v = i < nb ? blocksums[i] : 0;
    long long total;
    const long long ex = block_scan_excl(v, lds, &total);
    if (i < nb) blocksums[i] = carry + ex;
    carry += total;
  }
  if (threadIdx.x == 0) blocksums[nb] = carry;
}

// pass 3: new offsets and capacities
__global__ __launch_bounds__(kScanThreads) void k_relayout_offsets(long long n, const int *len, float slack,
                                                                   int min_slack, const long long *blocksums,
                                                                   long long *new_off, int *new_cap) {
  __shared__ long long lds[kScanThreads / kWave + 1];
  const long long base = static_cast<long long>(blockIdx.x) * kScanPerBlock + threadIdx.x * kScanPerThread;
  int caps[kScanPerThread];
  long long s = 0;
  for (int i = 0; i < kScanPerThread; ++i) {
    caps[i] = base + i < n ? relayout_cap(len[base + i], slack, min_slack) : 0;
    s += caps[i];
  }
  long long total;
  long long pos = blocksums[blockIdx.x] + block_scan_excl(s, lds, &total);
  for (int i = 0; i < kScanPerThread; ++i) {
    if (base + i < n) {
      new_off[base + i] = pos;
      new_cap[base + i] = caps[i];
      pos += caps[i];
    }
  }
}

// pass 5: install the new row table and arena top
__global__ void k_relayout_install(long long n, const long long *new_off, const int *new_cap, long long *off,
                                   int *cap, const long long *blocksums, int nb, u64 *top) {
  const long long stride = static_cast<long long>(gridDim.x) * blockDim.x;
  for (long long u = blockIdx.x * blockDim.x + threadIdx.x; u < n; u += stride) {
    off[u] = new_off[u];
    cap[u] = new_cap[u];
  }
  if (blockIdx.x == 0 && threadIdx.x == 0) *top = static_cast<u64>(blocksums[nb]);
}

}  // namespace

int relayout_blocks(long long n) { return static_cast<int>((n + kScanPerBlock - 1) / kScanPerBlock); }

void launch_relayout_sums(hipStream_t s, long long n, float slack, int min_slack, const int *len,
                          long long *blocksums) {
  const int nb = relayout_blocks(n);
  RP_LAUNCH(k_relayout_sums, dim3(nb), dim3(kScanThreads), 0, s, n, len, slack, min_slack, blocksums);
  RP_LAUNCH(k_relayout_scan_sums, dim3(1), dim3(kScanThreads), 0, s, blocksums, nb);
}

void launch_relayout_apply(hipStream_t s, long long n, float slack, int min_slack, Adj a, int *new_col,
                           float *new_wt, const long long *blocksums, long long *new_off, int *new_cap, u64 *top) {
  const int nb = relayout_blocks(n);
  RP_LAUNCH(k_relayout_offsets, dim3(nb), dim3(kScanThreads), 0, s, n, a.len, slack, min_slack, blocksums,
                     new_off, new_cap);
  RP_LAUNCH(k_repack_copy, dim3(blocks_for(n * kWave, 256, 8192)), dim3(256), 0, s, n, a.col, a.off, a.len,
                     new_col, new_off, a.wt, new_wt);
  long long ib = (n + 255) / 256;
  if (ib > 4096) ib = 4096;
  RP_LAUNCH(k_relayout_install, dim3(ib), dim3(256), 0, s, n, new_off, new_cap, a.off, a.cap, blocksums, nb,
                     top);
}

}  // namespace rp
