// Batch netting and the dynamic adjacency update.
//
// Netting (sequential semantics of a batch): an insert sets an arc present and a
// delete sets it absent, so the last op naming an edge decides its final state.
// One pass hashes every edge op and keeps the largest op index per edge; a second
// pass lets each winning op compare the final state with the pre-batch adjacency
// and emit the net inserted / deleted arcs. The last feature write per vertex is
// found the same way with a per-vertex atomicMax.
//
// Adjacency update: row slots are [off, off+cap), the first len used, in no
// particular order. Deletes tombstone their slot, then each hole in the part of
// the row that survives is filled from the row's tail; inserts append at
// len + rank. Rows that would overflow are first moved to the spare arena; the
// arena demand is checked before anything is mutated, so an arena that is too
// small aborts the batch with the state intact (the host then re-lays the rows
// out and runs the batch again).
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

// Position of `target` in row[0, len) or -1; all lanes of the wave get the answer.
__device__ inline int wave_find(const int *row, int len, int target) {
  const int lane = lane_id();
  for (int base = 0; base < len; base += kWave) {
    const int e = base + lane;
    const bool hit = e < len && row[e] == target;
    const u64 m = __ballot(hit);
    if (m) return base + __ffsll(static_cast<long long>(m)) - 1;
  }
  return -1;
}

__global__ void k_net_hash(const ripple_op *ops, int B, int undirected, long long n, u64 *ht_key,
                           int *ht_val, unsigned mask, int *op_slot, int *fop, Counters *c) {
  const int i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= B) return;
  const ripple_op op = ops[i];
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
  int a = op.u, b = op.v;
  if (undirected && a > b) {
    const int t = a;
    a = b;
    b = t;
  }
  const u64 key = static_cast<u64>(a) * static_cast<u64>(n) + static_cast<u64>(b);
  unsigned s = hash_slot(key, mask);
  while (true) {
    const u64 prev = atomicCAS(&ht_key[s], kEmptyKey, key);
    if (prev == kEmptyKey || prev == key) break;
    s = (s + 1) & mask;
  }
  atomicMax(&ht_val[s], i);
  op_slot[i] = static_cast<int>(s);
}

__global__ void k_net_decide(const ripple_op *ops, int B, int undirected, const int *ht_val,
                             const int *op_slot, const int *fop, Adj out, Adj in, int *ins_src,
                             int *ins_dst, int *del_src, int *del_dst, int *flist, Counters *c) {
  const int lane = lane_id();
  for (long long i = global_wave(); i < B; i += num_waves()) {
    const ripple_op op = ops[i];
    if (op.kind == RIPPLE_OP_FEATURE) {
      if (lane == 0 && fop[op.u] == i) {
        const u64 j = atomicAdd(&c->n_feat, 1ull);
        flist[j] = op.u;
      }
      continue;
    }
    const int s = op_slot[i];
    if (s < 0 || ht_val[s] != i) continue;  // self-loop, or a later op names this edge
    int a = op.u, b = op.v;
    if (undirected && a > b) {
      const int t = a;
      a = b;
      b = t;
    }
    const int la = out.len[a], lb = in.len[b];
    const bool use_out = la <= lb;
    const int *row = use_out ? out.col + out.off[a] : in.col + in.off[b];
    const int pos = wave_find(row, use_out ? la : lb, use_out ? b : a);
    const bool present = pos >= 0;
    const bool want = op.kind == RIPPLE_OP_INSERT;
    if (lane == 0) {
      atomicAdd(&c->edge_keys, 1ull);
      if (want == present) {
        atomicAdd(&c->noop_edge, 1ull);
      } else {
        int *ps = want ? ins_src : del_src;
        int *pd = want ? ins_dst : del_dst;
        const u64 j = atomicAdd(want ? &c->n_ins : &c->n_del, undirected ? 2ull : 1ull);
        ps[j] = a;
        pd[j] = b;
        if (undirected) {
          ps[j + 1] = b;
          pd[j + 1] = a;
        }
      }
    }
  }
}

// Work items over arcs x directions: item w -> arc w >> 1, direction w & 1.
// Direction 0 (out-adjacency): row = src, entry = dst; direction 1: row = dst, entry = src.
__device__ inline void item_row(long long w, const int *src, const int *dst, int &dir, int &row, int &entry) {
  const long long arc = w >> 1;
  dir = static_cast<int>(w & 1);
  row = dir == 0 ? src[arc] : dst[arc];
  entry = dir == 0 ? dst[arc] : src[arc];
}

__global__ void k_topo_count(int cap_arcs, Adj out, Adj in, const int *ins_src, const int *ins_dst,
                             const int *del_src, const int *del_dst, int *ins_rank, int *del_rank,
                             Counters *c) {
  const long long ni = 2 * static_cast<long long>(c->n_ins);
  const long long nd = 2 * static_cast<long long>(c->n_del);
  const long long stride = static_cast<long long>(gridDim.x) * blockDim.x;
  for (long long w = blockIdx.x * blockDim.x + threadIdx.x; w < ni + nd; w += stride) {
    int dir, row, entry;
    if (w < ni) {
      item_row(w, ins_src, ins_dst, dir, row, entry);
      ins_rank[w] = atomicAdd(&(dir ? in : out).inscnt[row], 1);
    } else {
      item_row(w - ni, del_src, del_dst, dir, row, entry);
      del_rank[w - ni] = atomicAdd(&(dir ? in : out).delcnt[row], 1);
    }
  }
}

__device__ inline int grow_cap(int newlen) {
  const long long g = static_cast<long long>(newlen) + newlen / 2 + 4;
  return static_cast<int>(((g + 3) / 4) * 4);
}

__global__ void k_topo_plan(int cap_arcs, Adj out, Adj in, const int *ins_src, const int *ins_dst,
                            const int *ins_rank, RelocItem *reloc, Counters *c) {
  const long long ni = 2 * static_cast<long long>(c->n_ins);
  const long long stride = static_cast<long long>(gridDim.x) * blockDim.x;
  for (long long w = blockIdx.x * blockDim.x + threadIdx.x; w < ni; w += stride) {
    if (ins_rank[w] != 0) continue;  // one planner per row
    int dir, row, entry;
    item_row(w, ins_src, ins_dst, dir, row, entry);
    const Adj &a = dir ? in : out;
    const int newlen = a.len[row] - a.delcnt[row] + a.inscnt[row];
    if (newlen > a.cap[row]) {
      const int nc = grow_cap(newlen);
      const u64 j = atomicAdd(&c->n_reloc, 1ull);
      reloc[j] = RelocItem{row, dir, nc, 0};
      atomicAdd(&c->arena_need[dir], static_cast<u64>(nc));
    }
  }
}

__global__ void k_topo_check(Counters *c, const Persist *p, long long cap_out, long long cap_in) {
  if (threadIdx.x != 0 || blockIdx.x != 0) return;
  const bool over0 = p->top[0] + c->arena_need[0] > static_cast<u64>(cap_out);
  const bool over1 = p->top[1] + c->arena_need[1] > static_cast<u64>(cap_in);
  if (over0 || over1) c->abort = 1;
}

// Pre-batch corrections, one per net arc (u,v) and layer l: an inserted arc adds
// u's pre-batch contribution to S^l_v, a deleted arc removes it (an insert is a
// message whose old embedding is zero, a delete one whose new embedding is zero).
// Runs before any adjacency, feature or embedding write, so H and degrees are the
// pre-batch ones.
__global__ void k_corrections(int agg, LayerPtrs lp, const int *out_len, const int *ins_src,
                              const int *ins_dst, const int *del_src, const int *del_dst, Counters *c) {
  if (c->abort) return;
  const int lane = lane_id();
  const long long ni = static_cast<long long>(c->n_ins);
  const long long na = ni + static_cast<long long>(c->n_del);
  const long long items = na * lp.L;
  for (long long it = global_wave(); it < items; it += num_waves()) {
    const long long arc = it / lp.L;
    const int l = static_cast<int>(it % lp.L) + 1;
    const bool ins = arc < ni;
    const int u = ins ? ins_src[arc] : del_src[arc - ni];
    const int v = ins ? ins_dst[arc] : del_dst[arc - ni];
    float coef = ins ? 1.0f : -1.0f;
    if (agg == kGcn) coef *= 1.0f / sqrtf(static_cast<float>(out_len[u]) + 1.0f);
    const int d = lp.dims[l - 1];
    const float *hu = lp.H[l - 1] + static_cast<long long>(u) * d;
    float *sv = lp.S[l] + static_cast<long long>(v) * d;
    for (int k = lane; k < d; k += kWave) unsafeAtomicAdd(&sv[k], coef * hu[k]);
  }
}

// Deletes: tombstone, fill surviving holes from the tail, shrink the row.
__global__ void k_del_find(Adj out, Adj in, const int *del_src, const int *del_dst, int *del_pos,
                           Counters *c) {
  if (c->abort) return;
  const long long nd = 2 * static_cast<long long>(c->n_del);
  for (long long w = global_wave(); w < nd; w += num_waves()) {
    int dir, row, entry;
    item_row(w, del_src, del_dst, dir, row, entry);
    const Adj &a = dir ? in : out;
    int *r = a.col + a.off[row];
    const int pos = wave_find(r, a.len[row], entry);
    if (lane_id() == 0) {
      del_pos[w] = pos;
      if (pos < 0) {
        atomicOr(&c->err, 1ull);
      } else {
        r[pos] = -1;
      }
    }
  }
}

__global__ void k_del_fill(Adj out, Adj in, const int *del_src, const int *del_dst, const int *del_pos,
                           Counters *c) {
  if (c->abort) return;
  const long long nd = 2 * static_cast<long long>(c->n_del);
  const long long stride = static_cast<long long>(gridDim.x) * blockDim.x;
  for (long long w = blockIdx.x * blockDim.x + threadIdx.x; w < nd; w += stride) {
    int dir, row, entry;
    item_row(w, del_src, del_dst, dir, row, entry);
    const Adj &a = dir ? in : out;
    const int p = del_pos[w];
    const int len = a.len[row], k = a.delcnt[row];
    if (p < 0 || p >= len - k) continue;  // hole lies in the part that is cut off
    const int j = atomicAdd(&a.fillcnt[row], 1);
    int *r = a.col + a.off[row];
    int seen = 0;
    for (int e = len - k; e < len; ++e) {
      const int val = r[e];
      if (val < 0) continue;
      if (seen == j) {
        r[p] = val;
        break;
      }
      ++seen;
    }
  }
}

__global__ void k_del_finish(Adj out, Adj in, const int *del_src, const int *del_dst, const int *del_rank,
                             int *ddeg, Counters *c) {
  if (c->abort) return;
  const long long nd = 2 * static_cast<long long>(c->n_del);
  const long long stride = static_cast<long long>(gridDim.x) * blockDim.x;
  for (long long w = blockIdx.x * blockDim.x + threadIdx.x; w < nd; w += stride) {
    if (del_rank[w] != 0) continue;
    int dir, row, entry;
    item_row(w, del_src, del_dst, dir, row, entry);
    const Adj &a = dir ? in : out;
    const int k = a.delcnt[row];
    a.len[row] -= k;
    if (dir == 0) ddeg[row] -= k;
  }
}

__global__ void k_reloc(Adj out, Adj in, const RelocItem *reloc, Persist *p, Counters *c) {
  if (c->abort) return;
  const long long nr = static_cast<long long>(c->n_reloc);
  const int lane = lane_id();
  for (long long j = global_wave(); j < nr; j += num_waves()) {
    const RelocItem it = reloc[j];
    const Adj &a = it.dir ? in : out;
    long long base = 0;
    if (lane == 0) base = static_cast<long long>(atomicAdd(&p->top[it.dir], static_cast<u64>(it.newcap)));
    base = __shfl(base, 0);
    const int *src = a.col + a.off[it.row];
    int *dst = a.col + base;
    const int len = a.len[it.row];
    for (int e = lane; e < len; e += kWave) dst[e] = src[e];
    if (lane == 0) {
      a.off[it.row] = base;
      a.cap[it.row] = it.newcap;
    }
  }
}

__global__ void k_ins_put(Adj out, Adj in, const int *ins_src, const int *ins_dst, const int *ins_rank,
                          Counters *c) {
  if (c->abort) return;
  const long long ni = 2 * static_cast<long long>(c->n_ins);
  const long long stride = static_cast<long long>(gridDim.x) * blockDim.x;
  for (long long w = blockIdx.x * blockDim.x + threadIdx.x; w < ni; w += stride) {
    int dir, row, entry;
    item_row(w, ins_src, ins_dst, dir, row, entry);
    const Adj &a = dir ? in : out;
    a.col[a.off[row] + a.len[row] + ins_rank[w]] = entry;
  }
}

__global__ void k_ins_finish(Adj out, Adj in, const int *ins_src, const int *ins_dst, const int *ins_rank,
                             int *ddeg, Counters *c) {
  if (c->abort) return;
  const long long ni = 2 * static_cast<long long>(c->n_ins);
  const long long stride = static_cast<long long>(gridDim.x) * blockDim.x;
  for (long long w = blockIdx.x * blockDim.x + threadIdx.x; w < ni; w += stride) {
    if (ins_rank[w] != 0) continue;
    int dir, row, entry;
    item_row(w, ins_src, ins_dst, dir, row, entry);
    const Adj &a = dir ? in : out;
    const int k = a.inscnt[row];
    a.len[row] += k;
    if (dir == 0) ddeg[row] += k;
  }
}

// Resets every per-batch scratch word the batch touched (runs even after an abort).
__global__ void k_cleanup(int B, const ripple_op *ops, const int *op_slot, u64 *ht_key, int *ht_val,
                          int *fop, Adj out, Adj in, const int *ins_src, const int *ins_dst,
                          const int *del_src, const int *del_dst, int *ddeg, const Counters *c) {
  const long long ni = 2 * static_cast<long long>(c->n_ins);
  const long long nd = 2 * static_cast<long long>(c->n_del);
  const long long stride = static_cast<long long>(gridDim.x) * blockDim.x;
  const long long t0 = blockIdx.x * blockDim.x + threadIdx.x;
  for (long long w = t0; w < ni; w += stride) {
    int dir, row, entry;
    item_row(w, ins_src, ins_dst, dir, row, entry);
    (dir ? in : out).inscnt[row] = 0;
    if (dir == 0) ddeg[row] = 0;
  }
  for (long long w = t0; w < nd; w += stride) {
    int dir, row, entry;
    item_row(w, del_src, del_dst, dir, row, entry);
    const Adj &a = dir ? in : out;
    a.delcnt[row] = 0;
    a.fillcnt[row] = 0;
    if (dir == 0) ddeg[row] = 0;
  }
  for (long long i = t0; i < B; i += stride) {
    const int s = op_slot[i];
    if (s >= 0) {
      ht_key[s] = kEmptyKey;
      ht_val[s] = -1;
    }
    if (ops[i].kind == RIPPLE_OP_FEATURE) fop[ops[i].u] = -1;
  }
}

inline int blocks_for(long long items, int threads, int cap = 4096) {
  long long b = (items + threads - 1) / threads;
  if (b < 1) b = 1;
  if (b > cap) b = cap;
  return static_cast<int>(b);
}

}  // namespace

void launch_net_hash(hipStream_t s, const ripple_op *ops, int B, int undirected, long long n, u64 *ht_key,
                     int *ht_val, unsigned mask, int *op_slot, int *fop, Counters *c) {
  if (B <= 0) return;
  hipLaunchKernelGGL(k_net_hash, dim3(blocks_for(B, 256, 1 << 20)), dim3(256), 0, s, ops, B, undirected, n,
                     ht_key, ht_val, mask, op_slot, fop, c);
}

void launch_net_decide(hipStream_t s, const ripple_op *ops, int B, int undirected, const int *ht_val,
                       const int *op_slot, const int *fop, Adj out, Adj in, int *ins_src, int *ins_dst,
                       int *del_src, int *del_dst, int *flist, Counters *c) {
  if (B <= 0) return;
  hipLaunchKernelGGL(k_net_decide, dim3(blocks_for(static_cast<long long>(B) * kWave, 256)), dim3(256), 0, s,
                     ops, B, undirected, ht_val, op_slot, fop, out, in, ins_src, ins_dst, del_src, del_dst,
                     flist, c);
}

void launch_topo_count(hipStream_t s, int cap_arcs, Adj out, Adj in, const int *ins_src, const int *ins_dst,
                       const int *del_src, const int *del_dst, int *ins_rank, int *del_rank, Counters *c) {
  hipLaunchKernelGGL(k_topo_count, dim3(blocks_for(4LL * cap_arcs, 256)), dim3(256), 0, s, cap_arcs, out, in,
                     ins_src, ins_dst, del_src, del_dst, ins_rank, del_rank, c);
}

void launch_topo_plan(hipStream_t s, int cap_arcs, Adj out, Adj in, const int *ins_src, const int *ins_dst,
                      const int *ins_rank, RelocItem *reloc, Counters *c) {
  hipLaunchKernelGGL(k_topo_plan, dim3(blocks_for(2LL * cap_arcs, 256)), dim3(256), 0, s, cap_arcs, out, in,
                     ins_src, ins_dst, ins_rank, reloc, c);
}

void launch_topo_check(hipStream_t s, Counters *c, const Persist *p, long long cap_out, long long cap_in) {
  hipLaunchKernelGGL(k_topo_check, dim3(1), dim3(64), 0, s, c, p, cap_out, cap_in);
}

void launch_corrections(hipStream_t s, int cap_arcs, int agg, LayerPtrs lp, const int *out_len,
                        const int *ins_src, const int *ins_dst, const int *del_src, const int *del_dst,
                        Counters *c) {
  hipLaunchKernelGGL(k_corrections, dim3(blocks_for(2LL * cap_arcs * lp.L * kWave, 256)), dim3(256), 0, s,
                     agg, lp, out_len, ins_src, ins_dst, del_src, del_dst, c);
}

void launch_del_apply(hipStream_t s, int cap_arcs, Adj out, Adj in, const int *del_src, const int *del_dst,
                      const int *del_rank, int *del_pos, int *ddeg, Counters *c) {
  hipLaunchKernelGGL(k_del_find, dim3(blocks_for(2LL * cap_arcs * kWave, 256)), dim3(256), 0, s, out, in,
                     del_src, del_dst, del_pos, c);
  hipLaunchKernelGGL(k_del_fill, dim3(blocks_for(2LL * cap_arcs, 256)), dim3(256), 0, s, out, in, del_src,
                     del_dst, del_pos, c);
  hipLaunchKernelGGL(k_del_finish, dim3(blocks_for(2LL * cap_arcs, 256)), dim3(256), 0, s, out, in, del_src,
                     del_dst, del_rank, ddeg, c);
}

void launch_reloc(hipStream_t s, int cap_reloc, Adj out, Adj in, const RelocItem *reloc, Persist *p,
                  Counters *c) {
  hipLaunchKernelGGL(k_reloc, dim3(blocks_for(static_cast<long long>(cap_reloc) * kWave, 256)), dim3(256), 0, s,
                     out, in, reloc, p, c);
}

void launch_ins_apply(hipStream_t s, int cap_arcs, Adj out, Adj in, const int *ins_src, const int *ins_dst,
                      const int *ins_rank, int *ddeg, Counters *c) {
  hipLaunchKernelGGL(k_ins_put, dim3(blocks_for(2LL * cap_arcs, 256)), dim3(256), 0, s, out, in, ins_src,
                     ins_dst, ins_rank, c);
  hipLaunchKernelGGL(k_ins_finish, dim3(blocks_for(2LL * cap_arcs, 256)), dim3(256), 0, s, out, in, ins_src,
                     ins_dst, ins_rank, ddeg, c);
}

void launch_cleanup(hipStream_t s, int B, int cap_arcs, const ripple_op *ops, const int *op_slot, u64 *ht_key,
                    int *ht_val, int *fop, Adj out, Adj in, const int *ins_src, const int *ins_dst,
                    const int *del_src, const int *del_dst, int *ddeg, const Counters *c) {
  const long long items = 2LL * cap_arcs > B ? 2LL * cap_arcs : B;
  hipLaunchKernelGGL(k_cleanup, dim3(blocks_for(items, 256)), dim3(256), 0, s, B, ops, op_slot, ht_key, ht_val,
                     fop, out, in, ins_src, ins_dst, del_src, del_dst, ddeg, c);
}

}  // namespace rp

namespace rp {

namespace {

// Re-layout: row u's used entries move from old_col[old_off[u]..] to new_col[new_off[u]..].
__global__ void k_repack_copy(long long n, const int *old_col, const long long *old_off, const int *len,
                              int *new_col, const long long *new_off) {
  const int lane = threadIdx.x & (kWave - 1);
  const long long nw = static_cast<long long>(gridDim.x) * blockDim.x / kWave;
  for (long long u = (static_cast<long long>(blockIdx.x) * blockDim.x + threadIdx.x) / kWave; u < n; u += nw) {
    const int *src = old_col + old_off[u];
    int *dst = new_col + new_off[u];
    const int l = len[u];
    for (int e = lane; e < l; e += kWave) dst[e] = src[e];
  }
}

}  // namespace

void launch_repack_copy(hipStream_t s, long long n, const int *old_col, const long long *old_off, const int *len,
                        int *new_col, const long long *new_off) {
  long long blocks = (n * kWave + 255) / 256;
  if (blocks > 8192) blocks = 8192;
  if (blocks < 1) blocks = 1;
  hipLaunchKernelGGL(k_repack_copy, dim3(blocks), dim3(256), 0, s, n, old_col, old_off, len, new_col, new_off);
}

}  // namespace rp
