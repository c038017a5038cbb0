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

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "ripple.h"

namespace rp {

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
  u64 err;                // device-detected inconsistency (bit 0: deleted arc not found)
  u64 count[kMaxL + 1];   // [0] = |dirty set of layer 1|, [l] = |A^l|
  u64 pushed[kMaxL + 1];  // [l] = out-arcs pushed at layer l
  u64 dest[kMaxL + 1];    // [l] = distinct sinks of those arcs
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
  int *inscnt;            // per-row scratch, zero between batches
  int *delcnt;
  int *fillcnt;
};

struct RelocItem {
  int row;
  int dir;
  int newcap;
  int pad;
};

struct LayerPtrs {
  float *H[kMaxL + 1];
  float *S[kMaxL + 1];
  int dims[kMaxL + 1];
  int L;
};

enum Agg { kSum = 0, kMean = 1, kGcn = 2 };

// --- launchers (each defined in the translation unit that holds its kernel) ---

// netting
void launch_net_hash(hipStream_t s, const ripple_op *ops, int B, int undirected, long long n,
                     u64 *ht_key, int *ht_val, unsigned mask, int *op_slot, int *fop, Counters *c);
void launch_net_decide(hipStream_t s, const ripple_op *ops, int B, int undirected, const int *ht_val,
                       const int *op_slot, const int *fop, Adj out, Adj in, int *ins_src, int *ins_dst,
                       int *del_src, int *del_dst, int *flist, Counters *c);

// topology (cap_arcs bounds n_ins and n_del)
void launch_topo_count(hipStream_t s, int cap_arcs, Adj out, Adj in, const int *ins_src, const int *ins_dst,
                       const int *del_src, const int *del_dst, int *ins_rank, int *del_rank, Counters *c);
void launch_topo_plan(hipStream_t s, int cap_arcs, Adj out, Adj in, const int *ins_src, const int *ins_dst,
                      const int *ins_rank, RelocItem *reloc, Counters *c);
void launch_topo_check(hipStream_t s, Counters *c, const Persist *p, long long cap_out, long long cap_in);
void launch_corrections(hipStream_t s, int cap_arcs, int agg, LayerPtrs lp, const int *out_len,
                        const int *ins_src, const int *ins_dst, const int *del_src, const int *del_dst,
                        Counters *c);
void launch_del_apply(hipStream_t s, int cap_arcs, Adj out, Adj in, const int *del_src, const int *del_dst,
                      const int *del_rank, int *del_pos, int *ddeg, Counters *c);
void launch_reloc(hipStream_t s, int cap_reloc, Adj out, Adj in, const RelocItem *reloc, Persist *p,
                  Counters *c);
void launch_ins_apply(hipStream_t s, int cap_arcs, Adj out, Adj in, const int *ins_src, const int *ins_dst,
                      const int *ins_rank, int *ddeg, Counters *c);
void launch_cleanup(hipStream_t s, int B, int cap_arcs, const ripple_op *ops, const int *op_slot,
                    u64 *ht_key, int *ht_val, int *fop, Adj out, Adj in, const int *ins_src,
                    const int *ins_dst, const int *del_src, const int *del_dst, int *ddeg,
                    const Counters *c);

// frontier
void launch_mark_dirty0(hipStream_t s, int cap_feat, int cap_arcs, int gcn, const int *flist,
                        const int *ins_src, const int *del_src, const int *ddeg, unsigned *bm, Counters *c);
int compact_blocks(long long n);
void launch_compact(hipStream_t s, long long n, unsigned *bm_a, unsigned *bm_b, int *blocksum,
                    int *list_out, u64 *count_out);

// layer 0 deltas
void launch_delta0(hipStream_t s, long long n, int agg, int d0, const int *list, const u64 *count,
                   const ripple_op *ops, const float *feat, const int *fop, float *X, const int *out_len,
                   const int *ddeg, float *delta, const Counters *c);

// scatter: S^l[v] += delta[j] for every post-batch out-arc (list[j] -> v); marks sinks
// in bm_out, the dirty vertices and the sinks of net arcs in bm_x.
void launch_scatter(hipStream_t s, long long n, int d, const int *list, const u64 *count, const float *delta,
                    Adj out, float *S, unsigned *bm_out, unsigned *bm_x, const int *ins_dst,
                    const int *del_dst, int cap_arcs, u64 *pushed, u64 *dest, const Counters *c);

// bootstrap pull: S[v] = sum over in-arcs c_u H[u]
void launch_pull(hipStream_t s, long long n, int d, int agg, const float *Hprev, Adj in, const int *out_len,
                 float *S);

// transform: for rows r < M (M = *count or count_fixed), v = rows ? rows[r] : r:
//   y = act(W [h_v || t_v S_v] + b)      (SAGE; t_v = 1 or 1/din(v))
//   y = act(W t_v (S_v + s_v h_v) + b)   (GCN; t_v = 1/sqrt(din+1), s_v = 1/sqrt(dout+1))
// then, when delta != nullptr, delta[r] = c'_v y - c_v H[v] (c = 1, or s_v post/pre
// batch under GCN), and H[v] = y.
struct GemmArgs {
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
  int K;
  int N;
  const float *bias;
  int relu;
  float *H;
  float *delta;
  int agg;
  const u64 *abort;
};
void launch_gemm(hipStream_t s, const GemmArgs &a, long long max_rows);

// re-layout of one adjacency direction
void launch_repack_copy(hipStream_t s, long long n, const int *old_col, const long long *old_off, const int *len,
                        int *new_col, const long long *new_off);

// utilities
void launch_fill_i32(hipStream_t s, int *p, long long count, int value);
void launch_fill_u64(hipStream_t s, u64 *p, long long count, u64 value);
void launch_gather_rows(hipStream_t s, const float *src, int d, const int *ids, long long count, float *out);

}  // namespace rp
