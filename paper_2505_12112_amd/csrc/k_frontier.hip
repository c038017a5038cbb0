// Frontier and message kernels.
//
// Per layer l the dirty set D^l (vertices whose layer-(l-1) contribution changed)
// pushes its delta rows along every post-batch out-arc into the cached aggregate
// S^l (Sec. IV-C.1: a message carries the new minus the old embedding and the
// receiver adds it to its mailbox), and the affected set
//   A^l = out(D^l) u sinks(net arcs) u D^l
// is collected in two bitmaps (one for the out-arc sinks, so that their distinct
// count is known exactly) and compacted into a sorted list by a popcount prefix
// sum, which also yields each listed vertex's first out-arc index for the next
// layer's scatter.
#include "internal.h"

namespace rp {

namespace {

constexpr int kCompactThreads = 256;
constexpr int kCompactWaves = kCompactThreads / kWave;
constexpr int kWordsPerThread = 4;
constexpr int kWordsPerBlock = kCompactThreads * kWordsPerThread;

__device__ inline int lane_id() { return threadIdx.x & (kWave - 1); }

__device__ inline long long global_wave() {
  return (static_cast<long long>(blockIdx.x) * blockDim.x + threadIdx.x) / kWave;
}

__device__ inline long long num_waves() {
  return static_cast<long long>(gridDim.x) * blockDim.x / kWave;
}

__device__ inline bool mark(unsigned *bm, int v) {
  const unsigned bit = 1u << (v & 31);
  return (atomicOr(&bm[v >> 5], bit) & bit) == 0;
}

inline int blocks_for(long long items, int threads, int cap = 4096) {
  long long b = (items + threads - 1) / threads;
  if (b < 1) b = 1;
  if (b > cap) b = cap;
  return static_cast<int>(b);
}

// Exclusive scan of v over the block; *total receives the block sum.
template <typename T>
__device__ inline T block_exclusive_scan(T v, T *lds, T *total) {
  const int lane = lane_id(), wave = threadIdx.x / kWave;
  T x = v;
#pragma unroll
  for (int o = 1; o < kWave; o <<= 1) {
    const T y = __shfl_up(x, o);
    if (lane >= o) x += y;
  }
  if (lane == kWave - 1) lds[wave] = x;
  __syncthreads();
  if (threadIdx.x == 0) {
    T run = 0;
    for (int w = 0; w < kCompactWaves; ++w) {
      const T t = lds[w];
      lds[w] = run;
      run += t;
    }
    lds[kCompactWaves] = run;
  }
  __syncthreads();
  const T excl = x - v + lds[wave];
  *total = lds[kCompactWaves];
  __syncthreads();
  return excl;
}

template <typename T>
__device__ inline T block_sum(T v, T *lds) {
  T total;
  block_exclusive_scan(v, lds, &total);
  return total;
}

// Pre-batch corrections and the layer-1 dirty marks (see launch_corr_mark).
__global__ void k_corr_mark(int agg, LayerPtrs lp, const int *out_len, const int *ddeg, const int *flist,
                            const int *ins_src, const int *ins_dst, const int *del_src, const int *del_dst,
                            unsigned *bm, Counters *c) {
  if (c->abort) return;
  const int lane = lane_id();
  const long long nf = static_cast<long long>(c->n_feat);
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
    if (agg == kGcn) coef *= 1.0f / sqrtf(static_cast<float>(out_len[u] - ddeg[u]) + 1.0f);
    const int d = lp.sw[l];
    const float *hu = lp.src[l] + static_cast<long long>(u) * d;
    float *sv = lp.S[l] + static_cast<long long>(v) * d;
    for (int k = lane; k < d; k += kWave) unsafeAtomicAdd(&sv[k], coef * hu[k]);
  }
  const long long total = nf + (agg == kGcn ? na : 0);
  const long long stride = static_cast<long long>(gridDim.x) * blockDim.x;
  for (long long i = blockIdx.x * blockDim.x + threadIdx.x; i < total; i += stride) {
    if (i < nf) {
      mark(bm, flist[i]);
    } else {
      const long long a = i - nf;
      const int u = a < ni ? ins_src[a] : del_src[a - ni];
      if (ddeg[u] != 0) mark(bm, u);
    }
  }
}

__device__ inline void word_stats(unsigned w, long long vbase, const int *odeg, const int *ideg, int &cnt,
                                  long long &dsum, long long &isum) {
  cnt += __popc(w);
  if (odeg != nullptr || ideg != nullptr) {
    while (w) {
      const int b = __ffs(w) - 1;
      if (odeg != nullptr) dsum += odeg[vbase + b];
      if (ideg != nullptr) isum += ideg[vbase + b];
      w &= w - 1;
    }
  }
}

__global__ __launch_bounds__(kCompactThreads) void k_compact_count(const unsigned *bm_a, const unsigned *bm_b,
                                                                   long long words, const int *odeg,
                                                                   const int *ideg, int *blocksum,
                                                                   long long *blockdeg) {
  __shared__ long long red[kCompactWaves + 1];
  const long long w0 = static_cast<long long>(blockIdx.x) * kWordsPerBlock + threadIdx.x * kWordsPerThread;
  int cnt = 0;
  long long dsum = 0, isum = 0;
#pragma unroll
  for (int i = 0; i < kWordsPerThread; ++i) {
    const long long w = w0 + i;
    if (w < words) word_stats(bm_a[w] | bm_b[w], w * 32, odeg, ideg, cnt, dsum, isum);
  }
  const long long tc = block_sum<long long>(cnt, red);
  const long long td = block_sum<long long>(dsum, red);
  const long long ti = block_sum<long long>(isum, red);
  if (threadIdx.x == 0) {
    blocksum[blockIdx.x] = static_cast<int>(tc);
    blockdeg[2 * blockIdx.x] = td;
    blockdeg[2 * blockIdx.x + 1] = ti;
  }
}

__global__ __launch_bounds__(kCompactThreads) void k_compact_emit(unsigned *bm_a, unsigned *bm_b, long long words,
                                                                  const int *blocksum, const long long *blockdeg,
                                                                  CompactOut o) {
  __shared__ long long red[kCompactWaves + 1];
  long long pre = 0, pred = 0, prei = 0;
  for (int b = threadIdx.x; b < static_cast<int>(blockIdx.x); b += kCompactThreads) {
    pre += blocksum[b];
    pred += blockdeg[2 * b];
    prei += blockdeg[2 * b + 1];
  }
  const long long base = block_sum<long long>(pre, red);
  const long long dbase = block_sum<long long>(pred, red);
  const long long ibase = block_sum<long long>(prei, red);
  const long long w0 = static_cast<long long>(blockIdx.x) * kWordsPerBlock + threadIdx.x * kWordsPerThread;
  const int *odeg = o.doff != nullptr ? o.out_deg : nullptr;
  const int *ideg = o.ioff != nullptr ? o.in_deg : nullptr;  // prefix only when wanted
  unsigned wv[kWordsPerThread];
  int cnt = 0;
  long long dsum = 0, isum = 0;
#pragma unroll
  for (int i = 0; i < kWordsPerThread; ++i) {
    const long long w = w0 + i;
    wv[i] = w < words ? (bm_a[w] | bm_b[w]) : 0u;
    word_stats(wv[i], w * 32, odeg, ideg, cnt, dsum, isum);
  }
  long long tot_c, tot_d, tot_i;
  long long pos = base + block_exclusive_scan<long long>(cnt, red, &tot_c);
  long long dpos = dbase + block_exclusive_scan<long long>(dsum, red, &tot_d);
  long long ipos = ibase + block_exclusive_scan<long long>(isum, red, &tot_i);
#pragma unroll
  for (int i = 0; i < kWordsPerThread; ++i) {
    unsigned m = wv[i];
    const long long vbase = (w0 + i) * 32;
    while (m) {
      const int b = __ffs(m) - 1;
      const int v = static_cast<int>(vbase + b);
      o.list[pos] = v;
      if (odeg != nullptr) {
        o.doff[pos] = dpos;
        dpos += odeg[v];
      }
      if (ideg != nullptr) {
        o.ioff[pos] = ipos;
        ipos += ideg[v];
      }
      if (o.slot != nullptr) o.slot[v] = static_cast<int>(pos);
      ++pos;
      m &= m - 1;
    }
    const long long w = w0 + i;
    if (w < words) {
      if (o.keep != nullptr) o.keep[w] = wv[i];
      bm_a[w] = 0u;
      bm_b[w] = 0u;
    }
  }
  if (blockIdx.x == gridDim.x - 1 && threadIdx.x == 0) {
    const long long total = base + tot_c;
    *o.count = static_cast<u64>(total);
    if (odeg != nullptr) o.doff[total] = dbase + tot_d;
    if (ideg != nullptr) o.ioff[total] = ibase + tot_i;
    // the count kernel summed in-degrees per block, also when no prefix is wanted
    if (o.in_total != nullptr) *o.in_total = static_cast<u64>(ibase + blockdeg[2 * blockIdx.x + 1]);
  }
}

// One-block form of the compaction for small graphs (one launch instead of two):
// 1024 threads walk the bitmap words in rounds, carrying the running offsets.
constexpr int kSingleThreads = 1024;
constexpr int kSingleWaves = kSingleThreads / kWave;

__device__ inline long long single_scan(long long v, long long *lds, long long *total) {
  const int lane = lane_id(), wave = threadIdx.x / kWave;
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
    for (int w = 0; w < kSingleWaves; ++w) {
      const long long t = lds[w];
      lds[w] = run;
      run += t;
    }
    lds[kSingleWaves] = run;
  }
  __syncthreads();
  const long long excl = x - v + lds[wave];
  *total = lds[kSingleWaves];
  __syncthreads();
  return excl;
}

__global__ __launch_bounds__(kSingleThreads) void k_compact_single(unsigned *bm_a, unsigned *bm_b, long long words,
                                                                   CompactOut o) {
  __shared__ long long red[kSingleWaves + 1];
  const int *odeg = o.doff != nullptr ? o.out_deg : nullptr;
  const int *ideg = (o.ioff != nullptr || o.in_total != nullptr) ? o.in_deg : nullptr;
  long long pos = 0, dpos = 0, ipos = 0;
  for (long long r0 = 0; r0 < words; r0 += static_cast<long long>(kSingleThreads) * kWordsPerThread) {
    const long long w0 = r0 + static_cast<long long>(threadIdx.x) * kWordsPerThread;
    unsigned wv[kWordsPerThread];
    int cnt = 0;
    long long dsum = 0, isum = 0;
#pragma unroll
    for (int i = 0; i < kWordsPerThread; ++i) {
      const long long w = w0 + i;
      wv[i] = w < words ? (bm_a[w] | bm_b[w]) : 0u;
      word_stats(wv[i], w * 32, odeg, ideg, cnt, dsum, isum);
    }
    long long tc, td, ti;
    long long p = pos + single_scan(cnt, red, &tc);
    long long dp = dpos + single_scan(dsum, red, &td);
    long long ip = ipos + single_scan(isum, red, &ti);
#pragma unroll
    for (int i = 0; i < kWordsPerThread; ++i) {
      unsigned m = wv[i];
      const long long vbase = (w0 + i) * 32;
      while (m) {
        const int b = __ffs(m) - 1;
        const int v = static_cast<int>(vbase + b);
        o.list[p] = v;
        if (odeg != nullptr) {
          o.doff[p] = dp;
          dp += odeg[v];
        }
        if (o.ioff != nullptr) {
          o.ioff[p] = ip;
          ip += ideg[v];
        }
        if (o.slot != nullptr) o.slot[v] = static_cast<int>(p);
        ++p;
        m &= m - 1;
      }
      const long long w = w0 + i;
      if (w < words) {
        if (o.keep != nullptr) o.keep[w] = wv[i];
        bm_a[w] = 0u;
        bm_b[w] = 0u;
      }
    }
    pos += tc;
    dpos += td;
    ipos += ti;
  }
  if (threadIdx.x == 0) {
    *o.count = static_cast<u64>(pos);
    if (odeg != nullptr) o.doff[pos] = dpos;
    if (o.ioff != nullptr) o.ioff[pos] = ipos;
    if (o.in_total != nullptr) *o.in_total = static_cast<u64>(ipos);
  }
}

// Layer-0 deltas: for each dirty vertex u (slot j), the new feature row is the
// last write of the batch (or the unchanged row), delta = c'_u x'_u - c_u x_u, and
// the feature row is overwritten.
__global__ void k_delta0(int agg, int d0, const int *list, const u64 *count, const ripple_op *ops,
                         const float *feat, const int *fop, float *X, const int *out_len, const int *ddeg,
                         float *delta, const Counters *c) {
  if (c->abort) return;
  const long long m = static_cast<long long>(*count);
  const int lane = lane_id();
  for (long long j = global_wave(); j < m; j += num_waves()) {
    const int u = list[j];
    const int fo = fop[u];
    float cn = 1.0f, co = 1.0f;
    if (agg == kGcn) {
      cn = 1.0f / sqrtf(static_cast<float>(out_len[u]) + 1.0f);
      co = 1.0f / sqrtf(static_cast<float>(out_len[u] - ddeg[u]) + 1.0f);
    }
    float *xu = X + static_cast<long long>(u) * d0;
    const float *xn = fo >= 0 ? feat + static_cast<long long>(ops[fo].feat_row) * d0 : xu;
    float *dj = delta + j * d0;
    for (int k = lane; k < d0; k += kWave) {
      const float xo = xu[k];
      const float x1 = xn[k];
      dj[k] = cn * x1 - co * xo;
      xu[k] = x1;
    }
  }
}

// First index i in [lo, hi) with a[i] > x (hi if none).
__device__ inline long long upper_bound(const long long *a, long long lo, long long hi, long long x) {
  while (lo < hi) {
    const long long mid = (lo + hi) >> 1;
    if (a[mid] <= x) lo = mid + 1;
    else hi = mid;
  }
  return lo;
}

// Last index j in [lo, hi) with a[j] <= x, for non-decreasing a with a[lo] <= x.
// The whole wave searches together: each round probes 64 evenly spaced entries
// with one load and keeps the gap after the last probe that is <= x, so a search
// over m entries takes ceil(log64 m) dependent loads instead of log2 m.
__device__ inline long long wave_last_le(const long long *a, long long lo, long long hi, long long x) {
  const int lane = lane_id();
  while (hi - lo > kWave) {
    const long long step = (hi - lo + kWave - 1) / kWave;
    const long long idx = lo + lane * step;
    const bool le = idx < hi && a[idx] <= x;
    const int last = __popcll(__ballot(le)) - 1;  // probes <= x form a prefix
    lo = lo + last * step;
    hi = lo + step < hi ? lo + step : hi;
  }
  const long long idx = lo + lane;
  const bool le = idx < hi && a[idx] <= x;
  return lo + __popcll(__ballot(le)) - 1;
}

// Edge-parallel scatter. Pushed arcs are numbered: arc e of listed vertex j has
// index doff[j] + its position in j's out-row. A wave takes a chunk of C
// consecutive arcs (C = 1 when there are few arcs, so that many waves run at
// once; up to 64 when there are many), each lane resolves one arc's source slot
// and sink and marks the sink, then G lanes per arc add the source's delta row
// into the sink's row of S with fp32 atomics (coalesced across the G lanes). The
// delta row stays in registers while consecutive arcs share a source, so a hub's
// arcs cost one row load per chunk; hubs spread over many waves.
template <int G, int NC, bool PUSH>
__global__ __launch_bounds__(256) void k_scatter(int d, const int *list, const u64 *count, const long long *doff,
                                                 const float *delta, Adj out, float *S, unsigned *bm_out,
                                                 unsigned *bm_x, const int *ins_dst, const int *del_dst,
                                                 u64 *pushed, u64 *dest, const Counters *c) {
  if (c->abort) return;
  const int lane = lane_id();
  const long long nD = static_cast<long long>(*count);
  const long long E = doff[nD];
  {
    const long long ni = static_cast<long long>(c->n_ins);
    const long long na = ni + static_cast<long long>(c->n_del);
    const long long stride = static_cast<long long>(gridDim.x) * blockDim.x;
    const long long t0 = blockIdx.x * blockDim.x + threadIdx.x;
    for (long long i = t0; i < na; i += stride) mark(bm_x, i < ni ? ins_dst[i] : del_dst[i - ni]);
    for (long long j = t0; j < nD; j += stride) mark(bm_x, list[j]);
    if (t0 == 0) *pushed = static_cast<u64>(E);
  }
  const long long waves = num_waves();
  int C = 1;
  while (C < kWave && static_cast<long long>(C) * waves < E) C <<= 1;
  constexpr int kEdgesPerStep = kWave / G;
  const int grp = lane / G, k0 = lane % G;
  u64 my_dest = 0;
  int cached = -1;
  float dreg[NC];
  const long long chunks = (E + C - 1) / C;
  for (long long ch = global_wave(); ch < chunks; ch += waves) {
    const long long e0 = ch * C;
    const long long elast = e0 + C - 1 < E - 1 ? e0 + C - 1 : E - 1;
    const long long ja = wave_last_le(doff, 0, nD + 1, e0);
    const long long jb = C == 1 ? ja : wave_last_le(doff, ja, nD + 1, elast);
    const long long e = e0 + lane;
    const bool active = e <= elast;
    int j = static_cast<int>(ja);
    if (jb > ja) {
      if (jb - ja < kWave) {
        // the window's offsets, one per lane; every lane takes part in the shuffles
        const long long mine = ja + lane <= jb ? doff[ja + lane] : (1LL << 62);
        int cnt_le = 0;
        for (int t = 0; t <= static_cast<int>(jb - ja); ++t) cnt_le += __shfl(mine, t) <= e ? 1 : 0;
        j = static_cast<int>(ja) + cnt_le - 1;
      } else if (active) {
        j = static_cast<int>(upper_bound(doff, ja, jb + 1, e) - 1);
      }
    }
    int v = -1;
    if (active) {
      const int u = list[j];
      v = out.col[out.off[u] + (e - doff[j])];
    }
    const bool fresh = v >= 0 && mark(bm_out, v);
    my_dest += __popcll(__ballot(fresh));
    const int cnt = PUSH ? static_cast<int>(elast - e0 + 1) : 0;
    for (int i = 0; i < cnt; i += kEdgesPerStep) {
      const int vv = __shfl(v, i + grp);
      const int jj = __shfl(j, i + grp);
      if (vv >= 0) {
        if (jj != cached) {
          const float *dj = delta + static_cast<long long>(jj) * d;
#pragma unroll
          for (int q = 0; q < NC; ++q) {
            const int k = k0 + q * G;
            dreg[q] = k < d ? dj[k] : 0.0f;
          }
          cached = jj;
        }
        float *sv = S + static_cast<long long>(vv) * d;
#pragma unroll
        for (int q = 0; q < NC; ++q) {
          const int k = k0 + q * G;
          if (k < d) unsafeAtomicAdd(&sv[k], dreg[q]);
        }
      }
    }
  }
  if (lane == 0 && my_dest) atomicAdd(dest, my_dest);
}

// Pull form of the message step (for dense frontiers). In-arcs of the sorted
// list A are numbered like the scatter's out-arcs (ioff gives each listed
// vertex's first in-arc). A wave takes C consecutive in-arcs; each lane resolves
// one arc's sink v and source u and keeps it if u is dirty (member bit), with the
// source's message row msg[slot[u]]. The wave then walks its kept arcs in order,
// summing message rows into registers while the sink stays the same, and adds
// the sum to S[v] with one row of fp32 atomics per sink: a sink's messages cost
// one read each and one row update per wave instead of one atomic row each.
template <int NC>
__global__ __launch_bounds__(256) void k_pull_msgs(int d, const int *list, const u64 *count, const long long *ioff,
                                                   Adj in, const unsigned *member, const int *slot,
                                                   const float *msg, float *S, const Counters *c) {
  if (c->abort) return;
  const int lane = lane_id();
  const long long nA = static_cast<long long>(*count);
  const long long E = ioff[nA];
  const long long waves = num_waves();
  int C = 1;
  while (C < kWave && static_cast<long long>(C) * waves < E) C <<= 1;
  const long long chunks = (E + C - 1) / C;
  for (long long ch = global_wave(); ch < chunks; ch += waves) {
    const long long e0 = ch * C;
    const long long elast = e0 + C - 1 < E - 1 ? e0 + C - 1 : E - 1;
    const long long ja = wave_last_le(ioff, 0, nA + 1, e0);
    const long long jb = C == 1 ? ja : wave_last_le(ioff, ja, nA + 1, elast);
    const long long e = e0 + lane;
    const bool active = e <= elast;
    int r = static_cast<int>(ja);
    if (jb > ja) {
      if (jb - ja < kWave) {
        const long long mine = ja + lane <= jb ? ioff[ja + lane] : (1LL << 62);
        int cnt_le = 0;
        for (int t = 0; t <= static_cast<int>(jb - ja); ++t) cnt_le += __shfl(mine, t) <= e ? 1 : 0;
        r = static_cast<int>(ja) + cnt_le - 1;
      } else if (active) {
        r = static_cast<int>(upper_bound(ioff, ja, jb + 1, e) - 1);
      }
    }
    int v = -1, j = -1;
    if (active) {
      v = list[r];
      const int u = in.col[in.off[v] + (e - ioff[r])];
      if ((member[u >> 5] >> (u & 31)) & 1u) j = slot[u];
    }
    u64 keep = __ballot(j >= 0);
    int cur = -1;
    float acc[NC];
#pragma unroll
    for (int q = 0; q < NC; ++q) acc[q] = 0.0f;
    while (keep) {
      const int i = __ffsll(static_cast<long long>(keep)) - 1;
      keep &= keep - 1;
      const int vv = __shfl(v, i);
      const int jj = __shfl(j, i);
      if (vv != cur) {
        if (cur >= 0) {
          float *sv = S + static_cast<long long>(cur) * d;
#pragma unroll
          for (int q = 0; q < NC; ++q) {
            const int k = lane + q * kWave;
            if (k < d) unsafeAtomicAdd(&sv[k], acc[q]);
            acc[q] = 0.0f;
          }
        }
        cur = vv;
      }
      const float *mj = msg + static_cast<long long>(jj) * d;
#pragma unroll
      for (int q = 0; q < NC; ++q) {
        const int k = lane + q * kWave;
        if (k < d) acc[q] += mj[k];
      }
    }
    if (cur >= 0) {
      float *sv = S + static_cast<long long>(cur) * d;
#pragma unroll
      for (int q = 0; q < NC; ++q) {
        const int k = lane + q * kWave;
        if (k < d) unsafeAtomicAdd(&sv[k], acc[q]);
      }
    }
  }
}

// Bootstrap: S[v] = sum over in-arcs (u -> v) of c_u H[u], one wave per vertex,
// in the in-row's order.
template <int NC>
__global__ __launch_bounds__(256) void k_pull(long long n, int d, int agg, const float *Hprev, Adj in,
                                              const int *out_len, float *S) {
  const int lane = lane_id();
  for (long long v = global_wave(); v < n; v += num_waves()) {
    float acc[NC];
#pragma unroll
    for (int q = 0; q < NC; ++q) acc[q] = 0.0f;
    const int deg = in.len[v];
    const int *row = in.col + in.off[v];
    for (int e0 = 0; e0 < deg; e0 += kWave) {
      const int e = e0 + lane;
      const int uid = e < deg ? row[e] : 0;
      float cu = 1.0f;
      if (agg == kGcn && e < deg) cu = 1.0f / sqrtf(static_cast<float>(out_len[uid]) + 1.0f);
      const int cnt = deg - e0 < kWave ? deg - e0 : kWave;
      for (int i = 0; i < cnt; ++i) {
        const int u = __shfl(uid, i);
        const float cf = __shfl(cu, i);
        const float *hu = Hprev + static_cast<long long>(u) * d;
#pragma unroll
        for (int q = 0; q < NC; ++q) {
          const int k = lane + q * kWave;
          if (k < d) acc[q] += cf * hu[k];
        }
      }
    }
    float *sv = S + v * d;
#pragma unroll
    for (int q = 0; q < NC; ++q) {
      const int k = lane + q * kWave;
      if (k < d) sv[k] = acc[q];
    }
  }
}

__global__ void k_fill_i32(int *p, long long count, int value) {
  const long long stride = static_cast<long long>(gridDim.x) * blockDim.x;
  for (long long i = blockIdx.x * blockDim.x + threadIdx.x; i < count; i += stride) p[i] = value;
}

__global__ void k_fill_u64(u64 *p, long long count, u64 value) {
  const long long stride = static_cast<long long>(gridDim.x) * blockDim.x;
  for (long long i = blockIdx.x * blockDim.x + threadIdx.x; i < count; i += stride) p[i] = value;
}

__global__ void k_gather_rows(const float *src, int d, const int *ids, long long count, float *out) {
  const long long total = count * d;
  const long long stride = static_cast<long long>(gridDim.x) * blockDim.x;
  for (long long i = blockIdx.x * blockDim.x + threadIdx.x; i < total; i += stride) {
    const long long r = i / d;
    const int k = static_cast<int>(i % d);
    out[i] = src[static_cast<long long>(ids[r]) * d + k];
  }
}

}  // namespace

void launch_corr_mark(hipStream_t s, int cap_feat, int cap_arcs, int agg, LayerPtrs lp, const int *out_len,
                      const int *ddeg, const int *flist, const int *ins_src, const int *ins_dst, const int *del_src,
                      const int *del_dst, unsigned *bm, Counters *c) {
  const long long waves = 2LL * cap_arcs * lp.L;
  const long long threads = static_cast<long long>(cap_feat) + 2LL * cap_arcs;
  const long long items = waves * kWave > threads ? waves * kWave : threads;
  hipLaunchKernelGGL(k_corr_mark, dim3(blocks_for(items, 256)), dim3(256), 0, s, agg, lp, out_len, ddeg, flist,
                     ins_src, ins_dst, del_src, del_dst, bm, c);
}

int compact_blocks(long long n) {
  const long long words = (n + 31) / 32;
  return static_cast<int>((words + kWordsPerBlock - 1) / kWordsPerBlock);
}

void launch_compact(hipStream_t s, long long n, unsigned *bm_a, unsigned *bm_b, int *blocksum, long long *blockdeg,
                    const CompactOut &o, bool single_block) {
  const long long words = (n + 31) / 32;
  if (single_block) {
    hipLaunchKernelGGL(k_compact_single, dim3(1), dim3(kSingleThreads), 0, s, bm_a, bm_b, words, o);
    return;
  }
  const int nb = compact_blocks(n);
  hipLaunchKernelGGL(k_compact_count, dim3(nb), dim3(kCompactThreads), 0, s, bm_a, bm_b, words,
                     o.doff != nullptr ? o.out_deg : nullptr,
                     (o.ioff != nullptr || o.in_total != nullptr) ? o.in_deg : nullptr, blocksum, blockdeg);
  hipLaunchKernelGGL(k_compact_emit, dim3(nb), dim3(kCompactThreads), 0, s, bm_a, bm_b, words, blocksum, blockdeg, o);
}

void launch_delta0(hipStream_t s, long long n, int agg, int d0, const int *list, const u64 *count,
                   const ripple_op *ops, const float *feat, const int *fop, float *X, const int *out_len,
                   const int *ddeg, float *delta, const Counters *c) {
  hipLaunchKernelGGL(k_delta0, dim3(blocks_for(n * kWave, 256, 2048)), dim3(256), 0, s, agg, d0, list, count,
                     ops, feat, fop, X, out_len, ddeg, delta, c);
}

void launch_scatter(hipStream_t s, long long n, int d, const int *list, const u64 *count, const long long *doff,
                    const float *delta, Adj out, float *S, unsigned *bm_out, unsigned *bm_x, const int *ins_dst,
                    const int *del_dst, u64 *pushed, u64 *dest, const Counters *c, bool push) {
  const int blocks = 2048;
#define RP_SCATTER(GV, NCV, P)                                                                                     \
  hipLaunchKernelGGL((k_scatter<GV, NCV, P>), dim3(blocks), dim3(256), 0, s, d, list, count, doff, delta, out, S, \
                     bm_out, bm_x, ins_dst, del_dst, pushed, dest, c)
  if (!push) RP_SCATTER(64, 1, false);
  else if (d <= 16) RP_SCATTER(16, 1, true);
  else if (d <= 32) RP_SCATTER(32, 1, true);
  else if (d <= 64) RP_SCATTER(64, 1, true);
  else if (d <= 128) RP_SCATTER(64, 2, true);
  else if (d <= 256) RP_SCATTER(64, 4, true);
  else if (d <= 512) RP_SCATTER(64, 8, true);
  else RP_SCATTER(64, 16, true);
#undef RP_SCATTER
}

void launch_pull_msgs(hipStream_t s, long long n, int d, const int *list, const u64 *count, const long long *ioff,
                      Adj in, const unsigned *member, const int *slot, const float *msg, float *S, const Counters *c) {
  const int blocks = 2048;
#define RP_PULLM(NCV)                                                                                         \
  hipLaunchKernelGGL((k_pull_msgs<NCV>), dim3(blocks), dim3(256), 0, s, d, list, count, ioff, in, member, slot, \
                     msg, S, c)
  if (d <= 64) RP_PULLM(1);
  else if (d <= 128) RP_PULLM(2);
  else if (d <= 256) RP_PULLM(4);
  else if (d <= 512) RP_PULLM(8);
  else RP_PULLM(16);
#undef RP_PULLM
}

void launch_pull(hipStream_t s, long long n, int d, int agg, const float *Hprev, Adj in, const int *out_len,
                 float *S) {
  const int blocks = blocks_for(n * kWave, 256, 8192);
  const int nc = (d + kWave - 1) / kWave;
#define RP_PULL(NCV) hipLaunchKernelGGL(k_pull<NCV>, dim3(blocks), dim3(256), 0, s, n, d, agg, Hprev, in, out_len, S)
  if (nc <= 1) RP_PULL(1);
  else if (nc == 2) RP_PULL(2);
  else if (nc <= 4) RP_PULL(4);
  else if (nc <= 8) RP_PULL(8);
  else RP_PULL(16);
#undef RP_PULL
}

void launch_fill_i32(hipStream_t s, int *p, long long count, int value) {
  if (count <= 0) return;
  hipLaunchKernelGGL(k_fill_i32, dim3(blocks_for(count, 256)), dim3(256), 0, s, p, count, value);
}

void launch_fill_u64(hipStream_t s, u64 *p, long long count, u64 value) {
  if (count <= 0) return;
  hipLaunchKernelGGL(k_fill_u64, dim3(blocks_for(count, 256)), dim3(256), 0, s, p, count, value);
}

void launch_gather_rows(hipStream_t s, const float *src, int d, const int *ids, long long count, float *out) {
  if (count <= 0) return;
  hipLaunchKernelGGL(k_gather_rows, dim3(blocks_for(count * d, 256)), dim3(256), 0, s, src, d, ids, count, out);
}

}  // namespace rp
