// Frontier and message kernels.
//
// Per layer l the dirty set D^l (vertices whose layer-(l-1) contribution changed)
// pushes its delta rows along every post-batch out-arc into the cached aggregate
// S^l (Sec. IV-C.1: a message carries the new minus the old embedding and the
// receiver adds it to its mailbox), and the affected set
//   A^l = out(D^l) u sinks(net arcs) u D^l
// is collected in two bitmaps (one for the out-arc sinks, so that their distinct
// count is known exactly) and compacted into a sorted list by a popcount prefix sum.
#include "internal.h"

namespace rp {

namespace {

constexpr int kCompactThreads = 256;
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

// Dirty set of layer 1: vertices with a feature write, and under GCN every vertex
// whose out-degree changed (its coefficient 1/sqrt(dout+1) scales all it sends).
__global__ void k_mark_dirty0(int gcn, const int *flist, const int *ins_src, const int *del_src,
                              const int *ddeg, unsigned *bm, Counters *c) {
  if (c->abort) return;
  const long long nf = static_cast<long long>(c->n_feat);
  const long long ni = static_cast<long long>(c->n_ins);
  const long long nd = static_cast<long long>(c->n_del);
  const long long total = nf + (gcn ? ni + nd : 0);
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

__device__ inline int block_reduce_sum(int v, int *red) {
  for (int o = kWave / 2; o > 0; o >>= 1) v += __shfl_down(v, o);
  const int w = threadIdx.x / kWave;
  if (lane_id() == 0) red[w] = v;
  __syncthreads();
  int t = 0;
  if (threadIdx.x == 0) {
    for (int i = 0; i < kCompactThreads / kWave; ++i) t += red[i];
    red[kCompactThreads / kWave] = t;
  }
  __syncthreads();
  t = red[kCompactThreads / kWave];
  __syncthreads();
  return t;
}

__global__ __launch_bounds__(kCompactThreads) void k_compact_count(const unsigned *bm_a, const unsigned *bm_b,
                                                                   long long words, int *blocksum) {
  __shared__ int red[kCompactThreads / kWave + 1];
  const long long w0 = static_cast<long long>(blockIdx.x) * kWordsPerBlock + threadIdx.x * kWordsPerThread;
  int cnt = 0;
#pragma unroll
  for (int i = 0; i < kWordsPerThread; ++i) {
    const long long w = w0 + i;
    if (w < words) cnt += __popc(bm_a[w] | bm_b[w]);
  }
  const int t = block_reduce_sum(cnt, red);
  if (threadIdx.x == 0) blocksum[blockIdx.x] = t;
}

__global__ __launch_bounds__(kCompactThreads) void k_compact_emit(unsigned *bm_a, unsigned *bm_b,
                                                                  long long words, const int *blocksum,
                                                                  int *list_out, u64 *count_out) {
  __shared__ int red[kCompactThreads / kWave + 1];
  __shared__ int scan[kCompactThreads];
  // exclusive prefix of earlier blocks
  int pre = 0;
  for (int b = threadIdx.x; b < static_cast<int>(blockIdx.x); b += kCompactThreads) pre += blocksum[b];
  const int base = block_reduce_sum(pre, red);
  const long long w0 = static_cast<long long>(blockIdx.x) * kWordsPerBlock + threadIdx.x * kWordsPerThread;
  unsigned wv[kWordsPerThread];
  int cnt = 0;
#pragma unroll
  for (int i = 0; i < kWordsPerThread; ++i) {
    const long long w = w0 + i;
    wv[i] = w < words ? (bm_a[w] | bm_b[w]) : 0u;
    cnt += __popc(wv[i]);
  }
  // block exclusive scan of cnt (Hillis-Steele in LDS)
  scan[threadIdx.x] = cnt;
  __syncthreads();
  for (int o = 1; o < kCompactThreads; o <<= 1) {
    const int v = threadIdx.x >= o ? scan[threadIdx.x - o] : 0;
    __syncthreads();
    scan[threadIdx.x] += v;
    __syncthreads();
  }
  int pos = base + scan[threadIdx.x] - cnt;
#pragma unroll
  for (int i = 0; i < kWordsPerThread; ++i) {
    unsigned m = wv[i];
    const long long vbase = (w0 + i) * 32;
    while (m) {
      const int b = __ffs(m) - 1;
      list_out[pos++] = static_cast<int>(vbase + b);
      m &= m - 1;
    }
    const long long w = w0 + i;
    if (w < words) {
      bm_a[w] = 0u;
      bm_b[w] = 0u;
    }
  }
  if (blockIdx.x == gridDim.x - 1 && threadIdx.x == kCompactThreads - 1) {
    *count_out = static_cast<u64>(base + scan[threadIdx.x]);
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

// One wave per dirty vertex: its delta row sits in registers (NC floats per lane),
// its out-row is read 64 ids at a time, and each id's row of S gets one coalesced
// row of fp32 atomic adds.
template <int NC>
__global__ __launch_bounds__(256) void k_scatter(int d, const int *list, const u64 *count, const float *delta,
                                                 Adj out, float *S, unsigned *bm_out, unsigned *bm_x,
                                                 const int *ins_dst, const int *del_dst, u64 *pushed,
                                                 u64 *dest, const Counters *c) {
  if (c->abort) return;
  const int lane = lane_id();
  // sinks of net arcs are affected at every layer
  {
    const long long ni = static_cast<long long>(c->n_ins);
    const long long na = ni + static_cast<long long>(c->n_del);
    const long long stride = static_cast<long long>(gridDim.x) * blockDim.x;
    for (long long i = blockIdx.x * blockDim.x + threadIdx.x; i < na; i += stride)
      mark(bm_x, i < ni ? ins_dst[i] : del_dst[i - ni]);
  }
  const long long m = static_cast<long long>(*count);
  u64 my_pushed = 0, my_dest = 0;
  for (long long j = global_wave(); j < m; j += num_waves()) {
    const int u = list[j];
    if (lane == 0) mark(bm_x, u);
    float dreg[NC];
    const float *dj = delta + j * d;
#pragma unroll
    for (int q = 0; q < NC; ++q) {
      const int k = lane + q * kWave;
      dreg[q] = k < d ? dj[k] : 0.0f;
    }
    const int deg = out.len[u];
    const int *row = out.col + out.off[u];
    my_pushed += deg;
    for (int e0 = 0; e0 < deg; e0 += kWave) {
      const int e = e0 + lane;
      const int cidx = e < deg ? row[e] : -1;
      const bool fresh = cidx >= 0 && mark(bm_out, cidx);
      my_dest += __popcll(__ballot(fresh));
      const int cnt = deg - e0 < kWave ? deg - e0 : kWave;
      for (int i = 0; i < cnt; ++i) {
        const int v = __shfl(cidx, i);
        float *sv = S + static_cast<long long>(v) * d;
#pragma unroll
        for (int q = 0; q < NC; ++q) {
          const int k = lane + q * kWave;
          if (k < d) unsafeAtomicAdd(&sv[k], dreg[q]);
        }
      }
    }
  }
  if (lane == 0 && (my_pushed | my_dest)) {
    atomicAdd(pushed, my_pushed);
    atomicAdd(dest, my_dest);
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

void launch_mark_dirty0(hipStream_t s, int cap_feat, int cap_arcs, int gcn, const int *flist,
                        const int *ins_src, const int *del_src, const int *ddeg, unsigned *bm, Counters *c) {
  hipLaunchKernelGGL(k_mark_dirty0, dim3(blocks_for(static_cast<long long>(cap_feat) + 2LL * cap_arcs, 256)),
                     dim3(256), 0, s, gcn, flist, ins_src, del_src, ddeg, bm, c);
}

int compact_blocks(long long n) {
  const long long words = (n + 31) / 32;
  return static_cast<int>((words + kWordsPerBlock - 1) / kWordsPerBlock);
}

void launch_compact(hipStream_t s, long long n, unsigned *bm_a, unsigned *bm_b, int *blocksum, int *list_out,
                    u64 *count_out) {
  const long long words = (n + 31) / 32;
  const int nb = compact_blocks(n);
  hipLaunchKernelGGL(k_compact_count, dim3(nb), dim3(kCompactThreads), 0, s, bm_a, bm_b, words, blocksum);
  hipLaunchKernelGGL(k_compact_emit, dim3(nb), dim3(kCompactThreads), 0, s, bm_a, bm_b, words, blocksum,
                     list_out, count_out);
}

void launch_delta0(hipStream_t s, long long n, int agg, int d0, const int *list, const u64 *count,
                   const ripple_op *ops, const float *feat, const int *fop, float *X, const int *out_len,
                   const int *ddeg, float *delta, const Counters *c) {
  hipLaunchKernelGGL(k_delta0, dim3(blocks_for(n * kWave, 256, 2048)), dim3(256), 0, s, agg, d0, list, count,
                     ops, feat, fop, X, out_len, ddeg, delta, c);
}

void launch_scatter(hipStream_t s, long long n, int d, const int *list, const u64 *count, const float *delta,
                    Adj out, float *S, unsigned *bm_out, unsigned *bm_x, const int *ins_dst, const int *del_dst,
                    int cap_arcs, u64 *pushed, u64 *dest, const Counters *c) {
  const int blocks = blocks_for(n * kWave, 256, 2048);
  const int nc = (d + kWave - 1) / kWave;
#define RP_SCATTER(NCV)                                                                                  \
  hipLaunchKernelGGL(k_scatter<NCV>, dim3(blocks), dim3(256), 0, s, d, list, count, delta, out, S, bm_out, \
                     bm_x, ins_dst, del_dst, pushed, dest, c)
  if (nc <= 1) RP_SCATTER(1);
  else if (nc == 2) RP_SCATTER(2);
  else if (nc <= 4) RP_SCATTER(4);
  else if (nc <= 8) RP_SCATTER(8);
  else RP_SCATTER(16);
#undef RP_SCATTER
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
