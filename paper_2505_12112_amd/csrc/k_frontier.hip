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
// layer's scatter. A pushing layer with a small frontier instead lists A^l in its
// own scatter, in no particular order: the first setter of a member's bit appends
// it (see ScatterList). The layer-1 dirty set of a batch without GCN terms is
// listed by the correction kernel itself, with its deltas.
#include <type_traits>

#include "internal.h"

namespace rp {

namespace {

constexpr int kCompactThreads = 256;
constexpr int kCompactWaves = kCompactThreads / kWave;
constexpr int kWordsPerThread = 4;
constexpr int kWordsPerBlock = kCompactThreads * kWordsPerThread;
// Tiles that are placed by block index: far fewer than the compute units, so all are
// resident at once (graphs up to 2M vertices; larger ones, whose compactions take
// long enough not to notice a round trip, go in ticket order).
constexpr long long kIndexTiles = 64;
static_assert(kIndexTiles <= kWave, "one lane per predecessor tile");

__device__ inline int lane_id() { return threadIdx.x & (kWave - 1); }

__device__ inline long long global_wave() {
  return (static_cast<long long>(blockIdx.x) * blockDim.x + threadIdx.x) / kWave;
}

__device__ inline long long num_waves() {
  return static_cast<long long>(gridDim.x) * blockDim.x / kWave;
}

// Sets v's bit; the old word is not read back, so nothing waits on it.
__device__ inline void mark_only(unsigned *bm, int v) { atomicOr(&bm[v >> 5], 1u << (v & 31)); }

inline int blocks_for(long long items, int threads, int cap = 4096) {
  long long b = (items + threads - 1) / threads;
  if (b < 1) b = 1;
  if (b > cap) b = cap;
  return static_cast<int>(b);
}

// The inserted arcs' slots, the pre-batch corrections and the layer-1 dirty marks
// (see launch_corr_mark).
__global__ void k_corr_mark(int agg, LayerPtrs lp, Adj out, Adj in, const int *ins_rank, const float *arc_w,
                            const int *ddeg, const int *flist, const int *ins_src, const int *ins_dst,
                            const int *del_src, const int *del_dst, const float *ins_w, const float *del_w,
                            unsigned *bm, Counters *c, DirectList dl) {
  const long long nf = static_cast<long long>(c->n_feat);
  const long long ni = static_cast<long long>(c->n_ins);
  const long long na = ni + static_cast<long long>(c->n_del);
  if (aborted_with(c->abort, nf, na)) return;
  const int lane = lane_id();
  const int *out_len = out.len;
  if (dl.list != nullptr && blockIdx.x == 0) {
    // block 0 lists the dirty set (flist[0, nf), distinct vertices) with the
    // exclusive prefix of their post-batch out-degrees: four entries per thread
    constexpr int kPer = kDirectListMax / 256;
    static_assert(kPer * 256 == kDirectListMax, "four entries per thread");
    __shared__ long long wsum[4];
    int v[kPer], dg[kPer];
    long long sum = 0;
#pragma unroll
    for (int q = 0; q < kPer; ++q) {
      const long long i = static_cast<long long>(threadIdx.x) * kPer + q;
      v[q] = i < nf ? flist[i] : -1;
    }
#pragma unroll
    for (int q = 0; q < kPer; ++q) {
      dg[q] = v[q] >= 0 ? out_len[v[q]] : 0;
      sum += dg[q];
    }
    long long incl = sum;
#pragma unroll
    for (int o = 1; o < kWave; o <<= 1) {
      const long long y = __shfl_up(incl, o);
      if (lane >= o) incl += y;
    }
    const int wave = threadIdx.x / kWave;
    if (lane == kWave - 1) wsum[wave] = incl;
    __syncthreads();
    long long pos = incl - sum, total = 0;
    for (int w = 0; w < 4; ++w) {
      if (w < wave) pos += wsum[w];
      total += wsum[w];
    }
#pragma unroll
    for (int q = 0; q < kPer; ++q) {
      const long long i = static_cast<long long>(threadIdx.x) * kPer + q;
      if (i < nf) {
        dl.list[i] = v[q];
        dl.doff[i] = pos;
      }
      pos += dg[q];
    }
    if (threadIdx.x == 0) {
      const long long listed = nf < kDirectListMax ? nf : kDirectListMax;
      dl.doff[listed] = total;
      *dl.count = static_cast<u64>(listed);
      *dl.out_total = static_cast<u64>(total);
      if (nf > kDirectListMax) atomicOr(&c->err, 2ull);
    }
  }
  if (dl.delta != nullptr) {
    // layer-0 deltas of the listed vertices, one wave per row from the grid's last
    // wave down (the corrections start at wave 0); x' is staged, X keeps x
    const float *feat = dl.in->feat;
    const long long nl = nf < kDirectListMax ? nf : kDirectListMax;
    for (long long j = num_waves() - 1 - global_wave(); j < nl; j += num_waves()) {
      const int u = flist[j];
      const float *xu = dl.X + static_cast<long long>(u) * dl.d0;
      const float *xn = feat + static_cast<long long>(dl.frow[j]) * dl.d0;
      float *dj = dl.delta + j * dl.ld;
      float *sj = dl.stage + j * dl.ld;
      for (int k = lane; k < dl.d0; k += kWave) {
        const float x1 = xn[k];
        dj[k] = x1 - xu[k];
        sj[k] = x1;
      }
    }
  }
  {
    // item w = 2 * arc + direction: its row's inserts follow the kept entries, in
    // rank order
    const long long stride = static_cast<long long>(gridDim.x) * blockDim.x;
    for (long long w = blockIdx.x * blockDim.x + threadIdx.x; w < 2 * ni; w += stride) {
      const long long arc = w >> 1;
      const int dir = static_cast<int>(w & 1);
      const int row = dir == 0 ? ins_src[arc] : ins_dst[arc];
      const int entry = dir == 0 ? ins_dst[arc] : ins_src[arc];
      const Adj &a = dir ? in : out;
      const long long slot = a.off[row] + (a.len[row] - a.inscnt[row]) + ins_rank[w];
      a.col[slot] = entry;
      if (a.wt != nullptr) a.wt[slot] = arc_w[arc];
    }
  }
  const long long items = na * lp.L;
  for (long long it = global_wave(); it < items; it += num_waves()) {
    const long long arc = it / lp.L;
    const int l = static_cast<int>(it % lp.L) + 1;
    const bool ins = arc < ni;
    const int u = ins ? ins_src[arc] : del_src[arc - ni];
    const int v = ins ? ins_dst[arc] : del_dst[arc - ni];
    float coef = ins ? 1.0f : -1.0f;
    if (agg == kGcn) coef *= 1.0f / sqrtf(static_cast<float>(out_len[u] - ddeg[u]) + 1.0f);
    if (ins_w != nullptr) coef *= ins ? ins_w[arc] : del_w[arc - ni];  // the arc's weight
    const int d = lp.sw[l];
    const float *hu = lp.src[l] + static_cast<long long>(u) * d;
    float *sv = lp.S[l] + static_cast<long long>(v) * d;
    for (int k = lane; k < d; k += kWave) unsafeAtomicAdd(&sv[k], coef * hu[k]);
  }
  const long long total = nf + (agg == kGcn ? na : 0);
  const long long stride = static_cast<long long>(gridDim.x) * blockDim.x;
  for (long long i = blockIdx.x * blockDim.x + threadIdx.x + (dl.list != nullptr ? nf : 0); i < total; i += stride) {
    if (i < nf) {
      mark_only(bm, flist[i]);
    } else {
      const long long a = i - nf;
      const int u = a < ni ? ins_src[a] : del_src[a - ni];
      if (ddeg[u] != 0) mark_only(bm, u);
    }
  }
}

// The set bits of a thread's kWordsPerThread (= 4) bitmap words, walked in vertex
// order from two 64-bit halves (no dynamically indexed register arrays).
struct BitCursor {
  unsigned long long lo, hi;
  long long base;  // vertex id of bit 0
  __device__ BitCursor(const unsigned (&w)[kWordsPerThread], long long first_word)
      : lo(w[0] | static_cast<unsigned long long>(w[1]) << 32),
        hi(w[2] | static_cast<unsigned long long>(w[3]) << 32), base(first_word * 32) {}
  __device__ bool empty() const { return (lo | hi) == 0; }
  __device__ int next() {  // -1 when exhausted
    if (lo) {
      const int b = __ffsll(lo) - 1;
      lo &= lo - 1;
      return static_cast<int>(base + b);
    }
    if (hi) {
      const int b = __ffsll(hi) - 1;
      hi &= hi - 1;
      return static_cast<int>(base + 64 + b);
    }
    return -1;
  }
};
static_assert(kWordsPerThread == 4, "BitCursor covers four words");

// Vertices and degrees are fetched kBatch at a time so that the loads of one
// thread overlap instead of forming a chain of dependent round trips.
constexpr int kBatch = 8;

// Loads a thread's words of both bitmaps; pop_a counts the first bitmap's bits.
__device__ inline void load_words(const unsigned *bm_a, const unsigned *bm_b, long long w0, long long words,
                                  unsigned (&wv)[kWordsPerThread], int &pop_a) {
  pop_a = 0;
#pragma unroll
  for (int i = 0; i < kWordsPerThread; ++i) {
    const unsigned a = w0 + i < words ? bm_a[w0 + i] : 0u;
    const unsigned b = w0 + i < words ? bm_b[w0 + i] : 0u;
    wv[i] = a | b;
    pop_a += __popc(a);
  }
}

// The bucket form's sinks, from their counts: bit b of word w is set when
// cnt[32 w + b] > 0; they count as first-bitmap bits. The counter array covers
// every word of every compaction tile (bucket_counter_slots), so all loads are in
// bounds and go out together; counters past n stay zero.
__device__ inline void count_words(const int *cnt, long long w0, unsigned (&wv)[kWordsPerThread], int &pop_a) {
  int4 x[kWordsPerThread][8];
#pragma unroll
  for (int i = 0; i < kWordsPerThread; ++i) {
    const int4 *q = reinterpret_cast<const int4 *>(cnt + (w0 + i) * 32);
#pragma unroll
    for (int k = 0; k < 8; ++k) x[i][k] = q[k];
  }
#pragma unroll
  for (int i = 0; i < kWordsPerThread; ++i) {
    unsigned bits = 0u;
#pragma unroll
    for (int k = 0; k < 8; ++k)
      bits |= (x[i][k].x > 0 ? 1u : 0u) << (4 * k) | (x[i][k].y > 0 ? 2u : 0u) << (4 * k) |
              (x[i][k].z > 0 ? 4u : 0u) << (4 * k) | (x[i][k].w > 0 ? 8u : 0u) << (4 * k);
    wv[i] |= bits;
    pop_a += __popc(bits);
  }
}

// Sums of the out- and in-degrees and bucket counts (any may be null) over the
// cursor's bits. The values of the first kBatch bits are kept in d0 / i0 / b0
// (most threads have no more), so the pass that writes the offsets need not fetch
// them again.
__device__ inline void degree_sums(BitCursor c, const int *odeg, const int *ideg, const int *bcnt, long long &dsum,
                                   long long &isum, long long &bsum, int (&d0)[kBatch], int (&i0)[kBatch],
                                   int (&b0)[kBatch]) {
  if (odeg == nullptr && ideg == nullptr && bcnt == nullptr) return;
  bool first = true;
  while (!c.empty()) {
    int v[kBatch];
#pragma unroll
    for (int j = 0; j < kBatch; ++j) v[j] = c.next();
#pragma unroll
    for (int j = 0; j < kBatch; ++j) {
      const int dv = odeg != nullptr && v[j] >= 0 ? odeg[v[j]] : 0;
      const int iv = ideg != nullptr && v[j] >= 0 ? ideg[v[j]] : 0;
      const int bv = bcnt != nullptr && v[j] >= 0 ? bcnt[v[j]] : 0;
      dsum += dv;
      isum += iv;
      bsum += bv;
      if (first) {
        d0[j] = dv;
        i0[j] = iv;
        b0[j] = bv;
      }
    }
    first = false;
  }
}

// Per-tile sums carried by the compaction: marked vertices, their out-degrees,
// their in-degrees, marked vertices of the first bitmap, their bucket counts.
constexpr int kVals = 5;

// Exclusive block scan of kVals values at once (one LDS round).
__device__ inline void block_scan(const long long (&v)[kVals], long long (&excl)[kVals], long long (&total)[kVals],
                                  long long (*lds)[kVals]) {
  const int lane = lane_id(), wave = threadIdx.x / kWave;
  long long x[kVals];
#pragma unroll
  for (int k = 0; k < kVals; ++k) x[k] = v[k];
#pragma unroll
  for (int o = 1; o < kWave; o <<= 1) {
#pragma unroll
    for (int k = 0; k < kVals; ++k) {
      const long long y = __shfl_up(x[k], o);
      if (lane >= o) x[k] += y;
    }
  }
  if (lane == kWave - 1) {
#pragma unroll
    for (int k = 0; k < kVals; ++k) lds[wave][k] = x[k];
  }
  __syncthreads();
  long long before[kVals] = {}, all[kVals] = {};
  for (int w = 0; w < kCompactWaves; ++w) {
#pragma unroll
    for (int k = 0; k < kVals; ++k) {
      const long long t = lds[w][k];
      if (w < wave) before[k] += t;
      all[k] += t;
    }
  }
#pragma unroll
  for (int k = 0; k < kVals; ++k) {
    excl[k] = before[k] + x[k] - v[k];
    total[k] = all[k];
  }
  __syncthreads();
}

// Published tile sums: each 64-bit word holds the launch epoch (1..65535) above a
// 48-bit value, so a word is valid on its own and words of earlier launches are
// never mistaken for current ones (the tiles of every launch rewrite all words).
constexpr int kEpochShift = 48;
constexpr u64 kValueMask = (1ull << kEpochShift) - 1;
constexpr int kSpinLimit = 1 << 20;

__device__ inline void publish(u64 *p, u64 epoch, const long long (&v)[kVals]) {
#pragma unroll
  for (int k = 0; k < kVals; ++k)
    __hip_atomic_store(p + k, epoch << kEpochShift | (static_cast<u64>(v[k]) & kValueMask), __ATOMIC_RELAXED,
                       __HIP_MEMORY_SCOPE_AGENT);
}

__device__ inline bool fetch(const u64 *p, u64 epoch, long long (&v)[kVals]) {
  bool ok = true;
#pragma unroll
  for (int k = 0; k < kVals; ++k) {
    const u64 w = __hip_atomic_load(p + k, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    ok = ok && (w >> kEpochShift) == epoch;
    v[k] = static_cast<long long>(w & kValueMask);
  }
  return ok;
}

// Single-pass compaction (a decoupled look-back prefix scan). Tiles of
// kWordsPerBlock bitmap words go to blocks by index when all tiles fit on the GPU at
// once, else in ticket order; either way a tile's predecessors are running or done
// when it waits for them. Each tile publishes its sums at once. A tile placed by
// index then reads all its predecessors' sums in one round (one lane each); in
// ticket order, wave 0 walks back over the predecessors (64 per step), adding
// their tile sums until it meets one that has published its inclusive prefix. A
// tile publishes its own sums before it waits, so every wait is for work that
// needs no waiting: all waits end. A wait that outlasts kSpinLimit polls (a predecessor
// that never ran) sets bit 2 of the error word and counts the tile as empty (the
// batch then fails loudly instead of hanging).
// Output: the marked vertices of both bitmaps as a sorted list with prefix sums of
// their out- and in-degrees, membership words and per-word prefix counts; both
// bitmaps are cleared. A full compaction lists every vertex without reading them.
__global__ __launch_bounds__(kCompactThreads) void k_compact(unsigned *bm_a, unsigned *bm_b, long long words,
                                                             CompactOut o, u64 *agg, u64 *inc, u64 *ticket,
                                                             u64 *err) {
  __shared__ long long red[kCompactWaves][kVals];
  __shared__ long long base_s[kVals];
  __shared__ u64 epoch_s, ticket_s;
  constexpr int kZeroList = 1024;  // long rows a tile zeroes cooperatively (more: by their own thread)
  __shared__ int zlist[kZeroList];
  __shared__ int zcount;
  if (threadIdx.x == 0) zcount = 0;  // published by the scan's barriers
  const long long tiles = gridDim.x;
  // Up to kIndexTiles tiles all fit on the GPU at once, so block b takes tile b and
  // its ticket (for the epoch) is in flight beside the bitmap loads. Beyond that,
  // tiles go in ticket order, so a tile's predecessors are running or done however
  // the blocks are dispatched.
  const bool by_ticket = tiles > kIndexTiles;
  u64 ticket_no = 0;
  if (by_ticket) {
    if (threadIdx.x == 0) ticket_s = atomicAdd(ticket, 1ull);
    __syncthreads();
    ticket_no = ticket_s;
  }
  const long long tile = by_ticket ? static_cast<long long>(ticket_no % static_cast<u64>(tiles)) : blockIdx.x;
  const long long w0 = tile * kWordsPerBlock + threadIdx.x * kWordsPerThread;
  const int *odeg = o.doff != nullptr || o.out_total != nullptr ? o.out_deg : nullptr;
  const int *ideg = o.ioff != nullptr || o.in_total != nullptr ? o.in_deg : nullptr;
  unsigned wv[kWordsPerThread];
  int pop_a = 0;
  if (o.full_n > 0) {
#pragma unroll
    for (int i = 0; i < kWordsPerThread; ++i) {
      const long long w = w0 + i;
      const long long left = o.full_n - w * 32;  // vertices from this word on
      wv[i] = left >= 32 ? ~0u : left > 0 ? (1u << left) - 1u : 0u;
    }
  } else {
    load_words(bm_a, bm_b, w0, words, wv, pop_a);
    if (o.bkt_cnt != nullptr) count_words(o.bkt_cnt, w0, wv, pop_a);
  }
  if (!by_ticket && threadIdx.x == 0) ticket_no = atomicAdd(ticket, 1ull);  // in flight beside the loads
  long long st[kVals] = {0, 0, 0, pop_a, 0};
#pragma unroll
  for (int i = 0; i < kWordsPerThread; ++i) st[0] += __popc(wv[i]);
  int d0[kBatch], i0[kBatch], b0[kBatch];
  degree_sums(BitCursor(wv, w0), odeg, ideg, o.bkt_cnt, st[1], st[2], st[4], d0, i0, b0);
  // The ticket counter only grows and every launch on this scratch has the same
  // number of blocks, each taking one ticket, so launch k holds tickets k * tiles
  // .. k * tiles + tiles - 1: the ticket's quotient names the launch.
  if (threadIdx.x == 0) epoch_s = ticket_no / static_cast<u64>(tiles) % 65535 + 1;
  long long ex[kVals], tot[kVals];
  block_scan(st, ex, tot, red);  // its barriers also publish epoch_s
  const u64 epoch = epoch_s;
  // Tiles by index publish their sums only: every predecessor's are read in one
  // round (one lane each). Tiles in ticket order also publish inclusive prefixes.
  if (threadIdx.x == 0) publish((by_ticket && tile == 0 ? inc : agg) + tile * kVals, epoch, tot);
  if (threadIdx.x < kWave && !by_ticket) {
    const int lane = lane_id();
    long long v[kVals] = {};
    bool timed_out = false;
    if (lane < tile) {
      for (int it = 0;; ++it) {
        if (fetch(agg + lane * kVals, epoch, v)) break;
        if (it >= kSpinLimit) {
          timed_out = true;
#pragma unroll
          for (int k = 0; k < kVals; ++k) v[k] = 0;
          break;
        }
        __builtin_amdgcn_s_sleep(2);
      }
    }
#pragma unroll
    for (int k = 0; k < kVals; ++k) {
#pragma unroll
      for (int o2 = kWave / 2; o2 > 0; o2 >>= 1) v[k] += __shfl_xor(v[k], o2);
    }
    if (timed_out) atomicOr(err, 4ull);
    if (lane == 0) {
#pragma unroll
      for (int k = 0; k < kVals; ++k) base_s[k] = v[k];
    }
  } else if (threadIdx.x < kWave) {
    const int lane = lane_id();
    long long acc[kVals] = {};
    bool timed_out = false;
    for (long long j = tile - 1; j >= 0; j -= kWave) {
      const long long p = j - lane;
      long long v[kVals] = {};
      bool incl = true;  // lanes before tile 0 end the walk with zeros
      if (p >= 0) {
        for (int it = 0;; ++it) {
          long long va[kVals];  // both words are read in the same round
          const bool got_inc = fetch(inc + p * kVals, epoch, v);
          const bool got_agg = fetch(agg + p * kVals, epoch, va);
          if (got_inc) break;
          if (got_agg) {
#pragma unroll
            for (int k = 0; k < kVals; ++k) v[k] = va[k];
            incl = false;
            break;
          }
          if (it >= kSpinLimit) {
            timed_out = true;
#pragma unroll
            for (int k = 0; k < kVals; ++k) v[k] = 0;
            break;
          }
          __builtin_amdgcn_s_sleep(2);
        }
      }
      const u64 im = __ballot(incl);
      const int first = im ? __ffsll(im) - 1 : kWave;  // nearest inclusive predecessor
#pragma unroll
      for (int k = 0; k < kVals; ++k) {
        long long x = lane <= first ? v[k] : 0;
#pragma unroll
        for (int o2 = kWave / 2; o2 > 0; o2 >>= 1) x += __shfl_xor(x, o2);
        acc[k] += x;
      }
      if (first < kWave) break;
    }
    if (timed_out) atomicOr(err, 4ull);
    if (lane == 0) {
#pragma unroll
      for (int k = 0; k < kVals; ++k) base_s[k] = acc[k];
      if (tile > 0) {
        long long incv[kVals];
#pragma unroll
        for (int k = 0; k < kVals; ++k) incv[k] = acc[k] + tot[k];
        publish(inc + tile * kVals, epoch, incv);
      }
    }
  }
  __syncthreads();
  long long base[kVals];
#pragma unroll
  for (int k = 0; k < kVals; ++k) base[k] = base_s[k];
  long long pos = base[0] + ex[0], dpos = base[1] + ex[1], ipos = base[2] + ex[2], bpos = base[4] + ex[4];
  if (o.memb != nullptr) {
    long long wp = pos;
#pragma unroll
    for (int i = 0; i < kWordsPerThread; ++i) {
      if (w0 + i < words) o.memb[w0 + i] = make_uint2(wv[i], static_cast<unsigned>(wp));
      wp += __popc(wv[i]);
    }
  }
  BitCursor c(wv, w0);
  bool first = true;  // the cursor repeats the first pass's order: its first batch is cached
  while ((o.list != nullptr || o.doff != nullptr || o.ioff != nullptr || o.boff != nullptr) && !c.empty()) {
    int v[kBatch], dv[kBatch], iv[kBatch], bv[kBatch];
#pragma unroll
    for (int j = 0; j < kBatch; ++j) v[j] = c.next();
#pragma unroll
    for (int j = 0; j < kBatch; ++j) {
      dv[j] = o.doff == nullptr || v[j] < 0 ? 0 : first ? d0[j] : odeg[v[j]];
      iv[j] = o.ioff == nullptr || v[j] < 0 ? 0 : first ? i0[j] : ideg[v[j]];
      bv[j] = o.boff == nullptr || v[j] < 0 ? 0 : first ? b0[j] : o.bkt_cnt[v[j]];
    }
    first = false;
#pragma unroll
    for (int j = 0; j < kBatch; ++j) {
      if (v[j] < 0) continue;
      if (o.list != nullptr) o.list[pos] = v[j];
      if (o.doff != nullptr) {
        o.doff[pos] = dpos;
        dpos += dv[j];
      }
      if (o.ioff != nullptr) {
        o.ioff[pos] = ipos;
        ipos += iv[j];
      }
      if (o.boff != nullptr) {  // the count is read above before its start is written over it
        o.boff[pos] = bpos;
        if (bv[j] > 0) o.bkt_start[v[j]] = static_cast<int>(bpos);
        bpos += bv[j];
      }
      if (o.zero_rows != nullptr && iv[j] > kRecomputeSeg) {  // summed in segments by the recompute
        const int slot = atomicAdd(&zcount, 1);
        if (slot < kZeroList) {
          zlist[slot] = v[j];  // zeroed by the whole block below
        } else {
          float *r = o.zero_rows + static_cast<long long>(v[j]) * o.zero_w;
          for (int k = 0; k < o.zero_w; ++k) r[k] = 0.f;
        }
      }
      ++pos;
    }
  }
  if (o.zero_rows != nullptr) {
    // the tile's long rows, a wave per row and a lane per element
    __syncthreads();
    const int nz = zcount < kZeroList ? zcount : kZeroList;
    for (int r = threadIdx.x / kWave; r < nz; r += kCompactWaves) {
      float *row = o.zero_rows + static_cast<long long>(zlist[r]) * o.zero_w;
      for (int k = lane_id(); k < o.zero_w; k += kWave) row[k] = 0.f;
    }
  }
#pragma unroll
  for (int i = 0; i < kWordsPerThread; ++i) {
    const long long w = w0 + i;
    if (w < words) {
      if (o.full_n == 0) {
        bm_a[w] = 0u;
        bm_b[w] = 0u;
      }
    }
  }
  if (tile == tiles - 1 && threadIdx.x == 0) {
    const long long total = base[0] + tot[0];
    *o.count = static_cast<u64>(total);
    if (o.doff != nullptr) o.doff[total] = base[1] + tot[1];
    if (o.ioff != nullptr) o.ioff[total] = base[2] + tot[2];
    if (o.boff != nullptr) o.boff[total] = base[4] + tot[4];
    if (o.out_total != nullptr) *o.out_total = static_cast<u64>(base[1] + tot[1]);
    if (o.in_total != nullptr) *o.in_total = static_cast<u64>(base[2] + tot[2]);
    if (o.sinks_a != nullptr) *o.sinks_a = static_cast<u64>(base[3] + tot[3]);
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

// wave_last_le over [0, n) that also hands back its last round's loads: lane t
// holds a[w0 + t] (1 << 62 past n), w0 <= the answer.
__device__ inline long long wave_last_le_win(const long long *a, long long n, long long x, long long &win,
                                             long long &w0) {
  const int lane = lane_id();
  long long lo = 0, hi = n;
  while (hi - lo > kWave) {
    const long long step = (hi - lo + kWave - 1) / kWave;
    const long long idx = lo + lane * step;
    const bool le = idx < hi && a[idx] <= x;
    const int last = __popcll(__ballot(le)) - 1;
    lo = lo + last * step;
    hi = lo + step < hi ? lo + step : hi;
  }
  const long long idx = lo + lane;
  win = idx < n ? a[idx] : (1LL << 62);
  w0 = lo;
  return lo + __popcll(__ballot(idx < hi && win <= x)) - 1;
}

// Same answer as wave_last_le(a, from, n1, x), for a lower bound `from` whose
// answer is usually close: one round of 64 probes from `from`, and the full
// search only when every probe is <= x. Used when a wave walks consecutive arcs.
__device__ inline long long owner_from(const long long *a, long long from, long long n1, long long x) {
  const int lane = lane_id();
  const long long hi = from + kWave < n1 ? from + kWave : n1;
  const long long idx = from + lane;
  const bool le = idx < hi && a[idx] <= x;
  const int cnt = __popcll(__ballot(le));
  if (cnt == hi - from && hi < n1) return wave_last_le(a, hi - 1, n1, x);
  return from + cnt - 1;
}

// One wave per listed vertex (see Delta0Args). list holds cap entries: the wave's
// first vertex is fetched with the count (an entry past the count is dropped).
__global__ void k_delta0(Delta0Args z, const int *list, const u64 *count, long long cap) {
  const long long j0 = global_wave();
  const int u0 = j0 < cap ? list[j0] : 0;
  const long long m = static_cast<long long>(*count);
  const float *feat = z.in->feat;
  // (an entry past the count may hold anything: it joins the test as an unsigned
  // half, which is never negative)
  if (aborted_with(z.c->abort, m, static_cast<unsigned>(u0) >> 1)) return;
  const int lane = lane_id();
  for (long long j = j0; j < m; j += num_waves()) {
    const int u = j == j0 ? u0 : list[j];
    const int fo = z.fop[u];
    float cn = 1.0f, co = 1.0f;
    if (z.agg == kGcn) {
      const int dout = z.out_len[u];
      cn = 1.0f / sqrtf(static_cast<float>(dout) + 1.0f);
      co = 1.0f / sqrtf(static_cast<float>(dout - z.ddeg[u]) + 1.0f);
    }
    float *xu = z.X + static_cast<long long>(u) * z.d0;
    const float *xn = fo >= 0 ? feat + static_cast<long long>(z.ops[fo].feat_row) * z.d0 : xu;
    float *dj = z.delta + j * z.ld;
    for (int k = lane; k < z.d0; k += kWave) {
      const float xo = xu[k];
      const float x1 = xn[k];
      dj[k] = cn * x1 - co * xo;
      xu[k] = x1;
    }
  }
}

// Arc e = e0 + lane (e <= elast) of the scatter's numbering, for a run whose first
// and last arcs belong to list positions ja and jb: its sink (-1 past elast).
__device__ inline int run_sink(const long long *doff, const int *list, const Adj &out, long long e0,
                               long long elast, long long ja, long long jb) {
  const int lane = lane_id();
  const long long e = e0 + lane;
  const bool active = e <= elast;
  int j = static_cast<int>(ja);
  if (jb > ja) {
    if (jb - ja < kWave) {
      const long long mine = ja + lane <= jb ? doff[ja + lane] : (1LL << 62);
      int cnt_le = 0;
      for (int t = 0; t <= static_cast<int>(jb - ja); ++t) cnt_le += __shfl(mine, t) <= e ? 1 : 0;
      j = static_cast<int>(ja) + cnt_le - 1;
    } else if (active) {
      j = static_cast<int>(upper_bound(doff, ja, jb + 1, e) - 1);
    }
  }
  if (!active) return -1;
  const int u = list[j];
  return out.col[out.off[u] + (e - doff[j])];
}

// One mark per lane (v < 0: none) by a scatter that lists A^l itself (see
// ScatterList): the membership and sink bits are set with returning atomics, the
// degrees are read beside them, and the lanes that set a membership bit first take
// consecutive list positions and out-arc offsets with one atomic for the wave.
__device__ inline void list_mark(int v, bool sink, const ScatterList &lo, unsigned *bm_out, unsigned *bm_x) {
  const int lane = lane_id();
  bool fresh = false, fresh_sink = false;
  long long dv = 0, iv = 0;
  if (v >= 0) {
    const unsigned bit = 1u << (v & 31);
    const unsigned om = atomicOr(&bm_x[v >> 5], bit);
    const unsigned os = sink ? atomicOr(&bm_out[v >> 5], bit) : bit;
    dv = lo.doff != nullptr ? lo.out_len[v] : 0;
    iv = lo.in_len[v];
    fresh = (om & bit) == 0;
    fresh_sink = (os & bit) == 0;
  }
  const u64 ms = __ballot(fresh_sink);
  const u64 m = __ballot(fresh);
  if ((m | ms) == 0) return;
  if (!fresh) dv = iv = 0;
  long long dinc = dv, itot = iv;
#pragma unroll
  for (int o = 1; o < kWave; o <<= 1) {
    const long long y = __shfl_up(dinc, o);
    if (lane >= o) dinc += y;
    itot += __shfl_xor(itot, o);
  }
  const long long dtot = __shfl(dinc, kWave - 1);
  const int leader = __ffsll(static_cast<long long>(m | ms)) - 1;
  u64 base = 0;
  if (lane == leader) {
    if (m != 0) base = atomicAdd(lo.app, static_cast<u64>(__popcll(m)) << kAppShift | static_cast<u64>(dtot));
    atomicAdd(lo.sinks, static_cast<u64>(__popcll(ms)) << kAppShift | static_cast<u64>(itot));
  }
  base = __shfl(base, leader);
  if (fresh) {
    const int below = static_cast<int>(__builtin_amdgcn_mbcnt_hi(
        static_cast<unsigned>(m >> 32), __builtin_amdgcn_mbcnt_lo(static_cast<unsigned>(m), 0u)));
    const long long pos = static_cast<long long>(base >> kAppShift) + below;
    lo.list[pos] = v;
    if (lo.doff != nullptr) lo.doff[pos] = static_cast<long long>(base & kAppMask) + dinc - dv;
  }
}

// Edge-parallel scatter. Pushed arcs are numbered: arc e of listed vertex j has
// index doff[j] + its position in j's out-row. A wave takes a chunk of C
// consecutive arcs (C = 1 when there are few arcs, so that many waves run at
// once; up to 64 when there are many), each lane resolves one arc's source slot
// and sink and marks the sink, then G lanes per arc add the source's delta row
// into the sink's row of S with fp32 atomics (coalesced across the G lanes). The
// delta row stays in registers while consecutive arcs share a source, so a hub's
// arcs cost one row load per chunk; hubs spread over many waves.
template <int G, int NC, bool PUSH, bool LIST>
__global__ __launch_bounds__(256) void k_scatter(int d, int ld, const int *list, const u64 *count, const long long *doff,
                                                 const float *delta, Adj out, float *S, unsigned *bm_out,
                                                 unsigned *bm_x, const int *ins_dst, const int *del_dst,
                                                 const u64 *pushed, const Counters *c, int mark_list,
                                                 ScatterCopy copy, ScatterList lo, int packed_in) {
  const u64 cw = *count;
  const long long nD = static_cast<long long>(packed_in ? cw >> kAppShift : cw);
  const long long E = static_cast<long long>(packed_in ? cw & kAppMask : *pushed);
  const long long ni = static_cast<long long>(c->n_ins);
  const long long na = ni + static_cast<long long>(c->n_del);
  if (aborted_with(c->abort, nD, E, na)) return;
  const int lane = lane_id();
  {
    const long long stride = static_cast<long long>(gridDim.x) * blockDim.x;
    const long long t0 = blockIdx.x * blockDim.x + threadIdx.x;
    if (!LIST) {
      for (long long i = t0; i < na; i += stride) mark_only(bm_x, i < ni ? ins_dst[i] : del_dst[i - ni]);
      if (mark_list)
        for (long long j = t0; j < nD; j += stride) mark_only(bm_x, list[j]);
    } else {
      // the net arcs' heads, then D when it joins A^l: whole waves step together
      const long long marks = na + (mark_list ? nD : 0);
      for (long long b = t0 - lane; b < marks; b += stride) {
        const long long i = b + lane;
        const int v = i >= marks ? -1 : i < ni ? ins_dst[i] : i < na ? del_dst[i - ni] : list[i - na];
        list_mark(v, false, lo, bm_out, bm_x);
      }
    }
  }
  if (copy.dst != nullptr) {
    // the staged rows of the listed vertices, one wave each from the grid's last
    // wave down (nothing in this kernel reads them)
    for (long long j = num_waves() - 1 - global_wave(); j < nD; j += num_waves()) {
      float *xu = copy.dst + static_cast<long long>(list[j]) * copy.d;
      const float *sj = copy.stage + j * copy.ld;
      for (int k = lane; k < copy.d; k += kWave) xu[k] = sj[k];
    }
  }
  const long long waves = num_waves();
  if (LIST) {
    // A^l listed here: the sinks are marked 64 arcs per wave (one list append per
    // wave), by waves from the grid's last one down (the adds below start at wave 0)
    const long long groups = (E + kWave - 1) / kWave;
    for (long long g = waves - 1 - global_wave(); g < groups; g += waves) {
      const long long e0 = g * kWave;
      const long long elast = e0 + kWave - 1 < E - 1 ? e0 + kWave - 1 : E - 1;
      // the search's last round leaves doff[w0 .. w0 + 63] in the lanes (w0 <= ja):
      // when the group's last arc falls in that window (no more than 64 - (ja - w0)
      // owners), each arc's owner and offset come from it by shuffles, with no
      // further load of the offsets
      long long mine, w0;
      const long long ja = wave_last_le_win(doff, nD, e0, mine, w0);
      const int owners = __popcll(__ballot(mine <= elast));  // window entries starting at or before elast
      int v = -1;
      if (owners < kWave || w0 + kWave >= nD) {
        const long long e = e0 + lane;
        int cnt_le = 0;
        for (int t = static_cast<int>(ja - w0); t < owners; ++t) cnt_le += __shfl(mine, t) <= e ? 1 : 0;
        const int at = static_cast<int>(ja - w0) + (cnt_le > 0 ? cnt_le - 1 : 0);
        const long long start = __shfl(mine, at);
        if (e <= elast) {
          const int u = list[w0 + at];
          v = out.col[out.off[u] + (e - start)];
        }
      } else {
        v = run_sink(doff, list, out, e0, elast, ja, owner_from(doff, ja, nD, elast));
      }
      list_mark(v, true, lo, bm_out, bm_x);
    }
  }
  // the owner searches run over doff[0, n1): a compacted list's doff[nD] holds the
  // arc total; a scatter-built list has no such entry, and needs none, as every
  // arc index is below the total
  const long long n1 = packed_in ? nD : nD + 1;
  int C = 1;
  while (C < kWave && static_cast<long long>(C) * waves < E) C <<= 1;
  constexpr int kEdgesPerStep = kWave / G;
  const int grp = lane / G, k0 = lane % G;
  int cached = -1;
  float dreg[NC];
  const long long chunks = (E + C - 1) / C;
  // a wave takes a contiguous run of chunks, so each chunk's first source is
  // found from the previous chunk's
  const long long per = (chunks + waves - 1) / waves;
  const long long c0 = global_wave() * per;
  const long long c1 = c0 + per < chunks ? c0 + per : chunks;
  long long ja = -1;
  for (long long ch = c0; ch < c1; ++ch) {
    const long long e0 = ch * C;
    const long long elast = e0 + C - 1 < E - 1 ? e0 + C - 1 : E - 1;
    ja = ja < 0 ? wave_last_le(doff, 0, n1, e0) : owner_from(doff, ja, n1, e0);
    if (PUSH && ja != cached) {
      // the chunk's first source is known before its arcs are resolved: fetch its
      // delta row now so that the load overlaps the list / offset / column reads
      const float *dj = delta + ja * ld;
#pragma unroll
      for (int q = 0; q < NC; ++q) {
        const int k = k0 + q * G;
        dreg[q] = k < d ? dj[k] : 0.0f;
      }
      cached = static_cast<int>(ja);
    }
    const long long jb = C == 1 ? ja : owner_from(doff, ja, n1, elast);
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
    float wv = 1.0f;  // the arc's weight (weighted graphs)
    if (active) {
      const int u = list[j];
      const long long slot = out.off[u] + (e - doff[j]);
      v = out.col[slot];
      if (PUSH && out.wt != nullptr) wv = out.wt[slot];
    }
    if (!LIST && v >= 0) mark_only(bm_out, v);
    const int cnt = PUSH ? static_cast<int>(elast - e0 + 1) : 0;
    for (int i = 0; i < cnt; i += kEdgesPerStep) {
      const int vv = __shfl(v, i + grp);
      const int jj = __shfl(j, i + grp);
      const float ww = __shfl(wv, i + grp);
      if (vv >= 0) {
        if (jj != cached) {
          const float *dj = delta + static_cast<long long>(jj) * ld;
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
          if (k < d) unsafeAtomicAdd(&sv[k], ww * dreg[q]);
        }
      }
    }
  }
}

constexpr int kPullArcs = 4;  // arcs per lane per chunk (the pull and the bucket passes)
constexpr int kPullChunk = kWave * kPullArcs;

// Exclusive prefix sums of a[0, n) in LDS, in place, by a block of kBinThreads
// threads (each a run of consecutive entries); ends with a barrier.
__device__ inline void block_exclusive_scan(int *a, int n, int *wave_sums) {
  const int t = threadIdx.x, lane = lane_id(), wave = t / kWave;
  const int per = (n + kBinThreads - 1) / kBinThreads;
  int s = 0;
  for (int i = 0; i < per; ++i) {
    const int k = t * per + i;
    if (k < n) s += a[k];
  }
  int incl = s;
#pragma unroll
  for (int o = 1; o < kWave; o <<= 1) {
    const int y = __shfl_up(incl, o);
    if (lane >= o) incl += y;
  }
  if (lane == kWave - 1) wave_sums[wave] = incl;
  __syncthreads();
  int base = incl - s;
  for (int w = 0; w < wave; ++w) base += wave_sums[w];
  for (int i = 0; i < per; ++i) {
    const int k = t * per + i;
    if (k < n) {
      const int x = a[k];
      a[k] = base;
      base += x;
    }
  }
  __syncthreads();
}

// The bucket form's passes over the pushed arcs (numbered as in the scatter), in
// chunks of up to kPullChunk consecutive arcs per wave (a contiguous run of chunks
// per wave, so that a block owns the same arcs in both passes), each lane up to
// kPullArcs consecutive arcs with all their loads in flight together. The arcs are
// sorted by sink in two levels: into bins of 2^shift consecutive sinks here, then
// by sink within each bin (k_bin_sort). Counting pass (SCATTER false): marks the
// net arcs' heads and, under a self term, D in bm_x, counts the block's arcs per
// bin in LDS, and adds each count to its bin's total with one atomic, which hands
// back the block's place in the bin. Scatter pass: the bins' first slots are the
// exclusive prefix of their totals (block 0 also stores them); each arc takes the
// next place of its block in its bin (an LDS cursor) and leaves its sink, its
// source's list position (its message row) and, when the model weights arcs, its
// weight there.
template <bool SCATTER>
__global__ __launch_bounds__(kBinThreads) void k_bin_arcs(const int *list, const u64 *count, const long long *doff,
                                                           Adj out, const u64 *pushed, Buckets b, unsigned *bm_x,
                                                           const int *ins_dst, const int *del_dst, int mark_list,
                                                           const Counters *c) {
  extern __shared__ int bins[];  // per bin: the block's count, or its cursor
  __shared__ int wave_sums[kBinThreads / kWave];
  const long long nD = static_cast<long long>(*count);
  const long long E = static_cast<long long>(*pushed);
  const long long ni = static_cast<long long>(c->n_ins);
  const long long na = ni + static_cast<long long>(c->n_del);
  if (aborted_with(c->abort, nD, E, na)) return;  // the same for the whole block
  const int lane = lane_id();
  const int nb = b.nbins;
  if (!SCATTER) {
    for (int i = threadIdx.x; i < nb; i += kBinThreads) bins[i] = 0;
    const long long stride = static_cast<long long>(gridDim.x) * kBinThreads;
    const long long t0 = blockIdx.x * static_cast<long long>(kBinThreads) + threadIdx.x;
    for (long long i = t0; i < na; i += stride) mark_only(bm_x, i < ni ? ins_dst[i] : del_dst[i - ni]);
    if (mark_list)
      for (long long j = t0; j < nD; j += stride) mark_only(bm_x, list[j]);
    __syncthreads();
  } else {
    for (int i = threadIdx.x; i < nb; i += kBinThreads) bins[i] = b.bin_total[i];
    __syncthreads();
    block_exclusive_scan(bins, nb, wave_sums);
    const int *own = b.block_off + static_cast<long long>(blockIdx.x) * nb;
    for (int i = threadIdx.x; i < nb; i += kBinThreads) {
      if (blockIdx.x == 0) b.bin_base[i] = bins[i];
      bins[i] += own[i];
    }
    __syncthreads();
  }
  const long long waves = num_waves();
  const long long n1 = nD + 1;  // a compacted list: doff[nD] holds the arc total
  int C = 1;
  while (C < kPullChunk && static_cast<long long>(C) * waves < E) C <<= 1;
  const int per_lane = C > kWave ? C / kWave : 1;
  const long long chunks = (E + C - 1) / C;
  const long long per = (chunks + waves - 1) / waves;
  const long long c0 = global_wave() * per;
  const long long c1 = c0 + per < chunks ? c0 + per : chunks;
  long long ja = -1;
  for (long long ch = c0; ch < c1; ++ch) {
    const long long e0 = ch * C;
    const long long elast = e0 + C - 1 < E - 1 ? e0 + C - 1 : E - 1;
    ja = ja < 0 ? wave_last_le(doff, 0, n1, e0) : owner_from(doff, ja, n1, e0);
    const long long jb = C == 1 ? ja : owner_from(doff, ja, n1, elast);
    long long e[kPullArcs];
    int r[kPullArcs];
    bool on[kPullArcs];
#pragma unroll
    for (int a = 0; a < kPullArcs; ++a) {
      e[a] = e0 + static_cast<long long>(lane) * per_lane + a;
      on[a] = a < per_lane && e[a] <= elast;
      r[a] = static_cast<int>(ja);
    }
    if (jb > ja) {
      if (jb - ja < kWave) {
        // the window's offsets, one per lane; every lane takes part in the shuffles
        const long long mine = ja + lane <= jb ? doff[ja + lane] : (1LL << 62);
        int cnt[kPullArcs] = {};
        for (int t = 0; t <= static_cast<int>(jb - ja); ++t) {
          const long long o = __shfl(mine, t);
#pragma unroll
          for (int a = 0; a < kPullArcs; ++a) cnt[a] += o <= e[a] ? 1 : 0;
        }
#pragma unroll
        for (int a = 0; a < kPullArcs; ++a) r[a] = static_cast<int>(ja) + cnt[a] - 1;
      } else {
#pragma unroll
        for (int a = 0; a < kPullArcs; ++a)
          if (on[a]) r[a] = static_cast<int>(upper_bound(doff, ja, jb + 1, e[a]) - 1);
      }
    }
    long long slot[kPullArcs];
    int v[kPullArcs];
#pragma unroll
    for (int a = 0; a < kPullArcs; ++a) {
      const int u = on[a] ? list[r[a]] : 0;
      slot[a] = on[a] ? out.off[u] + (e[a] - doff[r[a]]) : 0;
    }
#pragma unroll
    for (int a = 0; a < kPullArcs; ++a) v[a] = on[a] ? out.col[slot[a]] : 0;
    if (!SCATTER) {
#pragma unroll
      for (int a = 0; a < kPullArcs; ++a)
        if (on[a]) atomicAdd(&bins[v[a] >> b.shift], 1);
    } else {
      float w[kPullArcs];
#pragma unroll
      for (int a = 0; a < kPullArcs; ++a) w[a] = on[a] && b.tw != nullptr ? out.wt[slot[a]] : 1.0f;
#pragma unroll
      for (int a = 0; a < kPullArcs; ++a) {
        if (!on[a]) continue;
        const int p = atomicAdd(&bins[v[a] >> b.shift], 1);
        b.tv[p] = v[a];
        b.tj[p] = r[a];
        if (b.tw != nullptr) b.tw[p] = w[a];
      }
    }
  }
  if (!SCATTER) {
    // the block's counts into the bins' totals; a bin it has no arc in gets place 0
    __syncthreads();
    int *own = b.block_off + static_cast<long long>(blockIdx.x) * nb;
    for (int i = threadIdx.x; i < nb; i += kBinThreads) own[i] = bins[i] > 0 ? atomicAdd(&b.bin_total[i], bins[i]) : 0;
  }
}

// Second level of the bucket sort: block i takes bin i (sinks i 2^shift ..
// (i + 1) 2^shift - 1, its arcs in slots bin_base[i] .. + bin_total[i]). It counts
// the arcs per sink in LDS, stores the counts in cnt (from which the compaction
// lists the sinks and forms their buckets' offsets, the same prefix sums in vertex
// order), then places each arc at its sink's next slot: idx (and wt) hold each
// sink's bucket contiguously, buckets in vertex order. Resets the bin's total.
__global__ __launch_bounds__(kBinThreads) void k_bin_sort(long long n, const u64 *pushed, Buckets b,
                                                           const Counters *c) {
  extern __shared__ int cur[];  // per sink of the bin: its count, then its next slot
  __shared__ int wave_sums[kBinThreads / kWave];
  const long long E = static_cast<long long>(*pushed);
  if (aborted_with(c->abort, E)) return;
  const int bin = blockIdx.x;
  const int total = b.bin_total[bin];
  if (total == 0) return;  // the same for the whole block; its sinks' counters stay zero
  const int base = b.bin_base[bin];
  const int span = 1 << b.shift;
  const long long v0 = static_cast<long long>(bin) << b.shift;
  const int nv = static_cast<int>(n - v0 < span ? n - v0 : span);
  const int t = threadIdx.x;
  for (int i = t; i < span; i += kBinThreads) cur[i] = 0;
  __syncthreads();
  if (t == 0) b.bin_total[bin] = 0;  // every thread has read it
  constexpr int kU = 8;  // arcs per thread in flight
  for (int p0 = t; p0 < total; p0 += kU * kBinThreads) {
    int vv[kU];
#pragma unroll
    for (int q = 0; q < kU; ++q) {
      const int p = p0 + q * kBinThreads;
      vv[q] = p < total ? b.tv[base + p] : -1;
    }
#pragma unroll
    for (int q = 0; q < kU; ++q)
      if (vv[q] >= 0) atomicAdd(&cur[vv[q] - v0], 1);
  }
  __syncthreads();
  for (int i = t; i < nv; i += kBinThreads) b.cnt[v0 + i] = cur[i];
  block_exclusive_scan(cur, span, wave_sums);
  for (int p0 = t; p0 < total; p0 += kU * kBinThreads) {
    int vv[kU], jj[kU];
    float ww[kU];
#pragma unroll
    for (int q = 0; q < kU; ++q) {
      const int p = p0 + q * kBinThreads;
      const bool on = p < total;
      vv[q] = on ? b.tv[base + p] : -1;
      jj[q] = on ? b.tj[base + p] : 0;
      ww[q] = on && b.tw != nullptr ? b.tw[base + p] : 1.0f;
    }
#pragma unroll
    for (int q = 0; q < kU; ++q) {
      if (vv[q] < 0) continue;
      const int at = base + atomicAdd(&cur[vv[q] - v0], 1);
      b.idx[at] = jj[q];
      if (b.wt != nullptr) b.wt[at] = ww[q];
    }
  }
}

// Pull form of the message step (for dense frontiers). In-arcs of the sorted
// list A are numbered like the scatter's out-arcs (ioff gives each listed
// vertex's first in-arc). A wave takes chunks of up to 256 consecutive in-arcs (a
// contiguous run of chunks per wave), each lane up to four consecutive arcs: it
// resolves their sinks v and sources u, all loads of its arcs in flight together,
// and keeps an arc if u is dirty (member bit), with the source's message row (u's
// rank among the members, from the member word and the count of members before
// it). The (sink, row) pairs go to LDS in arc order. Groups of G lanes then walk
// the arcs of their own window (a quarter of the chunk when G = 16, all of it when
// G = 64), U message rows in flight at a time, summing rows into registers while
// the sink stays the same and adding each sum to S[v] with one row of fp32
// atomics: a sink's messages cost one read each, and one row update per window it
// spans. G = 16 for rows of at most 64 floats (four rows per wave instruction).

template <int G, int NC, int U>
__global__ __launch_bounds__(256) void k_pull_msgs(int d, int ld, const int *list, const u64 *count,
                                                   const long long *ioff, Adj in, const uint2 *memb,
                                                   const float *msg, float *S, unsigned *mark,
                                                   const Counters *c) {
  __shared__ int2 pairs[256 / kWave][kPullChunk];
  __shared__ float pair_w[256 / kWave][kPullChunk];  // the in-arcs' weights (weighted graphs)
  const long long nA = static_cast<long long>(*count);
  if (aborted_with(c->abort, nA)) return;
  const int lane = lane_id();
  const int grp = lane / G, k0 = lane % G;
  int2 *wp = pairs[threadIdx.x / kWave];
  float *ww = pair_w[threadIdx.x / kWave];
  const bool weighted = in.wt != nullptr;
  const long long E = ioff[nA];
  const long long waves = num_waves();
  int C = 1;
  while (C < kPullChunk && static_cast<long long>(C) * waves < E) C <<= 1;
  const int per_lane = C > kWave ? C / kWave : 1;  // arcs per lane
  const int window = C / (kWave / G) > 0 ? C / (kWave / G) : 1;  // chunk positions per group
  const long long chunks = (E + C - 1) / C;
  const long long per = (chunks + waves - 1) / waves;
  const long long c0 = global_wave() * per;
  const long long c1 = c0 + per < chunks ? c0 + per : chunks;
  long long ja = -1;
  for (long long ch = c0; ch < c1; ++ch) {
    const long long e0 = ch * C;
    const long long elast = e0 + C - 1 < E - 1 ? e0 + C - 1 : E - 1;
    ja = ja < 0 ? wave_last_le(ioff, 0, nA + 1, e0) : owner_from(ioff, ja, nA + 1, e0);
    const long long jb = C == 1 ? ja : owner_from(ioff, ja, nA + 1, elast);
    // this lane's arcs: chunk positions lane * per_lane + a
    long long e[kPullArcs];
    int r[kPullArcs];
#pragma unroll
    for (int a = 0; a < kPullArcs; ++a) {
      e[a] = e0 + static_cast<long long>(lane) * per_lane + a;
      r[a] = static_cast<int>(ja);
    }
    if (jb > ja) {
      if (jb - ja < kWave) {
        // the window's offsets, one per lane; every lane takes part in the shuffles
        const long long mine = ja + lane <= jb ? ioff[ja + lane] : (1LL << 62);
        int cnt[kPullArcs] = {};
        for (int t = 0; t <= static_cast<int>(jb - ja); ++t) {
          const long long o = __shfl(mine, t);
#pragma unroll
          for (int a = 0; a < kPullArcs; ++a) cnt[a] += o <= e[a] ? 1 : 0;
        }
#pragma unroll
        for (int a = 0; a < kPullArcs; ++a) r[a] = static_cast<int>(ja) + cnt[a] - 1;
      } else {
#pragma unroll
        for (int a = 0; a < kPullArcs; ++a)
          if (a < per_lane && e[a] <= elast) r[a] = static_cast<int>(upper_bound(ioff, ja, jb + 1, e[a]) - 1);
      }
    }
    int v[kPullArcs], u[kPullArcs];
    float w[kPullArcs];
#pragma unroll
    for (int a = 0; a < kPullArcs; ++a) {
      const bool active = a < per_lane && e[a] <= elast;
      v[a] = active ? (list != nullptr ? list[r[a]] : r[a]) : -1;
    }
#pragma unroll
    for (int a = 0; a < kPullArcs; ++a) {
      const long long slot = v[a] >= 0 ? in.off[v[a]] + (e[a] - ioff[r[a]]) : 0;
      u[a] = v[a] >= 0 ? __builtin_nontemporal_load(in.col + slot) : -1;
      w[a] = weighted && v[a] >= 0 ? __builtin_nontemporal_load(in.wt + slot) : 1.0f;
    }
#pragma unroll
    for (int a = 0; a < kPullArcs; ++a) {
      int j = -1;
      if (u[a] >= 0) {
        const uint2 mw = memb[u[a] >> 5];  // the member word and the members before it
        const unsigned bit = 1u << (u[a] & 31);
        if (mw.x & bit) j = static_cast<int>(mw.y) + __popc(mw.x & (bit - 1u));
      }
      if (a < per_lane) {
        wp[lane * per_lane + a] = make_int2(v[a], j);
        if (weighted) ww[lane * per_lane + a] = w[a];
      }
    }
    // the pairs are read back by other lanes of this wave only
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
    int cur = -1;
    float acc[NC];
#pragma unroll
    for (int q = 0; q < NC; ++q) acc[q] = 0.0f;
    const int base = grp * window;
    for (int t0 = 0; t0 < window; t0 += U) {  // trip count is the same for the whole wave
      int vv[U], jj[U];
      float wt[U];
#pragma unroll
      for (int t = 0; t < U; ++t) {
        const int pos = t0 + t;
        int2 pr = make_int2(-1, -1);
        float pw = 1.0f;
        if (pos < window && base + pos < C) {
          pr = wp[base + pos];
          if (weighted) pw = ww[base + pos];
        }
        vv[t] = pr.x;
        jj[t] = pr.y;
        wt[t] = pw;
      }
      // unconditional loads (an empty slot reads message row 0, a column past the
      // end the last column) masked to zero afterwards: no branch between the
      // loads (columns past the end are summed but never flushed)
      float row[U][NC];
#pragma unroll
      for (int t = 0; t < U; ++t) {
        // the group's whole span from the row start, column offsets as immediates
        // (columns past d read the next row or the table's tail, kRowTail)
        const float *mj = msg + static_cast<long long>(jj[t] >= 0 ? jj[t] : 0) * ld + k0;
        const unsigned keep = jj[t] >= 0 ? ~0u : 0u;
#pragma unroll
        for (int q = 0; q < NC; ++q) row[t][q] = __uint_as_float(__float_as_uint(mj[q * G]) & keep);
      }
#pragma unroll
      for (int t = 0; t < U; ++t) {
        if (jj[t] < 0) continue;
        if (vv[t] != cur) {
          if (cur >= 0) {
            float *sv = S + static_cast<long long>(cur) * d;
#pragma unroll
            for (int q = 0; q < NC; ++q) {
              const int k = k0 + q * G;
              if (k < d) unsafeAtomicAdd(&sv[k], acc[q]);
              acc[q] = 0.0f;
            }
            if (mark != nullptr && k0 == 0) mark_only(mark, cur);
          }
          cur = vv[t];
        }
#pragma unroll
        for (int q = 0; q < NC; ++q) acc[q] += wt[t] * row[t][q];
      }
    }
    if (cur >= 0) {
      float *sv = S + static_cast<long long>(cur) * d;
#pragma unroll
      for (int q = 0; q < NC; ++q) {
        const int k = k0 + q * G;
        if (k < d) unsafeAtomicAdd(&sv[k], acc[q]);
      }
      if (mark != nullptr && k0 == 0) mark_only(mark, cur);
    }
    // the next chunk overwrites the pairs only after every lane has read them
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
  }
}

// Recompute form of the message step (see launch_recompute). The in-arcs of the
// sorted list A are numbered by ioff. A wave takes ranges of C consecutive arc
// numbers (a contiguous run of ranges per wave, so that each range's sinks are
// found from the previous range's) and owns every segment that starts in its
// range: a segment is up to kRecomputeSeg consecutive in-arcs of one sink, the
// sink's own arcs from ioff_j + s kRecomputeSeg on. So a range owns segment 0 of
// the sinks that start in it (with C <= kRecomputeSeg no other segment of those),
// and at most one later segment of the sink that covers its first arc. The
// range's segments go round-robin to the wave's G-lane groups. A group fetches
// its segment's source ids, weights and coefficients in one round (each lane
// kRecomputeSeg / G arcs), then its source rows U at a time, summing in fp64. A
// sink of one segment is stored once, rounded to fp32; the segments of longer
// sinks are added with fp32 atomics into rows the compaction zeroed. The last
// range also owns the sinks past the last arc (rows without in-arcs, stored as
// zeros).
template <int G, int NC, int U>
__global__ __launch_bounds__(256) void k_recompute(int d, int gcn, const int *list, const u64 *count,
                                                   const long long *ioff, Adj in, const int *out_len,
                                                   const float *src, float *S, const Counters *c) {
  static_assert(G % U == 0 && kRecomputeSeg % G == 0, "steps of U arcs stay within one fetch slot");
  // the first kWave sinks of a range, fetched by the wave in one round when the range
  // starts: their first arc, their end and their vertex (read back by their groups)
  __shared__ long long sink_a[256 / kWave][kWave], sink_b[256 / kWave][kWave];
  __shared__ int sink_v[256 / kWave][kWave];
  long long *pa = sink_a[threadIdx.x / kWave], *pb = sink_b[threadIdx.x / kWave];
  int *pv = sink_v[threadIdx.x / kWave];
  constexpr int kPer = kRecomputeSeg / G;  // arcs fetched per lane
  constexpr int kSteps = kRecomputeSeg / U;
  const long long nA = static_cast<long long>(*count);
  if (aborted_with(c->abort, nA)) return;
  const int lane = lane_id();
  constexpr int kGroups = kWave / G;
  const int grp = lane / G, k0 = lane % G;
  const bool weighted = in.wt != nullptr;
  const long long E = ioff[nA];
  const long long waves = num_waves();
  long long C = 16;
  while (C < kRecomputeSeg && C * waves < E) C <<= 1;
  const long long ranges = E > 0 ? (E + C - 1) / C : 1;
  const long long per = (ranges + waves - 1) / waves;
  const long long r0 = global_wave() * per;
  const long long r1 = r0 + per < ranges ? r0 + per : ranges;
  long long jlast = -1;  // the last sink of the previous range (its successor starts this one's)
  for (long long r = r0; r < r1; ++r) {
    const long long R0 = r * C;
    const bool last_range = r == ranges - 1;
    const long long R1 = last_range ? (1LL << 62) : R0 + C;
    // first sink starting at or after R0, then the last one starting before R1
    const long long jf = r == r0 ? (R0 == 0 ? 0 : wave_last_le(ioff, 0, nA + 1, R0 - 1) + 1) : jlast + 1;
    long long jl = last_range ? nA - 1 : owner_from(ioff, jf > 0 ? jf - 1 : 0, nA + 1, R1 - 1);
    if (jl > nA - 1) jl = nA - 1;
    jlast = jl;
    // the sink before jf covers arc R0 when it ends past it: it may have a segment
    // starting in this range
    long long pstart = -1, pend = 0, pj = jf - 1;
    if (pj >= 0) {
      const long long a = ioff[pj], b = ioff[pj + 1];
      if (b > R0) {
        const long long s = (R0 - a + kRecomputeSeg - 1) / kRecomputeSeg;
        const long long st = a + s * kRecomputeSeg;
        if (st < R1 && st < b) {
          pstart = st;
          pend = st + kRecomputeSeg < b ? st + kRecomputeSeg : b;
        }
      }
    }
    const long long has_pred = pstart >= 0 ? 1 : 0;
    const long long sinks = jl >= jf ? jl - jf + 1 : 0;
    const long long items = has_pred + sinks;
    if (lane < sinks) {
      const long long j = jf + lane;
      pa[lane] = ioff[j];
      pb[lane] = ioff[j + 1];
      pv[lane] = list != nullptr ? list[j] : static_cast<int>(j);
    }
    // the sinks are read back by other lanes of this wave only
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
    for (long long it = grp; it < items; it += kGroups) {  // the same bounds for a group's lanes
      long long j, a0, a1;
      bool whole;
      int v;
      if (it < has_pred) {
        j = pj;
        a0 = pstart;
        a1 = pend;
        whole = false;
        v = list != nullptr ? list[j] : static_cast<int>(j);
      } else {
        const long long q = it - has_pred;
        j = jf + q;
        long long a, b;
        if (q < kWave) {
          a = pa[q];
          b = pb[q];
          v = pv[q];
        } else {
          a = ioff[j];
          b = ioff[j + 1];
          v = list != nullptr ? list[j] : static_cast<int>(j);
        }
        a0 = a;
        whole = b - a <= kRecomputeSeg;
        a1 = whole ? b : a + kRecomputeSeg;
      }
      const int na = static_cast<int>(a1 - a0);  // arcs in the segment (<= kRecomputeSeg)
      float *sv = S + static_cast<long long>(v) * d;
      // in-arc a0 + i of the sink's row
      const long long row0 = in.off[v] - ioff[j] + a0;
      // arc i of the segment is fetched by lane i % G of the group, into slot i / G
      int uq[kPer];
      double cq[kPer];
#pragma unroll
      for (int q = 0; q < kPer; ++q) {
        const int i = k0 + q * G;
        uq[q] = i < na ? in.col[row0 + i] : -1;
        cq[q] = i < na && weighted ? static_cast<double>(in.wt[row0 + i]) : 1.0;
      }
      if (gcn) {
#pragma unroll
        for (int q = 0; q < kPer; ++q)
          if (uq[q] >= 0) cq[q] /= sqrt(static_cast<double>(out_len[uq[q]]) + 1.0);
      }
      double acc[NC];
#pragma unroll
      for (int q = 0; q < NC; ++q) acc[q] = 0;
#pragma unroll
      for (int st = 0; st < kSteps; ++st) {
        if (st * U >= na) break;  // the same for the group's lanes
        const int q = st * U / G;  // the fetch slot of this step's arcs
        int uu[U];
        double cc[U];
#pragma unroll
        for (int t = 0; t < U; ++t) {
          const int from = grp * G + (st * U + t) % G;
          uu[t] = __shfl(uq[q], from);
          cc[t] = __shfl(cq[q], from);
        }
        // every lane loads (an empty slot reads row 0, a column past the end the
        // last column) and the value is masked to zero afterwards: the loads carry
        // no branch and are all in flight together (columns past the end are
        // summed but never stored)
        float row[U][NC];
#pragma unroll
        for (int t = 0; t < U; ++t) {
          // the group's whole span from the row start, column offsets as immediates
          // (columns past d read the next row or the table's tail, kRowTail)
          const float *su = src + static_cast<long long>(uu[t] >= 0 ? uu[t] : 0) * d + k0;
          const unsigned keep = uu[t] >= 0 ? ~0u : 0u;
#pragma unroll
          for (int p = 0; p < NC; ++p) row[t][p] = __uint_as_float(__float_as_uint(su[p * G]) & keep);
        }
#pragma unroll
        for (int t = 0; t < U; ++t)
#pragma unroll
          for (int p = 0; p < NC; ++p) acc[p] += cc[t] * static_cast<double>(row[t][p]);
      }
#pragma unroll
      for (int p = 0; p < NC; ++p) {
        const int k = k0 + p * G;
        if (k < d) {
          if (whole) sv[k] = static_cast<float>(acc[p]);
          else unsafeAtomicAdd(&sv[k], static_cast<float>(acc[p]));
        }
      }
    }
    // the next range overwrites the sinks only after every group has read them
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
  }
}

// The bucket form's sums (see launch_bucket_sum), on the recompute's split with
// bucket slots for in-arcs: ranges of C <= kRecomputeSeg consecutive slots, a
// contiguous run of them per wave; a range owns the first segment (up to
// kRecomputeSeg slots) of each sink whose bucket starts in it and at most one
// later segment of the sink before. Besides the message and aggregate rows, a
// range reads only three windows, which its wave fetches in one round of loads:
// the bucket starts and the vertices of the 64 sinks from the one before the
// range's first (lane t: boff and list at jf - 1 + t), and the 128 slots (message
// row and weight) from the range start, since a segment that starts in a range of
// at most 64 slots ends within 128 slots of its start. The windows of the wave's
// next range are fetched while the groups sum this range's segments, so a segment
// costs one round trip: its message rows, loaded together with its aggregate row.
// Sums are fp32; a one-segment bucket is added with a plain load and store, longer
// ones with atomics. Sinks with empty buckets are left alone; each sink's first
// segment resets its counter.
template <int G, int NC, int U>
__global__ __launch_bounds__(256) void k_bucket_sum(int d, int ld, const int *list, const u64 *count,
                                                    const long long *boff, Buckets bk, const float *msg, float *S,
                                                    const Counters *c) {
  static_assert(kWave % G == 0 && G % U == 0 && kRecomputeSeg % U == 0, "steps of U slots");
  static_assert(kRecomputeSeg <= kWave, "a segment starting in a range ends within two windows of slots");
  constexpr int kSlots = 2 * kWave;
  constexpr int kSteps = kRecomputeSeg / U;
  constexpr int kGroups = kWave / G;
  __shared__ long long win_b[256 / kWave][kWave];
  __shared__ int win_v[256 / kWave][kWave];
  __shared__ int win_u[256 / kWave][kSlots];
  __shared__ float win_w[256 / kWave][kSlots];
  const int w = threadIdx.x / kWave;
  long long *wb = win_b[w];
  int *wv = win_v[w], *wu = win_u[w];
  float *ww = win_w[w];
  const long long nA = static_cast<long long>(*count);
  if (aborted_with(c->abort, nA) || nA == 0) return;
  const long long E = boff[nA];
  if (E == 0) return;  // no message reached any sink
  const int lane = lane_id();
  const int grp = lane / G, k0 = lane % G;
  const bool weighted = bk.wt != nullptr;
  // the weight window is loaded unconditionally (from the slot array when there are no weights)
  const float *wsrc = weighted ? bk.wt : reinterpret_cast<const float *>(bk.idx);
  const long long waves = num_waves();
  long long C = 16;
  while (C < kRecomputeSeg && C * waves < E) C <<= 1;
  const long long ranges = (E + C - 1) / C;
  const long long per = (ranges + waves - 1) / waves;
  const long long r0 = global_wave() * per;
  const long long r1 = r0 + per < ranges ? r0 + per : ranges;
  if (r0 >= r1) return;
  // the window registers of the next range (clamped loads: entries outside the
  // list or the slots repeat its ends and are never used, except boff past nA,
  // which reads E and so ends the search for the range's last sink)
  long long nb;
  int nv, nu0, nu1;
  float nw0, nw1;
  const auto fetch = [&](long long jf, long long R0) {
    const long long i = jf - 1 + lane;
    const long long ib = i < 0 ? 0 : i > nA ? nA : i;
    const long long iv = i < 0 ? 0 : i > nA - 1 ? nA - 1 : i;
    const long long s0 = R0 + lane < E ? R0 + lane : E - 1;
    const long long s1 = R0 + kWave + lane < E ? R0 + kWave + lane : E - 1;
    nb = boff[ib];
    nv = list[iv];
    nu0 = bk.idx[s0];
    nu1 = bk.idx[s1];
    nw0 = wsrc[s0];
    nw1 = wsrc[s1];
  };
  // first sink starting at or after the first range's start
  long long jf = r0 == 0 ? 0 : wave_last_le(boff, 0, nA + 1, r0 * C - 1) + 1;
  fetch(jf, r0 * C);
  for (long long r = r0; r < r1; ++r) {
    const long long R0 = r * C;
    const bool last_range = r == ranges - 1;
    const long long R1 = last_range ? (1LL << 62) : R0 + C;
    // the previous range's groups have read the windows: publish this range's
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
    wb[lane] = nb;
    wv[lane] = nv;
    wu[lane] = nu0;
    wu[kWave + lane] = nu1;
    ww[lane] = nw0;
    ww[kWave + lane] = nw1;
    // the last sink starting before R1: the window's entries <= R1 - 1 form a prefix
    // (lane 0 stands for the sink before jf, or for nothing when jf = 0)
    long long jl = nA - 1;
    if (!last_range) {
      const bool le = jf - 1 + lane < 0 || nb <= R1 - 1;
      const int cnt = __popcll(__ballot(le));
      jl = jf + cnt - 2;
      if (cnt == kWave && jf - 1 + kWave <= nA) jl = wave_last_le(boff, jf - 2 + kWave, nA + 1, R1 - 1);
      if (jl > nA - 1) jl = nA - 1;
    }
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
    if (r + 1 < r1) fetch(jl + 1, R0 + C);
    // the sink before jf covers slot R0 when its bucket ends past it: it may have a
    // segment starting in this range
    long long pstart = -1, pend = 0;
    if (jf >= 1) {
      const long long a = wb[0], b = wb[1];
      if (b > R0) {
        const long long s = (R0 - a + kRecomputeSeg - 1) / kRecomputeSeg;
        const long long st = a + s * kRecomputeSeg;
        if (st < R1 && st < b) {
          pstart = st;
          pend = st + kRecomputeSeg < b ? st + kRecomputeSeg : b;
        }
      }
    }
    const long long has_pred = pstart >= 0 ? 1 : 0;
    const long long sinks = jl >= jf ? jl - jf + 1 : 0;
    const long long items = has_pred + sinks;
    for (long long it = grp; it < items; it += kGroups) {  // the same bounds for a group's lanes
      long long a0, a1;
      bool whole, first;
      int v;
      if (it < has_pred) {
        a0 = pstart;
        a1 = pend;
        whole = false;
        first = false;  // a segment starting in this range is not the sink's first
        v = wv[0];
      } else {
        const long long q = it - has_pred;  // sink jf + q: window entries q + 1 and q + 2
        long long a, b;
        if (q + 2 < kWave) {
          a = wb[q + 1];
          b = wb[q + 2];
          v = wv[q + 1];
        } else {
          a = boff[jf + q];
          b = boff[jf + q + 1];
          v = list[jf + q];
        }
        a0 = a;
        whole = b - a <= kRecomputeSeg;
        a1 = whole ? b : a + kRecomputeSeg;
        first = true;
      }
      const int na = static_cast<int>(a1 - a0);  // slots in the segment (<= kRecomputeSeg)
      if (na == 0) continue;                      // no message reached the sink (the same for the group)
      float *sv = S + static_cast<long long>(v) * d;
      // the row's current values, loaded with the message rows (used when the
      // bucket is one segment)
      float prev[NC];
#pragma unroll
      for (int p = 0; p < NC; ++p) prev[p] = sv[k0 + p * G];  // past d: the next row or the tail (never used)
      if (k0 == 0 && first) bk.cnt[v] = 0;                   // the bucket's start is no longer needed
      const int o0 = static_cast<int>(a0 - R0);  // the segment's first slot in the window
      float acc[NC];
#pragma unroll
      for (int p = 0; p < NC; ++p) acc[p] = 0.0f;
#pragma unroll
      for (int st = 0; st < kSteps; ++st) {
        if (st * U >= na) break;  // the same for the group's lanes
        // every lane loads (a slot past the segment repeats its last one, a column
        // past the end reads the next row or the tail) and the value is masked to
        // zero afterwards: the loads carry no branch and go out together
        float row[U][NC];
        float cc[U];
#pragma unroll
        for (int t = 0; t < U; ++t) {
          const int i = st * U + t;
          const int o = o0 + (i < na ? i : na - 1);
          const float *su = msg + static_cast<long long>(wu[o]) * ld + k0;
          cc[t] = weighted ? ww[o] : 1.0f;
          const unsigned keep = i < na ? ~0u : 0u;
#pragma unroll
          for (int p = 0; p < NC; ++p) row[t][p] = __uint_as_float(__float_as_uint(su[p * G]) & keep);
        }
#pragma unroll
        for (int t = 0; t < U; ++t)
#pragma unroll
          for (int p = 0; p < NC; ++p) acc[p] += cc[t] * row[t][p];
      }
#pragma unroll
      for (int p = 0; p < NC; ++p) {
        const int k = k0 + p * G;
        if (k < d) {
          if (whole) sv[k] = prev[p] + acc[p];
          else unsafeAtomicAdd(&sv[k], acc[p]);
        }
      }
    }
    jf = jl + 1;
  }
}

// Bootstrap: S[v] = sum over in-arcs (u -> v) of c_u H[u], one wave per vertex,
// in the in-row's order, summed in fp64 and rounded once.
template <int NC>
__global__ __launch_bounds__(256) void k_pull(long long n, int d, int agg, const float *Hprev, Adj in,
                                              const int *out_len, float *S) {
  const int lane = lane_id();
  for (long long v = global_wave(); v < n; v += num_waves()) {
    double acc[NC];
#pragma unroll
    for (int q = 0; q < NC; ++q) acc[q] = 0.0;
    const int deg = in.len[v];
    const int *row = in.col + in.off[v];
    for (int e0 = 0; e0 < deg; e0 += kWave) {
      const int e = e0 + lane;
      const int uid = e < deg ? row[e] : 0;
      double cu = 1.0;
      if (agg == kGcn && e < deg) cu = 1.0 / sqrt(static_cast<double>(out_len[uid]) + 1.0);
      if (in.wt != nullptr && e < deg) cu *= static_cast<double>(in.wt[in.off[v] + e]);  // the arc's weight
      const int cnt = deg - e0 < kWave ? deg - e0 : kWave;
      for (int i = 0; i < cnt; ++i) {
        const int u = __shfl(uid, i);
        const double cf = __shfl(cu, i);
        const float *hu = Hprev + static_cast<long long>(u) * d;
#pragma unroll
        for (int q = 0; q < NC; ++q) {
          const int k = lane + q * kWave;
          if (k < d) acc[q] += cf * static_cast<double>(hu[k]);
        }
      }
    }
    float *sv = S + v * d;
#pragma unroll
    for (int q = 0; q < NC; ++q) {
      const int k = lane + q * kWave;
      if (k < d) sv[k] = static_cast<float>(acc[q]);
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

void launch_corr_mark(hipStream_t s, int cap_feat, int cap_arcs, int agg, LayerPtrs lp, Adj out, Adj in,
                      const int *ins_rank, const float *arc_w, const int *ddeg, const int *flist, const int *ins_src,
                      const int *ins_dst, const int *del_src, const int *del_dst, const float *ins_w,
                      const float *del_w, unsigned *bm, Counters *c, const DirectList &direct) {
  const long long waves = 2LL * cap_arcs * lp.L;
  const long long threads = static_cast<long long>(cap_feat) + 2LL * cap_arcs;
  const long long items = waves * kWave > threads ? waves * kWave : threads;
  RP_LAUNCH(k_corr_mark, dim3(blocks_for(items, 256)), dim3(256), 0, s, agg, lp, out, in, ins_rank, arc_w,
                     ddeg, flist, ins_src, ins_dst, del_src, del_dst, ins_w, del_w, bm, c, direct);
}

int compact_blocks(long long n) {
  const long long words = (n + 31) / 32;
  return static_cast<int>((words + kWordsPerBlock - 1) / kWordsPerBlock);
}

long long bucket_counter_slots(long long n) { return static_cast<long long>(compact_blocks(n)) * kWordsPerBlock * 32; }

void launch_compact(hipStream_t s, long long n, unsigned *bm_a, unsigned *bm_b, const CompactScratch &cs,
                    const CompactOut &o) {
  const long long words = (n + 31) / 32;
  const int tiles = compact_blocks(n);
  RP_LAUNCH(k_compact, dim3(tiles), dim3(kCompactThreads), 0, s, bm_a, bm_b, words, o, cs.words,
                     cs.words + static_cast<long long>(tiles) * kVals, cs.words + 2LL * tiles * kVals, cs.err);
}

void launch_delta0(hipStream_t s, long long n, const Delta0Args &z, const int *list, const u64 *count) {
  RP_LAUNCH(k_delta0, dim3(blocks_for(n * kWave, 256, 2048)), dim3(256), 0, s, z, list, count, n);
}

long long compact_scratch_words(long long n) { return 2LL * compact_blocks(n) * kVals + 1; }

void launch_scatter(hipStream_t s, long long n, int d, int ld, const int *list, const u64 *count, const long long *doff,
                    const float *delta, Adj out, float *S, unsigned *bm_out, unsigned *bm_x, const int *ins_dst,
                    const int *del_dst, const u64 *pushed, const Counters *c, bool push, bool mark_list,
                    const ScatterCopy &copy, const ScatterList &lo, bool packed_in) {
  const int blocks = 2048;
#define RP_SCATTER_L(GV, NCV, P, LV)                                                                               \
  RP_LAUNCH((k_scatter<GV, NCV, P, LV>), dim3(blocks), dim3(256), 0, s, d, ld, list, count, doff, delta, out, \
                     S, bm_out, bm_x, ins_dst, del_dst, pushed, c, mark_list ? 1 : 0, copy, lo, packed_in ? 1 : 0)
#define RP_SCATTER(GV, NCV, P)                \
  do {                                        \
    if (P && lo.list != nullptr)              \
      RP_SCATTER_L(GV, NCV, P, P);            \
    else                                      \
      RP_SCATTER_L(GV, NCV, P, false);        \
  } while (0)
  if (!push) RP_SCATTER(64, 1, false);
  else if (d <= 16) RP_SCATTER(16, 1, true);
  else if (d <= 32) RP_SCATTER(32, 1, true);
  else if (d <= 64) RP_SCATTER(64, 1, true);
  else if (d <= 128) RP_SCATTER(64, 2, true);
  else if (d <= 256) RP_SCATTER(64, 4, true);
  else if (d <= 512) RP_SCATTER(64, 8, true);
  else RP_SCATTER(64, 16, true);
#undef RP_SCATTER
#undef RP_SCATTER_L
}

int bin_shift(long long n) {
  // bins of 8192 sinks (few enough bins that the scatter's runs into them combine
  // in L2), at most kMaxBins of them
  const int s = 13;
  return (n + (1LL << s) - 1) >> s <= kMaxBins ? s : -1;
}

void launch_bin_count(hipStream_t s, const int *list, const u64 *count, const long long *doff, Adj out,
                      const u64 *pushed, const Buckets &b, unsigned *bm_x, const int *ins_dst, const int *del_dst,
                      bool mark_list, const Counters *c) {
  RP_LAUNCH(k_bin_arcs<false>, dim3(kBinBlocks), dim3(kBinThreads), b.nbins * sizeof(int), s, list, count, doff, out,
            pushed, b, bm_x, ins_dst, del_dst, mark_list ? 1 : 0, c);
}

void launch_bin_scatter(hipStream_t s, const int *list, const u64 *count, const long long *doff, Adj out,
                        const u64 *pushed, const Buckets &b, const Counters *c) {
  RP_LAUNCH(k_bin_arcs<true>, dim3(kBinBlocks), dim3(kBinThreads), b.nbins * sizeof(int), s, list, count, doff, out,
            pushed, b, nullptr, nullptr, nullptr, 0, c);
}

void launch_bin_sort(hipStream_t s, long long n, const u64 *pushed, const Buckets &b, const Counters *c) {
  RP_LAUNCH(k_bin_sort, dim3(static_cast<unsigned>(b.nbins)), dim3(kBinThreads), (sizeof(int) << b.shift), s, n,
            pushed, b, c);
}

void launch_pull_msgs(hipStream_t s, long long n, int d, int ld, const int *list, const u64 *count,
                      const long long *ioff, Adj in, const uint2 *memb, const float *msg,
                      float *S, unsigned *mark, const Counters *c) {
  const int blocks = 2048;
#define RP_PULLM(GV, NCV, UV)                                                                                    \
  RP_LAUNCH((k_pull_msgs<GV, NCV, UV>), dim3(blocks), dim3(256), 0, s, d, ld, list, count, ioff, in, \
                     memb, msg, S, mark, c)
  if (d <= 16) RP_PULLM(16, 1, 8);
  else if (d <= 32) RP_PULLM(16, 2, 8);
  else if (d <= 48) RP_PULLM(16, 3, 16);  // sixteen rows in flight: 3% faster on 47-wide rows (four waves per
                                          // SIMD instead of six); for 64-wide rows the registers cost more
                                          // (three waves, 5% slower)
  else if (d <= 64) RP_PULLM(16, 4, 8);
  else if (d <= 128) RP_PULLM(64, 2, 8);
  else if (d <= 256) RP_PULLM(64, 4, 8);
  else if (d <= 512) RP_PULLM(64, 8, 4);
  else RP_PULLM(64, 16, 2);
#undef RP_PULLM
}

// (G, NC, U) by row width: lane groups of 16 up to 64 columns, whole waves above
#define RP_BY_WIDTH(M)                                                                                         \
  do {                                                                                                         \
    if (d <= 16) M(16, 1, 8);                                                                                  \
    else if (d <= 32) M(16, 2, 8);                                                                             \
    else if (d <= 48) M(16, 3, 8);                                                                             \
    else if (d <= 64) M(16, 4, 8);                                                                             \
    else if (d <= 128) M(64, 2, 8);                                                                            \
    else if (d <= 256) M(64, 4, 8);                                                                            \
    else if (d <= 512) M(64, 8, 4);                                                                            \
    else M(64, 16, 2);                                                                                         \
  } while (0)

void launch_recompute(hipStream_t s, long long n, int d, int gcn, const int *list, const u64 *count,
                      const long long *ioff, Adj in, const int *out_len, const float *src, float *S, const Counters *c) {
  const int blocks = 2048;
#define RP_RECOMP(GV, NCV, UV)                                                                                   \
  RP_LAUNCH((k_recompute<GV, NCV, UV>), dim3(blocks), dim3(256), 0, s, d, gcn, list, count, ioff, in, out_len, \
            src, S, c)
  RP_BY_WIDTH(RP_RECOMP);
#undef RP_RECOMP
}

// Rows per step of the bucket sums: whole-wave groups (rows over 64 wide) take at
// most four, since a bucket holds a handful of slots and the masked rows of a step
// of eight reload a 1 KB row (1% on dense_large's 256-wide second layer); 16-lane
// groups keep eight (with four, buckets of 5-8 slots cost a second round trip).
constexpr int bucket_rows_per_step(int g, int u) { return g == kWave && u > 4 ? 4 : u; }

void launch_bucket_sum(hipStream_t s, int d, int ld, const int *list, const u64 *count, const long long *boff,
                       const Buckets &bk, const float *msg, float *S, const Counters *c) {
  const int blocks = 2048;
#define RP_BSUM(GV, NCV, UV)                                                                                     \
  RP_LAUNCH((k_bucket_sum<GV, NCV, bucket_rows_per_step(GV, UV)>), dim3(blocks), dim3(256), 0, s, d, ld, list,    \
            count, boff, bk, msg, S, c)
  RP_BY_WIDTH(RP_BSUM);
#undef RP_BSUM
}
#undef RP_BY_WIDTH

void launch_pull(hipStream_t s, long long n, int d, int agg, const float *Hprev, Adj in, const int *out_len,
                 float *S) {
  const int blocks = blocks_for(n * kWave, 256, 8192);
  const int nc = (d + kWave - 1) / kWave;
#define RP_PULL(NCV) RP_LAUNCH(k_pull<NCV>, dim3(blocks), dim3(256), 0, s, n, d, agg, Hprev, in, out_len, S)
  if (nc <= 1) RP_PULL(1);
  else if (nc == 2) RP_PULL(2);
  else if (nc <= 4) RP_PULL(4);
  else if (nc <= 8) RP_PULL(8);
  else RP_PULL(16);
#undef RP_PULL
}

void launch_fill_i32(hipStream_t s, int *p, long long count, int value) {
  if (count <= 0) return;
  RP_LAUNCH(k_fill_i32, dim3(blocks_for(count, 256)), dim3(256), 0, s, p, count, value);
}

void launch_fill_u64(hipStream_t s, u64 *p, long long count, u64 value) {
  if (count <= 0) return;
  RP_LAUNCH(k_fill_u64, dim3(blocks_for(count, 256)), dim3(256), 0, s, p, count, value);
}

void launch_gather_rows(hipStream_t s, const float *src, int d, const int *ids, long long count, float *out) {
  if (count <= 0) return;
  RP_LAUNCH(k_gather_rows, dim3(blocks_for(count * d, 256)), dim3(256), 0, s, src, d, ids, count, out);
}

}  // namespace rp
