// Layer transform on the affected rows: Y = act(Z W^T + b) with fp32 MFMA
// (v_mfma_f32_16x16x4_f32), where each row of Z is gathered on the fly from the
// cached aggregate and the previous layer's embeddings (Eq. (2): Update^l then
// sigma). SAGE: z_v = [h_v || t_v S_v]; GCN: z_v = t_v (S_v + s_v h_v).
//
// A block of four waves owns a BM x BN output tile and walks K in steps of 32:
// the next step's A (gathered rows) and B (weight rows) are loaded into registers
// as float4 while the current step's MFMAs run from LDS, then stored into the
// other half of a double buffer, so there is one barrier per K step. Tiles are
// visited by a grid-stride loop so the row count can stay on the device. BN
// follows the layer width (16, 32, 48, 64, 128). Short row lists (the common
// case for small batches) go to a 16-row kernel that loads operands straight
// into registers and is bound by memory latency rather than throughput.
// The epilogue adds the bias, applies ReLU, forms the next layer's delta row
// (c'_v y - c_v h_old) and overwrites the embedding row.
//
// Modes. kLayer: Z = [h_v || t_v S_v] (SAGE) or t_v (S_v + s_v h_v) (GCN).
// kTransformFirst: the layer caches T_v = W_neigh S_v (width N) instead of S_v,
// Z is h_v (K = d_{l-1}) against W_self (SAGE) or W (GCN), and the epilogue adds
// the cached part: y = Z W_self^T + t_v T_v (SAGE) or y = t_v (T_v + s_v Z W^T)
// (GCN). kPlain: y = h_v W^T with no bias or activation; used for the rows
// P_v = W_neigh h_v that a transform-first layer caches, and its messages
// c'_v P'_v - c_v P_v formed by the same epilogue as the layer deltas.
// GraphConv (no self term): kLayer with z_v = t_v S_v (t = 1, or 1/d_in for the
// mean). GIN: kGin1 forms z_v = S_v + (1 + eps) h_v and writes ReLU(z W1^T + b1)
// to a buffer row per list position; kGin2 reads those rows as its operand and
// finishes with W2, b2 and the kLayer epilogue (the MLP of GINConv).
#include "internal.h"

namespace rp {

namespace {

typedef float floatx4 __attribute__((ext_vector_type(4)));
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));

// bf16 transforms use v_mfma_f32_16x16x32_bf16: per lane eight consecutive k
// values of its A row and of its B column, the same eight on both sides (the
// product is a sum over k, so which eight a lane holds does not matter as long as
// A and B agree); the 16 x 16 fp32 result has the layout of the fp32 MFMA's.
__device__ inline bf16x4 to_bf16(float4 x) {
  bf16x4 r;
  r[0] = static_cast<__bf16>(x.x);  // v_cvt_pk_bf16_f32: round to nearest even
  r[1] = static_cast<__bf16>(x.y);
  r[2] = static_cast<__bf16>(x.z);
  r[3] = static_cast<__bf16>(x.w);
  return r;
}

constexpr int kBK = 32;
constexpr int kLdk = kBK + 4;  // LDS row stride (floats)
constexpr int kThreads = 256;

template <int BM, int BN, int WM, int WN>
struct Shape {
  static constexpr int kWavesM = BM / (16 * WM);
  static constexpr int kWavesN = BN / (16 * WN);
  static_assert(kWavesM * kWavesN == 4, "four waves per block");
  static constexpr int kAChunks = BM * (kBK / 4);  // float4 chunks per A tile
  static constexpr int kBChunks = BN * (kBK / 4);
  static constexpr int kAPer = (kAChunks + kThreads - 1) / kThreads;
  static constexpr int kBPer = (kBChunks + kThreads - 1) / kThreads;
};

// True when Z = t (S + s h) with K = dprev: GCN (t, s from degrees) and GIN's
// first GEMM (t = 1, s = 1 + eps).
template <int AGG, int MODE>
__device__ constexpr bool sum_form() {
  return (MODE == kLayer && AGG == kGcn) || MODE == kGin1;
}
// True when Z = t S with K = dprev (GraphConv).
template <int AGG, int MODE>
__device__ constexpr bool neigh_only() {
  return MODE == kLayer && (AGG == kGcSum || AGG == kGcMean);
}

// Operand row v (kGin2: list position v), columns k .. k+3.
template <int AGG, bool VEC, int MODE>
__device__ inline float4 load_a(const GemmArgs &a, long long v, float tv, float sv, int k) {
  float4 r = make_float4(0.f, 0.f, 0.f, 0.f);
  if (v < 0 || k >= a.K) return r;
  const int dp = a.dprev;
  const long long base = v * dp;
  if (neigh_only<AGG, MODE>()) {
    if (VEC) {
      const float4 q = *reinterpret_cast<const float4 *>(a.S + base + k);
      return make_float4(tv * q.x, tv * q.y, tv * q.z, tv * q.w);
    }
    float t[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) t[i] = k + i < a.K ? tv * a.S[base + k + i] : 0.f;
    return make_float4(t[0], t[1], t[2], t[3]);
  }
  if (MODE != kLayer && MODE != kGin1) {  // plain rows of the previous layer (K == dprev)
    if (VEC) return *reinterpret_cast<const float4 *>(a.Hprev + base + k);
    float t[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) t[i] = k + i < a.K ? a.Hprev[base + k + i] : 0.f;
    return make_float4(t[0], t[1], t[2], t[3]);
  }
  if (VEC) {
    if (sum_form<AGG, MODE>()) {
      const float4 s = *reinterpret_cast<const float4 *>(a.S + base + k);
      const float4 h = *reinterpret_cast<const float4 *>(a.Hprev + base + k);
      r = make_float4(tv * (s.x + sv * h.x), tv * (s.y + sv * h.y), tv * (s.z + sv * h.z), tv * (s.w + sv * h.w));
    } else if (k < dp) {
      r = *reinterpret_cast<const float4 *>(a.Hprev + base + k);
    } else {
      const float4 s = *reinterpret_cast<const float4 *>(a.S + base + (k - dp));
      r = make_float4(tv * s.x, tv * s.y, tv * s.z, tv * s.w);
    }
    return r;
  }
  float t[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int kk = k + i;
    float val = 0.f;
    if (kk < a.K) {
      if (sum_form<AGG, MODE>()) {
        val = tv * (a.S[base + kk] + sv * a.Hprev[base + kk]);
      } else {
        val = kk < dp ? a.Hprev[base + kk] : tv * a.S[base + (kk - dp)];
      }
    }
    t[i] = val;
  }
  return make_float4(t[0], t[1], t[2], t[3]);
}

template <bool VEC>
__device__ inline float4 load_b(const GemmArgs &a, int col, int k) {
  if (col >= a.N || k >= a.K) return make_float4(0.f, 0.f, 0.f, 0.f);
  const float *w = a.W + static_cast<long long>(col) * a.K + k;
  if (VEC) return *reinterpret_cast<const float4 *>(w);
  float t[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) t[i] = k + i < a.K ? w[i] : 0.f;
  return make_float4(t[0], t[1], t[2], t[3]);
}

// The raw operand data of one float4 chunk (columns k .. k+3) of A row v (kGin2: a
// list position), fetched without a branch so that every load of a round is in
// flight together: a row past the count (v < 0) reads row 0 and a chunk past K the
// last chunk; finish_a drops them and applies the row's scales. x holds the S part
// or the plain row, h the previous layer's row of a sum form. (Widths are multiples
// of 4 here, so no chunk straddles h and S.)
struct AChunk {
  float4 x, h;
};

template <int AGG, int MODE>
__device__ inline AChunk fetch_a(const GemmArgs &a, long long v, int k) {
  const long long base = (v < 0 ? 0 : v) * a.dprev;
  const int kk = k < a.K ? k : a.K - 4;
  AChunk c;
  c.h = make_float4(0.f, 0.f, 0.f, 0.f);
  if (neigh_only<AGG, MODE>()) {
    c.x = *reinterpret_cast<const float4 *>(a.S + base + kk);
  } else if (MODE != kLayer && MODE != kGin1) {
    c.x = *reinterpret_cast<const float4 *>(a.Hprev + base + kk);
  } else if (sum_form<AGG, MODE>()) {
    c.x = *reinterpret_cast<const float4 *>(a.S + base + kk);
    c.h = *reinterpret_cast<const float4 *>(a.Hprev + base + kk);
  } else {
    const float *p = kk < a.dprev ? a.Hprev + base + kk : a.S + base + (kk - a.dprev);
    c.x = *reinterpret_cast<const float4 *>(p);
  }
  return c;
}

template <int AGG, int MODE>
__device__ inline float4 finish_a(const GemmArgs &a, const AChunk &c, bool valid, float tv, float sv, int k) {
  if (!valid || k >= a.K) return make_float4(0.f, 0.f, 0.f, 0.f);
  if (neigh_only<AGG, MODE>() || (MODE == kLayer && !sum_form<AGG, MODE>() && k >= a.dprev))
    return make_float4(tv * c.x.x, tv * c.x.y, tv * c.x.z, tv * c.x.w);
  if (sum_form<AGG, MODE>())
    return make_float4(tv * (c.x.x + sv * c.h.x), tv * (c.x.y + sv * c.h.y), tv * (c.x.z + sv * c.h.z),
                       tv * (c.x.w + sv * c.h.w));
  return c.x;
}

// W row `col`, columns k .. k+3, fetched without a branch (a column past N reads
// the last row and a chunk past K the last chunk; finish_b drops them).
__device__ inline float4 fetch_b(const GemmArgs &a, int col, int k) {
  const int cc = col < a.N ? col : a.N - 1;
  const int kk = k < a.K ? k : a.K - 4;
  return *reinterpret_cast<const float4 *>(a.W + static_cast<long long>(cc) * a.K + kk);
}

__device__ inline float4 finish_b(const GemmArgs &a, float4 b, int col, int k) {
  return col < a.N && k < a.K ? b : make_float4(0.f, 0.f, 0.f, 0.f);
}

// The same four weights in bf16 (raw bits, 8 bytes).
__device__ inline uint2 fetch_b_bf(const GemmArgs &a, int col, int k) {
  const int cc = col < a.N ? col : a.N - 1;
  const int kk = k < a.K ? k : a.K - 4;
  return *reinterpret_cast<const uint2 *>(a.Wb + static_cast<long long>(cc) * a.K + kk);
}

__device__ inline uint2 finish_b_bf(const GemmArgs &a, uint2 b, int col, int k) {
  return col < a.N && k < a.K ? b : make_uint2(0u, 0u);
}

// Bias, cached transformed aggregate (kTransformFirst), activation, delta and write-back for
// output element (row slot m with vertex v, column col).
template <int AGG, int MODE>
__device__ inline void epilogue(const GemmArgs &a, long long m, int v, int col, float y, float tv, float sv) {
  const int N = a.N;
  if (MODE == kTransformFirst) {
    const float Tv = a.S[static_cast<long long>(v) * N + col];
    y = AGG == kGcn ? tv * (Tv + sv * y) : y + tv * Tv;
  }
  y += a.bias != nullptr ? a.bias[col] : 0.f;
  if (a.relu) y = fmaxf(y, 0.f);
  float *hp = a.H + (MODE == kGin1 ? m : static_cast<long long>(v)) * N + col;
  if (MODE != kGin1 && a.delta != nullptr) {
    float cn = 1.f, co = 1.f;
    if (AGG == kGcn) {
      cn = sv;
      co = 1.0f / sqrtf(static_cast<float>(a.out_len[v] - a.ddeg[v]) + 1.0f);
    }
    a.delta[m * a.dld + col] = cn * y - co * (*hp);
  }
  *hp = y;
}

// Reads the abort flag and the row count (batch launches have both, bootstrap
// launches neither) in one round of loads, together with whatever loads produced
// `more` (non-negative values); true if the batch aborted.
template <typename... T>
__device__ inline bool abort_or_rows(const GemmArgs &a, long long &M, T... more) {
  if (a.abort != nullptr && a.count != nullptr) {
    const u64 ab = *a.abort;
    M = static_cast<long long>(*a.count >> a.count_shift);
    return aborted_with(ab, M, more...);
  }
  M = a.count_fixed;
  return a.abort != nullptr && *a.abort != 0;
}

// The epilogue for four consecutive columns col .. col+3 of row slot m (vertex v),
// all inside the layer (N % 4 == 0, so every row of H, S and delta is 16-byte
// aligned there): the scalar epilogue's arithmetic with float4 loads and stores.
template <int AGG, int MODE>
__device__ inline void epilogue4(const GemmArgs &a, long long m, int v, int col, float4 y, float tv, float sv) {
  const int N = a.N;
  float yy[4] = {y.x, y.y, y.z, y.w};
  if (MODE == kTransformFirst) {
    const float4 T = *reinterpret_cast<const float4 *>(a.S + static_cast<long long>(v) * N + col);
    const float tt[4] = {T.x, T.y, T.z, T.w};
#pragma unroll
    for (int i = 0; i < 4; ++i) yy[i] = AGG == kGcn ? tv * (tt[i] + sv * yy[i]) : yy[i] + tv * tt[i];
  }
  if (a.bias != nullptr) {
    const float4 b = *reinterpret_cast<const float4 *>(a.bias + col);
    yy[0] += b.x;
    yy[1] += b.y;
    yy[2] += b.z;
    yy[3] += b.w;
  }
  if (a.relu) {
#pragma unroll
    for (int i = 0; i < 4; ++i) yy[i] = fmaxf(yy[i], 0.f);
  }
  float4 *hp = reinterpret_cast<float4 *>(a.H + (MODE == kGin1 ? m : static_cast<long long>(v)) * N + col);
  if (MODE != kGin1 && a.delta != nullptr) {
    float cn = 1.f, co = 1.f;
    if (AGG == kGcn) {
      cn = sv;
      co = 1.0f / sqrtf(static_cast<float>(a.out_len[v] - a.ddeg[v]) + 1.0f);
    }
    const float4 o = *hp;
    *reinterpret_cast<float4 *>(a.delta + m * a.dld + col) =
        make_float4(cn * yy[0] - co * o.x, cn * yy[1] - co * o.y, cn * yy[2] - co * o.z, cn * yy[3] - co * o.w);
  }
  *hp = make_float4(yy[0], yy[1], yy[2], yy[3]);
}

// The launch's last a.cleanup_blocks blocks reset the batch's scratch instead of
// computing tiles (true for them); the others take tiles with stride gemm_grid.
__device__ inline bool cleanup_role(const GemmArgs &a, unsigned &gemm_grid) {
  gemm_grid = gridDim.x - static_cast<unsigned>(a.cleanup_blocks);
  if (blockIdx.x < gemm_grid) return false;
  const int b = static_cast<int>(blockIdx.x - gemm_grid);
  batch_cleanup(a.cleanup, b, static_cast<long long>(b) * blockDim.x + threadIdx.x,
                static_cast<long long>(a.cleanup_blocks) * blockDim.x);
  return true;
}

template <int BM, int BN, int WM, int WN, int AGG, bool VEC, int MODE, bool BF = false>
__global__ __launch_bounds__(kThreads) void k_gemm(GemmArgs a) {
  static_assert(!BF || VEC, "bf16 operands are gathered as float4 chunks");
  using Sh = Shape<BM, BN, WM, WN>;
  unsigned gemm_grid;
  if (cleanup_role(a, gemm_grid)) return;
  long long M;
  if (abort_or_rows(a, M)) return;
  const int N = a.N, K = a.K;
  const long long tiles_n = (N + BN - 1) / BN;
  const long long tiles = ((M + BM - 1) / BM) * tiles_n;

  // the double-buffered operand tiles, and after the K loop the output tile (row
  // stride BN + 4 floats keeps its rows 16-byte aligned), share one LDS block
  constexpr int kAsz = 2 * BM * kLdk, kBsz = 2 * BN * kLdk, kLdo = BN + 4;
  constexpr int kSmem = kAsz + kBsz > BM * kLdo ? kAsz + kBsz : BM * kLdo;
  __shared__ __attribute__((aligned(16))) float smem[kSmem];
  float(*As)[BM][kLdk] = reinterpret_cast<float(*)[BM][kLdk]>(smem);
  float(*Bs)[BN][kLdk] = reinterpret_cast<float(*)[BN][kLdk]>(smem + kAsz);
  // bf16 operand tiles in the same buffer: rows of kBK + 8 bf16 (80 bytes), so each
  // lane's eight k values are one aligned 16-byte read
  constexpr int kLdb = kBK + 8;
  unsigned short(*Ab)[BM][kLdb] = reinterpret_cast<unsigned short(*)[BM][kLdb]>(smem);
  unsigned short(*Bb)[BN][kLdb] = reinterpret_cast<unsigned short(*)[BN][kLdb]>(smem + kAsz);
  __shared__ int rv[BM];
  __shared__ float rt[BM];
  __shared__ float rs[BM];

  const int tid = threadIdx.x;
  const int lane = tid & (kWave - 1);
  const int wave = tid / kWave;
  const int wm0 = (wave / Sh::kWavesN) * (16 * WM);
  const int wn0 = (wave % Sh::kWavesN) * (16 * WN);
  const int lr = lane & 15;      // row (A) / column (B) within a 16-wide MFMA tile
  const int lk = lane >> 4;      // k within a 4-deep MFMA step

  for (long long t = blockIdx.x; t < tiles; t += gemm_grid) {
    const long long m0 = (t / tiles_n) * BM;
    const int n0 = static_cast<int>(t % tiles_n) * BN;
    __syncthreads();
    for (int r = tid; r < BM; r += kThreads) {
      const long long row = m0 + r;
      int v = -1;
      float tv = 0.f, sv = 0.f;
      if (row < M) {
        v = a.rows != nullptr ? a.rows[row] : static_cast<int>(row);
        if (AGG == kMean || AGG == kGcMean) {
          const int din = a.in_len[v];
          tv = din > 0 ? 1.0f / static_cast<float>(din) : 0.f;
        } else if (AGG == kGcn) {
          tv = 1.0f / sqrtf(static_cast<float>(a.in_len[v]) + 1.0f);
          sv = 1.0f / sqrtf(static_cast<float>(a.out_len[v]) + 1.0f);
        } else {
          tv = 1.0f;
          if (MODE == kGin1) sv = a.eps1;
        }
      }
      if (v >= 0 && n0 == 0 && a.clear_a != nullptr) {  // a scatter-built list's marks
        a.clear_a[v >> 5] = 0u;
        a.clear_b[v >> 5] = 0u;
      }
      rv[r] = v;
      rt[r] = tv;
      rs[r] = sv;
    }
    __syncthreads();

    // the next K step's operands: VEC kernels issue the raw loads here (no branch,
    // no arithmetic, so none of them waits) and finish the chunks (scales, dropped
    // rows and columns) when they are stored to LDS, after the current step's MFMAs
    float4 ra[Sh::kAPer], rb[Sh::kBPer];
    uint2 rbb[Sh::kBPer];
    AChunk rc[Sh::kAPer];
    int kload = 0;
    auto load_regs = [&](int k0) {
      kload = k0;
#pragma unroll
      for (int i = 0; i < Sh::kAPer; ++i) {
        const int c = tid + i * kThreads;
        if (c < Sh::kAChunks) {
          const int m = c / (kBK / 4);
          const int q = c % (kBK / 4);
          const long long arow = MODE == kGin2 ? (rv[m] >= 0 ? m0 + m : -1) : rv[m];
          if (VEC) rc[i] = fetch_a<AGG, MODE>(a, arow, k0 + 4 * q);
          else ra[i] = load_a<AGG, VEC, MODE>(a, arow, rt[m], rs[m], k0 + 4 * q);
        }
      }
#pragma unroll
      for (int i = 0; i < Sh::kBPer; ++i) {
        const int c = tid + i * kThreads;
        if (c < Sh::kBChunks) {
          const int nn = c / (kBK / 4);
          const int q = c % (kBK / 4);
          if (BF) rbb[i] = fetch_b_bf(a, n0 + nn, k0 + 4 * q);
          else rb[i] = VEC ? fetch_b(a, n0 + nn, k0 + 4 * q) : load_b<VEC>(a, n0 + nn, k0 + 4 * q);
        }
      }
    };
    auto store_lds = [&](int buf) {
#pragma unroll
      for (int i = 0; i < Sh::kAPer; ++i) {
        const int c = tid + i * kThreads;
        if (c < Sh::kAChunks) {
          const int m = c / (kBK / 4);
          const int q = c % (kBK / 4);
          float4 x = ra[i];
          if (VEC) {
            const bool valid = MODE == kGin2 ? rv[m] >= 0 : rv[m] >= 0;
            x = finish_a<AGG, MODE>(a, rc[i], valid, rt[m], rs[m], kload + 4 * q);
          }
          if (BF) *reinterpret_cast<bf16x4 *>(&Ab[buf][m][4 * q]) = to_bf16(x);
          else *reinterpret_cast<float4 *>(&As[buf][m][4 * q]) = x;
        }
      }
#pragma unroll
      for (int i = 0; i < Sh::kBPer; ++i) {
        const int c = tid + i * kThreads;
        if (c < Sh::kBChunks) {
          const int nn = c / (kBK / 4);
          const int q = c % (kBK / 4);
          if (BF)
            *reinterpret_cast<uint2 *>(&Bb[buf][nn][4 * q]) = finish_b_bf(a, rbb[i], n0 + nn, kload + 4 * q);
          else
            *reinterpret_cast<float4 *>(&Bs[buf][nn][4 * q]) =
                VEC ? finish_b(a, rb[i], n0 + nn, kload + 4 * q) : rb[i];
        }
      }
    };

    floatx4 acc[WM][WN];
#pragma unroll
    for (int i = 0; i < WM; ++i)
#pragma unroll
      for (int j = 0; j < WN; ++j) acc[i][j] = floatx4{0.f, 0.f, 0.f, 0.f};

    load_regs(0);
    store_lds(0);
    __syncthreads();
    int buf = 0;
    for (int k0 = 0; k0 < K; k0 += kBK) {
      const bool more = k0 + kBK < K;
      if (more) load_regs(k0 + kBK);
      if constexpr (BF) {
        // the step's 32 k values in one MFMA per output tile: lane (r, q) holds k
        // values 8q .. 8q+7 of its A row and B column
        bf16x8 av[WM], bv[WN];
#pragma unroll
        for (int i = 0; i < WM; ++i) av[i] = *reinterpret_cast<const bf16x8 *>(&Ab[buf][wm0 + i * 16 + lr][8 * lk]);
#pragma unroll
        for (int j = 0; j < WN; ++j) bv[j] = *reinterpret_cast<const bf16x8 *>(&Bb[buf][wn0 + j * 16 + lr][8 * lk]);
#pragma unroll
        for (int i = 0; i < WM; ++i)
#pragma unroll
          for (int j = 0; j < WN; ++j)
            acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(av[i], bv[j], acc[i][j], 0, 0, 0);
      } else {
#pragma unroll
        for (int kk = 0; kk < kBK; kk += 4) {
          float av[WM], bv[WN];
#pragma unroll
          for (int i = 0; i < WM; ++i) av[i] = As[buf][wm0 + i * 16 + lr][kk + lk];
#pragma unroll
          for (int j = 0; j < WN; ++j) bv[j] = Bs[buf][wn0 + j * 16 + lr][kk + lk];
#pragma unroll
          for (int i = 0; i < WM; ++i)
#pragma unroll
            for (int j = 0; j < WN; ++j)
              acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x4f32(av[i], bv[j], acc[i][j], 0, 0, 0);
        }
      }
      if (more) store_lds(buf ^ 1);
      __syncthreads();
      buf ^= 1;
    }

    // epilogue: lane holds C[4*(lane/16) + r][lane % 16] of each 16 x 16 tile
    if (VEC && N % 4 == 0) {
      // through LDS, so that each row's outputs are read, written and loaded as
      // float4 runs of up to BN columns (the K loop's last barrier has released the
      // operand tiles)
#pragma unroll
      for (int i = 0; i < WM; ++i)
#pragma unroll
        for (int j = 0; j < WN; ++j)
#pragma unroll
          for (int r = 0; r < 4; ++r) smem[(wm0 + i * 16 + lk * 4 + r) * kLdo + wn0 + j * 16 + lr] = acc[i][j][r];
      __syncthreads();
      for (int q = tid; q < BM * (BN / 4); q += kThreads) {
        const int ml = q / (BN / 4), c4 = q % (BN / 4);
        const int col = n0 + 4 * c4;
        const int v = rv[ml];
        if (v < 0 || col >= N) continue;
        const float4 y = *reinterpret_cast<const float4 *>(&smem[ml * kLdo + 4 * c4]);
        epilogue4<AGG, MODE>(a, m0 + ml, v, col, y, rt[ml], rs[ml]);
      }
    } else {
#pragma unroll
      for (int i = 0; i < WM; ++i) {
#pragma unroll
        for (int j = 0; j < WN; ++j) {
          const int col = n0 + wn0 + j * 16 + lr;
#pragma unroll
          for (int r = 0; r < 4; ++r) {
            const int ml = wm0 + i * 16 + lk * 4 + r;
            const int v = rv[ml];
            if (v < 0 || col >= N) continue;
            epilogue<AGG, MODE>(a, m0 + ml, v, col, acc[i][j][r], rt[ml], rs[ml]);
          }
        }
      }
    }
  }
}

// Small-row-count variant, built for latency: a block owns a 16 x BN output tile
// and its W waves split K into W contiguous ranges. Every lane loads its
// operands straight from global memory into registers as float4: lane (r, q)
// holds A row r and B column r at k = 16 f + 4 q .. 16 f + 4 q + 3 of its range,
// and at MFMA sub-step i both operands give component i, the same permutation of
// k on both sides. A range of up to 64 (W = 8) or 128 (W = 4) k values thus costs one round of loads and
// no LDS staging. The epilogue's inputs (old embedding row, cached transform,
// degrees, bias) are fetched as soon as the row ids are known, together with the
// operands, so a tile takes three dependent rounds of memory access: row count,
// row ids, then everything else. The W partial tiles meet in LDS.
constexpr int kRowsBM = 16;
// Lists of up to this many expected rows take eight waves per tile (64 k values
// per wave per round: the MFMA chain of a wave is half as long); longer ones four
// (128 k values per round, twice the tiles per compute unit).
constexpr long long kRowsWideMax = 2048;

template <int BN, int AGG, int MODE, int W, bool BF = false>
__global__ __launch_bounds__(W * kWave) void k_gemm_rows(GemmArgs a) {
  constexpr int kRowsWaves = W;  // waves per tile, each on its own range of k
  constexpr int kRowsThreads = W * kWave;
  constexpr int kRowsKC = W == 8 ? 64 : 128;  // k values per wave per round of loads
  constexpr int WN = BN / 16;
  constexpr int kF = kRowsKC / 16;  // float4 per lane per operand row and round
  constexpr int kTile = kRowsBM * BN;
  constexpr int kEl = (kTile + kRowsThreads - 1) / kRowsThreads;  // output elements per thread (at most)
  unsigned gemm_grid;
  if (cleanup_role(a, gemm_grid)) return;
  const int N = a.N, K = a.K, dp = a.dprev;
  const long long tiles_n = (N + BN - 1) / BN;
  const int tid = threadIdx.x;
  const int lane = tid & (kWave - 1);
  const int wave = tid / kWave;
  const int lr = lane & 15;
  const int lq = lane >> 4;
  // row ids of tile t up to `limit`: the lane's operand row and the rows of its
  // output elements (-1 past the limit)
  int va, ve[kEl];
  const auto row_ids = [&](long long t, long long limit) {
    const long long m0 = (t / tiles_n) * kRowsBM;
    const long long ar = m0 + lr;
    va = ar < limit ? (a.rows != nullptr ? a.rows[ar] : static_cast<int>(ar)) : -1;
#pragma unroll
    for (int i = 0; i < kEl; ++i) {
      const int e = tid + i * kRowsThreads;
      const long long row = m0 + e / BN;
      ve[i] = e < kTile && row < limit ? (a.rows != nullptr ? a.rows[row] : static_cast<int>(row)) : -1;
    }
  };
  // The first tile's ids are fetched with the row count: the list holds max_rows
  // ids, so ids read past the count stay in bounds; they are dropped below.
  row_ids(blockIdx.x, a.max_rows);
  long long M;
  // (ids past the count may hold anything: they join the test as unsigned halves,
  // which are never negative)
  if (abort_or_rows(a, M, static_cast<unsigned>(va) >> 1, static_cast<unsigned>(ve[0]) >> 1)) return;
  const long long tiles = ((M + kRowsBM - 1) / kRowsBM) * tiles_n;

  __shared__ float red[kRowsWaves][kRowsBM][BN + 1];

  const int kw = (K + kRowsWaves * 16 - 1) / (kRowsWaves * 16) * 16;  // k values per wave, a multiple of 16
  const int kb = wave * kw;
  const int ke = K < kb + kw ? K : kb + kw;

  for (long long t = blockIdx.x; t < tiles; t += gemm_grid) {
    const long long m0 = (t / tiles_n) * kRowsBM;
    const int n0 = static_cast<int>(t % tiles_n) * BN;
    if (t == blockIdx.x) {  // the prefetched ids: drop those past the count
      if (m0 + lr >= M) va = -1;
#pragma unroll
      for (int i = 0; i < kEl; ++i)
        if (m0 + (tid + i * kRowsThreads) / BN >= M) ve[i] = -1;
    } else {
      row_ids(t, M);
    }
    const long long ar = m0 + lr;
    const long long arow = MODE == kGin2 ? (ar < M ? ar : -1) : va;  // operand row (kGin2: list position)
    if (va >= 0 && n0 == 0 && wave == 0 && lq == 0 && a.clear_a != nullptr) {  // a scatter-built list's marks
      a.clear_a[va >> 5] = 0u;
      a.clear_b[va >> 5] = 0u;
    }
    // operand-row scales (layer mode): mean t = 1/deg_in; GCN t = (deg_in+1)^-1/2,
    // s = (deg_out+1)^-1/2
    float ta = 1.f, sa = 0.f;
    if (MODE == kLayer && va >= 0) {
      if (AGG == kMean || AGG == kGcMean) {
        const int din = a.in_len[va];
        ta = din > 0 ? 1.0f / static_cast<float>(din) : 0.f;
      } else if (AGG == kGcn) {
        ta = 1.0f / sqrtf(static_cast<float>(a.in_len[va]) + 1.0f);
        sa = 1.0f / sqrtf(static_cast<float>(a.out_len[va]) + 1.0f);
      }
    }
    if (MODE == kGin1) sa = a.eps1;
    // epilogue inputs
    float e_old[kEl], e_t[kEl], e_tv[kEl], e_sv[kEl], e_co[kEl], e_b[kEl];
#pragma unroll
    for (int i = 0; i < kEl; ++i) {
      const int col = n0 + (tid + i * kRowsThreads) % BN;
      const int v = ve[i];
      e_old[i] = 0.f;
      e_t[i] = 0.f;
      e_tv[i] = 1.f;
      e_sv[i] = 0.f;
      e_co[i] = 1.f;
      e_b[i] = 0.f;
      if (v < 0 || col >= N) continue;
      const long long idx = static_cast<long long>(v) * N + col;
      if (MODE != kGin1 && a.delta != nullptr) e_old[i] = a.H[idx];
      if (a.bias != nullptr) e_b[i] = a.bias[col];
      if (MODE == kTransformFirst) {
        e_t[i] = a.S[idx];
        if (AGG == kMean) {
          const int din = a.in_len[v];
          e_tv[i] = din > 0 ? 1.0f / static_cast<float>(din) : 0.f;
        } else if (AGG == kGcn) {
          e_tv[i] = 1.0f / sqrtf(static_cast<float>(a.in_len[v]) + 1.0f);
        }
      }
      if (AGG == kGcn) {
        const int dout = a.out_len[v];
        e_sv[i] = 1.0f / sqrtf(static_cast<float>(dout) + 1.0f);
        e_co[i] = 1.0f / sqrtf(static_cast<float>(dout - a.ddeg[v]) + 1.0f);
      }
    }

    floatx4 acc[WN];
#pragma unroll
    for (int j = 0; j < WN; ++j) acc[j] = floatx4{0.f, 0.f, 0.f, 0.f};
    const long long abase = arow * dp;
    if constexpr (BF) {
      // bf16: per round each lane takes eight consecutive k values (two float4 of
      // its A row, each all h or all S since the widths are multiples of 4) and the
      // same eight weights of each B column, one MFMA per 32 k values and column tile
      for (int kc = kb; kc < ke; kc += kRowsKC) {
        constexpr int kG = kRowsKC / 32;
        float4 zh[kG][2], zs[kG][2];
        uint2 wb[WN][kG][2];
#pragma unroll
        for (int g = 0; g < kG; ++g)
#pragma unroll
          for (int hh = 0; hh < 2; ++hh) {
            const int k = kc + 32 * g + 8 * lq + 4 * hh;
            const bool ok = arow >= 0 && k < ke;
            float4 x = make_float4(0.f, 0.f, 0.f, 0.f), h = x;
            if (ok) {
              if (neigh_only<AGG, MODE>()) {
                x = *reinterpret_cast<const float4 *>(a.S + abase + k);
              } else if (sum_form<AGG, MODE>()) {
                x = *reinterpret_cast<const float4 *>(a.S + abase + k);
                h = *reinterpret_cast<const float4 *>(a.Hprev + abase + k);
              } else if (MODE != kLayer) {
                x = *reinterpret_cast<const float4 *>(a.Hprev + abase + k);
              } else {
                x = k < dp ? *reinterpret_cast<const float4 *>(a.Hprev + abase + k)
                           : *reinterpret_cast<const float4 *>(a.S + abase + (k - dp));
              }
            }
            zs[g][hh] = x;
            zh[g][hh] = h;
#pragma unroll
            for (int j = 0; j < WN; ++j) {
              const int col = n0 + 16 * j + lr;
              wb[j][g][hh] = col < N && k < ke
                                 ? *reinterpret_cast<const uint2 *>(a.Wb + static_cast<long long>(col) * K + k)
                                 : make_uint2(0u, 0u);
            }
          }
#pragma unroll
        for (int g = 0; g < kG; ++g) {
          if (kc + 32 * g >= ke) break;  // the wave's k range ends inside the round (uniform)
          float4 z[2];
#pragma unroll
          for (int hh = 0; hh < 2; ++hh) {
            const int k = kc + 32 * g + 8 * lq + 4 * hh;
            const float4 x = zs[g][hh], h = zh[g][hh];
            if (sum_form<AGG, MODE>() && ((MODE == kLayer && AGG != kSum && AGG != kGcSum) || MODE == kGin1))
              z[hh] = make_float4(ta * (x.x + sa * h.x), ta * (x.y + sa * h.y), ta * (x.z + sa * h.z),
                                  ta * (x.w + sa * h.w));
            else if (((MODE == kLayer && AGG != kSum && AGG != kGcSum) || MODE == kGin1) &&
                     (neigh_only<AGG, MODE>() || k >= dp))
              z[hh] = make_float4(ta * x.x, ta * x.y, ta * x.z, ta * x.w);
            else
              z[hh] = x;
          }
          const bf16x4 lo = to_bf16(z[0]), hi = to_bf16(z[1]);
          const bf16x8 a8 = {lo[0], lo[1], lo[2], lo[3], hi[0], hi[1], hi[2], hi[3]};
#pragma unroll
          for (int j = 0; j < WN; ++j) {
            const uint4 w4 = make_uint4(wb[j][g][0].x, wb[j][g][0].y, wb[j][g][1].x, wb[j][g][1].y);
            bf16x8 b8;
            __builtin_memcpy(&b8, &w4, sizeof(b8));
            acc[j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a8, b8, acc[j], 0, 0, 0);
          }
        }
      }
    } else
    for (int kc = kb; kc < ke; kc += kRowsKC) {
      float4 av[kF], ah[kF], bv[WN][kF];
#pragma unroll
      for (int f = 0; f < kF; ++f) {
        const int k = kc + 16 * f + 4 * lq;
        const bool ok = arow >= 0 && k < ke;
        float4 x = make_float4(0.f, 0.f, 0.f, 0.f), h = x;
        if (ok) {
          if (neigh_only<AGG, MODE>()) {  // K == dp: z = t S
            x = *reinterpret_cast<const float4 *>(a.S + abase + k);
          } else if (sum_form<AGG, MODE>()) {  // K == dp: z = t (S + s h)
            x = *reinterpret_cast<const float4 *>(a.S + abase + k);
            h = *reinterpret_cast<const float4 *>(a.Hprev + abase + k);
          } else if (MODE != kLayer) {  // plain rows (kGin2: the first GEMM's rows)
            x = *reinterpret_cast<const float4 *>(a.Hprev + abase + k);
          } else {  // z = [h || t S]
            x = k < dp ? *reinterpret_cast<const float4 *>(a.Hprev + abase + k)
                       : *reinterpret_cast<const float4 *>(a.S + abase + (k - dp));
          }
        }
        av[f] = x;
        ah[f] = h;
      }
#pragma unroll
      for (int j = 0; j < WN; ++j) {
        const int col = n0 + 16 * j + lr;
#pragma unroll
        for (int f = 0; f < kF; ++f) {
          const int k = kc + 16 * f + 4 * lq;
          bv[j][f] = col < N && k < ke ? *reinterpret_cast<const float4 *>(a.W + static_cast<long long>(col) * K + k)
                                       : make_float4(0.f, 0.f, 0.f, 0.f);
        }
      }
      if ((MODE == kLayer && AGG != kSum && AGG != kGcSum) || MODE == kGin1) {
#pragma unroll
        for (int f = 0; f < kF; ++f) {
          const int k = kc + 16 * f + 4 * lq;
          if (sum_form<AGG, MODE>()) {
            av[f] = make_float4(ta * (av[f].x + sa * ah[f].x), ta * (av[f].y + sa * ah[f].y),
                                ta * (av[f].z + sa * ah[f].z), ta * (av[f].w + sa * ah[f].w));
          } else if (neigh_only<AGG, MODE>() || k >= dp) {
            av[f] = make_float4(ta * av[f].x, ta * av[f].y, ta * av[f].z, ta * av[f].w);
          }
        }
      }
#pragma unroll
      for (int f = 0; f < kF; ++f) {
        if (kc + 16 * f >= ke) break;  // the wave's k range ends inside the round (uniform)
        const float ax[4] = {av[f].x, av[f].y, av[f].z, av[f].w};
#pragma unroll
        for (int j = 0; j < WN; ++j) {
          const float bx[4] = {bv[j][f].x, bv[j][f].y, bv[j][f].z, bv[j][f].w};
#pragma unroll
          for (int i = 0; i < 4; ++i) acc[j] = __builtin_amdgcn_mfma_f32_16x16x4f32(ax[i], bx[i], acc[j], 0, 0, 0);
        }
      }
    }
    // lane holds C[4 q + r][r'] of each 16 x 16 tile (q = lane / 16, r' = lane % 16)
#pragma unroll
    for (int j = 0; j < WN; ++j)
#pragma unroll
      for (int r = 0; r < 4; ++r) red[wave][lq * 4 + r][j * 16 + lr] = acc[j][r];
    __syncthreads();
#pragma unroll
    for (int i = 0; i < kEl; ++i) {
      const int e = tid + i * kRowsThreads;
      const int ml = e / BN, cl = e % BN;
      const int col = n0 + cl;
      const int v = ve[i];
      if (v < 0 || col >= N) continue;
      float y = 0.f;
#pragma unroll
      for (int w = 0; w < kRowsWaves; ++w) y += red[w][ml][cl];
      if (MODE == kTransformFirst) y = AGG == kGcn ? e_tv[i] * (e_t[i] + e_sv[i] * y) : y + e_tv[i] * e_t[i];
      y += e_b[i];
      if (a.relu) y = fmaxf(y, 0.f);
      const long long idx = (MODE == kGin1 ? m0 + ml : static_cast<long long>(v)) * N + col;
      if (MODE != kGin1 && a.delta != nullptr) {
        const float cn = AGG == kGcn ? e_sv[i] : 1.f;
        a.delta[(m0 + ml) * a.dld + col] = cn * y - e_co[i] * e_old[i];
      }
      a.H[idx] = y;
    }
    __syncthreads();  // red is reused by the next tile
  }
}

template <int BN, int AGG, int MODE>
void launch_rows(hipStream_t s, const GemmArgs &a, long long max_rows, bool wide) {
  const long long tiles = ((max_rows + kRowsBM - 1) / kRowsBM) * ((a.N + BN - 1) / BN);
  long long blocks = tiles < 1 ? 1 : tiles;
  if (blocks > 2048) blocks = 2048;
  const dim3 grid(static_cast<unsigned>(blocks + a.cleanup_blocks));
  if (a.bf16 && wide) RP_LAUNCH((k_gemm_rows<BN, AGG, MODE, 8, true>), grid, dim3(8 * kWave), 0, s, a);
  else if (a.bf16) RP_LAUNCH((k_gemm_rows<BN, AGG, MODE, 4, true>), grid, dim3(4 * kWave), 0, s, a);
  else if (wide) RP_LAUNCH((k_gemm_rows<BN, AGG, MODE, 8>), grid, dim3(8 * kWave), 0, s, a);
  else RP_LAUNCH((k_gemm_rows<BN, AGG, MODE, 4>), grid, dim3(4 * kWave), 0, s, a);
}

template <int BM, int BN, int WM, int WN, int AGG, bool VEC, int MODE>
void launch_shape(hipStream_t s, const GemmArgs &a, long long max_rows) {
  const long long tiles = ((max_rows + BM - 1) / BM) * ((a.N + BN - 1) / BN);
  long long blocks = tiles < 1 ? 1 : tiles;
  if (blocks > 2048) blocks = 2048;
  const dim3 grid(static_cast<unsigned>(blocks + a.cleanup_blocks));
  if constexpr (VEC) {
    if (a.bf16) {
      RP_LAUNCH((k_gemm<BM, BN, WM, WN, AGG, VEC, MODE, true>), grid, dim3(kThreads), 0, s, a);
      return;
    }
  }
  RP_LAUNCH((k_gemm<BM, BN, WM, WN, AGG, VEC, MODE>), grid, dim3(kThreads), 0, s, a);
}

// BN follows N. Few expected rows: the 16-row split-K kernel; many: 128-row tiles
// (variant: see gemm_variant).
template <int AGG, bool VEC, int MODE>
void launch_agg(hipStream_t s, const GemmArgs &a, long long max_rows, int variant) {
  const bool big = variant == 1, wide = variant == 0;
  const int N = a.N;
  if (!VEC) {
    if (N <= 16) launch_shape<64, 16, 1, 1, AGG, VEC, MODE>(s, a, max_rows);
    else if (N <= 32) launch_shape<64, 32, 2, 1, AGG, VEC, MODE>(s, a, max_rows);
    else if (N <= 48) launch_shape<64, 48, 1, 3, AGG, VEC, MODE>(s, a, max_rows);
    else if (N <= 64) launch_shape<32, 64, 1, 2, AGG, VEC, MODE>(s, a, max_rows);
    else launch_shape<32, 128, 2, 2, AGG, VEC, MODE>(s, a, max_rows);
    return;
  }
  if (!big) {
    if (N <= 16) launch_rows<16, AGG, MODE>(s, a, max_rows, wide);
    else if (N <= 32) launch_rows<32, AGG, MODE>(s, a, max_rows, wide);
    else if (N <= 48) launch_rows<48, AGG, MODE>(s, a, max_rows, wide);
    else launch_rows<64, AGG, MODE>(s, a, max_rows, wide);  // N > 64: several 64-wide column tiles
    return;
  }
  if (N <= 16) launch_shape<64, 16, 1, 1, AGG, VEC, MODE>(s, a, max_rows);
  else if (N <= 32) launch_shape<64, 32, 2, 1, AGG, VEC, MODE>(s, a, max_rows);
  else if (N <= 48) launch_shape<128, 48, 2, 3, AGG, VEC, MODE>(s, a, max_rows);
  else if (N <= 64) launch_shape<128, 64, 4, 2, AGG, VEC, MODE>(s, a, max_rows);
  else launch_shape<128, 128, 4, 4, AGG, VEC, MODE>(s, a, max_rows);
}

template <int AGG, int MODE>
void launch_vec(hipStream_t s, const GemmArgs &a, long long max_rows, int variant) {
  const bool vec = (a.dprev % 4 == 0) && (a.K % 4 == 0);
  if (vec) launch_agg<AGG, true, MODE>(s, a, max_rows, variant);
  else launch_agg<AGG, false, MODE>(s, a, max_rows, variant);
}

template <int MODE>
void launch_mode(hipStream_t s, const GemmArgs &a, long long max_rows, int variant) {
  if constexpr (MODE == kGin1 || MODE == kGin2) {
    launch_vec<kSum, MODE>(s, a, max_rows, variant);  // GIN sums with coefficient 1
  } else {
    switch (a.agg) {
      case kMean:
        launch_vec<kMean, MODE>(s, a, max_rows, variant);
        break;
      case kGcn:
        launch_vec<kGcn, MODE>(s, a, max_rows, variant);
        break;
      case kGcSum:
        if constexpr (MODE == kLayer) launch_vec<kGcSum, MODE>(s, a, max_rows, variant);
        break;
      case kGcMean:
        if constexpr (MODE == kLayer) launch_vec<kGcMean, MODE>(s, a, max_rows, variant);
        break;
      default:
        launch_vec<kSum, MODE>(s, a, max_rows, variant);
        break;
    }
  }
}

}  // namespace

int gemm_variant(long long expected_rows, int n_cols) {
  // 128-row tiles from 32768 expected rows, or from 8192 when the output is at least
  // 128 wide (the 3-layer mean workload's 256-wide middle layer at ~15K rows: 5%
  // faster at batch 1000; narrow layers lose by it, and from 4096 rows the tiles
  // left too many compute units idle at batch 100)
  const long long big = n_cols >= 128 ? 8192 : 32768;
  return expected_rows >= big ? 1 : expected_rows > kRowsWideMax ? 2 : 0;
}

int cleanup_blocks_for(long long cap_ops) {
  // up to 4 * cap_ops (arc, direction) items and cap_ops ops, grid-strided
  const long long b = (4 * cap_ops + kThreads - 1) / kThreads;
  return static_cast<int>(b < 1 ? 1 : b > 256 ? 256 : b);
}

void launch_gemm(hipStream_t s, const GemmArgs &args, long long max_rows, long long expected_rows) {
  GemmArgs a = args;
  a.max_rows = max_rows;
  const int variant = gemm_variant(expected_rows, a.N);
  if (a.mode == kTransformFirst) launch_mode<kTransformFirst>(s, a, max_rows, variant);
  else if (a.mode == kPlain) launch_mode<kPlain>(s, a, max_rows, variant);
  else if (a.mode == kGin1) launch_mode<kGin1>(s, a, max_rows, variant);
  else if (a.mode == kGin2) launch_mode<kGin2>(s, a, max_rows, variant);
  else launch_mode<kLayer>(s, a, max_rows, variant);
}

}  // namespace rp
