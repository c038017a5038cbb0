// Layer transform on the affected rows: Y = act(Z W^T + b) with fp32 MFMA
// (v_mfma_f32_16x16x4_f32), where Z is gathered on the fly from the cached
// aggregate and the previous layer's embeddings (Eq. (2): Update^l then sigma).
//
// Block tile 64 x 64 over (rows of the affected list) x (output columns), K in
// steps of 16 staged through LDS; four waves each own a 32 x 32 quarter as 2 x 2
// MFMA tiles. The epilogue adds the bias, applies ReLU, forms the next layer's
// delta row (new minus old contribution) and overwrites the embedding row.
// Tiles are visited by a grid-stride loop so that the row count can stay on the
// device.
#include "internal.h"

namespace rp {

namespace {

typedef float floatx4 __attribute__((ext_vector_type(4)));

constexpr int kBM = 64;
constexpr int kBN = 64;
constexpr int kBK = 16;
constexpr int kThreads = 256;

template <int AGG>
__global__ __launch_bounds__(kThreads) void k_gemm_f32(GemmArgs a) {
  if (a.abort != nullptr && *a.abort) return;
  const long long M = a.count != nullptr ? static_cast<long long>(*a.count) : a.count_fixed;
  const int N = a.N, K = a.K, dp = a.dprev;
  const long long tiles_n = (N + kBN - 1) / kBN;
  const long long tiles = ((M + kBM - 1) / kBM) * tiles_n;

  __shared__ float As[kBK][kBM + 4];  // As[k][m] = Z[m0+m][k0+k]
  __shared__ float Bs[kBK][kBN + 4];  // Bs[k][n] = W[n0+n][k0+k]
  __shared__ int rv[kBM];             // vertex of each tile row, -1 past M
  __shared__ float rt[kBM];           // aggregate scale t_v
  __shared__ float rs[kBM];           // GCN self coefficient s_v (post-batch)

  const int tid = threadIdx.x;
  const int lane = tid & (kWave - 1);
  const int wave = tid / kWave;
  const int wm = (wave >> 1) * 32;
  const int wn = (wave & 1) * 32;

  for (long long t = blockIdx.x; t < tiles; t += gridDim.x) {
    const long long m0 = (t / tiles_n) * kBM;
    const int n0 = static_cast<int>(t % tiles_n) * kBN;
    __syncthreads();
    if (tid < kBM) {
      const long long r = m0 + tid;
      int v = -1;
      float tv = 0.0f, sv = 0.0f;
      if (r < M) {
        v = a.rows != nullptr ? a.rows[r] : static_cast<int>(r);
        if (AGG == kMean) {
          const int din = a.in_len[v];
          tv = din > 0 ? 1.0f / static_cast<float>(din) : 0.0f;
        } else if (AGG == kGcn) {
          tv = 1.0f / sqrtf(static_cast<float>(a.in_len[v]) + 1.0f);
          sv = 1.0f / sqrtf(static_cast<float>(a.out_len[v]) + 1.0f);
        } else {
          tv = 1.0f;
        }
      }
      rv[tid] = v;
      rt[tid] = tv;
      rs[tid] = sv;
    }
    floatx4 acc[2][2];
#pragma unroll
    for (int i = 0; i < 2; ++i)
#pragma unroll
      for (int j = 0; j < 2; ++j) acc[i][j] = floatx4{0.0f, 0.0f, 0.0f, 0.0f};

    for (int k0 = 0; k0 < K; k0 += kBK) {
      __syncthreads();
      {
        const int m = tid >> 2;
        const int kb = (tid & 3) * 4;
        const int v = rv[m];
        const long long rowoff = static_cast<long long>(v) * dp;
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const int k = k0 + kb + i;
          float val = 0.0f;
          if (v >= 0 && k < K) {
            if (AGG == kGcn) {
              val = rt[m] * (a.S[rowoff + k] + rs[m] * a.Hprev[rowoff + k]);
            } else {
              val = k < dp ? a.Hprev[rowoff + k] : rt[m] * a.S[rowoff + (k - dp)];
            }
          }
          As[kb + i][m] = val;
        }
      }
      {
        const int nn = tid >> 2;
        const int kb = (tid & 3) * 4;
        const int col = n0 + nn;
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const int k = k0 + kb + i;
          Bs[kb + i][nn] = (col < N && k < K) ? a.W[static_cast<long long>(col) * K + k] : 0.0f;
        }
      }
      __syncthreads();
#pragma unroll
      for (int kk = 0; kk < kBK; kk += 4) {
        const int kr = kk + (lane >> 4);
        float av[2], bv[2];
#pragma unroll
        for (int i = 0; i < 2; ++i) av[i] = As[kr][wm + i * 16 + (lane & 15)];
#pragma unroll
        for (int j = 0; j < 2; ++j) bv[j] = Bs[kr][wn + j * 16 + (lane & 15)];
#pragma unroll
        for (int i = 0; i < 2; ++i)
#pragma unroll
          for (int j = 0; j < 2; ++j)
            acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x4f32(av[i], bv[j], acc[i][j], 0, 0, 0);
      }
    }
    // epilogue: lane holds C[4*(lane/16) + r][lane % 16] of each 16 x 16 tile
#pragma unroll
    for (int i = 0; i < 2; ++i) {
#pragma unroll
      for (int j = 0; j < 2; ++j) {
        const int col = n0 + wn + j * 16 + (lane & 15);
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const int ml = wm + i * 16 + (lane >> 4) * 4 + r;
          const int v = rv[ml];
          if (v < 0 || col >= N) continue;
          float y = acc[i][j][r] + (a.bias != nullptr ? a.bias[col] : 0.0f);
          if (a.relu) y = fmaxf(y, 0.0f);
          float *hp = a.H + static_cast<long long>(v) * N + col;
          if (a.delta != nullptr) {
            float cn = 1.0f, co = 1.0f;
            if (AGG == kGcn) {
              cn = rs[ml];
              co = 1.0f / sqrtf(static_cast<float>(a.out_len[v] - a.ddeg[v]) + 1.0f);
            }
            a.delta[(m0 + ml) * N + col] = cn * y - co * (*hp);
          }
          *hp = y;
        }
      }
    }
  }
}

}  // namespace

void launch_gemm(hipStream_t s, const GemmArgs &a, long long max_rows) {
  const long long tiles = ((max_rows + kBM - 1) / kBM) * ((a.N + kBN - 1) / kBN);
  long long blocks = tiles < 1 ? 1 : tiles;
  if (blocks > 2048) blocks = 2048;
  switch (a.agg) {
    case kMean:
      hipLaunchKernelGGL(k_gemm_f32<kMean>, dim3(blocks), dim3(kThreads), 0, s, a);
      break;
    case kGcn:
      hipLaunchKernelGGL(k_gemm_f32<kGcn>, dim3(blocks), dim3(kThreads), 0, s, a);
      break;
    default:
      hipLaunchKernelGGL(k_gemm_f32<kSum>, dim3(blocks), dim3(kThreads), 0, s, a);
      break;
  }
}

}  // namespace rp
