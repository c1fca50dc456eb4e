// Loss-side work of one local SGD step: split-K reduction with the bias, the
// softmax cross-entropy gradient (mean over the minibatch, Algorithm 1 in
// Sec. 3.1 scales the summed gradient by 1/B), and the hidden-layer error.
#include "internal.h"

namespace hav {

// Z[p][m][n] = sum_ks part[ks][p][m][n] + b_p[n] for m < M; rows M..Mp-1 = 0.
__global__ __launch_bounds__(256) void k_reduce_bias(const float* __restrict__ part, int KS,
                                                     const float* __restrict__ bias, int64_t w_pitch,
                                                     float* __restrict__ Z, int P, int M, int Mp, int N) {
  const int64_t per = (int64_t)Mp * N;
  const int64_t total = (int64_t)P * per;
  const int64_t stride = total;  // part is [KS][P][Mp][N]
  for (int64_t e = blockIdx.x * 256ll + threadIdx.x; e < total; e += (int64_t)gridDim.x * 256) {
    const int p = (int)(e / per);
    const int64_t r = e - (int64_t)p * per;
    const int m = (int)(r / N), n = (int)(r % N);
    float v = 0.0f;
    if (m < M) {
      for (int ks = 0; ks < KS; ++ks) v += part[ks * stride + e];
      v += bias[(int64_t)p * w_pitch + n];
    }
    Z[e] = v;
  }
}

__device__ inline float wave_max(float v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v = fmaxf(v, __shfl_xor(v, o, 64));
  return v;
}
__device__ inline float wave_sum(float v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, 64);
  return v;
}

// One wave per (learner p, sample m < M): logits l_c = sum_ks part + b_c for
// c < C, G[c] = (softmax(l)_c - [c == y]) / M.  Columns C..Cp-1 stay zero.
__global__ __launch_bounds__(256) void k_softmax_grad(const float* __restrict__ part, int KS,
                                                      const float* __restrict__ bias, int64_t w_pitch,
                                                      const int32_t* __restrict__ labels,
                                                      const int32_t* __restrict__ idx, float* __restrict__ G,
                                                      int P, int M, int Mp, int C, int Cp) {
  const int row = blockIdx.x * 4 + (threadIdx.x >> 6);
  const int lane = threadIdx.x & 63;
  if (row >= P * M) return;
  const int p = row / M, m = row % M;
  const int64_t stride = (int64_t)P * Mp * Cp;
  const int64_t base = ((int64_t)p * Mp + m) * Cp;
  const float* b = bias + (int64_t)p * w_pitch;
  float* g = G + base;
  float mx = -INFINITY;
  for (int c = lane; c < C; c += 64) {
    float v = b[c];
    for (int ks = 0; ks < KS; ++ks) v += part[ks * stride + base + c];
    g[c] = v;
    mx = fmaxf(mx, v);
  }
  mx = wave_max(mx);
  float sum = 0.0f;
  for (int c = lane; c < C; c += 64) {
    const float e = expf(g[c] - mx);
    g[c] = e;
    sum += e;
  }
  sum = wave_sum(sum);
  const int y = labels[idx[(int64_t)p * M + m]];
  const float invB = 1.0f / (float)M;
  for (int c = lane; c < C; c += 64) g[c] = (g[c] / sum - (c == y ? 1.0f : 0.0f)) * invB;
}

// G1[p][m][h] = (sum_{c<C} G2[p][m][c] * W2_p[c][h]) * [Z1[p][m][h] > 0] for
// m < M; one thread per hidden unit h, 16 samples at a time, G2 staged in LDS.
__global__ __launch_bounds__(256) void k_bwd_hidden(const float* __restrict__ G2, const float* __restrict__ W2,
                                                    int64_t w_pitch, const float* __restrict__ Z1,
                                                    float* __restrict__ G1, int M, int Mp, int C, int Cp, int Hp,
                                                    int htiles) {
  constexpr int MC = 16, CC = 64;
  __shared__ float gs[MC][CC];
  const int p = blockIdx.x / htiles;
  const int h = (blockIdx.x % htiles) * 256 + threadIdx.x;
  const bool hok = h < Hp;
  const float* w2 = W2 + (int64_t)p * w_pitch;
  const float* g2 = G2 + (int64_t)p * Mp * Cp;
  for (int m0 = 0; m0 < M; m0 += MC) {
    float acc[MC];
#pragma unroll
    for (int i = 0; i < MC; ++i) acc[i] = 0.0f;
    for (int c0 = 0; c0 < C; c0 += CC) {
      __syncthreads();
      for (int e = threadIdx.x; e < MC * CC; e += 256) {
        const int mm = e / CC, cc = e % CC;
        gs[mm][cc] = (m0 + mm < M && c0 + cc < C) ? g2[(int64_t)(m0 + mm) * Cp + c0 + cc] : 0.0f;
      }
      __syncthreads();
      if (hok) {
        const int cn = min(CC, C - c0);
        for (int cc = 0; cc < cn; ++cc) {
          const float w = w2[(int64_t)(c0 + cc) * Hp + h];
#pragma unroll
          for (int i = 0; i < MC; ++i) acc[i] += gs[i][cc] * w;
        }
      }
    }
    if (hok) {
#pragma unroll
      for (int i = 0; i < MC; ++i) {
        const int m = m0 + i;
        if (m < M) {
          const int64_t o = ((int64_t)p * Mp + m) * Hp + h;
          G1[o] = Z1[o] > 0.0f ? acc[i] : 0.0f;
        }
      }
    }
  }
}

static int grid_cap(int64_t n, int cap) {
  int64_t g = (n + 255) / 256;
  return (int)(g < 1 ? 1 : (g < cap ? g : cap));
}

void launch_reduce_bias(hipStream_t s, const float* part, int KS, const float* bias, int64_t w_pitch, float* Z,
                        int P, int M, int Mp, int N) {
  k_reduce_bias<<<grid_cap((int64_t)P * Mp * N, 4096), 256, 0, s>>>(part, KS, bias, w_pitch, Z, P, M, Mp, N);
}

void launch_softmax_grad(hipStream_t s, const float* part, int KS, const float* bias, int64_t w_pitch,
                         const int32_t* labels, const int32_t* idx, float* G, int P, int M, int Mp, int C,
                         int Cp) {
  const int rows = P * M;
  k_softmax_grad<<<(rows + 3) / 4, 256, 0, s>>>(part, KS, bias, w_pitch, labels, idx, G, P, M, Mp, C, Cp);
}

void launch_bwd_hidden(hipStream_t s, const float* G2, const float* W2, int64_t w_pitch, const float* Z1,
                       float* G1, int P, int M, int Mp, int C, int Cp, int Hp) {
  const int htiles = (Hp + 255) / 256;
  k_bwd_hidden<<<P * htiles, 256, 0, s>>>(G2, W2, w_pitch, Z1, G1, M, Mp, C, Cp, Hp, htiles);
}

}  // namespace hav
