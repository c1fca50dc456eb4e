// Synthetic inputs, initial state and the minibatch index draw.
//
// Algorithm 1 (Sec. 3.1) has every learner draw a random minibatch of size B
// at every local step; Sec. 2 makes the draws i.i.d. across learners and
// steps.  Draws here are i.i.d. with replacement from a counter-based
// generator, so any implementation reproduces them bit for bit:
//   idx = H(k_index, t << 32 | j << 16 | s) mod N
// for sample s of learner j at global step t.
#include "internal.h"

namespace hav {

__global__ __launch_bounds__(256) void k_gen_labels(int32_t* __restrict__ y, int64_t N, uint64_t key, uint64_t C) {
  for (int64_t i = blockIdx.x * 256ll + threadIdx.x; i < N; i += (int64_t)gridDim.x * 256)
    y[i] = (int32_t)(hash64(key, (uint64_t)i) % C);
}

// One workgroup per dataset row i: X[i][d] = fp32(mu[y_i][d] + sigma * z_noise),
// computed as a single fused multiply-add (sigma * z is exact for the noise
// levels used, and the fused form rounds the exact sum once in any case).
__global__ __launch_bounds__(256) void k_gen_data(float* __restrict__ X, const int32_t* __restrict__ y, int64_t IN,
                                                  int64_t INp, uint64_t key_mean, uint64_t key_noise, float sigma) {
  const int64_t i = blockIdx.x;
  const uint64_t c = (uint64_t)y[i];
  float* row = X + i * INp;
  for (int64_t d = threadIdx.x; d < INp; d += 256) {
    float v = 0.0f;
    if (d < IN) {
      float mu = irwin_hall(key_mean, c * (uint64_t)IN + (uint64_t)d);
      float nz = irwin_hall(key_noise, (uint64_t)i * (uint64_t)IN + (uint64_t)d);
      v = __fmaf_rn(sigma, nz, mu);
    }
    row[d] = v;
  }
}

// Weight block [rows][cols] (leading dimension ld) of replica 0:
// (2u - 1) * scale, u = (H(key, layer << 48 | o*cols + i) >> 40) * 2^-24.
__global__ __launch_bounds__(256) void k_init_matrix(float* __restrict__ W, int64_t cols, int64_t ld, uint64_t key,
                                                     uint64_t layer, float scale) {
  const int64_t o = blockIdx.x;
  for (int64_t i = threadIdx.x; i < cols; i += 256) {
    uint64_t hv = hash64(key, (layer << 48) + (uint64_t)(o * cols + i));
    float u = (float)(hv >> 40) * 0x1p-24f;
    W[o * ld + i] = (2.0f * u - 1.0f) * scale;
  }
}

__global__ __launch_bounds__(256) void k_init_vector(float* __restrict__ w, int64_t D, uint64_t key, float std) {
  for (int64_t d = blockIdx.x * 256ll + threadIdx.x; d < D; d += (int64_t)gridDim.x * 256)
    w[d] = std * irwin_hall(key, (uint64_t)d);
}

// Given gradients of the averaging-only workload, [T][P][Dp]:
// G[k][j][d] = fp32(std * z(key, (k * 2^16 + j) * D + d)); padding is zero.
__global__ __launch_bounds__(256) void k_gen_grads(float* __restrict__ G, int64_t D, int64_t Dp, int P,
                                                   uint64_t key, float std) {
  const int kj = blockIdx.y;  // k * P + j
  const uint64_t k = (uint64_t)(kj / P), j = (uint64_t)(kj % P);
  float* row = G + (int64_t)kj * Dp;
  const uint64_t base = (k * 65536ull + j) * (uint64_t)D;
  for (int64_t d = blockIdx.x * 256ll + threadIdx.x; d < Dp; d += (int64_t)gridDim.x * 256)
    row[d] = d < D ? std * irwin_hall(key, base + (uint64_t)d) : 0.0f;
}

// Indices of one whole round, [T][P][B] with T = K1*K2 global steps starting
// at *step_ctr.  The last workgroup to finish advances *step_ctr by T, so the
// counter lives on the device and a round needs no host-side argument.
__global__ __launch_bounds__(256) void k_draw_indices(int32_t* __restrict__ idx, uint64_t* step_ctr,
                                                      uint32_t* done_ctr, int P, int B, int T, uint64_t N,
                                                      uint64_t key, const int32_t* __restrict__ labels,
                                                      int32_t* __restrict__ ylab, BlkTables tb) {
  const uint64_t t0 = *step_ctr;
  const int64_t total = (int64_t)T * P * B;
  for (int64_t e = blockIdx.x * 256ll + threadIdx.x; e < total; e += (int64_t)gridDim.x * 256) {
    const int64_t s = e % B;
    const int64_t j = (e / B) % P;
    const int64_t tt = e / ((int64_t)B * P);
    const uint64_t ctr = ((t0 + (uint64_t)tt) << 32) | ((uint64_t)j << 16) | (uint64_t)s;
    const int32_t i = (int32_t)(hash64(key, ctr) % N);
    idx[e] = i;
    if (ylab) ylab[e] = labels[i];
    if (tb.gtab) {
      // Row r = (k*S + learner-in-cluster)*B + s of cluster j/S in block tt/K1
      // (the last block with global_last: row (k*P + j)*B + s of one table).
      const int64_t b = tt / tb.K1, k = tt - b * tb.K1, g = j / tb.S, jc = j - g * tb.S;
      const int64_t o = tb.global_last && b == tb.K2 - 1 ? b * (P / tb.S) * tb.Rp + (k * P + j) * B + s
                                                         : (b * (P / tb.S) + g) * tb.Rp + (k * tb.S + jc) * B + s;
      const uint32_t go = (uint32_t)((((k * P + j) * tb.Mp + s) * tb.ldg) >> 6);
      const uint32_t xo = (uint32_t)(((int64_t)i * tb.ldx) >> 6);
      tb.gtab[o] = go;
      tb.xtab[o] = xo;
      if (tb.gtab1) {  // learner j's own rows, r = k*B + s
        const int64_t o1 = (b * P + j) * tb.Rp1 + k * B + s;
        tb.gtab1[o1] = go;
        tb.xtab1[o1] = xo;
      }
    }
  }
  __syncthreads();
  if (threadIdx.x == 0) {
    __threadfence();
    const uint32_t prev = atomicAdd(done_ctr, 1u);
    if (prev == gridDim.x - 1) {
      *step_ctr = t0 + (uint64_t)T;
      *done_ctr = 0u;
      __threadfence();
    }
  }
}

// dst[i] = i for i < n (the row list of an evaluation chunk).
__global__ __launch_bounds__(256) void k_iota(int32_t* __restrict__ dst, int n) {
  const int i = blockIdx.x * 256 + threadIdx.x;
  if (i < n) dst[i] = i;
}

static int grid_for(int64_t n, int cap = 8192) {
  int64_t g = (n + 255) / 256;
  if (g < 1) g = 1;
  return (int)(g < cap ? g : cap);
}

void launch_iota(hipStream_t s, int32_t* dst, int n) { launch(k_iota, (n + 255) / 256, 256, 0, s, dst, n); }

void launch_gen_labels(hipStream_t s, int32_t* y, int64_t N, uint64_t key, uint64_t C) {
  launch(k_gen_labels, grid_for(N), 256, 0, s, y, N, key, C);
}

void launch_gen_data(hipStream_t s, float* X, const int32_t* y, int64_t N, int64_t IN, int64_t INp,
                     uint64_t key_mean, uint64_t key_noise, float sigma) {
  launch(k_gen_data, (unsigned)N, 256, 0, s, X, y, IN, INp, key_mean, key_noise, sigma);
}

void launch_init_matrix(hipStream_t s, float* W, int64_t rows, int64_t cols, int64_t ld, uint64_t key,
                        uint64_t layer, float scale) {
  launch(k_init_matrix, (unsigned)rows, 256, 0, s, W, cols, ld, key, layer, scale);
}

void launch_init_vector(hipStream_t s, float* w, int64_t D, uint64_t key, float std) {
  launch(k_init_vector, grid_for(D), 256, 0, s, w, D, key, std);
}

void launch_gen_grads(hipStream_t s, float* G, int64_t D, int64_t Dp, int P, int T, uint64_t key, float std) {
  dim3 grid((unsigned)grid_for(Dp, 1024), (unsigned)(T * P));
  launch(k_gen_grads, grid, 256, 0, s, G, D, Dp, P, key, std);
}

void launch_draw_indices(hipStream_t s, int32_t* idx, uint64_t* step_ctr, uint32_t* done_ctr, int P, int B,
                         int T, uint64_t N, uint64_t key, const int32_t* labels, int32_t* ylab,
                         const BlkTables& tables) {
  launch(k_draw_indices, grid_for((int64_t)T * P * B, 1024), 256, 0, s, idx, step_ctr, done_ctr, P, B, T, N, key,
         labels, ylab, tables);
}

}  // namespace hav
