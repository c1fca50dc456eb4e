// Averaging of replicas (Algorithm 1, Sec. 3.1): the local mean over each
// cluster of S learners after every block of K1 steps, and the global mean
// over all P learners at the end of the round.  Both are HBM streams over the
// [P][Dp] replica array: every lane owns one 16-byte column slice and walks
// the S rows of its group, so each row is read once, coalesced along D, the
// sum over replicas stays in registers in the fixed order 0..S-1 (identical
// results on every run), and the mean is written back to all S rows.
//
// The averaging-only workload fuses its heavy-ball update v <- mu*v + g,
// w <- w - lr*v into the same pass (momentum buffers are per learner and are
// not averaged: Algorithm 1 averages parameters only).
#include "internal.h"

namespace hav {

__device__ inline f32x4 ld_stream(const f32x4* p) { return __builtin_nontemporal_load(p); }
__device__ inline void st_stream(f32x4* p, f32x4 v) { __builtin_nontemporal_store(v, p); }

// grid (x: column blocks, y: group).  Rows g*S .. g*S+S-1, columns [0, n4) in
// float4 units, row pitch pitch4.
__global__ __launch_bounds__(256) void k_group_mean(f32x4* __restrict__ W, int64_t pitch4, int64_t n4, int S) {
  f32x4* base = W + (int64_t)blockIdx.y * S * pitch4;
  const float inv = 1.0f / (float)S;
  const bool pow2 = (S & (S - 1)) == 0;
  for (int64_t i = blockIdx.x * 256ll + threadIdx.x; i < n4; i += (int64_t)gridDim.x * 256) {
    f32x4 sum = ld_stream(base + i);
    int u = 1;
    for (; u + 4 <= S; u += 4) {
      f32x4 a = ld_stream(base + (int64_t)u * pitch4 + i);
      f32x4 b = ld_stream(base + (int64_t)(u + 1) * pitch4 + i);
      f32x4 c = ld_stream(base + (int64_t)(u + 2) * pitch4 + i);
      f32x4 d = ld_stream(base + (int64_t)(u + 3) * pitch4 + i);
      sum += a;
      sum += b;
      sum += c;
      sum += d;
    }
    for (; u < S; ++u) sum += ld_stream(base + (int64_t)u * pitch4 + i);
    // Exact division by S (a power of two is an exact scaling either way).
    f32x4 mean = pow2 ? sum * inv : sum / (float)S;
    for (int v = 0; v < S; ++v) st_stream(base + (int64_t)v * pitch4 + i, mean);
  }
}

// Heavy-ball step of rows g*S .. g*S+S-1 with the given gradients Gr (row
// pitch pitch4); with `average`, the S updated rows are replaced by their mean
// in the same pass.
template <bool AVERAGE>
__global__ __launch_bounds__(256) void k_momentum(f32x4* __restrict__ W, f32x4* __restrict__ V,
                                                  const f32x4* __restrict__ Gr, int64_t pitch4, int64_t n4, int S,
                                                  float lr, float mu) {
  const int64_t row0 = (int64_t)blockIdx.y * S;
  const bool pow2 = (S & (S - 1)) == 0;
  const float inv = 1.0f / (float)S;
  for (int64_t i = blockIdx.x * 256ll + threadIdx.x; i < n4; i += (int64_t)gridDim.x * 256) {
    f32x4 sum = {0.f, 0.f, 0.f, 0.f};
#pragma unroll 4
    for (int u = 0; u < S; ++u) {
      const int64_t o = (row0 + u) * pitch4 + i;
      f32x4 w = ld_stream(W + o);
      f32x4 v = ld_stream(V + o);
      const f32x4 g = ld_stream(Gr + o);
      v = mu * v + g;
      w = w - lr * v;
      st_stream(V + o, v);
      if (AVERAGE)
        sum += w;
      else
        st_stream(W + o, w);
    }
    if (AVERAGE) {
      const f32x4 mean = pow2 ? sum * inv : sum / (float)S;
      for (int u = 0; u < S; ++u) st_stream(W + (row0 + u) * pitch4 + i, mean);
    }
  }
}

static unsigned col_blocks(int64_t n4, int groups) {
  // About 8 resident workgroups per CU over the whole launch.
  int64_t want = (2048 + groups - 1) / groups;
  int64_t need = (n4 + 255) / 256;
  int64_t g = want < need ? want : need;
  return (unsigned)(g < 1 ? 1 : g);
}

void launch_group_mean(hipStream_t s, float* W, int64_t Dp, int P, int S) {
  const int64_t n4 = Dp / 4;
  dim3 grid(col_blocks(n4, P / S), (unsigned)(P / S));
  k_group_mean<<<grid, 256, 0, s>>>((f32x4*)W, n4, n4, S);
}

void launch_momentum_step(hipStream_t s, float* W, float* V, const float* Gr, int64_t Dp, int P, int S,
                          bool average, float lr, float mu) {
  const int64_t n4 = Dp / 4;
  const int groups = average ? P / S : P;
  const int rows = average ? S : 1;
  dim3 grid(col_blocks(n4, groups), (unsigned)groups);
  if (average)
    k_momentum<true><<<grid, 256, 0, s>>>((f32x4*)W, (f32x4*)V, (const f32x4*)Gr, n4, n4, rows, lr, mu);
  else
    k_momentum<false><<<grid, 256, 0, s>>>((f32x4*)W, (f32x4*)V, (const f32x4*)Gr, n4, n4, rows, lr, mu);
}

}  // namespace hav
