// Averaging of replicas (Algorithm 1, Sec. 3.1): the local mean over each
// cluster of S learners after every block of K1 steps, and the global mean
// over all P learners at the end of the round.  Both are HBM streams over the
// [P][Dp] replica array, coalesced along D: a workgroup owns a run of 16-byte
// column pieces of one cluster; each thread takes one column piece and RG
// consecutive rows of the cluster (NG = S / RG threads per column), keeps its
// rows' partial sum in registers (rows in order), and the NG partial sums of a
// column are added through LDS in group order, so every run produces the same
// bits.  The mean is then written back to all S rows.
//
// The averaging-only workload fuses its heavy-ball step v <- mu*v + g +
// lambda*w, w <- w - lr*v into the same pass (the momentum buffers are per
// learner; Algorithm 1 averages parameters only, and the variant that also
// averages the buffers runs the plain mean over them as a second pass).
// After the global mean every learner holds the same parameters, so that pass
// writes the mean once, to a vector of its own, and the first step of the
// next round reads every learner's parameters from it: a pass over S rows
// of every column runs at about 0.75 of HBM peak for S = 4 and 0.68 for
// S = 32 on MI355X (more distinct rows in flight per column), and the single
// write takes a fifth of the global pass's bytes away.
#include <algorithm>

#include "internal.h"

namespace hav {

#ifndef HAV_AVG_RG
#define HAV_AVG_RG 1
#endif
#ifndef HAV_AVG_NT
#define HAV_AVG_NT 1
#endif
#if HAV_AVG_NT
__device__ inline f32x4 ld_stream(const f32x4* p) { return __builtin_nontemporal_load(p); }
__device__ inline void st_stream(f32x4* p, f32x4 v) { __builtin_nontemporal_store(v, p); }
#else
__device__ inline f32x4 ld_stream(const f32x4* p) { return *p; }
__device__ inline void st_stream(f32x4* p, f32x4 v) { *p = v; }
#endif

// grid (x: column runs, y: cluster).  MOM: apply the heavy-ball step with the
// given gradients Gr first.  MEAN: replace the S rows by their mean (else each
// updated row is written back as it is); ONE: write the mean to M instead (the
// global mean, one group).  The rows' parameters are read from Wsrc, rows wp4
// f32x4 apart (Wsrc = W, wp4 = pitch4; or the shared vector, wp4 = 0).  M may
// be the shared vector: a column's reads all come before its one write.
template <bool MOM, bool MEAN, int RG, int NG, int TB, bool ONE = false>
__global__ __launch_bounds__(TB) void k_rows(f32x4* W, f32x4* __restrict__ V, const f32x4* __restrict__ Gr,
                                             int64_t pitch4, int64_t n4, const float* __restrict__ lr_ptr, float mu,
                                             float wd, const f32x4* Wsrc, int64_t wp4, f32x4* M) {
  const float lr = MOM ? *lr_ptr : 0.0f;
  constexpr int S = RG * NG;
  constexpr int CPB = TB / NG;  // columns per workgroup
  __shared__ f32x4 part[NG > 1 ? NG : 1][CPB];
  const int tid = threadIdx.x, cl = tid % CPB, g = tid / CPB;
  const int64_t row0 = (int64_t)blockIdx.y * S + g * RG;
  for (int64_t c0 = (int64_t)blockIdx.x * CPB; c0 < n4; c0 += (int64_t)gridDim.x * CPB) {
    const int64_t i = c0 + cl;
    const bool ok = i < n4;
    const int64_t ic = ok ? i : 0;
    f32x4 w[RG];
#pragma unroll
    for (int u = 0; u < RG; ++u) w[u] = ld_stream(Wsrc + (row0 + u) * wp4 + ic);
    if (MOM) {
      f32x4 v[RG], gr[RG];
#pragma unroll
      for (int u = 0; u < RG; ++u) {
        v[u] = ld_stream(V + (row0 + u) * pitch4 + ic);
        gr[u] = ld_stream(Gr + (row0 + u) * pitch4 + ic);
      }
#pragma unroll
      for (int u = 0; u < RG; ++u) {
        v[u] = mu * v[u] + (gr[u] + wd * w[u]);
        w[u] = w[u] - lr * v[u];
        if (ok) st_stream(V + (row0 + u) * pitch4 + i, v[u]);
      }
    }
    if (!MEAN) {
#pragma unroll
      for (int u = 0; u < RG; ++u)
        if (ok) st_stream(W + (row0 + u) * pitch4 + i, w[u]);
      continue;
    }
    f32x4 sum = w[0];
#pragma unroll
    for (int u = 1; u < RG; ++u) sum += w[u];
    if (NG > 1) {
      part[g][cl] = sum;
      __syncthreads();
      sum = part[0][cl];
#pragma unroll
      for (int k = 1; k < NG; ++k) sum += part[k][cl];
      __syncthreads();
    }
    // S is a power of two here, so the scaling by 1/S is exact.
    const f32x4 mean = sum * (1.0f / (float)S);
    if (ONE) {
      if (ok && g == 0) st_stream(M + i, mean);
    } else {
#pragma unroll
      for (int u = 0; u < RG; ++u)
        if (ok) st_stream(W + (row0 + u) * pitch4 + i, mean);
    }
  }
}

// Any S: one thread per column piece walks all S rows (runtime count).
// Wsrc, wp4 and M (non-null: the mean goes there instead of the S rows) as in
// k_rows.
template <bool MOM>
__global__ __launch_bounds__(256) void k_rows_any(f32x4* W, f32x4* __restrict__ V, const f32x4* __restrict__ Gr,
                                                  int64_t pitch4, int64_t n4, int S, const float* __restrict__ lr_ptr,
                                                  float mu, float wd, const f32x4* Wsrc, int64_t wp4,
                                                  f32x4* M) {
  const float lr = MOM ? *lr_ptr : 0.0f;
  const int64_t row0 = (int64_t)blockIdx.y * S;
  for (int64_t i = blockIdx.x * 256ll + threadIdx.x; i < n4; i += (int64_t)gridDim.x * 256) {
    f32x4 sum = {0.f, 0.f, 0.f, 0.f};
#pragma unroll 4
    for (int u = 0; u < S; ++u) {
      const int64_t o = (row0 + u) * pitch4 + i;
      f32x4 w = ld_stream(Wsrc + (row0 + u) * wp4 + i);
      if (MOM) {
        f32x4 v = ld_stream(V + o);
        const f32x4 g = ld_stream(Gr + o);
        v = mu * v + (g + wd * w);
        w = w - lr * v;
        st_stream(V + o, v);
      }
      sum += w;
    }
    const f32x4 mean = sum / (float)S;
    if (M)
      st_stream(M + i, mean);
    else
      for (int u = 0; u < S; ++u) st_stream(W + (row0 + u) * pitch4 + i, mean);
  }
}

static unsigned col_runs(int64_t n4, int cpb, int groups) {
  // One column piece per thread, up to about 2^20 workgroups in all.
  int64_t need = (n4 + cpb - 1) / cpb;
  int64_t cap = std::max<int64_t>(1, (int64_t(1) << 20) / groups);
  return (unsigned)(need < cap ? need : cap);
}

// Where a pass reads the learners' parameters and where a global mean goes.
struct RowIO {
  const float* src;  // nullptr: the rows themselves
  int64_t src_pitch4;
  float* mean_out;   // nullptr: the mean goes to the rows
};

template <bool MOM, bool MEAN, int RG, int NG, int TB = 256, bool ONE = false>
static void launch_rows(hipStream_t s, float* W, float* V, const float* Gr, int64_t p4, int64_t n4, int groups,
                        const float* lr, float mu, float wd, const RowIO& io) {
  dim3 grid(col_runs(n4, TB / NG, groups), (unsigned)groups);
  launch(k_rows<MOM, MEAN, RG, NG, TB, ONE>, grid, TB, 0, s, (f32x4*)W, (f32x4*)V, (const f32x4*)Gr, p4, n4, lr, mu,
         wd, (const f32x4*)(io.src ? io.src : W), io.src ? io.src_pitch4 : p4, (f32x4*)io.mean_out);
}

// Cluster of S rows with S a power of two up to 64.  Up to 16 rows: one row per
// thread and S threads per column (more threads keep more loads in flight than
// more rows per thread); 32 and 64 rows: four rows per thread in 1024-thread
// workgroups (longer row segments per workgroup).  Measured on MI355X.
// Returns false for other S.
#ifndef HAV_AVG_RG_BIG
#define HAV_AVG_RG_BIG 4
#endif
#ifndef HAV_AVG_TB_BIG
#define HAV_AVG_TB_BIG 1024
#endif
template <bool MOM, int S, bool ONE>
static void launch_s(hipStream_t s, float* W, float* V, const float* Gr, int64_t p4, int64_t n4, int groups,
                     const float* lr, float mu, float wd, const RowIO& io) {
  constexpr int kR = S <= 16 ? HAV_AVG_RG : HAV_AVG_RG_BIG;
  constexpr int RG = S < kR ? S : kR;
  constexpr int TB = S <= 16 ? 256 : HAV_AVG_TB_BIG;
  launch_rows<MOM, true, RG, S / RG, TB, ONE>(s, W, V, Gr, p4, n4, groups, lr, mu, wd, io);
}

template <bool MOM, bool ONE = false>
static bool launch_mean_pow2(hipStream_t s, float* W, float* V, const float* Gr, int64_t p4, int64_t n4, int P,
                             int S, const float* lr, float mu, float wd, const RowIO& io) {
  const int groups = P / S;
  switch (S) {
    case 2: launch_s<MOM, 2, ONE>(s, W, V, Gr, p4, n4, groups, lr, mu, wd, io); return true;
    case 4: launch_s<MOM, 4, ONE>(s, W, V, Gr, p4, n4, groups, lr, mu, wd, io); return true;
    case 8: launch_s<MOM, 8, ONE>(s, W, V, Gr, p4, n4, groups, lr, mu, wd, io); return true;
    case 16: launch_s<MOM, 16, ONE>(s, W, V, Gr, p4, n4, groups, lr, mu, wd, io); return true;
    case 32: launch_s<MOM, 32, ONE>(s, W, V, Gr, p4, n4, groups, lr, mu, wd, io); return true;
    case 64: launch_s<MOM, 64, ONE>(s, W, V, Gr, p4, n4, groups, lr, mu, wd, io); return true;
    default: return false;
  }
}

void launch_group_mean(hipStream_t s, float* W, int64_t pitch, int64_t len, int P, int S) {
  const int64_t p4 = pitch / 4, n4 = len / 4;
  const RowIO io{nullptr, 0, nullptr};
  if (launch_mean_pow2<false>(s, W, nullptr, nullptr, p4, n4, P, S, nullptr, 0.0f, 0.0f, io)) return;
  dim3 grid(col_runs(n4, 256, P / S), (unsigned)(P / S));
  launch(k_rows_any<false>, grid, 256, 0, s, (f32x4*)W, nullptr, nullptr, p4, n4, S, (const float*)nullptr, 0.0f,
         0.0f, (const f32x4*)W, p4, (f32x4*)nullptr);
}

// Workgroups below g1: dst = mean of the n rows of src.  The others (when W
// is set): each column of the first n4b pieces of W's nb rows replaced by the
// rows' mean, rows added in order.
__global__ __launch_bounds__(256) void k_mean_rows(f32x4* __restrict__ dst, const f32x4* __restrict__ src,
                                                   int64_t pitch4, int64_t n4, int n, int g1, f32x4* __restrict__ W,
                                                   int64_t pitchb4, int64_t n4b, int nb) {
  // Rows are read eight at a time, all loads of a group issued before its
  // adds (a row past the last re-reads the last one and is not added), and
  // added in row order.
  auto row_sum = [](const f32x4* __restrict__ base, int64_t pitch, int rows) {
    f32x4 sum = base[0];
    for (int r0 = 1; r0 < rows; r0 += 8) {
      f32x4 v[8];
#pragma unroll
      for (int j = 0; j < 8; ++j) v[j] = base[(int64_t)(r0 + j < rows ? r0 + j : rows - 1) * pitch];
#pragma unroll
      for (int j = 0; j < 8; ++j)
        if (r0 + j < rows) sum += v[j];
    }
    return sum;
  };
  if ((int)blockIdx.x < g1) {
    for (int64_t i = blockIdx.x * 256ll + threadIdx.x; i < n4; i += (int64_t)g1 * 256)
      dst[i] = row_sum(src + i, pitch4, n) / (float)n;
    return;
  }
  const int gb = gridDim.x - g1;
  for (int64_t i = (blockIdx.x - g1) * 256ll + threadIdx.x; i < n4b; i += (int64_t)gb * 256) {
    const f32x4 mean = row_sum(W + i, pitchb4, nb) / (float)nb;
    for (int r = 0; r < nb; ++r) W[r * pitchb4 + i] = mean;
  }
}

void launch_mean_rows(hipStream_t s, float* dst, const float* src, int64_t pitch, int64_t len, int n, float* W,
                      int64_t pitch_b, int64_t len_b, int nb) {
  const int64_t n4 = len / 4;
  const unsigned g1 = col_runs(n4, 256, 1), gb = W ? col_runs(len_b / 4, 256, 1) : 0;
  launch(k_mean_rows, g1 + gb, 256, 0, s, (f32x4*)dst, (const f32x4*)src, pitch / 4, n4, n, (int)g1, (f32x4*)W,
         pitch_b / 4, len_b / 4, nb);
}

__global__ __launch_bounds__(256) void k_rows_differ(const int4* __restrict__ W, int64_t pitch4, int64_t n4, int n,
                                                     int* __restrict__ flag) {
  const int64_t total = (int64_t)(n - 1) * n4;
  for (int64_t e = blockIdx.x * 256ll + threadIdx.x; e < total; e += (int64_t)gridDim.x * 256) {
    const int64_t r = 1 + e / n4, i = e % n4;
    const int4 a = W[r * pitch4 + i], b = W[i];
    if (a.x != b.x || a.y != b.y || a.z != b.z || a.w != b.w) *flag = 1;
  }
}

void launch_rows_differ(hipStream_t s, const float* W, int64_t pitch, int64_t len, int n, int* flag) {
  if (n < 2) return;
  launch(k_rows_differ, col_runs((int64_t)(n - 1) * (len / 4), 256, 1), 256, 0, s, (const int4*)W, pitch / 4,
         len / 4, n, flag);
}

__global__ __launch_bounds__(256) void k_any_nonfinite(const f32x4* __restrict__ W, int64_t n4,
                                                       int* __restrict__ flag) {
  bool bad = false;
  for (int64_t i = blockIdx.x * 256ll + threadIdx.x; i < n4; i += (int64_t)gridDim.x * 256) {
    const f32x4 v = W[i];
    bad |= !(isfinite(v.x) && isfinite(v.y) && isfinite(v.z) && isfinite(v.w));
  }
  if (bad) *flag = 1;
}

void launch_any_nonfinite(hipStream_t s, const float* W, int64_t n, int* flag) {
  launch(k_any_nonfinite, col_runs(n / 4, 256, 1) < 4096 ? col_runs(n / 4, 256, 1) : 4096u, 256, 0, s,
         (const f32x4*)W, n / 4, flag);
}

void launch_momentum_step(hipStream_t s, float* W, float* V, const float* Gr, int64_t Dp, int P, int S,
                          bool average, const float* lr, float mu, float wd, const float* shared_in,
                          float* mean_out) {
  const int64_t n4 = Dp / 4;
  const RowIO io{shared_in, 0, S == P ? mean_out : nullptr};
  if (!average) {
    launch_rows<true, false, 1, 1>(s, W, V, Gr, n4, n4, P, lr, mu, wd, io);
    return;
  }
  if (io.mean_out ? launch_mean_pow2<true, true>(s, W, V, Gr, n4, n4, P, S, lr, mu, wd, io)
               : launch_mean_pow2<true, false>(s, W, V, Gr, n4, n4, P, S, lr, mu, wd, io))
    return;
  dim3 grid(col_runs(n4, 256, P / S), (unsigned)(P / S));
  launch(k_rows_any<true>, grid, 256, 0, s, (f32x4*)W, (f32x4*)V, (const f32x4*)Gr, n4, n4, S, lr, mu, wd,
         (const f32x4*)(shared_in ? shared_in : W), shared_in ? 0 : n4, (f32x4*)io.mean_out);
}

}  // namespace hav
