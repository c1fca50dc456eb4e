// Per-learner dense contractions of one local SGD step (Algorithm 1, Sec. 3.1:
// each learner's minibatch gradient of the softmax cross-entropy, followed by
// w <- w - lr * g), batched over the P learners and run on fp32 MFMA.
//
// k_fwd_nt:    part[ks][p][m][n] = sum_{k in split ks} A_p[m][k] * W_p[n][k]
//              (A = gathered minibatch rows of X, or ReLU of the hidden
//              pre-activations; W = a weight block, K-contiguous), split
//              over K so the launch fills the GPU.  The consumer adds the
//              partials in split order 0..KS-1 and the bias (deterministic; no
//              synchronisation between workgroups inside a kernel).
// k_update_tn: W_p[m][n] -= lr * sum_s G_p[s][m] * Bsrc_p[s][n], the weight
//              gradient of a layer fused with the SGD update (the gradient is
//              never stored), plus b_p[m] -= lr * sum_s G_p[s][m].
#include <algorithm>

#include "internal.h"

namespace hav {

constexpr int kKC = 64;         // K floats per pipeline stage of k_fwd_nt
constexpr int kLdsStride = 68;  // LDS row stride in floats (64 + 4: conflict-free 128-bit reads)
#ifndef HAV_FWD_TARGET_WG
#define HAV_FWD_TARGET_WG 512
#endif
constexpr int kFwdTargetWG = HAV_FWD_TARGET_WG;  // workgroups a forward launch aims for

__device__ inline f32x4 relu4(f32x4 v) {
  v.x = fmaxf(v.x, 0.0f);
  v.y = fmaxf(v.y, 0.0f);
  v.z = fmaxf(v.z, 0.0f);
  v.w = fmaxf(v.w, 0.0f);
  return v;
}

// Workgroup tile: MB*16 rows (minibatch samples) x 128 columns (output units),
// one K split.  Wave w owns columns [32w, 32w + 32) as two 16x16 MFMA blocks.
// The A tile is staged through LDS (double-buffered, one barrier per stage)
// because all four waves use it; W is streamed straight into registers in the
// 16x16x4 operand layout (lane l holds row l%16, four consecutive k at
// 16q + 4*(l/16)), prefetched one 64-wide stage ahead.  Within a 16-wide k
// group the four MFMAs take k = 4g + i (g = lane group, i = MFMA index): a
// permutation of the k order that A and W share, so the contraction is
// unchanged.
template <int ASRC, int MB>
__global__ __launch_bounds__(256) void k_fwd_nt(FwdArgs a, int ntiles, int mtiles) {
  constexpr int MT = MB * 16;
  constexpr int NLOAD = MT * (kKC / 4);
  constexpr int LPT = (NLOAD + 255) / 256;
  __shared__ __attribute__((aligned(16))) float As[2][MT * kLdsStride];

  const int bid = xcd_remap(blockIdx.x, gridDim.x);
  const int nt = bid % ntiles;
  const int mt = (bid / ntiles) % mtiles;
  const int ks = (bid / (ntiles * mtiles)) % a.KS;
  const int p = bid / (ntiles * mtiles * a.KS);
  const int nch = a.K / kKC;
  const int c0 = ks * a.cps;
  const int c1 = min(nch, c0 + a.cps);

  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  const int lrow = lane & 15, lgrp = lane >> 4;
  const int nw = nt * 128 + wave * 32;
  const bool v0 = nw < a.N, v1 = nw + 16 < a.N;
  const int mbase = mt * MT;

  // Loads are branch-free (out-of-range rows read row 0 and are zeroed by a
  // select): the compiler can then count outstanding loads exactly, and the
  // next stage's loads stay in flight while the current stage computes.
  const float* arow[LPT];
  bool aok[LPT];
  int lds_off[LPT];
#pragma unroll
  for (int i = 0; i < LPT; ++i) {
    const int q = tid + 256 * i;
    const int r = q >> 4, c4 = q & 15;
    lds_off[i] = r * kLdsStride + 4 * c4;
    const int m = mbase + r;
    aok[i] = m < a.M;
    const int mc = aok[i] ? m : 0;
    int64_t row;
    if (ASRC == A_GATHER)
      row = a.idx[(int64_t)p * a.M + mc];
    else
      row = (int64_t)p * a.Mp + mc;
    arow[i] = a.A + row * a.lda + 4 * c4;
  }
  const float* wp = a.W + (int64_t)p * a.w_pitch;
  const float* wrow0 = wp + (int64_t)(v0 ? nw + lrow : lrow) * a.ldw + 4 * lgrp;
  const float* wrow1 = wp + (int64_t)(v1 ? nw + 16 + lrow : lrow) * a.ldw + 4 * lgrp;

  f32x4 acc[MB][2];
#pragma unroll
  for (int m = 0; m < MB; ++m) acc[m][0] = acc[m][1] = f32x4{0.f, 0.f, 0.f, 0.f};
  f32x4 ar[LPT];
  f32x4 wa[2][4], wb[2][4];
  const f32x4 zero4 = {0.f, 0.f, 0.f, 0.f};

  auto load_a = [&](int c) {
#pragma unroll
    for (int i = 0; i < LPT; ++i) ar[i] = *(const f32x4*)(arow[i] + (int64_t)c * kKC);
  };
  auto store_a = [&](int buf) {
#pragma unroll
    for (int i = 0; i < LPT; ++i) {
      f32x4 v = aok[i] ? ar[i] : zero4;
      *(f32x4*)&As[buf][lds_off[i]] = ASRC == A_RELU ? relu4(v) : v;
    }
  };
  auto load_w = [&](int c, f32x4 (&w)[2][4]) {
    const int64_t o = (int64_t)c * kKC;
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      w[0][q] = *(const f32x4*)(wrow0 + o + 16 * q);
      w[1][q] = *(const f32x4*)(wrow1 + o + 16 * q);
    }
  };
  // Waves whose columns lie past N compute on row 0 and store nothing.
  auto compute = [&](int buf, const f32x4 (&w)[2][4]) {
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      f32x4 af[MB];
#pragma unroll
      for (int m = 0; m < MB; ++m)
        af[m] = *(const f32x4*)&As[buf][(16 * m + lrow) * kLdsStride + 16 * q + 4 * lgrp];
#pragma unroll
      for (int i = 0; i < 4; ++i) {
#pragma unroll
        for (int m = 0; m < MB; ++m) {
          acc[m][0] = __builtin_amdgcn_mfma_f32_16x16x4f32(af[m][i], w[0][q][i], acc[m][0], 0, 0, 0);
          acc[m][1] = __builtin_amdgcn_mfma_f32_16x16x4f32(af[m][i], w[1][q][i], acc[m][1], 0, 0, 0);
        }
      }
    }
  };

  // Two register sets for W alternate (no copies), so the wait for a stage's
  // W is placed right before its MFMAs and the next stage's loads stay in
  // flight meanwhile.  Prefetches past the last stage re-read the last stage
  // (in range, unused), which keeps the loads unconditional.
  if (c0 < c1) {
    load_a(c0);
    load_w(c0, wa);
    store_a(0);
    __syncthreads();
    for (int c = c0; c < c1; c += 2) {
      const int n1 = min(c + 1, c1 - 1), n2 = min(c + 2, c1 - 1);
      load_a(n1);
      load_w(n1, wb);
      __builtin_amdgcn_sched_barrier(0);  // issue the prefetch before the MFMAs
      compute(0, wa);
      store_a(1);
      __syncthreads();
      if (c + 1 >= c1) break;
      load_a(n2);
      load_w(n2, wa);
      __builtin_amdgcn_sched_barrier(0);
      compute(1, wb);
      store_a(0);
      __syncthreads();
    }
  }

  float* part = a.part + ((int64_t)ks * a.P + p) * a.Mp * a.N;
#pragma unroll
  for (int m = 0; m < MB; ++m)
#pragma unroll
    for (int j = 0; j < 2; ++j) {
      if (j == 0 ? !v0 : !v1) continue;
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int row = mbase + 16 * m + 4 * lgrp + r;
        if (row < a.Mp) part[(int64_t)row * a.N + nw + 16 * j + lrow] = acc[m][j][r];
      }
    }
}

static int pick_mb(int Mp) { return Mp >= 128 ? 8 : Mp >= 64 ? 4 : Mp >= 32 ? 2 : 1; }

void plan_split(int P, int Mp, int N, int K, int* KS, int* cps) {
  // Enough K splits that the launch has about kFwdTargetWG workgroups (the GEMMs have
  // few output tiles per learner: M is the minibatch), and no empty split.
  const int MB = pick_mb(Mp);
  const int mtiles = (Mp + MB * 16 - 1) / (MB * 16);
  const int nch = K / kKC;
  const int64_t tiles = (int64_t)P * mtiles * ((N + 127) / 128);
  int ks = (int)std::max<int64_t>(1, (kFwdTargetWG + tiles - 1) / tiles);
  ks = std::min(ks, nch);
  const int c = (nch + ks - 1) / ks;
  *KS = (nch + c - 1) / c;
  *cps = c;
}

int fwd_tiles(int P, int Mp, int N) {
  const int MB = pick_mb(Mp);
  const int mtiles = (Mp + MB * 16 - 1) / (MB * 16);
  return P * mtiles * ((N + 127) / 128);
}

void launch_fwd(hipStream_t s, const FwdArgs& a, ASource src) {
  const int MB = pick_mb(a.Mp);
  const int mtiles = (a.Mp + MB * 16 - 1) / (MB * 16);
  const int ntiles = (a.N + 127) / 128;
  const unsigned grid = (unsigned)((int64_t)a.P * a.KS * mtiles * ntiles);
#define HAV_FWD(S_, MB_) launch(k_fwd_nt<S_, MB_>, grid, 256, 0, s, a, ntiles, mtiles)
#define HAV_FWD_MB(S_)   \
  switch (MB) {          \
    case 1: HAV_FWD(S_, 1); break; \
    case 2: HAV_FWD(S_, 2); break; \
    case 4: HAV_FWD(S_, 4); break; \
    default: HAV_FWD(S_, 8); break; \
  }
  if (src == A_GATHER) {
    HAV_FWD_MB(A_GATHER)
  } else {
    HAV_FWD_MB(A_RELU)
  }
#undef HAV_FWD_MB
#undef HAV_FWD
}

// Workgroup tile 64 (rows m of W) x 256 (columns n of W).  The contraction
// runs over the minibatch (K = B) in stages of 32 samples: the stage's error
// rows G[s][m-tile] and input rows Bsrc[s][n-tile] (gathered through the
// sample indices) are copied into LDS with 16-byte loads; wave w computes the
// 64 x 64 block of columns [64w, 64w + 64) as 2 x 2 32x32x2 MFMA blocks, lane
// l taking G[s + l/32][m0 + l%32] and Bsrc[s + l/32][n0 + l%32] from LDS.
// The W tile is read before the first stage with 16-byte loads (one 1 KB row
// segment per wave instruction) so its latency overlaps the staging and the
// MFMAs; the accumulators (lane l, register r: row 8*(r/4) + 4*(l/32) + r%4,
// column l%32) are written to LDS and read back in the same 16-byte layout as
// the W tile for the update w - lr * g.
#ifndef HAV_UPD_UN
#define HAV_UPD_UN 128
#endif
constexpr int kUM = 64;           // W rows per workgroup
constexpr int kUN = HAV_UPD_UN;   // W columns per workgroup (64 per wave)
constexpr int kWC = kUN / 64;     // waves across the columns (64 columns each)
constexpr int kMI = kUM / (4 / kWC) / 32;  // 32-row MFMA blocks per wave
static_assert(kUN == 128 || kUN == 256, "update tile width");
constexpr int kSC = 32;           // samples per LDS stage
constexpr int kLA = kUM + 4;      // LDS row length of the G stage
constexpr int kLB = kUN + 4;      // LDS row length of the input stage and of the gradient tile
constexpr int kUpdLds = (kUM * kLB > kSC * (kLA + kLB)) ? kUM * kLB : kSC * (kLA + kLB);

template <int BSRC>
__global__ __launch_bounds__(256) void k_update_tn(UpdArgs a, int mtiles, int ntiles) {
  __shared__ __attribute__((aligned(16))) float lds[kUpdLds];
  float* As = lds;               // [kSC][kLA]
  float* Bs = lds + kSC * kLA;   // [kSC][kLB]
  float* Gt = lds;               // [kUM][kLB] gradient tile (after the stages)
  const int bid = xcd_remap(blockIdx.x, gridDim.x);
  const int nt = bid % ntiles;
  const int mt = (bid / ntiles) % mtiles;
  const int p = bid / (ntiles * mtiles);
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  const int l32 = lane & 31, lhi = lane >> 5;
  const int mrow0 = mt * kUM, ncol0 = nt * kUN;
  const int wn = (wave % kWC) * 64, wm = (wave / kWC) * kMI * 32;
  const bool wave_on = ncol0 + wn < a.Ncols;
  float* Wp = a.W + (int64_t)p * a.w_pitch;
  const float* Gp = a.G + (int64_t)p * a.Mp * a.ldg;
  const f32x4 zero4 = {0.f, 0.f, 0.f, 0.f};

  // The stage operands are loaded before the W tile: loads complete in issue
  // order, so waiting for the operands then leaves the W loads in flight
  // through the staging and the MFMAs.
  // All loads are branch-free (out-of-range pieces read an in-range address
  // and are zeroed by a select), so the compiler counts outstanding loads
  // exactly; the sample indices of a stage are read before its input rows.
  constexpr int kXP = kUN / 4;          // 16-byte pieces per input row
  constexpr int kXR = 256 / kXP;         // input rows per pass of the workgroup
  constexpr int kXL = kSC / kXR;         // input pieces per thread
  f32x4 ga[2], xb[kXL];
  bool gok[2], xok[kXL];
  const int xc4 = tid % kXP, xr0 = tid / kXP;
  const bool xcol_ok = ncol0 + 4 * xc4 < a.Ncols;
  const int xcol = xcol_ok ? ncol0 + 4 * xc4 : 0;
  auto load_stage = [&](int s0) {
#pragma unroll
    for (int i = 0; i < 2; ++i) {  // G[s0 .. s0+32)[mrow0 .. +64): 512 pieces
      const int q = tid + 256 * i;
      const int r = q >> 4, c4 = q & 15;
      const int s = s0 + r, m = mrow0 + 4 * c4;
      gok[i] = s < a.Kb && m < a.Mrows;
      ga[i] = *(const f32x4*)(Gp + (int64_t)(s < a.Kb ? s : 0) * a.ldg + (m < a.Mrows ? m : 0));
    }
    int64_t rows[kXL];
#pragma unroll
    for (int i = 0; i < kXL; ++i) {  // Bsrc[s0 .. s0+32)[ncol0 .. +kUN)
      const int s = s0 + xr0 + kXR * i;
      xok[i] = s < a.Kb && xcol_ok;
      const int sc = s < a.Kb ? s : 0;
      rows[i] = BSRC == A_GATHER ? (int64_t)a.idx[(int64_t)p * a.Kb + sc] : (int64_t)p * a.Mp + sc;
    }
#pragma unroll
    for (int i = 0; i < kXL; ++i) xb[i] = *(const f32x4*)(a.Bsrc + rows[i] * a.ldb + xcol);
  };
  auto store_stage = [&]() {
#pragma unroll
    for (int i = 0; i < 2; ++i) {
      const int q = tid + 256 * i;
      *(f32x4*)&As[(q >> 4) * kLA + 4 * (q & 15)] = gok[i] ? ga[i] : zero4;
    }
#pragma unroll
    for (int i = 0; i < kXL; ++i) {
      f32x4 v = xok[i] ? xb[i] : zero4;
      *(f32x4*)&Bs[(xr0 + kXR * i) * kLB + 4 * xc4] = BSRC == A_RELU ? relu4(v) : v;
    }
  };
  load_stage(0);
  __builtin_amdgcn_sched_barrier(0);  // keep the W loads behind the stage loads

  // W tile in 16-byte pieces: thread t takes column piece t%kXP of rows
  // t/kXP + kXR*i.
  const int wc4 = tid % kXP, wr0 = tid / kXP;
  const int wcol = ncol0 + 4 * wc4;
  const bool col_ok = wcol < a.Ncols;
  constexpr int kWL = kUM / kXR;
  f32x4 wv[kWL];
#pragma unroll
  for (int i = 0; i < kWL; ++i) {
    const int row = mrow0 + wr0 + kXR * i;
    wv[i] = *(const f32x4*)(Wp + (int64_t)(row < a.Mrows ? row : 0) * a.ldw + (col_ok ? wcol : 0));
  }

  f32x16 acc[kMI][2];
#pragma unroll
  for (int i = 0; i < kMI; ++i)
#pragma unroll
    for (int j = 0; j < 2; ++j)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.0f;

  for (int s0 = 0; s0 < a.Kb; s0 += kSC) {
    if (s0 > 0) load_stage(s0);
    store_stage();
    __syncthreads();
    if (wave_on) {
#pragma unroll
      for (int ss = 0; ss < kSC; ss += 2) {
        const int sr = ss + lhi;
        const float b0 = Bs[sr * kLB + wn + l32];
        const float b1 = Bs[sr * kLB + wn + 32 + l32];
#pragma unroll
        for (int i = 0; i < kMI; ++i) {
          const float av = As[sr * kLA + wm + 32 * i + l32];
          acc[i][0] = __builtin_amdgcn_mfma_f32_32x32x2f32(av, b0, acc[i][0], 0, 0, 0);
          acc[i][1] = __builtin_amdgcn_mfma_f32_32x32x2f32(av, b1, acc[i][1], 0, 0, 0);
        }
      }
    }
    __syncthreads();
  }

  // Gradient tile through LDS into the 16-byte layout of the W tile.
#pragma unroll
  for (int i = 0; i < kMI; ++i)
#pragma unroll
    for (int j = 0; j < 2; ++j)
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int row = wm + 32 * i + 8 * (r >> 2) + 4 * lhi + (r & 3);
        Gt[row * kLB + wn + 32 * j + l32] = acc[i][j][r];
      }
  __syncthreads();
  const float lr = a.lr;
#pragma unroll
  for (int i = 0; i < kWL; ++i) {
    const int rl = wr0 + kXR * i, row = mrow0 + rl;
    if (col_ok && row < a.Mrows) {
      const f32x4 g = *(const f32x4*)&Gt[rl * kLB + 4 * wc4];
      *(f32x4*)(Wp + (int64_t)row * a.ldw + wcol) = wv[i] - lr * g;
    }
  }

  if (nt == 0 && a.bias != nullptr && tid < kUM) {
    const int m = mrow0 + tid;
    if (m < a.Mrows) {
      float sum = 0.0f;
      for (int s = 0; s < a.Kb; ++s) sum += Gp[(int64_t)s * a.ldg + m];
      a.bias[(int64_t)p * a.w_pitch + m] -= a.lr * sum;
    }
  }
}

void launch_update(hipStream_t s, const UpdArgs& a, ASource bsrc) {
  const int mtiles = (a.Mrows + kUM - 1) / kUM;
  const int ntiles = (a.Ncols + kUN - 1) / kUN;
  const unsigned grid = (unsigned)((int64_t)a.P * mtiles * ntiles);
  if (bsrc == A_GATHER)
    launch(k_update_tn<A_GATHER>, grid, 256, 0, s, a, mtiles, ntiles);
  else
    launch(k_update_tn<A_RELU>, grid, 256, 0, s, a, mtiles, ntiles);
}

}  // namespace hav
