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
// k_step_w1:   the update of the first weight block at one step, optionally
//              followed by the mean over each group of SG learners (the local
//              average of Algorithm 1 for this block), and the forward
//              partials of the next step computed from the new tile while it
//              is still on chip, so the block is read and written once per
//              step instead of twice.
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

// Workgroup tile: MB*16 rows (minibatch samples; SG learners' minibatches
// stacked when they share one weight copy) x 128 columns (output units), one K
// split.  Wave w owns columns [32w, 32w + 32) as two 16x16 MFMA blocks.
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
  const int g = bid / (ntiles * mtiles * a.KS);  // row group: learners g*SG ..
  const int GM = a.SG * a.Mp;                     // rows of the group
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
    const int jj = m / a.Mp, sm = m - jj * a.Mp;
    aok[i] = m < GM && sm < a.M;
    const int v = aok[i] ? jj : 0;
    const int64_t p = a.vS > 0 ? (int64_t)(v / a.vS) * a.P + (int64_t)g * a.vS + v % a.vS : (int64_t)g * a.SG + v;
    const int sc = aok[i] ? sm : 0;
    int64_t row;
    if (ASRC == A_GATHER)
      row = a.idx[p * a.M + sc];
    else
      row = p * a.Mp + sc;
    arow[i] = a.A + row * a.lda + 4 * c4;
  }
  const float* wp = a.W + (int64_t)(g / a.wdiv) * a.w_pitch;
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

  const int64_t PT = a.PT > 0 ? a.PT : a.P;
#pragma unroll
  for (int m = 0; m < MB; ++m)
#pragma unroll
    for (int j = 0; j < 2; ++j) {
      if (j == 0 ? !v0 : !v1) continue;
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int row = mbase + 16 * m + 4 * lgrp + r;
        if (row >= GM) continue;
        const int v = row / a.Mp, sm = row - v * a.Mp;
        const int64_t p =
            a.vS > 0 ? (int64_t)(v / a.vS) * a.P + (int64_t)g * a.vS + v % a.vS : (int64_t)g * a.SG + v;
        a.part[(((int64_t)ks * PT + p) * a.Mp + sm) * a.N + nw + 16 * j + lrow] = acc[m][j][r];
      }
    }
}

static int pick_mb(int Mp, int mb_max = 8) {
  const int mb = Mp >= 128 ? 8 : Mp >= 64 ? 4 : Mp >= 32 ? 2 : 1;
  return mb < mb_max ? mb : mb_max;
}

void plan_split(int P, int Mp, int N, int K, int* KS, int* cps, int target_wg, int mb_max) {
  // Enough K splits that the launch has about target_wg workgroups (the GEMMs
  // have few output tiles per learner: M is the minibatch), and no empty split.
  if (target_wg <= 0) target_wg = kFwdTargetWG;
  const int MB = pick_mb(Mp, mb_max);
  const int mtiles = (Mp + MB * 16 - 1) / (MB * 16);
  const int nch = K / kKC;
  const int64_t tiles = (int64_t)P * mtiles * ((N + 127) / 128);
  int ks = (int)std::max<int64_t>(1, (target_wg + tiles - 1) / tiles);
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
  const int GM = a.SG * a.Mp;
  const int MB = pick_mb(GM, a.mb_max);
  const int mtiles = (GM + MB * 16 - 1) / (MB * 16);
  const int ntiles = (a.N + 127) / 128;
  const int groups = a.vS > 0 ? a.P / a.vS : a.P / a.SG;
  const unsigned grid = (unsigned)((int64_t)groups * a.KS * mtiles * ntiles);
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

// Four waves per SIMD (128 registers: the stage and tile registers fit).
template <int BSRC>
__global__ __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(4))) void k_update_tn(UpdArgs a, int mtiles,
                                                                                          int ntiles) {
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
  const float lr = *a.lr;
  // d = g + wd*w; with buffers v <- mu*v + d and the step takes v.
  float* Vp = a.V ? a.V + (int64_t)p * a.w_pitch : nullptr;
#pragma unroll
  for (int i = 0; i < kWL; ++i) {
    const int rl = wr0 + kXR * i, row = mrow0 + rl;
    if (col_ok && row < a.Mrows) {
      f32x4 d = *(const f32x4*)&Gt[rl * kLB + 4 * wc4];
      if (a.wd != 0.0f) d += a.wd * wv[i];
      if (Vp) {
        f32x4* vp = (f32x4*)(Vp + (int64_t)row * a.ldw + wcol);
        d = a.mu * *vp + d;
        *vp = d;
      }
      *(f32x4*)(Wp + (int64_t)row * a.ldw + wcol) = wv[i] - lr * d;
    }
  }

  if (nt == 0 && a.bias != nullptr && tid < kUM) {
    const int m = mrow0 + tid;
    if (m < a.Mrows) {
      float sum = 0.0f;
      for (int s = 0; s < a.Kb; ++s) sum += Gp[(int64_t)s * a.ldg + m];
      float* bp = a.bias + (int64_t)p * a.w_pitch + m;
      const float b = *bp;
      float d = sum + a.wd * b;
      if (a.vbias) {
        float* vp = a.vbias + (int64_t)p * a.w_pitch + m;
        d = a.mu * *vp + d;
        *vp = d;
      }
      *bp = b - lr * d;
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

// ------------------------------------------------------------ fused step
// Workgroup: one 64-row x kSN-column tile range of W1 for one group of SG
// learners, over NT consecutive column tiles (one split of the next step's
// forward contraction).  Per tile:
//   1. for each learner of the group: the update of k_update_tn (the same
//      stage layout; each wave owns a 32 x kSN/2 block of 32x32x2 MFMAs); the
//      new tile stays in registers;
//   2. SG > 1: the group mean of the new tiles (learners in order), written
//      to every learner of the group;
//   3. the new tile goes to LDS; for each learner, its next-step minibatch
//      rows (gathered, this tile's columns) are staged in LDS and the 16x16x4
//      MFMAs add X'[s][cols] . W[h][cols] to the learner's accumulators (same
//      k permutation as k_fwd_nt).
// After the last tile the accumulators are the split's partial sums of the
// next step's first-layer outputs, [split][P][Mp][Mrows].
//
// Loads run one work item ahead: as soon as the registers of the current
// item's stage operands, W tile and next-step rows have been consumed, the
// same registers receive the next item's (the next learner of the group, or
// the next tile), so every load is in flight through at least one block of
// MFMAs.  Past the last item the prefetch reads the last item again (in range,
// cached, unused), so no load depends on a branch.  The sample indices of the
// group are copied to LDS once.  The narrow tile keeps the registers and LDS
// of a workgroup small, so several workgroups share a CU and one's MFMAs run
// while another waits for memory.
#ifndef HAV_STEP_SN
#define HAV_STEP_SN 64
#endif
constexpr int kSN = HAV_STEP_SN;  // W1 columns per tile
static_assert(kSN == 64 || kSN == 128, "fused step tile width");
constexpr int kSL = kSN + 4;      // LDS row length of tile-wide rows
constexpr int kSP = kSN / 4;      // 16-byte pieces per tile-wide row
constexpr int kRP = 256 / kSP;    // tile-wide rows per pass of the workgroup
constexpr int kNA = kSN / 64;     // 32x32 update accumulators per wave
constexpr int kSU = (kUM * kSL > kSC * (kLA + kSL)) ? kUM * kSL : kSC * (kLA + kSL);
#ifndef HAV_STEP_TARGET_WG
#define HAV_STEP_TARGET_WG 768
#endif
constexpr int kStepTargetWG = HAV_STEP_TARGET_WG;
#ifndef HAV_STEP_UNROLL_U
#define HAV_STEP_UNROLL_U 4
#endif
#ifndef HAV_STEP_UNROLL_F
#define HAV_STEP_UNROLL_F 2
#endif
constexpr int kStepMaxB = 64;  // largest minibatch of the fused step

// Occupancy: at least four waves per SIMD for a single learner per group
// (its prefetch registers then fit in 128 VGPRs), three with the group mean
// of up to 8 x 16 forward rows (larger groups would spill).
// FWD = false: the update and the group mean only (no forward of the next
// step, no partials); the next step's forward then runs as one GEMM per
// group from the common result.
template <int SG, int MBF, bool FWD = true>
__global__ __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(!FWD || SG == 1 ? 4 : SG * MBF <= 8 ? 3 : 1))) void k_step_w1(
    StepArgs a, int mtiles, int ntiles, int nchunks) {
  constexpr int MP = MBF * 16;        // rows of the next-step forward (padded minibatch)
  constexpr int kWL = kUM / kRP;      // W pieces per thread
  constexpr int kXL = kSC / kRP;      // stage input pieces per thread
  constexpr int kXN = (MP + kRP - 1) / kRP;  // next-step input pieces per thread
  __shared__ __attribute__((aligned(16))) float lds[kSU + (FWD ? MP * kSL : 0)];
  __shared__ int32_t rows_t[SG][kStepMaxB], rows_n[FWD ? SG : 1][FWD ? kStepMaxB : 1];
  float* As = lds;               // [kSC][kLA] error rows of a stage
  float* Bs = lds + kSC * kLA;   // [kSC][kSL] input rows of a stage
  float* Wt = lds;               // [kUM][kSL] gradient tile, then the new tile
  float* Xs = lds + kSU;         // [MP][kSL] next-step input rows
  const UpdArgs& u = a.u;
  const int bid = xcd_remap(blockIdx.x, gridDim.x);
  const int mt = bid % mtiles;
  const int chunk = (bid / mtiles) % nchunks;
  const int pg = bid / (mtiles * nchunks);
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  const int l32 = lane & 31, lhi = lane >> 5;
  const int lrow = lane & 15, lgrp = lane >> 4;
  const int mrow0 = mt * kUM;
  const int wn = (wave & 1) * (kSN / 2), wm = (wave >> 1) * 32;  // update: the wave's block
  const int pc4 = tid % kSP, pr0 = tid / kSP;            // 16-byte piece of tile-wide rows
  const bool fwd_on = mrow0 + 16 * wave < u.Mrows;       // forward: the wave's 16 rows of W
  const f32x4 zero4 = {0.f, 0.f, 0.f, 0.f};
  const float lr = *u.lr;
  const int Kb = u.Kb;

  for (int e = tid; e < SG * Kb; e += 256) {
    const int64_t g = (int64_t)pg * SG * Kb + e;
    rows_t[e / Kb][e % Kb] = u.idx[g];
    if constexpr (FWD) rows_n[e / Kb][e % Kb] = a.idx_next[g];
  }
  __syncthreads();

  f32x4 ga[2], xb[kXL], wv[kWL], xn[kXN];
  bool gok[2], xok[kXL], xnok[kXN];
  // Stage s0 of item (tile n, learner j): G[s0 .. s0+32)[mrow0 .. +64) and
  // X[idx[s]][tile columns] for s = s0 + pr0 + kRP*i.
  auto load_stage = [&](int n, int j, int s0) {
    const float* Gp = u.G + (int64_t)(pg * SG + j) * u.Mp * u.ldg;
    const int col = n * kSN + 4 * pc4;
    const bool cok = col < u.Ncols;
#pragma unroll
    for (int i = 0; i < 2; ++i) {
      const int q = tid + 256 * i;
      const int s = s0 + (q >> 4), m = mrow0 + 4 * (q & 15);
      gok[i] = s < Kb && m < u.Mrows;
      ga[i] = *(const f32x4*)(Gp + (gok[i] ? (int64_t)s * u.ldg + m : 0));
    }
#pragma unroll
    for (int i = 0; i < kXL; ++i) {
      const int s = s0 + pr0 + kRP * i;
      xok[i] = s < Kb && cok;
      const int64_t row = rows_t[j][s < Kb ? s : 0];
      xb[i] = *(const f32x4*)(u.Bsrc + (xok[i] ? row * u.ldb + col : 0));
    }
  };
  auto store_stage = [&]() {
#pragma unroll
    for (int i = 0; i < 2; ++i) {
      const int q = tid + 256 * i;
      *(f32x4*)&As[(q >> 4) * kLA + 4 * (q & 15)] = gok[i] ? ga[i] : zero4;
    }
#pragma unroll
    for (int i = 0; i < kXL; ++i) *(f32x4*)&Bs[(pr0 + kRP * i) * kSL + 4 * pc4] = xok[i] ? xb[i] : zero4;
  };
  auto load_w = [&](int n, int j) {
    const float* Wp = u.W + (int64_t)(pg * SG + j) * u.w_pitch;
    const int col = n * kSN + 4 * pc4;
#pragma unroll
    for (int i = 0; i < kWL; ++i) {
      const int row = mrow0 + pr0 + kRP * i;
      const bool ok = row < u.Mrows && col < u.Ncols;
      wv[i] = *(const f32x4*)(Wp + (ok ? (int64_t)row * u.ldw + col : 0));
    }
  };
  auto load_next = [&](int n, int j) {  // X'[s][tile columns], s = pr0 + kRP*i
    if constexpr (!FWD) return;
    const int col = n * kSN + 4 * pc4;
    const bool cok = col < u.Ncols;
#pragma unroll
    for (int i = 0; i < kXN; ++i) {
      const int s = pr0 + kRP * i;
      xnok[i] = s < Kb && cok;
      const int64_t row = rows_n[j][s < Kb ? s : 0];
      xn[i] = *(const f32x4*)(u.Bsrc + (xnok[i] ? row * u.ldb + col : 0));
    }
  };

  f32x4 accf[SG][MBF];
#pragma unroll
  for (int j = 0; j < SG; ++j)
#pragma unroll
    for (int b = 0; b < MBF; ++b) accf[j][b] = zero4;
  f32x16 acc[kNA];
  auto mfma_stage = [&](bool on) {
    if (!on) return;
#pragma unroll HAV_STEP_UNROLL_U
    for (int ss = 0; ss < kSC; ss += 2) {
      const int sr = ss + lhi;
      const float av = As[sr * kLA + wm + l32];
#pragma unroll
      for (int jj = 0; jj < kNA; ++jj)
        acc[jj] = __builtin_amdgcn_mfma_f32_32x32x2f32(av, Bs[sr * kSL + wn + 32 * jj + l32], acc[jj], 0, 0, 0);
    }
  };

  const int n_begin = chunk * a.NT, n_end = min(ntiles, n_begin + a.NT);
  load_stage(n_begin, 0, 0);
  load_w(n_begin, 0);
  if constexpr (FWD) load_next(n_begin, 0);
  f32x4 msum[kWL];
  for (int n = n_begin; n < n_end; ++n) {
    const int ncol0 = n * kSN;
    const bool wave_on = ncol0 + wn < u.Ncols;
    const int col = ncol0 + 4 * pc4;
    const bool col_ok = col < u.Ncols;

#pragma unroll 1
    for (int j = 0; j < SG; ++j) {
      // next item: the next learner, else the next tile, else this item again
      const bool more = j + 1 < SG || n + 1 < n_end;
      const int jn = j + 1 < SG ? j + 1 : more ? 0 : j;
      const int nn = j + 1 < SG ? n : more ? n + 1 : n;
#pragma unroll
      for (int jj = 0; jj < kNA; ++jj)
#pragma unroll
        for (int r = 0; r < 16; ++r) acc[jj][r] = 0.0f;
      store_stage();
      for (int s0 = kSC; s0 < Kb; s0 += kSC) {  // minibatches over 32: further stages
        __syncthreads();
        mfma_stage(wave_on);
        __syncthreads();
        load_stage(n, j, s0);
        store_stage();
      }
      load_stage(nn, jn, 0);
      __builtin_amdgcn_sched_barrier(0);  // the prefetch goes out before the MFMAs
      __syncthreads();
      mfma_stage(wave_on);
      __syncthreads();
#pragma unroll
      for (int jj = 0; jj < kNA; ++jj)
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const int row = wm + 8 * (r >> 2) + 4 * lhi + (r & 3);
          Wt[row * kSL + wn + 32 * jj + l32] = acc[jj][r];
        }
      __syncthreads();
      // New tile: each thread reads its gradient pieces and, for SG == 1,
      // writes the new values over them (the same LDS words), so no other
      // thread's data is touched.  Rows past Mrows and columns past Ncols hold
      // zeros in LDS.
      float* Wp = u.W + (int64_t)(pg * SG + j) * u.w_pitch;
#pragma unroll
      for (int i = 0; i < kWL; ++i) {
        const int rl = pr0 + kRP * i, row = mrow0 + rl;
        const bool ok = col_ok && row < u.Mrows;
        f32x4* t = (f32x4*)&Wt[rl * kSL + 4 * pc4];
        const f32x4 wnew = wv[i] - lr * *t;
        if (SG == 1) {
          if (ok) *(f32x4*)(Wp + (int64_t)row * u.ldw + col) = wnew;
          if constexpr (FWD) *t = ok ? wnew : zero4;
        } else {
          msum[i] = j == 0 ? wnew : msum[i] + wnew;
        }
      }
      load_w(nn, jn);
      __builtin_amdgcn_sched_barrier(0);
      if (SG > 1) __syncthreads();  // the next learner's stage overwrites the gradient tile
    }

    if (SG > 1) {
      // SG is a power of two: scaling by 1/SG is exact.
#pragma unroll
      for (int i = 0; i < kWL; ++i) {
        const int rl = pr0 + kRP * i, row = mrow0 + rl;
        const bool ok = col_ok && row < u.Mrows;
        const f32x4 mean = msum[i] * (1.0f / (float)SG);
        if (ok)
          for (int j = 0; j < SG; ++j)
            *(f32x4*)(u.W + (int64_t)(pg * SG + j) * u.w_pitch + (int64_t)row * u.ldw + col) = mean;
        if constexpr (FWD) *(f32x4*)&Wt[rl * kSL + 4 * pc4] = ok ? mean : zero4;
      }
    }
    if constexpr (!FWD) {
      __syncthreads();  // the next tile's stage overwrites the gradient tile
      continue;
    }

    // Forward partials of the next step for every learner of the group.
#pragma unroll
    for (int j = 0; j < SG; ++j) {
#pragma unroll
      for (int i = 0; i < kXN; ++i)
        if (pr0 + kRP * i < MP) *(f32x4*)&Xs[(pr0 + kRP * i) * kSL + 4 * pc4] = xnok[i] ? xn[i] : zero4;
      const bool more = j + 1 < SG || n + 1 < n_end;
      load_next(j + 1 < SG ? n : more ? n + 1 : n, j + 1 < SG ? j + 1 : more ? 0 : j);
      __builtin_amdgcn_sched_barrier(0);
      __syncthreads();
      if (fwd_on) {
#pragma unroll HAV_STEP_UNROLL_F
        for (int q = 0; q < kSN / 16; ++q) {
          const f32x4 b = *(const f32x4*)&Wt[(16 * wave + lrow) * kSL + 16 * q + 4 * lgrp];
          f32x4 af[MBF];
#pragma unroll
          for (int m = 0; m < MBF; ++m) af[m] = *(const f32x4*)&Xs[(16 * m + lrow) * kSL + 16 * q + 4 * lgrp];
#pragma unroll
          for (int i = 0; i < 4; ++i)
#pragma unroll
            for (int m = 0; m < MBF; ++m)
              accf[j][m] = __builtin_amdgcn_mfma_f32_16x16x4f32(af[m][i], b[i], accf[j][m], 0, 0, 0);
        }
      }
      __syncthreads();
    }
  }

  if (FWD && fwd_on) {
    const int h = mrow0 + 16 * wave + lrow;
#pragma unroll
    for (int j = 0; j < SG; ++j) {
      float* part = a.part + ((int64_t)chunk * u.P + pg * SG + j) * u.Mp * u.Mrows;
#pragma unroll
      for (int m = 0; m < MBF; ++m)
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const int s = 16 * m + 4 * lgrp + r;
          if (s < u.Mp) part[(int64_t)s * u.Mrows + h] = accf[j][m][r];
        }
    }
  }
  // Bias step (softmax model, large-C MLP), once per learner and row tile.
  if (chunk == 0 && u.bias != nullptr && tid < kUM) {
    const int m = mrow0 + tid;
    if (m < u.Mrows)
      for (int j = 0; j < SG; ++j) {
        const int p = pg * SG + j;
        const float* Gp = u.G + (int64_t)p * u.Mp * u.ldg;
        float sum = 0.0f;
        for (int s = 0; s < Kb; ++s) sum += Gp[(int64_t)s * u.ldg + m];
        u.bias[(int64_t)p * u.w_pitch + m] -= lr * sum;
      }
  }
}

// Full-tile form of k_step_w1 for SG = 1: every sample, row and column of
// the launch in range (B a multiple of 32, Mrows of 64, Ncols of kSN) and the
// dataset, the learner's error rows and its weight block each below 4 GiB.
// Every global access is a buffer access: a per-lane 32-bit byte offset that
// stays fixed for the whole kernel (the gathered rows' offsets are read from
// LDS once) plus a wave-uniform offset in a scalar register (the tile's
// column, the piece's row group).  Nothing is selected or bounds-checked per
// tile, so the tile loop runs the MFMAs, the update itself and the LDS
// traffic and next to no other vector instruction (on gfx950 those stall
// the SIMD's matrix core).  The whole input tile of the step is loaded one
// tile ahead.  The step's error rows of the row tile sit
// in LDS for the whole workgroup (they do not depend on the column tile), and
// the waves raise their priority over the MFMA loops so that the SIMD keeps
// issuing MFMAs while other workgroups stage data.  Same tiles, operand
// layouts, k order and outputs as k_step_w1.
template <int MBF>
__global__ __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(MBF > 2 ? 3 : 4))) void k_step_w1_full(
    StepArgs a, int mtiles, int ntiles, int nchunks) {
  constexpr int MP = MBF * 16;   // samples of a step (= Kb = Mp)
  constexpr int kWL = kUM / kRP;
  constexpr int kXN = MP / kRP;  // pieces per thread of a 64-column tile of MP rows
  constexpr int kGL = MP * 16 / 256;  // pieces per thread of the G tile (MP rows x 64 units)
  constexpr int kUF = MBF > 2 ? 1 : HAV_STEP_UNROLL_F;  // forward unroll (64 samples: register pressure)
  constexpr int kBR = MP > kUM ? MP : kUM;
  static_assert(MP % kSC == 0 && kXN * kRP == MP, "full-tile step shapes");
  // Gs: the step's errors of this row tile (constant over the column tiles);
  // Bs: the tile's input rows, then (aliased) the gradient / new tile Wt;
  // Xs: the next step's input rows of the tile.
  __shared__ __attribute__((aligned(16))) float Gs[MP * kLA];
  __shared__ __attribute__((aligned(16))) float Bs[kBR * kSL];
  __shared__ __attribute__((aligned(16))) float Xs[MP * kSL];
  __shared__ uint32_t roff_t[MP], roff_n[MP];
  float* Wt = Bs;
  const UpdArgs& u = a.u;
  const int bid = xcd_remap(blockIdx.x, gridDim.x);
  const int mt = bid % mtiles;
  const int chunk = (bid / mtiles) % nchunks;
  const int p = bid / (mtiles * nchunks);
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  const int l32 = lane & 31, lhi = lane >> 5;
  const int lrow = lane & 15, lgrp = lane >> 4;
  const int mrow0 = mt * kUM;
  const int wn = (wave & 1) * (kSN / 2), wm = (wave >> 1) * 32;
  const int pc4 = tid % kSP, pr0 = tid / kSP;
  const float lr = *u.lr;

  // Byte offsets of this learner's gathered rows (this step and the next).
  for (int e = tid; e < MP; e += 256) {
    roff_t[e] = (uint32_t)((uint64_t)u.idx[(int64_t)p * MP + e] * (uint64_t)u.ldb * 4u);
    roff_n[e] = (uint32_t)((uint64_t)a.idx_next[(int64_t)p * MP + e] * (uint64_t)u.ldb * 4u);
  }
  const __amdgpu_buffer_rsrc_t rG =
      buf_rsrc(u.G + (int64_t)p * u.Mp * u.ldg + mrow0, (uint64_t)u.Mp * u.ldg * 4);
  const __amdgpu_buffer_rsrc_t rW =
      buf_rsrc(u.W + (int64_t)p * u.w_pitch + (int64_t)mrow0 * u.ldw, (uint64_t)kUM * u.ldw * 4);
  const __amdgpu_buffer_rsrc_t rWi =
      a.w_src ? buf_rsrc(a.w_src + (int64_t)(p / a.src_group) * a.src_pitch + (int64_t)mrow0 * u.ldw,
                         (uint64_t)kUM * u.ldw * 4)
              : rW;
  const __amdgpu_buffer_rsrc_t rX = buf_rsrc(u.Bsrc, (uint64_t)a.x_rows * u.ldb * 4);
  {
    // G[s][mrow0 + 4pc4], s = pr0 + 16i, once for the whole workgroup.
    const uint32_t vo_g = (uint32_t)(pr0 * u.ldg + 4 * pc4) * 4u;
    f32x4 g[kGL];
#pragma unroll
    for (int i = 0; i < kGL; ++i) g[i] = buf_ld16(rG, vo_g, i * kRP * (int)u.ldg * 4);
#pragma unroll
    for (int i = 0; i < kGL; ++i) *(f32x4*)&Gs[(pr0 + kRP * i) * kLA + 4 * pc4] = g[i];
  }
  __syncthreads();
  uint32_t xo_t[kXN], xo_n[kXN];
#pragma unroll
  for (int i = 0; i < kXN; ++i) {
    xo_t[i] = roff_t[pr0 + kRP * i] + 16u * pc4;
    xo_n[i] = roff_n[pr0 + kRP * i] + 16u * pc4;
  }
  const uint32_t vo_w = (uint32_t)(pr0 * u.ldw + 4 * pc4) * 4u;  // W[mrow0 + pr0 + 16i][n*kSN + 4pc4]
  const int w16 = kRP * (int)u.ldw * 4;

  f32x4 xb[kXN], wv[kWL], xn[kXN];
  auto load_x = [&](int n) {
#pragma unroll
    for (int i = 0; i < kXN; ++i) xb[i] = buf_ld16(rX, xo_t[i], n * kSN * 4);
  };
  auto load_w = [&](int n) {
#pragma unroll
    for (int i = 0; i < kWL; ++i) wv[i] = buf_ld16(rWi, vo_w, n * kSN * 4 + i * w16);
  };
  auto load_next = [&](int n) {
#pragma unroll
    for (int i = 0; i < kXN; ++i) xn[i] = buf_ld16(rX, xo_n[i], n * kSN * 4);
  };

  const f32x4 zero4 = {0.f, 0.f, 0.f, 0.f};
  f32x4 accf[MBF];
#pragma unroll
  for (int b = 0; b < MBF; ++b) accf[b] = zero4;
  f32x16 acc[kNA];

  const int n_begin = chunk * a.NT, n_end = min(ntiles, n_begin + a.NT);
  load_x(n_begin);
  load_w(n_begin);
  load_next(n_begin);
  for (int n = n_begin; n < n_end; ++n) {
    const int nn = n + 1 < n_end ? n + 1 : n;  // the last tile loads itself again: in range, unused
#pragma unroll
    for (int i = 0; i < kXN; ++i) *(f32x4*)&Bs[(pr0 + kRP * i) * kSL + 4 * pc4] = xb[i];
    load_x(nn);
#pragma unroll
    for (int jj = 0; jj < kNA; ++jj)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[jj][r] = 0.0f;
    __builtin_amdgcn_sched_barrier(0);
    __syncthreads();
    __builtin_amdgcn_s_setprio(1);
#pragma unroll HAV_STEP_UNROLL_U
    for (int ss = 0; ss < MP; ss += 2) {
      const int sr = ss + lhi;
      const float av = Gs[sr * kLA + wm + l32];
#pragma unroll
      for (int jj = 0; jj < kNA; ++jj)
        acc[jj] = __builtin_amdgcn_mfma_f32_32x32x2f32(av, Bs[sr * kSL + wn + 32 * jj + l32], acc[jj], 0, 0, 0);
    }
    __builtin_amdgcn_s_setprio(0);
    __syncthreads();
#pragma unroll
    for (int jj = 0; jj < kNA; ++jj)
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int row = wm + 8 * (r >> 2) + 4 * lhi + (r & 3);
        Wt[row * kSL + wn + 32 * jj + l32] = acc[jj][r];
      }
    __syncthreads();
    // New tile: each thread overwrites its own gradient pieces with the new
    // values and stores them.
#pragma unroll
    for (int i = 0; i < kWL; ++i) {
      f32x4* t = (f32x4*)&Wt[(pr0 + kRP * i) * kSL + 4 * pc4];
      const f32x4 wnew = wv[i] - lr * *t;
      buf_st16(rW, vo_w, n * kSN * 4 + i * w16, wnew);
      *t = wnew;
    }
    load_w(nn);
#pragma unroll
    for (int i = 0; i < kXN; ++i) *(f32x4*)&Xs[(pr0 + kRP * i) * kSL + 4 * pc4] = xn[i];
    load_next(nn);
    __builtin_amdgcn_sched_barrier(0);
    __syncthreads();
    __builtin_amdgcn_s_setprio(1);
#pragma unroll kUF
    for (int q = 0; q < kSN / 16; ++q) {
      const f32x4 b = *(const f32x4*)&Wt[(16 * wave + lrow) * kSL + 16 * q + 4 * lgrp];
      f32x4 af[MBF];
#pragma unroll
      for (int m = 0; m < MBF; ++m) af[m] = *(const f32x4*)&Xs[(16 * m + lrow) * kSL + 16 * q + 4 * lgrp];
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int m = 0; m < MBF; ++m) accf[m] = __builtin_amdgcn_mfma_f32_16x16x4f32(af[m][i], b[i], accf[m], 0, 0, 0);
    }
    __builtin_amdgcn_s_setprio(0);
    __syncthreads();
  }

  {
    const int h = mrow0 + 16 * wave + lrow;
    float* part = a.part + ((int64_t)chunk * u.P + p) * u.Mp * u.Mrows;
#pragma unroll
    for (int m = 0; m < MBF; ++m)
#pragma unroll
      for (int r = 0; r < 4; ++r) part[(int64_t)(16 * m + 4 * lgrp + r) * u.Mrows + h] = accf[m][r];
  }
  if (chunk == 0 && u.bias != nullptr && tid < kUM) {
    const int m = mrow0 + tid;
    const float* Gp = u.G + (int64_t)p * u.Mp * u.ldg;
    float sum = 0.0f;
    for (int s = 0; s < MP; ++s) sum += Gp[(int64_t)s * u.ldg + m];
    u.bias[(int64_t)p * u.w_pitch + m] -= lr * sum;
  }
}

// Full-tile update with the group mean (no forward) for groups of SG
// learners: per 64-column tile, each learner's new tile W_j - lr * G_j^T X_j
// (the update of k_step_w1_full), added in learner order and scaled by 1/SG
// (SG a power of two: exact), the mean written to every learner's row (or
// once, to w_dst).  Per
// learner the errors and input rows of the tile are staged through LDS while
// the next learner's are loaded; every global access is a buffer access with
// a fixed per-lane offset (the gathered rows' byte offsets from LDS) and a
// scalar offset.  Same launch conditions as k_step_w1_full.
template <int SG>
__global__ __launch_bounds__(256) void k_step_mean_full(StepArgs a, int mtiles, int ntiles, int nchunks) {
  constexpr int MP = 64;            // largest minibatch of the full-tile forms
  constexpr int kWL = kUM / kRP;    // W pieces per thread (4)
  constexpr int kXL = MP / kRP;     // G and X pieces per thread (4 each, 64 rows)
  __shared__ __attribute__((aligned(16))) float Gs[MP * kLA];  // then the gradient tile Wt
  __shared__ __attribute__((aligned(16))) float Bs[MP * kSL];
  __shared__ uint32_t roff[SG][MP];
  float* Wt = Gs;
  static_assert(kUM * kSL <= MP * kLA, "gradient tile fits in the error stage");
  const UpdArgs& u = a.u;
  const int bid = xcd_remap(blockIdx.x, gridDim.x);
  const int mt = bid % mtiles;
  const int chunk = (bid / mtiles) % nchunks;
  const int pg = bid / (mtiles * nchunks);
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  const int l32 = lane & 31, lhi = lane >> 5;
  const int mrow0 = mt * kUM;
  const int wn = (wave & 1) * (kSN / 2), wm = (wave >> 1) * 32;
  const int pc4 = tid % kSP, pr0 = tid / kSP;
  const float lr = *u.lr;
  const int Kb = u.Kb;  // = u.Mp, a multiple of 32 up to MP
  for (int e = tid; e < SG * Kb; e += 256)
    roff[e / Kb][e % Kb] = (uint32_t)((uint64_t)u.idx[(int64_t)pg * SG * Kb + e] * (uint64_t)u.ldb * 4u);
  __syncthreads();
  const uint32_t vo_g = (uint32_t)(pr0 * u.ldg + 4 * pc4) * 4u;
  const uint32_t vo_w = (uint32_t)(pr0 * u.ldw + 4 * pc4) * 4u;
  const int g16 = kRP * (int)u.ldg * 4, w16 = kRP * (int)u.ldw * 4;
  const __amdgpu_buffer_rsrc_t rX = buf_rsrc(u.Bsrc, (uint64_t)a.x_rows * u.ldb * 4);
  auto rG = [&](int j) {
    return buf_rsrc(u.G + (int64_t)(pg * SG + j) * u.Mp * u.ldg + mrow0, (uint64_t)u.Mp * u.ldg * 4);
  };
  auto rW = [&](int j) {
    return buf_rsrc(u.W + (int64_t)(pg * SG + j) * u.w_pitch + (int64_t)mrow0 * u.ldw, (uint64_t)kUM * u.ldw * 4);
  };
  auto rWi = [&](int j) {  // learner j's old block
    return a.w_src ? buf_rsrc(a.w_src + (int64_t)((pg * SG + j) / a.src_group) * a.src_pitch +
                                  (int64_t)mrow0 * u.ldw,
                              (uint64_t)kUM * u.ldw * 4)
                   : rW(j);
  };
  const int nst = Kb / kRP;  // 16-row passes of the minibatch (2 or 4)

  f32x4 ga[kXL], xb[kXL], wv[kWL], msum[kWL];
  auto load_item = [&](int n, int j) {  // errors and input rows of learner j, tile n
    const __amdgpu_buffer_rsrc_t r = rG(j);
#pragma unroll
    for (int i = 0; i < kXL; ++i) {
      const int ii = i < nst ? i : 0;  // passes past the minibatch repeat pass 0 (not stored)
      ga[i] = buf_ld16(r, vo_g, ii * g16);
      xb[i] = buf_ld16(rX, roff[j][pr0 + kRP * ii] + 16u * pc4, n * kSN * 4);
    }
  };
  auto load_w = [&](int n, int j) {
    const __amdgpu_buffer_rsrc_t r = rWi(j);
#pragma unroll
    for (int i = 0; i < kWL; ++i) wv[i] = buf_ld16(r, vo_w, n * kSN * 4 + i * w16);
  };
  f32x16 acc[kNA];

  const int n_begin = chunk * a.NT, n_end = min(ntiles, n_begin + a.NT);
  load_item(n_begin, 0);
  load_w(n_begin, 0);
  for (int n = n_begin; n < n_end; ++n) {
#pragma unroll 1
    for (int j = 0; j < SG; ++j) {
      // next item: the next learner, else the next tile, else this item again
      const bool more = j + 1 < SG || n + 1 < n_end;
      const int jn = j + 1 < SG ? j + 1 : more ? 0 : j;
      const int nn = j + 1 < SG ? n : more ? n + 1 : n;
#pragma unroll
      for (int i = 0; i < kXL; ++i)
        if (i < nst) {
          *(f32x4*)&Gs[(pr0 + kRP * i) * kLA + 4 * pc4] = ga[i];
          *(f32x4*)&Bs[(pr0 + kRP * i) * kSL + 4 * pc4] = xb[i];
        }
      load_item(nn, jn);
#pragma unroll
      for (int jj = 0; jj < kNA; ++jj)
#pragma unroll
        for (int r = 0; r < 16; ++r) acc[jj][r] = 0.0f;
      __builtin_amdgcn_sched_barrier(0);
      __syncthreads();
      __builtin_amdgcn_s_setprio(1);
      for (int s0 = 0; s0 < Kb; s0 += kSC) {  // 32-sample stages, each fully unrolled
#pragma unroll
        for (int ss = 0; ss < kSC; ss += 2) {
          const int sr = s0 + ss + lhi;
          const float av = Gs[sr * kLA + wm + l32];
#pragma unroll
          for (int jj = 0; jj < kNA; ++jj)
            acc[jj] = __builtin_amdgcn_mfma_f32_32x32x2f32(av, Bs[sr * kSL + wn + 32 * jj + l32], acc[jj], 0, 0, 0);
        }
      }
      __builtin_amdgcn_s_setprio(0);
      __syncthreads();
#pragma unroll
      for (int jj = 0; jj < kNA; ++jj)
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const int row = wm + 8 * (r >> 2) + 4 * lhi + (r & 3);
          Wt[row * kSL + wn + 32 * jj + l32] = acc[jj][r];
        }
      __syncthreads();
#pragma unroll
      for (int i = 0; i < kWL; ++i) {
        const f32x4 wnew = wv[i] - lr * *(const f32x4*)&Wt[(pr0 + kRP * i) * kSL + 4 * pc4];
        msum[i] = j == 0 ? wnew : msum[i] + wnew;
      }
      load_w(nn, jn);
      __syncthreads();  // the next item's stage overwrites the gradient tile
    }
#pragma unroll
    for (int i = 0; i < kWL; ++i) msum[i] = msum[i] * (1.0f / (float)SG);
    if (a.w_dst) {  // the group's mean once (a tile's loads above all precede its store)
      const __amdgpu_buffer_rsrc_t r =
          buf_rsrc(a.w_dst + (int64_t)pg * a.dst_pitch + (int64_t)mrow0 * u.ldw, (uint64_t)kUM * u.ldw * 4);
#pragma unroll
      for (int i = 0; i < kWL; ++i) buf_st16(r, vo_w, n * kSN * 4 + i * w16, msum[i]);
    } else {
      for (int j = 0; j < SG; ++j) {
        const __amdgpu_buffer_rsrc_t r = rW(j);
#pragma unroll
        for (int i = 0; i < kWL; ++i) buf_st16(r, vo_w, n * kSN * 4 + i * w16, msum[i]);
      }
    }
  }
  // Bias step (more than 32 classes), once per learner and row tile.
  if (chunk == 0 && u.bias != nullptr && tid < kUM) {
    const int m = mrow0 + tid;
    for (int j = 0; j < SG; ++j) {
      const int p = pg * SG + j;
      const float* Gp = u.G + (int64_t)p * u.Mp * u.ldg;
      float sum = 0.0f;
      for (int s = 0; s < Kb; ++s) sum += Gp[(int64_t)s * u.ldg + m];
      u.bias[(int64_t)p * u.w_pitch + m] -= lr * sum;
    }
  }
}

bool step_w1_supported(int Mp, int SG) {
  if (Mp < 1 || Mp > kStepMaxB || Mp % 16 != 0) return false;
  if (SG != 1 && SG != 2 && SG != 4 && SG != 8) return false;
  return SG * (Mp / 16) <= 16;
}

bool step_w1_mean_supported(int Mp, int SG) {
  return Mp >= 1 && Mp <= kStepMaxB && Mp % 16 == 0 && SG >= 2 && SG <= 64 && (SG & (SG - 1)) == 0;
}

#ifndef HAV_STEP_TARGET_WG64
#define HAV_STEP_TARGET_WG64 1536
#endif
// Workgroups a step launch aims for: about four per CU, or two waves of three
// per CU for 64-sample steps of one learner (the full-tile kernel's LDS
// allows three workgroups per CU there).
#ifndef HAV_STEP_TARGET_MEAN
#define HAV_STEP_TARGET_MEAN 1536
#endif
static int step_target(int SG, int Mp) { return SG == 1 && Mp == 64 ? HAV_STEP_TARGET_WG64 : kStepTargetWG; }

// no_fwd: the update with the group mean alone (its column chunks write no
// forward partials), with a grid target of its own.
static void step_plan(int P, int SG, int Mp, int Mrows, int Ncols, int* mtiles, int* ntiles, int* nchunks, int* NT,
                      bool no_fwd = false) {
  *mtiles = (Mrows + kUM - 1) / kUM;
  *ntiles = (Ncols + kSN - 1) / kSN;
  const int64_t base = (int64_t)(P / SG) * *mtiles;
  const int target = no_fwd ? HAV_STEP_TARGET_MEAN : step_target(SG, Mp);
  int nc = (int)std::min<int64_t>(*ntiles, std::max<int64_t>(1, (target + base - 1) / base));
  *NT = (*ntiles + nc - 1) / nc;
  *nchunks = (*ntiles + *NT - 1) / *NT;
}

bool step_full_shape(int Kb, int Mp, int Mrows, int Ncols, int64_t x_rows, int64_t ldb, int64_t ldg, int64_t ldw) {
  const uint64_t lim = 0xffffffffull;
  return Kb == Mp && Mp % kSC == 0 && Mp <= kStepMaxB && Mrows % kUM == 0 && Ncols % kSN == 0 && x_rows > 0 &&
         (uint64_t)x_rows * ldb * 4 < lim && (uint64_t)Mp * ldg * 4 < lim && (uint64_t)kUM * ldw * 4 < lim;
}

int step_w1_splits(int P, int SG, int Mp, int Mrows, int Ncols) {
  int mt, ntl, nc, NT;
  step_plan(P, SG, Mp, Mrows, Ncols, &mt, &ntl, &nc, &NT);
  return nc;
}

bool launch_step_w1(hipStream_t s, StepArgs a) {
  int mtiles, ntiles, nchunks;
  step_plan(a.u.P, a.SG, a.u.Mp, a.u.Mrows, a.u.Ncols, &mtiles, &ntiles, &nchunks, &a.NT, a.no_fwd);
  const unsigned grid = (unsigned)((int64_t)(a.u.P / a.SG) * mtiles * nchunks);
  const bool full =
      step_full_shape(a.u.Kb, a.u.Mp, a.u.Mrows, a.u.Ncols, a.x_rows, a.u.ldb, a.u.ldg, a.u.ldw);
  if ((a.w_src || a.w_dst) && !(full && (a.no_fwd || a.SG == 1))) return false;  // only the full-tile kernels redirect
  if (a.no_fwd && full) {
    switch (a.SG) {
      case 2: launch(k_step_mean_full<2>, grid, 256, 0, s, a, mtiles, ntiles, nchunks); break;
      case 4: launch(k_step_mean_full<4>, grid, 256, 0, s, a, mtiles, ntiles, nchunks); break;
      case 8: launch(k_step_mean_full<8>, grid, 256, 0, s, a, mtiles, ntiles, nchunks); break;
      case 16: launch(k_step_mean_full<16>, grid, 256, 0, s, a, mtiles, ntiles, nchunks); break;
      case 32: launch(k_step_mean_full<32>, grid, 256, 0, s, a, mtiles, ntiles, nchunks); break;
      default: launch(k_step_mean_full<64>, grid, 256, 0, s, a, mtiles, ntiles, nchunks); break;
    }
    return true;
  }
  if (a.no_fwd) {
    switch (a.SG) {
      case 2: launch(k_step_w1<2, 1, false>, grid, 256, 0, s, a, mtiles, ntiles, nchunks); break;
      case 4: launch(k_step_w1<4, 1, false>, grid, 256, 0, s, a, mtiles, ntiles, nchunks); break;
      case 8: launch(k_step_w1<8, 1, false>, grid, 256, 0, s, a, mtiles, ntiles, nchunks); break;
      case 16: launch(k_step_w1<16, 1, false>, grid, 256, 0, s, a, mtiles, ntiles, nchunks); break;
      case 32: launch(k_step_w1<32, 1, false>, grid, 256, 0, s, a, mtiles, ntiles, nchunks); break;
      default: launch(k_step_w1<64, 1, false>, grid, 256, 0, s, a, mtiles, ntiles, nchunks); break;
    }
    return true;
  }
  if (full && a.SG == 1) {
    if (a.u.Mp == 32)
      launch(k_step_w1_full<2>, grid, 256, 0, s, a, mtiles, ntiles, nchunks);
    else
      launch(k_step_w1_full<4>, grid, 256, 0, s, a, mtiles, ntiles, nchunks);
    return true;
  }
#define HAV_STEP(SG_, MBF_) launch(k_step_w1<SG_, MBF_>, grid, 256, 0, s, a, mtiles, ntiles, nchunks)
#define HAV_STEP_MBF(SG_)           \
  switch (a.u.Mp / 16) {            \
    case 1: HAV_STEP(SG_, 1); break; \
    case 2: HAV_STEP(SG_, 2); break; \
    case 3: HAV_STEP(SG_, 3); break; \
    default: HAV_STEP(SG_, 4); break; \
  }
  switch (a.SG) {
    case 1: HAV_STEP_MBF(1) break;
    case 2: HAV_STEP_MBF(2) break;
    case 4: HAV_STEP_MBF(4) break;
    default:
      if (a.u.Mp / 16 == 1)
        HAV_STEP(8, 1);
      else
        HAV_STEP(8, 2);
      break;
  }
#undef HAV_STEP_MBF
#undef HAV_STEP
  return true;
}

}  // namespace hav
