// Per-learner dense contractions of one local SGD step (Algorithm 1, Sec. 3.1:
// each learner's minibatch gradient of the softmax cross-entropy, followed by
// w <- w - lr * g), batched over the P learners and run on fp32 MFMA.
//
// k_fwd_nt:    part[ks][p][m][n] = sum_{k in split ks} A_p[m][k] * W_p[n][k]
//              (A = gathered minibatch rows of X, or ReLU of the hidden
//              pre-activations; W = a weight block, K-contiguous).  Split-K
//              partials are summed later in a fixed order, so results are
//              deterministic.
// k_update_tn: W_p[m][n] -= lr * sum_s G_p[s][m] * Bsrc_p[s][n], the weight
//              gradient of a layer fused with the SGD update (the gradient is
//              never stored), plus b_p[m] -= lr * sum_s G_p[s][m].
#include <algorithm>

#include "internal.h"

namespace hav {

constexpr int kKC = 32;         // K floats per pipeline stage of k_fwd_nt
constexpr int kLdsStride = 36;  // LDS row stride in floats (32 + 4: conflict-free 128-bit reads)

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
// 4*(l/16)), prefetched one stage ahead.  Within a 16-wide k group the four
// MFMAs take k = 4g + i (g = lane group, i = MFMA index): a permutation of the
// k order that A and W share, so the contraction is unchanged.
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

  const float* arow[LPT];
  int lds_off[LPT];
  bool aload[LPT];
#pragma unroll
  for (int i = 0; i < LPT; ++i) {
    const int q = tid + 256 * i;
    aload[i] = q < NLOAD;
    const int r = q >> 3, c4 = q & 7;
    lds_off[i] = r * kLdsStride + 4 * c4;
    const float* src = nullptr;
    const int m = mbase + r;
    if (aload[i] && m < a.M) {
      if (ASRC == A_GATHER)
        src = a.A + (int64_t)a.idx[(int64_t)p * a.M + m] * a.lda;
      else
        src = a.A + ((int64_t)p * a.Mp + m) * a.lda;
      src += 4 * c4;
    }
    arow[i] = src;
  }
  const float* wp = a.W + (int64_t)p * a.w_pitch;
  const float* wrow0 = wp + (int64_t)(nw + lrow) * a.ldw + 4 * lgrp;
  const float* wrow1 = wrow0 + 16 * a.ldw;

  f32x4 acc[MB][2];
#pragma unroll
  for (int m = 0; m < MB; ++m) acc[m][0] = acc[m][1] = f32x4{0.f, 0.f, 0.f, 0.f};
  f32x4 ar[LPT];
  f32x4 wc[2][2], wn[2][2];
  const f32x4 zero4 = {0.f, 0.f, 0.f, 0.f};

  auto load_a = [&](int c) {
#pragma unroll
    for (int i = 0; i < LPT; ++i) {
      f32x4 v = zero4;
      if (arow[i]) v = *(const f32x4*)(arow[i] + (int64_t)c * kKC);
      ar[i] = ASRC == A_RELU ? relu4(v) : v;
    }
  };
  auto store_a = [&](int buf) {
#pragma unroll
    for (int i = 0; i < LPT; ++i)
      if (aload[i]) *(f32x4*)&As[buf][lds_off[i]] = ar[i];
  };
  auto load_w = [&](int c, f32x4 (&w)[2][2]) {
    const int64_t o = (int64_t)c * kKC;
    if (v0) {
      w[0][0] = *(const f32x4*)(wrow0 + o);
      w[0][1] = *(const f32x4*)(wrow0 + o + 16);
    }
    if (v1) {
      w[1][0] = *(const f32x4*)(wrow1 + o);
      w[1][1] = *(const f32x4*)(wrow1 + o + 16);
    }
  };

  if (c0 < c1) {
    load_a(c0);
    store_a(0);
    load_w(c0, wc);
    __syncthreads();
    for (int c = c0; c < c1; ++c) {
      const int buf = (c - c0) & 1;
      const bool more = c + 1 < c1;
      if (more) {
        load_a(c + 1);
        load_w(c + 1, wn);
      }
      if (v0) {
#pragma unroll
        for (int h = 0; h < 2; ++h) {
          f32x4 af[MB];
#pragma unroll
          for (int m = 0; m < MB; ++m)
            af[m] = *(const f32x4*)&As[buf][(16 * m + lrow) * kLdsStride + 16 * h + 4 * lgrp];
#pragma unroll
          for (int i = 0; i < 4; ++i) {
#pragma unroll
            for (int m = 0; m < MB; ++m) {
              acc[m][0] = __builtin_amdgcn_mfma_f32_16x16x4f32(af[m][i], wc[0][h][i], acc[m][0], 0, 0, 0);
              if (v1) acc[m][1] = __builtin_amdgcn_mfma_f32_16x16x4f32(af[m][i], wc[1][h][i], acc[m][1], 0, 0, 0);
            }
          }
        }
      }
      if (more) store_a(buf ^ 1);
      __syncthreads();
#pragma unroll
      for (int j = 0; j < 2; ++j) {
        wc[j][0] = wn[j][0];
        wc[j][1] = wn[j][1];
      }
    }
  }

  float* out = a.part + ((int64_t)ks * a.P + p) * a.Mp * a.N;
#pragma unroll
  for (int m = 0; m < MB; ++m) {
#pragma unroll
    for (int j = 0; j < 2; ++j) {
      if (j == 0 ? !v0 : !v1) continue;
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int row = mbase + 16 * m + 4 * lgrp + r;
        if (row < a.Mp) out[(int64_t)row * a.N + nw + 16 * j + lrow] = acc[m][j][r];
      }
    }
  }
}

static int pick_mb(int Mp) { return Mp >= 128 ? 8 : Mp >= 64 ? 4 : Mp >= 32 ? 2 : 1; }

void plan_split(int P, int N, int K, int* KS, int* cps) {
  // Enough K splits that the launch has about 512 workgroups (the GEMMs have
  // few output tiles per learner: M is the minibatch), and no empty split.
  const int nch = K / kKC;
  const int64_t tiles = (int64_t)P * ((N + 127) / 128);
  int ks = (int)std::max<int64_t>(1, (512 + tiles - 1) / tiles);
  ks = std::min(ks, nch);
  const int c = (nch + ks - 1) / ks;
  *KS = (nch + c - 1) / c;
  *cps = c;
}

void launch_fwd(hipStream_t s, const FwdArgs& a, ASource src) {
  const int MB = pick_mb(a.Mp);
  const int mtiles = (a.Mp + MB * 16 - 1) / (MB * 16);
  const int ntiles = (a.N + 127) / 128;
  const unsigned grid = (unsigned)((int64_t)a.P * a.KS * mtiles * ntiles);
#define HAV_FWD(S_, MB_) k_fwd_nt<S_, MB_><<<grid, 256, 0, s>>>(a, ntiles, mtiles)
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

// Workgroup tile 64 (rows m of W) x 128 (columns n of W); wave w owns rows
// [32*(w/2), +32) and columns [64*(w%2), +64) as two 32x32 MFMA blocks.  The
// contraction runs over the minibatch (K = B), two samples per 32x32x2 MFMA:
// lane l supplies G[s + l/32][m0 + l%32] and Bsrc[s + l/32][n0 + l%32], both
// 128-byte coalesced rows.  The W tile is loaded before the contraction so its
// latency overlaps the MFMAs, then updated in place in the accumulator layout
// (lane l, register r: row 8*(r/4) + 4*(l/32) + r%4, column l%32).
template <int BSRC>
__global__ __launch_bounds__(256) void k_update_tn(UpdArgs a, int mtiles, int ntiles) {
  const int bid = xcd_remap(blockIdx.x, gridDim.x);
  const int nt = bid % ntiles;
  const int mt = (bid / ntiles) % mtiles;
  const int p = bid / (ntiles * mtiles);
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  const int l32 = lane & 31, lhi = lane >> 5;
  const int m0 = mt * 64 + (wave >> 1) * 32;
  const int n0 = nt * 128 + (wave & 1) * 64;
  const bool vb0 = n0 < a.Ncols, vb1 = n0 + 32 < a.Ncols;
  float* Wp = a.W + (int64_t)p * a.w_pitch;
  const float* Gp = a.G + (int64_t)p * a.Mp * a.ldg;

  if (m0 < a.Mrows && vb0) {
    f32x16 w0, w1;
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      const int row = m0 + 8 * (r >> 2) + 4 * lhi + (r & 3);
      const bool ok = row < a.Mrows;
      const float* wr = Wp + (int64_t)row * a.ldw + n0 + l32;
      w0[r] = ok ? wr[0] : 0.0f;
      w1[r] = (ok && vb1) ? wr[32] : 0.0f;
    }
    f32x16 acc0, acc1;
#pragma unroll
    for (int r = 0; r < 16; ++r) acc0[r] = acc1[r] = 0.0f;
    const bool mok = m0 + l32 < a.Mrows;
#pragma unroll 8
    for (int s = 0; s < a.Kb; s += 2) {
      const int ss = s + lhi;
      const bool sok = ss < a.Kb;
      const float av = (sok && mok) ? Gp[(int64_t)ss * a.ldg + m0 + l32] : 0.0f;
      float b0 = 0.0f, b1 = 0.0f;
      if (sok) {
        const float* br = BSRC == A_GATHER ? a.Bsrc + (int64_t)a.idx[(int64_t)p * a.Kb + ss] * a.ldb
                                           : a.Bsrc + ((int64_t)p * a.Mp + ss) * a.ldb;
        b0 = br[n0 + l32];
        if (vb1) b1 = br[n0 + 32 + l32];
        if (BSRC == A_RELU) {
          b0 = fmaxf(b0, 0.0f);
          b1 = fmaxf(b1, 0.0f);
        }
      }
      acc0 = __builtin_amdgcn_mfma_f32_32x32x2f32(av, b0, acc0, 0, 0, 0);
      acc1 = __builtin_amdgcn_mfma_f32_32x32x2f32(av, b1, acc1, 0, 0, 0);
    }
    const float lr = a.lr;
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      const int row = m0 + 8 * (r >> 2) + 4 * lhi + (r & 3);
      if (row < a.Mrows) {
        float* wr = Wp + (int64_t)row * a.ldw + n0 + l32;
        wr[0] = w0[r] - lr * acc0[r];
        if (vb1) wr[32] = w1[r] - lr * acc1[r];
      }
    }
  }

  if (nt == 0 && a.bias != nullptr && tid < 64) {
    const int m = mt * 64 + tid;
    if (m < a.Mrows) {
      float sum = 0.0f;
      for (int s = 0; s < a.Kb; ++s) sum += Gp[(int64_t)s * a.ldg + m];
      a.bias[(int64_t)p * a.w_pitch + m] -= a.lr * sum;
    }
  }
}

void launch_update(hipStream_t s, const UpdArgs& a, ASource bsrc) {
  const int mtiles = (a.Mrows + 63) / 64;
  const int ntiles = (a.Ncols + 127) / 128;
  const unsigned grid = (unsigned)((int64_t)a.P * mtiles * ntiles);
  if (bsrc == A_GATHER)
    k_update_tn<A_GATHER><<<grid, 256, 0, s>>>(a, mtiles, ntiles);
  else
    k_update_tn<A_RELU><<<grid, 256, 0, s>>>(a, mtiles, ntiles);
}

}  // namespace hav
