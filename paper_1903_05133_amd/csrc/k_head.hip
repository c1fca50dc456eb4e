// Loss-side work of one local SGD step: the softmax cross-entropy gradient
// (mean over the minibatch: Algorithm 1 in Sec. 3.1 scales the summed
// gradient by 1/B), the hidden-layer error, and the second layer's update.
//
// Two forms:
//  * small class count (C <= kSmallC): two fused kernels per step, each with
//    one workgroup per learner and 32 hidden units.  k_head_a sums the
//    layer-1 split-K partials with the bias (Z1) and forms this slice's
//    partial logits; k_head_b adds the slices' partial logits, takes the
//    softmax gradient, the hidden error, and the second-layer weight and both
//    bias updates;
//  * any class count: k_reduce_bias, the layer-2 forward GEMM,
//    k_softmax_grad and k_bwd_hidden; the second-layer update is the update
//    GEMM.
// Every kernel issues its global loads in batches before using them, so a
// workgroup waits for memory a few times, not once per element.
#include "internal.h"

namespace hav {

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

// Z[p][m][n] = b_p[n] + sum_ks part[ks][p][m][n] for m < M; rows M..Mp-1 = 0.
__global__ __launch_bounds__(256) void k_reduce_bias(const float* __restrict__ part, int KS,
                                                     const float* __restrict__ bias, int64_t w_pitch,
                                                     float* __restrict__ Z, int P, int M, int Mp, int N) {
  const int64_t per = (int64_t)Mp * N;
  const int64_t total = (int64_t)P * per;
  for (int64_t e = blockIdx.x * 256ll + threadIdx.x; e < total; e += (int64_t)gridDim.x * 256) {
    const int p = (int)(e / per);
    const int64_t r = e - (int64_t)p * per;
    const int m = (int)(r / N), n = (int)(r % N);
    float v = 0.0f;
    if (m < M) {
      v = bias[(int64_t)p * w_pitch + n];
#pragma unroll 8
      for (int ks = 0; ks < KS; ++ks) v += part[ks * total + e];
    }
    Z[e] = v;
  }
}

// One wave per (learner p, sample m < M): logits l_c = b_c + sum_ks part for
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
#pragma unroll 8
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

// The same for C <= 64 * NPL with the logits in registers (lane: classes
// lane + 64j): one pass over the partials, no logits written and read back,
// the label issued first.  Same arithmetic in the same order as
// k_softmax_grad.
template <int NPL>
__global__ __launch_bounds__(256) void k_softmax_grad_reg(const float* __restrict__ part, int KS,
                                                          const float* __restrict__ bias, int64_t w_pitch,
                                                          const int32_t* __restrict__ labels,
                                                          const int32_t* __restrict__ idx, float* __restrict__ G,
                                                          int P, int M, int Mp, int C, int Cp) {
  const int row = blockIdx.x * 4 + (threadIdx.x >> 6);
  const int lane = threadIdx.x & 63;
  if (row >= P * M) return;
  const int p = row / M, m = row % M;
  const int y = labels[idx[(int64_t)p * M + m]];
  const int64_t stride = (int64_t)P * Mp * Cp;
  const int64_t base = ((int64_t)p * Mp + m) * Cp;
  const float* b = bias + (int64_t)p * w_pitch;
  float v[NPL];
#pragma unroll
  for (int j = 0; j < NPL; ++j) {
    const int c = lane + 64 * j;
    const float bv = b[c < C ? c : C - 1];
    v[j] = c < C ? bv : -INFINITY;
  }
  for (int ks = 0; ks < KS; ++ks) {
    const float* pk = part + ks * stride + base;
#pragma unroll
    for (int j = 0; j < NPL; ++j) {
      const int c = lane + 64 * j;
      const float pv = pk[c < C ? c : C - 1];
      v[j] += c < C ? pv : 0.0f;
    }
  }
  float mx = -INFINITY;
#pragma unroll
  for (int j = 0; j < NPL; ++j) mx = fmaxf(mx, v[j]);
  mx = wave_max(mx);
  float sum = 0.0f;
#pragma unroll
  for (int j = 0; j < NPL; ++j) {
    v[j] = lane + 64 * j < C ? expf(v[j] - mx) : 0.0f;
    sum += v[j];
  }
  sum = wave_sum(sum);
  const float invB = 1.0f / (float)M;
  float* g = G + base;
#pragma unroll
  for (int j = 0; j < NPL; ++j) {
    const int c = lane + 64 * j;
    if (c < C) g[c] = (v[j] / sum - (c == y ? 1.0f : 0.0f)) * invB;
  }
}

// G1[p][m][h] = (sum_{c<C} G2[p][m][c] * W2_p[c][h]) * [Z1[p][m][h] > 0] for
// m < M.  Workgroup (p, 64 hidden units): lane = unit, wave w = a quarter of
// each 64-class chunk of G2 (staged in LDS, 16 samples at a time); the four
// waves' partial sums are added in wave order through LDS.  With b1, the
// unit's sum over the samples also takes the SGD step of b1[h].
__global__ __launch_bounds__(256) void k_bwd_hidden(const float* __restrict__ G2, const float* __restrict__ W2,
                                                    int64_t w_pitch, const float* __restrict__ Z1,
                                                    float* __restrict__ G1, int M, int Mp, int C, int Cp, int Hp,
                                                    int htiles, float* __restrict__ b1,
                                                    const float* __restrict__ lr_ptr) {
  constexpr int MC = 16, CC = 64, HU = 64, NW = 4, CW = CC / NW;
  __shared__ float gs[MC][CC];
  __shared__ float red[NW][MC][HU];
  const int p = blockIdx.x / htiles;
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const int h = (blockIdx.x % htiles) * HU + lane;
  const bool hok = h < Hp;
  const float* w2 = W2 + (int64_t)p * w_pitch;
  const float* g2 = G2 + (int64_t)p * Mp * Cp;
  float db1 = 0.0f;
  for (int m0 = 0; m0 < M; m0 += MC) {
    float acc[MC];
#pragma unroll
    for (int i = 0; i < MC; ++i) acc[i] = 0.0f;
    for (int c0 = 0; c0 < C; c0 += CC) {
      __syncthreads();
      for (int e = tid; e < MC * CC; e += 256) {
        const int mm = e / CC, cc = e % CC;
        const bool ok = m0 + mm < M && c0 + cc < C;
        const float v = g2[(int64_t)(ok ? m0 + mm : 0) * Cp + (ok ? c0 + cc : 0)];
        gs[mm][cc] = ok ? v : 0.0f;
      }
      __syncthreads();
      const int cb = c0 + CW * w;
#pragma unroll 4
      for (int cc = 0; cc < CW; ++cc) {
        const int c = cb + cc;
        const float wv = w2[(int64_t)(c < C ? c : 0) * Hp + (hok ? h : 0)];
        const float wt = c < C ? wv : 0.0f;
#pragma unroll
        for (int i = 0; i < MC; ++i) acc[i] += gs[i][CW * w + cc] * wt;
      }
    }
#pragma unroll
    for (int i = 0; i < MC; ++i) red[w][i][lane] = acc[i];
    __syncthreads();
    // wave w finishes samples w*4 .. w*4+3 of the chunk
#pragma unroll
    for (int j = 0; j < MC / NW; ++j) {
      const int i = MC / NW * w + j, m = m0 + i;
      const float g = ((red[0][i][lane] + red[1][i][lane]) + red[2][i][lane]) + red[3][i][lane];
      if (hok && m < M) {
        const int64_t o = ((int64_t)p * Mp + m) * Hp + h;
        const float g1 = Z1[o] > 0.0f ? g : 0.0f;
        G1[o] = g1;
        db1 += g1;
      }
    }
  }
  if (b1) {  // the four waves' sample sums, in wave order
    __syncthreads();
    red[w][0][lane] = db1;
    __syncthreads();
    if (w == 0 && hok)
      b1[(int64_t)p * w_pitch + h] -= *lr_ptr * (((red[0][0][lane] + red[1][0][lane]) + red[2][0][lane]) + red[3][0][lane]);
  }
}

// The same product on the matrix cores: G1[p][m][h] = [Z1 > 0] * sum_c
// G2[p][m][c] W2[p][c][h].  Workgroup (learner p, 32 samples, 32 hidden
// units): wave w takes classes [16w, 16w + 16) of each 64-class chunk with
// 32x32x2 MFMAs into its own 32x32 accumulator block.  Chunks are staged in
// LDS (G2 transposed, class-major, so a wave's operand reads are consecutive
// words), double-buffered, with two register sets so that the loads of chunk
// c + 2 are in flight while chunk c is multiplied; the four partial blocks
// are added in wave order through LDS.  Rows past M and classes past Cp read
// as zero.  b1 (M <= 32 only): also the step b1[h] -= lr * sum_m G1[m][h].
//
// UPD (one sample tile, plain SGD): the workgroup also takes the second
// layer's SGD step on its slab W2[:, h0 .. h0+32) while each chunk is in LDS:
// dW2 = G2^T relu(Z1) for the chunk's classes on 16x16x4 MFMAs (wave w:
// classes 16w .. 16w+15 of the chunk, both 16-unit halves; k = the 32
// samples), the new values written once from the old ones in LDS after
// they fed the hidden error.  The workgroup of slice 0 also steps b2.  No
// other workgroup reads or writes these columns of W2, so the update-GEMM's
// separate pass over W2 is not needed.
constexpr int kBhM = 32, kBhN = 32, kBhC = 64;
constexpr int kBhMaxC = 1024;  // most class slots Cp of the second-layer step (UPD): b2 sums in registers
constexpr int kBhLG = kBhM + 1, kBhLW = kBhN + 4;  // odd G2 stride: the transposing stores spread over the banks
constexpr int kBhLds = 2 * kBhC * (kBhLG + kBhLW);
template <bool UPD>
__global__ __launch_bounds__(256) void k_bwd_hidden_mfma(const float* __restrict__ G2, float* __restrict__ W2,
                                                         int64_t w_pitch, const float* __restrict__ Z1,
                                                         float* __restrict__ G1, int M, int Mp, int Cp, int Hp,
                                                         int htiles, int mtiles, float* __restrict__ b1,
                                                         const float* __restrict__ lr_ptr, float* __restrict__ vb1,
                                                         float mu, float wd, float* __restrict__ b2) {
  __shared__ __attribute__((aligned(16))) float lds[kBhLds];
  __shared__ float a1s[UPD ? kBhM : 1][kBhN + 1];  // relu(Z1) of the tile (UPD)
  // buffer b: G2 chunk [class][sample] at gsb(b), W2 chunk [class][unit] at wsb(b)
  auto gsb = [&](int b) { return lds + b * (kBhC * kBhLG); };
  auto wsb = [&](int b) { return lds + 2 * kBhC * kBhLG + b * (kBhC * kBhLW); };
  const int ht = blockIdx.x % htiles;
  const int mt = (blockIdx.x / htiles) % mtiles;
  const int p = blockIdx.x / (htiles * mtiles);
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  const int l32 = lane & 31, lhi = lane >> 5;
  const int m0 = mt * kBhM, h0 = ht * kBhN;
  const float* g2 = G2 + (int64_t)p * Mp * Cp;
  float* w2 = W2 + (int64_t)p * w_pitch;
  const f32x4 zero4 = {0.f, 0.f, 0.f, 0.f};
  const int nch = (Cp + kBhC - 1) / kBhC;
  const float lr = lr_ptr ? *lr_ptr : 0.0f;  // the eager form without steps passes no step size
  if constexpr (UPD) {  // relu(Z1)[m][h0 + 4(t%8) ..] of the tile; rows past M are zero
    const int m = tid >> 3, hq = 4 * (tid & 7);
    const f32x4 z = *(const f32x4*)(Z1 + ((int64_t)p * Mp + (m < M ? m : 0)) * Hp + h0 + hq);
    a1s[m][hq + 0] = m < M ? fmaxf(z.x, 0.0f) : 0.0f;
    a1s[m][hq + 1] = m < M ? fmaxf(z.y, 0.0f) : 0.0f;
    a1s[m][hq + 2] = m < M ? fmaxf(z.z, 0.0f) : 0.0f;
    a1s[m][hq + 3] = m < M ? fmaxf(z.w, 0.0f) : 0.0f;
  }

  // G2 pieces: q = tid + 256*i, sample q >> 4, classes 4*(q & 15) .. +3.
  // W2 pieces: q = tid + 256*i, class q >> 3, units 4*(q & 7) .. +3.
  // Loads are unconditional from clamped in-range addresses (a load whose
  // value is used in its own branch is waited for at once); rows past M and
  // classes past Cp become zero when stored to LDS.
  f32x4 ga0[2], wa0[2], ga1[2], wa1[2];
  auto load = [&](int c0, f32x4 (&g)[2], f32x4 (&w)[2]) {
#pragma unroll
    for (int i = 0; i < 2; ++i) {
      const int q = tid + 256 * i, r = q >> 4, c = c0 + 4 * (q & 15);
      g[i] = *(const f32x4*)(g2 + (int64_t)min(m0 + r, M - 1) * Cp + min(c, Cp - 4));
    }
#pragma unroll
    for (int i = 0; i < 2; ++i) {
      const int q = tid + 256 * i, c = c0 + (q >> 3);
      w[i] = *(const f32x4*)(w2 + (int64_t)min(c, Cp - 1) * Hp + h0 + 4 * (q & 7));
    }
  };
  auto store = [&](int buf, int c0, const f32x4 (&g)[2], const f32x4 (&w)[2]) {
#pragma unroll
    for (int i = 0; i < 2; ++i) {
      const int q = tid + 256 * i, r = q >> 4, c4 = 4 * (q & 15);
      const bool ok = m0 + r < M && c0 + c4 < Cp;
#pragma unroll
      for (int j = 0; j < 4; ++j) gsb(buf)[(c4 + j) * kBhLG + r] = ok ? g[i][j] : 0.0f;
    }
#pragma unroll
    for (int i = 0; i < 2; ++i) {
      const int q = tid + 256 * i;
      *(f32x4*)&wsb(buf)[(q >> 3) * kBhLW + 4 * (q & 7)] = c0 + (q >> 3) < Cp ? w[i] : zero4;
    }
  };

  f32x16 acc;
#pragma unroll
  for (int r = 0; r < 16; ++r) acc[r] = 0.0f;
  // b2 (slice 0, UPD): thread t < 64 sums class 64 ch + t of every chunk;
  // the step is taken once at the end.
  float sb2[UPD ? (kBhMaxC + kBhC - 1) / kBhC : 1];
#pragma unroll
  for (int k = 0; k < (UPD ? (kBhMaxC + kBhC - 1) / kBhC : 1); ++k) sb2[k] = 0.0f;
  auto chunk = [&](int ch) {  // the products of chunk ch, which sits in LDS buffer ch & 1
    const float* gb = gsb(ch & 1);
    const float* wb = wsb(ch & 1);
#pragma unroll
    for (int ss = 0; ss < kBhC / 4; ss += 2) {
      const int k = wave * (kBhC / 4) + ss + lhi;
      acc = __builtin_amdgcn_mfma_f32_32x32x2f32(gb[k * kBhLG + l32], wb[k * kBhLW + l32], acc, 0, 0, 0);
    }
    if constexpr (UPD) {
      // dW2 of classes 16w + i (i = lane%16 for A, rows 4(lane/16) + r of the
      // result) and units j = lane%16 of each half, over the 32 samples.
      const int i16 = lane & 15, k16 = lane >> 4;
      f32x4 d0 = zero4, d1 = zero4;
#pragma unroll
      for (int kk = 0; kk < kBhM / 4; ++kk) {
        const int m = 4 * kk + k16;
        const float av = gb[(16 * wave + i16) * kBhLG + m];
        d0 = __builtin_amdgcn_mfma_f32_16x16x4f32(av, a1s[m][i16], d0, 0, 0, 0);
        d1 = __builtin_amdgcn_mfma_f32_16x16x4f32(av, a1s[m][16 + i16], d1, 0, 0, 0);
      }
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int cl = 16 * wave + 4 * k16 + r, c = ch * kBhC + cl;
        if (c < Cp) {
          w2[(int64_t)c * Hp + h0 + i16] = wb[cl * kBhLW + i16] - lr * d0[r];
          w2[(int64_t)c * Hp + h0 + 16 + i16] = wb[cl * kBhLW + 16 + i16] - lr * d1[r];
        }
      }
      if (ht == 0 && tid < kBhC) {  // b2: column sums of G2 over the samples
        float sb = 0.0f;
#pragma unroll 8
        for (int m = 0; m < kBhM; ++m) sb += gb[tid * kBhLG + m];
#pragma unroll
        for (int k = 0; k < (kBhMaxC + kBhC - 1) / kBhC; ++k)
          if (k == ch) sb2[k] = sb;
      }
    }
  };
  // Chunks alternate between register sets 0 / 1 and LDS buffers 0 / 1; the
  // loads of chunk ch + 2 are in flight while chunk ch is multiplied (past
  // the last chunk they read an in-range chunk again, not stored).
  load(0, ga0, wa0);
  load(kBhC, ga1, wa1);
  store(0, 0, ga0, wa0);
  __syncthreads();
  for (int ch = 0; ch < nch; ch += 2) {
    load((ch + 2) * kBhC, ga0, wa0);
    __builtin_amdgcn_sched_barrier(0);  // those loads go out before the MFMAs
    chunk(ch);
    if (ch + 1 < nch) store(1, (ch + 1) * kBhC, ga1, wa1);
    __syncthreads();
    if (ch + 1 >= nch) break;
    load((ch + 3) * kBhC, ga1, wa1);
    __builtin_amdgcn_sched_barrier(0);
    chunk(ch + 1);
    if (ch + 2 < nch) store(0, (ch + 2) * kBhC, ga0, wa0);
    __syncthreads();
  }
  if constexpr (UPD) {
    if (ht == 0 && tid < kBhC) {
      float bo[(kBhMaxC + kBhC - 1) / kBhC];
#pragma unroll
      for (int k = 0; k < (kBhMaxC + kBhC - 1) / kBhC; ++k)
        bo[k] = b2[(int64_t)p * w_pitch + min(k * kBhC + tid, Cp - 1)];
#pragma unroll
      for (int k = 0; k < (kBhMaxC + kBhC - 1) / kBhC; ++k)
        if (k < nch && k * kBhC + tid < Cp) b2[(int64_t)p * w_pitch + k * kBhC + tid] = bo[k] - lr * sb2[k];
    }
  }
  // Waves 1-3 hand their blocks to wave 0 through LDS ([3][32][33]).
  if (wave > 0) {
#pragma unroll
    for (int r = 0; r < 16; ++r)
      lds[((wave - 1) * 32 + 8 * (r >> 2) + 4 * lhi + (r & 3)) * 33 + l32] = acc[r];
  }
  __syncthreads();
  if (wave == 0) {
    const int h = h0 + l32;
    // the ReLU masks of the 16 rows in one batch of loads (rows past M: clamped, unused)
    float zv[16];
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      const int m = m0 + 8 * (r >> 2) + 4 * lhi + (r & 3);
      zv[r] = Z1[((int64_t)p * Mp + min(m, M - 1)) * Hp + h];
    }
    float db = 0.0f;
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      const int row = 8 * (r >> 2) + 4 * lhi + (r & 3), m = m0 + row;
      const float g = ((acc[r] + lds[row * 33 + l32]) + lds[(32 + row) * 33 + l32]) + lds[(64 + row) * 33 + l32];
      if (m < M) {
        const float g1 = zv[r] > 0.0f ? g : 0.0f;
        G1[((int64_t)p * Mp + m) * Hp + h] = g1;
        db += g1;
      }
    }
    if (b1) {  // rows 0-3, 8-11, ... of lanes 0-31, then the other rows of lanes 32-63
      const float other = __shfl_xor(db, 32, 64);
      if (lhi == 0) {
        float* bp = b1 + (int64_t)p * w_pitch + h;
        if (mu == 0.0f && wd == 0.0f) {
          *bp -= lr * (db + other);
        } else {  // heavy-ball step with decay: d = g + wd*b; v <- mu*v + d; b <- b - lr*v
          float d = (db + other) + wd * *bp;
          if (vb1) {
            float* vp = vb1 + (int64_t)p * w_pitch + h;
            d = mu * *vp + d;
            *vp = d;
          }
          *bp -= lr * d;
        }
      }
    }
  }
}

// Heavy-ball delayed updates: the block's hidden errors scaled by their
// step's block-end coefficients, Gu[k] = u_{K1-1-k} Gs[k] (for the update of
// the parameters) and Gt[k] = t_{K1-1-k} Gs[k] (for the buffers).
__global__ __launch_bounds__(256) void k_scale_errors(const f32x4* __restrict__ Gs, f32x4* __restrict__ Gu,
                                                      f32x4* __restrict__ Gt, const float* __restrict__ hb, int K1,
                                                      int64_t n4) {
  const int k = blockIdx.y;
  const float cu = hb[hb_index(HB_U, K1 - 1 - k)], ct = hb[hb_index(HB_T, K1 - 1 - k)];
  for (int64_t i = blockIdx.x * 256ll + threadIdx.x; i < n4; i += (int64_t)gridDim.x * 256) {
    const f32x4 g = Gs[k * n4 + i];
    Gu[k * n4 + i] = cu * g;
    if (Gt) Gt[k * n4 + i] = ct * g;
  }
}

// Delayed-update pre-activations for the head with more than 32 classes
// (Z1Args): workgroup (p, slice of 32 hidden units); the Gram correction as in
// k_head_step (32x32x2 MFMAs over the earlier steps, split over the waves).
__global__ __launch_bounds__(256) void k_z1_delayed(Z1Args a, int htiles) {
  constexpr int kHS = 32, kMS = 32, kGrlS = kMS + 1, kMaxK = 7;
  __shared__ __attribute__((aligned(16))) float gsl[kMaxK][kMS][kHS];
  __shared__ float grl[kMaxK][kMS][kGrlS];
  __shared__ float cbuf[4][kMS][kMS + 1];
  const int p = blockIdx.x / htiles, ht = blockIdx.x % htiles;
  const int tid = threadIdx.x, u4 = tid & 7, rr = tid >> 3;
  const int M = a.M, Mp = a.Mp, Hp = a.Hp, kc = a.k;
  const int h4 = ht * kHS + 4 * u4;
  const f32x4 zero4 = {0.f, 0.f, 0.f, 0.f};
  f32x4 z = zero4;
  const float* pm = a.part + ((int64_t)p * Mp + (rr < M ? rr : 0)) * Hp + h4;
#pragma unroll 8
  for (int ks = 0; ks < a.KS; ++ks) z += *(const f32x4*)(pm + ks * a.split);
  if (a.hb) {  // heavy-ball block: p_k X_k W^T + q_k X_k V^T
    z = a.hb[hb_index(HB_P, kc)] * z;
    if (a.partv && kc > 0) {
      const float* pv = a.partv + ((int64_t)p * Mp + (rr < M ? rr : 0)) * Hp + h4;
      f32x4 zv = zero4;
#pragma unroll 8
      for (int ks = 0; ks < a.KSv; ++ks) zv += *(const f32x4*)(pv + ks * a.splitv);
      z += a.hb[hb_index(HB_Q, kc)] * zv;
    }
  }
  z += *(const f32x4*)(a.b1 + (int64_t)p * a.w_pitch + h4);
  if (kc > 0) {
    const int gsm = tid / (kHS / 4), gc4 = tid % (kHS / 4);
    for (int k2 = 0; k2 < kc; ++k2) {
      f32x4 v =
          *(const f32x4*)(a.gs + (((int64_t)k2 * a.P + p) * Mp + (gsm < M ? gsm : 0)) * Hp + ht * kHS + 4 * gc4);
      if (a.hb) v = a.hb[hb_index(HB_U, kc - 1 - k2)] * v;  // the step's own coefficient
      *(f32x4*)&gsl[k2][gsm][4 * gc4] = gsm < M ? v : zero4;
    }
    const float* gk = a.gram + (((int64_t)p * a.K1 + a.k) * a.K1) * Mp * Mp;
    for (int e = tid; e < kc * Mp * Mp; e += 256) {
      const int k2 = e / (Mp * Mp), rem = e % (Mp * Mp);
      grl[k2][rem / Mp][rem % Mp] = gk[(int64_t)k2 * Mp * Mp + rem];
    }
    __syncthreads();
    const int wave = tid >> 6, lane = tid & 63, l32 = lane & 31, lhi = lane >> 5;
    if (wave < kc) {
      f32x16 acc;
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[r] = 0.0f;
      for (int k2 = wave; k2 < kc; k2 += 4)
        for (int j = 0; j < Mp / 2; ++j)
          acc = __builtin_amdgcn_mfma_f32_32x32x2f32(grl[k2][l32][2 * j + lhi], gsl[k2][2 * j + lhi][l32], acc, 0,
                                                     0, 0);
#pragma unroll
      for (int r = 0; r < 16; ++r) cbuf[wave][8 * (r >> 2) + 4 * lhi + (r & 3)][l32] = acc[r];
    }
    __syncthreads();
    f32x4 c = zero4;
    for (int w = 0; w < (kc < 4 ? kc : 4); ++w)
      c += f32x4{cbuf[w][rr][4 * u4], cbuf[w][rr][4 * u4 + 1], cbuf[w][rr][4 * u4 + 2], cbuf[w][rr][4 * u4 + 3]};
    if (a.hb)
      z += c;  // the coefficients (u_n, which carry -lr) are in the staged errors
    else
      z -= *a.lr * c;
  }
  if (rr < M) *(f32x4*)(a.Z1 + ((int64_t)p * Mp + rr) * Hp + h4) = z;
}

void launch_z1_delayed(hipStream_t s, const Z1Args& a) {
  const int htiles = a.Hp / 32;
  launch(k_z1_delayed, a.P * htiles, 256, 0, s, a, htiles);
}

// ------------------------------------------------------------ small C
// Tile = learner p (blockIdx.x / htiles) and hidden units [32*ht, 32*ht + 32);
// samples in chunks of 32.  KC (16 or 32) is the class capacity, C <= KC.
// Loads never sit behind a branch: out-of-range rows read a clamped, in-range
// address and are zeroed by a select, so the compiler can keep many loads in
// flight and wait for exactly the ones it needs.
constexpr int kHU = 32;  // hidden units per workgroup
constexpr int kHM = 32;  // samples per chunk

// Z1 = b1 + sum of the layer-1 partials (stored for k_head_b and the ReLU
// masks), and this slice's partial logits
//   PL[p][m][c][ht] = [ht == 0] b2[c] + sum_{h in slice} ReLU(Z1[m][h]) * W2[c][h]
// (b2 is folded into slice 0's, so k_head_b never reads the b2 it updates).
// Thread t reads 16-byte pieces (units 4*(t%8) .. +3) of row t/8 of the chunk.
constexpr int kCorrMaxK = 7;  // earlier steps in a block (K1 <= 8) of the delayed head's corrections
template <int KC>
__global__ __launch_bounds__(256) void k_head_a(const float* __restrict__ part, int KS, const float* __restrict__ b1,
                                                const float* __restrict__ W2, const float* __restrict__ b2,
                                                int64_t w_pitch,
                                                float* __restrict__ Z1, float* __restrict__ PL, int P, int M, int Mp,
                                                int C, int Cp, int Hp, int htiles, int64_t split) {
  __shared__ float zs[kHM][kHU + 1];
  __shared__ float ws[KC][kHU + 1];
  const int p = blockIdx.x / htiles, ht = blockIdx.x % htiles;
  const int tid = threadIdx.x, u4 = tid & 7, rr = tid >> 3;
  const int h4 = ht * kHU + 4 * u4;
  const float* w2 = W2 + (int64_t)p * w_pitch;
#pragma unroll
  for (int i = 0; i < KC * kHU / 256; ++i) {
    const int e = tid + 256 * i;
    const int c = e / kHU, hh = e % kHU;
    const float v = w2[(int64_t)(c < C ? c : 0) * Hp + ht * kHU + hh];
    ws[c][hh] = c < C ? v : 0.0f;
  }
  const f32x4 bias = *(const f32x4*)(b1 + (int64_t)p * w_pitch + h4);
  const float* p0 = part + (int64_t)p * Mp * Hp + h4;
  auto part_sum = [&](int m0) {  // sum of the split-K partials of row m0 + rr, in split order
    const int m = m0 + rr;
    const float* pm = p0 + (int64_t)(m < M ? m : 0) * Hp;
    f32x4 z = {0.f, 0.f, 0.f, 0.f};
#pragma unroll 8
    for (int ks = 0; ks < KS; ++ks) z += *(const f32x4*)(pm + ks * split);
    return z;
  };
  for (int m0 = 0; m0 < M; m0 += kHM) {
    const int m = m0 + rr;
    const bool mok = m < M;
    f32x4 z = part_sum(m0);
    z += bias;
    if (mok) *(f32x4*)(Z1 + ((int64_t)p * Mp + m) * Hp + h4) = z;
    zs[rr][4 * u4 + 0] = mok ? fmaxf(z.x, 0.0f) : 0.0f;
    zs[rr][4 * u4 + 1] = mok ? fmaxf(z.y, 0.0f) : 0.0f;
    zs[rr][4 * u4 + 2] = mok ? fmaxf(z.z, 0.0f) : 0.0f;
    zs[rr][4 * u4 + 3] = mok ? fmaxf(z.w, 0.0f) : 0.0f;
    __syncthreads();
#pragma unroll
    for (int k = 0; k < kHM * KC / 256; ++k) {
      const int e = tid + 256 * k, mm = e / KC, c = e % KC;
      float acc = ht == 0 && c < C ? b2[(int64_t)p * w_pitch + c] : 0.0f;
#pragma unroll
      for (int hh = 0; hh < kHU; ++hh) acc += zs[mm][hh] * ws[c][hh];
      if (m0 + mm < M && c < C) PL[(((int64_t)p * Mp + m0 + mm) * Cp + c) * htiles + ht] = acc;
    }
    __syncthreads();
  }
}

// Per 32-sample chunk: the logits of each sample (the slices' partial logits,
// b2 included, added in slice order), its softmax cross-entropy gradient
// G2 = (softmax - onehot) / M (kept in LDS), then for this slice of units the
// hidden error G1 = (G2 W2)[m][h] * [Z1 > 0] (W2[:, h] held in registers)
// and the gradients of b1[h] and W2[:, h].  Thread (u = t%32, g = t/32) owns
// unit h = 32*ht + u and samples g + 8i of the chunk.  The eight sample groups
// are combined in LDS in a fixed order; then W2[:, h] and b1[h] take their SGD
// step after every use of the old column (no other workgroup touches column
// h).  Slice ht = 0 also updates b2.
template <int KC>
__global__ __launch_bounds__(256) void k_head_b(const float* __restrict__ PL, float* __restrict__ W2,
                                                float* __restrict__ b1, float* __restrict__ b2, int64_t w_pitch,
                                                const float* __restrict__ Z1, float* __restrict__ G1,
                                                const int32_t* __restrict__ labels, const int32_t* __restrict__ idx,
                                                int P, int M, int Mp, int C, int Cp, int Hp, int htiles,
                                                const float* __restrict__ lr_ptr, HeadMom mom) {
  const float lr = *lr_ptr;
  constexpr int kG = 256 / kHU;     // sample groups
  constexpr int kR = kHM / kG;      // samples per thread per chunk
  __shared__ float gs[kHM][KC + 1];
  __shared__ float red[kG][KC + 1][kHU];
  __shared__ int ys[kHM];
  const int p = blockIdx.x / htiles, ht = blockIdx.x % htiles;
  const int tid = threadIdx.x, u = tid % kHU, g = tid / kHU;
  const int h = ht * kHU + u;
  float* w2 = W2 + (int64_t)p * w_pitch;
  float wc[KC];
#pragma unroll
  for (int c = 0; c < KC; ++c) {
    const float v = w2[(int64_t)(c < C ? c : 0) * Hp + h];
    wc[c] = c < C ? v : 0.0f;
  }
  float db1 = 0.0f, db2 = 0.0f;
  float dw2[KC];
#pragma unroll
  for (int c = 0; c < KC; ++c) dw2[c] = 0.0f;
  const float invB = 1.0f / (float)M;
  for (int m0 = 0; m0 < M; m0 += kHM) {
    const int mn = min(kHM, M - m0);
    if (tid < kHM) ys[tid] = labels[idx[(int64_t)p * M + m0 + min(tid, mn - 1)]];
    float z[kR];
#pragma unroll
    for (int i = 0; i < kR; ++i) {
      const int mm = g + kG * i;
      const float v = Z1[((int64_t)p * Mp + m0 + (mm < mn ? mm : 0)) * Hp + h];
      z[i] = mm < mn ? v : 0.0f;
    }
#pragma unroll
    for (int k = 0; k < kHM * KC / 256; ++k) {
      const int e = tid + 256 * k, mm = e / KC, c = e % KC;
      const bool ok = mm < mn && c < C;
      const float* pl = PL + (((int64_t)p * Mp + m0 + (mm < mn ? mm : 0)) * Cp + (c < C ? c : 0)) * htiles;
      float l = 0.0f;
#pragma unroll 8
      for (int t = 0; t < htiles; ++t) l += pl[t];
      gs[mm][c] = ok ? l : 0.0f;
    }
    __syncthreads();
    if (tid < mn) {
      float mx = -INFINITY;
      for (int c = 0; c < C; ++c) mx = fmaxf(mx, gs[tid][c]);
      float sum = 0.0f;
      for (int c = 0; c < C; ++c) {
        const float e = expf(gs[tid][c] - mx);
        gs[tid][c] = e;
        sum += e;
      }
      const int y = ys[tid];
      for (int c = 0; c < C; ++c) gs[tid][c] = (gs[tid][c] / sum - (c == y ? 1.0f : 0.0f)) * invB;
    }
    __syncthreads();
#pragma unroll
    for (int i = 0; i < kR; ++i) {
      const int mm = g + kG * i;
      if (mm < mn) {
        const float a = fmaxf(z[i], 0.0f);
        float da = 0.0f;
#pragma unroll
        for (int c = 0; c < KC; ++c) da += gs[mm][c] * wc[c];
        const float g1 = z[i] > 0.0f ? da : 0.0f;
        G1[((int64_t)p * Mp + m0 + mm) * Hp + h] = g1;
        db1 += g1;
#pragma unroll
        for (int c = 0; c < KC; ++c) dw2[c] += gs[mm][c] * a;
      }
    }
    if (ht == 0 && tid < C)
      for (int mm = 0; mm < mn; ++mm) db2 += gs[mm][tid];
    __syncthreads();
  }
  red[g][KC][u] = db1;
#pragma unroll
  for (int c = 0; c < KC; ++c) red[g][c][u] = dw2[c];
  __syncthreads();
  // d = g + wd*w; with buffers v <- mu*v + d and the step takes v.
  auto step = [&](float* w, float* v, float wold, float gsum) {
    float d = gsum + mom.wd * wold;
    if (v) {
      d = mom.mu * *v + d;
      *v = d;
    }
    *w = wold - lr * d;
  };
  const int64_t po = (int64_t)p * w_pitch;
  if (g == 0) {
    float s = 0.0f;
#pragma unroll
    for (int k = 0; k < kG; ++k) s += red[k][KC][u];
    step(b1 + po + h, mom.vb1 ? mom.vb1 + po + h : nullptr, b1[po + h], s);
#pragma unroll
    for (int c = 0; c < KC; ++c)
      if (c < C) {
        float gsum = 0.0f;
#pragma unroll
        for (int k = 0; k < kG; ++k) gsum += red[k][c][u];
        const int64_t o = po + (int64_t)c * Hp + h;
        step(W2 + o, mom.vw2 ? mom.vw2 + o : nullptr, wc[c], gsum);
      }
  }
  if (ht == 0 && tid < C)
    step(b2 + po + tid, mom.vb2 ? mom.vb2 + po + tid : nullptr, b2[po + tid], db2);
}

// The loss side of an eager step (C <= 32), before the second layer's
// step.  Workgroup = learner p and the 16 samples [16q, 16q + 16) with every
// hidden unit, eight waves:
//  * Z1 = (split-K partials added in split order) + b1 and the learner's W2
//    (rows C..KC-1 zero) are staged in LDS;
//  * logits = b2 + ReLU(Z1) W2^T as 16x16x4 MFMAs, the 16-unit runs dealt
//    to the waves in turn and the waves' partial logits added in wave order;
//    then the softmax cross-entropy gradient G2 = (softmax - onehot) / M,
//    four lanes per sample;
//  * G1 = (G2 W2) * [Z1 > 0] (stored) and the group's dW2 = G2^T ReLU(Z1),
//    db1 = sum of G1 and db2 = sum of G2 over its samples, per 16-unit run
//    as 16x16x4 MFMAs.
// The group's dW2, db1, db2 go to its scratch row; k_head_w2_step adds the
// rows and takes the step (a cross-workgroup sum inside this kernel would
// need device-scope fences, each of which writes back and invalidates the
// L2 of its XCD).  Samples M..Mp-1 have Z1 = 0 and G2 = 0 (their G1 rows
// are written as zeros).
// Scratch row of (p, q), HS = (C + 1) Hp + 32 floats: [db1 (Hp) | dW2 (C x Hp) | db2 (C)],
// the order of b1 and W2 in the parameter vector.
constexpr int kHfWaves = 8;  // waves of k_head_fused
template <int KC, int HPM, int KSN>
__global__ __launch_bounds__(64 * kHfWaves) void k_head_fused(HeadFusedArgs a) {
  constexpr int NT = 64 * kHfWaves;
  constexpr int kZL = HPM + 4;  // LDS row length (rows 4 banks apart: conflict-free 16-byte reads of 16 rows)
  constexpr int kNB = 4 * HPM / NT;  // Z1 pieces per thread (at Hp = HPM: one batch of loads)
  constexpr int kNW = (KC * HPM / 4 + NT - 1) / NT;  // most W2 pieces per thread
  constexpr int kCT = KC / 16;                        // 16-class tiles
  __shared__ __attribute__((aligned(16))) float zs[16 * kZL];
  __shared__ __attribute__((aligned(16))) float ws[KC * kZL];
  __shared__ float ls[kHfWaves][16][KC + 1];
  __shared__ float g2s[16][KC + 1];
  __shared__ int ys[16];
  const int NS = a.Mp / 16;
  const int p = blockIdx.x / NS, q = blockIdx.x % NS;
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  const int li = lane & 15, lg = lane >> 4;
  const int Hp = a.Hp, C = a.C, M = a.M, H4 = Hp / 4, runs = Hp / 16;
  const int64_t po = (int64_t)p * a.w_pitch;
  const float* W2 = a.W2 + po;

  // Sample 16q + (tid & 15)'s row index now, its label once the loads
  // below are in flight (clamped to an in-range sample, no branch).
  const int sy = 16 * q + (tid & 15);
  const int ixv = a.idx[(int64_t)p * M + (sy < M ? sy : M - 1)];
  int yv = 0;
  // W2 rows c < KC (KC Hp / 4 pieces) and Z1 of the group's 16 rows (4 Hp
  // pieces, in batches) into LDS.  Every load is issued unconditionally:
  // piece indices past the count repeat the last piece (the same value to
  // the same LDS address), since a load behind a branch is waited for before
  // the next one is issued.
  {
    const int lw = KC * H4 - 1, lz = 4 * Hp - 1;
    f32x4 wr[kNW];
#pragma unroll
    for (int i = 0; i < kNW; ++i) {
      const int e = min(tid + NT * i, lw), c = e / H4, c4 = e % H4;
      const f32x4 v = *(const f32x4*)(W2 + (int64_t)(c < C ? c : 0) * Hp + 4 * c4);
      const f32x4 z4 = {0.f, 0.f, 0.f, 0.f};
      wr[i] = c < C ? v : z4;
    }
    const float* pbase = a.part + ((int64_t)p * a.Mp + 16 * q) * Hp;
    const float* b1 = a.b1 + po;
    const int nz = (4 * Hp + NT - 1) / NT;
    for (int i0 = 0; i0 < nz; i0 += kNB) {
      f32x4 zr[kNB][KSN > 0 ? KSN : 1], br[kNB];
#pragma unroll
      for (int i = 0; i < kNB; ++i) {
        const int e = min(tid + NT * min(i0 + i, nz - 1), lz), s = e / H4, c4 = e % H4;
        const float* src = pbase + (int64_t)s * Hp + 4 * c4;
        br[i] = *(const f32x4*)(b1 + 4 * c4);
#pragma unroll
        for (int k = 0; k < (KSN > 0 ? KSN : 1); ++k)
          zr[i][k] = KSN > 0 ? *(const f32x4*)(src + k * a.split) : f32x4{0.f, 0.f, 0.f, 0.f};
      }
      if (KSN == 0) {
        // Any split count: kKG splits of every piece per batch of loads, all
        // issued before the first add (split indices past the count load the
        // last split again and add zero), the splits added in order.
        constexpr int kKG = kNB > 4 ? 2 : 4;
        for (int k0 = 0; k0 < a.KS; k0 += kKG) {
          f32x4 zk[kNB][kKG];
#pragma unroll
          for (int i = 0; i < kNB; ++i) {
            const int e = min(tid + NT * min(i0 + i, nz - 1), lz), s = e / H4, c4 = e % H4;
            const float* src = pbase + (int64_t)s * Hp + 4 * c4;
#pragma unroll
            for (int k = 0; k < kKG; ++k) zk[i][k] = *(const f32x4*)(src + (int64_t)min(k0 + k, a.KS - 1) * a.split);
          }
#pragma unroll
          for (int i = 0; i < kNB; ++i)
#pragma unroll
            for (int k = 0; k < kKG; ++k) zr[i][0] += k0 + k < a.KS ? zk[i][k] : f32x4{0.f, 0.f, 0.f, 0.f};
        }
      }
      if (i0 == 0) yv = a.labels[ixv];
#pragma unroll
      for (int i = 0; i < kNB; ++i) {
        const int e = min(tid + NT * min(i0 + i, nz - 1), lz), s = e / H4, c4 = e % H4;
        f32x4 z = zr[i][0];
#pragma unroll
        for (int k = 1; k < KSN; ++k) z += zr[i][k];
        z += br[i];
        const f32x4 z4 = {0.f, 0.f, 0.f, 0.f};
        *(f32x4*)&zs[s * kZL + 4 * c4] = 16 * q + s < M ? z : z4;
      }
    }
#pragma unroll
    for (int i = 0; i < kNW; ++i) {
      const int e = min(tid + NT * i, lw), c = e / H4, c4 = e % H4;
      *(f32x4*)&ws[c * kZL + 4 * c4] = wr[i];
    }
  }
  if (tid < 16) ys[tid] = sy < M ? yv : 0;
  float b2v[KC / 4];  // b2 of the classes lane & 3 + 4k (softmax lanes of wave 0)
#pragma unroll
  for (int k = 0; k < KC / 4; ++k) {
    const int c = (lane & 3) + 4 * k;
    const float v = a.b2[po + (c < C ? c : 0)];
    b2v[k] = c < C ? v : 0.0f;
  }
  __syncthreads();

  // Partial logits over this wave's 16-unit runs (runs wave, wave + 8, ...):
  // lane group lg takes units 16 run + 4lg .. + 3 in the four k slots of four
  // MFMAs (the same units for both operands).
  {
    f32x4 acc[kCT];
#pragma unroll
    for (int ct = 0; ct < kCT; ++ct) acc[ct] = f32x4{0.f, 0.f, 0.f, 0.f};
    for (int run = wave; run < runs; run += kHfWaves) {
      const int col = 16 * run + 4 * lg;
      const f32x4 z = *(const f32x4*)&zs[li * kZL + col];
      const f32x4 av = {fmaxf(z.x, 0.0f), fmaxf(z.y, 0.0f), fmaxf(z.z, 0.0f), fmaxf(z.w, 0.0f)};
#pragma unroll
      for (int ct = 0; ct < kCT; ++ct) {
        const f32x4 bv = *(const f32x4*)&ws[(16 * ct + li) * kZL + col];
#pragma unroll
        for (int e = 0; e < 4; ++e) acc[ct] = __builtin_amdgcn_mfma_f32_16x16x4f32(av[e], bv[e], acc[ct], 0, 0, 0);
      }
    }
#pragma unroll
    for (int ct = 0; ct < kCT; ++ct)
#pragma unroll
      for (int r = 0; r < 4; ++r) ls[wave][4 * lg + r][16 * ct + li] = acc[ct][r];
  }
  __syncthreads();

  // Softmax gradient: wave 0, lanes 4s .. 4s + 3 for sample s, classes
  // (lane & 3) + 4k; the waves' partial logits added in wave order.
  if (wave == 0) {
    const int s = lane >> 2;
    float lv[KC / 4];
    float mx = -INFINITY;
#pragma unroll
    for (int k = 0; k < KC / 4; ++k) {
      const int c = (lane & 3) + 4 * k;
      float v = b2v[k];
#pragma unroll
      for (int w = 0; w < kHfWaves; ++w) v += ls[w][s][c];
      lv[k] = v;
      if (c < C) mx = fmaxf(mx, v);
    }
    mx = fmaxf(mx, __shfl_xor(mx, 1, 64));
    mx = fmaxf(mx, __shfl_xor(mx, 2, 64));
    float sum = 0.0f;
#pragma unroll
    for (int k = 0; k < KC / 4; ++k) {
      const int c = (lane & 3) + 4 * k;
      const float e = c < C ? expf(lv[k] - mx) : 0.0f;
      lv[k] = e;
      sum += e;
    }
    sum += __shfl_xor(sum, 1, 64);
    sum += __shfl_xor(sum, 2, 64);
    const bool valid = 16 * q + s < M;
    const int y = ys[s];
    const float invM = 1.0f / (float)M;
#pragma unroll
    for (int k = 0; k < KC / 4; ++k) {
      const int c = (lane & 3) + 4 * k;
      g2s[s][c] = valid && c < C ? (lv[k] / sum - (c == y ? 1.0f : 0.0f)) * invM : 0.0f;
    }
  }
  __syncthreads();

  // Per 16-unit run of this wave: G1 (samples 4lg + r, unit u) and dW2
  // (classes 16ct + 4lg + r, unit u), u = 16 run + li.
  float* hrow = a.scratch + ((int64_t)p * NS + q) * ((int64_t)(C + 1) * Hp + 32);
  float* g1 = a.G1 + ((int64_t)p * a.Mp + 16 * q) * Hp;
  for (int run = wave; run < runs; run += kHfWaves) {
    const int u = 16 * run + li;
    f32x4 d1 = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int t = 0; t < KC / 4; ++t)
      d1 = __builtin_amdgcn_mfma_f32_16x16x4f32(g2s[li][4 * t + lg], ws[(4 * t + lg) * kZL + u], d1, 0, 0, 0);
    f32x4 d2[kCT];
#pragma unroll
    for (int ct = 0; ct < kCT; ++ct) {
      d2[ct] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int t = 0; t < 4; ++t)
        d2[ct] = __builtin_amdgcn_mfma_f32_16x16x4f32(g2s[4 * t + lg][16 * ct + li],
                                                      fmaxf(zs[(4 * t + lg) * kZL + u], 0.0f), d2[ct], 0, 0, 0);
    }
    float db1 = 0.0f;
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const float g = zs[(4 * lg + r) * kZL + u] > 0.0f ? d1[r] : 0.0f;
      g1[(int64_t)(4 * lg + r) * Hp + u] = g;
      db1 += g;
    }
    db1 += __shfl_xor(db1, 16, 64);
    db1 += __shfl_xor(db1, 32, 64);
    if (lg == 0) hrow[u] = db1;
#pragma unroll
    for (int ct = 0; ct < kCT; ++ct)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int c = 16 * ct + 4 * lg + r;
        if (c < C) hrow[Hp + (int64_t)c * Hp + u] = d2[ct][r];
      }
  }
  if (tid < C) {
    float s2 = 0.0f;
#pragma unroll
    for (int s = 0; s < 16; ++s) s2 += g2s[s][tid];
    hrow[(int64_t)(C + 1) * Hp + tid] = s2;
  }
}

// The step of b1, W2 and b2 after k_head_fused: per learner the groups'
// gradient rows added in group order, then the SGD step (heavy-ball and
// decay as in k_head_b).  Workgroup = learner p and 1024 consecutive floats
// of [b1 | W2] (contiguous in the parameters, the buffers and the rows);
// block 0 of a learner also steps b2.
__global__ __launch_bounds__(256) void k_head_w2_step(HeadFusedArgs a, int nblk) {
  const int p = blockIdx.x / nblk, blk = blockIdx.x % nblk;
  const int tid = threadIdx.x;
  const int NS = a.Mp / 16, C = a.C, Hp = a.Hp;
  const int64_t HS = (int64_t)(C + 1) * Hp + 32;
  const int64_t po = (int64_t)p * a.w_pitch;
  const float* h0 = a.scratch + (int64_t)p * NS * HS;
  const float lr = *a.lr;
  const HeadMom& mom = a.mom;
  const int e = blk * 256 + tid;
  // The groups' rows in batches of eight loads issued together (indices past
  // NS repeat the last row and are not added).
  constexpr int kB = 8;
  if (e < (C + 1) * (Hp / 4)) {
    const bool isb = 4 * e < Hp;
    const int64_t o = isb ? 4 * e : 4 * e - Hp;
    f32x4* w = (f32x4*)((isb ? a.b1 : a.W2) + po + o);
    float* vbase = isb ? mom.vb1 : mom.vw2;
    const f32x4 wo = *w;  // issued with the rows below
    f32x4 g = {0.f, 0.f, 0.f, 0.f};
    for (int k0 = 0; k0 < NS; k0 += kB) {
      f32x4 v[kB];
#pragma unroll
      for (int k = 0; k < kB; ++k) v[k] = *(const f32x4*)(h0 + min(k0 + k, NS - 1) * HS + 4 * e);
#pragma unroll
      for (int k = 0; k < kB; ++k)
        if (k0 + k < NS) g = k0 + k == 0 ? v[k] : g + v[k];
    }
    f32x4 d = g + mom.wd * wo;
    if (vbase) {
      f32x4* v = (f32x4*)(vbase + po + o);
      d = mom.mu * *v + d;
      *v = d;
    }
    *w = wo - lr * d;
  }
  if (blk == 0 && tid < C) {
    float* w = a.b2 + po + tid;
    const float wo = *w;
    float g = 0.0f;
    for (int k0 = 0; k0 < NS; k0 += kB) {
      float v[kB];
#pragma unroll
      for (int k = 0; k < kB; ++k) v[k] = h0[min(k0 + k, NS - 1) * HS + (int64_t)(C + 1) * Hp + tid];
#pragma unroll
      for (int k = 0; k < kB; ++k)
        if (k0 + k < NS) g = k0 + k == 0 ? v[k] : g + v[k];
    }
    float d = g + mom.wd * wo;
    if (mom.vb2) {
      float* v = mom.vb2 + po + tid;
      d = mom.mu * *v + d;
      *v = d;
    }
    *w = wo - lr * d;
  }
}

// Value of another lane in the same group of eight by a DPP move: control
// 0xB1 (quad_perm 1,0,3,2) takes lane i^1, 0x4E (quad_perm 2,3,0,1) lane
// i^2, 0x141 (row_half_mirror) lane 7-i of the eight.
template <int kCtrl>
__device__ inline float dpp8(float x) {
  return __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(0, __builtin_bit_cast(int, x), kCtrl, 0xF, 0xF, false));
}

// Fused head of the delayed schedule (HeadStepArgs).  Workgroup (p, ht) owns
// hidden units h = 32*ht + u of learner p; M <= 32 samples, one chunk.  Step k
// of a block:
//  (A) k > 0, the rest of step k-1: logits of every sample from the partial
//      logits of all slices (b2 is folded into slice 0's), its softmax
//      cross-entropy gradient G2 (mean over the minibatch; eight threads per
//      sample), then for this slice, on the matrix cores: G1 = (G2 W2)[m][h]
//      * [Z1 > 0] into gs[k-1] and into LDS for (B), with its column sums
//      stepping b1[h] (waves 0 and 1, 16 units each), and the step of
//      W2[:, h] from G2^T relu(Z1) (waves 2 and 3); the new values stay in
//      LDS for (B); slice 0 steps b2.
//  (B) k < K1, step k: Z1 = b1 + sum of the split-K partials
//      - lr * sum_{k2<k} gram[k][k2] G1[k2] for this slice, its ReLU, and the
//      slice's partial logits into PL[k&1] (slice 0 adds b2).
// (A) reads PL[(k-1)&1] of every slice while (B) writes PL[k&1], and b2 is
// read and written by slice 0 only, so no workgroup depends on another
// within a launch.  Every global load the launch needs is issued before the
// first wait: step k's partials, the Gram rows and the earlier steps' hidden
// errors of (B), this slice's W2, Z1, b1 (and b2) and the partial logits
// and labels of (A).
// NK: slots for the earlier steps of a block (K1 - 1 <= NK).
template <int KC, int NK>
__global__ __launch_bounds__(256) void k_head_step(HeadStepArgs a, int htiles, int k) {
  constexpr int kG = 256 / kHU, kR = kHM / kG;
  static_assert(KC % kG == 0, "class tiles are whole sample groups");
  constexpr int kGsl = NK * kHM * kHU;     // G1 slices of the block's steps
  constexpr int kGrlS = kHM + 1;                    // Gram row stride (conflict-free column reads)
  constexpr int kGrl = NK * kHM * kGrlS;   // Gram rows of step k
  constexpr int kGS = KC + 4;  // G2 row stride (16-byte rows)
  constexpr int kPhaseA = kHM * kGS + (KC + kHM) * (kHU + 1);
  constexpr int kZs = kHM * (kHU + 1);
  constexpr int kCbuf = 4 * kHM * (kHM + 1);          // per-wave partial corrections
  constexpr int kRegion = kPhaseA > kZs + kCbuf ? kPhaseA : kZs + kCbuf;
  __shared__ __attribute__((aligned(16))) float lds[kGsl + kGrl + kRegion + KC * (kHU + 1) + kHU + KC];
  __shared__ int ys[kHM];
  auto gsl = [&](int k2, int s, int u) -> float& { return lds[(k2 * kHM + s) * kHU + u]; };
  float* grl = lds + kGsl;          // [NK][kHM][kGrlS]
  float* region = grl + kGrl;
  float* ws = region + kRegion;     // [KC][kHU + 1] W2 slice (after (A))
  float* bs = ws + KC * (kHU + 1);  // [kHU] b1 slice (after (A))
  float* b2l = bs + kHU;            // [KC] b2 (slice 0, after (A))

  // The slices of a learner run on one XCD (consecutive ids after the
  // remap), so the partial logits they exchange stay within one L2.
  const int bid = xcd_remap(blockIdx.x, gridDim.x);
  const int p = bid / htiles, ht = bid % htiles;
  const int tid = threadIdx.x;
  const int M = a.M, C = a.C, Cp = a.Cp, Hp = a.Hp, Mp = a.Mp;
  const float lr = *a.lr;
  float* w2 = a.W2 + (int64_t)p * a.w_pitch;
  float* b1 = a.b1 + (int64_t)p * a.w_pitch;
  float* b2 = a.b2 + (int64_t)p * a.w_pitch;
  const f32x4 zero4 = {0.f, 0.f, 0.f, 0.f};
  const int u4 = tid & 7, rr = tid >> 3;
  const int h4 = ht * kHU + 4 * u4;
  const int gsm = tid / (kHU / 4), gc4 = tid % (kHU / 4);
  const int u = tid % kHU, g = tid / kHU, h = ht * kHU + u;
  const int64_t step_floats = (int64_t)a.P * Mp * Hp;  // one step of the block's partials

  // Every global load that does not depend on (A) is issued here, with no
  // wait between them: the addresses are clamped into the buffers instead of
  // branched around per thread, and values are masked where they are used.
  // Step k's partials, first kPv splits (the rest, if any, are added in (B)).
  constexpr int kPv = 4;
  const int kc = k < a.K1 ? k : 0;  // earlier steps whose correction (B) applies
  f32x4 pv[kPv];
  if (k < a.K1) {
    const float* pm = a.part + k * step_floats + ((int64_t)p * Mp + (rr < M ? rr : 0)) * Hp + h4;
#pragma unroll
    for (int ks = 0; ks < kPv; ++ks) pv[ks] = *(const f32x4*)(pm + (ks < a.KS ? ks : a.KS - 1) * a.split);
  }
  // (B)'s operands: the hidden errors of steps k2 < k-1 (16-byte piece tid of
  // each step's 32 x 32 slice; step k-1 comes from (A)) and the Gram rows
  // gram[k][k2] (piece tid of each Mp x Mp block).
  f32x4 gv[NK - 1], gr[NK];
  if (kc > 1) {
    const float* gb = a.gs + ((int64_t)p * Mp + (gsm < M ? gsm : M - 1)) * Hp + ht * kHU + 4 * gc4;
#pragma unroll
    for (int k2 = 0; k2 < NK - 1; ++k2)
      gv[k2] = *(const f32x4*)(gb + (int64_t)(k2 < kc - 1 ? k2 : kc - 2) * a.P * Mp * Hp);
  }
  if (kc > 0) {
    const float* gk = a.gram + (((int64_t)p * a.K1 + k) * a.K1) * Mp * Mp +
                      4 * (tid < Mp * Mp / 4 ? tid : Mp * Mp / 4 - 1);
#pragma unroll
    for (int k2 = 0; k2 < NK; ++k2) gr[k2] = *(const f32x4*)(gk + (int64_t)(k2 < kc ? k2 : kc - 1) * Mp * Mp);
  }
  // (A)'s operands of this slice: W2[c][h] for c = g + 8q (classes past C
  // read row 0) and the pre-activations of step k-1 at samples g + 8i (past
  // M: row 0, never used), all written by this workgroup only; b1[h], and
  // b2, which only slice 0 uses (and alone writes).  Step 0 stages the same
  // W2 values for (B).
  constexpr int kWq = KC * kHU / 256;
  float wv[kWq], zp[kR];
  const float b1h = b1[h], b2v = b2[u < C ? u : 0];
#pragma unroll
  for (int q = 0; q < kWq; ++q) {
    const int c = g + kG * q;
    wv[q] = w2[(int64_t)(c < C ? c : 0) * Hp + h];
  }
  if (k > 0) {
#pragma unroll
    for (int i = 0; i < kR; ++i) {
      const int mm = g + kG * i;
      zp[i] = a.Z1[((int64_t)p * Mp + (mm < M ? mm : 0)) * Hp + h];
    }
  }
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6), lane = tid & 63;
  if (k > 0) {  // (A): the rest of step k-1
    const int kp = k - 1;
    float* g2s = region;                 // [kHM][kGS] G2
    float* wold = g2s + kHM * kGS;       // [KC][kHU + 1] the W2 slice before the step
    float* z1p = wold + KC * (kHU + 1);  // [kHM][kHU + 1] Z1 of step k-1
    const int yv = a.ylab[((int64_t)kp * a.P + p) * M + (tid < M ? tid : 0)];
    const float* plp = a.PL + (int64_t)(kp & 1) * a.pl_half;
    constexpr int kQ = kHM * KC / 256;
    const float* pl[kQ];
    bool ok[kQ];
#pragma unroll
    for (int q = 0; q < kQ; ++q) {
      const int e = tid + 256 * q, mm = e / KC, c = e % KC;
      ok[q] = mm < M && c < C;
      pl[q] = plp + (((int64_t)p * Mp + (ok[q] ? mm : 0)) * Cp + (ok[q] ? c : 0)) * htiles;
    }
    float l[kQ];
#pragma unroll
    for (int q = 0; q < kQ; ++q) l[q] = 0.0f;
    if ((htiles & 3) == 0) {
      // 16-byte pieces, four per logit and pass, all issued before the
      // pass's first add (pieces past htiles re-read the last one and are
      // not added); the slices are still added in order.
      for (int t0 = 0; t0 < htiles; t0 += 16) {
        f32x4 v[kQ][4];
#pragma unroll
        for (int q = 0; q < kQ; ++q)
#pragma unroll
          for (int t = 0; t < 4; ++t)
            v[q][t] = *(const f32x4*)(pl[q] + (t0 + 4 * t < htiles ? t0 + 4 * t : htiles - 4));
        __builtin_amdgcn_sched_barrier(0);  // keep the pass's loads ahead of its adds
#pragma unroll
        for (int q = 0; q < kQ; ++q)
#pragma unroll
          for (int t = 0; t < 4; ++t) {
            const bool in = t0 + 4 * t < htiles;
            l[q] += in ? v[q][t].x : 0.0f;
            l[q] += in ? v[q][t].y : 0.0f;
            l[q] += in ? v[q][t].z : 0.0f;
            l[q] += in ? v[q][t].w : 0.0f;
          }
      }
    } else {
#pragma unroll
      for (int q = 0; q < kQ; ++q) {
#pragma unroll 8
        for (int t = 0; t < htiles; ++t) l[q] += pl[q][t];
      }
    }
#pragma unroll
    for (int q = 0; q < kQ; ++q) {
      const int e = tid + 256 * q;
      g2s[(e / KC) * kGS + e % KC] = ok[q] ? l[q] : 0.0f;
    }
    if (tid < kHM) ys[tid] = yv;
    __syncthreads();
    // Staged here, not before the barrier above, so that these loads may
    // still be in flight while the logits are summed.
#pragma unroll
    for (int q = 0; q < kWq; ++q) wold[(g + kG * q) * (kHU + 1) + u] = wv[q];  // rows c >= C: row 0, met by zero G2
#pragma unroll
    for (int i = 0; i < kR; ++i) z1p[(g + kG * i) * (kHU + 1) + u] = zp[i];
    {  // softmax gradient: eight threads per sample, KC/8 classes each
      const int row = tid >> 3, l8 = tid & 7;
      float* rowp = g2s + row * kGS;
      float v[KC / 8];
      float mx = -INFINITY;
#pragma unroll
      for (int j = 0; j < KC / 8; ++j) {
        const int c = l8 + 8 * j;
        v[j] = rowp[c];
        if (c < C) mx = fmaxf(mx, v[j]);
      }
      mx = fmaxf(mx, dpp8<0xB1>(mx));  // the eight lanes of a sample by DPP moves:
      mx = fmaxf(mx, dpp8<0x4E>(mx));  // partner lane i^1, then i^2, then the
      mx = fmaxf(mx, dpp8<0x141>(mx)); // mirror 7-i (a lane of the other quad)
      float sum = 0.0f;
#pragma unroll
      for (int j = 0; j < KC / 8; ++j) {
        v[j] = l8 + 8 * j < C ? expf(v[j] - mx) : 0.0f;
        sum += v[j];
      }
      sum += dpp8<0xB1>(sum);
      sum += dpp8<0x4E>(sum);
      sum += dpp8<0x141>(sum);
      const int y = ys[row];
      const float invB = 1.0f / (float)M;
      if (row < M)
#pragma unroll
        for (int j = 0; j < KC / 8; ++j) {
          const int c = l8 + 8 * j;
          if (c < C) rowp[c] = (v[j] / sum - (c == y ? 1.0f : 0.0f)) * invB;
        }
    }
    __syncthreads();
    const int l16 = lane & 15, lq = lane >> 4;
    if (wave < 2) {
      // G1 = (G2 W2)[m][h] * [Z1 > 0] for units u0 = 16 w .. +15 as 16x16x4
      // MFMAs over the classes, two 16-sample tiles (lane (i, q): G2 row
      // m0 + i and W2 row 4s + q of unit u0 + i; acc[t][r] is sample
      // m0 + 4q + r of unit u0 + i); its column sums step b1.  Rows past M
      // are zero (their G2 rows are).
      const int u0 = 16 * wave, uu = u0 + l16;
      f32x4 acc[2] = {zero4, zero4};
#pragma unroll
      for (int s4 = 0; s4 < KC / 4; ++s4) {
        const float b = wold[(4 * s4 + lq) * (kHU + 1) + uu];
#pragma unroll
        for (int t = 0; t < 2; ++t)
          acc[t] = __builtin_amdgcn_mfma_f32_16x16x4f32(g2s[(16 * t + l16) * kGS + 4 * s4 + lq], b, acc[t], 0, 0, 0);
      }
      // The eight Z1 values are read before any is used, and the stores sit
      // after all of them, so no wait separates the rows.
      float g1[8];
#pragma unroll
      for (int e = 0; e < 8; ++e) g1[e] = z1p[(16 * (e >> 2) + 4 * lq + (e & 3)) * (kHU + 1) + uu];
      __builtin_amdgcn_sched_barrier(0);
      float db1 = 0.0f;
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        const f32x4 av = acc[e >> 2];
        const float v = (e & 3) == 0 ? av.x : (e & 3) == 1 ? av.y : (e & 3) == 2 ? av.z : av.w;
        g1[e] = g1[e] > 0.0f ? v : 0.0f;
        db1 += g1[e];
      }
      if (k < a.K1) {  // for (B) (k-1 <= K1-2 < NK); heavy-ball: scaled by u_0
        const float cu = a.hb ? a.hb[hb_index(HB_U, 0)] : 1.0f;
#pragma unroll
        for (int e = 0; e < 8; ++e) gsl(kp, 16 * (e >> 2) + 4 * lq + (e & 3), uu) = a.hb ? cu * g1[e] : g1[e];
      }
      float* g1out = a.gs + ((int64_t)kp * a.P + p) * Mp * Hp + ht * kHU + uu;
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        const int mm = 16 * (e >> 2) + 4 * lq + (e & 3);
        if (mm < M) g1out[(int64_t)mm * Hp] = g1[e];
      }
      db1 += __shfl_xor(db1, 16);
      db1 += __shfl_xor(db1, 32);
      if (lq == wave) {  // this thread's unit u is uu (tid % 32 = 16 w + i)
        float nb;
        if (a.hb) {  // heavy-ball step with decay
          float d = db1 + a.wd * b1h;
          if (a.vb1) {
            float* vp = a.vb1 + (int64_t)p * a.w_pitch + h;
            d = a.mu * *vp + d;
            *vp = d;
          }
          nb = b1h - lr * d;
        } else {
          nb = b1h - lr * db1;
        }
        b1[h] = nb;
        bs[u] = nb;
      }
    } else {
      // dW2[c][h] = sum_m G2[m][c] relu(Z1)[m][h] as 16x16x4 MFMAs over the
      // samples, 16 x 16 tiles (c0, u0) split over waves 2 and 3 (lane
      // (i, q): class c0 + i and unit u0 + i at sample 4s + q; acc[r] is
      // class c0 + 4q + r of unit u0 + i); W2 takes its step.
      for (int t = wave - 2; t < 2 * (KC / 16); t += 2) {
        const int c0 = 16 * (t >> 1), u0 = 16 * (t & 1);
        f32x4 acc = zero4;
#pragma unroll
        for (int s4 = 0; s4 < kHM / 4; ++s4) {
          const int mm = 4 * s4 + lq;
          acc = __builtin_amdgcn_mfma_f32_16x16x4f32(g2s[mm * kGS + c0 + l16],
                                                     fmaxf(z1p[mm * (kHU + 1) + u0 + l16], 0.0f), acc, 0, 0, 0);
        }
        const float accs[4] = {acc.x, acc.y, acc.z, acc.w};
        const int uu = u0 + l16;
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const int c = c0 + 4 * lq + r;
          const float wo = wold[c * (kHU + 1) + uu];
          float nw;
          if (a.hb) {  // heavy-ball step with decay
            float d = accs[r] + a.wd * wo;
            if (a.vw2 && c < C) {
              float* vp = a.vw2 + (int64_t)p * a.w_pitch + (int64_t)c * Hp + ht * kHU + uu;
              d = a.mu * *vp + d;
              *vp = d;
            }
            nw = wo - lr * d;
          } else {
            nw = wo - lr * accs[r];
          }
          if (c < C) w2[(int64_t)c * Hp + ht * kHU + uu] = nw;
          ws[c * (kHU + 1) + uu] = c < C ? nw : 0.0f;
        }
      }
    }
    if (ht == 0 && wave == 3 && lane < KC) {  // slice 0: b2[c = lane] (= u)
      float sb = 0.0f;
      for (int mm = 0; mm < M; ++mm) sb += g2s[mm * kGS + lane];
      if (a.hb && lane < C) {  // heavy-ball step with decay
        sb += a.wd * b2v;
        if (a.vb2) {
          float* vp = a.vb2 + (int64_t)p * a.w_pitch + lane;
          sb = a.mu * *vp + sb;
          *vp = sb;
        }
      }
      const float nb2 = lane < C ? b2v - lr * sb : 0.0f;
      if (lane < C) b2[lane] = nb2;
      b2l[lane] = nb2;
    }
  } else {  // step 0: (B)'s W2 slice, b1 and b2 as they are
#pragma unroll
    for (int q = 0; q < kWq; ++q) {
      const int c = g + kG * q;
      ws[c * (kHU + 1) + u] = c < C ? wv[q] : 0.0f;
    }
    if (tid < kHU) bs[tid] = b1h;
    if (ht == 0 && tid < KC) b2l[tid] = tid < C ? b2v : 0.0f;  // tid = u here
  }
  if (k >= a.K1) return;

  // (B): step k's forward for this slice.
#pragma unroll
  for (int k2 = 0; k2 < NK - 1; ++k2)
    if (k2 < kc - 1) {
      const f32x4 v = a.hb ? a.hb[hb_index(HB_U, kc - 1 - k2)] * gv[k2] : gv[k2];  // heavy-ball: u_{k-1-k2}
      *(f32x4*)&gsl(k2, gsm, 4 * gc4) = gsm < M ? v : zero4;
    }
#pragma unroll
  for (int k2 = 0; k2 < NK; ++k2)
    if (k2 < kc && tid < Mp * Mp / 4) {
      const int rem = 4 * tid;
      float* gp = &grl[(k2 * kHM + rem / Mp) * kGrlS + rem % Mp];
      gp[0] = gr[k2].x;
      gp[1] = gr[k2].y;
      gp[2] = gr[k2].z;
      gp[3] = gr[k2].w;
    }
  float* zs = region;           // [kHM][kHU + 1]
  float* cbuf = region + kZs;   // [4][kHM][kHM + 1]
  // Step k's partial sums (splits added in order), then b1.
  f32x4 z = zero4;
#pragma unroll
  for (int ks = 0; ks < kPv; ++ks)
    if (ks < a.KS) z += pv[ks];
  for (int ks = kPv; ks < a.KS; ++ks) {
    const float* pm = a.part + k * step_floats + ((int64_t)p * Mp + (rr < M ? rr : 0)) * Hp + h4;
    z += *(const f32x4*)(pm + ks * a.split);
  }
  if (a.hb) {  // heavy-ball block: p_k X_k W^T + q_k X_k V^T
    z = a.hb[hb_index(HB_P, k)] * z;
    if (a.partv && k > 0) {
      const float* pv = a.partv + k * step_floats + ((int64_t)p * Mp + (rr < M ? rr : 0)) * Hp + h4;
      f32x4 zv = zero4;
      for (int ks = 0; ks < a.KSv; ++ks) zv += *(const f32x4*)(pv + ks * a.splitv);
      z += a.hb[hb_index(HB_Q, k)] * zv;
    }
  }
  __syncthreads();
  z += f32x4{bs[4 * u4], bs[4 * u4 + 1], bs[4 * u4 + 2], bs[4 * u4 + 3]};
  if (kc > 0) {
    // The correction sum_{k2<k} gram[k][k2] G1[k2] of this slice is a 32 x 32
    // product with k*Mp terms, as 32x32x2 MFMAs (lane (l, h): Gram row l and
    // error row l of unit l at s2 = 2j + h).  Wave w takes the pairs j of
    // its quarter of the minibatch for every k2; the four partial tiles are
    // added in wave order.  Staged errors are zero past row M, so the sum
    // runs over the padded minibatch (Mp = 16 or 32).
    const int l32 = lane & 31, lhi = lane >> 5, jq = Mp / 8;
    f32x16 acc;
#pragma unroll
    for (int r = 0; r < 16; ++r) acc[r] = 0.0f;
    for (int k2 = 0; k2 < kc; ++k2)
      for (int jj = 0; jj < jq; ++jj) {
        const int j = wave * jq + jj;
        acc = __builtin_amdgcn_mfma_f32_32x32x2f32(grl[(k2 * kHM + l32) * kGrlS + 2 * j + lhi],
                                                   gsl(k2, 2 * j + lhi, l32), acc, 0, 0, 0);
      }
#pragma unroll
    for (int r = 0; r < 16; ++r)
      cbuf[(wave * kHM + 8 * (r >> 2) + 4 * lhi + (r & 3)) * (kHM + 1) + l32] = acc[r];
    __syncthreads();
    f32x4 c = zero4;
#pragma unroll
    for (int w = 0; w < 4; ++w) {
      const float* cr = cbuf + (w * kHM + rr) * (kHM + 1) + 4 * u4;
      c += f32x4{cr[0], cr[1], cr[2], cr[3]};
    }
    if (a.hb)
      z += c;  // the coefficients (u_n, which carry -lr) are in the staged errors
    else
      z -= lr * c;
  }
  const bool mok = rr < M;
  if (mok) *(f32x4*)(a.Z1 + ((int64_t)p * Mp + rr) * Hp + h4) = z;
  zs[rr * (kHU + 1) + 4 * u4 + 0] = mok ? fmaxf(z.x, 0.0f) : 0.0f;
  zs[rr * (kHU + 1) + 4 * u4 + 1] = mok ? fmaxf(z.y, 0.0f) : 0.0f;
  zs[rr * (kHU + 1) + 4 * u4 + 2] = mok ? fmaxf(z.z, 0.0f) : 0.0f;
  zs[rr * (kHU + 1) + 4 * u4 + 3] = mok ? fmaxf(z.w, 0.0f) : 0.0f;
  __syncthreads();
  // Partial logits of this slice, relu(Z1) (32 x 32) times the W2 slice
  // transposed, as 16x16x4 MFMAs: wave w takes samples 16 (w & 1) .. +15
  // and classes 16 (w >> 1) .. +15 (lane (i, q): sample row i and class
  // row i at unit 4s + q; result rows 4q .. 4q+3 of class column i).
  if (wave < 2 * (KC / 16)) {
    const int l16 = lane & 15, lq = lane >> 4, m0 = 16 * (wave & 1), c0 = 16 * (wave >> 1);
    f32x4 acc = zero4;
#pragma unroll
    for (int s4 = 0; s4 < kHU / 4; ++s4)
      acc = __builtin_amdgcn_mfma_f32_16x16x4f32(zs[(m0 + l16) * (kHU + 1) + 4 * s4 + lq],
                                                 ws[(c0 + l16) * (kHU + 1) + 4 * s4 + lq], acc, 0, 0, 0);
    float* plo = a.PL + (int64_t)(k & 1) * a.pl_half;
    const int c = c0 + l16;
    const float bb = ht == 0 ? b2l[c] : 0.0f;  // slice 0 adds b2
    const float accs[4] = {acc.x, acc.y, acc.z, acc.w};
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const int mm = m0 + 4 * lq + r;
      if (mm < M && c < C) plo[(((int64_t)p * Mp + mm) * Cp + c) * htiles + ht] = accs[r] + bb;
    }
  }
}

void launch_head_step(hipStream_t s, const HeadStepArgs& a, int k) {
  const int htiles = a.Hp / kHU;
  // Blocks of up to 4 steps take the 3-slot variant (fewer idle prefetches).
  if (a.C <= 16) {
    if (a.K1 <= 4)
      launch(k_head_step<16, 3>, a.P * htiles, 256, 0, s, a, htiles, k);
    else
      launch(k_head_step<16, kCorrMaxK>, a.P * htiles, 256, 0, s, a, htiles, k);
  } else {
    if (a.K1 <= 4)
      launch(k_head_step<32, 3>, a.P * htiles, 256, 0, s, a, htiles, k);
    else
      launch(k_head_step<32, kCorrMaxK>, a.P * htiles, 256, 0, s, a, htiles, k);
  }
}

// Evaluation: one wave per row m < M of a chunk.  Logits l_c = b_c + sum_ks
// part[ks][m][c] for c < C (splits added in order); the row's softmax
// cross-entropy log(sum_c exp(l_c - max)) + max - l_y and whether the first
// largest logit is the label's.
__global__ __launch_bounds__(256) void k_eval_rows(const float* __restrict__ part, int KS, int64_t split,
                                                   const float* __restrict__ bias, const int32_t* __restrict__ y,
                                                   int M, int Cp, int C, float* __restrict__ loss,
                                                   int32_t* __restrict__ hit) {
  const int m = blockIdx.x * 4 + (threadIdx.x >> 6);
  const int lane = threadIdx.x & 63;
  if (m >= M) return;
  const float* pr = part + (int64_t)m * Cp;
  auto logit = [&](int c) {
    float v = bias[c];
    for (int ks = 0; ks < KS; ++ks) v += pr[ks * split + c];
    return v;
  };
  float best = -INFINITY;
  int bestc = 0x7fffffff;
  for (int c = lane; c < C; c += 64) {
    const float v = logit(c);
    if (v > best) {  // c increases within a lane: the first index wins ties
      best = v;
      bestc = c;
    }
  }
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) {
    const float ob = __shfl_xor(best, o, 64);
    const int oc = __shfl_xor(bestc, o, 64);
    if (ob > best || (ob == best && oc < bestc)) {
      best = ob;
      bestc = oc;
    }
  }
  float sum = 0.0f;
  for (int c = lane; c < C; c += 64) sum += expf(logit(c) - best);
  sum = wave_sum(sum);
  if (lane == 0) {
    const int yy = y[m];
    loss[m] = logf(sum) + best - logit(yy);
    hit[m] = bestc == yy ? 1 : 0;
  }
}

void launch_eval_rows(hipStream_t s, const float* part, int KS, int64_t split, const float* bias, const int32_t* y,
                      int M, int Cp, int C, float* loss, int32_t* hit) {
  launch(k_eval_rows, (M + 3) / 4, 256, 0, s, part, KS, split, bias, y, M, Cp, C, loss, hit);
}

void launch_reduce_bias(hipStream_t s, const float* part, int KS, const float* bias, int64_t w_pitch, float* Z,
                        int P, int M, int Mp, int N) {
  int64_t g = ((int64_t)P * Mp * N + 255) / 256;
  launch(k_reduce_bias, (unsigned)(g < 4096 ? g : 4096), 256, 0, s, part, KS, bias, w_pitch, Z, P, M, Mp, N);
}

void launch_softmax_grad(hipStream_t s, const float* part, int KS, const float* bias, int64_t w_pitch,
                         const int32_t* labels, const int32_t* idx, float* G, int P, int M, int Mp, int C, int Cp) {
  const int rows = P * M;
  const unsigned grid = (unsigned)((rows + 3) / 4);
  // Up to 64 classes the plain kernel (measured faster there: 4.1 against
  // 7.0 us at 10 classes); the register form from 65 to 1024 classes (6.9
  // against 18.7 us at 1000).
  const int npl = (C + 63) / 64;
  if (npl <= 1)
    launch(k_softmax_grad, grid, 256, 0, s, part, KS, bias, w_pitch, labels, idx, G, P, M, Mp, C, Cp);
  else if (npl <= 2)
    launch(k_softmax_grad_reg<2>, grid, 256, 0, s, part, KS, bias, w_pitch, labels, idx, G, P, M, Mp, C, Cp);
  else if (npl <= 4)
    launch(k_softmax_grad_reg<4>, grid, 256, 0, s, part, KS, bias, w_pitch, labels, idx, G, P, M, Mp, C, Cp);
  else if (npl <= 8)
    launch(k_softmax_grad_reg<8>, grid, 256, 0, s, part, KS, bias, w_pitch, labels, idx, G, P, M, Mp, C, Cp);
  else if (npl <= 16)
    launch(k_softmax_grad_reg<16>, grid, 256, 0, s, part, KS, bias, w_pitch, labels, idx, G, P, M, Mp, C, Cp);
  else
    launch(k_softmax_grad, grid, 256, 0, s, part, KS, bias, w_pitch, labels, idx, G, P, M, Mp, C, Cp);
}

void launch_scale_errors(hipStream_t s, const float* Gs, float* Gu, float* Gt, const float* hb, int K1, int64_t n) {
  const int64_t n4 = n / 4;
  int64_t gx = (n4 + 255) / 256;
  if (gx > 2048) gx = 2048;
  launch(k_scale_errors, dim3((unsigned)gx, (unsigned)K1), 256, 0, s, (const f32x4*)Gs, (f32x4*)Gu, (f32x4*)Gt, hb, K1,
         n4);
}

void launch_bwd_hidden(hipStream_t s, const float* G2, float* W2, int64_t w_pitch, const float* Z1, float* G1, int P,
                       int M, int Mp, int C, int Cp, int Hp, float* b1, const float* lr, float* vb1, float mu, float wd,
                       float* b2) {
  if (b1 && M > kBhM) {  // the b1 step needs every sample in one workgroup
    const int htiles = (Hp + 63) / 64;
    launch(k_bwd_hidden, P * htiles, 256, 0, s, G2, W2, w_pitch, Z1, G1, M, Mp, C, Cp, Hp, htiles, b1, lr);
    return;
  }
  const int htiles = Hp / kBhN, mtiles = (M + kBhM - 1) / kBhM;
  const unsigned grid = (unsigned)((int64_t)P * mtiles * htiles);
  if (b2)
    launch(k_bwd_hidden_mfma<true>, grid, 256, 0, s, G2, W2, w_pitch, Z1, G1, M, Mp, Cp, Hp, htiles, mtiles, b1, lr, vb1,
           mu, wd, b2);
  else
    launch(k_bwd_hidden_mfma<false>, grid, 256, 0, s, G2, W2, w_pitch, Z1, G1, M, Mp, Cp, Hp, htiles, mtiles, b1, lr,
           vb1, mu, wd, (float*)nullptr);
}

bool bwd_hidden_update_supported(int M, int Cp) { return M <= kBhM && Cp <= kBhMaxC; }

bool head_fused_supported(int Hp, int Cp) { return Cp <= 16 ? Hp <= 1024 : Cp <= 32 && Hp <= 512; }

int64_t head_fused_scratch_floats(int P, int Mp, int C, int Hp) {
  return (int64_t)P * (Mp / 16) * ((int64_t)(C + 1) * Hp + 32);
}

void launch_head_fused(hipStream_t s, const HeadFusedArgs& a) {
  const int grid = a.P * (a.Mp / 16), nt = 64 * kHfWaves;
  const int ks = a.KS >= 1 && a.KS <= 3 ? a.KS : 0;
#define HAV_HEAD_FUSED(KC_, HPM_)                                                 \
  do {                                                                           \
    if (ks == 1) launch(k_head_fused<KC_, HPM_, 1>, grid, nt, 0, s, a);          \
    else if (ks == 2) launch(k_head_fused<KC_, HPM_, 2>, grid, nt, 0, s, a);     \
    else if (ks == 3) launch(k_head_fused<KC_, HPM_, 3>, grid, nt, 0, s, a);     \
    else launch(k_head_fused<KC_, HPM_, 0>, grid, nt, 0, s, a);                  \
  } while (0)
  if (a.Cp <= 16 && a.Hp <= 512)
    HAV_HEAD_FUSED(16, 512);
  else if (a.Cp <= 16)
    HAV_HEAD_FUSED(16, 1024);
  else
    HAV_HEAD_FUSED(32, 512);
#undef HAV_HEAD_FUSED
}

void launch_head_w2_step(hipStream_t s, const HeadFusedArgs& a) {
  const int nblk = ((a.C + 1) * (a.Hp / 4) + 255) / 256;
  launch(k_head_w2_step, a.P * nblk, 256, 0, s, a, nblk);
}

void launch_head_a(hipStream_t s, const float* part, int KS, const float* b1, const float* W2, const float* b2,
                   int64_t w_pitch, float* Z1, float* PL, int P, int M, int Mp, int C, int Cp, int Hp,
                   int64_t part_split) {
  const int htiles = Hp / kHU;
  const int64_t split = part_split > 0 ? part_split : (int64_t)P * Mp * Hp;
  if (C <= 16)
    launch(k_head_a<16>, P * htiles, 256, 0, s, part, KS, b1, W2, b2, w_pitch, Z1, PL, P, M, Mp, C, Cp, Hp, htiles,
           split);
  else
    launch(k_head_a<32>, P * htiles, 256, 0, s, part, KS, b1, W2, b2, w_pitch, Z1, PL, P, M, Mp, C, Cp, Hp, htiles,
           split);
}

void launch_head_b(hipStream_t s, const float* PL, float* W2, float* b1, float* b2, int64_t w_pitch,
                   const float* Z1, float* G1, const int32_t* labels, const int32_t* idx, int P, int M, int Mp, int C,
                   int Cp, int Hp, const float* lr, HeadMom mom) {
  const int htiles = Hp / kHU;
  if (C <= 16)
    launch(k_head_b<16>, P * htiles, 256, 0, s, PL, W2, b1, b2, w_pitch, Z1, G1, labels, idx, P, M, Mp, C, Cp, Hp,
           htiles, lr, mom);
  else
    launch(k_head_b<32>, P * htiles, 256, 0, s, PL, W2, b1, b2, w_pitch, Z1, G1, labels, idx, P, M, Mp, C, Cp, Hp,
           htiles, lr, mom);
}

}  // namespace hav
