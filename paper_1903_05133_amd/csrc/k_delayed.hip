// Kernels of the delayed first-layer update (include/hieravg.h,
// HIERAVG_UPDATE_DELAYED): within a block of K1 local steps (Algorithm 1,
// Sec. 3.1) every learner of a cluster starts from the same first weight
// block Wb, and after k steps its block is Wb - lr * sum_{k'<k} G_k'^T X_k'.
//
// k_fwd_blk:      the first-layer forward partials of all K1 steps of a block
//                 from the cluster copies (one GEMM per cluster and block).
// k_gram:         the Gram blocks X_k X_k'^T (k' < k) of each learner's
//                 minibatches in each block, which turn the forward from Wb
//                 into the forward from the learner's current block.
// k_block_update: the block-end cluster mean of the first weight block, as one
//                 update of the copy by the summed G^T X of the cluster.
#include <algorithm>

#include "internal.h"

namespace hav {

constexpr int kKC = 64;         // K floats per LDS chunk
constexpr int kLdsStride = 68;  // LDS row stride in floats (64 + 4: conflict-free 128-bit reads)
constexpr int kUM = 64;         // W rows per block-update workgroup
constexpr int kUN = 128;        // W columns per block-update workgroup
constexpr int kSC = 32;         // contraction rows per LDS stage
constexpr int kLA = kUM + 4;    // LDS row length of the error stage
constexpr int kLB = kUN + 4;    // LDS row length of the input stage and of the gradient tile

// Large-tile variant for the block-wide forward of delayed updates (many rows
// per weight copy): 1024 threads, output tile 128 rows x 128 columns, both
// operands staged through LDS (double-buffered, one barrier per 64-wide K
// chunk, the next chunk's loads in flight during the current chunk's MFMAs).
// Wave w owns the 32 x 32 block (rows 32*(w/4), columns 32*(w%4)) as one
// chain of 32x32x2 MFMAs (one accumulator chain per wave keeps the matrix
// pipe fuller than four interleaved 16x16x4 chains), so each SIMD
// interleaves four waves.  Lane (l, h) reads the 16-byte piece of k values
// 8q + 4h .. +3 of its row in both operands and feeds them to four MFMAs:
// MFMA e contracts k = 8q + e and 8q + 4 + e, a permutation of the chunk's k.
constexpr int kBT = 128;  // tile rows and columns
__global__ __launch_bounds__(1024) void k_fwd_blk(FwdArgs a, int ntiles, int mtiles) {
  __shared__ __attribute__((aligned(16))) float As[2][kBT * kLdsStride];
  __shared__ __attribute__((aligned(16))) float Ws[2][kBT * kLdsStride];
  const int bid = xcd_remap(blockIdx.x, gridDim.x);
  const int nt = bid % ntiles;
  const int mt = (bid / ntiles) % mtiles;
  const int ks = (bid / (ntiles * mtiles)) % a.KS;
  const int g = bid / (ntiles * mtiles * a.KS);
  const int GM = a.SG * a.Mp;
  const int nch = a.K / kKC;
  const int c0 = ks * a.cps;
  const int c1 = min(nch, c0 + a.cps);
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  const int l32 = lane & 31, lhi = lane >> 5;
  const int wm = (wave >> 2) * 32, wn = (wave & 3) * 32;
  const int mbase = mt * kBT, nbase = nt * kBT;
  const f32x4 zero4 = {0.f, 0.f, 0.f, 0.f};

  // Thread t stages pieces t and t + 1024 of each 128 x 64 chunk: row q/16,
  // 16-byte column piece q%16.
  const float* arow[2];
  const float* wrow[2];
  bool aok[2], wok[2];
  int off[2];
  const float* wp = a.W + (int64_t)(g / a.wdiv) * a.w_pitch;
  const float inv_mp = 1.0f / (float)a.Mp, inv_vs = 1.0f / (float)(a.vS > 0 ? a.vS : 1);
#pragma unroll
  for (int i = 0; i < 2; ++i) {
    const int q = tid + 1024 * i;
    const int r = q >> 4, c4 = q & 15;
    off[i] = r * kLdsStride + 4 * c4;
    const int m = mbase + r;
    const int jj = qdiv_small(m, a.Mp, inv_mp), sm = m - jj * a.Mp;
    aok[i] = m < GM && sm < a.M;
    const int v = aok[i] ? jj : 0;
    int64_t p = (int64_t)g * a.SG + v;
    if (a.vS > 0) {
      const int k = qdiv_small(v, a.vS, inv_vs);
      p = (int64_t)k * a.P + (int64_t)g * a.vS + (v - k * a.vS);
    }
    arow[i] = a.A + (int64_t)a.idx[p * a.M + (aok[i] ? sm : 0)] * a.lda + 4 * c4;
    const int n = nbase + r;
    wok[i] = n < a.N;
    wrow[i] = wp + (int64_t)(wok[i] ? n : 0) * a.ldw + 4 * c4;
  }
  f32x4 av[2], wv[2];
  auto load = [&](int c) {
    const int64_t o = (int64_t)c * kKC;
#pragma unroll
    for (int i = 0; i < 2; ++i) {
      av[i] = *(const f32x4*)(arow[i] + o);
      wv[i] = *(const f32x4*)(wrow[i] + o);
    }
  };
  auto store = [&](int buf) {
#pragma unroll
    for (int i = 0; i < 2; ++i) {
      *(f32x4*)&As[buf][off[i]] = aok[i] ? av[i] : zero4;
      *(f32x4*)&Ws[buf][off[i]] = wok[i] ? wv[i] : zero4;
    }
  };
  f32x16 acc;
#pragma unroll
  for (int r = 0; r < 16; ++r) acc[r] = 0.0f;
  auto compute = [&](int buf) {
#pragma unroll
    for (int q = 0; q < kKC / 8; ++q) {
      const f32x4 x = *(const f32x4*)&As[buf][(wm + l32) * kLdsStride + 8 * q + 4 * lhi];
      const f32x4 y = *(const f32x4*)&Ws[buf][(wn + l32) * kLdsStride + 8 * q + 4 * lhi];
#pragma unroll
      for (int e = 0; e < 4; ++e) acc = __builtin_amdgcn_mfma_f32_32x32x2f32(x[e], y[e], acc, 0, 0, 0);
    }
  };
  if (c0 < c1) {
    load(c0);
    store(0);
    __syncthreads();
    for (int c = c0; c < c1; ++c) {
      load(c + 1 < c1 ? c + 1 : c);  // the last chunk again at the end: in range, unused
      __builtin_amdgcn_sched_barrier(0);
      compute((c - c0) & 1);
      store((c - c0 + 1) & 1);
      __syncthreads();
    }
  }
  const int64_t PT = a.PT > 0 ? a.PT : a.P;
  const int col = nbase + wn + l32;
  if (col < a.N) {
    // The lane's rows 8i + e (e < 4) share one member (Mp is a multiple of
    // 16, GM of 16), so the row -> (member, sample) split runs once per i.
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int row0 = mbase + wm + 8 * i + 4 * lhi;
      if (row0 >= GM) continue;
      const int v = qdiv_small(row0, a.Mp, inv_mp), sm = row0 - v * a.Mp;
      int64_t p = (int64_t)g * a.SG + v;
      if (a.vS > 0) {
        const int k = qdiv_small(v, a.vS, inv_vs);
        p = (int64_t)k * a.P + (int64_t)g * a.vS + (v - k * a.vS);
      }
      float* dst = a.part + (((int64_t)ks * PT + p) * a.Mp + sm) * a.N + col;
#pragma unroll
      for (int e = 0; e < 4; ++e) dst[(int64_t)e * a.N] = acc[4 * i + e];
    }
  }
}

void launch_fwd_blk(hipStream_t s, const FwdArgs& a) {
  const int GM = a.SG * a.Mp;
  const int mtiles = (GM + kBT - 1) / kBT;
  const int ntiles = (a.N + kBT - 1) / kBT;
  const int groups = a.vS > 0 ? a.P / a.vS : a.P / a.SG;
  const unsigned grid = (unsigned)((int64_t)groups * a.KS * mtiles * ntiles);
  launch(k_fwd_blk, grid, 1024, 0, s, a, ntiles, mtiles);
}

// Split count of k_fwd_blk: about target_wg workgroups, no empty split.
void plan_split_blk(int groups, int rows, int N, int K, int* KS, int* cps, int target_wg) {
  const int64_t tiles = (int64_t)groups * ((rows + kBT - 1) / kBT) * ((N + kBT - 1) / kBT);
  const int nch = K / kKC;
  int ks = (int)std::max<int64_t>(1, (target_wg + tiles - 1) / tiles);
  ks = std::min(ks, nch);
  const int c = (nch + ks - 1) / ks;
  *KS = (nch + c - 1) / c;
  *cps = c;
}

// ------------------------------------------------------------ delayed update
// Tile of k_update_tn (64 rows x kUN columns of one group's W1), contracted
// over the K1*SG*B rows (step k, learner j, sample s) of the group in stages
// of 32 rows through two LDS buffers: each stage's loads are issued two
// stages ahead (two register sets) and each stage costs one barrier.  NTH/64
// waves split the tile into 32-row x (2*kUN/NW)-column blocks of 32x32x2
// MFMAs.
//
// Address arithmetic stays out of the stage loop (a SIMD's matrix core idles
// while it executes vector ALU instructions, so every such instruction per
// stage costs MFMA time): the input-row offset of every contraction row is
// tabulated in LDS once, in 64-float units, and with kAligned (B a multiple
// of 32) a stage is 32 consecutive samples of one (step, learner), whose
// error rows follow from scalar counters.  Input rows past the contraction
// and columns past the block are read from valid rows and columns instead of
// being masked: they only meet zero error rows or feed discarded outputs.
template <int NTH, bool kAligned>
__global__ __launch_bounds__(NTH) __attribute__((amdgpu_waves_per_eu(6))) void k_block_update(BlkArgs a, int mtiles,
                                                                                         int ntiles) {
  constexpr int NW = NTH / 64;            // waves
  constexpr int kWCn = NW / 2;            // waves across the columns (two 32-row blocks)
  constexpr int kWN = kUN / kWCn;         // columns per wave
  constexpr int kNA = kWN / 32;           // 32x32 accumulators per wave
  constexpr int kStage = kSC * (kLA + kLB);
  constexpr int kLds = 2 * kStage > kUM * kLB ? 2 * kStage : kUM * kLB;
  __shared__ __attribute__((aligned(16))) float lds[kLds];
  extern __shared__ uint32_t xtb[];  // [K1*SG*B] input row offset of each contraction row, / 64
  float* Gt = lds;  // [kUM][kLB] gradient tile (after the stages)
  // Tiles that share minibatch rows (same group and columns) are neighbours.
  const int bid = xcd_remap(blockIdx.x, gridDim.x);
  const int mt = bid % mtiles;
  const int nt = (bid / mtiles) % ntiles;
  const int g = bid / (ntiles * mtiles);
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  const int l32 = lane & 31, lhi = lane >> 5;
  const int mrow0 = mt * kUM, ncol0 = nt * kUN;
  const int wn = (wave % kWCn) * kWN, wm = (wave / kWCn) * 32;
  const bool wave_on = ncol0 + wn < a.Ncols;
  const int SB = a.SG * a.B;
  const int R = a.K1 * SB;  // contraction rows
  const int nst = (R + kSC - 1) / kSC;
  const f32x4 zero4 = {0.f, 0.f, 0.f, 0.f};

  constexpr int kXP = kUN / 4, kXR = NTH / kXP, kXL = kSC / kXR;
  constexpr int kGL = kSC * (kUM / 4) / NTH;  // G pieces per thread per stage
  const int xc4 = tid % kXP, xr0 = tid / kXP;
  const bool xcol_ok = ncol0 + 4 * xc4 < a.Ncols;
  const int xcol = xcol_ok ? ncol0 + 4 * xc4 : 0;
  const float* Xc = a.X + xcol;
  // G piece i of this thread: stage row (qq >> 4), columns m .. m+3 (a row
  // past Mrows reads row 0: its gradient row is discarded).
  int64_t goff[kGL];
#pragma unroll
  for (int i = 0; i < kGL; ++i) {
    const int qq = tid + NTH * i, m = mrow0 + 4 * (qq & 15);
    goff[i] = (int64_t)(qq >> 4) * a.ldg + (m < a.Mrows ? m : 0);
  }
  // Row r of the contraction: step k, learner g*SG + j, sample s (r < 2^24).
  const float inv_sb = 1.0f / (float)SB, inv_b = 1.0f / (float)a.B;
  auto gx_row = [&](int r, int64_t& grow, int64_t& irow) {
    const int k = qdiv_small(r, SB, inv_sb), rem = r - k * SB;
    const int j = qdiv_small(rem, a.B, inv_b), sm = rem - j * a.B;
    const int64_t kp = (int64_t)k * a.P + (int64_t)g * a.SG + j;
    grow = kp * a.Mp + sm;
    irow = kp * a.B + sm;
  };
  // Stage registers: two sets, so each stage's loads are issued two stages
  // before its rows go to LDS (two blocks of MFMAs of latency hiding).
  struct StageRegs {
    f32x4 ga[kGL], xb[kXL];
    bool gok[kGL];
  };
  StageRegs RA, RB;
  // The input row of every contraction row, read once into LDS: the stage
  // loads then depend on no other global load (loads complete in issue
  // order, so an index load in the loop would make the wait for it a wait
  // for the stage data issued before it).  The launcher checks that the
  // offsets fit 32 bits in 64-float units.
  for (int r = tid; r < R; r += NTH) {
    int64_t grow, irow;
    gx_row(r, grow, irow);
    xtb[r] = (uint32_t)(((int64_t)a.idx[irow] * a.ldx) >> 6);
  }
  __syncthreads();
  // kAligned (Mp = B): the SG learners of a step are consecutive error rows,
  // so the next stage to load starts gb_off floats into G and the offset
  // grows by 32 rows per stage, plus the other learners' rows at each step
  // boundary (every SB/32 stages).  load_stage runs for st = 0, 1, 2, ... in
  // order; past the end it reloads the last stage.
  int64_t gb_off = (int64_t)g * a.SG * a.Mp * a.ldg;
  int st_in_step = 0;
  const int stages_per_step = SB / kSC;
  const int64_t stage_step = (int64_t)kSC * a.ldg;
  const int64_t step_jump = (int64_t)(a.P - a.SG) * a.Mp * a.ldg;
  auto load_stage = [&](int st, StageRegs& q) {
    const int s0 = (st < nst ? st : nst - 1) * kSC;  // past the end: the last stage again
    if constexpr (kAligned) {
      const float* gb = a.G + gb_off;
#pragma unroll
      for (int i = 0; i < kGL; ++i) q.ga[i] = *(const f32x4*)(gb + goff[i]);
      if (st < nst - 1) {
        gb_off += stage_step;
        if (++st_in_step == stages_per_step) {
          st_in_step = 0;
          gb_off += step_jump;
        }
      }
    } else {
#pragma unroll
      for (int i = 0; i < kGL; ++i) {  // G rows s0 .. s0+32, columns mrow0 .. +64
        const int qq = tid + NTH * i;
        const int r = s0 + (qq >> 4), m = mrow0 + 4 * (qq & 15);
        q.gok[i] = r < R;
        int64_t grow, irow;
        gx_row(q.gok[i] ? r : 0, grow, irow);
        q.ga[i] = *(const f32x4*)(a.G + grow * a.ldg + (m < a.Mrows ? m : 0));
      }
    }
#pragma unroll
    for (int i = 0; i < kXL; ++i) {  // X rows of contraction rows s0 + xr0 + kXR*i
      const int r = s0 + xr0 + kXR * i;
      q.xb[i] = *(const f32x4*)(Xc + ((uint64_t)xtb[kAligned || r < R ? r : 0] << 6));
    }
  };
  auto store_stage = [&](int buf, const StageRegs& q) {
    float* As = lds + buf * kStage;
    float* Bs = As + kSC * kLA;
#pragma unroll
    for (int i = 0; i < kGL; ++i) {
      const int qq = tid + NTH * i;
      *(f32x4*)&As[(qq >> 4) * kLA + 4 * (qq & 15)] = kAligned || q.gok[i] ? q.ga[i] : zero4;
    }
#pragma unroll
    for (int i = 0; i < kXL; ++i) *(f32x4*)&Bs[(xr0 + kXR * i) * kLB + 4 * xc4] = q.xb[i];
  };

  f32x16 acc[kNA];
#pragma unroll
  for (int j = 0; j < kNA; ++j)
#pragma unroll
    for (int r = 0; r < 16; ++r) acc[j][r] = 0.0f;
  auto mfma_stage = [&](int buf) {
    if (!wave_on) return;
    const float* As = lds + buf * kStage;
    const float* Bs = As + kSC * kLA;
    __builtin_amdgcn_s_setprio(1);
#pragma unroll
    for (int ss = 0; ss < kSC; ss += 2) {
      const int sr = ss + lhi;
      const float av = As[sr * kLA + wm + l32];
#pragma unroll
      for (int j = 0; j < kNA; ++j)
        acc[j] = __builtin_amdgcn_mfma_f32_32x32x2f32(av, Bs[sr * kLB + wn + 32 * j + l32], acc[j], 0, 0, 0);
    }
    __builtin_amdgcn_s_setprio(0);
  };

  load_stage(0, RA);
  load_stage(1, RB);
  store_stage(0, RA);
  __syncthreads();
  // Iteration st: loads of stage st+2 go out, the MFMAs of stage st (LDS
  // buffer st&1) run, stage st+1 goes to the other buffer.  Unrolled by two
  // so each register set is named statically.
  for (int st = 0; st < nst; st += 2) {
    load_stage(st + 2, RA);
    __builtin_amdgcn_sched_barrier(0);
    mfma_stage(0);
    store_stage(1, RB);
    __syncthreads();
    if (st + 1 >= nst) break;
    load_stage(st + 3, RB);
    __builtin_amdgcn_sched_barrier(0);
    mfma_stage(1);
    store_stage(0, RA);
    __syncthreads();
  }

  // Base tile (16-byte pieces, thread t: column piece t%kXP of rows t/kXP +
  // kXR*i), loaded only now so that its registers are free during the
  // contraction (three workgroups per CU); its latency overlaps the
  // accumulator transfer to LDS.
  constexpr int kWL = kUM / kXR;
  const float* Wb = a.Wb + (int64_t)g * a.wb_pitch;
  f32x4 wv[kWL];
#pragma unroll
  for (int i = 0; i < kWL; ++i) {
    const int row = mrow0 + xr0 + kXR * i;
    wv[i] = *(const f32x4*)(Wb + (row < a.Mrows && xcol_ok ? (int64_t)row * a.ldw + xcol : 0));
  }
#pragma unroll
  for (int j = 0; j < kNA; ++j)
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      const int row = wm + 8 * (r >> 2) + 4 * lhi + (r & 3);
      Gt[row * kLB + wn + 32 * j + l32] = acc[j][r];
    }
  __syncthreads();
  float* Wo = a.Wo + (int64_t)g * a.wo_pitch;
  const float lr_eff = *a.lr / a.lr_div;
#pragma unroll
  for (int i = 0; i < kWL; ++i) {
    const int rl = xr0 + kXR * i, row = mrow0 + rl;
    if (xcol_ok && row < a.Mrows) {
      const f32x4 gsum = *(const f32x4*)&Gt[rl * kLB + 4 * xc4];
      *(f32x4*)(Wo + (int64_t)row * a.ldw + xcol) = wv[i] - lr_eff * gsum;
    }
  }
}

#ifndef HAV_BLK_THREADS
#define HAV_BLK_THREADS 512
#endif
void launch_block_update(hipStream_t s, const BlkArgs& a) {
  const int mtiles = (a.Mrows + kUM - 1) / kUM;
  const int ntiles = (a.Ncols + kUN - 1) / kUN;
  const unsigned grid = (unsigned)((int64_t)(a.P / a.SG) * mtiles * ntiles);
  const uint32_t shmem = sizeof(uint32_t) * a.K1 * a.SG * a.B;
  if (a.B % kSC == 0)
    launch(k_block_update<HAV_BLK_THREADS, true>, grid, HAV_BLK_THREADS, shmem, s, a, mtiles, ntiles);
  else
    launch(k_block_update<HAV_BLK_THREADS, false>, grid, HAV_BLK_THREADS, shmem, s, a, mtiles, ntiles);
}

// ------------------------------------------------------------ Gram blocks
// One workgroup per (learner p, block b, K split ks): all step pairs k2 < k of
// the block at once.  The K1*Bp minibatch rows of the block (gathered, this
// split's input features) are staged through LDS 64 features at a time, the
// next chunk's loads in flight during the current chunk's MFMAs; each wave
// owns a fixed set of the 16x16 output blocks of the lower block triangle
// (16x16x4 MFMAs, the k permutation of k_fwd_nt).  Every minibatch row is
// read once per split; the consumer adds the KSG partial sums.
constexpr int kGramMaxBlocks = 28;  // 16x16 output blocks per wave (K1 <= 8, Bp <= 32)
template <int NB, int ROWS>
__global__ __launch_bounds__(256) void k_gram(const float* __restrict__ X, int64_t ldx, int K,
                                              const int32_t* __restrict__ idx, float* __restrict__ gram, int P,
                                              int K1, int B, int Bp, int KSG) {
  constexpr int kRows = ROWS;         // LDS capacity in rows (K1 * Bp <= ROWS)
  constexpr int kL = kKC + 4;         // LDS row length
  constexpr int kLPT = kRows * (kKC / 4) / 256;  // 16-byte pieces per thread per chunk (at most)
  __shared__ __attribute__((aligned(16))) float xs[kRows * kL];
  const int ks = blockIdx.x % KSG;
  const int pb = blockIdx.x / KSG;  // p + P * b
  const int p = pb % P, b = pb / P;
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  const int lrow = lane & 15, lgrp = lane >> 4;
  const int rows = K1 * Bp;
  const int nch = K / kKC;
  const int c0 = (int)((int64_t)nch * ks / KSG), c1 = (int)((int64_t)nch * (ks + 1) / KSG);
  // Row r = k*Bp + s of the block: sample s of step b*K1 + k (rows past B: zero).
  const float* src[kLPT];
  bool ok[kLPT];
  int off[kLPT];
#pragma unroll
  for (int i = 0; i < kLPT; ++i) {
    const int q = tid + 256 * i;
    const int r = q >> 4, c4 = q & 15;
    const int k = r / Bp, sm = r - k * Bp;
    ok[i] = r < rows && sm < B;
    const int64_t e = ((int64_t)(b * K1 + (ok[i] ? k : 0)) * P + p) * B + (ok[i] ? sm : 0);
    src[i] = X + (int64_t)idx[e] * ldx + 4 * c4;
    off[i] = (r < kRows ? r : 0) * kL + 4 * c4;
  }
  // Output blocks of this wave: block e = wave + 4*t over the lower triangle
  // (pair (k, k2), row block mb, column block nb).
  const int mbs = Bp / 16;
  const int nblk = K1 * (K1 - 1) / 2 * mbs * mbs;
  int arow[NB], brow[NB];
  bool bon[NB];
#pragma unroll
  for (int t = 0; t < NB; ++t) {
    const int e = wave + 4 * t;
    bon[t] = e < nblk;
    int pr = (bon[t] ? e : 0) / (mbs * mbs), rem = (bon[t] ? e : 0) % (mbs * mbs);
    int k = 1, k2 = pr;
    while (k2 >= k) {
      k2 -= k;
      ++k;
    }
    arow[t] = (k * Bp + 16 * (rem / mbs) + lrow) * kL + 4 * lgrp;
    brow[t] = (k2 * Bp + 16 * (rem % mbs) + lrow) * kL + 4 * lgrp;
  }
  const f32x4 zero4 = {0.f, 0.f, 0.f, 0.f};
  f32x4 acc[NB];
#pragma unroll
  for (int t = 0; t < NB; ++t) acc[t] = zero4;
  f32x4 v[kLPT];
  auto load = [&](int c) {
#pragma unroll
    for (int i = 0; i < kLPT; ++i) v[i] = *(const f32x4*)(src[i] + (int64_t)c * kKC);
  };
  auto store = [&]() {
#pragma unroll
    for (int i = 0; i < kLPT; ++i)
      if (tid + 256 * i < rows * (kKC / 4)) *(f32x4*)&xs[off[i]] = ok[i] ? v[i] : zero4;
  };
  if (c0 < c1) {
    load(c0);
    for (int c = c0; c < c1; ++c) {
      store();
      __syncthreads();
      load(c + 1 < c1 ? c + 1 : c);  // next chunk in flight (the last again at the end)
      __builtin_amdgcn_sched_barrier(0);
#pragma unroll
      for (int t = 0; t < NB; ++t) {
        if (!bon[t]) continue;
#pragma unroll
        for (int q = 0; q < kKC / 16; ++q) {
          const f32x4 x = *(const f32x4*)&xs[arow[t] + 16 * q];
          const f32x4 y = *(const f32x4*)&xs[brow[t] + 16 * q];
#pragma unroll
          for (int i = 0; i < 4; ++i) acc[t] = __builtin_amdgcn_mfma_f32_16x16x4f32(x[i], y[i], acc[t], 0, 0, 0);
        }
      }
      __syncthreads();
    }
  }
  // gram[ks][b][p][k][k2][s][s2]
#pragma unroll
  for (int t = 0; t < NB; ++t) {
    if (!bon[t]) continue;
    const int e = wave + 4 * t;
    const int pr = e / (mbs * mbs), rem = e % (mbs * mbs);
    int k = 1, k2 = pr;
    while (k2 >= k) {
      k2 -= k;
      ++k;
    }
    const int K2n = gridDim.x / (KSG * P);
    float* out = gram + (((((int64_t)ks * K2n + b) * P + p) * K1 + k) * K1 + k2) * Bp * Bp;
#pragma unroll
    for (int r = 0; r < 4; ++r)
      out[(16 * (rem / mbs) + 4 * lgrp + r) * Bp + 16 * (rem % mbs) + lrow] = acc[t][r];
  }
}

// gram[0] += gram[1] + ... + gram[KSG-1] over the blocks k2 < k (added in
// split order), so the consumer reads one sum.  Element i enumerates
// (block and learner bp, step pair, 16-byte piece q of the Bp x Bp block).
__global__ __launch_bounds__(256) void k_gram_reduce(float* __restrict__ gram, int64_t split, int64_t n4, int K1,
                                                     int pairs, int blk4, int KSG) {
  f32x4* g = (f32x4*)gram;
  const int64_t s4 = split / 4;
  for (int64_t i = blockIdx.x * 256ll + threadIdx.x; i < n4; i += (int64_t)gridDim.x * 256) {
    const int q = (int)(i % blk4);
    const int64_t t = i / blk4;
    const int pr = (int)(t % pairs);
    const int64_t bp = t / pairs;
    int k = 1, k2 = pr;
    while (k2 >= k) {
      k2 -= k;
      ++k;
    }
    const int64_t o = ((bp * K1 + k) * K1 + k2) * blk4 + q;
    f32x4 v = g[o];
    for (int t2 = 1; t2 < KSG; ++t2) v += g[t2 * s4 + o];
    g[o] = v;
  }
}

int gram_splits(int P, int K2, int K) {
  // about two workgroups per CU, at least two 64-wide chunks per split
  const int target = 512;
  int ksg = (target + P * K2 - 1) / (P * K2);
  return std::max(1, std::min(ksg, K / kKC / 2));
}

void launch_gram(hipStream_t s, const float* X, int64_t ldx, int K, const int32_t* idx, float* gram, int P, int K1,
                 int K2, int B, int Bp, int KSG) {
  const int nblk = K1 * (K1 - 1) / 2 * (Bp / 16) * (Bp / 16);
  if (nblk == 0) return;
  const unsigned grid = (unsigned)((int64_t)P * K2 * KSG);
  const int nb = (nblk + 3) / 4;
#define HAV_GRAM(N_, R_) launch(k_gram<N_, R_>, grid, 256, 0, s, X, ldx, K, idx, gram, P, K1, B, Bp, KSG)
  if (K1 * Bp <= 128) {
    if (nb <= 2)
      HAV_GRAM(2, 128);
    else if (nb <= 6)
      HAV_GRAM(6, 128);
    else
      HAV_GRAM(12, 128);
  } else {
    if (nb <= 12)
      HAV_GRAM(12, 256);
    else
      HAV_GRAM(kGramMaxBlocks, 256);
  }
#undef HAV_GRAM
}

void launch_gram_reduce(hipStream_t s, float* gram, int P, int K1, int K2, int Bp, int KSG) {
  const int64_t split = (int64_t)K2 * P * K1 * K1 * Bp * Bp;
  const int pairs = K1 * (K1 - 1) / 2, blk4 = Bp * Bp / 4;
  const int64_t n4 = (int64_t)K2 * P * pairs * blk4;
  const int64_t g = std::min<int64_t>((n4 + 255) / 256, 2048);
  launch(k_gram_reduce, (unsigned)g, 256, 0, s, gram, split, n4, K1, pairs, blk4, KSG);
}

}  // namespace hav
