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
constexpr int kLB = kUN + 4;    // LDS row length of the input stage and of the gradient tile

// Large-tile variant for the block-wide forward of delayed updates (many rows
// per weight copy): 1024 threads, output tile 128 rows x 128 columns, both
// operands staged through LDS (double-buffered, one barrier per 64-wide K
// chunk).  The global loads run two chunks ahead in two register sets: the
// set that goes to LDS after a chunk's MFMAs was loaded a whole chunk
// earlier, so no wave waits on memory in the middle of its MFMA chain (with
// loads one chunk ahead, the four waves of a SIMD all stalled on the same
// fresh loads early in every chunk).
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
  // Tile (nt, mt, ks, g) of this workgroup: float-reciprocal quotients (a few
  // vector instructions each, where an integer division takes dozens).
  const int bid = xcd_remap(blockIdx.x, gridDim.x);
  const int q1 = qdiv_small(bid, ntiles, qdiv_inv(ntiles)), nt = bid - q1 * ntiles;
  const int q2 = qdiv_small(q1, mtiles, qdiv_inv(mtiles)), mt = q1 - q2 * mtiles;
  const int g = qdiv_small(q2, a.KS, qdiv_inv(a.KS)), ks = q2 - g * a.KS;
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
  const float inv_mp = qdiv_inv(a.Mp), inv_vs = qdiv_inv(a.vS > 0 ? a.vS : 1);
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
  // Two register sets: the loads of chunk c + 2 go out while chunk c is
  // contracted and chunk c + 1 (loaded one chunk earlier) goes to LDS.
  f32x4 av2[2], wv2[2];
  auto load2 = [&](int c) {
    const int64_t o = (int64_t)c * kKC;
#pragma unroll
    for (int i = 0; i < 2; ++i) {
      av2[i] = *(const f32x4*)(arow[i] + o);
      wv2[i] = *(const f32x4*)(wrow[i] + o);
    }
  };
  auto store2 = [&](int buf) {
#pragma unroll
    for (int i = 0; i < 2; ++i) {
      *(f32x4*)&As[buf][off[i]] = aok[i] ? av2[i] : zero4;
      *(f32x4*)&Ws[buf][off[i]] = wok[i] ? wv2[i] : zero4;
    }
  };
  if (c0 < c1) {
    load(c0);
    load2(c0 + 1 < c1 ? c0 + 1 : c0);
    store(0);
    __syncthreads();
    for (int c = c0; c < c1; c += 2) {
      load(c + 2 < c1 ? c + 2 : c1 - 1);  // clamped: in range, unused past the end
      __builtin_amdgcn_sched_barrier(0);
      compute(0);
      store2(1);
      __syncthreads();
      if (c + 1 >= c1) break;
      load2(c + 3 < c1 ? c + 3 : c1 - 1);
      __builtin_amdgcn_sched_barrier(0);
      compute(1);
      store(0);
      __syncthreads();
    }
  }
  const int64_t PT = a.PT > 0 ? a.PT : a.P;
  const int col = nbase + wn + l32;
  if (col < a.N) {
    // The lane's rows 8i + e (e < 4) share one member (Mp is a multiple of
    // 16, GM of 16).  The (member, sample) split of row 8i follows from that
    // of row 8(i-1): 8 < Mp, so the sample wraps into the next member at
    // most once, and the member's (step, learner) advances the same way.
    int row0 = mbase + wm + 4 * lhi;
    int v = qdiv_small(row0, a.Mp, inv_mp), sm = row0 - v * a.Mp;
    int vk = 0, vj = v;  // v = vk * vS + vj
    if (a.vS > 0) {
      vk = qdiv_small(v, a.vS, inv_vs);
      vj = v - vk * a.vS;
    }
    const int64_t gbase = a.vS > 0 ? (int64_t)g * a.vS : (int64_t)g * a.SG;
    const int64_t kstride = a.vS > 0 ? a.P : 0;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      if (i > 0) {
        row0 += 8;
        sm += 8;
        if (sm >= a.Mp) {
          sm -= a.Mp;
          if (a.vS > 0 && ++vj == a.vS) {
            vj = 0;
            ++vk;
          } else if (a.vS <= 0) {
            ++vj;
          }
        }
      }
      if (row0 >= GM) break;
      const int64_t p = vk * kstride + gbase + vj;
      float* dst = a.part + (((int64_t)ks * PT + p) * a.Mp + sm) * a.N + col;
#pragma unroll
      for (int e = 0; e < 4; ++e) dst[(int64_t)e * a.N] = acc[4 * i + e];
    }
  }
}

// Large-tile form for full tiles and long splits: 256 x 256 output tile,
// 32-wide K chunks in two LDS buffers (147 KB: one workgroup per CU), the
// next chunk's loads in flight during the current chunk's MFMAs (a second
// register set for loads two chunks ahead does not fit beside the four
// accumulators).  No row is out of range, so no load feeds a select.  Wave w owns rows 64*(w/4) and
// columns 64*(w%4) as four 32x32x2 chains (2 x 2 blocks), so a chunk's 64
// MFMAs per wave share one barrier and every 16-byte operand read feeds
// eight MFMAs instead of four.  Same k permutation and output layout as
// k_fwd_blk.
constexpr int kBT2 = 256;
constexpr int kKC2 = 32;
constexpr int kL2 = kKC2 + 4;
__global__ __launch_bounds__(1024) void k_fwd_blk256(FwdArgs a, int ntiles, int mtiles) {
  __shared__ __attribute__((aligned(16))) float As[2][kBT2 * kL2];
  __shared__ __attribute__((aligned(16))) float Ws[2][kBT2 * kL2];
  const int bid = xcd_remap(blockIdx.x, gridDim.x);
  const int q1 = qdiv_small(bid, ntiles, qdiv_inv(ntiles)), nt = bid - q1 * ntiles;
  const int q2 = qdiv_small(q1, mtiles, qdiv_inv(mtiles)), mt = q1 - q2 * mtiles;
  const int g = qdiv_small(q2, a.KS, qdiv_inv(a.KS)), ks = q2 - g * a.KS;
  const int nch = a.K / kKC;
  const int c0 = 2 * (ks * a.cps);
  const int c1 = 2 * min(nch, ks * a.cps + a.cps);
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  const int l32 = lane & 31, lhi = lane >> 5;
  const int wm = (wave >> 2) * 64, wn = (wave & 3) * 64;
  const int mbase = mt * kBT2, nbase = nt * kBT2;

  // Thread t stages pieces t and t + 1024 of each 256 x 32 chunk: row q/8,
  // 16-byte column piece q%8.  Every row is in range (full tiles).
  const float* arow[2];
  const float* wrow[2];
  int off[2];
  const float* wp = a.W + (int64_t)(g / a.wdiv) * a.w_pitch;
  const float inv_mp = qdiv_inv(a.Mp), inv_vs = qdiv_inv(a.vS > 0 ? a.vS : 1);
#pragma unroll
  for (int i = 0; i < 2; ++i) {
    const int q = tid + 1024 * i;
    const int r = q >> 3, c4 = q & 7;
    off[i] = r * kL2 + 4 * c4;
    const int m = mbase + r;
    const int jj = qdiv_small(m, a.Mp, inv_mp), sm = m - jj * a.Mp;
    int64_t p = (int64_t)g * a.SG + jj;
    if (a.vS > 0) {
      const int k = qdiv_small(jj, a.vS, inv_vs);
      p = (int64_t)k * a.P + (int64_t)g * a.vS + (jj - k * a.vS);
    }
    arow[i] = a.A + (int64_t)a.idx[p * a.M + sm] * a.lda + 4 * c4;
    wrow[i] = wp + (int64_t)(nbase + r) * a.ldw + 4 * c4;
  }
  f32x4 av[2], wv[2];
  auto load = [&](int c) {
    const int64_t o = (int64_t)c * kKC2;
#pragma unroll
    for (int i = 0; i < 2; ++i) {
      av[i] = *(const f32x4*)(arow[i] + o);
      wv[i] = *(const f32x4*)(wrow[i] + o);
    }
  };
  auto store = [&](int buf) {
#pragma unroll
    for (int i = 0; i < 2; ++i) {
      *(f32x4*)&As[buf][off[i]] = av[i];
      *(f32x4*)&Ws[buf][off[i]] = wv[i];
    }
  };
  f32x16 acc[2][2];
#pragma unroll
  for (int x = 0; x < 2; ++x)
#pragma unroll
    for (int y = 0; y < 2; ++y)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[x][y][r] = 0.0f;
  auto compute = [&](int buf) {
#pragma unroll
    for (int q = 0; q < kKC2 / 8; ++q) {
      f32x4 xa[2], yb[2];
#pragma unroll
      for (int x = 0; x < 2; ++x) xa[x] = *(const f32x4*)&As[buf][(wm + 32 * x + l32) * kL2 + 8 * q + 4 * lhi];
#pragma unroll
      for (int y = 0; y < 2; ++y) yb[y] = *(const f32x4*)&Ws[buf][(wn + 32 * y + l32) * kL2 + 8 * q + 4 * lhi];
#pragma unroll
      for (int e = 0; e < 4; ++e)
#pragma unroll
        for (int x = 0; x < 2; ++x)
#pragma unroll
          for (int y = 0; y < 2; ++y)
            acc[x][y] = __builtin_amdgcn_mfma_f32_32x32x2f32(xa[x][e], yb[y][e], acc[x][y], 0, 0, 0);
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
  const int64_t gbase = a.vS > 0 ? (int64_t)g * a.vS : (int64_t)g * a.SG;
  const int64_t kstride = a.vS > 0 ? a.P : 0;
#pragma unroll
  for (int x = 0; x < 2; ++x) {
    // Rows 8i + e of block x share one member (as in k_fwd_blk).
    int row0 = mbase + wm + 32 * x + 4 * lhi;
    int v = qdiv_small(row0, a.Mp, inv_mp), sm = row0 - v * a.Mp;
    int vk = 0, vj = v;
    if (a.vS > 0) {
      vk = qdiv_small(v, a.vS, inv_vs);
      vj = v - vk * a.vS;
    }
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      if (i > 0) {
        row0 += 8;
        sm += 8;
        if (sm >= a.Mp) {
          sm -= a.Mp;
          if (a.vS > 0 && ++vj == a.vS) {
            vj = 0;
            ++vk;
          } else if (a.vS <= 0) {
            ++vj;
          }
        }
      }
      const int64_t p = vk * kstride + gbase + vj;
      float* dst = a.part + (((int64_t)ks * PT + p) * a.Mp + sm) * a.N + nbase + wn + l32;
#pragma unroll
      for (int y = 0; y < 2; ++y)
#pragma unroll
        for (int e = 0; e < 4; ++e) dst[(int64_t)e * a.N + 32 * y] = acc[x][y][4 * i + e];
    }
  }
}

// Whether a block forward over `groups` row groups of `rows` rows takes the
// 256 x 256 tile: every tile full, and with the split count that brings the
// grid to about HAV_FWD_BLOCK_TARGET workgroups each split still at least 64
// 32-wide chunks long (the pipeline start is then a small share).  The split
// planner and the launcher both decide by this, so a launch runs the tile its
// split count was planned for (a split count planned for 128 x 128 tiles
// fills a quarter as many 256 x 256 workgroups).
static bool blk256_planned(int64_t groups, int rows, int N, int K) {
  if (rows % kBT2 != 0 || N % kBT2 != 0) return false;
  const int nch = K / kKC;
  const int64_t t2 = groups * (rows / kBT2) * (N / kBT2);
  const int64_t ks2 = std::min<int64_t>(nch, std::max<int64_t>(1, (HAV_FWD_BLOCK_TARGET + t2 - 1) / t2));
  return 2 * ((nch + ks2 - 1) / ks2) >= 64;
}

void launch_fwd_blk(hipStream_t s, const FwdArgs& a) {
  const int GM = a.SG * a.Mp;
  const int mtiles = (GM + kBT - 1) / kBT;
  const int ntiles = (a.N + kBT - 1) / kBT;
  const int groups = a.vS > 0 ? a.P / a.vS : a.P / a.SG;
  const unsigned grid = (unsigned)((int64_t)groups * a.KS * mtiles * ntiles);
  if (a.M == a.Mp && a.Mp % 8 == 0 && blk256_planned(groups, GM, a.N, a.K)) {
    const int mt2 = GM / kBT2, nt2 = a.N / kBT2;
    launch(k_fwd_blk256, (unsigned)((int64_t)groups * a.KS * mt2 * nt2), 1024, 0, s, a, nt2, mt2);
    return;
  }
  launch(k_fwd_blk, grid, 1024, 0, s, a, ntiles, mtiles);
}

// Split count of k_fwd_blk: about HAV_FWD_BLOCK_TARGET workgroups of the
// tile blk256_planned picks, no empty split.
void plan_split_blk(int groups, int rows, int N, int K, int* KS, int* cps) {
  const int64_t tiles = blk256_planned(groups, rows, N, K)
                            ? (int64_t)groups * (rows / kBT2) * (N / kBT2)
                            : (int64_t)groups * ((rows + kBT - 1) / kBT) * ((N + kBT - 1) / kBT);
  const int nch = K / kKC;
  int ks = (int)std::max<int64_t>(1, (HAV_FWD_BLOCK_TARGET + tiles - 1) / tiles);
  ks = std::min(ks, nch);
  const int c = (nch + ks - 1) / ks;
  *KS = (nch + c - 1) / c;
  *cps = c;
}

// ------------------------------------------------------------ delayed update
// Tile of the block update: 64 rows (hidden units m) x kUN columns (inputs n)
// of one group's W1, contracted over the K1*SG*B rows r = (step k, learner
// g*SG + j, sample s) of the group in stages of 32 rows through two LDS
// buffers (one barrier per stage; each stage's loads are issued two stages
// ahead).  Wave w owns the 32 x 32 block (rows 32*(w/4), columns 32*(w%4))
// as one chain of 32x32x2 MFMAs.
//
// The stage tiles sit in LDS transposed, contraction index innermost
// (At[m][r], Bt[n][r], 32 floats per row with no padding): lane (l, h) then
// reads four consecutive r of its row with one 16-byte read and feeds them
// to four MFMAs (MFMA (q, e) of a stage contracts r = 4q + e for lanes with
// h = 0 and 16 + 4q + e for h = 1, a permutation of the stage's rows that
// both operands share).  The 16-byte chunk c of row x is stored at chunk
// c ^ ((x >> 1) & 7), so the 16 rows a quarter-wave reads or writes fall
// into 16 distinct bank groups.  Wave w loads the stage's rows 4w .. 4w+3
// (lane l: error column m = l, input columns n = l and l + 64) with 4-byte
// loads, so each lane holds four consecutive r of one column: the
// transposed 16-byte chunk it writes.
//
// No vector arithmetic runs per stage (a SIMD's matrix core idles while it
// executes vector ALU instructions): the error-row and input-row offsets of
// every contraction row come from tables (64-float units) that the index
// draw writes, read with scalar loads, so each row's address is a scalar
// base plus the lane's fixed column.  Rows past the contraction point at row
// 0 and have their error rows zeroed; columns past the block read valid
// columns and feed discarded outputs.
constexpr int kBU = 32;  // LDS row length of the transposed stage tiles (= kSC)
__device__ inline int bu_swz(int x, int c) { return (x << 5) + ((c ^ ((x >> 1) & 7)) << 2); }

template <int NTH>
__global__ __launch_bounds__(NTH) __attribute__((amdgpu_waves_per_eu(6))) void k_block_update(
    BlkArgs a, const uint32_t* __restrict__ gtab, const uint32_t* __restrict__ xtab, int mtiles, int ntiles) {
  static_assert(NTH == 512 && kUN == 128 && kUM == 64 && kSC == 32, "block update tiling");
  constexpr int kStage = (kUM + kUN) * kBU;  // floats per LDS stage: At then Bt
  constexpr int kLds = 2 * kStage > kUM * kLB ? 2 * kStage : kUM * kLB;
  __shared__ __attribute__((aligned(16))) float lds[kLds];
  float* Gt = lds;  // [kUM][kLB] gradient tile (after the stages)
  // Tiles that share minibatch rows (same group and columns) are neighbours.
  const int bid = xcd_remap(blockIdx.x, gridDim.x);
  const int mt = bid % mtiles;
  const int nt = (bid / mtiles) % ntiles;
  const int g = bid / (ntiles * mtiles);
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);  // uniform: scalar row arithmetic
  const int l32 = lane & 31, lhi = lane >> 5;
  const int mrow0 = mt * kUM, ncol0 = nt * kUN;
  const int wn = (wave & 3) * 32, wm = (wave >> 2) * 32;
  const bool wave_on = ncol0 + wn < a.Ncols;
  const int R = a.K1 * a.SG * a.B;  // contraction rows
  const int nst = (R + kSC - 1) / kSC;
  const uint32_t* gt = gtab + (int64_t)g * nst * kSC;
  const uint32_t* xt = xtab + (int64_t)g * nst * kSC;
  if (a.tail && mt == 0) {
    // This group's cluster mean of the parameters after the first block: the
    // workgroups of row tile 0 take one run of columns each (rows in order).
    f32x4* T = (f32x4*)a.tail + (int64_t)g * a.SG * (a.tail_pitch / 4);
    const int64_t p4 = a.tail_pitch / 4, n4 = a.tail_len / 4, per = (n4 + ntiles - 1) / ntiles;
    const int64_t i1 = min(n4, (nt + 1) * per);
    for (int64_t i = nt * per + tid; i < i1; i += NTH) {
      f32x4 sum = T[i];
      for (int j = 1; j < a.SG; ++j) sum += T[j * p4 + i];
      const f32x4 mean = sum / (float)a.SG;
      for (int j = 0; j < a.SG; ++j) T[j * p4 + i] = mean;
    }
  }
  // This lane's columns as byte offsets within a row.  Each row is read
  // through a buffer resource whose range ends at the row's last valid
  // column, so columns past the block read 0 (their outputs are discarded).
  const int gcol = 4 * (mrow0 + lane), xcol0 = 4 * (ncol0 + lane), xcol1 = xcol0 + 256;
  const int grow_bytes = 4 * a.Mrows, xrow_bytes = 4 * a.Ncols;
  constexpr int kRsrcWord3 = 0x00020000;  // raw 32-bit buffer access (gfx9 family)

  struct StageRegs {
    float gv[4], x0[4], x1[4];
  };
  StageRegs RA, RB;
  auto load_stage = [&](int st, StageRegs& q) {
    const int r0 = (st < nst ? st : nst - 1) * kSC + 4 * wave;  // past the end: the last stage again
    const uint4 go = *(const uint4*)(gt + r0);
    const uint4 xo = *(const uint4*)(xt + r0);
    const uint32_t gr[4] = {go.x, go.y, go.z, go.w}, xr[4] = {xo.x, xo.y, xo.z, xo.w};
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const __amdgpu_buffer_rsrc_t grs = __builtin_amdgcn_make_buffer_rsrc(
          const_cast<float*>(a.G) + ((uint64_t)gr[i] << 6), 0, grow_bytes, kRsrcWord3);
      const __amdgpu_buffer_rsrc_t xrs = __builtin_amdgcn_make_buffer_rsrc(
          const_cast<float*>(a.X) + ((uint64_t)xr[i] << 6), 0, xrow_bytes, kRsrcWord3);
      q.gv[i] = __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(grs, gcol, 0, 0));
      q.x0[i] = __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(xrs, xcol0, 0, 0));
      q.x1[i] = __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(xrs, xcol1, 0, 0));
    }
  };
  auto store_stage = [&](int st, int buf, StageRegs& q) {
    float* S = lds + buf * kStage;
    const int r0 = st * kSC + 4 * wave;
    if (r0 + 4 > R) {  // rows past the contraction: zero error rows
#pragma unroll
      for (int i = 0; i < 4; ++i)
        if (r0 + i >= R) q.gv[i] = 0.0f;
    }
    *(f32x4*)&S[bu_swz(lane, wave)] = f32x4{q.gv[0], q.gv[1], q.gv[2], q.gv[3]};
    float* Bt = S + kUM * kBU;
    *(f32x4*)&Bt[bu_swz(lane, wave)] = f32x4{q.x0[0], q.x0[1], q.x0[2], q.x0[3]};
    *(f32x4*)&Bt[bu_swz(lane + 64, wave)] = f32x4{q.x1[0], q.x1[1], q.x1[2], q.x1[3]};
  };

  f32x16 acc;
#pragma unroll
  for (int r = 0; r < 16; ++r) acc[r] = 0.0f;
  // Operand rows of this lane and their swizzled chunk bases.
  const int arow = wm + l32, brow = wn + l32;
  const int aoff = arow << 5, boff = (kUM + brow) << 5;
  const int asw = (4 * lhi) ^ ((arow >> 1) & 7), bsw = (4 * lhi) ^ ((brow >> 1) & 7);
  auto mfma_stage = [&](int buf) {
    if (!wave_on) return;
    const float* S = lds + buf * kStage;
    __builtin_amdgcn_s_setprio(1);
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const f32x4 x = *(const f32x4*)&S[aoff + ((asw ^ q) << 2)];
      const f32x4 y = *(const f32x4*)&S[boff + ((bsw ^ q) << 2)];
#pragma unroll
      for (int e = 0; e < 4; ++e) acc = __builtin_amdgcn_mfma_f32_32x32x2f32(x[e], y[e], acc, 0, 0, 0);
    }
    __builtin_amdgcn_s_setprio(0);
  };

  load_stage(0, RA);
  load_stage(1, RB);
  store_stage(0, 0, RA);
  __syncthreads();
  // Iteration st: loads of stage st+2 go out, the MFMAs of stage st (buffer
  // 0) run, stage st+1 goes to buffer 1; then the same one stage later with
  // the buffers and register sets swapped.  A single loop exit and the odd
  // last stage after the loop keep the load waits where the data is used.
  int st = 0;
  for (; st + 1 < nst; st += 2) {
    load_stage(st + 2, RA);
    __builtin_amdgcn_sched_barrier(0);
    mfma_stage(0);
    store_stage(st + 1, 1, RB);
    __syncthreads();
    load_stage(st + 3, RB);
    __builtin_amdgcn_sched_barrier(0);
    mfma_stage(1);
    store_stage(st + 2, 0, RA);
    __syncthreads();
  }
  if (st < nst) {  // an odd stage count: the last stage is in buffer 0
    mfma_stage(0);
    __syncthreads();
  }

  // Base tile (16-byte pieces, thread t: column piece t%32 of rows t/32 +
  // 16*i), loaded only now so that its registers are free during the
  // contraction (three workgroups per CU); its latency overlaps the
  // accumulator transfer to LDS.
  constexpr int kXP = kUN / 4, kXR = NTH / kXP, kWL = kUM / kXR;
  const int xc4 = tid % kXP, xr0 = tid / kXP;
  const bool xcol_ok = ncol0 + 4 * xc4 < a.Ncols;
  const int xcol = xcol_ok ? ncol0 + 4 * xc4 : 0;
  const float* Wb = a.Wb + (int64_t)(g / a.base_div) * a.nbase * a.wb_pitch;
  f32x4 wv[kWL];
#pragma unroll
  for (int i = 0; i < kWL; ++i) {
    const int row = mrow0 + xr0 + kXR * i;
    wv[i] = *(const f32x4*)(Wb + (row < a.Mrows && xcol_ok ? (int64_t)row * a.ldw + xcol : 0));
  }
  if (a.nbase > 1) {  // the mean of the bases, added in order
    for (int c = 1; c < a.nbase; ++c) {
      f32x4 v[kWL];
#pragma unroll
      for (int i = 0; i < kWL; ++i) {
        const int row = mrow0 + xr0 + kXR * i;
        v[i] = *(const f32x4*)(Wb + (int64_t)c * a.wb_pitch +
                               (row < a.Mrows && xcol_ok ? (int64_t)row * a.ldw + xcol : 0));
      }
#pragma unroll
      for (int i = 0; i < kWL; ++i) wv[i] += v[i];
    }
#pragma unroll
    for (int i = 0; i < kWL; ++i) wv[i] = wv[i] / (float)a.nbase;
  }
#pragma unroll
  for (int r = 0; r < 16; ++r) {
    const int row = wm + 8 * (r >> 2) + 4 * lhi + (r & 3);
    Gt[row * kLB + wn + l32] = acc[r];
  }
  __syncthreads();
  float* Wo = a.Wo + (int64_t)g * a.wo_pitch;
  if (a.hb) {
    // Heavy-ball block end: hb[c1] * base + hb[c2] * (mean of the group's
    // rows of B2) + sum / lr_div, the errors already scaled per step.
    const float c1 = a.hb[a.hb_c1], c2 = a.hb[a.hb_c2], c3 = 1.0f / a.lr_div;
    f32x4 bm[kWL];
#pragma unroll
    for (int i = 0; i < kWL; ++i) bm[i] = f32x4{0.f, 0.f, 0.f, 0.f};
    if (a.B2) {
      const float* b2 = a.B2 + (int64_t)g * a.b2_rows * a.b2_pitch;
      for (int j = 0; j < a.b2_rows; ++j) {
#pragma unroll
        for (int i = 0; i < kWL; ++i) {
          const int row = mrow0 + xr0 + kXR * i;
          bm[i] += *(const f32x4*)(b2 + (int64_t)j * a.b2_pitch +
                                   (row < a.Mrows && xcol_ok ? (int64_t)row * a.ldw + xcol : 0));
        }
      }
#pragma unroll
      for (int i = 0; i < kWL; ++i) bm[i] = bm[i] / (float)a.b2_rows;
    }
#pragma unroll
    for (int i = 0; i < kWL; ++i) {
      const int rl = xr0 + kXR * i, row = mrow0 + rl;
      if (xcol_ok && row < a.Mrows) {
        const f32x4 gsum = *(const f32x4*)&Gt[rl * kLB + 4 * xc4];
        *(f32x4*)(Wo + (int64_t)row * a.ldw + xcol) = c1 * wv[i] + c2 * bm[i] + c3 * gsum;
      }
    }
    return;
  }
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

// Two-chain form of the block update for full tiles and large grids (plain
// SGD): 128 x 128 tile of W1 per workgroup, 8 waves, wave w owns rows
// 32*(w%4) and columns 64*(w/4) as two 32x32x2 chains, so a 32-row stage's
// 32 MFMAs per wave share one barrier (16 in k_block_update) and each
// error-operand read feeds eight MFMAs; two workgroups per CU.  Stage loads
// (wave w: rows 4w .. 4w+3 of the stage, every column of both operands),
// row tables, transposed swizzled LDS tiles and the k order are those of
// k_block_update.
constexpr int kUM3 = 128, kUN3 = 128, kLB3 = kUN3 + 4;
__global__ __launch_bounds__(512) void k_block_update2(BlkArgs a, const uint32_t* __restrict__ gtab,
                                                        const uint32_t* __restrict__ xtab, int mtiles, int ntiles) {
  constexpr int NTH = 512;
  constexpr int kStage = (kUM3 + kUN3) * kBU;
  constexpr int kLds = 2 * kStage > kUM3 * kLB3 ? 2 * kStage : kUM3 * kLB3;
  __shared__ __attribute__((aligned(16))) float lds[kLds];
  float* Gt = lds;
  const int bid = xcd_remap(blockIdx.x, gridDim.x);
  const int mt = bid % mtiles;
  const int nt = (bid / mtiles) % ntiles;
  const int g = bid / (ntiles * mtiles);
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int l32 = lane & 31, lhi = lane >> 5;
  const int mrow0 = mt * kUM3, ncol0 = nt * kUN3;
  const int wm = (wave & 3) * 32, wn = (wave >> 2) * 64;
  const int R = a.K1 * a.SG * a.B;
  const int nst = (R + kSC - 1) / kSC;
  const uint32_t* gt = gtab + (int64_t)g * nst * kSC;
  const uint32_t* xt = xtab + (int64_t)g * nst * kSC;
  if (a.tail && mt == 0) {
    f32x4* T = (f32x4*)a.tail + (int64_t)g * a.SG * (a.tail_pitch / 4);
    const int64_t p4 = a.tail_pitch / 4, n4 = a.tail_len / 4, per = (n4 + ntiles - 1) / ntiles;
    const int64_t i1 = min(n4, (nt + 1) * per);
    for (int64_t i = nt * per + tid; i < i1; i += NTH) {
      f32x4 sum = T[i];
      for (int j = 1; j < a.SG; ++j) sum += T[j * p4 + i];
      const f32x4 mean = sum / (float)a.SG;
      for (int j = 0; j < a.SG; ++j) T[j * p4 + i] = mean;
    }
  }
  const int gcol0 = 4 * (mrow0 + lane), gcol1 = gcol0 + 256, xcol0 = 4 * (ncol0 + lane), xcol1 = xcol0 + 256;
  const int grow_bytes = 4 * a.Mrows, xrow_bytes = 4 * a.Ncols;
  constexpr int kRsrcWord3 = 0x00020000;

  struct StageRegs {
    float g0[4], g1[4], x0[4], x1[4];
  };
  StageRegs RA, RB;
  auto load_stage = [&](int st, StageRegs& q) {
    const int r0 = (st < nst ? st : nst - 1) * kSC + 4 * wave;
    const uint4 go = *(const uint4*)(gt + r0);
    const uint4 xo = *(const uint4*)(xt + r0);
    const uint32_t gr[4] = {go.x, go.y, go.z, go.w}, xr[4] = {xo.x, xo.y, xo.z, xo.w};
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const __amdgpu_buffer_rsrc_t grs = __builtin_amdgcn_make_buffer_rsrc(
          const_cast<float*>(a.G) + ((uint64_t)gr[i] << 6), 0, grow_bytes, kRsrcWord3);
      const __amdgpu_buffer_rsrc_t xrs = __builtin_amdgcn_make_buffer_rsrc(
          const_cast<float*>(a.X) + ((uint64_t)xr[i] << 6), 0, xrow_bytes, kRsrcWord3);
      q.g0[i] = __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(grs, gcol0, 0, 0));
      q.g1[i] = __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(grs, gcol1, 0, 0));
      q.x0[i] = __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(xrs, xcol0, 0, 0));
      q.x1[i] = __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(xrs, xcol1, 0, 0));
    }
  };
  auto store_stage = [&](int st, int buf, StageRegs& q) {
    float* S = lds + buf * kStage;
    const int r0 = st * kSC + 4 * wave;
    if (r0 + 4 > R) {
#pragma unroll
      for (int i = 0; i < 4; ++i)
        if (r0 + i >= R) q.g0[i] = q.g1[i] = 0.0f;
    }
    *(f32x4*)&S[bu_swz(lane, wave)] = f32x4{q.g0[0], q.g0[1], q.g0[2], q.g0[3]};
    *(f32x4*)&S[bu_swz(lane + 64, wave)] = f32x4{q.g1[0], q.g1[1], q.g1[2], q.g1[3]};
    float* Bt = S + kUM3 * kBU;
    *(f32x4*)&Bt[bu_swz(lane, wave)] = f32x4{q.x0[0], q.x0[1], q.x0[2], q.x0[3]};
    *(f32x4*)&Bt[bu_swz(lane + 64, wave)] = f32x4{q.x1[0], q.x1[1], q.x1[2], q.x1[3]};
  };

  f32x16 acc[2];
#pragma unroll
  for (int y = 0; y < 2; ++y)
#pragma unroll
    for (int r = 0; r < 16; ++r) acc[y][r] = 0.0f;
  const int arow = wm + l32;
  const int aoff = arow << 5, asw = (4 * lhi) ^ ((arow >> 1) & 7);
  int boff[2], bsw[2];
#pragma unroll
  for (int y = 0; y < 2; ++y) {
    const int brow = wn + 32 * y + l32;
    boff[y] = (kUM3 + brow) << 5;
    bsw[y] = (4 * lhi) ^ ((brow >> 1) & 7);
  }
  auto mfma_stage = [&](int buf) {
    const float* S = lds + buf * kStage;
    __builtin_amdgcn_s_setprio(1);
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const f32x4 x = *(const f32x4*)&S[aoff + ((asw ^ q) << 2)];
      const f32x4 y0 = *(const f32x4*)&S[boff[0] + ((bsw[0] ^ q) << 2)];
      const f32x4 y1 = *(const f32x4*)&S[boff[1] + ((bsw[1] ^ q) << 2)];
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        acc[0] = __builtin_amdgcn_mfma_f32_32x32x2f32(x[e], y0[e], acc[0], 0, 0, 0);
        acc[1] = __builtin_amdgcn_mfma_f32_32x32x2f32(x[e], y1[e], acc[1], 0, 0, 0);
      }
    }
    __builtin_amdgcn_s_setprio(0);
  };

  load_stage(0, RA);
  load_stage(1, RB);
  store_stage(0, 0, RA);
  __syncthreads();
  int st = 0;
  for (; st + 1 < nst; st += 2) {
    load_stage(st + 2, RA);
    __builtin_amdgcn_sched_barrier(0);
    mfma_stage(0);
    store_stage(st + 1, 1, RB);
    __syncthreads();
    load_stage(st + 3, RB);
    __builtin_amdgcn_sched_barrier(0);
    mfma_stage(1);
    store_stage(st + 2, 0, RA);
    __syncthreads();
  }
  if (st < nst) {
    mfma_stage(0);
    __syncthreads();
  }
  // The gradient tile to LDS first (its registers are then free for the
  // base tile and the mean of the bases).
#pragma unroll
  for (int y = 0; y < 2; ++y)
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      const int row = wm + 8 * (r >> 2) + 4 * lhi + (r & 3);
      Gt[row * kLB3 + wn + 32 * y + l32] = acc[y][r];
    }
  // Base tile: thread t takes column piece t%32 of rows t/32 + 16*i.
  constexpr int kXP = kUN3 / 4, kXR = NTH / kXP, kWL = kUM3 / kXR;
  const int xc4 = tid % kXP, xr0 = tid / kXP;
  const int xcol = ncol0 + 4 * xc4;
  const float* Wb = a.Wb + (int64_t)(g / a.base_div) * a.nbase * a.wb_pitch;
  f32x4 wv[kWL];
#pragma unroll
  for (int i = 0; i < kWL; ++i) wv[i] = *(const f32x4*)(Wb + (int64_t)(mrow0 + xr0 + kXR * i) * a.ldw + xcol);
  if (a.nbase > 1) {  // the mean of the bases, added in order
    for (int c = 1; c < a.nbase; ++c) {
      f32x4 v[kWL];
#pragma unroll
      for (int i = 0; i < kWL; ++i)
        v[i] = *(const f32x4*)(Wb + (int64_t)c * a.wb_pitch + (int64_t)(mrow0 + xr0 + kXR * i) * a.ldw + xcol);
#pragma unroll
      for (int i = 0; i < kWL; ++i) wv[i] += v[i];
    }
#pragma unroll
    for (int i = 0; i < kWL; ++i) wv[i] = wv[i] / (float)a.nbase;
  }
  __syncthreads();
  float* Wo = a.Wo + (int64_t)g * a.wo_pitch;
  const float lr_eff = *a.lr / a.lr_div;
#pragma unroll
  for (int i = 0; i < kWL; ++i) {
    const int rl = xr0 + kXR * i;
    const f32x4 gsum = *(const f32x4*)&Gt[rl * kLB3 + 4 * xc4];
    *(f32x4*)(Wo + (int64_t)(mrow0 + rl) * a.ldw + xcol) = wv[i] - lr_eff * gsum;
  }
}

#ifndef HAV_BLK_THREADS
#define HAV_BLK_THREADS 512
#endif
void launch_block_update(hipStream_t s, const BlkArgs& a) {
  {  // the two-chain tile where every tile is full and the grid has at least eight per CU
    const int groups = a.P / a.SG;
    if (!a.hb && a.Mrows % kUM3 == 0 && a.Ncols % kUN3 == 0 &&
        (int64_t)groups * (a.Mrows / kUM3) * (a.Ncols / kUN3) >= 2048) {
      const int mt2 = a.Mrows / kUM3, nt2 = a.Ncols / kUN3;
      launch(k_block_update2, (unsigned)((int64_t)groups * mt2 * nt2), 512, 0, s, a, a.gtab, a.xtab, mt2, nt2);
      return;
    }
  }
  const int mtiles = (a.Mrows + kUM - 1) / kUM;
  const int ntiles = (a.Ncols + kUN - 1) / kUN;
  const unsigned grid = (unsigned)((int64_t)(a.P / a.SG) * mtiles * ntiles);
  launch(k_block_update<HAV_BLK_THREADS>, grid, HAV_BLK_THREADS, 0, s, a, a.gtab, a.xtab, mtiles, ntiles);
}

// ------------------------------------------------------------ Gram blocks
// One workgroup per (learner p, block b, K split ks): all step pairs k2 < k of
// the block at once.  The K1*Bp minibatch rows of the block (gathered, this
// split's input features) are staged through LDS 64 features at a time, the
// next chunk's loads in flight during the current chunk's MFMAs; each wave
// owns a fixed set of the 16x16 output blocks of the lower block triangle
// (16x16x4 MFMAs, the k permutation of k_fwd_nt).  Every minibatch row is
// read once per split; the consumer adds the KSG partial sums.
constexpr int kGT = 512, kGW = kGT / 64;  // threads and waves per workgroup
constexpr int kGramMaxBlocks = 14;  // 16x16 output blocks per wave (K1 <= 8, Bp <= 32)
template <int NB, int ROWS>
__global__ __launch_bounds__(kGT) void k_gram(const float* __restrict__ X, int64_t ldx, int K,
                                              const int32_t* __restrict__ idx, float* __restrict__ gram, int P,
                                              int K1, int B, int Bp, int KSG) {
  constexpr int kRows = ROWS;         // LDS capacity in rows (K1 * Bp <= ROWS)
  constexpr int kL = kKC + 4;         // LDS row length
  constexpr int kLPT = kRows * (kKC / 4) / kGT;  // 16-byte pieces per thread per chunk (at most)
  __shared__ __attribute__((aligned(16))) float xs[kRows * kL];
  const int ks = blockIdx.x % KSG;
  const int pb = blockIdx.x / KSG;  // p + P * b
  const int p = pb % P, b = pb / P;
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);  // uniform: scalar block bookkeeping
  const int lrow = lane & 15, lgrp = lane >> 4;
  const int rows = K1 * Bp;
  const int nch = K / kKC;
  const int c0 = (int)((int64_t)nch * ks / KSG), c1 = (int)((int64_t)nch * (ks + 1) / KSG);
  // Bp is 16 or 32 (B <= 32): row and block indices split with shifts.
  const int lg_bp = Bp == 32 ? 5 : 4, lg_mbs = lg_bp - 4;
  // Row r = k*Bp + s of the block: sample s of step b*K1 + k (rows past B: zero).
  const float* src[kLPT];
  bool ok[kLPT];
  int off[kLPT];
#pragma unroll
  for (int i = 0; i < kLPT; ++i) {
    const int q = tid + kGT * i;
    const int r = q >> 4, c4 = q & 15;
    const int k = r >> lg_bp, sm = r & (Bp - 1);
    ok[i] = r < rows && sm < B;
    const int64_t e = ((int64_t)(b * K1 + (ok[i] ? k : 0)) * P + p) * B + (ok[i] ? sm : 0);
    src[i] = X + (int64_t)idx[e] * ldx + 4 * c4;
    off[i] = (r < kRows ? r : 0) * kL + 4 * c4;
  }
  // Output blocks of this wave: block e = wave + kGW*t over the lower triangle
  // (pair (k, k2), row block mb, column block nb); wave-uniform.
  const int mbs = 1 << lg_mbs;
  const int nblk = K1 * (K1 - 1) / 2 * mbs * mbs;
  int bk[NB], bk2[NB], bmb[NB], bnb[NB];
  int arow[NB], brow[NB];
  bool bon[NB];
#pragma unroll
  for (int t = 0; t < NB; ++t) {
    const int e = wave + kGW * t;
    bon[t] = e < nblk;
    const int ee = bon[t] ? e : 0;
    const int pr = ee >> (2 * lg_mbs), rem = ee & (mbs * mbs - 1);
    int k = 1, k2 = pr;
    while (k2 >= k) {
      k2 -= k;
      ++k;
    }
    bk[t] = k;
    bk2[t] = k2;
    bmb[t] = rem >> lg_mbs;
    bnb[t] = rem & (mbs - 1);
    arow[t] = (k * Bp + 16 * bmb[t] + lrow) * kL + 4 * lgrp;
    brow[t] = (k2 * Bp + 16 * bnb[t] + lrow) * kL + 4 * lgrp;
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
  // Piece i holds row (tid >> 4) + 32*i; with B == Bp every staged row is a
  // sample.
  const bool all_rows = B == Bp;
  auto store = [&]() {
    if (all_rows) {
#pragma unroll
      for (int i = 0; i < kLPT; ++i)
        if ((tid >> 4) + 32 * i < rows) *(f32x4*)&xs[off[i]] = v[i];
    } else {
#pragma unroll
      for (int i = 0; i < kLPT; ++i)
        if ((tid >> 4) + 32 * i < rows) *(f32x4*)&xs[off[i]] = ok[i] ? v[i] : zero4;
    }
  };
  if (c0 < c1) {
    load(c0);
    for (int c = c0; c < c1; ++c) {
      store();
      __syncthreads();
      load(c + 1 < c1 ? c + 1 : c);  // next chunk in flight (the last again at the end)
      __builtin_amdgcn_sched_barrier(0);
      // Blocks past nblk repeat block 0 (their sums are not stored): no
      // branch around the MFMAs, so the accumulators stay in place.
#pragma unroll
      for (int t = 0; t < NB; ++t) {
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
  const int K2n = gridDim.x / (KSG * P);
#pragma unroll
  for (int t = 0; t < NB; ++t) {
    if (!bon[t]) continue;
    float* out = gram + (((((int64_t)ks * K2n + b) * P + p) * K1 + bk[t]) * K1 + bk2[t]) * Bp * Bp +
                 (16 * bmb[t] + 4 * lgrp) * Bp + 16 * bnb[t] + lrow;
#pragma unroll
    for (int r = 0; r < 4; ++r) out[r * Bp] = acc[t][r];
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

#ifndef HAV_GRAM_TARGET
#define HAV_GRAM_TARGET 512
#endif
int gram_splits(int P, int K2, int K) {
  // about two workgroups per CU, at least two 64-wide chunks per split
  const int target = HAV_GRAM_TARGET;
  int ksg = (target + P * K2 - 1) / (P * K2);
  return std::max(1, std::min(ksg, K / kKC / 2));
}

void launch_gram(hipStream_t s, const float* X, int64_t ldx, int K, const int32_t* idx, float* gram, int P, int K1,
                 int K2, int B, int Bp, int KSG) {
  const int nblk = K1 * (K1 - 1) / 2 * (Bp / 16) * (Bp / 16);
  if (nblk == 0 || (Bp != 16 && Bp != 32)) return;  // the delayed schedule has B <= 32
  const unsigned grid = (unsigned)((int64_t)P * K2 * KSG);
  const int nb = (nblk + kGW - 1) / kGW;
#define HAV_GRAM(N_, R_) launch(k_gram<N_, R_>, grid, kGT, 0, s, X, ldx, K, idx, gram, P, K1, B, Bp, KSG)
  if (K1 * Bp <= 128) {
    if (nb <= 1)
      HAV_GRAM(1, 128);
    else if (nb <= 3)
      HAV_GRAM(3, 128);
    else
      HAV_GRAM(6, 128);
  } else {
    if (nb <= 6)
      HAV_GRAM(6, 256);
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
