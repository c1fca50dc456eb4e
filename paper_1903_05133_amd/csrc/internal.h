// Internal declarations of the Hier-AVG HIP library (gfx950).
//
// Replica layout in HBM.  Every learner j owns row j of one [P][Dp] float32
// array.  A row holds the model's parameter blocks at offsets that are
// multiples of 16 floats, each block stored with padded dimensions
// (INp = roundup(IN, 64), Hp = roundup(H, 64), Cp = roundup(C, 16)) so that the
// GEMM kernels need no ragged-edge handling along K.  Padding entries are
// zero when the handle is created and stay zero: a zero input column, a zero
// hidden unit (ReLU(0) has derivative 0) and a zero class (masked out of the
// softmax) all receive zero gradient, and means of zeros are zero.
#pragma once

#include <hip/hip_ext.h>
#include <hip/hip_runtime.h>

#include <cstdint>

#include "hieravg.h"

namespace hav {

typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef float f32x16 __attribute__((ext_vector_type(16)));

// ------------------------------------------------------------ SplitMix64
constexpr uint64_t kGolden = 0x9E3779B97F4A7C15ull;

__host__ __device__ inline uint64_t mix64(uint64_t z) {
  z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
  z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
  return z ^ (z >> 31);
}

// H(key, c): SplitMix64 output at counter c of the stream `key`.
__host__ __device__ inline uint64_t hash64(uint64_t key, uint64_t c) { return mix64(key + (c + 1) * kGolden); }

// Exact Irwin-Hall(12) normal surrogate: the twelve 16-bit fields of three
// hashes, summed, centred and scaled by 2^-16 (exactly representable).
__device__ inline float irwin_hall(uint64_t key, uint64_t e) {
  int64_t acc = 0;
#pragma unroll
  for (int r = 0; r < 3; ++r) {
    uint64_t v = hash64(key, e * 3 + r);
    acc += (int64_t)(v & 0xFFFF) + (int64_t)((v >> 16) & 0xFFFF) + (int64_t)((v >> 32) & 0xFFFF) +
           (int64_t)(v >> 48);
  }
  return (float)(acc - 393210) * (1.0f / 65536.0f);
}

// Stream tags (ASCII names, big-endian).
constexpr uint64_t kTagIndex = 0x68762e696e646578ull;  // "hv.index"
constexpr uint64_t kTagLabel = 0x68762e6c6162656cull;  // "hv.label"
constexpr uint64_t kTagMean = 0x68762e636d65616eull;   // "hv.cmean"
constexpr uint64_t kTagNoise = 0x68762e6e6f697365ull;  // "hv.noise"
constexpr uint64_t kTagInit = 0x68762e77696e6974ull;   // "hv.winit"
constexpr uint64_t kTagGrad = 0x68762e6772616473ull;   // "hv.grads"
constexpr uint64_t kTagTestLabel = 0x68762e746c61626cull;  // "hv.tlabl" (held-out rows)
constexpr uint64_t kTagTestNoise = 0x68762e746e6f6973ull;  // "hv.tnois"

inline int64_t round_up(int64_t x, int64_t m) { return (x + m - 1) / m * m; }

// n / d for 0 <= n < 2^22, d >= 1, from inv = qdiv_inv(d) (1/d to within an
// ulp, computed once by the caller): n * inv is within one of n / d, so the
// truncated quotient is off by at most one, and one correction step each way
// makes it exact.  A few vector instructions instead of the long sequence of
// an integer division.
__device__ inline float qdiv_inv(int d) { return __builtin_amdgcn_rcpf((float)d); }
__device__ inline int qdiv_small(int n, int d, float inv) {
  int q = (int)((float)n * inv);
  q += (q + 1) * d <= n ? 1 : 0;
  q -= q * d > n ? 1 : 0;
  return q;
}

// Workgroup index -> logical tile index such that consecutive logical tiles
// run on the same XCD (the hardware deals workgroups to the 8 XCDs round
// robin).  Tiles that share operands then share an L2.
// Buffer accesses: a resource of (base, size in bytes), a per-lane 32-bit
// byte offset and a wave-uniform one; reads past the size return zero.
// The base address and size pass through readfirstlane: the resource then
// sits in scalar registers (the caller's values are uniform), and no access
// turns into a per-lane loop over resource values.
__device__ inline __amdgpu_buffer_rsrc_t buf_rsrc(const void* base, uint64_t bytes) {
  const uint64_t b = (uint64_t)base;
  const uint32_t lo = __builtin_amdgcn_readfirstlane((uint32_t)b), hi = __builtin_amdgcn_readfirstlane((uint32_t)(b >> 32));
  const int n = __builtin_amdgcn_readfirstlane((int)(bytes < 0xffffffffull ? bytes : 0xffffffffull));
  return __builtin_amdgcn_make_buffer_rsrc((void*)(((uint64_t)hi << 32) | lo), (short)0, n, 0x00020000);
}
__device__ inline f32x4 buf_ld16(__amdgpu_buffer_rsrc_t r, uint32_t voff, int soff) {
  return __builtin_bit_cast(f32x4, __builtin_amdgcn_raw_buffer_load_b128(r, voff, soff, 0));
}
__device__ inline void buf_st16(__amdgpu_buffer_rsrc_t r, uint32_t voff, int soff, f32x4 v) {
  typedef unsigned u32x4 __attribute__((ext_vector_type(4)));
  __builtin_amdgcn_raw_buffer_store_b128(__builtin_bit_cast(u32x4, v), r, voff, soff, 0);
}

__device__ inline int xcd_remap(int bid, int nblocks) {
  constexpr int kXcd = 8;
  int q = nblocks / kXcd, r = nblocks % kXcd;
  int x = bid % kXcd, i = bid / kXcd;
  return x * q + (x < r ? x : r) + i;
}

// ------------------------------------------------------------ kernel classes
enum KernelClass {
  KC_DRAW = 0,       // minibatch index draw (once per round)
  KC_FWD1,           // layer-1 forward GEMM (split-K partials)
  KC_REDUCE1,        // large C: split-K reduction + bias of layer 1
  KC_FWD2,           // large C: layer-2 forward GEMM (split-K partials)
  KC_SOFTMAX,        // logits reduction, softmax cross-entropy gradient
  KC_BWD_HIDDEN,     // large C: hidden-layer error (G2 W2) masked by ReLU'
  KC_HEAD_A,         // small C: layer-1 reduction + bias, partial logits
  KC_HEAD_B,         // small C: softmax, hidden error, layer-2 and bias updates
  KC_UPDATE2,        // layer-2 weight gradient fused with the SGD update
  KC_UPDATE1,        // layer-1 weight gradient fused with the SGD update
  KC_GROUP_MEAN,     // local mean over each cluster of S replicas
  KC_GLOBAL_MEAN,    // global mean over all P replicas
  KC_MOMENTUM,       // averaging kind: momentum update (no mean)
  KC_MOMENTUM_GROUP, // averaging kind: momentum update fused with the local mean
  KC_MOMENTUM_GLOBAL,// averaging kind: momentum update fused with the global mean
  KC_STEP1,          // layer-1 update fused with the next step's layer-1 forward
  KC_STEP1_MEAN,     // same, with the local mean of layer 1 in between
  KC_TAIL_MEAN,      // local mean of the parameters after layer 1
  KC_GRAM,           // delayed updates: Gram blocks of the round's minibatches
  KC_FWD1_BLOCK,     // delayed updates: layer-1 forward of a block's steps from the cluster copies
  KC_BLOCK_UPDATE,   // delayed updates: block-end update of the cluster copies
  KC_W1_MEAN,        // delayed updates: global mean of the cluster copies
  KC_TAIL_GLOBAL,    // global mean of the parameters after layer 1
  KC_GRAM_REDUCE,    // delayed updates: sum of the Gram blocks' feature splits
  KC_HEAD_STEP,      // delayed updates: backward of step k-1 + forward and loss gradient of step k
  KC_HEAD_END,       // delayed updates: backward of a block's last step
  KC_Z1_DELAYED,     // delayed updates, more than 32 classes: pre-activations with the Gram correction
  KC_VMEAN_GROUP,    // averaged momentum buffers: cluster mean of v
  KC_VMEAN_GLOBAL,   // averaged momentum buffers: global mean of v
  KC_MOMENTUM_FIRST, // averaging kind: a round's first step, from the stored global mean
  KC_FWD1_BLOCK_V,   // heavy-ball delayed updates: X_k V^T of a block's steps from each learner's buffer
  KC_SCALE_ERRORS,   // heavy-ball delayed updates: the block's errors scaled for the block-end updates
  KC_BUF_UPDATE,     // heavy-ball delayed updates: block-end update of each learner's first-layer buffer
  KC_UPD1_MEAN,      // layer-1 update of every learner with the local mean, no forward
  KC_FWD1_GROUP,     // layer-1 forward of a step from each cluster's common first layer (one GEMM per cluster)
  KC_UPD1_GLOBAL,    // layer-1 update of every learner with the global mean (a round's last step)
  KC_HEAD_FUSED,     // small C, eager: the loss side of a step (G1, gradient rows of W2, b1, b2)
  KC_HEAD_W2,        // small C, eager: the step of W2, b1, b2 from those rows
  KC_COUNT
};

// Largest class count handled by the fused small-C head kernels.
constexpr int kSmallC = 32;

// ------------------------------------------------------------ heavy-ball blocks
// Heavy-ball SGD with L2 decay (d = g + wd*w; v <- mu*v + d; w <- w - lr*v)
// over the steps of a block is linear in the block-start (w, v) and the
// steps' gradients g_m: with A = [[1 - lr*wd, -lr*mu], [wd, mu]] acting on
// (w, v) and e = (-lr, 1), after n steps
//   w_n = p_n w + q_n v + sum_{m<n} u_{n-1-m} g_m,
//   v_n = r_n w + s_n v + sum_{m<n} t_{n-1-m} g_m,
// where A^n = [[p_n, q_n], [r_n, s_n]], u_n = (A^n e)_w, t_n = (A^n e)_v.
// The device table (after the step size in the handle's hyperparameters)
// holds p, q, r, s, u, t for n = 0..K1, kHbStride floats apart.
constexpr int kHbOff = 16, kHbStride = 16;
enum HbCoef { HB_P = 0, HB_Q, HB_R, HB_S, HB_U, HB_T, HB_COUNT };
__host__ __device__ inline int hb_index(int which, int n) { return kHbOff + which * kHbStride + n; }
constexpr int kHyperFloats = kHbOff + HB_COUNT * kHbStride;

// ------------------------------------------------------------ launching
// Events that time the next launch on this thread (both null: not timing).
// When set, the launch goes through hipExtLaunchKernelGGL, whose dispatch
// packet itself records the kernel's start and end in the two events.
struct LaunchTiming {
  hipEvent_t start = nullptr, stop = nullptr;
};
extern thread_local LaunchTiming g_launch_timing;

template <class K, class... Args>
inline void launch(K kernel, dim3 grid, dim3 block, uint32_t shmem, hipStream_t s, Args... args) {
  if (g_launch_timing.start)
    hipExtLaunchKernelGGL(kernel, grid, block, shmem, s, g_launch_timing.start, g_launch_timing.stop, 0u, args...);
  else
    kernel<<<grid, block, shmem, s>>>(args...);
}

// ------------------------------------------------------------ launchers
// Data and initial state (k_data.hip).
void launch_gen_labels(hipStream_t s, int32_t* y, int64_t N, uint64_t key, uint64_t C);
void launch_gen_data(hipStream_t s, float* X, const int32_t* y, int64_t N, int64_t IN, int64_t INp,
                     uint64_t key_mean, uint64_t key_noise, float sigma);
void launch_init_matrix(hipStream_t s, float* W, int64_t rows, int64_t cols, int64_t ld, uint64_t key,
                        uint64_t layer, float scale);
void launch_init_vector(hipStream_t s, float* w, int64_t D, uint64_t key, float std);
void launch_gen_grads(hipStream_t s, float* G, int64_t D, int64_t Dp, int P, int T, uint64_t key, float std);
// dst[i] = i, i < n (n >= 1).
void launch_iota(hipStream_t s, int32_t* dst, int n);
// Row tables of the block update (delayed updates): for block b, cluster g
// and contraction row r = (k*S + j)*B + s (step k of the block, learner
// g*S + j, sample s) at [(b*(P/S) + g)*Rp + r], the offsets in 64-float
// units of that row's hidden-error row (row (k*P + g*S + j)*Mp + s of pitch
// ldg) and of its sample's dataset row (pitch ldx).  Rows R..Rp-1 of each
// table (R = K1*S*B, Rp = R rounded up to 32) stay 0.
// With global_last, the last block (b = K2-1) instead holds one table over
// all P learners, row r = (k*P + j)*B + s at [(b*(P/S))*Rp + r], for the
// block update that takes the global mean in the same launch.
// gtab1 (optional): the same rows per learner, row r = k*B + s of learner j
// in block b at [(b*P + j)*Rp1 + r] (the heavy-ball buffer updates).
struct BlkTables {
  uint32_t* gtab = nullptr;
  uint32_t* xtab = nullptr;
  int K1 = 1, S = 1, Mp = 0, Rp = 0;
  int64_t ldg = 0, ldx = 0;
  int K2 = 0;
  bool global_last = false;
  uint32_t* gtab1 = nullptr;
  uint32_t* xtab1 = nullptr;
  int Rp1 = 0;
};
// ylab (optional): the label of every drawn sample, same layout as idx.
// tables.gtab (optional): also write the block update's row tables.
void launch_draw_indices(hipStream_t s, int32_t* idx, uint64_t* step_ctr, uint32_t* done_ctr, int P, int B,
                         int T, uint64_t N, uint64_t key, const int32_t* labels = nullptr, int32_t* ylab = nullptr,
                         const BlkTables& tables = BlkTables());

// GEMMs (k_gemm.hip).
struct FwdArgs {
  const float* A;       // gathered: dataset X [N][lda]; relu: Z [P][Mp][lda]
  const int32_t* idx;   // [P][M] sample indices (gathered A)
  int64_t lda;
  const float* W;       // weight block of copy 0 ([N][ldw]); copy c at W + c*w_pitch
  int64_t w_pitch, ldw;
  float* part;          // [KS][P][Mp][N] split-K partial sums
  int P, M, Mp, N, K;   // N multiple of 16, K multiple of 64
  int KS, cps;          // split count and 64-wide K chunks per split
  // Learners p = g*SG .. g*SG+SG-1 form row group g (SG*Mp rows of one GEMM)
  // and read weight copy g / wdiv (w_pitch 0: one copy for all).
  int SG = 1, wdiv = 1;
  int mb_max = 8;  // largest row tile, in 16-row blocks (1, 2, 4 or 8)
  // vS > 0: the SG members of group g are (step k, learner g*vS + j) for
  // v = k*vS + j, whose sample indices sit at idx + (k*P + g*vS + j)*M and
  // whose outputs go to part[ks][k][P][Mp][N] (PT = steps * P members per
  // split).  idx then points at the first step's indices.
  int vS = 0, PT = 0;
};
enum ASource { A_GATHER = 0, A_RELU = 1 };
void launch_fwd(hipStream_t s, const FwdArgs& a, ASource src);
// Split count for a forward over P row groups of Mp rows each.
void plan_split(int P, int Mp, int N, int K, int* KS, int* cps, int target_wg = 0, int mb_max = 8);
// Large-tile forward (128 x 128 tiles, 1024 threads) for many rows per weight
// copy, and its split count.
void launch_fwd_blk(hipStream_t s, const FwdArgs& a);
void plan_split_blk(int groups, int rows, int N, int K, int* KS, int* cps);
// Workgroup target of the block-wide forward from the cluster copies.
#ifndef HAV_FWD_BLOCK_TARGET
#define HAV_FWD_BLOCK_TARGET 256
#endif
int fwd_tiles(int P, int Mp, int N);

struct UpdArgs {
  const float* G;       // [P][Mp][ldg] error rows (row s = sample, column m = output unit)
  int64_t ldg;
  int Mp;               // rows per learner in G and in the relu source
  const float* Bsrc;    // gathered: dataset X [N][ldb]; relu: Z [P][Mp][ldb]
  const int32_t* idx;   // [P][Kb]
  int64_t ldb;
  float* W;             // weight block of replica 0 ([Mrows][ldw]); replica p at W + p*w_pitch
  int64_t w_pitch, ldw;
  float* bias;          // bias block of replica 0 (or nullptr); replica p at bias + p*w_pitch
  int P, Kb, Mrows, Ncols;
  const float* lr;      // device scalar: the step size (read at kernel start)
  // Heavy-ball step with L2 decay (d = g + wd*w; v <- mu*v + d; w <- w - lr*v):
  // V, vbias are the buffers laid out like W, bias (nullptr: v = d, no state).
  float* V = nullptr;
  float* vbias = nullptr;
  float mu = 0.0f, wd = 0.0f;
};
void launch_update(hipStream_t s, const UpdArgs& a, ASource bsrc);

// Delayed first-layer update at the end of a block of K1 steps (the local
// averaging of Algorithm 1 applied to the first weight block): for each group
// g of SG learners,
//   Wo_g = Wb_g - lr_eff * sum_{k<K1, j in g, s<B} G[k][j][s][:]^T X[idx[k][j][s]][:]
// with lr_eff = lr / SG (the mean of the SG learners' K1 updates).
struct BlkArgs {
  const float* G;       // [K1][P][Mp][ldg] hidden errors of the block's steps
  int64_t ldg;
  const float* X;       // dataset [N][ldx]
  const int32_t* idx;   // [K1][P][B] indices of the block's steps
  int64_t ldx;
  const float* Wb;      // base of group g at Wb + g*wb_pitch (0: one base for all)
  int64_t wb_pitch;
  float* Wo;            // result of group g at Wo + g*wo_pitch (may equal the base)
  int64_t wo_pitch, ldw;
  int P, SG, K1, B, Mp, Mrows, Ncols;
  const float* lr;      // device scalar step size; the mean takes lr / lr_div
  float lr_div;
  const uint32_t* gtab;  // this block's row tables (BlkTables): [P/SG][Rp] each
  const uint32_t* xtab;
  // Optional (tail set): also replace the columns [0, tail_len) of each
  // group's SG replica rows (replica 0's at tail, tail_pitch floats apart) by
  // the group's mean: the cluster mean of the parameters after the first
  // block, which no other part of the launch touches.
  float* tail = nullptr;
  int64_t tail_pitch = 0, tail_len = 0;
  // The base of a group is the mean of nbase blocks wb_pitch apart (added in
  // order): the global update of the last block starts from the mean of the
  // cluster copies.  Group g reads base g / base_div (its cluster's copy for
  // a per-learner update).
  int nbase = 1, base_div = 1;
  // Heavy-ball block end (hb set, the coefficient table): the result is
  //   hb[c1] * base + hb[c2] * (mean of the group's b2_rows rows of B2)
  //   + sum / lr_div
  // with the contraction's error rows already scaled by their step's
  // coefficient (G = the scaled errors); group g's rows of B2 are
  // g*b2_rows .. +b2_rows-1, b2_pitch floats apart.
  const float* hb = nullptr;
  int hb_c1 = 0, hb_c2 = 0;
  const float* B2 = nullptr;
  int64_t b2_pitch = 0;
  int b2_rows = 0;
};
// Largest contraction (K1 * SG * B rows) of a block update.
constexpr int kBlkMaxRows = 16384;
void launch_block_update(hipStream_t s, const BlkArgs& a);

// Gram blocks of each learner's minibatches within each block of a round, as
// KSG partial sums over splits of the input features:
// sum_ks gram[ks][b][p][k][k2][s][s2] = X[idx_(b,k,p,s)] . X[idx_(b,k2,p,s2)]
// for k2 < k (rows and columns past B are zero), shape
// [KSG][K2][P][K1][K1][Bp][Bp]; launch_gram_reduce then adds the partial sums
// into split 0.  K1 * Bp <= 256.
int gram_splits(int P, int K2, int K);
void launch_gram(hipStream_t s, const float* X, int64_t ldx, int K, const int32_t* idx, float* gram, int P,
                 int K1, int K2, int B, int Bp, int KSG);
void launch_gram_reduce(hipStream_t s, float* gram, int P, int K1, int K2, int Bp, int KSG);

// Fused step of the first weight block: the update of step t (Bsrc = the
// dataset gathered through u.idx), optionally the mean over each group of SG
// learners, and optionally the forward of step t+1 on the new weights.
struct StepArgs {
  UpdArgs u;                // u.Bsrc is the dataset, gathered through u.idx
  const int32_t* idx_next;  // [P][Kb] sample indices of the next step
  float* part;              // [KS][P][Mp][Mrows] forward partials of the next step
  int SG;                   // learners averaged per group (1: no mean); SG | P
  int NT;                   // set by the launcher: 128-column tiles per workgroup
  int64_t x_rows = 0;       // rows of the dataset u.Bsrc (0: unknown)
  bool no_fwd = false;      // SG > 1: the update and the group mean only (no partials)
  // Full tiles only (step_full_shape): learner p reads its old block from
  // w_src + (p / src_group) * src_pitch (a mean written once) instead of its
  // own row; the update with the group mean writes group g's mean once, to
  // w_dst + g * dst_pitch, instead of to every learner's row.  Both blocks
  // are [Mrows][ldw] like W.
  const float* w_src = nullptr;
  int64_t src_pitch = 0;
  int src_group = 1;
  float* w_dst = nullptr;
  int64_t dst_pitch = 0;
};
// Whether the full-tile step kernels take a launch of this shape (the only
// ones that read w_src or write w_dst).
bool step_full_shape(int Kb, int Mp, int Mrows, int Ncols, int64_t x_rows, int64_t ldb, int64_t ldg, int64_t ldw);
// Whether the fused kernel handles this shape (Mp a multiple of 16 up to 64,
// SG in {1, 2, 4, 8}, SG * Mp / 16 <= 16).
bool step_w1_supported(int Mp, int SG);
// Whether the update-and-group-mean form without the forward (no_fwd) takes
// this shape: Mp a multiple of 16 up to 64, SG a power of two in [2, 64].
bool step_w1_mean_supported(int Mp, int SG);
// Number of forward splits KS the fused kernel writes for this shape.
int step_w1_splits(int P, int SG, int Mp, int Mrows, int Ncols);
// False (nothing launched) for a w_src / w_dst launch the full-tile kernels do not take.
bool launch_step_w1(hipStream_t s, StepArgs a);

// Head of the network (k_head.hip).
void launch_reduce_bias(hipStream_t s, const float* part, int KS, const float* bias, int64_t w_pitch, float* Z,
                        int P, int M, int Mp, int N);
void launch_softmax_grad(hipStream_t s, const float* part, int KS, const float* bias, int64_t w_pitch,
                         const int32_t* labels, const int32_t* idx, float* G, int P, int M, int Mp, int C, int Cp);
// b1 (optional, replica 0's; replica p at + p*w_pitch): also take the SGD step
// b1[h] -= lr * sum_m G1[m][h] (delayed updates, where no update GEMM steps b1).
// vb1 (optional, with b1): heavy-ball buffer of b1 (laid out like it) for the
// step with momentum mu and decay wd (d = sum + wd*b1; v <- mu*v + d).
// b2 (M <= 32, plain SGD; lr required): also the second layer's step,
// W2 -= lr * G2^T relu(Z1) and b2 -= lr * column sums of G2, in the same pass
// over W2 (no update GEMM for this layer).
void launch_bwd_hidden(hipStream_t s, const float* G2, float* W2, int64_t w_pitch, const float* Z1, float* G1, int P,
                       int M, int Mp, int C, int Cp, int Hp, float* b1 = nullptr, const float* lr = nullptr,
                       float* vb1 = nullptr, float mu = 0.0f, float wd = 0.0f, float* b2 = nullptr);
// Whether launch_bwd_hidden takes the second layer's step for M samples.
bool bwd_hidden_update_supported(int M, int Cp);
// Heavy-ball delayed updates, after a block's last step: Gu[k] = u_{K1-1-k}
// Gs[k] and (Gt set) Gt[k] = t_{K1-1-k} Gs[k] for k < K1, n floats per step
// (n a multiple of 4).
void launch_scale_errors(hipStream_t s, const float* Gs, float* Gu, float* Gt, const float* hb, int K1, int64_t n);
// Pre-activations of step k of a block under delayed updates for the head
// with more than 32 classes: Z1 = b1 + sum of the split-K partials
// - lr * sum_{k2<k} gram[k][k2] G1[k2] (M <= 32, K1 <= 8).
struct Z1Args {
  const float* part;      // step k's layer-1 split-K partials (split floats apart)
  int KS;
  int64_t split;
  const float* b1;        // replica 0's b1; replica p at + p*w_pitch
  int64_t w_pitch;
  const float* gs;        // [K1][P][Mp][Hp] hidden errors of the block's steps
  const float* gram;      // [P][K1][K1][Mp][Mp] of the block
  float* Z1;              // [P][Mp][Hp]
  const float* lr;
  int P, M, Mp, Hp, K1, k;
  // Heavy-ball delayed updates (hb set): Z1 = p_k (partials) + q_k (partv
  // partials, if set) + b1 + sum_{k2<k} u_{k-1-k2} gram[k][k2] G1[k2].
  const float* hb = nullptr;
  const float* partv = nullptr;  // step k's partials of X_k V^T, splits splitv apart
  int KSv = 0;
  int64_t splitv = 0;
};
void launch_z1_delayed(hipStream_t s, const Z1Args& a);
// part_split: floats between split-K partial sums (0: P * Mp * Hp).
void launch_head_a(hipStream_t s, const float* part, int KS, const float* b1, const float* W2, const float* b2,
                   int64_t w_pitch, float* Z1, float* PL, int P, int M, int Mp, int C, int Cp, int Hp,
                   int64_t part_split = 0);
// Heavy-ball step with L2 decay of the second layer and the biases in
// k_head_b: buffers laid out like W2, b1, b2 (nullptr: no buffers).
struct HeadMom {
  float* vw2 = nullptr;
  float* vb1 = nullptr;
  float* vb2 = nullptr;
  float mu = 0.0f, wd = 0.0f;
};
void launch_head_b(hipStream_t s, const float* PL, float* W2, float* b1, float* b2, int64_t w_pitch,
                   const float* Z1, float* G1, const int32_t* labels, const int32_t* idx, int P, int M, int Mp, int C,
                   int Cp, int Hp, const float* lr, HeadMom mom = HeadMom());
// The eager loss side (C <= 32) in two launches: one workgroup per learner
// and 16 samples (G1 and the group's gradient rows of b1, W2, b2:
// launch_head_fused), then the step of b1, W2, b2 from the rows
// (launch_head_w2_step).  Supported when head_fused_supported(Hp, Cp).
struct HeadFusedArgs {
  const float* part = nullptr;  // [KS][P][Mp][Hp] split-K partials of the layer-1 product, `split` floats apart
  int KS = 1;
  int64_t split = 0;
  float* b1 = nullptr;  // learner 0's b1, W2 ([Cp][Hp], rows C.. zero), b2; learners w_pitch apart
  float* W2 = nullptr;
  float* b2 = nullptr;
  int64_t w_pitch = 0;
  float* G1 = nullptr;  // [P][Mp][Hp] hidden error (rows M..Mp-1 written as zeros)
  const int32_t* labels = nullptr;
  const int32_t* idx = nullptr;  // [P][M]
  int P = 0, M = 0, Mp = 0, C = 0, Cp = 0, Hp = 0;
  const float* lr = nullptr;
  HeadMom mom;
  float* scratch = nullptr;  // head_fused_scratch_floats(P, Mp, C, Hp) floats
};
bool head_fused_supported(int Hp, int Cp);
int64_t head_fused_scratch_floats(int P, int Mp, int C, int Hp);
void launch_head_fused(hipStream_t s, const HeadFusedArgs& a);
void launch_head_w2_step(hipStream_t s, const HeadFusedArgs& a);

// Head of the delayed schedule (C <= 32, M <= 32, K1 <= 8), step k of a
// block: workgroup (p, slice of 32 hidden units) finishes step k-1's backward
// for its units (logits from every slice's partial logits, softmax gradient,
// hidden error into gs[k-1], SGD steps of b1, W2 and, on slice 0, b2) and
// runs step k's forward for them (pre-activations with the Gram correction,
// partial logits).  k = 0: forward only; k = K1: backward of the block's last
// step.
struct HeadStepArgs {
  const float* part;      // the block's layer-1 split-K partials: step k at + k*P*Mp*Hp, splits `split` apart
  int KS;
  int64_t split;
  float* W2;              // replica 0's second weight block; replica p at + p*w_pitch
  float* b1;
  float* b2;
  int64_t w_pitch;
  float* Z1;              // [P][Mp][Hp] pre-activations of the current step
  float* PL;              // [2][P][Mp][Cp][Hp/32] partial logits (step parity)
  int64_t pl_half;        // floats per parity
  float* gs;              // [K1][P][Mp][Hp] hidden errors of the block's steps
  const float* gram;      // [P][K1][K1][Mp][Mp] of the block
  const int32_t* ylab;    // [K1][P][M] labels of the block's samples
  const float* lr;        // device scalar step size
  int P, M, Mp, C, Cp, Hp, K1;
  // Heavy-ball delayed updates (hb set: the coefficient table): the forward
  // of step k is p_k (part) + q_k (partv, if set) + b1 + sum_{k2<k}
  // u_{k-1-k2} gram[k][k2] G1[k2], and b1, W2, b2 take heavy-ball steps with
  // decay (buffers vb1, vw2, vb2 laid out like b1, W2, b2; null when mu = 0).
  const float* hb = nullptr;
  const float* partv = nullptr;
  int KSv = 0;
  int64_t splitv = 0;
  float* vw2 = nullptr;
  float* vb1 = nullptr;
  float* vb2 = nullptr;
  float mu = 0.0f, wd = 0.0f;
};
// One launch for step k.
void launch_head_step(hipStream_t s, const HeadStepArgs& a, int k);

// Per-row softmax cross-entropy and first-argmax hit of an evaluation chunk
// from split-K logit partials part[ks][m][Cp] (split floats apart) and bias.
void launch_eval_rows(hipStream_t s, const float* part, int KS, int64_t split, const float* bias, const int32_t* y,
                      int M, int Cp, int C, float* loss, int32_t* hit);

// Averaging (k_avg.hip).
// Mean over each cluster of S rows of the columns [0, len) of W (row pitch
// `pitch`, both multiples of 4 floats).
void launch_group_mean(hipStream_t s, float* W, int64_t pitch, int64_t len, int P, int S);
// dst[i] = mean over r < n of src[r*pitch + i], i < len (multiples of 4
// floats); in the same launch (W set) the columns [0, len_b) of the nb rows
// of W (pitch_b apart) replaced by their mean.
void launch_mean_rows(hipStream_t s, float* dst, const float* src, int64_t pitch, int64_t len, int n,
                      float* W = nullptr, int64_t pitch_b = 0, int64_t len_b = 0, int nb = 0);
// flag = 1 if any of rows 1..n-1 of W (pitch floats apart) differs from row 0
// in columns [0, len) (bit patterns; len a multiple of 4); flag untouched otherwise.
void launch_rows_differ(hipStream_t s, const float* W, int64_t pitch, int64_t len, int n, int* flag);
// flag = 1 if any of the n floats at W is inf or NaN (n a multiple of 4).
void launch_any_nonfinite(hipStream_t s, const float* W, int64_t n, int* flag);
// Heavy-ball step of every learner on its given gradient, optionally followed
// by the mean over each cluster of S rows (average).  shared_in (optional,
// Dp floats): every learner's parameters are read from this vector instead of
// its row (after a global mean they are the same); mean_out (optional, Dp
// floats, S = P): the global mean goes there instead of to the P rows.  The
// two never alias the rows.
void launch_momentum_step(hipStream_t s, float* W, float* V, const float* Gr, int64_t Dp, int P, int S,
                          bool average, const float* lr, float mu, float wd, const float* shared_in = nullptr,
                          float* mean_out = nullptr);

}  // namespace hav
