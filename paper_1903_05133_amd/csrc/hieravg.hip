// C ABI, handle and round scheduler of the Hier-AVG hot path (Algorithm 1,
// Sec. 3.1).  A round is enqueued on one HIP stream with no host
// synchronisation inside it:
//
//   draw the round's minibatch indices
//   for b in 0..K2-1, k in 0..K1-1:    one local SGD step of all P learners
//     (after the last step of block b < K2-1: local mean over each cluster)
//   global mean over all P learners
//
// The local mean right before the global mean is left out: means of
// equal-size cluster means equal the global mean, so it changes nothing but
// rounding.
//
// Two schedules compute this round (include/hieravg.h, update_mode):
//  - eager: every step updates every learner's first weight block.  Where the
//    fused step kernel applies (padded minibatch up to 64), the update at
//    step t also computes the first-layer forward partials of step t+1 from
//    the new weights, and at the end of a block also takes the cluster mean
//    of that block in between; a small kernel then takes the cluster mean of
//    the remaining parameters.  Only step 0 of a round runs the stand-alone
//    forward kernel, and the last step the plain update before the global
//    mean.
//  - delayed (MLP): within a block the first weight block of every learner of
//    a cluster is the cluster's block-start copy minus the rank-B updates of
//    its earlier steps, so one GEMM per cluster gives the forward of all K1
//    steps (plus Gram corrections), and one GEMM per cluster at the block end
//    applies the K1*S learners' updates and the cluster mean together.
#include <algorithm>
#include <cmath>
#include <cstdlib>
#include <cstring>
#include <mutex>
#include <string>
#include <vector>

#include "internal.h"

using namespace hav;

namespace hav {
thread_local LaunchTiming g_launch_timing;
}

namespace {

thread_local std::string g_last_error;

void set_error(const std::string& s) { g_last_error = s; }

const char* kClassNames[KC_COUNT] = {
    "draw_indices", "fwd1_gemm",    "reduce1",      "fwd2_gemm",   "softmax_grad", "bwd_hidden",
    "head_a",       "head_b",       "update2_gemm", "update1_gemm", "group_mean",  "global_mean",
    "momentum",     "momentum_group_mean",          "momentum_global_mean",        "step1_gemm",
    "step1_gemm_group_mean",     "tail_group_mean", "gram", "fwd1_block_gemm", "block_update_gemm",
    "w1_global_mean", "tail_global_mean", "gram_reduce", "head_step", "head_step_end",
    "z1_delayed", "momentum_buffer_group_mean", "momentum_buffer_global_mean", "momentum_first_step",
    "fwd1_block_gemm_v", "scale_errors", "buffer_update_gemm", "update1_gemm_group_mean", "fwd1_group_gemm",
    "update1_gemm_global_mean", "head_fused", "head_w2_step"};

struct ProfRec {
  hipEvent_t a, b;
  int kc;
};

#define HAV_CHECK(expr)                                                                 \
  do {                                                                                  \
    hipError_t e_ = (expr);                                                             \
    if (e_ != hipSuccess) {                                                             \
      set_error(std::string(#expr) + " failed: " + hipGetErrorString(e_));             \
      return HIERAVG_EHIP;                                                              \
    }                                                                                   \
  } while (0)

}  // namespace

struct hieravg {
  hieravg_config cfg{};
  int64_t IN = 0, H = 0, C = 0, N = 0;
  int64_t INp = 0, Hp = 0, Cp = 0;
  int64_t D = 0, Dp = 0;
  int Bp = 0;
  int64_t off_W1 = 0, off_b1 = 0, off_W2 = 0, off_b2 = 0;

  float* W = nullptr;    // [P][Dp] replicas
  float* V = nullptr;    // [P][Dp] momentum buffers (momentum > 0, or the averaging kind)
  float* Gr = nullptr;   // [K1*K2][P][Dp] given gradients (averaging kind)
  float* Wm = nullptr;   // [Dp] averaging kind: every learner's parameters after a global mean
  float* X = nullptr;    // [N][INp] dataset
  int32_t* y = nullptr;  // [N] labels
  int32_t* idx = nullptr;  // [K2][K1][P][B] indices of the current round
  float* part = nullptr;   // split-K partial sums
  float* Z1 = nullptr;     // [P][Bp][Hp] hidden pre-activations
  float* PL = nullptr;     // [P][Bp][Cp][Hp/32] partial logits (small-C MLP)
  float* G2 = nullptr;     // [P][Bp][Cp] output error
  float* G1 = nullptr;     // [P][Bp][Hp] hidden error
  uint64_t* ctr = nullptr;  // [0]: global step counter; [1]: workgroup counter of the draw
  int* flag = nullptr;       // result word of device-side checks
  int n_allocs = 0, fail_alloc = 0;  // allocation count of create; the forced failure (debug)
  float* hyper = nullptr;   // [0]: step size lr read by the kernels (hieravg_set_lr); the heavy-ball
                            // coefficient table of the delayed schedule (internal.h)

  uint64_t key_index = 0;
  int KS1 = 1, cps1 = 1, KS2 = 1, cps2 = 1;
  int Bmax = 0;             // minibatch size at create: the buffers' capacity
  bool rows_stale = false;  // replicas 1..P-1 hold an old W1 (after a delayed round);
                            // averaging kind: every row is old, Wm holds the parameters
  bool in_shared = false;   // averaging kind: the round being enqueued starts from Wm
  bool fused = false;       // the fused step kernel applies (SG = 1)
  bool fused_mean = false;  // ... and also with the cluster mean (SG = S)
  int KS_step = 1, KS_mean = 1;  // forward splits written by the fused kernel
  // Block ends the fused mean step cannot take (S * B too large for its
  // forward registers): the update with the cluster mean, then the next
  // step's forward as one GEMM per cluster from the common first layer.
  bool upd_mean = false;
  int KS_g = 1, cps_g = 1;
  bool upd_global = false;  // the round's last step: update with the global mean (SG = P)
  // More than 32 classes, B <= 32, plain SGD: the hidden-error kernel also
  // steps W2 and b2 (no update GEMM for the second layer).
  bool w2_fused = false;
  // At most 32 classes, eager steps: the loss side as k_head_fused and the
  // second layer's step from its per-group gradient rows.
  bool head_fused = false;
  float* hgrad = nullptr;
  // Eager rounds whose steps take the full-tile kernels: the round-end global
  // mean of W1 goes once to Wg (once_global) and the block-end cluster means
  // once to the cluster copies Wc (once_block); the next step reads its old
  // W1 there, and the next round's first forward is one GEMM from Wg.  With
  // rows_stale, w1_wg says that every learner's W1 is Wg (not replica 0's).
  bool once_cond = false, once_alloc = false, once_global = false, once_block = false;
  float* Wg = nullptr;
  bool w1_wg = false;
  bool in_wg = false;         // the round being enqueued starts from Wg
  int KS_g0 = 1, cps_g0 = 1;  // splits of that first forward
  bool launch_failed = false; // a launch the plan promised was refused
  int ks_cur = 1;                // splits of the partials currently in `part`
  // Delayed first-layer updates (see hieravg.h, HIERAVG_UPDATE_DELAYED).
  bool delayed = false;    // the handle uses them for rounds that start with equal W1
  bool global_last = false; // the last block's update takes the global mean (K1*P*B rows fit)
  bool hb = false;          // delayed updates with momentum or weight decay (heavy-ball blocks)
  int KSv = 1, cpsv = 1;    // splits of the block-wide forward from the learners' buffers
  float* partv = nullptr;   // [KSv][K1][P][Bp][Hp] partials of X_k V^T (momentum > 0)
  float* Gu = nullptr;      // [K1][P][Bp][Hp] errors scaled for the block-end parameter update
  float* Gt = nullptr;      // [K1][P][Bp][Hp] errors scaled for the buffer update (momentum > 0)
  float* Wc2 = nullptr;     // second set of cluster copies (heavy-ball: the block-start copies stay
                            // intact for the buffer update)
  uint32_t* btab1 = nullptr;  // per-learner row tables of the buffer update
  bool w1_shared = true;   // every learner's W1 equals replica 0's (other rows may be stale)
  bool in_delayed = false; // the round being enqueued uses them
  int KS_b = 1, cps_b = 1; // splits of the block-wide forward
  float* Wc = nullptr;     // [P/S][Hp*INp] cluster copies of W1
  float* Gs = nullptr;     // [K1][P][Bp][Hp] hidden errors of the block's steps
  float* gram = nullptr;   // [KSG][K2][P][K1][K1][Bp][Bp] Gram blocks of the round
  int32_t* ylab = nullptr; // [T][P][B] labels of the drawn samples (delayed schedule)
  uint32_t* btab = nullptr; // [2][K2][P/S][Rp] row tables of the block update (BlkTables)
  float* part2 = nullptr;  // layer-2 split-K partials of the delayed schedule with more than 32 classes
  // Evaluation (allocated at the first hieravg_evaluate).
  int eval_rows = 0;                  // chunk capacity (multiple of 16)
  int64_t eval_part_cap = 0, eval_part2_cap = 0;  // floats in eval_part, eval_part2
  int32_t* eval_iota = nullptr;       // [eval_rows] 0, 1, 2, ...
  float *eval_part = nullptr, *eval_part2 = nullptr, *eval_Z1 = nullptr, *eval_loss = nullptr;
  int32_t* eval_hit = nullptr;
  int64_t n_test = 0;                 // held-out rows generated so far
  float* Xtest = nullptr;             // [n_test][INp]
  int32_t* ytest = nullptr;           // [n_test]
  int KSG = 1;             // feature splits of the Gram blocks
  hipStream_t own_stream = nullptr, stream = nullptr;
  int device = 0;  // the device current at create (every buffer lives there)
  int64_t steps = 0;
  int T = 1;  // SGD steps per round
  // One round's kernels, captured on first use and replayed for every round
  // that is not profiled (every launch argument is the same in every round).
  hipGraphExec_t round_exec[3] = {nullptr, nullptr, nullptr};  // [eager, delayed, eager from Wg]

  bool profiling = false;
  std::vector<ProfRec> recs;
  std::vector<hipEvent_t> pool;
};

namespace {

// Run `fn`, which makes exactly one kernel launch.  When profiling, the launch
// goes out with two events that its dispatch packet stamps; the recorded
// interval includes a few microseconds of dispatch latency per launch, so
// profiling gives launch counts and time shares, and hieravg_time_kernel
// gives per-launch durations.
template <class F>
void run(hieravg* h, int kc, F&& fn) {
  if (!h->profiling) {
    fn();
    return;
  }
  hipEvent_t ev[2];
  for (int i = 0; i < 2; ++i) {
    if (!h->pool.empty()) {
      ev[i] = h->pool.back();
      h->pool.pop_back();
    } else if (hipEventCreate(&ev[i]) != hipSuccess) {
      if (i == 1) h->pool.push_back(ev[0]);
      fn();
      return;
    }
  }
  g_launch_timing = {ev[0], ev[1]};
  fn();
  g_launch_timing = {};
  h->recs.push_back({ev[0], ev[1], kc});
}

void release(hieravg* h) {
  if (!h) return;
  if (h->stream) (void)hipStreamSynchronize(h->stream);
  void* bufs[] = {h->W,  h->V,  h->Gr, h->Wm, h->X,  h->y,  h->idx, h->part, h->Z1, h->hyper, h->btab,
                  h->PL, h->G2, h->G1, h->ctr, h->Wc, h->Gs, h->gram, h->ylab, h->part2, h->flag, h->eval_iota,
                  h->partv, h->Gu, h->Gt, h->Wc2, h->btab1, h->hgrad, h->Wg,
                  h->eval_part, h->eval_part2, h->eval_Z1, h->eval_loss, h->eval_hit, h->Xtest, h->ytest};
  for (void* b : bufs)
    if (b) (void)hipFree(b);
  for (auto& r : h->recs) {
    (void)hipEventDestroy(r.a);
    (void)hipEventDestroy(r.b);
  }
  for (auto e : h->pool) (void)hipEventDestroy(e);
  for (auto e : h->round_exec)
    if (e) (void)hipGraphExecDestroy(e);
  if (h->own_stream) (void)hipStreamDestroy(h->own_stream);

  delete h;
}

// Debug hook for the failure paths of create: HIERAVG_FAIL_ALLOC=n makes the
// n-th device allocation of a create (counted from 1) fail.
int forced_alloc_failure() {
  const char* v = std::getenv("HIERAVG_FAIL_ALLOC");
  return v ? std::atoi(v) : 0;
}

int alloc_zero(hieravg* h, void** p, size_t bytes, const char* what) {
  if (bytes == 0) bytes = 16;
  ++h->n_allocs;
  if (h->fail_alloc > 0 && h->n_allocs == h->fail_alloc) {
    *p = nullptr;
    set_error(std::string("hipMalloc of ") + what + " failed (HIERAVG_FAIL_ALLOC)");
    return HIERAVG_EHIP;
  }
  hipError_t e = hipMalloc(p, bytes);
  if (e != hipSuccess) {
    *p = nullptr;
    set_error(std::string("hipMalloc of ") + what + " (" + std::to_string(bytes) + " bytes) failed: " +
              hipGetErrorString(e));
    return HIERAVG_EHIP;
  }
  e = hipMemsetAsync(*p, 0, bytes, h->stream);
  if (e != hipSuccess) {
    set_error(std::string("hipMemsetAsync failed: ") + hipGetErrorString(e));
    return HIERAVG_EHIP;
  }
  return HIERAVG_OK;
}

bool delayed_applies(const hieravg_config& c) {
  const bool whole_blocks = c.k_global == 0 || c.k_global % c.K1 == 0;
  // The block update addresses dataset rows by 32-bit offsets in 64-float
  // units (a dataset below 2^38 floats).
  const bool rows_fit = (double)c.n_samples * (double)round_up(c.in_dim, 64) < 274877906944.0;
  return c.kind == HIERAVG_KIND_MLP && c.B <= 32 && c.K1 <= 8 && whole_blocks && rows_fit &&
         (int64_t)c.K1 * c.S * c.B <= kBlkMaxRows && c.avg_momentum == 0;
}

// Heavy-ball coefficient table (see internal.h) for step size lr, momentum
// mu and decay wd over blocks of up to K1 steps: A^n and A^n e in double,
// stored as float.
void hb_table(float lr, float mu, float wd, int K1, float* hyper) {
  const double g = lr, m = mu, l = wd;
  double a00 = 1.0, a01 = 0.0, a10 = 0.0, a11 = 1.0;  // A^0
  for (int n = 0; n <= K1 && n < kHbStride; ++n) {
    hyper[hb_index(HB_P, n)] = (float)a00;
    hyper[hb_index(HB_Q, n)] = (float)a01;
    hyper[hb_index(HB_R, n)] = (float)a10;
    hyper[hb_index(HB_S, n)] = (float)a11;
    hyper[hb_index(HB_U, n)] = (float)(-g * a00 + a01);
    hyper[hb_index(HB_T, n)] = (float)(-g * a10 + a11);
    // A^(n+1) = A A^n with A = [[1 - g l, -g m], [l, m]]
    const double b00 = (1.0 - g * l) * a00 - g * m * a10, b01 = (1.0 - g * l) * a01 - g * m * a11;
    const double b10 = l * a00 + m * a10, b11 = l * a01 + m * a11;
    a00 = b00;
    a01 = b01;
    a10 = b10;
    a11 = b11;
  }
}

int validate(const hieravg_config& c) {
  auto bad = [](const char* m) {
    set_error(m);
    return HIERAVG_EINVAL;
  };
  if (c.P < 1 || c.P > 65535) return bad("P must be in [1, 65535]");
  if (c.S < 1) return bad("S must be >= 1");
  if (c.P % c.S != 0) return bad("S must divide P (Sec. 2: S | P)");
  if (c.K1 < 1) return bad("K1 must be >= 1");
  if (c.k_global < 0) return bad("k_global must be >= 0");
  if (c.k_global == 0 && c.K2 < 1) return bad("K2 must be >= 1");
  const int64_t T = c.k_global > 0 ? (int64_t)c.k_global : (int64_t)c.K1 * c.K2;
  if (T > (1 << 20)) return bad("steps per round (K1*K2 or k_global) must be <= 2^20");
  if (!std::isfinite(c.lr) || c.lr < 0.0f) return bad("lr must be finite and >= 0");
  if (c.update_mode < HIERAVG_UPDATE_AUTO || c.update_mode > HIERAVG_UPDATE_DELAYED)
    return bad("update_mode must be one of HIERAVG_UPDATE_*");
  if (!std::isfinite(c.momentum) || c.momentum < 0.0f || c.momentum >= 1.0f)
    return bad("momentum must be in [0, 1)");
  if (!std::isfinite(c.weight_decay) || c.weight_decay < 0.0f) return bad("weight_decay must be finite and >= 0");
  if (c.avg_momentum != 0 && c.avg_momentum != 1) return bad("avg_momentum must be 0 or 1");
  if (c.update_mode == HIERAVG_UPDATE_DELAYED && !delayed_applies(c))
    return bad("delayed updates need the MLP with B <= 32, K1 <= 8, K1*S*B <= 16384, whole blocks and momentum "
               "buffers that are not averaged (avg_momentum = 0)");
  if (c.kind == HIERAVG_KIND_AVERAGING) {
    if (c.in_dim < 1 || c.in_dim > (int64_t(1) << 36)) return bad("averaging: D must be in [1, 2^36]");
    if (!std::isfinite(c.init_std) || !std::isfinite(c.grad_std)) return bad("averaging: stds must be finite");
    if (T * c.P > 65535) return bad("averaging: steps per round * P must be <= 65535");
    return HIERAVG_OK;
  }
  if (c.kind != HIERAVG_KIND_SOFTMAX && c.kind != HIERAVG_KIND_MLP) return bad("unknown model kind");
  if (c.B < 1 || c.B > 65535) return bad("B must be in [1, 65535]");
  if (c.in_dim < 1 || c.in_dim > (1 << 24)) return bad("in_dim must be in [1, 2^24]");
  if (c.classes < 1 || c.classes > (1 << 20)) return bad("classes must be in [1, 2^20]");
  if (c.kind == HIERAVG_KIND_MLP && (c.hidden < 1 || c.hidden > (1 << 20))) return bad("hidden must be in [1, 2^20]");
  if (c.n_samples < 1 || c.n_samples > 0x7fffffffLL) return bad("n_samples must be in [1, 2^31 - 1]");
  if (!std::isfinite(c.noise_std)) return bad("noise_std must be finite");
  if (T * c.P * c.B > 0x7fffffffLL) return bad("steps per round * P * B must be < 2^31");
  return HIERAVG_OK;
}

float fan_in_scale(int64_t fan_in) { return (float)(1.0 / std::sqrt((double)fan_in)); }

// Launch plan for minibatch size B (softmax / MLP kinds): padded batch,
// split counts, which fused and delayed kernels apply.  Returns the partial
// buffer size the plan needs, in floats.
int64_t plan(hieravg* h, int B) {
  const hieravg_config& c = h->cfg;
  const int P = c.P;
  const bool mlp = c.kind == HIERAVG_KIND_MLP;
  const int64_t n1 = mlp ? h->Hp : h->Cp;
  h->Bp = (int)round_up(B, 16);
  h->KS2 = h->cps2 = 1;
  plan_split(P, h->Bp, (int)n1, (int)h->INp, &h->KS1, &h->cps1);
  if (mlp) plan_split(P, h->Bp, (int)h->Cp, (int)h->Hp, &h->KS2, &h->cps2);
  // The fused step kernels take the plain SGD step only.
  h->fused = h->T >= 2 && step_w1_supported(h->Bp, 1) && c.momentum == 0.0f && c.weight_decay == 0.0f;
  h->fused_mean = h->fused && c.S > 1 && step_w1_supported(h->Bp, c.S);
  int64_t ks_max = h->KS1;
  if (h->fused) {
    h->KS_step = step_w1_splits(P, 1, h->Bp, (int)n1, (int)h->INp);
    ks_max = std::max<int64_t>(ks_max, h->KS_step);
  }
  h->upd_mean = mlp && h->fused && c.S > 1 && !h->fused_mean && step_w1_mean_supported(h->Bp, c.S);
  h->upd_global = mlp && h->fused && step_w1_mean_supported(h->Bp, P);
  h->w2_fused = mlp && c.classes > kSmallC && bwd_hidden_update_supported(B, (int)round_up(c.classes, 16)) && c.momentum == 0.0f &&
                c.weight_decay == 0.0f;
  h->head_fused = mlp && c.classes <= kSmallC && head_fused_supported((int)h->Hp, (int)round_up(c.classes, 16));
  if (h->upd_mean) {
    plan_split_blk(P / c.S, c.S * h->Bp, (int)n1, (int)h->INp, &h->KS_g, &h->cps_g);
    ks_max = std::max<int64_t>(ks_max, h->KS_g);
  }
  if (h->fused_mean) {
    h->KS_mean = step_w1_splits(P, c.S, h->Bp, (int)n1, (int)h->INp);
    ks_max = std::max<int64_t>(ks_max, h->KS_mean);
  }
  // Step 0 must be a kernel that reads a redirected old W1: a full-tile step
  // or update with the mean (not the fused mean step or the update GEMM).
  h->once_cond = mlp && h->fused && h->upd_global && (c.K1 > 1 || c.S == 1 || h->upd_mean) &&
                 step_full_shape(B, h->Bp, (int)h->Hp, (int)h->INp, h->N, h->INp, h->Hp, h->INp);
  h->once_global = h->once_cond && h->once_alloc;
  h->once_block = h->once_global && h->upd_mean && c.S > 1;
  if (h->once_cond) {
    plan_split_blk(1, P * h->Bp, (int)h->Hp, (int)h->INp, &h->KS_g0, &h->cps_g0);
    ks_max = std::max<int64_t>(ks_max, h->KS_g0);
  }
  h->delayed = false;
  hieravg_config cb = c;
  cb.B = B;
  if (mlp && delayed_applies(cb)) {
    const bool cheap = (int64_t)(c.K1 - 1) * h->Bp * 2 <= h->Hp;
    h->delayed = c.update_mode == HIERAVG_UPDATE_DELAYED || (c.update_mode == HIERAVG_UPDATE_AUTO && cheap);
  }
  // The last block's update over all P learners has one group of output
  // tiles (64 x 128); with fewer than two per CU the G cluster updates and a
  // separate mean of the copies fill the GPU better.  Heavy-ball blocks with
  // one block per round keep the cluster updates: the buffers' update needs
  // the block-start parameters, which the global update would overwrite.
  h->hb = h->delayed && (c.momentum > 0.0f || c.weight_decay > 0.0f);
  h->global_last = h->delayed && (int64_t)c.K1 * P * B <= kBlkMaxRows && (h->Hp / 64) * (h->INp / 128) >= 512 &&
                   !(h->hb && c.K2 < 2);
  if (h->delayed) {
    // One GEMM per cluster and block: the K1*S minibatches against the copy.
    plan_split_blk(P / c.S, c.K1 * c.S * h->Bp, (int)h->Hp, (int)h->INp, &h->KS_b, &h->cps_b);
    ks_max = std::max<int64_t>(ks_max, (int64_t)h->KS_b * c.K1);
    // Heavy-ball with momentum: one more per learner, its K1 minibatches
    // against its own buffer.
    if (h->hb && c.momentum > 0.0f)
      plan_split_blk(P, c.K1 * h->Bp, (int)h->Hp, (int)h->INp, &h->KSv, &h->cpsv);
  }
  h->ks_cur = h->KS1;
  return std::max<int64_t>(ks_max * P * h->Bp * n1, mlp ? (int64_t)h->KS2 * P * h->Bp * h->Cp : 0);
}

// The step size and the heavy-ball coefficient table, to the device.
hipError_t write_hyper(hieravg* h) {
  float hyper[kHyperFloats] = {};
  hyper[0] = h->cfg.lr;
  hb_table(h->cfg.lr, h->cfg.momentum, h->cfg.weight_decay, std::min(h->cfg.K1, kHbStride - 1), hyper);
  const hipError_t e = hipMemcpyAsync(h->hyper, hyper, sizeof(hyper), hipMemcpyHostToDevice, h->stream);
  if (e != hipSuccess) return e;
  return hipStreamSynchronize(h->stream);
}

int build(hieravg* h) {
  const hieravg_config& c = h->cfg;
  HAV_CHECK(hipGetDevice(&h->device));
  HAV_CHECK(hipStreamCreateWithFlags(&h->own_stream, hipStreamNonBlocking));
  h->stream = h->own_stream;
  {
    int rc;
    if ((rc = alloc_zero(h, (void**)&h->hyper, kHyperFloats * sizeof(float), "hyperparameters"))) return rc;
    HAV_CHECK(write_hyper(h));
  }
  const int P = c.P;
  const uint64_t seed = c.seed;

  if (c.kind == HIERAVG_KIND_AVERAGING) {
    h->D = c.in_dim;
    h->Dp = round_up(h->D, 64);
    const int T = h->T;
    int rc;
    if ((rc = alloc_zero(h, (void**)&h->W, sizeof(float) * P * h->Dp, "replicas"))) return rc;
    if ((rc = alloc_zero(h, (void**)&h->V, sizeof(float) * P * h->Dp, "momentum buffers"))) return rc;
    if ((rc = alloc_zero(h, (void**)&h->Gr, sizeof(float) * (size_t)T * P * h->Dp, "given gradients"))) return rc;
    if ((rc = alloc_zero(h, (void**)&h->ctr, 2 * sizeof(uint64_t), "counters"))) return rc;
    if ((rc = alloc_zero(h, (void**)&h->Wm, sizeof(float) * h->Dp, "common parameters"))) return rc;
    launch_init_vector(h->stream, h->W, h->D, hash64(seed, kTagInit), c.init_std);
    launch_gen_grads(h->stream, h->Gr, h->D, h->Dp, P, T, hash64(seed, kTagGrad), c.grad_std);
    // Every learner starts from w~_1: the first round reads it from Wm.
    HAV_CHECK(hipMemcpyAsync(h->Wm, h->W, sizeof(float) * h->Dp, hipMemcpyDeviceToDevice, h->stream));
  } else {
    const bool mlp = c.kind == HIERAVG_KIND_MLP;
    h->IN = c.in_dim;
    h->C = c.classes;
    h->H = mlp ? c.hidden : 0;
    h->N = c.n_samples;
    h->INp = round_up(h->IN, 64);
    h->Cp = round_up(h->C, 16);
    h->Hp = mlp ? round_up(h->H, 64) : 0;
    if (mlp) {
      h->off_W1 = 0;
      h->off_b1 = h->Hp * h->INp;
      h->off_W2 = h->off_b1 + h->Hp;
      h->off_b2 = h->off_W2 + h->Cp * h->Hp;
      h->Dp = round_up(h->off_b2 + h->Cp, 64);
      h->D = h->H * h->IN + h->H + h->C * h->H + h->C;
    } else {
      h->off_W1 = 0;
      h->off_b1 = h->Cp * h->INp;
      h->Dp = round_up(h->off_b1 + h->Cp, 64);
      h->D = h->C * h->IN + h->C;
    }
    const int T = h->T;
    // Buffers hold the largest launch plan over every batch size up to the
    // create-time B (hieravg_set_batch may lower it).
    h->Bmax = c.B;
    int64_t part_floats = 0, part2_floats = 0, partv_floats = 0;
    bool any_delayed = false, any_hb = false, any_once = false;
    int Bp_del = 0;
    for (int b = 16; b <= round_up(c.B, 16); b += 16) {
      const int64_t pf = plan(h, std::min(b, c.B));
      part_floats = std::max(part_floats, pf);
      any_once = any_once || h->once_cond;
      if (h->delayed) {
        any_delayed = true;
        any_hb = any_hb || h->hb;
        Bp_del = std::max(Bp_del, h->Bp);
        part2_floats = std::max<int64_t>(part2_floats, (int64_t)h->KS2 * P * h->Bp * h->Cp);
        if (h->hb) partv_floats = std::max<int64_t>(partv_floats, (int64_t)h->KSv * c.K1 * P * h->Bp * h->Hp);
      }
    }
    plan(h, c.B);
    h->Bp = (int)round_up(c.B, 16);
    int rc;
    if ((rc = alloc_zero(h, (void**)&h->W, sizeof(float) * P * h->Dp, "replicas"))) return rc;
    if (c.momentum > 0.0f &&
        (rc = alloc_zero(h, (void**)&h->V, sizeof(float) * P * h->Dp, "momentum buffers")))
      return rc;
    if ((rc = alloc_zero(h, (void**)&h->X, sizeof(float) * h->N * h->INp, "dataset"))) return rc;
    if ((rc = alloc_zero(h, (void**)&h->y, sizeof(int32_t) * h->N, "labels"))) return rc;
    if ((rc = alloc_zero(h, (void**)&h->idx, sizeof(int32_t) * (size_t)T * P * c.B, "indices"))) return rc;
    if ((rc = alloc_zero(h, (void**)&h->part, sizeof(float) * part_floats, "split-K partials"))) return rc;
    if ((rc = alloc_zero(h, (void**)&h->G2, sizeof(float) * P * h->Bp * h->Cp, "output error"))) return rc;
    if (mlp && h->C <= kSmallC &&
        (rc = alloc_zero(h, (void**)&h->PL, sizeof(float) * 2 * P * (h->Hp / 32) * h->Bp * h->Cp, "partial logits")))
      return rc;
    if (mlp) {
      if ((rc = alloc_zero(h, (void**)&h->Z1, sizeof(float) * P * h->Bp * h->Hp, "hidden activations"))) return rc;
      if ((rc = alloc_zero(h, (void**)&h->G1, sizeof(float) * P * h->Bp * h->Hp, "hidden error"))) return rc;
      if (any_once) {
        const size_t w1 = sizeof(float) * h->Hp * h->INp;
        if ((rc = alloc_zero(h, (void**)&h->Wg, w1, "common first layer")) ||
            (c.S > 1 && (rc = alloc_zero(h, (void**)&h->Wc, w1 * (P / c.S), "cluster copies of W1"))))
          return rc;
        h->once_alloc = true;
      }
      if (h->head_fused) {
        if ((rc = alloc_zero(h, (void**)&h->hgrad,
                             sizeof(float) * head_fused_scratch_floats(P, h->Bp, h->C, (int)h->Hp),
                             "head gradient rows")))
          return rc;
      }
    }
    if ((rc = alloc_zero(h, (void**)&h->ctr, 2 * sizeof(uint64_t), "counters"))) return rc;
    if (any_delayed) {
      const int64_t w1 = h->Hp * h->INp;
      if (!h->Wc && (rc = alloc_zero(h, (void**)&h->Wc, sizeof(float) * (P / c.S) * w1, "cluster copies of W1")))
        return rc;
      if ((rc = alloc_zero(h, (void**)&h->Gs, sizeof(float) * c.K1 * P * Bp_del * h->Hp, "block errors"))) return rc;
      if (any_hb) {
        if ((rc = alloc_zero(h, (void**)&h->Wc2, sizeof(float) * (P / c.S) * w1, "second cluster copies of W1")) ||
            (rc = alloc_zero(h, (void**)&h->Gu, sizeof(float) * c.K1 * P * Bp_del * h->Hp, "scaled block errors")))
          return rc;
        if (c.momentum > 0.0f) {
          const int64_t rp1 = round_up((int64_t)c.K1 * c.B, 32);
          if ((rc = alloc_zero(h, (void**)&h->Gt, sizeof(float) * c.K1 * P * Bp_del * h->Hp, "buffer block errors")) ||
              (rc = alloc_zero(h, (void**)&h->partv, sizeof(float) * partv_floats, "buffer partials")) ||
              (rc = alloc_zero(h, (void**)&h->btab1, 2 * sizeof(uint32_t) * (size_t)c.K2 * P * rp1,
                               "buffer update row tables")))
            return rc;
        }
      }
      if ((rc = alloc_zero(h, (void**)&h->ylab, sizeof(int32_t) * (size_t)T * P * c.B, "sample labels"))) return rc;
      const int64_t rp = round_up((int64_t)c.K1 * c.S * c.B, 32);
      if ((rc = alloc_zero(h, (void**)&h->btab, 2 * sizeof(uint32_t) * (size_t)c.K2 * (P / c.S) * rp,
                           "block update row tables")))
        return rc;
      // more than 32 classes: the layer-2 partials of a step must not overwrite
      // the block forward's partials of the later steps
      if (h->C > kSmallC &&
          (rc = alloc_zero(h, (void**)&h->part2, sizeof(float) * part2_floats, "layer-2 partials")))
        return rc;
      h->KSG = gram_splits(P, c.K2, (int)h->INp);
      if (c.K1 > 1 && (rc = alloc_zero(h, (void**)&h->gram,
                                       sizeof(float) * h->KSG * c.K2 * P * c.K1 * c.K1 * Bp_del * Bp_del, "Gram blocks")))
        return rc;
    }
    plan(h, c.B);  // again, now that the buffers of the once-written means exist
    h->key_index = hash64(seed, kTagIndex);
    launch_gen_labels(h->stream, h->y, h->N, hash64(seed, kTagLabel), (uint64_t)h->C);
    launch_gen_data(h->stream, h->X, h->y, h->N, h->IN, h->INp, hash64(seed, kTagMean), hash64(seed, kTagNoise),
                    c.noise_std);
    const uint64_t kinit = hash64(seed, kTagInit);
    if (mlp) {
      launch_init_matrix(h->stream, h->W + h->off_W1, h->H, h->IN, h->INp, kinit, 0, fan_in_scale(h->IN));
      launch_init_matrix(h->stream, h->W + h->off_W2, h->C, h->H, h->Hp, kinit, 1, fan_in_scale(h->H));
    } else {
      launch_init_matrix(h->stream, h->W + h->off_W1, h->C, h->IN, h->INp, kinit, 0, fan_in_scale(h->IN));
    }
  }
  HAV_CHECK(hipGetLastError());
  // Synchronize every learner with w~_1 (Algorithm 1, first lines).
  for (int p = 1; p < P; ++p)
    HAV_CHECK(hipMemcpyAsync(h->W + (int64_t)p * h->Dp, h->W, sizeof(float) * h->Dp, hipMemcpyDeviceToDevice,
                             h->stream));
  HAV_CHECK(hipStreamSynchronize(h->stream));
  return HIERAVG_OK;
}

// The heavy-ball buffers and decay of an update GEMM over the parameter block
// at offset `off` (bias at `boff`) of the replica rows.
void with_momentum(const hieravg* h, UpdArgs& u, int64_t off, int64_t boff) {
  u.mu = h->cfg.momentum;
  u.wd = h->cfg.weight_decay;
  if (h->V) {
    u.V = h->V + off;
    u.vbias = u.bias ? h->V + boff : nullptr;
  }
}

// Cluster copies written by the update of block b (read by block b + 1):
// one set, updated in place, for plain SGD; heavy-ball blocks alternate two
// sets so that the buffer update still reads the block-start copies.
float* wc_buf(const hieravg* h, int b) { return h->hb && (b & 1) ? h->Wc2 : h->Wc; }

// Averaging kind: the launch class of step tt of a round (the heavy-ball step
// alone, with the cluster mean at the end of a block, or with the global mean
// at the end of the round).
int avg_step_mean(const hieravg* h, int tt) {
  const hieravg_config& c = h->cfg;
  const bool end_round = tt == h->T - 1, end_block = (tt + 1) % c.K1 == 0;
  if (end_round && c.P > 1) return KC_MOMENTUM_GLOBAL;
  if (end_block && !end_round && c.S > 1) return KC_MOMENTUM_GROUP;
  return KC_MOMENTUM;
}

// The single kernel launch of class `kc` for step tt of the current round
// (tt selects the step's sample indices, or the averaging workload's given
// gradients).  Returns false for a class this workload does not launch.
bool launch_class(hieravg* h, int kc, int tt) {
  const hieravg_config& c = h->cfg;
  const int P = c.P, B = c.B, S = c.S;
  hipStream_t s = h->stream;
  float* W = h->W;
  if (c.kind == HIERAVG_KIND_AVERAGING) {
    const float* g = h->Gr + (int64_t)tt * P * h->Dp;
    switch (kc) {
      case KC_MOMENTUM:
        launch_momentum_step(s, W, h->V, g, h->Dp, P, 1, false, h->hyper, c.momentum, c.weight_decay);
        return true;
      case KC_MOMENTUM_GROUP:
        launch_momentum_step(s, W, h->V, g, h->Dp, P, S, true, h->hyper, c.momentum, c.weight_decay);
        return true;
      case KC_MOMENTUM_GLOBAL:  // every learner shares the result: it goes to Wm once
        launch_momentum_step(s, W, h->V, g, h->Dp, P, P, true, h->hyper, c.momentum, c.weight_decay, nullptr,
                             h->Wm);
        return true;
      case KC_MOMENTUM_FIRST: {  // the round's first step, every learner starting from Wm
        if (!h->in_shared) return false;
        const int v = avg_step_mean(h, 0);
        launch_momentum_step(s, W, h->V, g, h->Dp, P, v == KC_MOMENTUM_GLOBAL ? P : S, v != KC_MOMENTUM, h->hyper,
                             c.momentum, c.weight_decay, h->Wm, h->Wm);
        return true;
      }
      case KC_VMEAN_GROUP:
      case KC_VMEAN_GLOBAL: launch_group_mean(s, h->V, h->Dp, h->Dp, P, kc == KC_VMEAN_GROUP ? S : P); return true;
      default: return false;
    }
  }
  const int32_t* ix = h->idx + (int64_t)tt * P * B;
  const int Bp = h->Bp, C = (int)h->C, Cp = (int)h->Cp, Hp = (int)h->Hp, INp = (int)h->INp;
  const bool mlp = c.kind == HIERAVG_KIND_MLP, small = mlp && C <= kSmallC;
  const int64_t w1 = (int64_t)h->Hp * h->INp;
  // Where step tt reads its old W1: Wg for a round's first step after a
  // round that wrote it, a cluster copy for the step after a block end
  // (once_block), else the learner's row.
  auto old_w1 = [&](StepArgs& a) {
    if (tt == 0 && h->in_wg) {
      a.w_src = h->Wg;
      a.src_pitch = 0;
      a.src_group = P;
    } else if (h->once_block && tt > 0 && tt % c.K1 == 0) {
      a.w_src = h->Wc;
      a.src_pitch = w1;
      a.src_group = S;
    }
  };
  auto step = [&](const StepArgs& a) {
    if (!launch_step_w1(s, a)) h->launch_failed = true;
  };
  switch (kc) {
    case KC_DRAW: {
      BlkTables tb;
      if (h->in_delayed) {
        tb.Rp = (int)round_up((int64_t)c.K1 * S * B, 32);
        tb.gtab = h->btab;
        tb.xtab = h->btab + (int64_t)c.K2 * (P / S) * tb.Rp;
        tb.K1 = c.K1;
        tb.S = S;
        tb.Mp = Bp;
        tb.ldg = h->Hp;
        tb.ldx = h->INp;
        tb.K2 = c.K2;
        tb.global_last = h->global_last;
        if (h->hb && h->V) {
          tb.Rp1 = (int)round_up((int64_t)c.K1 * B, 32);
          tb.gtab1 = h->btab1;
          tb.xtab1 = h->btab1 + (int64_t)c.K2 * P * tb.Rp1;
        }
      }
      launch_draw_indices(s, h->idx, h->ctr, (uint32_t*)(h->ctr + 1), P, B, h->T, (uint64_t)h->N,
                          h->key_index, h->y, h->in_delayed ? h->ylab : nullptr, tb);
      return true;
    }
    case KC_FWD1: {
      if (tt == 0 && h->in_wg) {  // every learner's W1 is Wg: one GEMM over all P minibatches
        FwdArgs f{h->X, ix, h->INp, h->Wg, 0, h->INp, h->part, P, B, Bp, Hp, INp, h->KS_g0, h->cps_g0};
        f.SG = P;
        launch_fwd_blk(s, f);
        h->ks_cur = h->KS_g0;
        return true;
      }
      FwdArgs f{h->X, ix, h->INp, W + h->off_W1, h->Dp, h->INp, h->part, P, B, Bp, mlp ? Hp : Cp, INp, h->KS1,
                h->cps1};
      launch_fwd(s, f, A_GATHER);
      h->ks_cur = h->KS1;
      return true;
    }
    case KC_SOFTMAX:
      if (small) return false;
      launch_softmax_grad(s, h->in_delayed ? h->part2 : h->part, mlp ? h->KS2 : h->ks_cur,
                          W + (mlp ? h->off_b2 : h->off_b1), h->Dp, h->y, ix, h->G2, P, B, Bp, C, Cp);
      return true;
    case KC_UPDATE1: {
      // With the small-C head, b1 took its step in k_head_b; the softmax
      // model's layer is the first and only one.
      if (!mlp) {
        UpdArgs u{h->G2, h->Cp, Bp, h->X, ix, h->INp, W + h->off_W1, h->Dp, h->INp, W + h->off_b1, P, B, Cp, INp,
                  h->hyper};
        with_momentum(h, u, h->off_W1, h->off_b1);
        launch_update(s, u, A_GATHER);
      } else {
        UpdArgs u{h->G1, h->Hp, Bp, h->X, ix, h->INp, W + h->off_W1, h->Dp, h->INp,
                  small ? nullptr : W + h->off_b1, P, B, Hp, INp, h->hyper};
        with_momentum(h, u, h->off_W1, h->off_b1);
        launch_update(s, u, A_GATHER);
      }
      return true;
    }
    case KC_STEP1:
    case KC_STEP1_MEAN: {
      const bool mean = kc == KC_STEP1_MEAN;
      if (!(mean ? h->fused_mean : h->fused) || tt + 1 >= h->T) return false;
      StepArgs a{};
      if (!mlp)
        a.u = UpdArgs{h->G2, h->Cp, Bp, h->X, ix, h->INp, W + h->off_W1, h->Dp, h->INp, W + h->off_b1, P, B, Cp, INp,
                      h->hyper};
      else
        a.u = UpdArgs{h->G1, h->Hp, Bp, h->X, ix, h->INp, W + h->off_W1, h->Dp, h->INp,
                      small ? nullptr : W + h->off_b1, P, B, Hp, INp, h->hyper};
      a.idx_next = ix + (int64_t)P * B;
      a.part = h->part;
      a.SG = mean ? S : 1;
      a.x_rows = h->N;
      if (!mean) old_w1(a);
      step(a);
      h->ks_cur = mean ? h->KS_mean : h->KS_step;
      return true;
    }
    case KC_UPD1_MEAN:
    case KC_UPD1_GLOBAL: {
      const bool global = kc == KC_UPD1_GLOBAL;
      // (the cluster form also ends an eager round whose means go to the copies)
      if (global ? !h->upd_global : !h->upd_mean || (tt + 1 >= h->T && !h->once_block)) return false;
      StepArgs a{};
      a.u = UpdArgs{h->G1, h->Hp, Bp, h->X, ix, h->INp, W + h->off_W1, h->Dp, h->INp,
                    small ? nullptr : W + h->off_b1, P, B, Hp, INp, h->hyper};
      a.SG = global ? P : S;
      a.no_fwd = true;
      a.x_rows = h->N;
      old_w1(a);
      if (global ? h->once_global : h->once_block) {
        a.w_dst = global ? h->Wg : h->Wc;
        a.dst_pitch = global ? 0 : w1;
      }
      step(a);
      return true;
    }
    case KC_FWD1_GROUP: {
      // Step tt's forward from each cluster's common first layer (every row of
      // the cluster holds it; row g*S is read): SG = S learners per GEMM.
      if (!h->upd_mean) return false;
      FwdArgs f{h->X, ix, h->INp, h->once_block ? h->Wc : W + h->off_W1, h->once_block ? w1 : (int64_t)S * h->Dp,
                h->INp, h->part, P, B, Bp, Hp, INp, h->KS_g, h->cps_g};
      f.SG = S;
      launch_fwd_blk(s, f);
      h->ks_cur = h->KS_g;
      return true;
    }
    case KC_TAIL_MEAN: launch_group_mean(s, W + h->off_b1, h->Dp, h->Dp - h->off_b1, P, S); return true;
    case KC_TAIL_GLOBAL: launch_group_mean(s, W + h->off_b1, h->Dp, h->Dp - h->off_b1, P, P); return true;
    case KC_GRAM:
      if (!h->delayed || h->gram == nullptr) return false;
      launch_gram(s, h->X, h->INp, INp, h->idx, h->gram, P, c.K1, c.K2, B, Bp, h->KSG);
      return true;
    case KC_GRAM_REDUCE:
      if (!h->delayed || h->gram == nullptr || h->KSG < 2) return false;
      launch_gram_reduce(s, h->gram, P, c.K1, c.K2, Bp, h->KSG);
      return true;
    case KC_FWD1_BLOCK: {
      if (!h->delayed) return false;
      // All K1 steps of block b at once: they read the block-start copy
      // (the round-start W1 in replica 0 for b = 0, else the cluster's copy);
      // partials go to part[ks][k][P][Bp][Hp].
      const int b = tt / c.K1;
      FwdArgs f{h->X, h->idx + (int64_t)b * c.K1 * P * B, h->INp, b == 0 ? W + h->off_W1 : wc_buf(h, b - 1),
                b == 0 ? 0 : h->Hp * h->INp, h->INp, h->part, P, B, Bp, Hp, INp, h->KS_b, h->cps_b};
      f.SG = c.K1 * S;
      f.vS = S;
      f.PT = c.K1 * P;
      launch_fwd_blk(s, f);
      h->ks_cur = h->KS_b;
      return true;
    }
    case KC_FWD1_BLOCK_V: {
      // Heavy-ball with momentum: X_k V^T of learner j's K1 steps from its own
      // buffer (groups of K1 members, the block's steps of one learner).
      if (!h->delayed || !h->hb || !h->V) return false;
      const int b = tt / c.K1;
      FwdArgs f{h->X, h->idx + (int64_t)b * c.K1 * P * B, h->INp, h->V + h->off_W1, h->Dp, h->INp, h->partv, P, B,
                Bp, Hp, INp, h->KSv, h->cpsv};
      f.SG = c.K1;
      f.vS = 1;
      f.PT = c.K1 * P;
      launch_fwd_blk(s, f);
      return true;
    }
    case KC_SCALE_ERRORS:
      if (!h->delayed || !h->hb) return false;
      launch_scale_errors(s, h->Gs, h->Gu, h->V ? h->Gt : nullptr, h->hyper, c.K1, (int64_t)P * Bp * Hp);
      return true;
    case KC_BUF_UPDATE: {
      // Heavy-ball with momentum, block end: each learner's buffer of W1,
      // v = r_K W_b + s_K v + sum_k t_{K-1-k} G_k^T X_k (its own rows).
      if (!h->delayed || !h->hb || !h->V) return false;
      const int b = tt / c.K1;
      const int64_t rp1 = round_up((int64_t)c.K1 * B, 32), blk1 = (int64_t)P * rp1;
      BlkArgs a{h->Gt, h->Hp, h->X, h->idx + (int64_t)b * c.K1 * P * B, h->INp,
                b == 0 ? W + h->off_W1 : wc_buf(h, b - 1), b == 0 ? 0 : w1, h->V + h->off_W1, h->Dp, h->INp, P, 1,
                c.K1, B, Bp, Hp, INp, h->hyper, 1.0f, h->btab1 + b * blk1, h->btab1 + (int64_t)c.K2 * blk1 + b * blk1};
      a.base_div = S;
      a.hb = h->hyper;
      a.hb_c1 = hb_index(HB_R, c.K1);
      a.hb_c2 = hb_index(HB_S, c.K1);
      a.B2 = h->V + h->off_W1;
      a.b2_pitch = h->Dp;
      a.b2_rows = 1;
      launch_block_update(s, a);
      return true;
    }
    case KC_BLOCK_UPDATE: {
      if (!h->delayed) return false;
      const int b = tt / c.K1;
      const int64_t rp = round_up((int64_t)c.K1 * S * B, 32), blk = (int64_t)(P / S) * rp;
      BlkArgs a{h->hb ? h->Gu : h->Gs, h->Hp, h->X, h->idx + (int64_t)b * c.K1 * P * B, h->INp,
                b == 0 ? W + h->off_W1 : wc_buf(h, b - 1), b == 0 ? 0 : w1, wc_buf(h, b), w1, h->INp, P, S, c.K1, B,
                Bp, Hp, INp, h->hyper, (float)S, h->btab + b * blk, h->btab + (int64_t)c.K2 * blk + b * blk};
      if (h->hb) {  // p_K W_b + q_K mean_j V_j + the errors scaled by u / S
        a.hb = h->hyper;
        a.hb_c1 = hb_index(HB_P, c.K1);
        a.hb_c2 = hb_index(HB_Q, c.K1);
        if (h->V) {
          a.B2 = h->V + h->off_W1;
          a.b2_pitch = h->Dp;
          a.b2_rows = S;
        }
      }
      if (b == c.K2 - 1 && h->global_last) {
        // The last block: one update over all P learners from the mean of the
        // cluster copies (the global mean of Algorithm 1, which skips the
        // cluster mean before it), into replica 0's W1, and the global mean
        // of b1, W2, b2.
        a.SG = P;
        a.lr_div = (float)P;
        a.nbase = b == 0 ? 1 : P / S;
        if (a.B2) a.b2_rows = P;
        a.Wo = W + h->off_W1;
        a.wo_pitch = 0;
        if (P > 1) {
          a.tail = W + h->off_b1;
          a.tail_pitch = h->Dp;
          a.tail_len = h->Dp - h->off_b1;
        }
      } else if (b < c.K2 - 1 && S > 1) {  // the block-end cluster mean of b1, W2, b2
        a.tail = W + h->off_b1;
        a.tail_pitch = h->Dp;
        a.tail_len = h->Dp - h->off_b1;
      }
      launch_block_update(s, a);
      return true;
    }
    case KC_W1_MEAN:  // with the global mean of b1, W2, b2 in the same launch
      if (!h->in_delayed) {  // eager, cluster copies: their mean into the common copy
        if (!h->once_block) return false;
        launch_mean_rows(s, h->Wg, h->Wc, w1, w1, P / S, W + h->off_b1, h->Dp, h->Dp - h->off_b1, P);
        return true;
      }
      launch_mean_rows(s, W + h->off_W1, wc_buf(h, c.K2 - 1), h->Hp * h->INp, h->Hp * h->INp, P / S,
                       P > 1 ? W + h->off_b1 : nullptr,
                       h->Dp, h->Dp - h->off_b1, P);
      return true;
    case KC_GROUP_MEAN: launch_group_mean(s, W, h->Dp, h->Dp, P, S); return true;
    case KC_GLOBAL_MEAN: launch_group_mean(s, W, h->Dp, h->Dp, P, P); return true;
    case KC_VMEAN_GROUP:
    case KC_VMEAN_GLOBAL:
      if (!h->V) return false;
      launch_group_mean(s, h->V, h->Dp, h->Dp, P, kc == KC_VMEAN_GROUP ? S : P);
      return true;
    default: break;
  }
  if (!mlp) return false;
  switch (kc) {
    case KC_HEAD_A:  // eager schedule (the delayed one runs KC_HEAD_STEP)
      if (!small || h->in_delayed) return false;
      launch_head_a(s, h->part, h->ks_cur, W + h->off_b1, W + h->off_W2, W + h->off_b2, h->Dp, h->Z1, h->PL, P, B,
                    Bp, C, Cp, Hp);
      return true;
    case KC_HEAD_B: {  // eager schedule
      if (!small || h->in_delayed) return false;
      HeadMom mom;
      mom.mu = c.momentum;
      mom.wd = c.weight_decay;
      if (h->V) {
        mom.vw2 = h->V + h->off_W2;
        mom.vb1 = h->V + h->off_b1;
        mom.vb2 = h->V + h->off_b2;
      }
      launch_head_b(s, h->PL, W + h->off_W2, W + h->off_b1, W + h->off_b2, h->Dp, h->Z1, h->G1, h->y, ix, P, B, Bp,
                    C, Cp, Hp, h->hyper, mom);
      return true;
    }
    case KC_HEAD_FUSED:
    case KC_HEAD_W2: {  // eager schedule
      if (!small || h->in_delayed || !h->head_fused) return false;
      HeadFusedArgs a;
      a.part = h->part;
      a.KS = h->ks_cur;
      a.split = (int64_t)P * Bp * Hp;
      a.b1 = W + h->off_b1;
      a.W2 = W + h->off_W2;
      a.b2 = W + h->off_b2;
      a.w_pitch = h->Dp;
      a.G1 = h->G1;
      a.labels = h->y;
      a.idx = ix;
      a.P = P;
      a.M = B;
      a.Mp = Bp;
      a.C = C;
      a.Cp = Cp;
      a.Hp = Hp;
      a.lr = h->hyper;
      a.mom.mu = c.momentum;
      a.mom.wd = c.weight_decay;
      if (h->V) {
        a.mom.vw2 = h->V + h->off_W2;
        a.mom.vb1 = h->V + h->off_b1;
        a.mom.vb2 = h->V + h->off_b2;
      }
      a.scratch = h->hgrad;
      if (kc == KC_HEAD_FUSED)
        launch_head_fused(s, a);
      else
        launch_head_w2_step(s, a);
      return true;
    }
    case KC_HEAD_STEP:
    case KC_HEAD_END: {
      if (!h->in_delayed) return false;
      // HEAD_STEP at step tt: backward of step tt-1 of the block (if any),
      // forward and output error of step tt; HEAD_END at a block's last step
      // tt: its backward.
      const int k = kc == KC_HEAD_END ? c.K1 : tt % c.K1;
      const int blk = tt / c.K1;
      HeadStepArgs a{};
      a.part = h->part;
      a.KS = h->ks_cur;
      a.split = (int64_t)c.K1 * P * Bp * Hp;
      a.W2 = W + h->off_W2;
      a.b1 = W + h->off_b1;
      a.b2 = W + h->off_b2;
      a.w_pitch = h->Dp;
      a.Z1 = h->Z1;
      a.PL = h->PL;
      a.pl_half = (int64_t)P * (Hp / 32) * Bp * Cp;
      a.gs = h->Gs;
      a.gram = h->gram ? h->gram + (int64_t)blk * P * c.K1 * c.K1 * Bp * Bp : nullptr;
      a.ylab = h->ylab + (int64_t)blk * c.K1 * P * B;
      a.lr = h->hyper;
      a.P = P;
      a.M = B;
      a.Mp = Bp;
      a.C = C;
      a.Cp = Cp;
      a.Hp = Hp;
      a.K1 = c.K1;
      if (h->hb) {  // heavy-ball blocks: coefficients, buffer partials, head buffers
        a.hb = h->hyper;
        a.partv = h->partv;
        a.KSv = h->KSv;
        a.splitv = (int64_t)c.K1 * P * Bp * Hp;
        a.mu = c.momentum;
        a.wd = c.weight_decay;
        if (h->V) {
          a.vw2 = h->V + h->off_W2;
          a.vb1 = h->V + h->off_b1;
          a.vb2 = h->V + h->off_b2;
        }
      }
      launch_head_step(s, a, k);
      return true;
    }
    case KC_REDUCE1:
      if (small) return false;
      launch_reduce_bias(s, h->part, h->ks_cur, W + h->off_b1, h->Dp, h->Z1, P, B, Bp, Hp);
      return true;
    case KC_FWD2: {
      if (small) return false;
      FwdArgs f{h->Z1, nullptr, h->Hp, W + h->off_W2, h->Dp, h->Hp, h->in_delayed ? h->part2 : h->part, P, B, Bp, Cp,
                Hp, h->KS2, h->cps2};
      launch_fwd(s, f, A_RELU);
      return true;
    }
    case KC_BWD_HIDDEN:
      if (small) return false;
      if (h->in_delayed)  // the hidden errors are kept for the block end; b1 takes its step here
        launch_bwd_hidden(s, h->G2, W + h->off_W2, h->Dp, h->Z1, h->Gs + (int64_t)(tt % c.K1) * P * Bp * Hp, P, B,
                          Bp, C, Cp, Hp, W + h->off_b1, h->hyper, h->hb && h->V ? h->V + h->off_b1 : nullptr,
                          h->hb ? c.momentum : 0.0f, h->hb ? c.weight_decay : 0.0f,
                          h->w2_fused ? W + h->off_b2 : nullptr);
      else if (h->w2_fused)
        launch_bwd_hidden(s, h->G2, W + h->off_W2, h->Dp, h->Z1, h->G1, P, B, Bp, C, Cp, Hp, nullptr, h->hyper,
                          nullptr, 0.0f, 0.0f, W + h->off_b2);
      else
        launch_bwd_hidden(s, h->G2, W + h->off_W2, h->Dp, h->Z1, h->G1, P, B, Bp, C, Cp, Hp);
      return true;
    case KC_Z1_DELAYED: {
      if (!h->in_delayed || small) return false;
      Z1Args a{};
      const int k = tt % c.K1;
      a.part = h->part + (int64_t)k * P * Bp * Hp;
      a.KS = h->ks_cur;
      a.split = (int64_t)c.K1 * P * Bp * Hp;
      a.b1 = W + h->off_b1;
      a.w_pitch = h->Dp;
      a.gs = h->Gs;
      a.gram = h->gram ? h->gram + (int64_t)(tt / c.K1) * P * c.K1 * c.K1 * Bp * Bp : nullptr;
      a.Z1 = h->Z1;
      a.lr = h->hyper;
      a.P = P;
      a.M = B;
      a.Mp = Bp;
      a.Hp = Hp;
      a.K1 = c.K1;
      a.k = k;
      if (h->hb) {
        a.hb = h->hyper;
        if (h->V) {
          a.partv = h->partv + (int64_t)k * P * Bp * Hp;
          a.KSv = h->KSv;
          a.splitv = (int64_t)c.K1 * P * Bp * Hp;
        }
      }
      launch_z1_delayed(s, a);
      return true;
    }
    case KC_UPDATE2: {
      if (small || h->w2_fused) return false;
      UpdArgs u{h->G2, h->Cp, Bp, h->Z1, nullptr, h->Hp, W + h->off_W2, h->Dp, h->Hp, W + h->off_b2, P, B, Cp, Hp,
                h->hyper};
      with_momentum(h, u, h->off_W2, h->off_b2);
      launch_update(s, u, A_RELU);
      return true;
    }
    default: return false;
  }
}

// One local SGD step of all P learners at step tt of the round (Algorithm 1:
// w <- w - lr/B * sum_s grad f(w; xi_s) for every learner concurrently),
// followed by the cluster mean when the step ends a block that is not the
// last one.  `have_fwd`: the first-layer forward partials of this step are
// already in `part` (computed by the previous step's fused kernel); on return
// it says the same of the next step.
void enqueue_step(hieravg* h, int tt, bool& have_fwd) {
  static const int kSoftmax[] = {KC_SOFTMAX};
  static const int kSmall[] = {KC_HEAD_A, KC_HEAD_B};
  static const int kSmallFused[] = {KC_HEAD_FUSED};
  static const int kLarge[] = {KC_REDUCE1, KC_FWD2, KC_SOFTMAX, KC_BWD_HIDDEN, KC_UPDATE2};
  const hieravg_config& c = h->cfg;
  const int* seq;
  int n;
  if (c.kind == HIERAVG_KIND_SOFTMAX) {
    seq = kSoftmax;
    n = 1;
  } else if (h->C <= kSmallC) {
    seq = h->head_fused ? kSmallFused : kSmall;
    n = h->head_fused ? 1 : 2;
  } else {
    seq = kLarge;
    n = h->w2_fused ? 4 : 5;  // KC_UPDATE2 last: the hidden-error kernel steps W2 and b2
  }
  auto go = [&](int kc) { run(h, kc, [&] { launch_class(h, kc, tt); }); };
  if (!have_fwd) go(KC_FWD1);
  for (int i = 0; i < n; ++i) go(seq[i]);
  // Small-C head: then the step of W2, b1, b2 from its gradient rows (on a
  // second stream beside the first-layer kernel below, which reads none of
  // them, the captured round was 0.13 ms slower on the 64-learner MLP).
  if (seq == kSmallFused) go(KC_HEAD_W2);
  const int T = h->T;
  const bool last = tt == T - 1;
  const bool mean = !last && (tt + 1) % c.K1 == 0 && c.S > 1;
  have_fwd = false;
  if (last && h->upd_global && h->once_block) {
    // the cluster means, once, to the copies, then their mean into the
    // common copy with the global mean of b1, W2, b2 (one group of P
    // learners per tile would leave the GPU half idle)
    go(KC_UPD1_MEAN);
    go(KC_W1_MEAN);
  } else if (last && h->upd_global) {  // with the global mean of every block
    go(KC_UPD1_GLOBAL);
    go(KC_TAIL_GLOBAL);
  } else if (last || !h->fused || (mean && !h->fused_mean && !h->upd_mean)) {
    go(KC_UPDATE1);
    if (mean) go(KC_GROUP_MEAN);
    if (mean && h->cfg.avg_momentum && h->V) go(KC_VMEAN_GROUP);
  } else if (mean && h->fused_mean) {
    go(KC_STEP1_MEAN);
    go(KC_TAIL_MEAN);
    have_fwd = true;
  } else if (mean) {
    go(KC_UPD1_MEAN);
    go(KC_TAIL_MEAN);
    run(h, KC_FWD1_GROUP, [&] { launch_class(h, KC_FWD1_GROUP, tt + 1); });
    have_fwd = true;
  } else {
    go(KC_STEP1);
    have_fwd = true;
  }
}

struct Segment {
  int64_t rows, cols, src_ld, src_off, dst_off;
};

std::vector<Segment> segments(const hieravg* h) {
  if (h->cfg.kind == HIERAVG_KIND_AVERAGING) return {{1, h->D, h->D, 0, 0}};
  if (h->cfg.kind == HIERAVG_KIND_SOFTMAX)
    return {{h->C, h->IN, h->INp, h->off_W1, 0}, {1, h->C, h->C, h->off_b1, h->C * h->IN}};
  const int64_t o1 = h->H * h->IN, o2 = o1 + h->H, o3 = o2 + h->C * h->H;
  return {{h->H, h->IN, h->INp, h->off_W1, 0},
          {1, h->H, h->H, h->off_b1, o1},
          {h->C, h->H, h->Hp, h->off_W2, o2},
          {1, h->C, h->C, h->off_b2, o3}};
}

}  // namespace

extern "C" {

const char* hieravg_last_error(void) { return g_last_error.c_str(); }

hieravg_t hieravg_create_config(const hieravg_config* cfg) {
  if (!cfg) {
    set_error("cfg is NULL");
    return nullptr;
  }
  if (validate(*cfg) != HIERAVG_OK) return nullptr;
  hieravg* h = new (std::nothrow) hieravg;
  if (!h) {
    set_error("out of host memory");
    return nullptr;
  }
  h->cfg = *cfg;
  h->fail_alloc = forced_alloc_failure();
  // Steps per round; K2 becomes the number of blocks (the last one shorter
  // when K1 does not divide k_global).
  h->T = cfg->k_global > 0 ? cfg->k_global : cfg->K1 * cfg->K2;
  h->cfg.k_global = h->T;
  h->cfg.K2 = (h->T + cfg->K1 - 1) / cfg->K1;
  if (build(h) != HIERAVG_OK) {
    std::string msg = g_last_error;
    release(h);
    set_error(msg);
    return nullptr;
  }
  g_last_error.clear();
  return h;
}

hieravg_t hieravg_create(int32_t P, int32_t S, int32_t K1, int32_t K2, int32_t model, float lr, int32_t B,
                         uint64_t seed) {
  hieravg_config c{};
  c.P = P;
  c.S = S;
  c.K1 = K1;
  c.K2 = K2;
  c.B = B;
  c.lr = lr;
  c.seed = seed;
  switch (model) {
    case HIERAVG_MODEL_SOFTMAX_3072_10:
      c.kind = HIERAVG_KIND_SOFTMAX;
      c.in_dim = 3072;
      c.classes = 10;
      c.n_samples = 2048;
      c.noise_std = 1.0f;
      break;
    case HIERAVG_MODEL_MLP_3072_512_10:
      c.kind = HIERAVG_KIND_MLP;
      c.in_dim = 3072;
      c.hidden = 512;
      c.classes = 10;
      c.n_samples = 50000;
      c.noise_std = 0.5f;
      break;
    case HIERAVG_MODEL_MLP_150528_1024_1000:
      c.kind = HIERAVG_KIND_MLP;
      c.in_dim = 150528;
      c.hidden = 1024;
      c.classes = 1000;
      c.n_samples = 100000;
      c.noise_std = 1.0f;
      break;
    case HIERAVG_MODEL_AVERAGING_11_7M:
      c.kind = HIERAVG_KIND_AVERAGING;
      c.in_dim = 11700000;
      c.momentum = 0.9f;
      c.init_std = 0.01f;
      c.grad_std = 0.01f;
      break;
    default:
      set_error("unknown model id " + std::to_string(model));
      return nullptr;
  }
  return hieravg_create_config(&c);
}

}  // extern "C"

namespace {

// Every kernel of one round, enqueued on the handle's stream.
void enqueue_round(hieravg* h) {
  const hieravg_config& c = h->cfg;
  const int T = h->T;
  const int P = c.P;
  if (c.kind == HIERAVG_KIND_AVERAGING) {
    // The first step reads every learner's parameters from Wm when the round
    // starts from a common value; the global mean writes Wm.
    for (int tt = 0; tt < T; ++tt) {
      const int kc = avg_step_mean(h, tt);
      const int lk = tt == 0 && h->in_shared ? KC_MOMENTUM_FIRST : kc;
      run(h, lk, [&] { launch_class(h, lk, tt); });
      if (c.avg_momentum && kc != KC_MOMENTUM) {
        const int vk = kc == KC_MOMENTUM_GLOBAL ? KC_VMEAN_GLOBAL : KC_VMEAN_GROUP;
        run(h, vk, [&] { launch_class(h, vk, tt); });
      }
    }
  } else if (h->in_delayed) {
    // Delayed first-layer updates: per block, the forward of its K1 steps
    // from the block-start copies, then per step the head (with the Gram
    // corrections of the earlier steps) and the hidden error, then one update
    // of each cluster's copy; at the end the global mean of the copies goes
    // to replica 0 (every learner's W1) and the other parameters take their
    // global mean.
    auto go = [&](int kc, int tt) { run(h, kc, [&] { launch_class(h, kc, tt); }); };
    go(KC_DRAW, 0);
    if (c.K1 > 1) {
      go(KC_GRAM, 0);
      if (h->KSG > 1) go(KC_GRAM_REDUCE, 0);
    }
    for (int b = 0; b < c.K2; ++b) {
      go(KC_FWD1_BLOCK, b * c.K1);
      if (h->hb && h->V) go(KC_FWD1_BLOCK_V, b * c.K1);  // heavy-ball: X_k V^T of every learner
      if (h->C <= kSmallC) {
        for (int k = 0; k < c.K1; ++k) go(KC_HEAD_STEP, b * c.K1 + k);
        go(KC_HEAD_END, b * c.K1 + c.K1 - 1);
      } else {  // more than 32 classes: the layer-2 GEMMs of the eager head, per step
        for (int k = 0; k < c.K1; ++k)
          for (int kc : {KC_Z1_DELAYED, KC_FWD2, KC_SOFTMAX, KC_BWD_HIDDEN, KC_UPDATE2})
            if (kc != KC_UPDATE2 || !h->w2_fused) go(kc, b * c.K1 + k);
      }
      if (h->hb) go(KC_SCALE_ERRORS, b * c.K1);
      // with the cluster mean of b1, W2, b2 for b < K2 - 1; the last block's
      // update takes the global mean of every block
      go(KC_BLOCK_UPDATE, b * c.K1);
      // heavy-ball with momentum: each learner's buffer, from the block-start
      // copies the update above left intact
      if (h->hb && h->V) go(KC_BUF_UPDATE, b * c.K1);
    }
    if (!h->global_last) go(KC_W1_MEAN, 0);  // with the global mean of b1, W2, b2
  } else {
    run(h, KC_DRAW, [&] { launch_class(h, KC_DRAW, 0); });
    bool have_fwd = false;
    for (int tt = 0; tt < T; ++tt) enqueue_step(h, tt, have_fwd);
    if (P > 1 && !h->upd_global) run(h, KC_GLOBAL_MEAN, [&] { launch_class(h, KC_GLOBAL_MEAN, 0); });
    if (P > 1 && c.avg_momentum && h->V) run(h, KC_VMEAN_GLOBAL, [&] { launch_class(h, KC_VMEAN_GLOBAL, 0); });
  }
}

// ------------------------------------------------------------ evaluation
constexpr int kEvalMaxChunk = 4096;  // rows per evaluation chunk

// Device buffers of one evaluation: a chunk of `rows` rows at a time.
struct EvalBufs {
  int rows = 0;
  int32_t* iota = nullptr;   // [rows] 0, 1, 2, ...
  float* part = nullptr;     // first-layer split-K partials, capacity part_cap floats
  int64_t part_cap = 0;
  float* Z1 = nullptr;       // [rows][Hp] (MLP)
  float* part2 = nullptr;    // logit split-K partials (MLP), capacity part2_cap floats
  int64_t part2_cap = 0;
  float* loss = nullptr;     // [rows]
  int32_t* hit = nullptr;    // [rows]
};

int eval_check(hieravg* h, int32_t replica, int32_t split, int64_t n_rows, const double* mean_loss,
               const int64_t* correct) {
  if (!h || !mean_loss || !correct) {
    set_error("NULL handle or output");
    return HIERAVG_EINVAL;
  }
  if (h->cfg.kind == HIERAVG_KIND_AVERAGING) {
    set_error("the averaging-only workload has no model to evaluate");
    return HIERAVG_EINVAL;
  }
  if (replica < 0 || replica >= h->cfg.P || (split != 0 && split != 1) || n_rows < 1 ||
      (split == 0 && n_rows > h->N) || n_rows > (int64_t(1) << 31)) {
    set_error("bad replica, split or row count (split 0 takes at most N rows)");
    return HIERAVG_EINVAL;
  }
  return HIERAVG_OK;
}

// Split count of a forward over one row group of Mp rows whose partials must
// fit in `cap` floats (cap >= Mp * N).
void split_within(int Mp, int N, int K, int64_t cap, int* KS, int* cps) {
  plan_split(1, Mp, N, K, KS, cps);
  const int nch = K / 64;
  const int64_t ks_max = std::max<int64_t>(1, cap / ((int64_t)Mp * N));
  if (*KS > ks_max) {
    const int c = (int)((nch + ks_max - 1) / ks_max);
    *cps = c;
    *KS = (nch + c - 1) / c;
  }
}

// Loss and hits of rows 0 .. n_rows-1 of a split, chunk by chunk: the forward
// kernels of the round (first layer from the dataset rows, split-K partials),
// then per row the softmax cross-entropy at the label and the first argmax;
// the host adds the per-row values in double.
int eval_chunks(hieravg* h, const EvalBufs& b, int replica, int split, int64_t n_rows, double* mean_loss,
                int64_t* correct) {
  const bool mlp = h->cfg.kind == HIERAVG_KIND_MLP;
  const int Hp = (int)h->Hp, Cp = (int)h->Cp, INp = (int)h->INp, C = (int)h->C;
  const int n1 = mlp ? Hp : Cp;
  hipStream_t s = h->stream;
  const float* Xs = split == 0 ? h->X : h->Xtest;
  const int32_t* ys = split == 0 ? h->y : h->ytest;
  // Replica `replica`; its first weight block lives in replica 0 while the
  // learners share it under delayed updates.
  const float* Wr = h->W + (int64_t)replica * h->Dp;
  const float* W1r = h->rows_stale ? (h->w1_wg ? h->Wg : h->W + h->off_W1) : Wr + h->off_W1;
  double total = 0.0;
  int64_t hits = 0;
  float lh[kEvalMaxChunk];
  int32_t hh[kEvalMaxChunk];
  for (int64_t r0 = 0; r0 < n_rows; r0 += b.rows) {
    const int M = (int)std::min<int64_t>(b.rows, n_rows - r0);
    const int Mp = (int)round_up(M, 16);
    int KS1, cps1;
    split_within(Mp, n1, INp, b.part_cap, &KS1, &cps1);
    FwdArgs f{Xs + r0 * h->INp, b.iota, h->INp, W1r, 0, h->INp, b.part, 1, M, Mp, n1, INp, KS1, cps1};
    launch_fwd(s, f, A_GATHER);
    if (mlp) {
      launch_reduce_bias(s, b.part, KS1, Wr + h->off_b1, 0, b.Z1, 1, M, Mp, Hp);
      int KS2, cps2;
      split_within(Mp, Cp, Hp, b.part2_cap, &KS2, &cps2);
      FwdArgs f2{b.Z1, nullptr, h->Hp, Wr + h->off_W2, 0, h->Hp, b.part2, 1, M, Mp, Cp, Hp, KS2, cps2};
      launch_fwd(s, f2, A_RELU);
      launch_eval_rows(s, b.part2, KS2, (int64_t)Mp * Cp, Wr + h->off_b2, ys + r0, M, Cp, C, b.loss, b.hit);
    } else {
      launch_eval_rows(s, b.part, KS1, (int64_t)Mp * Cp, Wr + h->off_b1, ys + r0, M, Cp, C, b.loss, b.hit);
    }
    HAV_CHECK(hipGetLastError());
    HAV_CHECK(hipMemcpyAsync(lh, b.loss, sizeof(float) * M, hipMemcpyDeviceToHost, s));
    HAV_CHECK(hipMemcpyAsync(hh, b.hit, sizeof(int32_t) * M, hipMemcpyDeviceToHost, s));
    HAV_CHECK(hipStreamSynchronize(s));
    for (int i = 0; i < M; ++i) {
      total += lh[i];
      hits += hh[i];
    }
  }
  *mean_loss = total / (double)n_rows;
  *correct = hits;
  return HIERAVG_OK;
}

// The device scratch array of hieravg_evaluate_noalloc: one per GPU (a
// file-scope device array exists once on every device the library runs on),
// kept until the process ends.  Host code never passes `scratch` itself to a
// kernel (on the host it names a stand-in, not device memory): it looks up
// the array's device address once per device and uses that.
constexpr int64_t kScratchFloats = HIERAVG_EVAL_SCRATCH_BYTES / sizeof(float);
static __device__ __align__(256) float scratch[kScratchFloats];

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
float* g_scratch_ptr[kMaxDevices] = {};

// The device address of `scratch` on device `dev` (the current device).
int scratch_on_device(int dev, float** out) {
  if (dev < 0 || dev >= kMaxDevices) {
    set_error("device id out of the range of the scratch table");
    return HIERAVG_EINVAL;
  }
  std::lock_guard<std::mutex> lk(g_scratch_mu);
  if (!g_scratch_ptr[dev]) {
    void* p = nullptr;
    const hipError_t e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess || !p) {
      set_error(std::string("hipGetSymbolAddress of the evaluation scratch failed: ") + hipGetErrorString(e));
      return HIERAVG_EHIP;
    }
    g_scratch_ptr[dev] = (float*)p;
  }
  *out = g_scratch_ptr[dev];
  return HIERAVG_OK;
}

// Makes `dev` current for a scope and restores the caller's device.
struct DeviceGuard {
  int prev = -1;
  int enter(int dev) {
    if (hipGetDevice(&prev) != hipSuccess) {
      prev = -1;
      set_error("hipGetDevice failed");
      return HIERAVG_EHIP;
    }
    if (prev != dev && hipSetDevice(dev) != hipSuccess) {
      set_error("hipSetDevice to the handle's device failed");
      return HIERAVG_EHIP;
    }
    return HIERAVG_OK;
  }
  ~DeviceGuard() {
    if (prev >= 0) (void)hipSetDevice(prev);
  }
};

// Largest chunk (rows, a multiple of 16 up to kEvalMaxChunk) whose buffers fit
// in the scratch array with one split each, and the partial capacities.
int eval_scratch_plan(const hieravg* h, int* rows, int64_t* part_cap, int64_t* part2_cap) {
  const bool mlp = h->cfg.kind == HIERAVG_KIND_MLP;
  const int64_t n1 = mlp ? h->Hp : h->Cp;
  for (int r = kEvalMaxChunk; r >= 16; r /= 2) {
    const int64_t fixed = 3 * round_up(r, 64) + (mlp ? round_up((int64_t)r * h->Hp, 64) : 0);
    int64_t p2 = 0;
    if (mlp) {
      int KS2, cps2;
      plan_split(1, r, (int)h->Cp, (int)h->Hp, &KS2, &cps2);
      p2 = round_up((int64_t)KS2 * r * h->Cp, 64);
      if (fixed + p2 + r * n1 > kScratchFloats) p2 = round_up((int64_t)r * h->Cp, 64);
    }
    const int64_t left = kScratchFloats - fixed - p2;
    if (left >= r * n1) {
      *rows = r;
      *part_cap = left;
      *part2_cap = p2;
      return HIERAVG_OK;
    }
  }
  const int64_t need = 4 * (3 * 64 + 16 * n1 + (mlp ? 16 * (h->Hp + h->Cp) : 0));
  set_error("hieravg_evaluate_noalloc: a 16-row chunk of this model needs " + std::to_string(need) +
            " bytes of scratch, more than its " + std::to_string((long long)HIERAVG_EVAL_SCRATCH_BYTES));
  return HIERAVG_ESIZE;
}

}  // namespace

extern "C" {

int hieravg_round(hieravg_t h) {
  if (!h) {
    set_error("NULL handle");
    return HIERAVG_EINVAL;
  }
  const bool avg = h->cfg.kind == HIERAVG_KIND_AVERAGING;
  // Delayed updates need every learner to start the round from replica 0's
  // W1; the averaging kind starts from Wm when the learners share it.
  h->in_delayed = h->delayed && h->w1_shared;
  h->in_shared = avg && h->w1_shared;
  h->in_wg = !avg && !h->in_delayed && h->once_global && h->rows_stale && h->w1_wg;
  if (!avg && h->rows_stale && h->w1_wg && !h->in_wg) {
    // Every learner's W1 is Wg: a delayed round reads it in replica 0, any
    // other eager round in every row.
    const size_t w1 = sizeof(float) * h->Hp * h->INp;
    for (int p = 0; p < (h->in_delayed ? 1 : h->cfg.P); ++p)
      HAV_CHECK(hipMemcpyAsync(h->W + (int64_t)p * h->Dp + h->off_W1, h->Wg, w1, hipMemcpyDeviceToDevice,
                               h->stream));
    h->w1_wg = false;
    h->rows_stale = h->in_delayed;
  }
  if (!avg && !h->in_delayed && h->rows_stale && !h->in_wg) {
    // An eager round reads every replica's W1: copy replica 0's to the others.
    const size_t w1 = sizeof(float) * h->Hp * h->INp;
    for (int p = 1; p < h->cfg.P; ++p)
      HAV_CHECK(hipMemcpyAsync(h->W + (int64_t)p * h->Dp + h->off_W1, h->W + h->off_W1, w1,
                               hipMemcpyDeviceToDevice, h->stream));
    h->rows_stale = false;
  }
  h->launch_failed = false;
  const char* refused = "a step launch of the round's plan was refused (internal error)";
  if (h->profiling) {
    enqueue_round(h);
  } else {
    hipGraphExec_t& exec = h->round_exec[h->in_delayed || h->in_shared ? 1 : h->in_wg ? 2 : 0];
    if (!exec) {
      HAV_CHECK(hipStreamBeginCapture(h->stream, hipStreamCaptureModeThreadLocal));
      enqueue_round(h);
      hipGraph_t graph = nullptr;
      HAV_CHECK(hipStreamEndCapture(h->stream, &graph));
      if (h->launch_failed) {
        (void)hipGraphDestroy(graph);
        set_error(refused);
        return HIERAVG_EINVAL;
      }
      const hipError_t e = hipGraphInstantiate(&exec, graph, nullptr, nullptr, 0);
      (void)hipGraphDestroy(graph);
      if (e != hipSuccess) {
        exec = nullptr;
        set_error(std::string("hipGraphInstantiate of the round failed: ") + hipGetErrorString(e));
        return HIERAVG_EHIP;
      }
    }
    HAV_CHECK(hipGraphLaunch(exec, h->stream));
  }
  HAV_CHECK(hipGetLastError());
  if (h->launch_failed) {
    set_error(refused);
    return HIERAVG_EINVAL;
  }
  // After the global mean every learner holds replica 0's W1 (under delayed
  // updates only replica 0's copy is written); averaging kind: Wm holds every
  // learner's parameters (with P = 1 the round's last step writes row 0).
  if (avg && h->cfg.P > 1) {
    h->rows_stale = true;
  } else if (avg) {
    HAV_CHECK(hipMemcpyAsync(h->Wm, h->W, sizeof(float) * h->Dp, hipMemcpyDeviceToDevice, h->stream));
  }
  h->w1_shared = true;
  if (h->in_delayed) h->rows_stale = true;
  if (!avg && !h->in_delayed && h->once_global) {  // the global mean of W1 went to Wg only
    h->rows_stale = true;
    h->w1_wg = true;
  }
  h->steps += h->T;
  return HIERAVG_OK;
}

int hieravg_set_batch(hieravg_t h, int32_t B) {
  if (!h) {
    set_error("NULL handle");
    return HIERAVG_EINVAL;
  }
  if (h->cfg.kind == HIERAVG_KIND_AVERAGING) {
    set_error("the averaging-only workload has no minibatch");
    return HIERAVG_EINVAL;
  }
  if (B < 1 || B > h->Bmax) {
    set_error("B must be in [1, the minibatch size given at create]");
    return HIERAVG_EINVAL;
  }
  HAV_CHECK(hipStreamSynchronize(h->stream));
  h->cfg.B = B;
  plan(h, B);
  // The captured rounds carry the old launch shapes.
  for (auto& e : h->round_exec)
    if (e) {
      (void)hipGraphExecDestroy(e);
      e = nullptr;
    }
  return HIERAVG_OK;
}

int hieravg_set_lr(hieravg_t h, float lr) {
  if (!h) {
    set_error("NULL handle");
    return HIERAVG_EINVAL;
  }
  if (!std::isfinite(lr) || lr < 0.0f) {
    set_error("lr must be finite and >= 0");
    return HIERAVG_EINVAL;
  }
  h->cfg.lr = lr;
  HAV_CHECK(hipStreamSynchronize(h->stream));
  HAV_CHECK(write_hyper(h));  // the step size and the heavy-ball coefficients
  return HIERAVG_OK;
}

int hieravg_evaluate(hieravg_t h, int32_t replica, int32_t split, int64_t n_rows, double* mean_loss,
                     int64_t* correct) {
  int rc = eval_check(h, replica, split, n_rows, mean_loss, correct);
  if (rc != HIERAVG_OK) return rc;
  const hieravg_config& c = h->cfg;
  const bool mlp = c.kind == HIERAVG_KIND_MLP;
  const int Hp = (int)h->Hp, Cp = (int)h->Cp, INp = (int)h->INp, C = (int)h->C;
  hipStream_t s = h->stream;
  HAV_CHECK(hipStreamSynchronize(s));
  // Buffers for chunks of up to kEvalMaxChunk rows.
  const int chunk = (int)std::min<int64_t>(kEvalMaxChunk, round_up(n_rows, 16));
  // Partials for the split counts of a full chunk (a shorter last chunk
  // takes at most as many floats: split_within caps its splits).
  int ks1, ks2 = 1, cps;
  plan_split(1, chunk, mlp ? Hp : Cp, INp, &ks1, &cps);
  if (mlp) plan_split(1, chunk, Cp, Hp, &ks2, &cps);
  if (chunk > h->eval_rows) {
    void* old[] = {h->eval_iota, h->eval_part, h->eval_part2, h->eval_Z1, h->eval_loss, h->eval_hit};
    for (void* b : old)
      if (b) (void)hipFree(b);
    h->eval_iota = nullptr;
    h->eval_part = h->eval_part2 = h->eval_Z1 = h->eval_loss = nullptr;
    h->eval_hit = nullptr;
    h->eval_rows = 0;
    if ((rc = alloc_zero(h, (void**)&h->eval_iota, sizeof(int32_t) * chunk, "evaluation rows")) ||
        (rc = alloc_zero(h, (void**)&h->eval_part, sizeof(float) * ks1 * chunk * (mlp ? Hp : Cp), "evaluation partials")) ||
        (rc = alloc_zero(h, (void**)&h->eval_loss, sizeof(float) * chunk, "evaluation losses")) ||
        (rc = alloc_zero(h, (void**)&h->eval_hit, sizeof(int32_t) * chunk, "evaluation hits")))
      return rc;
    if (mlp && ((rc = alloc_zero(h, (void**)&h->eval_part2, sizeof(float) * ks2 * chunk * Cp, "evaluation logits")) ||
                (rc = alloc_zero(h, (void**)&h->eval_Z1, sizeof(float) * chunk * Hp, "evaluation activations"))))
      return rc;
    launch_iota(s, h->eval_iota, chunk);
    HAV_CHECK(hipGetLastError());
    HAV_CHECK(hipStreamSynchronize(s));
    h->eval_rows = chunk;
    h->eval_part_cap = (int64_t)ks1 * chunk * (mlp ? Hp : Cp);
    h->eval_part2_cap = mlp ? (int64_t)ks2 * chunk * Cp : 0;
  }
  // Held-out rows: the dataset recipe with its own label and noise streams.
  if (split == 1 && n_rows > h->n_test) {
    if (h->Xtest) (void)hipFree(h->Xtest);
    if (h->ytest) (void)hipFree(h->ytest);
    h->Xtest = nullptr;
    h->ytest = nullptr;
    h->n_test = 0;
    if ((rc = alloc_zero(h, (void**)&h->Xtest, sizeof(float) * n_rows * h->INp, "held-out rows")) ||
        (rc = alloc_zero(h, (void**)&h->ytest, sizeof(int32_t) * n_rows, "held-out labels")))
      return rc;
    launch_gen_labels(s, h->ytest, n_rows, hash64(c.seed, kTagTestLabel), (uint64_t)C);
    launch_gen_data(s, h->Xtest, h->ytest, n_rows, h->IN, h->INp, hash64(c.seed, kTagMean),
                    hash64(c.seed, kTagTestNoise), c.noise_std);
    HAV_CHECK(hipGetLastError());
    h->n_test = n_rows;
  }
  EvalBufs b;
  b.rows = chunk;
  b.iota = h->eval_iota;
  b.part = h->eval_part;
  b.part_cap = h->eval_part_cap;
  b.Z1 = h->eval_Z1;
  b.part2 = h->eval_part2;
  b.part2_cap = h->eval_part2_cap;
  b.loss = h->eval_loss;
  b.hit = h->eval_hit;
  return eval_chunks(h, b, replica, split, n_rows, mean_loss, correct);
}

int hieravg_evaluate_noalloc(hieravg_t h, int32_t replica, int32_t split, int64_t n_rows, double* mean_loss,
                             int64_t* correct) {
  int rc = eval_check(h, replica, split, n_rows, mean_loss, correct);
  if (rc != HIERAVG_OK) return rc;
  if (split == 1 && n_rows > h->n_test) {
    set_error("hieravg_evaluate_noalloc: the held-out rows are generated (and allocated) by hieravg_evaluate; " +
              std::to_string(h->n_test) + " exist, " + std::to_string(n_rows) + " requested");
    return HIERAVG_ESIZE;
  }
  EvalBufs b;
  if ((rc = eval_scratch_plan(h, &b.rows, &b.part_cap, &b.part2_cap)) != HIERAVG_OK) return rc;
  DeviceGuard dg;
  if ((rc = dg.enter(h->device)) != HIERAVG_OK) return rc;
  float* base = nullptr;
  if ((rc = scratch_on_device(h->device, &base)) != HIERAVG_OK) return rc;
  // Regions of the scratch array (offsets in floats, each a multiple of 64).
  const bool mlp = h->cfg.kind == HIERAVG_KIND_MLP;
  const int64_t rows64 = round_up(b.rows, 64);
  int64_t off = 0;
  b.iota = (int32_t*)(base + off);
  off += rows64;
  b.loss = base + off;
  off += rows64;
  b.hit = (int32_t*)(base + off);
  off += rows64;
  b.Z1 = mlp ? base + off : nullptr;
  off += mlp ? round_up((int64_t)b.rows * h->Hp, 64) : 0;
  b.part2 = mlp ? base + off : nullptr;
  off += mlp ? round_up(b.part2_cap, 64) : 0;
  b.part = base + off;
  HAV_CHECK(hipStreamSynchronize(h->stream));
  launch_iota(h->stream, b.iota, b.rows);
  HAV_CHECK(hipGetLastError());
  return eval_chunks(h, b, replica, split, n_rows, mean_loss, correct);
}

int hieravg_params(hieravg_t h, float* dst, size_t n_floats) {
  if (!h || !dst) {
    set_error("NULL handle or destination");
    return HIERAVG_EINVAL;
  }
  const int P = h->cfg.P;
  if (n_floats < (size_t)P * (size_t)h->D) {
    set_error("destination holds " + std::to_string(n_floats) + " floats, need P*D = " +
              std::to_string((int64_t)P * h->D));
    return HIERAVG_ESIZE;
  }
  HAV_CHECK(hipStreamSynchronize(h->stream));
  const std::vector<Segment> segs = segments(h);
  for (int p = 0; p < P; ++p)
    for (size_t i = 0; i < segs.size(); ++i) {
      const Segment& g = segs[i];
      // After delayed updates only replica 0 holds the (common) W1; after an
      // averaging-kind round Wm holds every learner's parameters.
      const float* src = h->W + (int64_t)p * h->Dp;
      if (i == 0 && h->rows_stale) src = h->cfg.kind == HIERAVG_KIND_AVERAGING ? h->Wm : h->w1_wg ? h->Wg : h->W;
      HAV_CHECK(hipMemcpy2DAsync(dst + (int64_t)p * h->D + g.dst_off, sizeof(float) * g.cols, src + g.src_off,
                                 sizeof(float) * g.src_ld, sizeof(float) * g.cols, g.rows, hipMemcpyDefault,
                                 h->stream));
    }
  HAV_CHECK(hipStreamSynchronize(h->stream));
  return HIERAVG_OK;
}

int hieravg_set_params(hieravg_t h, const float* src, size_t n_floats) {
  if (!h || !src) {
    set_error("NULL handle or source");
    return HIERAVG_EINVAL;
  }
  const int P = h->cfg.P;
  if (n_floats < (size_t)P * (size_t)h->D) {
    set_error("source holds fewer than P*D floats");
    return HIERAVG_ESIZE;
  }
  HAV_CHECK(hipStreamSynchronize(h->stream));
  for (int p = 0; p < P; ++p)
    for (const Segment& g : segments(h))
      HAV_CHECK(hipMemcpy2DAsync(h->W + (int64_t)p * h->Dp + g.src_off, sizeof(float) * g.src_ld,
                                 src + (int64_t)p * h->D + g.dst_off, sizeof(float) * g.cols,
                                 sizeof(float) * g.cols, g.rows, hipMemcpyDefault, h->stream));
  h->w1_shared = false;  // unless every row's W1 equals row 0's (a round-boundary checkpoint)
  h->rows_stale = false;
  h->w1_wg = false;
  const bool avg = h->cfg.kind == HIERAVG_KIND_AVERAGING;
  if (h->cfg.kind == HIERAVG_KIND_MLP || avg) {
    // MLP: equal W1 rows allow delayed updates; averaging kind: equal rows
    // let the next round start from Wm.
    if (!h->flag) HAV_CHECK(hipMalloc((void**)&h->flag, sizeof(int)));
    HAV_CHECK(hipMemsetAsync(h->flag, 0, sizeof(int), h->stream));
    launch_rows_differ(h->stream, h->W + h->off_W1, h->Dp, avg ? h->Dp : h->Hp * h->INp, P, h->flag);
    HAV_CHECK(hipGetLastError());
    int differ = 0;
    HAV_CHECK(hipMemcpyAsync(&differ, h->flag, sizeof(int), hipMemcpyDeviceToHost, h->stream));
    HAV_CHECK(hipStreamSynchronize(h->stream));
    h->w1_shared = differ == 0;
    if (avg && h->w1_shared)
      HAV_CHECK(hipMemcpyAsync(h->Wm, h->W, sizeof(float) * h->Dp, hipMemcpyDeviceToDevice, h->stream));
    // Equal rows where eager rounds write the global mean of W1 once: the
    // state such a round leaves, so the next round starts from the common
    // copy as it would have (the same launches and rounding: checkpoints at
    // a round boundary resume exactly).
    if (!avg && h->w1_shared && h->once_global) {
      HAV_CHECK(hipMemcpyAsync(h->Wg, h->W + h->off_W1, sizeof(float) * h->Hp * h->INp, hipMemcpyDeviceToDevice,
                               h->stream));
      h->rows_stale = true;
      h->w1_wg = true;
    }
  }
  HAV_CHECK(hipStreamSynchronize(h->stream));
  return HIERAVG_OK;
}

int hieravg_momentum(hieravg_t h, float* dst, size_t n_floats) {
  if (!h || !dst) {
    set_error("NULL handle or destination");
    return HIERAVG_EINVAL;
  }
  if (!h->V) {
    set_error("no momentum buffers (momentum is 0)");
    return HIERAVG_EINVAL;
  }
  const int P = h->cfg.P;
  if (n_floats < (size_t)P * (size_t)h->D) {
    set_error("destination holds fewer than P*D floats");
    return HIERAVG_ESIZE;
  }
  HAV_CHECK(hipStreamSynchronize(h->stream));
  for (int p = 0; p < P; ++p)
    for (const Segment& g : segments(h))
      HAV_CHECK(hipMemcpy2DAsync(dst + (int64_t)p * h->D + g.dst_off, sizeof(float) * g.cols,
                                 h->V + (int64_t)p * h->Dp + g.src_off, sizeof(float) * g.src_ld,
                                 sizeof(float) * g.cols, g.rows, hipMemcpyDefault, h->stream));
  HAV_CHECK(hipStreamSynchronize(h->stream));
  return HIERAVG_OK;
}

int hieravg_set_momentum(hieravg_t h, const float* src, size_t n_floats) {
  if (!h || !src) {
    set_error("NULL handle or source");
    return HIERAVG_EINVAL;
  }
  if (!h->V) {
    set_error("no momentum buffers (momentum is 0)");
    return HIERAVG_EINVAL;
  }
  const int P = h->cfg.P;
  if (n_floats < (size_t)P * (size_t)h->D) {
    set_error("source holds fewer than P*D floats");
    return HIERAVG_ESIZE;
  }
  HAV_CHECK(hipStreamSynchronize(h->stream));
  for (int p = 0; p < P; ++p)
    for (const Segment& g : segments(h))
      HAV_CHECK(hipMemcpy2DAsync(h->V + (int64_t)p * h->Dp + g.src_off, sizeof(float) * g.src_ld,
                                 src + (int64_t)p * h->D + g.dst_off, sizeof(float) * g.cols,
                                 sizeof(float) * g.cols, g.rows, hipMemcpyDefault, h->stream));
  HAV_CHECK(hipStreamSynchronize(h->stream));
  return HIERAVG_OK;
}

void hieravg_destroy(hieravg_t h) { release(h); }

int64_t hieravg_dim(hieravg_t h) {
  if (!h) {
    set_error("NULL handle");
    return HIERAVG_EINVAL;
  }
  return h->D;
}

int hieravg_check_finite(hieravg_t h) {
  if (!h) {
    set_error("NULL handle");
    return HIERAVG_EINVAL;
  }
  if (!h->flag) HAV_CHECK(hipMalloc((void**)&h->flag, sizeof(int)));
  HAV_CHECK(hipMemsetAsync(h->flag, 0, sizeof(int), h->stream));
  // After a round every learner's parameters are replica 0's (Wm for the
  // averaging kind); the other rows may hold older values.
  if (h->rows_stale && h->w1_wg) {
    launch_any_nonfinite(h->stream, h->Wg, h->Hp * h->INp, h->flag);
    launch_any_nonfinite(h->stream, h->W + h->off_b1, h->Dp - h->off_b1, h->flag);
  } else if (h->rows_stale)
    launch_any_nonfinite(h->stream, h->cfg.kind == HIERAVG_KIND_AVERAGING ? h->Wm : h->W, h->Dp, h->flag);
  else
    launch_any_nonfinite(h->stream, h->W, (int64_t)h->cfg.P * h->Dp, h->flag);
  HAV_CHECK(hipGetLastError());
  int bad = 0;
  HAV_CHECK(hipMemcpyAsync(&bad, h->flag, sizeof(int), hipMemcpyDeviceToHost, h->stream));
  HAV_CHECK(hipStreamSynchronize(h->stream));
  if (bad) {
    set_error("a replica holds inf or NaN");
    return HIERAVG_ENONFINITE;
  }
  return HIERAVG_OK;
}

int hieravg_set_step_count(hieravg_t h, int64_t t) {
  if (!h) {
    set_error("NULL handle");
    return HIERAVG_EINVAL;
  }
  if (t < 0) {
    set_error("the step count must be >= 0");
    return HIERAVG_EINVAL;
  }
  HAV_CHECK(hipStreamSynchronize(h->stream));
  const uint64_t v[2] = {(uint64_t)t, 0};
  HAV_CHECK(hipMemcpy(h->ctr, v, sizeof(v), hipMemcpyHostToDevice));
  h->steps = t;
  return HIERAVG_OK;
}

int64_t hieravg_step_count(hieravg_t h) {
  if (!h) {
    set_error("NULL handle");
    return HIERAVG_EINVAL;
  }
  return h->steps;
}

int hieravg_last_indices(hieravg_t h, int32_t* dst, size_t n) {
  if (!h || !dst) {
    set_error("NULL handle or destination");
    return HIERAVG_EINVAL;
  }
  if (h->cfg.kind == HIERAVG_KIND_AVERAGING) {
    set_error("the averaging-only workload draws no samples");
    return HIERAVG_EINVAL;
  }
  const size_t need = (size_t)h->T * h->cfg.P * h->cfg.B;
  if (n < need) {
    set_error("destination holds fewer than T*P*B indices");
    return HIERAVG_ESIZE;
  }
  HAV_CHECK(hipStreamSynchronize(h->stream));
  HAV_CHECK(hipMemcpy(dst, h->idx, need * sizeof(int32_t), hipMemcpyDefault));
  return HIERAVG_OK;
}

int hieravg_set_stream(hieravg_t h, void* hip_stream) {
  if (!h) {
    set_error("NULL handle");
    return HIERAVG_EINVAL;
  }
  HAV_CHECK(hipStreamSynchronize(h->stream));
  h->stream = hip_stream ? (hipStream_t)hip_stream : h->own_stream;
  return HIERAVG_OK;
}

int hieravg_sync(hieravg_t h) {
  if (!h) {
    set_error("NULL handle");
    return HIERAVG_EINVAL;
  }
  HAV_CHECK(hipStreamSynchronize(h->stream));
  return HIERAVG_OK;
}

int hieravg_profile(hieravg_t h, int enable) {
  if (!h) {
    set_error("NULL handle");
    return HIERAVG_EINVAL;
  }
  HAV_CHECK(hipStreamSynchronize(h->stream));
  for (auto& r : h->recs) {
    h->pool.push_back(r.a);
    h->pool.push_back(r.b);
  }
  h->recs.clear();
  h->profiling = enable != 0;
  return HIERAVG_OK;
}

int hieravg_profile_read(hieravg_t h, int64_t* launches, double* total_ms, int n) {
  if (!h || !launches || !total_ms || n < 0) {
    set_error("bad arguments");
    return HIERAVG_EINVAL;
  }
  HAV_CHECK(hipStreamSynchronize(h->stream));
  for (int i = 0; i < n; ++i) {
    launches[i] = 0;
    total_ms[i] = 0.0;
  }
  for (auto& r : h->recs) {
    float ms = 0.0f;
    HAV_CHECK(hipEventElapsedTime(&ms, r.a, r.b));
    if (r.kc < n) {
      launches[r.kc] += 1;
      total_ms[r.kc] += ms;
    }
  }
  return HIERAVG_OK;
}

int hieravg_time_kernel(hieravg_t h, int kernel_class, int reps, double* mean_ms) {
  if (!h || !mean_ms || reps < 1 || reps > 100000 || kernel_class < 0 || kernel_class >= KC_COUNT ||
      kernel_class == KC_DRAW) {
    set_error("bad arguments");
    return HIERAVG_EINVAL;
  }
  if (h->profiling) {
    set_error("disable hieravg_profile first");
    return HIERAVG_EINVAL;
  }
  // The launches are captured into a graph (kernel nodes only) and the graph
  // is launched once between the two events, so the host's per-launch cost
  // stays out of the timed interval.
  HAV_CHECK(hipStreamSynchronize(h->stream));
  HAV_CHECK(hipStreamBeginCapture(h->stream, hipStreamCaptureModeThreadLocal));
  bool ok = true;
  for (int i = 0; i < reps && ok; ++i) ok = launch_class(h, kernel_class, 0);
  hipGraph_t graph = nullptr;
  HAV_CHECK(hipStreamEndCapture(h->stream, &graph));
  if (!ok) {
    (void)hipGraphDestroy(graph);
    set_error("this workload does not launch that kernel class");
    return HIERAVG_EINVAL;
  }
  hipGraphExec_t exec = nullptr;
  hipEvent_t a = nullptr, b = nullptr;
  int rc = HIERAVG_OK;
  if (hipGraphInstantiate(&exec, graph, nullptr, nullptr, 0) != hipSuccess) rc = HIERAVG_EHIP;
  if (rc == HIERAVG_OK && (hipEventCreate(&a) != hipSuccess || hipEventCreate(&b) != hipSuccess)) rc = HIERAVG_EHIP;
  if (rc == HIERAVG_OK && hipEventRecord(a, h->stream) != hipSuccess) rc = HIERAVG_EHIP;
  if (rc == HIERAVG_OK && hipGraphLaunch(exec, h->stream) != hipSuccess) rc = HIERAVG_EHIP;
  if (rc == HIERAVG_OK && hipEventRecord(b, h->stream) != hipSuccess) rc = HIERAVG_EHIP;
  if (rc == HIERAVG_OK && hipEventSynchronize(b) != hipSuccess) rc = HIERAVG_EHIP;
  float ms = 0.0f;
  if (rc == HIERAVG_OK && hipEventElapsedTime(&ms, a, b) != hipSuccess) rc = HIERAVG_EHIP;
  if (a) (void)hipEventDestroy(a);
  if (b) (void)hipEventDestroy(b);
  if (exec) (void)hipGraphExecDestroy(exec);
  (void)hipGraphDestroy(graph);
  if (rc != HIERAVG_OK) {
    set_error("timing the kernel failed");
    return rc;
  }
  *mean_ms = ms / reps;
  return HIERAVG_OK;
}

int hieravg_kernel_classes(void) { return KC_COUNT; }

const char* hieravg_kernel_class_name(int c) { return (c >= 0 && c < KC_COUNT) ? kClassNames[c] : ""; }

}  // extern "C"
