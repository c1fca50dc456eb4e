/*
 * hieravg.h -- C ABI of the Hier-AVG data-parallel hot path on one MI355X.
 *
 * Hier-AVG (Zhou & Cong, "A Distributed Hierarchical Averaging SGD
 * Algorithm: Trading Local Reductions for Global Reductions", arXiv
 * 1903.05133), Algorithm 1 in Sec. 3.1: P learners each run K1 local SGD
 * steps on their own minibatch of size B, then every local cluster of S
 * learners replaces its parameters by their mean; after K2 such blocks all P
 * learners replace their parameters by the global mean.  Sec. 2 fixes
 * S | P and S >= 1.
 *
 * Units.  K2 here counts local-averaging blocks per round (the paper's beta,
 * Sec. 3.1), so one round is K1*K2 SGD steps per learner and the paper's
 * global averaging interval is K1*K2 steps.
 *
 * All P learners are rows of one replica array on one GPU; a round is a
 * sequence of kernels enqueued on the handle's HIP stream.  The handle owns
 * every device buffer it allocates; callers own the buffers they pass in.
 * A handle is not thread-safe; distinct handles are independent.
 *
 * Errors.  Functions returning int return HIERAVG_OK (0) or a negative code;
 * hieravg_last_error() then describes the failure (thread-local string,
 * valid until the next failing call on the same thread).  Constructors return
 * NULL on failure.  Asynchronous GPU faults surface as HIERAVG_EHIP at the
 * next call that synchronises.
 */
#ifndef HIERAVG_H
#define HIERAVG_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef struct hieravg* hieravg_t;

/* Return codes. */
#define HIERAVG_OK 0
#define HIERAVG_EINVAL (-1) /* bad argument or handle                      */
#define HIERAVG_EHIP (-2)   /* HIP runtime or kernel error                 */
#define HIERAVG_ENONFINITE (-3) /* hieravg_check_finite: a replica holds inf or NaN */
#define HIERAVG_ESIZE (-4)  /* destination/source size too small / too big */

/* Model kinds (what one learner's SGD step computes). */
#define HIERAVG_KIND_SOFTMAX 0   /* softmax regression, IN -> C             */
#define HIERAVG_KIND_MLP 1       /* IN -> H (ReLU) -> C, softmax CE         */
#define HIERAVG_KIND_AVERAGING 2 /* momentum SGD on given gradients, no model */

/* Named workloads accepted by hieravg_create (the `model` argument). */
#define HIERAVG_MODEL_SOFTMAX_3072_10 0      /* N=2048, class means z, noise std 1 */
#define HIERAVG_MODEL_MLP_3072_512_10 1      /* N=50000, noise std 0.5             */
#define HIERAVG_MODEL_MLP_150528_1024_1000 2 /* N=100000, noise std 1              */
#define HIERAVG_MODEL_AVERAGING_11_7M 3      /* D=11.7e6, momentum 0.9, stds 0.01  */

/*
 * How the first weight block (W1 of the MLP) takes its SGD steps inside a
 * round.  Both give the result of Algorithm 1 up to float32 rounding.
 *  EAGER:   every step reads and writes each learner's W1 (the fused
 *           update-and-next-forward kernel).
 *  DELAYED: within a block of K1 steps each learner's W1 is its cluster's
 *           block-start copy minus lr times the sum of its steps' rank-B
 *           updates G^T X.  The forward uses the block-start copy plus the
 *           correction -lr * sum_{k'<k} (X_k X_k'^T) G_k' and the cluster
 *           mean at the block end is one update of the copy by the summed
 *           G^T X of the cluster's learners and steps.  Needs the MLP with
 *           B <= 32, K1 <= 8, K1*S*B <= 16384, whole blocks (k_global a
 *           multiple of K1), a dataset under 2^38 floats, momentum buffers
 *           that the means leave alone (avg_momentum = 0), and a round that
 *           starts with equal W1 in every replica (true after create, after
 *           every round, and after hieravg_set_params with equal W1 rows;
 *           otherwise that next round runs EAGER).  With momentum or weight
 *           decay the K1 heavy-ball steps of a block are linear in (W1, V1):
 *           W1 and its buffer at step n are fixed multiples of the block-start
 *           pair plus weighted sums of the step gradients, and the block end
 *           applies those weights in the same cluster GEMM.
 *  AUTO:    DELAYED where it applies and its extra Gram products cost at most
 *           an eighth of the step's flops ((K1 - 1) * B <= H / 2), else EAGER.
 */
#define HIERAVG_UPDATE_AUTO 0
#define HIERAVG_UPDATE_EAGER 1
#define HIERAVG_UPDATE_DELAYED 2

/*
 * Full description of a workload.  Synthetic data, minibatch draws, initial
 * parameters and (averaging kind) the given gradients are all generated on
 * the GPU from `seed` with the SplitMix64 counter generator (Steele, Lea &
 * Flood, OOPSLA 2014), H(key, c) = mix64(key + (c + 1) * 0x9E3779B97F4A7C15):
 *   sample s of learner j at global step t: H(k_index, t<<32 | j<<16 | s) mod N
 *   label of row i:                         H(k_label, i) mod C
 *   X[i][d] = fp32(mu[y_i][d] + noise_std * z(k_noise, i*IN + d)),
 *   mu[c][d] = z(k_mean, c*IN + d),  z = exact Irwin-Hall(12) normal surrogate,
 *   weights (2u - 1) * fp32(1/sqrt(fan_in)), u = (H(k_init, layer<<48 | e) >> 40) / 2^24,
 *   biases 0; averaging kind: w0[d] = fp32(init_std * z(k_init, d)) and
 *   gradient of learner j at step-in-round k: fp32(grad_std * z(k_grad, (k*2^16 + j)*D + d)).
 * Stream keys are k_x = H(seed, tag_x) for fixed 64-bit tags.
 */
typedef struct hieravg_config {
  int32_t P;        /* learners, 1 <= P < 65536                            */
  int32_t S;        /* learners per local cluster, S | P                    */
  int32_t K1;       /* local SGD steps per block, >= 1                      */
  int32_t K2;       /* blocks per round (the paper's beta), >= 1            */
  int32_t B;        /* minibatch size, 1 <= B < 65536 (ignored: averaging)  */
  int32_t kind;     /* HIERAVG_KIND_*                                        */
  int64_t in_dim;   /* softmax/MLP: input features; averaging: D            */
  int64_t hidden;   /* MLP hidden width; 0 otherwise                        */
  int64_t classes;  /* softmax/MLP classes; 0 for averaging                 */
  int64_t n_samples;/* dataset rows N (softmax/MLP), N < 2^32               */
  float noise_std;  /* data noise std                                       */
  float lr;         /* step size gamma, finite and >= 0                     */
  float momentum;   /* heavy-ball coefficient mu in [0, 1) (every kind):    */
                    /*   d = g + weight_decay*w, v <- mu*v + d, w <- w - lr*v */
  float init_std;   /* averaging kind: std of the initial replica           */
  float grad_std;   /* averaging kind: std of the given gradients           */
  uint64_t seed;
  int32_t update_mode; /* HIERAVG_UPDATE_* (how the first weight block is updated) */
  int32_t k_global;    /* SGD steps per round (the paper's global interval K2 in steps,
                          Sec. 3.1); 0: K1*K2.  When set, K2 is not used: a local mean
                          follows every K1 steps of the round except its last step, which
                          takes the global mean, so a round of k_global steps that K1
                          does not divide ends with a shorter block (a non-integer beta);
                          the count of local steps restarts at every global mean */
  float weight_decay;  /* L2 coefficient lambda >= 0 of the step above; with
                          momentum = weight_decay = 0 the step is Algorithm 1's
                          plain SGD step.  The paper states no optimizer beyond
                          SGD; these follow the usual heavy-ball convention.
                          Softmax/MLP with either set run EAGER updates. */
  int32_t avg_momentum; /* 1: every local and global mean also averages the
                           momentum buffers v; 0: v stays per learner (Algorithm 1
                           averages parameters only) */
} hieravg_config;

/*
 * Create a handle for one of the named workloads (HIERAVG_MODEL_*), as
 * Algorithm 1's first line: builds the dataset, draws the initial global
 * parameter w~_1 and copies it into all P replica rows.  Blocks until the
 * set-up kernels have finished.  Returns NULL (and sets the last error) on
 * invalid arguments (P<1, S<1, S not dividing P, K1<1, K2<1, B<1, P or B >=
 * 65536, lr not finite or negative, unknown model) or allocation failure.
 */
hieravg_t hieravg_create(int32_t P, int32_t S, int32_t K1, int32_t K2, int32_t model, float lr,
                         int32_t B, uint64_t seed);

/* Same, for an explicit workload description (any dimensions).  Also NULL for
 * an update_mode outside HIERAVG_UPDATE_* or DELAYED where it does not apply. */
hieravg_t hieravg_create_config(const hieravg_config* cfg);

/*
 * Enqueue one round (one outer iteration n of Algorithm 1): K2 blocks of K1
 * local SGD steps, a local mean over each cluster after every block but the
 * last, and the global mean at the end (the local mean right before the
 * global mean does not change the exact result and is skipped).
 * Asynchronous with respect to the host.  The first call captures the
 * round's kernels into a HIP graph; later calls launch that graph on the
 * handle's current stream (while profiling, the kernels are launched one by
 * one instead).  Returns HIERAVG_OK or an error.
 */
int hieravg_round(hieravg_t h);

/*
 * Synchronise the handle's stream and copy all replicas to `dst` as a dense
 * row-major [P][D] float32 array (D = hieravg_dim(h)), each row packed as
 * softmax [W (C x IN row-major) | b (C)], MLP [W1 (H x IN) | b1 (H) |
 * W2 (C x H) | b2 (C)], averaging [w (D)].  `dst` may be host or device
 * memory; `n_floats` is its capacity and must be >= P*D (else HIERAVG_ESIZE).
 */
int hieravg_params(hieravg_t h, float* dst, size_t n_floats);

/* Overwrite all replicas from a dense [P][D] array laid out as above (host
 * or device memory, n_floats >= P*D).  Momentum buffers are left as they are.
 * Synchronous.  When every replica's first weight block is then the same
 * (a checkpoint taken at a round boundary), the next round may take delayed
 * updates; otherwise it runs EAGER. */
int hieravg_set_params(hieravg_t h, const float* src, size_t n_floats);

/* The momentum buffers v of all learners, copied out / in as a dense [P][D]
 * array in the layout of hieravg_params (host or device memory, n_floats >=
 * P*D, else HIERAVG_ESIZE).  Synchronous.  HIERAVG_EINVAL when the handle has
 * no buffers (momentum = 0: the step keeps no state). */
int hieravg_momentum(hieravg_t h, float* dst, size_t n_floats);
int hieravg_set_momentum(hieravg_t h, const float* src, size_t n_floats);

/*
 * Minibatch size of the rounds enqueued from now on (a per-round schedule
 * B_n, Thm 3.3), 1 <= B <= the B given at create (the buffers' capacity).
 * The draws of sample s keep their counters, so the first B samples of a
 * step are the same for any B.  Synchronises; the next round rebuilds its
 * launch plan.  HIERAVG_EINVAL for the averaging kind or B out of range.
 */
int hieravg_set_batch(hieravg_t h, int32_t B);

/*
 * Step size of the rounds enqueued from now on (a per-round schedule, e.g.
 * the step decay 0.1 -> 0.01 of Sec. 4 or the gamma_n of Thm 3.3).  The value
 * lives in device memory and every kernel reads it, so a change needs no new
 * launch plan.  Synchronises the handle's stream.  HIERAVG_EINVAL for a
 * non-finite or negative lr.
 */
int hieravg_set_lr(hieravg_t h, float lr);

/*
 * Quality of one replica's model (softmax or MLP kinds): the mean softmax
 * cross-entropy F(w; xi) over `n_rows` rows (the empirical risk of Sec. 2)
 * and the number of rows whose first largest logit is the label's.  split 0
 * takes the training rows 0 .. n_rows-1 (n_rows <= N); split 1 takes held-out
 * rows 0 .. n_rows-1 of a second synthetic set with the same class means and
 * its own label and noise streams (labels H(k_tlabel, i) mod C, noise
 * z(k_tnoise, i*IN + d)), generated on the GPU at the first call that needs
 * them.  Runs on the handle's stream and synchronises; allocates its
 * buffers at the first call.  HIERAVG_EINVAL for the averaging kind, a bad
 * replica or split, or n_rows out of range.
 */
int hieravg_evaluate(hieravg_t h, int32_t replica, int32_t split, int64_t n_rows, double* mean_loss,
                     int64_t* correct);

/*
 * hieravg_evaluate for callers that cannot allocate device memory (code that
 * must not call hipMalloc or hipFree: tight serving or evaluation loops,
 * harnesses that forbid allocation).  Same arguments, results and errors as
 * hieravg_evaluate; it allocates nothing.  Its chunk buffers (row list,
 * split-K partials, activations, per-row losses and hits) live in one
 * file-scope device array of HIERAVG_EVAL_SCRATCH_BYTES bytes that exists
 * once on every GPU the library runs on and is held until the process ends;
 * the chunk is the largest of 4096, 2048, ..., 16 rows whose buffers fit.
 * Every call on a GPU shares that GPU's array (nothing in it needs to start
 * at zero), so calls that overlap on one GPU, from any handles or threads,
 * race and must be serialised by the caller.  Split 1 evaluates held-out
 * rows that an earlier hieravg_evaluate call of the handle generated
 * (n_rows above that count: HIERAVG_ESIZE).  A model whose 16-row chunk does
 * not fit the array (2*hidden + classes above about 262000 for the MLP,
 * classes above that for softmax regression) gets HIERAVG_ESIZE with the
 * size it would need.  Runs on the handle's stream,
 * on the handle's device, and synchronises.
 */
#define HIERAVG_EVAL_SCRATCH_BYTES ((size_t)16 << 20)
int hieravg_evaluate_noalloc(hieravg_t h, int32_t replica, int32_t split, int64_t n_rows, double* mean_loss,
                             int64_t* correct);

/* Release every resource of the handle.  NULL-safe. */
void hieravg_destroy(hieravg_t h);

/* Thread-local description of the last failure ("" if none). */
const char* hieravg_last_error(void);

/* Parameters per replica D, or a negative code for a NULL handle. */
int64_t hieravg_dim(hieravg_t h);

/* Global SGD steps taken since creation (K1*K2 per round). */
int64_t hieravg_step_count(hieravg_t h);

/* Divergence check: synchronise and scan every replica; HIERAVG_OK when all
 * parameters are finite, HIERAVG_ENONFINITE when any is inf or NaN (for
 * example after a step size too large for the data). */
int hieravg_check_finite(hieravg_t h);

/* Set the global step counter t (t >= 0): the next round draws its
 * minibatches for steps t, t+1, ...  With hieravg_set_params (and
 * hieravg_set_momentum) this resumes a run exactly from a checkpoint taken
 * at a round boundary.  Synchronous; HIERAVG_EINVAL for t < 0. */
int hieravg_set_step_count(hieravg_t h, int64_t t);

/*
 * Copy the minibatch indices the last round drew, as int32 [T][P][B] with T
 * the steps per round (K2*K1 or k_global) and B the current minibatch size
 * (hieravg_set_batch), to `dst` (host or device,
 * n >= T*P*B).  Synchronises.  HIERAVG_EINVAL for the averaging kind (it
 * draws no samples).
 */
int hieravg_last_indices(hieravg_t h, int32_t* dst, size_t n);

/*
 * Make the handle enqueue on `hip_stream` (a hipStream_t, e.g. a torch
 * stream's handle; NULL selects the handle's own stream).  The caller keeps
 * ownership of the stream and must keep it alive while the handle uses it.
 * Synchronises the previous stream first.
 */
int hieravg_set_stream(hieravg_t h, void* hip_stream);

/* Block until all work enqueued by the handle has finished. */
int hieravg_sync(hieravg_t h);

/*
 * Per-kernel timing with HIP events: while enabled, every launch carries two
 * events that its dispatch packet stamps at kernel start and end, so the
 * recorded durations are the kernels' execution times.  enable != 0 starts
 * recording (clearing earlier records); enable == 0 stops.  hieravg_profile_read synchronises and writes, for every
 * kernel class c < min(n, hieravg_kernel_classes()), the number of launches
 * and their summed duration in milliseconds.
 */
int hieravg_profile(hieravg_t h, int enable);
int hieravg_profile_read(hieravg_t h, int64_t* launches, double* total_ms, int n);
int hieravg_kernel_classes(void);

/*
 * Mean duration in milliseconds of one launch of kernel class
 * `kernel_class` (see hieravg_kernel_class_name), from HIP events around one
 * launch of a graph of `reps` back-to-back launches of it (captured on the
 * handle's stream) with the arguments of step 0 of the current round.  For measurement only: the launches act on the replicas as
 * `reps` extra applications of that kernel would.  HIERAVG_EINVAL for a class
 * the workload does not launch, for the index draw, or while profiling.
 * Synchronises.
 */
int hieravg_time_kernel(hieravg_t h, int kernel_class, int reps, double* mean_ms);
const char* hieravg_kernel_class_name(int c);

#ifdef __cplusplus
}
#endif

#endif /* HIERAVG_H */
