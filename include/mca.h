/*
 * mca.h -- C ABI of the MI355X (gfx950) library for the hot path of the Monte
 * Carlo mutation-selection method (MCA): mutate one parameter, evaluate the
 * loss incrementally from cached local fields, accept or roll back.
 *
 * The calls follow the paper's statement of the problem:
 *   - training set D = {(x_mu, y_mu)} and network f_W (Sec. 3.1, Eq. 2);
 *   - mutation W' = W + dW of a single entry, w -> w + delta * rand with rand
 *     uniform on [-1, 1], or a jump to another discrete state (Sec. 2, Eq. 1;
 *     Eq. 5; Eq. 12);
 *   - loss L(W') = average cross-entropy over the whole sample set (Sec. 2,
 *     Eq. 2 with R = 0);
 *   - greedy selection: keep W' if the loss change passes the test, else keep W
 *     (Eq. 6);
 *   - incremental evaluation from the local fields cached after the last
 *     accepted mutation (Sec. 2.4; Sec. 2.1 for the layer-local cache).
 *
 * Conventions shared by every call:
 *   - Ownership: host arrays passed in are owned by the caller, read during the
 *     call and never retained.  The device workspace is owned by the caller
 *     (e.g. a torch uint8 tensor), must be at least mca_plan() bytes, 256-byte
 *     aligned, and must outlive the context.  The context owns only its host
 *     struct and, once created, a few HIP events.
 *   - Stream: all device work is enqueued on the hip_stream given to mca_init
 *     (hipStream_t passed as void*; NULL = the null stream).  Every call that
 *     returns host values synchronises that stream before returning.
 *   - Errors: calls return MCA_OK (0) or a negative MCA_E* code.  Arguments are
 *     validated before anything is enqueued, so a call that fails validation
 *     changes nothing.  A HIP runtime error poisons the context: every later
 *     call returns MCA_EPOISONED.  mca_last_error(ctx) returns the message of
 *     the last failure (ctx may be NULL for failures before a context exists;
 *     that message is thread-local).  No C++ exception crosses this ABI.
 *   - Layout of an MLP: weight l (0-based) has shape [n_{l+1}][n_l], row j is
 *     the output unit, column i the input unit (z = W a, Sec. 3.6), row-major.
 *     Biases: none (the MLP weights are the only mutable parameters).
 *   - Threading: a context must not be used by two threads at once.
 */
#ifndef MCA_H_
#define MCA_H_

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define MCA_ABI_VERSION 3
#define MCA_MAX_LAYERS 32  /* maximum number of MLP weight matrices */
#define MCA_MAX_CLASSES 16 /* maximum MLP output width (logits kept in registers) */

/* status codes */
#define MCA_OK 0
#define MCA_EINVAL (-1)       /* bad shape, enum, K, index or pointer */
#define MCA_ESTATE (-2)       /* commit/rollback without a pending batch, eval while pending */
#define MCA_ENOSPACE (-3)     /* workspace smaller than mca_plan() */
#define MCA_EDEVICE (-4)      /* HIP runtime error; the context is now poisoned */
#define MCA_EPOISONED (-5)    /* context poisoned by an earlier device error */
#define MCA_EUNSUPPORTED (-6) /* valid request this build does not implement */

/* network kinds */
#define MCA_NET_MLP 0
#define MCA_NET_TRANSFORMER 1

/* transfer functions of hidden MLP layers (Sec. 2) */
#define MCA_ACT_TANH 0
#define MCA_ACT_GAUSS 1 /* exp(-gamma z^2) */
#define MCA_ACT_RELU 2  /* max(0, z) */

/* weight modes */
#define MCA_WEIGHTS_FP32 0    /* continuous fp32 weights, w -> fl32(w + d) (Eq. 1) */
#define MCA_WEIGHTS_TERNARY 1 /* w = code * scale_l, code in {-1, 0, 1} (Eq. 12) */

/* selection rules */
#define MCA_RULE_GREEDY 0     /* accept iff dL < 0 (dL <= 0 with accept_ties) (Eq. 6) */
#define MCA_RULE_METROPOLIS 1 /* accept with probability min{1, exp(-beta dL)} (Eq. 7) */

/* what one candidate changes (MLPs) */
#define MCA_MUTATE_SINGLE 0         /* one parameter (Eq. 1) */
#define MCA_MUTATE_CHANNEL_REDRAW 1 /* a channel: one weight per layer on an input-to-output
                                     * path, each re-drawn as fl32(sqrt(8 / fan_in)) * r (Sec. 2.3) */
#define MCA_MUTATE_CHANNEL_ZERO 2   /* a channel whose weights are all set to zero (Sec. 2.3) */

/* how a candidate picks its parameter */
#define MCA_PICK_WEIGHT 0 /* uniform over all parameters */
#define MCA_PICK_LAYER 1  /* uniform layer, then uniform inside it */
#define MCA_PICK_STICKY 2 /* Sec. 2.1's current-layer schedule: the steps of block
                           * e = floor(t / sticky_steps) all mutate layer
                           * floor(w0 L / 2^64), w0 = word 0 of the Philox block at
                           * counter (e, 0, 0, 1); uniform inside that layer */

typedef struct mca_net_desc {
  int32_t kind;                         /* MCA_NET_* */
  /* MLP */
  int32_t n_layers;                     /* number of weight matrices L, 1..MCA_MAX_LAYERS */
  int32_t widths[MCA_MAX_LAYERS + 1];   /* n_0 .. n_L; n_L <= MCA_MAX_CLASSES */
  int32_t act;                          /* MCA_ACT_* for hidden layers; logits are linear */
  float gamma;                          /* Gaussian coefficient (MCA_ACT_GAUSS) */
  int32_t weight_mode;                  /* MCA_WEIGHTS_* */
  float scales[MCA_MAX_LAYERS];         /* ternary: per-layer scale s_l (fp32) */
  /* mutation and selection */
  int32_t pick;                         /* MCA_PICK_* */
  float delta;                          /* amplitude: d = fl32(delta * r), r in [-1, 1 - 2^-23] */
  float bound;                          /* > 0: reject unevaluated if |w'| >= bound (Eq. 1 Delta) */
  int32_t accept_ties;                  /* 0: accept iff dL < 0; 1: dL <= 0 (Eq. 6) */
  uint64_t seed;                        /* Philox key word 0 */
  uint64_t stream_tag;                  /* Philox key word 1 */
  /* Transformer (MCA_NET_TRANSFORMER) */
  int32_t vocab, ctx, d_model, n_block, n_head, d_mlp;
  float ln_eps;
  /* selection rule (Eq. 6 / Eq. 7).  Metropolis: candidate k of step t draws
   * U from Philox block (t, k, 1, 0), word 0: U = (w0 >> 11) * 2^-53, and passes
   * iff dL < -ln(U) / beta (the same event as U < exp(-beta dL)). */
  int32_t accept_rule;                  /* MCA_RULE_* */
  /* pruning (Sec. 2.2, "w -> 0"): in every step candidates 0 .. n_prune-1
   * set their weight to zero (d = -w; ternary: code 0), the rest are the
   * ordinary mutations; n_prune >= K gives pure pruning, 0 none.  Pruning
   * candidates come first in stream order, so they are preferred. */
  int32_t n_prune;
  double beta;                          /* Metropolis selection intensity, > 0 */
  /* minibatch (Sec. 2.2, MLPs): 0 = every sample; otherwise the loss
   * changes of steps t with floor(t / subset_period) = e are averaged over
   * the subset_size samples n = ((e mod N) * subset_size + m) mod N,
   * m < subset_size (consecutive windows of the sample order, wrapping).
   * The explicit mca_eval_losses scores the window of the device's next step
   * (mca_set_step).  Caches stay exact for every sample, and the committed
   * loss is the mean over every sample. */
  int64_t subset_size;
  int64_t subset_period;
  /* MCA_MUTATE_*.  Channel mutations (Sec. 2.3) need an MLP of fp32 weights
   * with L >= 2 whose hidden layers are all 256, 512 or 1024 wide, every
   * sample in each step (subset_size 0) and no pruning candidates
   * (n_prune 0); their candidates are mca_channel records (mca_propose_channels,
   * mca_eval_channels), scored against the committed state like single
   * mutations and committed, rolled back and run (mca_run_steps) the same way. */
  int32_t mutation;
  /* Deep nets of Sec. 2.1 (MLPs).  biases = 1: layer l has one bias per
   * unit; its parameter tensor is the augmented matrix [n_{l+1}][n_l + 1]
   * (row j: unit j's incoming weights, then its bias), and a candidate with
   * i = n_l mutates that bias.  layer_norm = 1: every hidden local field is
   * normalized over the units of its layer, sample by sample,
   * h = (z - mean z) / sqrt(var z + ln_eps) (population variance, no gain or
   * bias), before the transfer function; the logits are not normalized.
   * Either needs L >= 2, every hidden layer 256, 512 or 1024 units wide,
   * fp32 weights and single mutations.  sticky_steps: block length of
   * MCA_PICK_STICKY (>= 1), ignored by the other picks. */
  int32_t biases;
  int32_t layer_norm;
  int32_t sticky_steps;
} mca_net_desc;

/* mca_cand.flags */
#define MCA_CAND_PRUNE 1 /* set the weight to zero (Sec. 2.2): w' = 0, d = -w, code 0 */

/* One proposed single-parameter mutation (32 bytes). */
typedef struct mca_cand {
  int64_t flat;  /* index over all parameters in canonical order */
  int32_t layer; /* parameter tensor (MLP: weight matrix) index */
  int32_t j;     /* row: output unit (1-D tensors: element) */
  int32_t i;     /* column: input unit (1-D tensors: 0) */
  float d;       /* continuous: fp32 increment fl32(delta * r); ternary or pruning: fl32(w' - w) */
  int32_t code;  /* ternary: the new code (-1, 0, 1); continuous: 0 */
  int32_t flags; /* MCA_CAND_* */
} mca_cand;

/* One proposed channel mutation (Sec. 2.3): units[m] is the path's unit in
 * layer m (units[0] an input, units[L] a class; entries past L unused); the
 * path's weight of layer m is W_m[units[m + 1]][units[m]] and becomes
 * w_new[m].  Drawn from the Philox blocks at counters (t, k, 2 + b, 0),
 * words in order: word m gives units[m] = floor(word * n_m / 2^64), m = 0..L;
 * word L + 1 + m re-draws w_new[m] = fl32(fl32(sqrt(8 / n_m)) * r) with
 * r = (word >> 40) * 2^-23 - 1 (zero for MCA_MUTATE_CHANNEL_ZERO).  260 bytes. */
typedef struct mca_channel {
  int32_t units[MCA_MAX_LAYERS + 1];
  float w_new[MCA_MAX_LAYERS];
} mca_channel;

/* Data set.  MLP: x is [n_samples][n_0] fp32 row-major, y the labels in
 * [0, n_L).  Transformer: tokens is [n_seq][ctx] int32, y the next-symbol
 * targets [n_seq][ctx]; n_samples = n_seq * ctx positions. */
typedef struct mca_data {
  int64_t n_samples;
  const float* x;
  const int32_t* tokens;
  const int32_t* y;
  int32_t n_seq;
  int32_t reserved;
} mca_data;

typedef struct mca_stats {
  uint64_t steps;     /* steps completed by this call */
  uint64_t evaluated; /* candidate evaluations that count: K per completed step */
  uint64_t accepted;  /* committed mutations */
  uint64_t wasted;    /* speculative evaluations discarded (not counted above) */
  uint64_t tie_band;  /* decision-relevant candidates with |dL| < 1e-6 */
  double loss;        /* committed loss after the call */
  uint64_t next_step; /* step index t of the next step */
} mca_stats;

/* Optional per-step record of mca_run_steps (host arrays, caller-owned). */
typedef struct mca_trace {
  int32_t* chosen; /* [n_steps]: committed candidate k of each step, or -1 */
  double* dloss;   /* [n_steps * K]: every candidate's dL, or NULL */
} mca_trace;

/* Accumulated device time per phase (HIP events on the context's stream). */
typedef struct mca_timing {
  double ms[8];        /* by phase: 0 propose, 1 eval, 2 select, 3 commit, 4 step loop,
                          5 forward, 6 one-workgroup step loop */
  uint64_t launches[8];
} mca_timing;

typedef struct mca_ctx mca_ctx;

/* ABI version (MCA_ABI_VERSION). */
int mca_abi_version(void);

/* sizeof of the ABI structs, so bindings can check their mirrors:
 * which = 0 mca_net_desc, 1 mca_cand, 2 mca_data, 3 mca_stats, 4 mca_trace,
 * 5 mca_timing, 6 mca_channel; 0 for any other value. */
size_t mca_struct_size(int32_t which);

/* Device workspace bytes for a net, n_samples and at most k_max candidates per
 * step.  Pure: touches no device.  Returns MCA_EINVAL on a bad description and
 * MCA_EUNSUPPORTED for a valid net this build does not run: MLPs of three or
 * more layers whose last hidden layer has more than 1024 units, MLPs of four
 * or more layers whose hidden layers are not all 256 units wide, and
 * Transformers outside d_model = 32 * n_head <= 256, d_mlp a multiple of 32,
 * ctx <= 128, vocab <= 128, n_block <= 8, fp32 weights with the uniform
 * parameter pick. */
int mca_plan(const mca_net_desc* net, int64_t n_samples, int32_t k_max,
             size_t* workspace_bytes);

/* Create a context: validate, copy the host parameters and data into the
 * workspace, run the full forward pass over all samples to fill the local-field
 * and per-sample loss caches (Sec. 2.1, Sec. 2.4), set the step counter to 0.
 * params: n_params host pointers in canonical order (MLP: the L weight
 * matrices, augmented with their bias column when biases = 1).  codes: ternary only, L host int8 arrays of the same shapes
 * (params must then equal code * scale); NULL otherwise.  Synchronises. */
int mca_init(mca_ctx** out, const mca_net_desc* net, const float* const* params,
             int32_t n_params, const int8_t* const* codes, const mca_data* data,
             int32_t k_max, void* workspace, size_t workspace_bytes, void* hip_stream);

/* Candidates k = 0..K-1 of step `step`: Philox4x64-10 with key (seed, tag),
 * counter (step, k, 0, 0), decoded as in Eq. 1 / Eq. 12 (the ternary move reads
 * the committed codes).  Pure with respect to the committed state.  Writes K
 * records to out_host.  1 <= K <= k_max.  MCA_ESTATE while a batch is pending
 * (it reuses the pending batch's device buffers).  Synchronises. */
int mca_propose(mca_ctx* ctx, uint64_t step, int32_t K, mca_cand* out_host);

/* Score K candidates against the committed state: loss_out[k] = L + dL_k and
 * dloss_out[k] = dL_k, dL_k = (1/N) sum_n (l'_n - l_n) over the samples the
 * mutation changes (Eq. 2 difference).  A candidate whose |w'| >= bound gets
 * +inf.  Either output may be NULL.  Leaves the committed state untouched and
 * marks the batch pending (MCA_ESTATE if one is already pending).  Synchronises. */
int mca_eval_losses(mca_ctx* ctx, const mca_cand* cands_host, int32_t K,
                    double* loss_out, double* dloss_out);

/* Channel contexts (mutation MCA_MUTATE_CHANNEL_*, Sec. 2.3): candidates
 * k = 0..K-1 of step `step` as channel records (the draw described at
 * mca_channel), 1 <= K <= k_max.  Pure with respect to the committed state.
 * MCA_ESTATE while a batch is pending, MCA_EINVAL on a single-mutation
 * context.  Synchronises. */
int mca_propose_channels(mca_ctx* ctx, uint64_t step, int32_t K, mca_channel* out_host);

/* Channel contexts: score K channel records against the committed state, as
 * mca_eval_losses does for single mutations: dL_k = L(W with every path
 * weight of channel k replaced) - L(W), computed on every sample from the
 * cached fields (the first field's path column, then each later layer's
 * dense change plus its own path weight's change).  A channel with any
 * |w_new| >= bound gets +inf.  Records are validated (units in range, finite
 * values) before anything is enqueued.  Marks the batch pending; commit it
 * with mca_commit(k) or drop it with mca_rollback.  Synchronises. */
int mca_eval_channels(mca_ctx* ctx, const mca_channel* chans_host, int32_t K,
                      double* loss_out, double* dloss_out);

/* Accept candidate k of the pending batch (Eq. 6): write the new parameter and
 * update the cached local fields and per-sample losses in place; L += dL_k.
 * Clears the pending batch.  MCA_ESTATE without a pending batch, MCA_EINVAL
 * for k outside [0, K).  Does not synchronise. */
int mca_commit(mca_ctx* ctx, int32_t k);

/* Reject the pending batch (Eq. 6, W_{t+1} = W_t).  The committed state is
 * byte-identical to before the evaluation.  MCA_ESTATE without a pending batch. */
int mca_rollback(mca_ctx* ctx);

/* For callers that cannot allocate device memory (code under HIP graph
 * capture, tight serving loops, harnesses that forbid it): mca_eval_losses
 * without any use of the context's per-call buffers.  The per-call device
 * buffers (the candidates' device copy, prepared values, tile sums, the
 * three-layer and deep nets' affected-sample lists, loss changes) live in one
 * static array per GPU of 8 MiB, held until the process ends; a request that
 * needs more (K x (N or tiles) too large) fails with MCA_EINVAL before
 * anything is enqueued.  The call allocates nothing, scores K candidates
 * (1 <= K <= 1024, K not bounded by k_max) against the committed state
 * exactly as mca_eval_losses does (same kernels, same results), leaves no
 * pending batch and touches no pending batch's buffers, and synchronises.
 * MLP contexts only (MCA_EUNSUPPORTED otherwise).  Every call on a GPU shares
 * that GPU's array: calls that overlap on one GPU (several streams or
 * threads) race on it. */
int mca_eval_losses_noalloc(mca_ctx* ctx, const mca_cand* cands_host, int32_t K,
                            double* loss_out, double* dloss_out);

/* Tuning options of mca_run_steps (mca_set_option):
 *   MCA_OPT_PERSISTENT_LOOP  1 (default): run eligible nets (mutations reach
 *                            at most the last two layers, K <= 64) in one
 *                            launch per call: one workgroup when the samples
 *                            and weights fit it (N <= 1024, K <= 2, at most 10
 *                            classes and 3072 weights; with K = 1 it scores
 *                            steps t and t + 1 against one state and counts a
 *                            discarded second score in stats.wasted), else a
 *                            grid of workgroups; 0: one launch per phase per
 *                            step.  All give the same decisions up to the
 *                            order of the loss-change sums.
 *   MCA_OPT_LOOP_TILE        samples per workgroup of the persistent loop,
 *                            16..64 (default 64).
 *   MCA_OPT_LOOP_LAUNCH      1 (default): an ordinary launch of the
 *                            persistent loop's grid, relying on the library's
 *                            occupancy check for all workgroups to be resident
 *                            together (on a GPU shared with other work, a
 *                            workgroup kept out makes the loop's bounded waits
 *                            give up: MCA_EDEVICE, never a hang); 0: a
 *                            cooperative launch, where the runtime guarantees
 *                            it (about 15 us more per call). */
#define MCA_OPT_PERSISTENT_LOOP 1
#define MCA_OPT_LOOP_TILE 2
#define MCA_OPT_LOOP_LAUNCH 3
/* Set a tuning option; MCA_EINVAL for an unknown option or value. */
int mca_set_option(mca_ctx* ctx, int32_t option, int64_t value);

/* Set the device's next step index (the step mca_run_steps starts from).  The
 * explicit path (mca_propose with an explicit step, mca_eval_losses,
 * mca_commit / mca_rollback) never changes it.  MCA_ESTATE while a batch is
 * pending.  Does not synchronise. */
int mca_set_step(mca_ctx* ctx, uint64_t next_step);

/* Run steps t .. t+n_steps-1 on the device with K candidates each: propose,
 * evaluate, commit the first candidate in stream order that passes the test,
 * no host round trip per step.  trace may be NULL.  stats (may be NULL) gets
 * this call's counters.  MCA_ESTATE while a batch is pending.  Synchronises. */
int mca_run_steps(mca_ctx* ctx, uint64_t n_steps, int32_t K, mca_trace* trace,
                  mca_stats* stats);

/* Copy the committed parameters (and ternary codes; codes may be NULL) to host
 * arrays in canonical order.  Synchronises. */
int mca_get_params(mca_ctx* ctx, float* const* params_out, int8_t* const* codes_out);

/* Committed loss L and the next step index.  Synchronises. */
int mca_get_loss(mca_ctx* ctx, double* loss, uint64_t* next_step);

/* Replace the committed state (resume from a checkpoint): parameters, codes
 * (ternary), next step index; recomputes every cache.  Synchronises. */
int mca_set_state(mca_ctx* ctx, const float* const* params, const int8_t* const* codes,
                  uint64_t next_step);

/* Recompute every cache from the committed parameters with the full forward
 * pass (removes drift of the incremental updates).  Synchronises. */
int mca_refresh(mca_ctx* ctx);

/* Copy the cached per-sample losses l_n (fp32, n_samples values).  A
 * Transformer context first completes the dense recomputation of its last
 * incrementally scored winner (Sec. 2.5), which the next evaluation would
 * otherwise do.  Synchronises. */
int mca_get_sample_losses(mca_ctx* ctx, float* out_host);

/* Phase timers: phase_mask bit p enables recording a pair of HIP events on the
 * context's stream around every launch of phase p (phases as in mca_timing;
 * 0 disables all); no synchronisation per launch.  mca_get_timing reads (and
 * optionally resets) the accumulated device time per phase and synchronises.
 * The events add a little launch overhead.  A non-zero mask also makes up to
 * 32 events ahead (kept until mca_destroy), so the first timed launches
 * create none. */
int mca_set_timing(mca_ctx* ctx, int32_t phase_mask);
int mca_get_timing(mca_ctx* ctx, mca_timing* out, int32_t reset);

/* Release the context (not the caller's workspace).  NULL is ignored. */
void mca_destroy(mca_ctx* ctx);

/* Message of the last failure on ctx, or of the calling thread when ctx is NULL. */
const char* mca_last_error(const mca_ctx* ctx);

#ifdef __cplusplus
}
#endif

#endif /* MCA_H_ */
