/*
 * oscars.h - C ABI of the Oscars local-SGD hot path on one MI355X (gfx950).
 *
 * The method (Huang, "Oscars: Adaptive Semi-Synchronous Parallel Model for
 * Distributed Deep Learning with Global View", arXiv 2102.08550):
 *   - Problem Formulation, Eq. 1-3: a common barrier T and per-worker local
 *     step counts tau_i = floor(T / t_i^iter) chosen to minimise the largest
 *     idle time max_i mod(T, t_i^iter) under a bound M on the step spread;
 *   - Approach, Algorithm 1 (Load-Balance): the scan that finds T*;
 *   - Approach, Eq. 4: each worker runs tau_i local SGD steps
 *     x <- x - eta g(x); at its tau_i-th step the models of all N workers are
 *     averaged with weight 1/N and every worker continues from the average.
 *
 * Here the N workers are K simulated replicas that live side by side in one
 * GPU's memory; the parameter server's aggregation is a K-way reduction kernel.
 *
 * Conventions for every function:
 *   - returns an oscars_status (0 = OSCARS_OK, < 0 = error); never throws;
 *   - arguments are validated before anything is changed or enqueued; on an
 *     OSCARS_E_INVALID / OSCARS_E_INFEASIBLE return nothing was modified;
 *   - device pointers are HIP device memory owned by the caller; host arrays
 *     are only read (or written, for outputs) during the call;
 *   - GPU work is enqueued on the given HIP stream (NULL = the null stream)
 *     and the call returns without waiting, unless stated otherwise;
 *   - on OSCARS_E_HIP the contents of device outputs are unspecified and
 *     oscars_last_hip_error() gives the HIP error code;
 *   - a context is not thread-safe; distinct contexts are independent.
 */
#ifndef OSCARS_H
#define OSCARS_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef int32_t oscars_status;

enum {
  OSCARS_OK = 0,
  OSCARS_E_INVALID = -1,    /* bad argument: null, out of range, misaligned  */
  OSCARS_E_NOMEM = -2,      /* host or device allocation failed              */
  OSCARS_E_HIP = -3,        /* a HIP runtime call or kernel launch failed    */
  OSCARS_E_INFEASIBLE = -4, /* Algorithm 1: constraint false at T = max t    */
  OSCARS_E_STATE = -5       /* call not valid in the context's current state */
};

enum { OSCARS_FP32 = 0, OSCARS_BF16 = 1 };

/* Largest number of replicas one aggregation accepts. */
#define OSCARS_MAX_K 64
/* Largest mini-batch size and layer width the local-step kernels accept. */
#define OSCARS_MAX_BATCH 1024
#define OSCARS_MAX_WIDTH 65536
#define OSCARS_MAX_LAYERS 16

/* Opaque context: model shape, K, device workspace, per-worker cursors. */
typedef struct oscars_ctx oscars_ctx;

/*
 * Model: a fully connected ReLU network with a softmax cross-entropy loss.
 *   n_layers  L >= 1 (L = 1 is softmax regression);
 *   dims      host [L + 1]: dims[0] = input width d, dims[L] = classes C,
 *             every entry in [1, OSCARS_MAX_WIDTH]; all but dims[L] must be
 *             multiples of 8 (16-byte rows for the kernels' vector loads);
 *   dtype     OSCARS_FP32: inputs, weights and arithmetic in fp32;
 *             OSCARS_BF16: bf16 inputs and weights in the products, fp32
 *             accumulation, fp32 master parameters.
 * Flat parameter layout of one replica (what oscars_num_params counts):
 *   [W_1 (dims[1] x dims[0], row-major), b_1 (dims[1]), W_2, b_2, ...],
 *   each segment starting on a 64-element (256-byte) boundary; the padding
 *   between segments is zero and stays zero.
 */
typedef struct {
  int32_t n_layers;
  const int32_t* dims;
  int32_t dtype;
} oscars_model;

/*
 * Training data and the workers' shards (Introduction: each worker of a
 * parameter server holds different training data).
 *   x        device [n_rows][d]: fp32, or bf16 bit patterns for OSCARS_BF16;
 *            16-byte aligned;
 *   y        device [n_rows] int32 labels in [0, C) (a row with a label
 *            outside that range gets a NaN loss and no one-hot term);
 *   n_rows   number of rows;
 *   offsets  host [K + 1], non-decreasing, offsets[0] = 0,
 *            offsets[K] = n_rows; worker k owns rows [offsets[k], offsets[k+1]),
 *            which must not be empty;
 *   seed     seed of the mini-batch sampler (see oscars_sample_indices).
 */
typedef struct {
  const void* x;
  const int32_t* y;
  int64_t n_rows;
  const int64_t* offsets;
  uint64_t seed;
} oscars_shards;

/* Create a context for K replicas of `model`, mini-batches up to max_batch.
 * Allocates, on the current HIP device, the whole device workspace the
 * local steps use: activations, bf16 weight copies, split-K partials, the
 * index table and loss buffer for rounds of up to 64 local steps per worker
 * (with pinned host staging), and, for bf16 models, the scratch replicas
 * on which OSCARS_BACKWARD_AUTO times the backward paths (K x the widest
 * layer, fp32 + bf16; left out where they would take
 * more than a quarter of the free device memory, and then nothing is timed).
 * `hip_stream` (a hipStream_t, NULL = null stream) is the stream
 * oscars_local_steps enqueues on.  The context owns its tuning state (GEMM
 * tilings, backward path): contexts do not share it. */
oscars_status oscars_create(oscars_ctx** out, const oscars_model* model, int32_t K,
                            int32_t max_batch, void* hip_stream);
/*
 * Convolutional model: the stand-in for the paper's own workload, a
 * convolutional network trained on CIFAR-10 images (Evaluation Setup).  fp32
 * throughout, like the paper's PyTorch.
 *   height, width, channels  the input image; a dataset row holds
 *             height x width x channels fp32 values, channels fastest (NHWC);
 *             height, width <= 4096, the row at most 2^24 values, and
 *             max_batch x every layer's activations below 2^31 values;
 *   n_conv    1 <= n_conv <= OSCARS_MAX_LAYERS - 1 conv layers, each a 3 x 3
 *             convolution with one row and column of zero padding on every
 *             side, a bias per output channel and ReLU:
 *               Z[b][i][j][o] = bias[o] + sum_{r,s,c} X[b][s i + r - 1][s j + s' - 1][c] W[o][r][s'][c]
 *             with output extent (input - 1) / stride + 1;
 *   conv_channels  host [n_conv]: output channels, 1 .. OSCARS_MAX_WIDTH;
 *   conv_strides   host [n_conv]: 1 or 2;
 *   classes   then every channel averaged over all positions, a linear
 *             classifier to `classes` logits (with bias), softmax cross-entropy
 *             averaged over the batch;
 *   conv_skip host [n_conv] or NULL (none): nonzero where conv layer l (1-based)
 *             ends a residual block, the identity shortcut of the paper's
 *             ResNet: the output of layer l - 2 (the block's input) is added to
 *             Z before the ReLU.  Such a layer needs l >= 3, stride 1 for
 *             layers l - 1 and l, as many channels as layer l - 2 and at least
 *             4 input channels; else OSCARS_E_INVALID.
 * Flat parameter layout of one replica: [W_1 ([C_1][3][3][C_0]), b_1, ...,
 * W_n, b_n, W_fc ([classes][C_n]), b_fc], each segment starting on a
 * 64-element boundary (oscars_layer_offsets: layers 1 .. n_conv + 1).
 * Every other call (local steps, rounds, aggregation, evaluation, cursors)
 * takes the context as for the fully connected model; x is the fp32 images.
 */
typedef struct {
  int32_t height, width, channels;
  int32_t n_conv;
  const int32_t* conv_channels;
  const int32_t* conv_strides;
  int32_t classes;
  const int32_t* conv_skip;
} oscars_cnn_model;

/* Create a context for K replicas of a convolutional model (see above), mini-
 * batches up to max_batch; allocates its whole device workspace (activations
 * and their gradients per conv layer, pooled features, logits, weight-gradient
 * partials, the index table) on the current device. */
oscars_status oscars_create_cnn(oscars_ctx** out, const oscars_cnn_model* model, int32_t K,
                                int32_t max_batch, void* hip_stream);

/* Free the workspace.  NULL is allowed.  Waits for the context's stream. */
void oscars_destroy(oscars_ctx* ctx);
/* Replace the stream later calls enqueue on. */
oscars_status oscars_set_stream(oscars_ctx* ctx, void* hip_stream);
/* Padded flat length of one replica (the stride between replicas). */
int64_t oscars_num_params(const oscars_ctx* ctx);
/* Element offsets of W_l and b_l (l = 1..L) in the flat layout. */
oscars_status oscars_layer_offsets(const oscars_ctx* ctx, int32_t l, int64_t* w_off,
                                   int64_t* b_off);

/* Algorithm 1 (Approach; Problem Formulation Eq. 1-3), host only.
 *   t_iter  host [N] per-worker iteration times in integer ticks, >= 1;
 *   M       bound on floor(T/min t) - floor(T/max t), >= 1;
 *   T_star  out: chosen barrier;  tau  out host [N]: floor(T_star / t_iter[i]).
 * Scans T = max t, max t + 1, ... while the constraint holds, keeps the first
 * T of least maximal wait, and stops early at the first zero wait.
 * OSCARS_E_INFEASIBLE if the constraint already fails at T = max t. */
oscars_status oscars_load_balance(const int64_t* t_iter, int32_t N, int64_t M, int64_t* T_star,
                                  int32_t* tau);

/* The load-balancing controller's plan from measured iteration times
 * (Problem Formulation: each worker's iteration time is steady; Approach: the
 * global view measures them and runs Algorithm 1), host only.
 *   t_measured  host [N] per-worker iteration times, finite and > 0, any one
 *               unit (e.g. milliseconds);
 *   resolution  1 <= R <= OSCARS_MAX_RESOLUTION: the tick is min(t) / R, so
 *               the fastest worker takes R ticks;
 *   ticks       out host [N] or NULL: t_i in ticks, max(1, floor(t_i / tick + 0.5));
 *   M, T_star, tau as oscars_load_balance, which then runs on the ticks.
 * OSCARS_E_INVALID for a bad time, resolution, or a time above
 * OSCARS_MAX_TICKS ticks; OSCARS_E_INFEASIBLE as oscars_load_balance.
 * The scan of Algorithm 1 grows with R: it ends within about M * R ticks. */
#define OSCARS_MAX_RESOLUTION 4096
#define OSCARS_MAX_TICKS 1073741824
oscars_status oscars_plan_tau(const double* t_measured, int32_t N, int32_t resolution, int64_t M,
                              int64_t* ticks, int64_t* T_star, int32_t* tau);

/* Eq. 4 weights, host only: w[k] = 1/K as fp32 for every k.  `staleness`
 * (host [K], may be NULL) is accepted and has no effect: the update rule
 * averages uniformly. */
oscars_status oscars_paper_weights(const int32_t* staleness, int32_t K, float* w);

/* Contiguous shards, host only: offsets[k] = floor(k * n_rows / K), k = 0..K. */
oscars_status oscars_shard_offsets(int64_t n_rows, int32_t K, int64_t* offsets);

/* Mini-batch rows of worker k, host only.  Worker k draws its shard without
 * replacement, epoch by epoch; sample number p = step * batch + b lies in
 * epoch e = p / n_k at position p mod n_k; the epoch-e order is a Durstenfeld
 * shuffle of 0..n_k-1 (i from n_k-1 down to 1, j = r mod (i+1)) driven by
 * SplitMix64 started at seed ^ ((k << 32) | e).
 *   rows_out  host [steps][batch]: global row indices for steps
 *             first_step .. first_step + steps - 1. */
oscars_status oscars_sample_indices(const oscars_shards* shards, int32_t K, int32_t k,
                                    int64_t first_step, int32_t steps, int32_t batch,
                                    int64_t* rows_out);

/* Local SGD of Eq. 4 (second branch) for every worker, batched on the GPU.
 * Allocates no device memory unless some worker runs more than 64 steps in
 * one call (the index table then grows, once, after waiting for the stream).
 *   replicas  device [K][oscars_num_params] fp32 master parameters, one replica
 *             per worker, 16-byte aligned; updated in place;
 *   shards    training data and shards (K + 1 offsets);
 *   tau       host [K]: worker k runs tau[k] >= 0 steps (0 leaves replica k
 *             untouched); at most 4096;
 *   lr        learning rate eta, finite and > 0;
 *   batch     mini-batch size, 1 <= batch <= max_batch of the context.
 * Worker k continues its sample stream where its previous call stopped (its
 * cursor advances by tau[k]).  Replicas with tau[k] <= j get no work in step j.
 * The batches' rows are drawn on the host and uploaded from a staging buffer
 * that the next call reuses: a call first waits until the stream has run the
 * previous call's upload (the host stays at most one call ahead).  Hence
 * OSCARS_E_STATE, with no side effects, when the context's stream is being
 * captured into a graph. */
oscars_status oscars_local_steps(oscars_ctx* ctx, float* replicas, const oscars_shards* shards,
                                 const int32_t* tau, float lr, int32_t batch);

/* One round of Eq. 4 (Approach): every worker starts from the global model,
 * runs its tau[k] local SGD steps (as oscars_local_steps), and the parameter
 * server's average of the K results becomes the new global model (as
 * oscars_aggregate with broadcast = 0, n = ld = oscars_num_params).
 *   global    device [oscars_num_params] fp32, in: the model every worker
 *             starts from (the workers' pull), out: the average; 16-byte
 *             aligned, not overlapping replicas;
 *   replicas  device [K][oscars_num_params] fp32, out: the workers' models at
 *             the barrier, before averaging (their previous contents are not
 *             read; a worker with tau[k] = 0 gets a copy of the start model);
 *   weights   host [K] fp32, finite.
 * Equivalent to copying global into every replica, oscars_local_steps and
 * oscars_aggregate(global, replicas, weights, K, n, n, 0), bit for bit, but
 * without writing K copies of the model: the first step reads the global
 * model directly.  Waits for the previous upload, and refuses a stream being
 * captured into a graph (OSCARS_E_STATE), as oscars_local_steps. */
oscars_status oscars_round(oscars_ctx* ctx, float* global, float* replicas,
                           const oscars_shards* shards, const int32_t* tau, float lr,
                           int32_t batch, const float* weights);

/* Mean training loss of each worker over its steps in the last
 * oscars_local_steps or oscars_round call (NaN for a worker that ran no step).  Waits for the
 * context's stream.  losses: host [K]. */
oscars_status oscars_round_losses(oscars_ctx* ctx, float* losses);

/* Held-out evaluation of one model (the convergence measure of Evaluation:
 * loss and accuracy of the trained classifier).  The forward pass of the
 * local steps (same GEMMs, same rounding points) over rows 0 .. n_rows-1 of
 * x, max_batch rows at a time, on the context's stream:
 *   params    device [n_pad] fp32, flat layout (e.g. the global model);
 *   x, y      device, as in oscars_shards (dtype of the model);
 *   n_rows    1 <= n_rows <= 2^31 - 65;
 *   loss_sum  out: summed softmax cross-entropy (fp32 per row, summed on the
 *             GPU in double in a fixed order: 256 contiguous runs of rows,
 *             each in row order, the run sums left to right);
 *   correct   out: rows whose label's logit is the largest (ties count).
 * Uses the context's activation workspace (not the losses of the last
 * local steps), allocates and frees temporary device buffers (the row
 * table, per-row losses and flags: 12 bytes per row), times GEMM tilings
 * the context has not decided yet, and waits for the stream.  Not for a
 * stream being captured into a graph. */
oscars_status oscars_evaluate(oscars_ctx* ctx, const float* params, const void* x,
                              const int32_t* y, int64_t n_rows, double* loss_sum,
                              int64_t* correct);

/* oscars_evaluate for callers that cannot allocate device memory: serving
 * loops that evaluate a model over and over, code that must not call
 * hipMalloc / hipFree (e.g. next to a graph being captured on another
 * stream), harnesses that forbid allocation.  Same arguments and the same
 * results, bit for bit, as oscars_evaluate; it differs in three ways:
 *   - its temporaries (row table, per-row losses and flags, results) live in
 *     one library-wide device array of about 3 MB per GPU, set aside when the
 *     first context on that GPU is created and held until the process ends,
 *     so n_rows <= OSCARS_EVAL_NOALLOC_MAX_ROWS (else OSCARS_E_INVALID);
 *   - it allocates nothing and creates no HIP objects: GEMM tilings the
 *     context has not decided yet take the fixed rule instead of being timed
 *     (every tiling gives the same bits);
 *   - every call on one GPU shares that array: calls that overlap on one GPU
 *     (two host threads, or two contexts on different streams) race and
 *     their results are undefined.  The call waits for the context's
 *     stream before it returns, so calls from one thread never overlap.
 * OSCARS_E_STATE if the current device is not the context's. */
#define OSCARS_EVAL_NOALLOC_MAX_ROWS 262144
oscars_status oscars_evaluate_noalloc(oscars_ctx* ctx, const float* params, const void* x,
                                      const int32_t* y, int64_t n_rows, double* loss_sum,
                                      int64_t* correct);

/* Parameter-server aggregation (Approach, Eq. 4, first branch).
 *   global    device [n] fp32 out: g[i] = sum_k w_k * replicas[k * ld + i],
 *             summed as a balanced pairwise tree over P = next power of two
 *             >= K leaves (leaf k = fl(w_k * x_k[i]) for k < K, +0 otherwise;
 *             each node fl(left + right)); with K a power of two and
 *             w_k = 1/K the result is exact up to that tree's roundings;
 *   replicas  device [K][ld] fp32; if broadcast != 0 every replica is
 *             overwritten with g after the reduction (replicas[k*ld + i] = g[i]
 *             for i < n); otherwise only read;
 *   weights   host [K] fp32 (oscars_paper_weights gives the paper's 1/K);
 *   K         1 <= K <= OSCARS_MAX_K;  n >= 1;  ld >= n, ld % 4 == 0;
 *   global and replicas 16-byte aligned and not overlapping. */
oscars_status oscars_aggregate(float* global, float* replicas, const float* weights, int32_t K,
                               int64_t n, int64_t ld, int32_t broadcast, void* hip_stream);

/* Broadcast of the global model to every worker (Approach, Eq. 4: after the
 * average every worker continues from it):
 *   replicas[k * ld + i] = global[i] for k < K, i < n, non-temporal stores;
 *   the same K, n, ld rules, alignment and no-overlap requirement as
 *   oscars_aggregate.  oscars_round needs no broadcast (its workers start
 *   from the global model itself); this is the separate step for callers
 *   that keep K materialised replicas.  With K = 1 it is a plain copy. */
oscars_status oscars_broadcast(const float* global, float* replicas, int32_t K, int64_t n,
                               int64_t ld, void* hip_stream);

/* Resume support: per-worker count of local steps done so far. host [K]. */
oscars_status oscars_get_cursors(const oscars_ctx* ctx, int64_t* steps_done);
oscars_status oscars_set_cursors(oscars_ctx* ctx, const int64_t* steps_done);

/* Per-kernel timing with HIP events recorded on the context's stream around
 * every launch of the selected kernel kinds (bit mask of 1 << OSCARS_KERNEL_*).
 * oscars_profile_end waits for the stream and returns, per kind, the summed
 * milliseconds and the number of launches since oscars_profile_begin
 * (host [OSCARS_KERNEL_COUNT] each). */
enum {
  OSCARS_KERNEL_CAST = 0,
  OSCARS_KERNEL_FWD = 1,
  OSCARS_KERNEL_SOFTMAX = 2,
  OSCARS_KERNEL_DGRAD = 3,
  OSCARS_KERNEL_WGRAD = 4,
  OSCARS_KERNEL_AGGREGATE = 5, /* the aggregation inside oscars_round */
  OSCARS_KERNEL_BWD_FUSED = 6, /* backward-data + backward-weight + update, one launch */
  OSCARS_KERNEL_COUNT = 7
};
oscars_status oscars_profile_begin(oscars_ctx* ctx, uint32_t kind_mask);
oscars_status oscars_profile_end(oscars_ctx* ctx, double* ms, int64_t* launches);

/* Tiling of the forward and backward-data GEMMs of one context (a tuning and
 * testing aid).  Every tiling sums each output in the same order (K in
 * chunks of 1024 summed left to right), so results are bit-identical
 * whatever the tiling; only the speed differs.
 *   OSCARS_TILING_AUTO (default): the launches of each GEMM configuration
 *     (layer shape, batch, number of active replicas) in the process are
 *     tuned online: while the configuration is being tuned, each launch runs
 *     one feasible tiling between two events on the stream (two timed
 *     launches per tiling, read later without waiting), after which the
 *     tiling with the fastest launch is kept (oscars_tuning_pending counts the
 *     configurations still being tuned); while the stream is being captured
 *     into a graph
 *     a fixed rule chooses instead.
 *   L, M, S: 128 x 128, 64 x 128, 64 x 64 output tiles; LS: 128 x 128 with
 *     the K chunks split over workgroups (more than one K chunk);
 *   W: 128 x 256 (bf16 models, batches above 128); WS, VS: 128 x 256 and
 *     64 x 256 with the K chunks split over workgroups (bf16, batches above
 *     128, more than one K chunk) -- where a forced tiling does not apply, W
 *     or L is used.
 * Every call (AUTO included) restarts the tuning of every configuration.
 * Returns OSCARS_E_INVALID for a value outside [0, OSCARS_TILING_COUNT). */
enum {
  OSCARS_TILING_AUTO = 0,
  OSCARS_TILING_L = 1,
  OSCARS_TILING_M = 2,
  OSCARS_TILING_S = 3,
  OSCARS_TILING_W = 4,
  OSCARS_TILING_WS = 5,
  OSCARS_TILING_VS = 6,
  OSCARS_TILING_LS = 7,
  OSCARS_TILING_COUNT = 8
};
oscars_status oscars_set_gemm_tiling(oscars_ctx* ctx, int32_t tiling);

/* Number of forward / backward-data GEMM configurations of this context
 * whose tiling OSCARS_TILING_AUTO is still tuning (seen at least once, not
 * yet decided), into *configurations.  A caller that times the steady state
 * runs rounds until it reads 0.  Returns OSCARS_E_INVALID for a null
 * pointer. */
oscars_status oscars_tuning_pending(const oscars_ctx* ctx, int32_t* configurations);

/* Backward pass of the layers of a bf16 model, per context (a tuning and
 * testing aid).  By default one launch per hidden layer (l >= 2) does
 * backward-data, backward-weight and the SGD update of Eq. 4 (Approach): it
 * rounds the fp32 master it streams for the update to the bf16 weights the
 * forward pass used, so backward-data reads no weights of its own.  Layer 1
 * (no backward-data) may take the same streamed launch for backward-weight
 * and the update alone.  The results are bit-identical to the separate
 * backward-data and update launches, whichever mode runs (a weight that is
 * exactly -0 may come out as +0 in one and -0 in the other).  The bias
 * gradient of every update sums the batch in blocks of 64 rows, block sums
 * left to right.
 *   OSCARS_BACKWARD_AUTO (default): the fastest at the first launch of the
 *     configuration (inputs, outputs, batch, active replicas, layer 1 or
 *     hidden) in this context of: the fused launch with each feasible
 *     number of 1024-output chunks per workgroup (all; then half, a quarter,
 *     ... down to one, where the context's partial buffer holds the split;
 *     layer 1 needs no partials), and the separate launches.  Each runs
 *     three times there on the scratch replicas oscars_create allocated, the
 *     faster of its last two runs counting; a later candidate is taken only
 *     when it is more than 5% faster than the earlier pick (the separate
 *     update comes first for layer 1, last for the hidden layers).
 *     Untimed -- on a stream being captured into a graph, or where
 *     oscars_create left the scratch out --: fused, split over the number of
 *     workgroups per 64-wide input strip that fills the last pass over the
 *     CUs best (the fewest on ties);
 *   OSCARS_BACKWARD_SEPARATE: backward-data and update launches;
 *   OSCARS_BACKWARD_FUSED: fused, never split;
 *   OSCARS_BACKWARD_FUSED_SPLIT: fused, split wherever there is more than one
 *     chunk of output features and the context's partial buffer holds them.
 * Fusion applies to batches of at most 256 rows; larger batches always use
 * the separate launches.  Returns OSCARS_E_INVALID for a value outside
 * [0, OSCARS_BACKWARD_COUNT). */
enum {
  OSCARS_BACKWARD_AUTO = 0,
  OSCARS_BACKWARD_SEPARATE = 1,
  OSCARS_BACKWARD_FUSED = 2,
  OSCARS_BACKWARD_FUSED_SPLIT = 3,
  OSCARS_BACKWARD_COUNT = 4
};
oscars_status oscars_set_backward(oscars_ctx* ctx, int32_t mode);

/* The backward path of layer `layer` (1..L) in oscars_local_steps and
 * oscars_round of this context with `replicas` active replicas (1..K) and
 * batch `batch` (1..max_batch): *fused = 1 for the fused launch of
 * backward-data (none for layer 1), backward-weight and update, 0 for the
 * separate launches (always for fp32 MLPs, OSCARS_BACKWARD_SEPARATE,
 * batches above 256 and layers whose input width is not a multiple of 8),
 * -1 where OSCARS_BACKWARD_AUTO times configurations and has not timed that
 * one in this context yet.  Convolutional contexts: 1 where backward-data
 * and backward-weight of a conv layer (2..L-1, channel counts multiples of
 * 4) share one launch (the updates follow in their own launch), else 0.
 * Returns OSCARS_E_INVALID for an argument out of range. */
oscars_status oscars_backward_path(const oscars_ctx* ctx, int32_t layer, int32_t batch,
                                   int32_t replicas, int32_t* fused);

const char* oscars_status_str(oscars_status s);
/* HIP error code of the last OSCARS_E_HIP in this thread (0 if none). */
int32_t oscars_last_hip_error(void);

#ifdef __cplusplus
}
#endif

#endif /* OSCARS_H */
