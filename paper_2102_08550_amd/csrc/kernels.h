// Launchers of the hot-path kernels (device code in kernels.hip).
#pragma once

#include <hip/hip_runtime.h>

#include <cstdint>

namespace oscars {

enum GemmMode { GEMM_FWD = 0, GEMM_DGRAD = 1, GEMM_WGRAD = 2 };

// Forward and backward-data sum K in chunks of this many elements (each
// chunk from zero, chunk sums left to right); a split-K launch has one
// partial per chunk.
constexpr int GEMM_KCHUNK = 1024;

// One grouped GEMM launch over `n_slots` replicas (grid y = slot).  Slot z
// works on replica order[z].  Every per-slot pointer is the slot-0 address;
// the kernel adds z (or order[z] where *_by_order is set) times its stride.
// C[m][n] = sum_k A(m, k) B(n, k); the M side is always a weight dimension so
// that each lane's four consecutive accumulator rows are four consecutive
// elements in memory (weights and activations are both stored with the
// feature index fastest).
//
//   FWD   C[o][b] = sum_i W[o][i] act[b][i];  out[b][o] = C + bias[o]
//         (ReLU if relu).  A = W [M=out][K=in]; B = act [N=batch][K=in]
//         (b_ld), or dataset rows x[gather[b]] when gather != nullptr, which
//         are then also copied to rows_out.
//   DGRAD C[i][b] = sum_o W[o][i] D[b][o];  out[b][i] = C where
//         mask[b][i] > 0, else 0.  A = W as [K=out][M=in]; B = D [N=batch][K=out].
//   WGRAD C[i][o] = sum_b act[b][i] D[b][o] = dW[o][i];  W <- W - lr dW
//         (fp32 master), bias[o] <- bias[o] - lr sum_b D[b][o], bf16 copy of
//         W refreshed if wcopy.  A = act as [K=batch][M=in] (layer 1: the
//         rows the forward pass gathered); B = D as [K=batch][N=out].
struct GemmArgs {
  int M, N, K;
  // Chunked extent of each operand's contiguous dimension (K for a
  // K-contiguous operand, M or N otherwise): a multiple of 8 elements, with
  // readable (zero) padding between the logical size and the extent.
  int a_ext, b_ext;
  const void* a;  // operand A (FWD, DGRAD: weights; WGRAD: activations / x)
  int64_t a_ld, a_slot;
  int a_by_order;  // a's slot offset uses order[z] (fp32 masters) instead of z
  const void* b;  // operand B (FWD: activations / x; DGRAD, WGRAD: delta)
  int64_t b_ld, b_slot;
  const int32_t* gather;  // FWD layer 1: dataset rows of the batch (B rows)
  int64_t gather_slot;
  void* rows_out;  // FWD layer 1: the gathered rows, [batch][rows_out_ld] per slot
  int64_t rows_out_ld, rows_out_slot;
  void* out;  // FWD: activations or logits; DGRAD: delta of the layer below
  int64_t out_ld, out_slot;
  const void* mask;  // DGRAD: activations of the layer below
  int64_t mask_ld, mask_slot;
  float* master;  // fp32 replicas written by WGRAD (by order[z])
  int64_t master_slot;  // replica stride
  // fp32 parameters read: the bias in FWD, W and bias in WGRAD.  Normally the
  // replicas themselves (master_in = master); in the first local step of a
  // round that starts from the global model, the global model with stride 0.
  const float* master_in;
  int64_t master_in_slot;
  int64_t w_off, b_off;  // W_l and b_l offsets within a replica
  uint16_t* wcopy;  // WGRAD, bf16 models: slot-indexed bf16 weight copies
  int64_t wcopy_slot;
  int wcopy_slots;  // WGRAD: only slots z < wcopy_slots refresh their copy (the
                    // others take their last local step: nothing reads it)
  // FWD / DGRAD split-K partials: fp32 [slot][chunk][N][out_ld], capacity
  // part_cap floats (nullptr or too small: no split).  part_slot is set by the
  // launcher.
  float* part;
  int64_t part_cap, part_slot;
  const int32_t* order;  // [slots] replica id of each slot
  float lr;
  int relu;  // FWD: apply ReLU
  int out_bf16;  // FWD / DGRAD: store bf16 (else fp32)
};

// The tiling state of one context (forced tiling, online tuning, choices).
struct GemmTuner;
GemmTuner* gemm_tuner_create();  // nullptr when out of host memory
void gemm_tuner_destroy(GemmTuner* t);

// tuner: the context's tiling state (nullptr: the fixed rule, nothing timed);
// tune = false: nothing is timed and no event is created -- a configuration
// the tuner has decided keeps its choice, any other takes the fixed rule.
hipError_t launch_gemm(const GemmArgs& g, GemmMode mode, bool bf16, int n_slots, hipStream_t s,
                       GemmTuner* tuner, bool tune = true);

// Forward / backward-data tilings (backward-weight always uses one):
//   L 128 x 128, M 64 x 128, S 64 x 64 (register-staged operands), and LS,
//   L split over K chunks;
//   W 128 x 256 and, split over K chunks, WS (128 x 256) and VS (64 x 256)
//   (bf16, batches above 128, operands streamed into LDS).
// AUTO tunes each configuration online: its launches run the feasible
// tilings in turn, timed (two launches each), until the fastest is kept.
// Any other value forces that tiling where it applies (L for LS without
// room for the partials, W for another infeasible split, L where no
// whole-batch tiling applies).
enum GemmTiling {
  GEMM_TILING_AUTO = 0,
  GEMM_TILING_L = 1,
  GEMM_TILING_M = 2,
  GEMM_TILING_S = 3,
  GEMM_TILING_W = 4,
  GEMM_TILING_WS = 5,
  GEMM_TILING_VS = 6,
  GEMM_TILING_LS = 7,
  GEMM_TILING_COUNT = 8
};
void gemm_tuner_set_tiling(GemmTuner* t, int tiling);
// Configurations whose AUTO tiling is still being tuned by this tuner.
int gemm_tuner_pending(GemmTuner* t);
// While on (for the calling thread), an AUTO configuration not decided yet is
// decided at its next launch: every feasible tiling timed there and then, the
// fastest kept (for launches that are themselves being timed).
void set_gemm_tune_now(bool on);

// Backward pass of a hidden layer (l >= 2) of a bf16 model in one launch:
// backward-data, backward-weight and the SGD update, with the arguments of
// the backward-data launch plus those of the update (master, master_in,
// w_off, b_off, wcopy, lr):  M = inputs, N = batch, K = outputs; a = the
// activations of the layer below [N][a_ld] (also the ReLU mask), b = delta
// [N][b_ld], out = the delta of the layer below.  Same results, bit for
// bit, as GEMM_DGRAD followed by GEMM_WGRAD (but for the sign of a weight
// that is exactly -0).  Batches of at most 256 rows, inputs a multiple of 8,
// W_l within 32-bit buffer offsets (backward_fusable).
bool backward_fusable(const GemmArgs& g);
bool backward_fused_enabled(int mode);
// mode: the context's BackwardMode; cps_forced > 0: each workgroup covers
// that many KCHUNK ranges of outputs (all of them where the partial buffer
// cannot hold the split); 0: by mode.  dgrad = false: backward-weight and the
// update only, for layer 1 (GEMM_WGRAD's operands: a = the gathered input
// rows, b = delta; out, mask and part unused), the same results as
// GEMM_WGRAD bit for bit (but for the sign of a weight that is exactly -0).
hipError_t launch_bwd_fused(const GemmArgs& g, int n_slots, hipStream_t s, int mode,
                            int cps_forced = 0, bool dgrad = true);
// The feasible ranges per workgroup (all chunks first, then halving down to
// one), at most `max` of them written to cps; returns their number.
int bwd_fused_splits(const GemmArgs& g, int n_slots, int* cps, int max, bool dgrad = true);
// Backward of hidden bf16 layers (a per-context setting): AUTO (fused, the
// o chunks split over the workgroup count that best fills the last CU pass,
// or the separate launches, whichever the caller timed faster for the
// configuration),
// SEPARATE (backward-data and update kernels), FUSED (never split),
// FUSED_SPLIT (one chunk per workgroup wherever there is more than one chunk
// and the partial buffer holds them).
enum BackwardMode { BACKWARD_AUTO = 0, BACKWARD_SEPARATE = 1, BACKWARD_FUSED = 2,
                    BACKWARD_FUSED_SPLIT = 3, BACKWARD_MODE_COUNT = 4 };

// Softmax cross-entropy on logits [slot][B][ld]: delta = (softmax - onehot)/B
// stored as bf16 or fp32 into delta [slot][B][ld] (columns C..ld-1 zeroed),
// per-row loss into loss[slot][B]; if correct != nullptr, correct[slot][B] =
// 1 where the label's logit is the largest (ties count), else 0.
hipError_t launch_softmax_ce(const float* logits, int64_t ld, int64_t slot_stride, int C, int B,
                             const int32_t* y, const int32_t* gather, int64_t gather_slot,
                             void* delta, bool delta_bf16, float* loss, int64_t loss_slot,
                             int n_slots, hipStream_t s, int32_t* correct = nullptr);

// wcopy[z][i] = bf16(master[order[z]][i]) for i < n, z < n_slots.
hipError_t launch_cast_bf16(const float* master, int64_t master_slot, const int32_t* order,
                            uint16_t* wcopy, int64_t wcopy_slot, int64_t n, int n_slots,
                            hipStream_t s);

// Held-out evaluation: the row table [64 slot entries = 0][i = 0 .. n-1]
// that the forward pass gathers through, and the reduction of the per-row
// losses (double: 256 contiguous runs of rows, each in row order, the run
// sums left to right) and correct flags (int64) into *out_loss, *out_hits.
hipError_t launch_eval_rows(int32_t* table, int64_t n, hipStream_t s);
hipError_t launch_eval_reduce(const float* loss, const int32_t* hit, int64_t n, double* out_loss,
                              int64_t* out_hits, hipStream_t s);

// replicas[k * ld + i] = g[i] for k < K, i < n (non-temporal stores).
hipError_t launch_broadcast(const float* g, float* replicas, int K, int64_t n, int64_t ld,
                            hipStream_t s);

// Pairwise-tree weighted K-way reduction with optional broadcast.
hipError_t launch_aggregate(float* g, float* replicas, const float* w, int K, int64_t n,
                            int64_t ld, int broadcast, hipStream_t s);

}  // namespace oscars
