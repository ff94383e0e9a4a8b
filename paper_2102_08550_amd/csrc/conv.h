// Launchers of the convolutional workload's kernels (device code in
// conv_kernels.hip): 3 x 3 convolutions with padding 1 as implicit GEMMs on
// fp32 MFMA, global average pooling, and the linear classifier, grouped over
// the active replica slots like the fully connected kernels.
#pragma once

#include <hip/hip_runtime.h>

#include <cstdint>

namespace oscars {

enum ConvPass {
  CONV_FWD = 0,    // Z[p][o] = b[o] + sum_{r,s,c} in[tap(p, r, s)][c] W[o][r][s][c]; ReLU
  CONV_DGRAD = 1,  // dIn[q][c] = sum_{r,s,o} dZ[p(q, r, s)][o] W[o][r][s][c] where mask > 0
  CONV_WGRAD = 2,  // dW[o][r][s][c] = sum_p dZ[p][o] in[tap(p, r, s)][c]; db[o] = sum_p dZ[p][o]
  FC_FWD = 3,      // logits[b][o] = bias[o] + sum_c pooled[b][c] W[o][c]
  FC_DGRAD = 4,    // dpooled[b][c] = sum_o delta[b][o] W[o][c]
  FC_WGRAD = 5     // dW[o][c] = sum_b delta[b][o] pooled[b][c]; db[o] = sum_b delta[b][o]
};

// One grouped launch over n_slots replica slots (slot z works on replica
// order[z]).  Every per-slot pointer is the slot-0 address; the kernel adds z
// (activations, gradients, partials) or order[z] (parameters) times its
// stride.  Layouts: images and activations [batch][H][W][C] fp32 (channels
// fastest); conv weights [Cout][3][3][Cin], classifier weights
// [classes][channels], each followed by its bias, at w_off / b_off of the
// flat replica.
struct ConvArgs {
  int B;                  // batch rows
  int H, W, C;            // the layer's input (FC: C = pooled channels, H = W = 1)
  int Ho, Wo, Co;         // the layer's output (FC: Co = classes)
  int stride;             // 1 or 2 (conv)
  int cls;                // CONV_DGRAD with stride 2: parity class of the input pixels, 2 (hi & 1)
                          // + (wi & 1), or -1 for all four classes in one launch (see
                          // conv_kernels.hip)
  const float* in;        // conv input [B][H][W][C] (or, with gather, dataset rows); FC: pooled
  int64_t in_slot, in_ld;             // slot stride; row stride of a gathered dataset row
  const int32_t* gather;  // layer 1: dataset row of each batch row, [slot] stride gather_slot
  int64_t gather_slot;
  const float* dout;      // DGRAD / WGRAD: gradient of the layer output [B][Ho][Wo][Co]
  int64_t dout_slot, dout_ld;         // FC: delta [B][dout_ld]
  const float* master_in; // parameters read (weights; bias in FWD), by order[z]
  int64_t master_in_slot;
  int64_t w_off, b_off;
  float* out;             // FWD: activations (FC: logits [B][out_ld]); DGRAD: gradient of the input
  int64_t out_slot, out_ld;
  const float* mask;      // CONV_DGRAD: the input activation (ReLU mask, > 0)
  int64_t mask_slot;
  const float* skip;      // residual shortcut or nullptr: CONV_FWD adds skip[p][o] to Z before
  int64_t skip_slot;      // the ReLU (the block's input); CONV_DGRAD adds skip[q][c] to the
                          // input gradient before the mask (the gradient at the block's end)
  float* part;            // WGRAD: partial sums [slot][split][Co][N] (launch_conv_updates)
  int64_t part_slot;
  int splits;             // WGRAD: number of K ranges (of output pixels, output rows of layers
  int64_t k_per_split;    // with at most 3 input channels, or batch rows; conv_wgrad_ranges)
  const int32_t* order;
};

hipError_t launch_conv(const ConvArgs& a, ConvPass pass, int n_slots, hipStream_t s);

// CONV_DGRAD of d and CONV_WGRAD of w (the same layer; each as launch_conv
// takes it) in one launch, where that applies: channel counts multiples of 4
// and no gathered rows (conv_pair_fits; otherwise hipErrorInvalidValue and
// nothing launched).
bool conv_pair_fits(const ConvArgs& d, const ConvArgs& w, int n_slots);
hipError_t launch_conv_pair(const ConvArgs& d, const ConvArgs& w, int n_slots, hipStream_t s);

// Output pixels per weight-gradient range of the 64 x 64 conv tiles.
constexpr int CONV_WGRAD_PIXELS = 256;

// The K ranges a CONV_WGRAD launch of these sizes expects (ConvArgs.splits,
// ConvArgs.k_per_split): ranges of CONV_WGRAD_PIXELS output pixels, or, for
// layers with at most three input channels whose staged input rows fit a
// workgroup's LDS, of whole output rows (as many as fill 512 pixel slots of
// the row width rounded up to 32).
void conv_wgrad_ranges(const ConvArgs& a, int* splits, int64_t* k_per_split);


// pooled[z][b][c] = (sum over the H W positions of act[z][b][.][c]: eight
// groups of consecutive positions, each in position order, the group sums in
// order) / (H W).
hipError_t launch_avgpool(const float* act, int64_t act_slot, float* pooled, int64_t pooled_slot,
                          int B, int HW, int C, int n_slots, hipStream_t s);
// dZ[z][b][p][c] = dpooled[z][b][c] / (H W) where act[z][b][p][c] > 0, else 0.
hipError_t launch_avgpool_backward(const float* dpooled, int64_t dpooled_slot, const float* act,
                                   int64_t act_slot, float* dz, int B, int HW, int C,
                                   int n_slots, hipStream_t s);

// The classifier head of one local step (average pooling, linear classifier,
// softmax cross-entropy, the classifier's backward-data and the pooling
// backward), grouped over slots like ConvArgs: slot z uses the parameters of
// replica order[z].
struct HeadArgs {
  int B, HW, C, classes;          // batch rows, positions and channels of the last conv
                                  // layer's output, classes
  const float* act;               // that output [B][HW][C] (after ReLU), slot stride act_slot
  int64_t act_slot;
  const float* master_in;         // parameters read, by order[z]: classifier W [classes][C]
  int64_t master_in_slot;         // at w_off, its bias at b_off
  int64_t w_off, b_off;
  const int32_t* order;
  const int32_t* y;               // labels of the dataset rows
  const int32_t* gather;          // dataset row of each batch row, [slot] stride gather_slot
  int64_t gather_slot;
  float* pooled;                  // out: pooled[b][c], slot stride pooled_slot
  int64_t pooled_slot;
  float* delta;                   // out: logit gradient [b][delta_ld], slot stride delta_slot
  int64_t delta_slot, delta_ld;
  float* loss;                    // out: per-row loss, slot stride loss_slot
  int64_t loss_slot;
  float* dz;                      // out: gradient at the last conv output [B][HW][C]
  int64_t dz_slot;
};

// Whether the head of these sizes fits one workgroup's LDS (else the
// separate pooling, classifier and softmax launches are used).
bool conv_head_fits(int HW, int C, int classes);

// Forward and backward of the head up to the last conv output's gradient,
// one workgroup per (slot, batch row): pooled, logits, loss, delta (the
// classifier's input to its weight gradient) and dz.
hipError_t launch_conv_head(const HeadArgs& h, int n_slots, hipStream_t s);

// One layer's parameters for launch_conv_updates: W [M][N - 1] at w_off and
// the bias [M] at b_off of the flat replica, and their gradient as
// weight-gradient partials [slot][split][M][N] (bias last; slot stride
// part_slot), or, with part == nullptr, the classifier's gradient formed from
// HeadArgs' pooled and delta (M = classes, N = C + 1).
struct UpdateBlock {
  const float* part;
  int64_t part_slot;
  int splits, M, N;
  int64_t w_off, b_off;
};
constexpr int MAX_UPDATE_BLOCKS = 4;

// The SGD updates of up to MAX_UPDATE_BLOCKS layers in one launch (after every
// backward-data launch that reads their weights): each gradient summed in a
// fixed order (partials: eight groups of consecutive ranges, each in range
// order, the group sums in order; the classifier's: eight groups of
// consecutive batch rows likewise), then master[order[z]] <- master_in - lr
// gradient (master_in likewise by order[z]).
hipError_t launch_conv_updates(const UpdateBlock* blocks, int n_blocks, const HeadArgs* head,
                               const float* master_in, int64_t master_in_slot, const int32_t* order,
                               float* master, int64_t master_slot, float lr, int n_slots,
                               hipStream_t s);

}  // namespace oscars
