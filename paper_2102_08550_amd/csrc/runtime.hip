// Context, workspace and round scheduler of the Oscars hot path.
//
// oscars_local_steps runs Eq. 4's second branch for all K workers at once:
// workers are sorted by tau (descending, ties by index) into slots, so the
// workers still running in local step j are the slot prefix
// {z : tau[order[z]] > j}.  Each step launches, for that prefix only,
// forward GEMMs, softmax cross-entropy, and per layer (top down) the
// backward-data GEMM followed by the backward-weight GEMM with the fused SGD
// update.  Workers whose tau is used up get no work and no writes: the GPU
// counterpart of the idle time before the barrier (Eq. 1).
#include <hip/hip_runtime.h>

#include <algorithm>
#include <array>
#include <cmath>
#include <cstring>
#include <map>
#include <mutex>
#include <new>
#include <vector>

#include "../../include/oscars.h"
#include "conv.h"
#include "host_logic.h"
#include "kernels.h"

using namespace oscars;

namespace {

thread_local int32_t g_last_hip = 0;

oscars_status hip_fail(hipError_t e) {
  g_last_hip = static_cast<int32_t>(e);
  return OSCARS_E_HIP;
}

int64_t round_up(int64_t v, int64_t a) { return (v + a - 1) / a * a; }

bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

constexpr int kMaxTau = 4096;
// Index-table, loss and staging capacity allocated by oscars_create: rounds
// of up to this many local steps per worker need no allocation later.
constexpr int kPreTau = 64;
// Backward path timing: how much faster a later candidate must be to be taken.
constexpr float kBackwardMargin = 0.05f;

}  // namespace

// Device memory of oscars_evaluate_noalloc: the temporaries of one
// evaluation of up to OSCARS_EVAL_NOALLOC_MAX_ROWS rows (results, row table,
// per-row losses and flags; EvalLayout below), one copy per GPU, held until
// the process ends.  Host code never uses this name as an address: it takes
// the device address each GPU reports for it (scratch_address).
constexpr size_t kNoAllocScratchBytes =
    256 + (64 + OSCARS_EVAL_NOALLOC_MAX_ROWS) * 4 + 2 * OSCARS_EVAL_NOALLOC_MAX_ROWS * 4;
static_assert(OSCARS_EVAL_NOALLOC_MAX_ROWS % 64 == 0, "whole 256-byte parts");
static __device__ __align__(256) unsigned char scratch[kNoAllocScratchBytes];

namespace {

std::mutex g_scratch_mu;
std::map<int, void*> g_scratch_ptr;  // device -> address of `scratch` there

// The address of `scratch` on `device`, which must be the current device;
// looked up once per device.
hipError_t scratch_address(int device, void** out) {
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  auto it = g_scratch_ptr.find(device);
  if (it != g_scratch_ptr.end()) {
    *out = it->second;
    return hipSuccess;
  }
  void* p = nullptr;
  const hipError_t e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
  if (e != hipSuccess) return e;
  g_scratch_ptr[device] = p;
  *out = p;
  return hipSuccess;
}

}  // namespace

struct oscars_ctx {
  int L = 0;
  std::vector<int32_t> dims;
  bool bf16 = false;
  int K = 0, max_batch = 0;
  hipStream_t stream = nullptr;
  int device = 0;
  std::vector<int64_t> w_off, b_off, ld;  // per layer l = 1..L (index 0 unused for offsets)
  int64_t n_pad = 0;
  size_t esize = 4;  // bytes per activation / delta element

  std::vector<void*> allocs;
  uint16_t* wcopy = nullptr;       // [K][n_pad] bf16 weight copies (bf16 models)
  uint16_t* gq = nullptr;          // [n_pad] bf16 copy of a round's start model (bf16 models)
  std::vector<void*> act;          // act[l], l = 0..L-1: [K][max_batch][ld[l]] (act[0]: batch rows)
  float* logits = nullptr;         // [K][max_batch][ld[L]]
  float* part = nullptr;           // split-K partials of forward / backward-data GEMMs
  int64_t part_cap = 0;            // floats
  std::vector<void*> delta;        // delta[l], l = 1..L: [K][max_batch][ld[l]]
  int32_t* table_dev = nullptr;    // order [64] then index table [slots][tau_max][B]
  int64_t table_cap = 0;           // int32 elements
  float* loss_dev = nullptr;       // [slots][tau_max][B]
  int64_t loss_cap = 0;
  int32_t* pinned = nullptr;       // host staging of table_dev
  int64_t pinned_cap = 0;
  hipEvent_t upload_done = nullptr;
  bool upload_pending = false;

  std::vector<int64_t> cursors;
  std::vector<WorkerSampler> samplers;

  std::vector<int32_t> last_order, last_tau;
  int last_tau_max = 0, last_B = 0;

  // Backward of hidden bf16 layers without a forced mode, per (inputs,
  // outputs, batch, replicas): fused with this many 1024-output chunks per
  // workgroup (> 0), or the separate launches (0); timed at the first launch
  // on scratch replicas (cal_*, allocated then).
  std::map<std::array<int, 5>, int> bwd_fused_choice;  // (M, K, N, replicas, backward-data)
  float* cal_master = nullptr;   // [K][cal_layer] fp32: W_l then b_l
  uint16_t* cal_copy = nullptr;  // [K][cal_w] bf16 copies of W_l
  int32_t* cal_order = nullptr;  // [K] = 0 .. K-1
  int64_t cal_layer = 0, cal_w = 0;
  bool cal_off = false;  // scratch too large for the free device memory: no timing
  hipEvent_t cal_ev[2] = {nullptr, nullptr};

  void* noalloc_scratch = nullptr;   // this device's `scratch` (oscars_evaluate_noalloc)
  // Convolutional model (oscars_create_cnn): conv layers l = 1..L-1, the
  // classifier is layer L.  geometry[l] for l = 0 (the image) .. L-1.
  bool cnn = false;
  std::vector<int> img_h, img_w, img_c, conv_stride;
  std::vector<int> conv_skip;      // conv layer l adds the output of layer l - 2 (l = 1..L-1)
  std::vector<float*> cact, cdz;   // [K][max_batch][h][w][c] per conv layer (1..L-1)
  float* pooled = nullptr;         // [K][max_batch][c of layer L-1]
  float* dpooled = nullptr;
  float* cpart = nullptr;          // weight-gradient partials, one region per layer
  std::vector<float*> cpart_l;     // layer l's region [K][cpart_slot_l[l]] (l = 1..L; L: the
  std::vector<int64_t> cpart_slot_l;  // classifier), kept until the step's updates
  int64_t cnn_slot(int l) const {
    return static_cast<int64_t>(max_batch) * img_h[l] * img_w[l] * img_c[l];
  }

  GemmTuner* tuner = nullptr;        // tiling of this context's GEMM launches
  int backward_mode = BACKWARD_AUTO;  // backward of hidden bf16 layers

  uint32_t prof_mask = 0;
  std::vector<hipEvent_t> ev_pool;
  std::vector<std::pair<int, int>> prof_recs;  // (kind, first event index)

  int64_t act_slot(int l) const { return static_cast<int64_t>(max_batch) * ld[l]; }
};

namespace {

void free_ctx(oscars_ctx* c) {
  if (!c) return;
  (void)hipStreamSynchronize(c->stream);
  for (void* p : c->allocs) (void)hipFree(p);
  if (c->table_dev) (void)hipFree(c->table_dev);
  if (c->loss_dev) (void)hipFree(c->loss_dev);
  if (c->pinned) (void)hipHostFree(c->pinned);
  if (c->upload_done) (void)hipEventDestroy(c->upload_done);
  for (hipEvent_t e : c->cal_ev)
    if (e) (void)hipEventDestroy(e);
  for (hipEvent_t e : c->ev_pool) (void)hipEventDestroy(e);
  gemm_tuner_destroy(c->tuner);
  delete c;
}

hipError_t dev_alloc(oscars_ctx* c, size_t bytes, void** out) {
  void* p = nullptr;
  hipError_t e = hipMalloc(&p, bytes);
  if (e != hipSuccess) return e;
  c->allocs.push_back(p);
  e = hipMemsetAsync(p, 0, bytes, c->stream);
  *out = p;
  return e;
}

// Index table (with host staging) and loss buffer for `need` table entries
// and `loss_need` losses; grows them only when they are too small (waiting
// for the stream first).  On failure the context keeps its old buffers.
hipError_t ensure_tables(oscars_ctx* c, int64_t need, int64_t loss_need) {
  hipError_t e = hipSuccess;
  if (need > c->table_cap || loss_need > c->loss_cap || need > c->pinned_cap) {
    e = hipStreamSynchronize(c->stream);
    if (e != hipSuccess) return e;
    c->upload_pending = false;
  }
  if (need > c->pinned_cap) {
    int32_t* p = nullptr;
    e = hipHostMalloc(reinterpret_cast<void**>(&p), need * sizeof(int32_t));
    if (e != hipSuccess) return e;
    if (c->pinned) (void)hipHostFree(c->pinned);
    c->pinned = p;
    c->pinned_cap = need;
  }
  if (need > c->table_cap) {
    int32_t* p = nullptr;
    e = hipMalloc(reinterpret_cast<void**>(&p), need * sizeof(int32_t));
    if (e != hipSuccess) return e;
    if (c->table_dev) (void)hipFree(c->table_dev);
    c->table_dev = p;
    c->table_cap = need;
  }
  if (loss_need > c->loss_cap) {
    float* p = nullptr;
    e = hipMalloc(reinterpret_cast<void**>(&p), loss_need * sizeof(float));
    if (e != hipSuccess) return e;
    if (c->loss_dev) (void)hipFree(c->loss_dev);
    c->loss_dev = p;
    c->loss_cap = loss_need;
  }
  return hipSuccess;
}

// Scratch replicas on which OSCARS_BACKWARD_AUTO times the backward paths of
// the hidden layers of a bf16 model: K x the widest hidden layer (fp32 W and
// b, bf16 W).  Skipped (no timing: c->cal_off) where it would take more than
// a quarter of the free device memory.
hipError_t alloc_calibration(oscars_ctx* c) {
  if (!c->bf16) return hipSuccess;
  for (int l = 1; l <= c->L; ++l) {
    const int64_t w = static_cast<int64_t>(c->dims[l]) * c->dims[l - 1];
    c->cal_w = std::max(c->cal_w, round_up(w, 8));
    c->cal_layer = std::max(c->cal_layer, round_up(w + c->dims[l], 8));
  }
  size_t free_b = 0, total_b = 0;
  hipError_t e = hipMemGetInfo(&free_b, &total_b);
  if (e != hipSuccess) return e;
  const double need = static_cast<double>(c->K) * (c->cal_layer * 4.0 + c->cal_w * 2.0);
  if (need > static_cast<double>(free_b) / 4.0) {
    c->cal_off = true;
    return hipSuccess;
  }
  void* p = nullptr;
  e = dev_alloc(c, static_cast<size_t>(c->K) * c->cal_layer * 4, &p);
  c->cal_master = static_cast<float*>(p);
  if (e == hipSuccess) e = dev_alloc(c, static_cast<size_t>(c->K) * c->cal_w * 2, &p);
  c->cal_copy = static_cast<uint16_t*>(p);
  if (e == hipSuccess) e = dev_alloc(c, static_cast<size_t>(c->K) * 4, &p);
  c->cal_order = static_cast<int32_t*>(p);
  std::vector<int32_t> ident(c->K);
  for (int k = 0; k < c->K; ++k) ident[k] = k;
  if (e == hipSuccess)
    e = hipMemcpyAsync(c->cal_order, ident.data(), ident.size() * 4, hipMemcpyHostToDevice,
                       c->stream);
  if (e == hipSuccess) e = hipStreamSynchronize(c->stream);
  for (int i = 0; i < 2 && e == hipSuccess; ++i) e = hipEventCreate(&c->cal_ev[i]);
  return e;
}

// Run `launch` (returns hipError_t), bracketed by profiling events if the
// kind is selected.
template <typename F>
hipError_t timed(oscars_ctx* c, int kind, F&& launch) {
  if (!(c->prof_mask & (1u << kind))) return launch();
  const int i = static_cast<int>(c->prof_recs.size()) * 2;
  while (static_cast<int>(c->ev_pool.size()) < i + 2) {
    hipEvent_t e;
    hipError_t err = hipEventCreate(&e);
    if (err != hipSuccess) return err;
    c->ev_pool.push_back(e);
  }
  hipError_t err = hipEventRecord(c->ev_pool[i], c->stream);
  if (err != hipSuccess) return err;
  err = launch();
  if (err != hipSuccess) return err;
  err = hipEventRecord(c->ev_pool[i + 1], c->stream);
  if (err != hipSuccess) return err;
  c->prof_recs.emplace_back(kind, i);
  return hipSuccess;
}

}  // namespace

extern "C" {

oscars_status oscars_create(oscars_ctx** out, const oscars_model* m, int32_t K, int32_t max_batch,
                            void* hip_stream) {
  if (!out || !m || !m->dims) return OSCARS_E_INVALID;
  if (m->n_layers < 1 || m->n_layers > OSCARS_MAX_LAYERS) return OSCARS_E_INVALID;
  if (m->dtype != OSCARS_FP32 && m->dtype != OSCARS_BF16) return OSCARS_E_INVALID;
  if (K < 1 || K > OSCARS_MAX_K || max_batch < 1 || max_batch > OSCARS_MAX_BATCH)
    return OSCARS_E_INVALID;
  for (int l = 0; l <= m->n_layers; ++l) {
    const int32_t w = m->dims[l];
    if (w < 1 || w > OSCARS_MAX_WIDTH) return OSCARS_E_INVALID;
    if (l < m->n_layers && w % 8 != 0) return OSCARS_E_INVALID;
  }
  oscars_ctx* c = new (std::nothrow) oscars_ctx();
  if (!c) return OSCARS_E_NOMEM;
  c->L = m->n_layers;
  c->dims.assign(m->dims, m->dims + m->n_layers + 1);
  c->bf16 = m->dtype == OSCARS_BF16;
  c->esize = c->bf16 ? 2 : 4;
  c->K = K;
  c->max_batch = max_batch;
  c->stream = static_cast<hipStream_t>(hip_stream);
  c->w_off.assign(c->L + 1, 0);
  c->b_off.assign(c->L + 1, 0);
  c->ld.assign(c->L + 1, 0);
  int64_t off = 0;
  for (int l = 1; l <= c->L; ++l) {
    c->w_off[l] = off;
    off = round_up(off + static_cast<int64_t>(c->dims[l]) * c->dims[l - 1], 64);
    c->b_off[l] = off;
    off = round_up(off + c->dims[l], 64);
    c->ld[l] = round_up(c->dims[l], 64);
  }
  c->ld[0] = c->dims[0];
  c->n_pad = off;
  c->cursors.assign(K, 0);
  c->samplers.resize(K);
  c->tuner = gemm_tuner_create();
  if (!c->tuner) {
    delete c;
    return OSCARS_E_NOMEM;
  }

  hipError_t e = hipGetDevice(&c->device);
  if (e == hipSuccess) e = scratch_address(c->device, &c->noalloc_scratch);
  if (e == hipSuccess && c->bf16) {
    void* p = nullptr;
    e = dev_alloc(c, static_cast<size_t>(K) * c->n_pad * 2, &p);
    c->wcopy = static_cast<uint16_t*>(p);
    if (e == hipSuccess) e = dev_alloc(c, static_cast<size_t>(c->n_pad) * 2, &p);
    c->gq = static_cast<uint16_t*>(p);
  }
  c->act.assign(c->L + 1, nullptr);
  c->delta.assign(c->L + 1, nullptr);
  if (e == hipSuccess)  // act[0]: the gathered batch rows of the current step
    e = dev_alloc(c, static_cast<size_t>(K) * c->act_slot(0) * c->esize, &c->act[0]);
  for (int l = 1; l <= c->L && e == hipSuccess; ++l) {
    const size_t n = static_cast<size_t>(K) * c->act_slot(l);
    if (l < c->L) e = dev_alloc(c, n * c->esize, &c->act[l]);
    if (e == hipSuccess) e = dev_alloc(c, n * c->esize, &c->delta[l]);
  }
  if (e == hipSuccess) {
    void* p = nullptr;
    e = dev_alloc(c, static_cast<size_t>(K) * c->act_slot(c->L) * 4, &p);
    c->logits = static_cast<float*>(p);
  }
  // Split-K partials ([slot][chunk][batch][ld] fp32) for launches of every
  // active replica; the kernels split only whole-batch tiles (batches above
  // 128) whose K has more than one chunk.
  if (e == hipSuccess && max_batch > 128) {
    constexpr int64_t kChunk = GEMM_KCHUNK;
    const int64_t kSplitSlots = K;
    int64_t need = 0;
    for (int l = 1; l <= c->L; ++l) {
      const int64_t fwd = (c->dims[l - 1] + kChunk - 1) / kChunk;
      if (fwd > 1) need = std::max(need, fwd * max_batch * c->ld[l]);
      const int64_t bwd = (c->dims[l] + kChunk - 1) / kChunk;
      if (l > 1 && bwd > 1) need = std::max(need, bwd * max_batch * c->ld[l - 1]);
    }
    if (need > 0) {
      c->part_cap = need * std::min<int64_t>(K, kSplitSlots);
      void* p = nullptr;
      e = dev_alloc(c, static_cast<size_t>(c->part_cap) * 4, &p);
      c->part = static_cast<float*>(p);
    }
  }
  if (e == hipSuccess) e = hipEventCreateWithFlags(&c->upload_done, hipEventDisableTiming);
  if (e == hipSuccess) {
    const int64_t rows = static_cast<int64_t>(K) * kPreTau * max_batch;
    e = ensure_tables(c, 64 + rows, rows);
  }
  if (e == hipSuccess) e = alloc_calibration(c);
  if (e == hipSuccess) e = hipStreamSynchronize(c->stream);
  if (e != hipSuccess) {
    free_ctx(c);
    return e == hipErrorOutOfMemory ? OSCARS_E_NOMEM : hip_fail(e);
  }
  *out = c;
  return OSCARS_OK;
}

oscars_status oscars_create_cnn(oscars_ctx** out, const oscars_cnn_model* m, int32_t K,
                                int32_t max_batch, void* hip_stream) {
  if (!out || !m || !m->conv_channels || !m->conv_strides) return OSCARS_E_INVALID;
  if (m->n_conv < 1 || m->n_conv > OSCARS_MAX_LAYERS - 1) return OSCARS_E_INVALID;
  if (m->height < 1 || m->width < 1 || m->channels < 1 || m->height > 4096 ||
      m->width > 4096 || m->channels > OSCARS_MAX_WIDTH)
    return OSCARS_E_INVALID;
  if (static_cast<int64_t>(m->height) * m->width * m->channels > (int64_t{1} << 24))
    return OSCARS_E_INVALID;
  if (m->classes < 1 || m->classes > OSCARS_MAX_WIDTH) return OSCARS_E_INVALID;
  if (K < 1 || K > OSCARS_MAX_K || max_batch < 1 || max_batch > OSCARS_MAX_BATCH)
    return OSCARS_E_INVALID;
  for (int l = 0; l < m->n_conv; ++l) {
    if (m->conv_channels[l] < 1 || m->conv_channels[l] > OSCARS_MAX_WIDTH) return OSCARS_E_INVALID;
    if (m->conv_strides[l] != 1 && m->conv_strides[l] != 2) return OSCARS_E_INVALID;
    // a shortcut at 0-based layer l adds the output of layer l - 2 (1-based l - 1)
    if (m->conv_skip && m->conv_skip[l] &&
        (l < 2 || m->conv_strides[l] != 1 || m->conv_strides[l - 1] != 1 ||
         m->conv_channels[l] != m->conv_channels[l - 2] || m->conv_channels[l - 1] < 4))
      return OSCARS_E_INVALID;
  }
  oscars_ctx* c = new (std::nothrow) oscars_ctx();
  if (!c) return OSCARS_E_NOMEM;
  const int Lc = m->n_conv;
  c->cnn = true;
  c->L = Lc + 1;
  c->dims.assign(c->L + 1, 0);
  c->dims[0] = m->height * m->width * m->channels;
  for (int l = 1; l <= Lc; ++l) c->dims[l] = m->conv_channels[l - 1];
  c->dims[c->L] = m->classes;
  c->bf16 = false;
  c->esize = 4;
  c->K = K;
  c->max_batch = max_batch;
  c->stream = static_cast<hipStream_t>(hip_stream);
  c->img_h.assign(Lc + 1, 0);
  c->img_w.assign(Lc + 1, 0);
  c->img_c.assign(Lc + 1, 0);
  c->conv_stride.assign(Lc + 1, 1);
  c->conv_skip.assign(Lc + 2, 0);
  for (int l = 1; l <= Lc; ++l) c->conv_skip[l] = m->conv_skip && m->conv_skip[l - 1] ? 1 : 0;
  c->img_h[0] = m->height;
  c->img_w[0] = m->width;
  c->img_c[0] = m->channels;
  for (int l = 1; l <= Lc; ++l) {
    c->conv_stride[l] = m->conv_strides[l - 1];
    c->img_h[l] = (c->img_h[l - 1] - 1) / c->conv_stride[l] + 1;
    c->img_w[l] = (c->img_w[l - 1] - 1) / c->conv_stride[l] + 1;
    c->img_c[l] = m->conv_channels[l - 1];
  }
  for (int l = 0; l <= Lc; ++l) {  // per-slot activations within 32-bit indices
    if (static_cast<int64_t>(max_batch) * c->img_h[l] * c->img_w[l] * c->img_c[l] >=
        (int64_t{1} << 31)) {
      delete c;
      return OSCARS_E_INVALID;
    }
  }
  c->w_off.assign(c->L + 1, 0);
  c->b_off.assign(c->L + 1, 0);
  c->ld.assign(c->L + 1, 0);
  int64_t off = 0;
  for (int l = 1; l <= c->L; ++l) {
    const int64_t w = l <= Lc ? 9LL * c->img_c[l - 1] * c->img_c[l]
                              : static_cast<int64_t>(m->classes) * c->img_c[Lc];
    c->w_off[l] = off;
    off = round_up(off + w, 64);
    c->b_off[l] = off;
    off = round_up(off + c->dims[l], 64);
  }
  c->ld[c->L] = round_up(m->classes, 64);
  c->n_pad = off;
  c->cursors.assign(K, 0);
  c->samplers.resize(K);
  c->act.assign(c->L + 1, nullptr);
  c->delta.assign(c->L + 1, nullptr);
  c->cact.assign(Lc + 1, nullptr);
  c->cdz.assign(Lc + 1, nullptr);
  c->tuner = gemm_tuner_create();
  if (!c->tuner) {
    delete c;
    return OSCARS_E_NOMEM;
  }
  // weight-gradient partials per slot and layer: splits x outputs (all layers'
  // partials of a step live until its updates, which run after every
  // backward-data launch)
  c->cpart_l.assign(Lc + 2, nullptr);
  c->cpart_slot_l.assign(Lc + 2, 0);
  c->cpart_slot_l[Lc + 1] = round_up(static_cast<int64_t>(m->classes) * (c->img_c[Lc] + 1), 64);
  for (int l = 1; l <= Lc; ++l) {
    ConvArgs a{};
    a.B = max_batch;
    a.H = c->img_h[l - 1];
    a.W = c->img_w[l - 1];
    a.C = c->img_c[l - 1];
    a.Ho = c->img_h[l];
    a.Wo = c->img_w[l];
    a.Co = c->img_c[l];
    a.stride = c->conv_stride[l];
    int splits = 0;
    int64_t per = 0;
    conv_wgrad_ranges(a, &splits, &per);
    c->cpart_slot_l[l] = round_up(static_cast<int64_t>(splits) * a.Co * (9LL * a.C + 1), 64);
  }
  int64_t part_total = 0;
  for (int l = 1; l <= Lc + 1; ++l) part_total += c->cpart_slot_l[l];

  hipError_t e = hipGetDevice(&c->device);
  if (e == hipSuccess) e = scratch_address(c->device, &c->noalloc_scratch);
  void* p = nullptr;
  for (int l = 1; l <= Lc && e == hipSuccess; ++l) {
    const size_t bytes = static_cast<size_t>(K) * c->cnn_slot(l) * 4;
    e = dev_alloc(c, bytes, &p);
    c->cact[l] = static_cast<float*>(p);
    if (e == hipSuccess) e = dev_alloc(c, bytes, &p);
    c->cdz[l] = static_cast<float*>(p);
  }
  const size_t pooled_bytes = static_cast<size_t>(K) * max_batch * c->img_c[Lc] * 4;
  if (e == hipSuccess) e = dev_alloc(c, pooled_bytes, &p);
  c->pooled = static_cast<float*>(p);
  if (e == hipSuccess) e = dev_alloc(c, pooled_bytes, &p);
  c->dpooled = static_cast<float*>(p);
  if (e == hipSuccess) e = dev_alloc(c, static_cast<size_t>(K) * c->act_slot(c->L) * 4, &p);
  c->logits = static_cast<float*>(p);
  if (e == hipSuccess) e = dev_alloc(c, static_cast<size_t>(K) * c->act_slot(c->L) * 4, &p);
  c->delta[c->L] = p;
  if (e == hipSuccess) e = dev_alloc(c, static_cast<size_t>(K) * part_total * 4, &p);
  c->cpart = static_cast<float*>(p);
  int64_t part_off = 0;
  for (int l = 1; l <= Lc + 1 && e == hipSuccess; ++l) {
    c->cpart_l[l] = c->cpart + part_off;
    part_off += static_cast<int64_t>(K) * c->cpart_slot_l[l];
  }
  if (e == hipSuccess) e = hipEventCreateWithFlags(&c->upload_done, hipEventDisableTiming);
  if (e == hipSuccess) {
    const int64_t rows = static_cast<int64_t>(K) * kPreTau * max_batch;
    e = ensure_tables(c, 64 + rows, rows);
  }
  if (e == hipSuccess) e = hipStreamSynchronize(c->stream);
  if (e != hipSuccess) {
    free_ctx(c);
    return e == hipErrorOutOfMemory ? OSCARS_E_NOMEM : hip_fail(e);
  }
  *out = c;
  return OSCARS_OK;
}

void oscars_destroy(oscars_ctx* ctx) { free_ctx(ctx); }

oscars_status oscars_set_stream(oscars_ctx* ctx, void* hip_stream) {
  if (!ctx) return OSCARS_E_INVALID;
  hipError_t e = hipStreamSynchronize(ctx->stream);
  if (e != hipSuccess) return hip_fail(e);
  ctx->stream = static_cast<hipStream_t>(hip_stream);
  return OSCARS_OK;
}

int64_t oscars_num_params(const oscars_ctx* ctx) { return ctx ? ctx->n_pad : -1; }

oscars_status oscars_layer_offsets(const oscars_ctx* ctx, int32_t l, int64_t* w_off,
                                   int64_t* b_off) {
  if (!ctx || !w_off || !b_off || l < 1 || l > ctx->L) return OSCARS_E_INVALID;
  *w_off = ctx->w_off[l];
  *b_off = ctx->b_off[l];
  return OSCARS_OK;
}

oscars_status oscars_get_cursors(const oscars_ctx* ctx, int64_t* steps_done) {
  if (!ctx || !steps_done) return OSCARS_E_INVALID;
  std::copy(ctx->cursors.begin(), ctx->cursors.end(), steps_done);
  return OSCARS_OK;
}

oscars_status oscars_set_cursors(oscars_ctx* ctx, const int64_t* steps_done) {
  if (!ctx || !steps_done) return OSCARS_E_INVALID;
  for (int k = 0; k < ctx->K; ++k)
    if (steps_done[k] < 0) return OSCARS_E_INVALID;
  std::copy(steps_done, steps_done + ctx->K, ctx->cursors.begin());
  return OSCARS_OK;
}

}  // extern "C"

namespace {

ConvArgs conv_layer_args(const oscars_ctx* c, int l, const float* master_in, int64_t master_in_slot,
                         const int32_t* order, int B) {
  ConvArgs a{};
  a.B = B;
  a.order = order;
  a.master_in = master_in;
  a.master_in_slot = master_in_slot;
  a.w_off = c->w_off[l];
  a.b_off = c->b_off[l];
  if (l < c->L) {
    a.H = c->img_h[l - 1];
    a.W = c->img_w[l - 1];
    a.C = c->img_c[l - 1];
    a.Ho = c->img_h[l];
    a.Wo = c->img_w[l];
    a.Co = c->img_c[l];
    a.stride = c->conv_stride[l];
  } else {  // classifier
    a.H = a.W = a.Ho = a.Wo = 1;
    a.C = c->img_c[c->L - 1];
    a.Co = c->dims[c->L];
    a.stride = 1;
  }
  return a;
}

// The classifier head of local step j (conv_head_kernel): whether it fits
// one workgroup is checked by the caller (conv_head_fits).
HeadArgs head_args(const oscars_ctx* c, const float* master_in, int64_t master_in_slot,
                   const int32_t* order, const int32_t* y, const int32_t* rows,
                   int64_t rows_slot, int B, float* loss) {
  const int L = c->L;
  HeadArgs h{};
  h.B = B;
  h.HW = c->img_h[L - 1] * c->img_w[L - 1];
  h.C = c->img_c[L - 1];
  h.classes = c->dims[L];
  h.act = c->cact[L - 1];
  h.act_slot = c->cnn_slot(L - 1);
  h.master_in = master_in;
  h.master_in_slot = master_in_slot;
  h.w_off = c->w_off[L];
  h.b_off = c->b_off[L];
  h.order = order;
  h.y = y;
  h.gather = rows;
  h.gather_slot = rows_slot;
  h.pooled = c->pooled;
  h.pooled_slot = static_cast<int64_t>(c->max_batch) * h.C;
  h.delta = static_cast<float*>(c->delta[L]);
  h.delta_slot = c->act_slot(L);
  h.delta_ld = c->ld[L];
  h.loss = loss;
  h.loss_slot = rows_slot;
  h.dz = c->cdz[L - 1];
  h.dz_slot = c->cnn_slot(L - 1);
  return h;
}

// Forward pass of the convolutional model for n_slots slots: conv layers
// (layer 1 gathers the dataset rows `rows` of each slot), then, with
// `with_head`, average pooling and the classifier logits into c->logits.
hipError_t cnn_forward(oscars_ctx* c, const float* master_in, int64_t master_in_slot,
                       const int32_t* order, const void* x, const int32_t* rows,
                       int64_t rows_slot, int B, int ns, bool with_head = true) {
  const int L = c->L;
  hipError_t e = hipSuccess;
  for (int l = 1; l < L && e == hipSuccess; ++l) {
    ConvArgs a = conv_layer_args(c, l, master_in, master_in_slot, order, B);
    if (l == 1) {
      a.in = static_cast<const float*>(x);
      a.in_ld = c->dims[0];
      a.gather = rows;
      a.gather_slot = rows_slot;
    } else {
      a.in = c->cact[l - 1];
      a.in_slot = c->cnn_slot(l - 1);
    }
    if (c->conv_skip[l]) {  // the residual block's input
      a.skip = c->cact[l - 2];
      a.skip_slot = c->cnn_slot(l - 2);
    }
    a.out = c->cact[l];
    a.out_slot = c->cnn_slot(l);
    e = timed(c, OSCARS_KERNEL_FWD, [&] { return launch_conv(a, CONV_FWD, ns, c->stream); });
  }
  if (!with_head) return e;
  const int HW = c->img_h[L - 1] * c->img_w[L - 1], Cl = c->img_c[L - 1];
  const int64_t pslot = static_cast<int64_t>(c->max_batch) * Cl;
  if (e == hipSuccess)
    e = timed(c, OSCARS_KERNEL_FWD, [&] {
      return launch_avgpool(c->cact[L - 1], c->cnn_slot(L - 1), c->pooled, pslot, B, HW, Cl, ns,
                            c->stream);
    });
  if (e == hipSuccess) {
    ConvArgs a = conv_layer_args(c, L, master_in, master_in_slot, order, B);
    a.in = c->pooled;
    a.in_slot = pslot;
    a.out = c->logits;
    a.out_slot = c->act_slot(L);
    a.out_ld = c->ld[L];
    e = timed(c, OSCARS_KERNEL_FWD, [&] { return launch_conv(a, FC_FWD, ns, c->stream); });
  }
  return e;
}

// One local step of every active slot of the convolutional model after its
// forward pass and loss gradient (in c->delta[L]): classifier backward-data
// and weight-gradient partials, pooling backward with the last ReLU mask,
// then per conv layer (top down) backward-data (masked by the layer below)
// and its weight-gradient partials; last, the SGD updates of all layers in
// launches of up to MAX_UPDATE_BLOCKS layers, after every backward-data launch
// has read the weights they overwrite.  With `head` (conv_head_kernel ran
// instead of the pooling, classifier and softmax launches and already wrote
// the gradient at the last conv output), the classifier's update forms its
// gradient from pooled and delta.
hipError_t cnn_backward(oscars_ctx* c, float* replicas, const float* master_in,
                        int64_t master_in_slot, const int32_t* order, const void* x,
                        const int32_t* rows, int64_t rows_slot, int B, int ns, float lr,
                        const HeadArgs* head) {
  const int L = c->L;
  const int Cl = c->img_c[L - 1], HW = c->img_h[L - 1] * c->img_w[L - 1];
  const int64_t pslot = static_cast<int64_t>(c->max_batch) * Cl;
  hipError_t e = hipSuccess;
  std::vector<UpdateBlock> upd;
  {
    ConvArgs a = conv_layer_args(c, L, master_in, master_in_slot, order, B);
    UpdateBlock u{};
    u.M = a.Co;
    u.N = a.C + 1;
    u.w_off = a.w_off;
    u.b_off = a.b_off;
    if (!head) {
      a.in = c->pooled;
      a.in_slot = pslot;
      a.dout = static_cast<const float*>(c->delta[L]);
      a.dout_slot = c->act_slot(L);
      a.dout_ld = c->ld[L];
      a.out = c->dpooled;
      a.out_slot = pslot;
      a.out_ld = Cl;
      e = timed(c, OSCARS_KERNEL_DGRAD, [&] { return launch_conv(a, FC_DGRAD, ns, c->stream); });
      a.part = c->cpart_l[L];
      a.part_slot = c->cpart_slot_l[L];
      a.splits = 1;
      a.k_per_split = B;
      if (e == hipSuccess)
        e = timed(c, OSCARS_KERNEL_WGRAD, [&] { return launch_conv(a, FC_WGRAD, ns, c->stream); });
      if (e == hipSuccess)
        e = timed(c, OSCARS_KERNEL_DGRAD, [&] {
          return launch_avgpool_backward(c->dpooled, pslot, c->cact[L - 1], c->cnn_slot(L - 1),
                                         c->cdz[L - 1], B, HW, Cl, ns, c->stream);
        });
      u.part = a.part;
      u.part_slot = a.part_slot;
      u.splits = 1;
    }
    upd.push_back(u);
  }
  for (int l = L - 1; l >= 1 && e == hipSuccess; --l) {
    ConvArgs a = conv_layer_args(c, l, master_in, master_in_slot, order, B);
    a.dout = c->cdz[l];
    a.dout_slot = c->cnn_slot(l);
    ConvArgs ad = a;  // backward-data (l > 1)
    if (l > 1) {
      ad.out = c->cdz[l - 1];
      ad.out_slot = c->cnn_slot(l - 1);
      ad.mask = c->cact[l - 1];
      ad.mask_slot = c->cnn_slot(l - 1);
      if (c->conv_skip[l + 1]) {  // layer l + 1 adds this layer's input: its Z gradient too
        ad.skip = c->cdz[l + 1];
        ad.skip_slot = c->cnn_slot(l + 1);
      }
      // stride 2: the four parity classes of the input pixels in one launch
      ad.cls = -1;
      a.in = c->cact[l - 1];
      a.in_slot = c->cnn_slot(l - 1);
    } else {
      a.in = static_cast<const float*>(x);
      a.in_ld = c->dims[0];
      a.gather = rows;
      a.gather_slot = rows_slot;
    }
    conv_wgrad_ranges(a, &a.splits, &a.k_per_split);
    a.part = c->cpart_l[l];
    a.part_slot = c->cpart_slot_l[l];
    if (l > 1 && conv_pair_fits(ad, a, ns)) {
      // one or two replicas: backward-data and backward-weight in one launch
      e = timed(c, OSCARS_KERNEL_BWD_FUSED,
                [&] { return launch_conv_pair(ad, a, ns, c->stream); });
    } else {
      if (l > 1) {
        e = timed(c, OSCARS_KERNEL_DGRAD,
                  [&] { return launch_conv(ad, CONV_DGRAD, ns, c->stream); });
        if (e != hipSuccess) break;
      }
      e = timed(c, OSCARS_KERNEL_WGRAD, [&] { return launch_conv(a, CONV_WGRAD, ns, c->stream); });
    }
    UpdateBlock u{};
    u.part = a.part;
    u.part_slot = a.part_slot;
    u.splits = a.splits;
    u.M = a.Co;
    u.N = 9 * a.C + 1;
    u.w_off = a.w_off;
    u.b_off = a.b_off;
    upd.push_back(u);
  }
  for (size_t i = 0; i < upd.size() && e == hipSuccess; i += MAX_UPDATE_BLOCKS) {
    const int n = static_cast<int>(std::min<size_t>(MAX_UPDATE_BLOCKS, upd.size() - i));
    e = timed(c, OSCARS_KERNEL_WGRAD, [&] {
      return launch_conv_updates(upd.data() + i, n, head, master_in, master_in_slot, order, replicas,
                                 c->n_pad, lr, ns, c->stream);
    });
  }
  return e;
}

// Backward of layer l of a bf16 model without a forced mode: at the first
// launch of each (inputs, outputs, batch, replicas, layer 1 or hidden) the
// fused launch (gf) with every feasible number of output chunks per
// workgroup (all, then halving down to one), and the separate backward-data
// + update launches (gd, gw; layer 1: gd == nullptr, the fused launch
// without backward-data against the update alone), each run three times on
// the scratch replicas oscars_create allocated, timed; the fastest of the
// last two runs of each decides (the earlier candidate on ties).  The real
// replicas and weight copies are untouched; every hidden-layer candidate
// writes the delta of the layer below, which the real launch that follows
// recomputes.  *cps: the chunks per workgroup of the fused launch, or 0 for
// the separate launches.  On a stream being captured into a graph, or
// without scratch, nothing is timed: the fused launch with the split its
// launcher picks (*cps = -1).
hipError_t choose_backward(oscars_ctx* c, int ns, const GemmArgs& gf, const GemmArgs* gd,
                           const GemmArgs& gw, int* cps) {
  *cps = -1;
  hipStreamCaptureStatus cap = hipStreamCaptureStatusNone;
  if (hipStreamIsCapturing(c->stream, &cap) != hipSuccess || cap != hipStreamCaptureStatusNone)
    return hipSuccess;
  const bool dgrad = gd != nullptr;
  const std::array<int, 5> key{gf.M, gf.K, gf.N, ns, dgrad ? 1 : 0};
  auto it = c->bwd_fused_choice.find(key);
  if (it != c->bwd_fused_choice.end()) {
    *cps = it->second;
    return hipSuccess;
  }
  // no scratch (too large for the free memory, see alloc_calibration): untimed
  if (c->cal_off || !c->cal_master) return hipSuccess;
  hipError_t e = hipSuccess;
  const int64_t wsize = static_cast<int64_t>(gf.M) * gf.K;  // W_l: outputs x inputs
  auto to_scratch = [&](GemmArgs& a) {
    a.master = c->cal_master;
    a.master_slot = c->cal_layer;
    a.master_in = c->cal_master;
    a.master_in_slot = c->cal_layer;
    a.w_off = 0;
    a.b_off = wsize;
    a.order = c->cal_order;
    if (a.wcopy) {
      a.wcopy = c->cal_copy;
      a.wcopy_slot = c->cal_w;
    }
  };
  GemmArgs f = gf, d = dgrad ? *gd : gw, w = gw;
  to_scratch(f);
  to_scratch(d);
  to_scratch(w);
  d.a = c->cal_copy;  // backward-data reads the slots' bf16 weights
  d.a_slot = c->cal_w;
  d.a_by_order = 0;
  // candidates: fused with each feasible split, then separate (0) (layer 1:
  // separate first); three runs of each, round robin; the first (which also
  // picks the backward-data tiling) is not counted, the faster of the other
  // two is
  int cand[8];
  // Layer 1's separate update comes first, so that the streamed launch
  // replaces it only when faster by the margin (picked first, within the
  // margin, the streamed launch ran a 4096 x 4096 layer 1 at 3 replicas in
  // 117 against 96 us for the separate update).
  int nc = 0;
  if (!dgrad) cand[nc++] = 0;
  nc += bwd_fused_splits(f, ns, cand + nc, 7, dgrad);
  if (dgrad) cand[nc++] = 0;
  float best[8] = {};
  struct TuneNow {  // the separate path's backward-data tiling decided at its first run
    TuneNow() { set_gemm_tune_now(true); }
    ~TuneNow() { set_gemm_tune_now(false); }
  } tune_now;
  for (int rep = 0; rep < 3 && e == hipSuccess; ++rep) {
    for (int i = 0; i < nc && e == hipSuccess; ++i) {
      float ms = 0.0f;
      e = hipEventRecord(c->cal_ev[0], c->stream);
      if (cand[i] > 0) {
        if (e == hipSuccess)
          e = launch_bwd_fused(f, ns, c->stream, c->backward_mode, cand[i], dgrad);
      } else {
        if (e == hipSuccess && dgrad)
          e = launch_gemm(d, GEMM_DGRAD, true, ns, c->stream, c->tuner);
        if (e == hipSuccess) e = launch_gemm(w, GEMM_WGRAD, true, ns, c->stream, c->tuner);
      }
      if (e == hipSuccess) e = hipEventRecord(c->cal_ev[1], c->stream);
      if (e == hipSuccess) e = hipEventSynchronize(c->cal_ev[1]);
      if (e == hipSuccess) e = hipEventElapsedTime(&ms, c->cal_ev[0], c->cal_ev[1]);
      if (rep == 1 || (rep > 1 && ms < best[i])) best[i] = ms;
    }
  }
  if (e != hipSuccess) return e;
  // A later candidate replaces the pick only when it is faster by more than
  // kBackwardMargin: near ties (within the run-to-run spread of these
  // timings) go to the earlier candidate, so that separate processes on one
  // box take the same paths.
  int pick = 0;
  for (int i = 1; i < nc; ++i)
    if (best[i] < best[pick] * (1.0f - kBackwardMargin)) pick = i;
  *cps = cand[pick];
  c->bwd_fused_choice[key] = *cps;
  return hipSuccess;
}

// tau_k local steps of every worker.  start == nullptr: worker k starts from
// replica k.  Otherwise every worker starts from `start` (the global model of
// a round): the first step reads `start` and writes replica k; workers with
// tau_k = 0 get a copy of `start`.
oscars_status run_local_steps(oscars_ctx* c, float* replicas, const float* start,
                              const oscars_shards* s, const int32_t* tau, float lr, int32_t batch) {
  // ---- validation (no side effects on failure) ----
  if (!c || !replicas || !s || !tau || !s->x || !s->y || !s->offsets) return OSCARS_E_INVALID;
  if (!aligned16(replicas) || !aligned16(s->x)) return OSCARS_E_INVALID;
  if (!std::isfinite(lr) || !(lr > 0.0f)) return OSCARS_E_INVALID;
  if (batch < 1 || batch > c->max_batch) return OSCARS_E_INVALID;
  if (s->n_rows < 1 || s->n_rows > 0x7FFFFFFF) return OSCARS_E_INVALID;
  const int K = c->K;
  if (s->offsets[0] != 0 || s->offsets[K] != s->n_rows) return OSCARS_E_INVALID;
  for (int k = 0; k < K; ++k) {
    if (s->offsets[k + 1] <= s->offsets[k]) return OSCARS_E_INVALID;
    if (tau[k] < 0 || tau[k] > kMaxTau) return OSCARS_E_INVALID;
  }
  // Not on a stream being captured into a graph: every call draws its
  // batches on the host and waits for the previous call's index upload, which
  // a graph could neither redraw nor wait for.
  hipStreamCaptureStatus cap = hipStreamCaptureStatusNone;
  hipError_t e = hipStreamIsCapturing(c->stream, &cap);
  if (e != hipSuccess) return hip_fail(e);
  if (cap != hipStreamCaptureStatusNone) return OSCARS_E_STATE;

  // ---- slots: workers with work, by tau descending, ties by index ----
  std::vector<int32_t> order;
  for (int k = 0; k < K; ++k)
    if (tau[k] > 0) order.push_back(k);
  std::stable_sort(order.begin(), order.end(),
                   [&](int32_t a, int32_t b) { return tau[a] > tau[b]; });
  const int n_slots = static_cast<int>(order.size());
  const int tau_max = n_slots ? tau[order[0]] : 0;
  const int B = batch;

  // ---- index table capacity: order[64] then rows[slot][j][b] (grown only
  // for more than kPreTau steps per worker; failures leave no side effects) ----
  const int64_t need = 64 + static_cast<int64_t>(n_slots) * tau_max * B;
  const int64_t loss_need = static_cast<int64_t>(n_slots) * tau_max * B;
  if (c->upload_pending) {
    e = hipEventSynchronize(c->upload_done);
    if (e != hipSuccess) return hip_fail(e);
    c->upload_pending = false;
  }
  e = ensure_tables(c, need, loss_need);
  if (e == hipErrorOutOfMemory || e == hipErrorMemoryAllocation) return OSCARS_E_NOMEM;
  if (e != hipSuccess) return hip_fail(e);

  c->last_order = order;
  c->last_tau.assign(tau, tau + K);
  c->last_B = batch;
  c->last_tau_max = tau_max;
  if (start) {
    for (int k = 0; k < K; ++k) {
      if (tau[k] > 0) continue;
      e = hipMemcpyAsync(replicas + static_cast<int64_t>(k) * c->n_pad, start,
                         c->n_pad * sizeof(float), hipMemcpyDeviceToDevice, c->stream);
      if (e != hipSuccess) return hip_fail(e);
    }
  }
  if (n_slots == 0) return OSCARS_OK;
  int32_t* h_order = c->pinned;
  int32_t* h_rows = c->pinned + 64;
  for (int z = 0; z < 64; ++z) h_order[z] = z < n_slots ? order[z] : 0;
  for (int z = 0; z < n_slots; ++z) {
    const int k = order[z];
    WorkerSampler& ws = c->samplers[k];
    ws.reset(s->seed, static_cast<uint32_t>(k), s->offsets[k], s->offsets[k + 1] - s->offsets[k]);
    for (int j = 0; j < tau[k]; ++j)
      for (int b = 0; b < B; ++b)
        h_rows[(static_cast<int64_t>(z) * tau_max + j) * B + b] =
            static_cast<int32_t>(ws.row((c->cursors[k] + j) * B + b));
  }
  e = hipMemcpyAsync(c->table_dev, c->pinned, need * sizeof(int32_t), hipMemcpyHostToDevice,
                     c->stream);
  if (e == hipSuccess) e = hipEventRecord(c->upload_done, c->stream);
  if (e != hipSuccess) return hip_fail(e);
  c->upload_pending = true;
  const int32_t* d_order = c->table_dev;
  const int32_t* d_rows = c->table_dev + 64;

  if (c->cnn) {
    for (int j = 0; j < tau_max; ++j) {
      int ns = 0;
      while (ns < n_slots && tau[order[ns]] > j) ++ns;
      const int32_t* rows_j = d_rows + static_cast<int64_t>(j) * B;
      const int64_t rows_slot = static_cast<int64_t>(tau_max) * B;
      const bool from_start = start && j == 0;
      const float* min = from_start ? start : replicas;
      const int64_t min_slot = from_start ? 0 : c->n_pad;
      float* loss_j = c->loss_dev + static_cast<int64_t>(j) * B;
      const HeadArgs head =
          head_args(c, min, min_slot, d_order, s->y, rows_j, rows_slot, B, loss_j);
      const bool fused_head = conv_head_fits(head.HW, head.C, head.classes);
      e = cnn_forward(c, min, min_slot, d_order, s->x, rows_j, rows_slot, B, ns, !fused_head);
      if (e == hipSuccess)
        e = timed(c, OSCARS_KERNEL_SOFTMAX, [&] {
          if (fused_head) return launch_conv_head(head, ns, c->stream);
          return launch_softmax_ce(c->logits, c->ld[c->L], c->act_slot(c->L), c->dims[c->L], B,
                                   s->y, rows_j, rows_slot, c->delta[c->L], false, loss_j,
                                   rows_slot, ns, c->stream);
        });
      if (e == hipSuccess)
        e = cnn_backward(c, replicas, min, min_slot, d_order, s->x, rows_j, rows_slot, B, ns, lr,
                         fused_head ? &head : nullptr);
      if (e != hipSuccess) return hip_fail(e);
    }
    for (int k = 0; k < K; ++k) c->cursors[k] += tau[k];
    return OSCARS_OK;
  }

  // ---- bf16 working copies: of the start model once, else of every active replica ----
  if (c->bf16) {
    e = timed(c, OSCARS_KERNEL_CAST, [&] {
      return start ? launch_cast_bf16(start, 0, d_order, c->gq, 0, c->n_pad, 1, c->stream)
                   : launch_cast_bf16(replicas, c->n_pad, d_order, c->wcopy, c->n_pad, c->n_pad,
                                      n_slots, c->stream);
    });
    if (e != hipSuccess) return hip_fail(e);
  }

  const int L = c->L;
  const int64_t rows_slot = static_cast<int64_t>(tau_max) * B;
  for (int j = 0; j < tau_max; ++j) {
    int ns = 0, ns_next = 0;
    while (ns < n_slots && tau[order[ns]] > j) ++ns;
    while (ns_next < n_slots && tau[order[ns_next]] > j + 1) ++ns_next;
    const int32_t* rows_j = d_rows + static_cast<int64_t>(j) * B;

    // Weights as operand A: slot-indexed bf16 copies, or the fp32 masters
    // themselves (reached through order[]); in the first step of a round that
    // starts from the global model, that model (shared by every slot).
    const bool from_start = start && j == 0;
    auto weights = [&](GemmArgs& g, int l) {
      if (from_start) {
        g.a = c->bf16 ? static_cast<const void*>(c->gq + c->w_off[l])
                      : static_cast<const void*>(start + c->w_off[l]);
        g.a_by_order = 0;
        g.a_slot = 0;
      } else if (c->bf16) {
        g.a = c->wcopy + c->w_off[l];
        g.a_by_order = 0;
        g.a_slot = c->n_pad;
      } else {
        g.a = replicas + c->w_off[l];
        g.a_by_order = 1;
        g.a_slot = c->n_pad;
      }
      g.a_ld = c->dims[l - 1];
    };
    auto common = [&](GemmArgs& g, int l) {
      g.master = replicas;
      g.master_slot = c->n_pad;
      g.master_in = from_start ? start : replicas;
      g.master_in_slot = from_start ? 0 : c->n_pad;
      g.w_off = c->w_off[l];
      g.b_off = c->b_off[l];
      g.order = d_order;
      g.lr = lr;
      g.part = c->part;
      g.part_cap = c->part_cap;
    };

    // forward: C[o][b] = W_l . act_{l-1}
    for (int l = 1; l <= L; ++l) {
      GemmArgs g{};
      g.M = c->dims[l];
      g.N = B;
      g.K = c->dims[l - 1];
      g.a_ext = g.K;
      g.b_ext = g.K;
      weights(g, l);
      if (l == 1) {
        g.b = s->x;
        g.b_ld = c->dims[0];
        g.b_slot = 0;
        g.gather = rows_j;
        g.gather_slot = rows_slot;
        g.rows_out = c->act[0];
        g.rows_out_ld = c->ld[0];
        g.rows_out_slot = c->act_slot(0);
      } else {
        g.b = c->act[l - 1];
        g.b_ld = c->ld[l - 1];
        g.b_slot = c->act_slot(l - 1);
      }
      common(g, l);
      if (l < L) {
        g.out = c->act[l];
        g.relu = 1;
        g.out_bf16 = c->bf16;
      } else {
        g.out = c->logits;
        g.relu = 0;
        g.out_bf16 = 0;
      }
      g.out_ld = c->ld[l];
      g.out_slot = c->act_slot(l);
      e = timed(c, OSCARS_KERNEL_FWD, [&] { return launch_gemm(g, GEMM_FWD, c->bf16, ns, c->stream, c->tuner); });
      if (e != hipSuccess) return hip_fail(e);
    }
    // loss gradient
    e = timed(c, OSCARS_KERNEL_SOFTMAX, [&] {
      return launch_softmax_ce(c->logits, c->ld[L], c->act_slot(L), c->dims[L], B, s->y, rows_j,
                               rows_slot, c->delta[L], c->bf16, c->loss_dev + static_cast<int64_t>(j) * B,
                               rows_slot, ns, c->stream);
    });
    if (e != hipSuccess) return hip_fail(e);
    // backward-data of layer l > 1: C[i][b] = sum_o W_l[o][i] delta_l[b][o],
    // masked by act_{l-1} > 0
    auto dgrad_args = [&](int l) {
      GemmArgs g{};
      g.M = c->dims[l - 1];
      g.N = B;
      g.K = c->dims[l];
      g.a_ext = g.M;                                 // W rows, m chunks
      g.b_ext = static_cast<int>(round_up(g.K, 8));  // delta rows are zero-padded
      weights(g, l);
      g.b = c->delta[l];
      g.b_ld = c->ld[l];
      g.b_slot = c->act_slot(l);
      common(g, l);
      g.out = c->delta[l - 1];
      g.out_ld = c->ld[l - 1];
      g.out_slot = c->act_slot(l - 1);
      g.out_bf16 = c->bf16;
      g.mask = c->act[l - 1];
      g.mask_ld = c->ld[l - 1];
      g.mask_slot = c->act_slot(l - 1);
      return g;
    };
    // backward-weight + SGD update of layer l:
    // C[i][o] = sum_b act_{l-1}[b][i] delta_l[b][o] = dW_l[o][i]
    auto wgrad_args = [&](int l) {
      GemmArgs g{};
      g.M = c->dims[l - 1];
      g.N = c->dims[l];
      g.K = B;
      g.a_ext = g.M;
      g.b_ext = static_cast<int>(round_up(g.N, 8));  // delta rows are zero-padded
      g.a = c->act[l - 1];  // for l = 1: the batch rows the forward pass gathered
      g.a_ld = c->ld[l - 1];
      g.a_slot = c->act_slot(l - 1);
      g.a_by_order = 0;
      g.b = c->delta[l];
      g.b_ld = c->ld[l];
      g.b_slot = c->act_slot(l);
      common(g, l);
      g.wcopy = c->bf16 ? c->wcopy : nullptr;
      g.wcopy_slot = c->n_pad;
      g.wcopy_slots = ns_next;  // slots ns_next .. ns-1 take their last step now
      return g;
    };
    // backward, top layer first; dgrad(l) reads W_l before wgrad(l) updates it
    for (int l = L; l >= 1; --l) {
      if (l > 1 && c->bf16 && backward_fused_enabled(c->backward_mode)) {
        // hidden layer of a bf16 model: backward-data, backward-weight and the
        // update in one launch (bit-identical to the two launches below)
        GemmArgs g{};
        g.M = c->dims[l - 1];
        g.N = B;
        g.K = c->dims[l];
        g.a = c->act[l - 1];
        g.a_ld = c->ld[l - 1];
        g.a_slot = c->act_slot(l - 1);
        g.b = c->delta[l];
        g.b_ld = c->ld[l];
        g.b_slot = c->act_slot(l);
        common(g, l);
        g.out = c->delta[l - 1];
        g.out_ld = c->ld[l - 1];
        g.out_slot = c->act_slot(l - 1);
        g.out_bf16 = 1;
        g.mask = c->act[l - 1];
        g.mask_ld = c->ld[l - 1];
        g.mask_slot = c->act_slot(l - 1);
        g.wcopy = c->wcopy;
        g.wcopy_slot = c->n_pad;
        g.wcopy_slots = ns_next;  // slots ns_next .. ns-1 take their last step now
        if (backward_fusable(g)) {
          int cps = -1;  // fused, split by the launcher's rule
          if (c->backward_mode == BACKWARD_AUTO) {
            const GemmArgs gd = dgrad_args(l);
            e = choose_backward(c, ns, g, &gd, wgrad_args(l), &cps);
            if (e != hipSuccess) return hip_fail(e);
          }
          if (cps != 0) {
            e = timed(c, OSCARS_KERNEL_BWD_FUSED,
                      [&] {
                        return launch_bwd_fused(g, ns, c->stream, c->backward_mode,
                                                cps > 0 ? cps : 0);
                      });
            if (e != hipSuccess) return hip_fail(e);
            continue;
          }
        }
      }
      if (l == 1 && c->bf16 && backward_fused_enabled(c->backward_mode)) {
        // layer 1: backward-weight and the update streamed like the fused
        // backward of the hidden layers, without backward-data
        GemmArgs g{};
        g.M = c->dims[0];
        g.N = B;
        g.K = c->dims[1];
        g.a = c->act[0];  // the batch rows the forward pass gathered
        g.a_ld = c->ld[0];
        g.a_slot = c->act_slot(0);
        g.b = c->delta[1];
        g.b_ld = c->ld[1];
        g.b_slot = c->act_slot(1);
        common(g, 1);
        g.wcopy = c->wcopy;
        g.wcopy_slot = c->n_pad;
        g.wcopy_slots = ns_next;  // slots ns_next .. ns-1 take their last step now
        if (backward_fusable(g)) {
          int cps = -1;
          if (c->backward_mode == BACKWARD_AUTO) {
            e = choose_backward(c, ns, g, nullptr, wgrad_args(1), &cps);
            if (e != hipSuccess) return hip_fail(e);
          }
          if (cps != 0) {
            e = timed(c, OSCARS_KERNEL_WGRAD,
                      [&] {
                        return launch_bwd_fused(g, ns, c->stream, c->backward_mode,
                                                cps > 0 ? cps : 0, false);
                      });
            if (e != hipSuccess) return hip_fail(e);
            continue;
          }
        }
      }
      if (l > 1) {
        const GemmArgs g = dgrad_args(l);
        e = timed(c, OSCARS_KERNEL_DGRAD,
                  [&] { return launch_gemm(g, GEMM_DGRAD, c->bf16, ns, c->stream, c->tuner); });
        if (e != hipSuccess) return hip_fail(e);
      }
      const GemmArgs g = wgrad_args(l);
      e = timed(c, OSCARS_KERNEL_WGRAD,
                [&] { return launch_gemm(g, GEMM_WGRAD, c->bf16, ns, c->stream, c->tuner); });
      if (e != hipSuccess) return hip_fail(e);
    }
  }
  for (int k = 0; k < K; ++k) c->cursors[k] += tau[k];
  return OSCARS_OK;
}

oscars_status check_evaluate(const oscars_ctx* c, const float* params, const void* x,
                             const int32_t* y, int64_t n_rows, const double* loss_sum,
                             const int64_t* correct) {
  if (!c || !params || !x || !y || !loss_sum || !correct) return OSCARS_E_INVALID;
  if (!aligned16(params) || !aligned16(x)) return OSCARS_E_INVALID;
  if (n_rows < 1 || n_rows > 0x7FFFFFFF - 64) return OSCARS_E_INVALID;
  return OSCARS_OK;
}

// Device bytes of an evaluation's temporaries: results (double loss, int64
// count), then the row table [64 + n] int32, per-row losses [n] fp32 and
// correct flags [n] int32, each part 256-byte aligned.
struct EvalLayout {  // kNoAllocScratchBytes holds it for OSCARS_EVAL_NOALLOC_MAX_ROWS rows
  int64_t table, loss, hit, end;
  explicit EvalLayout(int64_t n) {
    table = 256;
    loss = table + round_up((64 + n) * 4, 256);
    hit = loss + round_up(n * 4, 256);
    end = hit + round_up(n * 4, 256);
  }
};

size_t eval_bytes(int64_t n_rows) { return static_cast<size_t>(EvalLayout(n_rows).end); }

// The forward pass of the local steps over rows 0 .. n_rows-1, max_batch rows
// at a time, into the temporaries at `buf` (eval_bytes(n_rows) bytes of
// device memory); then the fixed-order reduction and a copy of its two
// results to the host.  tune = false: no GEMM tiling is timed (no events are
// created); the tilings the context has decided, else the fixed rule.  Every
// tiling gives the same bits.  Waits for the context's stream.
hipError_t run_evaluate(oscars_ctx* c, const float* params, const void* x, const int32_t* y,
                        int64_t n_rows, void* buf, bool tune, double* loss_sum, int64_t* correct) {
  const EvalLayout lay(n_rows);
  char* base = static_cast<char*>(buf);
  struct Results {
    double loss;
    int64_t hits;
  };
  Results* d_res = reinterpret_cast<Results*>(base);
  int32_t* d_tab = reinterpret_cast<int32_t*>(base + lay.table);
  float* d_loss = reinterpret_cast<float*>(base + lay.loss);
  int32_t* d_hit = reinterpret_cast<int32_t*>(base + lay.hit);
  const int L = c->L, Bmax = c->max_batch;
  const uint32_t prof_mask = c->prof_mask;  // evaluation launches are never profiled
  c->prof_mask = 0;
  hipError_t e = launch_eval_rows(d_tab, n_rows, c->stream);
  // Weights as the forward pass reads them: the bf16 copy of params (one
  // cast into the start-model buffer) or params themselves.
  if (e == hipSuccess && c->bf16)
    e = launch_cast_bf16(params, 0, d_tab, c->gq, 0, c->n_pad, 1, c->stream);
  for (int64_t i0 = 0; i0 < n_rows && e == hipSuccess; i0 += Bmax) {
    const int N = static_cast<int>(std::min<int64_t>(Bmax, n_rows - i0));
    const int32_t* rows = d_tab + 64 + i0;
    if (c->cnn) {
      e = cnn_forward(c, params, 0, d_tab, x, rows, 0, N, 1);
      if (e == hipSuccess)
        e = launch_softmax_ce(c->logits, c->ld[L], c->act_slot(L), c->dims[L], N, y, rows, 0,
                              c->delta[L], false, d_loss + i0, 0, 1, c->stream, d_hit + i0);
      continue;
    }
    for (int l = 1; l <= L && e == hipSuccess; ++l) {
      GemmArgs g{};
      g.M = c->dims[l];
      g.N = N;
      g.K = c->dims[l - 1];
      g.a_ext = g.K;
      g.b_ext = g.K;
      g.a = c->bf16 ? static_cast<const void*>(c->gq + c->w_off[l])
                    : static_cast<const void*>(params + c->w_off[l]);
      g.a_ld = c->dims[l - 1];
      if (l == 1) {
        g.b = x;
        g.b_ld = c->dims[0];
        g.gather = rows;
        g.rows_out = c->act[0];
        g.rows_out_ld = c->ld[0];
      } else {
        g.b = c->act[l - 1];
        g.b_ld = c->ld[l - 1];
      }
      g.master = const_cast<float*>(params);  // not written by the forward pass
      g.master_in = params;
      g.b_off = c->b_off[l];
      g.w_off = c->w_off[l];
      g.order = d_tab;
      g.part = c->part;
      g.part_cap = c->part_cap;
      g.out = l < L ? c->act[l] : static_cast<void*>(c->logits);
      g.relu = l < L;
      g.out_bf16 = l < L && c->bf16;
      g.out_ld = c->ld[l];
      e = launch_gemm(g, GEMM_FWD, c->bf16, 1, c->stream, c->tuner, tune);
    }
    if (e == hipSuccess)
      e = launch_softmax_ce(c->logits, c->ld[L], c->act_slot(L), c->dims[L], N, y, rows, 0,
                            c->delta[L], c->bf16, d_loss + i0, 0, 1, c->stream, d_hit + i0);
  }
  c->prof_mask = prof_mask;
  if (e == hipSuccess)
    e = launch_eval_reduce(d_loss, d_hit, n_rows, &d_res->loss, &d_res->hits, c->stream);
  Results h{};
  if (e == hipSuccess)
    e = hipMemcpyAsync(&h, d_res, sizeof(Results), hipMemcpyDeviceToHost, c->stream);
  if (e == hipSuccess) e = hipStreamSynchronize(c->stream);
  if (e != hipSuccess) return e;
  *loss_sum = h.loss;
  *correct = h.hits;
  return hipSuccess;
}

}  // namespace

extern "C" {

oscars_status oscars_local_steps(oscars_ctx* c, float* replicas, const oscars_shards* s,
                                 const int32_t* tau, float lr, int32_t batch) {
  return run_local_steps(c, replicas, nullptr, s, tau, lr, batch);
}

oscars_status oscars_round(oscars_ctx* c, float* global, float* replicas, const oscars_shards* s,
                           const int32_t* tau, float lr, int32_t batch, const float* weights) {
  if (!c || !global || !replicas || !weights) return OSCARS_E_INVALID;
  if (!aligned16(global)) return OSCARS_E_INVALID;
  for (int k = 0; k < c->K; ++k)
    if (!std::isfinite(weights[k])) return OSCARS_E_INVALID;
  const uintptr_t g0 = reinterpret_cast<uintptr_t>(global), g1 = g0 + c->n_pad * sizeof(float);
  const uintptr_t r0 = reinterpret_cast<uintptr_t>(replicas),
                  r1 = r0 + static_cast<uintptr_t>(c->K) * c->n_pad * sizeof(float);
  if (g0 < r1 && r0 < g1) return OSCARS_E_INVALID;
  oscars_status st = run_local_steps(c, replicas, global, s, tau, lr, batch);
  if (st != OSCARS_OK) return st;
  hipError_t e = timed(c, OSCARS_KERNEL_AGGREGATE, [&] {
    return launch_aggregate(global, replicas, weights, c->K, c->n_pad, c->n_pad, 0, c->stream);
  });
  return e == hipSuccess ? OSCARS_OK : hip_fail(e);
}

oscars_status oscars_round_losses(oscars_ctx* c, float* losses) {
  if (!c || !losses) return OSCARS_E_INVALID;
  for (int k = 0; k < c->K; ++k) losses[k] = NAN;
  const int n_slots = static_cast<int>(c->last_order.size());
  if (n_slots == 0) return OSCARS_OK;
  const int64_t cnt = static_cast<int64_t>(n_slots) * c->last_tau_max * c->last_B;
  std::vector<float> h(cnt);
  hipError_t e = hipStreamSynchronize(c->stream);
  if (e == hipSuccess)
    e = hipMemcpy(h.data(), c->loss_dev, cnt * sizeof(float), hipMemcpyDeviceToHost);
  if (e != hipSuccess) return hip_fail(e);
  for (int z = 0; z < n_slots; ++z) {
    const int k = c->last_order[z];
    double acc = 0.0;
    for (int j = 0; j < c->last_tau[k]; ++j)
      for (int b = 0; b < c->last_B; ++b)
        acc += h[(static_cast<int64_t>(z) * c->last_tau_max + j) * c->last_B + b];
    losses[k] = static_cast<float>(acc / (static_cast<double>(c->last_tau[k]) * c->last_B));
  }
  return OSCARS_OK;
}

oscars_status oscars_evaluate(oscars_ctx* c, const float* params, const void* x, const int32_t* y,
                              int64_t n_rows, double* loss_sum, int64_t* correct) {
  oscars_status st = check_evaluate(c, params, x, y, n_rows, loss_sum, correct);
  if (st != OSCARS_OK) return st;
  void* buf = nullptr;
  hipError_t e = hipMalloc(&buf, eval_bytes(n_rows));
  if (e != hipSuccess) return e == hipErrorOutOfMemory ? OSCARS_E_NOMEM : hip_fail(e);
  e = run_evaluate(c, params, x, y, n_rows, buf, true, loss_sum, correct);
  const hipError_t f = hipFree(buf);  // waits for the device
  if (e == hipSuccess) e = f;
  return e == hipSuccess ? OSCARS_OK : hip_fail(e);
}

oscars_status oscars_evaluate_noalloc(oscars_ctx* c, const float* params, const void* x,
                                      const int32_t* y, int64_t n_rows, double* loss_sum,
                                      int64_t* correct) {
  oscars_status st = check_evaluate(c, params, x, y, n_rows, loss_sum, correct);
  if (st != OSCARS_OK) return st;
  if (n_rows > OSCARS_EVAL_NOALLOC_MAX_ROWS) return OSCARS_E_INVALID;
  if (eval_bytes(n_rows) > kNoAllocScratchBytes) return OSCARS_E_INVALID;
  int dev = -1;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return hip_fail(e);
  if (dev != c->device || !c->noalloc_scratch) return OSCARS_E_STATE;
  e = run_evaluate(c, params, x, y, n_rows, c->noalloc_scratch, false, loss_sum, correct);
  return e == hipSuccess ? OSCARS_OK : hip_fail(e);
}

oscars_status oscars_aggregate(float* global, float* replicas, const float* weights, int32_t K,
                               int64_t n, int64_t ld, int32_t broadcast, void* hip_stream) {
  if (!global || !replicas || !weights) return OSCARS_E_INVALID;
  if (K < 1 || K > OSCARS_MAX_K || n < 1 || ld < n || ld % 4 != 0) return OSCARS_E_INVALID;
  if (!aligned16(global) || !aligned16(replicas)) return OSCARS_E_INVALID;
  for (int k = 0; k < K; ++k)
    if (!std::isfinite(weights[k])) return OSCARS_E_INVALID;
  const uintptr_t g0 = reinterpret_cast<uintptr_t>(global), g1 = g0 + n * sizeof(float);
  const uintptr_t r0 = reinterpret_cast<uintptr_t>(replicas),
                  r1 = r0 + ((K - 1) * ld + n) * sizeof(float);
  if (g0 < r1 && r0 < g1) return OSCARS_E_INVALID;
  hipError_t e = launch_aggregate(global, replicas, weights, K, n, ld, broadcast,
                                  static_cast<hipStream_t>(hip_stream));
  return e == hipSuccess ? OSCARS_OK : hip_fail(e);
}

oscars_status oscars_broadcast(const float* global, float* replicas, int32_t K, int64_t n,
                               int64_t ld, void* hip_stream) {
  if (!global || !replicas) return OSCARS_E_INVALID;
  if (K < 1 || K > OSCARS_MAX_K || n < 1 || ld < n || ld % 4 != 0) return OSCARS_E_INVALID;
  if (!aligned16(global) || !aligned16(replicas)) return OSCARS_E_INVALID;
  const uintptr_t g0 = reinterpret_cast<uintptr_t>(global), g1 = g0 + n * sizeof(float);
  const uintptr_t r0 = reinterpret_cast<uintptr_t>(replicas),
                  r1 = r0 + ((K - 1) * ld + n) * sizeof(float);
  if (g0 < r1 && r0 < g1) return OSCARS_E_INVALID;
  hipError_t e = launch_broadcast(global, replicas, K, n, ld, static_cast<hipStream_t>(hip_stream));
  return e == hipSuccess ? OSCARS_OK : hip_fail(e);
}

oscars_status oscars_set_gemm_tiling(oscars_ctx* c, int32_t tiling) {
  static_assert(OSCARS_TILING_COUNT == GEMM_TILING_COUNT && OSCARS_TILING_VS == GEMM_TILING_VS &&
                    OSCARS_TILING_LS == GEMM_TILING_LS,
                "tiling codes of the C ABI and of the launchers agree");
  if (!c || tiling < 0 || tiling >= OSCARS_TILING_COUNT) return OSCARS_E_INVALID;
  gemm_tuner_set_tiling(c->tuner, tiling);
  return OSCARS_OK;
}

oscars_status oscars_tuning_pending(const oscars_ctx* c, int32_t* configurations) {
  if (!c || !configurations) return OSCARS_E_INVALID;
  *configurations = gemm_tuner_pending(c->tuner);
  return OSCARS_OK;
}

oscars_status oscars_backward_path(const oscars_ctx* c, int32_t layer, int32_t batch,
                                   int32_t replicas, int32_t* fused) {
  if (!c || !fused || layer < 1 || layer > c->L || batch < 1 || batch > c->max_batch ||
      replicas < 1 || replicas > c->K)
    return OSCARS_E_INVALID;
  *fused = 0;
  if (c->cnn) {
    // conv layers 2 .. L - 1: backward-data and backward-weight in one launch
    if (layer < 2 || layer >= c->L) return OSCARS_OK;
    ConvArgs a = conv_layer_args(c, layer, nullptr, 0, nullptr, batch);
    ConvArgs ad = a;
    ad.cls = -1;
    conv_wgrad_ranges(a, &a.splits, &a.k_per_split);
    *fused = conv_pair_fits(ad, a, replicas) ? 1 : 0;
    return OSCARS_OK;
  }
  if (!c->bf16 || !backward_fused_enabled(c->backward_mode)) return OSCARS_OK;
  GemmArgs g{};
  g.M = c->dims[layer - 1];
  g.N = batch;
  g.K = c->dims[layer];
  if (!backward_fusable(g)) return OSCARS_OK;
  if (c->backward_mode != BACKWARD_AUTO) {
    *fused = 1;
    return OSCARS_OK;
  }
  if (c->cal_off) {  // no timing: fused
    *fused = 1;
    return OSCARS_OK;
  }
  const auto it = c->bwd_fused_choice.find(
      std::array<int, 5>{g.M, g.K, g.N, replicas, layer > 1 ? 1 : 0});
  *fused = it == c->bwd_fused_choice.end() ? -1 : (it->second > 0 ? 1 : 0);
  return OSCARS_OK;
}

oscars_status oscars_set_backward(oscars_ctx* c, int32_t mode) {
  static_assert(OSCARS_BACKWARD_COUNT == BACKWARD_MODE_COUNT &&
                    OSCARS_BACKWARD_FUSED_SPLIT == BACKWARD_FUSED_SPLIT,
                "backward modes of the C ABI and of the launchers agree");
  if (!c || mode < 0 || mode >= OSCARS_BACKWARD_COUNT) return OSCARS_E_INVALID;
  c->backward_mode = mode;
  return OSCARS_OK;
}

oscars_status oscars_profile_begin(oscars_ctx* c, uint32_t kind_mask) {
  if (!c || (kind_mask >> OSCARS_KERNEL_COUNT) != 0) return OSCARS_E_INVALID;
  c->prof_mask = kind_mask;
  c->prof_recs.clear();
  while (c->ev_pool.size() < 8192) {
    hipEvent_t ev;
    hipError_t e = hipEventCreate(&ev);
    if (e != hipSuccess) return hip_fail(e);
    c->ev_pool.push_back(ev);
  }
  return OSCARS_OK;
}

oscars_status oscars_profile_end(oscars_ctx* c, double* ms, int64_t* launches) {
  if (!c || !ms || !launches) return OSCARS_E_INVALID;
  for (int i = 0; i < OSCARS_KERNEL_COUNT; ++i) {
    ms[i] = 0.0;
    launches[i] = 0;
  }
  hipError_t e = hipStreamSynchronize(c->stream);
  if (e != hipSuccess) return hip_fail(e);
  for (const auto& r : c->prof_recs) {
    float t = 0.0f;
    e = hipEventElapsedTime(&t, c->ev_pool[r.second], c->ev_pool[r.second + 1]);
    if (e != hipSuccess) return hip_fail(e);
    ms[r.first] += t;
    launches[r.first] += 1;
  }
  c->prof_mask = 0;
  c->prof_recs.clear();
  return OSCARS_OK;
}

int32_t oscars_last_hip_error(void) { return g_last_hip; }

}  // extern "C"
