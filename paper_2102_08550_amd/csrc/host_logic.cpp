// Algorithm 1, Eq. 4 weights, shard offsets and the mini-batch sampler.
// Host only; see oscars.h for the contract of each entry point.
#include "host_logic.h"

#include <cmath>
#include <cstring>

#include "../../include/oscars.h"

namespace oscars {

void epoch_order(uint64_t seed, uint32_t k, uint64_t e, int64_t n, std::vector<int32_t>& out) {
  out.resize(static_cast<size_t>(n));
  for (int64_t i = 0; i < n; ++i) out[i] = static_cast<int32_t>(i);
  SplitMix64 rng(seed ^ ((static_cast<uint64_t>(k) << 32) | e));
  for (int64_t i = n - 1; i >= 1; --i) {
    const uint64_t j = rng.next() % static_cast<uint64_t>(i + 1);
    const int32_t t = out[i];
    out[i] = out[j];
    out[j] = t;
  }
}

void WorkerSampler::reset(uint64_t seed, uint32_t k, int64_t first, int64_t n_k) {
  if (seed != seed_ || k != k_ || first != first_ || n_k != n_k_) epoch_ = -1;
  seed_ = seed;
  k_ = k;
  first_ = first;
  n_k_ = n_k;
}

int64_t WorkerSampler::row(int64_t p) {
  const int64_t e = p / n_k_;
  if (e != epoch_) {
    epoch_order(seed_, k_, static_cast<uint64_t>(e), n_k_, order_);
    epoch_ = e;
  }
  return first_ + order_[static_cast<size_t>(p % n_k_)];
}

}  // namespace oscars

using namespace oscars;

extern "C" {

oscars_status oscars_load_balance(const int64_t* t_iter, int32_t N, int64_t M, int64_t* T_star,
                                  int32_t* tau) {
  if (!t_iter || !T_star || !tau || N < 1 || M < 1) return OSCARS_E_INVALID;
  int64_t tmin = t_iter[0], tmax = t_iter[0];
  for (int32_t i = 0; i < N; ++i) {
    if (t_iter[i] < 1) return OSCARS_E_INVALID;
    if (t_iter[i] < tmin) tmin = t_iter[i];
    if (t_iter[i] > tmax) tmax = t_iter[i];
  }
  // Side condition of Eq. 3: floor(T/min t) - floor(T/max t) < M.
  auto feasible = [&](int64_t T) { return T / tmin - T / tmax < M; };
  int64_t T = tmax;
  if (!feasible(T)) return OSCARS_E_INFEASIBLE;
  int64_t best_T = T, best_wait = INT64_MAX;
  // Algorithm 1: each candidate T has maximal wait max_i mod(T, t_i) (Eq. 1, 2);
  // keep the first T with the least maximal wait.  A zero wait cannot be
  // beaten, and stopping there also ends the scan for equal t_i.
  while (feasible(T)) {
    int64_t w = 0;
    for (int32_t i = 0; i < N; ++i) {
      const int64_t r = T % t_iter[i];
      if (r > w) w = r;
    }
    if (w < best_wait) {
      best_wait = w;
      best_T = T;
    }
    if (w == 0) break;
    if (T == INT64_MAX) break;
    ++T;
  }
  *T_star = best_T;
  for (int32_t i = 0; i < N; ++i) tau[i] = static_cast<int32_t>(best_T / t_iter[i]);
  return OSCARS_OK;
}

oscars_status oscars_plan_tau(const double* t_measured, int32_t N, int32_t resolution, int64_t M,
                              int64_t* ticks, int64_t* T_star, int32_t* tau) {
  if (!t_measured || !T_star || !tau || N < 1 || M < 1) return OSCARS_E_INVALID;
  if (resolution < 1 || resolution > OSCARS_MAX_RESOLUTION) return OSCARS_E_INVALID;
  double tmin = t_measured[0];
  for (int32_t i = 0; i < N; ++i) {
    const double v = t_measured[i];
    if (!std::isfinite(v) || !(v > 0.0)) return OSCARS_E_INVALID;
    if (v < tmin) tmin = v;
  }
  // The fastest worker is `resolution` ticks; every time becomes the nearest
  // whole number of ticks (halves up), at least one.
  const double tick = tmin / resolution;
  std::vector<int64_t> q(N);
  for (int32_t i = 0; i < N; ++i) {
    const double x = std::floor(t_measured[i] / tick + 0.5);
    if (!(x <= static_cast<double>(OSCARS_MAX_TICKS))) return OSCARS_E_INVALID;
    q[i] = x < 1.0 ? 1 : static_cast<int64_t>(x);
  }
  const oscars_status st = oscars_load_balance(q.data(), N, M, T_star, tau);
  if (st == OSCARS_OK && ticks) std::copy(q.begin(), q.end(), ticks);
  return st;
}

oscars_status oscars_paper_weights(const int32_t* staleness, int32_t K, float* w) {
  (void)staleness;  // Eq. 4 averages uniformly; staleness does not enter.
  if (!w || K < 1) return OSCARS_E_INVALID;
  const float v = 1.0f / static_cast<float>(K);
  for (int32_t k = 0; k < K; ++k) w[k] = v;
  return OSCARS_OK;
}

oscars_status oscars_shard_offsets(int64_t n_rows, int32_t K, int64_t* offsets) {
  if (!offsets || K < 1 || n_rows < 0) return OSCARS_E_INVALID;
  for (int32_t k = 0; k <= K; ++k) {
    // floor(k * n / K) without overflow for n < 2^62, K < 2^31.
    const int64_t q = n_rows / K, r = n_rows % K;
    offsets[k] = q * k + (r * k) / K;
  }
  return OSCARS_OK;
}

oscars_status oscars_sample_indices(const oscars_shards* s, int32_t K, int32_t k,
                                    int64_t first_step, int32_t steps, int32_t batch,
                                    int64_t* rows_out) {
  if (!s || !s->offsets || !rows_out || K < 1 || k < 0 || k >= K || first_step < 0 ||
      steps < 0 || batch < 1)
    return OSCARS_E_INVALID;
  const int64_t lo = s->offsets[k], hi = s->offsets[k + 1];
  if (lo < 0 || hi <= lo || hi > s->n_rows) return OSCARS_E_INVALID;
  WorkerSampler ws;
  ws.reset(s->seed, static_cast<uint32_t>(k), lo, hi - lo);
  for (int64_t j = 0; j < steps; ++j)
    for (int32_t b = 0; b < batch; ++b)
      rows_out[j * batch + b] = ws.row((first_step + j) * batch + b);
  return OSCARS_OK;
}

const char* oscars_status_str(oscars_status s) {
  switch (s) {
    case OSCARS_OK: return "ok";
    case OSCARS_E_INVALID: return "invalid argument";
    case OSCARS_E_NOMEM: return "out of memory";
    case OSCARS_E_HIP: return "HIP error";
    case OSCARS_E_INFEASIBLE: return "barrier constraint infeasible at T = max t";
    case OSCARS_E_STATE: return "invalid state";
    default: return "unknown status";
  }
}

}  // extern "C"
