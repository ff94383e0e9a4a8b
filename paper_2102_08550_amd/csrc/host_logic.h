// Host-side parts of the hot path that need no GPU: Algorithm 1, shard
// assignment and the mini-batch sampler.  Pure C++17 (no HIP), so the same
// source also builds into a host-only library for CPU tests.
#pragma once

#include <cstdint>
#include <vector>

namespace oscars {

// SplitMix64 (Steele, Lea and Flood, OOPSLA 2014): the state advances by the
// golden gamma and each output is the state through the variant-13 finaliser.
struct SplitMix64 {
  uint64_t state;
  explicit SplitMix64(uint64_t s) : state(s) {}
  uint64_t next() {
    state += 0x9E3779B97F4A7C15ull;
    uint64_t z = state;
    z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
    z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
    return z ^ (z >> 31);
  }
};

// Epoch order of one worker's shard: Durstenfeld shuffle of 0..n-1 with
// j = r mod (i + 1), r from SplitMix64 seeded with seed ^ ((k << 32) | e).
void epoch_order(uint64_t seed, uint32_t k, uint64_t e, int64_t n, std::vector<int32_t>& out);

// Streams one worker's sample rows, keeping the current epoch's order cached.
class WorkerSampler {
 public:
  void reset(uint64_t seed, uint32_t k, int64_t first, int64_t n_k);
  // Global row of sample number p (p = step * batch + b) of this worker.
  int64_t row(int64_t p);

 private:
  uint64_t seed_ = 0;
  uint32_t k_ = 0;
  int64_t first_ = 0, n_k_ = 0;
  int64_t epoch_ = -1;
  std::vector<int32_t> order_;
};

}  // namespace oscars
