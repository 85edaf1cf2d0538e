// Random draws of retraining: the uniform training subset of the window
// (section 4.3, "Training data sampling") and the per-epoch visiting order.
//
// Generator: SplitMix64 (Steele, Lea and Flood, OOPSLA 2014): the state
// advances by the golden-ratio increment 0x9E3779B97F4A7C15 and each output is
// the state passed through the variant-13 finaliser (xor-shift 30, multiply
// 0xBF58476D1CE4E5B9, xor-shift 27, multiply 0x94D049BB133111EB, xor-shift 31).
// Shuffle: Fisher-Yates in Durstenfeld's in-place form, run forwards: step i
// swaps position i with a position drawn uniformly from [i, n), the draw being
// (next output) mod (n - i).  Running only `count` steps gives a uniform
// ordered sample of `count` distinct items.
// Seeds: the subset uses start state `seed`; epoch e (0-based) uses
// seed + (e + 1) * 0xD1B54A32D192ED03 (mod 2^64).
#include "rng.hpp"

#include <cmath>
#include <numeric>

namespace ekya {

namespace {
struct SplitMix64 {
  uint64_t s;
  explicit SplitMix64(uint64_t seed) : s(seed) {}
  uint64_t operator()() {
    s += 0x9E3779B97F4A7C15ULL;
    uint64_t z = s;
    z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ULL;
    z = (z ^ (z >> 27)) * 0x94D049BB133111EBULL;
    return z ^ (z >> 31);
  }
};
}  // namespace

int subset_count(int n_frames, double frac) {
  double v = std::floor(frac * (double)n_frames + 0.5);
  int c = (int)v;
  return c < 1 ? 1 : c;
}

std::vector<int32_t> partial_shuffle(int n, int count, uint64_t seed) {
  std::vector<int32_t> a(n);
  std::iota(a.begin(), a.end(), 0);
  SplitMix64 g(seed);
  for (int i = 0; i < count; ++i) {
    const uint64_t span = (uint64_t)(n - i);
    const int j = i + (int)(g() % span);
    std::swap(a[i], a[j]);
  }
  a.resize(count);
  return a;
}

std::vector<int32_t> training_subset(int n_frames, double frac, uint64_t seed) {
  return partial_shuffle(n_frames, subset_count(n_frames, frac), seed);
}

std::vector<int32_t> epoch_order(int n, uint64_t seed, int epoch) {
  return partial_shuffle(n, n, seed + (uint64_t)(epoch + 1) * 0xD1B54A32D192ED03ULL);
}

}  // namespace ekya
