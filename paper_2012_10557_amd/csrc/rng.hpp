#pragma once
#include <stdint.h>

#include <vector>

namespace ekya {
int subset_count(int n_frames, double frac);
std::vector<int32_t> partial_shuffle(int n, int count, uint64_t seed);
std::vector<int32_t> training_subset(int n_frames, double frac, uint64_t seed);
std::vector<int32_t> epoch_order(int n, uint64_t seed, int epoch);
}  // namespace ekya
