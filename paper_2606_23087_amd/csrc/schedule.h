// Dynamic packing scheduler (paper Alg. 1, Sec. 3.4): host code, no GPU.
// Not part of the public ABI; include/flowpool.h exposes it as
// plan_dynamic_packing and plan_pool_packing.
#pragma once

#include <stdint.h>

#include <vector>

namespace fp {

struct PackingPlan {
  std::vector<int32_t> mb_of_seq;   // microbatch of each sequence (creation order)
  std::vector<int32_t> tokens;      // per microbatch
  std::vector<int32_t> max_len;
  std::vector<int64_t> cost;        // L * sum(l) + l_max^2 = L^2 * Cost(B) of Eq. 3
  std::vector<int32_t> bucket;      // cost bucket, 0 = lowest centroid
  std::vector<int32_t> rank;        // data-parallel rank it is dealt to
  std::vector<int32_t> slot;        // position in that rank's dispatch order
};

constexpr int kKmeansRounds = 100;

// Preconditions (checked by the caller): n >= 0, 1 <= capacity <= 2^20,
// every length in [1, capacity], n_ranks >= 1, n_buckets >= 1.
void dynamic_packing(const int32_t* lengths, int32_t n, int32_t capacity, int32_t n_ranks,
                     int32_t n_buckets, PackingPlan* out);

}  // namespace fp
