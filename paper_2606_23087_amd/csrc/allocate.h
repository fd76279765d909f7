// Heterogeneous parallel allocator (paper Sec. 3.3, Eq. 1-2): host code, no
// GPU. Not part of the public ABI; include/flowpool.h exposes it as
// alloc_candidates and plan_allocation.
#pragma once

#include <stdint.h>

#include <vector>

namespace fp {

struct Config {
  int32_t dp, tp, pp;
};

struct FlowChoice {
  std::vector<int32_t> choice;   // configuration index per module (encoders, then the backbone)
  int64_t G = 0, F = 0, devices = 0;
};

// Pruned configurations of one module in increasing (dp, tp, pp) order.
std::vector<Config> prune_candidates(bool backbone, int32_t devices, int32_t per_node, int32_t global_batch,
                                     int32_t layers);

// lexmax (G, -F) over one configuration per module within `budget` devices;
// tau/cost[i] list module i's configurations, the backbone last. Returns
// false when nothing fits.
bool flow_match(const std::vector<std::vector<int64_t>>& tau, const std::vector<std::vector<int64_t>>& cost,
                int64_t budget, FlowChoice* out);

}  // namespace fp
