// Heterogeneous parallel allocator of the paper (Sec. 3.3, Eq. 1-2), host side.
//
// Candidate pruning: encoders run DP x TP, the backbone DP x TP x PP. The
// paper's three pruning conditions become: DP divides the global batch; the
// configuration's device count DP x TP x PP (its module budget) fits the
// cluster, and PP divides the backbone's layers when a layer count is given
// (layers = 0: no layer rule); TP divides the devices of a node, so TP groups
// on consecutive devices never straddle two nodes.
//
// Flow matching: one configuration per module, total devices <= R,
// lexmax (G, -F) with G = min(T_enc, T_bb) and F = |T_enc - T_bb|. For a
// fixed backbone configuration (throughput t_b, budget left B) the best
// encoder choice is the smallest encoder sum >= t_b that fits B (then
// G = t_b and F is least), else the largest sum that fits B. So every
// encoder combination is listed once, grouped by sum, and a min-tree over
// the groups (cheapest combination of each sum) answers both questions per
// backbone configuration in O(log groups), instead of trying every
// combination against every backbone configuration.
// Ties: fewer devices, then the smallest choice vector (encoders, backbone).

#include "allocate.h"

#include <algorithm>
#include <limits>
#include <numeric>

namespace fp {
namespace {

struct Combo {
  int64_t sum;
  int64_t cost;
  std::vector<int32_t> idx;
};

// Min-tree over groups 0..n-1 holding each group's cheapest cost.
class MinTree {
 public:
  explicit MinTree(const std::vector<int64_t>& v) {
    n_ = 1;
    while (n_ < (int64_t)v.size()) n_ <<= 1;
    t_.assign(2 * (size_t)n_, std::numeric_limits<int64_t>::max());
    for (size_t i = 0; i < v.size(); ++i) t_[(size_t)n_ + i] = v[i];
    for (int64_t i = n_ - 1; i >= 1; --i) t_[(size_t)i] = std::min(t_[2 * (size_t)i], t_[2 * (size_t)i + 1]);
  }
  // Leftmost group >= lo whose cost <= budget, or -1.
  int64_t first_from(int64_t lo, int64_t budget) const { return first(1, 0, n_, lo, budget); }
  // Rightmost group whose cost <= budget, or -1.
  int64_t last_fit(int64_t budget) const {
    if (t_[1] > budget) return -1;
    size_t i = 1;
    while (i < (size_t)n_) i = (t_[2 * i + 1] <= budget) ? 2 * i + 1 : 2 * i;
    return (int64_t)i - n_;
  }

 private:
  int64_t first(size_t node, int64_t l, int64_t r, int64_t lo, int64_t budget) const {
    if (r <= lo || t_[node] > budget) return -1;
    if (r - l == 1) return l;
    const int64_t m = (l + r) / 2;
    const int64_t a = first(2 * node, l, m, lo, budget);
    return a >= 0 ? a : first(2 * node + 1, m, r, lo, budget);
  }
  int64_t n_;
  std::vector<int64_t> t_;
};

}  // namespace

std::vector<Config> prune_candidates(bool backbone, int32_t devices, int32_t per_node, int32_t global_batch,
                                     int32_t layers) {
  std::vector<Config> out;
  // PP ranges over the divisors of the layer count, or (layers = 0) over
  // every degree the device budget allows; encoders have PP = 1.
  const int32_t pp_max = !backbone ? 1 : (layers > 0 ? layers : devices);
  for (int32_t dp = 1; dp <= global_batch; ++dp) {
    if (global_batch % dp) continue;
    for (int32_t tp = 1; tp <= per_node; ++tp) {
      if (per_node % tp) continue;
      for (int32_t pp = 1; pp <= pp_max; ++pp) {
        if (layers > 0 && layers % pp) continue;
        if ((int64_t)dp * tp * pp > devices) break;   // larger pp only grows the product
        out.push_back(Config{dp, tp, pp});
      }
    }
  }
  return out;  // generated in increasing (dp, tp, pp) order
}

bool flow_match(const std::vector<std::vector<int64_t>>& tau, const std::vector<std::vector<int64_t>>& cost,
                int64_t budget, FlowChoice* out) {
  const size_t n_mod = tau.size();
  const size_t n_enc = n_mod - 1;
  // Every encoder combination that fits the budget on its own.
  std::vector<Combo> combos;
  std::vector<int32_t> idx(n_enc, 0);
  for (;;) {
    Combo c{0, 0, idx};
    for (size_t e = 0; e < n_enc; ++e) {
      c.sum += tau[e][(size_t)idx[e]];
      c.cost += cost[e][(size_t)idx[e]];
    }
    if (c.cost <= budget) combos.push_back(std::move(c));
    int64_t e = (int64_t)n_enc - 1;
    while (e >= 0 && ++idx[(size_t)e] == (int32_t)tau[(size_t)e].size()) idx[(size_t)e--] = 0;
    if (e < 0) break;
  }
  std::stable_sort(combos.begin(), combos.end(), [](const Combo& a, const Combo& b) {
    if (a.sum != b.sum) return a.sum < b.sum;
    if (a.cost != b.cost) return a.cost < b.cost;
    return a.idx < b.idx;
  });
  // Groups of equal sum; the first combination of a group is its best
  // (fewest devices, then smallest indices).
  std::vector<size_t> head;
  std::vector<int64_t> gsum, gcost;
  for (size_t i = 0; i < combos.size(); ++i) {
    if (i == 0 || combos[i].sum != combos[i - 1].sum) {
      head.push_back(i);
      gsum.push_back(combos[i].sum);
      gcost.push_back(combos[i].cost);
    }
  }
  if (head.empty()) return false;
  MinTree tree(gcost);
  bool found = false;
  FlowChoice best;
  const std::vector<int64_t>& tb = tau[n_mod - 1];
  const std::vector<int64_t>& cb = cost[n_mod - 1];
  for (size_t b = 0; b < tb.size(); ++b) {
    const int64_t left = budget - cb[b];
    if (left < 0) continue;
    const int64_t lo = (int64_t)(std::lower_bound(gsum.begin(), gsum.end(), tb[b]) - gsum.begin());
    int64_t g = tree.first_from(lo, left);
    if (g < 0) g = tree.last_fit(left);
    if (g < 0) continue;
    // The group's head is its cheapest combination (then smallest indices),
    // and it fits: the tree only returns groups whose cheapest cost fits.
    const Combo& c = combos[head[(size_t)g]];
    FlowChoice cand;
    cand.G = std::min(c.sum, tb[b]);
    cand.F = c.sum > tb[b] ? c.sum - tb[b] : tb[b] - c.sum;
    cand.devices = c.cost + cb[b];
    cand.choice = c.idx;
    cand.choice.push_back((int32_t)b);
    auto key_less = [](const FlowChoice& x, const FlowChoice& y) {
      if (x.G != y.G) return x.G > y.G;
      if (x.F != y.F) return x.F < y.F;
      if (x.devices != y.devices) return x.devices < y.devices;
      return x.choice < y.choice;
    };
    if (!found || key_less(cand, best)) {
      best = std::move(cand);
      found = true;
    }
  }
  if (found) *out = std::move(best);
  return found;
}

}  // namespace fp
