// Dynamic packing scheduler of the paper's Alg. 1 (Sec. 3.4), host side.
//
// Phase 1, best-fit packing: a segment tree over the residual capacities
// [0, L] keeps, at each internal node, the largest residual of the non-empty
// leaves below it. A sequence of length l descends to the leftmost leaf
// r >= l, i.e. the open microbatch with the smallest residual that still
// holds it, in O(log L); within a leaf the microbatch opened first wins. A
// sequence that fits nowhere opens a new microbatch. A microbatch whose
// residual drops below the shortest length of the call leaves the tree.
//
// Phase 2, two-dimension load balancing: Eq. 3 cost of every microbatch
// (kept exact as L * sum(l) + l_max^2), buckets of similar cost by
// one-dimensional k-means with exact rational centroids, then each bucket's
// microbatches in decreasing cost dealt to the ranks in zig-zag order.

#include "schedule.h"

#include <algorithm>
#include <numeric>
#include <set>
#include <unordered_map>

namespace fp {
namespace {

// Max-tree over leaves 0..L; a leaf holds r when some open microbatch has
// residual r, else -1.
class ResidualTree {
 public:
  explicit ResidualTree(int32_t capacity) {
    size_ = 1;
    while (size_ < capacity + 1) size_ <<= 1;
    t_.assign(2 * (size_t)size_, -1);
  }
  void set(int32_t r, bool occupied) {
    size_t i = (size_t)r + size_;
    t_[i] = occupied ? r : -1;
    for (i >>= 1; i; i >>= 1) t_[i] = std::max(t_[2 * i], t_[2 * i + 1]);
  }
  // Smallest occupied leaf r >= l, or -1.
  int32_t best_fit(int32_t l) const {
    if (t_[1] < l) return -1;
    size_t i = 1;
    while (i < (size_t)size_) i = (t_[2 * i] >= l) ? 2 * i : 2 * i + 1;
    return (int32_t)(i - size_);
  }

 private:
  int32_t size_;
  std::vector<int32_t> t_;
};

void best_fit(const int32_t* lengths, int32_t n, int32_t capacity, PackingPlan* out) {
  out->mb_of_seq.assign((size_t)n, -1);
  if (n == 0) return;
  const int32_t l_min = *std::min_element(lengths, lengths + n);
  ResidualTree tree(capacity);
  std::unordered_map<int32_t, std::set<int32_t>> at;   // residual -> open microbatches
  std::vector<int32_t> residual;
  auto leave = [&](int32_t j) {
    auto it = at.find(residual[(size_t)j]);
    it->second.erase(j);
    if (it->second.empty()) {
      tree.set(it->first, false);
      at.erase(it);
    }
  };
  auto enter = [&](int32_t j) {
    auto& s = at[residual[(size_t)j]];
    if (s.empty()) tree.set(residual[(size_t)j], true);
    s.insert(j);
  };
  for (int32_t i = 0; i < n; ++i) {
    const int32_t l = lengths[i];
    const int32_t r = tree.best_fit(l);
    int32_t j;
    if (r >= 0) {
      j = *at[r].begin();
      leave(j);
    } else {
      j = (int32_t)residual.size();
      residual.push_back(capacity);
      out->tokens.push_back(0);
      out->max_len.push_back(0);
    }
    residual[(size_t)j] -= l;
    out->tokens[(size_t)j] += l;
    out->max_len[(size_t)j] = std::max(out->max_len[(size_t)j], l);
    out->mb_of_seq[(size_t)i] = j;
    if (residual[(size_t)j] >= l_min) enter(j);
  }
}

// |x - S/c| for centroid S/c, compared exactly: |x c_a - S_a| c_b < |x c_b - S_b| c_a.
struct Centroid {
  __int128 sum;
  int64_t count;
};

bool closer(int64_t x, const Centroid& a, const Centroid& b) {
  __int128 da = (__int128)x * a.count - a.sum;
  __int128 db = (__int128)x * b.count - b.sum;
  if (da < 0) da = -da;
  if (db < 0) db = -db;
  return da * b.count < db * a.count;
}

void kmeans(const std::vector<int64_t>& x, int32_t n_buckets, std::vector<int32_t>* bucket) {
  const int64_t m = (int64_t)x.size();
  bucket->assign((size_t)m, 0);
  if (m == 0) return;
  const int64_t k_n = std::min<int64_t>(n_buckets, m);
  std::vector<int32_t> order((size_t)m);
  std::iota(order.begin(), order.end(), 0);
  std::stable_sort(order.begin(), order.end(), [&](int32_t a, int32_t b) { return x[(size_t)a] < x[(size_t)b]; });
  std::vector<Centroid> c((size_t)k_n);
  for (int64_t k = 0; k < k_n; ++k) c[(size_t)k] = Centroid{x[(size_t)order[(size_t)((2 * k + 1) * m / (2 * k_n))]], 1};
  std::vector<int32_t> assign((size_t)m, -1), next((size_t)m);
  for (int round = 0; round < kKmeansRounds; ++round) {
    for (int64_t j = 0; j < m; ++j) {
      int32_t best = 0;
      for (int32_t k = 1; k < (int32_t)k_n; ++k)
        if (closer(x[(size_t)j], c[(size_t)k], c[(size_t)best])) best = k;
      next[(size_t)j] = best;
    }
    if (next == assign) break;
    assign.swap(next);
    std::vector<Centroid> acc((size_t)k_n, Centroid{0, 0});
    for (int64_t j = 0; j < m; ++j) {
      acc[(size_t)assign[(size_t)j]].sum += x[(size_t)j];
      acc[(size_t)assign[(size_t)j]].count += 1;
    }
    for (int64_t k = 0; k < k_n; ++k)
      if (acc[(size_t)k].count) c[(size_t)k] = acc[(size_t)k];
  }
  *bucket = assign;
}

}  // namespace

void dynamic_packing(const int32_t* lengths, int32_t n, int32_t capacity, int32_t n_ranks,
                     int32_t n_buckets, PackingPlan* out) {
  *out = PackingPlan{};
  best_fit(lengths, n, capacity, out);
  const size_t m = out->tokens.size();
  out->cost.resize(m);
  for (size_t j = 0; j < m; ++j)
    out->cost[j] = (int64_t)capacity * out->tokens[j] + (int64_t)out->max_len[j] * out->max_len[j];
  kmeans(out->cost, n_buckets, &out->bucket);

  out->rank.assign(m, -1);
  out->slot.assign(m, -1);
  std::vector<int32_t> next_slot((size_t)n_ranks, 0);
  const int32_t n_b = m ? *std::max_element(out->bucket.begin(), out->bucket.end()) + 1 : 0;
  std::vector<std::vector<int32_t>> lists((size_t)n_b);
  for (size_t j = 0; j < m; ++j) lists[(size_t)out->bucket[j]].push_back((int32_t)j);
  for (int32_t b = n_b - 1; b >= 0; --b) {
    std::vector<int32_t>& lst = lists[(size_t)b];
    std::stable_sort(lst.begin(), lst.end(),
                     [&](int32_t u, int32_t v) { return out->cost[(size_t)u] > out->cost[(size_t)v]; });
    // Zig-zag: ranks 0..N-1, then N-1..0, restarting forward for each bucket.
    size_t a = 0;
    bool forward = true;
    while (a < lst.size()) {
      for (int32_t s = 0; s < n_ranks && a < lst.size(); ++s, ++a) {
        const int32_t r = forward ? s : n_ranks - 1 - s;
        out->rank[(size_t)lst[a]] = r;
        out->slot[(size_t)lst[a]] = next_slot[(size_t)r]++;
      }
      forward = !forward;
    }
  }
}

}  // namespace fp
