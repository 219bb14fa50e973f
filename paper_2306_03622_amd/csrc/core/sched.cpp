#include "sched.hpp"

#include <algorithm>
#include <cmath>
#include <numeric>

namespace tp {

double rrc(uint64_t n, uint64_t m, double p) { return (p * (double)n - (double)m) / (1.0 - p); }

std::vector<uint8_t> high_group(const std::vector<double>& r, double alpha) {
  const size_t nf = r.size();
  std::vector<size_t> order(nf);
  std::iota(order.begin(), order.end(), 0);
  std::stable_sort(order.begin(), order.end(), [&](size_t a, size_t b) { return r[a] < r[b]; });
  double total = 0;
  for (double v : r) total += std::max(v, 0.0);
  const double limit = alpha * total;
  std::vector<uint8_t> high(nf, 0);
  double prefix = 0;
  for (size_t j = 0; j < nf; ++j) {
    prefix += std::max(r[order[j]], 0.0);
    if (prefix > limit) break;
    high[order[j]] = 1;
  }
  return high;
}

int32_t sched_pick(const std::vector<double>& r, const std::vector<uint8_t>& high,
                   const std::vector<int32_t>& pending_func) {
  int32_t best_f = -1;
  bool best_high = false;
  for (int32_t f : pending_func) {
    const bool h = high[f] != 0;
    if (best_f < 0 || (h && !best_high)) {
      best_f = f;
      best_high = h;
      continue;
    }
    if (h != best_high) continue;
    // high group: larger RRC first; low group: smaller RRC first; ties: lower index
    const bool better = h ? (r[f] > r[best_f] || (r[f] == r[best_f] && f < best_f))
                          : (r[f] < r[best_f] || (r[f] == r[best_f] && f < best_f));
    if (better) best_f = f;
  }
  if (best_f < 0) return -1;
  for (size_t i = 0; i < pending_func.size(); ++i)
    if (pending_func[i] == best_f) return (int32_t)i;
  return -1;
}

double alpha_update(double alpha, double last_ratio, double new_ratio, double scalar, double threshold) {
  // TCP-like: the change in the compliant share, outside a dead band of +-|threshold|, sets
  // the direction; alpha moves one factor of `scalar` that way and stays at most 1
  const double band = std::fabs(threshold), change = new_ratio - last_ratio;
  const int direction = (change > band) - (change < -band);
  return std::min(alpha * std::pow(scalar, direction), 1.0);
}

}  // namespace tp
