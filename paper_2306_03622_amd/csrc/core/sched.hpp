// SLO-aware request queueing (paper Sec. 5.3 "Request queueing" and the appendix "Function
// request prioritization"): the required request count (RRC) of each function, the split of
// functions into a high- and a low-priority group by a threshold alpha, the choice of the
// next queued request, and the periodic adjustment of alpha. Host-only C++.
#pragma once
#include <cstdint>
#include <vector>

namespace tp {

// RRC = (p n - m) / (1 - p): the number of further requests a function must serve within
// its deadline for m' / n' to reach the tail percentile p, from (m + RRC) / (n + RRC) = p,
// with n requests served so far and m of them within the deadline. 0 < p < 1.
double rrc(uint64_t n, uint64_t m, double p);

// Functions sorted by RRC ascending (ties: lower index first); the first k form the high-
// priority group, k the largest with sum_{j<=k} max(RRC_j, 0) <= alpha * sum_i max(RRC_i, 0).
// Returns 1 for members of the high group.
std::vector<uint8_t> high_group(const std::vector<double>& rrc, double alpha);

// The queued request to run next. pending_func lists the function of every queued request in
// arrival order. High-priority functions go first, the one with the largest RRC first (ties:
// lower index); otherwise the low-priority function with the smallest RRC (ties: lower
// index); within a function, the earliest arrival. Returns an index into pending_func, or -1
// if it is empty.
int32_t sched_pick(const std::vector<double>& rrc, const std::vector<uint8_t>& high,
                   const std::vector<int32_t>& pending_func);

// The periodic alpha auto-configuration (appendix "Function request prioritization", the
// algorithm of that name): when the share of SLO-compliant functions moved by more than
// |threshold| since the last period, alpha is scaled by scalar in the direction of the move
// (up when compliance improved, down when it worsened), never above 1; otherwise unchanged.
double alpha_update(double alpha, double last_ratio, double new_ratio, double scalar, double threshold);

}  // namespace tp
