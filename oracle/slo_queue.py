"""SLO-aware request queueing (oracle).

Test infrastructure only. Paper Sec. 5.3 ("Request queueing") and the appendix "Function
request prioritization":

* A function's required request count is RRC = (p n - m) / (1 - p), where n requests have
  been served, m of them within the deadline, and p is the SLO's tail percentile; it solves
  (m + RRC) / (n + RRC) = p. A smaller RRC means the function is closer to meeting its SLO.
* With the functions sorted by RRC, the first k form the high-priority group, k the largest
  integer with sum_{j<=k} max(RRC_j, 0) <= alpha * sum_i max(RRC_i, 0).
* Requests of the high-priority group run first, in reverse order of RRC (largest first);
  those of the low-priority group in order of RRC (smallest first).
* alpha is adjusted periodically from the share of SLO-compliant functions, in the manner
  of TCP congestion control (the appendix's alpha auto-configuration): a rise of the share
  by more than |threshold| since the last period grows alpha by the factor `scalar`, a fall
  by more than |threshold| shrinks it by the same factor, and alpha never exceeds 1.

Readings where the paper is silent: ties in RRC go to the lower function index, both when
sorting and when choosing; within a function, requests run in arrival order; the sums run
over every function of the node.
"""
from __future__ import annotations


def rrc(n: int, m: int, p: float) -> float:
    return (p * n - m) / (1.0 - p)


def high_group(rrcs, alpha: float):
    order = sorted(range(len(rrcs)), key=lambda f: (rrcs[f], f))
    total = sum(max(r, 0.0) for r in rrcs)
    high = [False] * len(rrcs)
    prefix = 0.0
    for f in order:                      # grow the group while the prefix stays within the limit
        prefix += max(rrcs[f], 0.0)
        if prefix > alpha * total:
            break
        high[f] = True
    return high


def pick(rrcs, high, pending_func):
    """Index into pending_func (the function of each queued request, in arrival order) of the
    request to run next, or -1."""
    funcs = set(pending_func)
    if not funcs:
        return -1
    hi = [f for f in funcs if high[f]]
    if hi:
        target = sorted(hi, key=lambda f: (-rrcs[f], f))[0]
    else:
        target = sorted(funcs, key=lambda f: (rrcs[f], f))[0]
    return pending_func.index(target)


def alpha_update(alpha: float, last_ratio: float, new_ratio: float, scalar: float = 2.0,
                 threshold: float = 0.04) -> float:
    band = abs(threshold)
    change = new_ratio - last_ratio
    direction = (change > band) - (change < -band)     # +1 grow, -1 shrink, 0 hold
    return min(alpha * scalar ** direction, 1.0)
