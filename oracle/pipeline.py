"""Modelled completion time of a pipelined cold request, and the best grouping by exhaustion.

Test infrastructure only. Paper Sec. 4.3 ("Model swapping and pipeline execution"): the
layers' transfers are grouped; each group is one transfer whose completion lets the
layers it holds start, so later transfers overlap earlier layers' computation; groups
that are too small pay a fixed synchronisation cost per transfer, groups that are too
large delay the layers waiting for them.

Reading (the paper gives no formula): one copy engine moves the groups back to back, a
group costing a fixed ``chunk_us`` plus its bytes at ``rate`` bytes per microsecond; the
compute engine runs the layers in order, layer ``u`` for ``unit_us[u]``; the first layer of
a group may start only ``wait_us`` after its group has landed. The completion time is when
the last layer ends. Groups are contiguous runs of layers; group 0 starts at byte 0 and
the last group ends at the buffer end.

``simulate`` steps through the two engines one event at a time; ``best_grouping`` tries
every grouping (2^(n-1) of them) and keeps the fastest, preferring fewer groups on ties.
Both are for small n; they share nothing with the library's dynamic program.
"""
from __future__ import annotations

import itertools


def _group_bytes(unit_begin, total_bytes, first):
    ends = list(first[1:]) + [None]
    out = []
    for g, (a, b) in enumerate(zip(first, ends)):
        lo = 0 if g == 0 else unit_begin[a]
        hi = total_bytes if b is None else unit_begin[b]
        out.append(hi - lo)
    return out


def simulate(unit_begin, total_bytes, unit_us, first, rate, chunk_us, wait_us):
    """Completion time (us) of the grouping whose groups start at units ``first``."""
    n = len(unit_begin)
    assert first and first[0] == 0 and all(a < b for a, b in zip(first, first[1:])) and first[-1] < n
    sizes = _group_bytes(unit_begin, total_bytes, first)
    # copy engine: the events "group g has landed"
    landed = []
    clock = 0.0
    for nb in sizes:
        clock = clock + chunk_us + nb / rate
        landed.append(clock)
    # compute engine: layers in order
    group_of = {}
    for g, a in enumerate(first):
        b = first[g + 1] if g + 1 < len(first) else n
        for u in range(a, b):
            group_of[u] = g
    now = 0.0
    for u in range(n):
        g = group_of[u]
        if u == first[g]:
            now = max(now, landed[g] + wait_us)
        now = now + unit_us[u]
    return now


def best_grouping(unit_begin, total_bytes, unit_us, rate, chunk_us, wait_us, rel_tol=1e-9):
    """(first units, time) of the fastest grouping; among equally fast ones the fewest groups."""
    n = len(unit_begin)
    best = None
    for k in range(n):                      # k boundaries -> k + 1 groups, fewest first
        for cut in itertools.combinations(range(1, n), k):
            first = [0, *cut]
            t = simulate(unit_begin, total_bytes, unit_us, first, rate, chunk_us, wait_us)
            if best is None or t < best[1] * (1 - rel_tol) - 1e-12:
                best = (first, t)
    return best
