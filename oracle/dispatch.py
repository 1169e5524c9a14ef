"""Reference for skewness-aware dispatching (StreamRL Algorithm 2 with Equation 2).

TEST INFRASTRUCTURE ONLY: only ``tests/``, ``__graft_entry__.smoke()`` and the
benchmark's ``cpu_baseline`` leg may import this module. Plain Python, written
step by step from the algorithm.

What it computes (Section 5.3, "Skewness-aware Scheduling", the "Dispatching" part). A batch of
prompts with estimated output lengths is to be spread over N generation
instances. The prompts are sorted by estimate, longest first; the first
alpha fraction are long-tail samples, the rest regular. The P90 and P50 of an
output-length distribution D stand for the average output length of the two
groups. For every split N = N_l + N_r the latency of each group is estimated
with Equation 2,

    Latency = PTL(BS) * L_avg * ceil(M / BS),

where M is the number of prompts one instance of the group receives and
PTL(BS) the per-token decode latency at batch size BS (profiled beforehand),
and the split with the smallest total is chosen. Within each group the
samples are then spread evenly over the group's instances.

Readings where the paper is silent or ambiguous:
  * the long-tail group is the first floor(alpha * |P|) prompts; ties in the
    estimate keep index order;
  * P50 / P90 are lower-rank percentiles: element floor(q * (n - 1)) of the
    sorted sample;
  * M of an instance is ceil(group size / instances of the group), and BS is
    min(M, max_batch), max_batch standing for the KV-memory limit the paper
    mentions; Equation 2 is 0 for an empty group;
  * PTL between profiled batch sizes is linear interpolation; below the first
    point it is the first value, beyond the last it continues the last segment
    (a single profiled point gives a flat curve);
  * a group with samples needs at least one instance, an empty group may get
    none; splits are visited with N_l ascending and the first minimum is kept;
  * combining the two groups: Algorithm 2 adds the two latencies
    (combine="sum", the default); since the groups run on disjoint instances at
    the same time, the generation time is their maximum, available as
    combine="max";
  * "evenly distributed" within a group: the group's samples, in sorted order,
    are dealt round-robin to its instances (long-tail instances first, then
    regular ones).
"""
from __future__ import annotations

import math


def percentile_lower(values, q: float) -> int:
    """Lower-rank percentile: the sorted sample's element at floor(q * (n - 1))."""
    v = sorted(int(x) for x in values)
    return v[int(math.floor(q * (len(v) - 1)))]


def ptl(batch: int, table_batch, table_seconds) -> float:
    """Per-token latency at ``batch`` from profiled points (piecewise linear)."""
    xs = [int(x) for x in table_batch]
    ys = [float(y) for y in table_seconds]
    if batch <= xs[0] or len(xs) == 1:      # one profiled point: a flat curve
        return ys[0]
    for k in range(1, len(xs)):
        if batch <= xs[k]:
            x0, x1, y0, y1 = xs[k - 1], xs[k], ys[k - 1], ys[k]
            return y0 + (y1 - y0) * (batch - x0) / (x1 - x0)
    x0, x1, y0, y1 = xs[-2], xs[-1], ys[-2], ys[-1]
    return y1 + (y1 - y0) * (batch - x1) / (x1 - x0)


def generation_latency(l_avg: float, m: int, max_batch: int, table_batch, table_seconds) -> float:
    """Equation 2 for one instance that receives ``m`` prompts."""
    if m == 0:
        return 0.0
    bs = min(m, max_batch)
    rounds = -(-m // bs)
    return ptl(bs, table_batch, table_seconds) * l_avg * rounds


def dispatch(est_len, alpha: float, dist, num_instances: int, table_batch, table_seconds, max_batch: int,
             combine: str = "sum"):
    """Algorithm 2. Returns (N_l, N_r, estimated latency, instance of every prompt)."""
    n = len(est_len)
    order = sorted(range(n), key=lambda i: (-int(est_len[i]), i))
    n_long = int(math.floor(alpha * n))
    long_tail, regular = order[:n_long], order[n_long:]
    l_alpha = percentile_lower(dist, 0.9)
    l_r = percentile_lower(dist, 0.5)
    best = None
    for n_l in range(0, num_instances + 1):
        n_r = num_instances - n_l
        if (long_tail and n_l == 0) or (regular and n_r == 0):
            continue
        lat_l = generation_latency(l_alpha, -(-len(long_tail) // n_l) if n_l else 0, max_batch,
                                   table_batch, table_seconds)
        lat_r = generation_latency(l_r, -(-len(regular) // n_r) if n_r else 0, max_batch,
                                   table_batch, table_seconds)
        total = lat_l + lat_r if combine == "sum" else max(lat_l, lat_r)
        if best is None or total < best[2]:
            best = (n_l, n_r, total)
    if best is None:
        raise ValueError("no valid split (N too small for the non-empty groups)")
    n_l, n_r, total = best
    instance = [-1] * n
    for k, i in enumerate(long_tail):
        instance[i] = k % n_l
    for k, i in enumerate(regular):
        instance[i] = n_l + k % n_r
    return n_l, n_r, total, instance
