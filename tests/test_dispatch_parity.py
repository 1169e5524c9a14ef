"""The library's skewness-aware dispatching (C++, include/sl_dispatch.h) against the oracle.

Both sides perform the same binary64 operations in the same order, so the
plans (split, instance of every prompt) and the latency estimates must be
equal exactly. Host code only: this runs without a GPU.
"""
import numpy as np
import pytest

from oracle import dispatch as Dp
from paper_2504_15930_amd import dispatch, sl


def _profile(rng):
    pts = sorted(set(int(x) for x in rng.integers(1, 300, int(rng.integers(1, 9)))))
    base = np.cumsum(rng.uniform(0.0, 0.5, len(pts))) + rng.uniform(0.1, 1.0)
    return pts, [float(x) for x in base]


@pytest.mark.parametrize("combine", ["sum", "max"])
def test_plan_matches_oracle(combine):
    rng = np.random.default_rng(7 if combine == "sum" else 8)
    for trial in range(300):
        n = int(rng.integers(1, 400))
        est = rng.integers(1, 9000, n)
        if trial % 5 == 0:
            est = rng.integers(1, 6, n)                       # many ties
        dist = rng.integers(1, 9000, int(rng.integers(1, 300)))
        N = int(rng.integers(1, 17))
        alpha = float(rng.choice([0.0, 0.05, 0.2, 0.5, 1.0, rng.uniform()]))
        pb, ps = _profile(rng)
        max_batch = int(rng.integers(1, 300))
        try:
            want = Dp.dispatch(est, alpha, dist, N, pb, ps, max_batch, combine)
        except ValueError:
            with pytest.raises(sl.SlError):
                dispatch.plan(est, alpha, dist, N, pb, ps, max_batch, combine)
            continue
        got = dispatch.plan(est, alpha, dist, N, pb, ps, max_batch, combine)
        assert got[:3] == want[:3], (trial, got[:3], want[:3])
        assert got[3].tolist() == want[3], trial


def test_generation_latency_matches_equation2():
    rng = np.random.default_rng(9)
    for _ in range(500):
        pb, ps = _profile(rng)
        m = int(rng.integers(0, 2000))
        mb = int(rng.integers(1, 400))
        l_avg = float(rng.integers(1, 9000))
        assert dispatch.generation_latency(l_avg, m, mb, pb, ps) == Dp.generation_latency(l_avg, m, mb, pb, ps)


def test_plan_rejects_bad_arguments():
    pb, ps = [1, 8], [1.0, 2.0]
    with pytest.raises(sl.SlError):
        dispatch.plan([1, 2, 3], 1.5, [5], 2, pb, ps, 4)            # alpha > 1
    with pytest.raises(sl.SlError):
        dispatch.plan([1, 2, 3], 0.3, [5], 0, pb, ps, 4)            # no instances
    with pytest.raises(sl.SlError):
        dispatch.plan([1, 2, 3], 0.3, [5], 2, [8, 1], ps, 4)        # profile not ascending
    with pytest.raises(sl.SlError):
        dispatch.plan([1, 2, 3], 0.5, [5], 1, pb, ps, 4)            # two groups, one instance
