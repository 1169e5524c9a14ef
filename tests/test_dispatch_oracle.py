"""Pins for the skewness-aware dispatching oracle (oracle/dispatch.py), CPU only.

Fixed independently of the code: numpy's lower-rank percentile and linear
interpolation (library routines), a hand-worked four-instance example, the
paper's two-instance illustration (two long-tail samples of twice the regular
length get a dedicated instance), and the closed form for a flat PTL curve.
"""
import numpy as np
import pytest

from oracle import dispatch as Dp


def pin_percentile_matches_numpy(D):
    rng = np.random.default_rng(1)
    for n in (1, 2, 5, 10, 101, 1000):
        v = rng.integers(1, 10000, n)
        for q in (0.5, 0.9):
            assert D.percentile_lower(v, q) == int(np.percentile(v, 100 * q, method="lower")), (n, q)


def pin_ptl_interpolation(D):
    xb, ys = [1, 4, 16, 64], [1.0, 1.3, 2.0, 5.0]
    for b in range(1, 65):
        assert abs(D.ptl(b, xb, ys) - float(np.interp(b, xb, ys))) <= 1e-12 * 5.0, b
    assert D.ptl(0, xb, ys) == 1.0
    assert abs(D.ptl(112, xb, ys) - (5.0 + 3.0 * 48 / 48)) < 1e-12    # continues the last segment


def pin_hand_worked(D):
    """10 prompts, N = 4, alpha = 0.2, D = 10..100 (P90 = 90, P50 = 50), PTL points
    (1, 1.0), (2, 1.2), (4, 2.0), max batch 2. Long-tail = prompts 1 and 3.
      N_l = 1: long M = 2 -> 1.2 * 90 * 1 = 108; regular M = ceil(8/3) = 3 -> BS 2, 2 rounds
               -> 1.2 * 50 * 2 = 120; sum 228, max 120
      N_l = 2: long M = 1 -> 1.0 * 90 = 90; regular M = 4 -> 2 rounds -> 120; sum 210, max 120
      N_l = 3: long 90; regular M = 8 -> 4 rounds -> 240; sum 330, max 240
    Sum picks N_l = 2; max ties at N_l = 1 and 2 and keeps the first."""
    est = [5, 100, 7, 90, 3, 8, 2, 60, 1, 4]
    dist = list(range(10, 101, 10))
    tb, ts = [1, 2, 4], [1.0, 1.2, 2.0]
    n_l, n_r, lat, inst = D.dispatch(est, 0.2, dist, 4, tb, ts, 2, "sum")
    assert (n_l, n_r) == (2, 2) and abs(lat - 210.0) < 1e-9
    # regular order 7, 5, 2, 0, 9, 4, 6, 8 dealt to instances 2, 3, 2, 3, ...
    assert inst == [3, 0, 2, 1, 3, 3, 2, 2, 3, 2]
    n_l, n_r, lat, inst = D.dispatch(est, 0.2, dist, 4, tb, ts, 2, "max")
    assert (n_l, n_r) == (1, 3) and abs(lat - 120.0) < 1e-9
    assert inst[1] == 0 and inst[3] == 0


def pin_paper_two_instances(D):
    """Two instances; two long-tail prompts twice as long as the 64 regular ones: the two
    long-tail prompts share one instance, the 64 regular ones the other."""
    L = 1000
    est = [L] * 32 + [2 * L] + [L] * 32 + [2 * L]
    dist = [L] * 8 + [2 * L] * 2
    n_l, n_r, lat, inst = D.dispatch(est, 0.031, dist, 2, [1, 64], [1.0, 2.0], 64)
    assert (n_l, n_r) == (1, 1)
    assert inst[32] == 0 and inst[65] == 0 and all(inst[i] == 1 for i in range(66) if i not in (32, 65))
    assert abs(lat - (D.ptl(2, [1, 64], [1.0, 2.0]) * 2 * L + D.ptl(64, [1, 64], [1.0, 2.0]) * L)) < 1e-9


def pin_flat_ptl_closed_form(D):
    """With a flat PTL and one round everywhere, every split costs c * (P90 + P50): the first is kept."""
    rng = np.random.default_rng(2)
    est = rng.integers(1, 5000, 200)
    dist = rng.integers(1, 5000, 300)
    n_l, n_r, lat, inst = D.dispatch(est, 0.2, dist, 8, [1, 1000], [0.5, 0.5], 1000)
    assert (n_l, n_r) == (1, 7)
    want = 0.5 * (np.percentile(dist, 90, method="lower") + np.percentile(dist, 50, method="lower"))
    assert abs(lat - want) < 1e-9
    # long-tail = the 40 largest estimates (ties by index), all on instance 0
    order = sorted(range(200), key=lambda i: (-int(est[i]), i))
    assert sorted(i for i in range(200) if inst[i] == 0) == sorted(order[:40])


def pin_groups_balanced(D):
    rng = np.random.default_rng(3)
    est = rng.integers(1, 9000, 777)
    dist = rng.integers(1, 9000, 500)
    tb = [1, 2, 4, 8, 16, 32, 64, 128, 256]
    ts = [1.0, 1.01, 1.03, 1.07, 1.15, 1.3, 1.7, 2.6, 4.5]
    for combine in ("sum", "max"):
        n_l, n_r, lat, inst = D.dispatch(est, 0.2, dist, 8, tb, ts, 128, combine)
        assert n_l + n_r == 8 and n_l >= 1 and n_r >= 1
        counts = np.bincount(inst, minlength=8)
        assert counts[:n_l].max() - counts[:n_l].min() <= 1 and counts[n_l:].max() - counts[n_l:].min() <= 1
        assert counts[:n_l].sum() == int(np.floor(0.2 * 777))
        # the chosen split is the cheapest one, the per-instance sizes being ceil(group / instances)
        costs = []
        for k in range(1, 8):
            m_l, m_r = -(-155 // k), -(-622 // (8 - k))
            a = D.generation_latency(int(np.percentile(dist, 90, method="lower")), m_l, 128, tb, ts)
            b = D.generation_latency(int(np.percentile(dist, 50, method="lower")), m_r, 128, tb, ts)
            costs.append(a + b if combine == "sum" else max(a, b))
        assert abs(lat - min(costs)) <= 1e-9 * min(costs) and n_l == 1 + int(np.argmin(costs))


ALL_PINS = [pin_percentile_matches_numpy, pin_ptl_interpolation, pin_hand_worked, pin_paper_two_instances,
            pin_flat_ptl_closed_form, pin_groups_balanced]


@pytest.mark.parametrize("pin", ALL_PINS, ids=lambda f: f.__name__)
def test_pin(pin):
    pin(Dp)
