"""Planted mistakes in the dispatching oracle (oracle/dispatch.py) must trip a pin."""
import importlib.util
import os
import sys

import pytest

import test_dispatch_oracle as pins
from oracle import dispatch as Dp

MUTANTS = [
    ("sort_ascending", "key=lambda i: (-int(est_len[i]), i)", "key=lambda i: (int(est_len[i]), i)"),
    ("percentiles_swapped", "l_alpha = percentile_lower(dist, 0.9)", "l_alpha = percentile_lower(dist, 0.5)"),
    ("percentile_upper_rank", "v[int(math.floor(q * (len(v) - 1)))]", "v[int(math.ceil(q * (len(v) - 1)))]"),
    ("rounds_floor", "rounds = -(-m // bs)", "rounds = m // bs"),
    ("batch_ignores_limit", "bs = min(m, max_batch)", "bs = m"),
    ("m_floor_division", "-(-len(long_tail) // n_l) if n_l else 0", "len(long_tail) // n_l if n_l else 0"),
    ("interp_step_function", "return y0 + (y1 - y0) * (batch - x0) / (x1 - x0)", "return y0"),
    ("combine_ignored", "total = lat_l + lat_r if combine == \"sum\" else max(lat_l, lat_r)", "total = lat_l + lat_r"),
    ("last_minimum_kept", "if best is None or total < best[2]:", "if best is None or total <= best[2]:"),
    ("long_tail_ceil", "n_long = int(math.floor(alpha * n))", "n_long = int(math.ceil(alpha * n))"),
    ("regular_not_offset", "instance[i] = n_l + k % n_r", "instance[i] = k % n_r"),
]


def _load_mutant(tmp_path, name, old, new):
    src = open(Dp.__file__).read()
    assert old in src, f"mutation target not found: {old!r}"
    path = os.path.join(tmp_path, f"dispatch_{name}.py")
    with open(path, "w") as f:
        f.write(src.replace(old, new, 1))
    spec = importlib.util.spec_from_file_location(f"dispatch_{name}", path)
    mod = importlib.util.module_from_spec(spec)
    sys.modules[spec.name] = mod
    try:
        spec.loader.exec_module(mod)
    finally:
        sys.modules.pop(spec.name, None)
    return mod


@pytest.mark.parametrize("name,old,new", MUTANTS, ids=[m[0] for m in MUTANTS])
def test_mutant_is_caught(tmp_path, name, old, new):
    mod = _load_mutant(str(tmp_path), name, old, new)
    failed = []
    for pin in pins.ALL_PINS:
        try:
            pin(mod)
        except (AssertionError, IndexError, ValueError, ZeroDivisionError):
            failed.append(pin.__name__)
    assert failed, f"mutant {name} survived every pin"
