"""The CPU oracle against facts fixed outside it (library routines, closed forms, invariants)."""
import pytest

import oracle_pins


@pytest.mark.parametrize("pin", oracle_pins.ALL_PINS, ids=lambda f: f.__name__)
def test_oracle_pin(pin, oracle_lib):
    pin(oracle_lib)


def test_oracle_rejects_bad_arguments(oracle_lib):
    import numpy as np
    import oracle
    rng = np.random.default_rng(0)
    case, _ = oracle_pins.random_case(rng, 2, 4, 2, 64, 16, [5, 20])
    bad = dict(case)
    bad["block_table"] = case["block_table"].copy()
    bad["block_table"][1, 1] = case["k_pages"].shape[0]          # page id past the pool
    with pytest.raises(ValueError):
        oracle_pins.run(oracle_lib, bad)
    bad = dict(case)
    bad["seq_lens"] = np.array([5, 16 * case["block_table"].shape[1] + 1], dtype=np.int32)
    with pytest.raises(ValueError):
        oracle_pins.run(oracle_lib, bad)
    bad = dict(case)
    bad["seq_lens"] = np.array([-1, 20], dtype=np.int32)
    with pytest.raises(ValueError):
        oracle_pins.run(oracle_lib, bad)
    with pytest.raises(ValueError):
        oracle.decode_attn(case["q"][:, :3], case["k_pages"], case["v_pages"],
                           case["block_table"], case["seq_lens"], case["scale"], lib=oracle_lib)
