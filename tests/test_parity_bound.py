"""The GPU tests' tolerance check itself (CPU only): it must reject errors the
stated bound forbids, including ones the relative term alone would let pass."""
import numpy as np
import pytest

from parity import assert_parity


def _ref():
    rng = np.random.default_rng(5)
    return rng.normal(0.0, 1.5, (3, 4, 64))


def test_accepts_bf16_rounding():
    ref = _ref()
    # round to bf16 (nearest even) through float32 bit manipulation
    f = ref.astype(np.float32).view(np.uint32)
    r = ((f + 0x7FFF + ((f >> 16) & 1)) & 0xFFFF0000).astype(np.uint32).view(np.float32)
    assert_parity(r.astype(np.float64), ref, "bf16 rounding only")


def test_rejects_small_output_error_the_relative_term_allows():
    ref = _ref()
    g = ref.copy()
    i = np.unravel_index(np.argmin(np.abs(np.abs(ref) - 1.0)), ref.shape)
    g[i] += 0.012   # within 1e-2 + 2e-2 * |ref| at |ref| ~ 1, beyond the bare 1e-2
    with pytest.raises(AssertionError, match="where"):
        assert_parity(g, ref, "planted 0.012 at |ref| ~ 1")


def test_large_outputs_keep_the_relative_allowance():
    ref = np.sign(_ref()) * (np.abs(_ref()) + 5.0)   # every |ref| >= 5
    g = ref * (1 + 2.0 ** -8)   # one bf16 ulp relative, > 1e-2 absolute
    assert_parity(g, ref, "relative error at |ref| >= 4")


def test_rejects_nonfinite_and_row_error():
    ref = _ref()
    g = ref.copy()
    g[0, 0, 0] = np.nan
    with pytest.raises(AssertionError, match="non-finite"):
        assert_parity(g, ref)
    g = ref * 1.03
    with pytest.raises(AssertionError):
        assert_parity(g, ref)


def test_value_scale_widens_the_absolute_bound():
    ref = _ref()
    g = ref.copy()
    i = np.unravel_index(np.argmin(np.abs(np.abs(ref) - 1.0)), ref.shape)
    g[i] += 0.03
    with pytest.raises(AssertionError):
        assert_parity(g, ref, "unit scale")
    assert_parity(g, ref, "values at scale 5", value_scale=np.full(ref.shape[:-1] + (1,), 5.0))


def test_value_rms_rows_hand_worked():
    from parity import value_rms_rows
    # one KV head, pages of 2 tokens, D = 2; sequence 0 has 3 tokens on pages 1, 0
    v = np.zeros((3, 1, 2, 2))
    v[1, 0] = [[3.0, 4.0], [0.0, 0.0]]
    v[0, 0] = [[1.0, 1.0], [np.nan, np.nan]]   # slot past the end: never read
    got = value_rms_rows(v, np.array([[1, 0], [2, 2]]), np.array([3, 0]), num_q_heads=2)
    assert got.shape == (2, 2, 1)
    assert np.allclose(got[0, :, 0], np.sqrt((9 + 16 + 0 + 0 + 1 + 1) / 6))
    assert np.all(got[1] == 1.0)
