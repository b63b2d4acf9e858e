"""The parity metrics themselves (CPU): an error confined to one query head of
one sequence passes the whole-output L1 ratio but fails the per-row bound."""
import numpy as np
import pytest

from tests.gpu_util import MEAN_REL, assert_close, elementwise_rel, errors, row_l1_ratios


def test_row_bound_catches_an_error_confined_to_one_head():
    rng = np.random.default_rng(0)
    ref = rng.standard_normal((16, 32, 128)) * 0.007      # |O| at long context
    x = ref.copy()
    x[5, 17, 32:48] *= 1.05                               # 16 columns of one head, 5 % off
    ma, mr = errors(x, ref)
    assert ma < 1e-2 and mr < MEAN_REL                    # the global bounds would pass it
    rows = row_l1_ratios(x, ref)
    assert rows.shape == (16 * 32,) and rows.argmax() == 5 * 32 + 17 and rows.max() > MEAN_REL
    with pytest.raises(AssertionError):
        assert_close(x, ref, "planted one-head error")
    assert_close(ref + 1e-9, ref, "unperturbed")


def test_row_ratios_skip_empty_rows_and_elementwise_floor():
    ref = np.zeros((2, 4))
    ref[1] = [1.0, -2.0, 0.0, 4.0]
    x = ref + np.array([[0.0] * 4, [0.1, 0.0, 2e-6, 0.0]])
    r = row_l1_ratios(x, ref)
    assert r.shape == (1,) and abs(r[0] - (0.1 + 2e-6) / 7.0) < 1e-15
    mean, mx = elementwise_rel(x, ref)
    assert abs(mx - 2.0) < 1e-12                           # 2e-6 over the 1e-6 floor
    assert abs(mean - (0.1 + 2.0) / 8) < 1e-12
