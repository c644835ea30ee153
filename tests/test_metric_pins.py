"""Pins of the parity metric: max|x - ref| / max|ref| per output tensor, the reading taken of the
relative error that section 3.2 quotes without a definition.  Every expected value below is worked
out by hand from that definition; each case targets one way the metric could be wrong."""
import numpy as np
import pytest

import oracle


def test_one_sided_negative_error():
    ref = np.array([1.0, 2.0, -4.0])
    x = ref - np.array([0.0, 0.5, 0.0])       # the result falls short: x - ref = -0.5
    assert oracle.max_rel_err(x, ref) == 0.125     # 0.5 / 4


def test_errors_above_and_below_count_alike():
    ref = np.array([3.0, -1.0, 0.5])
    up, down = ref + np.array([0.0, 0.3, 0.0]), ref - np.array([0.0, 0.3, 0.0])
    assert oracle.max_rel_err(up, ref) == pytest.approx(0.1)
    assert oracle.max_rel_err(down, ref) == pytest.approx(0.1)


def test_largest_magnitude_of_the_reference_is_the_scale():
    ref = np.array([-8.0, 1.0])                # the scale comes from the negative entry
    x = np.array([-8.0, 1.8])
    assert oracle.max_rel_err(x, ref) == pytest.approx(0.1)


def test_scale_is_the_reference_not_the_result():
    ref = np.array([1.0, 1.0])
    x = np.array([1.0, 3.0])
    assert oracle.max_rel_err(x, ref) == 2.0   # 2 / max|ref| = 2, not 2 / max|x| = 2/3


def test_zeros_in_the_reference():
    ref = np.array([0.0, 0.0, 2.0])
    x = np.array([0.1, 0.0, 2.0])
    assert oracle.max_rel_err(x, ref) == pytest.approx(0.05)


def test_all_zero_reference_gives_the_absolute_error():
    ref = np.zeros(4)
    x = np.array([0.0, 0.3, -0.5, 0.0])
    assert oracle.max_rel_err(x, ref) == 0.5
    assert oracle.max_rel_err(ref, ref) == 0.0


def test_exact_and_empty():
    ref = np.array([[1.0, -2.0], [3.0, 0.25]])
    assert oracle.max_rel_err(ref.copy(), ref) == 0.0
    assert oracle.max_rel_err(np.zeros((0, 3)), np.zeros((0, 3))) == 0.0


def test_shapes_must_match():
    with pytest.raises(ValueError):
        oracle.max_rel_err(np.zeros(3), np.zeros(1))       # would broadcast silently
    with pytest.raises(ValueError):
        oracle.max_rel_err(np.zeros((2, 3)), np.zeros((3, 2)))
    with pytest.raises(ValueError):
        oracle.max_rel_err_slices(np.zeros((2, 3)), np.zeros((2, 4)), [0, 1])


def test_per_slice_metric_sees_a_local_error():
    """Slice 0 is off by 10 % of its own scale; against the whole tensor's scale (set by slice 1)
    that is 0.1 %, which a global bar would pass."""
    ref = np.array([[1.0, 1.0], [100.0, 100.0]])
    x = np.array([[1.0, 1.1], [100.0, 100.0]])
    assert oracle.max_rel_err(x, ref) == pytest.approx(0.001)
    assert oracle.max_rel_err_slices(x, ref, [0, 1]) == pytest.approx(0.1)
    assert oracle.max_rel_err_slices(x, ref, [1]) == 0.0
    # index tuples address (sequence, head) slices of [B, T, H, d] tensors
    o_ref = np.ones((2, 3, 4, 2))
    o = o_ref.copy()
    o[1, :, 2, :] += 0.25
    assert oracle.max_rel_err_slices(o, o_ref, [(b, slice(None), h) for b in range(2) for h in range(4)]) == 0.25


def test_p99_of_elementwise_errors():
    ref = np.ones(1000)
    x = ref.copy()
    x[:20] += 0.5                                            # 2 % of the elements off by 0.5
    assert oracle.p99_rel_err(x, ref) == pytest.approx(0.5 / (1.0 + 1e-3))
    assert oracle.p99_rel_err(ref, ref) == 0.0
