"""Pins of the oracle's offline budgets (end of Sec. 3.2: layer budgets fixed
ahead of time from a few calibration chunks) to facts other than the
oracle itself: averaging, softmax invariances, closed forms and the
relation to the online step."""
import math

import numpy as np
import pytest
import scipy.special

from oracle import omnimem_oracle as om

from test_oracle_pins import _tiny_layers


def test_two_steps_equal_one_step_of_their_mean():
    c1 = np.array([0.31, 0.52, 0.44, 0.12])
    c2 = np.array([0.29, 0.18, 0.61, 0.40])
    two = om.calibration_budgets([c1, c2], 4 * 4096)
    one = om.calibration_budgets([(c1 + c2) / 2], 4 * 4096)
    assert two.tolist() == one.tolist()
    # a sum instead of a mean changes C/T and with it the budgets
    assert om.calibration_budgets([c1 + c2], 4 * 4096).tolist() != two.tolist()


def test_shift_of_every_layer_leaves_budgets():
    c = np.array([[0.2, 0.5, 0.45, 0.9, 0.1], [0.3, 0.4, 0.5, 0.7, 0.2]])
    assert om.calibration_budgets(c, 20480).tolist() == om.calibration_budgets(c + 2.5, 20480).tolist()


def test_equal_compressibility_splits_evenly_remainder_to_lower_layers():
    b = om.calibration_budgets([[0.4] * 5, [0.4] * 5], 5 * 4096 + 3)
    assert b.tolist() == [4097, 4097, 4097, 4096, 4096]


def test_two_layers_unclamped_closed_form():
    # Two layers whose shares stay inside [B_min, B_max]: x_0 = B sigma((c0 - c1) / T).
    c0, c1, t, total = 0.50, 0.46, 0.2, 10000
    x0 = total * scipy.special.expit((c0 - c1) / t)
    assert 0.5 * total / 2 < x0 < 2.0 * total / 2
    b = om.calibration_budgets([[c0, c1]], total, temperature=t)
    assert b.sum() == total
    assert abs(b[0] - x0) < 1.0
    assert b[0] in (math.floor(x0), math.ceil(x0))


def test_large_temperature_tends_to_uniform():
    rng = np.random.default_rng(3)
    c = rng.uniform(0, 1, (4, 7))
    b = om.calibration_budgets(c, 7 * 1000, temperature=1e9)
    assert b.tolist() == [1000] * 7


def test_budgets_sum_and_bounds():
    rng = np.random.default_rng(4)
    for _ in range(20):
        L = int(rng.integers(2, 12))
        total = int(rng.integers(L * 10, L * 5000))
        c = rng.uniform(0, 1, (int(rng.integers(1, 6)), L))
        b = om.calibration_budgets(c, total, temperature=float(rng.uniform(0.05, 1.0)))
        lo = math.ceil(0.5 * total / L)
        hi = math.floor(2.0 * total / L)
        assert b.sum() == total
        assert ((b >= lo) & (b <= hi)).all()


def test_no_token_count_caps_calibrated_budgets():
    # Online, a layer with fewer tokens than its share keeps only its tokens;
    # the calibrated budget of the same values is not capped.
    c = np.array([0.9, 0.1, 0.1])
    n = [500, 6144, 6144]
    online = om.integer_budgets(om.layer_shares(c, n, 3000), n, 3000)
    offline = om.calibration_budgets([c], 3000)
    assert online[0] == 500
    assert offline[0] > 500
    assert offline.sum() == 3000


def test_fixed_split_cases():
    assert om.fixed_split(9999, 0.7, 40, 10) == (40, 10)     # more budget than rows: keep all
    assert om.fixed_split(-3, 0.7, 40, 10) == (0, 0)
    assert om.fixed_split(20, 0.75, 40, 10) == om.split_budget(20, 0.75, 40, 10) == (15, 5)
    assert om.fixed_split(45, 0.95, 40, 10) == (40, 5)       # visual capped at its rows


def test_step_with_its_own_budgets_matches_the_online_step():
    layers = _tiny_layers()
    online = om.compression_step(layers, 60)
    fixed = om.compression_step(layers, 60, layer_budgets=online["layer_budgets"])
    assert fixed["budgets"] == online["budgets"]
    for a, b in zip(online["idx"], fixed["idx"]):
        np.testing.assert_array_equal(a, b)


def test_step_keeps_everything_under_large_fixed_budgets():
    layers = _tiny_layers()
    out = om.compression_step(layers, 60, layer_budgets=[10**6] * len(layers))
    for layer, (mv, ma) in zip(layers, out["budgets"]):
        mod = layer["modality"]
        assert (mv, ma) == (int((mod == 0).sum()), int((mod == 1).sum()))


def test_calibration_needs_a_step():
    with pytest.raises(ValueError):
        om.calibration_budgets(np.zeros((0, 3)), 100)
