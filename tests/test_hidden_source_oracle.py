"""Pins of the oracle's hidden-state redundancy (Eq. 7 as printed, on hidden
states; reading R23) to facts other than the oracle itself."""
import json
import os

import numpy as np
import pytest

from oracle import omnimem_oracle as om

from test_oracle_pins import GOLDEN, _tiny_layers


def test_golden_three_tokens_on_hidden_states():
    # The same worked example as the value-vector pin, given as hidden states.
    with open(os.path.join(GOLDEN, "adjacent_cosine_3tok.json")) as f:
        g = json.load(f)
    h = np.array(g["vectors"], dtype=np.float64)
    s = om.hidden_redundancy(h, np.zeros(len(h), dtype=np.uint8), 2, "adj")
    np.testing.assert_allclose(s, np.repeat(np.array(g["s_adj"])[None], 2, axis=0), rtol=0, atol=1e-12)


def test_one_head_of_values_as_hidden_states():
    rng = np.random.default_rng(7)
    v = rng.standard_normal((1, 20, 12))
    mod = np.array([0, 1] * 10, dtype=np.uint8)
    for mode in ("adj", "max"):
        np.testing.assert_allclose(om.hidden_redundancy(v[0], mod, 3, mode),
                                   np.repeat(om.redundancy(v, mod, mode), 3, axis=0), rtol=1e-13)


def test_row_scaling_leaves_cosines():
    rng = np.random.default_rng(8)
    h = rng.standard_normal((15, 40))
    mod = np.array([0] * 10 + [1] * 5, dtype=np.uint8)
    scaled = h * rng.uniform(0.1, 10.0, (15, 1))
    np.testing.assert_allclose(om.hidden_redundancy(h, mod, 2), om.hidden_redundancy(scaled, mod, 2),
                               rtol=1e-12, atol=1e-14)


def test_orthogonal_neighbours_give_zero():
    # Standard basis vectors: every adjacent cosine is 0.
    h = np.eye(6)
    s = om.hidden_redundancy(h, np.zeros(6, dtype=np.uint8), 1)
    np.testing.assert_array_equal(s, np.zeros((1, 6)))


def test_step_carries_the_kept_hidden_states():
    layers = _tiny_layers()
    rng = np.random.default_rng(9)
    for lay in layers:
        lay["h"] = rng.standard_normal((len(lay["modality"]), 24))
    out = om.compression_step(layers, 60, mode="adj", shared_selection=True, use_hidden=True)
    for lay, idx, h_out, s in zip(layers, out["idx"], out["h_out"], out["s"]):
        np.testing.assert_array_equal(h_out, lay["h"][idx[0]])
        assert (s == s[0]).all()              # one redundancy per token
    with pytest.raises(ValueError):
        om.compression_step(layers, 60, mode="adj", use_hidden=True)
