"""Pins of the oracle's layer-shared selection (Eqs. 4-5 keep one index set
per layer; reading R22) to facts other than the oracle itself."""
import itertools

import numpy as np

from oracle import omnimem_oracle as om

from test_oracle_pins import _tiny_layers


def _scores(seed, h_kv=3, n=14):
    rng = np.random.default_rng(seed)
    mod = np.array([0] * 9 + [1] * 5, dtype=np.uint8)[:n]
    a = rng.exponential(1.0, (h_kv, n))
    s = rng.uniform(-0.2, 0.95, (h_kv, n))
    return a, s, mod


def test_one_kv_head_is_the_per_head_selection():
    a, s, mod = _scores(1, h_kv=1)
    np.testing.assert_array_equal(om.layer_shared_select(a, s, mod, 4, 2),
                                  om.select(om.retention_score(a, s), mod, 4, 2))


def test_identical_heads_reduce_to_the_per_head_selection():
    a, s, mod = _scores(2, h_kv=1)
    a3, s3 = np.repeat(a, 3, axis=0), np.repeat(s, 3, axis=0)
    np.testing.assert_array_equal(om.layer_shared_select(a3, s3, mod, 5, 3),
                                  om.select(om.retention_score(a3, s3), mod, 5, 3))


def test_head_order_does_not_matter_and_rows_are_shared():
    a, s, mod = _scores(3)
    idx = om.layer_shared_select(a, s, mod, 5, 2)
    perm = [2, 0, 1]
    np.testing.assert_array_equal(idx, om.layer_shared_select(a[perm], s[perm], mod, 5, 2))
    assert (idx == idx[0]).all()


def test_importance_sum_or_mean_rank_alike():
    # psi = a^lambda (1 - s): scaling a by H_kv scales psi by H_kv^lambda.
    a, s, mod = _scores(4)
    mean_a = np.repeat(a.mean(axis=0, keepdims=True), 3, axis=0)
    np.testing.assert_array_equal(om.layer_shared_select(a, s, mod, 4, 2),
                                  om.layer_shared_select(mean_a, s, mod, 4, 2))


def test_brute_force_best_shared_subset():
    # The kept rows of each modality maximise the summed layer psi over all
    # subsets of that size (ties to the earliest rows), with the layer psi
    # written out from its definition here.
    a, s, mod = _scores(5, n=10)
    mod = np.array([0] * 6 + [1] * 4, dtype=np.uint8)
    psi = (a.sum(axis=0) ** om.DEFAULT_LAMBDA) * (1.0 - s.mean(axis=0))
    idx = om.layer_shared_select(a, s, mod, 3, 2)[0]
    for mu, m, got in ((0, 3, idx[:3]), (1, 2, idx[3:])):
        pos = np.flatnonzero(mod == mu)
        best = max(itertools.combinations(pos.tolist(), m),
                   key=lambda c: (round(psi[list(c)].sum(), 12), [-x for x in c]))
        assert sorted(best) == got.tolist()


def test_step_with_shared_selection():
    layers = _tiny_layers()
    per_head = om.compression_step(layers, 60)
    shared = om.compression_step(layers, 60, shared_selection=True)
    assert shared["budgets"] == per_head["budgets"]      # the allocation does not change
    for layer, idx, ko in zip(layers, shared["idx"], shared["k_out"]):
        assert (idx == idx[0]).all()
        for g in range(idx.shape[0]):
            np.testing.assert_array_equal(ko[g], layer["k"][g, idx[g]])
