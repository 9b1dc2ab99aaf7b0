"""Pins of the CPU oracle to facts other than itself.

Closed forms, invariants, special cases that reduce to library routines,
values printed in the paper (tests/golden/) and brute force on tiny inputs.
Each group names the passage of the paper it pins.
"""
import itertools
import json
import math
import os

import numpy as np
import pytest
import scipy.optimize
import scipy.special
import scipy.stats

from oracle import omnimem_oracle as om

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _rand_layer(seed, h_q=4, h_kv=2, d=8, n_cache=7, n_chunk=5, scale=1.0):
    rng = np.random.default_rng(seed)
    q = rng.standard_normal((h_q, n_chunk, d))
    k = rng.standard_normal((h_kv, n_cache + n_chunk, d))
    return q, k, scale / math.sqrt(d)


# --------------------------------------------------------------------------
# Eq. (6): accumulated attention importance
# --------------------------------------------------------------------------

@pytest.mark.parametrize("causal", [True, False])
def test_importance_total_is_queries_times_group(causal):
    # Every softmax row sums to one, so a KV head's total is G * C.
    q, k, sc = _rand_layer(1)
    a = om.attention_importance(q, k, 7, sc, causal)
    g = q.shape[0] // k.shape[0]
    np.testing.assert_allclose(a.sum(axis=1), g * q.shape[1], rtol=1e-12)


def test_importance_zero_query_noncausal_is_uniform():
    q, k, sc = _rand_layer(2)
    q[:] = 0.0
    a = om.attention_importance(q, k, 7, sc, causal=False)
    n = k.shape[1]
    np.testing.assert_allclose(a, 2 * 5 / n, rtol=1e-12)
    assert om.normalized_entropy(a[0]) == pytest.approx(1.0, abs=1e-12)


def test_importance_zero_query_causal_harmonic_closed_form():
    # With equal scores, query i spreads 1/(n_cache + i + 1) over its rows.
    n_cache, n_chunk, g = 7, 5, 2
    q, k, sc = _rand_layer(3, n_cache=n_cache, n_chunk=n_chunk)
    q[:] = 0.0
    a = om.attention_importance(q, k, n_cache, sc, causal=True)
    want = np.empty(n_cache + n_chunk)
    want[:n_cache] = g * sum(1.0 / (n_cache + i + 1) for i in range(n_chunk))
    for t in range(n_chunk):
        want[n_cache + t] = g * sum(1.0 / (n_cache + i + 1) for i in range(t, n_chunk))
    np.testing.assert_allclose(a[0], want, rtol=1e-12)
    np.testing.assert_allclose(a[1], want, rtol=1e-12)


def test_lse_zero_query_is_log_visible_count():
    n_cache, n_chunk = 7, 5
    q, k, sc = _rand_layer(4, n_cache=n_cache, n_chunk=n_chunk)
    q[:] = 0.0
    lse = om.attention_lse(q, k, n_cache, sc, causal=True)
    want = np.log(n_cache + np.arange(n_chunk) + 1.0)
    np.testing.assert_allclose(lse, np.broadcast_to(want, lse.shape), rtol=1e-12)


def test_importance_invariant_to_per_query_score_shift():
    # Appending a coordinate with k = 1 adds a per-(head, query) constant to
    # every score of that query; a softmax over keys must not change.  A
    # normalisation over the wrong axis fails this.
    q, k, sc = _rand_layer(5)
    rng = np.random.default_rng(55)
    shift = rng.standard_normal(q.shape[:2] + (1,)) * 3.0
    q2 = np.concatenate([q, shift], axis=2)
    k2 = np.concatenate([k, np.ones(k.shape[:2] + (1,))], axis=2)
    a1 = om.attention_importance(q, k, 7, sc)
    a2 = om.attention_importance(q2, k2, 7, sc)
    np.testing.assert_allclose(a1, a2, rtol=1e-10)


def test_importance_sharp_limit_counts_argmax():
    # As the scale grows the softmax becomes one-hot on the argmax, so a_k
    # counts the (query head of group g, query) pairs whose best visible key
    # is k.  Pins the visibility rule and the query-head -> KV-head grouping.
    h_q, h_kv, n_cache, n_chunk, d = 6, 2, 9, 6, 5
    rng = np.random.default_rng(6)
    q = rng.integers(-3, 4, size=(h_q, n_chunk, d)).astype(float)
    k = rng.integers(-3, 4, size=(h_kv, n_cache + n_chunk, d)).astype(float)
    k += rng.standard_normal(k.shape) * 0.01  # break exact ties
    counts = np.zeros((h_kv, n_cache + n_chunk))
    group = h_q // h_kv
    for h in range(h_q):
        for i in range(n_chunk):
            best, best_j, second = -np.inf, -1, -np.inf
            for j in range(n_cache + n_chunk):
                if j >= n_cache and j - n_cache > i:
                    continue
                val = sum(q[h, i, x] * k[h // group, j, x] for x in range(d))
                if val > best:
                    best, best_j, second = val, j, best
                elif val > second:
                    second = val
            assert best - second > 1e-3
            counts[h // group, best_j] += 1
    a = om.attention_importance(q, k, n_cache, 1e6, causal=True)
    np.testing.assert_allclose(a, counts, atol=1e-9)


def test_importance_subsets_match_full():
    q, k, sc = _rand_layer(7)
    full = om.attention_importance(q, k, 7, sc)
    keys = [0, 3, 8, 11]
    np.testing.assert_allclose(om.attention_importance(q, k, 7, sc, keys=keys), full[:, keys],
                               rtol=1e-12)
    lse = om.attention_lse(q, k, 7, sc)
    np.testing.assert_allclose(om.attention_lse(q, k, 7, sc, queries=[1, 4]), lse[:, [1, 4]],
                               rtol=1e-12)


# --------------------------------------------------------------------------
# Eq. (7): cosine redundancy
# --------------------------------------------------------------------------

def test_golden_three_token_cosines():
    with open(os.path.join(GOLDEN, "adjacent_cosine_3tok.json")) as f:
        gold = json.load(f)
    u = np.array(gold["vectors"])[None]
    mod = np.zeros(3, dtype=np.uint8)
    np.testing.assert_allclose(om.redundancy(u, mod, "adj")[0], gold["s_adj"], atol=1e-12)
    np.testing.assert_allclose(om.redundancy(u, mod, "max")[0], gold["s_max"], atol=1e-12)


def test_cosine_from_angles_closed_form():
    # Planar vectors at angles theta with random lengths: cos = cos(dtheta).
    rng = np.random.default_rng(8)
    n = 9
    theta = rng.uniform(0, 2 * math.pi, size=n)
    length = rng.uniform(0.1, 5.0, size=n)
    u = np.zeros((1, n, 4))
    u[0, :, 0] = length * np.cos(theta)
    u[0, :, 1] = length * np.sin(theta)
    mod = np.array([0, 1, 0, 0, 1, 1, 0, 1, 0], dtype=np.uint8)
    s_max = om.redundancy(u, mod, "max")[0]
    s_adj = om.redundancy(u, mod, "adj")[0]
    for mu in (0, 1):
        pos = [p for p in range(n) if mod[p] == mu]
        for t, p in enumerate(pos):
            others = [math.cos(theta[p] - theta[o]) for o in pos if o != p]
            assert s_max[p] == pytest.approx(max(others), abs=1e-12)
            nbrs = [pos[x] for x in (t - 1, t + 1) if 0 <= x < len(pos)]
            want = sum(math.cos(theta[p] - theta[o]) for o in nbrs) / len(nbrs)
            assert s_adj[p] == pytest.approx(want, abs=1e-12)


def test_cosine_special_cases():
    d = 6
    u = np.zeros((1, 6, d))
    u[0, 0, 0] = 1.0          # one-hot rows: orthogonal
    u[0, 1, 1] = 2.0
    u[0, 2, 2] = 3.0
    u[0, 3] = [1, 2, 3, 4, 5, 6]
    u[0, 4] = -u[0, 3] * 0.5  # antipodal to row 3
    u[0, 5] = 0.0             # zero vector
    mod = np.array([0, 0, 0, 1, 1, 1], dtype=np.uint8)
    s = om.redundancy(u, mod, "max")[0]
    np.testing.assert_allclose(s[:3], 0.0, atol=1e-15)
    assert s[3] == pytest.approx(0.0)  # max(cos to antipode = -1, cos to zero vector = 0)
    assert s[5] == pytest.approx(0.0)
    only_pair = om.redundancy(u[:, 3:5], np.array([1, 1], dtype=np.uint8), "max")[0]
    np.testing.assert_allclose(only_pair, -1.0, atol=1e-15)


def test_exact_duplicate_gives_one_and_scale_invariance():
    rng = np.random.default_rng(9)
    u = rng.standard_normal((2, 10, 16))
    u[:, 7] = u[:, 2] * 3.5
    mod = np.zeros(10, dtype=np.uint8)
    s = om.redundancy(u, mod, "max")
    np.testing.assert_allclose(s[:, [2, 7]], 1.0, atol=1e-12)
    scaled = u * rng.uniform(0.1, 10.0, size=(2, 10, 1))
    np.testing.assert_allclose(om.redundancy(scaled, mod, "max"), s, atol=1e-12)
    np.testing.assert_allclose(om.redundancy(scaled, mod, "adj"), om.redundancy(u, mod, "adj"),
                               atol=1e-12)


def test_redundancy_ignores_other_modality_and_lone_token():
    rng = np.random.default_rng(10)
    u = rng.standard_normal((1, 5, 8))
    u[0, 4] = u[0, 1]  # audio row duplicates a visual row
    mod = np.array([0, 0, 0, 0, 1], dtype=np.uint8)
    s = om.redundancy(u, mod, "max")[0]
    assert s[1] < 0.99
    assert s[4] == 0.0  # the only audio token
    rows = om.redundancy(u, mod, "max", rows=[4, 1])[0]
    np.testing.assert_allclose(rows, [s[4], s[1]])


# --------------------------------------------------------------------------
# Eq. (8): retention score
# --------------------------------------------------------------------------

def test_retention_special_cases():
    a = np.array([0.0, 0.5, 2.0, 7.0])
    s = np.array([0.3, 1.0, -1.0, 0.0])
    np.testing.assert_allclose(om.retention_score(a, s, 0.0), 1.0 - s)  # cosine-only ablation
    psi = om.retention_score(a, s, 0.02)
    assert psi[0] == 0.0 and psi[1] == 0.0
    assert psi[2] == pytest.approx(2.0 * 2.0 ** 0.02)
    assert (psi >= 0).all()
    np.testing.assert_allclose(om.retention_score(a, np.zeros(4), 1.0), a)


# --------------------------------------------------------------------------
# Eqs. (9), (10), (13): normalised entropy and compressibility
# --------------------------------------------------------------------------

def test_normalized_entropy_closed_forms_and_library():
    assert om.normalized_entropy(np.full(17, 3.0)) == pytest.approx(1.0, abs=1e-14)
    assert om.normalized_entropy(np.eye(1, 9, 4)[0]) == 0.0
    p = 0.2
    binary = -(p * math.log(p) + (1 - p) * math.log(1 - p))
    assert om.normalized_entropy([p, 1 - p, 0, 0]) == pytest.approx(binary / math.log(4))
    rng = np.random.default_rng(11)
    x = rng.exponential(size=50)
    assert om.normalized_entropy(x) == pytest.approx(scipy.stats.entropy(x) / math.log(50))
    assert om.normalized_entropy([5.0]) == 0.0


def test_avba_statistics_closed_forms():
    # Uniform importance inside each modality -> both normalised entropies 1;
    # identical values -> mean cosine 1 -> compressibility 0.
    mod = np.array([0, 0, 0, 1, 1, 0, 1], dtype=np.uint8)
    a = np.where(mod == 0, 2.0, 5.0)[None].repeat(3, axis=0)
    s = np.ones((3, 7))
    st = om.avba_statistics(a, s, mod)
    assert st["H_v"] == pytest.approx(1.0) and st["H_a"] == pytest.approx(1.0)
    assert st["C_v"] == 0.0 and st["C_a"] == 0.0 and st["C_l"] == 0.0
    s = np.zeros((3, 7))
    s[:, mod == 1] = 0.5
    st = om.avba_statistics(a, s, mod)
    assert st["C_v"] == pytest.approx(1.0)
    assert st["C_a"] == pytest.approx(0.5)
    assert st["sbar_l"] == pytest.approx(0.5 * 3 / 7)
    p = np.where(mod == 0, 2.0, 5.0)
    assert st["H_l"] == pytest.approx(scipy.stats.entropy(p) / math.log(7))


def test_avba_statistics_per_head_entropy_is_averaged():
    mod = np.zeros(4, dtype=np.uint8)
    a = np.array([[1.0, 1.0, 1.0, 1.0], [1.0, 0.0, 0.0, 0.0]])
    st = om.avba_statistics(a, np.zeros((2, 4)), mod)
    assert st["H_v"] == pytest.approx(0.5)
    assert st["H_a"] == 0.0 and st["C_a"] == 0.0


# --------------------------------------------------------------------------
# Eqs. (11), (12): modality split
# --------------------------------------------------------------------------

def test_modality_weights_closed_forms():
    assert om.modality_weights(0.7, 0.7, 5.0) == pytest.approx((5 / 6, 1 / 6))
    wv, wa = om.modality_weights(0.3, 0.9, 5.0)
    assert wv + wa == pytest.approx(1.0)
    assert wv == pytest.approx(1.5 / 2.4)
    assert om.modality_weights(0.0, 0.0, 5.0) == pytest.approx((5 / 6, 1 / 6))
    assert om.modality_weights(0.4, 0.0, 5.0) == (1.0, 0.0)


def test_golden_memory_size_split_is_consistent_with_paper():
    # The paper prints ~800 audio at r = 5 and ~400 audio at r = 10 for a 4k
    # budget.  One compressibility ratio C_a / C_v must explain both, which
    # holds only if r multiplies C_v (Eq. 11) and not C_a.
    with open(os.path.join(GOLDEN, "avba_memory_size.json")) as f:
        gold = json.load(f)
    b, tol = gold["budget"], gold["relative_tolerance"]
    ratio = scipy.optimize.brentq(
        lambda x: om.modality_weights(1.0, x, gold["r_default"])[1] * b - gold["audio_at_r5"],
        1e-6, 1e3)
    audio_r10 = om.modality_weights(1.0, ratio, gold["r_alt"])[1] * b
    assert abs(audio_r10 - gold["audio_at_r10"]) <= tol * gold["audio_at_r10"]
    visual_r5 = om.modality_weights(1.0, ratio, gold["r_default"])[0] * b
    assert abs(visual_r5 - gold["visual_at_r5_approx"]) <= 0.15 * b


# --------------------------------------------------------------------------
# Eq. (14) with the [B_min, B_max] constraint, integer budgets, the split
# --------------------------------------------------------------------------

def test_single_layer_gets_whole_budget():
    x = om.layer_shares([0.37], [6144], 4096)
    assert x[0] == pytest.approx(4096.0)
    assert om.integer_budgets(x, [6144], 4096).tolist() == [4096]
    # fewer tokens than budget: keep them all
    assert om.integer_budgets(om.layer_shares([0.1], [300], 4096), [300], 4096).tolist() == [300]


def test_equal_compressibility_equal_budgets_and_shift_invariance():
    n = [6144] * 5
    x = om.layer_shares([0.4] * 5, n, 5 * 4096 + 3)
    np.testing.assert_allclose(x, (5 * 4096 + 3) / 5)
    c = np.array([0.2, 0.5, 0.45, 0.9, 0.1])
    np.testing.assert_allclose(om.layer_shares(c, n, 20480), om.layer_shares(c + 3.0, n, 20480),
                               rtol=1e-12)


def test_equal_shares_leftover_goes_to_lower_layers():
    # Five equal layers and three spare units: layers 0, 1 and 2 get them.
    n = [6144] * 5
    x = om.layer_shares([0.4] * 5, n, 5 * 4096 + 3)
    assert om.integer_budgets(x, n, 5 * 4096 + 3).tolist() == [4097, 4097, 4097, 4096, 4096]


def test_budgets_respect_real_valued_bounds():
    # One dominant layer: the others sit at the smallest integer budget that
    # is at least B_min = 0.5 B_tot / L, the dominant one at most B_max.
    n = [1000] * 3
    c = [5.0, 0.0, 0.0]
    x = om.layer_shares(c, n, 100, 0.2)
    b = om.integer_budgets(x, n, 100)
    assert b.sum() == 100
    assert b[1] == b[2] == 17  # ceil(100 / 6)
    assert b[0] == 66          # 100 - 2 * 17 <= floor(200 / 3)
    assert all(bl >= 0.5 * 100 / 3 and bl <= 2.0 * 100 / 3 for bl in b)
    wide = om.integer_budgets(om.layer_shares(c, n, 100, 0.2, bmax_frac=3.0), n, 100,
                              bmax_frac=3.0)
    assert wide.tolist() == [66, 17, 17]


def test_shares_keep_every_token_when_budget_exceeds_them():
    x = om.layer_shares([0.1, 0.9], [1500, 2000], 4096)
    np.testing.assert_array_equal(x, [1500.0, 2000.0])
    assert om.integer_budgets(x, [1500, 2000], 4096).tolist() == [1500, 2000]


def test_unclamped_shares_are_softmax_library():
    c = np.array([0.3, 0.35, 0.25, 0.31])
    x = om.layer_shares(c, [10 ** 6] * 4, 1000, 0.2, bmin_frac=0.0, bmax_frac=4.0)
    np.testing.assert_allclose(x, 1000 * scipy.special.softmax(c / 0.2), rtol=1e-12)


def test_waterfill_matches_independent_root_finder():
    rng = np.random.default_rng(12)
    for trial in range(20):
        L = int(rng.integers(2, 30))
        c = rng.uniform(0.0, 1.0, size=L)
        n = rng.integers(1000, 9000, size=L)
        b = int(rng.integers(L * 500, min(int(n.sum()) - 1, L * 6000)))
        t = float(rng.uniform(0.05, 1.0))
        lo, hi = om.layer_bounds(n, b)
        if lo.sum() > b:
            continue
        x = om.layer_shares(c, n, b, t)
        assert x.sum() == pytest.approx(min(b, hi.sum()), rel=1e-12)
        assert (x >= lo - 1e-9).all() and (x <= hi + 1e-9).all()
        if hi.sum() <= b:
            continue
        p = scipy.special.softmax(c / t)
        f = lambda kap: np.clip(kap * b * p, lo, hi).sum() - b
        kap = scipy.optimize.brentq(f, 0.0, 1e6, xtol=1e-15, rtol=1e-15)
        np.testing.assert_allclose(x, np.clip(kap * b * p, lo, hi), rtol=1e-9, atol=1e-7)


def test_integer_budgets_are_the_closest_apportionment():
    # Largest remainder = the integer vector with entries in {floor x, ceil x},
    # sum B_tot, closest to x in squared error; ties -> earlier layers first.
    rng = np.random.default_rng(13)
    for trial in range(30):
        L = int(rng.integers(2, 7))
        n = rng.integers(50, 200, size=L)
        b = int(rng.integers(L * 40, int(n.sum())))
        c = rng.uniform(0, 1, size=L)
        lo, hi = om.layer_bounds(n, b)
        if lo.sum() > b or hi.sum() <= b:
            continue
        x = om.layer_shares(c, n, b, 0.3)
        got = om.integer_budgets(x, n, b)
        best = None
        for choice in itertools.product(*[sorted({math.floor(v), math.ceil(v)}) for v in x]):
            if sum(choice) != b or any(ch > h for ch, h in zip(choice, hi)):
                continue
            err = sum((ch - v) ** 2 for ch, v in zip(choice, x))
            key = (round(err, 9), [-ch for ch in choice])
            if best is None or key < best[0]:
                best = (key, choice)
        assert list(got) == list(best[1])
        assert got.sum() == b


def test_infeasible_minimum_budgets():
    with pytest.raises(om.InfeasibleBudget):
        om.layer_shares([0.1, 0.2], [5000, 5000], 100, bmin_frac=3.0, bmax_frac=4.0)


def test_split_budget_cases():
    assert om.split_budget(4096, 5 / 6, 4608, 1536) == (3413, 683)
    assert om.split_budget(100, 1.0, 60, 80) == (60, 40)     # visual capped by K_v
    assert om.split_budget(95, 0.0, 90, 5) == (90, 5)        # audio capped by K_a
    assert om.split_budget(7, 0.5, 10, 10) == (4, 3)         # round half up
    for bl, w, kv, ka in [(50, 0.3, 40, 40), (0, 0.9, 3, 3), (80, 0.99, 30, 60)]:
        mv, ma = om.split_budget(bl, w, kv, ka)
        assert mv + ma == bl and 0 <= mv <= kv and 0 <= ma <= ka


# --------------------------------------------------------------------------
# Eqs. (4), (5): Select by top-M psi, and the compaction
# --------------------------------------------------------------------------

def _brute_force_select(psi_row, positions, m):
    best = None
    for subset in itertools.combinations(positions, m):
        total = sum(psi_row[p] for p in subset)
        key = (-total, list(subset))
        if best is None or key < best:
            best = key
    return sorted(best[1]) if best else []


def test_select_is_max_sum_subset_with_earliest_ties():
    rng = np.random.default_rng(14)
    for trial in range(40):
        n = int(rng.integers(2, 13))
        mod = rng.integers(0, 2, size=n).astype(np.uint8)
        # coarse values make ties frequent
        psi = rng.integers(0, 4, size=(2, n)).astype(float) / 4.0
        kv, ka = int((mod == 0).sum()), int((mod == 1).sum())
        mv, ma = int(rng.integers(0, kv + 1)), int(rng.integers(0, ka + 1))
        idx = om.select(psi, mod, mv, ma)
        for g in range(2):
            vis = [p for p in range(n) if mod[p] == 0]
            aud = [p for p in range(n) if mod[p] == 1]
            want = _brute_force_select(psi[g], vis, mv) + _brute_force_select(psi[g], aud, ma)
            assert idx[g].tolist() == want


def test_compact_moves_rows_to_their_slots():
    x = np.arange(10, dtype=float)[None, :, None].repeat(2, axis=0).repeat(3, axis=2)
    psi = np.array([[0.1, 0.9, 0.5, 0.7, 0.2, 0.8, 0.3, 0.6, 0.4, 0.0]] * 2)
    mod = np.array([0, 1, 0, 1, 0, 1, 0, 1, 0, 1], dtype=np.uint8)
    idx = om.select(psi, mod, 2, 3)
    assert idx[0].tolist() == [2, 8, 1, 3, 5]
    out = om.compact(x, idx)
    np.testing.assert_array_equal(out[:, :, 0], idx.astype(float))


# --------------------------------------------------------------------------
# The whole step
# --------------------------------------------------------------------------

def _tiny_layers(n_layers=3, seed=20):
    rng = np.random.default_rng(seed)
    layers = []
    for l in range(n_layers):
        n_cache, n_chunk = 24, 12
        mod = np.array(([0] * 18 + [1] * 6) + ([0] * 4 + [1] * 2) * 2, dtype=np.uint8)
        v = rng.standard_normal((2, 36, 8))
        v[:, 10] = v[:, 3] + 0.01 * rng.standard_normal((2, 8))
        layers.append(dict(q=rng.standard_normal((4, n_chunk, 8)) * (l + 1),
                           k=rng.standard_normal((2, 36, 8)), v=v, modality=mod,
                           n_cache=n_cache, sm_scale=1 / math.sqrt(8)))
    return layers


@pytest.mark.parametrize("mode", ["max", "adj"])
def test_step_invariants(mode):
    layers = _tiny_layers()
    out = om.compression_step(layers, 3 * 20, mode=mode)
    assert sum(mv + ma for mv, ma in out["budgets"]) == 60
    for layer, (mv, ma), idx, ko in zip(layers, out["budgets"], out["idx"], out["k_out"]):
        mod = layer["modality"]
        assert idx.shape == (2, mv + ma)
        for g in range(2):
            assert (mod[idx[g, :mv]] == 0).all() and (mod[idx[g, mv:]] == 1).all()
            assert (np.diff(idx[g, :mv]) > 0).all() and (np.diff(idx[g, mv:]) > 0).all()
        np.testing.assert_array_equal(ko[1], layer["k"][1, idx[1]])
    lo, hi = om.layer_bounds([36] * 3, 60)
    assert all(lo[l] <= out["layer_budgets"][l] <= hi[l] for l in range(3))


def test_step_drops_the_redundant_twin_first():
    # A token with an exact twin in its modality has psi = 0 under 'max':
    # with a budget that cannot keep every token, both twins go first.
    layers = _tiny_layers(1, seed=21)
    layers[0]["v"][:, 10] = layers[0]["v"][:, 3]
    out = om.compression_step(layers, 30)
    kept = set(out["idx"][0][0].tolist())
    assert 3 not in kept and 10 not in kept
