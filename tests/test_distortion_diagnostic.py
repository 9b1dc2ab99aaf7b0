"""Attention-output distortion of the psi-selected cache (diagnostic, CPU).

Sec. 3.1 motivates the retention score psi = a^lambda (1 - s) (Eq. 8): keep
the rows the chunk's queries attend to (Eq. 6) and drop the rows that other
rows already stand for (Eq. 7), so that attention over the kept rows stays
close to attention over all of them.  On tiny duplicate-rich working sets
this test enumerates every subset S of M rows and measures the distortion

    D(S) = || softmax(sigma Q K_S^T) V_S - softmax(sigma Q K^T) V ||^2

of the chunk queries' outputs (all rows visible, summed over heads and
queries).  It reports where the oracle's psi-selected subset ranks among all
C(N, M) subsets (the fraction of subsets with a smaller distortion), beside
the "uniform" selection that keeps every (N/M)-th row.  The paper fixes no
value for this, so it is a diagnostic: the only assertion is the survey's,
that on duplicate-rich inputs psi does better than the median subset, made
for the redundancy form the paper prints (Eq. 7, adjacent rows) on inputs
whose near-duplicates come in runs, as consecutive video frames do.

What it shows: with the all-pairs maximum (reading R6), the two members of a
tight near-duplicate pair have the same s (cosine is symmetric), so both are
dropped together and psi's subset ranks among the worst; Eq. 7 as printed
keeps the ends of a run and ranks better than the median; uniform selection
beats both on run-structured data.  Printed with ``pytest -s``.
"""
import itertools
import math

import numpy as np

from oracle import omnimem_oracle as om

RUNS = [1, 3, 1, 2, 1, 3, 1, 2]   # 8 distinct rows, 14 rows in all
KEEP = 8
SEEDS = range(10)


def _working_set(seed, runs, shuffle, d=8, h_q=2, n_q=4, noise=0.02):
    """Rows in runs of near-identical keys and values (each run one
    underlying row plus small noise); optionally in random order."""
    rng = np.random.default_rng(seed)
    base_k = rng.standard_normal((len(runs), d))
    base_v = rng.standard_normal((len(runs), d))
    which = [i for i, r in enumerate(runs) for _ in range(r)]
    k = base_k[which] + noise * rng.standard_normal((len(which), d))
    v = base_v[which] + noise * rng.standard_normal((len(which), d))
    if shuffle:
        order = rng.permutation(len(which))
        k, v = k[order], v[order]
    q = rng.standard_normal((h_q, n_q, d))
    return q, k[None], v[None]


def _outputs(q, k, v, rows, sigma):
    logits = np.einsum("hcd,nd->hcn", q, k[0, rows]) * sigma
    logits -= logits.max(axis=-1, keepdims=True)
    p = np.exp(logits)
    p /= p.sum(axis=-1, keepdims=True)
    return np.einsum("hcn,nd->hcd", p, v[0, rows])


def _ranks(q, k, v, keep, mode):
    """(rank of the psi subset, rank of the uniform subset) among all subsets."""
    n, d = k.shape[1], k.shape[2]
    sigma = 1.0 / math.sqrt(d)
    modality = np.zeros(n, dtype=np.uint8)
    a = om.attention_importance(q, k, n - q.shape[1], sigma, causal=False)
    s = om.redundancy(v, modality, mode)
    chosen = om.select(om.retention_score(a, s), modality, keep, 0)[0]
    full = _outputs(q, k, v, np.arange(n), sigma)

    def distortion(rows):
        return float(((_outputs(q, k, v, np.asarray(rows), sigma) - full) ** 2).sum())

    every = np.array([distortion(c) for c in itertools.combinations(range(n), keep)])
    uniform = [math.floor(i * n / keep) for i in range(keep)]
    return float((every < distortion(chosen)).mean()), float((every < distortion(uniform)).mean())


def test_distortion_is_zero_for_the_whole_set():
    q, k, v = _working_set(0, RUNS, shuffle=False)
    n = k.shape[1]
    sigma = 1.0 / math.sqrt(k.shape[2])
    full = _outputs(q, k, v, np.arange(n), sigma)
    assert np.array_equal(_outputs(q, k, v, np.arange(n), sigma), full)


def test_psi_subset_rank_diagnostic():
    table = {}
    for mode in ("adj", "max"):
        for shuffle in (False, True):
            r = np.array([_ranks(*_working_set(seed, RUNS, shuffle), KEEP, mode) for seed in SEEDS])
            assert np.isfinite(r).all() and ((0.0 <= r) & (r <= 1.0)).all()
            table[(mode, shuffle)] = r
    print("\nfraction of the C(14, 8) subsets with less distortion (median / worst over 10 seeds)")
    for (mode, shuffle), r in table.items():
        print(f"  redundancy {mode:3s} {'shuffled rows' if shuffle else 'runs of rows ':13s}: "
              f"psi {np.median(r[:, 0]):.3f} / {r[:, 0].max():.3f}   uniform {np.median(r[:, 1]):.3f}")
    # Eq. 7 as printed, near-duplicates in runs: psi does better than the median subset.
    assert np.median(table[("adj", False)][:, 0]) < 0.5
