"""Comparison rules between the HIP path and the oracle.

Tolerances (bf16/fp32 inputs, fp32 accumulation on the GPU, fp64 oracle):
  a, lse, normalised entropy, C, w:  |d| <= 1e-3 |ref| + 1e-6 mean|ref|
  s:                                 |d| <= 1e-3 |ref| + 1e-5
Integer work (budgets from identical inputs, gathers) is bit-exact.  Kept
index sets are bit-exact where the oracle's psi margin at the M-th boundary
exceeds 1e-3 relative; otherwise every kept row must have psi >= psi_(M)
(1 - 1e-3) and every dropped row psi <= psi_(M) (1 + 1e-3).
"""
import math

import numpy as np

from oracle import omnimem_oracle as om

# The library's configuration values are fp32; the oracle takes the same
# numbers widened to fp64.
LAMBDA = float(np.float32(om.DEFAULT_LAMBDA))
TEMPERATURE = float(np.float32(om.DEFAULT_T))
RATIO = float(np.float32(om.DEFAULT_R))
REL = 1e-3


def assert_close_a(got, ref, what="a"):
    got = np.asarray(got, dtype=np.float64)
    ref = np.asarray(ref, dtype=np.float64)
    tol = REL * np.abs(ref) + 1e-6 * np.abs(ref).mean()
    bad = np.abs(got - ref) > tol
    if bad.any():
        i = np.argmax(np.abs(got - ref) - tol)
        raise AssertionError(f"{what}: {bad.sum()} of {bad.size} beyond tolerance; worst at flat {i}: "
                             f"got {got.flat[i]!r} ref {ref.flat[i]!r}")


def assert_close_s(got, ref, what="s"):
    got = np.asarray(got, dtype=np.float64)
    ref = np.asarray(ref, dtype=np.float64)
    tol = REL * np.abs(ref) + 1e-5
    bad = np.abs(got - ref) > tol
    if bad.any():
        i = np.argmax(np.abs(got - ref) - tol)
        raise AssertionError(f"{what}: {bad.sum()} of {bad.size} beyond tolerance; worst at flat {i}: "
                             f"got {got.flat[i]!r} ref {ref.flat[i]!r}")


def check_selection(idx_row, psi_row, modality, m_v, m_a, rel=REL):
    """One KV head: GPU kept rows vs the oracle's psi.  Returns #exact blocks."""
    modality = np.asarray(modality)
    exact = 0
    for mu, lo, hi in ((0, 0, m_v), (1, m_v, m_v + m_a)):
        got = np.asarray(idx_row[lo:hi], dtype=np.int64)
        m = hi - lo
        pos = om.segment_positions(modality, mu)
        assert len(got) == m
        if m:
            assert (np.diff(got) > 0).all(), "kept rows not ascending"
            assert (modality[got] == mu).all(), "kept row of the wrong modality"
        order = sorted(pos.tolist(), key=lambda p: (-psi_row[p], p))
        ref = np.sort(np.array(order[:m], dtype=np.int64))
        if m == 0 or m == len(pos):
            np.testing.assert_array_equal(got, ref)
            exact += 1
            continue
        psi_m, psi_next = psi_row[order[m - 1]], psi_row[order[m]]
        margin = (psi_m - psi_next) / psi_m if psi_m > 0 else 0.0
        if margin > rel:
            np.testing.assert_array_equal(got, ref)
            exact += 1
        else:
            kept = set(got.tolist())
            dropped = [p for p in pos.tolist() if p not in kept]
            assert all(psi_row[p] >= psi_m * (1 - rel) for p in kept)
            assert all(psi_row[p] <= psi_m * (1 + rel) for p in dropped)
    return exact


def check_topk_property(idx_row, a_row, s_row, modality, m_v, m_a, lam=LAMBDA, rel=1e-5):
    """One KV head of the GPU's own chain: the kept rows of each modality
    are ascending, of that modality, M of them, and no dropped row has a
    larger psi = a^lam (1 - s) than a kept one.  psi is recomputed here in
    float64 from the GPU's fp32 a and s; the GPU orders by its fp32 psi, so
    a relative slack of `rel` is allowed."""
    modality = np.asarray(modality)
    psi = np.power(np.asarray(a_row, dtype=np.float64), lam) * (1.0 - np.asarray(s_row, dtype=np.float64))
    for mu, lo, hi in ((0, 0, m_v), (1, m_v, m_v + m_a)):
        got = np.asarray(idx_row[lo:hi], dtype=np.int64)
        pos = np.flatnonzero(modality == mu)
        assert len(got) == hi - lo
        if len(got) == 0:
            continue
        assert (np.diff(got) > 0).all(), "kept rows not ascending"
        assert (modality[got] == mu).all(), "kept row of the wrong modality"
        dropped = np.setdiff1d(pos, got)
        if len(dropped):
            assert psi[dropped].max() <= psi[got].min() * (1 + rel), "a dropped row outranks a kept one"


def oracle_allocation(a_list, s_list, layers, total_budget, bmin=om.DEFAULT_BMIN_FRAC,
                      bmax=om.DEFAULT_BMAX_FRAC, temperature=TEMPERATURE, r=RATIO):
    """Oracle stats, shares and (M_v, M_a) per layer from given a, s."""
    stats = [om.avba_statistics(a, s, l["modality"]) for a, s, l in zip(a_list, s_list, layers)]
    n_tok = [len(l["modality"]) for l in layers]
    shares = om.layer_shares([st["C_l"] for st in stats], n_tok, total_budget, temperature, bmin, bmax)
    b_l = om.integer_budgets(shares, n_tok, total_budget, bmin, bmax)
    budgets = []
    for st, b, l in zip(stats, b_l, layers):
        mod = np.asarray(l["modality"])
        w_v, _ = om.modality_weights(st["C_v"], st["C_a"], r)
        st["w_v"] = w_v
        budgets.append(om.split_budget(int(b), w_v, int((mod == 0).sum()), int((mod == 1).sum())))
    return stats, shares, np.array(budgets, dtype=np.int64)


STAT_KEYS = ["H_v", "H_a", "H_l", "sbar_v", "sbar_a", "sbar_l", "C_v", "C_a", "C_l", "w_v"]


def as_f64(layer):
    out = dict(layer)
    for key in ("q", "k", "v"):
        out[key] = np.asarray(layer[key], dtype=np.float64)
    return out


def free_running_budget_bounds(gpu_stats, ref_stats, shares, ref_budgets, temperature=TEMPERATURE):
    """Per-layer bounds on |M_v - M_v_ref| and |M_a - M_a_ref| when the
    budgets come from the GPU's own a and s, derived from the measured
    differences of the statistics (Eqs. 13, 14 and readings R16-R18):

    x_l = clamp(kappa B_tot p_l, lo_l, hi_l), p = softmax(C / T).  If every
    C_l moves by at most dC, each p_l moves by a factor within exp(+-2 dC/T),
    kappa (fixed by sum x = B_tot) by at most the same, and the clamp does not
    amplify: |dx_l| <= x_l (exp(4 dC/T) - 1).  The integer budgets (R17) add
    at most one unit (a floor crossing or a change in the remainder order):
    |dB_l| <= ceil(|dx_l|) + 1.  The split M_v = floor(w_v B_l + 1/2), clamped
    (R18), moves by at most |dB_l| + B_l |dw_v| + 1, and M_a = B_l - M_v by
    at most |dB_l| + |dM_v|.
    """
    d_c = max(abs(float(g[8]) - float(r["C_l"])) for g, r in zip(gpu_stats, ref_stats))
    grow = math.expm1(4.0 * d_c / temperature)
    out = []
    for l, (g, r) in enumerate(zip(gpu_stats, ref_stats)):
        d_b = math.ceil(float(shares[l]) * grow) + 1
        b_l = int(ref_budgets[l].sum())
        d_mv = d_b + math.ceil(b_l * abs(float(g[9]) - float(r["w_v"]))) + 1
        out.append((d_mv, d_b + d_mv))
    return np.array(out, dtype=np.int64)
