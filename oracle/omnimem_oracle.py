"""Plain CPU oracle of OmniMem's per-chunk KV-cache compression step.

TEST INFRASTRUCTURE ONLY.  Nothing on the product path may import, call or
execute this module: only the test suite, the package smoke check and the
benchmark's CPU-baseline leg use it.  It shares no code, constants or helpers
with the HIP library; both sides receive the same seeded inputs.

Everything is float64 numpy on inputs already rounded to the working dtype.
Each function follows one passage of the paper (OmniMem, arXiv 2606.07577)
in the paper's order and notation:

  * Eq. (1)  chunk attention over [visual cache; audio cache; chunk]   -> attention_lse
  * Eq. (6)  accumulated attention importance a_k                     -> attention_importance
  * Eq. (7)  cosine redundancy s_k (value vectors, Sec. 3.1)          -> redundancy
    (hidden states, as Eq. (7) is printed)                            -> hidden_redundancy
  * Eq. (8)  retention score psi_k = a_k^lambda (1 - s_k)              -> retention_score
  * Eqs. (9), (10), (13)  normalised entropy x (1 - mean cosine)      -> avba_statistics
  * Eqs. (11), (12)  audio/visual proportions w_v, w_a                -> modality_weights
  * Eq. (14) + the [B_min, B_max] constraint of Sec. 3.2              -> layer_budgets
  * the layer budget divided between the modalities by w_v and w_a
    (Sec. 3.2, after Eqs. (11), (12))                                 -> split_budget
  * layer budgets fixed in advance from calibration data
    (end of Sec. 3.2)                                                 -> calibration_budgets,
                                                                         fixed_split
  * Eqs. (4), (5) Select: top-M by psi per modality (Sec. 3.1)         -> select
    (one index set per layer, as Eqs. (4), (5) write it)              -> layer_shared_select
  * Eq. (3) / Eq. (2): the retained pairs form the next caches         -> compact

Where the paper is silent the oracle takes these readings (each one is
listed with its justification in the design notes):
  R2  causal attention inside the chunk; cache rows visible to every query.
  R4  one joint softmax over cache and chunk rows of both modalities.
  R5  importance and selection per KV head; a_k sums the G query heads of
      that KV head.
  R6  two redundancy modes: 'max' = max cosine to any other member of the
      same (KV head, modality) segment; 'adj' = Eq. (7) literally, with the
      neighbours taken in the modality's own order.
  R9  0^lambda = 0 for lambda > 0, x^0 = 1; cosine clamped to [-1, 1] and 0
      when either vector has zero norm.
  R10 ties in the top-M go to the lower working-set position.
  R12 normalised entropy per KV head, averaged over KV heads; mean cosine
      over all heads and tokens of the modality.
  R14 Eq. (13) is normalised by ln N (the layer's token count).
  R15 B_tot * Softmax(C/T) is the layer's real-valued budget.
  R16 the clamp to [B_min, B_max] keeps the sum: x_l = clamp(kappa B_tot p_l,
      lo_l, hi_l) with the unique kappa giving sum x_l = B_tot.  The values
      B_min = 0.5 B_tot/L and B_max = 2 B_tot/L are a proposal: the paper
      gives none.  PARITY UNPINNED for those two constants.
  R17 integer layer budgets by largest remainder, ties to the lower layer.
  R18 M_v = round-half-up(w_v B_l) clamped so that both modalities fit.
  R21 offline budgets: C^(l) of Eq. (13) averaged over the calibration
      steps, then Eq. (14), the clamp and the integer rounding (R15-R17) on
      the means, with no cap by a layer's token count; a step under these
      budgets keeps min(B^(l), N_l) rows of layer l, split by its own w_v.
  R22 layer-shared selection: the layer's psi takes a summed over the KV
      heads (every query head's attention, Eq. (6) over all heads) and s
      averaged over them; every KV head keeps the rows chosen from it.
  R23 hidden-state source: Eq. (7) on the layer's hidden states (one per
      token, shared by its KV heads), adjacent form as printed; the kept
      rows' hidden states are carried with the cache, which needs one
      index set per layer (R22).
"""
from __future__ import annotations

import math

import numpy as np

VISUAL = 0
AUDIO = 1

# Sec. 4.3 (inference specifications): lambda = 0.02, T = 0.2.  Sec. 3.2: r = 5.
DEFAULT_LAMBDA = 0.02
DEFAULT_T = 0.2
DEFAULT_R = 5.0
# Reading R16 (the paper states that the clamp exists but not its values).
DEFAULT_BMIN_FRAC = 0.5
DEFAULT_BMAX_FRAC = 2.0


class InfeasibleBudget(ValueError):
    """The per-layer minimum budgets exceed the total budget."""


# ---------------------------------------------------------------------------
# Eq. (1) and Eq. (6): attention of the chunk queries over the working set
# ---------------------------------------------------------------------------

def visibility(n_cache: int, n_chunk: int, causal: bool = True) -> np.ndarray:
    """[C, N] boolean: may chunk query i attend to working-set row j.

    Rows 0..n_cache-1 are the retained caches (both modalities), rows
    n_cache.. are the chunk in time order (Eq. 3 appends the chunk after the
    cache).  Reading R2: every cache row is visible; chunk row n_cache + t is
    visible to chunk query i iff t <= i.
    """
    n = n_cache + n_chunk
    i = np.arange(n_chunk)[:, None]
    j = np.arange(n)[None, :]
    if not causal:
        return np.ones((n_chunk, n), dtype=bool)
    return (j < n_cache) | (j - n_cache <= i)


def attention_lse(q, k, n_cache, sm_scale, causal=True, queries=None):
    """log sum_j exp(sm_scale <q_{h,i}, k_{g(h),j}>) over the rows visible to i.

    This is the normaliser of the softmax in the chunk attention of Eq. (1);
    query head h reads KV head g(h) = h // G with G = H_q / H_kv.
    q: [H_q, C, d]; k: [H_kv, N, d].  Returns [H_q, len(queries)].
    """
    h_q, c, _ = q.shape
    h_kv, n, _ = k.shape
    group = h_q // h_kv
    qs = np.arange(c) if queries is None else np.asarray(queries)
    vis = visibility(n_cache, n - n_cache, causal)[qs]
    lse = np.empty((h_q, len(qs)))
    for h in range(h_q):
        scores = sm_scale * (q[h, qs] @ k[h // group].T)
        scores = np.where(vis, scores, -np.inf)
        m = scores.max(axis=1, keepdims=True)
        lse[h] = m[:, 0] + np.log(np.exp(scores - m).sum(axis=1))
    return lse


def attention_importance(q, k, n_cache, sm_scale, causal=True, lse=None, keys=None):
    """Eq. (6): a_k = sum over chunk queries q of the attention A_{q,k}.

    Reading R5: per KV head g, the sum runs over every chunk query of every
    query head in g's group.  A is the softmax of Eq. (1) (reading R4: one
    softmax over all visible rows of both modalities).  `lse` may be given
    (shape [H_q, C]); `keys` restricts the output to those working-set rows.
    Returns [H_kv, len(keys)].
    """
    h_q, c, _ = q.shape
    h_kv, n, _ = k.shape
    group = h_q // h_kv
    if lse is None:
        lse = attention_lse(q, k, n_cache, sm_scale, causal)
    ks = np.arange(n) if keys is None else np.asarray(keys)
    vis = visibility(n_cache, n - n_cache, causal)[:, ks]
    a = np.zeros((h_kv, len(ks)))
    for h in range(h_q):
        g = h // group
        scores = sm_scale * (q[h] @ k[g, ks].T)
        probs = np.exp(np.where(vis, scores - lse[h][:, None], -np.inf))
        a[g] += probs.sum(axis=0)
    return a


# ---------------------------------------------------------------------------
# Eq. (7): cosine-similarity redundancy (value vectors, Sec. 3.1)
# ---------------------------------------------------------------------------

def segment_positions(modality, mu):
    """Working-set rows of modality mu, ascending (the order of Eq. 3)."""
    return np.flatnonzero(np.asarray(modality) == mu)


def cosine_matrix(x, y):
    """cos(x_i, y_j); 0 where either vector has zero norm; clamped to [-1, 1]."""
    nx = np.sqrt((x * x).sum(axis=1))
    ny = np.sqrt((y * y).sum(axis=1))
    den = np.outer(nx, ny)
    dots = x @ y.T
    safe = np.where(den > 0, den, 1.0)
    return np.clip(np.where(den > 0, dots / safe, 0.0), -1.0, 1.0)


def redundancy(u, modality, mode="max", rows=None):
    """s_k for every row of u ([H_kv, N, d], values by default, reading R7).

    mode 'adj' is Eq. (7): the mean of the cosine with the previous and the
    next member of the same modality (one neighbour at either end, 0 for a
    modality with a single token, reading R8).  mode 'max' (reading R6) is
    the largest cosine with any other member of the same modality.
    `rows` restricts the output to those working-set rows.  Returns
    [H_kv, len(rows)].
    """
    h_kv, n, _ = u.shape
    modality = np.asarray(modality)
    rows = np.arange(n) if rows is None else np.asarray(rows)
    out = np.zeros((h_kv, len(rows)))
    for mu in (VISUAL, AUDIO):
        pos = segment_positions(modality, mu)
        if len(pos) < 2:
            continue  # a lone token has nothing to be redundant with: s = 0
        rank = {int(p): t for t, p in enumerate(pos)}
        want = [(r_out, rank[int(p)]) for r_out, p in enumerate(rows) if int(p) in rank]
        if not want:
            continue
        r_out = np.array([w[0] for w in want])
        t_seg = np.array([w[1] for w in want])
        for g in range(h_kv):
            seg = u[g, pos]
            if mode == "max":
                cos = cosine_matrix(seg[t_seg], seg)
                cos[np.arange(len(t_seg)), t_seg] = -np.inf
                out[g, r_out] = cos.max(axis=1)
            elif mode == "adj":
                for ro, t in zip(r_out, t_seg):
                    nbrs = [x for x in (t - 1, t + 1) if 0 <= x < len(pos)]
                    cos = cosine_matrix(seg[[t]], seg[nbrs])[0]
                    out[g, ro] = cos.mean()
            else:
                raise ValueError(mode)
    return out


def hidden_redundancy(h, modality, h_kv, mode="adj"):
    """Eq. (7) as printed (reading R23): s_k from the hidden states
    h [N, d_model] of the layer's tokens, one value per token, repeated for
    each of the h_kv KV heads.  Returns [h_kv, N]."""
    s = redundancy(np.asarray(h, dtype=np.float64)[None], modality, mode)
    return np.repeat(s, h_kv, axis=0)


# ---------------------------------------------------------------------------
# Eq. (8): retention score
# ---------------------------------------------------------------------------

def retention_score(a, s, lam=DEFAULT_LAMBDA):
    """psi_k = a_k^lambda (1 - s_k)  (reading R9: 0^lambda = 0, x^0 = 1)."""
    return np.power(a, lam) * (1.0 - s)


# ---------------------------------------------------------------------------
# Eqs. (9), (10), (13): compressibility statistics
# ---------------------------------------------------------------------------

def normalized_entropy(x):
    """H[x / sum x] / ln K for K = len(x) entries (0 ln 0 = 0).

    K <= 1, or an all-zero x, gives 0.
    """
    x = np.asarray(x, dtype=np.float64)
    if x.size <= 1:
        return 0.0
    total = x.sum()
    if total <= 0:
        return 0.0
    p = x / total
    p = p[p > 0]
    return float(-(p * np.log(p)).sum() / math.log(x.size))


def avba_statistics(a, s, modality):
    """Per-layer AVBA inputs from importance a and redundancy s ([H_kv, N]).

    Eqs. (9)-(10): C_mu = Hn[a_mu] (1 - sbar_mu) where Hn is the entropy of
    the attention normalised over the modality's tokens divided by ln K_mu.
    Eq. (13): C_l = Hn[a] (1 - sbar) over all N tokens (reading R14: also
    divided by ln N).  Reading R12: Hn is computed per KV head and averaged;
    sbar averages s over every head and token of the set.
    """
    modality = np.asarray(modality)
    h_kv = a.shape[0]
    stats = {}
    sets = {
        "v": modality == VISUAL,
        "a": modality == AUDIO,
        "l": np.ones_like(modality, dtype=bool),
    }
    for name, sel in sets.items():
        ent = float(np.mean([normalized_entropy(a[g, sel]) for g in range(h_kv)]))
        sbar = float(s[:, sel].mean()) if sel.any() else 0.0
        stats["H_" + name] = ent
        stats["sbar_" + name] = sbar
        stats["C_" + name] = ent * (1.0 - sbar)
    return stats


# ---------------------------------------------------------------------------
# Eqs. (11), (12): audio/visual proportions
# ---------------------------------------------------------------------------

def modality_weights(c_v, c_a, r=DEFAULT_R):
    """w_v = C_v r / (C_v r + C_a), w_a = C_a / (C_v r + C_a).

    A zero denominator (no signal in either modality) falls back to the
    prior ratio: w_v = r / (r + 1).
    """
    den = c_v * r + c_a
    if den <= 0:
        return r / (r + 1.0), 1.0 / (r + 1.0)
    return c_v * r / den, c_a / den


# ---------------------------------------------------------------------------
# Eq. (14) and the [B_min, B_max] constraint (Sec. 3.2)
# ---------------------------------------------------------------------------

def layer_softmax(c_layers, temperature=DEFAULT_T):
    """Softmax over layers of C^(l) / T (Eq. 14)."""
    c = np.asarray(c_layers, dtype=np.float64) / temperature
    e = np.exp(c - c.max())
    return e / e.sum()


def layer_bounds(n_tokens, total_budget, bmin_frac=DEFAULT_BMIN_FRAC,
                 bmax_frac=DEFAULT_BMAX_FRAC):
    """lo_l = min(ceil(bmin_frac B_tot / L), N_l), hi_l = min(floor(bmax_frac B_tot / L), N_l)."""
    n_tokens = np.asarray(n_tokens, dtype=np.int64)
    n_layers = len(n_tokens)
    lo_base = math.ceil((float(bmin_frac) * float(total_budget)) / n_layers)
    hi_base = math.floor((float(bmax_frac) * float(total_budget)) / n_layers)
    lo = np.minimum(lo_base, n_tokens)
    hi = np.minimum(hi_base, n_tokens)
    return lo, hi


def layer_shares(c_layers, n_tokens, total_budget, temperature=DEFAULT_T,
                 bmin_frac=DEFAULT_BMIN_FRAC, bmax_frac=DEFAULT_BMAX_FRAC):
    """Real-valued layer budgets x_l (readings R15, R16).

    x_l = clamp(kappa * B_tot * p_l, lo_l, hi_l) with p = Softmax(C/T) and
    the unique kappa for which sum_l x_l = B_tot, found from the sorted
    breakpoints of the piecewise-linear sum.  If even the upper bounds do
    not reach B_tot every layer keeps hi_l.
    """
    p = layer_softmax(c_layers, temperature)
    lo, hi = layer_bounds(n_tokens, total_budget, bmin_frac, bmax_frac)
    lo = lo.astype(np.float64)
    hi = hi.astype(np.float64)
    b = float(total_budget)
    if lo.sum() > b:
        raise InfeasibleBudget("sum of per-layer minimum budgets exceeds the total")
    if hi.sum() <= b:
        return hi.copy()

    def total(kappa):
        return np.clip(kappa * b * p, lo, hi).sum()

    live = p > 0
    breaks = np.sort(np.concatenate([lo[live] / (b * p[live]), hi[live] / (b * p[live])]))
    values = np.array([total(kb) for kb in breaks])
    first = int(np.argmax(values >= b))  # values is nondecreasing and ends at sum(hi) > b
    if first == 0:
        kappa = breaks[0]
    else:
        k0, k1 = breaks[first - 1], breaks[first]
        f0, f1 = values[first - 1], values[first]
        kappa = k0 + (b - f0) * (k1 - k0) / (f1 - f0)
    return np.clip(kappa * b * p, lo, hi)


def integer_budgets(shares, n_tokens, total_budget, bmin_frac=DEFAULT_BMIN_FRAC,
                    bmax_frac=DEFAULT_BMAX_FRAC):
    """Reading R17: floor, then the leftover units one each to the layers with
    the largest fractional part among those below hi_l, ties to lower l."""
    shares = np.asarray(shares, dtype=np.float64)
    _, hi = layer_bounds(n_tokens, total_budget, bmin_frac, bmax_frac)
    budgets = np.floor(shares).astype(np.int64)
    if hi.sum() <= total_budget:
        return hi.astype(np.int64)
    leftover = int(total_budget - budgets.sum())
    frac = shares - np.floor(shares)
    order = sorted((l for l in range(len(shares)) if budgets[l] < hi[l]),
                   key=lambda l: (-frac[l], l))
    if leftover < 0 or leftover > len(order):
        raise AssertionError("largest-remainder rounding out of range")
    for l in order[:leftover]:
        budgets[l] += 1
    return budgets


def split_budget(layer_budget, w_v, k_visual, k_audio):
    """Reading R18: M_v = floor(w_v B_l + 1/2) clamped to
    [max(0, B_l - K_a), min(K_v, B_l)]; M_a = B_l - M_v."""
    m_v = math.floor(w_v * layer_budget + 0.5)
    m_v = min(max(m_v, max(0, layer_budget - k_audio)), min(k_visual, layer_budget))
    return int(m_v), int(layer_budget - m_v)


# ---------------------------------------------------------------------------
# Offline budgets (end of Sec. 3.2): B^(l) fixed from a calibration set
# ---------------------------------------------------------------------------

def calibration_budgets(c_layer_steps, total_budget, temperature=DEFAULT_T,
                        bmin_frac=DEFAULT_BMIN_FRAC, bmax_frac=DEFAULT_BMAX_FRAC):
    """Per-layer budgets fixed in advance (reading R21).

    c_layer_steps: [steps, L] values of C^(l) (Eq. 13), one row per
    calibration step.  Their mean over the steps goes through Eq. (14) with
    the clamp to [B_min, B_max] (R15, R16) and the integer rounding (R17).
    Token counts of any one step do not cap these budgets, so the bounds are
    taken with counts large enough never to bind.
    """
    c = np.asarray(c_layer_steps, dtype=np.float64)
    if c.ndim != 2 or c.shape[0] == 0:
        raise ValueError("calibration needs at least one step of per-layer values")
    c_mean = c.mean(axis=0)
    never_binding = (math.floor(float(bmax_frac) * float(total_budget))
                     + math.ceil(float(bmin_frac) * float(total_budget)) + 1)
    n_free = [never_binding] * c.shape[1]
    shares = layer_shares(c_mean, n_free, total_budget, temperature, bmin_frac, bmax_frac)
    return integer_budgets(shares, n_free, total_budget, bmin_frac, bmax_frac)


def fixed_split(layer_budget, w_v, k_visual, k_audio):
    """One layer of a step under offline budgets (reading R21): it keeps
    min(B^(l), N_l) rows (a negative budget keeps none), split between the
    modalities by this step's w_v as in the online mode (R18)."""
    b = min(max(int(layer_budget), 0), int(k_visual) + int(k_audio))
    return split_budget(b, w_v, k_visual, k_audio)


# ---------------------------------------------------------------------------
# Eqs. (4), (5): Select, and the compaction into the next caches
# ---------------------------------------------------------------------------

def select(psi, modality, m_visual, m_audio):
    """Top-M_mu rows of each modality by psi (Sec. 3.1), per KV head.

    Reading R10: order by (psi descending, position ascending); reading R11:
    the kept rows are emitted in ascending position, visual block first.
    psi: [H_kv, N].  Returns int64 [H_kv, M_v + M_a].
    """
    modality = np.asarray(modality)
    rows = []
    for g in range(psi.shape[0]):
        kept = []
        for mu, m in ((VISUAL, m_visual), (AUDIO, m_audio)):
            pos = segment_positions(modality, mu)
            order = sorted(pos.tolist(), key=lambda p: (-psi[g, p], p))
            kept.append(np.sort(np.array(order[:m], dtype=np.int64)))
        rows.append(np.concatenate(kept))
    return np.stack(rows)


def layer_shared_select(a, s, modality, m_visual, m_audio, lam=DEFAULT_LAMBDA):
    """One index set per layer (reading R22): rows ranked by psi of the
    layer's importance sum_g a_g and redundancy mean_g s_g, top-M per
    modality as in select(); every KV head keeps those rows.
    a, s: [H_kv, N].  Returns int64 [H_kv, M_v + M_a] with identical rows.
    """
    a_layer = np.asarray(a, dtype=np.float64).sum(axis=0, keepdims=True)
    s_layer = np.asarray(s, dtype=np.float64).mean(axis=0, keepdims=True)
    idx = select(retention_score(a_layer, s_layer, lam), modality, m_visual, m_audio)
    return np.repeat(idx, np.asarray(a).shape[0], axis=0)


def compact(x, idx):
    """Next cache rows: x_out[g, i] = x[g, idx[g, i]]  ([H_kv, M, d])."""
    return np.stack([x[g, idx[g]] for g in range(x.shape[0])])


# ---------------------------------------------------------------------------
# One whole compression step over all layers
# ---------------------------------------------------------------------------

def compression_step(layers, total_budget, lam=DEFAULT_LAMBDA, r=DEFAULT_R,
                     temperature=DEFAULT_T, bmin_frac=DEFAULT_BMIN_FRAC,
                     bmax_frac=DEFAULT_BMAX_FRAC, mode="max", causal=True,
                     use_keys=False, layer_budgets=None, shared_selection=False,
                     use_hidden=False):
    """Run the whole step.  `layers` is a list of dicts with keys
    q [H_q,C,d], k and v [H_kv,N,d], modality [N], n_cache, sm_scale.
    With `layer_budgets` (offline budgets B^(l), reading R21) the layers
    keep those, capped at their token counts, instead of the budgets of
    Eq. (14) from this step.  With `shared_selection` every KV head of a
    layer keeps the same rows (reading R22).  With `use_hidden` the
    redundancy comes from each layer's hidden states `h` [N, d_model]
    (Eq. 7 as printed, reading R23; adjacent form) and the kept rows' hidden
    states are compacted too (out["h_out"]), which needs shared_selection.

    Returns a dict of per-layer lists: a, s, stats, budgets (M_v, M_a), idx,
    k_out, v_out, plus the real-valued shares x_l and integer B_l.
    """
    if use_hidden and not shared_selection:
        raise ValueError("hidden states are carried per token: they need shared_selection")
    out = {"a": [], "s": [], "stats": [], "idx": [], "k_out": [], "v_out": [],
           "budgets": [], "h_out": []}
    for layer in layers:
        a = attention_importance(layer["q"], layer["k"], layer["n_cache"],
                                 layer["sm_scale"], causal)
        if use_hidden:
            s = hidden_redundancy(layer["h"], layer["modality"], layer["k"].shape[0], mode)
        else:
            src = layer["k"] if use_keys else layer["v"]
            s = redundancy(src, layer["modality"], mode)
        out["a"].append(a)
        out["s"].append(s)
        out["stats"].append(avba_statistics(a, s, layer["modality"]))
    c_layers = [st["C_l"] for st in out["stats"]]
    n_tokens = [len(layer["modality"]) for layer in layers]
    if layer_budgets is None:
        shares = layer_shares(c_layers, n_tokens, total_budget, temperature,
                              bmin_frac, bmax_frac)
        budgets = integer_budgets(shares, n_tokens, total_budget, bmin_frac, bmax_frac)
    else:
        budgets = np.minimum(np.maximum(np.asarray(layer_budgets, dtype=np.int64), 0), n_tokens)
        shares = budgets.astype(np.float64)
    out["shares"] = shares
    out["layer_budgets"] = budgets
    for layer, st, b_l, a, s in zip(layers, out["stats"], budgets, out["a"], out["s"]):
        mod = np.asarray(layer["modality"])
        w_v, _ = modality_weights(st["C_v"], st["C_a"], r)
        st["w_v"] = w_v
        m_v, m_a = split_budget(int(b_l), w_v, int((mod == VISUAL).sum()),
                                int((mod == AUDIO).sum()))
        if shared_selection:
            idx = layer_shared_select(a, s, mod, m_v, m_a, lam)
        else:
            idx = select(retention_score(a, s, lam), mod, m_v, m_a)
        out["budgets"].append((m_v, m_a))
        out["idx"].append(idx)
        out["k_out"].append(compact(layer["k"], idx))
        if use_hidden:
            out["h_out"].append(np.asarray(layer["h"])[idx[0]])
        out["v_out"].append(compact(layer["v"], idx))
    return out
