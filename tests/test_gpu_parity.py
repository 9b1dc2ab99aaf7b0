"""Parity of the HIP path (through the C ABI) with the CPU oracle.

Each stage is checked on its own ("teacher-forced": the GPU stage gets the
oracle's inputs where a stage has inputs) and the whole chain free-running.
Small workloads are compared element by element; the full-size Qwen-7B
shaped layer (6144 tokens) likewise; the 28-layer and 40960-token workloads
on sampled queries/keys/rows the oracle computes one by one, plus
properties that hold at any size.
"""
import math

import numpy as np
import pytest
import torch

from oracle import omnimem_oracle as om
from paper_2606_07577_amd import omnimem, synth
from paper_2606_07577_amd.step import DeviceStep
from tests import parity as P

pytestmark = pytest.mark.gpu


def _sync():
    torch.cuda.synchronize()


class Case:
    """Run every stage of one workload on the GPU and keep host copies."""

    def __init__(self, layers, budget, **opts):
        self.layers = layers
        self.budget = budget
        self.opts = opts
        self.step = st = DeviceStep(layers, budget, **opts)
        st.score(lse_out=True)
        st.redundancy()
        st.allocate()
        st.select_compact()
        _sync()
        L = len(layers)
        self.lse = [st.host("lse", l) for l in range(L)]
        self.a = [st.host("a", l) for l in range(L)]
        self.s = [st.host("s", l) for l in range(L)]
        self.budgets = st.budgets.cpu().numpy().astype(np.int64)
        self.stats = st.stats.cpu().numpy()
        self.idx = [st.host("idx", l) for l in range(L)]
        self.k_out = [st.k_out[l].float().cpu().numpy() for l in range(L)]
        self.v_out = [st.v_out[l].float().cpu().numpy() for l in range(L)]
        self.layers64 = [P.as_f64(x) for x in layers]

    @property
    def causal(self):
        return bool(self.opts.get("causal", 1))

    @property
    def mode(self):
        return "adj" if self.opts.get("sim", omnimem.SIM_MAX) == omnimem.SIM_ADJ else "max"


def ragged_layers(n_layers=1, d=128, dtype="bf16", seed=100, caches=((200, 77),), frames=(3, 41, 13),
                  h_q=8, h_kv=2, hidden_dim=0):
    out = []
    for l in range(n_layers):
        cv, ca = caches[l % len(caches)]
        out.append(synth.make_layer([seed, l], h_q=h_q, h_kv=h_kv, d=d, n_cache_v=cv, n_cache_a=ca,
                                    n_frames=frames[0], frame_v=frames[1], frame_a=frames[2],
                                    dup_frac=0.3, head_scale=(0.5, 2.0), dtype=dtype,
                                    sm_scale=1.0 / ((0.5 + l) * math.sqrt(d)), hidden_dim=hidden_dim))
    return out


_cache = {}


def get_case(name):
    if name in _cache:
        return _cache[name]
    if name == "tiny-f32":
        case = Case(synth.make_workload("tiny-f32-640"), 256)
    elif name == "qwen-layer":
        case = Case(synth.make_workload("qwen7b-layer-6144"), 4096)
    elif name == "ragged-bf16":
        case = Case(ragged_layers(), 300)
    elif name == "ragged-bf16-d64":
        case = Case(ragged_layers(d=64, seed=101), 250)
    elif name == "ragged-3layer":
        case = Case(ragged_layers(3, seed=102, caches=((200, 77), (333, 111), (64, 17))), 3 * 260)
    elif name == "ragged-adj-noncausal":
        case = Case(ragged_layers(seed=103), 300, sim=omnimem.SIM_ADJ, causal=0)
    else:
        raise KeyError(name)
    _cache[name] = case
    return case


FULL_CASES = ["tiny-f32", "ragged-bf16", "ragged-bf16-d64", "ragged-3layer", "ragged-adj-noncausal",
              "qwen-layer"]


@pytest.mark.parametrize("name", FULL_CASES)
def test_lse_and_importance(name):
    c = get_case(name)
    for l, lay in enumerate(c.layers64):
        lse = om.attention_lse(lay["q"], lay["k"], lay["n_cache"], lay["sm_scale"], c.causal)
        P.assert_close_a(c.lse[l], lse, f"lse layer {l}")
        a = om.attention_importance(lay["q"], lay["k"], lay["n_cache"], lay["sm_scale"], c.causal, lse=lse)
        P.assert_close_a(c.a[l], a, f"a layer {l}")
        group = lay["q"].shape[0] // lay["k"].shape[0]
        np.testing.assert_allclose(c.a[l].sum(axis=1, dtype=np.float64), group * lay["q"].shape[1], rtol=1e-4)


@pytest.mark.parametrize("h_q,h_kv,causal", [(3, 3, 1), (6, 2, 1), (6, 2, 0)])
def test_importance_head_groups(h_q, h_kv, causal):
    # The column-sum pass sums over the G query heads of a KV head inside
    # one work row, the query head changing between streamed tiles (and
    # chunk boundaries falling inside a head's tiles): G = 1 and G = 3.
    layers = ragged_layers(seed=109, h_q=h_q, h_kv=h_kv, caches=((400, 130),), frames=(3, 90, 30))
    step = DeviceStep(layers, 300, causal=causal)
    step.score(lse_out=True)
    _sync()
    lay = P.as_f64(layers[0])
    lse = om.attention_lse(lay["q"], lay["k"], lay["n_cache"], lay["sm_scale"], bool(causal))
    P.assert_close_a(step.host("lse", 0), lse, "lse")
    a = om.attention_importance(lay["q"], lay["k"], lay["n_cache"], lay["sm_scale"], bool(causal), lse=lse)
    P.assert_close_a(step.host("a", 0), a, "a")
    step.close()


@pytest.mark.parametrize("name", FULL_CASES)
def test_redundancy(name):
    c = get_case(name)
    for l, lay in enumerate(c.layers64):
        s = om.redundancy(lay["v"], lay["modality"], c.mode)
        P.assert_close_s(c.s[l], s, f"s layer {l}")


@pytest.mark.parametrize("name", FULL_CASES)
def test_allocate_teacher_forced(name):
    # The GPU allocation from the oracle's own a and s (rounded to fp32, the
    # ABI's type) must give the oracle's integer budgets exactly.
    c = get_case(name)
    a_ref, s_ref = [], []
    for lay in c.layers64:
        a_ref.append(om.attention_importance(lay["q"], lay["k"], lay["n_cache"], lay["sm_scale"], c.causal)
                     .astype(np.float32))
        s_ref.append(om.redundancy(lay["v"], lay["modality"], c.mode).astype(np.float32))
    st = c.step
    a_dev, s_dev = st.to_device_f32(a_ref), st.to_device_f32(s_ref)
    budgets = torch.zeros_like(st.budgets)
    stats = torch.zeros_like(st.stats)
    st.ctx.omnimem_allocate(st.descs, a_dev, s_dev, c.budget, budgets, stats)
    _sync()
    ref_stats, shares, ref_budgets = P.oracle_allocation(
        [x.astype(np.float64) for x in a_ref], [x.astype(np.float64) for x in s_ref], c.layers, c.budget)
    np.testing.assert_array_equal(budgets.cpu().numpy(), ref_budgets)
    got = stats.cpu().numpy()
    for l, rs in enumerate(ref_stats):
        P.assert_close_a(got[l], [rs[k] for k in P.STAT_KEYS], f"stats layer {l}")
    total = sum(min(n, c.budget) for n in [len(x["modality"]) for x in c.layers])
    assert ref_budgets.sum() == min(c.budget, total)


@pytest.mark.parametrize("name", FULL_CASES)
def test_select_compact_teacher_forced(name):
    c = get_case(name)
    st = c.step
    L = len(c.layers)
    a_ref, s_ref = [], []
    for lay in c.layers64:
        a_ref.append(om.attention_importance(lay["q"], lay["k"], lay["n_cache"], lay["sm_scale"], c.causal)
                     .astype(np.float32))
        s_ref.append(om.redundancy(lay["v"], lay["modality"], c.mode).astype(np.float32))
    _, _, budgets = P.oracle_allocation([x.astype(np.float64) for x in a_ref],
                                        [x.astype(np.float64) for x in s_ref], c.layers, c.budget)
    st.ctx.omnimem_select_compact(st.descs, st.to_device_f32(a_ref), st.to_device_f32(s_ref),
                                  torch.from_numpy(budgets.astype(np.int32)).to(st.device), st.idx)
    _sync()
    for l in range(L):
        mv, ma = budgets[l]
        psi = om.retention_score(a_ref[l].astype(np.float64), s_ref[l].astype(np.float64), P.LAMBDA)
        idx = st.host("idx", l)[:, : mv + ma]
        for g in range(st.h_kv):
            P.check_selection(idx[g], psi[g], c.layers[l]["modality"], mv, ma)
        k_out = st.k_out[l].float().cpu().numpy()
        v_out = st.v_out[l].float().cpu().numpy()
        for g in range(st.h_kv):
            np.testing.assert_array_equal(k_out[g, : mv + ma], c.layers[l]["k"][g, idx[g]])
            np.testing.assert_array_equal(v_out[g, : mv + ma], c.layers[l]["v"][g, idx[g]])


@pytest.mark.parametrize("name", FULL_CASES)
def test_chain_free_running(name):
    # The GPU's own a, s -> budgets -> kept rows; budgets within the bounds
    # that the measured differences of the statistics imply, the kept rows a
    # valid top-M of the oracle's psi under the GPU's budgets, and the
    # compacted caches exactly the kept rows.
    c = get_case(name)
    a_o, s_o = [], []
    for lay in c.layers64:
        a_o.append(om.attention_importance(lay["q"], lay["k"], lay["n_cache"], lay["sm_scale"], c.causal))
        s_o.append(om.redundancy(lay["v"], lay["modality"], c.mode))
    ref_stats, shares, ref_budgets = P.oracle_allocation(a_o, s_o, c.layers, c.budget)
    assert c.budgets.sum() == ref_budgets.sum()
    bounds = P.free_running_budget_bounds(c.stats, ref_stats, shares, ref_budgets)
    print(f"{name}: budget differences {np.abs(c.budgets - ref_budgets).max()} within bounds up to {bounds.max()}")
    assert (np.abs(c.budgets - ref_budgets) <= bounds).all(), (c.budgets, ref_budgets, bounds)
    for l, lay in enumerate(c.layers):
        mv, ma = c.budgets[l]
        psi = om.retention_score(a_o[l], s_o[l], P.LAMBDA)
        for g in range(c.step.h_kv):
            row = c.idx[l][g, : mv + ma]
            P.check_selection(row, psi[g], lay["modality"], mv, ma, rel=5e-3)
            np.testing.assert_array_equal(c.k_out[l][g, : mv + ma], lay["k"][g, row])
            np.testing.assert_array_equal(c.v_out[l][g, : mv + ma], lay["v"][g, row])


def test_determinism_bitwise():
    c = get_case("ragged-3layer")
    st = c.step
    st.run()
    _sync()
    again = [st.host("a", l) for l in range(3)], [st.host("s", l) for l in range(3)]
    for l in range(3):
        np.testing.assert_array_equal(again[0][l], c.a[l])
        np.testing.assert_array_equal(again[1][l], c.s[l])
    np.testing.assert_array_equal(st.budgets.cpu().numpy(), c.budgets)
    for l in range(3):
        np.testing.assert_array_equal(st.host("idx", l), c.idx[l])


def test_caller_supplied_lse_matches_computed():
    c = get_case("ragged-bf16")
    layers = c.layers
    step = DeviceStep(layers, 300)
    lse = [torch.from_numpy(c.lse[0]).contiguous().cuda()]
    step.set_lse_inputs(lse)
    step.score(lse_out=True)
    _sync()
    np.testing.assert_array_equal(step.host("lse", 0), c.lse[0])  # passed through unchanged
    # the given lse is the computed one rounded to natural log: a agrees to a few ulp
    np.testing.assert_allclose(step.host("a", 0), c.a[0], rtol=2e-6, atol=0)
    step.close()


# ---------------------------------------------------------------------------
# Large workloads: sampled outputs and properties
# ---------------------------------------------------------------------------

def _chain_properties(c):
    """What the GPU's own chain must satisfy at any size: budgets that sum
    to the total and fit each modality, a kept set that is a top-M of the
    GPU's own psi per (layer, head, modality), and compacted rows equal to
    the kept input rows."""
    total = sum(len(lay["modality"]) for lay in c.layers)
    assert c.budgets.sum() == min(c.budget, total)
    for l, lay in enumerate(c.layers):
        mod = np.asarray(lay["modality"])
        mv, ma = c.budgets[l]
        assert 0 <= mv <= (mod == 0).sum() and 0 <= ma <= (mod == 1).sum()
        for g in range(c.step.h_kv):
            row = c.idx[l][g, : mv + ma]
            P.check_topk_property(row, c.a[l][g], c.s[l][g], mod, mv, ma)
            np.testing.assert_array_equal(c.k_out[l][g, : mv + ma], lay["k"][g, row])
            np.testing.assert_array_equal(c.v_out[l][g, : mv + ma], lay["v"][g, row])


def _teacher_forced_full_size(c, seed):
    """Allocation and selection at full size from generator-drawn a and s
    (the ABI lets a caller supply them): budgets exactly the oracle's,
    statistics within tolerance, kept rows the oracle's top-M."""
    st = c.step
    a_syn, s_syn = synth.make_scores([lay["modality"] for lay in c.layers], st.h_kv, seed)
    a_dev, s_dev = st.to_device_f32(a_syn), st.to_device_f32(s_syn)
    budgets = torch.zeros_like(st.budgets)
    stats = torch.zeros_like(st.stats)
    st.ctx.omnimem_allocate(st.descs, a_dev, s_dev, c.budget, budgets, stats)
    _sync()
    a64 = [x.astype(np.float64) for x in a_syn]
    s64 = [x.astype(np.float64) for x in s_syn]
    ref_stats, _, ref_budgets = P.oracle_allocation(a64, s64, c.layers, c.budget)
    np.testing.assert_array_equal(budgets.cpu().numpy(), ref_budgets)
    got = stats.cpu().numpy()
    for l, rs in enumerate(ref_stats):
        P.assert_close_a(got[l], [rs[k] for k in P.STAT_KEYS], f"stats layer {l}")
    st.ctx.omnimem_select_compact(st.descs, a_dev, s_dev, budgets, st.idx)
    _sync()
    for l, lay in enumerate(c.layers):
        mv, ma = ref_budgets[l]
        psi = om.retention_score(a64[l], s64[l], P.LAMBDA)
        idx = st.host("idx", l)[:, : mv + ma]
        k_out = st.k_out[l].float().cpu().numpy()
        for g in range(st.h_kv):
            P.check_selection(idx[g], psi[g], lay["modality"], mv, ma)
            np.testing.assert_array_equal(k_out[g, : mv + ma], lay["k"][g, idx[g]])


def _oracle_full(layers64, causal, mode, q_block=512, k_block=2048, s_block=4096):
    """The oracle's lse, a and s of every query, row and head of `layers64`,
    computed in blocks of queries, keys and rows as jobs on the host's cores
    (BLAS one thread per job): first every lse, then a (which needs the lse
    of all of a group's queries) and s.  Returns per layer
    (lse [H_q, C], a [H_kv, N], s [H_kv, N])."""
    import os
    from concurrent.futures import ThreadPoolExecutor
    from threadpoolctl import threadpool_limits

    def group_of(lay, g):
        group = lay["q"].shape[0] // lay["k"].shape[0]
        return lay["q"][g * group:(g + 1) * group], lay["k"][g:g + 1]

    def lse_job(l, g, q0):
        lay = layers64[l]
        q_g, k_g = group_of(lay, g)
        qs = np.arange(q0, min(q0 + q_block, q_g.shape[1]))
        return om.attention_lse(q_g, k_g, lay["n_cache"], lay["sm_scale"], causal, queries=qs)

    def a_job(l, g, k0, lse_g):
        lay = layers64[l]
        q_g, k_g = group_of(lay, g)
        ks = np.arange(k0, min(k0 + k_block, k_g.shape[1]))
        return om.attention_importance(q_g, k_g, lay["n_cache"], lay["sm_scale"], causal, lse=lse_g, keys=ks)[0]

    def s_job(l, g, r0):
        lay = layers64[l]
        rows = np.arange(r0, min(r0 + s_block, lay["v"].shape[1]))
        return om.redundancy(lay["v"][g:g + 1], lay["modality"], mode, rows=rows)[0]

    L = len(layers64)
    units = [(l, g) for l in range(L) for g in range(layers64[l]["k"].shape[0])]
    workers = max(1, min(16, os.cpu_count() or 1))
    with threadpool_limits(limits=1), ThreadPoolExecutor(max_workers=workers) as ex:
        lse_jobs = [(l, g, q0) for (l, g) in units for q0 in range(0, layers64[l]["q"].shape[1], q_block)]
        lse_parts = list(ex.map(lambda j: lse_job(*j), lse_jobs))
        lse = {}
        for (l, g, _), part in zip(lse_jobs, lse_parts):
            lse.setdefault((l, g), []).append(part)
        lse = {key: np.concatenate(v, axis=1) for key, v in lse.items()}
        a_jobs = [(l, g, k0) for (l, g) in units for k0 in range(0, layers64[l]["k"].shape[1], k_block)]
        s_jobs = [(l, g, r0) for (l, g) in units for r0 in range(0, layers64[l]["v"].shape[1], s_block)]
        a_fut = [ex.submit(a_job, l, g, k0, lse[(l, g)]) for (l, g, k0) in a_jobs]
        s_fut = [ex.submit(s_job, l, g, r0) for (l, g, r0) in s_jobs]
        a_parts = [f.result() for f in a_fut]
        s_parts = [f.result() for f in s_fut]
    out = []
    for l in range(L):
        h_kv = layers64[l]["k"].shape[0]
        lse_l = np.concatenate([lse[(l, g)] for g in range(h_kv)])
        a_l = np.stack([np.concatenate([p for (ll, g, _), p in zip(a_jobs, a_parts) if ll == l and g == gg])
                        for gg in range(h_kv)])
        s_l = np.stack([np.concatenate([p for (ll, g, _), p in zip(s_jobs, s_parts) if ll == l and g == gg])
                        for gg in range(h_kv)])
        out.append((lse_l, a_l, s_l))
    return out


def _full_size_checks(c):
    """Every query, row and KV head against the oracle (lse, a, s), then the
    GPU's own chain: budgets within the bounds the measured statistics imply
    and the kept rows a valid top-M of the oracle's psi."""
    ref = _oracle_full(c.layers64, True, "max")
    for l, (lse, a, s) in enumerate(ref):
        P.assert_close_a(c.lse[l], lse, f"lse layer {l}")
        P.assert_close_a(c.a[l], a, f"a layer {l}")
        P.assert_close_s(c.s[l], s, f"s layer {l}")
    a_o = [r[1] for r in ref]
    s_o = [r[2] for r in ref]
    ref_stats, shares, ref_budgets = P.oracle_allocation(a_o, s_o, c.layers, c.budget)
    assert c.budgets.sum() == ref_budgets.sum()
    bounds = P.free_running_budget_bounds(c.stats, ref_stats, shares, ref_budgets)
    print(f"budget differences {np.abs(c.budgets - ref_budgets).max()} within bounds up to {bounds.max()}")
    assert (np.abs(c.budgets - ref_budgets) <= bounds).all(), (c.budgets, ref_budgets, bounds)
    for l, lay in enumerate(c.layers):
        mv, ma = c.budgets[l]
        psi = om.retention_score(a_o[l], s_o[l], P.LAMBDA)
        for g in range(c.step.h_kv):
            P.check_selection(c.idx[l][g, : mv + ma], psi[g], lay["modality"], mv, ma, rel=5e-3)


@pytest.mark.timeout(900)
def test_28_layer_workload_full_size():
    layers = synth.make_workload("qwen7b-28layer-6144")
    c = Case(layers, 28 * 4096)
    _full_size_checks(c)
    _chain_properties(c)
    _teacher_forced_full_size(c, 11)
    c.step.close()


@pytest.mark.timeout(900)
def test_long_cache_workload_full_size():
    layers = synth.make_workload("qwen7b-longcache-40960")
    c = Case(layers, 32768)
    _full_size_checks(c)
    _chain_properties(c)
    _teacher_forced_full_size(c, 12)
    c.step.close()


# ---------------------------------------------------------------------------
# Layer-shared selection (Eqs. 4-5 carry no head index; reading R22)
# ---------------------------------------------------------------------------

@pytest.mark.parametrize("name", ["ragged-bf16", "ragged-3layer", "qwen-layer"])
def test_shared_selection_teacher_forced(name):
    # The oracle's a and s through the GPU's selection with one index set per
    # layer: every head keeps the same rows, a top-M of the oracle's layer
    # psi (ties within the fp32 rounding of the head sums), compacted.
    base = get_case(name)
    layers = base.layers
    st = DeviceStep(layers, base.budget, shared_selection=1)
    a_ref, s_ref = [], []
    for lay in base.layers64:
        a_ref.append(om.attention_importance(lay["q"], lay["k"], lay["n_cache"], lay["sm_scale"], True)
                     .astype(np.float32))
        s_ref.append(om.redundancy(lay["v"], lay["modality"], "max").astype(np.float32))
    _, _, budgets = P.oracle_allocation([x.astype(np.float64) for x in a_ref],
                                        [x.astype(np.float64) for x in s_ref], layers, base.budget)
    st.budgets.copy_(torch.from_numpy(budgets.astype(np.int32)))
    st.select_compact(a=st.to_device_f32(a_ref), s=st.to_device_f32(s_ref))
    _sync()
    for l, lay in enumerate(layers):
        mod = np.asarray(lay["modality"])
        mv, ma = (int(x) for x in budgets[l])
        idx = st.host("idx", l)[:, : mv + ma]
        assert (idx == idx[0]).all(), f"layer {l}: heads keep different rows"
        a64, s64 = a_ref[l].astype(np.float64), s_ref[l].astype(np.float64)
        psi = om.retention_score(a64.sum(axis=0), s64.mean(axis=0), P.LAMBDA)
        P.check_selection(idx[0], psi, mod, mv, ma, rel=1e-5)
        k_out = st.k_out[l].float().cpu().numpy()
        for g in range(st.h_kv):
            np.testing.assert_array_equal(k_out[g, : mv + ma], lay["k"][g, idx[0]])
    st.close()


def test_shared_selection_chain_and_one_head_equivalence():
    # The whole GPU step with shared selection keeps, per layer, a top-M of
    # the layer psi of its own a and s; with one KV head it is the per-head
    # step bit for bit.
    layers = ragged_layers(2, seed=112, caches=((300, 90), (120, 60)))
    st = DeviceStep(layers, 500, shared_selection=1)
    st.run()
    _sync()
    budgets = st.budgets.cpu().numpy()
    for l, lay in enumerate(layers):
        mod = np.asarray(lay["modality"])
        mv, ma = (int(x) for x in budgets[l])
        idx = st.host("idx", l)[:, : mv + ma]
        assert (idx == idx[0]).all()
        a64, s64 = st.host("a", l).astype(np.float64), st.host("s", l).astype(np.float64)
        P.check_topk_property(idx[0], a64.sum(axis=0), s64.mean(axis=0), mod, mv, ma)
    st.close()
    one = ragged_layers(1, seed=113, h_q=4, h_kv=1)
    per_head, shared = DeviceStep(one, 200), DeviceStep(one, 200, shared_selection=1)
    for x in (per_head, shared):
        x.run()
    _sync()
    np.testing.assert_array_equal(per_head.idx.cpu().numpy(), shared.idx.cpu().numpy())
    np.testing.assert_array_equal(per_head.k_out[0].view(torch.int16).cpu().numpy(),
                                  shared.k_out[0].view(torch.int16).cpu().numpy())
    per_head.close()
    shared.close()


# ---------------------------------------------------------------------------
# Redundancy from hidden states (Eq. 7 as printed; reading R23)
# ---------------------------------------------------------------------------

def _hidden_step(layers, budget, dh, sim=omnimem.SIM_ADJ):
    return DeviceStep(layers, budget, sim=sim, sim_source=omnimem.SRC_HIDDEN, hidden_dim=dh, shared_selection=1)


@pytest.mark.parametrize("dtype,dh,mode", [("bf16", 3584, "adj"), ("f32", 200, "adj"),
                                           ("bf16", 3584, "max"), ("f32", 192, "max")])
def test_hidden_state_redundancy(dtype, dh, mode):
    # One value per token from its hidden state, in every KV head's row;
    # 'max' spans several row blocks per segment (256 rows for bf16, 128 for
    # fp32: pairs on and off the diagonal, a ragged last block).
    layers = ragged_layers(2, dtype=dtype, seed=114, caches=((200, 77), (90, 31)), hidden_dim=dh)
    st = _hidden_step(layers, 300, dh, omnimem.SIM_ADJ if mode == "adj" else omnimem.SIM_MAX)
    st.redundancy()
    _sync()
    for l, lay in enumerate(layers):
        ref = om.hidden_redundancy(lay["h"].astype(np.float64), lay["modality"], st.h_kv, mode)
        P.assert_close_s(st.host("s", l), ref, f"s layer {l}")
    st.close()


@pytest.mark.parametrize("mode", ["adj", "max"])
@pytest.mark.parametrize("cache_v", [128, 256])
def test_hidden_state_small_segments(mode, cache_v):
    # A visual segment of cache_v + 1 rows (a last block of one row for the
    # all-pairs kernel's 128- and 256-row blocks) and a lone audio row (no
    # partner: s = 0), next to a layer of two rows per modality.
    layers = (ragged_layers(1, seed=117, caches=((cache_v, 1),), frames=(1, 1, 0), hidden_dim=256)
              + ragged_layers(1, seed=118, caches=((1, 1),), frames=(1, 1, 1), hidden_dim=256))
    st = _hidden_step(layers, 100, 256, omnimem.SIM_ADJ if mode == "adj" else omnimem.SIM_MAX)
    st.redundancy()
    _sync()
    for l, lay in enumerate(layers):
        ref = om.hidden_redundancy(lay["h"].astype(np.float64), lay["modality"], st.h_kv, mode)
        P.assert_close_s(st.host("s", l), ref, f"s layer {l}")
    assert (st.host("s", 0)[:, np.asarray(layers[0]["modality"]) == 1] == 0).all()
    st.close()


def test_hidden_state_step_carries_kept_rows():
    # The whole step with hidden states: shared kept rows, the hidden states
    # of exactly those rows compacted bit for bit, K and V too.
    layers = ragged_layers(2, seed=115, caches=((300, 90), (120, 60)), hidden_dim=1024)
    st = _hidden_step(layers, 500, 1024)
    st.run()
    _sync()
    budgets = st.budgets.cpu().numpy()
    for l, lay in enumerate(layers):
        mod = np.asarray(lay["modality"])
        mv, ma = (int(x) for x in budgets[l])
        idx = st.host("idx", l)[:, : mv + ma]
        s = st.host("s", l)
        assert (idx == idx[0]).all() and (s == s[0]).all()
        a64 = st.host("a", l).astype(np.float64)
        P.check_topk_property(idx[0], a64.sum(axis=0), s[0].astype(np.float64), mod, mv, ma)
        h_out = st.h_out[l][: mv + ma].view(torch.int16).cpu().numpy()
        h_in = st.h[l].view(torch.int16).cpu().numpy()
        np.testing.assert_array_equal(h_out, h_in[idx[0]])
        k_out = st.k_out[l].float().cpu().numpy()
        for g in range(st.h_kv):
            np.testing.assert_array_equal(k_out[g, : mv + ma], lay["k"][g, idx[0]])
    st.close()


@pytest.mark.parametrize("mode", ["adj", "max"])
def test_hidden_state_workload_full_size(mode):
    layers = synth.make_workload("qwen7b-layer-6144-hidden")
    st = _hidden_step(layers, 4096, 3584, omnimem.SIM_ADJ if mode == "adj" else omnimem.SIM_MAX)
    st.run()
    _sync()
    lay = layers[0]
    ref = om.hidden_redundancy(lay["h"].astype(np.float64), lay["modality"], st.h_kv, mode)
    P.assert_close_s(st.host("s", 0), ref, "s")
    mv, ma = (int(x) for x in st.budgets.cpu().numpy()[0])
    assert mv + ma == 4096
    idx = st.host("idx", 0)[:, :4096]
    np.testing.assert_array_equal(st.h_out[0][:4096].view(torch.int16).cpu().numpy(),
                                  st.h[0].view(torch.int16).cpu().numpy()[idx[0]])
    st.close()


def test_hidden_state_errors():
    layers = ragged_layers(seed=116, hidden_dim=512)
    with pytest.raises(omnimem.OmnimemError) as e:   # all pairs on hidden states: d_model in multiples of 64
        DeviceStep(layers, 300, sim=omnimem.SIM_MAX, sim_source=omnimem.SRC_HIDDEN, hidden_dim=520)
    assert e.value.status == omnimem.ERR_UNSUPPORTED
    with pytest.raises(omnimem.OmnimemError) as e:
        DeviceStep(layers, 300, sim=omnimem.SIM_ADJ, sim_source=omnimem.SRC_HIDDEN, hidden_dim=100)  # 200 B rows
    assert e.value.status == omnimem.ERR_INVALID_ARG
    st = DeviceStep(layers, 300, sim=omnimem.SIM_ADJ, sim_source=omnimem.SRC_HIDDEN, hidden_dim=512)
    st.redundancy()
    st.allocate()
    with pytest.raises(omnimem.OmnimemError) as e:   # kept hidden states need one index set per layer
        st.select_compact()
    assert e.value.status == omnimem.ERR_INVALID_ARG
    st.close()


# ---------------------------------------------------------------------------
# Offline budgets (end of Sec. 3.2; reading R21)
# ---------------------------------------------------------------------------

def _calib_layers():
    # five layers of different sizes; the smallest has fewer rows (243) than
    # the calibrated budgets can reach, so the cap of a fixed step is met
    return ragged_layers(5, seed=110, caches=((200, 77), (333, 111), (64, 17), (500, 40), (150, 150)))


def test_offline_budgets_teacher_forced():
    # Calibration over four steps of generator-drawn a and s, then two steps
    # under the fixed layer budgets: layer budgets and (M_v, M_a) exactly
    # the oracle's, each step's statistics within tolerance.
    layers = _calib_layers()
    total = 5 * 200
    st = DeviceStep(layers, total)
    mods = [lay["modality"] for lay in layers]
    st.ctx.omnimem_calibration_reset()
    c_steps = []
    for seed in range(4):
        a_syn, s_syn = synth.make_scores(mods, st.h_kv, 500 + seed)
        stats = torch.zeros_like(st.stats)
        st.ctx.omnimem_calibrate(st.descs, st.to_device_f32(a_syn), st.to_device_f32(s_syn), stats)
        _sync()
        ref = [om.avba_statistics(a.astype(np.float64), s.astype(np.float64), m)
               for a, s, m in zip(a_syn, s_syn, mods)]
        got = stats.cpu().numpy()
        for l, rs in enumerate(ref):
            w_v, _ = om.modality_weights(rs["C_v"], rs["C_a"], P.RATIO)
            rs["w_v"] = w_v
            P.assert_close_a(got[l], [rs[k] for k in P.STAT_KEYS], f"calibration step {seed} stats layer {l}")
        c_steps.append([rs["C_l"] for rs in ref])
    st.calibration_budgets()
    _sync()
    ref_lb = om.calibration_budgets(c_steps, total, P.TEMPERATURE)
    got_lb = st.layer_budgets.cpu().numpy()
    np.testing.assert_array_equal(got_lb, ref_lb)
    for seed in (600, 601):
        a_syn, s_syn = synth.make_scores(mods, st.h_kv, seed)
        budgets = torch.zeros_like(st.budgets)
        st.ctx.omnimem_allocate_fixed(st.descs, st.to_device_f32(a_syn), st.to_device_f32(s_syn),
                                      st.layer_budgets, budgets)
        _sync()
        want = []
        for a, s, m, b in zip(a_syn, s_syn, mods, ref_lb):
            rs = om.avba_statistics(a.astype(np.float64), s.astype(np.float64), m)
            w_v, _ = om.modality_weights(rs["C_v"], rs["C_a"], P.RATIO)
            want.append(om.fixed_split(int(b), w_v, int((m == 0).sum()), int((m == 1).sum())))
        np.testing.assert_array_equal(budgets.cpu().numpy(), np.array(want))
    # a reset and a single step: the budgets of that step's values alone
    st.ctx.omnimem_calibration_reset()
    a_syn, s_syn = synth.make_scores(mods, st.h_kv, 700)
    st.ctx.omnimem_calibrate(st.descs, st.to_device_f32(a_syn), st.to_device_f32(s_syn))
    st.calibration_budgets()
    _sync()
    one = [om.avba_statistics(a.astype(np.float64), s.astype(np.float64), m)["C_l"]
           for a, s, m in zip(a_syn, s_syn, mods)]
    np.testing.assert_array_equal(st.layer_budgets.cpu().numpy(), om.calibration_budgets([one], total,
                                                                                           P.TEMPERATURE))
    st.close()


def test_step_under_fixed_budgets_end_to_end():
    # The whole GPU step with the layer budgets fixed: each layer keeps
    # min(B_l, N_l) rows, a valid top-M of the GPU's own psi, compacted.
    layers = _calib_layers()
    st = DeviceStep(layers, 1000)
    lb = np.array([150, 400, 10**6, 0, 231], dtype=np.int32)
    st.layer_budgets.copy_(torch.from_numpy(lb))
    st.fixed_budgets = True
    st.run()
    _sync()
    budgets = st.budgets.cpu().numpy()
    for l, lay in enumerate(layers):
        mod = np.asarray(lay["modality"])
        mv, ma = budgets[l]
        assert mv + ma == min(lb[l], len(mod))
        assert 0 <= mv <= (mod == 0).sum() and 0 <= ma <= (mod == 1).sum()
        a, s, idx = st.host("a", l), st.host("s", l), st.host("idx", l)
        k_out = st.k_out[l].float().cpu().numpy()
        for g in range(st.h_kv):
            row = idx[g, : mv + ma]
            P.check_topk_property(row, a[g], s[g], mod, mv, ma)
            np.testing.assert_array_equal(k_out[g, : mv + ma], lay["k"][g, row])
    st.close()


def test_offline_budgets_errors():
    layers = ragged_layers(seed=111)
    st = DeviceStep(layers, 300)
    st.ctx.omnimem_calibration_reset()
    with pytest.raises(omnimem.OmnimemError) as e:
        st.calibration_budgets()            # no calibration step yet
    assert e.value.status == omnimem.ERR_INVALID_ARG
    with pytest.raises(omnimem.OmnimemError) as e:
        st.ctx.omnimem_allocate_fixed(st.descs, st.a, st.s, None, st.budgets)
    assert e.value.status == omnimem.ERR_INVALID_ARG
    st.close()


# ---------------------------------------------------------------------------
# Degenerate cases and argument validation
# ---------------------------------------------------------------------------

def _mixed_layers():
    """Layers of very different shapes in one call: a long chunk, a cache
    with a one-row chunk, a chunk without cache, a lone audio row, and a
    layer larger than the others (different row counts per work plan)."""
    shapes = [((300, 90), (2, 101, 37)), ((700, 260), (1, 1, 0)), ((0, 0), (3, 64, 21)),
              ((130, 1), (1, 33, 0)), ((1500, 500), (4, 120, 40))]
    out = []
    for l, ((cv, ca), frames) in enumerate(shapes):
        out.append(synth.make_layer([107, l], h_q=8, h_kv=2, d=128, n_cache_v=cv, n_cache_a=ca,
                                    n_frames=frames[0], frame_v=frames[1], frame_a=frames[2],
                                    dup_frac=0.3, head_scale=(0.5, 2.0), dtype="bf16",
                                    sm_scale=1.0 / ((0.7 + 0.4 * l) * math.sqrt(128))))
    return out


def test_mixed_layer_shapes_in_one_call():
    # Every stage on layers whose sizes differ widely, so the score-pass and
    # Gram plans split rows across workgroups, mix layers in one chunk and
    # meet one-row chunks, cache-free layers and a lone audio row.
    layers = _mixed_layers()
    budget = sum(len(x["modality"]) for x in layers) // 3
    c = Case(layers, budget)
    for l, lay in enumerate(c.layers64):
        lse = om.attention_lse(lay["q"], lay["k"], lay["n_cache"], lay["sm_scale"], True)
        P.assert_close_a(c.lse[l], lse, f"lse layer {l}")
        a = om.attention_importance(lay["q"], lay["k"], lay["n_cache"], lay["sm_scale"], True, lse=lse)
        P.assert_close_a(c.a[l], a, f"a layer {l}")
        P.assert_close_s(c.s[l], om.redundancy(lay["v"], lay["modality"], "max"), f"s layer {l}")
    _chain_properties(c)
    c.step.close()


def test_mixed_shapes_with_caller_lse_on_some_layers():
    # Layers with a caller-supplied lse drop out of the LSE pass's plan; the
    # others must be unaffected.
    layers = _mixed_layers()
    lay64 = [P.as_f64(x) for x in layers]
    ref_lse = [om.attention_lse(x["q"], x["k"], x["n_cache"], x["sm_scale"], True) for x in lay64]
    step = DeviceStep(layers, 1000)
    given = [torch.from_numpy(ref_lse[l].astype(np.float32)).contiguous().cuda() if l in (1, 3) else None
             for l in range(len(layers))]
    step.set_lse_inputs(given)
    step.score(lse_out=True)
    _sync()
    for l, lay in enumerate(lay64):
        P.assert_close_a(step.host("lse", l), ref_lse[l], f"lse layer {l}")
        a = om.attention_importance(lay["q"], lay["k"], lay["n_cache"], lay["sm_scale"], True, lse=ref_lse[l])
        P.assert_close_a(step.host("a", l), a, f"a layer {l}")
    step.close()


def test_fp32_head_dim_128():
    # fp32 inputs at d = 128 (the widest register footprint of the Gram pass).
    layers = [synth.make_layer([108, 0], h_q=4, h_kv=2, d=128, n_cache_v=150, n_cache_a=50, n_frames=2,
                               frame_v=40, frame_a=10, dup_frac=0.3, dtype="f32")]
    c = Case(layers, 120)
    lay = c.layers64[0]
    lse = om.attention_lse(lay["q"], lay["k"], lay["n_cache"], lay["sm_scale"], True)
    P.assert_close_a(c.a[0], om.attention_importance(lay["q"], lay["k"], lay["n_cache"], lay["sm_scale"], True,
                                                     lse=lse))
    P.assert_close_s(c.s[0], om.redundancy(lay["v"], lay["modality"], "max"))
    _chain_properties(c)
    c.step.close()


def test_visual_only_layer_and_budget_beyond_tokens():
    layers = ragged_layers(seed=104, caches=((150, 0),), frames=(2, 30, 0))
    c = Case(layers, 1000)   # more budget than the 210 rows: keep everything
    assert c.budgets.tolist() == [[210, 0]]
    np.testing.assert_array_equal(c.idx[0][:, :210], np.tile(np.arange(210), (2, 1)))
    lay = c.layers64[0]
    P.assert_close_s(c.s[0], om.redundancy(lay["v"], lay["modality"], "max"))
    c.step.close()


def test_exact_duplicates_and_zero_rows():
    layers = ragged_layers(seed=105)
    lay = layers[0]
    lay["v"][:, 5] = lay["v"][:, 9]        # exact twins
    lay["v"][:, 11] = 0.0                  # zero vector: cosine 0 with everything
    c = Case(layers, 300)
    assert (c.s[0][:, [5, 9]] == 1.0).all()
    P.assert_close_s(c.s[0], om.redundancy(P.as_f64(lay)["v"], lay["modality"], "max"))
    c.step.close()


def test_validation_errors():
    layers = ragged_layers(seed=106)
    st = DeviceStep(layers, 300)
    with pytest.raises(omnimem.OmnimemError) as e:
        st.ctx.omnimem_allocate(st.descs, st.a, st.s, -1, st.budgets)
    assert e.value.status == omnimem.ERR_INVALID_ARG
    with pytest.raises(omnimem.OmnimemError) as e:
        omnimem.Context(1, 8, 3, 128, 1024, 512)
    assert e.value.status == omnimem.ERR_INVALID_ARG
    with pytest.raises(omnimem.OmnimemError) as e:
        omnimem.Context(1, 8, 2, 96, 1024, 512)
    assert e.value.status == omnimem.ERR_UNSUPPORTED
    small = omnimem.Context(1, 8, 2, 128, 100, 50)
    with pytest.raises(omnimem.OmnimemError) as e:
        small.omnimem_score(st.descs, st.a)
    assert e.value.status == omnimem.ERR_CAPACITY
    small.close()
    bad = omnimem.make_layer(st.q[0], st.k[0], st.v[0], st.mod[0], st.n_cache[0], 0.0, None,
                             st.k[0], st.v_out[0])  # output aliases the input
    with pytest.raises(omnimem.OmnimemError) as e:
        st.ctx.omnimem_select_compact([bad], st.a, st.s, st.budgets, st.idx)
    assert e.value.status == omnimem.ERR_INVALID_ARG
    tight = omnimem.Context(1, 8, 2, 128, st.max_tokens, st.max_chunk, b_min_frac=1.5, b_max_frac=2.0)
    with pytest.raises(omnimem.OmnimemError) as e:
        tight.omnimem_allocate(st.descs, st.a, st.s, 100, st.budgets)
    assert e.value.status == omnimem.ERR_INFEASIBLE
    tight.close()
    st.close()


# ---------------------------------------------------------------------------
# The LSE pass's redo path and redundancy on key vectors
# ---------------------------------------------------------------------------

@pytest.mark.parametrize("d", [128, 64])
def test_lse_redo_when_later_keys_dominate(d):
    # The bf16 LSE pass takes each query's exponent reference from the first
    # 32 keys of its key range and redoes a range whose sums leave the fp32
    # headroom.  Keys 1000 times larger than the rest, at offsets 40..47 of
    # every 64-key tile (never among the first 32 keys of a range), give
    # later scores far above that reference; lse and a (Eq. 6) must still
    # match the oracle.
    layers = ragged_layers(seed=110, d=d, caches=((300, 100),), frames=(3, 70, 20))
    lay = layers[0]
    n = lay["k"].shape[1]
    planted = np.flatnonzero((np.arange(n) % 64 >= 40) & (np.arange(n) % 64 < 48))
    lay["k"][:, planted] = synth.round_to_bf16(lay["k"][:, planted] * 1000.0)
    step = DeviceStep(layers, 300)
    step.score(lse_out=True)
    _sync()
    x = P.as_f64(lay)
    lse = om.attention_lse(x["q"], x["k"], x["n_cache"], x["sm_scale"], True)
    # the planted keys lift lse far above what the first 32 keys give (ln 2^100 = 69.3)
    import scipy.special
    group = x["q"].shape[0] // x["k"].shape[0]
    first = np.stack([scipy.special.logsumexp(x["sm_scale"] * x["q"][h] @ x["k"][h // group, :32].T, axis=1)
                      for h in range(x["q"].shape[0])])
    assert (lse - first > 80).mean() > 0.5
    P.assert_close_a(step.host("lse", 0), lse, "lse")
    a = om.attention_importance(x["q"], x["k"], x["n_cache"], x["sm_scale"], True, lse=lse)
    P.assert_close_a(step.host("a", 0), a, "a")
    assert np.isfinite(step.host("a", 0)).all()
    step.close()


@pytest.mark.parametrize("sim", [omnimem.SIM_MAX, omnimem.SIM_ADJ])
def test_redundancy_on_keys(sim):
    # Eq. (7) on the key vectors (Sec. 3.1 allows the cache's own vectors):
    # s from k instead of v, then the whole step against the oracle's step
    # run on keys.
    mode = "max" if sim == omnimem.SIM_MAX else "adj"
    layers = ragged_layers(2, seed=111, caches=((200, 77), (150, 60)))
    c = Case(layers, 2 * 250, sim=sim, sim_source=omnimem.SRC_KEYS)
    ref = om.compression_step(c.layers64, c.budget, lam=P.LAMBDA, temperature=P.TEMPERATURE, r=P.RATIO,
                              mode=mode, use_keys=True)
    for l, lay in enumerate(c.layers64):
        P.assert_close_s(c.s[l], om.redundancy(lay["k"], lay["modality"], mode), f"s on keys, layer {l}")
        assert not np.allclose(c.s[l], om.redundancy(lay["v"], lay["modality"], mode), atol=1e-3)
    assert c.budgets.sum() == np.array(ref["budgets"]).sum()
    assert np.abs(c.budgets - np.array(ref["budgets"])).max() <= 1
    for l, lay in enumerate(c.layers):
        mv, ma = c.budgets[l]
        psi = om.retention_score(ref["a"][l], ref["s"][l], P.LAMBDA)
        for g in range(c.step.h_kv):
            row = c.idx[l][g, : mv + ma]
            P.check_selection(row, psi[g], lay["modality"], mv, ma, rel=5e-3)
            np.testing.assert_array_equal(c.k_out[l][g, : mv + ma], lay["k"][g, row])
    c.step.close()


def test_redundancy_on_keys_full_size():
    layers = synth.make_workload("qwen7b-layer-6144")
    step = DeviceStep(layers, 4096, sim_source=omnimem.SRC_KEYS)
    step.redundancy()
    _sync()
    lay = P.as_f64(layers[0])
    rows = np.sort(np.random.default_rng(5).choice(lay["k"].shape[1], size=128, replace=False))
    P.assert_close_s(step.host("s", 0)[:, rows], om.redundancy(lay["k"], lay["modality"], "max", rows=rows),
                     "s on keys (sampled rows)")
    step.close()
