"""The three ranking paths of the selection (Eqs. 4, 5 and 8) against each
other and against the oracle's top-M, through the C ABI: one workgroup per
(layer, KV head, modality) with keys in LDS (psi_topk), the same with every
key in registers for working sets of at most 8192 rows (psi_topk_reg), and
several workgroups per (layer, KV head) (topk_hist, topk_bin, topk_emit).

All paths must keep exactly the same rows (the top M of each modality by
the fp32 psi key, ties to the lower row), so idx and the compacted K/V must
agree bit for bit; the kept rows are also checked against the oracle's psi.
Inputs: the synthetic a, s of the selection stage on small ragged layers
(one slice), a 6144-token layer (three slices) and a 20001-token layer (ten
slices, the last ragged; the register path does not take it and falls back
to one workgroup), plus a, s built to stress the ranking: psi quantised to
a few values (ties across slices), one psi for every row (the threshold
bin's candidates exceed what LDS holds), and zero and NaN scores; budgets
of 0, 1, all rows, beyond the rows and beyond the output capacity;
layer-shared selection and compaction in place.  With the "half" budgets
most segments of the 6144-token and ragged layers end the register path's
select by ranking a threshold bin of at most 256 keys directly, with equal
keys among them in the quantised case.
"""
import numpy as np
import pytest
import torch

from oracle import omnimem_oracle as om
from paper_2606_07577_amd import omnimem, synth
from paper_2606_07577_amd.step import DeviceStep
from tests import parity as P
from tests.test_gpu_inplace import _compare
from tests.test_gpu_parity import ragged_layers

pytestmark = pytest.mark.gpu

PATHS = (omnimem.TOPK_ONE_WORKGROUP, omnimem.TOPK_REGISTERS, omnimem.TOPK_SPLIT)
ONE, REG, SPLIT = PATHS


def _long_layer(seed=500, n_cache_v=12000, n_cache_a=4001, frames=(4, 900, 100), h_kv=2):
    return [synth.make_layer([seed], h_q=4, h_kv=h_kv, d=128, n_cache_v=n_cache_v, n_cache_a=n_cache_a,
                             n_frames=frames[0], frame_v=frames[1], frame_a=frames[2], dtype="bf16")]


def _workload(name):
    if name == "ragged-3layer":
        return ragged_layers(3, seed=102, caches=((200, 77), (333, 111), (64, 17)))
    if name == "qwen-layer":
        return synth.make_workload("qwen7b-layer-6144")
    if name == "long-20001":
        return _long_layer()
    raise KeyError(name)


def _scores(layers, h_kv, kind, seed=7):
    mods = [l["modality"] for l in layers]
    a, s = synth.make_scores(mods, h_kv, seed)
    rng = np.random.default_rng([seed, 99])
    if kind == "ties":         # a few psi values, each shared by rows all over the working set
        a = [np.float32(2.0) ** rng.integers(-3, 3, size=x.shape).astype(np.float32) for x in a]
        s = [rng.choice(np.float32([0.0, 0.25, 0.5]), size=x.shape) for x in s]
    elif kind == "constant":   # every row the same psi
        a = [np.ones_like(x) for x in a]
        s = [np.zeros_like(x) for x in s]
    elif kind == "zeros-nans":
        for x in a:
            x[:, rng.random(x.shape[1]) < 0.2] = 0.0
            x[:, rng.random(x.shape[1]) < 0.01] = np.nan
        for x in s:
            x[:, rng.random(x.shape[1]) < 0.01] = np.nan
    return [x.astype(np.float32) for x in a], [x.astype(np.float32) for x in s]


def _applied(budget, mod, cap):
    """Budgets as the library applies them."""
    kv, ka = int((mod == 0).sum()), int((mod == 1).sum())
    mv = min(max(budget[0], 0), kv, cap)
    ma = min(max(budget[1], 0), ka, cap - mv)
    return mv, ma


def _budgets(layers, which):
    out = []
    for l in layers:
        kv, ka = int((l["modality"] == 0).sum()), int((l["modality"] == 1).sum())
        out.append({"half": (kv // 2, ka // 3), "one": (1, 1), "zero": (0, 0), "all": (kv, ka),
                    "beyond": (kv + 5, ka + 9), "mixed": (kv - 1, 0)}[which])
    return out


def _run(step, a, s, budgets, path):
    step.ctx.omnimem_set_topk_path(path)
    for t in step.k_out + step.v_out:
        t.zero_()
    step.idx.fill_(-1)
    step.select_compact(a=a, s=s, budgets=torch.tensor(budgets, dtype=torch.int32, device=step.device))
    torch.cuda.synchronize()
    return (step.idx.clone(), [t.clone() for t in step.k_out], [t.clone() for t in step.v_out])


def _check(step, layers, a_h, s_h, budgets, shared=False):
    a, s = step.to_device_f32(a_h), step.to_device_f32(s_h)
    one = _run(step, a, s, budgets, ONE)
    others = [_run(step, a, s, budgets, path) for path in (REG, SPLIT)]
    split = others[1]
    for l, lay in enumerate(layers):
        n = len(lay["modality"])
        mv, ma = _applied(budgets[l], lay["modality"], n)
        m = mv + ma
        for path, res in zip((REG, SPLIT), others):
            assert torch.equal(one[0][l, :, :m], res[0][l, :, :m]), f"path {path}, layer {l}: kept rows differ"
            assert torch.equal(one[1][l][:, :m], res[1][l][:, :m]) and torch.equal(one[2][l][:, :m], res[2][l][:, :m])
        a64 = np.asarray(a_h[l], dtype=np.float64)
        s64 = np.asarray(s_h[l], dtype=np.float64)
        if shared:   # one ranking per layer: a summed over the heads, s averaged (fp32, head order)
            a64 = np.asarray(np.sum(np.asarray(a_h[l], np.float32), axis=0, dtype=np.float32), np.float64)[None]
            s64 = np.asarray(np.sum(np.asarray(s_h[l], np.float32), axis=0, dtype=np.float32)
                             / np.float32(step.h_kv), np.float64)[None]
        # the library's key: s clamped to [-1, 1] (a NaN s clamps to -1), a NaN a ranks as 0
        s64 = np.clip(np.nan_to_num(s64, nan=-1.0), -1.0, 1.0)
        psi = om.retention_score(np.nan_to_num(a64, nan=0.0), s64, P.LAMBDA)
        idx = split[0][l].cpu().numpy()
        for g in range(step.h_kv):
            P.check_selection(idx[g, :m], psi[0 if shared else g], lay["modality"], mv, ma)
    return one, split


@pytest.mark.parametrize("name", ["ragged-3layer", "qwen-layer", "long-20001"])
@pytest.mark.parametrize("kind", ["synthetic", "ties", "constant", "zeros-nans"])
def test_paths_keep_the_same_rows(name, kind):
    layers = _workload(name)
    h_kv = layers[0]["k"].shape[0]
    step = DeviceStep(layers, 1000)
    a_h, s_h = _scores(layers, h_kv, kind)
    for which in ("half", "one", "zero", "all", "beyond", "mixed"):
        print(f"{name} {kind} budgets {which}", flush=True)
        _check(step, layers, a_h, s_h, _budgets(layers, which))
    step.close()


def test_paths_output_capacity():
    layers = _workload("qwen-layer")
    n = len(layers[0]["modality"])
    cap = 2500
    step = DeviceStep(layers, 1000)
    k_small = torch.zeros((step.h_kv, cap, step.d), device=step.device, dtype=step.tdtype)
    v_small = torch.zeros_like(k_small)
    a_h, s_h = _scores(layers, step.h_kv, "synthetic")
    a, s = step.to_device_f32(a_h), step.to_device_f32(s_h)
    desc = [omnimem.make_layer(step.q[0], step.k[0], step.v[0], step.mod[0], step.n_cache[0], step.sm_scale[0],
                               None, k_small, v_small, out_rows=cap)]
    bud = torch.tensor([(2000, 1500)], dtype=torch.int32, device=step.device)
    res = []
    for path in PATHS:
        step.ctx.omnimem_set_topk_path(path)
        step.idx.fill_(-1)
        k_small.zero_()
        v_small.zero_()
        step.ctx.omnimem_select_compact(desc, a, s, bud, step.idx)
        torch.cuda.synchronize()
        res.append((step.idx.clone(), k_small.clone(), v_small.clone()))
    mv, ma = _applied((2000, 1500), layers[0]["modality"], cap)
    assert (mv, ma) == (2000, 500) and n > cap
    for r in res[1:]:
        assert torch.equal(res[0][0][0, :, :cap], r[0][0, :, :cap])
        assert torch.equal(res[0][1], r[1]) and torch.equal(res[0][2], r[2])
    step.close()


@pytest.mark.parametrize("kind", ["synthetic", "ties"])
def test_paths_shared_selection(kind):
    layers = _workload("long-20001") if kind == "synthetic" else _workload("ragged-3layer")
    step = DeviceStep(layers, 1000, shared_selection=1)
    a_h, s_h = _scores(layers, step.h_kv, kind)
    for which in ("half", "all", "one"):
        one, _ = _check(step, layers, a_h, s_h, _budgets(layers, which), shared=True)
        for l in range(len(layers)):   # every head keeps the same rows
            assert torch.equal(one[0][l, 0], one[0][l, 1])
    step.close()


@pytest.mark.parametrize("path", [REG, SPLIT])
@pytest.mark.parametrize("budget", [(260, 90), (150, 50), (0, 116), (323, 0), (300, 1)])
def test_paths_in_place(budget, path):
    layers = ragged_layers(seed=200)
    step = DeviceStep(layers, 300, inplace_stage_rows=128)
    a, s = synth.make_scores([l["modality"] for l in layers], step.h_kv, 1)
    a, s = step.to_device_f32(a), step.to_device_f32(s)
    ref = _run(step, a, s, [budget], ONE)[0]
    step.ctx.omnimem_set_topk_path(path)
    _compare(step, layers, [budget], a, s)
    m = sum(_applied(budget, layers[0]["modality"], len(layers[0]["modality"])))
    got = _run(step, a, s, [budget], path)[0]
    assert torch.equal(ref[0, :, :m], got[0, :, :m])
    step.close()


def test_split_path_repeated_calls_leave_no_state():
    # The global histograms are cleared by each call: the same inputs give
    # the same rows on every call, and a call on other inputs in between
    # does not leak into the next one.
    layers = _workload("qwen-layer")
    step = DeviceStep(layers, 1000)
    a1, s1 = _scores(layers, step.h_kv, "synthetic", seed=1)
    a2, s2 = _scores(layers, step.h_kv, "ties", seed=2)
    d1 = step.to_device_f32(a1), step.to_device_f32(s1)
    d2 = step.to_device_f32(a2), step.to_device_f32(s2)
    bud = _budgets(layers, "half")
    first = _run(step, *d1, bud, SPLIT)[0]
    for _ in range(3):
        _run(step, *d2, bud, SPLIT)
        again = _run(step, *d1, bud, SPLIT)[0]
        assert torch.equal(first, again)
    step.close()


def test_unknown_path_is_refused():
    step = DeviceStep(_workload("ragged-3layer"), 300)
    with pytest.raises(omnimem.OmnimemError):
        step.ctx.omnimem_set_topk_path(7)
    step.ctx.omnimem_set_topk_path(omnimem.TOPK_AUTO)
    step.close()


def test_paths_single_modality_layers_and_tiny_working_sets():
    # A visual-only layer, an audio-only layer and a 3-row layer in one call:
    # one modality's segment is empty, budgets reach past it, and the split
    # path's only slice is nearly empty.
    layers = [ragged_layers(seed=106, caches=((150, 0),), frames=(2, 30, 0))[0],
              ragged_layers(seed=107, caches=((0, 90),), frames=(2, 0, 20))[0],
              ragged_layers(seed=108, caches=((1, 1),), frames=(1, 1, 0))[0]]
    step = DeviceStep(layers, 200)
    a_h, s_h = _scores(layers, step.h_kv, "synthetic")
    for budgets in ([(100, 5), (5, 60), (1, 1)], [(500, 500), (500, 500), (500, 500)], [(0, 0), (0, 1), (2, 0)]):
        _check(step, layers, a_h, s_h, budgets)
    step.close()
