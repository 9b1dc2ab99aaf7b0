"""Compaction in place (k_out is k, v_out is v; Eqs. 2-5: each cache is
pruned into its own next state) against compaction out of place, bit for
bit, through the C ABI.

The kept rows come from the same selection in both runs (same a, s and
budgets), so the in-place result must equal the out-of-place one exactly,
whatever order the in-place pass moves rows in.  Cases cover budgets where
every kept row moves toward the front, where kept audio rows land behind
their own row (the visual budget exceeds the visual rows in front of them:
those rows go through the staging rows), where nothing moves, mixed
in-place and out-of-place layers in one call, layer-shared selection,
fp32 at head_dim 64, full-size layers, a shortfall of staging rows (nothing
may move), an output capacity below the budget, and the chunk append
(Eq. 3) that follows a step in a stream.
"""
import numpy as np
import pytest
import torch

from paper_2606_07577_amd import omnimem, synth
from paper_2606_07577_amd.step import DeviceStep
from tests.test_gpu_parity import ragged_layers

pytestmark = pytest.mark.gpu


def _scores(step, layers, seed):
    a, s = synth.make_scores([l["modality"] for l in layers], step.h_kv, seed)
    return step.to_device_f32(a), step.to_device_f32(s)


def _compare(step, layers, budgets, a, s, inplace_layers=None, check_rest=True):
    """Run select_compact out of place and in place (on copies of k, v and
    the modality) with the same inputs; assert equal results."""
    L = len(layers)
    inplace_layers = set(range(L)) if inplace_layers is None else set(inplace_layers)
    bud = torch.tensor(budgets, dtype=torch.int32, device=step.device)
    idx_oop = torch.full_like(step.idx, -1)
    mod_oop = [torch.full_like(m, 7) for m in step.mod]
    descs = [omnimem.make_layer(step.q[l], step.k[l], step.v[l], step.mod[l], step.n_cache[l], step.sm_scale[l],
                                None, step.k_out[l], step.v_out[l], modality_out=mod_oop[l]) for l in range(L)]
    step.ctx.omnimem_select_compact(descs, a, s, bud, idx_oop)
    torch.cuda.synchronize()
    k_in = [step.k[l].clone() for l in range(L)]
    v_in = [step.v[l].clone() for l in range(L)]
    m_in = [step.mod[l].clone() for l in range(L)]
    kw = [x.clone() for x in k_in]
    vw = [x.clone() for x in v_in]
    mw = [x.clone() for x in m_in]
    ko = [torch.zeros_like(x) for x in k_in]
    vo = [torch.zeros_like(x) for x in v_in]
    descs = []
    for l in range(L):
        if l in inplace_layers:
            descs.append(omnimem.make_layer(step.q[l], kw[l], vw[l], mw[l], step.n_cache[l], step.sm_scale[l], None,
                                            kw[l], vw[l], modality_out=mw[l]))
        else:
            descs.append(omnimem.make_layer(step.q[l], kw[l], vw[l], mw[l], step.n_cache[l], step.sm_scale[l], None,
                                            ko[l], vo[l], modality_out=mw[l]))
    idx_ip = torch.full_like(step.idx, -1)
    step.ctx.omnimem_select_compact(descs, a, s, bud, idx_ip)
    torch.cuda.synchronize()
    assert step.ctx.omnimem_inplace_status() >= 0
    assert torch.equal(idx_ip, idx_oop)
    moved_back = 0
    for l in range(L):
        mv, ma = (int(x) for x in budgets[l])
        m = mv + ma
        kk, vv = (kw[l], vw[l]) if l in inplace_layers else (ko[l], vo[l])
        assert torch.equal(kk[:, :m], step.k_out[l][:, :m]), f"layer {l}: k differs"
        assert torch.equal(vv[:, :m], step.v_out[l][:, :m]), f"layer {l}: v differs"
        want_mod = torch.cat([torch.zeros(mv, dtype=torch.uint8), torch.ones(ma, dtype=torch.uint8)])
        assert torch.equal(mw[l][:m].cpu(), want_mod)
        assert torch.equal(mod_oop[l][:m].cpu(), want_mod)
        if check_rest:
            # rows from M on are never written, in place or not
            assert torch.equal(mw[l][m:], m_in[l][m:])
            if l in inplace_layers:
                assert torch.equal(kw[l][:, m:], k_in[l][:, m:]) and torch.equal(vw[l][:, m:], v_in[l][:, m:])
            else:
                assert torch.equal(kw[l], k_in[l]) and torch.equal(vw[l], v_in[l])
        idx = idx_oop[l, :, :m].cpu().numpy()
        moved_back += int((idx[:, mv:] < np.arange(mv, m)[None, :]).sum())
    return moved_back


@pytest.mark.parametrize("budget", [(260, 90), (150, 50), (323, 116), (0, 116), (323, 0), (0, 0), (300, 1)])
def test_inplace_equals_out_of_place_ragged(budget):
    layers = ragged_layers(seed=200)   # cache 200 v + 77 a, chunk 3 x (41 v + 13 a): K_v 323, K_a 116
    step = DeviceStep(layers, 300, inplace_stage_rows=128)
    a, s = _scores(step, layers, 1)
    moved_back = _compare(step, layers, [budget], a, s)
    print(f"budget {budget}: {moved_back} kept rows staged", flush=True)
    if budget == (260, 90):
        assert moved_back > 0          # the staging path ran
    if budget[0] <= 200:
        assert moved_back == 0
    step.close()


def test_inplace_mixed_layers_and_fp32():
    layers = ragged_layers(3, seed=201, caches=((200, 77), (333, 111), (64, 17)))
    step = DeviceStep(layers, 3 * 260, inplace_stage_rows=256)
    a, s = _scores(step, layers, 2)
    budgets = [(250, 60), (300, 100), (150, 30)]
    assert _compare(step, layers, budgets, a, s, inplace_layers=[0, 2]) > 0
    assert _compare(step, layers, budgets, a, s) > 0
    step.close()
    tiny = synth.make_workload("tiny-f32-640")
    step = DeviceStep(tiny, 256, inplace_stage_rows=160)
    a, s = _scores(step, tiny, 3)
    assert _compare(step, tiny, [(420, 100)], a, s) > 0   # visual cache is 384 rows
    assert _compare(step, tiny, [(200, 56)], a, s) == 0
    step.close()


def test_inplace_shared_selection():
    layers = ragged_layers(2, seed=202, caches=((200, 77), (120, 40)))
    step = DeviceStep(layers, 2 * 260, inplace_stage_rows=128, shared_selection=1)
    a, s = _scores(step, layers, 4)
    assert _compare(step, layers, [(260, 90), (200, 50)], a, s) > 0
    step.close()


def test_inplace_full_size_layer():
    # 6144 rows, 4 KV heads: once with the GPU's own AVBA budgets, once with
    # a visual budget beyond the 3072 visual cache rows (the 1024 audio cache
    # rows, when kept, land behind their row).
    layers = synth.make_workload("qwen7b-layer-6144")
    step = DeviceStep(layers, 4096, inplace_stage_rows=2048)
    step.score()
    step.redundancy()
    step.allocate()
    torch.cuda.synchronize()
    own = step.budgets.cpu().numpy().tolist()
    _compare(step, layers, own, step.a, step.s)
    assert _compare(step, layers, [(3800, 600)], step.a, step.s) > 0
    step.close()


def test_inplace_stream_first_chunk_shape():
    # A stream's first step: an empty cache and a chunk of interleaved frames
    # [384 v | 128 a] x 4 kept whole: every audio row but the last ones lands
    # behind its own row.
    src = synth.StreamSource("qwen7b-stream-64x28", n_layers=2)
    ch = src.chunk(0)
    layers = [dict(q=c["q"], k=c["k"], v=c["v"], modality=c["modality"], n_cache=0, sm_scale=c["sm_scale"],
                   dtype="bf16") for c in ch]
    step = DeviceStep(layers, 2 * 2048, inplace_stage_rows=512)
    a, s = _scores(step, layers, 5)
    assert _compare(step, layers, [(1536, 512), (1536, 512)], a, s) > 400
    step.close()


def test_inplace_staging_shortfall_moves_nothing():
    layers = ragged_layers(seed=203)
    step = DeviceStep(layers, 300, inplace_stage_rows=4)
    a, s = _scores(step, layers, 6)
    k0, v0, m0 = step.k[0].clone(), step.v[0].clone(), step.mod[0].clone()
    desc = omnimem.make_layer(step.q[0], step.k[0], step.v[0], step.mod[0], step.n_cache[0], 0.0, None,
                              step.k[0], step.v[0], modality_out=step.mod[0])
    bud = torch.tensor([[260, 90]], dtype=torch.int32, device=step.device)
    step.ctx.omnimem_select_compact([desc], a, s, bud, step.idx)
    torch.cuda.synchronize()
    with pytest.raises(omnimem.OmnimemError) as e:
        step.ctx.omnimem_inplace_status()
    assert e.value.status == omnimem.ERR_CAPACITY
    assert torch.equal(step.k[0], k0) and torch.equal(step.v[0], v0) and torch.equal(step.mod[0], m0)
    idx = step.idx[0, :, :350].cpu().numpy()
    assert (np.diff(idx[:, :260], axis=1) > 0).all() and (np.diff(idx[:, 260:], axis=1) > 0).all()
    # the reported need is the longest run of audio slots whose row lies in front of them
    slots = np.arange(260, 350)
    need = max(int(((idx[g, 260:] >= 0) & (idx[g, 260:] < slots)).sum()) for g in range(idx.shape[0]))
    assert need > 4 and f"needed {need} staging rows" in str(e.value), (need, str(e.value))
    assert step.ctx.omnimem_inplace_status() == 0      # the record was cleared
    # A call that needs no staging rows still runs on the same context.
    bud = torch.tensor([[150, 50]], dtype=torch.int32, device=step.device)
    step.ctx.omnimem_select_compact([desc], a, s, bud, step.idx)
    torch.cuda.synchronize()
    assert step.ctx.omnimem_inplace_status() == 0
    idx = step.idx[0, :, :200].long()
    for g in range(2):
        assert torch.equal(step.k[0][g, :200], k0[g, idx[g]])
    step.close()


def test_inplace_long_shortfall_is_counted_whole():
    # A full-size layer whose visual budget exceeds the 3072 visual cache
    # rows: the kept audio cache rows all land behind their row, a run of
    # hundreds of slots against 100 staging rows (two staging tiles).  Nothing
    # moves, and the status reports the whole run.
    layers = synth.make_workload("qwen7b-layer-6144")
    step = DeviceStep(layers, 4096, inplace_stage_rows=100)
    a, s = _scores(step, layers, 8)
    k0, v0 = step.k[0].clone(), step.v[0].clone()
    desc = omnimem.make_layer(step.q[0], step.k[0], step.v[0], step.mod[0], step.n_cache[0], step.sm_scale[0], None,
                              step.k[0], step.v[0])
    mv, ma = 3900, 900
    bud = torch.tensor([[mv, ma]], dtype=torch.int32, device=step.device)
    step.ctx.omnimem_select_compact([desc], a, s, bud, step.idx)
    torch.cuda.synchronize()
    with pytest.raises(omnimem.OmnimemError) as e:
        step.ctx.omnimem_inplace_status()
    assert e.value.status == omnimem.ERR_CAPACITY
    assert torch.equal(step.k[0], k0) and torch.equal(step.v[0], v0)
    idx = step.idx[0, :, mv:mv + ma].cpu().numpy()
    slots = np.arange(mv, mv + ma)
    need = max(int(((idx[g] >= 0) & (idx[g] < slots)).sum()) for g in range(idx.shape[0]))
    assert need > 100 + 256 and f"needed {need} staging rows" in str(e.value), (need, str(e.value))
    step.close()


def test_output_capacity_below_budget():
    # Out of place into outputs of exactly M rows per head ([H_kv][M][d]),
    # and into outputs smaller than the budget: visual rows first.
    layers = ragged_layers(seed=204)
    step = DeviceStep(layers, 300)
    a, s = _scores(step, layers, 7)
    bud = torch.tensor([[220, 80]], dtype=torch.int32, device=step.device)
    ref = omnimem.make_layer(step.q[0], step.k[0], step.v[0], step.mod[0], step.n_cache[0], 0.0, None,
                             step.k_out[0], step.v_out[0])
    idx_ref = torch.full_like(step.idx, -1)
    step.ctx.omnimem_select_compact([ref], a, s, bud, idx_ref)
    torch.cuda.synchronize()
    for cap, mv, ma in ((300, 220, 80), (250, 220, 30), (200, 200, 0)):
        ko = torch.zeros((2, cap, 128), dtype=torch.bfloat16, device=step.device)
        vo = torch.zeros_like(ko)
        mo = torch.full((cap,), 9, dtype=torch.uint8, device=step.device)
        desc = omnimem.make_layer(step.q[0], step.k[0], step.v[0], step.mod[0], step.n_cache[0], 0.0, None, ko, vo,
                                  out_rows=cap, modality_out=mo)
        idx = torch.full_like(step.idx, -1)
        step.ctx.omnimem_select_compact([desc], a, s, bud, idx)
        torch.cuda.synchronize()
        # each block keeps the top rows of the same ranking: the full budget's
        # rows when it fits, else a subset of them, in row order
        for lo, hi, flo, fhi in ((0, mv, 0, 220), (mv, mv + ma, 220, 300)):
            got = idx[0, :, lo:hi].cpu().numpy()
            full = idx_ref[0, :, flo:fhi].cpu().numpy()
            for g in range(2):
                if hi - lo == fhi - flo:
                    np.testing.assert_array_equal(got[g], full[g])
                assert set(got[g].tolist()) <= set(full[g].tolist())
                assert (np.diff(got[g]) > 0).all()
        rows = idx[0, :, : mv + ma].long()
        for g in range(2):
            assert torch.equal(ko[g, : mv + ma], step.k[0][g, rows[g]])
            assert torch.equal(vo[g, : mv + ma], step.v[0][g, rows[g]])
        assert (mo[:mv] == 0).all() and (mo[mv:mv + ma] == 1).all() and (mo[mv + ma:] == 9).all()
    # An output buffer too small for its out_rows is refused.
    ko = torch.zeros((2, 100, 128), dtype=torch.bfloat16, device=step.device)
    bad = omnimem.make_layer(step.q[0], step.k[0], step.v[0], step.mod[0], step.n_cache[0], 0.0, None, ko,
                             torch.zeros_like(ko), out_rows=0)
    with pytest.raises(omnimem.OmnimemError) as e:
        step.ctx.omnimem_select_compact([bad], a, s, bud, step.idx)
    assert e.value.status == omnimem.ERR_INVALID_ARG
    step.close()


def test_aliasing_rules():
    layers = ragged_layers(seed=205)
    step = DeviceStep(layers, 300)                 # no staging rows reserved
    a, s = _scores(step, layers, 8)
    inplace = omnimem.make_layer(step.q[0], step.k[0], step.v[0], step.mod[0], step.n_cache[0], 0.0, None,
                                 step.k[0], step.v[0])
    with pytest.raises(omnimem.OmnimemError) as e:
        step.ctx.omnimem_select_compact([inplace], a, s, step.budgets, step.idx)
    assert e.value.status == omnimem.ERR_INVALID_ARG and "staging" in str(e.value)
    step.close()
    step = DeviceStep(layers, 300, inplace_stage_rows=64)
    shifted = omnimem.make_layer(step.q[0], step.k[0], step.v[0], step.mod[0], step.n_cache[0], 0.0, None,
                                 step.k[0][:, 1:], step.v[0][:, 1:])     # overlaps without being k, v
    with pytest.raises(omnimem.OmnimemError) as e:
        step.ctx.omnimem_select_compact([shifted], a, s, step.budgets, step.idx)
    assert e.value.status == omnimem.ERR_INVALID_ARG
    half = omnimem.make_layer(step.q[0], step.k[0], step.v[0], step.mod[0], step.n_cache[0], 0.0, None,
                              step.k[0], step.v_out[0])                  # only k in place
    with pytest.raises(omnimem.OmnimemError) as e:
        step.ctx.omnimem_select_compact([half], a, s, step.budgets, step.idx)
    assert e.value.status == omnimem.ERR_INVALID_ARG
    step.close()


def test_append_after_inplace_step():
    # Eq. (3): after an in-place step the next chunk goes behind the kept rows.
    layers = ragged_layers(2, seed=206, caches=((200, 77), (120, 40)))
    cap = 600
    step = DeviceStep(layers, 2 * 260, inplace_stage_rows=128)
    a, s = _scores(step, layers, 9)
    budgets = [(250, 60), (130, 50)]
    ks = [torch.zeros((2, cap, 128), dtype=torch.bfloat16, device=step.device) for _ in layers]
    vs = [torch.zeros_like(x) for x in ks]
    ms = [torch.full((cap,), 5, dtype=torch.uint8, device=step.device) for _ in layers]
    descs = []
    for l in range(2):
        n = step.n[l]
        ks[l][:, :n], vs[l][:, :n], ms[l][:n] = step.k[l], step.v[l], step.mod[l]
        descs.append(omnimem.make_layer(step.q[l], ks[l], vs[l], ms[l], step.n_cache[l], 0.0, None, ks[l], vs[l],
                                        modality_out=ms[l], n=n))
    bud = torch.tensor(budgets, dtype=torch.int32, device=step.device)
    step.ctx.omnimem_select_compact(descs, a, s, bud, step.idx)
    torch.cuda.synchronize()
    kept = [ks[l][:, :sum(budgets[l])].clone() for l in range(2)]
    gen = torch.Generator(device="cuda").manual_seed(3)
    chunks, new = [], []
    for l in range(2):
        ck = torch.randn((2, 50, 128), generator=gen, device="cuda").to(torch.bfloat16)
        cv = torch.randn((2, 50, 128), generator=gen, device="cuda").to(torch.bfloat16)
        cm = (torch.arange(50, device="cuda") % 5 == 4).to(torch.uint8)
        chunks.append(omnimem.make_chunk(ck, cv, cm))
        new.append((ck, cv, cm))
    m = [sum(b) for b in budgets]
    qs = [torch.zeros((8, 50, 128), dtype=torch.bfloat16, device="cuda") for _ in range(2)]
    nxt = [omnimem.make_layer(qs[l], ks[l], vs[l], ms[l], m[l], 0.0, n=m[l] + 50) for l in range(2)]
    step.ctx.omnimem_append(nxt, chunks)
    torch.cuda.synchronize()
    for l in range(2):
        ck, cv, cm = new[l]
        assert torch.equal(ks[l][:, :m[l]], kept[l]) and torch.equal(ks[l][:, m[l]:m[l] + 50], ck)
        assert torch.equal(vs[l][:, m[l]:m[l] + 50], cv)
        want = torch.cat([torch.zeros(budgets[l][0], dtype=torch.uint8), torch.ones(budgets[l][1], dtype=torch.uint8),
                          cm.cpu()])
        assert torch.equal(ms[l][: m[l] + 50].cpu(), want)
        assert (ms[l][max(m[l] + 50, step.n[l]):] == 5).all()
    bad = [omnimem.make_chunk(new[l][0][:, :49], new[l][1][:, :49], new[l][2][:49]) for l in range(2)]
    with pytest.raises(omnimem.OmnimemError) as e:
        step.ctx.omnimem_append(nxt, bad)
    assert e.value.status == omnimem.ERR_INVALID_ARG
    step.close()
