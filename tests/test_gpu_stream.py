"""The compression step after every chunk of a stream (caches carried over).

The runner keeps one cache buffer per layer: each chunk is appended behind
the kept rows (Eq. 3) and the step compacts the kept rows to the front in
place (Eqs. 2-5).

Small stream, oracle-driven: at every chunk the oracle runs the step on its
own state; the GPU runs the same working set (its cache is set to the
oracle's before the chunk is appended) and is compared stage by stage.

Post-eviction working sets at full size: caches of the shape the stream has
after many evictions (thousands of rows kept from earlier chunks, visual
block then audio block, then the new chunk), drawn on the host by a seeded
choice of earlier generator rows, go through the runner; the oracle
computes the same step on the same rows and is compared element by element.

Full-size stream (64 chunks x 28 layers, AR(1) visual tokens): the GPU's
own caches are carried from chunk to chunk.  Every chunk is checked for
properties that hold at any size; the first two chunks, whose working sets
are pure generator output (every token is kept while the budget exceeds the
cache), are also checked against the oracle on sampled rows.

In place against out of place: two runners fed the same chunks keep
bit-identical caches, also when the staging reserve is too small and the
runner falls back to compacting out of place.
"""
import numpy as np
import pytest
import torch

from oracle import omnimem_oracle as om
from paper_2606_07577_amd import synth
from paper_2606_07577_amd.step import StreamRunner
from tests import parity as P

pytestmark = pytest.mark.gpu


def _runner(src, **kw):
    sp = src.spec
    kw.setdefault("keep_working_set", True)
    return StreamRunner(sp["n_layers"], sp["h_q"], sp["h_kv"], sp["d"], src.chunk_len, sp["total_budget"],
                        dtype=sp["dtype"], **kw)


def _host(t):
    return t.float().cpu().numpy()


def test_small_stream_follows_the_oracle():
    src = synth.StreamSource("small-stream")
    sp = src.spec
    L, h_kv, d = sp["n_layers"], sp["h_kv"], sp["d"]
    run = _runner(src)
    state = [dict(k=np.zeros((h_kv, 0, d)), v=np.zeros((h_kv, 0, d)), m_v=0, m_a=0) for _ in range(L)]
    evicted = 0
    for t in range(sp["n_chunks"]):
        chunk = src.chunk(t)
        layers = []
        for l, ch in enumerate(chunk):
            st = state[l]
            mod = np.concatenate([np.zeros(st["m_v"], np.uint8), np.ones(st["m_a"], np.uint8), ch["modality"]])
            layers.append({"q": ch["q"].astype(np.float64),
                           "k": np.concatenate([st["k"], ch["k"]], axis=1).astype(np.float64),
                           "v": np.concatenate([st["v"], ch["v"]], axis=1).astype(np.float64),
                           "modality": mod, "n_cache": st["m_v"] + st["m_a"], "sm_scale": ch["sm_scale"]})
            run.set_cache(l, st["k"], st["v"], st["m_v"], st["m_a"])
        ref = om.compression_step(layers, sp["total_budget"], lam=P.LAMBDA, temperature=P.TEMPERATURE,
                                  r=P.RATIO)
        budgets = run.push(chunk).astype(np.int64)
        torch.cuda.synchronize()
        ref_b = np.array(ref["budgets"], dtype=np.int64)
        print(f"chunk {t}: N {[len(x['modality']) for x in layers]} budgets {budgets.tolist()}", flush=True)
        assert budgets.sum() == ref_b.sum() == min(sp["total_budget"], sum(len(x["modality"]) for x in layers))
        assert np.abs(budgets - ref_b).max() <= 1
        for l, lay in enumerate(layers):
            n = len(lay["modality"])
            P.assert_close_a(run.a[l, :, :n].cpu().numpy(), ref["a"][l], f"a chunk {t} layer {l}")
            P.assert_close_s(run.s[l, :, :n].cpu().numpy(), ref["s"][l], f"s chunk {t} layer {l}")
            mv, ma = budgets[l]
            idx = run.idx[l, :, : mv + ma].cpu().numpy()
            psi = om.retention_score(ref["a"][l], ref["s"][l], P.LAMBDA)
            k_ws, v_ws, m_ws = run.working_set[l]
            np.testing.assert_array_equal(_host(k_ws), lay["k"])       # the working set the GPU saw
            np.testing.assert_array_equal(m_ws.cpu().numpy(), lay["modality"])
            k_out, v_out = _host(run.cache_k(l)), _host(run.cache_v(l))
            np.testing.assert_array_equal(run.cache_modality(l).cpu().numpy(),
                                          np.repeat([0, 1], [mv, ma]).astype(np.uint8))
            for g in range(h_kv):
                P.check_selection(idx[g], psi[g], lay["modality"], mv, ma, rel=5e-3)
                np.testing.assert_array_equal(k_out[g], lay["k"][g, idx[g]])
                np.testing.assert_array_equal(v_out[g], lay["v"][g, idx[g]])
            evicted += n - mv - ma
        # The next working set starts from the oracle's caches.
        for l in range(L):
            mv, ma = ref["budgets"][l]
            state[l] = dict(k=ref["k_out"][l].astype(np.float32), v=ref["v_out"][l].astype(np.float32),
                            m_v=int(mv), m_a=int(ma))
    assert evicted > 0
    run.close()


def _gpu_topk_properties(run, l, n, mv, ma, mod):
    a = run.a[l, :, :n].cpu().numpy()
    s = run.s[l, :, :n].cpu().numpy()
    idx = run.idx[l, :, : mv + ma].cpu().numpy()
    assert np.all(np.abs(s) <= 1.0)
    for g in range(run.h_kv):
        P.check_topk_property(idx[g], a[g], s[g], mod, mv, ma)
    gidx = torch.from_numpy(idx.astype(np.int64)).to(run.device)
    k_ws, v_ws, _ = run.working_set[l]
    for src, got in ((k_ws, run.cache_k(l)), (v_ws, run.cache_v(l))):
        want = torch.gather(src, 1, gidx[:, :, None].expand(-1, -1, run.d))
        assert torch.equal(got, want)
    return a


def test_full_size_stream_64_chunks_28_layers():
    src = synth.StreamSource("qwen7b-stream-64x28", backend="torch")
    sp = src.spec
    L, C, G = sp["n_layers"], src.chunk_len, sp["h_q"] // sp["h_kv"]
    run = _runner(src)
    rng = np.random.default_rng(21)
    kept0 = None
    for t in range(sp["n_chunks"]):
        chunk = src.chunk(t)
        n_cache = list(run.n_cache)
        budgets = run.push(chunk).astype(np.int64)
        torch.cuda.synchronize()
        n_tok = [nc + C for nc in n_cache]
        assert budgets.sum() == min(sp["total_budget"], sum(n_tok)), t
        mods = [run.working_set[l][2].cpu().numpy() for l in range(L)]
        for l in range(L):
            assert len(mods[l]) == n_tok[l]
            assert budgets[l, 0] <= (mods[l] == 0).sum() and budgets[l, 1] <= (mods[l] == 1).sum()
        if t < 2:
            # The budget exceeds every cache so far: everything is kept.
            np.testing.assert_array_equal(budgets.sum(axis=1), n_tok)
        if t in (0, 1, 2, 3, 31, 63) or t % 16 == 5:
            print(f"chunk {t}: budgets {budgets[:, 0].min()}..{budgets[:, 0].max()} visual, "
                  f"{budgets[:, 1].min()}..{budgets[:, 1].max()} audio", flush=True)
            for l in (0, 13, 27):
                a = _gpu_topk_properties(run, l, n_tok[l], budgets[l, 0], budgets[l, 1], mods[l])
                np.testing.assert_allclose(a.sum(axis=1, dtype=np.float64), G * C, rtol=1e-4)
        if t == 0:
            kept0 = [(ch["k"].float().cpu().numpy(), ch["v"].float().cpu().numpy(), ch["modality"].cpu().numpy())
                     for ch in chunk]
            _oracle_sampled(run, chunk, None, 0, t, rng)
        if t == 1:
            _oracle_sampled(run, chunk, kept0, 27, t, rng)
    assert run.steps == sp["n_chunks"]
    assert run.fallbacks == 0
    run.close()


def _oracle_sampled(run, chunk, kept, l, t, rng):
    """Chunk 0 or 1: the working set is generator output (chunk 1 follows
    chunk 0's rows, all kept, visual first); compare lse-free quantities on
    samples with the oracle: a at sampled keys of one KV head, s at sampled
    rows."""
    ch = chunk[l]
    q = ch["q"].float().cpu().numpy().astype(np.float64)
    k = ch["k"].float().cpu().numpy().astype(np.float64)
    v = ch["v"].float().cpu().numpy().astype(np.float64)
    mod = ch["modality"].cpu().numpy()
    n_cache = 0
    if kept is not None:
        k0, v0, m0 = kept[l]
        order = np.concatenate([np.flatnonzero(m0 == 0), np.flatnonzero(m0 == 1)])
        k = np.concatenate([k0[:, order].astype(np.float64), k], axis=1)
        v = np.concatenate([v0[:, order].astype(np.float64), v], axis=1)
        mod = np.concatenate([m0[order], mod])
        n_cache = len(order)
    n = len(mod)
    np.testing.assert_array_equal(_host(run.working_set[l][0]), k)
    h_kv = k.shape[0]
    group = q.shape[0] // h_kv
    g = int(rng.integers(h_kv))
    keys = np.sort(rng.choice(n, size=64, replace=False))
    q_g = q[g * group:(g + 1) * group]
    lse_g = om.attention_lse(q_g, k[g:g + 1], n_cache, ch["sm_scale"], True)
    a_ref = om.attention_importance(q_g, k[g:g + 1], n_cache, ch["sm_scale"], True, lse=lse_g, keys=keys)
    P.assert_close_a(run.a[l, g, :n].cpu().numpy()[keys], a_ref[0], f"a chunk {t} layer {l} head {g}")
    rows = np.sort(rng.choice(n, size=64, replace=False))
    s_ref = om.redundancy(v, mod, "max", rows=rows)
    P.assert_close_s(run.s[l, :, :n].cpu().numpy()[:, rows], s_ref, f"s chunk {t} layer {l}")


# ---------------------------------------------------------------------------
# Post-eviction working sets at full size
# ---------------------------------------------------------------------------

def _post_eviction_layers(t, layers=(0, 1), keep=(3072, 1024), seed=77):
    """Working sets of two layers of the 64 x 28 stream at chunk t, built on
    the host: the cache is a seeded uniform choice of `keep` = (visual, audio)
    rows among all rows of chunks 0 .. t-1 of that layer (the same rows in
    every KV head, in age order, visual block then audio block), followed by
    chunk t.  Values are the generator's (numpy backend)."""
    src = synth.StreamSource("qwen7b-stream-64x28", n_layers=max(layers) + 1)
    rng = np.random.default_rng([seed, t])
    pools = {l: ([], [], []) for l in layers}     # visual k, v rows; audio k, v rows
    out_chunk = None
    for c in range(t + 1):
        ch = src.chunk(c)
        if c == t:
            out_chunk = ch
            break
        for l in layers:
            mod = ch[l]["modality"]
            kv, vv, ka_va = pools[l]
            kv.append(ch[l]["k"][:, mod == 0])
            vv.append(ch[l]["v"][:, mod == 0])
            ka_va.append((ch[l]["k"][:, mod == 1], ch[l]["v"][:, mod == 1]))
    work = []
    for l in layers:
        kv, vv, ka_va = pools[l]
        ch = out_chunk[l]
        if t == 0:
            k_c = np.zeros((ch["k"].shape[0], 0, ch["k"].shape[2]), np.float32)
            v_c, m_v, m_a = k_c, 0, 0
        else:
            kvis, vvis = np.concatenate(kv, axis=1), np.concatenate(vv, axis=1)
            kaud = np.concatenate([x[0] for x in ka_va], axis=1)
            vaud = np.concatenate([x[1] for x in ka_va], axis=1)
            m_v, m_a = min(keep[0], kvis.shape[1]), min(keep[1], kaud.shape[1])
            iv = np.sort(rng.choice(kvis.shape[1], size=m_v, replace=False))
            ia = np.sort(rng.choice(kaud.shape[1], size=m_a, replace=False))
            k_c = np.concatenate([kvis[:, iv], kaud[:, ia]], axis=1)
            v_c = np.concatenate([vvis[:, iv], vaud[:, ia]], axis=1)
        mod = np.concatenate([np.zeros(m_v, np.uint8), np.ones(m_a, np.uint8), ch["modality"]])
        work.append(dict(cache=(k_c, v_c, m_v, m_a), chunk=ch,
                         layer={"q": ch["q"].astype(np.float64),
                                "k": np.concatenate([k_c, ch["k"]], axis=1).astype(np.float64),
                                "v": np.concatenate([v_c, ch["v"]], axis=1).astype(np.float64),
                                "modality": mod, "n_cache": m_v + m_a, "sm_scale": ch["sm_scale"]}))
    return work, src


@pytest.mark.timeout(400)
@pytest.mark.parametrize("t", [2, 31, 63])
def test_post_eviction_working_sets_full_size(t):
    work, src = _post_eviction_layers(t)
    sp = src.spec
    L = len(work)
    run = StreamRunner(L, sp["h_q"], sp["h_kv"], sp["d"], src.chunk_len, L * 4096, dtype="bf16",
                       keep_working_set=True)
    for l, w in enumerate(work):
        run.set_cache(l, *w["cache"])
    budgets = run.push([w["chunk"] for w in work]).astype(np.int64)
    torch.cuda.synchronize()
    layers = [w["layer"] for w in work]
    a_ref, s_ref = [], []
    for l, lay in enumerate(layers):
        n = len(lay["modality"])
        np.testing.assert_array_equal(_host(run.working_set[l][0]), lay["k"])
        a = om.attention_importance(lay["q"], lay["k"], lay["n_cache"], lay["sm_scale"], True)
        s = om.redundancy(lay["v"], lay["modality"], "max")
        P.assert_close_a(run.a[l, :, :n].cpu().numpy(), a, f"a chunk {t} layer {l}")
        P.assert_close_s(run.s[l, :, :n].cpu().numpy(), s, f"s chunk {t} layer {l}")
        a_ref.append(a)
        s_ref.append(s)
    ref_stats, shares, ref_budgets = P.oracle_allocation(a_ref, s_ref, layers, L * 4096)
    print(f"chunk {t}: N {[len(x['modality']) for x in layers]} budgets gpu {budgets.tolist()} "
          f"oracle {ref_budgets.tolist()}", flush=True)
    assert budgets.sum() == ref_budgets.sum()
    bounds = P.free_running_budget_bounds(run.stats.cpu().numpy(), ref_stats, shares, ref_budgets)
    print(f"chunk {t}: budget differences {np.abs(budgets - ref_budgets).max()} within bounds up to {bounds.max()}")
    assert (np.abs(budgets - ref_budgets) <= bounds).all(), (budgets, ref_budgets, bounds)
    for l, lay in enumerate(layers):
        mv, ma = budgets[l]
        psi = om.retention_score(a_ref[l], s_ref[l], P.LAMBDA)
        idx = run.idx[l, :, : mv + ma].cpu().numpy()
        k_out, v_out = _host(run.cache_k(l)), _host(run.cache_v(l))
        for g in range(run.h_kv):
            P.check_selection(idx[g], psi[g], lay["modality"], mv, ma, rel=5e-3)
            np.testing.assert_array_equal(k_out[g], lay["k"][g, idx[g]])
            np.testing.assert_array_equal(v_out[g], lay["v"][g, idx[g]])
    # Teacher-forced: the oracle's a, s (fp32) into allocation and selection.
    st_a = torch.zeros_like(run.a)
    st_s = torch.zeros_like(run.s)
    for l, lay in enumerate(layers):
        n = len(lay["modality"])
        st_a[l, :, :n] = torch.from_numpy(a_ref[l].astype(np.float32))
        st_s[l, :, :n] = torch.from_numpy(s_ref[l].astype(np.float32))
    # (the runner's buffers now hold the compacted caches: describe the
    # working sets from their snapshots)
    from paper_2606_07577_amd import omnimem
    descs = [omnimem.make_layer(None, k_ws, v_ws, m_ws, layers[l]["n_cache"], layers[l]["sm_scale"])
             for l, (k_ws, v_ws, m_ws) in enumerate(run.working_set)]
    stats, _, forced = P.oracle_allocation([x.astype(np.float32).astype(np.float64) for x in a_ref],
                                           [x.astype(np.float32).astype(np.float64) for x in s_ref], layers, L * 4096)
    out = torch.zeros_like(run.budgets)
    run.ctx.omnimem_allocate(descs, st_a, st_s, L * 4096, out)
    torch.cuda.synchronize()
    np.testing.assert_array_equal(out.cpu().numpy(), forced)
    run.close()


# ---------------------------------------------------------------------------
# In place against out of place
# ---------------------------------------------------------------------------

def _same_caches(r1, r2, L):
    torch.cuda.synchronize()
    for l in range(L):
        assert r1.n_cache[l] == r2.n_cache[l]
        assert torch.equal(r1.cache_k(l), r2.cache_k(l)), l
        assert torch.equal(r1.cache_v(l), r2.cache_v(l)), l
        assert torch.equal(r1.cache_modality(l), r2.cache_modality(l)), l


@pytest.mark.parametrize("name,chunks,stage_rows", [("small-stream", 10, None), ("small-stream", 10, 1),
                                                    ("qwen7b-stream-64x28", 6, None)])
def test_stream_in_place_equals_out_of_place(name, chunks, stage_rows):
    src = synth.StreamSource(name, backend="torch")
    ip = _runner(src, keep_working_set=False, stage_rows=stage_rows)
    oop = _runner(src, keep_working_set=False, in_place=False)
    L = src.spec["n_layers"]
    for t in range(chunks):
        chunk = src.chunk(t)
        b1 = ip.push(chunk)
        b2 = oop.push(chunk)
        np.testing.assert_array_equal(b1, b2)
        _same_caches(ip, oop, L)
    if stage_rows == 1:
        assert ip.fallbacks > 0   # the reserve was too small for some step: compacted out of place
    else:
        assert ip.fallbacks == 0
    ip.close()
    oop.close()


@pytest.mark.parametrize("in_place,stage_rows", [(True, None), (True, 1), (False, None)])
def test_stream_without_waiting_equals_waiting(in_place, stage_rows):
    # push(wait=False) reads a step's budgets only when the next chunk has
    # been described (or at finish()): the same steps, the same caches.
    src = synth.StreamSource("small-stream", backend="torch")
    waiting = _runner(src, keep_working_set=False, in_place=in_place, stage_rows=stage_rows)
    pipelined = _runner(src, keep_working_set=False, in_place=in_place, stage_rows=stage_rows)
    L = src.spec["n_layers"]
    chunks = [src.chunk(t) for t in range(10)]
    for t, chunk in enumerate(chunks):
        b = waiting.push(chunk)
        assert pipelined.push(chunk, wait=False) is None
        if t == 4:   # finish() gives the step's budgets
            np.testing.assert_array_equal(pipelined.finish(), b)
            _same_caches(waiting, pipelined, L)
        if t == 7:   # so does a read of a cache
            pipelined.cache_k(0)
            _same_caches(waiting, pipelined, L)
    np.testing.assert_array_equal(pipelined.finish(), waiting.budgets_host.numpy())
    assert pipelined.finish() is None
    _same_caches(waiting, pipelined, L)
    assert (pipelined.steps, pipelined.tokens, pipelined.fallbacks) == (waiting.steps, waiting.tokens, waiting.fallbacks)
    waiting.close()
    pipelined.close()


def test_small_stream_with_offline_budgets():
    # Offline budgets (end of Sec. 3.2; reading R21) on a stream: the first
    # four chunks calibrate (their steps allocate online), the layer budgets
    # are then frozen and the remaining chunks only split them.  The GPU's
    # frozen budgets come from its own statistics, so they may differ from
    # the oracle's by a rounding unit; from the freeze on the GPU takes the
    # oracle's (teacher-forced) and each step must match the oracle's.
    src = synth.StreamSource("small-stream")
    sp = src.spec
    L, h_kv, d = sp["n_layers"], sp["h_kv"], sp["d"]
    total = sp["total_budget"]
    n_cal = 4
    run = _runner(src)
    run.ctx.omnimem_calibration_reset()
    run.calibrating = True
    state = [dict(k=np.zeros((h_kv, 0, d)), v=np.zeros((h_kv, 0, d)), m_v=0, m_a=0) for _ in range(L)]
    c_hist, ref_lb = [], None
    for t in range(sp["n_chunks"]):
        chunk = src.chunk(t)
        layers = []
        for l, ch in enumerate(chunk):
            st = state[l]
            mod = np.concatenate([np.zeros(st["m_v"], np.uint8), np.ones(st["m_a"], np.uint8), ch["modality"]])
            layers.append({"q": ch["q"].astype(np.float64),
                           "k": np.concatenate([st["k"], ch["k"]], axis=1).astype(np.float64),
                           "v": np.concatenate([st["v"], ch["v"]], axis=1).astype(np.float64),
                           "modality": mod, "n_cache": st["m_v"] + st["m_a"], "sm_scale": ch["sm_scale"]})
            run.set_cache(l, st["k"], st["v"], st["m_v"], st["m_a"])
        ref = om.compression_step(layers, total, lam=P.LAMBDA, temperature=P.TEMPERATURE, r=P.RATIO,
                                  layer_budgets=ref_lb)
        budgets = run.push(chunk).astype(np.int64)
        torch.cuda.synchronize()
        ref_b = np.array(ref["budgets"], dtype=np.int64)
        n_tok = np.array([len(x["modality"]) for x in layers])
        print(f"chunk {t}: N {n_tok.tolist()} budgets {budgets.tolist()}", flush=True)
        if ref_lb is None:
            c_hist.append([s["C_l"] for s in ref["stats"]])
            assert np.abs(budgets - ref_b).max() <= 1
        else:
            np.testing.assert_array_equal(budgets.sum(axis=1), np.minimum(ref_lb, n_tok))
            assert np.abs(budgets - ref_b).max() <= 1
        for l, lay in enumerate(layers):
            mv, ma = budgets[l]
            idx = run.idx[l, :, : mv + ma].cpu().numpy()
            k_out = _host(run.cache_k(l))
            np.testing.assert_array_equal(_host(run.working_set[l][0]), lay["k"])
            if (mv, ma) == tuple(ref_b[l]):
                psi = om.retention_score(ref["a"][l], ref["s"][l], P.LAMBDA)
                for g in range(h_kv):
                    P.check_selection(idx[g], psi[g], lay["modality"], mv, ma, rel=5e-3)
            for g in range(h_kv):
                np.testing.assert_array_equal(k_out[g], lay["k"][g, idx[g]])
        if t == n_cal - 1:
            run.freeze_budgets()
            ref_lb = om.calibration_budgets(c_hist, total, P.TEMPERATURE)
            got_lb = run.layer_budgets.cpu().numpy().astype(np.int64)
            print(f"frozen layer budgets: gpu {got_lb.tolist()} oracle {ref_lb.tolist()}", flush=True)
            assert got_lb.sum() == ref_lb.sum() == total
            assert np.abs(got_lb - ref_lb).max() <= 1
            run.layer_budgets.copy_(torch.from_numpy(ref_lb.astype(np.int32)))
        for l in range(L):
            mv, ma = ref["budgets"][l]
            state[l] = dict(k=ref["k_out"][l].astype(np.float32), v=ref["v_out"][l].astype(np.float32),
                            m_v=int(mv), m_a=int(ma))
    run.close()
