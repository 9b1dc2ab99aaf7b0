"""The compression step after every chunk of a stream (caches carried over).

Small stream, oracle-driven: at every chunk the oracle runs the step on its
own state; the GPU runs the same working set (its cache is set to the
oracle's before the chunk is appended) and is compared stage by stage.

Full-size stream (64 chunks x 28 layers, AR(1) visual tokens): the GPU's
own caches are carried from chunk to chunk.  Every chunk is checked for
properties that hold at any size; the first two chunks, whose working sets
are pure generator output (every token is kept while the budget exceeds the
cache), are also checked against the oracle on sampled rows.
"""
import numpy as np
import pytest
import torch

from oracle import omnimem_oracle as om
from paper_2606_07577_amd import synth
from paper_2606_07577_amd.step import StreamRunner
from tests import parity as P

pytestmark = pytest.mark.gpu


def _runner(src):
    sp = src.spec
    return StreamRunner(sp["n_layers"], sp["h_q"], sp["h_kv"], sp["d"], src.chunk_len, sp["total_budget"],
                        dtype=sp["dtype"])


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
        prev = 1 - run.cur
        for l, lay in enumerate(layers):
            n = len(lay["modality"])
            P.assert_close_a(run.a[l, :, :n].cpu().numpy(), ref["a"][l], f"a chunk {t} layer {l}")
            P.assert_close_s(run.s[l, :, :n].cpu().numpy(), ref["s"][l], f"s chunk {t} layer {l}")
            mv, ma = budgets[l]
            idx = run.idx[l, :, : mv + ma].cpu().numpy()
            psi = om.retention_score(ref["a"][l], ref["s"][l], P.LAMBDA)
            k_in = run.kbuf[prev][l][:, :n].float().cpu().numpy()
            k_out = run.kbuf[run.cur][l][:, : mv + ma].float().cpu().numpy()
            v_out = run.vbuf[run.cur][l][:, : mv + ma].float().cpu().numpy()
            np.testing.assert_array_equal(k_in, lay["k"])       # the working set the GPU saw
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
    prev = 1 - run.cur
    gidx = torch.from_numpy(idx.astype(np.int64)).to(run.device)
    for buf in (run.kbuf, run.vbuf):
        src = buf[prev][l][:, :n]
        want = torch.gather(src, 1, gidx[:, :, None].expand(-1, -1, run.d))
        assert torch.equal(buf[run.cur][l][:, : mv + ma], want)
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
        n_tok = [nc + C for nc in n_cache]
        assert budgets.sum() == min(sp["total_budget"], sum(n_tok)), t
        mods = [run.mbuf[1 - run.cur][l][:n].cpu().numpy() for l, n in enumerate(n_tok)]
        for l in range(L):
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
    np.testing.assert_array_equal(run.kbuf[1 - run.cur][l][:, :n].float().cpu().numpy(), k)
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
        prev = 1 - run.cur
        for l, lay in enumerate(layers):
            mv, ma = budgets[l]
            idx = run.idx[l, :, : mv + ma].cpu().numpy()
            k_out = run.kbuf[run.cur][l][:, : mv + ma].float().cpu().numpy()
            np.testing.assert_array_equal(run.kbuf[prev][l][:, : len(lay["modality"])].float().cpu().numpy(),
                                          lay["k"])
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
