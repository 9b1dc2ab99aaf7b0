"""The seeded input generator: shapes, determinism, bf16 rounding, structure."""
import numpy as np
import pytest
import torch

from paper_2606_07577_amd import synth


def test_round_to_bf16_matches_torch_cast():
    rng = np.random.default_rng(0)
    x = (rng.standard_normal(100000) * np.exp(rng.uniform(-20, 20, 100000))).astype(np.float32)
    x[:4] = [0.0, -0.0, 1.0 + 2 ** -8, 1.0 + 3 * 2 ** -8]  # exact ties round to even
    want = torch.from_numpy(x).to(torch.bfloat16).to(torch.float32).numpy()
    np.testing.assert_array_equal(synth.round_to_bf16(x), want)


def test_tiny_workload_shapes_and_layout():
    (layer,) = synth.make_workload("tiny-f32-640")
    assert layer["q"].shape == (8, 128, 64)
    assert layer["k"].shape == layer["v"].shape == (2, 640, 64)
    mod = layer["modality"]
    assert (mod == 0).sum() == 480 and (mod == 1).sum() == 160
    assert (mod[:384] == 0).all() and (mod[384:512] == 1).all()
    assert mod[512:560].tolist() == [0] * 48 and mod[560:576].tolist() == [1] * 16
    assert layer["n_cache"] == 512
    assert layer["sm_scale"] == np.float32(1 / 8)


def test_deterministic_and_layer_independent():
    a = synth.make_workload("qwen7b-28layer-6144", layers=[3], h_q=4, h_kv=1, d=16)
    b = synth.make_workload("qwen7b-28layer-6144", layers=[3], h_q=4, h_kv=1, d=16)
    c = synth.make_workload("qwen7b-28layer-6144", layers=[4], h_q=4, h_kv=1, d=16)
    for key in ("q", "k", "v"):
        np.testing.assert_array_equal(a[0][key], b[0][key])
        assert not np.array_equal(a[0][key], c[0][key])
    assert a[0]["sm_scale"] != c[0]["sm_scale"]


def test_bf16_values_are_representable():
    (layer,) = synth.make_workload("qwen7b-layer-6144", h_q=4, h_kv=2, d=32)
    for key in ("q", "k", "v"):
        np.testing.assert_array_equal(synth.round_to_bf16(layer[key]), layer[key])


def test_near_duplicate_fraction():
    (layer,) = synth.make_workload("tiny-f32-640")
    vis = np.flatnonzero(layer["modality"] == 0)
    v = layer["v"][0, vis]
    v = v / np.linalg.norm(v, axis=1, keepdims=True)
    cos = v @ v.T
    dup = [t for t in range(1, len(vis)) if cos[t, :t].max() > 0.99]
    assert abs(len(dup) - 0.25 * len(vis)) <= 2


def test_long_cache_audio_keys_are_smaller():
    spec = dict(h_q=4, h_kv=1, d=32, n_cache_v=768, n_cache_a=256, n_frames=2)
    (layer,) = synth.make_workload("qwen7b-longcache-40960", **spec)
    aud = layer["modality"] == 1
    ratio = np.linalg.norm(layer["k"][0, ~aud], axis=1).mean() / \
        np.linalg.norm(layer["k"][0, aud], axis=1).mean()
    assert 2.7 < ratio < 3.3


def test_stream_chunks_ar1_and_layout():
    src = synth.StreamSource("small-stream")
    sp = src.spec
    fv, fa = sp["frame_v"], sp["frame_a"]
    c0, c1 = src.chunk(0), src.chunk(1)
    assert len(c0) == sp["n_layers"]
    lay0, lay1 = c0[0], c1[0]
    assert lay0["q"].shape == (sp["h_q"], src.chunk_len, sp["d"])
    assert lay0["k"].shape == (sp["h_kv"], src.chunk_len, sp["d"])
    np.testing.assert_array_equal(lay0["modality"][:fv], 0)
    np.testing.assert_array_equal(lay0["modality"][fv:fv + fa], 1)
    # bf16-representable values
    np.testing.assert_array_equal(synth.round_to_bf16(lay0["k"]), lay0["k"])
    # neighbouring frames at the same spatial slot are correlated by rho,
    # across the chunk boundary too; audio rows are not
    first = lay0["k"][:, :fv].ravel()
    second = lay0["k"][:, fv + fa:2 * fv + fa].ravel()
    assert abs(np.corrcoef(first, second)[0, 1] - sp["rho"]) < 0.02
    last = lay0["k"][:, (sp["n_frames"] - 1) * (fv + fa):(sp["n_frames"] - 1) * (fv + fa) + fv].ravel()
    assert abs(np.corrcoef(last, lay1["k"][:, :fv].ravel())[0, 1] - sp["rho"]) < 0.02
    assert abs(np.corrcoef(lay0["k"][:, fv:fv + fa].ravel(), lay0["k"][:, 2 * fv + fa:2 * fv + 2 * fa].ravel())[0, 1]) < 0.05
    assert abs(lay1["v"][:, :fv].std() - 1.0) < 0.05
    # deterministic, generated in order only
    again = synth.StreamSource("small-stream")
    np.testing.assert_array_equal(again.chunk(0)[2]["v"], c0[2]["v"])
    with pytest.raises(ValueError):
        again.chunk(2)


def test_synthetic_scores_ranges():
    mods = [synth.modality_mask(30, 10, 2, 20, 5), synth.modality_mask(100, 20, 1, 8, 8)]
    a, s = synth.make_scores(mods, 3, seed=1)
    for ai, si, m in zip(a, s, mods):
        assert ai.shape == si.shape == (3, len(m))
        assert ai.dtype == si.dtype == np.float32
        assert (ai >= 0).all() and (ai == 0).any()
        assert (np.abs(si) <= 1).all() and (si > 0.99).any()
