"""Seeded synthetic inputs shaped like streaming audio-visual KV caches.

This module only draws random numbers and lays them out; it holds none of
the compression method's arithmetic.  The same arrays feed the HIP library
and the CPU oracle.  Values are float32 arrays; for the bf16 workloads every
value is already rounded (round-to-nearest-even) to a bf16-representable
number, so a cast to bfloat16 is exact.

Working-set row layout of one layer (the order of Eq. 3 in the paper: the
retained caches, then the new chunk):

    [cache visual (n_cache_v) | cache audio (n_cache_a) | chunk frames]

and every chunk frame is `frame_v` visual rows followed by `frame_a` audio
rows.  modality[j] is 0 for visual and 1 for audio.
"""
from __future__ import annotations

import math

import numpy as np

VISUAL = 0
AUDIO = 1


def round_to_bf16(x: np.ndarray) -> np.ndarray:
    """float32 -> nearest bf16 value (ties to even), returned as float32."""
    u = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32)
    lsb = (u >> np.uint32(16)) & np.uint32(1)
    r = (u + np.uint32(0x7FFF) + lsb) & np.uint32(0xFFFF0000)
    return r.view(np.float32)


def modality_mask(n_cache_v, n_cache_a, n_frames, frame_v, frame_a):
    frame = np.concatenate([np.full(frame_v, VISUAL), np.full(frame_a, AUDIO)])
    return np.concatenate([
        np.full(n_cache_v, VISUAL), np.full(n_cache_a, AUDIO), np.tile(frame, n_frames)
    ]).astype(np.uint8)


def _plant_near_duplicates(rng, k, v, visual_rows, frac, noise):
    """Make `frac` of the visual rows (never the first) noisy copies of a
    uniformly chosen earlier visual row, for K and V of every KV head."""
    n_vis = len(visual_rows)
    n_dup = int(round(frac * n_vis))
    if n_dup == 0 or n_vis < 2:
        return
    chosen = np.sort(rng.choice(np.arange(1, n_vis), size=min(n_dup, n_vis - 1), replace=False))
    for t in chosen:
        src = visual_rows[rng.integers(0, t)]
        dst = visual_rows[t]
        k[:, dst] = k[:, src] + noise * rng.standard_normal(k[:, dst].shape, dtype=np.float32)
        v[:, dst] = v[:, src] + noise * rng.standard_normal(v[:, dst].shape, dtype=np.float32)


def make_layer(seed, *, h_q, h_kv, d, n_cache_v, n_cache_a, n_frames, frame_v, frame_a,
               dup_frac=0.0, dup_noise=0.05, head_scale=None, audio_key_std=1.0,
               sm_scale=None, dtype="bf16", q_std=1.0):
    """One layer's working set: q [H_q, C, d], k and v [H_kv, N, d], modality [N]."""
    rng = np.random.default_rng(seed)
    modality = modality_mask(n_cache_v, n_cache_a, n_frames, frame_v, frame_a)
    n = len(modality)
    n_cache = n_cache_v + n_cache_a
    c = n - n_cache
    q = q_std * rng.standard_normal((h_q, c, d), dtype=np.float32)
    k = rng.standard_normal((h_kv, n, d), dtype=np.float32)
    v = rng.standard_normal((h_kv, n, d), dtype=np.float32)
    audio = modality == AUDIO
    if audio_key_std != 1.0:
        k[:, audio] *= np.float32(audio_key_std)
    _plant_near_duplicates(rng, k, v, np.flatnonzero(~audio), dup_frac, dup_noise)
    if head_scale is not None:
        lo, hi = head_scale
        k *= rng.uniform(lo, hi, size=(h_kv, 1, 1)).astype(np.float32)
        v *= rng.uniform(lo, hi, size=(h_kv, 1, 1)).astype(np.float32)
    if dtype == "bf16":
        q, k, v = round_to_bf16(q), round_to_bf16(k), round_to_bf16(v)
    elif dtype != "f32":
        raise ValueError(dtype)
    return {
        "q": q, "k": k, "v": v, "modality": modality, "n_cache": n_cache,
        "sm_scale": float(1.0 / math.sqrt(d)) if sm_scale is None else float(sm_scale),
        "dtype": dtype,
    }


# The measured and tested workloads.  Chunks are laid out as frames of
# [visual block, audio block]; caches not given a split take cfg 1's 3:1.
WORKLOADS = {
    "tiny-f32-640": dict(
        desc="1 layer, 8 query / 2 KV heads, head_dim 64, fp32, cache 512 (384 v, 128 a) + "
             "chunk 128 (96 v, 32 a), 25% near-duplicate visual tokens, budget 256",
        n_layers=1, h_q=8, h_kv=2, d=64, n_cache_v=384, n_cache_a=128, n_frames=2,
        frame_v=48, frame_a=16, dup_frac=0.25, head_scale=None, audio_key_std=1.0,
        temperature=None, dtype="f32", total_budget=256, seed=0),
    "qwen7b-layer-6144": dict(
        desc="1 layer, 28 query / 4 KV heads, head_dim 128, bf16, cache 4096 (3072 v, 1024 a) + "
             "chunk 2048 (1536 v, 512 a), per-head K/V scale U(0.5,2), 30% near-duplicate "
             "visual tokens, budget 4096",
        n_layers=1, h_q=28, h_kv=4, d=128, n_cache_v=3072, n_cache_a=1024, n_frames=4,
        frame_v=384, frame_a=128, dup_frac=0.30, head_scale=(0.5, 2.0), audio_key_std=1.0,
        temperature=None, dtype="bf16", total_budget=4096, seed=1),
    "qwen7b-28layer-6144": dict(
        desc="28 layers of the 6144-token Qwen-7B-shaped layer, per-layer softmax temperature "
             "U(0.3,3), budget 28x4096 split by AVBA",
        n_layers=28, h_q=28, h_kv=4, d=128, n_cache_v=3072, n_cache_a=1024, n_frames=4,
        frame_v=384, frame_a=128, dup_frac=0.30, head_scale=(0.5, 2.0), audio_key_std=1.0,
        temperature=(0.3, 3.0), dtype="bf16", total_budget=28 * 4096, seed=2),
    "qwen7b-longcache-40960": dict(
        desc="1 layer, 28 query / 4 KV heads, head_dim 128, bf16, cache 32768 (24576 v, 8192 a) "
             "+ chunk 8192 (6144 v, 2048 a), audio keys 3x smaller norm, 30% near-duplicate "
             "visual tokens, budget 32768",
        n_layers=1, h_q=28, h_kv=4, d=128, n_cache_v=24576, n_cache_a=8192, n_frames=16,
        frame_v=384, frame_a=128, dup_frac=0.30, head_scale=None, audio_key_std=1.0 / 3.0,
        temperature=None, dtype="bf16", total_budget=32768, seed=3),
}


def layer_temperatures(spec):
    """Per-layer softmax temperature tau_l (None -> all 1)."""
    if spec["temperature"] is None:
        return [1.0] * spec["n_layers"]
    rng = np.random.default_rng([spec["seed"], 7919])
    lo, hi = spec["temperature"]
    return [float(t) for t in rng.uniform(lo, hi, size=spec["n_layers"])]


def make_workload(name, layers=None, **overrides):
    """All (or the listed) layers of a named workload as a list of layer dicts."""
    spec = dict(WORKLOADS[name])
    spec.update(overrides)
    taus = layer_temperatures(spec)
    keep = range(spec["n_layers"]) if layers is None else layers
    out = []
    for l in keep:
        out.append(make_layer(
            [spec["seed"], l], h_q=spec["h_q"], h_kv=spec["h_kv"], d=spec["d"],
            n_cache_v=spec["n_cache_v"], n_cache_a=spec["n_cache_a"],
            n_frames=spec["n_frames"], frame_v=spec["frame_v"], frame_a=spec["frame_a"],
            dup_frac=spec["dup_frac"], head_scale=spec["head_scale"],
            audio_key_std=spec["audio_key_std"],
            sm_scale=1.0 / (taus[l] * math.sqrt(spec["d"])), dtype=spec["dtype"]))
    return out


def tokens_per_step(name):
    spec = WORKLOADS[name]
    n = spec["n_cache_v"] + spec["n_cache_a"] + spec["n_frames"] * (spec["frame_v"] + spec["frame_a"])
    return spec["n_layers"] * n
