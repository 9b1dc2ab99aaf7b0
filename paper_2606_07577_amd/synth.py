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
    uniformly chosen earlier visual row, for K and V of every KV head.
    Returns the (source, copy) row pairs."""
    n_vis = len(visual_rows)
    n_dup = int(round(frac * n_vis))
    pairs = []
    if n_dup == 0 or n_vis < 2:
        return pairs
    chosen = np.sort(rng.choice(np.arange(1, n_vis), size=min(n_dup, n_vis - 1), replace=False))
    for t in chosen:
        src = visual_rows[rng.integers(0, t)]
        dst = visual_rows[t]
        k[:, dst] = k[:, src] + noise * rng.standard_normal(k[:, dst].shape, dtype=np.float32)
        v[:, dst] = v[:, src] + noise * rng.standard_normal(v[:, dst].shape, dtype=np.float32)
        pairs.append((int(src), int(dst)))
    return pairs


def make_layer(seed, *, h_q, h_kv, d, n_cache_v, n_cache_a, n_frames, frame_v, frame_a,
               dup_frac=0.0, dup_noise=0.05, head_scale=None, audio_key_std=1.0,
               sm_scale=None, dtype="bf16", q_std=1.0, hidden_dim=0):
    """One layer's working set: q [H_q, C, d], k and v [H_kv, N, d], modality [N];
    with hidden_dim, also hidden states h [N, hidden_dim] ~ N(0, 1) in which
    the near-duplicate rows of K and V are noisy copies too (drawn from a
    stream of their own, so q, k and v do not depend on hidden_dim)."""
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
    pairs = _plant_near_duplicates(rng, k, v, np.flatnonzero(~audio), dup_frac, dup_noise)
    if head_scale is not None:
        lo, hi = head_scale
        k *= rng.uniform(lo, hi, size=(h_kv, 1, 1)).astype(np.float32)
        v *= rng.uniform(lo, hi, size=(h_kv, 1, 1)).astype(np.float32)
    h = None
    if hidden_dim:
        hrng = np.random.default_rng([*np.atleast_1d(seed).tolist(), 4093])
        h = hrng.standard_normal((n, hidden_dim), dtype=np.float32)
        for src, dst in pairs:
            h[dst] = h[src] + dup_noise * hrng.standard_normal(hidden_dim, dtype=np.float32)
    if dtype == "bf16":
        q, k, v = round_to_bf16(q), round_to_bf16(k), round_to_bf16(v)
        h = None if h is None else round_to_bf16(h)
    elif dtype != "f32":
        raise ValueError(dtype)
    out = {
        "q": q, "k": k, "v": v, "modality": modality, "n_cache": n_cache,
        "sm_scale": float(1.0 / math.sqrt(d)) if sm_scale is None else float(sm_scale),
        "dtype": dtype,
    }
    if h is not None:
        out["h"] = h
    return out


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
    "qwen7b-layer-6144-hidden": dict(
        desc="the 6144-token Qwen-7B-shaped layer with hidden states of width 3584 (Qwen2.5-7B's "
             "d_model) carrying the same near-duplicates; redundancy from them (Eq. 7 as printed), "
             "one index set per layer",
        n_layers=1, h_q=28, h_kv=4, d=128, n_cache_v=3072, n_cache_a=1024, n_frames=4,
        frame_v=384, frame_a=128, dup_frac=0.30, head_scale=(0.5, 2.0), audio_key_std=1.0,
        temperature=None, dtype="bf16", total_budget=4096, seed=1, hidden_dim=3584),
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
            sm_scale=1.0 / (taus[l] * math.sqrt(spec["d"])), dtype=spec["dtype"],
            hidden_dim=spec.get("hidden_dim", 0)))
    return out


def tokens_per_step(name):
    spec = WORKLOADS[name]
    n = spec["n_cache_v"] + spec["n_cache_a"] + spec["n_frames"] * (spec["frame_v"] + spec["frame_a"])
    return spec["n_layers"] * n


# ---------------------------------------------------------------------------
# Streams: the step after every chunk, caches carried from step to step
# ---------------------------------------------------------------------------

# Each chunk is `n_frames` frames of [frame_v visual | frame_a audio] rows.
# Visual K and V follow an AR(1) process over the global frame index, per
# (layer, KV head, spatial slot p in 0..frame_v-1):
#     x_f = rho x_{f-1} + sqrt(1 - rho^2) eps_f,   x_0 ~ N(0, 1),
# so every frame is N(0, 1) and neighbouring frames are correlated by rho.
# Audio K, V and the chunk queries are i.i.d. N(0, 1).  The stream starts
# from empty caches.
STREAMS = {
    "qwen7b-stream-64x28": dict(
        desc="64 chunks through 28 layers, 28 query / 4 KV heads, head_dim 128, bf16; each chunk "
             "4 frames of 384 visual + 128 audio tokens; visual K/V AR(1) over frames (rho 0.9); "
             "softmax temperature U(0.3,3) per layer; total budget 28x4096",
        n_layers=28, h_q=28, h_kv=4, d=128, n_chunks=64, n_frames=4, frame_v=384, frame_a=128,
        rho=0.9, temperature=(0.3, 3.0), dtype="bf16", total_budget=28 * 4096, seed=4),
    "small-stream": dict(
        desc="10 chunks through 3 layers, 8 query / 2 KV heads, head_dim 128, bf16; each chunk "
             "2 frames of 96 visual + 32 audio tokens; AR(1) rho 0.9; total budget 3x256",
        n_layers=3, h_q=8, h_kv=2, d=128, n_chunks=10, n_frames=2, frame_v=96, frame_a=32,
        rho=0.9, temperature=(0.3, 3.0), dtype="bf16", total_budget=3 * 256, seed=5),
}


class StreamSource:
    """The chunks of a named stream, generated in order.

    backend "numpy": host float32 arrays (bf16-rounded for bf16 streams).
    backend "torch": tensors on `device` in the stream's dtype, drawn with
    torch's generator (other values than the numpy backend, same recipe).
    chunk(t) must be called for t = 0, 1, 2, ... in order; it returns one
    dict per layer with q [H_q, C, d], k and v [H_kv, C, d], modality [C]
    and sm_scale.
    """

    def __init__(self, name, backend="numpy", device="cuda", **overrides):
        spec = dict(STREAMS[name])
        spec.update(overrides)
        self.spec = spec
        self.backend = backend
        self.device = device
        self.taus = layer_temperatures(spec)
        self.modality = modality_mask(0, 0, spec["n_frames"], spec["frame_v"], spec["frame_a"])
        self.chunk_len = len(self.modality)
        self._state = [None] * spec["n_layers"]   # last visual frame (k, v) per layer
        self._next = 0

    def sm_scale(self, l):
        return 1.0 / (self.taus[l] * math.sqrt(self.spec["d"]))

    def chunk(self, t):
        if t != self._next:
            raise ValueError(f"chunks are generated in order: expected {self._next}, got {t}")
        self._next += 1
        return [self._layer_chunk(t, l) for l in range(self.spec["n_layers"])]

    def _layer_chunk(self, t, l):
        sp = self.spec
        h_q, h_kv, d = sp["h_q"], sp["h_kv"], sp["d"]
        nf, fv, fa = sp["n_frames"], sp["frame_v"], sp["frame_a"]
        rho = sp["rho"]
        c = self.chunk_len
        if self.backend == "numpy":
            rng = np.random.default_rng([sp["seed"], t, l])
            normal = lambda *shape: rng.standard_normal(shape, dtype=np.float32)
            empty = lambda *shape: np.empty(shape, dtype=np.float32)
        else:
            import torch
            g = torch.Generator(device=self.device)
            g.manual_seed((sp["seed"] * 1_000_003 + t) * 1009 + l)
            normal = lambda *shape: torch.randn(shape, generator=g, device=self.device, dtype=torch.float32)
            empty = lambda *shape: torch.empty(shape, device=self.device, dtype=torch.float32)
        q = normal(h_q, c, d)
        k, v = empty(h_kv, c, d), empty(h_kv, c, d)
        innov = math.sqrt(1.0 - rho * rho)
        state = self._state[l]
        for f in range(nf):
            base = f * (fv + fa)
            if state is None:
                kf, vf = normal(h_kv, fv, d), normal(h_kv, fv, d)
            else:
                kf = rho * state[0] + innov * normal(h_kv, fv, d)
                vf = rho * state[1] + innov * normal(h_kv, fv, d)
            state = (kf, vf)
            k[:, base:base + fv], v[:, base:base + fv] = kf, vf
            k[:, base + fv:base + fv + fa] = normal(h_kv, fa, d)
            v[:, base + fv:base + fv + fa] = normal(h_kv, fa, d)
        self._state[l] = state
        if self.backend == "numpy":
            if sp["dtype"] == "bf16":
                q, k, v = round_to_bf16(q), round_to_bf16(k), round_to_bf16(v)
            modality = self.modality.copy()
        else:
            import torch
            td = torch.bfloat16 if sp["dtype"] == "bf16" else torch.float32
            q, k, v = q.to(td), k.to(td), v.to(td)
            modality = torch.from_numpy(self.modality).to(self.device)
        return {"q": q, "k": k, "v": v, "modality": modality, "sm_scale": self.sm_scale(l),
                "dtype": sp["dtype"]}


def make_scores(modalities, h_kv, seed, group_queries=2048 * 7):
    """Synthetic per-layer importance a [H_kv, N] and redundancy s [H_kv, N]
    (float32) for driving the allocation and selection stages on their own.

    a: log-normal with a per-layer spread U(0.3, 3) (so the normalised
    entropies differ between layers), scaled to sum to `group_queries` per
    head like a real column sum; a few exact zeros.  s: 70% of rows
    N(0.1, 0.15), 30% near-duplicates 1 - LogUniform(1e-3, 1e-1), clipped to
    [-1, 1]; a few exact ties of a and s between rows.
    """
    rng = np.random.default_rng([seed, 31337])
    a_out, s_out = [], []
    for mod in modalities:
        n = len(mod)
        spread = rng.uniform(0.3, 3.0)
        a = np.exp(spread * rng.standard_normal((h_kv, n)))
        a *= group_queries / a.sum(axis=1, keepdims=True)
        a[:, rng.choice(n, size=max(1, n // 500), replace=False)] = 0.0
        s = 0.1 + 0.15 * rng.standard_normal((h_kv, n))
        dup = rng.random((h_kv, n)) < 0.3
        s[dup] = 1.0 - np.exp(rng.uniform(np.log(1e-3), np.log(1e-1), size=dup.sum()))
        s = np.clip(s, -1.0, 1.0)
        twins = rng.choice(n, size=(max(1, n // 200), 2), replace=True)
        a[:, twins[:, 1]] = a[:, twins[:, 0]]
        s[:, twins[:, 1]] = s[:, twins[:, 0]]
        a_out.append(a.astype(np.float32))
        s_out.append(s.astype(np.float32))
    return a_out, s_out
