#!/usr/bin/env python3
"""Throughput of the OmniMem per-chunk KV-cache compression step on one MI355X.

One step = the four stages of the C ABI (importance score, redundancy,
AVBA allocation, select + compact) over one synthetic working set whose
inputs are already resident in HBM.  The metric is KV tokens entering the
step per second, summed over layers.  Prints one JSON line.
"""
import argparse
import json
import math
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

METRIC = "KV tokens compressed/sec per layer-step; % MFMA peak (score+Gram), % HBM (top-k+compact)"
PEAK_HBM_GBS = 8000.0                                   # MI355X HBM3E
PEAK_MFMA_TFLOPS = {"bf16": 2500.0, "f32": 157.3}       # dense MFMA

# HBM bytes per launch from two rocprofv3 counter passes (FETCH_SIZE, then
# WRITE_SIZE, KiB per dispatch), each divided by what that counter reads for a
# plain 1 GiB device-to-device copy (FETCH_SIZE 0.5x, WRITE_SIZE 1.0x), with
# the SHA-256 of the code of the library sources the counters were taken on
# (comments and blank lines left out).  A code change makes the figures
# stale: the roofline then reports traffic null.
KERNEL_SOURCES = ["include/omnimem.h"] + [f"paper_2606_07577_amd/csrc/{f}" for f in (
    "common.h", "api.hip", "score.hip", "redundancy.hip", "allocate.hip", "select.hip")]
MEASURED_TRAFFIC = {
    "qwen7b-stream-64x28": {
        "sources_sha256": "24c825019fb7279f0410ec26c325d4a26aea536854ca8f7aa8afde88e6a5ded8",
        "append_chunk": 235384164, "lse_pass": 604350999, "lse_merge": 19381020, "colsum_pass": 622659771,
        "head_sum": 21864299, "lists_norms": 181314004, "gram_sym": 816413190, "gram_finish": 6206188,
        "avba_partials": 6072666, "avba_allocate": 181106, "psi_topk_reg": 20871092,
        "stage_moved_back": 15224527, "gather_inplace": 417904305,
    },
    "qwen7b-28layer-6144": {
        "sources_sha256": "24c825019fb7279f0410ec26c325d4a26aea536854ca8f7aa8afde88e6a5ded8",
        "lse_pass": 608507806, "lse_merge": 19381186, "colsum_pass": 613571541, "head_sum": 22237014,
        "lists_norms": 184685541, "gram_sym": 823118569, "gram_finish": 6248350, "avba_partials": 6110176,
        "avba_allocate": 123965, "psi_topk_reg": 14505207, "gather_compact": 471744325,
    },
    "qwen7b-layer-6144": {
        "sources_sha256": "24c825019fb7279f0410ec26c325d4a26aea536854ca8f7aa8afde88e6a5ded8",
        "lse_pass": 31056374, "lse_merge": 1738778, "colsum_pass": 33076993, "head_sum": 1460231,
        "lists_norms": 6721705, "gram_sym": 14042062, "gram_finish": 245756, "avba_partials": 331903,
        "avba_allocate": 36191, "psi_topk_reg": 697023, "gather_compact": 16881639,
    },
    "qwen7b-layer-6144-hidden": {
        "sources_sha256": "24c825019fb7279f0410ec26c325d4a26aea536854ca8f7aa8afde88e6a5ded8",
        "lse_pass": 31055225, "lse_merge": 1738710, "colsum_pass": 33082548, "head_sum": 1460345,
        "modality_lists": 65832, "hidden_norms": 44175417, "gram_wide": 188173558, "hidden_finish": 138239,
        "avba_partials": 331903, "avba_allocate": 36191, "layer_inputs": 272514, "psi_topk_reg": 227003,
        "gather_compact": 16881708, "gather_hidden": 58879398,
    },
    "qwen7b-longcache-40960": {
        "sources_sha256": "24c825019fb7279f0410ec26c325d4a26aea536854ca8f7aa8afde88e6a5ded8",
        "lse_pass": 5085468639, "lse_merge": 3850240, "colsum_pass": 380252009, "head_sum": 5419069,
        "lists_norms": 44044125, "gram_sym": 947909492, "gram_finish": 1499112, "avba_partials": 1492173,
        "avba_allocate": 53599, "topk_hist": 2205441, "topk_bin": 1948912, "topk_emit": 2727622,
        "gather_compact": 134783809,
    },
}


def _code_only(text):
    """The source without its comments and blank lines: what the counters
    depend on is the code, so a comment edit does not make them stale."""
    out, i, n, quote = [], 0, len(text), None
    while i < n:
        c = text[i]
        if quote:
            out.append(c)
            if c == "\\" and i + 1 < n:
                out.append(text[i + 1])
                i += 2
                continue
            if c == quote:
                quote = None
            i += 1
        elif c in "\"'":
            quote = c
            out.append(c)
            i += 1
        elif text.startswith("//", i):
            j = text.find("\n", i)
            i = n if j < 0 else j
        elif text.startswith("/*", i):
            j = text.find("*/", i + 2)
            i = n if j < 0 else j + 2
            out.append(" ")
        else:
            out.append(c)
            i += 1
    return "\n".join(line.rstrip() for line in "".join(out).split("\n") if line.strip())


def sources_sha256():
    import hashlib
    h = hashlib.sha256()
    for rel in KERNEL_SOURCES:
        with open(os.path.join(ROOT, rel), encoding="utf-8") as f:
            h.update(_code_only(f.read()).encode())
    return h.hexdigest()


def measured_traffic(workload, kernel):
    rec = MEASURED_TRAFFIC.get(workload)
    if rec is None or kernel not in rec or rec["sources_sha256"] != sources_sha256():
        return None
    return rec[kernel]


def parse_args():
    p = argparse.ArgumentParser(description=__doc__)
    p.add_argument("--gpus", type=int, default=1)
    p.add_argument("--steps", type=int, default=None,
                   help="timed steps (default: every chunk of a stream, 50 for a fixed working set)")
    p.add_argument("--warmup", type=int, default=5)
    p.add_argument("--workload", default="qwen7b-stream-64x28",
                   help="a stream (default: 64 chunks through 28 layers) or a fixed working set")
    p.add_argument("--out-of-place", action="store_true",
                   help="streams: keep two cache buffers per layer and compact from one into the other "
                        "instead of compacting in place")
    p.add_argument("--no-cpu-baseline", action="store_true")
    p.add_argument("--offline-budgets", action="store_true",
                   help="fix the layer budgets in advance from a calibration (end of Sec. 3.2): static "
                        "workloads calibrate on their own step, streams on their warmup chunks; the timed "
                        "steps only split the fixed budgets")
    p.add_argument("--sim", choices=["max", "adj"], default=None,
                   help="redundancy form: all-pairs maximum (default on values) or the adjacent form of Eq. 7 "
                        "(default on hidden states)")
    p.add_argument("--shared-selection", action="store_true",
                   help="keep one index set per layer (Eqs. 4-5), ranked by the importance summed and the "
                        "redundancy averaged over the KV heads")
    p.add_argument("--no-graph", dest="graph", action="store_false",
                   help="time the four calls launched on the stream instead of replays of one HIP graph of "
                        "the whole step")
    p.add_argument("--lse-given", action="store_true",
                   help="take each layer's log-sum-exp as an input, as the model's chunk prefill attention "
                        "produces it (Eq. 1): the step then runs without the LSE pass")
    p.add_argument("--roof-probe", action="store_true",
                   help="only measure the instruction-mix ceiling of the score passes (MFMA alone, exp2 alone, "
                        "the passes' MFMA/exp2/FMA/add mix with and without LDS fragment reads) and exit")
    p.add_argument("--no-roof-probe", action="store_true",
                   help="leave the instruction-mix ceiling out of the bench line")
    p.add_argument("--copy-calibration", type=int, default=0, metavar="MIB",
                   help="only run 5 device-to-device copies of MIB MiB each (reference kernel for "
                        "scaling the FETCH_SIZE / WRITE_SIZE counters) and exit")
    return p.parse_args()


def copy_calibration(mib):
    """Plain copies of known size: each reads and writes exactly `mib` MiB."""
    import torch
    n = mib * (1 << 20) // 4
    src = torch.ones(n, dtype=torch.float32, device="cuda")
    dst = torch.empty_like(src)
    for _ in range(5):
        dst.copy_(src)
    torch.cuda.synchronize()
    print(json.dumps({"copy_bytes_read": n * 4, "copy_bytes_written": n * 4, "launches": 5}))


def roof_probe(torch):
    """Throughput of the score passes' instruction mix on this GPU, from the
    probe kernels of libomnimem_probe.so (registers only, plus LDS reads in
    one of them).  Returns MFMA-flop rates as fractions of the bf16 peak:
    MFMA alone, and the per-MFMA mix of the passes (one 32x32x16 bf16 MFMA,
    two exp2, two FMA, two adds) with and without its LDS fragment reads;
    the mix is the ceiling of a pass that does this work per MFMA.  Also the
    Gram pass's mix (one MFMA, two cosines: four multiplies, two running
    maxima, one v_max3; LDS fragments and a barrier per tile)."""
    import ctypes

    from paper_2606_07577_amd import build
    lib = ctypes.CDLL(build.PROBE_LIB)
    lib.omnimem_probe_run.argtypes = [ctypes.c_int, ctypes.c_int, ctypes.c_int, ctypes.c_void_p, ctypes.c_int,
                                      ctypes.c_void_p]
    lib.omnimem_probe_run.restype = ctypes.c_int
    cus = torch.cuda.get_device_properties(0).multi_processor_count
    out = torch.zeros(1, device="cuda")
    stream = torch.cuda.current_stream()
    mfma_flop = 32 * 32 * 16 * 2

    def best_ms(kind, blocks, iters, reps=5):
        best = float("inf")
        for _ in range(reps):
            a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            a.record(stream)
            rc = lib.omnimem_probe_run(kind, blocks, iters, ctypes.c_void_p(out.data_ptr()), 0,
                                       ctypes.c_void_p(stream.cuda_stream))
            b.record(stream)
            if rc != 0:
                raise RuntimeError(f"probe {kind}: hip error {rc}")
            torch.cuda.synchronize()
            best = min(best, a.elapsed_time(b))
        return best

    res = {"cus": cus}
    for waves in (2, 4):                       # waves per SIMD (workgroups of 4 waves per compute unit)
        blocks = cus * waves
        ms = best_ms(0, blocks, 20000)
        res[f"mfma_only_{waves}w"] = blocks * 4 * 4 * 20000 * mfma_flop / (ms / 1e3) / 1e12
        ms = best_ms(1, blocks, 20000)
        res[f"exp2_per_ns_{waves}w"] = blocks * 4 * 64 * 16 * 20000 / (ms * 1e6)
    for kind, name in ((2, "mix"), (3, "mix_lds"), (4, "mix_lds_barrier"), (5, "gram_mix")):
        blocks = cus * 2                        # the passes' occupancy: two 4-wave workgroups per compute unit
        ms = best_ms(kind, blocks, 2500)
        res[name] = blocks * 4 * 32 * 2500 * mfma_flop / (ms / 1e3) / 1e12
    peak = PEAK_MFMA_TFLOPS["bf16"]
    out_d = {"unit": "TFLOP/s of MFMA work", "peak": peak,
             "mfma_only": round(max(res["mfma_only_2w"], res["mfma_only_4w"]), 1),
             "mix": round(res["mix"], 1), "mix_lds": round(res["mix_lds"], 1),
             "mix_lds_barrier": round(res["mix_lds_barrier"], 1), "gram_mix": round(res["gram_mix"], 1),
             "exp2_per_ns": round(max(res["exp2_per_ns_2w"], res["exp2_per_ns_4w"]), 1)}
    for k in ("mfma_only", "mix", "mix_lds", "mix_lds_barrier", "gram_mix"):
        out_d[k + "_frac"] = round(out_d[k] / peak, 4)
    return out_d


def layer_work(h_q, c, n_cache, h_kv, n, d, elt, k_v, k_a, m, causal=True):
    """Algorithmic units of one layer in one step: score flops (per pass),
    Gram flops, top-k bytes read (a, s, modality) and written (idx),
    compaction bytes."""
    pairs = c * n_cache + c * (c + 1) // 2 if causal else c * n
    score = 2 * d * h_q * pairs
    gram = h_kv * (k_v * (k_v - 1) + k_a * (k_a - 1)) * d   # K(K-1)/2 pairs x 2d per segment
    topk_in = h_kv * n * (4 + 4) + n                         # a, s, modality in
    topk_out = 4 * h_kv * m                                   # idx out
    compact = 2 * 2 * h_kv * m * d * elt                      # K and V rows, read + write
    return score, gram, topk_in, topk_out, compact


# The kernels of the two stages the fractions cover: the MFMA contractions
# (score and Gram) and the top-k with the compaction (every ranking path,
# the layer-shared pre-reduction and both gathers; the staging copy and the
# pre-reduction count in time only).
SCORE_GRAM_KERNELS = ["lse_pass", "colsum_pass", "gram_pass", "gram_sym", "gram_wide"]
TOPK_COMPACT_KERNELS = ["layer_inputs", "psi_topk", "psi_topk_reg", "topk_hist", "topk_bin", "topk_emit",
                        "gather_compact", "stage_moved_back", "gather_inplace"]


def work_table(score, gram, topk_in, topk_out, compact):
    """Per-launch algorithmic units of each counted kernel (the split top-k's
    inputs are read by topk_hist and its output written by topk_emit)."""
    return {"lse_pass": ("mfma", score), "colsum_pass": ("mfma", score), "gram_pass": ("mfma", gram),
            "gram_sym": ("mfma", gram),
            "gram_wide": ("mfma", gram),
            "gather_compact": ("hbm", compact), "gather_inplace": ("hbm", compact),
            "psi_topk": ("hbm", topk_in + topk_out), "psi_topk_reg": ("hbm", topk_in + topk_out),
            "topk_hist": ("hbm", topk_in), "topk_emit": ("hbm", topk_out)}


def static_work(layers, budgets, hidden_dim=0):
    tot = [0, 0, 0, 0, 0]
    for lay, (mv, ma) in zip(layers, budgets):
        h_q, c, d = lay["q"].shape
        h_kv, n, _ = lay["k"].shape
        mod = lay["modality"]
        k_v, k_a = int((mod == 0).sum()), int((mod == 1).sum())
        w = layer_work(h_q, c, lay["n_cache"], h_kv, n, d, 2 if lay["dtype"] == "bf16" else 4,
                       k_v, k_a, int(mv) + int(ma))
        if hidden_dim:  # the Gram on the layer's hidden states: one per layer, d_model wide
            w = (w[0], (k_v * (k_v - 1) + k_a * (k_a - 1)) * hidden_dim) + tuple(w[2:])
        tot = [x + y for x, y in zip(tot, w)]
    return work_table(*tot)


def _host_cpu():
    """Host threads available to this process and the CPU model."""
    try:
        cores = len(os.sched_getaffinity(0))
    except AttributeError:
        cores = os.cpu_count() or 1
    model = "unknown"
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    model = line.split(":", 1)[1].strip()
                    break
    except OSError:
        pass
    return cores, model


def _time_oracle(layers, budget, threads, **kw):
    import threadpoolctl

    from oracle import omnimem_oracle as orc
    with threadpoolctl.threadpool_limits(limits=threads, user_api="blas"):
        t0 = time.perf_counter()
        orc.compression_step(layers, budget, **kw)
        return time.perf_counter() - t0


def cpu_baseline(layers, spec, sample_layers=1):
    """The oracle, as it stands, on `sample_layers` layers of the same
    working sets, with every host thread available to its BLAS and again
    with one (on one layer)."""
    import numpy as np

    lays = []
    for lay in layers[:sample_layers]:
        x = dict(lay)
        for key in ("q", "k", "v", "h"):
            if key in x:
                x[key] = x[key].astype(np.float64)
        lays.append(x)
    per_layer_budget = spec["total_budget"] // spec["n_layers"]
    hidden = bool(spec.get("hidden_dim"))
    kw = dict(mode="adj" if hidden else "max", shared_selection=hidden, use_hidden=hidden)
    cores, model = _host_cpu()
    dt = _time_oracle(lays, per_layer_budget * len(lays), cores, **kw)
    dt1 = _time_oracle(lays[:1], per_layer_budget, 1, **kw)
    n = sum(int(x["k"].shape[1]) for x in lays)
    n1 = int(lays[0]["k"].shape[1])
    return {"value": n / dt, "unit": "tokens/s", "cores": cores, "kind": "oracle",
            "cpu_model": model, "one_thread_value": n1 / dt1,
            "sample": f"{len(lays)} layer(s) of {n // len(lays)} tokens of the same workload through the whole "
                      f"numpy fp64 oracle step: {dt:.1f} s wall with its BLAS on {cores} threads "
                      f"(exp, sort and the Python loops single-threaded); one layer on one thread: {dt1:.1f} s"}


def stream_sample_layers(name, t=2, n_layers=2):
    """Working sets of the first `n_layers` layers of a stream at chunk t
    while every earlier row is still kept (true up to chunk 2 at the
    headline's budget): the rows of chunks 0 .. t-1, visual rows then audio
    rows in age order, followed by chunk t.  Host arrays (numpy generator)."""
    import numpy as np

    from paper_2606_07577_amd import synth
    src = synth.StreamSource(name, n_layers=n_layers)
    past = []
    for c in range(t + 1):
        ch = src.chunk(c)
        if c < t:
            past.append(ch)
    out = []
    for l in range(n_layers):
        ks = np.concatenate([p[l]["k"] for p in past], axis=1) if past else ch[l]["k"][:, :0]
        vs = np.concatenate([p[l]["v"] for p in past], axis=1) if past else ch[l]["v"][:, :0]
        ms = np.concatenate([p[l]["modality"] for p in past]) if past else ch[l]["modality"][:0]
        order = np.concatenate([np.flatnonzero(ms == 0), np.flatnonzero(ms == 1)])
        out.append({"q": ch[l]["q"], "k": np.concatenate([ks[:, order], ch[l]["k"]], axis=1),
                    "v": np.concatenate([vs[:, order], ch[l]["v"]], axis=1),
                    "modality": np.concatenate([ms[order], ch[l]["modality"]]), "n_cache": len(order),
                    "sm_scale": ch[l]["sm_scale"], "dtype": ch[l]["dtype"]})
    return out


def run_static(args, torch):
    """K steps of one fixed working set (every step sees the same inputs)."""
    from paper_2606_07577_amd import synth
    from paper_2606_07577_amd.step import DeviceStep

    spec = synth.WORKLOADS[args.workload]
    layers = synth.make_workload(args.workload)
    options = {"shared_selection": int(args.shared_selection)}
    if spec.get("hidden_dim"):
        # redundancy from the hidden states (Eq. 7 as printed, adjacent form); their kept rows are
        # carried with the cache, which takes one index set per layer
        from paper_2606_07577_amd import omnimem as om
        options.update(sim=om.SIM_MAX if args.sim == "max" else om.SIM_ADJ, sim_source=om.SRC_HIDDEN,
                       hidden_dim=spec["hidden_dim"], shared_selection=1)
    elif args.sim == "adj":
        from paper_2606_07577_amd import omnimem as om
        options.update(sim=om.SIM_ADJ)
    step = DeviceStep(layers, spec["total_budget"], **options)
    stream = torch.cuda.current_stream()
    if args.lse_given:
        # Stand-in for the prefill's log-sum-exp: the library's own, computed
        # once before timing and then passed in as every layer's input.
        step.score(stream, lse_out=True)
        torch.cuda.synchronize()
        step.set_lse_inputs([step.lse[l, :, : int(lay["q"].shape[1])].contiguous() for l, lay in enumerate(layers)])
        torch.cuda.synchronize()
    if args.offline_budgets:
        step.score(stream, lse_out=False)
        step.redundancy(stream)
        step.ctx.omnimem_calibration_reset()
        step.calibrate(stream)
        step.calibration_budgets(stream)
        step.fixed_budgets = True
        torch.cuda.synchronize()
    print(f"[bench] workload {args.workload}: inputs resident, warmup {args.warmup}", file=sys.stderr, flush=True)
    for _ in range(args.warmup):
        step.run(stream)
    torch.cuda.synchronize()

    graph, launch = None, "stream"
    if args.graph:
        # The step's layer table is uploaded by the warmup: the captured calls
        # launch kernels only.  A capture that fails leaves the stream mode.
        try:
            graph_stream = torch.cuda.Stream()
            graph_stream.wait_stream(stream)
            with torch.cuda.stream(graph_stream):
                step.run(graph_stream)
            torch.cuda.synchronize()
            graph = torch.cuda.CUDAGraph()
            with torch.cuda.graph(graph, stream=graph_stream):
                step.run(graph_stream)
            torch.cuda.synchronize()
            with torch.cuda.stream(graph_stream):
                graph.replay()
            torch.cuda.synchronize()
            stream, launch = graph_stream, "graph replay"
        except Exception as e:  # noqa: BLE001 - report and measure the stream launches instead
            print(f"[bench] graph capture failed ({e}); timing stream launches", file=sys.stderr, flush=True)
            graph, launch = None, "stream (graph capture failed)"
            torch.cuda.synchronize()

    # Timed region: K whole steps, nothing else.
    start, stop = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    with torch.cuda.stream(stream):  # graph replays launch on the current stream
        start.record(stream)
        for _ in range(args.steps):
            if graph is not None:
                graph.replay()
            else:
                step.run(stream)
        stop.record(stream)
    torch.cuda.synchronize()
    ms = start.elapsed_time(stop) / args.steps
    tokens = sum(int(l["k"].shape[1]) for l in layers)

    # Same K steps again with per-kernel HIP events on the launch stream.
    step.ctx.omnimem_profile(True)
    torch.cuda.synchronize()
    for _ in range(args.steps):
        step.run(stream)
    torch.cuda.synchronize()
    kernels = step.ctx.omnimem_profile_report()
    step.ctx.omnimem_profile(False)
    work = static_work(layers, step.budgets.cpu().numpy(), spec.get("hidden_dim", 0))
    config = {"workload": args.workload, "layers": spec["n_layers"], "q_heads": spec["h_q"],
              "kv_heads": spec["h_kv"], "head_dim": spec["d"], "cache": spec["n_cache_v"] + spec["n_cache_a"],
              "chunk": spec["n_frames"] * (spec["frame_v"] + spec["frame_a"]), "budget": spec["total_budget"],
              "lse": "input" if args.lse_given else "computed",
              "layer_budgets": "offline" if args.offline_budgets else "per step",
              "selection": "per layer" if options["shared_selection"] else "per KV head",
              "launch": launch,
              "redundancy": ("hidden states (%d), " % spec["hidden_dim"] if spec.get("hidden_dim") else "values, ")
                            + ("all pairs" if options.get("sim", 0) == 0 else "adjacent")}
    baseline = None
    if not args.no_cpu_baseline:
        print("[bench] timing the oracle on the host", file=sys.stderr, flush=True)
        baseline = cpu_baseline(layers, spec)
    step.close()
    return ms, tokens / (ms / 1e3), kernels, work, layers[0]["dtype"], config, baseline


def run_stream(args, torch):
    """The step after each of K consecutive chunks of a stream, from empty
    caches.  All chunks are generated on the device before timing; the timed
    region holds, per chunk, the append of its K/V behind the kept rows
    (Eq. 3), the four library calls and the read-back of the budgets (the
    host waits for the budgets only; the compaction overlaps the next
    step's preparation)."""
    from paper_2606_07577_amd import synth
    from paper_2606_07577_amd.step import StreamRunner

    spec = synth.STREAMS[args.workload]
    steps = args.steps = min(args.steps or spec["n_chunks"], spec["n_chunks"])
    src = synth.StreamSource(args.workload, backend="torch")
    chunks = [src.chunk(t) for t in range(steps)]
    torch.cuda.synchronize()

    def runner(**kw):
        return StreamRunner(spec["n_layers"], spec["h_q"], spec["h_kv"], spec["d"], src.chunk_len,
                            spec["total_budget"], dtype=spec["dtype"], in_place=not args.out_of_place,
                            shared_selection=int(args.shared_selection), **kw)

    print(f"[bench] stream {args.workload}: {steps} chunks resident, warmup {args.warmup} chunks",
          file=sys.stderr, flush=True)
    warm = runner()
    warm.calibrating = args.offline_budgets
    for t in range(min(args.warmup, steps)):
        warm.push(chunks[t])
    if args.offline_budgets:
        if min(args.warmup, steps) == 0:
            print("--offline-budgets calibrates on the warmup chunks: give --warmup >= 1", file=sys.stderr)
            sys.exit(1)
        warm.freeze_budgets()
    fixed_lb = warm.layer_budgets.clone() if args.offline_budgets else None
    torch.cuda.synchronize()
    warm.close()

    def fix(r):
        if fixed_lb is not None:
            r.layer_budgets.copy_(fixed_lb)
            r.fixed = True
        return r

    # Timed region: K steps of the stream, nothing else.  The host reads a
    # step's budgets when it has described the next chunk (push without
    # wait), as a serving loop would, so its work overlaps the GPU's.
    run = fix(runner())
    stream = torch.cuda.current_stream()
    start, stop = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    start.record(stream)
    for t in range(steps):
        run.push(chunks[t], stream, wait=False)
    stop.record(stream)
    torch.cuda.synchronize()
    run.finish()
    ms = start.elapsed_time(stop) / steps
    tokens = run.tokens / steps            # working-set rows per step, summed over layers
    fallbacks = run.fallbacks
    run.close()

    # The same stream again with events around the append and the four
    # stages of every step.
    run = fix(runner(timing=True))
    for t in range(steps):
        run.push(chunks[t], stream)
    app_ms, abi_ms = run.timings()
    run.close()

    # The shapes each step saw (kept rows, audio rows, budgets), read back in
    # a pass of their own (the stream is deterministic: every pass sees the
    # same), then the stream again with per-kernel HIP events and no
    # read-back beyond the budgets push itself waits for.
    run = fix(runner())
    shapes = []
    for t in range(steps):
        n_cache = list(run.n_cache)
        k_a = [int((run.cache_modality(l) == 1).sum()) for l in range(spec["n_layers"])]
        budgets = run.push(chunks[t], stream)
        shapes.append((n_cache, k_a, [int(budgets[l].sum()) for l in range(spec["n_layers"])]))
    torch.cuda.synchronize()
    run.close()
    run = fix(runner())
    run.ctx.omnimem_profile(True)
    for t in range(steps):
        run.push(chunks[t], stream)
    torch.cuda.synchronize()
    kernels = run.ctx.omnimem_profile_report()
    run.close()
    tot = [0, 0, 0, 0, 0]
    elt = 2 if spec["dtype"] == "bf16" else 4
    for n_cache, k_a, kept in shapes:
        for l in range(spec["n_layers"]):
            ka = k_a[l] + spec["n_frames"] * spec["frame_a"]
            n = n_cache[l] + src.chunk_len
            w = layer_work(spec["h_q"], src.chunk_len, n_cache[l], spec["h_kv"], n, spec["d"], elt,
                           n - ka, ka, kept[l])
            tot = [x + y for x, y in zip(tot, w)]
    work = work_table(*[x / steps for x in tot])
    config = {"workload": args.workload, "layers": spec["n_layers"], "q_heads": spec["h_q"],
              "kv_heads": spec["h_kv"], "head_dim": spec["d"], "chunks": steps,
              "chunk": src.chunk_len, "budget": spec["total_budget"], "launch": "stream",
              "compaction": "out of place (two buffers)" if args.out_of_place else "in place (one buffer)",
              "layer_budgets": "offline" if args.offline_budgets else "per step",
              "selection": "per layer" if args.shared_selection else "per KV head"}
    extra = {"append_ms_per_step": round(app_ms / steps, 5), "stages_ms_per_step": round(abi_ms / steps, 5),
             "stages_tokens_per_s": round(tokens / (abi_ms / steps / 1e3), 1), "fallback_steps": fallbacks}
    baseline = None
    if not args.no_cpu_baseline:
        print("[bench] timing the oracle on the host", file=sys.stderr, flush=True)
        sample = stream_sample_layers(args.workload, t=2, n_layers=2)
        baseline = cpu_baseline(sample, spec, sample_layers=2)
        baseline["sample"] = ("the stream's working sets at chunk 2 (4096 kept rows + a 2048-row chunk) of layers "
                              "0 and 1; " + baseline["sample"])
    return ms, tokens / (ms / 1e3), kernels, work, spec["dtype"], config, baseline, extra


def main():
    args = parse_args()
    if args.gpus != 1:
        print(f"bench.py measures one GPU only; --gpus {args.gpus} is not supported "
              "(the step is per layer and KV head; sharding is described in the design notes)",
              file=sys.stderr)
        sys.exit(1)
    if args.copy_calibration:
        copy_calibration(args.copy_calibration)
        return
    import torch

    if args.roof_probe:
        print(json.dumps({"score_pass_ceiling": roof_probe(torch)}))
        return

    from paper_2606_07577_amd import synth
    if args.lse_given and args.workload in synth.STREAMS:
        print("--lse-given applies to the fixed working sets, not to streams", file=sys.stderr)
        sys.exit(1)
    extra = {}
    if args.workload in synth.STREAMS:
        ms, value, kernels, work, dtype, config, base, extra = run_stream(args, torch)
    else:
        if args.out_of_place:
            print("--out-of-place applies to streams", file=sys.stderr)
            sys.exit(1)
        args.steps = args.steps or 50
        ms, value, kernels, work, dtype, config, base = run_static(args, torch)
    print(f"[bench] {ms:.4f} ms/step, {value:.4g} tokens/s", file=sys.stderr, flush=True)
    per_kernel = {}
    for name, (launches, total_ms) in kernels.items():
        avg_ms = total_ms / max(launches, 1)
        entry = {"avg_us": round(avg_ms * 1e3, 3), "launches": launches}
        if name in work:
            bound, units = work[name]
            if bound == "mfma":
                ach = units / (avg_ms / 1e3) / 1e12
                entry.update(bound="mfma", achieved=ach, unit="TFLOP/s", frac=ach / PEAK_MFMA_TFLOPS[dtype])
            else:
                ach = units / (avg_ms / 1e3) / 1e9
                entry.update(bound="hbm", achieved=ach, unit="GB/s", frac=ach / PEAK_HBM_GBS)
        per_kernel[name] = entry
    dominant = max((n for n in per_kernel if n in work), key=lambda n: per_kernel[n]["avg_us"])
    dk = per_kernel[dominant]
    peak = PEAK_MFMA_TFLOPS[dtype] if dk["bound"] == "mfma" else PEAK_HBM_GBS
    roofline = {"bound": dk["bound"], "achieved": round(dk["achieved"], 3), "peak": peak, "unit": dk["unit"],
                "frac": round(dk["frac"], 4), "traffic": measured_traffic(args.workload, dominant),
                "traffic_unit": "bytes", "kernel": dominant,
                "units_per_launch": work[dominant][1], "avg_launch_us": dk["avg_us"]}

    def stage_frac(names, peak_units, scale):
        # time of every listed kernel that ran; units of those with algorithmic units (the
        # in-place staging copy moves bytes beyond the out-of-place minimum: time only)
        t = sum(per_kernel[n]["avg_us"] for n in names if n in per_kernel) / 1e6
        u = sum(work[n][1] for n in names if n in per_kernel and n in work)
        return round(u / t / scale / peak_units, 4) if t > 0 else None

    fractions = {
        "mfma_frac_score_gram": stage_frac(SCORE_GRAM_KERNELS, PEAK_MFMA_TFLOPS[dtype], 1e12),
        "hbm_frac_topk_compact": stage_frac(TOPK_COMPACT_KERNELS, PEAK_HBM_GBS, 1e9),
    }
    out = {
        "metric": METRIC, "value": round(value, 1), "unit": "tokens/s", "n_gpus": 1, "steps": args.steps,
        "warmup": args.warmup, "ms_per_step": round(ms, 5), "higher_is_better": True, "scaling": "weak",
        "vs_baseline": None, "dtype": dtype, "data": "synthetic", "config": config,
        "roofline": roofline, "fractions": fractions, "kernels": per_kernel, "cpu_baseline": base,
    }
    out.update(extra)
    if not args.no_roof_probe:
        ceiling = roof_probe(torch)
        for name in ("lse_pass", "colsum_pass"):
            if name in per_kernel and "frac" in per_kernel[name]:
                ceiling[name + "_vs_mix"] = round(per_kernel[name]["frac"] / ceiling["mix_frac"], 4)
        if "gram_sym" in per_kernel and "frac" in per_kernel["gram_sym"]:
            ceiling["gram_sym_vs_gram_mix"] = round(per_kernel["gram_sym"]["frac"] / ceiling["gram_mix_frac"], 4)
        out["score_pass_ceiling"] = ceiling
    print(json.dumps(out))


if __name__ == "__main__":
    main()
