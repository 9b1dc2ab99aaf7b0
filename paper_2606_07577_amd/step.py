"""One compression step on the GPU through the C ABI.

`DeviceStep` uploads a workload (a list of layer dicts as produced by
`synth.make_workload`) to device buffers laid out as the library expects,
owns the output buffers and runs the four stages on a stream.
"""
from __future__ import annotations

import numpy as np
import torch

from . import omnimem as om


class DeviceStep:
    def __init__(self, layers, total_budget, device="cuda", max_tokens=None, max_chunk=None, **options):
        self.device = torch.device(device)
        self.n_layers = len(layers)
        first = layers[0]
        self.dtype_name = first["dtype"]
        self.tdtype = torch.bfloat16 if self.dtype_name == "bf16" else torch.float32
        h_q, _, d = first["q"].shape
        h_kv = first["k"].shape[0]
        self.h_q, self.h_kv, self.d = h_q, h_kv, d
        self.n = [int(l["k"].shape[1]) for l in layers]
        self.n_cache = [int(l["n_cache"]) for l in layers]
        self.max_tokens = max_tokens or max(self.n)
        self.max_chunk = max_chunk or max(n - c for n, c in zip(self.n, self.n_cache))
        self.total_budget = int(total_budget)
        self.ctx = om.Context(self.n_layers, h_q, h_kv, d, self.max_tokens, self.max_chunk,
                              dtype=om.BF16 if self.dtype_name == "bf16" else om.F32, **options)
        dev, td = self.device, self.tdtype
        self.q = [torch.from_numpy(np.ascontiguousarray(l["q"])).to(dev, td) for l in layers]
        self.k = [torch.from_numpy(np.ascontiguousarray(l["k"])).to(dev, td) for l in layers]
        self.v = [torch.from_numpy(np.ascontiguousarray(l["v"])).to(dev, td) for l in layers]
        self.mod = [torch.from_numpy(np.ascontiguousarray(l["modality"])).to(dev) for l in layers]
        self.k_out = [torch.zeros_like(k) for k in self.k]
        self.v_out = [torch.zeros_like(v) for v in self.v]
        # hidden states (redundancy source of Eq. 7 as printed), when the layers carry them
        self.h = [torch.from_numpy(np.ascontiguousarray(l["h"])).to(dev, self.tdtype) if "h" in l else None
                  for l in layers]
        self.h_out = [torch.zeros_like(h) if h is not None else None for h in self.h]
        self.sm_scale = [float(l["sm_scale"]) for l in layers]
        shape = (self.n_layers, h_kv, self.max_tokens)
        self.a = torch.zeros(shape, device=dev, dtype=torch.float32)
        self.s = torch.zeros(shape, device=dev, dtype=torch.float32)
        self.idx = torch.full(shape, -1, device=dev, dtype=torch.int32)
        self.lse = torch.zeros((self.n_layers, h_q, self.max_chunk), device=dev, dtype=torch.float32)
        self.budgets = torch.zeros((self.n_layers, 2), device=dev, dtype=torch.int32)
        self.stats = torch.zeros((self.n_layers, 10), device=dev, dtype=torch.float32)
        self.layer_budgets = torch.zeros(self.n_layers, device=dev, dtype=torch.int32)
        self.fixed_budgets = False          # run() splits self.layer_budgets instead of Eq. (14)
        self.lse_in = [None] * self.n_layers
        self.descs = self._descs()

    def _descs(self):
        return [om.make_layer(self.q[l], self.k[l], self.v[l], self.mod[l], self.n_cache[l],
                              self.sm_scale[l], self.lse_in[l], self.k_out[l], self.v_out[l],
                              self.h[l], self.h_out[l])
                for l in range(self.n_layers)]

    def set_lse_inputs(self, lse_list):
        """Give each layer a caller-side log-sum-exp ([H_q, C] fp32 device tensors)."""
        self.lse_in = list(lse_list)
        self.descs = self._descs()

    # stages ---------------------------------------------------------------
    def score(self, stream=None, lse_out=True):
        self.ctx.omnimem_score(self.descs, self.a, self.lse if lse_out else None, stream)

    def redundancy(self, stream=None):
        self.ctx.omnimem_redundancy(self.descs, self.s, stream)

    def allocate(self, stream=None, a=None, s=None):
        self.ctx.omnimem_allocate(self.descs, self.a if a is None else a, self.s if s is None else s,
                                  self.total_budget, self.budgets, self.stats, stream)

    def select_compact(self, stream=None, a=None, s=None, budgets=None):
        self.ctx.omnimem_select_compact(self.descs, self.a if a is None else a, self.s if s is None else s,
                                        self.budgets if budgets is None else budgets, self.idx, stream)

    # offline budgets (calibration) ----------------------------------------
    def calibrate(self, stream=None, a=None, s=None):
        self.ctx.omnimem_calibrate(self.descs, self.a if a is None else a, self.s if s is None else s,
                                   self.stats, stream)

    def calibration_budgets(self, stream=None):
        """The calibration's layer budgets into self.layer_budgets."""
        self.ctx.omnimem_calibration_budgets(self.total_budget, self.layer_budgets, stream)

    def allocate_fixed(self, stream=None, a=None, s=None, layer_budgets=None):
        self.ctx.omnimem_allocate_fixed(self.descs, self.a if a is None else a, self.s if s is None else s,
                                        self.layer_budgets if layer_budgets is None else layer_budgets,
                                        self.budgets, self.stats, stream)

    def run(self, stream=None):
        self.score(stream, lse_out=False)
        self.redundancy(stream)
        if self.fixed_budgets:
            self.allocate_fixed(stream)
        else:
            self.allocate(stream)
        self.select_compact(stream)

    # host views -----------------------------------------------------------
    def to_device_f32(self, per_layer):
        """[L] list of [H_kv, N_l] host arrays -> a [L, H_kv, max_tokens] device tensor."""
        out = torch.zeros((self.n_layers, self.h_kv, self.max_tokens), dtype=torch.float32)
        for l, arr in enumerate(per_layer):
            out[l, :, : arr.shape[1]] = torch.from_numpy(np.asarray(arr, dtype=np.float32))
        return out.to(self.device)

    def host(self, name, l):
        t = getattr(self, name)
        if name in ("a", "s", "idx"):
            return t[l, :, : self.n[l]].cpu().numpy()
        if name == "lse":
            return t[l, :, : self.n[l] - self.n_cache[l]].cpu().numpy()
        return t[l].cpu().numpy()

    def close(self):
        self.ctx.close()


class StreamRunner:
    """The compression step after every chunk of a stream, on the GPU.

    Each layer's cache is one buffer [H_kv, cap, d] for K, one for V and a
    modality buffer [cap].  A step's working set is the buffer's first
    N = n_cache + C rows: omnimem_append writes the chunk's K/V and modality
    behind the kept rows (Eq. 3), the four stages run, and
    omnimem_select_compact moves the kept rows to the front of the same
    buffers and rewrites their modality (in place, Eqs. 2-5).  With
    in_place=False two buffers per layer alternate instead (out of place).

    The host needs each layer's kept-row count to describe the next working
    set: it copies the budgets back after the allocation stage and waits for
    that copy only, so the compaction of one step overlaps the host's
    preparation of the next.  The descriptors are ctypes arrays built once;
    a step only updates the fields that change.

    In place, kept audio rows that land behind their own row are staged in
    the context's reserve of `stage_rows` rows per (layer, KV head); there
    are never more of them than the layer's audio budget.  When a step's
    audio budget exceeds the reserve, the runner asks the library whether
    that step's compaction ran and, if it moved nothing for lack of staging
    rows, compacts out of place into temporary buffers and copies back.
    """

    def __init__(self, n_layers, h_q, h_kv, d, chunk_len, total_budget, dtype="bf16", device="cuda",
                 in_place=True, stage_rows=None, keep_working_set=False, timing=False, **options):
        self.device = torch.device(device)
        self.L, self.h_q, self.h_kv, self.d, self.C = n_layers, h_q, h_kv, d, chunk_len
        self.total_budget = int(total_budget)
        self.tdtype = torch.bfloat16 if dtype == "bf16" else torch.float32
        cfg_probe = om.Context.default_config()
        bmax = options.get("b_max_frac", cfg_probe.b_max_frac)
        self.cache_cap = int(bmax * total_budget / n_layers)   # no layer keeps more
        self.cap = self.cache_cap + chunk_len
        self.in_place = bool(in_place)
        self.stage_rows = int(stage_rows if stage_rows is not None else self.cache_cap // 2) if in_place else 0
        self.ctx = om.Context(n_layers, h_q, h_kv, d, self.cap, chunk_len,
                              dtype=om.BF16 if dtype == "bf16" else om.F32,
                              inplace_stage_rows=self.stage_rows, **options)
        dev, td = self.device, self.tdtype
        n_sets = 1 if self.in_place else 2
        self.kbuf = [[torch.zeros((h_kv, self.cap, d), device=dev, dtype=td) for _ in range(n_layers)]
                     for _ in range(n_sets)]
        self.vbuf = [[torch.zeros((h_kv, self.cap, d), device=dev, dtype=td) for _ in range(n_layers)]
                     for _ in range(n_sets)]
        self.mbuf = [[torch.zeros(self.cap, device=dev, dtype=torch.uint8) for _ in range(n_layers)]
                     for _ in range(n_sets)]
        shape = (n_layers, h_kv, self.cap)
        self.a = torch.zeros(shape, device=dev, dtype=torch.float32)
        self.s = torch.zeros(shape, device=dev, dtype=torch.float32)
        self.idx = torch.full(shape, -1, device=dev, dtype=torch.int32)
        self.budgets = torch.zeros((n_layers, 2), device=dev, dtype=torch.int32)
        self.budgets_host = torch.zeros((n_layers, 2), dtype=torch.int32, pin_memory=True)
        self.stats = torch.zeros((n_layers, 10), device=dev, dtype=torch.float32)
        self.layer_budgets = torch.zeros(n_layers, device=dev, dtype=torch.int32)
        self.calibrating = False   # each step also adds its C^(l) to the calibration
        self.fixed = False         # steps split self.layer_budgets instead of Eq. (14)
        self.cur = 0               # buffer set holding the cache (out of place: alternates)
        self.n_cache = [0] * n_layers
        self.steps = 0
        self.tokens = 0            # sum over steps and layers of the working-set size
        self.fallbacks = 0         # steps compacted out of place for lack of staging rows
        self.keep_working_set = keep_working_set
        self.working_set = None    # [L] of (k, v, modality) copies of the last step's working set
        self._layers = (om.Layer * n_layers)()
        self._chunks = (om.Chunk * n_layers)()
        self._budget_ready = torch.cuda.Event()
        self._pending, self._pending_stream = False, None   # a pushed step whose budgets are unread
        self.timing = timing       # per step: events before the append, before score, after select_compact
        self.events = []

    # buffers ------------------------------------------------------------
    def cache_k(self, l):
        """Device view of layer l's kept keys [H_kv, n_cache, d]."""
        self.finish()
        return self.kbuf[self.cur][l][:, : self.n_cache[l]]

    def cache_v(self, l):
        self.finish()
        return self.vbuf[self.cur][l][:, : self.n_cache[l]]

    def cache_modality(self, l):
        self.finish()
        return self.mbuf[self.cur][l][: self.n_cache[l]]

    def set_cache(self, l, k, v, m_v, m_a):
        """Replace layer l's retained cache: k, v [H_kv, m_v + m_a, d] (host or
        device), visual rows first."""
        self.finish()
        m = int(m_v) + int(m_a)
        if m > self.cache_cap:
            raise ValueError(f"cache of {m} rows exceeds the capacity {self.cache_cap}")
        kb, vb, mb = self.kbuf[self.cur][l], self.vbuf[self.cur][l], self.mbuf[self.cur][l]
        kb[:, :m] = torch.as_tensor(k).to(self.device, self.tdtype)
        vb[:, :m] = torch.as_tensor(v).to(self.device, self.tdtype)
        mb[:m_v] = 0
        mb[m_v:m] = 1
        self.n_cache[l] = m

    # one step ----------------------------------------------------------
    def _describe(self, chunk, qs, cur):
        """Fill the persistent descriptor arrays for a step's working sets in
        buffer set `cur`, all but the kept-row counts (_set_cache_rows)."""
        other = cur if self.in_place else 1 - cur
        for l, ch in enumerate(chunk):
            kb, vb, mb = self.kbuf[cur][l], self.vbuf[cur][l], self.mbuf[cur][l]
            ko, vo, mo = self.kbuf[other][l], self.vbuf[other][l], self.mbuf[other][l]
            lay = self._layers[l]
            q = qs[l]
            lay.q, lay.q_head_stride, lay.q_row_stride = q.data_ptr(), q.stride(0), q.stride(1)
            lay.k, lay.v = kb.data_ptr(), vb.data_ptr()
            lay.kv_head_stride, lay.kv_row_stride = kb.stride(0), kb.stride(1)
            lay.modality = mb.data_ptr()
            lay.n_chunk = self.C
            lay.sm_scale = float(ch["sm_scale"])
            lay.k_out, lay.v_out = ko.data_ptr(), vo.data_ptr()
            lay.out_head_stride, lay.out_row_stride = ko.stride(0), ko.stride(1)
            lay.out_rows = self.cap
            lay.modality_out = mo.data_ptr()
            c = self._chunks[l]
            ck, cv, cm = ch["k"], ch["v"], ch["modality"]
            c.k, c.v, c.modality = ck.data_ptr(), cv.data_ptr(), cm.data_ptr()
            c.head_stride, c.row_stride, c.n_rows = ck.stride(0), ck.stride(1), ck.shape[1]

    def _set_cache_rows(self):
        for l in range(self.L):
            self._layers[l].n_cache = self.n_cache[l]

    def _on_device(self, chunk):
        dev, td = self.device, self.tdtype
        out = []
        for ch in chunk:
            x = dict(ch)
            for key in ("q", "k", "v"):
                t = torch.as_tensor(ch[key]).to(dev, td)
                x[key] = t if t.is_contiguous() else t.contiguous()
            x["modality"] = torch.as_tensor(ch["modality"]).to(dev, torch.uint8)
            out.append(x)
        return out

    def push(self, chunk, stream=None, wait=True):
        """Append one chunk (list of per-layer dicts from synth.StreamSource:
        q [H_q, C, d], k, v [H_kv, C, d], modality [C], sm_scale) and run the
        step.  With wait, returns the budgets [L, 2] as a host array (the
        compaction may still be running on the stream).  Without, returns
        None at once: the step's budgets are read by the next push (after it
        has described its chunk, so the host's work overlaps the GPU's) or
        by finish()."""
        stream = stream if stream is not None else torch.cuda.current_stream()
        chunk = self._on_device(chunk)
        cur = self.cur if self.in_place or not self._pending else 1 - self.cur
        self._describe(chunk, [ch["q"] for ch in chunk], cur)
        self.finish()              # the previous step's budgets give this step's kept rows
        self._chunk_refs = chunk   # keep the inputs alive while the stream uses them
        self._set_cache_rows()
        ctx, lays = self.ctx, self._layers
        ev = None
        if self.timing:
            ev = [torch.cuda.Event(enable_timing=True) for _ in range(3)]
            ev[0].record(stream)
        ctx.omnimem_append(lays, self._chunks, stream)
        if self.keep_working_set:
            with torch.cuda.stream(stream):
                self.working_set = [(self.kbuf[self.cur][l][:, : self.n_cache[l] + self.C].clone(),
                                     self.vbuf[self.cur][l][:, : self.n_cache[l] + self.C].clone(),
                                     self.mbuf[self.cur][l][: self.n_cache[l] + self.C].clone())
                                    for l in range(self.L)]
        if ev:
            ev[1].record(stream)
        ctx.omnimem_score(lays, self.a, None, stream)
        ctx.omnimem_redundancy(lays, self.s, stream)
        if self.calibrating:
            ctx.omnimem_calibrate(lays, self.a, self.s, None, stream)
        if self.fixed:
            ctx.omnimem_allocate_fixed(lays, self.a, self.s, self.layer_budgets, self.budgets, self.stats, stream)
        else:
            ctx.omnimem_allocate(lays, self.a, self.s, self.total_budget, self.budgets, self.stats, stream)
        with torch.cuda.stream(stream):
            self.budgets_host.copy_(self.budgets, non_blocking=True)
            self._budget_ready.record(stream)
        ctx.omnimem_select_compact(lays, self.a, self.s, self.budgets, self.idx, stream)
        if ev:
            ev[2].record(stream)
            self.events.append(ev)
        for l in range(self.L):
            self.tokens += self.n_cache[l] + self.C
        self._pending, self._pending_stream = True, stream
        return self.finish() if wait else None

    def finish(self):
        """Wait for the last pushed step's budgets and take its kept-row
        counts as the caches' sizes; returns the budgets [L, 2] (None when no
        step is pending)."""
        if not self._pending:
            return None
        self._pending = False
        self._budget_ready.synchronize()
        budgets = self.budgets_host.numpy().copy()
        if self.in_place and int(budgets[:, 1].max()) > self.stage_rows:
            self._check_staging(self._pending_stream)
        for l in range(self.L):
            self.n_cache[l] = int(budgets[l, 0]) + int(budgets[l, 1])
        if not self.in_place:
            self.cur = 1 - self.cur
        self.steps += 1
        return budgets

    def _check_staging(self, stream):
        """A step whose audio budget exceeds the staging reserve: if its
        in-place compaction moved nothing, compact out of place into
        temporaries and copy the kept rows back."""
        stream.synchronize()
        try:
            self.ctx.omnimem_inplace_status()
            return
        except om.OmnimemError as e:
            if e.status != om.ERR_CAPACITY:
                raise
        self.fallbacks += 1
        tmp = []
        lays = (om.Layer * self.L)()
        for l in range(self.L):
            lay = om.Layer.from_buffer_copy(self._layers[l])
            ko = torch.empty_like(self.kbuf[self.cur][l])
            vo = torch.empty_like(self.vbuf[self.cur][l])
            lay.k_out, lay.v_out = ko.data_ptr(), vo.data_ptr()
            tmp.append((ko, vo))
            lays[l] = lay
        self.ctx.omnimem_select_compact(lays, self.a, self.s, self.budgets, self.idx, stream)
        with torch.cuda.stream(stream):
            for l, (ko, vo) in enumerate(tmp):
                self.kbuf[self.cur][l].copy_(ko)
                self.vbuf[self.cur][l].copy_(vo)
        stream.synchronize()

    def timings(self):
        """Summed milliseconds over the timed steps: (appends, four stages)."""
        torch.cuda.synchronize()
        app = sum(e[0].elapsed_time(e[1]) for e in self.events)
        abi = sum(e[1].elapsed_time(e[2]) for e in self.events)
        return app, abi

    def freeze_budgets(self, stream=None):
        """Layer budgets from the steps calibrated so far; later steps split them."""
        self.finish()
        self.ctx.omnimem_calibration_budgets(self.total_budget, self.layer_budgets, stream)
        self.calibrating = False
        self.fixed = True

    def close(self):
        self.finish()
        self.ctx.close()
