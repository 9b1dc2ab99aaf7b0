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

    Each layer's cache lives in two ping-pong buffers [H_kv, cap, d]: the
    working set of a step is the current buffer's first N = n_cache + C rows
    (retained visual, retained audio, then the new chunk, Eq. 3), and
    omnimem_select_compact writes the kept rows to the front of the other
    buffer, which then receives the next chunk behind them.  Appending the
    chunk stands in for the model's prefill writing its K/V; it is a device
    copy outside the library.  After each step the budgets are read back (a
    stream synchronisation): the host needs them to describe the next
    working set.
    """

    def __init__(self, n_layers, h_q, h_kv, d, chunk_len, total_budget, dtype="bf16", device="cuda",
                 **options):
        self.device = torch.device(device)
        self.L, self.h_q, self.h_kv, self.d, self.C = n_layers, h_q, h_kv, d, chunk_len
        self.total_budget = int(total_budget)
        self.tdtype = torch.bfloat16 if dtype == "bf16" else torch.float32
        cfg_probe = om.Context.default_config()
        bmax = options.get("b_max_frac", cfg_probe.b_max_frac)
        self.cache_cap = int(bmax * total_budget / n_layers)   # no layer keeps more
        self.cap = self.cache_cap + chunk_len
        self.ctx = om.Context(n_layers, h_q, h_kv, d, self.cap, chunk_len,
                              dtype=om.BF16 if dtype == "bf16" else om.F32, **options)
        dev, td = self.device, self.tdtype
        self.kbuf = [[torch.zeros((h_kv, self.cap, d), device=dev, dtype=td) for _ in range(n_layers)]
                     for _ in range(2)]
        self.vbuf = [[torch.zeros((h_kv, self.cap, d), device=dev, dtype=td) for _ in range(n_layers)]
                     for _ in range(2)]
        self.mbuf = [[torch.zeros(self.cap, device=dev, dtype=torch.uint8) for _ in range(n_layers)]
                     for _ in range(2)]
        shape = (n_layers, h_kv, self.cap)
        self.a = torch.zeros(shape, device=dev, dtype=torch.float32)
        self.s = torch.zeros(shape, device=dev, dtype=torch.float32)
        self.idx = torch.full(shape, -1, device=dev, dtype=torch.int32)
        self.budgets = torch.zeros((n_layers, 2), device=dev, dtype=torch.int32)
        self.stats = torch.zeros((n_layers, 10), device=dev, dtype=torch.float32)
        self.layer_budgets = torch.zeros(n_layers, device=dev, dtype=torch.int32)
        self.calibrating = False   # each step also adds its C^(l) to the calibration
        self.fixed = False         # steps split self.layer_budgets instead of Eq. (14)
        self.cur = 0
        self.n_cache = [0] * n_layers
        self.steps = 0
        self.tokens = 0          # sum over steps and layers of the working-set size

    def set_cache(self, l, k, v, m_v, m_a):
        """Replace layer l's retained cache: k, v [H_kv, m_v + m_a, d] (host or
        device), visual rows first."""
        m = int(m_v) + int(m_a)
        if m > self.cache_cap:
            raise ValueError(f"cache of {m} rows exceeds the capacity {self.cache_cap}")
        kb, vb, mb = self.kbuf[self.cur][l], self.vbuf[self.cur][l], self.mbuf[self.cur][l]
        kb[:, :m] = torch.as_tensor(k).to(self.device, self.tdtype)
        vb[:, :m] = torch.as_tensor(v).to(self.device, self.tdtype)
        mb[:m_v] = 0
        mb[m_v:m] = 1
        self.n_cache[l] = m

    def working_set(self, l):
        """Device views of layer l's current working set (k, v, modality)."""
        n = self.n_cache[l] + self.C
        return (self.kbuf[self.cur][l][:, :n], self.vbuf[self.cur][l][:, :n], self.mbuf[self.cur][l][:n])

    def push(self, chunk, stream=None):
        """Append one chunk (list of per-layer dicts from synth.StreamSource)
        and run the step.  Returns the budgets [L, 2] as a host array."""
        dev, td = self.device, self.tdtype
        descs, qs = [], []
        other = 1 - self.cur
        for l, ch in enumerate(chunk):
            n0 = self.n_cache[l]
            n = n0 + self.C
            kb, vb, mb = self.kbuf[self.cur][l], self.vbuf[self.cur][l], self.mbuf[self.cur][l]
            kb[:, n0:n] = torch.as_tensor(ch["k"]).to(dev, td)
            vb[:, n0:n] = torch.as_tensor(ch["v"]).to(dev, td)
            mb[n0:n] = torch.as_tensor(ch["modality"]).to(dev)
            q = torch.as_tensor(ch["q"]).to(dev, td).contiguous()
            qs.append(q)
            descs.append(om.make_layer(q, kb[:, :n], vb[:, :n], mb[:n], n0, ch["sm_scale"], None,
                                       self.kbuf[other][l], self.vbuf[other][l]))
            self.tokens += n
        self._descs, self._qs = descs, qs
        self.ctx.omnimem_score(descs, self.a, None, stream)
        self.ctx.omnimem_redundancy(descs, self.s, stream)
        if self.calibrating:
            self.ctx.omnimem_calibrate(descs, self.a, self.s, None, stream)
        if self.fixed:
            self.ctx.omnimem_allocate_fixed(descs, self.a, self.s, self.layer_budgets, self.budgets, self.stats,
                                            stream)
        else:
            self.ctx.omnimem_allocate(descs, self.a, self.s, self.total_budget, self.budgets, self.stats, stream)
        self.ctx.omnimem_select_compact(descs, self.a, self.s, self.budgets, self.idx, stream)
        budgets = self.budgets.cpu().numpy()
        for l in range(self.L):
            m_v, m_a = int(budgets[l, 0]), int(budgets[l, 1])
            mb = self.mbuf[other][l]
            mb[:m_v] = 0
            mb[m_v:m_v + m_a] = 1
            self.n_cache[l] = m_v + m_a
        self.cur = other
        self.steps += 1
        return budgets

    def freeze_budgets(self, stream=None):
        """Layer budgets from the steps calibrated so far; later steps split them."""
        self.ctx.omnimem_calibration_budgets(self.total_budget, self.layer_budgets, stream)
        self.calibrating = False
        self.fixed = True

    def close(self):
        self.ctx.close()
