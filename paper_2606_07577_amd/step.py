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
        self.sm_scale = [float(l["sm_scale"]) for l in layers]
        shape = (self.n_layers, h_kv, self.max_tokens)
        self.a = torch.zeros(shape, device=dev, dtype=torch.float32)
        self.s = torch.zeros(shape, device=dev, dtype=torch.float32)
        self.idx = torch.full(shape, -1, device=dev, dtype=torch.int32)
        self.lse = torch.zeros((self.n_layers, h_q, self.max_chunk), device=dev, dtype=torch.float32)
        self.budgets = torch.zeros((self.n_layers, 2), device=dev, dtype=torch.int32)
        self.stats = torch.zeros((self.n_layers, 10), device=dev, dtype=torch.float32)
        self.lse_in = [None] * self.n_layers
        self.descs = self._descs()

    def _descs(self):
        return [om.make_layer(self.q[l], self.k[l], self.v[l], self.mod[l], self.n_cache[l],
                              self.sm_scale[l], self.lse_in[l], self.k_out[l], self.v_out[l])
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

    def run(self, stream=None):
        self.score(stream, lse_out=False)
        self.redundancy(stream)
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
