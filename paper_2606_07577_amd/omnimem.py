"""Thin ctypes binding of libomnimem.so (the C ABI in include/omnimem.h).

Argument marshalling only: every stage of the compression step runs in the
library's HIP kernels.  torch tensors serve as device buffers and streams.
There is no fallback: if the library is missing or fails to load, every
call raises.
"""
from __future__ import annotations

import ctypes
import math
import os

import torch

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libomnimem.so")

OK, ERR_INVALID_ARG, ERR_UNSUPPORTED, ERR_INFEASIBLE, ERR_CAPACITY, ERR_HIP = range(6)
BF16, F32 = 0, 1
SIM_MAX, SIM_ADJ = 0, 1
SRC_VALUES, SRC_KEYS, SRC_HIDDEN = 0, 1, 2
TOPK_AUTO, TOPK_REGISTERS, TOPK_ONE_WORKGROUP, TOPK_SPLIT = 0, 1, 2, 3

EXPORTED = [
    "omnimem_config_default", "omnimem_create", "omnimem_destroy", "omnimem_last_error",
    "omnimem_score", "omnimem_redundancy", "omnimem_allocate", "omnimem_select_compact",
    "omnimem_calibrate", "omnimem_calibration_reset", "omnimem_calibration_budgets",
    "omnimem_allocate_fixed", "omnimem_profile", "omnimem_profile_report", "omnimem_inplace_status",
    "omnimem_append", "omnimem_allocate_noalloc", "omnimem_set_topk_path",
]


class OmnimemError(RuntimeError):
    def __init__(self, status, message):
        super().__init__(f"omnimem status {status}: {message}")
        self.status = status


class Config(ctypes.Structure):
    _fields_ = [
        ("n_layers", ctypes.c_int32), ("n_q_heads", ctypes.c_int32), ("n_kv_heads", ctypes.c_int32),
        ("head_dim", ctypes.c_int32), ("dtype", ctypes.c_int32), ("lambda_", ctypes.c_float),
        ("ratio_r", ctypes.c_float), ("temperature", ctypes.c_float), ("b_min_frac", ctypes.c_float),
        ("b_max_frac", ctypes.c_float), ("causal", ctypes.c_int32), ("sim", ctypes.c_int32),
        ("sim_source", ctypes.c_int32), ("shared_selection", ctypes.c_int32), ("max_tokens", ctypes.c_int64),
        ("max_chunk", ctypes.c_int64), ("hidden_dim", ctypes.c_int32), ("inplace_stage_rows", ctypes.c_int32),
    ]


class Layer(ctypes.Structure):
    _fields_ = [
        ("q", ctypes.c_void_p), ("q_head_stride", ctypes.c_int64), ("q_row_stride", ctypes.c_int64),
        ("k", ctypes.c_void_p), ("v", ctypes.c_void_p), ("kv_head_stride", ctypes.c_int64),
        ("kv_row_stride", ctypes.c_int64), ("modality", ctypes.c_void_p), ("n_cache", ctypes.c_int64),
        ("n_chunk", ctypes.c_int64), ("sm_scale", ctypes.c_float), ("lse", ctypes.c_void_p),
        ("k_out", ctypes.c_void_p), ("v_out", ctypes.c_void_p), ("out_head_stride", ctypes.c_int64),
        ("out_row_stride", ctypes.c_int64), ("hidden", ctypes.c_void_p), ("hidden_row_stride", ctypes.c_int64),
        ("hidden_out", ctypes.c_void_p), ("hidden_out_row_stride", ctypes.c_int64), ("out_rows", ctypes.c_int64),
        ("modality_out", ctypes.c_void_p),
    ]


class Chunk(ctypes.Structure):
    _fields_ = [
        ("k", ctypes.c_void_p), ("v", ctypes.c_void_p), ("head_stride", ctypes.c_int64),
        ("row_stride", ctypes.c_int64), ("modality", ctypes.c_void_p), ("n_rows", ctypes.c_int64),
    ]


class KernelTime(ctypes.Structure):
    _fields_ = [("name", ctypes.c_char * 32), ("launches", ctypes.c_int32), ("total_ms", ctypes.c_double)]


_lib = None


def load_library(path=LIB_PATH):
    """Load libomnimem.so; raises if it is not built."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(path):
        raise RuntimeError(f"{path} is missing: build it with `python -m paper_2606_07577_amd.build`")
    lib = ctypes.CDLL(path)
    vp, i32, i64 = ctypes.c_void_p, ctypes.c_int, ctypes.c_int64
    lib.omnimem_config_default.argtypes = [ctypes.POINTER(Config)]
    lib.omnimem_config_default.restype = None
    lib.omnimem_create.argtypes = [ctypes.POINTER(Config), ctypes.POINTER(vp)]
    lib.omnimem_create.restype = i32
    lib.omnimem_destroy.argtypes = [vp]
    lib.omnimem_destroy.restype = i32
    lib.omnimem_last_error.argtypes = [vp]
    lib.omnimem_last_error.restype = ctypes.c_char_p
    lib.omnimem_score.argtypes = [vp, ctypes.POINTER(Layer), vp, vp, vp]
    lib.omnimem_score.restype = i32
    lib.omnimem_redundancy.argtypes = [vp, ctypes.POINTER(Layer), vp, vp]
    lib.omnimem_redundancy.restype = i32
    lib.omnimem_allocate.argtypes = [vp, ctypes.POINTER(Layer), vp, vp, i64, vp, vp, vp]
    lib.omnimem_allocate.restype = i32
    lib.omnimem_select_compact.argtypes = [vp, ctypes.POINTER(Layer), vp, vp, vp, vp, vp]
    lib.omnimem_select_compact.restype = i32
    lib.omnimem_calibrate.argtypes = [vp, ctypes.POINTER(Layer), vp, vp, vp, vp]
    lib.omnimem_calibrate.restype = i32
    lib.omnimem_calibration_reset.argtypes = [vp]
    lib.omnimem_calibration_reset.restype = i32
    lib.omnimem_calibration_budgets.argtypes = [vp, i64, vp, vp]
    lib.omnimem_calibration_budgets.restype = i32
    lib.omnimem_allocate_fixed.argtypes = [vp, ctypes.POINTER(Layer), vp, vp, vp, vp, vp, vp]
    lib.omnimem_allocate_fixed.restype = i32
    lib.omnimem_allocate_noalloc.argtypes = [ctypes.POINTER(Config), ctypes.POINTER(Layer), vp, vp, i64, vp, vp, vp]
    lib.omnimem_allocate_noalloc.restype = i32
    lib.omnimem_inplace_status.argtypes = [vp, ctypes.POINTER(ctypes.c_int64)]
    lib.omnimem_inplace_status.restype = i32
    lib.omnimem_append.argtypes = [vp, ctypes.POINTER(Layer), ctypes.POINTER(Chunk), vp]
    lib.omnimem_append.restype = i32
    lib.omnimem_set_topk_path.argtypes = [vp, i32]
    lib.omnimem_set_topk_path.restype = i32
    lib.omnimem_profile.argtypes = [vp, ctypes.c_int32]
    lib.omnimem_profile.restype = i32
    lib.omnimem_profile_report.argtypes = [vp, ctypes.POINTER(KernelTime), ctypes.c_int32,
                                           ctypes.POINTER(ctypes.c_int32)]
    lib.omnimem_profile_report.restype = i32
    _lib = lib
    return lib


def _ptr(t):
    if t is None:
        return None
    if not isinstance(t, torch.Tensor) or not t.is_cuda:
        raise TypeError("device tensors (torch, cuda) are required")
    return t.data_ptr()


def _stream(stream):
    s = stream if stream is not None else torch.cuda.current_stream()
    return ctypes.c_void_p(s.cuda_stream)


def make_layer(q, k, v, modality, n_cache, sm_scale=0.0, lse=None, k_out=None, v_out=None, hidden=None,
               hidden_out=None, out_rows=0, modality_out=None, n=None):
    """Descriptor of one layer's working set from device tensors.

    q [H_q, C, d]; k, v [H_kv, >=N, d] (the working set is their first N
    rows, N = k.shape[1] unless given); modality uint8 [>=N]; optional lse
    [H_q, C] fp32; optional k_out, v_out [H_kv, out_rows, d] (same strides;
    k_out is k and v_out is v for compaction in place); optional hidden
    [N, d_model] and hidden_out [>=M, d_model]; optional modality_out uint8.
    """
    if k.stride() != v.stride():
        raise ValueError("k and v must share strides")
    if k_out is not None and (v_out is None or k_out.stride() != v_out.stride()):
        raise ValueError("k_out and v_out must both be given with equal strides")
    if modality.dtype != torch.uint8:
        raise TypeError("modality must be uint8")
    n = k.shape[1] if n is None else int(n)
    lay = Layer()
    lay.q = _ptr(q)
    lay.q_head_stride, lay.q_row_stride = (q.stride(0), q.stride(1)) if q is not None else (0, 0)
    lay.k, lay.v = _ptr(k), _ptr(v)
    lay.kv_head_stride, lay.kv_row_stride = k.stride(0), k.stride(1)
    lay.modality = _ptr(modality)
    lay.n_cache = int(n_cache)
    lay.n_chunk = int(n - n_cache)
    lay.sm_scale = float(sm_scale)
    lay.lse = _ptr(lse)
    if k_out is not None:
        lay.k_out, lay.v_out = _ptr(k_out), _ptr(v_out)
        lay.out_head_stride, lay.out_row_stride = k_out.stride(0), k_out.stride(1)
        lay.out_rows = int(out_rows)
    if modality_out is not None:
        if modality_out.dtype != torch.uint8:
            raise TypeError("modality_out must be uint8")
        lay.modality_out = _ptr(modality_out)
    if hidden is not None:
        lay.hidden, lay.hidden_row_stride = _ptr(hidden), hidden.stride(0)
    if hidden_out is not None:
        lay.hidden_out, lay.hidden_out_row_stride = _ptr(hidden_out), hidden_out.stride(0)
    return lay


class Context:
    """An omnimem_ctx: workspace for the given capacities on the current device."""

    def __init__(self, n_layers, n_q_heads, n_kv_heads, head_dim, max_tokens, max_chunk,
                 dtype=BF16, **options):
        lib = load_library()
        cfg = Config()
        lib.omnimem_config_default(ctypes.byref(cfg))
        cfg.n_layers, cfg.n_q_heads, cfg.n_kv_heads, cfg.head_dim = n_layers, n_q_heads, n_kv_heads, head_dim
        cfg.dtype, cfg.max_tokens, cfg.max_chunk = dtype, max_tokens, max_chunk
        for key, val in options.items():
            setattr(cfg, "lambda_" if key == "lam" else key, val)
        self.cfg = cfg
        self._lib = lib
        handle = ctypes.c_void_p()
        st = lib.omnimem_create(ctypes.byref(cfg), ctypes.byref(handle))
        if st != OK:
            raise OmnimemError(st, lib.omnimem_last_error(None).decode())
        self.handle = handle

    @staticmethod
    def default_config():
        """The library's default omnimem_config (sizes 0)."""
        cfg = Config()
        load_library().omnimem_config_default(ctypes.byref(cfg))
        return cfg

    def _check(self, st):
        if st != OK:
            raise OmnimemError(st, self._lib.omnimem_last_error(self.handle).decode())

    def _layers(self, layers):
        if len(layers) != self.cfg.n_layers:
            raise ValueError(f"expected {self.cfg.n_layers} layer descriptors")
        if isinstance(layers, ctypes.Array) and layers._type_ is Layer:
            return layers
        return (Layer * len(layers))(*layers)

    def close(self):
        if self.handle:
            self._lib.omnimem_destroy(self.handle)
            self.handle = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    # The four stages of the C ABI, same names.
    def omnimem_score(self, layers, a, lse_out=None, stream=None):
        self._check(self._lib.omnimem_score(self.handle, self._layers(layers), _ptr(a), _ptr(lse_out),
                                            _stream(stream)))

    def omnimem_redundancy(self, layers, s, stream=None):
        self._check(self._lib.omnimem_redundancy(self.handle, self._layers(layers), _ptr(s), _stream(stream)))

    def omnimem_allocate(self, layers, a, s, total_budget, budgets, stats=None, stream=None):
        self._check(self._lib.omnimem_allocate(self.handle, self._layers(layers), _ptr(a), _ptr(s),
                                               int(total_budget), _ptr(budgets), _ptr(stats), _stream(stream)))

    def omnimem_select_compact(self, layers, a, s, budgets, idx=None, stream=None):
        self._check(self._lib.omnimem_select_compact(self.handle, self._layers(layers), _ptr(a), _ptr(s),
                                                     _ptr(budgets), _ptr(idx), _stream(stream)))

    # Offline budgets (calibration), same names as the C ABI.
    def omnimem_calibrate(self, layers, a, s, stats=None, stream=None):
        self._check(self._lib.omnimem_calibrate(self.handle, self._layers(layers), _ptr(a), _ptr(s), _ptr(stats),
                                                _stream(stream)))

    def omnimem_calibration_reset(self):
        self._check(self._lib.omnimem_calibration_reset(self.handle))

    def omnimem_calibration_budgets(self, total_budget, layer_budgets, stream=None):
        self._check(self._lib.omnimem_calibration_budgets(self.handle, int(total_budget), _ptr(layer_budgets),
                                                          _stream(stream)))

    def omnimem_allocate_fixed(self, layers, a, s, layer_budgets, budgets, stats=None, stream=None):
        self._check(self._lib.omnimem_allocate_fixed(self.handle, self._layers(layers), _ptr(a), _ptr(s),
                                                     _ptr(layer_budgets), _ptr(budgets), _ptr(stats),
                                                     _stream(stream)))


    def omnimem_inplace_status(self):
        """Largest staging need of the in-place compactions since the last
        query (0: none); raises OmnimemError when one moved nothing for lack
        of staging rows or an ordering wait gave up.  Synchronous."""
        need = ctypes.c_int64()
        self._check(self._lib.omnimem_inplace_status(self.handle, ctypes.byref(need)))
        return need.value

    def omnimem_append(self, layers, chunks, stream=None):
        if len(chunks) != self.cfg.n_layers:
            raise ValueError(f"expected {self.cfg.n_layers} chunk descriptors")
        arr = chunks if isinstance(chunks, ctypes.Array) else (Chunk * len(chunks))(*chunks)
        self._check(self._lib.omnimem_append(self.handle, self._layers(layers), arr, _stream(stream)))

    def omnimem_set_topk_path(self, path):
        """Ranking path of later select_compact calls (TOPK_AUTO,
        TOPK_REGISTERS, TOPK_ONE_WORKGROUP or TOPK_SPLIT)."""
        self._check(self._lib.omnimem_set_topk_path(self.handle, int(path)))

    def omnimem_profile(self, on):
        self._check(self._lib.omnimem_profile(self.handle, int(bool(on))))

    def omnimem_profile_report(self):
        """{kernel name: (launches, total milliseconds)} of the recorded launches."""
        buf = (KernelTime * 32)()
        n = ctypes.c_int32()
        self._check(self._lib.omnimem_profile_report(self.handle, buf, 32, ctypes.byref(n)))
        return {buf[i].name.decode(): (buf[i].launches, buf[i].total_ms) for i in range(n.value)}


def allocate_noalloc(cfg, layers, a, s, total_budget, budgets, stats=None, stream=None):
    """omnimem_allocate_noalloc: the allocation stage with no context and no
    device allocation (cfg is a Config; layers a list of Layer)."""
    lib = load_library()
    arr = layers if isinstance(layers, ctypes.Array) else (Layer * len(layers))(*layers)
    st = lib.omnimem_allocate_noalloc(ctypes.byref(cfg), arr, _ptr(a), _ptr(s), int(total_budget), _ptr(budgets),
                                      _ptr(stats), _stream(stream))
    if st != OK:
        raise OmnimemError(st, lib.omnimem_last_error(None).decode())


def make_chunk(k, v, modality):
    """Descriptor of one layer's new chunk rows: k, v [H_kv, C, d] (equal
    strides), modality uint8 [C] (device tensors)."""
    if k.stride() != v.stride():
        raise ValueError("chunk k and v must share strides")
    if modality.dtype != torch.uint8:
        raise TypeError("modality must be uint8")
    ch = Chunk()
    ch.k, ch.v = _ptr(k), _ptr(v)
    ch.head_stride, ch.row_stride = k.stride(0), k.stride(1)
    ch.modality = _ptr(modality)
    ch.n_rows = k.shape[1]
    return ch


def default_scale(head_dim):
    return 1.0 / math.sqrt(head_dim)
