"""The C-ABI library loads and exports every function include/omnimem.h
declares; host-only entry points behave without a GPU."""
import ctypes
import os
import re

from paper_2606_07577_amd import omnimem

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _declared():
    text = open(os.path.join(ROOT, "include", "omnimem.h")).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(omnimem_[a-z_]+)\s*\(", text)))


def test_header_declares_the_four_stages_and_lifecycle():
    names = _declared()
    for want in ("omnimem_score", "omnimem_redundancy", "omnimem_allocate", "omnimem_select_compact",
                 "omnimem_create", "omnimem_destroy", "omnimem_last_error", "omnimem_config_default"):
        assert want in names
    assert sorted(omnimem.EXPORTED) == names


def test_library_exports_every_declared_symbol():
    lib = ctypes.CDLL(omnimem.LIB_PATH)
    for name in _declared():
        assert hasattr(lib, name), name


def test_config_defaults_are_the_papers():
    lib = omnimem.load_library()
    cfg = omnimem.Config()
    lib.omnimem_config_default(ctypes.byref(cfg))
    assert abs(cfg.lambda_ - 0.02) < 1e-7 and cfg.ratio_r == 5.0 and abs(cfg.temperature - 0.2) < 1e-7
    assert cfg.causal == 1 and cfg.sim == omnimem.SIM_MAX and cfg.dtype == omnimem.BF16


def test_create_rejects_bad_config_before_touching_the_device():
    lib = omnimem.load_library()
    cfg = omnimem.Config()
    lib.omnimem_config_default(ctypes.byref(cfg))
    cfg.n_layers, cfg.n_q_heads, cfg.n_kv_heads, cfg.head_dim = 1, 8, 3, 128
    cfg.max_tokens, cfg.max_chunk = 100, 10
    h = ctypes.c_void_p()
    assert lib.omnimem_create(ctypes.byref(cfg), ctypes.byref(h)) == omnimem.ERR_INVALID_ARG
    assert b"H_kv" in lib.omnimem_last_error(None)
    cfg.n_kv_heads, cfg.head_dim = 2, 96
    assert lib.omnimem_create(ctypes.byref(cfg), ctypes.byref(h)) == omnimem.ERR_UNSUPPORTED
    assert lib.omnimem_score(None, None, None, None, None) == omnimem.ERR_INVALID_ARG
