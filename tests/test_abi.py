"""The C ABI library builds, loads without a GPU and exports every symbol
include/as2d.h declares; the binding covers exactly those symbols."""
import ctypes
import os
import re

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def header_symbols():
    src = open(os.path.join(ROOT, "include", "as2d.h")).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"\b(as2d_[a-z_0-9]+)\s*\(", src)))


@pytest.fixture(scope="module")
def lib():
    from tests.harness import ensure_built
    ensure_built()
    from paper_2609_37617_amd import as2d
    return as2d.load_library()


def test_header_declares_the_boundary_calls():
    syms = header_symbols()
    for name in ("as2d_load_weights", "as2d_prefill_kv", "as2d_verify", "as2d_decode_one",
                 "as2d_verify_batch", "as2d_free", "as2d_last_error"):
        assert name in syms


def test_library_exports_every_declared_symbol(lib):
    for name in header_symbols():
        assert hasattr(lib, name), name


def test_binding_matches_header():
    from paper_2609_37617_amd import as2d
    assert sorted(as2d.EXPORTS) == header_symbols()


def test_null_arguments_rejected_without_gpu(lib):
    from paper_2609_37617_amd import as2d
    out = ctypes.c_void_p()
    assert lib.as2d_load_weights(None, None, 0, None, ctypes.byref(out)) == as2d.EINVAL
    assert lib.as2d_verify(None, 0, None, 0, None) == as2d.EINVAL
    assert lib.as2d_decode_one(None, 0, None) == as2d.EINVAL
    assert lib.as2d_rollback(None, 0, 0, 0) == as2d.EINVAL
    assert lib.as2d_step_bytes(None, 1, 1) == -1
    assert lib.as2d_last_error(None) == b"null context"
    lib.as2d_free(None)


def test_config_validation_without_gpu(lib):
    """Shape checks run before any device call."""
    from paper_2609_37617_amd import as2d
    from workload import TINY
    cfg = as2d.Config(TINY.n_layers, 100, TINY.n_q_heads, TINY.n_kv_heads, TINY.head_dim, TINY.ffn,
                      TINY.vocab, 1e4, 1e-6, 0, 0, 1, 64, 4)   # hidden 100: not a multiple of 128
    ptrs = (ctypes.c_void_p * 21)(*([1] * 21))
    out = ctypes.c_void_p()
    assert lib.as2d_load_weights(ctypes.byref(cfg), ptrs, 21, None, ctypes.byref(out)) == as2d.EINVAL
    cfg.hidden, cfg.head_dim = 256, 96
    assert lib.as2d_load_weights(ctypes.byref(cfg), ptrs, 21, None, ctypes.byref(out)) == as2d.EINVAL
    cfg.head_dim, cfg.max_k = 64, 40
    assert lib.as2d_load_weights(ctypes.byref(cfg), ptrs, 21, None, ctypes.byref(out)) == as2d.EINVAL
    cfg.max_k = 4
    assert lib.as2d_load_weights(ctypes.byref(cfg), ptrs, 7, None, ctypes.byref(out)) == as2d.EINVAL
