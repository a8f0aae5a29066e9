"""Host-side checks of the C ABI that need no GPU: the library loads and
exports every entry point include/sd.h declares, and its pure host
functions behave as documented."""

import ctypes
import os
import re

import pytest

from paper_2309_08168_amd import binding

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _declared():
    src = open(os.path.join(ROOT, "include", "sd.h")).read()
    return sorted(set(re.findall(r"^\s*(?:sd_status|size_t|int32_t|const char \*)\s*\*?\s*(sd_\w+)\s*\(", src,
                                 flags=re.M)))


def test_every_declared_symbol_is_exported():
    lib = binding.load()
    declared = _declared()
    assert declared == sorted(binding.EXPORTS)
    for name in declared:
        assert hasattr(lib, name), name


def test_version_and_empty_error():
    lib = binding.load()
    assert b"gfx950" in lib.sd_version()
    assert lib.sd_last_error() is not None


def test_kv_cache_bytes_layout():
    import sd_synth as S

    lib = binding.load()
    for name in ("tiny", "7b", "13b", "70b"):
        cfg = S.MODELS[name]
        c = binding.make_config(cfg)
        es = 2 if cfg.dtype == "bf16" else 4
        assert lib.sd_kv_cache_bytes(ctypes.byref(c), 100) == cfg.n_layers * 2 * cfg.n_kv_heads * 100 * cfg.head_dim * es
    bad = binding.make_config(S.MODELS["tiny"])
    bad.head_dim = 12
    assert lib.sd_kv_cache_bytes(ctypes.byref(bad), 10) == 0


def test_null_arguments_are_rejected_without_a_gpu():
    lib = binding.load()
    out = ctypes.c_void_p()
    assert lib.sd_model_create(None, None, None, ctypes.byref(out)) == binding.SD_ERR_INVALID_ARG
    assert b"config" in lib.sd_last_error()
    assert lib.sd_model_destroy(None) == binding.SD_ERR_INVALID_ARG
    assert lib.sd_kv_cache_length(None) == -1
    assert lib.sd_kv_cache_truncate(None, 0) == binding.SD_ERR_INVALID_ARG
    assert lib.sd_forward(None, None, 1, None, None, None) == binding.SD_ERR_INVALID_ARG
    assert lib.sd_self_spec_generate(None, None, 1, 1, None, 1, ctypes.c_float(0.5), None, None) == \
        binding.SD_ERR_INVALID_ARG
    assert lib.sd_autoregressive_generate(None, None, 1, 1, None, None) == binding.SD_ERR_INVALID_ARG


@pytest.mark.parametrize("field,value", [("head_dim", 7), ("n_kv_heads", 3), ("vocab", 1), ("d_model", 12),
                                         ("head_dim", 256), ("dtype", 5)])
def test_bad_shapes_are_rejected(field, value):
    import sd_synth as S

    lib = binding.load()
    c = binding.make_config(S.MODELS["tiny"])
    setattr(c, field, value)
    w = binding.sd_weights()
    out = ctypes.c_void_p()
    assert lib.sd_model_create(ctypes.byref(c), ctypes.byref(w), None, ctypes.byref(out)) == \
        binding.SD_ERR_INVALID_ARG
    assert not out.value
