"""The C-ABI library builds for gfx950, loads, and exports every function
include/darts.h declares (no compute call: this runs without a GPU)."""
import ctypes
import os
import re

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "darts.h")


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(darts_[a-z0-9_]+)\s*\(", text)))


@pytest.fixture(scope="module")
def lib_path():
    from paper_2605_30859_amd import binding
    if not os.path.exists(binding.lib_path):
        from paper_2605_30859_amd.build import build
        build()
    return binding.lib_path


def test_header_declares_the_boundary():
    names = declared_functions()
    for required in ("darts_init", "darts_prefill", "darts_decode_step", "darts_select_and_prune",
                     "darts_attn_decode", "darts_sample", "darts_select_groups"):
        assert required in names


def test_library_exports_every_declared_symbol(lib_path):
    lib = ctypes.CDLL(lib_path)
    missing = [n for n in declared_functions() if not hasattr(lib, n)]
    assert not missing, missing


def test_binding_signatures_cover_header(lib_path):
    from paper_2605_30859_amd import binding
    binding.load_library()
    assert set(declared_functions()) == set(binding._SIGS)


def test_strerror_without_gpu(lib_path):
    from paper_2605_30859_amd import binding
    lib = binding.load_library()
    assert lib.darts_strerror(0) == b"ok"
    assert b"invalid" in lib.darts_strerror(1)


def test_invalid_config_rejected_before_any_device_call(lib_path):
    """k > m is rejected by host validation, before touching the device."""
    from paper_2605_30859_amd import binding
    from workload import get_config
    lib = binding.load_library()
    model, run = get_config("tiny")
    mc = binding.model_cfg_struct(model)
    rc = binding.run_cfg_struct(run, None)
    ctx = ctypes.c_void_p()
    assert lib.darts_init(ctypes.byref(mc), 4, 8, ctypes.byref(rc), ctypes.byref(ctx)) == binding.DARTS_EINVAL
    rc.prompt_len = 17
    assert lib.darts_init(ctypes.byref(mc), 8, 4, ctypes.byref(rc), ctypes.byref(ctx)) == binding.DARTS_EINVAL
    assert not ctx.value


def test_caller_weights_count_and_null_entry_rejected(lib_path):
    """darts_weight_count: 2 + n_layers * (7 dense, 8 MoE); a caller weight
    array with a null entry is rejected by host validation, before any device
    call, and *out stays untouched."""
    from paper_2605_30859_amd import binding
    from workload import get_config
    lib = binding.load_library()
    for name, per_layer in (("tiny", 7), ("dense-small", 7), ("qwen3-30b-a3b", 8)):
        model, _ = get_config(name)
        assert binding.darts_weight_count(model) == 2 + model.n_layers * per_layer
    assert lib.darts_weight_count(None) == 0
    model, run = get_config("tiny")
    n = binding.darts_weight_count(model)
    arr = (ctypes.c_void_p * n)()
    for i in range(n):
        arr[i] = 0x1000 * (i + 1)        # never dereferenced: entry 3 is null
    arr[3] = None
    mc = binding.model_cfg_struct(model, arr)
    rc = binding.run_cfg_struct(run, None)
    ctx = ctypes.c_void_p()
    assert lib.darts_init(ctypes.byref(mc), run.m, run.k, ctypes.byref(rc), ctypes.byref(ctx)) == binding.DARTS_EINVAL
    assert not ctx.value
