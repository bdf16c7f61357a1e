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
